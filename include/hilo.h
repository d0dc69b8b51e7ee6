/*
 * hilo.h -- C ABI of libhilo.so, the MI355X (gfx950) hot path of HiLo-Token: one diffusion-
 * transformer block run on an input-adaptively compressed token set.
 *
 * The six calls follow the method's own order (HiLo-Token, Sec. 2.3 "HiLo-Token Selection"):
 *   hilo_score      Sobel frequency energy of every latent patch
 *   hilo_select     2x2 regional pooling of the energy, threshold or top-k, dilated user mask kept
 *                   fine, and the index map of the compressed grid
 *   hilo_compress   fine patches copied, every other 2x2 block pooled into one low-frequency token,
 *                   text tokens appended (concatenation along the token dimension)
 *   hilo_attention  pre-LN adaLN joint attention over image + text tokens of each sample
 *   hilo_mlp        pre-LN adaLN GELU MLP
 *   hilo_decompress scatter fine tokens and broadcast pooled tokens back to the full grid
 * hilo_compress_norm + hilo_attention_normed are hilo_compress + hilo_attention with the attention
 * half's first row norm done in the compress pass, on the rows it just formed.
 *
 * Conventions shared by every call
 *   - Every tensor pointer is a caller-owned DEVICE pointer unless stated otherwise; tensors are
 *     dense, row-major, with the last index contiguous.  The library never allocates device memory
 *     and never synchronises; each call validates its arguments on the host, returns an error and
 *     enqueues nothing when they are wrong, and otherwise enqueues its kernels on `stream` (a
 *     hipStream_t passed as void*; NULL = the default stream) and returns HILO_OK.
 *   - A launch failure returns HILO_E_DEVICE.  A fault inside a kernel surfaces at the caller's
 *     next synchronisation.  No C++ exception crosses this boundary.
 *   - Token counts never travel back to the host: hilo_select leaves them in device memory and
 *     the later calls read them there, sizing their grids for the worst case (no compression).
 *   - Shapes: G = batch * images grids of N = grid_h * grid_w patches (raster order p = i*grid_w+j),
 *     NB = N / 4 coarse 2x2 blocks (b = (i/2)*(grid_w/2) + j/2), D = dim, L = text_len.
 *     T_max = batch * (images * (N + NB) + L) bounds the packed sequence of every token set
 *     (hilo_max_tokens; the PARTITION set of hilo_select never exceeds batch * (images * N + L)).
 *   - The packed sequence of sample s occupies rows [cu_seqlens[s], cu_seqlens[s+1]) of z:
 *     [grid 0: fine patches in raster order, then pooled blocks in block order ; grid 1 ... ;
 *      L text tokens].  seg_off[g] is the first row of grid g.
 *   - The residual stream z is float32 in every dtype; x_img, x_txt, weights and y are `dtype`.
 *   - Calls that touch disjoint buffers may run concurrently on different streams.
 */
#ifndef HILO_H
#define HILO_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define HILO_ABI_VERSION 6

typedef enum {
  HILO_OK = 0,
  HILO_E_NULL = 1,      /* a required pointer is NULL                                        */
  HILO_E_SHAPE = 2,     /* grid not even/positive, dim != heads*head_dim, size limits (below) */
  HILO_E_DTYPE = 3,     /* dtype unknown, or head_dim unsupported for the dtype               */
  HILO_E_PARAM = 4,     /* selection mode or token set unknown, tau not finite, keep out of   */
                        /* [0, NB], dilate_r negative, n_blocks negative                      */
  HILO_E_WORKSPACE = 5, /* workspace smaller than hilo_workspace_bytes()                      */
  HILO_E_DEVICE = 6     /* a HIP launch failed, or no GPU                                     */
} hilo_status;

typedef enum { HILO_F32 = 0, HILO_BF16 = 1 } hilo_dtype;

typedef enum { HILO_SELECT_THRESHOLD = 0, HILO_SELECT_TOPK = 1 } hilo_select_mode;

/* What a grid's compressed tokens are, besides the 4 fine patches of every kept block:
 *   PARTITION  one pooled (low-frequency) token per block that is not kept: every patch is
 *              represented exactly once (n_img = NB + 3 K)
 *   OVERLAP    one pooled token per block, kept blocks included (Sec. 2.3: all low-frequency
 *              tokens are retained and concatenated with the selected high-frequency tokens;
 *              n_img = NB + 4 K)
 *   DROP       nothing else (Sec. 3.2: for text-prompted generative fill the tokens outside the
 *              dilated mask can be pruned entirely; n_img = 4 K) -- patches of other blocks have
 *              no token (idx_map -1)                                                            */
typedef enum { HILO_TOKENS_PARTITION = 0, HILO_TOKENS_OVERLAP = 1, HILO_TOKENS_DROP = 2 } hilo_token_set;

/* Problem shape.  Limits (HILO_E_SHAPE otherwise): grid_h, grid_w even and > 0; N/4 <= 16384;
 * dim == heads * head_dim, dim % 64 == 0, dim <= 8192 (keeps energies exact in int64 and block
 * sums exact in double); mlp_dim % 64 == 0; text_len >= 0; T_max < 2^31.
 * head_dim must be 64 or 128 (HILO_E_DTYPE otherwise).                                         */
typedef struct {
  int32_t batch, images, grid_h, grid_w, text_len, dim, heads, head_dim, mlp_dim;
  int32_t dtype; /* hilo_dtype */
} hilo_shape;

/* Per-stream weights in nn.Linear layout [out][in], element type `dtype`.  Arrays of two:
 * index 0 = image tokens, index 1 = text tokens (the same pointers may be given for both).      */
typedef struct {
  const void *w_qkv; /* [3D][D]  rows 0..D-1 -> q, D..2D-1 -> k, 2D..3D-1 -> v; head h = cols h*hd */
  const void *b_qkv; /* [3D]                                                                     */
  const void *w_o;   /* [D][D]                                                                   */
  const void *b_o;   /* [D]                                                                      */
} hilo_attn_w;

typedef struct {
  const void *w1; /* [F][D]  F = mlp_dim */
  const void *b1; /* [F]                 */
  const void *w2; /* [D][F]              */
  const void *b2; /* [D]                 */
} hilo_mlp_w;

/* S1 -- frequency energy (Sec. 2.3: spatial-frequency map from two Sobel operators).
 * For every grid g, patch (i,j) and channel c, with x read as float32 and neighbours clamped to
 * the grid (replicated border):
 *   gx = ((x[i-1][j+1] + 2x[i][j+1]) + x[i+1][j+1]) - ((x[i-1][j-1] + 2x[i][j-1]) + x[i+1][j-1])
 *   gy = ((x[i+1][j-1] + 2x[i+1][j]) + x[i+1][j+1]) - ((x[i-1][j-1] + 2x[i-1][j]) + x[i-1][j+1])
 *   q  = floor(min(gx*gx + gy*gy, 2^22) * 2^16)   (float32, every operation rounded, no fusion;
 *                                                  a NaN energy counts as 2^22)
 * (for bf16 latents the device forms a + 2b as one fused multiply-add: 2b is exact, so the result
 * is the same for every input below 2^127 in magnitude)
 *   energy[g][p] = sum over c of q, exact in int64.
 * x_img [G][N][D] dtype  ->  energy [G][N] int64.                                               */
hilo_status hilo_score(const hilo_shape *shape, const void *x_img, int64_t *energy, void *stream);

/* S1 in pixel space (the paper's own selector input, Sec. 2.3: Sobel on the image, 16x pooling
 * onto the token grid).  rgb: DEVICE float32 [G][3][16 grid_h][16 grid_w] (planar channels, any
 * value range).  For every pixel and channel the energy and fixed point of hilo_score (same
 * formulas, neighbours clamped to the image), summed exactly over the token's 16 x 16 pixels and 3
 * channels: energy [G][N] int64, ready for hilo_select.  The paper cuts its normalised Sobel
 * magnitude at 0.1; the energy is the magnitude squared, so its counterpart here is THRESHOLD
 * with tau = 0.01.  HILO_E_SHAPE if the image has 2^31 or more values.                          */
hilo_status hilo_score_pixels(const hilo_shape *shape, const float *rgb, int64_t *energy, void *stream);

/* S2 -- selection (Sec. 2.3: 16x regional pooling of the frequency map onto the token grid,
 * threshold on the normalised map, dilated user mask combined with the selection).
 *   B_b  = sum of the 4 energies of block b (exact);  E_max = max_p energy[g][p]
 *   F    = blocks holding a patch within Chebyshev distance dilate_r of a force pixel
 *   THRESHOLD: fine_b = (b in F) or (E_max > 0 and (double)B_b > (4.0 * tau[g]) * (double)E_max)
 *              i.e. the block's mean normalised energy strictly exceeds tau[g]
 *   TOPK:      F plus the max(0, keep[g] - |F|) other blocks of largest B_b (ties: lower b first)
 * Outputs (device): idx_map [G][N] int32 (row of patch p within its grid's compressed tokens),
 * fine_idx [G][N] int32 (patch of fine row k, k < n_fine; rest unspecified), pool_idx [G][NB]
 * int32 (block of pooled row k, k < n_pool; rest unspecified), counts [G][2] int32
 * {n_fine = 4 |fine|, n_pool = NB - |fine|}, cu_seqlens [batch+1] int32, seg_off [G] int32.
 * force: [G][N] uint8 device pointer (nonzero = inside the user mask) or NULL (no mask).
 * tau, keep: HOST arrays [G]; only the one the mode uses is read (the other may be NULL).      */
hilo_status hilo_select(const hilo_shape *shape, const int64_t *energy, const uint8_t *force,
                        int32_t dilate_r, int32_t mode, const double *tau, const int32_t *keep,
                        int32_t *idx_map, int32_t *fine_idx, int32_t *pool_idx, int32_t *counts,
                        int32_t *cu_seqlens, int32_t *seg_off, void *stream);

/* S2 with a token set (hilo_token_set; hilo_select is PARTITION).  The kept blocks are chosen as
 * above.  OVERLAP: pool_idx[g][k] = k for all NB blocks, counts {4 |fine|, NB}, and idx_map of a
 * patch in a kept block is its fine row, otherwise n_fine + its block.  DROP: counts
 * {4 |fine|, 0}, idx_map -1 for patches outside kept blocks.  token_set unknown -> HILO_E_PARAM. */
hilo_status hilo_select_tokens(const hilo_shape *shape, const int64_t *energy, const uint8_t *force,
                               int32_t dilate_r, int32_t mode, const double *tau,
                               const int32_t *keep, int32_t token_set, int32_t *idx_map,
                               int32_t *fine_idx, int32_t *pool_idx, int32_t *counts,
                               int32_t *cu_seqlens, int32_t *seg_off, void *stream);

/* S3 -- compress (Sec. 2.3: selected high-frequency tokens concatenated with low-frequency tokens
 * along the token dimension).  Row seg_off[g] + k of z is x_img[g][fine_idx[g][k]] for k < n_fine
 * and ((x00 + x01) + (x10 + x11)) * 0.25 over the 4 patches of block pool_idx[g][k - n_fine]
 * (float32) for n_fine <= k < n_fine + n_pool; the L text rows of sample s (x_txt [B][L][D]
 * dtype) follow its image rows.  z [T_max][D] float32; rows past cu_seqlens[batch] untouched.  */
hilo_status hilo_compress(const hilo_shape *shape, const void *x_img, const void *x_txt,
                          const int32_t *fine_idx, const int32_t *pool_idx, const int32_t *counts,
                          const int32_t *cu_seqlens, const int32_t *seg_off, float *z, void *stream);

/* S4 -- attention half of the block, in place on z (Sec. 2.3: the concatenated HiLo tokens are
 * what the DiT processes; Sec. 2.2 and Sec. 4: attention over all tokens is the quadratic cost the
 * compression removes).  MMDiT-style joint attention over the image and text tokens of each
 * sample; image rows use w[0] / mod stream 0, text rows w[1] / stream 1:
 *   h = LN(z) * (1 + scale1) + shift1;  qkv = h W_qkv^T + b_qkv
 *   a = softmax(q k^T / sqrt(head_dim)) v per head over all rows of the sample (no mask)
 *   z = z + gate1 * (a W_o^T + b_o)
 * LN: biased variance over D, eps 1e-6, no affine.  mod [batch][2][6][D] float32 holds
 * shift1, scale1, gate1, shift2, scale2, gate2 per sample and stream.  bf16 products accumulate in
 * float32; h, qkv and a are rounded to `dtype` in the workspace.  workspace: device scratch of
 * ws_bytes >= hilo_workspace_bytes(shape), owned by the caller, contents undefined after.
 * The block needs only the sample boundaries (cu_seqlens) and the image/text split (the last
 * text_len rows of each sample): the per-grid counts and offsets of hilo_select do not change it,
 * since attention is equivariant to the order of a sample's rows and the weights depend only on
 * the stream.                                                                                   */
hilo_status hilo_attention(const hilo_shape *shape, float *z, const int32_t *cu_seqlens,
                           const hilo_attn_w w[2], const float *mod, void *workspace,
                           size_t ws_bytes, void *stream);

/* S3 and the first step of S4 in one pass (Sec. 2.3: the compressed tokens are what the DiT's
 * block normalises first): z exactly as hilo_compress, and the attention half's normalised,
 * modulated rows h = LN(z) * (1 + scale1) + shift1 (as hilo_attention forms them, bit for bit)
 * written into the first bytes of `workspace`, where hilo_attention_normed reads them; z is not
 * read back.  shape must also be a valid block shape (HILO_E_SHAPE / HILO_E_DTYPE as
 * hilo_attention); mod as hilo_attention; workspace: ws_bytes >= hilo_workspace_bytes(shape),
 * the same workspace then passed to hilo_attention_normed with nothing enqueued on it in between.
 * Errors as hilo_compress, plus HILO_E_NULL for mod or workspace and HILO_E_WORKSPACE.          */
hilo_status hilo_compress_norm(const hilo_shape *shape, const void *x_img, const void *x_txt,
                               const int32_t *fine_idx, const int32_t *pool_idx, const int32_t *counts,
                               const int32_t *cu_seqlens, const int32_t *seg_off, const float *mod,
                               float *z, void *workspace, size_t ws_bytes, void *stream);

/* S4 without its first step: hilo_attention on the normalised rows hilo_compress_norm left in the
 * workspace (the same z, cu_seqlens, mod and workspace; same results as hilo_compress followed by
 * hilo_attention).  Arguments and errors as hilo_attention.                                      */
hilo_status hilo_attention_normed(const hilo_shape *shape, float *z, const int32_t *cu_seqlens,
                                  const hilo_attn_w w[2], const float *mod, void *workspace,
                                  size_t ws_bytes, void *stream);

/* S5 -- MLP half of the block, in place on z (Sec. 2.3: the DiT runs on the HiLo tokens; Sec. 2.2:
 * the DiT is most of the model's latency):
 *   h2 = LN(z) * (1 + scale2) + shift2;  z = z + gate2 * (GELU_tanh(h2 W1^T + b1) W2^T + b2)
 * GELU_tanh(u) = 0.5 u (1 + tanh(sqrt(2/pi) (u + 0.044715 u^3))).  Arguments as hilo_attention. */
hilo_status hilo_mlp(const hilo_shape *shape, float *z, const int32_t *cu_seqlens,
                     const hilo_mlp_w w[2], const float *mod, void *workspace, size_t ws_bytes,
                     void *stream);

/* S4 + S5 for a stack of n_blocks blocks, in order, in place on z: block l runs hilo_attention
 * then hilo_mlp with attn_w[2l .. 2l+1], mlp_w[2l .. 2l+1] (image / text stream) and its
 * modulation mod + l * batch * 2 * 6 * dim.  This is the regime of the paper's speedups (Sec. 3.3):
 * the selection, compression and decompression run once per sampling step, the network's blocks
 * all run on the compressed sequence in between.  attn_w, mlp_w: HOST arrays [n_blocks][2] of
 * device weight pointers; mod: DEVICE float32 [n_blocks][batch][2][6][dim].  Every pointer is
 * checked before anything is enqueued.  n_blocks = 0 enqueues nothing; n_blocks < 0 ->
 * HILO_E_PARAM.  workspace as hilo_attention (ws_bytes >= hilo_workspace_bytes(shape)).        */
hilo_status hilo_blocks(const hilo_shape *shape, float *z, const int32_t *cu_seqlens,
                        const hilo_attn_w *attn_w, const hilo_mlp_w *mlp_w, const float *mod,
                        int32_t n_blocks, void *workspace, size_t ws_bytes, void *stream);

/* FP8 projections (Sec. 3.3: the token compression composes with FP8 quantisation of the network).
 * Format: OCP FP8 E4M3 (sign, 4 exponent bits with bias 7, 3 mantissa bits, subnormals, largest
 * finite 448, codes 0x7f / 0xff NaN, no infinity), one float32 scale per row.  A row x of C values
 * is quantised as (every step one float32 operation)
 *   amax = max |x|;  inv = 448 / amax (correctly rounded; 0 when amax == 0)
 *   code = round-to-nearest-even E4M3 of clamp(x * inv, -448, 448);  scale = amax / 448
 * so that value(code) * scale approximates x.  The FP8 block runs all four projections (QKV,
 * attention output, MLP up, MLP down) on such rows -- activations per token, weights per output
 * channel -- with exact products and float32 accumulation: acc = sum_k value(xcode[m][k])
 * value(wcode[n][k]), then out = acc * (xscale[m] * wscale[n]) + bias.  The normalised rows h and
 * h2 are quantised where they are formed (float32, no bf16 rounding first); the attention output
 * and the GELU output, which other kernels produce in bf16, by a pass over their rows.  Everything
 * else is as in the bf16 block.                                                                  */

/* Weights of the FP8 block: the four projection weights as E4M3 codes with one float32 scale per
 * output channel (per row of the [out][in] matrix, hilo_quantize_rows), biases bf16.  Arrays of
 * two per block: image stream, text stream.                                                      */
typedef struct {
  const uint8_t *w_qkv; /* [3D][D] E4M3 codes */
  const float *s_qkv;   /* [3D] row scales    */
  const void *b_qkv;    /* [3D] bf16          */
  const uint8_t *w_o;   /* [D][D] E4M3 codes  */
  const float *s_o;     /* [D] row scales     */
  const void *b_o;      /* [D] bf16           */
} hilo_attn_w_fp8;

typedef struct {
  const uint8_t *w1; /* [F][D] E4M3 codes */
  const float *s1;   /* [F] row scales    */
  const void *b1;    /* [F] bf16          */
  const uint8_t *w2; /* [D][F] E4M3 codes */
  const float *s2;   /* [D] row scales    */
  const void *b2;    /* [D] bf16          */
} hilo_mlp_w_fp8;

/* Per-row E4M3 quantisation (as above) of x [rows][cols], dtype HILO_F32 or HILO_BF16 (read
 * exactly as float32): codes [rows][cols] uint8, scale [rows] float32, all device memory.  For
 * preparing FP8 weights once per model.  cols > 0 and cols % 4 == 0, 0 <= rows < 2^31 - 4
 * (HILO_E_SHAPE otherwise); rows == 0 enqueues nothing.                                          */
hilo_status hilo_quantize_rows(int32_t dtype, const void *x, int64_t rows, int64_t cols,
                               uint8_t *codes, float *scale, void *stream);

/* Workspace of the FP8 block (hilo_attention_fp8, hilo_mlp_fp8): hilo_workspace_bytes plus one
 * region that holds the attention output's bf16 rows in the attention half and the hidden rows'
 * codes and scales in the MLP half; 0 if the shape is invalid for the FP8 block.                 */
size_t hilo_workspace_bytes_fp8(const hilo_shape *shape);

/* hilo_attention with both projections and the attention's score product in FP8 (Sec. 3.3): h =
 * LN(z) * (1 + scale1) + shift1 is formed in float32 and quantised per row straight from
 * registers, then multiplied by the FP8 W_qkv; that projection's q and k leave as E4M3 codes with a
 * power-of-two scale per (row, head) -- 2^k, k the least integer with 448 2^k >= the row's amax --
 * formed from its float32 values, v as bf16; the attention core multiplies the FP8 q and k
 * (hilo_attention_core_fp8), softmax and P V as in hilo_attention; its output rows are quantised
 * and multiplied by the FP8 W_o.  shape->dtype must be HILO_BF16 (HILO_E_DTYPE), dim a multiple of
 * 256 and mlp_dim of 128 (HILO_E_SHAPE).  workspace: ws_bytes >= hilo_workspace_bytes_fp8(shape). */
hilo_status hilo_attention_fp8(const hilo_shape *shape, float *z, const int32_t *cu_seqlens,
                               const hilo_attn_w_fp8 w[2], const float *mod, void *workspace,
                               size_t ws_bytes, void *stream);

/* hilo_mlp with both projections in FP8 (h2 quantised where it is formed, the GELU output by a pass
 * over its bf16 rows); the gated residual as in hilo_mlp.  Requirements as hilo_attention_fp8;
 * workspace: ws_bytes >= hilo_workspace_bytes_fp8(shape).                                        */
hilo_status hilo_mlp_fp8(const hilo_shape *shape, float *z, const int32_t *cu_seqlens,
                         const hilo_mlp_w_fp8 w[2], const float *mod, void *workspace,
                         size_t ws_bytes, void *stream);

/* The FP8 block's counterparts of hilo_compress_norm / hilo_attention_normed (Sec. 2.3 and
 * Sec. 3.3): z as hilo_compress, and the attention half's normalised rows as the FP8 block's
 * projection input (per-row E4M3 codes and row scales, as hilo_attention_fp8 forms them, bit for
 * bit) in the workspace; then hilo_attention_fp8 from its QKV projection on.  Shapes, pointers and
 * workspace (ws_bytes >= hilo_workspace_bytes_fp8(shape), the same one for both calls with nothing
 * enqueued on it in between) as hilo_attention_fp8 and hilo_compress_norm.                      */
hilo_status hilo_compress_norm_fp8(const hilo_shape *shape, const void *x_img, const void *x_txt,
                                   const int32_t *fine_idx, const int32_t *pool_idx, const int32_t *counts,
                                   const int32_t *cu_seqlens, const int32_t *seg_off, const float *mod,
                                   float *z, void *workspace, size_t ws_bytes, void *stream);
hilo_status hilo_attention_fp8_normed(const hilo_shape *shape, float *z, const int32_t *cu_seqlens,
                                      const hilo_attn_w_fp8 w[2], const float *mod, void *workspace,
                                      size_t ws_bytes, void *stream);

/* S6 -- decompress.  The paper does not say how the DiT's output on the HiLo tokens returns to the
 * full grid; this is the plain reading (each patch takes its token's output):
 * y_img[g][p] = z[seg_off[g] + idx_map[g][p]] (fine tokens scatter back to
 * their patch, pooled tokens broadcast to the 4 patches of their block), y_txt[s][t] = the text
 * rows of sample s; both rounded to dtype.  y_img [G][N][D], y_txt [B][L][D] or NULL.  A patch
 * without a token (idx_map -1, token set DROP) gets zeros: use hilo_decompress_delta there.     */
hilo_status hilo_decompress(const hilo_shape *shape, const float *z, const int32_t *idx_map,
                            const int32_t *cu_seqlens, const int32_t *seg_off, void *y_img,
                            void *y_txt, void *stream);

/* S6, delta form (for the OVERLAP and DROP token sets): the block's change of a token is added to
 * the patches it stands for, y_img[g][p] = x_img[g][p] + (z[row] - z0[row]) with row =
 * seg_off[g] + idx_map[g][p] and z0[row] the value hilo_compress wrote there, recomputed from
 * x_img with the same float32 operations (the patch itself for a fine row, the block mean
 * ((x00 + x01) + (x10 + x11)) * 0.25 for a pooled row; a row is fine when idx_map < counts[g][0]).
 * Patches without a token keep x_img.  A pooled token's update thus reaches its 4 patches on top
 * of their own high-frequency detail instead of replacing them by the block mean.  Text rows as
 * in hilo_decompress.  Float32 arithmetic, rounded to dtype once.                                */
hilo_status hilo_decompress_delta(const hilo_shape *shape, const float *z, const void *x_img,
                                  const int32_t *idx_map, const int32_t *counts,
                                  const int32_t *cu_seqlens, const int32_t *seg_off, void *y_img,
                                  void *y_txt, void *stream);

/* The attention core alone (the softmax(q k^T / sqrt(hd)) v step of hilo_attention), for
 * localising parity failures and timing: qkv [T_max][3D] dtype -> out [T_max][D] dtype, rows of
 * sample s attend to the rows of sample s.  workspace: device scratch of ws_bytes >=
 * hilo_workspace_bytes(shape) for the bf16 path (its partial results); may be NULL for F32.      */
hilo_status hilo_attention_core(const hilo_shape *shape, const void *qkv,
                                const int32_t *cu_seqlens, void *out, void *workspace,
                                size_t ws_bytes, void *stream);

/* The FP8 block's attention core alone (Sec. 3.3, "Compatibility with Quantization and
 * Distillation": FP8 on top of the compression; here the score product q k^T runs on FP8 operands):
 * qkv8 holds T_max rows of 6 D bytes -- bytes [0, D) the q codes, [D, 2 D) the k codes (OCP E4M3,
 * head h in bytes h hd .. of each), [2 D, 2 D + 2 H) one E8M0 scale byte per (row, head), q heads
 * then k heads (row scale 2^(byte - 127)), and bytes [4 D, 6 D) the v row in bf16 -- the layout
 * hilo_attention_fp8's QKV projection writes.  out [T_max][D] bf16 = softmax(q k^T / sqrt(hd)) v
 * with q, k dequantised (code value times scale) and the probabilities and v as in the bf16 core;
 * rows of sample s attend to the rows of sample s.  Shape: as hilo_attention_fp8 (bf16, dim a
 * multiple of 256).  workspace: device scratch of ws_bytes >= hilo_workspace_bytes(shape).      */
hilo_status hilo_attention_core_fp8(const hilo_shape *shape, const void *qkv8,
                                    const int32_t *cu_seqlens, void *out, void *workspace,
                                    size_t ws_bytes, void *stream);

/* hilo_attention_core without a workspace, for callers that cannot allocate device memory (code
 * under HIP graph capture, serving loops and harnesses that forbid hipMalloc): the same kernels and
 * launch, with the stream-K partial results in a scratch array the library holds on each device
 * it runs on (HILO_ATTN_SCRATCH_BYTES, set up on the first call on a device, kept until the process
 * ends).  It calls no allocating routine.  Nothing in the scratch needs clearing between calls,
 * but every call on one device shares it: calls that overlap on one device (on different streams,
 * or from several host threads) race and give undefined results.  The core sizes its launch so
 * that its partial results fit the scratch at any sequence length; HILO_E_WORKSPACE reports a
 * breach of that bound, HILO_E_DEVICE a failed lookup of the scratch; other statuses as
 * hilo_attention_core.  No kernel timing.                                                       */
#define HILO_ATTN_SCRATCH_BYTES ((size_t)72 * 1024 * 1024)
hilo_status hilo_attention_core_noalloc(const hilo_shape *shape, const void *qkv,
                                        const int32_t *cu_seqlens, void *out, void *stream);

size_t hilo_workspace_bytes(const hilo_shape *shape); /* 0 if the shape is invalid */
/* T_max = batch * (images * (N + N/4) + text_len): the most rows any token set can produce
 * (OVERLAP with every block kept); z and the workspace are sized for it, -1 if invalid.         */
int64_t hilo_max_tokens(const hilo_shape *shape);
const char *hilo_status_str(int32_t status);
int32_t hilo_abi_version(void);

/* Kernel timing.  While enabled, every kernel the library launches is bracketed by a pair of HIP
 * events recorded on its launch stream; hilo_profile_read returns, after the caller has
 * synchronised, the summed milliseconds and launch count of one kernel kind since the last
 * hilo_profile_enable(1).  kind in [0, hilo_profile_kinds()); hilo_profile_name(kind) names it.
 * Not thread safe; meant for benchmarks.                                                         */
hilo_status hilo_profile_enable(int32_t on);
hilo_status hilo_profile_read(int32_t kind, double *total_ms, int64_t *launches);
int32_t hilo_profile_kinds(void);
const char *hilo_profile_name(int32_t kind);

#ifdef __cplusplus
}
#endif

#endif /* HILO_H */
