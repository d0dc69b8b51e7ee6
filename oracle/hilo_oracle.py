"""CPU oracle for the HiLo-Token compressed DiT block.  TEST INFRASTRUCTURE ONLY.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may import this module; the
product path (the HIP library and its Python binding) never does.  It shares no code with the HIP
path: the only thing both sides have in common is the seeded input generator, which holds none of
the method's arithmetic.

The oracle is plain and slow on purpose.  It follows the method step by step, in the order of the
paper's description of HiLo-Token selection (Sec. 2.3, "HiLo-Token Selection"), followed by one
diffusion-transformer block on the shortened sequence and the reassembly of the full grid:

  score      Sobel frequency energy per latent patch              (Sec. 2.3, Sobel operators)
  score_pixels  the same energy on the RGB image, summed over each  (Sec. 2.3, Sobel on the image,
             token's 16 x 16 pixels                                 16x pooling to the token grid)
  select     2x2 regional pooling, threshold or top-k, dilated    (Sec. 2.3, regionalisation +
             user mask forced fine                                  dilated mask; Sec. 1)
  compact    index map: fine patches, pooled blocks, their ranks   (Sec. 2.3, token-dim concat)
  compress   fine rows copied, pooled rows = mean of 4 patches     (Sec. 2.3; Abstract: LF tokens
                                                                     carry the blurry global part)
  block      joint attention + MLP over image and text tokens      (Sec. 2.2 / Sec. 4: DiT whose
                                                                     cost is quadratic in tokens)
  stack      blocks in order; request = one selection, then per   (Sec. 2.3: selection once per
             step compress -> stack -> decompress                   request; Sec. 3.3: 8 steps)
  fp8        per-row E4M3 quantisation of the operands of the     (Sec. 3.3: FP8 quantisation
             four projections and of the attention's q and k        on top of the compression)
  decompress scatter fine rows, broadcast pooled rows to 4 patches

Precision.  Floating point that decides an integer (the energy that decides which blocks stay
fine) is computed in float32, one IEEE round-to-nearest operation at a time, in a fixed order and
never fused; the device takes the same decision in the same precision.  Everything else (pooling,
layer norm, projections, attention, MLP) is float64.  Matrix products use numpy's matmul as a
library primitive.

Readings of the paper where it is silent or loose are listed in the design notes; each function
below states the reading it implements.

Parity status per function (what pins it is in tests/test_oracle_*.py):
  score, score_pixels, dilate, block_sums, select_*, compact, layout, compress, decompress,
  attention, mlp, stack, request, e4m3_value, quantize_rows, pow2_exponent, quantize_rows_pow2,
  attend_codes:
  pinned by closed forms, library routines (scipy Sobel / binary dilation, torch SDPA / layer_norm
  / gelu), hand-worked fixtures under tests/golden/, and the identities of the method (0% compression
  equals the dense block, pooling a constant block then broadcasting is lossless, kept-token count
  equals the selection rule's count).  Against the paper's own numbers: parity unpinned -- the paper
  prints no worked example, intermediate value or error bound, and its weights and data are not
  available.
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

CAP = np.float32(2.0 ** 22)    # per-channel energy cap before quantisation
SCALE = np.float32(2.0 ** 16)  # fixed-point scale of the per-channel energy
LN_EPS = 1e-6


# ------------------------------------------------------------------------------------------------
# S1  score
# ------------------------------------------------------------------------------------------------

def score(x_img: np.ndarray, grid_h: int, grid_w: int) -> np.ndarray:
    """Per-patch Sobel frequency energy, summed over channels as 64-bit fixed point.

    Sec. 2.3 estimates a spatial-frequency map with two Sobel convolutions.  Reading used here: the
    Sobel pair runs across the latent patch grid, per channel, with replicated borders; the energy
    of one channel is gx^2 + gy^2 in float32, capped at 2^22, scaled by 2^16 and floored to an
    integer; a patch's energy is the exact int64 sum over channels (so the channel order cannot
    change the result).

    x_img [G][N][D] float32, N = grid_h * grid_w in raster order  ->  E [G][N] int64
    """
    x_all = np.asarray(x_img, dtype=np.float32)
    G, N, D = x_all.shape
    assert N == grid_h * grid_w
    E = np.empty((G, N), dtype=np.int64)
    two = np.float32(2.0)
    for g in range(G):
        x = x_all[g].reshape(grid_h, grid_w, D)
        xp = np.pad(x, ((1, 1), (1, 1), (0, 0)), mode="edge")  # replicate border

        def at(di: int, dj: int) -> np.ndarray:
            return xp[1 + di:1 + di + grid_h, 1 + dj:1 + dj + grid_w, :]

        # horizontal derivative: right column minus left column, rows weighted 1, 2, 1
        gx = ((at(-1, 1) + two * at(0, 1)) + at(1, 1)) - ((at(-1, -1) + two * at(0, -1)) + at(1, -1))
        # vertical derivative: lower row minus upper row, columns weighted 1, 2, 1
        gy = ((at(1, -1) + two * at(1, 0)) + at(1, 1)) - ((at(-1, -1) + two * at(-1, 0)) + at(-1, 1))
        t1 = gx * gx
        t2 = gy * gy
        v = t1 + t2
        q = np.floor(np.fmin(v, CAP) * SCALE).astype(np.int64)  # fmin: a NaN energy takes the cap
        E[g] = q.sum(axis=-1, dtype=np.int64).reshape(N)
    return E


PIX_PER_TOKEN = 16  # image pixels per token side: 8x VAE x 2x patch embedding (Sec. 2.3)


def score_pixels(rgb: np.ndarray, grid_h: int, grid_w: int) -> np.ndarray:
    """Per-token frequency energy from the image itself, the paper's selector (Sec. 2.3: Sobel
    operators on the image, then 16x spatial pooling onto the token grid).  The per-pixel energy is
    `score`'s (float32 per operation, capped, 2^-16 fixed point, replicated border) on the pixel
    grid with the 3 colour channels as channels; a token's energy is the exact sum over its 16 x 16
    pixels (a sum rather than a mean: the normalisation by the maximum cancels the factor).

    rgb [G][3][16 grid_h][16 grid_w] float32  ->  E [G][grid_h * grid_w] int64"""
    rgb = np.asarray(rgb, dtype=np.float32)
    G, C, Hp, Wp = rgb.shape
    T = PIX_PER_TOKEN
    assert Hp == T * grid_h and Wp == T * grid_w
    per_pixel = score(rgb.transpose(0, 2, 3, 1).reshape(G, Hp * Wp, C), Hp, Wp)
    return per_pixel.reshape(G, grid_h, T, grid_w, T).sum(axis=(2, 4), dtype=np.int64).reshape(G, grid_h * grid_w)


# ------------------------------------------------------------------------------------------------
# S2  select
# ------------------------------------------------------------------------------------------------

def block_of(grid_h: int, grid_w: int) -> np.ndarray:
    """Block index b = (i // 2) * (grid_w // 2) + (j // 2) of every patch p = i * grid_w + j."""
    i, j = np.divmod(np.arange(grid_h * grid_w), grid_w)
    return (i // 2) * (grid_w // 2) + (j // 2)


def block_sums(E: np.ndarray, grid_h: int, grid_w: int) -> np.ndarray:
    """Regional pooling of the frequency map onto the coarse grid (Sec. 2.3, regionalisation):
    B_b = sum of the 4 patch energies of 2x2 block b (exact int64).  [G][N] -> [G][N/4]."""
    G = E.shape[0]
    e = E.reshape(G, grid_h // 2, 2, grid_w // 2, 2)
    return (((e[:, :, 0, :, 0] + e[:, :, 0, :, 1]) + e[:, :, 1, :, 0]) + e[:, :, 1, :, 1]).reshape(G, -1)


def dilate(force: Optional[np.ndarray], grid_h: int, grid_w: int, r: int, G: int) -> np.ndarray:
    """Dilated user mask (Sec. 2.3: the user mask is dilated and combined with the HF map).

    Reading: square (Chebyshev) structuring element of radius r patches, clipped at the grid edge:
    force'(p) = 1 iff some force(q) = 1 with max(|di|, |dj|) <= r.  Returns bool [G][N]."""
    if force is None:
        return np.zeros((G, grid_h * grid_w), dtype=bool)
    f = np.asarray(force).reshape(G, grid_h, grid_w) != 0
    out = np.zeros_like(f)
    for di in range(-r, r + 1):
        for dj in range(-r, r + 1):
            src_i = slice(max(0, di), grid_h + min(0, di))
            dst_i = slice(max(0, -di), grid_h + min(0, -di))
            src_j = slice(max(0, dj), grid_w + min(0, dj))
            dst_j = slice(max(0, -dj), grid_w + min(0, -dj))
            out[:, dst_i, dst_j] |= f[:, src_i, src_j]
    return out.reshape(G, -1)


def forced_blocks(force: Optional[np.ndarray], grid_h: int, grid_w: int, r: int, G: int) -> np.ndarray:
    """F: blocks holding at least one patch of the dilated mask.  bool [G][N/4]."""
    d = dilate(force, grid_h, grid_w, r, G)
    blk = block_of(grid_h, grid_w)
    F = np.zeros((G, grid_h * grid_w // 4), dtype=bool)
    for g in range(G):
        np.logical_or.at(F[g], blk, d[g])
    return F


def select_threshold(E: np.ndarray, force: Optional[np.ndarray], grid_h: int, grid_w: int, r: int,
                     tau: Sequence[float]) -> np.ndarray:
    """Threshold selection (Sec. 2.3: keep tokens whose normalised frequency exceeds a threshold,
    e.g. 0.1, after regional pooling; the dilated mask is kept in any case).

    Reading: normalised map = E / max(E) per grid; a block stays fine when the mean of its 4
    normalised energies strictly exceeds tau, i.e. B_b > 4 tau E_max, compared in double with the
    right-hand side formed as one product (4.0 * tau) * E_max.  A flat grid (E_max = 0) keeps only
    forced blocks.  Returns bool fine[G][N/4]."""
    G = E.shape[0]
    B = block_sums(E, grid_h, grid_w)
    F = forced_blocks(force, grid_h, grid_w, r, G)
    fine = F.copy()
    for g in range(G):
        emax = int(E[g].max())
        if emax > 0:
            rhs = (4.0 * float(tau[g])) * float(emax)
            fine[g] |= B[g].astype(np.float64) > rhs
    return fine


def select_topk(E: np.ndarray, force: Optional[np.ndarray], grid_h: int, grid_w: int, r: int,
                keep: Sequence[int]) -> np.ndarray:
    """Top-k selection: the forced blocks first, then the highest-scoring other blocks until K blocks
    are fine (ties: lower block index first).  |fine| = max(K, |F|).  Returns bool fine[G][N/4]."""
    G = E.shape[0]
    B = block_sums(E, grid_h, grid_w)
    F = forced_blocks(force, grid_h, grid_w, r, G)
    fine = F.copy()
    for g in range(G):
        extra = max(0, int(keep[g]) - int(F[g].sum()))
        cand = np.flatnonzero(~F[g])
        order = np.lexsort((cand, -B[g][cand]))  # primary: B descending, secondary: index ascending
        fine[g][cand[order[:extra]]] = True
    return fine


TOKEN_SETS = ("partition", "overlap", "drop")


def compact(fine: np.ndarray, grid_h: int, grid_w: int, tokens: str = "partition") -> Tuple[np.ndarray, ...]:
    """Index map of the compressed grid (Sec. 2.3: selected HF tokens are concatenated with the LF
    tokens along the token dimension).

    Per grid the compressed image tokens are [fine patches in raster order ; pooled blocks in block
    raster order].  Which blocks get a pooled (LF) token depends on the token set:
      partition  the blocks that are not fine (every patch represented once)
      overlap    every block (Sec. 2.3: all LF tokens are kept, next to the selected HF tokens)
      drop       none (Sec. 3.2: for text-prompted fill the tokens outside the dilated mask can be
                 pruned entirely); patches of other blocks then have no row (idx_map -1)
    Returns
      idx_map  [G][N]    compressed row of every patch (a fine patch's own row, else its block's row,
                         or -1 without one)
      fine_idx [G][N]    patch index of compressed row k < n_fine (entries >= n_fine are -1)
      pool_idx [G][N/4]  block index of pooled row k < n_pool (rest -1)
      counts   [G][2]    (n_fine, n_pool)
    """
    G, NB = fine.shape
    N = grid_h * grid_w
    blk = block_of(grid_h, grid_w)
    idx_map = np.empty((G, N), dtype=np.int32)
    fine_idx = np.full((G, N), -1, dtype=np.int32)
    pool_idx = np.full((G, NB), -1, dtype=np.int32)
    counts = np.empty((G, 2), dtype=np.int32)
    if tokens not in TOKEN_SETS:
        raise ValueError(tokens)
    for g in range(G):
        fine_patch = fine[g][blk]
        fp = np.flatnonzero(fine_patch)
        pooled = {"partition": ~fine[g], "overlap": np.ones(NB, dtype=bool), "drop": np.zeros(NB, dtype=bool)}[tokens]
        pb = np.flatnonzero(pooled)
        n_fine, n_pool = fp.size, pb.size
        fine_idx[g, :n_fine] = fp
        pool_idx[g, :n_pool] = pb
        rank_fine = np.cumsum(fine_patch) - 1
        rank_pool = np.cumsum(pooled) - 1
        other = np.where(pooled[blk], n_fine + rank_pool[blk], -1)
        idx_map[g] = np.where(fine_patch, rank_fine, other)
        counts[g] = (n_fine, n_pool)
    return idx_map, fine_idx, pool_idx, counts


def layout(counts: np.ndarray, batch: int, images: int, text_len: int) -> Tuple[np.ndarray, np.ndarray]:
    """Packed ragged sequence: sample s = [grid 0 tokens ; grid 1 tokens ; ... ; text tokens].
    Returns cu_seqlens [B+1] (row offsets of samples) and seg_off [G] (first row of each grid)."""
    cu = np.zeros(batch + 1, dtype=np.int32)
    seg = np.zeros(batch * images, dtype=np.int32)
    for s in range(batch):
        row = int(cu[s])
        for i in range(images):
            g = s * images + i
            seg[g] = row
            row += int(counts[g, 0]) + int(counts[g, 1])
        cu[s + 1] = row + text_len
    return cu, seg


# ------------------------------------------------------------------------------------------------
# S3 / S6  compress, decompress
# ------------------------------------------------------------------------------------------------

def compress(x_img: np.ndarray, x_txt: np.ndarray, grid_h: int, grid_w: int, fine_idx: np.ndarray,
             pool_idx: np.ndarray, counts: np.ndarray, cu: np.ndarray, seg: np.ndarray,
             text_len: int) -> np.ndarray:
    """Build the compressed sequence Z [cu[B]][D] (float64).

    Fine rows are the patch tokens themselves (HF tokens).  Each pooled row is the mean of the 4
    patches of its 2x2 block (reading of the LF token under the partition of the grid into fine and
    pooled blocks).  Text rows are copied after the image rows of their sample."""
    G, N, D = x_img.shape
    B = x_txt.shape[0]
    Z = np.zeros((int(cu[B]), D), dtype=np.float64)
    W2 = grid_w // 2
    for g in range(G):
        x = x_img[g].astype(np.float64)
        nf, npool = int(counts[g, 0]), int(counts[g, 1])
        base = int(seg[g])
        Z[base:base + nf] = x[fine_idx[g, :nf]]
        b = pool_idx[g, :npool].astype(np.int64)
        p00 = (b // W2) * 2 * grid_w + (b % W2) * 2
        Z[base + nf:base + nf + npool] = (x[p00] + x[p00 + 1] + x[p00 + grid_w] + x[p00 + grid_w + 1]) / 4.0
    for s in range(B):
        Z[int(cu[s + 1]) - text_len:int(cu[s + 1])] = x_txt[s].astype(np.float64)
    return Z


def decompress(Z: np.ndarray, idx_map: np.ndarray, cu: np.ndarray, seg: np.ndarray,
               text_len: int, batch: int, x_img: Optional[np.ndarray] = None,
               Z_in: Optional[np.ndarray] = None) -> Tuple[np.ndarray, np.ndarray]:
    """Reassemble the full grid (the paper is silent on this step).

    Broadcast form (Z_in None): Y_img[g][p] = Z[seg[g] + idx_map[g][p]] -- fine rows scatter back
    to their patch, pooled rows broadcast to the 4 patches of their block; a patch without a row
    gets zeros.  Delta form (x_img and Z_in, the sequence as compressed): Y_img[g][p] = x[g][p] +
    (Z[row] - Z_in[row]) -- the block's change of the token is added to every patch it stands for;
    a patch without a row keeps x.  Y_txt = the text rows of Z in both forms."""
    G, N = idx_map.shape
    y_img = np.zeros((G, N, Z.shape[1]), dtype=np.float64)
    for g in range(G):
        has = idx_map[g] >= 0
        rows = int(seg[g]) + idx_map[g][has].astype(np.int64)
        if Z_in is None:
            y_img[g][has] = Z[rows]
        else:
            x = x_img[g].astype(np.float64)
            y_img[g] = x
            y_img[g][has] = x[has] + (Z[rows] - Z_in[rows])
    y_txt = np.stack([Z[int(cu[s + 1]) - text_len:int(cu[s + 1])] for s in range(batch)])
    return y_img, y_txt


# ------------------------------------------------------------------------------------------------
# S4 / S5  the DiT block on the compressed sequence
# ------------------------------------------------------------------------------------------------

def layer_norm(z: np.ndarray) -> np.ndarray:
    """LayerNorm over the last axis, biased variance, eps 1e-6, no affine (adaLN supplies it)."""
    mu = z.mean(axis=-1, keepdims=True)
    var = ((z - mu) ** 2).mean(axis=-1, keepdims=True)
    return (z - mu) / np.sqrt(var + LN_EPS)


def gelu_tanh(u: np.ndarray) -> np.ndarray:
    """GELU, tanh form: 0.5 u (1 + tanh(sqrt(2/pi) (u + 0.044715 u^3)))."""
    return 0.5 * u * (1.0 + np.tanh(np.sqrt(2.0 / np.pi) * (u + 0.044715 * u ** 3)))


def _segments(cu: np.ndarray, text_len: int):
    """(sample, stream, first row, end row) of every image/text segment of the packed sequence."""
    for s in range(len(cu) - 1):
        yield s, 0, int(cu[s]), int(cu[s + 1]) - text_len
        yield s, 1, int(cu[s + 1]) - text_len, int(cu[s + 1])


# ------------------------------------------------------------------------------------------------
# FP8 (Sec. 3.3: the compressed DiT combines with FP8 quantisation)
# ------------------------------------------------------------------------------------------------

E4M3_MAX = np.float32(448.0)


def e4m3_value(codes: np.ndarray) -> np.ndarray:
    """Value of OCP FP8 E4M3 codes (1 sign, 4 exponent bits with bias 7, 3 mantissa bits; exponent
    0 is subnormal; 0x7f / 0xff are NaN, there is no infinity), float64."""
    c = np.asarray(codes, dtype=np.uint8).astype(np.int64)
    sign = np.where(c & 0x80, -1.0, 1.0)
    e = (c >> 3) & 0xF
    m = (c & 0x7).astype(np.float64)
    v = np.where(e == 0, m / 8.0 * 2.0 ** -6, (1.0 + m / 8.0) * np.exp2(e.astype(np.float64) - 7.0))
    v = np.where((e == 15) & (m == 7), np.nan, v)
    return sign * v


def quantize_rows(x: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """Per-row FP8 E4M3 quantisation, every step one float32 operation:
      amax = max |x| over the row;  inv = 448 / amax (correctly rounded; 0 for an all-zero row)
      code = round-to-nearest-even E4M3 of clamp(x * inv, -448, 448);  scale = amax / 448
    so code value * scale approximates x.  x [R][C] float32 -> codes uint8 [R][C], scale float32 [R].
    (The rounding to E4M3 uses torch's float8_e4m3fn cast as a library primitive.)"""
    import torch

    x = np.asarray(x, dtype=np.float32)
    amax = np.abs(x).max(axis=1)
    with np.errstate(divide="ignore"):
        inv = np.where(amax > 0, E4M3_MAX / amax, np.float32(0)).astype(np.float32)
    y = np.clip(x * inv[:, None], -E4M3_MAX, E4M3_MAX).astype(np.float32)
    codes = torch.from_numpy(y).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    scale = (amax / E4M3_MAX).astype(np.float32)
    return codes, scale


def dequant_rows(codes: np.ndarray, scale: np.ndarray) -> np.ndarray:
    return e4m3_value(codes) * np.asarray(scale, dtype=np.float64)[:, None]


def pow2_exponent(amax: np.ndarray) -> np.ndarray:
    """Smallest integer k with 448 * 2^k >= amax (0 where amax is 0), from the exact binary
    decomposition amax = m * 2^E, m in [0.5, 1): 448 = 0.875 * 2^9, so k = E - 9 when m <= 0.875 and
    E - 8 otherwise; clamped below at -127, the least E8M0 scale (a row that small still fits:
    amax * 2^127 < 448).  amax float32 [R] -> int64 [R]."""
    m, E = np.frexp(np.asarray(amax, dtype=np.float64))
    k = np.maximum(np.where(m <= 0.875, E - 9, E - 8), -127).astype(np.int64)
    return np.where(np.asarray(amax) > 0, k, 0)


def quantize_rows_pow2(x: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """Per-row FP8 E4M3 quantisation with a power-of-two scale (the form an E8M0 block scale takes):
      k = pow2_exponent(max |x| over the row);  code = round-to-nearest-even E4M3 of x * 2^-k
    (x * 2^-k is exact and lies in [-448, 448], so nothing saturates), code value * 2^k approximates
    x.  x [R][C] float32 -> codes uint8 [R][C], exponents int64 [R].  (The rounding to E4M3 uses
    torch's float8_e4m3fn cast as a library primitive.)"""
    import torch

    x = np.asarray(x, dtype=np.float32)
    k = pow2_exponent(np.abs(x).max(axis=1))
    y = (x.astype(np.float64) * np.exp2(-k.astype(np.float64))[:, None]).astype(np.float32)
    codes = torch.from_numpy(y).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    return codes, k


def dequant_rows_pow2(codes: np.ndarray, k: np.ndarray) -> np.ndarray:
    return e4m3_value(codes) * np.exp2(np.asarray(k, dtype=np.float64))[:, None]


def _fp8_matmul(h: np.ndarray, q) -> np.ndarray:
    """h @ W^T with both operands FP8 per row: h quantised per row (rounded to float32 first), W given
    as its per-output-channel codes and scales q = quantize_rows(W)."""
    hc, hs = quantize_rows(h.astype(np.float32))
    wc, ws = q
    return dequant_rows(hc, hs) @ dequant_rows(wc, ws).T


def _w(weights, sigma: int, name: str) -> np.ndarray:
    return np.asarray(weights[sigma][name], dtype=np.float64)


def _attend(q: np.ndarray, k: np.ndarray, v: np.ndarray, heads: int) -> np.ndarray:
    """softmax(q k^T / sqrt(head_dim)) v per head (columns h*hd .. (h+1)*hd), float64."""
    D = q.shape[1]
    hd = D // heads
    out = np.empty((q.shape[0], D), dtype=np.float64)
    for hh in range(heads):
        cols = slice(hh * hd, (hh + 1) * hd)
        sc = (q[:, cols] @ k[:, cols].T) / np.sqrt(hd)
        sc = sc - sc.max(axis=1, keepdims=True)
        p = np.exp(sc)
        p /= p.sum(axis=1, keepdims=True)
        out[:, cols] = p @ v[:, cols]
    return out


def _attend_scores(qh: np.ndarray, kh: np.ndarray, v: np.ndarray) -> np.ndarray:
    """softmax(qh kh^T / sqrt(head_dim)) v for one head given its (dequantised) q and k, float64."""
    sc = (qh @ kh.T) / np.sqrt(qh.shape[1])
    sc = sc - sc.max(axis=1, keepdims=True)
    p = np.exp(sc)
    p /= p.sum(axis=1, keepdims=True)
    return p @ v


def _attend_fp8(q: np.ndarray, k: np.ndarray, v: np.ndarray, heads: int) -> np.ndarray:
    """_attend with the score product on FP8 operands: every (token, head) row of q and of k is
    quantised per row with a power-of-two scale (quantize_rows_pow2, from the computed value rounded
    once to float32); the probabilities and v are not quantised.  float64."""
    D = q.shape[1]
    hd = D // heads
    out = np.empty((q.shape[0], D), dtype=np.float64)
    for hh in range(heads):
        cols = slice(hh * hd, (hh + 1) * hd)
        qh = dequant_rows_pow2(*quantize_rows_pow2(q[:, cols].astype(np.float32)))
        kh = dequant_rows_pow2(*quantize_rows_pow2(k[:, cols].astype(np.float32)))
        out[:, cols] = _attend_scores(qh, kh, v[:, cols])
    return out


def attend_codes(q_codes: np.ndarray, q_exp: np.ndarray, k_codes: np.ndarray, k_exp: np.ndarray,
                 v: np.ndarray, heads: int) -> np.ndarray:
    """The FP8-score attention of one sample from given codes: q_codes / k_codes uint8 [n][D] (head h
    in columns h*hd ..), q_exp / k_exp int [n][heads] (row scale 2^exp of each (token, head)), v
    [n][D].  The step after the quantisation of _attend_fp8, float64."""
    D = q_codes.shape[1]
    hd = D // heads
    out = np.empty((q_codes.shape[0], D), dtype=np.float64)
    for hh in range(heads):
        cols = slice(hh * hd, (hh + 1) * hd)
        qh = dequant_rows_pow2(q_codes[:, cols], q_exp[:, hh])
        kh = dequant_rows_pow2(k_codes[:, cols], k_exp[:, hh])
        out[:, cols] = _attend_scores(qh, kh, np.asarray(v, dtype=np.float64)[:, cols])
    return out


def attention_core(qkv: np.ndarray, cu: np.ndarray, heads: int,
                   rows: Optional[np.ndarray] = None) -> np.ndarray:
    """The attention step alone on a packed [T][3D] projection: every row attends to all rows of
    its own sample.  Returns a for `rows` (all rows when None), float64 [len(rows)][D]."""
    qkv = np.asarray(qkv, dtype=np.float64)
    D = qkv.shape[1] // 3
    rows = np.arange(int(cu[-1])) if rows is None else np.asarray(rows)
    out = np.empty((rows.size, D), dtype=np.float64)
    for s in range(len(cu) - 1):
        lo, hi = int(cu[s]), int(cu[s + 1])
        sel = np.flatnonzero((rows >= lo) & (rows < hi))
        if sel.size:
            out[sel] = _attend(qkv[rows[sel], :D], qkv[lo:hi, D:2 * D], qkv[lo:hi, 2 * D:], heads)
    return out


def attention(Z: np.ndarray, cu: np.ndarray, text_len: int, heads: int, weights, mod: np.ndarray,
              rows: Optional[np.ndarray] = None, fp8=None) -> np.ndarray:
    """Attention half of an MMDiT-style pre-LN adaLN block with per-stream weights:

      h   = LN(z) * (1 + scale1) + shift1
      qkv = h W_qkv^T + b_qkv                       (image and text rows use their own weights)
      a   = softmax(q k^T / sqrt(head_dim)) v       per head, over all rows of the same sample
      z1  = z + gate1 * (a W_o^T + b_o)

    Joint attention over image + text tokens of one sample, no mask (Sec. 2.3: the HiLo tokens are
    processed by the DiT; Sec. 2.2: memory-efficient attention).  Returns z1 for `rows` (all rows
    when None), float64 [len(rows)][D].  With `fp8` (per stream {"w_qkv": (codes, scale), "w_o": ...})
    both projections multiply FP8 rows of their input by FP8 rows of the weight (quantize_rows): each
    input row is quantised from the value the block computes (h, then the attention output a), in
    float64 rounded once to float32 (Sec. 3.3 names FP8 quantisation of the network and nothing about
    an intermediate storage precision, so none is assumed); and the attention's score product runs
    on FP8 q and k, each (token, head) row with a power-of-two scale (_attend_fp8)."""
    T, D = Z.shape
    all_rows = np.arange(T) if rows is None else np.asarray(rows)
    out = np.empty((all_rows.size, D), dtype=np.float64)
    for s in range(len(cu) - 1):
        lo, hi = int(cu[s]), int(cu[s + 1])
        sel = np.flatnonzero((all_rows >= lo) & (all_rows < hi))
        if sel.size == 0:
            continue
        qkv = np.empty((hi - lo, 3 * D), dtype=np.float64)
        for (ss, sig, a, b) in _segments(cu, text_len):
            if ss != s or b <= a:
                continue
            h = layer_norm(Z[a:b]) * (1.0 + mod[s, sig, 1]) + mod[s, sig, 0]
            prod = _fp8_matmul(h, fp8[sig]["w_qkv"]) if fp8 is not None else h @ _w(weights, sig, "w_qkv").T
            qkv[a - lo:b - lo] = prod + _w(weights, sig, "b_qkv")
        r_loc = all_rows[sel] - lo
        attend = _attend_fp8 if fp8 is not None else _attend
        a_out = attend(qkv[r_loc, :D], qkv[:, D:2 * D], qkv[:, 2 * D:], heads)
        text_start = hi - text_len
        for sig in (0, 1):
            m = (all_rows[sel] >= text_start) if sig == 1 else (all_rows[sel] < text_start)
            if not m.any():
                continue
            prod = (_fp8_matmul(a_out[m], fp8[sig]["w_o"]) if fp8 is not None
                    else a_out[m] @ _w(weights, sig, "w_o").T)
            o = prod + _w(weights, sig, "b_o")
            out[sel[m]] = Z[all_rows[sel][m]] + mod[s, sig, 2] * o
    return out


def mlp(Z1: np.ndarray, row_ids: np.ndarray, cu: np.ndarray, text_len: int, weights,
        mod: np.ndarray, fp8=None) -> np.ndarray:
    """MLP half of the block: z2 = z1 + gate2 * (GELU_tanh(h2 W1^T + b1) W2^T + b2) with
    h2 = LN(z1) * (1 + scale2) + shift2.  Z1 holds the rows `row_ids` of the packed sequence (their
    sample and stream follow from cu_seqlens).  Returns float64 [len(row_ids)][D].  With `fp8`
    (per stream {"w1": (codes, scale), "w2": ...}) both projections multiply FP8 rows of their input
    by FP8 rows of the weight: h2 and the GELU output are quantised from their computed values."""
    out = np.empty_like(Z1, dtype=np.float64)
    row_ids = np.asarray(row_ids)
    for (s, sig, a, b) in _segments(cu, text_len):
        m = (row_ids >= a) & (row_ids < b)
        if not m.any():
            continue
        z = Z1[m]
        h2 = layer_norm(z) * (1.0 + mod[s, sig, 4]) + mod[s, sig, 3]
        prod = _fp8_matmul(h2, fp8[sig]["w1"]) if fp8 is not None else h2 @ _w(weights, sig, "w1").T
        u = prod + _w(weights, sig, "b1")
        g = gelu_tanh(u)
        prod = _fp8_matmul(g, fp8[sig]["w2"]) if fp8 is not None else g @ _w(weights, sig, "w2").T
        o = prod + _w(weights, sig, "b2")
        out[m] = z + mod[s, sig, 5] * o
    return out


def block(Z: np.ndarray, cu: np.ndarray, text_len: int, heads: int, weights, mod: np.ndarray,
          rows: Optional[np.ndarray] = None, fp8=None) -> Tuple[np.ndarray, np.ndarray]:
    """Whole block on the packed sequence: returns (z1, z2) for `rows` (all rows when None).
    `fp8`: per stream {name: (codes, scale)} for name in w_qkv, w_o, w1, w2: all four projections on
    FP8 operands (quantize_fp8_weights)."""
    rows = np.arange(Z.shape[0]) if rows is None else np.asarray(rows)
    z1 = attention(Z, cu, text_len, heads, weights, mod, rows, fp8)
    z2 = mlp(z1, rows, cu, text_len, weights, mod, fp8)
    return z1, z2


FP8_WEIGHTS = ("w_qkv", "w_o", "w1", "w2")


def quantize_fp8_weights(weights) -> List[Dict[str, Tuple[np.ndarray, np.ndarray]]]:
    """Per stream, the FP8 rows (per output channel) of the four projection weights."""
    return [{name: quantize_rows(np.asarray(w[name], dtype=np.float32)) for name in FP8_WEIGHTS}
            for w in weights]


# ------------------------------------------------------------------------------------------------
# end to end
# ------------------------------------------------------------------------------------------------

def select(E, force, grid_h, grid_w, r, mode: str, tau=None, keep=None) -> np.ndarray:
    if mode == "threshold":
        return select_threshold(E, force, grid_h, grid_w, r, tau)
    if mode == "topk":
        return select_topk(E, force, grid_h, grid_w, r, keep)
    raise ValueError(mode)


def pipeline(x_img, x_txt, shape, force, r: int, mode: str, tau=None, keep=None, weights=None,
             mod=None, rows: Optional[np.ndarray] = None, with_block: bool = True,
             tokens: str = "partition", delta: bool = False, fp8: bool = False) -> Dict[str, np.ndarray]:
    """All six steps on one batch.  `shape` needs grid_h, grid_w, batch, images, text_len, heads.
    With `rows` the block is evaluated only for those packed rows (z1, z2 and y are then partial:
    y_img / y_txt are not formed).  `tokens` picks the token set (compact), `delta` the delta form
    of the reassembly (decompress)."""
    H, W = shape.grid_h, shape.grid_w
    E = score(x_img, H, W)
    fine = select(E, force, H, W, r, mode, tau, keep)
    idx_map, fine_idx, pool_idx, counts = compact(fine, H, W, tokens)
    cu, seg = layout(counts, shape.batch, shape.images, shape.text_len)
    Z = compress(x_img, x_txt, H, W, fine_idx, pool_idx, counts, cu, seg, shape.text_len)
    res = dict(E=E, fine=fine, idx_map=idx_map, fine_idx=fine_idx, pool_idx=pool_idx, counts=counts,
               cu=cu, seg=seg, Z=Z)
    if with_block:
        z1, z2 = block(Z, cu, shape.text_len, shape.heads, weights, mod, rows,
                       quantize_fp8_weights(weights) if fp8 else None)
        res.update(z1=z1, z2=z2)
        if rows is None:
            y_img, y_txt = decompress(z2, idx_map, cu, seg, shape.text_len, shape.batch,
                                      x_img if delta else None, Z if delta else None)
            res.update(y_img=y_img, y_txt=y_txt)
    return res


def stack(Z: np.ndarray, cu: np.ndarray, text_len: int, heads: int, weights_per_block, mods) -> np.ndarray:
    """Blocks in order on the packed sequence, each one's output the next one's input (the DiT of
    the paper is a stack of such blocks run on the compressed tokens, Sec. 2.2 / Sec. 3.3)."""
    z = Z
    for weights, mod in zip(weights_per_block, mods):
        _, z = block(z, cu, text_len, heads, weights, mod)
    return z


def request(x_steps, x_txt, shape, force, r: int, mode: str, weights_per_block, mods, tau=None,
            keep=None) -> Dict[str, object]:
    """One editing request: the selection runs once, on step 0's latents (Sec. 2.3: it costs a few
    milliseconds per request), then every sampling step (Sec. 3.3: 8 steps) compresses its own
    latents with that selection, runs the block stack and decompresses.  mods[t][l] is block l's
    modulation at step t.  Returns the selection and per step the packed input Z and the outputs."""
    H, W = shape.grid_h, shape.grid_w
    E = score(x_steps[0], H, W)
    fine = select(E, force, H, W, r, mode, tau, keep)
    idx_map, fine_idx, pool_idx, counts = compact(fine, H, W)
    cu, seg = layout(counts, shape.batch, shape.images, shape.text_len)
    out = dict(E=E, fine=fine, idx_map=idx_map, fine_idx=fine_idx, pool_idx=pool_idx, counts=counts, cu=cu,
               seg=seg, Z=[], z=[], y_img=[], y_txt=[])
    for t, x in enumerate(x_steps):
        Z = compress(x, x_txt, H, W, fine_idx, pool_idx, counts, cu, seg, shape.text_len)
        z = stack(Z, cu, shape.text_len, shape.heads, weights_per_block, mods[t])
        y_img, y_txt = decompress(z, idx_map, cu, seg, shape.text_len, shape.batch)
        out["Z"].append(Z)
        out["z"].append(z)
        out["y_img"].append(y_img)
        out["y_txt"].append(y_txt)
    return out


def dense_sequence(x_img, x_txt, batch: int, images: int, text_len: int):
    """Uncompressed sequence of the same batch: [grid 0 raster ; grid 1 raster ; text] per sample."""
    G, N, D = x_img.shape
    rows = []
    cu = np.zeros(batch + 1, dtype=np.int32)
    for s in range(batch):
        for i in range(images):
            rows.append(x_img[s * images + i].astype(np.float64))
        rows.append(x_txt[s].astype(np.float64))
        cu[s + 1] = cu[s] + images * N + text_len
    return np.concatenate(rows, axis=0), cu
