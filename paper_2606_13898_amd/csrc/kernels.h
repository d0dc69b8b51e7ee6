// Internal launchers of libhilo (host side).  Every launcher enqueues on `st` and returns the
// launch status; argument validation happens in the C ABI layer before any of these is called.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace hilo {

constexpr int kSelMaxGrids = 64;  // grids per select launch (per-grid parameters ride in kernel args)

hipError_t launch_score(bool bf16, const void *x, long long *E, int G, int H, int W, int D,
                        hipStream_t st);
// rgb [G][3][16 H][16 W] float32 -> E [G][H * W]: per-token pixel-space Sobel energy
hipError_t launch_score_pixels(const float *rgb, long long *E, int G, int H, int W, hipStream_t st);
size_t select_lds_bytes(int NB);
// tokens: 0 partition, 1 overlap, 2 drop (see k_select).  With G == 1, cu and seg (both or
// neither) receive the sequence layout as well (L text rows), so launch_layout is not needed.
hipError_t launch_select(const long long *E, const uint8_t *force, int G, int H, int W, int r,
                         int mode, int tokens, const double *tau, const int *keep, int *idx_map,
                         int *fine_idx, int *pool_idx, int *counts, int *cu, int *seg, int L,
                         hipStream_t st);
hipError_t launch_layout(const int *counts, int B, int I, int L, int *cu, int *seg, hipStream_t st);

hipError_t launch_compress(bool bf16, const void *x_img, const void *x_txt, const int *fine_idx,
                           const int *pool_idx, const int *counts, const int *cu, const int *seg,
                           float *z, int B, int I, int H, int W, int D, int L, hipStream_t st);
// S3 fused with the attention half's row norm: z as launch_compress, and out = the normalised,
// modulated rows (bf16 for bf16 inputs, float32 otherwise), as launch_rownorm with set 0; with
// fp8 (bf16 inputs) their E4M3 codes and row scales, as launch_rownorm_fp8.
hipError_t launch_compress_norm(bool bf16, const void *x_img, const void *x_txt, const int *fine_idx,
                                const int *pool_idx, const int *counts, const int *cu, const int *seg,
                                const float *mod, float *z, int B, int I, int H, int W, int D, int L,
                                void *out, hipStream_t st, bool fp8 = false, float *row_scale = nullptr);
hipError_t launch_decompress(bool bf16, const float *z, const int *idx_map, const int *cu,
                             const int *seg, void *y_img, void *y_txt, int B, int I, int N, int D,
                             int L, hipStream_t st);
hipError_t launch_decompress_delta(bool bf16, const float *z, const void *x_img, const int *idx_map,
                                   const int *counts, const int *cu, const int *seg, void *y_img,
                                   void *y_txt, int B, int I, int H, int W, int D, int L, hipStream_t st);
// h = LN(z) * (1 + mod[s][stream][which*3 + 1]) + mod[s][stream][which*3], rows < cu[B]
hipError_t launch_rownorm(bool bf16, const float *z, const int *cu, const float *mod, int B, int L,
                          int D, int Tmax, int which, void *out, hipStream_t st);
// the same rows as FP8 E4M3 codes [Tmax][D] plus a float32 scale per row (D % 4 == 0)
hipError_t launch_rownorm_fp8(const float *z, const int *cu, const float *mod, int B, int L, int D,
                              int Tmax, int which, uint8_t *codes, float *row_scale, hipStream_t st);
// per-row FP8 E4M3 codes and scales of x [rows][cols] (cols % 4 == 0); with row_limit (device
// pointer), only rows below *row_limit
hipError_t launch_quantize_rows(bool bf16, const void *x, int rows, int cols, uint8_t *codes, float *scale,
                                hipStream_t st, const int *row_limit = nullptr);

enum Epilogue { EPI_BIAS = 0, EPI_GELU = 1, EPI_RESID = 2 };
// The four projections of the block; each gets its own kernel instantiation (so profiles and
// counters tell them apart) with the epilogue it needs.
enum GemmRole { GEMM_QKV = 0, GEMM_O = 1, GEMM_FC1 = 2, GEMM_FC2 = 3 };
constexpr int role_epilogue(int role) {
  return role == GEMM_QKV ? EPI_BIAS : role == GEMM_FC1 ? EPI_GELU : EPI_RESID;
}

// Segment-aware C = A W_sigma^T with the epilogue; rows of sample s split into the image segment
// (stream 0) and the text segment (stream 1), tiles never straddle a segment.
struct GemmProblem {
  const void *A;          // [Tmax][K] dtype (row stride lda)
  int lda;
  const void *W[2];       // [N][K] dtype per stream
  const void *bias[2];    // [N] dtype per stream
  int N, K;
  void *out;              // EPI_BIAS / EPI_GELU: [Tmax][ldo] dtype
  int ldo;
  float *z;               // EPI_RESID: z[m][n] += gate * (acc + bias)
  int ldz;
  const float *mod;       // [B][2][6][D]
  int gate_idx, D;
  const int *cu;          // [B+1]
  int B, L, max_img_rows; // max_img_rows = images * N
  float *part;            // bf16 path: partial tiles (kSkPartBytes)
  const float *a_scale;   // FP8 operands: A row m is codes * a_scale[m] ...
  const float *w_scale[2];  // ... and W row n of stream s is codes * w_scale[s][n]
  // FP8 attention scores (the FP8 block's QKV projection, 256 x 256 tiles): when set, the columns
  // below 2 D (q then k) leave as E4M3 codes with one power-of-two scale per (row, head) instead of
  // bf16 -- row m's codes at qk8 + m * ldq8 + column, its E8M0 scale bytes (127 + k) at qk8 + m *
  // ldq8 + 2 D + head (the q heads, then the k heads) -- and only the v columns go to out.
  uint8_t *qk8;
  int ldq8, head_dim;
};

// Partial-sum area of the GEMMs (part of the caller's workspace): one slot per data-parallel unit
// of a split wave plus two per workgroup for its stream-K range, one fp32 256 x 256 tile per slot,
// one workgroup per CU (at most 256).
constexpr int kBigMaxWorkgroups = 256;
constexpr size_t kSkPartBytes = size_t(kBigMaxWorkgroups) * 3 * 256 * 256 * sizeof(float);
hipError_t launch_gemm(bool bf16, int role, const GemmProblem &p, hipStream_t st);
// FP8 E4M3 operands (A [Tmax][K] codes, W[s] [N][K] codes, per-row scales), bf16 bias; the
// epilogue of the role (bf16 output or the float32 residual update); K % 128 == 0, N % 16 == 0.
hipError_t launch_gemm_fp8(int role, const GemmProblem &p, hipStream_t st);

// Stream-K partial results of the bf16 attention core (part of the caller's workspace): two
// slots per workgroup, each the unnormalised output and running max / sum of one query tile.
constexpr int kAttnMaxWorkgroups = 512;
constexpr size_t kAttnSlotFloats = size_t(4) * 2 * 8 * 64 * 4 + size_t(4) * 2 * 64 * 2;
constexpr size_t kAttnPartBytes = size_t(kAttnMaxWorkgroups) * 2 * kAttnSlotFloats * sizeof(float);

// qkv [Tmax][3D] -> out [Tmax][D] (ld = D), per sample and head over cu.  part: kAttnPartBytes of
// device scratch for the bf16 path (unused by the fp32 path).  qk8 (bf16 path only): the score
// product on FP8 q and k, codes and E8M0 scale bytes in rows of ldq8 bytes (GemmProblem::qk8); the
// v columns of qkv stay bf16.
hipError_t launch_attention(bool bf16, const void *qkv, const int *cu, void *out, float *part, int B,
                            int heads, int hd, int max_seq, hipStream_t st, const uint8_t *qk8 = nullptr,
                            int ldq8 = 0);
// Bytes of partial results launch_attention uses on the current device (0 for the fp32 path);
// never more than kAttnPartBytes.
size_t attention_part_bytes(bool bf16, int hd);

}  // namespace hilo
