// Projections of the block (QKV, attention output, MLP up and down): C = A W^T on the ragged
// packed sequence, image rows with the image-stream weights and text rows with the text-stream
// weights, tiles never straddling a segment.  Epilogues fuse the bias, the tanh-GELU, and the
// gated residual update of the float32 stream z.
//
// bf16 path: gfx950 MFMA v_mfma_f32_16x16x32_bf16, fp32 accumulation.  A workgroup of WM x WN
// waves owns a BM x BN output tile; K advances in steps of 64 through a double-buffered LDS tile
// (one barrier per step) while the next step's global loads are in flight.  LDS rows are 128 B
// (64 bf16); the 16-byte chunk c of row r is stored at chunk c ^ ((r >> 1) & 7) so that the 16
// lanes of an MFMA operand read (16 consecutive rows, same chunk) hit 16 distinct bank groups.
//
// The MFMA is issued with the weight fragment as its first operand, so each lane's 4
// accumulators are 4 consecutive output columns of one row (contiguous epilogue stores).
#include "common.h"
#include "kernels.h"

namespace hilo {

HILO_DEV float gelu_tanh(float u) {
  const float k0 = 0.7978845608028654f;  // sqrt(2 / pi)
  const float inner = k0 * (u + 0.044715f * u * u * u);
  return 0.5f * u * (1.0f + tanhf(inner));
}

// Row range of row-tile t: tiles of sample s are [image tiles][text tiles].
struct TileRows {
  int s, sigma, row0, nrows;
};

HILO_DEV TileRows tile_rows(const int *cu, int L, int imgTiles, int txtTiles, int BM, int t) {
  TileRows tr;
  const int per = imgTiles + txtTiles;
  tr.s = t / per;
  const int lt = t % per;
  const int lo = cu[tr.s], hi = cu[tr.s + 1];
  const int tstart = hi - L;
  if (lt < imgTiles) {
    tr.sigma = 0;
    tr.row0 = lo + lt * BM;
    tr.nrows = min(BM, tstart - tr.row0);
  } else {
    tr.sigma = 1;
    tr.row0 = tstart + (lt - imgTiles) * BM;
    tr.nrows = min(BM, hi - tr.row0);
  }
  return tr;
}

template <int EPI, bool BF16OUT>
HILO_DEV void epilogue4(const GemmProblem &p, const TileRows &tr, int m, int n, const float *acc) {
  // m: output row, n: first of 4 consecutive columns (n + 3 < N guaranteed by N % 4 == 0)
  float b[4];
  if (BF16OUT) {
    const uint2 bu = *reinterpret_cast<const uint2 *>(
        reinterpret_cast<const uint16_t *>(p.bias[tr.sigma]) + n);
    b[0] = __uint_as_float(bu.x << 16); b[1] = __uint_as_float(bu.x & 0xffff0000u);
    b[2] = __uint_as_float(bu.y << 16); b[3] = __uint_as_float(bu.y & 0xffff0000u);
  } else {
    const float4 bf = *reinterpret_cast<const float4 *>(reinterpret_cast<const float *>(p.bias[tr.sigma]) + n);
    b[0] = bf.x; b[1] = bf.y; b[2] = bf.z; b[3] = bf.w;
  }
  float v[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) v[e] = acc[e] + b[e];
  if constexpr (EPI == EPI_RESID) {
    const float4 gt = *reinterpret_cast<const float4 *>(
        p.mod + (size_t(tr.s * 2 + tr.sigma) * 6 + p.gate_idx) * p.D + n);
    float4 *zp = reinterpret_cast<float4 *>(p.z + size_t(m) * p.ldz + n);
    float4 zv = *zp;
    zv.x += gt.x * v[0];
    zv.y += gt.y * v[1];
    zv.z += gt.z * v[2];
    zv.w += gt.w * v[3];
    *zp = zv;
  } else {
    if constexpr (EPI == EPI_GELU) {
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = gelu_tanh(v[e]);
    }
    if (BF16OUT) {
      uint2 u;
      u.x = pack_bf16x2(v[0], v[1]);
      u.y = pack_bf16x2(v[2], v[3]);
      *reinterpret_cast<uint2 *>(reinterpret_cast<uint16_t *>(p.out) + size_t(m) * p.ldo + n) = u;
    } else {
      *reinterpret_cast<float4 *>(reinterpret_cast<float *>(p.out) + size_t(m) * p.ldo + n) =
          make_float4(v[0], v[1], v[2], v[3]);
    }
  }
}

// ------------------------------------------------------------------------------- bf16 MFMA

template <int BM, int BN, int WM, int WN, int EPI>
__global__ __launch_bounds__(WM *WN * 64) void k_gemm_bf16(GemmProblem p, int imgTiles,
                                                           int txtTiles, int tilesN) {
  constexpr int NT = WM * WN * 64;
  constexpr int BK = 64;
  constexpr int TM = BM / WM / 16;
  constexpr int TN = BN / WN / 16;
  constexpr int CA = BM * 8 / NT;  // 16-byte chunks per thread per A tile
  constexpr int CB = BN * 8 / NT;
  static_assert(CA * NT == BM * 8 && CB * NT == BN * 8, "tile/threads mismatch");
  __shared__ __attribute__((aligned(16))) uint16_t sA[2][BM * BK];
  __shared__ __attribute__((aligned(16))) uint16_t sB[2][BN * BK];

  const int bid = xcd_remap(blockIdx.x, gridDim.x);
  const int tn = bid % tilesN;
  const TileRows tr = tile_rows(p.cu, p.L, imgTiles, txtTiles, BM, bid / tilesN);
  if (tr.nrows <= 0) return;
  const int n0 = tn * BN;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int wm = wid / WN, wn = wid % WN;
  const uint16_t *A = reinterpret_cast<const uint16_t *>(p.A);
  const uint16_t *Wt = reinterpret_cast<const uint16_t *>(p.W[tr.sigma]);
  const int K = p.K;

  // global source offsets (elements) of this thread's chunks; rows/cols past the tile edge are
  // clamped to the last valid one (their results are never stored)
  size_t offA[CA], offB[CB];
  int ldsA[CA], ldsB[CB];
#pragma unroll
  for (int c = 0; c < CA; ++c) {
    const int idx = tid + c * NT, r = idx >> 3, ch = idx & 7;
    offA[c] = size_t(tr.row0 + min(r, tr.nrows - 1)) * p.lda + ch * 8;
    ldsA[c] = r * BK + ((ch ^ ((r >> 1) & 7)) * 8);
  }
#pragma unroll
  for (int c = 0; c < CB; ++c) {
    const int idx = tid + c * NT, r = idx >> 3, ch = idx & 7;
    offB[c] = size_t(min(n0 + r, p.N - 1)) * K + ch * 8;
    ldsB[c] = r * BK + ((ch ^ ((r >> 1) & 7)) * 8);
  }

  uint4 ra[CA], rb[CB];
  auto gload = [&](int k0) {
#pragma unroll
    for (int c = 0; c < CA; ++c) ra[c] = *reinterpret_cast<const uint4 *>(A + offA[c] + k0);
#pragma unroll
    for (int c = 0; c < CB; ++c) rb[c] = *reinterpret_cast<const uint4 *>(Wt + offB[c] + k0);
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int c = 0; c < CA; ++c) *reinterpret_cast<uint4 *>(&sA[buf][ldsA[c]]) = ra[c];
#pragma unroll
    for (int c = 0; c < CB; ++c) *reinterpret_cast<uint4 *>(&sB[buf][ldsB[c]]) = rb[c];
  };

  f32x4 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int wrow = wm * (BM / WM), wcol = wn * (BN / WN);
  const int lr = lane & 15, lg = lane >> 4;

  const int nk = K / BK;
  gload(0);
  sstore(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) gload((kt + 1) * BK);
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const int ch = ks * 4 + lg;
      bf16x8 fa[TM], fb[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int r = wrow + i * 16 + lr;
        fa[i] = *reinterpret_cast<const bf16x8 *>(&sA[buf][r * BK + ((ch ^ ((r >> 1) & 7)) * 8)]);
      }
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int r = wcol + j * 16 + lr;
        fb[j] = *reinterpret_cast<const bf16x8 *>(&sB[buf][r * BK + ((ch ^ ((r >> 1) & 7)) * 8)]);
      }
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fb[j], fa[i], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) sstore(buf ^ 1);
    __syncthreads();
  }

  // acc[i][j][e]: row wrow + i*16 + lr, column wcol + j*16 + 4*lg + e
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int rl = wrow + i * 16 + lr;
    if (rl >= tr.nrows) continue;
    const int m = tr.row0 + rl;
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int n = n0 + wcol + j * 16 + 4 * lg;
      if (n >= p.N) continue;
      float a4[4] = {acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]};
      epilogue4<EPI, true>(p, tr, m, n, a4);
    }
  }
}

// ------------------------------------------------------------------------------- fp32 path

// Plain LDS-tiled fp32 FMA kernel for the float32 problem sizes: 64 x 64 tile, 256 threads, 4 x 4
// outputs per thread.
template <int EPI>
__global__ __launch_bounds__(256) void k_gemm_f32(GemmProblem p, int imgTiles, int txtTiles,
                                                  int tilesN) {
  constexpr int BM = 64, BN = 64, BK = 16;
  __shared__ float sA[BK][BM + 4];
  __shared__ float sB[BK][BN + 4];
  const int bid = blockIdx.x;
  const int tn = bid % tilesN;
  const TileRows tr = tile_rows(p.cu, p.L, imgTiles, txtTiles, BM, bid / tilesN);
  if (tr.nrows <= 0) return;
  const int n0 = tn * BN;
  const float *A = reinterpret_cast<const float *>(p.A);
  const float *Wt = reinterpret_cast<const float *>(p.W[tr.sigma]);
  const int tid = threadIdx.x;
  const int tx = tid % 16, ty = tid / 16;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < p.K; k0 += BK) {
    for (int e = tid; e < BM * BK; e += 256) {
      const int r = e / BK, k = e % BK;
      sA[k][r] = A[size_t(tr.row0 + min(r, tr.nrows - 1)) * p.lda + k0 + k];
      sB[k][r] = Wt[size_t(min(n0 + r, p.N - 1)) * p.K + k0 + k];
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < BK; ++k) {
      float a[4], b[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) { a[u] = sA[k][ty * 4 + u]; b[u] = sB[k][tx * 4 + u]; }
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int v = 0; v < 4; ++v) acc[u][v] += a[u] * b[v];
    }
    __syncthreads();
  }
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int rl = ty * 4 + u;
    if (rl >= tr.nrows) continue;
    const int n = n0 + tx * 4;
    if (n >= p.N) continue;
    epilogue4<EPI, false>(p, tr, tr.row0 + rl, n, acc[u]);
  }
}

// ------------------------------------------------------------------------------- dispatch

template <int BM, int BN, int WM, int WN, int EPI>
static hipError_t run_bf16(const GemmProblem &p, hipStream_t st) {
  const int imgTiles = (p.max_img_rows + BM - 1) / BM;
  const int txtTiles = (p.L + BM - 1) / BM;
  const int tilesN = (p.N + BN - 1) / BN;
  const long long nblk = (long long)p.B * (imgTiles + txtTiles) * tilesN;
  if (nblk <= 0) return hipSuccess;
  hipLaunchKernelGGL((k_gemm_bf16<BM, BN, WM, WN, EPI>), dim3(unsigned(nblk)), dim3(WM * WN * 64),
                     0, st, p, imgTiles, txtTiles, tilesN);
  return hipGetLastError();
}

template <int EPI>
static hipError_t run_f32(const GemmProblem &p, hipStream_t st) {
  const int imgTiles = (p.max_img_rows + 63) / 64;
  const int txtTiles = (p.L + 63) / 64;
  const int tilesN = (p.N + 63) / 64;
  const long long nblk = (long long)p.B * (imgTiles + txtTiles) * tilesN;
  if (nblk <= 0) return hipSuccess;
  hipLaunchKernelGGL((k_gemm_f32<EPI>), dim3(unsigned(nblk)), dim3(256), 0, st, p, imgTiles,
                     txtTiles, tilesN);
  return hipGetLastError();
}

hipError_t launch_gemm(bool bf16, int epi, const GemmProblem &p, hipStream_t st) {
  if (!bf16) {
    switch (epi) {
      case EPI_BIAS: return run_f32<EPI_BIAS>(p, st);
      case EPI_GELU: return run_f32<EPI_GELU>(p, st);
      default: return run_f32<EPI_RESID>(p, st);
    }
  }
  // wide outputs (QKV, MLP up): 256 x 256 tiles; narrow outputs (D columns): 128 x 128 tiles
  switch (epi) {
    case EPI_BIAS: return run_bf16<256, 256, 2, 2, EPI_BIAS>(p, st);
    case EPI_GELU: return run_bf16<256, 256, 2, 2, EPI_GELU>(p, st);
    default: return run_bf16<128, 128, 2, 2, EPI_RESID>(p, st);
  }
}

}  // namespace hilo
