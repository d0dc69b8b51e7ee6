// Projections of the block (QKV, attention output, MLP up and down): C = A W^T on the ragged
// packed sequence, image rows with the image-stream weights and text rows with the text-stream
// weights, tiles never straddling a segment.  Epilogues fuse the bias, the tanh-GELU, and the
// gated residual update of the float32 stream z.
//
// bf16 path: gfx950 MFMA v_mfma_f32_16x16x32_bf16, fp32 accumulation in VGPRs; 256 x 256 tiles
// on 8 waves, K steps of 64 through a double-buffered LDS ring filled by direct global->LDS loads,
// scheduled stream-K over one persistent workgroup per CU.
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

// LDS rows hold BK bf16 = BK/8 chunks of 16 bytes; chunk c of row r lives at slot c ^ swz(r).
// An MFMA operand read touches one chunk of 16 consecutive rows: swz makes those 16 reads land
// in 16 distinct 16-byte bank groups of a 256-byte bank window (64 banks), and any 8 consecutive
// rows in 8 distinct groups of a 128-byte window (32 banks).
template <int BK>
HILO_DEV int swz(int r) {
  if constexpr (BK == 64) return (r & 7) ^ ((r >> 3) & 1);
  else return ((r >> 1) & 3) ^ ((r >> 3) & 1);
}

// One 16-byte global load per lane straight into LDS: lane l of the wave lands at byte 16*l of
// the wave's 1 KiB destination (the destination base is uniform, held in M0).
HILO_DEV void g2lds16(const void *g, void *lds_wave_base) {
  __builtin_amdgcn_global_load_lds(g, (__attribute__((address_space(3))) void *)lds_wave_base, 16, 0, 0);
}

template <int N>
HILO_DEV void wait_vmem_le() { asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory"); }

// Active row tiles of the ragged problem: per sample, ceil(image rows / BM) image tiles then
// ceil(L / BM) text tiles.  Only the device knows the row counts, so every workgroup walks the
// (few) segments itself.
HILO_DEV int row_tiles_total(const GemmProblem &p, int BM) {
  int R = 0;
  for (int s = 0; s < p.B; ++s) {
    const int nimg = p.cu[s + 1] - p.L - p.cu[s];
    R += (nimg + BM - 1) / BM + (p.L + BM - 1) / BM;
  }
  return R;
}

HILO_DEV TileRows decode_row_tile(const GemmProblem &p, int BM, int r) {
  TileRows tr{0, 0, 0, 0};
  for (int s = 0; s < p.B; ++s) {
    const int lo = p.cu[s], hi = p.cu[s + 1], ts = hi - p.L;
    const int ti = (ts - lo + BM - 1) / BM, tt = (p.L + BM - 1) / BM;
    if (r < ti) {
      tr = TileRows{s, 0, lo + r * BM, min(BM, ts - (lo + r * BM))};
      break;
    }
    r -= ti;
    if (r < tt) {
      tr = TileRows{s, 1, ts + r * BM, min(BM, hi - (ts + r * BM))};
      break;
    }
    r -= tt;
  }
  return tr;
}

// Stream-K schedule.  The iteration space is (tile, K step) with tiles ordered row-tile fastest
// (tile t = tn * R + r); the P persistent workgroups take equal contiguous ranges of it, so the
// load is balanced whatever the ragged tile count.  A tile fully inside one range is finished
// there; a tile cut by range boundaries leaves fp32 partial sums (at most two per workgroup: the
// first and the last tile of its range) that k_gemm_fix adds up in workgroup order and finishes
// with the same epilogue -- deterministic, and no workgroup ever waits for another.
struct SkRange {
  long long beg, end;
};

HILO_DEV SkRange sk_range(long long I, int P, int pid) {
  return SkRange{I * pid / P, I * (pid + 1) / P};
}

// WM x WN waves, wave tile (BM/WM) x (BN/WN), K step 64 through a double-buffered LDS ring filled
// by direct global->LDS loads one step ahead, one barrier per step.
template <int BM, int BN, int WM, int WN>
struct SkTile {
  static constexpr int NW = WM * WN;
  static constexpr int BK = 64;
  static constexpr int RPI = 8;              // rows per wave load instruction (1 KiB)
  static constexpr int TM = BM / WM / 16;
  static constexpr int TN = BN / WN / 16;
  static constexpr int IA = BM / RPI / NW;   // load instructions per wave per step
  static constexpr int IB = BN / RPI / NW;
  static_assert(IA * RPI * NW == BM && IB * RPI * NW == BN, "tile / wave mismatch");
  static constexpr size_t kPartFloats = size_t(BM) * BN;

  // partial-sum slot layout: register order, one float4 per lane per (wave, i, j)
  HILO_DEV static size_t part_index(int wid, int i, int j, int lane) {
    return ((size_t(wid) * TM * TN + i * TN + j) * 64 + lane) * 4;
  }

  template <int EPI>
  HILO_DEV static void epilogue(const GemmProblem &p, const TileRows &tr, int n0, int wid, int lane,
                                f32x4 (&acc)[TM][TN]) {
    const int wrow = (wid / WN) * (BM / WM), wcol = (wid % WN) * (BN / WN);
    const int lr = lane & 15, lg = lane >> 4;
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
};

template <int BM, int BN, int WM, int WN, int EPI>
__global__ __launch_bounds__(WM *WN * 64) void k_gemm_sk(GemmProblem p) {
  using T = SkTile<BM, BN, WM, WN>;
  constexpr int BK = T::BK, TM = T::TM, TN = T::TN, IA = T::IA, IB = T::IB, NW = T::NW;
  __shared__ __attribute__((aligned(1024))) uint16_t sA[2][BM * BK];
  __shared__ __attribute__((aligned(1024))) uint16_t sB[2][BN * BK];

  // logical workgroup index: each XCD gets a contiguous band of the iteration space (a narrow
  // band of weight columns for all rows), so its L2 serves the weight tiles to all of its CUs
  const int P = gridDim.x;
  const int pid = xcd_remap(blockIdx.x, P);
  const int R = row_tiles_total(p, BM);
  const int tilesN = (p.N + BN - 1) / BN;
  const int nk = p.K / BK;
  const long long I = (long long)R * tilesN * nk;
  const SkRange rg = sk_range(I, P, pid);
  if (rg.beg >= rg.end) return;
  const long long head = rg.beg / nk;

  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int wrow = (wid / WN) * (BM / WM), wcol = (wid % WN) * (BN / WN);
  const int lr = lane & 15, lg = lane >> 4;
  const int lrow = lane >> 3, lslot = lane & 7;
  const uint16_t *A = reinterpret_cast<const uint16_t *>(p.A);

  for (long long it = rg.beg; it < rg.end;) {
    const long long t = it / nk;
    const int kb = int(it - t * nk);
    const int ke = int(min((long long)nk, (long long)kb + (rg.end - it)));
    const int tn = int(t / R);
    const TileRows tr = decode_row_tile(p, BM, int(t % R));
    const int n0 = tn * BN;
    const uint16_t *Wt = reinterpret_cast<const uint16_t *>(p.W[tr.sigma]);

    // this lane's load sources: row (wave band + 8 i + lane / 8), chunk (lane % 8) ^ swz(row);
    // rows past the tile edge re-read the last valid row (their results are never stored)
    const uint16_t *srcA[IA];
    const uint16_t *srcB[IB];
#pragma unroll
    for (int i = 0; i < IA; ++i) {
      const int r = wid * (BM / NW) + 8 * i + lrow;
      srcA[i] = A + size_t(tr.row0 + min(r, tr.nrows - 1)) * p.lda + ((lslot ^ swz<BK>(r)) * 8);
    }
#pragma unroll
    for (int i = 0; i < IB; ++i) {
      const int r = wid * (BN / NW) + 8 * i + lrow;
      srcB[i] = Wt + size_t(min(n0 + r, p.N - 1)) * p.K + ((lslot ^ swz<BK>(r)) * 8);
    }
    auto issue = [&](int k0, int buf) {
#pragma unroll
      for (int i = 0; i < IA; ++i) g2lds16(srcA[i] + k0, &sA[buf][(wid * (BM / NW) + 8 * i) * BK]);
#pragma unroll
      for (int i = 0; i < IB; ++i) g2lds16(srcB[i] + k0, &sB[buf][(wid * (BN / NW) + 8 * i) * BK]);
    };

    f32x4 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    issue(kb * BK, 0);
    for (int kt = kb; kt < ke; ++kt) {
      const int buf = (kt - kb) & 1;
      wait_vmem_le<0>();
      __syncthreads();
      if (kt + 1 < ke) issue((kt + 1) * BK, buf ^ 1);
#pragma unroll
      for (int ks = 0; ks < BK / 32; ++ks) {
        const int ch = ks * 4 + lg;
        bf16x8 fa[TM], fb[TN];
#pragma unroll
        for (int i = 0; i < TM; ++i) {
          const int r = wrow + i * 16 + lr;
          fa[i] = *reinterpret_cast<const bf16x8 *>(&sA[buf][r * BK + ((ch ^ swz<BK>(r)) * 8)]);
        }
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const int r = wcol + j * 16 + lr;
          fb[j] = *reinterpret_cast<const bf16x8 *>(&sB[buf][r * BK + ((ch ^ swz<BK>(r)) * 8)]);
        }
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fb[j], fa[i], acc[i][j], 0, 0, 0);
        __builtin_amdgcn_iglp_opt(1);  // interleave the next step's LDS reads with the MFMAs
      }
    }

    if (kb == 0 && ke == nk) {
      T::template epilogue<EPI>(p, tr, n0, wid, lane, acc);
    } else {
      float *slot = p.part + (size_t(pid) * 2 + (t == head ? 0 : 1)) * T::kPartFloats;
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          *reinterpret_cast<f32x4 *>(slot + T::part_index(wid, i, j, lane)) = acc[i][j];
    }
    it += ke - kb;
    __syncthreads();  // the next tile's loads reuse the LDS ring
  }
}

// Finishes every tile cut by range boundaries: the workgroup whose range holds the tile's first
// K step sums the partials of all contributors in workgroup order, then runs the epilogue.
template <int BM, int BN, int WM, int WN, int EPI>
__global__ __launch_bounds__(WM *WN * 64) void k_gemm_fix(GemmProblem p) {
  using T = SkTile<BM, BN, WM, WN>;
  constexpr int BK = T::BK, TM = T::TM, TN = T::TN;
  const int P = gridDim.x;
  const int pid = blockIdx.x;
  const int R = row_tiles_total(p, BM);
  const int tilesN = (p.N + BN - 1) / BN;
  const int nk = p.K / BK;
  const long long I = (long long)R * tilesN * nk;
  const SkRange rg = sk_range(I, P, pid);
  if (rg.beg >= rg.end) return;
  const long long tl = (rg.end - 1) / nk;            // last tile touched by this range
  if (rg.end >= (tl + 1) * nk) return;                // it ends inside this range: not cut here
  if (rg.beg > tl * nk) return;                       // this range does not hold its first step
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;

  f32x4 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int q = pid; q < P; ++q) {
    const SkRange rq = sk_range(I, P, q);
    if (rq.beg >= rq.end) continue;
    if (rq.beg >= (tl + 1) * nk) break;
    const float *slot = p.part + (size_t(q) * 2 + (rq.beg / nk == tl ? 0 : 1)) * T::kPartFloats;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
        acc[i][j] += *reinterpret_cast<const f32x4 *>(slot + T::part_index(wid, i, j, lane));
    if (rq.end >= (tl + 1) * nk) break;
  }
  const TileRows tr = decode_row_tile(p, BM, int(tl % R));
  T::template epilogue<EPI>(p, tr, int(tl / R) * BN, wid, lane, acc);
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

int sk_workgroups() {
  static int ncu[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) dev = 0;
  if (ncu[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
      n = kSkMaxWorkgroups;
    ncu[dev] = n;
  }
  return ncu[dev] < kSkMaxWorkgroups ? ncu[dev] : kSkMaxWorkgroups;
}

template <int BM, int BN, int WM, int WN, int EPI>
static hipError_t run_bf16(const GemmProblem &p, hipStream_t st) {
  static_assert(size_t(BM) * BN <= kSkPartFloats, "partial slot too small");
  const int P = sk_workgroups();
  hipLaunchKernelGGL((k_gemm_sk<BM, BN, WM, WN, EPI>), dim3(P), dim3(WM * WN * 64), 0, st, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((k_gemm_fix<BM, BN, WM, WN, EPI>), dim3(P), dim3(WM * WN * 64), 0, st, p);
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
  switch (epi) {
    case EPI_BIAS: return run_bf16<256, 256, 2, 4, EPI_BIAS>(p, st);
    case EPI_GELU: return run_bf16<256, 256, 2, 4, EPI_GELU>(p, st);
    default: return run_bf16<256, 256, 2, 4, EPI_RESID>(p, st);
  }
}

}  // namespace hilo
