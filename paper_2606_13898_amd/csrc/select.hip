// S1 score and S2 select kernels (HiLo-Token, Sec. 2.3 "HiLo-Token Selection").
//
// k_score    one read of the latent grid: per patch the Sobel energy of every channel, floored to
//            2^-16 fixed point and summed exactly over channels (bit-reproducible in any order).
// k_select   one workgroup per grid: 2x2 block sums, E_max, dilated forced blocks, threshold or
//            top-k (MSB radix select on the exact 53-bit block sums), then the ordered prefix sums
//            that produce the compressed grid's index map.
// k_layout   row offsets of grids and samples in the packed sequence.
#include "common.h"
#include "kernels.h"

namespace hilo {

// ------------------------------------------------------------------------------------------ S1

// Channels per 16-byte load.
template <bool BF16> struct ScoreVec { static constexpr int V = BF16 ? 8 : 4; };

template <bool BF16>
HILO_DEV void load_vec(const void *base, size_t elem, float *f) {
  if constexpr (BF16) {
    uint4 u = *reinterpret_cast<const uint4 *>(reinterpret_cast<const uint16_t *>(base) + elem);
    unpack8(u, f);
  } else {
    float4 u = *reinterpret_cast<const float4 *>(reinterpret_cast<const float *>(base) + elem);
    f[0] = u.x; f[1] = u.y; f[2] = u.z; f[3] = u.w;
  }
}

// float32 latents: workgroup = one row i of one grid, TJ consecutive patches j0..j0+TJ-1; threads
// split the channels in 16-byte groups and slide a 3x3 window of columns along j.
template <bool BF16, int TJ>
__global__ __launch_bounds__(512) void k_score(const void *__restrict__ x, long long *__restrict__ E,
                                               int H, int W, int D, int tilesJ) {
#pragma clang fp contract(off)
  constexpr int V = ScoreVec<BF16>::V;
  const int CG = D / V;
  const int t = xcd_remap(blockIdx.x, gridDim.x);
  const int jt = t % tilesJ;
  const int gi = t / tilesJ;  // g * H + i
  const int i = gi % H;
  const int g = gi / H;
  const int j0 = jt * TJ;
  const int nj = min(TJ, W - j0);
  const size_t rU = (size_t(g) * H + max(i - 1, 0)) * W;
  const size_t rM = (size_t(g) * H + i) * W;
  const size_t rD = (size_t(g) * H + min(i + 1, H - 1)) * W;

  // Each per-channel term is an integer < 2^38 held exactly in a float; partial sums stay below
  // D * 2^38 <= 2^51, so double accumulation is exact and independent of order.
  double acc[TJ];
#pragma unroll
  for (int k = 0; k < TJ; ++k) acc[k] = 0.0;

  for (int cg = threadIdx.x; cg < CG; cg += blockDim.x) {
    const size_t c0 = size_t(cg) * V;
    // per column: the upper and lower rows (for gy) and the column sum (u + 2 m) + d (for gx),
    // formed once per column and slid along j; gx = sum(right) - sum(left) in the same order
    float Lu[V], Ld[V], Ls[V], Cu[V], Cd[V], Cs[V], Ru[V], Rm[V], Rd[V], Rs[V];
    const int jl = max(j0 - 1, 0);
    load_vec<BF16>(x, (rU + jl) * D + c0, Lu);
    load_vec<BF16>(x, (rM + jl) * D + c0, Rm);
    load_vec<BF16>(x, (rD + jl) * D + c0, Ld);
#pragma unroll
    for (int v = 0; v < V; ++v) Ls[v] = (Lu[v] + 2.0f * Rm[v]) + Ld[v];
    load_vec<BF16>(x, (rU + j0) * D + c0, Cu);
    load_vec<BF16>(x, (rM + j0) * D + c0, Rm);
    load_vec<BF16>(x, (rD + j0) * D + c0, Cd);
#pragma unroll
    for (int v = 0; v < V; ++v) Cs[v] = (Cu[v] + 2.0f * Rm[v]) + Cd[v];
#pragma unroll
    for (int k = 0; k < TJ; ++k) {
      if (k < nj) {
        const int jr = min(j0 + k + 1, W - 1);
        load_vec<BF16>(x, (rU + jr) * D + c0, Ru);
        load_vec<BF16>(x, (rM + jr) * D + c0, Rm);
        load_vec<BF16>(x, (rD + jr) * D + c0, Rd);
        double dpart = 0.0;
#pragma unroll
        for (int v = 0; v < V; ++v) {
          // horizontal: right column minus left column, rows weighted 1, 2, 1
          Rs[v] = (Ru[v] + 2.0f * Rm[v]) + Rd[v];
          float gx = Rs[v] - Ls[v];
          // vertical: lower row minus upper row, columns weighted 1, 2, 1
          float gy = ((Ld[v] + 2.0f * Cd[v]) + Rd[v]) - ((Lu[v] + 2.0f * Cu[v]) + Ru[v]);
          float t1 = gx * gx;
          float t2 = gy * gy;
          float e = t1 + t2;
          float q = floorf(fminf(e, 4194304.0f) * 65536.0f);  // fminf(NaN, cap) = cap
          dpart += double(q);
        }
        acc[k] += dpart;
#pragma unroll
        for (int v = 0; v < V; ++v) {
          Lu[v] = Cu[v]; Ld[v] = Cd[v]; Ls[v] = Cs[v];
          Cu[v] = Ru[v]; Cd[v] = Rd[v]; Cs[v] = Rs[v];
        }
      }
    }
  }

  __shared__ long long red[TJ][8];
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6, nw = blockDim.x >> 6;
#pragma unroll
  for (int k = 0; k < TJ; ++k) {
    long long s = wave_sum_i64(static_cast<long long>(acc[k]));
    if (lane == 0) red[k][wid] = s;
  }
  __syncthreads();
  if (threadIdx.x < nj) {
    long long s = 0;
    for (int w = 0; w < nw; ++w) s += red[threadIdx.x][w];
    E[rM + j0 + threadIdx.x] = s;
  }
}

// bf16 latents: workgroup = one patch row x TJ columns with every channel; a lane takes 4
// channels at a time (8-byte loads) of the 3 rows x (TJ + 2) columns it needs, all loaded before
// any arithmetic, and loops over its channel groups.  Workgroups of at most 256 threads leave
// several resident per CU, so the loads of one overlap the arithmetic of another (the kernel is
// bound by the vector ALU: 3072 channels, 64x64 grid, 15.8 us against 17.8 with 768 threads, one
// workgroup per CU; 128 threads 20.4, 192 17.3).  Per channel a slide along the columns forms the
// vertical sums once per column;
// (u + 2m) is one fma: 2m is exact, so its single rounding equals the two-step sum of the
// definition for every input below 2^127 in magnitude (above, the two-step form overflows to
// infinity first).  The per-output sums over channels meet in LDS (exact in double).
template <int TJ, int NT>
__global__ __launch_bounds__(NT) void k_score_bf16(const uint16_t *__restrict__ x, long long *__restrict__ E,
                                                   int H, int W, int D, int tilesJ) {
#pragma clang fp contract(off)
  const int CG = D / 4;
  const int t = xcd_remap(blockIdx.x, gridDim.x);
  const int jt = t % tilesJ, gi = t / tilesJ, i = gi % H, g = gi / H;
  const int j0 = jt * TJ, nj = min(TJ, W - j0);
  const size_t rU = (size_t(g) * H + max(i - 1, 0)) * W;
  const size_t rM = (size_t(g) * H + i) * W;
  const size_t rD = (size_t(g) * H + min(i + 1, H - 1)) * W;
  double acc[TJ];
#pragma unroll
  for (int k = 0; k < TJ; ++k) acc[k] = 0.0;
  for (int cg = threadIdx.x; cg < CG; cg += NT) {
    const size_t c0 = size_t(cg) * 4;
    uint2 u[TJ + 2], m[TJ + 2], d[TJ + 2];
#pragma unroll
    for (int c = 0; c < TJ + 2; ++c) {
      const int col = min(max(j0 - 1 + c, 0), W - 1);
      u[c] = *reinterpret_cast<const uint2 *>(x + (rU + col) * D + c0);
      m[c] = *reinterpret_cast<const uint2 *>(x + (rM + col) * D + c0);
      d[c] = *reinterpret_cast<const uint2 *>(x + (rD + col) * D + c0);
    }
#pragma unroll
    for (int w = 0; w < 2; ++w) {
#pragma unroll
      for (int hb = 0; hb < 2; ++hb) {
        auto f = [&](const uint2 &v) {
          const uint32_t b = w ? v.y : v.x;
          return __uint_as_float(hb ? (b & 0xffff0000u) : (b << 16));
        };
        float pu = f(u[0]), pd = f(d[0]);
        float cu = f(u[1]), cd = f(d[1]);
        float Vp = __builtin_fmaf(2.0f, f(m[0]), pu) + pd;  // vertical sums of columns j-1, j
        float Vc = __builtin_fmaf(2.0f, f(m[1]), cu) + cd;
#pragma unroll
        for (int k = 0; k < TJ; ++k) {
          const float nu = f(u[k + 2]), nd = f(d[k + 2]);
          const float Vn = __builtin_fmaf(2.0f, f(m[k + 2]), nu) + nd;
          const float gx = Vn - Vp;
          const float gy = (__builtin_fmaf(2.0f, cd, pd) + nd) - (__builtin_fmaf(2.0f, cu, pu) + nu);
          const float t1 = gx * gx;
          const float t2 = gy * gy;
          const float e = t1 + t2;
          acc[k] += double(floorf(fminf(e, 4194304.0f) * 65536.0f));  // fminf(NaN, cap) = cap
          pu = cu; pd = cd; cu = nu; cd = nd;
          Vp = Vc; Vc = Vn;
        }
      }
    }
  }
  __shared__ double red[TJ][NT];
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  constexpr int NW = NT / 64;
#pragma unroll
  for (int k = 0; k < TJ; ++k) red[k][tid] = acc[k];
  __syncthreads();
  for (int k = wid; k < nj; k += NW) {
    double s = 0.0;
#pragma unroll
    for (int w = 0; w < NW; ++w) s += red[k][w * 64 + lane];
    const long long v = wave_sum_i64(static_cast<long long>(s));
    if (lane == 0) E[rM + j0 + k] = v;
  }
}

constexpr int kScoreTJ = 8;

hipError_t launch_score(bool bf16, const void *x, long long *E, int G, int H, int W, int D,
                        hipStream_t st) {
  const int tilesJ = (W + kScoreTJ - 1) / kScoreTJ;
  const long long nblk = (long long)G * H * tilesJ;
  if (nblk <= 0) return hipSuccess;
  if (bf16) {
    const uint16_t *xb = reinterpret_cast<const uint16_t *>(x);
    const int lanes = D / 4;  // D % 64 == 0
#define HILO_SCORE(NTV) \
  hipLaunchKernelGGL((k_score_bf16<kScoreTJ, NTV>), dim3(unsigned(nblk)), dim3(NTV), 0, st, xb, E, H, W, D, tilesJ)
    if (lanes <= 64) HILO_SCORE(64);
    else if (lanes <= 128) HILO_SCORE(128);
    else HILO_SCORE(256);
#undef HILO_SCORE
    return hipGetLastError();
  }
  const int CG = D / 4;
  int threads = ((CG + 63) / 64) * 64;
  if (threads > 512) threads = 512;
  hipLaunchKernelGGL((k_score<false, kScoreTJ>), dim3(unsigned(nblk)), dim3(threads), 0, st, x, E,
                     H, W, D, tilesJ);
  return hipGetLastError();
}

// Pixel-space score (the paper's own selector input, Sec. 2.3): Sobel on each channel of the RGB
// image, with the per-pixel float32 energy, cap and 2^-16 fixed point of k_score, summed exactly
// over the 16 x 16 pixels and 3 channels of a token (the 16x pooling onto the token grid; the
// normalisation by the maximum cancels the 1/256 of a mean).  One workgroup per token: each
// channel's 18 x 18 pixel tile (token plus a one-pixel ring, replicated at the image edge) goes
// through LDS, one thread per pixel.
constexpr int kPixPerTok = 16;

__global__ __launch_bounds__(256) void k_score_pixels(const float *__restrict__ rgb,
                                                      long long *__restrict__ E, int H, int W) {
#pragma clang fp contract(off)
  constexpr int T = kPixPerTok, TT = T + 2;
  __shared__ float tile[TT][TT + 1];
  __shared__ long long red[4];
  const int Hp = H * T, Wp = W * T;
  const int tok = xcd_remap(blockIdx.x, gridDim.x);
  const int g = tok / (H * W), rem = tok - g * (H * W), ti = rem / W, tj = rem - ti * W;
  const int ty = threadIdx.x / T, tx = threadIdx.x % T;
  const int y = ty + 1, x = tx + 1;
  double acc = 0.0;  // integers < 2^38 each, three of them: exact
  for (int c = 0; c < 3; ++c) {
    const float *plane = rgb + (size_t(g) * 3 + c) * size_t(Hp) * Wp;
    for (int e = threadIdx.x; e < TT * TT; e += 256) {
      const int ly = e / TT, lx = e - ly * TT;
      const int py = min(max(ti * T + ly - 1, 0), Hp - 1), px = min(max(tj * T + lx - 1, 0), Wp - 1);
      tile[ly][lx] = plane[size_t(py) * Wp + px];
    }
    __syncthreads();
    const float gx = ((tile[y - 1][x + 1] + 2.0f * tile[y][x + 1]) + tile[y + 1][x + 1]) -
                     ((tile[y - 1][x - 1] + 2.0f * tile[y][x - 1]) + tile[y + 1][x - 1]);
    const float gy = ((tile[y + 1][x - 1] + 2.0f * tile[y + 1][x]) + tile[y + 1][x + 1]) -
                     ((tile[y - 1][x - 1] + 2.0f * tile[y - 1][x]) + tile[y - 1][x + 1]);
    const float t1 = gx * gx;
    const float t2 = gy * gy;
    const float e = t1 + t2;
    acc += double(floorf(fminf(e, 4194304.0f) * 65536.0f));  // fminf(NaN, cap) = cap
    __syncthreads();  // the tile is refilled for the next channel
  }
  const long long s = wave_sum_i64(static_cast<long long>(acc));
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) E[tok] = (red[0] + red[1]) + (red[2] + red[3]);
}

hipError_t launch_score_pixels(const float *rgb, long long *E, int G, int H, int W, hipStream_t st) {
  const long long nblk = (long long)G * H * W;
  if (nblk <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_score_pixels, dim3(unsigned(nblk)), dim3(256), 0, st, rgb, E, H, W);
  return hipGetLastError();
}

// ------------------------------------------------------------------------------------------ S2

constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / 64;

// Exclusive prefix sum over the workgroup in thread order; `total` receives the sum.
HILO_DEV int block_excl_scan(int v, int *tmp, int &total) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  int x = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    int y = __shfl_up(x, off, 64);
    if (lane >= off) x += y;
  }
  if (lane == 63) tmp[wid] = x;
  __syncthreads();
  if (threadIdx.x == 0) {
    int run = 0;
    for (int w = 0; w < kSelWaves; ++w) {
      int t = tmp[w];
      tmp[w] = run;
      run += t;
    }
    tmp[kSelWaves] = run;
  }
  __syncthreads();
  const int excl = tmp[wid] + x - v;
  total = tmp[kSelWaves];
  __syncthreads();
  return excl;
}

HILO_DEV long long block_max_i64(long long v, long long *tmp) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  v = wave_max_i64(v);
  if (lane == 0) tmp[wid] = v;
  __syncthreads();
  long long m = tmp[0];
  for (int w = 1; w < kSelWaves; ++w) m = tmp[w] > m ? tmp[w] : m;
  __syncthreads();
  return m;
}

struct SelChunk {
  double tau[kSelMaxGrids];
  int keep[kSelMaxGrids];
};

// flag bits per block: 1 = fine by score, 2 = forced by the dilated mask
// token set (what the compressed grid holds besides the fine patches of the kept blocks):
// 0 partition -- one pooled token per other block; 1 overlap -- one pooled token per block, kept
// blocks included; 2 drop -- nothing else (patches of other blocks get idx_map -1)
__global__ __launch_bounds__(kSelThreads) void k_select(
    const long long *__restrict__ E, const uint8_t *__restrict__ force, int H, int W, int r,
    int mode, int tokens, SelChunk prm, int g0, int *__restrict__ idx_map, int *__restrict__ fine_idx,
    int *__restrict__ pool_idx, int *__restrict__ counts, int *__restrict__ cu_out,
    int *__restrict__ seg_out, int L) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  const int gl = blockIdx.x;
  const int g = g0 + gl;
  const int N = H * W, NB = N / 4, W2 = W / 2;
  const int tid = threadIdx.x;
  long long *Bs = reinterpret_cast<long long *>(smem);                 // [NB] block sums
  uint8_t *flag = reinterpret_cast<uint8_t *>(Bs + NB);                  // [NB]
  int *itmp = reinterpret_cast<int *>(flag + ((NB + 15) & ~15));         // [kSelWaves + 1]
  int *hist = itmp + 32;                                                 // [256]
  long long *ltmp = reinterpret_cast<long long *>(hist + 256);          // [kSelWaves]
  unsigned long long *lor = reinterpret_cast<unsigned long long *>(ltmp + kSelWaves);  // [1]
  int *bcast = reinterpret_cast<int *>(lor + 1);                        // [4]
  if (tid == 0) *lor = 0;
  const long long *Eg = E + size_t(g) * N;

  // block sums and the grid maximum
  long long mx = 0;
  for (int b = tid; b < NB; b += kSelThreads) {
    const int I = b / W2, J = b % W2;
    const int p = 2 * I * W + 2 * J;
    const long long e00 = Eg[p], e01 = Eg[p + 1], e10 = Eg[p + W], e11 = Eg[p + W + 1];
    Bs[b] = ((e00 + e01) + e10) + e11;
    long long m = e00 > e01 ? e00 : e01;
    long long m2 = e10 > e11 ? e10 : e11;
    m = m > m2 ? m : m2;
    mx = m > mx ? m : mx;
    uint8_t f = 0;
    if (force) {
      const uint8_t *Fg = force + size_t(g) * N;
      const int i0 = max(2 * I - r, 0), i1 = min(2 * I + 1 + r, H - 1);
      const int jj0 = max(2 * J - r, 0), jj1 = min(2 * J + 1 + r, W - 1);
      for (int ii = i0; ii <= i1 && !f; ++ii)
        for (int jj = jj0; jj <= jj1; ++jj)
          if (Fg[ii * W + jj]) { f = 2; break; }
    }
    flag[b] = f;
  }
  // the grid maximum only enters the threshold rule; either way a barrier makes Bs and flag visible
  long long emax = 0;
  if (mode == 0) emax = block_max_i64(mx, ltmp);
  else __syncthreads();

  if (mode == 0) {  // threshold
    if (emax > 0) {
      const double rhs = (4.0 * prm.tau[gl]) * double(emax);
      for (int b = tid; b < NB; b += kSelThreads)
        if (double(Bs[b]) > rhs) flag[b] |= 1;
    }
    __syncthreads();
  } else {  // top-k
    // forced blocks, and the OR of the other blocks' sums: its top byte is where the radix starts
    int nf_local = 0;
    unsigned long long orv = 0;
    for (int b = tid; b < NB; b += kSelThreads) {
      const bool forced = flag[b] & 2;
      nf_local += forced ? 1 : 0;
      if (!forced) orv |= static_cast<unsigned long long>(Bs[b]);
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) orv |= __shfl_xor(orv, off, 64);
    if ((tid & 63) == 0 && orv != 0) atomicOr(lor, orv);
    int nF;
    (void)block_excl_scan(nf_local, itmp, nF);  // its barriers also complete the OR
    const unsigned long long allor = *lor;
    const int top = allor == 0 ? 0 : ((63 - __clzll(static_cast<long long>(allor))) / 8) * 8;
    const int kp = max(0, prm.keep[gl] - nF);
    const int nN = NB - nF;
    if (kp >= nN) {
      for (int b = tid; b < NB; b += kSelThreads) flag[b] |= 1;
      __syncthreads();
    } else if (kp > 0) {
      // MSB radix select of the kp-th largest block sum among non-forced blocks (sums < 2^53),
      // from the highest byte any of them has set (the bytes above are zero in all of them)
      long long prefix = 0, mask = 0;
      int rem = kp;
      bool whole_bin = false;  // the candidates with the resolved prefix are exactly the rem still needed
      for (int shift = top; shift >= 0; shift -= 8) {
        for (int d = tid; d < 256; d += kSelThreads) hist[d] = 0;
        __syncthreads();
        for (int b = tid; b < NB; b += kSelThreads) {
          const long long v = Bs[b];
          const bool cand = !(flag[b] & 2) && (v & mask) == prefix;
          const int dg = int((v >> shift) & 255);
          // a wave whose candidates share one digit (the leading digits of the sums mostly do)
          // adds their count with one atomic instead of 64 serialised on one address
          const unsigned long long cm = __ballot(cand);
          if (cm != 0) {
            const int first = __ffsll(cm) - 1;
            const int d0 = __shfl(dg, first, 64);
            if (__ballot(cand && dg != d0) == 0) {
              if ((tid & 63) == first) atomicAdd(&hist[d0], __popcll(cm));
            } else if (cand) {
              atomicAdd(&hist[dg], 1);
            }
          }
        }
        __syncthreads();
        if (tid < 64) {
          // lane l owns digits 255-4l .. 252-4l (descending); find the digit where the count of
          // larger-or-equal candidates reaches rem
          int h[4], s = 0;
#pragma unroll
          for (int u = 0; u < 4; ++u) { h[u] = hist[255 - 4 * tid - u]; s += h[u]; }
          int x = s;
#pragma unroll
          for (int off = 1; off < 64; off <<= 1) {
            int y = __shfl_up(x, off, 64);
            if (tid >= off) x += y;
          }
          const int excl = x - s;
          if (excl < rem && rem <= x) {
            int cum = excl, d = 0, hd = 0;
#pragma unroll
            for (int u = 0; u < 4; ++u) {
              if (cum + h[u] >= rem) { d = 255 - 4 * tid - u; hd = h[u]; break; }
              cum += h[u];
            }
            bcast[0] = d;
            bcast[1] = rem - cum;
            bcast[2] = rem - cum == hd ? 1 : 0;
          }
        }
        __syncthreads();
        prefix |= (long long)bcast[0] << shift;
        mask |= 255LL << shift;
        rem = bcast[1];
        whole_bin = bcast[2] != 0;
        __syncthreads();
        // every candidate of the digit's bin is selected: the lower bits cannot change the selection
        if (whole_bin) break;
      }
      // all candidates above the threshold value, and the first `rem` equal ones in block order
      const int chunk = (NB + kSelThreads - 1) / kSelThreads;
      const int b0 = tid * chunk, b1 = min(b0 + chunk, NB);
      if (whole_bin) {  // the bin is taken whole: every candidate at or above its prefix
        for (int b = b0; b < b1; ++b)
          if (!(flag[b] & 2) && (Bs[b] & mask) >= prefix) flag[b] |= 1;
        __syncthreads();
      } else {
        int neq = 0;
        for (int b = b0; b < b1; ++b)
          if (!(flag[b] & 2) && Bs[b] == prefix) ++neq;
        int tot;
        int before = block_excl_scan(neq, itmp, tot);
        for (int b = b0; b < b1; ++b) {
          if (flag[b] & 2) continue;
          if (Bs[b] > prefix) flag[b] |= 1;
          else if (Bs[b] == prefix) {
            if (before < rem) flag[b] |= 1;
            ++before;
          }
        }
        __syncthreads();
      }
    }
  }

  // pooled blocks: ranks in block order (stored over the no longer needed block sums)
  int *prank = reinterpret_cast<int *>(Bs);
  {
    const int chunk = (NB + kSelThreads - 1) / kSelThreads;
    const int b0 = tid * chunk, b1 = min(b0 + chunk, NB);
    auto pooled = [&](int b) { return tokens == 1 || (tokens == 0 && !flag[b]); };
    int np = 0;
    for (int b = b0; b < b1; ++b) np += pooled(b) ? 1 : 0;
    __syncthreads();  // every thread has read Bs-derived flags before prank overwrites Bs
    int ntot;
    int rk = block_excl_scan(np, itmp, ntot);
    for (int b = b0; b < b1; ++b) {
      if (pooled(b)) {
        prank[b] = rk;
        pool_idx[size_t(g) * NB + rk] = b;
        ++rk;
      }
    }
    if (tid == 0) counts[2 * g + 1] = ntot;
  }
  __syncthreads();
  // fine patches: ranks in raster order; pooled patches point at their block's row
  {
    const int chunk = (N + kSelThreads - 1) / kSelThreads;
    const int p0 = tid * chunk, p1 = min(p0 + chunk, N);
    int nfl = 0;
    for (int p = p0; p < p1; ++p) {
      const int i = p / W, j = p % W;
      nfl += flag[(i >> 1) * W2 + (j >> 1)] ? 1 : 0;
    }
    int nfine;
    int rk = block_excl_scan(nfl, itmp, nfine);
    int *im = idx_map + size_t(g) * N;
    int *fi = fine_idx + size_t(g) * N;
    for (int p = p0; p < p1; ++p) {
      const int i = p / W, j = p % W;
      const int b = (i >> 1) * W2 + (j >> 1);
      if (flag[b]) {
        fi[rk] = p;
        im[p] = rk;
        ++rk;
      } else {
        im[p] = tokens == 2 ? -1 : nfine + prank[b];
      }
    }
    if (tid == 0) {
      counts[2 * g] = nfine;
      // a selection of a single grid (one sample, one image) also writes the sequence layout: the
      // grid's rows start at 0 and the text rows follow them (the counts are this thread's own)
      if (cu_out != nullptr) {
        seg_out[0] = 0;
        cu_out[0] = 0;
        cu_out[1] = counts[2 * g + 1] + nfine + L;
      }
    }
  }
}

size_t select_lds_bytes(int NB) {
  return size_t(NB) * 8 + ((NB + 15) & ~15) + 32 * 4 + 256 * 4 + kSelWaves * 8 + 8 + 16;
}

hipError_t launch_select(const long long *E, const uint8_t *force, int G, int H, int W, int r,
                         int mode, int tokens, const double *tau, const int *keep, int *idx_map,
                         int *fine_idx, int *pool_idx, int *counts, int *cu, int *seg, int L,
                         hipStream_t st) {
  if ((cu != nullptr) != (seg != nullptr) || (cu != nullptr && G != 1)) return hipErrorInvalidValue;
  const int NB = H * W / 4;
  const size_t lds = select_lds_bytes(NB);
  for (int g0 = 0; g0 < G; g0 += kSelMaxGrids) {
    const int n = min(kSelMaxGrids, G - g0);
    SelChunk c;
    for (int k = 0; k < kSelMaxGrids; ++k) {
      c.tau[k] = (mode == 0 && k < n) ? tau[g0 + k] : 0.0;
      c.keep[k] = (mode == 1 && k < n) ? keep[g0 + k] : 0;
    }
    hipLaunchKernelGGL(k_select, dim3(n), dim3(kSelThreads), lds, st, E, force, H, W, r, mode, tokens,
                       c, g0, idx_map, fine_idx, pool_idx, counts, cu, seg, L);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

__global__ void k_layout(const int *__restrict__ counts, int B, int I, int L, int *__restrict__ cu,
                         int *__restrict__ seg) {
  if (threadIdx.x != 0) return;
  int row = 0;
  cu[0] = 0;
  for (int s = 0; s < B; ++s) {
    for (int i = 0; i < I; ++i) {
      const int g = s * I + i;
      seg[g] = row;
      row += counts[2 * g] + counts[2 * g + 1];
    }
    row += L;
    cu[s + 1] = row;
  }
}

hipError_t launch_layout(const int *counts, int B, int I, int L, int *cu, int *seg,
                         hipStream_t st) {
  hipLaunchKernelGGL(k_layout, dim3(1), dim3(64), 0, st, counts, B, I, L, cu, seg);
  return hipGetLastError();
}

}  // namespace hilo
