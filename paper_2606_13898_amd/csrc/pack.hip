// S3 compress, S6 decompress and the row normalisation feeding the block's projections.
//
// All three are HBM-bound row gathers/scatters: every thread moves 16-byte vectors along the
// contiguous channel axis, so each wave touches whole 1 KiB runs of a row.  Grids are sized for
// the uncompressed worst case (counts live on the device); surplus row slots exit at once.
#include "common.h"
#include "kernels.h"

namespace hilo {

constexpr int kPackThreads = 256;
constexpr int kPackRows = 4;  // row slots per workgroup, one wave each
static_assert(kPackThreads == 64 * kPackRows, "one wave per row slot");

template <bool BF16>
HILO_DEV void load8(const void *base, size_t elem, float *f) {
  if constexpr (BF16) {
    uint4 u = *reinterpret_cast<const uint4 *>(reinterpret_cast<const uint16_t *>(base) + elem);
    unpack8(u, f);
  } else {
    const float4 *p = reinterpret_cast<const float4 *>(reinterpret_cast<const float *>(base) + elem);
    float4 a = p[0], b = p[1];
    f[0] = a.x; f[1] = a.y; f[2] = a.z; f[3] = a.w; f[4] = b.x; f[5] = b.y; f[6] = b.z; f[7] = b.w;
  }
}

template <bool BF16>
HILO_DEV void store8(void *base, size_t elem, const float *f) {
  if constexpr (BF16) {
    uint4 u;
    u.x = pack_bf16x2(f[0], f[1]);
    u.y = pack_bf16x2(f[2], f[3]);
    u.z = pack_bf16x2(f[4], f[5]);
    u.w = pack_bf16x2(f[6], f[7]);
    *reinterpret_cast<uint4 *>(reinterpret_cast<uint16_t *>(base) + elem) = u;
  } else {
    float4 *p = reinterpret_cast<float4 *>(reinterpret_cast<float *>(base) + elem);
    p[0] = make_float4(f[0], f[1], f[2], f[3]);
    p[1] = make_float4(f[4], f[5], f[6], f[7]);
  }
}

HILO_DEV void store8_f32(float *z, size_t elem, const float *f) {
  float4 *p = reinterpret_cast<float4 *>(z + elem);
  p[0] = make_float4(f[0], f[1], f[2], f[3]);
  p[1] = make_float4(f[4], f[5], f[6], f[7]);
}

// Row slots: [0, G*N) are image rows (grid g, compressed row k = slot % N), then B*L text rows.
// One wave per row slot (kPackRows per workgroup): the rows of a workgroup proceed in parallel
// and each lane issues all of its loads for the row before the stores.
template <bool BF16>
__global__ __launch_bounds__(kPackThreads) void k_compress(
    const void *__restrict__ x_img, const void *__restrict__ x_txt, const int *__restrict__ fine_idx,
    const int *__restrict__ pool_idx, const int *__restrict__ counts, const int *__restrict__ cu,
    const int *__restrict__ seg, float *__restrict__ z, int G, int N, int W, int D, int L,
    long long nslots) {
#pragma clang fp contract(off)
  const int CGn = D / 8;
  const int lane = threadIdx.x & 63;
  const int R = N + N / 4;  // row slots per grid: at most N fine rows and N / 4 pooled ones
  const long long imgSlots = (long long)G * R;
  const long long slot = (long long)blockIdx.x * kPackRows + (threadIdx.x >> 6);
  if (slot >= nslots) return;
  size_t dst, s0, s1 = 0, s2 = 0, s3 = 0;
  bool pooled = false;
  const void *src = x_img;
  if (slot < imgSlots) {
    const int g = int(slot / R), k = int(slot % R);
    const int nf = counts[2 * g], np = counts[2 * g + 1];
    if (k >= nf + np) return;
    dst = size_t(seg[g] + k);
    if (k < nf) {
      s0 = size_t(g) * N + fine_idx[size_t(g) * N + k];
    } else {
      const int b = pool_idx[size_t(g) * (N / 4) + (k - nf)];
      const int W2 = W / 2;
      const size_t p00 = size_t(g) * N + size_t(b / W2) * 2 * W + size_t(b % W2) * 2;
      s0 = p00; s1 = p00 + 1; s2 = p00 + W; s3 = p00 + W + 1;
      pooled = true;
    }
  } else {
    const long long t = slot - imgSlots;
    const int s = int(t / L), j = int(t % L);
    dst = size_t(cu[s + 1] - L + j);
    s0 = size_t(s) * L + j;
    src = x_txt;
  }
  if (pooled) {
#pragma unroll 2
    for (int cg = lane; cg < CGn; cg += 64) {
      const size_t c = size_t(cg) * 8;
      float a[8], b[8], e[8], f[8];
      load8<BF16>(src, s0 * D + c, a);
      load8<BF16>(src, s1 * D + c, b);
      load8<BF16>(src, s2 * D + c, e);
      load8<BF16>(src, s3 * D + c, f);
#pragma unroll
      for (int v = 0; v < 8; ++v) a[v] = ((a[v] + b[v]) + (e[v] + f[v])) * 0.25f;
      store8_f32(z, dst * D + c, a);
    }
  } else {
#pragma unroll 4
    for (int cg = lane; cg < CGn; cg += 64) {
      const size_t c = size_t(cg) * 8;
      float a[8];
      load8<BF16>(src, s0 * D + c, a);
      store8_f32(z, dst * D + c, a);
    }
  }
}

hipError_t launch_compress(bool bf16, const void *x_img, const void *x_txt, const int *fine_idx,
                           const int *pool_idx, const int *counts, const int *cu, const int *seg,
                           float *z, int B, int I, int H, int W, int D, int L, hipStream_t st) {
  const int G = B * I, N = H * W;
  const long long nslots = (long long)G * (N + N / 4) + (long long)B * L;
  const long long nblk = (nslots + kPackRows - 1) / kPackRows;
  if (nblk <= 0) return hipSuccess;
  if (bf16)
    hipLaunchKernelGGL(k_compress<true>, dim3(unsigned(nblk)), dim3(kPackThreads), 0, st, x_img,
                       x_txt, fine_idx, pool_idx, counts, cu, seg, z, G, N, W, D, L, nslots);
  else
    hipLaunchKernelGGL(k_compress<false>, dim3(unsigned(nblk)), dim3(kPackThreads), 0, st, x_img,
                       x_txt, fine_idx, pool_idx, counts, cu, seg, z, G, N, W, D, L, nslots);
  return hipGetLastError();
}

// Output row slots: [0, G*N) image patches, then B*L text rows; one wave per row slot.
template <bool BF16>
__global__ __launch_bounds__(kPackThreads) void k_decompress(
    const float *__restrict__ z, const int *__restrict__ idx_map, const int *__restrict__ cu,
    const int *__restrict__ seg, void *__restrict__ y_img, void *__restrict__ y_txt, int G, int N,
    int D, int L, long long nslots) {
  const int CGn = D / 8;
  const int lane = threadIdx.x & 63;
  const long long imgSlots = (long long)G * N;
  const long long slot = (long long)blockIdx.x * kPackRows + (threadIdx.x >> 6);
  if (slot >= nslots) return;
  size_t src, dst;
  void *out;
  if (slot < imgSlots) {
    const int g = int(slot / N);
    const int idx = idx_map[slot];
    dst = size_t(slot);
    out = y_img;
    if (idx < 0) {  // a dropped patch (token set "drop"): no token, zeros
      const float f[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
      for (int cg = lane; cg < CGn; cg += 64) store8<BF16>(out, dst * D + size_t(cg) * 8, f);
      return;
    }
    src = size_t(seg[g]) + size_t(idx);
  } else {
    if (!y_txt) return;
    const long long t = slot - imgSlots;
    const int s = int(t / L), j = int(t % L);
    src = size_t(cu[s + 1] - L + j);
    dst = size_t(t);
    out = y_txt;
  }
#pragma unroll 4
  for (int cg = lane; cg < CGn; cg += 64) {
    const size_t c = size_t(cg) * 8;
    const float4 *p = reinterpret_cast<const float4 *>(z + src * D + c);
    const float4 a = p[0], b = p[1];
    float f[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
    store8<BF16>(out, dst * D + c, f);
  }
}

// Delta form: y[p] = x[p] + (z[row] - z0[row]) where z0 is what compress wrote to the row, rebuilt
// here from x with the same float32 operations (the patch itself for a fine row; for a pooled row
// ((x00 + x01) + (x10 + x11)) * 0.25 over its block); a patch without a token keeps x[p].  Text
// rows are copied as in k_decompress.
template <bool BF16>
__global__ __launch_bounds__(kPackThreads) void k_decompress_delta(
    const float *__restrict__ z, const void *__restrict__ x_img, const int *__restrict__ idx_map,
    const int *__restrict__ counts, const int *__restrict__ cu, const int *__restrict__ seg,
    void *__restrict__ y_img, void *__restrict__ y_txt, int G, int N, int W, int D, int L,
    long long nslots) {
#pragma clang fp contract(off)
  const int CGn = D / 8;
  const int lane = threadIdx.x & 63;
  const long long imgSlots = (long long)G * N;
  const long long slot = (long long)blockIdx.x * kPackRows + (threadIdx.x >> 6);
  if (slot >= nslots) return;
  if (slot >= imgSlots) {
    if (!y_txt) return;
    const long long t = slot - imgSlots;
    const int s = int(t / L), j = int(t % L);
    const size_t src = size_t(cu[s + 1] - L + j);
    for (int cg = lane; cg < CGn; cg += 64) {
      const size_t c = size_t(cg) * 8;
      const float4 *q = reinterpret_cast<const float4 *>(z + src * D + c);
      const float4 a = q[0], b = q[1];
      float f[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
      store8<BF16>(y_txt, size_t(t) * D + c, f);
    }
    return;
  }
  const int g = int(slot / N), p = int(slot % N);
  const int idx = idx_map[slot];
  const int nf = counts[2 * g];
  const size_t row = size_t(seg[g]) + size_t(idx < 0 ? 0 : idx);
  const int i = p / W, j = p % W;
  const size_t p00 = size_t(g) * N + size_t(i & ~1) * W + size_t(j & ~1);
#pragma unroll 2
  for (int cg = lane; cg < CGn; cg += 64) {
    const size_t c = size_t(cg) * 8;
    float x[8];
    load8<BF16>(x_img, slot * size_t(D) + c, x);
    if (idx >= 0) {
      float z0[8];
      if (idx < nf) {
#pragma unroll
        for (int v = 0; v < 8; ++v) z0[v] = x[v];
      } else {
        float a[8], b[8], e[8], f[8];
        load8<BF16>(x_img, p00 * D + c, a);
        load8<BF16>(x_img, (p00 + 1) * D + c, b);
        load8<BF16>(x_img, (p00 + W) * D + c, e);
        load8<BF16>(x_img, (p00 + W + 1) * D + c, f);
#pragma unroll
        for (int v = 0; v < 8; ++v) z0[v] = ((a[v] + b[v]) + (e[v] + f[v])) * 0.25f;
      }
      const float4 *q = reinterpret_cast<const float4 *>(z + row * D + c);
      const float4 za = q[0], zb = q[1];
      const float zz[8] = {za.x, za.y, za.z, za.w, zb.x, zb.y, zb.z, zb.w};
#pragma unroll
      for (int v = 0; v < 8; ++v) x[v] = x[v] + (zz[v] - z0[v]);
    }
    store8<BF16>(y_img, slot * size_t(D) + c, x);
  }
}

hipError_t launch_decompress_delta(bool bf16, const float *z, const void *x_img, const int *idx_map,
                                   const int *counts, const int *cu, const int *seg, void *y_img,
                                   void *y_txt, int B, int I, int H, int W, int D, int L, hipStream_t st) {
  const int G = B * I, N = H * W;
  const long long nslots = (long long)G * N + (long long)B * L;
  const long long nblk = (nslots + kPackRows - 1) / kPackRows;
  if (nblk <= 0) return hipSuccess;
  if (bf16)
    hipLaunchKernelGGL(k_decompress_delta<true>, dim3(unsigned(nblk)), dim3(kPackThreads), 0, st, z,
                       x_img, idx_map, counts, cu, seg, y_img, y_txt, G, N, W, D, L, nslots);
  else
    hipLaunchKernelGGL(k_decompress_delta<false>, dim3(unsigned(nblk)), dim3(kPackThreads), 0, st, z,
                       x_img, idx_map, counts, cu, seg, y_img, y_txt, G, N, W, D, L, nslots);
  return hipGetLastError();
}

hipError_t launch_decompress(bool bf16, const float *z, const int *idx_map, const int *cu,
                             const int *seg, void *y_img, void *y_txt, int B, int I, int N, int D,
                             int L, hipStream_t st) {
  const int G = B * I;
  const long long nslots = (long long)G * N + (long long)B * L;
  const long long nblk = (nslots + kPackRows - 1) / kPackRows;
  if (nblk <= 0) return hipSuccess;
  if (bf16)
    hipLaunchKernelGGL(k_decompress<true>, dim3(unsigned(nblk)), dim3(kPackThreads), 0, st, z,
                       idx_map, cu, seg, y_img, y_txt, G, N, D, L, nslots);
  else
    hipLaunchKernelGGL(k_decompress<false>, dim3(unsigned(nblk)), dim3(kPackThreads), 0, st, z,
                       idx_map, cu, seg, y_img, y_txt, G, N, D, L, nslots);
  return hipGetLastError();
}

// ------------------------------------------------------------------------------- row norm

// LN(v) (biased variance, eps 1e-6) * (1 + scale) + shift of one row held by a wave (lane l holds
// the float4 at columns (64 k + l) * 4, k < NV), written in the projection's input form: OUT 0
// float32, 1 bf16, 2 FP8 E4M3 codes plus the row's scale (amax / 448; codes of h * (448 / amax),
// both divisions correctly rounded).  shift points at the row's (sample, stream) shift vector, the
// scale vector follows it.  Every lane takes part (wave reductions).
template <int OUT, int NV>
HILO_DEV void norm_row(float4 (&v)[NV], int lane, int D, const float *__restrict__ shift, size_t row,
                       void *__restrict__ out, float *__restrict__ row_scale) {
  const float *scale = shift + D;
  float sum = 0.f;
#pragma unroll
  for (int k = 0; k < NV; ++k) sum += (v[k].x + v[k].y) + (v[k].z + v[k].w);
  const float mean = wave_sum_f32(sum) / float(D);
  float sq = 0.f;
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const int c = (k * 64 + lane) * 4;
    if (c < D) {
      const float a = v[k].x - mean, b = v[k].y - mean, e = v[k].z - mean, f = v[k].w - mean;
      sq += (a * a + b * b) + (e * e + f * f);
    }
  }
  const float var = wave_sum_f32(sq) / float(D);
  const float rstd = 1.0f / sqrtf(var + 1e-6f);
  if constexpr (OUT == 2) {
    float amax = 0.f;
#pragma unroll
    for (int k = 0; k < NV; ++k) {
      const int c = (k * 64 + lane) * 4;
      if (c < D) {
        const float4 sc = *reinterpret_cast<const float4 *>(scale + c);
        const float4 sh = *reinterpret_cast<const float4 *>(shift + c);
        v[k].x = (v[k].x - mean) * rstd * (1.f + sc.x) + sh.x;
        v[k].y = (v[k].y - mean) * rstd * (1.f + sc.y) + sh.y;
        v[k].z = (v[k].z - mean) * rstd * (1.f + sc.z) + sh.z;
        v[k].w = (v[k].w - mean) * rstd * (1.f + sc.w) + sh.w;
        amax = fmaxf(amax, fmaxf(fmaxf(fabsf(v[k].x), fabsf(v[k].y)), fmaxf(fabsf(v[k].z), fabsf(v[k].w))));
      }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) amax = fmaxf(amax, __shfl_xor(amax, off, 64));
    const float inv = amax > 0.f ? __fdiv_rn(448.0f, amax) : 0.f;
    if (lane == 0) row_scale[row] = __fdiv_rn(amax, 448.0f);
    uint8_t *o = reinterpret_cast<uint8_t *>(out) + row * D;
#pragma unroll
    for (int k = 0; k < NV; ++k) {
      const int c = (k * 64 + lane) * 4;
      if (c < D)
        *reinterpret_cast<uint32_t *>(o + c) = fp8x4(v[k].x * inv, v[k].y * inv, v[k].z * inv, v[k].w * inv);
    }
    return;
  }
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const int c = (k * 64 + lane) * 4;
    if (c < D) {
      const float4 sc = *reinterpret_cast<const float4 *>(scale + c);
      const float4 sh = *reinterpret_cast<const float4 *>(shift + c);
      const float h0 = (v[k].x - mean) * rstd * (1.f + sc.x) + sh.x;
      const float h1 = (v[k].y - mean) * rstd * (1.f + sc.y) + sh.y;
      const float h2 = (v[k].z - mean) * rstd * (1.f + sc.z) + sh.z;
      const float h3 = (v[k].w - mean) * rstd * (1.f + sc.w) + sh.w;
      if constexpr (OUT == 1) {
        uint2 u;
        u.x = pack_bf16x2(h0, h1);
        u.y = pack_bf16x2(h2, h3);
        *reinterpret_cast<uint2 *>(reinterpret_cast<uint16_t *>(out) + row * D + c) = u;
      } else {
        *reinterpret_cast<float4 *>(reinterpret_cast<float *>(out) + row * D + c) = make_float4(h0, h1, h2, h3);
      }
    }
  }
}

// One wave per row of z: norm_row with the row's sample and stream (modulation set `which`: 0 for
// the attention half, 1 for the MLP half).  NV = float4s per lane covers D <= 256 NV; the row stays
// in registers between the passes.
template <int OUT, int NV>
__global__ __launch_bounds__(256) void k_rownorm(const float *__restrict__ z, const int *__restrict__ cu,
                                                 const float *__restrict__ mod, int B, int L, int D,
                                                 int Tmax, int which, void *__restrict__ out,
                                                 float *__restrict__ row_scale) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= Tmax || row >= cu[B]) return;
  const int s = sample_of_row(cu, B, row);
  const int sigma = row >= cu[s + 1] - L ? 1 : 0;
  const float *shift = mod + (size_t(s * 2 + sigma) * 6 + which * 3) * D;
  const float *zr = z + size_t(row) * D;
  float4 v[NV];
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const int c = (k * 64 + lane) * 4;
    v[k] = c < D ? *reinterpret_cast<const float4 *>(zr + c) : make_float4(0.f, 0.f, 0.f, 0.f);
  }
  norm_row<OUT, NV>(v, lane, D, shift, size_t(row), out, row_scale);
}

// S3 and the attention half's row norm in one pass: the row slots of k_compress, one wave each,
// form the z row in registers in norm_row's lane layout (lane l: the float4 at columns (64 k + l) *
// 4), store it, and norm_row writes its normalised, modulated form (modulation set 0) -- the z
// values and the normalised rows are those of k_compress followed by k_rownorm, bit for bit, and
// z is not read back.  Image rows take the shift and scale of their grid's sample, text rows the
// text stream's.
template <bool BF16, int OUT, int NV>
__global__ __launch_bounds__(kPackThreads) void k_compress_norm(
    const void *__restrict__ x_img, const void *__restrict__ x_txt, const int *__restrict__ fine_idx,
    const int *__restrict__ pool_idx, const int *__restrict__ counts, const int *__restrict__ cu,
    const int *__restrict__ seg, const float *__restrict__ mod, float *__restrict__ z, int G, int I,
    int N, int W, int D, int L, long long nslots, void *__restrict__ out, float *__restrict__ row_scale) {
#pragma clang fp contract(off)
  const int lane = threadIdx.x & 63;
  const int R = N + N / 4;
  const long long imgSlots = (long long)G * R;
  const long long slot = (long long)blockIdx.x * kPackRows + (threadIdx.x >> 6);
  if (slot >= nslots) return;
  size_t dst, s0, s1 = 0, s2 = 0, s3 = 0;
  bool pooled = false;
  const void *src = x_img;
  int sample, sigma;
  if (slot < imgSlots) {
    const int g = int(slot / R), k = int(slot % R);
    const int nf = counts[2 * g], np = counts[2 * g + 1];
    if (k >= nf + np) return;
    dst = size_t(seg[g] + k);
    sample = g / I;
    sigma = 0;
    if (k < nf) {
      s0 = size_t(g) * N + fine_idx[size_t(g) * N + k];
    } else {
      const int b = pool_idx[size_t(g) * (N / 4) + (k - nf)];
      const int W2 = W / 2;
      const size_t p00 = size_t(g) * N + size_t(b / W2) * 2 * W + size_t(b % W2) * 2;
      s0 = p00; s1 = p00 + 1; s2 = p00 + W; s3 = p00 + W + 1;
      pooled = true;
    }
  } else {
    const long long t = slot - imgSlots;
    sample = int(t / L);
    const int j = int(t % L);
    dst = size_t(cu[sample + 1] - L + j);
    s0 = size_t(sample) * L + j;
    src = x_txt;
    sigma = 1;
  }
  auto load4 = [&](size_t e) __attribute__((always_inline)) {
    if constexpr (BF16) {
      const uint2 u = *reinterpret_cast<const uint2 *>(reinterpret_cast<const uint16_t *>(src) + e);
      return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u),
                         __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xffff0000u));
    } else {
      return *reinterpret_cast<const float4 *>(reinterpret_cast<const float *>(src) + e);
    }
  };
  float4 v[NV];
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const int c = (k * 64 + lane) * 4;
    if (c < D) {
      if (pooled) {
        const float4 a = load4(s0 * D + c), b = load4(s1 * D + c), e = load4(s2 * D + c), f = load4(s3 * D + c);
        v[k] = make_float4(((a.x + b.x) + (e.x + f.x)) * 0.25f, ((a.y + b.y) + (e.y + f.y)) * 0.25f,
                           ((a.z + b.z) + (e.z + f.z)) * 0.25f, ((a.w + b.w) + (e.w + f.w)) * 0.25f);
      } else {
        v[k] = load4(s0 * D + c);
      }
      *reinterpret_cast<float4 *>(z + dst * D + c) = v[k];
    } else {
      v[k] = make_float4(0.f, 0.f, 0.f, 0.f);
    }
  }
  norm_row<OUT, NV>(v, lane, D, mod + size_t(sample * 2 + sigma) * 6 * D, dst, out, row_scale);
}

template <bool BF16, int OUT>
static hipError_t run_compress_norm(const void *x_img, const void *x_txt, const int *fine_idx,
                                    const int *pool_idx, const int *counts, const int *cu, const int *seg,
                                    const float *mod, float *z, int G, int I, int N, int W, int D, int L,
                                    long long nslots, void *out, float *row_scale, hipStream_t st) {
  const long long nblk = (nslots + kPackRows - 1) / kPackRows;
  const int nv = (D + 255) / 256;
#define HILO_CN(NVV)                                                                                  \
  hipLaunchKernelGGL((k_compress_norm<BF16, OUT, NVV>), dim3(unsigned(nblk)), dim3(kPackThreads), 0, st, \
                     x_img, x_txt, fine_idx, pool_idx, counts, cu, seg, mod, z, G, I, N, W, D, L, nslots, \
                     out, row_scale)
  if (nv <= 4) HILO_CN(4);
  else if (nv <= 8) HILO_CN(8);
  else if (nv <= 12) HILO_CN(12);
  else if (nv <= 16) HILO_CN(16);
  else HILO_CN(32);
#undef HILO_CN
  return hipGetLastError();
}

hipError_t launch_compress_norm(bool bf16, const void *x_img, const void *x_txt, const int *fine_idx,
                                const int *pool_idx, const int *counts, const int *cu, const int *seg,
                                const float *mod, float *z, int B, int I, int H, int W, int D, int L,
                                void *out, hipStream_t st, bool fp8, float *row_scale) {
  const int G = B * I, N = H * W;
  const long long nslots = (long long)G * (N + N / 4) + (long long)B * L;
  if (nslots <= 0) return hipSuccess;
  if (fp8)
    return bf16 ? run_compress_norm<true, 2>(x_img, x_txt, fine_idx, pool_idx, counts, cu, seg, mod, z, G,
                                             I, N, W, D, L, nslots, out, row_scale, st)
                : hipErrorInvalidValue;
  return bf16 ? run_compress_norm<true, 1>(x_img, x_txt, fine_idx, pool_idx, counts, cu, seg, mod, z, G,
                                           I, N, W, D, L, nslots, out, nullptr, st)
              : run_compress_norm<false, 0>(x_img, x_txt, fine_idx, pool_idx, counts, cu, seg, mod, z,
                                            G, I, N, W, D, L, nslots, out, nullptr, st);
}

template <int OUT>
static hipError_t run_rownorm(const float *z, const int *cu, const float *mod, int B, int L, int D,
                              int Tmax, int which, void *out, float *row_scale, hipStream_t st) {
  const int nblk = (Tmax + 3) / 4;
  const int nv = (D + 255) / 256;
#define HILO_NORM(NVV)                                                                         \
  hipLaunchKernelGGL((k_rownorm<OUT, NVV>), dim3(nblk), dim3(256), 0, st, z, cu, mod, B, L, D, \
                     Tmax, which, out, row_scale)
  if (nv <= 4) HILO_NORM(4);
  else if (nv <= 8) HILO_NORM(8);
  else if (nv <= 12) HILO_NORM(12);
  else if (nv <= 16) HILO_NORM(16);
  else HILO_NORM(32);
#undef HILO_NORM
  return hipGetLastError();
}

hipError_t launch_rownorm(bool bf16, const float *z, const int *cu, const float *mod, int B, int L,
                          int D, int Tmax, int which, void *out, hipStream_t st) {
  if (Tmax <= 0) return hipSuccess;
  return bf16 ? run_rownorm<1>(z, cu, mod, B, L, D, Tmax, which, out, nullptr, st)
              : run_rownorm<0>(z, cu, mod, B, L, D, Tmax, which, out, nullptr, st);
}

hipError_t launch_rownorm_fp8(const float *z, const int *cu, const float *mod, int B, int L, int D,
                              int Tmax, int which, uint8_t *codes, float *row_scale, hipStream_t st) {
  if (Tmax <= 0) return hipSuccess;
  return run_rownorm<2>(z, cu, mod, B, L, D, Tmax, which, codes, row_scale, st);
}

// Per-row FP8 quantisation of a [rows][cols] matrix (bf16 or float32), one wave per row: the row's
// amax, then the codes of x * (448 / amax) and the scale amax / 448 (as k_rownorm's FP8 output).
template <bool BF16>
__global__ __launch_bounds__(256) void k_quantize_rows(const void *__restrict__ x, int rows, int cols,
                                                       uint8_t *__restrict__ codes, float *__restrict__ scale,
                                                       const int *__restrict__ row_limit) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows || (row_limit && row >= *row_limit)) return;
  auto ld4 = [&](int c, float *f) {
    if constexpr (BF16) {
      const uint2 u = *reinterpret_cast<const uint2 *>(reinterpret_cast<const uint16_t *>(x) + size_t(row) * cols + c);
      f[0] = __uint_as_float(u.x << 16); f[1] = __uint_as_float(u.x & 0xffff0000u);
      f[2] = __uint_as_float(u.y << 16); f[3] = __uint_as_float(u.y & 0xffff0000u);
    } else {
      const float4 u = *reinterpret_cast<const float4 *>(reinterpret_cast<const float *>(x) + size_t(row) * cols + c);
      f[0] = u.x; f[1] = u.y; f[2] = u.z; f[3] = u.w;
    }
  };
  float amax = 0.f;
  for (int c = lane * 4; c < cols; c += 256) {
    float f[4];
    ld4(c, f);
    amax = fmaxf(amax, fmaxf(fmaxf(fabsf(f[0]), fabsf(f[1])), fmaxf(fabsf(f[2]), fabsf(f[3]))));
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) amax = fmaxf(amax, __shfl_xor(amax, off, 64));
  const float inv = amax > 0.f ? __fdiv_rn(448.0f, amax) : 0.f;
  if (lane == 0) scale[row] = __fdiv_rn(amax, 448.0f);
  for (int c = lane * 4; c < cols; c += 256) {
    float f[4];
    ld4(c, f);
    *reinterpret_cast<uint32_t *>(codes + size_t(row) * cols + c) = fp8x4(f[0] * inv, f[1] * inv, f[2] * inv, f[3] * inv);
  }
}

// The same quantisation for bf16 rows of up to 16384 columns in one pass over HBM: one workgroup
// per row, the row held in registers (NC chunks of 4 columns per thread, packed bf16), the amax
// reduced over the workgroup.
template <int NC>
__global__ __launch_bounds__(256) void k_quantize_rows_wg(const uint16_t *__restrict__ x, int cols,
                                                          uint8_t *__restrict__ codes, float *__restrict__ scale,
                                                          const int *__restrict__ row_limit) {
  __shared__ float red[4];
  const int row = blockIdx.x, tid = threadIdx.x;
  if (row_limit && row >= *row_limit) return;
  const uint16_t *xr = x + size_t(row) * cols;
  uint2 v[NC];
  float amax = 0.f;
#pragma unroll
  for (int k = 0; k < NC; ++k) {
    const int c = (k * 256 + tid) * 4;
    v[k] = c < cols ? *reinterpret_cast<const uint2 *>(xr + c) : make_uint2(0u, 0u);
    amax = fmaxf(amax, fmaxf(fmaxf(fabsf(__uint_as_float(v[k].x << 16)), fabsf(__uint_as_float(v[k].x & 0xffff0000u))),
                             fmaxf(fabsf(__uint_as_float(v[k].y << 16)), fabsf(__uint_as_float(v[k].y & 0xffff0000u)))));
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) amax = fmaxf(amax, __shfl_xor(amax, off, 64));
  if ((tid & 63) == 0) red[tid >> 6] = amax;
  __syncthreads();
  amax = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  const float inv = amax > 0.f ? __fdiv_rn(448.0f, amax) : 0.f;
  if (tid == 0) scale[row] = __fdiv_rn(amax, 448.0f);
  uint8_t *o = codes + size_t(row) * cols;
#pragma unroll
  for (int k = 0; k < NC; ++k) {
    const int c = (k * 256 + tid) * 4;
    if (c < cols)
      *reinterpret_cast<uint32_t *>(o + c) =
          fp8x4(__uint_as_float(v[k].x << 16) * inv, __uint_as_float(v[k].x & 0xffff0000u) * inv,
                __uint_as_float(v[k].y << 16) * inv, __uint_as_float(v[k].y & 0xffff0000u) * inv);
  }
}

hipError_t launch_quantize_rows(bool bf16, const void *x, int rows, int cols, uint8_t *codes, float *scale,
                                hipStream_t st, const int *row_limit) {
  if (rows <= 0) return hipSuccess;
  if (bf16 && cols <= 16384) {
    const uint16_t *xb = reinterpret_cast<const uint16_t *>(x);
    const int nc = (cols + 1023) / 1024;
#define HILO_QWG(NCV) \
  hipLaunchKernelGGL(k_quantize_rows_wg<NCV>, dim3(rows), dim3(256), 0, st, xb, cols, codes, scale, row_limit)
    if (nc <= 1) HILO_QWG(1);
    else if (nc <= 2) HILO_QWG(2);
    else if (nc <= 3) HILO_QWG(3);
    else if (nc <= 4) HILO_QWG(4);
    else if (nc <= 6) HILO_QWG(6);
    else if (nc <= 8) HILO_QWG(8);
    else if (nc <= 12) HILO_QWG(12);
    else HILO_QWG(16);
#undef HILO_QWG
    return hipGetLastError();
  }
  const int nblk = (rows + 3) / 4;
  if (bf16)
    hipLaunchKernelGGL(k_quantize_rows<true>, dim3(nblk), dim3(256), 0, st, x, rows, cols, codes, scale, row_limit);
  else
    hipLaunchKernelGGL(k_quantize_rows<false>, dim3(nblk), dim3(256), 0, st, x, rows, cols, codes, scale, row_limit);
  return hipGetLastError();
}

}  // namespace hilo
