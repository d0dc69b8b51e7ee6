// Shared device helpers for the gfx950 kernels of libhilo.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#define HILO_DEV __device__ __forceinline__

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

namespace hilo {

constexpr int kXcds = 8;  // MI355X: 8 accelerator complex dies, each with its own L2

// The dispatcher hands workgroup b to XCD b % 8.  Remap so that each XCD receives a contiguous
// range of logical tiles (neighbouring tiles then share that XCD's L2).
HILO_DEV int xcd_remap(int b, int n) {
  int q = n / kXcds, r = n % kXcds;
  int x = b % kXcds, k = b / kXcds;
  return x * q + (x < r ? x : r) + k;
}

HILO_DEV float bf2f(uint16_t b) { return __uint_as_float(uint32_t(b) << 16); }

// float -> bf16 bits, round to nearest even (NaN stays NaN).
HILO_DEV uint16_t f2bf(float f) {
  return __builtin_bit_cast(uint16_t, static_cast<__bf16>(f));
}

HILO_DEV uint32_t pack_bf16x2(float lo, float hi) {
  return uint32_t(f2bf(lo)) | (uint32_t(f2bf(hi)) << 16);
}

// 8 bf16 (one 16-byte load) -> 8 floats
HILO_DEV void unpack8(const uint4 &u, float *f) {
  f[0] = __uint_as_float(u.x << 16); f[1] = __uint_as_float(u.x & 0xffff0000u);
  f[2] = __uint_as_float(u.y << 16); f[3] = __uint_as_float(u.y & 0xffff0000u);
  f[4] = __uint_as_float(u.z << 16); f[5] = __uint_as_float(u.z & 0xffff0000u);
  f[6] = __uint_as_float(u.w << 16); f[7] = __uint_as_float(u.w & 0xffff0000u);
}

HILO_DEV long long wave_sum_i64(long long v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

HILO_DEV long long wave_max_i64(long long v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    long long o = __shfl_xor(v, off, 64);
    v = o > v ? o : v;
  }
  return v;
}

HILO_DEV float wave_sum_f32(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// FP8 E4M3 codes of four values after scaling: clamp to the format's range (the conversion itself
// would turn an overflow into NaN), then round to nearest even.
HILO_DEV uint32_t fp8x4(float a, float b, float c, float d) {
  const float m = 448.0f;
  a = fminf(fmaxf(a, -m), m); b = fminf(fmaxf(b, -m), m);
  c = fminf(fmaxf(c, -m), m); d = fminf(fmaxf(d, -m), m);
  int w = __builtin_amdgcn_cvt_pk_fp8_f32(a, b, 0, false);
  w = __builtin_amdgcn_cvt_pk_fp8_f32(c, d, w, true);
  return uint32_t(w);
}

// Power-of-two scale of a row for E4M3 codes: the least k with 448 * 2^k >= amax (amax = f * 2^e,
// f in [1, 2): k = e - 8 when f <= 1.75, else e - 7), clamped below at -127, the least E8M0 scale;
// 0 for an all-zero row.  Codes are then x * 2^-k (exact), all within [-448, 448].
HILO_DEV int pow2_exponent(float amax) {
  const uint32_t b = __float_as_uint(amax);
  const int e = int((b >> 23) & 0xff);
  if (amax == 0.f) return 0;
  if (e == 0) return -127;  // subnormal: far below 448 * 2^-127
  const int k = e - 127 - ((b & 0x7fffff) <= 0x600000u ? 8 : 7);
  return k < -127 ? -127 : k;
}
// 2^-k for k in [-127, 127] as a float (always a normal number for the k above)
HILO_DEV float pow2_inverse(int k) { return __uint_as_float(uint32_t(127 - k) << 23); }

// Sample boundary i of the packed sequence.  The boundaries do not change while a kernel runs, so
// they are read through the constant address space: the compiler then uses scalar loads with their
// own wait, where a vector load inside a pipelined loop is followed by a wait for every global load
// in flight (a drained prefetch per tile or unit).
HILO_DEV int cu_at(const int *cu, int i) { return ((const __attribute__((address_space(4))) int *)cu)[i]; }

// Sample that packed row r belongs to: largest s with cu[s] <= r (cu has B+1 entries).
HILO_DEV int sample_of_row(const int32_t *cu, int B, int r) {
  int lo = 0, hi = B;  // answer in [lo, hi)
  while (hi - lo > 1) {
    int mid = (lo + hi) >> 1;
    if (cu[mid] <= r) lo = mid; else hi = mid;
  }
  return lo;
}

}  // namespace hilo
