// Attention core: a = softmax(q k^T / sqrt(hd)) v per sample and head over the packed ragged
// sequence (joint attention of a sample's image and text tokens, no mask).
//
// bf16 path (gfx950 MFMA v_mfma_f32_16x16x32_bf16, fp32 online softmax in base 2):
//   workgroup = NW waves x QW query rows of one (sample, head) (head dim 128: 8 x 32, one
//   workgroup per CU; 64: 4 x 32, two per CU); K/V stream through LDS in tiles of 64 keys, double
//   buffered.  Each wave computes S^T = K Q^T so that every lane owns one query
//   row's scores (4 keys per 16-key subtile): the running max stays lane-local, and the
//   probabilities are already in the register layout of the second MFMA operand for
//   O^T = V^T P^T.  The MFMA's k index may be permuted as long as both operands agree: the lane
//   holding keys {4g..4g+3} and {16+4g..16+4g+3} of a 32-key step feeds exactly those keys of V^T.
//   K and V both land in LDS in their natural [key][dim] layout by direct global->LDS loads; the
//   V^T fragments come out of gfx950's transposing LDS read (ds_read_b64_tr_b16), two per
//   fragment.  Fragments are read ahead of their MFMAs (K one key subtile, V two output subtiles)
//   through inline asm with explicit waits, and the next tile's transfer starts at the top of a
//   step.  Only the last key tile carries the sequence-end mask.  The row sums of P come from one
//   more MFMA against a fragment of ones, and the reference maximum of the online softmax moves
//   (rescaling O and l) only when a row maximum exceeds it by more than 2^8.
#include "common.h"
#include "kernels.h"

namespace hilo {

constexpr float kLog2e = 1.4426950408889634f;
// online softmax: the reference maximum lags the true one by at most this much (base 2)
constexpr float kLazyRescale = 8.0f;

// max with the lanes 16 and 32 apart (the 4 lanes holding the same query row)
HILO_DEV float xmax16_32(float x) {
  auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

// K tile rows (head_dim bf16) are stored with 16-byte chunk c of row r at slot c ^ kswz(r), so
// the 16 lanes reading one chunk of 16 consecutive rows hit 16 distinct bank groups.
template <int HD>
HILO_DEV int kswz(int r) {
  if constexpr (HD == 128) return r & 15;
  else return (r & 7) ^ ((r >> 3) & 1);
}

// V tile rows (head_dim bf16, [key][dim]) keep 16-byte chunk c of row r at slot c ^ vsw(r).  A
// transposing fragment read has the 16 lanes of a group read 8 bytes each from 4 consecutive rows
// (a multiple of 4 apart from the group's first) and 2 neighbouring chunks: 2 (r & 3) gives those
// 8 (row, chunk) pairs distinct slots, and 8 ((r >> 2) & 1) moves the next group (the next 4
// rows) to the other half of a 256-byte row.
template <int HD>
HILO_DEV int vsw(int r) {
  if constexpr (HD == 128) return (2 * (r & 3)) ^ (8 * ((r >> 2) & 1));
  else return 2 * (r & 3);
}

typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));

// MFMA fragments leave LDS through inline asm with explicit waits.  The compiler then sees no LDS
// load that might alias the global->LDS transfer in flight into the other buffer; for one it can
// see, it waits for that whole transfer before the first fragment read of the step.
template <int OFF>
HILO_DEV void lds_read_b128(bf16x8 &dst, uint32_t addr) {
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(dst) : "v"(addr), "n"(OFF) : "memory");
}
// Transposing LDS read: within each group of 16 lanes, lane i receives element i % 4 of the
// 8-byte words read by lanes 4m + i / 4 (m = 0..3) of its group.
template <int OFF>
HILO_DEV void lds_read_tr16(bf16x4 &dst, uint32_t addr) {
  asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(dst) : "v"(addr), "n"(OFF) : "memory");
}
// Waits until at most N LDS reads of this wave are outstanding (they complete in order) and makes
// x depend on the wait, so that no use of x is scheduled above it; lds_tie orders further values.
template <int N, typename T>
HILO_DEV void lds_wait(T &x) {
  asm volatile("s_waitcnt lgkmcnt(%1)" : "+v"(x) : "n"(N) : "memory");
}
// the same with n a constant once the caller's loops are unrolled (larger n wait for all reads)
template <typename T>
HILO_DEV void lds_wait_n(int n, T &x) {
  switch (n) {
    case 8: lds_wait<8>(x); break;
    case 7: lds_wait<7>(x); break;
    case 6: lds_wait<6>(x); break;
    case 5: lds_wait<5>(x); break;
    case 4: lds_wait<4>(x); break;
    case 3: lds_wait<3>(x); break;
    case 2: lds_wait<2>(x); break;
    case 1: lds_wait<1>(x); break;
    default: lds_wait<0>(x); break;
  }
}
template <typename T>
HILO_DEV void lds_tie(T &x) {
  asm volatile("" : "+v"(x));
}

// FP8 K tile rows (head_dim bytes) keep 16-byte chunk c of row r at slot c ^ kswz8(r): the 16
// lanes reading one chunk of 16 consecutive rows hit 16 distinct bank groups (rows of 128 bytes:
// even and odd rows fall in opposite halves of the 256 banked bytes, so the 8 rows of each parity
// need 8 distinct slots; rows of 64 bytes: the 4 rows r, r + 4, r + 8, r + 12 need 4).
template <int HD>
HILO_DEV int kswz8(int r) {
  if constexpr (HD == 128) return (r >> 1) & 7;
  else return ((r >> 1) & 3) ^ ((r >> 3) & 1);
}
template <int OFF>
HILO_DEV void lds_read_b32(uint32_t &dst, uint32_t addr) {
  asm volatile("ds_read_b32 %0, %1 offset:%2" : "=v"(dst) : "v"(addr), "n"(OFF) : "memory");
}
typedef int i32x8 __attribute__((ext_vector_type(8)));

HILO_DEV void g2lds4(const void *g, void *lds_wave_base) {
  __builtin_amdgcn_global_load_lds(g, (__attribute__((address_space(3))) void *)lds_wave_base, 4, 0, 0);
}

HILO_DEV void g2lds16(const void *g, void *lds_wave_base) {
  __builtin_amdgcn_global_load_lds(g, (__attribute__((address_space(3))) void *)lds_wave_base, 16, 0, 0);
}

// Stream-K schedule of the attention core.  A unit is (sample, head, query tile of QW*NW rows);
// it takes nkv(s) = ceil(n_s / 64) key steps.  Units are ordered sample-major, then head, then
// query tile (the query tiles of one head share its keys in L2), and the P persistent workgroups
// take equal contiguous ranges of the (unit, key step) space.  A unit fully inside one range is
// finished there; a cut unit leaves per-range partial results (unnormalised O, running max m and
// sum l per query row) that k_attn_fix merges in range order: M = max m_i,
// O = sum exp2(m_i - M) O_i / sum exp2(m_i - M) l_i.
struct AttnUnit {
  int s, h, qt, nkv;
  long long start;  // first iteration of the unit
};

HILO_DEV long long attn_iterations(const int *cu, int B, int heads, int BQ) {
  long long I = 0;
  for (int s = 0; s < B; ++s) {
    const int n = cu_at(cu, s + 1) - cu_at(cu, s);
    I += (long long)heads * ((n + BQ - 1) / BQ) * ((n + 63) / 64);
  }
  return I;
}

HILO_DEV AttnUnit attn_unit(const int *cu, int B, int heads, int BQ, long long it) {
  long long base = 0;
  for (int s = 0; s < B; ++s) {
    const int n = cu_at(cu, s + 1) - cu_at(cu, s);
    const int qtiles = (n + BQ - 1) / BQ, nkv = (n + 63) / 64;
    const long long span = (long long)heads * qtiles * nkv;
    if (it < base + span) {
      const long long u = (it - base) / nkv;
      return AttnUnit{s, int(u / qtiles), int(u % qtiles), nkv, base + u * nkv};
    }
    base += span;
  }
  return AttnUnit{0, 0, 0, 1, 0};
}

struct AttnArgs {
  const uint16_t *qkv;
  const int *cu;
  uint16_t *out;
  float *part;  // partial slots: 2 per workgroup
  int B, heads;
  float scale_log2;
  // FP8 scores: row m's q and k codes at qk8 + m * ldq8 (q heads, then k heads), its E8M0 scale
  // bytes at + 2 D (q heads, then k heads); v stays bf16 in qkv
  const uint8_t *qk8;
  int ldq8;
};

template <int HD, int QW, int NW>
struct AttnShape {
  static constexpr int QS = QW / 16;
  static constexpr int DS = HD / 16;
  static constexpr int BQ = QW * NW;
  // partial slot: O (QS*DS float4 per lane) then m and l (QS floats each per lane), per wave
  static constexpr int kOFloats = NW * QS * DS * 64 * 4;
  static constexpr int kSlotFloats = kOFloats + NW * QS * 64 * 2;
  HILO_DEV static size_t o_index(int wid, int qs, int d, int lane) {
    return ((size_t(wid) * QS + qs) * DS + d) * 256 + lane * 4;
  }
  HILO_DEV static size_t ml_index(int wid, int qs, int lane) {
    return kOFloats + ((size_t(wid) * QS + qs) * 64 + lane) * 2;
  }
};

template <int HD, int QW, int NW>
HILO_DEV void attn_store_out(const AttnArgs &a, const AttnUnit &u, int wid, int lane,
                             f32x4 (&o)[QW / 16][HD / 16], const float (&l)[QW / 16]) {
  constexpr int QS = QW / 16, DS = HD / 16;
  const int lo = cu_at(a.cu, u.s), n = cu_at(a.cu, u.s + 1) - lo;
  const int D = a.heads * HD;
  const int lr = lane & 15, lg = lane >> 4;
#pragma unroll
  for (int qs = 0; qs < QS; ++qs) {
    const float inv = 1.0f / l[qs];
    const int q = u.qt * (QW * NW) + wid * QW + qs * 16 + lr;
    if (q >= n) continue;
    uint16_t *orow = a.out + size_t(lo + q) * D + size_t(u.h) * HD;
#pragma unroll
    for (int d = 0; d < DS; ++d) {
      uint2 w;
      w.x = pack_bf16x2(o[qs][d][0] * inv, o[qs][d][1] * inv);
      w.y = pack_bf16x2(o[qs][d][2] * inv, o[qs][d][3] * inv);
      *reinterpret_cast<uint2 *>(orow + d * 16 + 4 * lg) = w;
    }
  }
}

template <int HD, int QW, int NW, bool F8S>
__global__ __launch_bounds__(NW * 64, 8 / NW) void k_attn_bf16(AttnArgs a) {
  using S = AttnShape<HD, QW, NW>;
  constexpr int BKV = 64;
  constexpr int QS = S::QS;         // query subtiles per wave
  constexpr int KK = HD / 32;       // k-steps of the score MFMA
  constexpr int DS = S::DS;         // d subtiles of the output
  constexpr int BQ = S::BQ;
  constexpr int CPR = HD / 8;       // 16-byte chunks per K row
  constexpr int RPI = 64 / CPR;     // K rows per wave load instruction (1 KiB)
  constexpr int KI = BKV / RPI / NW;  // K load instructions per wave per tile
  static_assert(KI * RPI * NW == BKV, "K tile / wave mismatch");
  __shared__ __attribute__((aligned(1024))) uint16_t sK[2][F8S ? 8 : BKV * HD];
  __shared__ __attribute__((aligned(1024))) uint16_t sV[2][BKV * HD];
  // FP8 scores: the K tile's codes (head_dim bytes per key) and its keys' scale dwords
  constexpr int K8I = BKV * HD / 1024 / NW;  // 1 KiB K-code load instructions per wave per tile
  static_assert(!F8S || K8I == 1, "FP8 K tile / wave mismatch");
  constexpr int R8 = 1024 / HD;              // K-code rows per load instruction
  __shared__ __attribute__((aligned(1024))) uint8_t sK8[2][F8S ? BKV * HD : 16];
  __shared__ __attribute__((aligned(256))) uint32_t sKs[2][F8S ? BKV : 4];

  const int P = gridDim.x;
  const int pid = xcd_remap(blockIdx.x, P);
  const long long I = attn_iterations(a.cu, a.B, a.heads, BQ);
  const long long beg = I * pid / P, end = I * (pid + 1) / P;
  if (beg >= end) return;
  const long long head_start = attn_unit(a.cu, a.B, a.heads, BQ, beg).start;
  const int D = a.heads * HD;
  const size_t ld = size_t(3) * D;
  const int tid = threadIdx.x, lane = tid & 63, wid = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lr = lane & 15, lg = lane >> 4;
  const int krow = lane / CPR, kslot = lane % CPR;

  for (long long it = beg; it < end;) {
    const AttnUnit u = attn_unit(a.cu, a.B, a.heads, BQ, it);
    const int kb = int(it - u.start);
    const int ke = int(min((long long)u.nkv, (long long)kb + (end - it)));
    const int lo = cu_at(a.cu, u.s);
    const int n = cu_at(a.cu, u.s + 1) - lo;
    const int q0 = u.qt * BQ;
    const uint16_t *Q = a.qkv + size_t(lo) * ld + size_t(u.h) * HD;
    const uint16_t *Kp = Q + D;
    const uint16_t *Vp = Q + 2 * D;

    // query fragments (second MFMA operand): row q, dims kk*32 + 8*lg .. +7; FP8 scores: codes
    // 32 lg .. 32 lg + 31 of the row's head (head dim 64: lanes 32..63 hold the 128-deep MFMA's K
    // range 64..127, zero) and the row's scale byte
    bf16x8 qf[F8S ? 1 : QS][F8S ? 1 : KK];
    i32x8 qf8[QS];
    uint32_t qsc[QS];
#pragma unroll
    for (int qs = 0; qs < QS; ++qs) {
      const int q = min(q0 + wid * QW + qs * 16 + lr, n - 1);
      if constexpr (F8S) {
        const uint8_t *qr = a.qk8 + size_t(lo + q) * a.ldq8;
        const i32x8 c = *reinterpret_cast<const i32x8 *>(qr + u.h * HD + 32 * (HD == 128 ? lg : (lg & 1)));
        qf8[qs] = (HD == 128 || lg < 2) ? c : i32x8{0, 0, 0, 0, 0, 0, 0, 0};
        qsc[qs] = qr[2 * D + u.h];
      } else {
#pragma unroll
        for (int kk = 0; kk < KK; ++kk)
          qf[qs][kk] = *reinterpret_cast<const bf16x8 *>(Q + size_t(q) * ld + kk * 32 + 8 * lg);
      }
    }

    // K and V: direct global->LDS, lane -> (row wid*KI*RPI + RPI*i + lane/CPR, slot lane%CPR),
    // V's chunks placed by vsw.  A tile's address is a uniform base (key row kv0, in scalar
    // registers) plus this lane's fixed 32-bit byte offset, so the loads of a step need no vector
    // address arithmetic; only a tile reaching past the sequence end (a unit's last, at most once)
    // re-forms the offsets with the rows clamped to the last one.
    const uint32_t ldb = uint32_t(ld) * 2;  // bytes per token row
    uint32_t koff[KI], voff[KI];
#pragma unroll
    for (int i = 0; i < KI; ++i) {
      const int r = (wid * KI + i) * RPI + krow;
      koff[i] = uint32_t(r) * ldb + uint32_t((kslot ^ kswz<HD>(r)) * 16);
      voff[i] = uint32_t(r) * ldb + uint32_t((kslot ^ vsw<HD>(r)) * 16);
    }
    // FP8 scores: the K codes, lane -> (row wid*R8 + lane/(HD/16), slot lane%(HD/16)), chunks placed
    // by kswz8; wave 0 also fetches the dword holding each of the tile's 64 keys' scale byte
    const uint32_t ld8 = uint32_t(a.ldq8);
    const int r8 = wid * R8 + lane / (HD / 16);
    const uint32_t k8off = uint32_t(r8) * ld8 + uint32_t(((lane % (HD / 16)) ^ kswz8<HD>(r8)) * 16);
    const int sbyte = 2 * D + a.heads + u.h;  // the k scale byte of this head within a row
    auto issue_kv = [&](int kv0, int buf) {
      const char *kb = reinterpret_cast<const char *>(Kp) + size_t(kv0) * ldb;
      const char *vb = reinterpret_cast<const char *>(Vp) + size_t(kv0) * ldb;
      if constexpr (F8S) {
        const uint8_t *k8b = a.qk8 + size_t(lo + kv0) * a.ldq8 + D + u.h * HD;
        const bool full = kv0 + BKV <= n;
        const uint32_t back8 = full ? 0u : uint32_t(r8 - (min(kv0 + r8, n - 1) - kv0)) * ld8;  // rows re-read
        g2lds16(k8b + (k8off - back8), &sK8[buf][wid * 1024]);
        if (wid == 0)
          g2lds4(a.qk8 + size_t(lo + min(kv0 + lane, n - 1)) * a.ldq8 + (sbyte & ~3), &sKs[buf][0]);
#pragma unroll
        for (int i = 0; i < KI; ++i) {
          const int r = (wid * KI + i) * RPI + krow;
          const uint32_t back = full ? 0u : uint32_t(r - (min(kv0 + r, n - 1) - kv0)) * ldb;
          g2lds16(vb + (voff[i] - back), &sV[buf][(wid * KI + i) * RPI * HD]);
        }
        return;
      }
      if (kv0 + BKV <= n) {
#pragma unroll
        for (int i = 0; i < KI; ++i) {
          g2lds16(kb + koff[i], &sK[buf][(wid * KI + i) * RPI * HD]);
          g2lds16(vb + voff[i], &sV[buf][(wid * KI + i) * RPI * HD]);
        }
      } else {
#pragma unroll
        for (int i = 0; i < KI; ++i) {
          const int r = (wid * KI + i) * RPI + krow;
          const uint32_t back = uint32_t(r - (min(kv0 + r, n - 1) - kv0)) * ldb;  // rows re-read
          g2lds16(kb + (koff[i] - back), &sK[buf][(wid * KI + i) * RPI * HD]);
          g2lds16(vb + (voff[i] - back), &sV[buf][(wid * KI + i) * RPI * HD]);
        }
      }
    };
    // LDS byte addresses of this lane's fragments in buffer 0 (buffer 1 is kTileBytes further).
    // K (first MFMA operand) of key subtile ks, k-step kk: row ks*16 + lr, chunk kk*4 + lg; the
    // swizzle depends on lr only, so ks is an immediate offset
    constexpr uint32_t kTileBytes = BKV * HD * 2;
    const uint32_t sK0 = (uint32_t)(uintptr_t)&sK[0][0], sV0 = (uint32_t)(uintptr_t)&sV[0][0];
    uint32_t kaddr[KK];
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) kaddr[kk] = sK0 + (lr * HD + (((kk * 4 + lg) ^ kswz<HD>(lr)) * 8)) * 2;
    // FP8 K of key subtile ks: row ks*16 + lr, chunks 2 lg and 2 lg + 1 (head dim 64: lanes 32..63
    // read the chunks of lanes 0..31, real codes that meet zero query entries); kswz8 depends on lr
    // only, so ks is an immediate offset.  The scale dword of key ks*16 + lr: immediate ks * 64.
    constexpr uint32_t kTile8 = BKV * HD;
    const uint32_t sK80 = (uint32_t)(uintptr_t)&sK8[0][0], sKs0 = (uint32_t)(uintptr_t)&sKs[0][0];
    const int lg8 = HD == 128 ? lg : (lg & 1);
    const uint32_t k8a0 = sK80 + lr * HD + (((2 * lg8) ^ kswz8<HD>(lr)) * 16);
    const uint32_t k8a1 = sK80 + lr * HD + (((2 * lg8 + 1) ^ kswz8<HD>(lr)) * 16);
    const int ssh = (sbyte & 3) * 8;
    // V^T of output subtile d: lane (g = lg, s = lr) reads dims d*16 + 4 (s % 4) .. +3 of key rows
    // 32 kk2 + 4 g + s / 4 and 16 rows further (the transpose gives lane s dim d*16 + s of those 8
    // keys); the swizzle of those rows depends on lane bits only, so kk2 and the +16 rows are
    // immediate offsets
    uint32_t vaddr[DS];
    {
      const int r1 = 4 * lg + (lr >> 2);
#pragma unroll
      for (int d = 0; d < DS; ++d) {
        const int c = 2 * d + ((lr & 3) >> 1);
        vaddr[d] = sV0 + (r1 * HD + ((c ^ vsw<HD>(r1)) << 3) + (lr & 1) * 4) * 2;
      }
    }
    // (the key subtile is the instruction's immediate offset)
    auto read_k = [&](const uint32_t (&kb)[KK], int ks, bf16x8 (&kf)[KK]) {
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) {
        switch (ks) {
          case 0: lds_read_b128<0>(kf[kk], kb[kk]); break;
          case 1: lds_read_b128<16 * HD * 2>(kf[kk], kb[kk]); break;
          case 2: lds_read_b128<32 * HD * 2>(kf[kk], kb[kk]); break;
          default: lds_read_b128<48 * HD * 2>(kf[kk], kb[kk]); break;
        }
      }
    };
    // two 8-byte halves per k-step: [kk2][0] rows r1, [kk2][1] rows r1 + 16
    auto read_v = [&](uint32_t boff, int d, bf16x4 (&vh)[2][2]) {
      const uint32_t ad = vaddr[d] + boff;
      lds_read_tr16<0>(vh[0][0], ad);
      lds_read_tr16<16 * HD * 2>(vh[0][1], ad);
      lds_read_tr16<32 * HD * 2>(vh[1][0], ad);
      lds_read_tr16<48 * HD * 2>(vh[1][1], ad);
    };

    f32x4 o[QS][DS];
#pragma unroll
    for (int qs = 0; qs < QS; ++qs)
#pragma unroll
      for (int d = 0; d < DS; ++d) o[qs][d] = f32x4{0.f, 0.f, 0.f, 0.f};
    // running reference maximum (scaled, base 2) and the row sums of P, accumulated by the MFMA
    // against a fragment of ones (every lane gets its query's full sum over the 32 keys of a
    // k-step, of the same bf16-rounded probabilities that weight V)
    float mrun[QS];
    f32x4 lacc[QS];
#pragma unroll
    for (int qs = 0; qs < QS; ++qs) { mrun[qs] = -INFINITY; lacc[qs] = f32x4{0.f, 0.f, 0.f, 0.f}; }
    bf16x8 ones;
#pragma unroll
    for (int e = 0; e < 8; ++e) ones[e] = static_cast<__bf16>(1.0f);

    // one 64-key step; keys >= n exist only in a unit's last step, the only one that masks.  The
    // next tile's transfer (into the buffer every wave left at the last barrier) starts first.
    auto step = [&](int buf, int kv0, bool mask, auto &&prefetch) {
      prefetch();
      const uint32_t boff = buf ? kTileBytes : 0u;
      uint32_t kb[KK];
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) kb[kk] = kaddr[kk] + boff;
      // S^T for 64 keys x QW queries: sc[ks][qs][e] = score(query qs*16+lr, key ks*16+4*lg+e);
      // K fragments are read one key subtile ahead of the MFMAs that use them
      f32x4 sc[4][QS];
#pragma unroll
      for (int ks = 0; ks < 4; ++ks)
#pragma unroll
        for (int qs = 0; qs < QS; ++qs) sc[ks][qs] = f32x4{0.f, 0.f, 0.f, 0.f};
      if constexpr (F8S) {
        // one 128-deep FP8 MFMA per (key subtile, query subtile); the E8M0 scales of the lane's key
        // row and query row scale the product in the matrix core
        const uint32_t b8 = buf ? kTile8 : 0u;
        const uint32_t sa = sKs0 + (buf ? BKV * 4 : 0) + lr * 4;
        uint32_t kw[4];
        lds_read_b32<0>(kw[0], sa);
        lds_read_b32<64>(kw[1], sa);
        lds_read_b32<128>(kw[2], sa);
        lds_read_b32<192>(kw[3], sa);
        bf16x8 kh[2][2];  // the two 16-byte halves of a 32-byte FP8 fragment
        auto read_k8 = [&](int ks, bf16x8 (&h)[2]) {
          switch (ks) {
            case 0: lds_read_b128<0>(h[0], k8a0 + b8); lds_read_b128<0>(h[1], k8a1 + b8); break;
            case 1: lds_read_b128<16 * HD>(h[0], k8a0 + b8); lds_read_b128<16 * HD>(h[1], k8a1 + b8); break;
            case 2: lds_read_b128<32 * HD>(h[0], k8a0 + b8); lds_read_b128<32 * HD>(h[1], k8a1 + b8); break;
            default: lds_read_b128<48 * HD>(h[0], k8a0 + b8); lds_read_b128<48 * HD>(h[1], k8a1 + b8); break;
          }
        };
        read_k8(0, kh[0]);
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
          if (ks + 1 < 4) read_k8(ks + 1, kh[(ks + 1) & 1]);
          lds_wait_n(ks + 1 < 4 ? 2 : 0, kh[ks & 1][1]);
          lds_tie(kh[ks & 1][0]);
          if (ks == 0) {  // the scale reads went first: complete with the first K fragment
            lds_tie(kw[0]); lds_tie(kw[1]); lds_tie(kw[2]); lds_tie(kw[3]);
          }
          const i32x8 kf = __builtin_bit_cast(i32x8, __builtin_shufflevector(kh[ks & 1][0], kh[ks & 1][1], 0, 1, 2, 3, 4, 5, 6, 7, 8, 9, 10, 11, 12, 13, 14, 15));
          const int ksc = int((kw[ks] >> ssh) & 0xffu);
#pragma unroll
          for (int qs = 0; qs < QS; ++qs)
            sc[ks][qs] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(kf, qf8[qs], sc[ks][qs], 0, 0, 0, ksc, 0, int(qsc[qs]));
        }
      } else {
        bf16x8 kf[2][KK];
        read_k(kb, 0, kf[0]);
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
          if (ks + 1 < 4) read_k(kb, ks + 1, kf[(ks + 1) & 1]);
#pragma unroll
          for (int kk = 0; kk < KK; ++kk) {
            lds_wait_n((KK - 1 - kk) + (ks + 1 < 4 ? KK : 0), kf[ks & 1][kk]);
#pragma unroll
            for (int qs = 0; qs < QS; ++qs)
              sc[ks][qs] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[ks & 1][kk], qf[qs][kk], sc[ks][qs], 0, 0, 0);
          }
        }
      }
      // the first two V^T subtiles load while the softmax runs, later ones two subtiles ahead
      bf16x4 vh[3][2][2];
      read_v(boff, 0, vh[0]);
      read_v(boff, 1, vh[1]);
      if (mask) {
#pragma unroll
        for (int ks = 0; ks < 4; ++ks)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (kv0 + ks * 16 + 4 * lg + e >= n)
#pragma unroll
              for (int qs = 0; qs < QS; ++qs) sc[ks][qs][e] = -INFINITY;
      }
      bf16x8 pf[QS][2];
#pragma unroll
      for (int qs = 0; qs < QS; ++qs) {
        float m4[4];
#pragma unroll
        for (int ks = 0; ks < 4; ++ks)
          m4[ks] = fmaxf(fmaxf(sc[ks][qs][0], sc[ks][qs][1]), fmaxf(sc[ks][qs][2], sc[ks][qs][3]));
        const float mt = xmax16_32(fmaxf(fmaxf(m4[0], m4[1]), fmaxf(m4[2], m4[3]))) * a.scale_log2;
        // The reference maximum moves only when some row's tile maximum exceeds it by more than
        // kLazyRescale: O and l share it, so the result does not depend on it, and the
        // probabilities stay below 2^kLazyRescale
        if (__any(mt > mrun[qs] + kLazyRescale)) {
          const float mnew = fmaxf(mrun[qs], mt);
          const float alpha = __builtin_amdgcn_exp2f(mrun[qs] - mnew);
          lacc[qs] *= alpha;
#pragma unroll
          for (int d = 0; d < DS; ++d) o[qs][d] *= alpha;
          mrun[qs] = mnew;
        }
#pragma unroll
        for (int kk2 = 0; kk2 < 2; ++kk2) {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            pf[qs][kk2][e] =
                static_cast<__bf16>(__builtin_amdgcn_exp2f(fmaf(sc[2 * kk2][qs][e], a.scale_log2, -mrun[qs])));
            pf[qs][kk2][4 + e] =
                static_cast<__bf16>(__builtin_amdgcn_exp2f(fmaf(sc[2 * kk2 + 1][qs][e], a.scale_log2, -mrun[qs])));
          }
          lacc[qs] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, pf[qs][kk2], lacc[qs], 0, 0, 0);
        }
      }
      // O^T += V^T P^T
#pragma unroll
      for (int d = 0; d < DS; ++d) {
        if (d + 2 < DS) read_v(boff, d + 2, vh[(d + 2) % 3]);
        bf16x4 (&h)[2][2] = vh[d % 3];
        lds_wait_n(4 * (d + 2 < DS ? 2 : DS - 1 - d), h[1][1]);
        lds_tie(h[0][0]);
        lds_tie(h[0][1]);
        lds_tie(h[1][0]);
#pragma unroll
        for (int kk2 = 0; kk2 < 2; ++kk2) {
          const bf16x8 vf = __builtin_shufflevector(h[kk2][0], h[kk2][1], 0, 1, 2, 3, 4, 5, 6, 7);
#pragma unroll
          for (int qs = 0; qs < QS; ++qs)
            o[qs][d] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pf[qs][kk2], o[qs][d], 0, 0, 0);
        }
      }
    };

    issue_kv(kb * BKV, 0);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    // all steps but the last load the next tile unconditionally and never mask: no branch splits
    // the loop body's schedule
    for (int kt = kb; kt < ke - 1; ++kt) {
      const int buf = (kt - kb) & 1;
      step(buf, kt * BKV, false, [&]() { issue_kv((kt + 1) * BKV, buf ^ 1); });
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      __syncthreads();
    }
    step((ke - 1 - kb) & 1, (ke - 1) * BKV, (ke - 1) * BKV + BKV > n, [] {});
    __syncthreads();

    float lsum[QS];
#pragma unroll
    for (int qs = 0; qs < QS; ++qs) lsum[qs] = lacc[qs][0];
    if (kb == 0 && ke == u.nkv) {
      attn_store_out<HD, QW, NW>(a, u, wid, lane, o, lsum);
    } else {
      float *slot = a.part + (size_t(pid) * 2 + (u.start == head_start ? 0 : 1)) * S::kSlotFloats;
#pragma unroll
      for (int qs = 0; qs < QS; ++qs) {
#pragma unroll
        for (int d = 0; d < DS; ++d)
          *reinterpret_cast<f32x4 *>(slot + S::o_index(wid, qs, d, lane)) = o[qs][d];
        *reinterpret_cast<float2 *>(slot + S::ml_index(wid, qs, lane)) = make_float2(mrun[qs], lsum[qs]);
      }
    }
    it += ke - kb;
  }
}

// Merges every unit cut by range boundaries; run by the range holding the unit's first key step.
template <int HD, int QW, int NW>
__global__ __launch_bounds__(NW * 64) __attribute__((amdgpu_waves_per_eu(2, 2))) void k_attn_fix(AttnArgs a) {
  using S = AttnShape<HD, QW, NW>;
  constexpr int QS = S::QS, DS = S::DS, BQ = S::BQ;
  const int P = gridDim.x;
  const int pid = blockIdx.x;
  const long long I = attn_iterations(a.cu, a.B, a.heads, BQ);
  const long long beg = I * pid / P, end = I * (pid + 1) / P;
  if (beg >= end) return;
  const AttnUnit u = attn_unit(a.cu, a.B, a.heads, BQ, end - 1);
  const long long ue = u.start + u.nkv;
  if (end >= ue) return;      // the unit ends inside this range: not cut here
  if (beg > u.start) return;  // this range does not hold the unit's first step
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;

  f32x4 o[QS][DS];
  float m[QS], l[QS];
#pragma unroll
  for (int qs = 0; qs < QS; ++qs) {
    m[qs] = -INFINITY;
    l[qs] = 0.f;
#pragma unroll
    for (int d = 0; d < DS; ++d) o[qs][d] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  // one contributor's partial: (m, l) per query subtile and the unnormalised O
  struct Part {
    float2 ml[QS];
    f32x4 o[QS][DS];
  };
  auto load = [&](const float *slot, Part &c) __attribute__((always_inline)) {
#pragma unroll
    for (int qs = 0; qs < QS; ++qs) {
      c.ml[qs] = *reinterpret_cast<const float2 *>(slot + S::ml_index(wid, qs, lane));
#pragma unroll
      for (int d = 0; d < DS; ++d) c.o[qs][d] = *reinterpret_cast<const f32x4 *>(slot + S::o_index(wid, qs, d, lane));
    }
  };
  auto merge = [&](const Part &c) __attribute__((always_inline)) {
#pragma unroll
    for (int qs = 0; qs < QS; ++qs) {
      const float mn = fmaxf(m[qs], c.ml[qs].x);
      const float ca = __builtin_amdgcn_exp2f(m[qs] - mn), cb = __builtin_amdgcn_exp2f(c.ml[qs].x - mn);
      l[qs] = l[qs] * ca + c.ml[qs].y * cb;
#pragma unroll
      for (int d = 0; d < DS; ++d) o[qs][d] = o[qs][d] * ca + c.o[qs][d] * cb;
      m[qs] = mn;
    }
  };
  // contributor ranges [b, e) in order; their starts floor(I q / P) advance by additions.  They are
  // merged in that order, two at a time: both partials' loads are in flight together
  const float *pend = nullptr;
  const long long qI = I / P, rI = I - qI * P;
  long long b = beg, r = I * pid - beg * P;
  for (int q = pid; q < P; ++q) {
    long long e = b + qI, rn = r + rI;
    if (rn >= P) {
      ++e;
      rn -= P;
    }
    const long long bq = b, eq = e;
    b = e;
    r = rn;
    if (bq >= eq) continue;
    if (bq >= ue) break;
    // slot 0 holds the partial of the range's first unit, slot 1 of its last
    const float *slot = a.part + (size_t(q) * 2 + (bq >= u.start ? 0 : 1)) * S::kSlotFloats;
    if (pend == nullptr) {
      pend = slot;
    } else {
      Part c0, c1;
      load(pend, c0);
      load(slot, c1);
      merge(c0);
      merge(c1);
      pend = nullptr;
    }
    if (eq >= ue) break;
  }
  if (pend != nullptr) {
    Part c0;
    load(pend, c0);
    merge(c0);
  }
  attn_store_out<HD, QW, NW>(a, u, wid, lane, o, l);
}

// fp32 path: one thread per query row, keys/values staged through LDS 32 rows at a time.
template <int HD>
__global__ __launch_bounds__(64) void k_attn_f32(const float *__restrict__ qkv,
                                                 const int *__restrict__ cu, float *__restrict__ out,
                                                 int heads, int qtiles, float scale_log2) {
  constexpr int BKV = 32;
  __shared__ float sK[BKV][HD];
  __shared__ float sV[BKV][HD];
  const int qt = blockIdx.x % qtiles;
  const int sh = blockIdx.x / qtiles;
  const int h = sh % heads, s = sh / heads;
  const int lo = cu[s], n = cu[s + 1] - lo;
  const int q0 = qt * 64;
  if (q0 >= n) return;
  const int D = heads * HD;
  const size_t ld = size_t(3) * D;
  const int q = min(q0 + int(threadIdx.x), n - 1);
  float qv[HD], o[HD];
  for (int d = 0; d < HD; ++d) { qv[d] = qkv[size_t(lo + q) * ld + h * HD + d]; o[d] = 0.f; }
  float m = -INFINITY, l = 0.f;
  for (int kv0 = 0; kv0 < n; kv0 += BKV) {
    __syncthreads();
    for (int e = threadIdx.x; e < BKV * HD; e += 64) {
      const int r = e / HD, d = e % HD;
      const int row = min(kv0 + r, n - 1);
      sK[r][d] = qkv[size_t(lo + row) * ld + D + h * HD + d];
      sV[r][d] = qkv[size_t(lo + row) * ld + 2 * D + h * HD + d];
    }
    __syncthreads();
    const int nk = min(BKV, n - kv0);
    for (int r = 0; r < nk; ++r) {
      float sdot = 0.f;
      for (int d = 0; d < HD; ++d) sdot += qv[d] * sK[r][d];
      const float x = sdot * scale_log2;
      const float mnew = fmaxf(m, x);
      const float alpha = exp2f(m - mnew);
      const float p = exp2f(x - mnew);
      l = l * alpha + p;
      for (int d = 0; d < HD; ++d) o[d] = o[d] * alpha + p * sV[r][d];
      m = mnew;
    }
  }
  if (q0 + int(threadIdx.x) < n) {
    const float inv = 1.0f / l;
    for (int d = 0; d < HD; ++d) out[size_t(lo + q) * D + h * HD + d] = o[d] * inv;
  }
}

// Persistent workgroups of the bf16 core: per_cu on every CU, capped so that their two partial
// slots each (slot_floats) fit the partial area of the workspace.
int attn_workgroups(int per_cu, size_t slot_floats) {
  static int ncu[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) dev = 0;
  if (ncu[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
      n = kAttnMaxWorkgroups / 2;
    ncu[dev] = n;
  }
  const int cap = int(kAttnPartBytes / (2 * slot_floats * sizeof(float)));
  const int p = per_cu * ncu[dev];
  return p < cap ? p : cap;
}

template <int HD, int QW, int NW>
static hipError_t run_attn_bf16(const void *qkv, const int *cu, void *out, float *part, int B,
                                int heads, const uint8_t *qk8, int ldq8, hipStream_t st) {
  using S = AttnShape<HD, QW, NW>;
  static_assert(S::kSlotFloats <= 2 * kAttnSlotFloats, "partial slot too large for the workspace");
  AttnArgs a{reinterpret_cast<const uint16_t *>(qkv), cu, reinterpret_cast<uint16_t *>(out), part, B,
             heads, kLog2e / sqrtf(float(HD)), qk8, ldq8};
  // 4 waves: two workgroups per CU; 8 waves: one (two waves per SIMD either way)
  const int P = attn_workgroups(NW == 8 ? 1 : 2, S::kSlotFloats);
  if (qk8) hipLaunchKernelGGL((k_attn_bf16<HD, QW, NW, true>), dim3(P), dim3(NW * 64), 0, st, a);
  else hipLaunchKernelGGL((k_attn_bf16<HD, QW, NW, false>), dim3(P), dim3(NW * 64), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((k_attn_fix<HD, QW, NW>), dim3(P), dim3(NW * 64), 0, st, a);
  return hipGetLastError();
}

template <int HD>
static hipError_t run_attn_f32(const void *qkv, const int *cu, void *out, int B, int heads,
                               int max_seq, hipStream_t st) {
  const int qtiles = (max_seq + 63) / 64;
  const long long nblk = (long long)B * heads * qtiles;
  if (nblk <= 0) return hipSuccess;
  const float sl2 = kLog2e / sqrtf(float(HD));
  hipLaunchKernelGGL((k_attn_f32<HD>), dim3(unsigned(nblk)), dim3(64), 0, st,
                     reinterpret_cast<const float *>(qkv), cu, reinterpret_cast<float *>(out),
                     heads, qtiles, sl2);
  return hipGetLastError();
}

size_t attention_part_bytes(bool bf16, int hd) {
  if (!bf16) return 0;
  const size_t slot = hd == 128 ? AttnShape<128, 32, 8>::kSlotFloats : AttnShape<64, 32, 4>::kSlotFloats;
  return size_t(2) * attn_workgroups(hd == 128 ? 1 : 2, slot) * slot * sizeof(float);
}

hipError_t launch_attention(bool bf16, const void *qkv, const int *cu, void *out, float *part, int B,
                            int heads, int hd, int max_seq, hipStream_t st, const uint8_t *qk8, int ldq8) {
  if (bf16) {
    if (hd == 128) return run_attn_bf16<128, 32, 8>(qkv, cu, out, part, B, heads, qk8, ldq8, st);
    return run_attn_bf16<64, 32, 4>(qkv, cu, out, part, B, heads, qk8, ldq8, st);
  }
  if (hd == 128) return run_attn_f32<128>(qkv, cu, out, B, heads, max_seq, st);
  return run_attn_f32<64>(qkv, cu, out, B, heads, max_seq, st);
}

}  // namespace hilo
