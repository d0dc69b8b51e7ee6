// Projections of the block (QKV, attention output, MLP up and down): C = A W^T on the ragged
// packed sequence, image rows with the image-stream weights and text rows with the text-stream
// weights, tiles never straddling a segment.  Epilogues fuse the bias, the tanh-GELU, and the
// gated residual update of the float32 stream z; for the FP8 block's QKV projection, the q and k
// columns leave as E4M3 codes with a power-of-two scale per (row, head).
//
// bf16 and FP8 paths: one MFMA kernel (k_gemm_big), one persistent workgroup per CU with 4 waves,
// 192 x 192 tiles (every projection but the FP8 QKV) or 256 x 256 (the FP8 QKV, which writes FP8
// q / k with one scale per row and head: a wave's 128 columns hold whole heads) as
// 32 x 32 MFMA blocks (v_mfma_f32_32x32x16_bf16, or v_mfma_f32_32x32x64_f8f6f4 on E4M3 codes),
// fp32 accumulators in AGPRs, K in 64-byte stages through a 4-slot LDS ring filled by direct
// global->LDS loads (192 x 192 tiles: 128-byte K-step windows, both stages of a row's K step
// together, through a 3-slot ring).  Whole data-parallel waves of tiles run first, then a stream-K remainder;
// cut tiles leave fp32 partials that k_gemm_fix adds in a fixed order before the epilogue.
// float32 path: a plain LDS-tiled FMA kernel for the small float32 workloads.
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace hilo {

// tanh-approximated GELU, 0.5 u (1 + tanh(y)) with y = sqrt(2/pi) (u + 0.044715 u^3), evaluated
// through the identity 0.5 (1 + tanh(y)) = 1 / (1 + exp(-2y)): one hardware exp2 and one
// reciprocal (about one ulp each) instead of a full tanh.  Very negative u gives exp2 -> inf and
// the result -0; very positive u gives exp2 -> 0 and the result u.
HILO_DEV float gelu_tanh(float u) {
  constexpr float c = -2.0f * 0.7978845608028654f * 1.4426950408889634f;  // -2 sqrt(2/pi) log2(e)
  const float t = c * u * (1.0f + 0.044715f * u * u);
  return u * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(t));
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

// One 16-byte global load per lane straight into LDS: lane l of the wave lands at byte 16*l of
// the wave's 1 KiB destination (the destination base is uniform, held in M0).
HILO_DEV void g2lds16(const void *g, void *lds_wave_base) {
  __builtin_amdgcn_global_load_lds(g, (__attribute__((address_space(3))) void *)lds_wave_base, 16, 0, 0);
}

// Active row tiles of the ragged problem: per sample, ceil(image rows / BM) image tiles then
// ceil(L / BM) text tiles.  Only the device knows the row counts, so every workgroup walks the
// (few) segments itself.
HILO_DEV int row_tiles_total(const GemmProblem &p, int BM) {
  int R = 0;
  for (int s = 0; s < p.B; ++s) {
    const int nimg = cu_at(p.cu, s + 1) - p.L - cu_at(p.cu, s);
    R += (nimg + BM - 1) / BM + (p.L + BM - 1) / BM;
  }
  return R;
}

HILO_DEV TileRows decode_row_tile(const GemmProblem &p, int BM, int r) {
  TileRows tr{0, 0, 0, 0};
  for (int s = 0; s < p.B; ++s) {
    const int lo = cu_at(p.cu, s), hi = cu_at(p.cu, s + 1), ts = hi - p.L;
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

// Schedule of the bf16 projections over P persistent workgroups (one per CU).  A unit is one
// K piece of one output tile: tiles are cut into s pieces when there are fewer tiles than
// workgroups (s = ceil(P / tiles), at most one K step per piece), else s = 1.  Units are ordered
// piece-major, row tile fastest within a piece.  The first floor(U / P) * P units run
// data-parallel in whole waves -- the workgroups of an XCD then work on neighbouring tiles at the
// same K step, so its L2 serves each weight and activation slice to all of them.  The
// remaining units (all of the same K length) are spread evenly over the P workgroups stream-K,
// so no CU idles through a partial last wave.  A unit not finished in one place leaves an fp32
// partial tile (data-parallel unit u: slot u; stream-K range of workgroup w: slots P + 2w for its
// first unit and P + 2w + 1 for its second); k_gemm_fix adds the partials of each such tile in a
// fixed order and runs the epilogue -- deterministic, and no workgroup ever waits for another.
struct SkPlan {
  int R, TN, T, nk;  // row tiles, column tiles, tiles, K steps
  int s, U, dp;    // pieces per tile, units, data-parallel units
  int len;         // K steps of a stream-K unit
  long long I;     // stream-K iterations
  int Pk;          // workgroups sharing them (0 .. Pk-1; the others get empty ranges)
};

// A problem with fewer tiles than workgroups and at most this many K steps runs one whole tile per
// workgroup (some CUs idle) instead of cutting tiles into K pieces: for short K the partial tiles
// and their fixup cost more than the idle CUs.
constexpr int kNoSplitSteps = 64;

// Stream-K ranges hold at least this many K steps: every range cut leaves a partial tile (256 KiB
// at 256 x 256) that the fixup reads back, so a short tail goes to fewer workgroups.
constexpr int kSkMinSteps = 12;

HILO_DEV SkPlan sk_plan(const GemmProblem &p, int BM, int BN, int P, int kstep = 64) {
  SkPlan q;
  q.R = row_tiles_total(p, BM);
  q.TN = (p.N + BN - 1) / BN;
  q.T = q.R * q.TN;
  q.nk = p.K / kstep;
  // a stream-K tail costs a partial tile (144 or 256 KiB) per piece; when the last wave holds at
  // least half of P tiles, whole tiles in ceil(T / P) waves finish sooner
  const bool whole_waves = q.T >= P && 2 * (q.T % P) >= P;
  // a single wave that fills at least 7/8 of the workgroups also runs whole tiles (cutting K would
  // add a partial per tile to save at most an eighth)
  const bool full_wave = q.T < P && 8 * q.T >= 7 * P;
  if ((q.T < P && q.nk <= kNoSplitSteps) || whole_waves || full_wave) {
    q.s = 1;
    q.U = q.dp = q.T;
    q.len = q.nk;
    q.I = 0;
    q.Pk = P;
    return q;
  }
  q.s = (q.T >= P || q.T == 0) ? 1 : min((P + q.T - 1) / q.T, q.nk);
  q.U = q.T * q.s;
  q.dp = q.U / P * P;
  // the stream-K units all lie in the last piece (or every piece is one K step long)
  const int tail = q.U - q.dp;
  const int pc = tail > 0 ? q.dp / q.T : 0;
  q.len = (pc + 1) * q.nk / q.s - pc * q.nk / q.s;
  q.I = (long long)tail * q.len;
  // at least one workgroup per tail unit, so no range is longer than a unit and a range touches at
  // most two units (the two partial slots of its workgroup)
  q.Pk = int(min((long long)P, max((long long)tail, (q.I + kSkMinSteps - 1) / kSkMinSteps)));
  return q;
}

struct SkRange {
  long long beg, end;
};

HILO_DEV SkRange sk_range(long long I, int P, int w) {
  return SkRange{I * w / P, I * (w + 1) / P};
}

// Workgroup w's stream-K range under plan q (empty past the plan's Pk workgroups).
HILO_DEV SkRange sk_range(const SkPlan &q, int w) {
  return w < q.Pk ? sk_range(q.I, q.Pk, w) : SkRange{q.I, q.I};
}

// The workgroup whose stream-K range holds iteration a.
HILO_DEV int sk_owner(long long I, int P, long long a) { return int(((a + 1) * P - 1) / I); }

HILO_DEV int piece_k0(const SkPlan &q, int piece) { return piece * q.nk / q.s; }

// Tile t -> (row tile, column tile): groups of kTileGroupRows row tiles by all column tiles, row
// tile fastest within a group, so one XCD's 32 workgroups of a wave (consecutive ids, xcd_remap)
// cover 8 row tiles by 4 column tiles: 12 operand slices per K step, the least any 32 tiles need,
// instead of 18 in plain row-fastest order over 15 row tiles.
constexpr int kTileGroupRows = 8;

HILO_DEV void tile_coords(const SkPlan &q, int t, int &r, int &tn) {
  const int grp = t / (kTileGroupRows * q.TN), in = t - grp * (kTileGroupRows * q.TN);
  const int gm = min(kTileGroupRows, q.R - grp * kTileGroupRows);
  r = grp * kTileGroupRows + in % gm;
  tn = in / gm;
}

// Work items of one workgroup, in order: its data-parallel units (u = pid, pid + P, ...), then the
// pieces of its stream-K range.  An item is (tile, 64-deep K steps [kb, ke), partial slot or null
// for a tile finished here).
struct SkItem {
  int t, kb, ke;
  float *slot;
  bool valid;
};

struct SkCursor {
  int u;          // next data-parallel unit
  long long it;   // next stream-K iteration
};

HILO_DEV SkItem sk_next_item(SkCursor &c, const SkPlan &q, const SkRange &rg, int P, int pid, float *part,
                             size_t part_floats) {
  SkItem x{0, 0, 0, nullptr, false};
  if (c.u < q.dp) {
    const int pc = c.u / q.T;
    x.t = c.u - pc * q.T;
    x.kb = piece_k0(q, pc);
    x.ke = piece_k0(q, pc + 1);
    x.slot = q.s == 1 ? nullptr : part + size_t(c.u) * part_floats;
    x.valid = true;
    c.u += P;
  } else if (c.it < rg.end) {
    const long long v = c.it / q.len;
    const int k0 = int(c.it - v * q.len);
    const int k1 = int(min((long long)q.len, k0 + (rg.end - c.it)));
    const int uu = q.dp + int(v);
    const int pc = uu / q.T;
    x.t = uu - pc * q.T;
    x.kb = piece_k0(q, pc) + k0;
    x.ke = piece_k0(q, pc) + k1;
    const bool whole = q.s == 1 && k0 == 0 && k1 == q.len;
    x.slot = whole ? nullptr : part + (size_t(P) + size_t(pid) * 2 + (c.it == rg.beg ? 0 : 1)) * part_floats;
    x.valid = true;
    c.it += k1 - k0;
  }
  return x;
}

// Partial tiles of a BM x BN tile on WM x WN waves, in the 16 x 16 fragment order the fixup
// reads, and the fixup's epilogue of one fragment row.
template <int BM, int BN, int WM, int WN>
struct SkTile {
  static constexpr int NW = WM * WN;
  static constexpr int TM = BM / WM / 16;
  static constexpr int TN = BN / WN / 16;
  static constexpr size_t kPartFloats = size_t(BM) * BN;

  // partial-sum slot layout: register order, one float4 per lane per (wave, i, j)
  HILO_DEV static size_t part_index(int wid, int i, int j, int lane) {
    return ((size_t(wid) * TM * TN + i * TN + j) * 64 + lane) * 4;
  }

  // The FP8 q / k codes of fragment row i0 of wave wid (the whole-tile form is big_epilogue_qk8):
  // the wave's BN / WN columns hold whole heads; a row's columns of one head are spread over the 4
  // lanes l % 16 + 16 m, each holding 4 columns of every 16.
  HILO_DEV static void epilogue_rows_qk8(const GemmProblem &p, const TileRows &tr, int n0, int wid, int i0,
                                         int lane, const f32x4 (&acc)[1][TN]) {
    const int rl = (wid / WN) * (BM / WM) + i0 * 16 + (lane & 15);
    const int wc0 = n0 + (wid % WN) * (BN / WN);
    const int cbase = wc0 + 4 * (lane >> 4);
    const int hd = p.head_dim, jph = hd / 16;  // fragment columns per head
    const uint16_t *bias = reinterpret_cast<const uint16_t *>(p.bias[tr.sigma]);
    const float *ws = tr.sigma ? p.w_scale[1] : p.w_scale[0];
    const float asc = p.a_scale[tr.row0 + min(rl, tr.nrows - 1)];
    float v[TN][4];
    float am0 = 0.f, am1 = 0.f;
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int nc = cbase + j * 16;
      const uint2 bu = *reinterpret_cast<const uint2 *>(bias + nc);
      const float4 wsc = *reinterpret_cast<const float4 *>(ws + nc);
      const float b[4] = {__uint_as_float(bu.x << 16), __uint_as_float(bu.x & 0xffff0000u),
                          __uint_as_float(bu.y << 16), __uint_as_float(bu.y & 0xffff0000u)};
      v[j][0] = acc[0][j][0] * (asc * wsc.x) + b[0];
      v[j][1] = acc[0][j][1] * (asc * wsc.y) + b[1];
      v[j][2] = acc[0][j][2] * (asc * wsc.z) + b[2];
      v[j][3] = acc[0][j][3] * (asc * wsc.w) + b[3];
      const float m = fmaxf(fmaxf(fabsf(v[j][0]), fabsf(v[j][1])), fmaxf(fabsf(v[j][2]), fabsf(v[j][3])));
      if (j / jph == 0) am0 = fmaxf(am0, m);
      else am1 = fmaxf(am1, m);
    }
    am0 = fmaxf(am0, __shfl_xor(am0, 16, 64));
    am0 = fmaxf(am0, __shfl_xor(am0, 32, 64));
    am1 = fmaxf(am1, __shfl_xor(am1, 16, 64));
    am1 = fmaxf(am1, __shfl_xor(am1, 32, 64));
    const int k0 = pow2_exponent(am0), k1 = pow2_exponent(am1);
    const float inv0 = pow2_inverse(k0), inv1 = pow2_inverse(k1);
    if (rl >= tr.nrows) return;
    uint8_t *row = p.qk8 + size_t(tr.row0 + rl) * p.ldq8;
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const float s = j / jph == 0 ? inv0 : inv1;
      *reinterpret_cast<uint32_t *>(row + cbase + j * 16) = fp8x4(v[j][0] * s, v[j][1] * s, v[j][2] * s, v[j][3] * s);
    }
    if ((lane >> 4) == 0) {
      row[2 * p.D + wc0 / hd] = uint8_t(127 + k0);
      if (jph * 2 == TN) row[2 * p.D + wc0 / hd + 1] = uint8_t(127 + k1);
    }
  }

  // Epilogue of fragment rows i0 .. i0 + ROWS - 1 of wave wid (each fragment: 4 consecutive
  // columns of one row).  Every load the epilogue needs (bias, gate, the old z) is issued before
  // the first store: the compiler cannot prove that the outputs do not alias the inputs, so an
  // interleaved order would serialise one memory round trip per fragment.  Loads use indices
  // clamped into the tile; values for rows or columns outside it are never stored.
  template <int EPI, int ROWS, bool F8 = false>
  HILO_DEV static void epilogue_rows(const GemmProblem &p, const TileRows &tr, int n0, int wid, int i0,
                                     int lane, const f32x4 (&acc)[ROWS][TN]) {
    const int rbase = (wid / WN) * (BM / WM) + i0 * 16 + (lane & 15);
    const int cbase = n0 + (wid % WN) * (BN / WN) + 4 * (lane >> 4);
    const uint16_t *bias = reinterpret_cast<const uint16_t *>(p.bias[tr.sigma]);
    float bv[TN][4];
    float4 gt[TN];
    float4 zv[ROWS][TN];
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int nc = min(cbase + j * 16, p.N - 4);
      const uint2 bu = *reinterpret_cast<const uint2 *>(bias + nc);
      bv[j][0] = __uint_as_float(bu.x << 16); bv[j][1] = __uint_as_float(bu.x & 0xffff0000u);
      bv[j][2] = __uint_as_float(bu.y << 16); bv[j][3] = __uint_as_float(bu.y & 0xffff0000u);
      if constexpr (EPI == EPI_RESID)
        gt[j] = *reinterpret_cast<const float4 *>(p.mod + (size_t(tr.s * 2 + tr.sigma) * 6 + p.gate_idx) * p.D + nc);
    }
    float4 wsc[TN];
    float asc[ROWS];
    if constexpr (F8) {
      const float *ws = tr.sigma ? p.w_scale[1] : p.w_scale[0];
#pragma unroll
      for (int j = 0; j < TN; ++j) wsc[j] = *reinterpret_cast<const float4 *>(ws + min(cbase + j * 16, p.N - 4));
#pragma unroll
      for (int i = 0; i < ROWS; ++i) asc[i] = p.a_scale[tr.row0 + min(rbase + i * 16, tr.nrows - 1)];
    }
    if constexpr (EPI == EPI_RESID) {
#pragma unroll
      for (int i = 0; i < ROWS; ++i) {
        const size_t m = size_t(tr.row0 + min(rbase + i * 16, tr.nrows - 1));
#pragma unroll
        for (int j = 0; j < TN; ++j)
          zv[i][j] = *reinterpret_cast<const float4 *>(p.z + m * p.ldz + min(cbase + j * 16, p.N - 4));
      }
    }
#pragma unroll
    for (int i = 0; i < ROWS; ++i) {
      const int rl = rbase + i * 16;
      if (rl >= tr.nrows) continue;
      const size_t m = size_t(tr.row0 + rl);
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int n = cbase + j * 16;
        if (n >= p.N) continue;
        float v[4];
        if constexpr (F8) {
          v[0] = acc[i][j][0] * (asc[i] * wsc[j].x) + bv[j][0];
          v[1] = acc[i][j][1] * (asc[i] * wsc[j].y) + bv[j][1];
          v[2] = acc[i][j][2] * (asc[i] * wsc[j].z) + bv[j][2];
          v[3] = acc[i][j][3] * (asc[i] * wsc[j].w) + bv[j][3];
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] = acc[i][j][e] + bv[j][e];
        }
        if constexpr (EPI == EPI_RESID) {
          float4 zn = zv[i][j];
          zn.x += gt[j].x * v[0];
          zn.y += gt[j].y * v[1];
          zn.z += gt[j].z * v[2];
          zn.w += gt[j].w * v[3];
          *reinterpret_cast<float4 *>(p.z + m * p.ldz + n) = zn;
        } else {
          if constexpr (EPI == EPI_GELU) {
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] = gelu_tanh(v[e]);
          }
          uint2 u;
          u.x = pack_bf16x2(v[0], v[1]);
          u.y = pack_bf16x2(v[2], v[3]);
          *reinterpret_cast<uint2 *>(reinterpret_cast<uint16_t *>(p.out) + m * p.ldo + n) = u;
        }
      }
    }
  }
};

// ------------------------------------------------------------------------------ MFMA tiles
//
// One persistent workgroup per CU, 4 waves (2 x 2).  For 256 x 256 tiles the wave tile is 128 x 128
// as 4 x 4 blocks of 32 x 32: 256 fp32 accumulators per lane, held in AGPRs, and per K step the CU
// loads half the operand bytes per FLOP of a 128 x 128 tile (BM x BN tiles: BM/64 x BN/64 blocks per
// wave, the same schedule).  K runs in stages of 64 bytes per row (32 bf16 or 64 FP8 values)
// through a 4-slot LDS ring (32 KiB per 256 x 256 stage: the stage's A rows, then its W rows, 16-byte
// chunks swizzled), loaded by direct global->LDS loads three stages ahead (window mode, below: the
// LDS holds three 128-byte K-step windows per row, loaded two K steps ahead).  A 256 x 256 stage is
// 16 blocks:
//   * bf16: two v_mfma_f32_32x32x16_bf16 per block, one per K half (chunks {h, h + 2});
//   * FP8:  one v_mfma_f32_32x32x64_f8f6f4 per block (all four chunks, 8 registers per operand).
// Either way lane (r, g) = (l % 32, l / 32) of a fragment reads chunks 2 g and 2 g + 1 of row r of a
// 32-row fragment: each half-wave reads one chunk of 32 consecutive rows, which the swizzle spreads
// over all banks (the 16 x 16 fragment order, 16 rows of two chunks per half-wave, measured 2-way
// bank conflicts on every read).  With one wave per SIMD nothing hides a stall of the wave, so the
// loop is a fixed schedule (inline asm pins the order):
//   * each block row waits only for its own fragment reads (DS reads complete in order, so an exact
//     lgkmcnt is known at every point);
//   * before block 4 the wave waits for its loads of the *next* stage and meets the others at the
//     barrier, which also tells it that every wave has finished reading the slot it is about to
//     refill;
//   * after each of blocks 4..11: one of the stage's 8 loads (three stages ahead) and two of the 16
//     fragment reads of the next stage.
// Fragments alternate between two register sets, so a scheduling unit is two stages (the K step of
// the stream-K plan: 64 bf16 or 128 FP8 values).  A second cursor over the workgroup's items drives
// the loads: at the end of an item they already fetch the next item's first stages, so its
// epilogue overlaps them.  Past the last item the loader repeats the last stage into free slots
// (valid addresses; keeps the vmcnt arithmetic uniform).  The epilogue's per-column and per-row
// operands (bias, FP8 scales, gate) reach LDS by a DMA issued in the item's first stage, so the
// epilogue never waits on the prefetch loads in flight behind them.
// Values that are the same on every lane, restated as such (the compiler otherwise keeps some of
// the stream-K bookkeeping in VGPRs and branches on it with exec masks).
HILO_DEV int uni(int v) { return __builtin_amdgcn_readfirstlane(v); }
HILO_DEV float *uni(float *ptr) {
  const uint64_t v = reinterpret_cast<uint64_t>(ptr);
  const uint32_t lo = __builtin_amdgcn_readfirstlane(uint32_t(v)), hi = __builtin_amdgcn_readfirstlane(uint32_t(v >> 32));
  return reinterpret_cast<float *>((uint64_t(hi) << 32) | lo);
}
HILO_DEV SkItem uni(const SkItem &x) { return SkItem{uni(x.t), uni(x.kb), uni(x.ke), uni(x.slot), uni(int(x.valid)) != 0}; }
HILO_DEV TileRows uni(const TileRows &x) { return TileRows{uni(x.s), uni(x.sigma), uni(x.row0), uni(x.nrows)}; }

namespace big {
constexpr int S = 4;                   // LDS ring slots
// per wave, behind the ring: the wave's columns of bias (bf16, <= 256 B), of the FP8 weight scales
// (float32, <= 512 B), its rows of FP8 activation scales (<= 512 B) and its columns of the residual
// gate (float32, <= 512 B)
constexpr int kEpiWave = 1792, kEpiBias = 0, kEpiCol = 256, kEpiRow = 768, kEpiGate = 1280;
HILO_DEV int swz(int r) { return ((r >> 1) & 3) ^ ((r >> 3) & 1); }
// W row read by fragment lane r.  The 32 x 32 MFMA's output row i (the W side) lands in
// accumulator register 4 (i / 8) + i % 4 of the lanes of half (i / 4) % 2; reading W row perm_w(i)
// there gives lane half g the columns 16 g .. 16 g + 15 in register order.  These LDS reads are
// conflict-free like the natural order (measured; shifting the second half by 8 rows is not).
HILO_DEV int perm_w(int r) { return ((r & 4) ? 16 : 0) + 4 * (r >> 3) + (r & 3); }
// A BM x BN tile on 4 waves (2 x 2), wave tile BM/2 x BN/2 as NBM x NBN blocks of 32 x 32.
template <int BM, int BN>
struct Geo {
  static_assert((BM == 256 && BN == 256) || (BM == 192 && BN == 192) || (BM == 256 && BN == 192),
                "tile shapes of the MFMA kernel");
  static constexpr int NBM = BM / 64;        // blocks per wave column (A side)
  static constexpr int NBN = BN / 64;        // blocks per wave row (W side)
  static constexpr int LQ = NBM + NBN;       // load instructions per wave per stage (A rows, then W rows)
  static constexpr int NR = 2 * LQ;          // fragment reads per wave per stage
  static constexpr int AB = BM * 64;         // bytes of a stage's A rows
  static constexpr int SB = (BM + BN) * 64;  // bytes of a stage
  // Window mode: when three K steps of the tile fit in LDS, each row's 128 bytes of a K step (both
  // of its stages) stay together, so one load instruction fetches 8 whole 128-byte lines instead of
  // 16 half lines (measured: fewer, fuller requests to the L2); three window slots keep the loads
  // two K steps ahead.  The 256-wide tiles hold only two windows, and one K step of prefetch
  // measured slower than the half-line ring.
  static constexpr int WS = 3;                          // window slots
  static constexpr int SBW = (BM + BN) * 128;           // bytes of a window
  static constexpr bool WIN = BM == BN && WS * SBW + 4 * kEpiWave <= 160 * 1024;
  static constexpr int LDS = WIN ? WS * SBW + 4 * kEpiWave : S * SB + 4 * kEpiWave;
  // every load and fragment read of a stage is issued after its barrier (block NBN) and before
  // its last block; in window mode a stage loads BM / 32 instructions of 8 rows (its wave's A rows
  // in the first stage of a K step, its W rows in the second), the same count as LQ for BM == BN
  static_assert(NBN + LQ <= NBM * NBN, "stage schedule does not fit the blocks");
  static_assert(!WIN || BM / 32 == LQ, "window loads per stage");
};
// Chunk swizzle of a 128-byte window row: the 16-byte chunk that global chunk c of row r occupies is
// c ^ swzw(r).  A ds_read_b128 serves 16 lanes per cycle from 64 banks; with it every 16-lane group
// of a fragment read (16 consecutive rows, or the perm_w rows of W) hits 16 distinct bank groups.
HILO_DEV int swzw(int r) { return ((r >> 1) & 3) ^ ((((r >> 3) ^ (r >> 4)) & 1) << 2); }
}  // namespace big

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

#define HILO_MFMA16_AGPR(ACC, FB, FA) \
  asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+a"(ACC) : "v"(FB), "v"(FA) : "memory")
// first MFMA of a tile: accumulate onto zero (no separate clearing of the AGPRs)
#define HILO_MFMA16_AGPR0(ACC, FB, FA) \
  asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, 0" : "=a"(ACC) : "v"(FB), "v"(FA) : "memory")
// The 8-register operands have no host counterpart: the host pass (which only needs the kernel's
// launch stub) would reject the constraint and silently drop the stub, so it sees no asm here.
#if defined(__HIP_DEVICE_COMPILE__)
#define HILO_MFMA8_AGPR(ACC, FB, FA) \
  asm volatile("v_mfma_f32_32x32x64_f8f6f4 %0, %1, %2, %0" : "+a"(ACC) : "v"(FB), "v"(FA) : "memory")
#define HILO_MFMA8_AGPR0(ACC, FB, FA) \
  asm volatile("v_mfma_f32_32x32x64_f8f6f4 %0, %1, %2, 0" : "=a"(ACC) : "v"(FB), "v"(FA) : "memory")
#else
#define HILO_MFMA8_AGPR(ACC, FB, FA) ((void)0)
#define HILO_MFMA8_AGPR0(ACC, FB, FA) ((void)0)
#endif
HILO_DEV u32x8 cat8(u32x4 lo, u32x4 hi) { return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7); }
#define HILO_DS_READ16(DST, ADDR, OFF) \
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(DST) : "v"(ADDR), "i"(OFF) : "memory")

// One 4-byte global load per lane straight into LDS: lane l lands at byte 4 l of the destination.
HILO_DEV void g2lds4(const void *g, void *lds_wave_base) {
  __builtin_amdgcn_global_load_lds(g, (__attribute__((address_space(3))) void *)lds_wave_base, 4, 0, 0);
}

template <int N>
HILO_DEV void wait_lgkm_le() { asm volatile("s_waitcnt lgkmcnt(%0)" ::"n"(N) : "memory"); }

HILO_DEV void wait_lgkm_rt(int n) {  // n is a compile-time constant after unrolling
  switch (n) {
    case 0: wait_lgkm_le<0>(); break;   case 1: wait_lgkm_le<1>(); break;
    case 2: wait_lgkm_le<2>(); break;   case 3: wait_lgkm_le<3>(); break;
    case 4: wait_lgkm_le<4>(); break;   case 5: wait_lgkm_le<5>(); break;
    case 6: wait_lgkm_le<6>(); break;   case 7: wait_lgkm_le<7>(); break;
    case 8: wait_lgkm_le<8>(); break;   case 9: wait_lgkm_le<9>(); break;
    case 10: wait_lgkm_le<10>(); break; case 11: wait_lgkm_le<11>(); break;
    case 12: wait_lgkm_le<12>(); break; case 13: wait_lgkm_le<13>(); break;
    case 14: wait_lgkm_le<14>(); break; default: wait_lgkm_le<15>(); break;
  }
}

// Epilogue of a BM x BN tile from the AGPR accumulators of wave wid.  The W fragments are read in
// the row order perm_w, so lane l of block (bi, bj) holds row 32 bi + l % 32 of the wave tile and, in
// register v, column 32 bj + 16 (l / 32) + v: 16 consecutive columns, stored as two 16-byte pieces
// (bf16) or four (float32 z).  Column operands (bias, FP8 weight scales, the gate) come from the
// wave's LDS area `epi`, once per block column; FP8 row scales once per tile.  Bias / GELU outputs
// are rounded to bf16, the residual update adds gate * (acc + bias) to the float32 z.  Blocks leave
// the AGPRs one at a time.
template <int BM, int BN, int EPI, bool F8>
HILO_DEV void big_epilogue(const GemmProblem &p, const TileRows &tr, int n0, int wid, int lane,
                           const uint8_t *epi, f32x16 (&acc)[BM / 64][BN / 64]) {
  using namespace big;
  constexpr int NBM = Geo<BM, BN>::NBM, NBN = Geo<BM, BN>::NBN;
  const int rbase = (wid >> 1) * (BM / 2) + (lane & 31);
  const int cl0 = 16 * (lane >> 5);              // this lane's first column within a 32-column block
  const int cbase = n0 + (wid & 1) * (BN / 2) + cl0;
  float sa[NBM];
#pragma unroll
  for (int bi = 0; bi < NBM; ++bi)
    sa[bi] = F8 ? *reinterpret_cast<const float *>(epi + kEpiRow + 4 * (32 * bi + (lane & 31))) : 1.f;
  // The residual update loads every z piece of the wave before it stores any: stores count in
  // vmcnt, so a z load issued after a block's stores would wait for them too (one memory round
  // trip per block: 16.4 us per 192 x 192 tile epilogue against 13.4-14.1 with one).
  // Lanes outside the tile load a valid element they do not store.
  constexpr int ZB = EPI == EPI_RESID ? NBM * NBN : 1;
  static_assert(EPI != EPI_RESID || ZB <= 9, "the wave's z pieces are held in registers");
  float4 zz[ZB][4];
  if constexpr (EPI == EPI_RESID) {
#pragma unroll
    for (int bj = 0; bj < NBN; ++bj)
#pragma unroll
      for (int bi = 0; bi < NBM; ++bi) {
        const int rl = rbase + 32 * bi, n = cbase + 32 * bj;
        const bool in = rl < tr.nrows && n < p.N;
        const float4 *zp =
            reinterpret_cast<const float4 *>(p.z + size_t(tr.row0 + (in ? rl : 0)) * p.ldz + (in ? n : 0));
#pragma unroll
        for (int h = 0; h < 4; ++h) zz[bj * NBM + bi][h] = zp[h];
      }
  }
#pragma unroll
  for (int bj = 0; bj < NBN; ++bj) {
    const int cl = cl0 + 32 * bj, n = cbase + 32 * bj;
    u32x4 bu[2];
    f32x4 cv[4], gv[4];  // FP8 weight scales and the residual gate of the lane's 16 columns
#pragma unroll
    for (int h = 0; h < 2; ++h) bu[h] = *reinterpret_cast<const u32x4 *>(epi + kEpiBias + 2 * cl + 16 * h);
    if constexpr (F8) {
#pragma unroll
      for (int h = 0; h < 4; ++h) cv[h] = *reinterpret_cast<const f32x4 *>(epi + kEpiCol + 4 * cl + 16 * h);
    }
    if constexpr (EPI == EPI_RESID) {
#pragma unroll
      for (int h = 0; h < 4; ++h) gv[h] = *reinterpret_cast<const f32x4 *>(epi + kEpiGate + 4 * cl + 16 * h);
    }
#pragma unroll
    for (int bi = 0; bi < NBM; ++bi) {
      f32x16 blk = acc[bi][bj];  // one block out of the AGPRs at a time
      asm volatile("" : "+v"(blk));
      const int rl = rbase + 32 * bi;
      if (rl < tr.nrows && n < p.N) {  // N % 16 == 0: a lane's 16 columns are all inside or all out
        const size_t m = size_t(tr.row0 + rl);
        float v[16];
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const uint32_t w = bu[e >> 3][(e >> 1) & 3];
          const float bias = __uint_as_float((e & 1) ? (w & 0xffff0000u) : (w << 16));
          if constexpr (F8) v[e] = blk[e] * (sa[bi] * cv[e >> 2][e & 3]) + bias;
          else v[e] = blk[e] + bias;
        }
        if constexpr (EPI == EPI_RESID) {
          float4 *zp = reinterpret_cast<float4 *>(p.z + m * p.ldz + n);
#pragma unroll
          for (int h = 0; h < 4; ++h) {
            float4 z = zz[bj * NBM + bi][h];
            z.x += gv[h][0] * v[4 * h + 0];
            z.y += gv[h][1] * v[4 * h + 1];
            z.z += gv[h][2] * v[4 * h + 2];
            z.w += gv[h][3] * v[4 * h + 3];
            zp[h] = z;
          }
        } else {
          if constexpr (EPI == EPI_GELU) {
#pragma unroll
            for (int e = 0; e < 16; ++e) v[e] = gelu_tanh(v[e]);
          }
          uint4 *op = reinterpret_cast<uint4 *>(reinterpret_cast<uint16_t *>(p.out) + m * p.ldo + n);
#pragma unroll
          for (int h = 0; h < 2; ++h)
            op[h] = make_uint4(pack_bf16x2(v[8 * h + 0], v[8 * h + 1]), pack_bf16x2(v[8 * h + 2], v[8 * h + 3]),
                               pack_bf16x2(v[8 * h + 4], v[8 * h + 5]), pack_bf16x2(v[8 * h + 6], v[8 * h + 7]));
        }
      }
      asm volatile("" ::: "memory");  // the next block's operands stay below these stores
    }
  }
}

// FP8 q and k for the attention's score product, from the QKV projection's accumulators of a
// 256 x 256 tile of FP8 operands whose columns lie below 2 D.  The wave's 128 columns hold whole
// heads (128 / head_dim of them); per (row, head): the values acc * (row scale * weight scale) +
// bias (as the bf16 output would take them), their amax over the head -- this lane's 16 columns of
// each block and those of lane l ^ 32, which holds the block's other 16 -- the power-of-two scale
// 2^k, and the E4M3 codes of the values times 2^-k (16 bytes per lane and block); then one E8M0
// byte 127 + k per (row, head).  The values are formed twice (amax, then codes) instead of held.
template <int BM, int BN>
HILO_DEV void big_epilogue_qk8(const GemmProblem &p, const TileRows &tr, int n0, int wid, int lane,
                               const uint8_t *epi, f32x16 (&acc)[BM / 64][BN / 64]) {
  using namespace big;
  static_assert(BN == 256, "a wave's 128 columns hold whole heads");
  constexpr int NBM = BM / 64, NBN = BN / 64;
  const int hd = p.head_dim, bph = hd / 32;  // blocks per head
  const int rbase = (wid >> 1) * (BM / 2) + (lane & 31);
  const int cl0 = 16 * (lane >> 5);
  const int wc0 = n0 + (wid & 1) * (BN / 2);
  auto values = [&](int bi, int bj, float sa, float (&v)[16]) __attribute__((always_inline)) {
    const int cl = cl0 + 32 * bj;
    u32x4 bu[2];
    f32x4 cv[4];
#pragma unroll
    for (int h = 0; h < 2; ++h) bu[h] = *reinterpret_cast<const u32x4 *>(epi + kEpiBias + 2 * cl + 16 * h);
#pragma unroll
    for (int h = 0; h < 4; ++h) cv[h] = *reinterpret_cast<const f32x4 *>(epi + kEpiCol + 4 * cl + 16 * h);
    f32x16 blk = acc[bi][bj];
    asm volatile("" : "+v"(blk));
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const uint32_t w = bu[e >> 3][(e >> 1) & 3];
      const float bias = __uint_as_float((e & 1) ? (w & 0xffff0000u) : (w << 16));
      v[e] = blk[e] * (sa * cv[e >> 2][e & 3]) + bias;
    }
  };
#pragma unroll
  for (int bi = 0; bi < NBM; ++bi) {
    const float sa = *reinterpret_cast<const float *>(epi + kEpiRow + 4 * (32 * bi + (lane & 31)));
    float am0 = 0.f, am1 = 0.f;
#pragma unroll
    for (int bj = 0; bj < NBN; ++bj) {
      float v[16];
      values(bi, bj, sa, v);
      float m = 0.f;
#pragma unroll
      for (int e = 0; e < 16; ++e) m = fmaxf(m, fabsf(v[e]));
      if (bj / bph == 0) am0 = fmaxf(am0, m);
      else am1 = fmaxf(am1, m);
    }
    am0 = fmaxf(am0, __shfl_xor(am0, 32, 64));
    am1 = fmaxf(am1, __shfl_xor(am1, 32, 64));
    const int k0 = pow2_exponent(am0), k1 = pow2_exponent(am1);
    const float i0 = pow2_inverse(k0), i1 = pow2_inverse(k1);
    const int rl = rbase + 32 * bi;
    if (rl < tr.nrows) {
      uint8_t *row = p.qk8 + size_t(tr.row0 + rl) * p.ldq8;
#pragma unroll
      for (int bj = 0; bj < NBN; ++bj) {
        float v[16];
        values(bi, bj, sa, v);
        const float s = bj / bph == 0 ? i0 : i1;
        uint4 c;
        c.x = fp8x4(v[0] * s, v[1] * s, v[2] * s, v[3] * s);
        c.y = fp8x4(v[4] * s, v[5] * s, v[6] * s, v[7] * s);
        c.z = fp8x4(v[8] * s, v[9] * s, v[10] * s, v[11] * s);
        c.w = fp8x4(v[12] * s, v[13] * s, v[14] * s, v[15] * s);
        *reinterpret_cast<uint4 *>(row + wc0 + cl0 + 32 * bj) = c;
      }
      if (lane < 32) {
        row[2 * p.D + wc0 / hd] = uint8_t(127 + k0);
        if (bph * 2 == NBN) row[2 * p.D + wc0 / hd + 1] = uint8_t(127 + k1);
      }
    }
    asm volatile("" ::: "memory");
  }
}

template <int BM, int BN, int EPI, int ROLE, bool F8>
__global__ __launch_bounds__(256) void k_gemm_big(GemmProblem p) {
  using namespace big;
  using G = Geo<BM, BN>;
  constexpr int NBM = G::NBM, NBN = G::NBN, LQ = G::LQ, NR = G::NR, AB = G::AB, SB = G::SB;
  constexpr bool WIN = G::WIN;
  constexpr int SBW = G::SBW, NLA = WIN ? 2 * NBM : NBM, NLB = WIN ? 2 * NBN : NBN;
  using T = SkTile<BM, BN, 2, 2>;       // partial slot size and layout (16 x 16 fragment order)
  constexpr int ESZ = F8 ? 1 : 2;       // operand bytes per element
  __shared__ __attribute__((aligned(1024))) uint8_t lds[G::LDS];

  const int P = gridDim.x;
  const int pid = xcd_remap(blockIdx.x, P);
  const SkPlan q = sk_plan(p, BM, BN, P, F8 ? 128 : 64);
  const SkRange rg = sk_range(q, pid);

  const int lane = threadIdx.x & 63;
  const int wid = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lrow = lane >> 2, lslot = lane & 3;
  const uint8_t *A = reinterpret_cast<const uint8_t *>(p.A);

  // ---- loader: its own cursor over this workgroup's items, three stages ahead of the MFMAs (window
  // mode: two K steps ahead); wave wid loads rows wid BM/4 .. + BM/4 - 1 of A and wid BN/4 .. +
  // BN/4 - 1 of W, 16 rows of 64 bytes (window mode: 8 rows of 128 bytes) per 1 KiB instruction
  SkCursor lc{pid, rg.beg};
  const uint8_t *la[NLA], *lb[NLB];
  int lk = 0, lke = 0;  // next stage (window mode: K step) to load, absolute in K, and its item's end
  auto ld_src = [&](int t) __attribute__((always_inline)) {
    int rt, tn;
    tile_coords(q, t, rt, tn);
    tn = uni(tn);
    const TileRows tr = uni(decode_row_tile(p, BM, uni(rt)));
    const uint8_t *Wt = reinterpret_cast<const uint8_t *>(tr.sigma ? p.W[1] : p.W[0]);
    if constexpr (WIN) {
#pragma unroll
      for (int i = 0; i < NLA; ++i) {
        const int r = wid * (BM / 4) + 8 * i + (lane >> 3);
        la[i] = A + size_t(tr.row0 + min(r, tr.nrows - 1)) * p.lda * ESZ + ((lane & 7) ^ swzw(r)) * 16;
      }
#pragma unroll
      for (int i = 0; i < NLB; ++i) {
        const int r = wid * (BN / 4) + 8 * i + (lane >> 3);
        lb[i] = Wt + size_t(min(tn * BN + r, p.N - 1)) * p.K * ESZ + ((lane & 7) ^ swzw(r)) * 16;
      }
    } else {
#pragma unroll
      for (int i = 0; i < NBM; ++i) {
        const int r = wid * (BM / 4) + 16 * i + lrow;
        la[i] = A + size_t(tr.row0 + min(r, tr.nrows - 1)) * p.lda * ESZ + (lslot ^ swz(r)) * 16;
      }
#pragma unroll
      for (int i = 0; i < NBN; ++i) {
        const int r = wid * (BN / 4) + 16 * i + lrow;
        lb[i] = Wt + size_t(min(tn * BN + r, p.N - 1)) * p.K * ESZ + (lslot ^ swz(r)) * 16;
      }
    }
  };
  auto ld_advance = [&]() __attribute__((always_inline)) {
    const SkItem x = uni(sk_next_item(lc, q, rg, P, pid, p.part, T::kPartFloats));
    if (x.valid) {
      ld_src(x.t);
      lk = WIN ? x.kb : 2 * x.kb;
      lke = WIN ? x.ke : 2 * x.ke;
    } else {
      lk = lke - 1;  // no further item: repeat the last stage
    }
    lk = uni(lk);
    lke = uni(lke);
  };
  // load instruction j (0..LQ-1) of the current loader stage into `slot`: A rows for j < NBM
  auto ld_one = [&](int slot, int j) __attribute__((always_inline)) {
    const int k0 = lk * 64;  // bytes
    if (j < NBM) g2lds16(la[j] + k0, lds + slot * SB + wid * (BM / 4) * 64 + j * 1024);
    else g2lds16(lb[j - NBM] + k0, lds + slot * SB + AB + wid * (BN / 4) * 64 + (j - NBM) * 1024);
  };
  // window mode: load instruction j of half h (0: the wave's A rows, 1: its W rows) of the loader's
  // K step into window slot `ws`
  auto ld_win = [&](int ws, int h, int j) __attribute__((always_inline)) {
    const int k0 = lk * 128;  // bytes
    if (h == 0) g2lds16(la[j] + k0, lds + ws * SBW + (wid * (BM / 4) + 8 * j) * 128);
    else g2lds16(lb[j] + k0, lds + ws * SBW + BM * 128 + (wid * (BN / 4) + 8 * j) * 128);
  };

  // ---- fragment reads: lane (r, g) = (lane % 32, lane / 32) reads chunk 2 g (low half) and 2 g + 1
  // (high half) of row r (A) or perm_w(r) (W) of a 32-row fragment; read t of a stage (slot byte
  // offset so) is half t % 2 of W fragment t / 2 for t < 2 NBN, then of A fragment (t - 2 NBN) / 2
  const int r8 = lane & 31, g8 = lane >> 5, w8 = perm_w(r8);
  const uint32_t lds0 = (uint32_t)(uintptr_t)lds;
  const uint32_t fa8 = lds0 + (wid >> 1) * (BM / 2) * 64, fb8 = lds0 + AB + (wid & 1) * (BN / 2) * 64;
  const uint32_t fa8l = fa8 + r8 * 64 + (((2 * g8) ^ swz(r8)) * 16), fa8h = fa8 + r8 * 64 + (((2 * g8 + 1) ^ swz(r8)) * 16);
  const uint32_t fb8l = fb8 + w8 * 64 + (((2 * g8) ^ swz(w8)) * 16), fb8h = fb8 + w8 * 64 + (((2 * g8 + 1) ^ swz(w8)) * 16);
  // window mode: the same lane mapping on 128-byte rows; half h (0, 1) of a K step holds its global
  // chunks 4 h .. 4 h + 3, and a fragment spans 32 rows of 128 bytes
  const uint32_t wa = lds0 + (wid >> 1) * (BM / 2) * 128 + r8 * 128;
  const uint32_t wb = lds0 + BM * 128 + (wid & 1) * (BN / 2) * 128 + w8 * 128;
  const uint32_t fwa[4] = {wa + (((2 * g8) ^ swzw(r8)) * 16), wa + (((2 * g8 + 1) ^ swzw(r8)) * 16),
                           wa + (((4 + 2 * g8) ^ swzw(r8)) * 16), wa + (((5 + 2 * g8) ^ swzw(r8)) * 16)};
  const uint32_t fwb[4] = {wb + (((2 * g8) ^ swzw(w8)) * 16), wb + (((2 * g8 + 1) ^ swzw(w8)) * 16),
                           wb + (((4 + 2 * g8) ^ swzw(w8)) * 16), wb + (((5 + 2 * g8) ^ swzw(w8)) * 16)};
  constexpr int FRB = WIN ? 4096 : 2048;  // bytes between fragments
  // read t of the stage at byte offset so; hs: the stage's half of its K step (window mode only)
  auto rd_one = [&](u32x4 (&fa)[2 * NBM], u32x4 (&fb)[2 * NBN], uint32_t so, int t, int hs) __attribute__((always_inline)) {
    const uint32_t al = WIN ? fwa[2 * hs] : fa8l, ah = WIN ? fwa[2 * hs + 1] : fa8h;
    const uint32_t bl = WIN ? fwb[2 * hs] : fb8l, bh = WIN ? fwb[2 * hs + 1] : fb8h;
#define HILO_RD_CASE(C)                                                                                     \
  case C:                                                                                                   \
    if constexpr (C < 2 * NBN)                                                                              \
      HILO_DS_READ16(fb[C % (2 * NBN)], ((C & 1) ? bh : bl) + so, ((C % (2 * NBN)) >> 1) * FRB);            \
    else if constexpr (C < 2 * NBN + 2 * NBM)                                                               \
      HILO_DS_READ16(fa[(C - 2 * NBN) % (2 * NBM)], ((C & 1) ? ah : al) + so, (((C - 2 * NBN) % (2 * NBM)) >> 1) * FRB); \
    break;
    switch (t) {
      HILO_RD_CASE(0) HILO_RD_CASE(1) HILO_RD_CASE(2) HILO_RD_CASE(3) HILO_RD_CASE(4) HILO_RD_CASE(5)
      HILO_RD_CASE(6) HILO_RD_CASE(7) HILO_RD_CASE(8) HILO_RD_CASE(9) HILO_RD_CASE(10) HILO_RD_CASE(11)
      HILO_RD_CASE(12) HILO_RD_CASE(13) HILO_RD_CASE(14) HILO_RD_CASE(15)
      default: break;
    }
#undef HILO_RD_CASE
  };

  // ---- epilogue operands of the current item: this wave's BN/2 columns (and FP8 rows) into its
  // LDS area, by DMA (4 bytes per lane), indices clamped into the tile
  uint8_t *epi = lds + (WIN ? G::WS * SBW : S * SB) + wid * kEpiWave;
  TileRows etr{0, 0, 0, 1};
  int en0 = 0;
  auto epi_load = [&]() __attribute__((always_inline)) {
    const int c0 = en0 + (wid & 1) * (BN / 2);
    const uint16_t *bias = reinterpret_cast<const uint16_t *>(etr.sigma ? p.bias[1] : p.bias[0]);
    g2lds4(bias + min(c0 + 2 * lane, p.N - 2), epi + kEpiBias);
    if constexpr (F8) {
      const float *ws = etr.sigma ? p.w_scale[1] : p.w_scale[0];
      g2lds4(ws + min(c0 + lane, p.N - 1), epi + kEpiCol);
      g2lds4(ws + min(c0 + 64 + lane, p.N - 1), epi + kEpiCol + 256);
    }
    if constexpr (EPI == EPI_RESID) {
      const float *gate = p.mod + (size_t(etr.s * 2 + etr.sigma) * 6 + p.gate_idx) * p.D;
      g2lds4(gate + min(c0 + lane, p.N - 1), epi + kEpiGate);
      g2lds4(gate + min(c0 + 64 + lane, p.N - 1), epi + kEpiGate + 256);
    }
    if constexpr (F8) {
      const int r0 = (wid >> 1) * (BM / 2);
      g2lds4(p.a_scale + etr.row0 + min(r0 + lane, etr.nrows - 1), epi + kEpiRow);
      g2lds4(p.a_scale + etr.row0 + min(r0 + 64 + lane, etr.nrows - 1), epi + kEpiRow + 256);
    }
  };

  f32x16 acc[NBM][NBN];
  u32x4 xa[2 * NBM], xb[2 * NBN], ya[2 * NBM], yb[2 * NBN];

  // one stage (ring slot gs % S) on fragments (fa, fb); reads stage gs + 1 into (na, nb); the first
  // stage of a tile (first = true_type) starts the accumulators from zero and, for a tile finished
  // here, fetches the epilogue operands after its loads.  Before block NBN: barrier; after each of
  // blocks NBN .. NBN + LQ - 1: one load of the stage three ahead and two fragment reads of the next.
  auto stage = [&](auto first, auto odd, u32x4 (&fa)[2 * NBM], u32x4 (&fb)[2 * NBN], u32x4 (&na)[2 * NBM],
                   u32x4 (&nb)[2 * NBN], int gs, bool with_epi) __attribute__((always_inline)) {
    constexpr bool ODD = decltype(odd)::value;  // second stage of its K step
    int lslot_w;
    uint32_t so;
    if constexpr (WIN) {
      // window slot of this K step; loads go two K steps ahead, reads to the next stage
      const int w3 = (gs >> 1) % G::WS;
      lslot_w = w3 == 0 ? G::WS - 1 : w3 - 1;
      so = uint32_t((ODD ? (w3 == G::WS - 1 ? 0 : w3 + 1) : w3) * SBW);
    } else {
      lslot_w = (gs + S - 1) & (S - 1);
      so = uint32_t(((gs + 1) & (S - 1)) * SB);
    }
#pragma unroll
    for (int bi = 0; bi < NBM; ++bi) {
      // outstanding reads allowed: this stage's A halves of blocks bi+1.., the next stage's so far
      wait_lgkm_rt(2 * (NBM - 1 - bi) + 2 * min(max(NBN * bi - NBN, 0), LQ));
#pragma unroll
      for (int bj = 0; bj < NBN; ++bj) {
        const int qq = NBN * bi + bj;
        if (qq == NBN) {
          // window mode: the second stage of K step w waits for K step w + 1 (only the loads of w + 2
          // issued by the first stage may be outstanding); the first stage reads the second half of
          // its own K step, which is complete already.  Either barrier also frees the slot the stage
          // loads into: every wave has finished the K step before.
          if constexpr (!WIN) asm volatile("s_waitcnt vmcnt(%0)\n s_barrier" ::"n"((S - 3) * LQ) : "memory");
          else if constexpr (ODD) asm volatile("s_waitcnt vmcnt(%0)\n s_barrier" ::"n"(LQ) : "memory");
          else asm volatile("s_barrier" ::: "memory");
        }
        if constexpr (F8) {
          if constexpr (decltype(first)::value)
            HILO_MFMA8_AGPR0(acc[bi][bj], cat8(fb[2 * bj], fb[2 * bj + 1]), cat8(fa[2 * bi], fa[2 * bi + 1]));
          else
            HILO_MFMA8_AGPR(acc[bi][bj], cat8(fb[2 * bj], fb[2 * bj + 1]), cat8(fa[2 * bi], fa[2 * bi + 1]));
        } else {
          if constexpr (decltype(first)::value) HILO_MFMA16_AGPR0(acc[bi][bj], fb[2 * bj], fa[2 * bi]);
          else HILO_MFMA16_AGPR(acc[bi][bj], fb[2 * bj], fa[2 * bi]);
          HILO_MFMA16_AGPR(acc[bi][bj], fb[2 * bj + 1], fa[2 * bi + 1]);
        }
        if (qq >= NBN && qq < NBN + LQ) {
          if constexpr (WIN) {
            // the epilogue DMA goes ahead of the stage's loads, so the next stage's vmcnt covers it
            if constexpr (decltype(first)::value) {
              if (qq == NBN && with_epi) epi_load();
            }
            ld_win(lslot_w, ODD ? 1 : 0, qq - NBN);
          } else {
            ld_one(lslot_w, qq - NBN);
          }
          rd_one(na, nb, so, 2 * (qq - NBN), ODD ? 0 : 1);
          rd_one(na, nb, so, 2 * (qq - NBN) + 1, ODD ? 0 : 1);
        }
        if constexpr (decltype(first)::value && !WIN) {
          if (qq == NBN + LQ - 1 && with_epi) epi_load();
        }
      }
    }
    if constexpr (!WIN || ODD) ++lk;
  };

  SkCursor cc{pid, rg.beg};
  SkItem cur = uni(sk_next_item(cc, q, rg, P, pid, p.part, T::kPartFloats));
  if (!cur.valid) return;
  ld_advance();  // the same first item
  if constexpr (WIN) {
    // the first two K steps, then wait for the first
#pragma unroll 1
    for (int wv = 0; wv < G::WS - 1; ++wv) {
      if (lk == lke) ld_advance();
#pragma unroll
      for (int j = 0; j < NLA; ++j) ld_win(wv, 0, j);
#pragma unroll
      for (int j = 0; j < NLB; ++j) ld_win(wv, 1, j);
      ++lk;
    }
    asm volatile("s_waitcnt vmcnt(%0)\n s_barrier" ::"n"(NLA + NLB) : "memory");
  } else {
#pragma unroll 1
    for (int st = 0; st < S - 1; ++st) {
      if (lk == lke) ld_advance();
#pragma unroll
      for (int j = 0; j < LQ; ++j) ld_one(st, j);
      ++lk;
    }
    asm volatile("s_waitcnt vmcnt(%0)\n s_barrier" ::"n"((S - 2) * LQ) : "memory");
  }
#pragma unroll
  for (int t = 0; t < NR; ++t) rd_one(xa, xb, 0, t, 0);

  // the loader moves to its next item between stages, outside the MFMA schedule
  auto ld_check = [&]() __attribute__((always_inline)) {
    if (lk == lke) ld_advance();
  };
  int gs = 0;
  while (true) {
    const bool whole = cur.slot == nullptr;
    if (whole) {
      int rt, tn;
      tile_coords(q, cur.t, rt, tn);
      en0 = uni(tn) * BN;
      etr = uni(decode_row_tile(p, BM, uni(rt)));
    }
    ld_check();
    stage(std::true_type{}, std::false_type{}, xa, xb, ya, yb, gs, whole);
    ld_check();
    stage(std::false_type{}, std::true_type{}, ya, yb, xa, xb, gs + 1, false);
    gs += 2;
#pragma unroll 1
    for (int kt = cur.kb + 1; kt < cur.ke; ++kt) {
      ld_check();
      stage(std::false_type{}, std::false_type{}, xa, xb, ya, yb, gs, false);
      ld_check();
      stage(std::false_type{}, std::true_type{}, ya, yb, xa, xb, gs + 1, false);
      gs += 2;
    }
    // The last MFMAs' results must land before the accumulators are read (the empty asm ties each
    // accumulator to this point, so no read is scheduled above it), and the reads of the next
    // stage's fragments must be complete before the compiler may move those registers.
    asm volatile("s_waitcnt lgkmcnt(0)\n s_nop 7\n s_nop 7\n s_nop 7\n s_nop 7" ::: "memory");
#pragma unroll
    for (int i = 0; i < NBM; ++i)
#pragma unroll
      for (int j = 0; j < NBN; ++j) asm volatile("" : "+a"(acc[i][j]));
    if (whole) {
      // the epilogue-operand DMA of the first stage is complete once two later stages have passed
      // their barriers (each waits for all but the last stage's loads); a one-step item waits here.
      // In window mode the item's second stage waited for it already.
      if (!WIN && cur.ke - cur.kb < 2) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      if constexpr (F8 && EPI == EPI_BIAS && BN == 256) {
        if (p.qk8 != nullptr && en0 < 2 * p.D) big_epilogue_qk8<BM, BN>(p, etr, en0, wid, lane, epi, acc);
        else big_epilogue<BM, BN, EPI, F8>(p, etr, en0, wid, lane, epi, acc);
      } else {
        big_epilogue<BM, BN, EPI, F8>(p, etr, en0, wid, lane, epi, acc);
      }
    } else {
      // the partial tile in the 16 x 16 fragment layout k_gemm_fix reads (2 NBM x 2 NBN fragments per
      // wave): row 32 bi + l % 32 is fragment row 2 bi + (l % 32) / 16; columns 32 bj + 16 (l / 32)
      // + 4 b .. + 3 are lane l % 16 + 16 b of fragment column 2 bj + l / 32
      constexpr int TFM = 2 * NBM, TFN = 2 * NBN;
      float *base = cur.slot + (size_t(wid) * TFM * TFN * 64 + ((lane & 31) >> 4) * TFN * 64 + (lane >> 5) * 64 + (lane & 15)) * 4;
#pragma unroll
      for (int bi = 0; bi < NBM; ++bi)
#pragma unroll
        for (int bj = 0; bj < NBN; ++bj) {
          f32x16 blk = acc[bi][bj];
          asm volatile("" : "+v"(blk));
#pragma unroll
          for (int b = 0; b < 4; ++b)
            *reinterpret_cast<f32x4 *>(base + ((2 * bi * TFN + 2 * bj) * 64 + 16 * b) * 4) =
                f32x4{blk[4 * b], blk[4 * b + 1], blk[4 * b + 2], blk[4 * b + 3]};
          asm volatile("" ::: "memory");
        }
    }
    cur = uni(sk_next_item(cc, q, rg, P, pid, p.part, T::kPartFloats));
    if (!cur.valid) break;
  }
  asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory");
}

// Finishes every tile left in partials.  A work item is one fragment row of one main-kernel wave
// of one tile, taken by one wave of the fixup: it adds the tile's partials (pieces in K order,
// stream-K contributors in workgroup order) and runs the epilogue on the row.  Contributions are
// loaded in batches of four (one memory round trip per batch instead of per contributor) and
// added in the fixed order, so the result does not depend on the batching.
constexpr int kFixThreads = 256;
constexpr int kFixBatch = 4;

template <int BM, int BN, int WM, int WN, int EPI, int ROLE, bool F8 = false>
__global__ __launch_bounds__(kFixThreads) void k_gemm_fix(GemmProblem p, int P) {
  using T = SkTile<BM, BN, WM, WN>;
  constexpr int TM = T::TM, TN = T::TN, NW = T::NW, FW = kFixThreads / 64;
  const SkPlan q = sk_plan(p, BM, BN, P, F8 ? 128 : 64);
  const int nfix = q.s > 1 ? q.T : q.U - q.dp;
  const int lane = threadIdx.x & 63;
  const int items = nfix * NW * TM;
  for (int x = blockIdx.x * FW + (threadIdx.x >> 6); x < items; x += gridDim.x * FW) {
    const int f = x / (NW * TM), rem = x - f * (NW * TM), wid = rem / TM, i = rem - wid * TM;
    const int t = q.s > 1 ? f : q.dp + f;
    f32x4 acc[1][TN];
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[0][j] = f32x4{0.f, 0.f, 0.f, 0.f};
    const float *b[kFixBatch];
    int nb = 0;
    auto flush = [&]() {
      f32x4 v[kFixBatch][TN];
#pragma unroll
      for (int c = 0; c < kFixBatch; ++c)
        if (c < nb) {
#pragma unroll
          for (int j = 0; j < TN; ++j) v[c][j] = *reinterpret_cast<const f32x4 *>(b[c] + T::part_index(wid, i, j, lane));
        }
#pragma unroll
      for (int c = 0; c < kFixBatch; ++c)
        if (c < nb) {
#pragma unroll
          for (int j = 0; j < TN; ++j) acc[0][j] += v[c][j];
        }
      nb = 0;
    };
    auto push = [&](const float *slot) {
#pragma unroll
      for (int c = 0; c < kFixBatch; ++c)
        if (c == nb) b[c] = slot;
      if (++nb == kFixBatch) flush();
    };
    bool done_whole = false;
    for (int pc = 0; pc < q.s; ++pc) {
      const int u = pc * q.T + t;
      if (u < q.dp) {
        push(p.part + size_t(u) * T::kPartFloats);
        continue;
      }
      const int v = u - q.dp;
      const long long a0 = (long long)v * q.len;
      const int w0 = sk_owner(q.I, q.Pk, a0), w1 = sk_owner(q.I, q.Pk, a0 + q.len - 1);
      if (q.s == 1 && w0 == w1) {  // one workgroup held the whole tile and finished it
        done_whole = true;
        break;
      }
      // contributors in workgroup order.  Range starts floor(I w / Pk) advance by additions (no
      // 64-bit division per contributor); a range's first unit is v exactly when it starts at or
      // after unit v's first iteration.
      const int Pk = q.Pk;
      const long long qI = q.I / Pk, rI = q.I - qI * Pk;
      long long qb = q.I * w0 / Pk, rb = q.I * w0 - qb * Pk;
      for (int w = w0; w <= w1; ++w) {
        long long qn = qb + qI, rn = rb + rI;
        if (rn >= Pk) {
          ++qn;
          rn -= Pk;
        }
        if (qb < qn) push(p.part + (size_t(P) + size_t(w) * 2 + (qb >= a0 ? 0 : 1)) * T::kPartFloats);
        qb = qn;
        rb = rn;
      }
    }
    if (done_whole) continue;
    flush();
    int rt, tn;
    tile_coords(q, t, rt, tn);
    const TileRows tr = decode_row_tile(p, BM, rt);
    if constexpr (F8 && EPI == EPI_BIAS && BN == 256) {
      if (p.qk8 != nullptr && tn * BN < 2 * p.D) {
        T::epilogue_rows_qk8(p, tr, tn * BN, wid, i, lane, acc);
        continue;
      }
    }
    T::template epilogue_rows<EPI, 1, F8>(p, tr, tn * BN, wid, i, lane, acc);
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

// CUs of the current device (cached per device).
int device_cus() {
  static int ncu[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) dev = 0;
  if (ncu[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
      n = kBigMaxWorkgroups;
    ncu[dev] = n;
  }
  return ncu[dev];
}

// BM x BN tiles: one persistent workgroup per CU.
template <int BM, int BN, int ROLE, bool F8 = false>
static hipError_t run_big(const GemmProblem &p, hipStream_t st) {
  static_assert(size_t(BM) * BN * 3 * kBigMaxWorkgroups * sizeof(float) <= kSkPartBytes, "partial area too small");
  const int P = device_cus() < kBigMaxWorkgroups ? device_cus() : kBigMaxWorkgroups;
  hipLaunchKernelGGL((k_gemm_big<BM, BN, role_epilogue(ROLE), ROLE, F8>), dim3(P), dim3(256), 0, st, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const bool long_k = p.K / (F8 ? 128 : 64) > kNoSplitSteps;
  const long long tiles_max = (long long)p.B * ((p.max_img_rows + BM - 1) / BM + (p.L + BM - 1) / BM) *
                              ((p.N + BN - 1) / BN);
  if (tiles_max < P && !long_k) return hipSuccess;
  // P workgroups stride over the fixup's items: few enough that a launch with nothing to finish
  // (the device's row counts led to whole tiles) costs little
  hipLaunchKernelGGL((k_gemm_fix<BM, BN, 2, 2, role_epilogue(ROLE), ROLE, F8>), dim3(P), dim3(kFixThreads), 0, st, p, P);
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

hipError_t launch_gemm(bool bf16, int role, const GemmProblem &p, hipStream_t st) {
  if (!bf16) {
    switch (role_epilogue(role)) {
      case EPI_BIAS: return run_f32<EPI_BIAS>(p, st);
      case EPI_GELU: return run_f32<EPI_GELU>(p, st);
      default: return run_f32<EPI_RESID>(p, st);
    }
  }
  // Every projection on 192 x 192 tiles, whose K steps run through the LDS as whole 128-byte
  // lines.  At 2766 rows (the 64 x 64 workload): QKV 720 tiles in three whole waves, MLP up 960 in
  // four, the attention output and MLP down (N = 3072) 240 tiles in one wave with no K split.  256 x
  // 256 tiles (half-line stages) cost slightly less per output but quantise these row counts worse:
  // QKV took 178 us as two launches (256 x 256, then 256 x 192 for the columns one wave could not
  // hold) against 161, MLP up 230 us as two waves plus a stream-K tail against 218.
  switch (role) {
    case GEMM_QKV: return run_big<192, 192, GEMM_QKV>(p, st);
    case GEMM_O: return run_big<192, 192, GEMM_O>(p, st);
    case GEMM_FC1: return run_big<192, 192, GEMM_FC1>(p, st);
    default: return run_big<192, 192, GEMM_FC2>(p, st);
  }
}

hipError_t launch_gemm_fp8(int role, const GemmProblem &p, hipStream_t st) {
  switch (role) {
    // the FP8 QKV projection always writes FP8 q / k: 256-column tiles (whole heads per wave)
    case GEMM_QKV: return p.qk8 ? run_big<256, 256, GEMM_QKV, true>(p, st) : hipErrorInvalidValue;
    case GEMM_O: return run_big<192, 192, GEMM_O, true>(p, st);
    case GEMM_FC1: return run_big<192, 192, GEMM_FC1, true>(p, st);
    default: return run_big<192, 192, GEMM_FC2, true>(p, st);
  }
}

}  // namespace hilo
