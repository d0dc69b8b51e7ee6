// C ABI of libhilo: argument validation, workspace layout, kernel sequencing and the optional
// per-kernel event timing.  Nothing here allocates device memory or synchronises.
#include <cmath>
#include <mutex>
#include <vector>

#include "../../include/hilo.h"
#include "kernels.h"

using namespace hilo;

namespace {

// ----------------------------------------------------------------------------- kernel timing

enum Kind {
  K_SCORE, K_SELECT, K_LAYOUT, K_COMPRESS, K_NORM_ATTN, K_GEMM_QKV, K_ATTN_CORE, K_GEMM_O,
  K_NORM_MLP, K_GEMM_FC1, K_GEMM_FC2, K_DECOMPRESS, K_QUANT_ATTN, K_QUANT_MLP, K_COUNT
};
const char *kKindNames[K_COUNT] = {"score", "select", "layout", "compress", "rownorm_attn",
                                   "gemm_qkv", "attention_core", "gemm_o", "rownorm_mlp",
                                   "gemm_fc1", "gemm_fc2", "decompress", "quantize_attn",
                                   "quantize_mlp"};

struct ProfRec {
  int kind;
  hipEvent_t a, b;
};
bool g_prof = false;
std::vector<ProfRec> g_recs;
size_t g_used = 0;
constexpr size_t kMaxRecs = 1 << 16;

// Runs `launch` bracketed by events when timing is on.
template <typename F>
hipError_t timed(int kind, hipStream_t st, F &&launch) {
  if (!g_prof || g_used >= kMaxRecs) return launch();
  if (g_used == g_recs.size()) {
    ProfRec r{kind, nullptr, nullptr};
    if (hipEventCreate(&r.a) != hipSuccess) return launch();
    if (hipEventCreate(&r.b) != hipSuccess) {
      (void)hipEventDestroy(r.a);
      return launch();
    }
    g_recs.push_back(r);
  }
  ProfRec &r = g_recs[g_used];
  r.kind = kind;
  hipError_t e = hipEventRecord(r.a, st);
  if (e != hipSuccess) return e;
  e = launch();
  if (e != hipSuccess) return e;
  e = hipEventRecord(r.b, st);
  if (e == hipSuccess) ++g_used;  // only a launch bracketed by both events is read back
  return e;
}

// ----------------------------------------------------------------------------- validation

int g_ndev = -1;
bool have_device() {
  if (g_ndev < 0) {
    int n = 0;
    if (hipGetDeviceCount(&n) != hipSuccess) n = 0;
    g_ndev = n;
  }
  return g_ndev > 0;
}

hilo_status check_grid(const hilo_shape *s) {
  if (!s) return HILO_E_NULL;
  if (s->dtype != HILO_F32 && s->dtype != HILO_BF16) return HILO_E_DTYPE;
  if (s->batch <= 0 || s->images <= 0 || s->grid_h <= 0 || s->grid_w <= 0) return HILO_E_SHAPE;
  if ((s->grid_h & 1) || (s->grid_w & 1)) return HILO_E_SHAPE;
  if (s->text_len < 0) return HILO_E_SHAPE;
  if (s->dim <= 0 || s->dim % 64 != 0 || s->dim > 8192) return HILO_E_SHAPE;
  const long long N = (long long)s->grid_h * s->grid_w;
  if (N / 4 > 16384) return HILO_E_SHAPE;
  const long long tmax = (long long)s->batch * (s->images * (N + N / 4) + s->text_len);
  if (tmax >= (1LL << 31) / 8) return HILO_E_SHAPE;
  return HILO_OK;
}

hilo_status check_block(const hilo_shape *s) {
  hilo_status e = check_grid(s);
  if (e != HILO_OK) return e;
  if (s->heads <= 0 || s->head_dim <= 0 || (long long)s->heads * s->head_dim != s->dim)
    return HILO_E_SHAPE;
  if (s->mlp_dim <= 0 || s->mlp_dim % 64 != 0 || s->mlp_dim > 65536) return HILO_E_SHAPE;
  if (s->head_dim != 64 && s->head_dim != 128) return HILO_E_DTYPE;
  return HILO_OK;
}

// image rows per grid: at most every patch fine plus one pooled token per block (token set
// "overlap"); partition and drop sets stay within N
long long grid_rows_max(const hilo_shape *s) {
  const long long N = (long long)s->grid_h * s->grid_w;
  return N + N / 4;
}

long long tmax_of(const hilo_shape *s) {
  return (long long)s->batch * ((long long)s->images * grid_rows_max(s) + s->text_len);
}

size_t esize(const hilo_shape *s) { return s->dtype == HILO_BF16 ? 2 : 4; }

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// Partial-result region shared by the stream-K GEMMs and the stream-K attention core (they never
// run at the same time on one stream).
constexpr size_t kPartBytes = kSkPartBytes > kAttnPartBytes ? kSkPartBytes : kAttnPartBytes;
size_t ws_part(const hilo_shape *s) { return s->dtype == HILO_BF16 ? kPartBytes : 0; }

// The normalised rows: T x D of dtype, or for the FP8 projections T x D codes followed (at
// align256(T D)) by T float32 row scales.  The attention output reuses the region.
size_t ws_h(const hilo_shape *s) {
  const size_t T = size_t(tmax_of(s)), D = size_t(s->dim);
  const size_t a = align256(T * D * esize(s)), f8 = align256(T * D) + align256(T * sizeof(float));
  return a > f8 ? a : f8;
}

size_t ws_attention(const hilo_shape *s) {
  const size_t T = size_t(tmax_of(s)), D = size_t(s->dim), e = esize(s);
  return ws_h(s) + align256(T * 3 * D * e) + ws_part(s);  // h (then a), qkv, partials
}

size_t ws_mlp(const hilo_shape *s) {
  const size_t T = size_t(tmax_of(s)), F = size_t(s->mlp_dim), e = esize(s);
  return ws_h(s) + align256(T * F * e) + ws_part(s);  // h2, hidden, partials
}

// The FP8 block keeps one more region behind everything the bf16 block uses (at
// hilo_workspace_bytes): the attention output's bf16 rows in the attention half (the normalised
// rows' codes in the first region stay intact), the hidden rows' codes [T][F] and T row scales in
// the MLP half.
size_t ws_fp8_base(const hilo_shape *s) {
  const size_t a = ws_attention(s), m = ws_mlp(s);
  return a > m ? a : m;
}

size_t ws_fp8_extra(const hilo_shape *s) {
  const size_t T = size_t(tmax_of(s)), D = size_t(s->dim), F = size_t(s->mlp_dim);
  const size_t codes = align256(T * F) + align256(T * sizeof(float)), aout = align256(T * D * 2);
  return codes > aout ? codes : aout;
}

size_t ws_fp8(const hilo_shape *s) { return ws_fp8_base(s) + ws_fp8_extra(s); }

hilo_status dev_status(hipError_t e) { return e == hipSuccess ? HILO_OK : HILO_E_DEVICE; }

GemmProblem base_problem(const hilo_shape *s, const int32_t *cu, const float *mod, float *part) {
  GemmProblem p{};
  p.part = part;
  p.mod = mod;
  p.D = s->dim;
  p.cu = cu;
  p.B = s->batch;
  p.L = s->text_len;
  p.max_img_rows = int(s->images * grid_rows_max(s));
  return p;
}

}  // namespace

extern "C" {

int32_t hilo_abi_version(void) { return HILO_ABI_VERSION; }

const char *hilo_status_str(int32_t st) {
  switch (st) {
    case HILO_OK: return "ok";
    case HILO_E_NULL: return "required pointer is NULL";
    case HILO_E_SHAPE: return "invalid or unsupported shape";
    case HILO_E_DTYPE: return "unsupported dtype or head_dim";
    case HILO_E_PARAM: return "invalid selection parameter";
    case HILO_E_WORKSPACE: return "workspace too small";
    case HILO_E_DEVICE: return "HIP launch failed or no GPU";
    default: return "unknown status";
  }
}

int64_t hilo_max_tokens(const hilo_shape *s) {
  if (check_grid(s) != HILO_OK) return -1;
  return tmax_of(s);
}

size_t hilo_workspace_bytes(const hilo_shape *s) {
  if (check_block(s) != HILO_OK) return 0;
  const size_t a = ws_attention(s), m = ws_mlp(s);
  return a > m ? a : m;
}

hilo_status hilo_score(const hilo_shape *s, const void *x_img, int64_t *energy, void *stream) {
  hilo_status e = check_grid(s);
  if (e != HILO_OK) return e;
  if (!x_img || !energy) return HILO_E_NULL;
  if (!have_device()) return HILO_E_DEVICE;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  return dev_status(timed(K_SCORE, st, [&] {
    return launch_score(s->dtype == HILO_BF16, x_img, reinterpret_cast<long long *>(energy),
                        s->batch * s->images, s->grid_h, s->grid_w, s->dim, st);
  }));
}

hilo_status hilo_score_pixels(const hilo_shape *s, const float *rgb, int64_t *energy, void *stream) {
  hilo_status e = check_grid(s);
  if (e != HILO_OK) return e;
  if (!rgb || !energy) return HILO_E_NULL;
  if ((long long)s->grid_h * 16 * s->grid_w * 16 * 3 * s->batch * s->images >= (1LL << 31)) return HILO_E_SHAPE;
  if (!have_device()) return HILO_E_DEVICE;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  return dev_status(timed(K_SCORE, st, [&] {
    return launch_score_pixels(rgb, reinterpret_cast<long long *>(energy), s->batch * s->images,
                               s->grid_h, s->grid_w, st);
  }));
}

hilo_status hilo_select(const hilo_shape *s, const int64_t *energy, const uint8_t *force,
                        int32_t dilate_r, int32_t mode, const double *tau, const int32_t *keep,
                        int32_t *idx_map, int32_t *fine_idx, int32_t *pool_idx, int32_t *counts,
                        int32_t *cu_seqlens, int32_t *seg_off, void *stream) {
  return hilo_select_tokens(s, energy, force, dilate_r, mode, tau, keep, HILO_TOKENS_PARTITION,
                            idx_map, fine_idx, pool_idx, counts, cu_seqlens, seg_off, stream);
}

hilo_status hilo_select_tokens(const hilo_shape *s, const int64_t *energy, const uint8_t *force,
                               int32_t dilate_r, int32_t mode, const double *tau,
                               const int32_t *keep, int32_t token_set, int32_t *idx_map,
                               int32_t *fine_idx, int32_t *pool_idx, int32_t *counts,
                               int32_t *cu_seqlens, int32_t *seg_off, void *stream) {
  hilo_status e = check_grid(s);
  if (e != HILO_OK) return e;
  if (!energy || !idx_map || !fine_idx || !pool_idx || !counts || !cu_seqlens || !seg_off)
    return HILO_E_NULL;
  if (mode != HILO_SELECT_THRESHOLD && mode != HILO_SELECT_TOPK) return HILO_E_PARAM;
  if (token_set != HILO_TOKENS_PARTITION && token_set != HILO_TOKENS_OVERLAP &&
      token_set != HILO_TOKENS_DROP)
    return HILO_E_PARAM;
  if (dilate_r < 0) return HILO_E_PARAM;
  const int G = s->batch * s->images;
  const int NB = s->grid_h * s->grid_w / 4;
  if (mode == HILO_SELECT_THRESHOLD) {
    if (!tau) return HILO_E_NULL;
    for (int g = 0; g < G; ++g)
      if (!std::isfinite(tau[g])) return HILO_E_PARAM;
  } else {
    if (!keep) return HILO_E_NULL;
    for (int g = 0; g < G; ++g)
      if (keep[g] < 0 || keep[g] > NB) return HILO_E_PARAM;
  }
  if (!have_device()) return HILO_E_DEVICE;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  const int r = dilate_r > s->grid_h + s->grid_w ? s->grid_h + s->grid_w : dilate_r;
  hipError_t he = timed(K_SELECT, st, [&] {
    // one grid: the selection writes the layout itself (one launch less)
    const bool one = G == 1;
    return launch_select(reinterpret_cast<const long long *>(energy), force, G, s->grid_h,
                         s->grid_w, r, mode, token_set, tau, keep, idx_map, fine_idx, pool_idx,
                         counts, one ? cu_seqlens : nullptr, one ? seg_off : nullptr, s->text_len, st);
  });
  if (he != hipSuccess) return HILO_E_DEVICE;
  if (G == 1) return HILO_OK;
  return dev_status(timed(K_LAYOUT, st, [&] {
    return launch_layout(counts, s->batch, s->images, s->text_len, cu_seqlens, seg_off, st);
  }));
}

hilo_status hilo_compress(const hilo_shape *s, const void *x_img, const void *x_txt,
                          const int32_t *fine_idx, const int32_t *pool_idx, const int32_t *counts,
                          const int32_t *cu_seqlens, const int32_t *seg_off, float *z,
                          void *stream) {
  hilo_status e = check_grid(s);
  if (e != HILO_OK) return e;
  if (!x_img || !fine_idx || !pool_idx || !counts || !cu_seqlens || !seg_off || !z)
    return HILO_E_NULL;
  if (s->text_len > 0 && !x_txt) return HILO_E_NULL;
  if (!have_device()) return HILO_E_DEVICE;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  return dev_status(timed(K_COMPRESS, st, [&] {
    return launch_compress(s->dtype == HILO_BF16, x_img, x_txt, fine_idx, pool_idx, counts,
                           cu_seqlens, seg_off, z, s->batch, s->images, s->grid_h, s->grid_w,
                           s->dim, s->text_len, st);
  }));
}

hilo_status hilo_decompress(const hilo_shape *s, const float *z, const int32_t *idx_map,
                            const int32_t *cu_seqlens, const int32_t *seg_off, void *y_img,
                            void *y_txt, void *stream) {
  hilo_status e = check_grid(s);
  if (e != HILO_OK) return e;
  if (!z || !idx_map || !cu_seqlens || !seg_off || !y_img) return HILO_E_NULL;
  if (!have_device()) return HILO_E_DEVICE;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  return dev_status(timed(K_DECOMPRESS, st, [&] {
    return launch_decompress(s->dtype == HILO_BF16, z, idx_map, cu_seqlens, seg_off, y_img,
                             s->text_len > 0 ? y_txt : nullptr, s->batch, s->images,
                             s->grid_h * s->grid_w, s->dim, s->text_len, st);
  }));
}

hilo_status hilo_decompress_delta(const hilo_shape *s, const float *z, const void *x_img,
                                  const int32_t *idx_map, const int32_t *counts,
                                  const int32_t *cu_seqlens, const int32_t *seg_off, void *y_img,
                                  void *y_txt, void *stream) {
  hilo_status e = check_grid(s);
  if (e != HILO_OK) return e;
  if (!z || !x_img || !idx_map || !counts || !cu_seqlens || !seg_off || !y_img) return HILO_E_NULL;
  if (!have_device()) return HILO_E_DEVICE;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  return dev_status(timed(K_DECOMPRESS, st, [&] {
    return launch_decompress_delta(s->dtype == HILO_BF16, z, x_img, idx_map, counts, cu_seqlens,
                                   seg_off, y_img, s->text_len > 0 ? y_txt : nullptr, s->batch,
                                   s->images, s->grid_h, s->grid_w, s->dim, s->text_len, st);
  }));
}

hilo_status hilo_attention_core(const hilo_shape *s, const void *qkv, const int32_t *cu_seqlens,
                                void *out, void *workspace, size_t ws_bytes, void *stream) {
  hilo_status e = check_block(s);
  if (e != HILO_OK) return e;
  if (!qkv || !cu_seqlens || !out) return HILO_E_NULL;
  if (ws_part(s) && !workspace) return HILO_E_NULL;
  if (ws_bytes < ws_part(s)) return HILO_E_WORKSPACE;
  if (!have_device()) return HILO_E_DEVICE;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  const int max_seq = int(s->images * grid_rows_max(s) + s->text_len);
  return dev_status(timed(K_ATTN_CORE, st, [&] {
    return launch_attention(s->dtype == HILO_BF16, qkv, cu_seqlens, out,
                            reinterpret_cast<float *>(workspace), s->batch, s->heads, s->head_dim,
                            max_seq, st);
  }));
}

}  // extern "C"

// ----------------------------------------------------------------- allocation-free attention core

// Scratch of hilo_attention_core_noalloc: the attention core's stream-K partial results, in a
// device array of the library's own (each GPU the library runs on holds one copy, allocated when
// the library's code is loaded there and kept until the process ends).  Host code never passes
// `scratch` itself to a kernel (on the host the name is only a stand-in for the symbol): it passes
// the device address hipGetSymbolAddress returns for the current device.
static __device__ __align__(256) uint8_t scratch[HILO_ATTN_SCRATCH_BYTES];
static_assert(HILO_ATTN_SCRATCH_BYTES >= kAttnPartBytes, "scratch smaller than the attention partials");

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};

// The current device's address of `scratch`, looked up once per device (with that device current:
// every device has its own copy at its own address); nullptr if the lookup fails.
void *scratch_ptr() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void *ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || ptr == nullptr) return nullptr;
    g_scratch_ptr[dev] = ptr;
  }
  return g_scratch_ptr[dev];
}

}  // namespace

extern "C" {

hilo_status hilo_attention_core_noalloc(const hilo_shape *s, const void *qkv,
                                        const int32_t *cu_seqlens, void *out, void *stream) {
  hilo_status e = check_block(s);
  if (e != HILO_OK) return e;
  if (!qkv || !cu_seqlens || !out) return HILO_E_NULL;
  if (!have_device()) return HILO_E_DEVICE;
  const bool bf = s->dtype == HILO_BF16;
  if (attention_part_bytes(bf, s->head_dim) > HILO_ATTN_SCRATCH_BYTES) return HILO_E_WORKSPACE;
  float *part = nullptr;
  if (bf) {
    part = reinterpret_cast<float *>(scratch_ptr());
    if (!part) return HILO_E_DEVICE;
  }
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  const int max_seq = int(s->images * grid_rows_max(s) + s->text_len);
  return dev_status(launch_attention(bf, qkv, cu_seqlens, out, part, s->batch, s->heads, s->head_dim,
                                     max_seq, st));
}

}  // extern "C"

namespace {

hilo_status check_attn_w(const hilo_attn_w *w) {
  if (!w) return HILO_E_NULL;
  for (int k = 0; k < 2; ++k)
    if (!w[k].w_qkv || !w[k].b_qkv || !w[k].w_o || !w[k].b_o) return HILO_E_NULL;
  return HILO_OK;
}

hilo_status check_mlp_w(const hilo_mlp_w *w) {
  if (!w) return HILO_E_NULL;
  for (int k = 0; k < 2; ++k)
    if (!w[k].w1 || !w[k].b1 || !w[k].w2 || !w[k].b2) return HILO_E_NULL;
  return HILO_OK;
}

hilo_status check_attn_w8(const hilo_attn_w_fp8 *w) {
  if (!w) return HILO_E_NULL;
  for (int k = 0; k < 2; ++k)
    if (!w[k].w_qkv || !w[k].s_qkv || !w[k].b_qkv || !w[k].w_o || !w[k].s_o || !w[k].b_o) return HILO_E_NULL;
  return HILO_OK;
}

hilo_status check_mlp_w8(const hilo_mlp_w_fp8 *w) {
  if (!w) return HILO_E_NULL;
  for (int k = 0; k < 2; ++k)
    if (!w[k].w1 || !w[k].s1 || !w[k].b1 || !w[k].w2 || !w[k].s2 || !w[k].b2) return HILO_E_NULL;
  return HILO_OK;
}

// The FP8 block: bf16 shape; every projection's K (dim, mlp_dim) in whole 128-deep steps, and dim a
// multiple of 256, so that the QKV projection's 256-column tiles hold whole heads of q and k.
hilo_status check_fp8_block(const hilo_shape *s) {
  hilo_status e = check_block(s);
  if (e != HILO_OK) return e;
  if (s->dtype != HILO_BF16) return HILO_E_DTYPE;
  if (s->dim % 256 != 0 || s->mlp_dim % 128 != 0) return HILO_E_SHAPE;
  return HILO_OK;
}

// Row scales of the FP8 normalised rows, behind their codes.
float *fp8_row_scales(const hilo_shape *s, void *h) {
  return reinterpret_cast<float *>(reinterpret_cast<char *>(h) + align256(size_t(tmax_of(s)) * s->dim));
}

// The attention half, arguments already validated: bf16 / float32 weights w, or (w8 non-null) the
// FP8 QKV projection.
hilo_status enqueue_attention(const hilo_shape *s, float *z, const int32_t *cu_seqlens,
                              const hilo_attn_w *w, const hilo_attn_w_fp8 *w8, const float *mod,
                              void *workspace, hipStream_t st, bool normed = false) {
  const bool bf = s->dtype == HILO_BF16;
  const int D = s->dim;
  const int T = int(tmax_of(s));
  char *ws = reinterpret_cast<char *>(workspace);
  void *h = ws;  // LN output, later the attention output
  void *qkv = ws + ws_h(s);
  float *part = reinterpret_cast<float *>(ws + ws_h(s) + align256(size_t(T) * 3 * D * esize(s)));
  float *hs = fp8_row_scales(s, h);

  hipError_t he = hipSuccess;
  // the normalised rows are already in place when hilo_compress_norm wrote them
  if (!normed) {
    he = timed(K_NORM_ATTN, st, [&] {
      return w8 ? launch_rownorm_fp8(z, cu_seqlens, mod, s->batch, s->text_len, D, T, 0,
                                     reinterpret_cast<uint8_t *>(h), hs, st)
                : launch_rownorm(bf, z, cu_seqlens, mod, s->batch, s->text_len, D, T, 0, h, st);
    });
    if (he != hipSuccess) return HILO_E_DEVICE;
  }

  GemmProblem p = base_problem(s, cu_seqlens, mod, part);
  p.A = h; p.lda = D;
  p.N = 3 * D; p.K = D;
  p.out = qkv; p.ldo = 3 * D;
  // FP8 block: q and k leave the projection as E4M3 codes with per-(row, head) power-of-two scales,
  // in the first 2 D bytes (codes) and the next 2 H bytes (scales) of each row of the qkv region;
  // v stays bf16 in its columns
  uint8_t *qk8 = w8 ? reinterpret_cast<uint8_t *>(qkv) : nullptr;
  const int ldq8 = 3 * D * 2;
  if (w8) {
    p.W[0] = w8[0].w_qkv; p.W[1] = w8[1].w_qkv;
    p.bias[0] = w8[0].b_qkv; p.bias[1] = w8[1].b_qkv;
    p.a_scale = hs;
    p.w_scale[0] = w8[0].s_qkv; p.w_scale[1] = w8[1].s_qkv;
    p.qk8 = qk8; p.ldq8 = ldq8; p.head_dim = s->head_dim;
    he = timed(K_GEMM_QKV, st, [&] { return launch_gemm_fp8(GEMM_QKV, p, st); });
  } else {
    p.W[0] = w[0].w_qkv; p.W[1] = w[1].w_qkv;
    p.bias[0] = w[0].b_qkv; p.bias[1] = w[1].b_qkv;
    he = timed(K_GEMM_QKV, st, [&] { return launch_gemm(bf, GEMM_QKV, p, st); });
  }
  if (he != hipSuccess) return HILO_E_DEVICE;

  const int max_seq = int(s->images * grid_rows_max(s) + s->text_len);
  // the attention output: over the normalised rows (bf16 block), or behind the bf16 block's
  // regions (FP8 block, whose normalised-row codes stay in place)
  void *aout = w8 ? static_cast<void *>(ws + ws_fp8_base(s)) : h;
  he = timed(K_ATTN_CORE, st, [&] {
    return launch_attention(bf, qkv, cu_seqlens, aout, part, s->batch, s->heads, s->head_dim,
                            max_seq, st, qk8, ldq8);
  });
  if (he != hipSuccess) return HILO_E_DEVICE;

  GemmProblem q = base_problem(s, cu_seqlens, mod, part);
  q.A = h; q.lda = D;
  q.N = D; q.K = D;
  q.z = z; q.ldz = D; q.gate_idx = 2;
  if (w8) {
    // the attention output's rows as FP8 codes and scales, in the QKV region (free again)
    uint8_t *ac = reinterpret_cast<uint8_t *>(qkv);
    float *as = reinterpret_cast<float *>(ac + align256(size_t(T) * D));
    he = timed(K_QUANT_ATTN, st, [&] { return launch_quantize_rows(true, aout, T, D, ac, as, st, cu_seqlens + s->batch); });
    if (he != hipSuccess) return HILO_E_DEVICE;
    q.A = ac;
    q.W[0] = w8[0].w_o; q.W[1] = w8[1].w_o;
    q.bias[0] = w8[0].b_o; q.bias[1] = w8[1].b_o;
    q.a_scale = as;
    q.w_scale[0] = w8[0].s_o; q.w_scale[1] = w8[1].s_o;
    return dev_status(timed(K_GEMM_O, st, [&] { return launch_gemm_fp8(GEMM_O, q, st); }));
  }
  q.W[0] = w[0].w_o; q.W[1] = w[1].w_o;
  q.bias[0] = w[0].b_o; q.bias[1] = w[1].b_o;
  return dev_status(timed(K_GEMM_O, st, [&] { return launch_gemm(bf, GEMM_O, q, st); }));
}

// The MLP half, arguments already validated: bf16 / float32 weights w, or (w8 non-null) the FP8
// up projection.
hilo_status enqueue_mlp(const hilo_shape *s, float *z, const int32_t *cu_seqlens,
                        const hilo_mlp_w *w, const hilo_mlp_w_fp8 *w8, const float *mod,
                        void *workspace, hipStream_t st) {
  const bool bf = s->dtype == HILO_BF16;
  const int D = s->dim, F = s->mlp_dim;
  const int T = int(tmax_of(s));
  char *ws = reinterpret_cast<char *>(workspace);
  void *h2 = ws;
  void *hid = ws + ws_h(s);
  float *part = reinterpret_cast<float *>(ws + ws_h(s) + align256(size_t(T) * F * esize(s)));
  float *hs = fp8_row_scales(s, h2);

  hipError_t he = timed(K_NORM_MLP, st, [&] {
    return w8 ? launch_rownorm_fp8(z, cu_seqlens, mod, s->batch, s->text_len, D, T, 1,
                                   reinterpret_cast<uint8_t *>(h2), hs, st)
              : launch_rownorm(bf, z, cu_seqlens, mod, s->batch, s->text_len, D, T, 1, h2, st);
  });
  if (he != hipSuccess) return HILO_E_DEVICE;

  GemmProblem p = base_problem(s, cu_seqlens, mod, part);
  p.A = h2; p.lda = D;
  p.N = F; p.K = D;
  p.out = hid; p.ldo = F;
  if (w8) {
    p.W[0] = w8[0].w1; p.W[1] = w8[1].w1;
    p.bias[0] = w8[0].b1; p.bias[1] = w8[1].b1;
    p.a_scale = hs;
    p.w_scale[0] = w8[0].s1; p.w_scale[1] = w8[1].s1;
    he = timed(K_GEMM_FC1, st, [&] { return launch_gemm_fp8(GEMM_FC1, p, st); });
  } else {
    p.W[0] = w[0].w1; p.W[1] = w[1].w1;
    p.bias[0] = w[0].b1; p.bias[1] = w[1].b1;
    he = timed(K_GEMM_FC1, st, [&] { return launch_gemm(bf, GEMM_FC1, p, st); });
  }
  if (he != hipSuccess) return HILO_E_DEVICE;

  GemmProblem q = base_problem(s, cu_seqlens, mod, part);
  q.A = hid; q.lda = F;
  q.N = D; q.K = F;
  q.z = z; q.ldz = D; q.gate_idx = 5;
  if (w8) {
    // the hidden rows as FP8 codes and scales, behind everything the bf16 block uses
    uint8_t *hc = reinterpret_cast<uint8_t *>(ws + ws_fp8_base(s));
    float *hs8 = reinterpret_cast<float *>(hc + align256(size_t(T) * F));
    he = timed(K_QUANT_MLP, st, [&] { return launch_quantize_rows(true, hid, T, F, hc, hs8, st, cu_seqlens + s->batch); });
    if (he != hipSuccess) return HILO_E_DEVICE;
    q.A = hc;
    q.W[0] = w8[0].w2; q.W[1] = w8[1].w2;
    q.bias[0] = w8[0].b2; q.bias[1] = w8[1].b2;
    q.a_scale = hs8;
    q.w_scale[0] = w8[0].s2; q.w_scale[1] = w8[1].s2;
    return dev_status(timed(K_GEMM_FC2, st, [&] { return launch_gemm_fp8(GEMM_FC2, q, st); }));
  }
  q.W[0] = w[0].w2; q.W[1] = w[1].w2;
  q.bias[0] = w[0].b2; q.bias[1] = w[1].b2;
  return dev_status(timed(K_GEMM_FC2, st, [&] { return launch_gemm(bf, GEMM_FC2, q, st); }));
}

}  // namespace

extern "C" {

hilo_status hilo_attention(const hilo_shape *s, float *z, const int32_t *cu_seqlens,
                           const hilo_attn_w w[2], const float *mod, void *workspace,
                           size_t ws_bytes, void *stream) {
  hilo_status e = check_block(s);
  if (e != HILO_OK) return e;
  if (!z || !cu_seqlens || !mod || !workspace) return HILO_E_NULL;
  if ((e = check_attn_w(w)) != HILO_OK) return e;
  if (ws_bytes < ws_attention(s)) return HILO_E_WORKSPACE;
  if (!have_device()) return HILO_E_DEVICE;
  return enqueue_attention(s, z, cu_seqlens, w, nullptr, mod, workspace, reinterpret_cast<hipStream_t>(stream));
}

hilo_status hilo_compress_norm(const hilo_shape *s, const void *x_img, const void *x_txt,
                               const int32_t *fine_idx, const int32_t *pool_idx, const int32_t *counts,
                               const int32_t *cu_seqlens, const int32_t *seg_off, const float *mod,
                               float *z, void *workspace, size_t ws_bytes, void *stream) {
  hilo_status e = check_block(s);
  if (e != HILO_OK) return e;
  if (!x_img || !fine_idx || !pool_idx || !counts || !cu_seqlens || !seg_off || !mod || !z || !workspace)
    return HILO_E_NULL;
  if (s->text_len > 0 && !x_txt) return HILO_E_NULL;
  if (ws_bytes < ws_attention(s)) return HILO_E_WORKSPACE;
  if (!have_device()) return HILO_E_DEVICE;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  return dev_status(timed(K_COMPRESS, st, [&] {
    return launch_compress_norm(s->dtype == HILO_BF16, x_img, x_txt, fine_idx, pool_idx, counts,
                                cu_seqlens, seg_off, mod, z, s->batch, s->images, s->grid_h,
                                s->grid_w, s->dim, s->text_len, workspace, st);
  }));
}

hilo_status hilo_attention_normed(const hilo_shape *s, float *z, const int32_t *cu_seqlens,
                                  const hilo_attn_w w[2], const float *mod, void *workspace,
                                  size_t ws_bytes, void *stream) {
  hilo_status e = check_block(s);
  if (e != HILO_OK) return e;
  if (!z || !cu_seqlens || !mod || !workspace) return HILO_E_NULL;
  if ((e = check_attn_w(w)) != HILO_OK) return e;
  if (ws_bytes < ws_attention(s)) return HILO_E_WORKSPACE;
  if (!have_device()) return HILO_E_DEVICE;
  return enqueue_attention(s, z, cu_seqlens, w, nullptr, mod, workspace, reinterpret_cast<hipStream_t>(stream),
                           true);
}

hilo_status hilo_mlp(const hilo_shape *s, float *z, const int32_t *cu_seqlens,
                     const hilo_mlp_w w[2], const float *mod, void *workspace, size_t ws_bytes,
                     void *stream) {
  hilo_status e = check_block(s);
  if (e != HILO_OK) return e;
  if (!z || !cu_seqlens || !mod || !workspace) return HILO_E_NULL;
  if ((e = check_mlp_w(w)) != HILO_OK) return e;
  if (ws_bytes < ws_mlp(s)) return HILO_E_WORKSPACE;
  if (!have_device()) return HILO_E_DEVICE;
  return enqueue_mlp(s, z, cu_seqlens, w, nullptr, mod, workspace, reinterpret_cast<hipStream_t>(stream));
}

size_t hilo_workspace_bytes_fp8(const hilo_shape *s) {
  if (check_fp8_block(s) != HILO_OK) return 0;
  return ws_fp8(s);
}

hilo_status hilo_attention_fp8(const hilo_shape *s, float *z, const int32_t *cu_seqlens,
                               const hilo_attn_w_fp8 w[2], const float *mod, void *workspace,
                               size_t ws_bytes, void *stream) {
  hilo_status e = check_fp8_block(s);
  if (e != HILO_OK) return e;
  if (!z || !cu_seqlens || !mod || !workspace) return HILO_E_NULL;
  if ((e = check_attn_w8(w)) != HILO_OK) return e;
  if (ws_bytes < ws_fp8(s)) return HILO_E_WORKSPACE;
  if (!have_device()) return HILO_E_DEVICE;
  return enqueue_attention(s, z, cu_seqlens, nullptr, w, mod, workspace, reinterpret_cast<hipStream_t>(stream));
}

hilo_status hilo_compress_norm_fp8(const hilo_shape *s, const void *x_img, const void *x_txt,
                                   const int32_t *fine_idx, const int32_t *pool_idx, const int32_t *counts,
                                   const int32_t *cu_seqlens, const int32_t *seg_off, const float *mod,
                                   float *z, void *workspace, size_t ws_bytes, void *stream) {
  hilo_status e = check_fp8_block(s);
  if (e != HILO_OK) return e;
  if (!x_img || !fine_idx || !pool_idx || !counts || !cu_seqlens || !seg_off || !mod || !z || !workspace)
    return HILO_E_NULL;
  if (s->text_len > 0 && !x_txt) return HILO_E_NULL;
  if (ws_bytes < ws_fp8(s)) return HILO_E_WORKSPACE;
  if (!have_device()) return HILO_E_DEVICE;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  return dev_status(timed(K_COMPRESS, st, [&] {
    return launch_compress_norm(true, x_img, x_txt, fine_idx, pool_idx, counts, cu_seqlens, seg_off, mod, z,
                                s->batch, s->images, s->grid_h, s->grid_w, s->dim, s->text_len, workspace, st,
                                true, fp8_row_scales(s, workspace));
  }));
}

hilo_status hilo_attention_fp8_normed(const hilo_shape *s, float *z, const int32_t *cu_seqlens,
                                      const hilo_attn_w_fp8 w[2], const float *mod, void *workspace,
                                      size_t ws_bytes, void *stream) {
  hilo_status e = check_fp8_block(s);
  if (e != HILO_OK) return e;
  if (!z || !cu_seqlens || !mod || !workspace) return HILO_E_NULL;
  if ((e = check_attn_w8(w)) != HILO_OK) return e;
  if (ws_bytes < ws_fp8(s)) return HILO_E_WORKSPACE;
  if (!have_device()) return HILO_E_DEVICE;
  return enqueue_attention(s, z, cu_seqlens, nullptr, w, mod, workspace, reinterpret_cast<hipStream_t>(stream),
                           true);
}

hilo_status hilo_mlp_fp8(const hilo_shape *s, float *z, const int32_t *cu_seqlens,
                         const hilo_mlp_w_fp8 w[2], const float *mod, void *workspace, size_t ws_bytes,
                         void *stream) {
  hilo_status e = check_fp8_block(s);
  if (e != HILO_OK) return e;
  if (!z || !cu_seqlens || !mod || !workspace) return HILO_E_NULL;
  if ((e = check_mlp_w8(w)) != HILO_OK) return e;
  if (ws_bytes < ws_fp8(s)) return HILO_E_WORKSPACE;
  if (!have_device()) return HILO_E_DEVICE;
  return enqueue_mlp(s, z, cu_seqlens, nullptr, w, mod, workspace, reinterpret_cast<hipStream_t>(stream));
}

hilo_status hilo_attention_core_fp8(const hilo_shape *s, const void *qkv8, const int32_t *cu_seqlens,
                                    void *out, void *workspace, size_t ws_bytes, void *stream) {
  hilo_status e = check_fp8_block(s);
  if (e != HILO_OK) return e;
  if (!qkv8 || !cu_seqlens || !out || !workspace) return HILO_E_NULL;
  if (ws_bytes < ws_part(s)) return HILO_E_WORKSPACE;
  if (!have_device()) return HILO_E_DEVICE;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  const int max_seq = int(s->images * grid_rows_max(s) + s->text_len);
  return dev_status(timed(K_ATTN_CORE, st, [&] {
    return launch_attention(true, qkv8, cu_seqlens, out, reinterpret_cast<float *>(workspace), s->batch,
                            s->heads, s->head_dim, max_seq, st, reinterpret_cast<const uint8_t *>(qkv8),
                            6 * s->dim);
  }));
}

hilo_status hilo_quantize_rows(int32_t dtype, const void *x, int64_t rows, int64_t cols, uint8_t *codes,
                               float *scale, void *stream) {
  if (dtype != HILO_F32 && dtype != HILO_BF16) return HILO_E_DTYPE;
  if (rows < 0 || rows >= (1LL << 31) - 4 || cols <= 0 || cols % 4 != 0 || cols > (1LL << 31) - 1)
    return HILO_E_SHAPE;
  if (!x || !codes || !scale) return HILO_E_NULL;
  if (rows == 0) return HILO_OK;
  if (!have_device()) return HILO_E_DEVICE;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  return dev_status(launch_quantize_rows(dtype == HILO_BF16, x, int(rows), int(cols), codes, scale, st));
}

hilo_status hilo_blocks(const hilo_shape *s, float *z, const int32_t *cu_seqlens,
                        const hilo_attn_w *attn_w, const hilo_mlp_w *mlp_w, const float *mod,
                        int32_t n_blocks, void *workspace, size_t ws_bytes, void *stream) {
  hilo_status e = check_block(s);
  if (e != HILO_OK) return e;
  if (n_blocks < 0) return HILO_E_PARAM;
  if (!z || !cu_seqlens || !attn_w || !mlp_w || !mod || !workspace) return HILO_E_NULL;
  for (int l = 0; l < n_blocks; ++l) {
    if ((e = check_attn_w(attn_w + 2 * l)) != HILO_OK) return e;
    if ((e = check_mlp_w(mlp_w + 2 * l)) != HILO_OK) return e;
  }
  if (ws_bytes < hilo_workspace_bytes(s)) return HILO_E_WORKSPACE;
  if (!have_device()) return HILO_E_DEVICE;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  const size_t mod_stride = size_t(s->batch) * 2 * 6 * s->dim;
  for (int l = 0; l < n_blocks; ++l) {
    const float *ml = mod + l * mod_stride;
    if ((e = enqueue_attention(s, z, cu_seqlens, attn_w + 2 * l, nullptr, ml, workspace, st)) != HILO_OK) return e;
    if ((e = enqueue_mlp(s, z, cu_seqlens, mlp_w + 2 * l, nullptr, ml, workspace, st)) != HILO_OK) return e;
  }
  return HILO_OK;
}

hilo_status hilo_profile_enable(int32_t on) {
  g_prof = on != 0;
  if (g_prof) g_used = 0;
  return HILO_OK;
}

hilo_status hilo_profile_read(int32_t kind, double *total_ms, int64_t *launches) {
  if (!total_ms || !launches) return HILO_E_NULL;
  if (kind < 0 || kind >= K_COUNT) return HILO_E_PARAM;
  double tot = 0.0;
  int64_t n = 0;
  for (size_t i = 0; i < g_used; ++i) {
    if (g_recs[i].kind != kind) continue;
    float ms = 0.f;
    if (hipEventSynchronize(g_recs[i].b) != hipSuccess) return HILO_E_DEVICE;
    if (hipEventElapsedTime(&ms, g_recs[i].a, g_recs[i].b) != hipSuccess) return HILO_E_DEVICE;
    tot += ms;
    ++n;
  }
  *total_ms = tot;
  *launches = n;
  return HILO_OK;
}

int32_t hilo_profile_kinds(void) { return K_COUNT; }

const char *hilo_profile_name(int32_t kind) {
  return (kind >= 0 && kind < K_COUNT) ? kKindNames[kind] : "unknown";
}

}  // extern "C"
