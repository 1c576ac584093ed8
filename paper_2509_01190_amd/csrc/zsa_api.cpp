// C-ABI of libzsa: argument validation, the Eq. 2 keep-count schedule,
// workspace layout and the orchestration of the per-layer kernels.
// Everything here runs on the host and only enqueues work on the caller's
// stream; no call synchronises, allocates device memory or copies from host
// memory (host values reach kernels as launch arguments).
#include <algorithm>
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <string>
#include <vector>

#include "../../include/zsa.h"
#include "zsa_internal.h"

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

int hip_fail(hipError_t e, const char* what) {
  return fail(ZSA_EHIP, "%s: %s", what, hipGetErrorString(e));
}

#define HIP_TRY(expr, what)                          \
  do {                                               \
    const hipError_t e_ = (expr);                    \
    if (e_ != hipSuccess) return hip_fail(e_, what); \
  } while (0)

#define CHECK(expr)            \
  do {                         \
    const int rc_ = (expr);    \
    if (rc_ != ZSA_OK) return rc_; \
  } while (0)

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
inline size_t esize(int dtype) { return dtype == ZSA_BF16 ? 2 : 4; }
inline size_t round256(size_t b) { return (b + 255) & ~static_cast<size_t>(255); }

// Eq. 2 for one sequence. The product and the sum are two separately
// rounded IEEE double operations (the volatile store keeps the compiler from
// fusing them), exactly as written: floor(alpha * n + 1e-9), clipped to
// [tau, n] (never above n).
int32_t keep_count_impl(int32_t n, double alpha, int32_t tau) {
  volatile double prod = alpha * static_cast<double>(n);
  const double v = prod + 1e-9;
  int64_t k = static_cast<int64_t>(floor(v));
  if (k < tau) k = tau;
  if (k > n) k = n;
  return static_cast<int32_t>(k);
}

int check_rate(double a) {
  if (!(a >= 0.0 && a <= 1.0))  // also rejects NaN
    return fail(ZSA_EINVAL, "keep rate %g is NaN or outside [0, 1]", a);
  return ZSA_OK;
}

// validate packed sequence offsets; returns total rows and the longest length
int check_seqs(int32_t batch, const int32_t* cu_host, const int32_t* cu_dev, int32_t* total,
               int32_t* max_len) {
  if (batch < 0) return fail(ZSA_EINVAL, "batch %d < 0", batch);
  if (cu_host == nullptr || cu_dev == nullptr) return fail(ZSA_EINVAL, "cu_host / cu_dev is NULL");
  if (cu_host[0] != 0) return fail(ZSA_ESHAPE, "cu[0] = %d, must be 0", cu_host[0]);
  int32_t ml = 0;
  for (int b = 0; b < batch; ++b) {
    const int32_t len = cu_host[b + 1] - cu_host[b];
    if (len < 0) return fail(ZSA_ESHAPE, "cu not monotone at sequence %d", b);
    if (len > ml) ml = len;
  }
  *total = cu_host[batch];
  *max_len = ml;
  return ZSA_OK;
}

int check_dtype(int32_t dtype) {
  if (dtype != ZSA_F32 && dtype != ZSA_BF16) return fail(ZSA_EINVAL, "dtype %d unknown", dtype);
  return ZSA_OK;
}

int check_ptr16(const void* p, const char* name, bool may_be_null = false) {
  if (p == nullptr) {
    if (may_be_null) return ZSA_OK;
    return fail(ZSA_EINVAL, "%s is NULL", name);
  }
  if (!aligned16(p)) return fail(ZSA_EALIGN, "%s is not 16-byte aligned", name);
  return ZSA_OK;
}

int check_width(int32_t dtype, int64_t width, const char* name) {
  if (width <= 0) return fail(ZSA_ESHAPE, "%s = %lld must be positive", name, (long long)width);
  if ((width * static_cast<int64_t>(esize(dtype))) % 16 != 0)
    return fail(ZSA_EALIGN, "%s = %lld rows are not a multiple of 16 bytes", name, (long long)width);
  return ZSA_OK;
}

// The bf16 attention kernels address one sequence's K/V rows (and the decode
// kernel one cache slot's rows) through a buffer resource whose byte range
// and per-tile offsets are 32-bit: the rows a kernel can reach must span
// less than 4 GiB (with a margin of 256 rows for the tile look-ahead).
int check_row_range(int64_t rows, int64_t row_elems, int dtype, const char* what) {
  if ((rows + 256) * row_elems * static_cast<int64_t>(esize(dtype)) >= (int64_t{1} << 32))
    return fail(ZSA_EUNSUPPORTED,
                "%s: %lld rows of %lld elements span 4 GiB or more (32-bit buffer offsets)", what,
                (long long)rows, (long long)row_elems);
  return ZSA_OK;
}

int check_head_dim(int32_t hd) {
  if (hd != 16 && hd != 32 && hd != 64 && hd != 128)
    return fail(ZSA_EUNSUPPORTED, "head_dim %d (supported: 16, 32, 64, 128)", hd);
  return ZSA_OK;
}

int check_cfg(const zsa_layer_cfg* c) {
  if (c == nullptr) return fail(ZSA_EINVAL, "cfg is NULL");
  if (c->kind != ZSA_ENCODER && c->kind != ZSA_DECODER) return fail(ZSA_EINVAL, "kind %d", c->kind);
  CHECK(check_dtype(c->dtype));
  if (c->n_heads <= 0 || c->head_dim <= 0 || c->n_heads * c->head_dim != c->d_model)
    return fail(ZSA_ESHAPE, "n_heads %d * head_dim %d != d_model %d", c->n_heads, c->head_dim,
                c->d_model);
  CHECK(check_head_dim(c->head_dim));
  CHECK(check_width(c->dtype, c->d_model, "d_model"));
  CHECK(check_width(c->dtype, c->d_ff, "d_ff"));
  if (c->d_model % 8 != 0 || c->d_ff % 8 != 0)
    return fail(ZSA_EUNSUPPORTED, "d_model and d_ff must be multiples of 8");
  if (c->d_model > (c->dtype == ZSA_BF16 ? 8192 : 4096))
    return fail(ZSA_EUNSUPPORTED, "d_model %d above the row-norm limit", c->d_model);
  if (c->tau < 1) return fail(ZSA_EINVAL, "tau %d < 1", c->tau);
  if (!(c->norm_eps >= 0.f)) return fail(ZSA_EINVAL, "norm_eps must be >= 0");
  if (c->kind == ZSA_DECODER && !(c->rope_theta > 0.f)) return fail(ZSA_EINVAL, "rope_theta <= 0");
  if (c->n_kv_heads < 0 || (c->n_kv_heads > 0 && c->n_heads % c->n_kv_heads != 0))
    return fail(ZSA_ESHAPE, "n_kv_heads %d must divide n_heads %d", c->n_kv_heads, c->n_heads);
  return ZSA_OK;
}

// key/value heads (grouped-query attention; 0 in the config means n_heads)
int kv_heads(const zsa_layer_cfg& c) { return c.n_kv_heads == 0 ? c.n_heads : c.n_kv_heads; }
// width of the fused [q | k | v] projection output
int64_t qkv_width(const zsa_layer_cfg& c) {
  return c.d_model + 2 * static_cast<int64_t>(kv_heads(c)) * c.head_dim;
}

int check_weights(const zsa_layer_cfg* c, const zsa_layer_weights* w) {
  if (w == nullptr) return fail(ZSA_EINVAL, "weights are NULL");
  CHECK(check_ptr16(w->norm1_w, "norm1_w"));
  CHECK(check_ptr16(w->w_qkv, "w_qkv"));
  CHECK(check_ptr16(w->w_o, "w_o"));
  CHECK(check_ptr16(w->norm2_w, "norm2_w"));
  CHECK(check_ptr16(w->w_up, "w_up"));
  CHECK(check_ptr16(w->w_down, "w_down"));
  CHECK(check_ptr16(w->b_qkv, "b_qkv", true));
  CHECK(check_ptr16(w->b_o, "b_o", true));
  CHECK(check_ptr16(w->b_up, "b_up", true));
  CHECK(check_ptr16(w->b_down, "b_down", true));
  if (c->kind == ZSA_ENCODER) {
    CHECK(check_ptr16(w->norm1_b, "norm1_b", true));
    CHECK(check_ptr16(w->norm2_b, "norm2_b", true));
  }
  return ZSA_OK;
}

// ---------------------------------------------------------------------------
// workspace layout
// ---------------------------------------------------------------------------
struct LayerBufs {
  void* h;
  void* qkv;
  void* o;
  void* f;
  void* xg;
  void* og;
  float* lse;
  float* partials;
  int32_t* kept;
  float* rope;  // per-row rotary table of the rows entering a decoder block
  void* splitk;
  size_t splitk_bytes;
};

struct Carver {
  size_t off = 0;
  size_t take(size_t bytes) {
    const size_t o = off;
    off += round256(bytes);
    return o;
  }
};

struct LayerLayout {
  size_t h, qkv, o, f, xg, og, lse, partials, kept, rope, rope_bytes, splitk, splitk_bytes, end;
};

LayerLayout layer_layout(const zsa_layer_cfg* c, int64_t T, Carver& cv) {
  const size_t e = esize(c->dtype);
  const int64_t d = c->d_model, F = c->d_ff;
  // a later (shorter) layer may pick more head groups; H is the upper bound
  const int G = c->n_heads;
  LayerLayout L;
  L.h = cv.take(T * d * e);
  L.qkv = cv.take(T * qkv_width(*c) * e);
  L.o = cv.take(T * d * e);
  L.f = cv.take(T * F * e);
  L.xg = cv.take(T * d * e);
  L.og = cv.take(T * d * e);
  L.lse = cv.take(static_cast<size_t>(c->n_heads) * T * 4);
  L.partials = cv.take(static_cast<size_t>(G) * T * 4);
  L.kept = cv.take(T * 4);
  L.rope_bytes = c->kind == ZSA_DECODER ? zsa::rope_table_bytes(static_cast<int>(T), c->head_dim) : 0;
  L.rope = cv.take(L.rope_bytes);
  // split-K partials of the projections, for any row count up to T
  const int dt = c->dtype;
  const int up_n = c->kind == ZSA_DECODER ? 2 * F : F;
  const int rows = static_cast<int>(T);
  L.splitk_bytes = std::max({zsa::gemm_workspace_bound(dt, rows, static_cast<int>(qkv_width(*c)), d),
                             zsa::gemm_workspace_bound(dt, rows, d, d),
                             zsa::gemm_workspace_bound(dt, rows, up_n, d),
                             zsa::gemm_workspace_bound(dt, rows, d, F)});
  L.splitk = cv.take(L.splitk_bytes);
  L.end = cv.off;
  return L;
}

LayerBufs carve_layer(const LayerLayout& L, void* ws) {
  char* base = static_cast<char*>(ws);
  LayerBufs b;
  b.h = base + L.h;
  b.qkv = base + L.qkv;
  b.o = base + L.o;
  b.f = base + L.f;
  b.xg = base + L.xg;
  b.og = base + L.og;
  b.lse = reinterpret_cast<float*>(base + L.lse);
  b.partials = reinterpret_cast<float*>(base + L.partials);
  b.kept = reinterpret_cast<int32_t*>(base + L.kept);
  b.rope = L.rope_bytes ? reinterpret_cast<float*>(base + L.rope) : nullptr;
  b.splitk = L.splitk_bytes ? base + L.splitk : nullptr;
  b.splitk_bytes = L.splitk_bytes;
  return b;
}

// ---------------------------------------------------------------------------
// one block
// ---------------------------------------------------------------------------
struct RowSet {
  int32_t B;
  const int32_t* cu_host;
  const int32_t* cu_dev;
  int32_t T;
  int32_t max_len;
};

void fill_rope(zsa::EpiParams& ep, int hd, float theta) {
  for (int i = 0; i < zsa::kMaxHalfHead; ++i)
    ep.inv_freq[i] = i < hd / 2 ? pow(static_cast<double>(theta), -2.0 * i / hd) : 0.0;
}

// rope_fresh: the rotary table in the workspace does not yet hold the rows
// entering this block (their positions changed, or it was never built); a
// decoder block then rebuilds it before its QKV projection
int run_layer(hipStream_t s, const zsa_layer_cfg& c, const zsa_layer_weights& w,
              const void* x_in, const int32_t* pos_in, const RowSet& in, bool prune,
              const RowSet& out, void* x_out, int32_t* pos_out, float* scores_out,
              int32_t* kept_out, const LayerBufs& wb, void* kv_layer = nullptr, int kv_cap = 0,
              int32_t* marks_pos = nullptr, bool rope_fresh = true) {
  using namespace zsa;
  const int dt = c.dtype;
  const size_t e = esize(dt);
  const int d = c.d_model, H = c.n_heads, hd = c.head_dim, F = c.d_ff;
  const int kvd = kv_heads(c) * hd;     // key (and value) columns
  const int qw = d + 2 * kvd;           // row width of the fused [q | k | v] output
  const int kvg = H / kv_heads(c);      // query heads per key/value head
  const bool dec = c.kind == ZSA_DECODER;
  const int norm_kind = dec ? ZSA_NORM_RMS : ZSA_NORM_LAYER;
  const float scale = 1.0f / sqrtf(static_cast<float>(hd));

  HIP_TRY(launch_norm(s, dt, norm_kind, x_in, w.norm1_w, dec ? nullptr : w.norm1_b, in.T, d,
                      c.norm_eps, wb.h),
          "norm1");
  {
    EpiParams ep{};
    ep.epi = dec ? EPI_ROPE : EPI_NONE;
    ep.bias = w.b_qkv;
    ep.y = wb.qkv;
    ep.ldy = qw;
    ep.pos = pos_in;
    ep.head_dim = hd;
    ep.rope_cols = dec ? d + kvd : 0;
    if (dec) {
      fill_rope(ep, hd, c.rope_theta);
      if (wb.rope != nullptr && dt == ZSA_BF16) {
        if (rope_fresh) HIP_TRY(launch_rope_table(s, pos_in, in.T, ep, wb.rope), "rotary table");
        ep.rope_cs = wb.rope;
      }
    }
    HIP_TRY(launch_gemm(s, dt, wb.h, in.T, d, w.w_qkv, qw, ep, wb.splitk, wb.splitk_bytes),
            "qkv projection");
  }
  if (kv_layer != nullptr)  // the rows entering this layer, for generation
    HIP_TRY(launch_kv_store(s, dt, wb.qkv, qw, d, kvd, in.B, in.max_len, in.cu_dev, nullptr,
                            kv_layer, kv_cap),
            "kv cache");
  const char* qkv = static_cast<const char*>(wb.qkv);
  const void* q = qkv;
  const void* k = qkv + d * e;
  const void* v = qkv + (d + kvd) * e;
  HIP_TRY(launch_attention(s, dt, q, k, v, qw, H, kvg, hd, c.causal, scale, in.B, in.max_len, in.T,
                           in.cu_dev, wb.o, d, wb.lse),
          "attention");
  const void* xr = x_in;
  const void* orows = wb.o;
  int rows = in.T;
  if (prune) {
    const int G = score_groups(dt, H, hd, in.T);
    HIP_TRY(launch_score(s, dt, q, k, qw, wb.lse, H, kvg, hd, c.causal, scale, in.B, in.max_len,
                         in.T, in.cu_dev, wb.partials, G),
            "score");
    int32_t* kept = kept_out != nullptr ? kept_out : wb.kept;
    HIP_TRY(launch_select(s, wb.partials, G, in.T, in.B, in.max_len, in.cu_dev, out.cu_dev, kept,
                          scores_out, c.force_keep_last != 0),
            "select");
    if (c.mark_only != 0) {
      // rows are marked, not removed: only the marked positions are gathered
      if (marks_pos != nullptr)
        HIP_TRY(launch_gather(s, dt, d, in.T, kept, out.T, nullptr, nullptr, nullptr, nullptr,
                              pos_in, marks_pos),
                "mark positions");
    } else {
      HIP_TRY(launch_gather(s, dt, d, in.T, kept, out.T, x_in, wb.xg, wb.o, wb.og, pos_in,
                            pos_out),
              "gather");
      xr = wb.xg;
      orows = wb.og;
      rows = out.T;
    }
  }
  {
    EpiParams ep{};
    ep.epi = EPI_RESIDUAL;
    ep.bias = w.b_o;
    ep.residual = xr;
    ep.y = x_out;
    ep.ldy = d;
    HIP_TRY(launch_gemm(s, dt, orows, rows, d, w.w_o, d, ep, wb.splitk, wb.splitk_bytes),
            "output projection");
  }
  HIP_TRY(launch_norm(s, dt, norm_kind, x_out, w.norm2_w, dec ? nullptr : w.norm2_b, rows, d,
                      c.norm_eps, wb.h),
          "norm2");
  {
    EpiParams ep{};
    ep.epi = dec ? EPI_SWIGLU : EPI_GELU;
    ep.bias = w.b_up;
    ep.y = wb.f;
    ep.ldy = F;
    HIP_TRY(launch_gemm(s, dt, wb.h, rows, d, w.w_up, dec ? 2 * F : F, ep, wb.splitk,
                        wb.splitk_bytes),
            "up projection");
  }
  {
    EpiParams ep{};
    ep.epi = EPI_RESIDUAL;
    ep.bias = w.b_down;
    ep.residual = x_out;
    ep.y = x_out;
    ep.ldy = d;
    HIP_TRY(launch_gemm(s, dt, wb.f, rows, F, w.w_down, d, ep, wb.splitk, wb.splitk_bytes),
            "down projection");
  }
  return ZSA_OK;
}

// ---------------------------------------------------------------------------
// timing hook
// ---------------------------------------------------------------------------
struct TimingState {
  bool armed = false;
  int used = 0;
  std::vector<hipEvent_t> start, stop;
};
TimingState g_timing[zsa::K_NCLASS];

}  // namespace

namespace zsa {
int set_error(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

bool timing_take(int kclass, hipEvent_t* start, hipEvent_t* stop) {
  if (kclass < 0 || kclass >= K_NCLASS) return false;
  TimingState& t = g_timing[kclass];
  if (!t.armed || t.used >= static_cast<int>(t.start.size())) return false;
  *start = t.start[t.used];
  *stop = t.stop[t.used];
  ++t.used;
  return true;
}
}  // namespace zsa

// ===========================================================================
// exported entry points
// ===========================================================================
extern "C" {

const char* zsa_last_error(void) { return g_err.c_str(); }
const char* zsa_version(void) { return "zsa 0.1 gfx950"; }

int zsa_keep_count(int32_t n, double keep_rate, int32_t tau, int32_t* k_out) {
  if (k_out == nullptr) return fail(ZSA_EINVAL, "k_out is NULL");
  CHECK(check_rate(keep_rate));
  if (tau < 1) return fail(ZSA_EINVAL, "tau %d < 1", tau);
  if (n < 0) return fail(ZSA_EINVAL, "n %d < 0", n);
  *k_out = keep_count_impl(n, keep_rate, tau);
  return ZSA_OK;
}

int zsa_keep_schedule(int32_t batch, const int32_t* lengths, const double* keep_rate, int32_t tau,
                      int32_t n_points, int32_t* counts_out) {
  if (batch < 0 || n_points < 0) return fail(ZSA_EINVAL, "negative batch or n_points");
  if (batch > 0 && (lengths == nullptr || keep_rate == nullptr || counts_out == nullptr))
    return fail(ZSA_EINVAL, "NULL array");
  if (tau < 1) return fail(ZSA_EINVAL, "tau %d < 1", tau);
  for (int b = 0; b < batch; ++b) {
    CHECK(check_rate(keep_rate[b]));
    if (lengths[b] < 0) return fail(ZSA_EINVAL, "length %d < 0", lengths[b]);
  }
  for (int b = 0; b < batch; ++b) {
    int32_t cur = lengths[b];
    for (int p = 0; p < n_points; ++p) {
      cur = keep_count_impl(cur, keep_rate[b], tau);
      counts_out[p * batch + b] = cur;
    }
  }
  return ZSA_OK;
}

int zsa_norm(void* stream, int32_t dtype, int32_t kind, const void* x, const void* gain,
             const void* shift, int32_t rows, int32_t d, float eps, void* y) {
  CHECK(check_dtype(dtype));
  if (kind != ZSA_NORM_LAYER && kind != ZSA_NORM_RMS) return fail(ZSA_EINVAL, "norm kind %d", kind);
  if (rows < 0) return fail(ZSA_EINVAL, "rows < 0");
  CHECK(check_width(dtype, d, "d"));
  if (d > (dtype == ZSA_BF16 ? 8192 : 4096)) return fail(ZSA_EUNSUPPORTED, "d %d too wide", d);
  // no rows: nothing is read or written, so x and y may be NULL
  CHECK(check_ptr16(x, "x", rows == 0));
  CHECK(check_ptr16(gain, "gain"));
  CHECK(check_ptr16(y, "y", rows == 0));
  CHECK(check_ptr16(shift, "shift", true));
  if (rows == 0) return ZSA_OK;
  HIP_TRY(zsa::launch_norm(static_cast<hipStream_t>(stream), dtype, kind, x, gain,
                           kind == ZSA_NORM_LAYER ? shift : nullptr, rows, d, eps, y),
          "norm");
  return ZSA_OK;
}

size_t zsa_linear_workspace_size(int32_t dtype, int32_t m, int32_t n, int32_t k) {
  if (m <= 0 || n <= 0 || k <= 0) return 0;
  return zsa::gemm_workspace_bytes(dtype, m, n, k);
}

int zsa_linear(void* stream, int32_t dtype, const void* x, int32_t m, int32_t k, const void* w,
               int32_t n, const void* bias, int32_t epilogue, const void* residual,
               const int32_t* pos, int32_t head_dim, int32_t rope_cols, float rope_theta,
               void* y, void* ws, size_t ws_bytes) {
  CHECK(check_dtype(dtype));
  if (m < 0) return fail(ZSA_EINVAL, "m < 0");
  CHECK(check_width(dtype, k, "k"));
  if (n <= 0 || n % 8 != 0) return fail(ZSA_ESHAPE, "n %d must be a positive multiple of 8", n);
  if (epilogue < ZSA_EPI_NONE || epilogue > ZSA_EPI_ROPE) return fail(ZSA_EINVAL, "epilogue %d", epilogue);
  if (epilogue == ZSA_EPI_SWIGLU && n % 16 != 0)
    return fail(ZSA_ESHAPE, "SwiGLU needs n %% 16 == 0 (n = %d)", n);
  // no rows: nothing is read or written, so the row operands may be NULL
  CHECK(check_ptr16(x, "x", m == 0));
  CHECK(check_ptr16(w, "w"));
  CHECK(check_ptr16(y, "y", m == 0));
  CHECK(check_ptr16(bias, "bias", true));
  if (epilogue == ZSA_EPI_RESIDUAL) CHECK(check_ptr16(residual, "residual", m == 0));
  zsa::EpiParams ep{};
  ep.epi = epilogue;
  ep.bias = bias;
  ep.residual = residual;
  ep.y = y;
  ep.ldy = epilogue == ZSA_EPI_SWIGLU ? n / 2 : n;
  if (epilogue == ZSA_EPI_ROPE) {
    if (head_dim != 16 && head_dim != 32 && head_dim != 64 && head_dim != 128)
      return fail(ZSA_EUNSUPPORTED, "rotary head_dim %d", head_dim);
    if (rope_cols < 0 || rope_cols % head_dim != 0 || rope_cols > n)
      return fail(ZSA_ESHAPE, "rope_cols %d", rope_cols);
    if (pos == nullptr && m > 0) return fail(ZSA_EINVAL, "pos is NULL");
    if (!(rope_theta > 0.f)) return fail(ZSA_EINVAL, "rope_theta <= 0");
    ep.pos = pos;
    ep.head_dim = head_dim;
    ep.rope_cols = rope_cols;
    fill_rope(ep, head_dim, rope_theta);
  }
  size_t need = 0;
  if (ws != nullptr) {
    CHECK(check_ptr16(ws, "ws"));
    need = zsa_linear_workspace_size(dtype, m, n, k);
    if (ws_bytes < need)
      return fail(ZSA_EWORKSPACE, "linear workspace %zu < %zu bytes", ws_bytes, need);
  }
  if (m == 0) return ZSA_OK;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (epilogue == ZSA_EPI_ROPE && dtype == ZSA_BF16 && ws != nullptr && m > 0 &&
      ws_bytes >= round256(need) + zsa::rope_table_bytes(m, head_dim)) {
    // room past the split-K partials: the rotary angles as a per-row table
    float* table = reinterpret_cast<float*>(static_cast<char*>(ws) + round256(need));
    HIP_TRY(zsa::launch_rope_table(s, pos, m, ep, table), "rotary table");
    ep.rope_cs = table;
    ws_bytes = need;
  }
  HIP_TRY(zsa::launch_gemm(s, dtype, x, m, k, w, n, ep, ws, ws_bytes), "linear");
  return ZSA_OK;
}

size_t zsa_attention_workspace_size(int32_t n_heads, int32_t total_rows, int32_t want_scores) {
  if (n_heads <= 0 || total_rows < 0) return 0;
  size_t b = round256(static_cast<size_t>(n_heads) * total_rows * 4);  // lse scratch
  if (want_scores) b += round256(static_cast<size_t>(n_heads) * total_rows * 4);  // partials
  return b;
}

int check_kv_heads(int32_t n_heads, int32_t n_kv_heads, int* group) {
  if (n_heads <= 0) return fail(ZSA_EINVAL, "n_heads %d", n_heads);
  const int32_t hkv = n_kv_heads == 0 ? n_heads : n_kv_heads;
  if (hkv < 0 || n_heads % hkv != 0)
    return fail(ZSA_ESHAPE, "n_kv_heads %d must divide n_heads %d", n_kv_heads, n_heads);
  *group = n_heads / hkv;
  return ZSA_OK;
}

int zsa_attention_with_scores(void* stream, int32_t dtype, const void* q, const void* k,
                              const void* v, int64_t row_stride, int32_t n_heads,
                              int32_t n_kv_heads, int32_t head_dim, int32_t causal, float scale,
                              int32_t batch, const int32_t* cu_host, const int32_t* cu_dev,
                              void* out, int64_t out_stride, float* lse, float* scores, void* ws,
                              size_t ws_bytes) {
  CHECK(check_dtype(dtype));
  CHECK(check_head_dim(head_dim));
  int kvg = 1;
  CHECK(check_kv_heads(n_heads, n_kv_heads, &kvg));
  int32_t T, max_len;
  CHECK(check_seqs(batch, cu_host, cu_dev, &T, &max_len));
  // no rows (every sequence empty): nothing is read or written, so the row
  // operands may be NULL
  CHECK(check_ptr16(q, "q", T == 0));
  CHECK(check_ptr16(k, "k", T == 0));
  CHECK(check_ptr16(v, "v", T == 0));
  CHECK(check_ptr16(out, "out", T == 0));
  CHECK(check_width(dtype, row_stride, "row_stride"));
  CHECK(check_width(dtype, out_stride, "out_stride"));
  if (row_stride < static_cast<int64_t>(n_heads) * head_dim || out_stride < static_cast<int64_t>(n_heads) * head_dim)
    return fail(ZSA_ESHAPE, "row stride shorter than n_heads * head_dim");
  if (!(scale > 0.f)) return fail(ZSA_EINVAL, "scale must be positive");
  CHECK(check_row_range(max_len, row_stride, dtype, "attention"));
  const size_t need = zsa_attention_workspace_size(n_heads, T, scores != nullptr);
  if (scores != nullptr || lse == nullptr) {
    if (ws_bytes < need || (need > 0 && ws == nullptr))
      return fail(ZSA_EWORKSPACE, "workspace %zu bytes < %zu", ws_bytes, need);
  }
  if (T == 0) return ZSA_OK;
  hipStream_t s = static_cast<hipStream_t>(stream);
  char* base = static_cast<char*>(ws);
  float* lse_buf = lse != nullptr ? lse : reinterpret_cast<float*>(base);
  HIP_TRY(zsa::launch_attention(s, dtype, q, k, v, row_stride, n_heads, kvg, head_dim, causal,
                                scale, batch, max_len, T, cu_dev, out, out_stride, lse_buf),
          "attention");
  if (scores != nullptr) {
    float* partials = reinterpret_cast<float*>(base + round256(static_cast<size_t>(n_heads) * T * 4));
    const int G = zsa::score_groups(dtype, n_heads, head_dim, T);
    HIP_TRY(zsa::launch_score(s, dtype, q, k, row_stride, lse_buf, n_heads, kvg, head_dim, causal,
                              scale, batch, max_len, T, cu_dev, partials, G),
            "score");
    HIP_TRY(zsa::launch_score_finalize(s, partials, G, T, scores), "score finalize");
  }
  return ZSA_OK;
}

size_t zsa_score_workspace_size(int32_t n_heads, int32_t total_rows) {
  if (n_heads <= 0 || total_rows < 0) return 0;
  return round256(static_cast<size_t>(n_heads) * total_rows * 4);
}

int zsa_score_positions(void* stream, int32_t dtype, const void* q, const void* k,
                        int64_t row_stride, const float* lse, int32_t n_heads,
                        int32_t n_kv_heads, int32_t head_dim, int32_t causal, float scale,
                        int32_t batch, const int32_t* cu_host, const int32_t* cu_dev,
                        float* scores, void* ws, size_t ws_bytes) {
  CHECK(check_dtype(dtype));
  CHECK(check_head_dim(head_dim));
  int kvg = 1;
  CHECK(check_kv_heads(n_heads, n_kv_heads, &kvg));
  int32_t T, max_len;
  CHECK(check_seqs(batch, cu_host, cu_dev, &T, &max_len));
  // no rows: nothing is read or written, so the row operands may be NULL
  CHECK(check_ptr16(q, "q", T == 0));
  CHECK(check_ptr16(k, "k", T == 0));
  if (T > 0 && (lse == nullptr || scores == nullptr)) return fail(ZSA_EINVAL, "lse / scores is NULL");
  CHECK(check_width(dtype, row_stride, "row_stride"));
  if (row_stride < static_cast<int64_t>(n_heads) * head_dim)
    return fail(ZSA_ESHAPE, "row stride shorter than n_heads * head_dim");
  if (!(scale > 0.f)) return fail(ZSA_EINVAL, "scale must be positive");
  CHECK(check_row_range(max_len, row_stride, dtype, "score"));
  const size_t need = zsa_score_workspace_size(n_heads, T);
  if (ws_bytes < need || (need > 0 && ws == nullptr))
    return fail(ZSA_EWORKSPACE, "workspace %zu bytes < %zu", ws_bytes, need);
  if (T == 0) return ZSA_OK;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int G = zsa::score_groups(dtype, n_heads, head_dim, T);
  float* partials = static_cast<float*>(ws);
  HIP_TRY(zsa::launch_score(s, dtype, q, k, row_stride, lse, n_heads, kvg, head_dim, causal,
                            scale, batch, max_len, T, cu_dev, partials, G),
          "score");
  HIP_TRY(zsa::launch_score_finalize(s, partials, G, T, scores), "score finalize");
  return ZSA_OK;
}

size_t zsa_select_workspace_size(int32_t batch) {
  return batch < 0 ? 0 : round256(static_cast<size_t>(batch + 1) * 4);
}

int zsa_select_topk(void* stream, const float* scores, int32_t batch, const int32_t* cu_host,
                    const int32_t* cu_dev, const int32_t* k_host, int32_t force_keep_last,
                    int32_t* kept_rows, void* ws, size_t ws_bytes) {
  int32_t T, max_len;
  CHECK(check_seqs(batch, cu_host, cu_dev, &T, &max_len));
  if (batch > 0 && k_host == nullptr) return fail(ZSA_EINVAL, "k_host is NULL");
  std::vector<int32_t> cu_out(batch + 1, 0);
  for (int b = 0; b < batch; ++b) {
    const int32_t n = cu_host[b + 1] - cu_host[b];
    if (k_host[b] < 0 || k_host[b] > n)
      return fail(ZSA_ESHAPE, "k[%d] = %d outside [0, %d]", b, k_host[b], n);
    cu_out[b + 1] = cu_out[b] + k_host[b];
  }
  if (T > 0 && scores == nullptr) return fail(ZSA_EINVAL, "scores is NULL");
  if (cu_out[batch] > 0 && kept_rows == nullptr) return fail(ZSA_EINVAL, "kept_rows is NULL");
  const size_t need = zsa_select_workspace_size(batch);
  if (ws_bytes < need || ws == nullptr) return fail(ZSA_EWORKSPACE, "workspace %zu < %zu", ws_bytes, need);
  hipStream_t s = static_cast<hipStream_t>(stream);
  int32_t* cu_out_dev = static_cast<int32_t*>(ws);
  HIP_TRY(zsa::launch_upload_i32(s, cu_out_dev, cu_out.data(), batch + 1), "upload");
  HIP_TRY(zsa::launch_select(s, scores, 1, T, batch, max_len, cu_dev, cu_out_dev, kept_rows, nullptr,
                             force_keep_last != 0),
          "select");
  return ZSA_OK;
}

int zsa_compact_gather(void* stream, int32_t dtype, const void* hidden, int32_t d,
                       const int32_t* pos, int32_t t_in, const int32_t* kept_rows, int32_t t_out,
                       void* hidden_out, int32_t* pos_out) {
  CHECK(check_dtype(dtype));
  CHECK(check_width(dtype, d, "d"));
  if (t_in < 0 || t_out < 0) return fail(ZSA_EINVAL, "negative row count");
  if ((pos == nullptr) != (pos_out == nullptr)) return fail(ZSA_EINVAL, "pos and pos_out must both be set or both NULL");
  if (t_out > 0) {
    CHECK(check_ptr16(hidden, "hidden"));
    CHECK(check_ptr16(hidden_out, "hidden_out"));
    if (kept_rows == nullptr) return fail(ZSA_EINVAL, "kept_rows is NULL");
  }
  HIP_TRY(zsa::launch_gather(static_cast<hipStream_t>(stream), dtype, d, t_in, kept_rows, t_out,
                             hidden, hidden_out, nullptr, nullptr, pos, pos_out),
          "gather");
  return ZSA_OK;
}

size_t zsa_layer_workspace_size(const zsa_layer_cfg* cfg, int32_t total_rows, int32_t batch) {
  if (cfg == nullptr || total_rows < 0 || batch < 0) return 0;
  Carver cv;
  layer_layout(cfg, total_rows, cv);
  cv.take(static_cast<size_t>(batch + 1) * 4);   // kept-list offsets (mark-only)
  return cv.off;
}

int zsa_layer_forward(void* stream, const zsa_layer_cfg* cfg, const zsa_layer_weights* w,
                      const void* hidden_in, const int32_t* pos_in, int32_t batch,
                      const int32_t* cu_host, const int32_t* cu_dev, const double* keep_rate,
                      void* hidden_out, int32_t* pos_out, int32_t* cu_out_host,
                      int32_t* cu_out_dev, float* scores_out, int32_t* kept_rows_out, void* ws,
                      size_t ws_bytes) {
  CHECK(check_cfg(cfg));
  CHECK(check_weights(cfg, w));
  int32_t T, max_len;
  CHECK(check_seqs(batch, cu_host, cu_dev, &T, &max_len));
  if (T > 0) {
    CHECK(check_ptr16(hidden_in, "hidden_in"));
    CHECK(check_ptr16(hidden_out, "hidden_out"));
    if (pos_in == nullptr || pos_out == nullptr) return fail(ZSA_EINVAL, "pos_in / pos_out is NULL");
  }
  if (cu_out_host == nullptr || cu_out_dev == nullptr) return fail(ZSA_EINVAL, "cu_out is NULL");
  CHECK(check_row_range(max_len, qkv_width(*cfg), cfg->dtype, "attention"));
  const bool prune = keep_rate != nullptr;
  std::vector<int32_t> cu_out(batch + 1, 0);
  int32_t max_out = 0;
  for (int b = 0; b < batch; ++b) {
    const int32_t n = cu_host[b + 1] - cu_host[b];
    int32_t kb = n;
    if (prune) {
      CHECK(check_rate(keep_rate[b]));
      kb = keep_count_impl(n, keep_rate[b], cfg->tau);
    }
    cu_out[b + 1] = cu_out[b] + kb;
    if (kb > max_out) max_out = kb;
  }
  const size_t need = zsa_layer_workspace_size(cfg, T, batch);
  if (ws_bytes < need || ws == nullptr) return fail(ZSA_EWORKSPACE, "workspace %zu < %zu", ws_bytes, need);

  hipStream_t s = static_cast<hipStream_t>(stream);
  Carver cv;
  const LayerBufs wb = carve_layer(layer_layout(cfg, T, cv), ws);
  // mark-only: the output keeps every row; the kept lists get offsets of their own
  const bool mark = prune && cfg->mark_only != 0;
  int32_t* marks_cu = reinterpret_cast<int32_t*>(static_cast<char*>(ws) +
                                                 cv.take(static_cast<size_t>(batch + 1) * 4));
  const RowSet in{batch, cu_host, cu_dev, T, max_len};
  int32_t* sel_cu = mark ? marks_cu : cu_out_dev;
  const RowSet sel{batch, cu_out.data(), sel_cu, cu_out[batch], max_out};
  HIP_TRY(zsa::launch_upload_i32(s, sel_cu, cu_out.data(), batch + 1), "upload");
  if (mark) HIP_TRY(zsa::launch_upload_i32(s, cu_out_dev, cu_host, batch + 1), "upload");
  if (T > 0) {
    CHECK(run_layer(s, *cfg, *w, hidden_in, pos_in, in, prune, sel, hidden_out, pos_out,
                    scores_out, kept_rows_out, wb));
    if (!prune || mark) HIP_TRY(zsa::launch_copy_i32(s, pos_out, pos_in, T), "pos copy");
  }
  memcpy(cu_out_host, mark ? cu_host : cu_out.data(), sizeof(int32_t) * (batch + 1));
  return ZSA_OK;
}

size_t zsa_stack_workspace_size(const zsa_layer_cfg* cfg, int32_t total_rows, int32_t batch,
                                int32_t n_prune) {
  if (cfg == nullptr || total_rows < 0 || batch < 0 || n_prune < 0) return 0;
  Carver cv;
  layer_layout(cfg, total_rows, cv);
  const size_t xb = static_cast<size_t>(total_rows) * cfg->d_model * esize(cfg->dtype);
  cv.take(xb);
  cv.take(xb);
  cv.take(static_cast<size_t>(total_rows) * 4);
  cv.take(static_cast<size_t>(total_rows) * 4);
  cv.take(static_cast<size_t>(n_prune) * (batch + 1) * 4);
  return cv.off;
}

int zsa_stack_forward(void* stream, const zsa_layer_cfg* cfg, const zsa_layer_weights* w,
                      int32_t n_layers, const int32_t* prune_after, int32_t n_prune,
                      const double* keep_rate, const void* hidden_in, const int32_t* pos_in,
                      int32_t batch, const int32_t* cu_host, const int32_t* cu_dev,
                      void* hidden_out, int32_t* pos_out, int32_t* cu_out_host,
                      int32_t* cu_out_dev, int32_t* counts_out_host, float* scores_dbg,
                      int32_t* pos_dbg, void* hidden_dbg, void* kv_cache, int32_t kv_capacity,
                      void* ws, size_t ws_bytes) {
  CHECK(check_cfg(cfg));
  if (n_layers < 1) return fail(ZSA_EINVAL, "n_layers %d < 1", n_layers);
  if (w == nullptr) return fail(ZSA_EINVAL, "weights are NULL");
  for (int l = 0; l < n_layers; ++l) {
    const int rc = check_weights(cfg, &w[l]);
    if (rc != ZSA_OK) return fail(rc, "layer %d: %s", l + 1, g_err.c_str());
  }
  if (n_prune < 0 || (n_prune > 0 && prune_after == nullptr)) return fail(ZSA_EINVAL, "prune_after");
  for (int p = 0; p < n_prune; ++p) {
    if (prune_after[p] < 1 || prune_after[p] > n_layers)
      return fail(ZSA_EINVAL, "prune_after[%d] = %d outside 1..%d", p, prune_after[p], n_layers);
    if (p > 0 && prune_after[p] <= prune_after[p - 1])
      return fail(ZSA_EINVAL, "prune_after must be strictly ascending");
  }
  int32_t T0, max_len0;
  CHECK(check_seqs(batch, cu_host, cu_dev, &T0, &max_len0));
  CHECK(check_row_range(max_len0, qkv_width(*cfg), cfg->dtype, "attention"));
  if (n_prune > 0 && batch > 0 && keep_rate == nullptr) return fail(ZSA_EINVAL, "keep_rate is NULL");
  for (int b = 0; n_prune > 0 && b < batch; ++b) CHECK(check_rate(keep_rate[b]));
  if (T0 > 0) {
    CHECK(check_ptr16(hidden_in, "hidden_in"));
    CHECK(check_ptr16(hidden_out, "hidden_out"));
    if (pos_in == nullptr || pos_out == nullptr) return fail(ZSA_EINVAL, "pos_in / pos_out is NULL");
  }
  if (cu_out_host == nullptr || cu_out_dev == nullptr) return fail(ZSA_EINVAL, "cu_out is NULL");
  if (kv_cache != nullptr) {
    if (!cfg->causal) return fail(ZSA_EINVAL, "a key/value cache needs the causal mask");
    CHECK(check_ptr16(kv_cache, "kv_cache"));
    if (kv_capacity < max_len0)
      return fail(ZSA_ESHAPE, "kv_capacity %d below the longest sequence %d", kv_capacity, max_len0);
  }
  const size_t need = zsa_stack_workspace_size(cfg, T0, batch, n_prune);
  if (ws_bytes < need || ws == nullptr) return fail(ZSA_EWORKSPACE, "workspace %zu < %zu", ws_bytes, need);

  // the whole schedule is known on the host before any launch
  std::vector<std::vector<int32_t>> cus(n_prune + 1, std::vector<int32_t>(batch + 1, 0));
  std::vector<int32_t> maxl(n_prune + 1, 0);
  for (int b = 0; b <= batch; ++b) cus[0][b] = cu_host[b];
  maxl[0] = max_len0;
  for (int p = 1; p <= n_prune; ++p) {
    for (int b = 0; b < batch; ++b) {
      const int32_t n = cus[p - 1][b + 1] - cus[p - 1][b];
      const int32_t kb = keep_count_impl(n, keep_rate[b], cfg->tau);
      cus[p][b + 1] = cus[p][b] + kb;
      if (kb > maxl[p]) maxl[p] = kb;
      if (counts_out_host != nullptr) counts_out_host[(p - 1) * batch + b] = kb;
    }
  }

  hipStream_t s = static_cast<hipStream_t>(stream);
  Carver cv;
  const LayerBufs wb = carve_layer(layer_layout(cfg, T0, cv), ws);
  char* base = static_cast<char*>(ws);
  const size_t xb = static_cast<size_t>(T0) * cfg->d_model * esize(cfg->dtype);
  void* xbuf[2] = {base + cv.take(xb), base + cv.take(xb)};
  int32_t* posbuf[2] = {reinterpret_cast<int32_t*>(base + cv.take(static_cast<size_t>(T0) * 4)),
                        reinterpret_cast<int32_t*>(base + cv.take(static_cast<size_t>(T0) * 4))};
  int32_t* meta = reinterpret_cast<int32_t*>(base + cv.take(static_cast<size_t>(n_prune) * (batch + 1) * 4));

  std::vector<int32_t> flat;
  for (int p = 1; p <= n_prune; ++p) flat.insert(flat.end(), cus[p].begin(), cus[p].end());
  if (!flat.empty()) HIP_TRY(zsa::launch_upload_i32(s, meta, flat.data(), static_cast<int>(flat.size())), "upload");
  const bool mark = cfg->mark_only != 0;
  HIP_TRY(zsa::launch_upload_i32(s, cu_out_dev, mark ? cus[0].data() : cus[n_prune].data(),
                                 batch + 1),
          "upload");

  const void* cur_x = hidden_in;
  const int32_t* cur_pos = pos_in;
  RowSet cur{batch, cus[0].data(), cu_dev, T0, max_len0};
  int point = 0;
  bool rope_fresh = true;  // the rows entering the block changed since the last table
  size_t score_off = 0, pos_off = 0, hid_off = 0;
  const size_t row_bytes = static_cast<size_t>(cfg->d_model) * esize(cfg->dtype);
  for (int l = 1; l <= n_layers && T0 > 0; ++l) {
    const bool last = l == n_layers;
    const bool prune = point < n_prune && prune_after[point] == l;
    void* x_out = last ? hidden_out : xbuf[(l - 1) & 1];
    void* kv_layer = kv_cache == nullptr
                         ? nullptr
                         : static_cast<char*>(kv_cache) + static_cast<size_t>(l - 1) * batch *
                                                              kv_capacity * 2 * kv_heads(*cfg) *
                                                              cfg->head_dim * esize(cfg->dtype);
    if (prune && mark) {
      // every row continues; the point's marked rows (Eq. 2 count) are listed
      const RowSet sel{batch, cus[point + 1].data(), meta + static_cast<size_t>(point) * (batch + 1),
                       cus[point + 1][batch], maxl[point + 1]};
      float* sdbg = scores_dbg != nullptr ? scores_dbg + score_off : nullptr;
      int32_t* mpos = pos_dbg != nullptr ? pos_dbg + pos_off : nullptr;
      CHECK(run_layer(s, *cfg, w[l - 1], cur_x, cur_pos, cur, true, sel, x_out, nullptr, sdbg,
                      nullptr, wb, kv_layer, kv_capacity, mpos, rope_fresh));
      rope_fresh = false;  // marking keeps every row
      score_off += cur.T;
      pos_off += sel.T;
      ++point;
    } else if (prune && scores_dbg == nullptr && cus[point + 1] == cus[point]) {
      // Eq. 2 keeps every row of every sequence here (each at its floor
      // tau): the kept set is all rows in order, so the layer runs unpruned
      // and the scores, the selection and the gather are skipped
      CHECK(run_layer(s, *cfg, w[l - 1], cur_x, cur_pos, cur, false, cur, x_out, nullptr, nullptr,
                      nullptr, wb, kv_layer, kv_capacity, nullptr, rope_fresh));
      rope_fresh = false;
      if (pos_dbg != nullptr)
        HIP_TRY(zsa::launch_copy_i32(s, pos_dbg + pos_off, cur_pos, cur.T), "pos debug copy");
      score_off += cur.T;
      pos_off += cur.T;
      ++point;
    } else if (prune) {
      const RowSet nxt{batch, cus[point + 1].data(), meta + static_cast<size_t>(point) * (batch + 1),
                       cus[point + 1][batch], maxl[point + 1]};
      int32_t* pos_next = last ? pos_out : posbuf[point & 1];
      float* sdbg = scores_dbg != nullptr ? scores_dbg + score_off : nullptr;
      CHECK(run_layer(s, *cfg, w[l - 1], cur_x, cur_pos, cur, true, nxt, x_out, pos_next, sdbg,
                      nullptr, wb, kv_layer, kv_capacity, nullptr, rope_fresh));
      rope_fresh = true;  // the next block's rows are the kept ones
      if (pos_dbg != nullptr)
        HIP_TRY(zsa::launch_copy_i32(s, pos_dbg + pos_off, pos_next, nxt.T), "pos debug copy");
      score_off += cur.T;
      pos_off += nxt.T;
      cur_pos = pos_next;
      cur = nxt;
      ++point;
    } else {
      CHECK(run_layer(s, *cfg, w[l - 1], cur_x, cur_pos, cur, false, cur, x_out, nullptr, nullptr,
                      nullptr, wb, kv_layer, kv_capacity, nullptr, rope_fresh));
      rope_fresh = false;
    }
    cur_x = x_out;
    if (hidden_dbg != nullptr) {  // this block's output rows (cur: the rows leaving it)
      const size_t bytes = static_cast<size_t>(cur.T) * row_bytes;
      HIP_TRY(hipMemcpyAsync(static_cast<char*>(hidden_dbg) + hid_off, x_out, bytes,
                             hipMemcpyDeviceToDevice, s),
              "hidden debug copy");
      hid_off += bytes;
    }
  }
  if (T0 > 0 && cur_pos != pos_out) HIP_TRY(zsa::launch_copy_i32(s, pos_out, cur_pos, cur.T), "pos copy");
  memcpy(cu_out_host, mark ? cus[0].data() : cus[n_prune].data(), sizeof(int32_t) * (batch + 1));
  return ZSA_OK;
}

// ---------------------------------------------------------------------------
// backward through the pruned stack
// ---------------------------------------------------------------------------
namespace {

int64_t round64(int64_t v) { return (v + 63) / 64 * 64; }

// buffers of one layer's backward, for up to T rows
struct BwdLayout {
  size_t h1, x1, h2, u, dF, du, dh2, dx1, dog, dofull, dxr, dqkv, dh1, D, stats, inv, wT, aT, bT,
      col, splitk, splitk_bytes, end;
};

BwdLayout bwd_layout(const zsa_layer_cfg* c, int64_t T, Carver& cv) {
  const size_t e = esize(c->dtype);
  const int64_t d = c->d_model, F = c->d_ff, qw = qkv_width(*c);
  const int64_t up_n = c->kind == ZSA_DECODER ? 2 * F : F;
  const int64_t maxc = std::max({d, qw, up_n, F});
  BwdLayout B;
  B.h1 = cv.take(T * d * e);
  B.x1 = cv.take(T * d * e);
  B.h2 = cv.take(T * d * e);
  B.u = cv.take(T * up_n * e);
  B.dF = cv.take(T * F * e);
  B.du = cv.take(T * up_n * e);
  B.dh2 = cv.take(T * d * e);
  B.dx1 = cv.take(T * d * e);
  B.dog = cv.take(T * d * e);
  B.dofull = cv.take(T * d * e);
  B.dxr = cv.take(T * d * e);
  B.dqkv = cv.take(T * qw * e);
  B.dh1 = cv.take(T * d * e);
  B.D = cv.take(static_cast<size_t>(c->n_heads) * T * 4);
  B.stats = cv.take(static_cast<size_t>(T) * 2 * 4);
  B.inv = cv.take(static_cast<size_t>(T) * 4);
  B.wT = cv.take(static_cast<size_t>(d) * maxc * e);
  B.aT = cv.take(static_cast<size_t>(round64(T)) * maxc * e);
  B.bT = cv.take(static_cast<size_t>(round64(T)) * maxc * e);
  B.col = cv.take(zsa::colsum_scratch_floats(static_cast<int>(T), static_cast<int>(maxc)) * 4);
  // split-K room for the backward's input-gradient products at any row count
  const int dt = c->dtype, rows = static_cast<int>(T);
  B.splitk_bytes = std::max({zsa::gemm_workspace_bound(dt, rows, static_cast<int>(F), static_cast<int>(d)),
                             zsa::gemm_workspace_bound(dt, rows, static_cast<int>(d), static_cast<int>(up_n)),
                             zsa::gemm_workspace_bound(dt, rows, static_cast<int>(d), static_cast<int>(d)),
                             zsa::gemm_workspace_bound(dt, rows, static_cast<int>(d), static_cast<int>(qw))});
  // ... and for the weight-gradient products (K = the rows, padded to 64)
  const int kp = static_cast<int>(round64(T));
  B.splitk_bytes = std::max({B.splitk_bytes,
                             zsa::gemm_f32_workspace_bound(static_cast<int>(d), static_cast<int>(F), kp),
                             zsa::gemm_f32_workspace_bound(static_cast<int>(up_n), static_cast<int>(d), kp),
                             zsa::gemm_f32_workspace_bound(static_cast<int>(d), static_cast<int>(d), kp),
                             zsa::gemm_f32_workspace_bound(static_cast<int>(qw), static_cast<int>(d), kp)});
  B.splitk = cv.take(B.splitk_bytes);
  B.end = cv.off;
  return B;
}

// one block's backward: recompute its forward, then dL/dx and dL/dW
int layer_backward(hipStream_t s, const zsa_layer_cfg& c, const zsa_layer_weights& w,
                   const zsa_layer_grads& gr, const void* x_in, const int32_t* pos_in,
                   const RowSet& in, bool prune, const RowSet& out, const int32_t* kept,
                   const void* dy, void* dx, const LayerBufs& wb, char* base, const BwdLayout& B) {
  using namespace zsa;
  const int dt = c.dtype;
  const size_t e = esize(dt);
  const int d = c.d_model, H = c.n_heads, hd = c.head_dim, F = c.d_ff;
  const int kvd = kv_heads(c) * hd, qw = static_cast<int>(qkv_width(c)), kvg = H / kv_heads(c);
  const bool dec = c.kind == ZSA_DECODER;
  const int norm_kind = dec ? ZSA_NORM_RMS : ZSA_NORM_LAYER;
  const int up_n = dec ? 2 * F : F;
  const float scale = 1.0f / sqrtf(static_cast<float>(hd));
  const int T = in.T, To = prune ? out.T : in.T;
  const int Tp = static_cast<int>(round64(T)), Top = static_cast<int>(round64(To));
  auto P = [&](size_t off) { return static_cast<void*>(base + off); };
  float* stats = reinterpret_cast<float*>(base + B.stats);
  float* col = reinterpret_cast<float*>(base + B.col);
  void* sk = B.splitk_bytes ? P(B.splitk) : nullptr;
  auto gemm = [&](const void* x, int M, int K, const void* wt, int N, void* y) {
    EpiParams ep{};
    ep.epi = EPI_NONE;
    ep.y = y;
    ep.ldy = N;
    return launch_gemm(s, dt, x, M, K, wt, N, ep, sk, B.splitk_bytes);
  };
  // dW = a^T b over `rows` rows: a [rows, na], b [rows, nb] -> out [na, nb]
  auto wgrad = [&](const void* a, int na, const void* b, int nb, int rows, int rows_p,
                   float* out) -> hipError_t {
    hipError_t er = launch_transpose(s, dt, a, rows, na, na, P(B.aT), rows_p);
    if (er != hipSuccess) return er;
    er = launch_transpose(s, dt, b, rows, nb, nb, P(B.bT), rows_p);
    if (er != hipSuccess) return er;
    return launch_gemm_f32(s, P(B.aT), na, rows_p, P(B.bT), nb, out, sk, B.splitk_bytes);
  };
  // y = x W for W [n_out_w, n_in_w] stored as a Linear weight: x [rows, n_out_w]
  auto xgrad = [&](const void* x, int rows, const void* W, int wn, int wk, void* y) -> hipError_t {
    hipError_t er = launch_transpose(s, dt, W, wn, wk, wk, P(B.wT), wn);  // W^T [wk, wn]
    if (er != hipSuccess) return er;
    return gemm(x, rows, wn, P(B.wT), wk, y);
  };
  auto colsum = [&](const void* a, int rows, int cols, const void* x, float* outp) -> hipError_t {
    if (outp == nullptr) return hipSuccess;
    return launch_colsum(s, dt, a, cols, x, cols, x != nullptr ? stats : nullptr, rows, cols, col,
                         outp);
  };

  // ---- the layer's forward again (deterministic: the same values)
  HIP_TRY(launch_norm(s, dt, norm_kind, x_in, w.norm1_w, dec ? nullptr : w.norm1_b, T, d,
                      c.norm_eps, P(B.h1)),
          "norm1");
  EpiParams rope{};
  if (dec) fill_rope(rope, hd, c.rope_theta);
  {
    EpiParams ep = rope;
    ep.epi = dec ? EPI_ROPE : EPI_NONE;
    ep.bias = w.b_qkv;
    ep.y = wb.qkv;
    ep.ldy = qw;
    ep.pos = pos_in;
    ep.head_dim = hd;
    ep.rope_cols = dec ? d + kvd : 0;
    HIP_TRY(launch_gemm(s, dt, P(B.h1), T, d, w.w_qkv, qw, ep, wb.splitk, wb.splitk_bytes),
            "qkv projection");
  }
  const char* qkv = static_cast<const char*>(wb.qkv);
  const void* q = qkv;
  const void* k = qkv + d * e;
  const void* v = qkv + (d + kvd) * e;
  HIP_TRY(launch_attention(s, dt, q, k, v, qw, H, kvg, hd, c.causal, scale, in.B, in.max_len, T,
                           in.cu_dev, wb.o, d, wb.lse),
          "attention");
  const void* xr = x_in;
  const void* og = wb.o;
  if (prune) {
    HIP_TRY(launch_gather(s, dt, d, T, kept, To, x_in, wb.xg, wb.o, wb.og, nullptr, nullptr),
            "gather");
    xr = wb.xg;
    og = wb.og;
  }
  {
    EpiParams ep{};
    ep.epi = EPI_RESIDUAL;
    ep.bias = w.b_o;
    ep.residual = xr;
    ep.y = P(B.x1);
    ep.ldy = d;
    HIP_TRY(launch_gemm(s, dt, og, To, d, w.w_o, d, ep, wb.splitk, wb.splitk_bytes),
            "output projection");
  }
  HIP_TRY(launch_norm(s, dt, norm_kind, P(B.x1), w.norm2_w, dec ? nullptr : w.norm2_b, To, d,
                      c.norm_eps, P(B.h2)),
          "norm2");
  {
    EpiParams ep{};
    ep.epi = EPI_NONE;
    ep.bias = w.b_up;
    ep.y = P(B.u);
    ep.ldy = up_n;
    HIP_TRY(launch_gemm(s, dt, P(B.h2), To, d, w.w_up, up_n, ep, wb.splitk, wb.splitk_bytes),
            "up projection");
  }
  HIP_TRY(launch_act_fwd(s, dt, P(B.u), wb.f, To, F, dec), "activation");

  // ---- backward: MLP
  HIP_TRY(wgrad(dy, d, wb.f, F, To, Top, gr.w_down), "down weight gradient");
  HIP_TRY(colsum(dy, To, d, nullptr, gr.b_down), "down bias gradient");
  HIP_TRY(xgrad(dy, To, w.w_down, d, F, P(B.dF)), "down input gradient");
  HIP_TRY(launch_act_bwd(s, dt, P(B.dF), P(B.u), P(B.du), To, F, dec), "activation gradient");
  HIP_TRY(wgrad(P(B.du), up_n, P(B.h2), d, To, Top, gr.w_up), "up weight gradient");
  HIP_TRY(colsum(P(B.du), To, up_n, nullptr, gr.b_up), "up bias gradient");
  HIP_TRY(xgrad(P(B.du), To, w.w_up, up_n, d, P(B.dh2)), "up input gradient");
  HIP_TRY(launch_norm_bwd(s, dt, norm_kind, P(B.x1), w.norm2_w, P(B.dh2), dy, P(B.dx1), To, d,
                          c.norm_eps, stats),
          "norm2 gradient");
  HIP_TRY(colsum(P(B.dh2), To, d, P(B.x1), gr.norm2_w), "norm2 gain gradient");
  if (!dec) HIP_TRY(colsum(P(B.dh2), To, d, nullptr, gr.norm2_b), "norm2 shift gradient");
  // ---- output projection
  HIP_TRY(wgrad(P(B.dx1), d, og, d, To, Top, gr.w_o), "output weight gradient");
  HIP_TRY(colsum(P(B.dx1), To, d, nullptr, gr.b_o), "output bias gradient");
  HIP_TRY(xgrad(P(B.dx1), To, w.w_o, d, d, P(B.dog)), "output input gradient");
  // ---- undo compaction: dropped rows get no gradient from the rows after them
  const void* dof = P(B.dog);
  const void* dxr = P(B.dx1);
  if (prune) {
    int32_t* inv = reinterpret_cast<int32_t*>(base + B.inv);
    HIP_TRY(launch_scatter_rows(s, dt, d, P(B.dog), kept, To, T, inv, P(B.dofull)), "scatter");
    HIP_TRY(launch_scatter_rows(s, dt, d, P(B.dx1), kept, To, T, inv, P(B.dxr)), "scatter");
    dof = P(B.dofull);
    dxr = P(B.dxr);
  }
  // ---- attention
  float* Dv = reinterpret_cast<float*>(base + B.D);
  HIP_TRY(launch_rowdot(s, dt, dof, wb.o, d, T, H, hd, Dv), "rowdot");
  char* dqkv = base + B.dqkv;
  HIP_TRY(launch_attention_bwd(s, q, k, v, qw, dof, d, wb.lse, Dv, H, kvg, hd, c.causal, scale,
                               in.B, in.max_len, T, in.cu_dev, dqkv, dqkv + d * e,
                               dqkv + (d + kvd) * e, qw),
          "attention gradient");
  if (dec) HIP_TRY(launch_rope_bwd(s, dt, dqkv, qw, T, d + kvd, hd, pos_in, rope), "rope gradient");
  // ---- qkv projection and norm1
  HIP_TRY(wgrad(dqkv, qw, P(B.h1), d, T, Tp, gr.w_qkv), "qkv weight gradient");
  HIP_TRY(colsum(dqkv, T, qw, nullptr, gr.b_qkv), "qkv bias gradient");
  HIP_TRY(xgrad(dqkv, T, w.w_qkv, qw, d, P(B.dh1)), "qkv input gradient");
  HIP_TRY(launch_norm_bwd(s, dt, norm_kind, x_in, w.norm1_w, P(B.dh1), dxr, dx, T, d, c.norm_eps,
                          stats),
          "norm1 gradient");
  HIP_TRY(colsum(P(B.dh1), T, d, x_in, gr.norm1_w), "norm1 gain gradient");
  if (!dec) HIP_TRY(colsum(P(B.dh1), T, d, nullptr, gr.norm1_b), "norm1 shift gradient");
  return ZSA_OK;
}

}  // namespace

size_t zsa_stack_backward_workspace_size(const zsa_layer_cfg* cfg, int32_t total_rows,
                                         int32_t batch, int32_t n_layers, int32_t n_prune) {
  if (cfg == nullptr || total_rows < 0 || batch < 0 || n_layers < 1 || n_prune < 0) return 0;
  const size_t T = static_cast<size_t>(total_rows);
  Carver cv;
  layer_layout(cfg, total_rows, cv);
  bwd_layout(cfg, total_rows, cv);
  cv.take(static_cast<size_t>(n_layers) * T * cfg->d_model * esize(cfg->dtype));  // layer inputs
  cv.take(static_cast<size_t>(n_layers) * T * 4);                                // positions
  cv.take(static_cast<size_t>(n_prune) * T * 4);                                 // kept rows
  cv.take(static_cast<size_t>(n_prune) * (batch + 1) * 4);                       // offsets
  cv.take(2 * T * cfg->d_model * esize(cfg->dtype));                             // gradients
  return cv.off;
}

int zsa_stack_backward(void* stream, const zsa_layer_cfg* cfg, const zsa_layer_weights* w,
                       const zsa_layer_grads* grads, int32_t n_layers, const int32_t* prune_after,
                       int32_t n_prune, const double* keep_rate, const void* hidden_in,
                       const int32_t* pos_in, int32_t batch, const int32_t* cu_host,
                       const int32_t* cu_dev, const void* dy, void* dx, void* ws,
                       size_t ws_bytes) {
  CHECK(check_cfg(cfg));
  if (!zsa::backward_supported(cfg->dtype, cfg->head_dim))
    return fail(ZSA_EUNSUPPORTED, "backward: bf16 with head_dim 64 or 128");
  if (cfg->mark_only) return fail(ZSA_EUNSUPPORTED, "backward of the mark-only mode");
  if (n_layers < 1 || w == nullptr || grads == nullptr)
    return fail(ZSA_EINVAL, "n_layers %d / weights / grads", n_layers);
  for (int l = 0; l < n_layers; ++l) {
    const zsa_layer_grads& g = grads[l];
    if (g.w_qkv == nullptr || g.w_o == nullptr || g.w_up == nullptr || g.w_down == nullptr ||
        g.norm1_w == nullptr || g.norm2_w == nullptr)
      return fail(ZSA_EINVAL, "layer %d: a weight gradient pointer is NULL", l + 1);
  }
  if (n_prune < 0 || (n_prune > 0 && prune_after == nullptr)) return fail(ZSA_EINVAL, "prune_after");
  for (int p = 0; p < n_prune; ++p) {
    if (prune_after[p] < 1 || prune_after[p] > n_layers || (p > 0 && prune_after[p] <= prune_after[p - 1]))
      return fail(ZSA_EINVAL, "prune_after must be strictly ascending in 1..%d", n_layers);
  }
  int32_t T0, max_len0;
  CHECK(check_seqs(batch, cu_host, cu_dev, &T0, &max_len0));
  CHECK(check_row_range(max_len0, qkv_width(*cfg), cfg->dtype, "attention"));
  if (n_prune > 0 && batch > 0 && keep_rate == nullptr) return fail(ZSA_EINVAL, "keep_rate is NULL");
  for (int b = 0; n_prune > 0 && b < batch; ++b) CHECK(check_rate(keep_rate[b]));
  if (T0 > 0) {
    CHECK(check_ptr16(hidden_in, "hidden_in"));
    CHECK(check_ptr16(dy, "dy"));
    CHECK(check_ptr16(dx, "dx"));
    if (pos_in == nullptr) return fail(ZSA_EINVAL, "pos_in is NULL");
  }
  const size_t need = zsa_stack_backward_workspace_size(cfg, T0, batch, n_layers, n_prune);
  if (ws == nullptr || ws_bytes < need) return fail(ZSA_EWORKSPACE, "workspace %zu < %zu", ws_bytes, need);
  if (T0 == 0) return ZSA_OK;

  // the schedule, as in the forward
  std::vector<std::vector<int32_t>> cus(n_prune + 1, std::vector<int32_t>(batch + 1, 0));
  std::vector<int32_t> maxl(n_prune + 1, 0);
  for (int b = 0; b <= batch; ++b) cus[0][b] = cu_host[b];
  maxl[0] = max_len0;
  for (int p = 1; p <= n_prune; ++p)
    for (int b = 0; b < batch; ++b) {
      const int32_t n = cus[p - 1][b + 1] - cus[p - 1][b];
      const int32_t kb = keep_count_impl(n, keep_rate[b], cfg->tau);
      cus[p][b + 1] = cus[p][b] + kb;
      maxl[p] = std::max(maxl[p], kb);
    }
  hipStream_t s = static_cast<hipStream_t>(stream);
  char* base = static_cast<char*>(ws);
  Carver cv;
  const LayerBufs wb = carve_layer(layer_layout(cfg, T0, cv), ws);
  const BwdLayout B = bwd_layout(cfg, T0, cv);
  const size_t e = esize(cfg->dtype);
  const size_t xrow = static_cast<size_t>(cfg->d_model) * e;
  char* xs = base + cv.take(static_cast<size_t>(n_layers) * T0 * xrow);
  int32_t* ps = reinterpret_cast<int32_t*>(base + cv.take(static_cast<size_t>(n_layers) * T0 * 4));
  int32_t* kept = reinterpret_cast<int32_t*>(base + cv.take(static_cast<size_t>(n_prune) * T0 * 4));
  int32_t* meta = reinterpret_cast<int32_t*>(base + cv.take(static_cast<size_t>(n_prune) * (batch + 1) * 4));
  char* gbuf = base + cv.take(2 * static_cast<size_t>(T0) * xrow);
  std::vector<int32_t> flat;
  for (int p = 1; p <= n_prune; ++p) flat.insert(flat.end(), cus[p].begin(), cus[p].end());
  if (!flat.empty()) HIP_TRY(zsa::launch_upload_i32(s, meta, flat.data(), static_cast<int>(flat.size())), "upload");

  // forward, keeping every layer's input rows, positions and kept rows
  std::vector<const void*> xin(n_layers + 1);
  std::vector<const int32_t*> pin(n_layers + 1);
  std::vector<RowSet> rin(n_layers + 1);
  std::vector<int> pt_of(n_layers + 1, -1);
  xin[1] = hidden_in;
  pin[1] = pos_in;
  rin[1] = RowSet{batch, cus[0].data(), cu_dev, T0, max_len0};
  int point = 0;
  for (int l = 1; l <= n_layers; ++l) {
    const bool prune = point < n_prune && prune_after[point] == l;
    RowSet nxt = rin[l];
    if (prune) {
      nxt = RowSet{batch, cus[point + 1].data(), meta + static_cast<size_t>(point) * (batch + 1),
                   cus[point + 1][batch], maxl[point + 1]};
      pt_of[l] = point;
    }
    if (l < n_layers) {
      void* x_out = xs + static_cast<size_t>(l) * T0 * xrow;
      int32_t* p_out = prune ? ps + static_cast<size_t>(l) * T0 : nullptr;
      CHECK(run_layer(s, *cfg, w[l - 1], xin[l], pin[l], rin[l], prune, nxt, x_out, p_out,
                      nullptr, prune ? kept + static_cast<size_t>(point) * T0 : nullptr, wb));
      xin[l + 1] = x_out;
      pin[l + 1] = prune ? p_out : pin[l];
      rin[l + 1] = nxt;
    } else if (prune) {
      // the last layer's kept rows, for its backward
      CHECK(run_layer(s, *cfg, w[l - 1], xin[l], pin[l], rin[l], true, nxt, gbuf, ps, nullptr,
                      kept + static_cast<size_t>(point) * T0, wb));
    }
    if (prune) ++point;
  }
  // backward, last layer first
  const void* g_in = dy;
  for (int l = n_layers; l >= 1; --l) {
    const bool prune = pt_of[l] >= 0;
    const RowSet out = prune ? RowSet{batch, cus[pt_of[l] + 1].data(),
                                      meta + static_cast<size_t>(pt_of[l]) * (batch + 1),
                                      cus[pt_of[l] + 1][batch], maxl[pt_of[l] + 1]}
                             : rin[l];
    void* g_out = l == 1 ? dx : gbuf + static_cast<size_t>(l & 1) * T0 * xrow;
    CHECK(layer_backward(s, *cfg, w[l - 1], grads[l - 1], xin[l], pin[l], rin[l], prune, out,
                         prune ? kept + static_cast<size_t>(pt_of[l]) * T0 : nullptr, g_in, g_out,
                         wb, base, B));
    g_in = g_out;
  }
  return ZSA_OK;
}

// ---------------------------------------------------------------------------
// generation after a pruned prefill
// ---------------------------------------------------------------------------
struct DecodeLayout {
  size_t h, qkv, o, f, m, l, op, pos, len, splitk, splitk_bytes, end;
};

// the four projections of a block: fused q|k|v, output, up, down (N, K)
void decode_gemm_shapes(const zsa_layer_cfg& c, int nk[4][2]) {
  const int d = c.d_model, F = c.d_ff, qw = static_cast<int>(qkv_width(c));
  const int up_n = c.kind == ZSA_DECODER ? 2 * F : F;
  const int shapes[4][2] = {{qw, d}, {d, d}, {up_n, d}, {d, F}};
  for (int g = 0; g < 4; ++g) {
    nk[g][0] = shapes[g][0];
    nk[g][1] = shapes[g][1];
  }
}

DecodeLayout decode_layout(const zsa_layer_cfg* c, int32_t batch, int32_t cap, int32_t n_layers) {
  const size_t e = esize(c->dtype);
  const int64_t d = c->d_model, F = c->d_ff, qw = qkv_width(*c);
  const int S = zsa::decode_splits_bound(cap);
  const size_t part = static_cast<size_t>(batch) * c->n_heads * S;
  Carver cv;
  DecodeLayout L;
  L.h = cv.take(batch * d * e);
  L.qkv = cv.take(batch * qw * e);
  L.o = cv.take(batch * d * e);
  L.f = cv.take(batch * F * e);
  L.m = cv.take(part * 4);
  L.l = cv.take(part * 4);
  L.op = cv.take(part * c->head_dim * 4);
  // host values of the step, uploaded together: pos [batch], then per layer
  // the cache row of the new row and the rows attended [2 batch]
  L.pos = cv.take(static_cast<size_t>(batch) * (1 + 2 * std::max(n_layers, 1)) * 4);
  L.len = L.pos + static_cast<size_t>(batch) * 4;
  // split-K partials of projections that do not take the few-row kernel
  int nk[4][2];
  decode_gemm_shapes(*c, nk);
  L.splitk_bytes = 0;
  for (int g = 0; g < 4; ++g)
    L.splitk_bytes = std::max(L.splitk_bytes,
                              zsa::gemm_workspace_bound(c->dtype, batch, nk[g][0], nk[g][1]));
  L.splitk = cv.take(L.splitk_bytes);
  L.end = cv.off;
  return L;
}

size_t zsa_decode_workspace_size(const zsa_layer_cfg* cfg, int32_t n_layers, int32_t batch,
                                 int32_t kv_capacity) {
  if (cfg == nullptr || n_layers < 1 || batch < 0 || kv_capacity < 1) return 0;
  return decode_layout(cfg, batch, kv_capacity, n_layers).end;
}

int zsa_decode_step(void* stream, const zsa_layer_cfg* cfg, const zsa_layer_weights* w,
                    int32_t n_layers, int32_t batch, const void* x_in, const int32_t* pos_host,
                    void* kv_cache, int32_t kv_capacity, const int32_t* kv_len_host, void* x_out,
                    void* ws, size_t ws_bytes) {
  using namespace zsa;
  CHECK(check_cfg(cfg));
  const zsa_layer_cfg& c = *cfg;
  const int d = c.d_model, H = c.n_heads, hd = c.head_dim, F = c.d_ff;
  const int kvd = kv_heads(c) * hd, qw = static_cast<int>(qkv_width(c)), kvg = H / kv_heads(c);
  if (!c.causal) return fail(ZSA_EINVAL, "decoding needs the causal mask");
  if (!decode_supported(c.dtype, hd, kvg))
    return fail(ZSA_EUNSUPPORTED, "decode: bf16 with head_dim 64 or 128 and 1, 2, 4 or 8 query "
                                  "heads per key/value head");
  if (n_layers < 1 || w == nullptr) return fail(ZSA_EINVAL, "n_layers %d / weights", n_layers);
  if (batch < 0) return fail(ZSA_EINVAL, "batch %d", batch);
  if (batch == 0) return ZSA_OK;
  if (kv_capacity < 1) return fail(ZSA_EINVAL, "kv_capacity %d", kv_capacity);
  CHECK(check_row_range(kv_capacity, 2 * static_cast<int64_t>(kvd), c.dtype, "kv cache"));
  CHECK(check_ptr16(x_in, "x_in"));
  CHECK(check_ptr16(x_out, "x_out"));
  CHECK(check_ptr16(kv_cache, "kv_cache"));
  if (reinterpret_cast<uintptr_t>(kv_cache) % 256 != 0)
    return fail(ZSA_EINVAL, "kv_cache must be 256-byte aligned");
  if (pos_host == nullptr || kv_len_host == nullptr) return fail(ZSA_EINVAL, "pos / kv_len is NULL");
  for (int i = 0; i < n_layers * batch; ++i)
    if (kv_len_host[i] < 0 || kv_len_host[i] >= kv_capacity)
      return fail(ZSA_ESHAPE, "kv_len[%d] = %d leaves no room below kv_capacity %d", i,
                  kv_len_host[i], kv_capacity);
  const DecodeLayout L = decode_layout(cfg, batch, kv_capacity, n_layers);
  if (ws == nullptr || ws_bytes < L.end)
    return fail(ZSA_EWORKSPACE, "workspace %zu < %zu", ws_bytes, L.end);
  hipStream_t s = static_cast<hipStream_t>(stream);
  char* base = static_cast<char*>(ws);
  void* h = base + L.h;
  void* qkv = base + L.qkv;
  void* o = base + L.o;
  void* f = base + L.f;
  int32_t* pos_dev = reinterpret_cast<int32_t*>(base + L.pos);
  int32_t* len_dev = reinterpret_cast<int32_t*>(base + L.len);
  void* splitk = L.splitk_bytes ? base + L.splitk : nullptr;
  const bool dec = c.kind == ZSA_DECODER;
  const int norm_kind = dec ? ZSA_NORM_RMS : ZSA_NORM_LAYER;
  const size_t e = esize(c.dtype);
  const size_t layer_bytes = static_cast<size_t>(batch) * kv_capacity * 2 * kvd * e;

  std::vector<int32_t> host_ints;
  host_ints.reserve(static_cast<size_t>(batch) * (1 + 2 * n_layers));
  host_ints.insert(host_ints.end(), pos_host, pos_host + batch);
  std::vector<int> max_n(n_layers, 0);
  for (int l = 0; l < n_layers; ++l) {
    for (int b = 0; b < batch; ++b) host_ints.push_back(kv_len_host[l * batch + b]);  // new row
    for (int b = 0; b < batch; ++b) {
      host_ints.push_back(kv_len_host[l * batch + b] + 1);  // rows attended, the new one included
      max_n[l] = std::max(max_n[l], kv_len_host[l * batch + b] + 1);
    }
  }
  HIP_TRY(launch_upload_i32(s, pos_dev, host_ints.data(), static_cast<int>(host_ints.size())),
          "upload");
  // few-row projections stream W through the matrix cores; other shapes
  // take the general GEMM
  auto proj = [&](const void* x, int K, const void* wt, int N, const EpiParams& ep) -> hipError_t {
    return launch_gemm(s, c.dtype, x, batch, K, wt, N, ep, splitk, L.splitk_bytes);
  };
  // the block's pre-norm and the projection that reads it: folded into the
  // few-row kernel when it can take it, else normalised into h first
  auto norm_proj = [&](const void* x, const void* g, const void* b, const void* wt, int N,
                       const EpiParams& ep) -> hipError_t {
    if (skinny_ok(c.dtype, batch, N, d, ep) && skinny_norm_ok(batch, N, d)) {
      const PreNorm pn{static_cast<const bf16_t*>(g), dec ? nullptr : static_cast<const bf16_t*>(b),
                       dec ? 1 : 0, c.norm_eps};
      return launch_gemm_skinny(s, x, batch, d, wt, N, ep, &pn);
    }
    hipError_t e = launch_norm(s, c.dtype, norm_kind, x, g, dec ? nullptr : b, batch, d,
                               c.norm_eps, h);
    if (e != hipSuccess) return e;
    return proj(h, d, wt, N, ep);
  };
  for (int l = 0; l < n_layers; ++l) {
    const zsa_layer_weights& wl = w[l];
    const void* xin = l == 0 ? x_in : x_out;
    void* cache_l = static_cast<char*>(kv_cache) + l * layer_bytes;
    int32_t* len_l = len_dev + 2 * batch * l;
    {
      EpiParams ep{};
      ep.epi = dec ? EPI_ROPE : EPI_NONE;
      ep.bias = wl.b_qkv;
      ep.y = qkv;
      ep.ldy = qw;
      ep.pos = pos_dev;
      ep.head_dim = hd;
      ep.rope_cols = dec ? d + kvd : 0;
      if (dec) fill_rope(ep, hd, c.rope_theta);
      HIP_TRY(norm_proj(xin, wl.norm1_w, wl.norm1_b, wl.w_qkv, qw, ep), "norm1, qkv projection");
    }
    HIP_TRY(launch_decode_attention(s, qkv, qw, d, cache_l, kv_capacity, hd, H, kv_heads(c),
                                    len_l + batch, batch, max_n[l],
                                    1.0f / sqrtf(static_cast<float>(hd)),
                                    reinterpret_cast<float*>(base + L.m),
                                    reinterpret_cast<float*>(base + L.l),
                                    reinterpret_cast<float*>(base + L.op), o, d),
            "decode attention");
    {
      EpiParams ep{};
      ep.epi = EPI_RESIDUAL;
      ep.bias = wl.b_o;
      ep.residual = xin;
      ep.y = x_out;
      ep.ldy = d;
      HIP_TRY(proj(o, d, wl.w_o, d, ep), "output projection");
    }
    {
      EpiParams ep{};
      ep.epi = dec ? EPI_SWIGLU : EPI_GELU;
      ep.bias = wl.b_up;
      ep.y = f;
      ep.ldy = F;
      HIP_TRY(norm_proj(x_out, wl.norm2_w, wl.norm2_b, wl.w_up, dec ? 2 * F : F, ep),
              "norm2, up projection");
    }
    {
      EpiParams ep{};
      ep.epi = EPI_RESIDUAL;
      ep.bias = wl.b_down;
      ep.residual = x_out;
      ep.y = x_out;
      ep.ldy = d;
      HIP_TRY(proj(f, F, wl.w_down, d, ep), "down projection");
    }
  }
  return ZSA_OK;
}

int zsa_timing_arm(int32_t kclass, int32_t capacity) {
  if (kclass < 0 || kclass >= zsa::K_NCLASS) return fail(ZSA_EINVAL, "kernel class %d", kclass);
  if (capacity < 1) return fail(ZSA_EINVAL, "capacity %d", capacity);
  TimingState& t = g_timing[kclass];
  while (static_cast<int>(t.start.size()) < capacity) {
    hipEvent_t a, b;
    HIP_TRY(hipEventCreate(&a), "event create");
    HIP_TRY(hipEventCreate(&b), "event create");
    t.start.push_back(a);
    t.stop.push_back(b);
  }
  t.armed = true;
  t.used = 0;
  return ZSA_OK;
}

int zsa_timing_read(int32_t kclass, int32_t* launches, double* total_ms) {
  if (kclass < 0 || kclass >= zsa::K_NCLASS) return fail(ZSA_EINVAL, "kernel class %d", kclass);
  if (launches == nullptr || total_ms == nullptr) return fail(ZSA_EINVAL, "NULL output");
  TimingState& t = g_timing[kclass];
  double sum = 0.0;
  for (int i = 0; i < t.used; ++i) {
    HIP_TRY(hipEventSynchronize(t.stop[i]), "event sync");
    float ms = 0.f;
    HIP_TRY(hipEventElapsedTime(&ms, t.start[i], t.stop[i]), "event time");
    sum += ms;
  }
  *launches = t.used;
  *total_ms = sum;
  t.armed = false;
  t.used = 0;
  return ZSA_OK;
}

}  // extern "C"
