// zsa_attention_with_scores_static: the attention-with-scores call for
// callers that cannot allocate device memory (code under HIP graph capture,
// tight serving loops). Its scratch -- the log-sum-exp rows when the caller
// does not want them, and the per-head-group score partials -- lives in a
// file-scope device array of fixed size instead of a caller workspace.
//
// The array's name is a host-side stand-in in host code: its device
// address is looked up once per device (with that device current) through
// hipGetSymbolAddress and kept; only that address reaches kernels.
#include <mutex>

#include "../../include/zsa.h"
#include "zsa_internal.h"

namespace {

constexpr size_t kScratchBytes = size_t{32} << 20;
constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

std::mutex g_lock;
void* g_scratch_ptr[kMaxDevices] = {};

// the current device's copy of the array (looked up on its first use there)
int scratch_on_current_device(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return zsa::set_error(ZSA_EHIP, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices)
    return zsa::set_error(ZSA_EUNSUPPORTED, "device %d beyond the %d the static scratch serves",
                          dev, kMaxDevices);
  std::lock_guard<std::mutex> guard(g_lock);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || p == nullptr)
      return zsa::set_error(ZSA_EHIP, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return ZSA_OK;
}

}  // namespace

extern "C" {

size_t zsa_static_scratch_bytes(void) { return kScratchBytes; }

int zsa_attention_with_scores_static(void* stream, int32_t dtype, const void* q, const void* k,
                                     const void* v, int64_t row_stride, int32_t n_heads,
                                     int32_t n_kv_heads, int32_t head_dim, int32_t causal,
                                     float scale, int32_t batch, const int32_t* cu_host,
                                     const int32_t* cu_dev, void* out, int64_t out_stride,
                                     float* lse, float* scores) {
  // the scratch this call needs, checked against the array before anything
  // else touches the GPU (malformed offsets are reported by the call below)
  if (batch >= 0 && cu_host != nullptr && n_heads > 0) {
    const int32_t rows = cu_host[batch];
    size_t need = 0;
    if (rows >= 0) {
      // the workspace rule of zsa_attention_with_scores: partials when scores
      // are wanted, the log-sum-exp rows when the caller passes none
      need = zsa_attention_workspace_size(n_heads, rows, scores != nullptr);
      if (lse != nullptr && scores == nullptr) need = 0;
    }
    if (need > kScratchBytes)
      return zsa::set_error(ZSA_EUNSUPPORTED,
                            "attention over %d rows x %d heads needs %zu bytes of scratch; the "
                            "static scratch holds %zu (use zsa_attention_with_scores with a "
                            "workspace)",
                            rows, n_heads, need, kScratchBytes);
  }
  void* ws = nullptr;
  const int rc = scratch_on_current_device(&ws);
  if (rc != ZSA_OK) return rc;
  return zsa_attention_with_scores(stream, dtype, q, k, v, row_stride, n_heads, n_kv_heads,
                                   head_dim, causal, scale, batch, cu_host, cu_dev, out,
                                   out_stride, lse, scores, ws, kScratchBytes);
}

}  // extern "C"
