// Stand-ins for everything the C-ABI's host code calls on the device side,
// for the sanitized host-only build of the argument validation and the
// Eq. 2 schedule. A launch stub must never run: every call the driver makes
// either is host-only or fails validation before the first launch, so
// reaching one aborts the driver (and fails the test). The shape helpers
// return fixed, harmless values: no workspace size is checked here.
#include <stdio.h>
#include <stdlib.h>

#include "../../paper_2509_01190_amd/csrc/zsa_internal.h"

namespace {
[[noreturn]] void reached(const char* what) {
  fprintf(stderr, "launch stub reached: %s\n", what);
  abort();
}
}  // namespace

extern "C" {
const char* hipGetErrorString(hipError_t) { return "hip stub"; }
hipError_t hipMemcpyAsync(void*, const void*, size_t, hipMemcpyKind, hipStream_t) {
  reached("hipMemcpyAsync");
}
hipError_t hipEventCreate(hipEvent_t*) { reached("hipEventCreate"); }
hipError_t hipEventSynchronize(hipEvent_t) { reached("hipEventSynchronize"); }
hipError_t hipEventElapsedTime(float*, hipEvent_t, hipEvent_t) { reached("hipEventElapsedTime"); }
}

namespace zsa {
hipError_t launch_norm(hipStream_t, int, int, const void*, const void*, const void*, int, int,
                       float, void*) {
  reached("launch_norm");
}
hipError_t launch_gemm(hipStream_t, int, const void*, int, int, const void*, int,
                       const EpiParams&, void*, size_t) {
  reached("launch_gemm");
}
size_t gemm_workspace_bytes(int, int, int, int) { return 0; }
size_t gemm_workspace_bound(int, int, int, int) { return 0; }
bool skinny_ok(int, int, int, int, const EpiParams&) { return false; }
bool skinny_norm_ok(int, int, int) { return false; }
hipError_t launch_gemm_skinny(hipStream_t, const void*, int, int, const void*, int,
                              const EpiParams&, const PreNorm*) {
  reached("launch_gemm_skinny");
}
hipError_t launch_attention(hipStream_t, int, const void*, const void*, const void*, int64_t, int,
                            int, int, int, float, int, int, int, const int32_t*, void*, int64_t,
                            float*) {
  reached("launch_attention");
}
hipError_t launch_score(hipStream_t, int, const void*, const void*, int64_t, const float*, int,
                        int, int, int, float, int, int, int, const int32_t*, float*, int) {
  reached("launch_score");
}
int score_groups(int, int, int, int) { return 1; }
hipError_t launch_score_finalize(hipStream_t, const float*, int, int, float*) {
  reached("launch_score_finalize");
}
hipError_t launch_select(hipStream_t, const float*, int, int, int, int, const int32_t*,
                         const int32_t*, int32_t*, float*, int) {
  reached("launch_select");
}
hipError_t launch_kv_store(hipStream_t, int, const void*, int64_t, int, int, int, int,
                           const int32_t*, const int32_t*, void*, int) {
  reached("launch_kv_store");
}
hipError_t launch_decode_attention(hipStream_t, const void*, int64_t, int, void*, int, int, int,
                                   int, const int32_t*, int, int, float, float*, float*, float*,
                                   void*, int64_t) {
  reached("launch_decode_attention");
}
int decode_splits_bound(int) { return 1; }
bool decode_supported(int dtype, int hd, int group) {
  return dtype == 1 && (hd == 64 || hd == 128) &&
         (group == 1 || group == 2 || group == 4 || group == 8);
}
bool backward_supported(int dtype, int hd) { return dtype == 1 && (hd == 64 || hd == 128); }
hipError_t launch_gemm_f32(hipStream_t, const void*, int, int, const void*, int, float*, void*,
                           size_t) {
  reached("launch_gemm_f32");
}
size_t gemm_f32_workspace_bound(int, int, int) { return 0; }
hipError_t launch_transpose(hipStream_t, int, const void*, int, int, int64_t, void*, int) {
  reached("launch_transpose");
}
size_t colsum_scratch_floats(int, int) { return 0; }
hipError_t launch_colsum(hipStream_t, int, const void*, int64_t, const void*, int64_t,
                         const float*, int, int, float*, float*) {
  reached("launch_colsum");
}
hipError_t launch_norm_bwd(hipStream_t, int, int, const void*, const void*, const void*,
                           const void*, void*, int, int, float, float*) {
  reached("launch_norm_bwd");
}
hipError_t launch_act_fwd(hipStream_t, int, const void*, void*, int, int, int) {
  reached("launch_act_fwd");
}
hipError_t launch_act_bwd(hipStream_t, int, const void*, const void*, void*, int, int, int) {
  reached("launch_act_bwd");
}
hipError_t launch_scatter_rows(hipStream_t, int, int, const void*, const int32_t*, int, int,
                               int32_t*, void*) {
  reached("launch_scatter_rows");
}
hipError_t launch_rowdot(hipStream_t, int, const void*, const void*, int64_t, int, int, int,
                         float*) {
  reached("launch_rowdot");
}
hipError_t launch_rope_bwd(hipStream_t, int, void*, int64_t, int, int, int, const int32_t*,
                           const EpiParams&) {
  reached("launch_rope_bwd");
}
hipError_t launch_attention_bwd(hipStream_t, const void*, const void*, const void*, int64_t,
                                const void*, int64_t, const float*, const float*, int, int, int,
                                int, float, int, int, int, const int32_t*, void*, void*, void*,
                                int64_t) {
  reached("launch_attention_bwd");
}
hipError_t launch_rope_table(hipStream_t, const int32_t*, int, const EpiParams&, float*) {
  reached("launch_rope_table");
}
hipError_t launch_gather(hipStream_t, int, int, int, const int32_t*, int, const void*, void*,
                         const void*, void*, const int32_t*, int32_t*) {
  reached("launch_gather");
}
hipError_t launch_upload_i32(hipStream_t, int32_t*, const int32_t*, int) {
  reached("launch_upload_i32");
}
hipError_t launch_copy_i32(hipStream_t, int32_t*, const int32_t*, int) {
  reached("launch_copy_i32");
}
}  // namespace zsa
