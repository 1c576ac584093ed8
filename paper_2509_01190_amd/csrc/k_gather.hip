// Compaction of kept rows (pruned rows take no part in later layers) and the
// small metadata kernels.
//
// gather_rows: every thread moves one 16-byte chunk of one kept row; a row of
// d bf16 values is d/8 chunks, so consecutive threads read and write
// consecutive 16-byte pieces of a row (coalesced). Up to two row arrays share
// one index read (the layer path moves the residual and the attention output
// of the kept rows together). The kernel is HBM-bound: 2 * t_out * d * size
// bytes per array plus the index and position words.
#include "zsa_internal.h"

namespace zsa {
namespace {

__global__ __launch_bounds__(256) void gather_rows_kernel(
    int chunks_per_row, int t_in, const int32_t* __restrict__ kept, int t_out,
    const uint4* __restrict__ src0, uint4* __restrict__ dst0, const uint4* __restrict__ src1,
    uint4* __restrict__ dst1, const int32_t* __restrict__ pos, int32_t* __restrict__ pos_out) {
  const int64_t total = static_cast<int64_t>(t_out) * chunks_per_row;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < total;
       i += stride) {
    const int r = static_cast<int>(i / chunks_per_row);
    const int c = static_cast<int>(i - static_cast<int64_t>(r) * chunks_per_row);
    const int src = kept[r];
    const bool ok = src >= 0 && src < t_in;
    const int64_t so = static_cast<int64_t>(src) * chunks_per_row + c;
    const int64_t d_o = static_cast<int64_t>(r) * chunks_per_row + c;
    uint4 v0 = make_uint4(0u, 0u, 0u, 0u), v1 = v0;
    if (ok) {
      v0 = src0[so];
      if (src1 != nullptr) v1 = src1[so];
    }
    dst0[d_o] = v0;
    if (src1 != nullptr) dst1[d_o] = v1;
    if (c == 0 && pos_out != nullptr) pos_out[r] = ok ? pos[src] : -1;
  }
}

__global__ void gather_pos_kernel(int t_in, const int32_t* __restrict__ kept, int t_out,
                                  const int32_t* __restrict__ pos, int32_t* __restrict__ pos_out) {
  const int r = blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= t_out) return;
  const int src = kept[r];
  pos_out[r] = (src >= 0 && src < t_in) ? pos[src] : -1;
}

constexpr int kUploadMax = 248;
struct I32Payload {
  int32_t n;
  int32_t v[kUploadMax];
};

__global__ void upload_kernel(int32_t* __restrict__ dst, I32Payload p) {
  for (int i = threadIdx.x; i < p.n; i += blockDim.x) dst[i] = p.v[i];
}

__global__ void copy_i32_kernel(int32_t* __restrict__ dst, const int32_t* __restrict__ src,
                                int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) dst[i] = src[i];
}

}  // namespace

hipError_t launch_gather(hipStream_t s, int dtype, int d, int t_in, const int32_t* kept,
                         int t_out, const void* src0, void* dst0, const void* src1, void* dst1,
                         const int32_t* pos, int32_t* pos_out) {
  if (t_out == 0) return hipSuccess;
  if (src0 == nullptr) {
    return launch(K_GATHER, gather_pos_kernel, dim3((t_out + 255) / 256), dim3(256), 0, s, t_in,
                  kept, t_out, pos, pos_out);
  }
  const int esz = dtype == 1 ? 2 : 4;
  const int cpr = d * esz / 16;
  const int64_t total = static_cast<int64_t>(t_out) * cpr;
  int64_t blocks = (total + 255) / 256;
  if (blocks > 256 * 64) blocks = 256 * 64;  // grid-stride beyond ~16 waves of workgroups per CU
  return launch(K_GATHER, gather_rows_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0,
                s, cpr, t_in, kept, t_out, static_cast<const uint4*>(src0),
                static_cast<uint4*>(dst0), static_cast<const uint4*>(src1),
                static_cast<uint4*>(dst1), pos, pos_out);
}

// Host values reach the device through kernel arguments (no host-to-device
// copy, so the call stays capturable in a HIP graph).
hipError_t launch_upload_i32(hipStream_t s, int32_t* dst, const int32_t* host_vals, int n) {
  for (int off = 0; off < n; off += kUploadMax) {
    I32Payload p;
    p.n = n - off < kUploadMax ? n - off : kUploadMax;
    for (int i = 0; i < p.n; ++i) p.v[i] = host_vals[off + i];
    const hipError_t e = launch(K_MISC, upload_kernel, dim3(1), dim3(256), 0, s, dst + off, p);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_copy_i32(hipStream_t s, int32_t* dst, const int32_t* src, int n) {
  if (n == 0) return hipSuccess;
  return launch(K_MISC, copy_i32_kernel, dim3((n + 255) / 256), dim3(256), 0, s, dst, src, n);
}

}  // namespace zsa
