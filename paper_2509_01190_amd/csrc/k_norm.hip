// Row normalisation of the pre-norm block (LayerNorm / RMSNorm).
// LW lanes per row (a 64-lane wave, or half of one for rows of up to 96
// 16-byte chunks), 256 / LW rows per workgroup; each lane keeps its 16-byte
// chunks of the row in registers, so the row is read from HBM once and the
// statistics are exact two-pass (mean, then centred sum of squares) in fp32.
#include "zsa_internal.h"

namespace zsa {
namespace {

// sum over the LW lanes of a row (xor offsets below LW stay inside it)
template <int LW>
__device__ __forceinline__ float row_sum(float v) {
#pragma unroll
  for (int off = LW / 2; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

template <typename T, int MAXC, bool RMS, int LW>
__global__ __launch_bounds__(256) void norm_kernel(const T* __restrict__ x,
                                                   const T* __restrict__ g,
                                                   const T* __restrict__ b, int rows, int d,
                                                   float eps, T* __restrict__ y) {
  constexpr int V = Vec16<T>::N;
  const int lane = threadIdx.x & (LW - 1);
  const int row = blockIdx.x * (256 / LW) + threadIdx.x / LW;
  if (row >= rows) return;
  const int C = d / V;
  const uint4* xr = reinterpret_cast<const uint4*>(x + static_cast<size_t>(row) * d);
  float v[MAXC][V];
  float sum = 0.f;
#pragma unroll
  for (int i = 0; i < MAXC; ++i) {
    const int c = lane + i * LW;
    if (c < C) {
      unpack16(xr[c], v[i], T());
#pragma unroll
      for (int e = 0; e < V; ++e) sum += v[i][e];
    } else {
#pragma unroll
      for (int e = 0; e < V; ++e) v[i][e] = 0.f;
    }
  }
  const float inv_d = 1.0f / static_cast<float>(d);
  float mean = 0.f;
  float sq = 0.f;
  if (!RMS) {
    mean = row_sum<LW>(sum) * inv_d;
#pragma unroll
    for (int i = 0; i < MAXC; ++i) {
      if (lane + i * LW < C) {
#pragma unroll
        for (int e = 0; e < V; ++e) {
          const float t = v[i][e] - mean;
          sq += t * t;
        }
      }
    }
  } else {
#pragma unroll
    for (int i = 0; i < MAXC; ++i)
#pragma unroll
      for (int e = 0; e < V; ++e) sq += v[i][e] * v[i][e];
  }
  const float rstd = 1.0f / sqrtf(row_sum<LW>(sq) * inv_d + eps);
  const uint4* gr = reinterpret_cast<const uint4*>(g);
  const uint4* br = reinterpret_cast<const uint4*>(b);
  uint4* yr = reinterpret_cast<uint4*>(y + static_cast<size_t>(row) * d);
#pragma unroll
  for (int i = 0; i < MAXC; ++i) {
    const int c = lane + i * LW;
    if (c < C) {
      float gv[V], bv[V], o[V];
      unpack16(gr[c], gv, T());
      if (!RMS && b != nullptr) {
        unpack16(br[c], bv, T());
      } else {
#pragma unroll
        for (int e = 0; e < V; ++e) bv[e] = 0.f;
      }
#pragma unroll
      for (int e = 0; e < V; ++e) o[e] = (v[i][e] - mean) * rstd * gv[e] + bv[e];
      yr[c] = pack16(o, T());
    }
  }
}

template <typename T, bool RMS>
hipError_t dispatch(hipStream_t s, const void* x, const void* g, const void* b, int rows, int d,
                    float eps, void* y) {
  constexpr int V = Vec16<T>::N;
  const int C = d / V;
  const dim3 block(256);
  const T* xp = static_cast<const T*>(x);
  const T* gp = static_cast<const T*>(g);
  const T* bp = static_cast<const T*>(b);
  T* yp = static_cast<T*>(y);
  // rows of up to 96 chunks (768 bf16): half a wave per row
  if (C <= 96) {
    const dim3 grid((rows + 7) / 8);
    if (C <= 32) return launch(K_NORM, norm_kernel<T, 1, RMS, 32>, grid, block, 0, s, xp, gp, bp, rows, d, eps, yp);
    if (C <= 64) return launch(K_NORM, norm_kernel<T, 2, RMS, 32>, grid, block, 0, s, xp, gp, bp, rows, d, eps, yp);
    return launch(K_NORM, norm_kernel<T, 3, RMS, 32>, grid, block, 0, s, xp, gp, bp, rows, d, eps, yp);
  }
  const dim3 grid((rows + 3) / 4);
  if (C <= 128) return launch(K_NORM, norm_kernel<T, 2, RMS, 64>, grid, block, 0, s, xp, gp, bp, rows, d, eps, yp);
  if (C <= 256) return launch(K_NORM, norm_kernel<T, 4, RMS, 64>, grid, block, 0, s, xp, gp, bp, rows, d, eps, yp);
  if (C <= 512) return launch(K_NORM, norm_kernel<T, 8, RMS, 64>, grid, block, 0, s, xp, gp, bp, rows, d, eps, yp);
  if (C <= 1024) return launch(K_NORM, norm_kernel<T, 16, RMS, 64>, grid, block, 0, s, xp, gp, bp, rows, d, eps, yp);
  return hipErrorInvalidValue;
}

}  // namespace

hipError_t launch_norm(hipStream_t s, int dtype, int kind, const void* x, const void* g,
                       const void* b, int rows, int d, float eps, void* y) {
  if (rows == 0) return hipSuccess;
  if (dtype == 1)
    return kind == 1 ? dispatch<bf16_t, true>(s, x, g, b, rows, d, eps, y)
                     : dispatch<bf16_t, false>(s, x, g, b, rows, d, eps, y);
  return kind == 1 ? dispatch<float, true>(s, x, g, b, rows, d, eps, y)
                   : dispatch<float, false>(s, x, g, b, rows, d, eps, y);
}

}  // namespace zsa
