// Contribution score of every row at a pruning layer: the column sums of
// the normalised soft-score matrices, summed over heads,
//     s[j] = sum_h sum_i exp(q_i . k_j * scale - lse_h[i]),
// over the rows i the mask lets see row j. The normalised probability needs
// each query row's final log-sum-exp, which the attention pass has already
// written, so this is a second sweep over Q K^T that never stores P.
//
// bf16, head_dim 64/128 (MFMA): one 256-thread workgroup per (128-key block,
// head group, sequence). Its K tile sits in registers as the B operand; the
// 4 waves stride over 32-query tiles and compute S = Q K^T with
// v_mfma_f32_32x32x16_bf16 in the *non*-transposed layout, where a lane owns
// one key column and 16 query rows, so the column sum is in-lane adds. The
// log-sum-exp values of the query rows are staged in LDS (2048 at a time).
// Lane halves and waves are combined in a fixed order and the workgroup
// writes one partial vector per head group ([G][T]); the top-k kernel adds
// the G partials in a fixed order. No atomics: the result is bitwise
// reproducible. Causal workgroups start at the first query that can see
// their keys.
//
// fp32 / other head dims: one thread per key, vector ALU.
#include <math.h>

#include "zsa_internal.h"

namespace zsa {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr int kLseChunk = 2048;
// keys per workgroup: every workgroup reads the query rows of its heads once,
// so wider key blocks move fewer bytes per score
constexpr int kScoreKeys = 128;

template <int HD, int KB>
__global__ __launch_bounds__(256) void score_mfma_kernel(
    const bf16_t* __restrict__ Q, const bf16_t* __restrict__ K, int64_t rs,
    const float* __restrict__ lse, int H, int kv_group, int causal, float scale_log2,
    const int32_t* __restrict__ cu, int T, int groups, float* __restrict__ partials) {
  constexpr int KLD = HD + 8;
  constexpr int KK = HD / 16;
  constexpr int KS = KB / 32;  // 32-key column blocks
  __shared__ __align__(16) bf16_t Ks[KB * KLD];
  __shared__ __align__(16) float Ls[kLseChunk];
  __shared__ float red[4][KB];

  const int b = blockIdx.z, g = blockIdx.y;
  const int lo = cu[b];
  const int n = cu[b + 1] - lo;
  const int j0 = blockIdx.x * KB;
  if (j0 >= n) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5, l32 = lane & 31;
  float colsum[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) colsum[ks] = 0.f;

  const int qs = causal ? (j0 & ~31) : 0;
  for (int h = g; h < H; h += groups) {
    __syncthreads();  // previous head's readers are done with Ks / Ls
    for (int c = tid; c < KB * HD / 8; c += 256) {
      const int r = c / (HD / 8), ch = (c % (HD / 8)) * 8;
      const int jr = j0 + r;
      // keys past the sequence repeat the last row; their columns are not written
      *reinterpret_cast<uint4*>(Ks + r * KLD + ch) =
          *reinterpret_cast<const uint4*>(K + static_cast<int64_t>(lo + min(jr, n - 1)) * rs +
                                          (h / kv_group) * HD + ch);
    }
    __syncthreads();
    bf16x8_t kf[KS][KK];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int kk = 0; kk < KK; ++kk)
        kf[ks][kk] = __builtin_bit_cast(
            bf16x8_t, *reinterpret_cast<const uint4*>(Ks + (ks * 32 + l32) * KLD + kk * 16 + half * 8));

    const bf16_t* qh = Q + static_cast<int64_t>(lo) * rs + h * HD + half * 8;
    for (int c0 = qs; c0 < n; c0 += kLseChunk) {
      const int cend = min(n, c0 + kLseChunk);
      __syncthreads();
      for (int i = c0 + tid; i < cend; i += 256)
        Ls[i - c0] = lse[static_cast<int64_t>(h) * T + lo + i] * kLog2e;
      __syncthreads();
      // query tiles of 32 rows, strided over the 4 waves; the next tile's Q
      // fragments are loaded while this tile's products and exps run. Rows
      // past the sequence are clamped and masked.
      int i0 = c0 + wave * 32;
      u32x4 qn[KK];
      if (i0 < cend) {
#pragma unroll
        for (int kk = 0; kk < KK; ++kk)
          qn[kk] = *reinterpret_cast<const u32x4*>(qh + static_cast<int64_t>(min(i0 + l32, n - 1)) * rs + kk * 16);
      }
      for (; i0 < cend; i0 += 128) {
        bf16x8_t qa[KK];
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) qa[kk] = __builtin_bit_cast(bf16x8_t, qn[kk]);
        const int inext = i0 + 128;
        if (inext < cend) {
#pragma unroll
          for (int kk = 0; kk < KK; ++kk)
            qn[kk] = *reinterpret_cast<const u32x4*>(qh + static_cast<int64_t>(min(inext + l32, n - 1)) * rs + kk * 16);
        }
        // this lane's 16 query rows: i0 + 8 (r/4) + 4 half + r%4, four runs of 4
        float4 lq[4];
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4)
          lq[q4] = *reinterpret_cast<const float4*>(Ls + (i0 - c0) + 8 * q4 + 4 * half);
        // masks matter only where the tile crosses the sequence end or, under
        // the causal mask, reaches keys after some of its queries
        const bool edge = i0 + 32 > cend || (causal && j0 + KB - 1 > i0);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          f32x16_t acc;
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[r] = 0.f;
#pragma unroll
          for (int kk = 0; kk < KK; ++kk)
            acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qa[kk], kf[ks][kk], acc, 0, 0, 0);
          // acc[r]: query i0 + 8 (r/4) + 4 half + r%4, key j0 + 32 ks + l32
          float tsum = 0.f;
          if (!edge) {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
              const float4 l4 = lq[r >> 2];
              const float L = (r & 3) == 0 ? l4.x : (r & 3) == 1 ? l4.y : (r & 3) == 2 ? l4.z : l4.w;
              tsum += __builtin_amdgcn_exp2f(fmaf(acc[r], scale_log2, -L));
            }
          } else {
            const int j = j0 + ks * 32 + l32;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
              const int i = i0 + 8 * (r >> 2) + 4 * half + (r & 3);
              const float4 l4 = lq[r >> 2];
              const float L = (r & 3) == 0 ? l4.x : (r & 3) == 1 ? l4.y : (r & 3) == 2 ? l4.z : l4.w;
              const bool ok = i < cend && (!causal || j <= i);
              tsum += ok ? __builtin_amdgcn_exp2f(fmaf(acc[r], scale_log2, -L)) : 0.f;
            }
          }
          colsum[ks] += tsum;
        }
      }
    }
  }
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) colsum[ks] = half_swap_sum(colsum[ks]);
  if (half == 0) {
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) red[wave][32 * ks + l32] = colsum[ks];
  }
  __syncthreads();
  if (tid < KB) {
    const int j = j0 + tid;
    const float v = ((red[0][tid] + red[1][tid]) + red[2][tid]) + red[3][tid];
    if (j < n) partials[static_cast<int64_t>(g) * T + lo + j] = v;
  }
}

template <typename T, int HD>
__global__ __launch_bounds__(64) void score_valu_kernel(const T* __restrict__ Q,
                                                        const T* __restrict__ K, int64_t rs,
                                                        const float* __restrict__ lse, int H,
                                                        int kv_group, int causal, float scale,
                                                        const int32_t* __restrict__ cu, int Tn,
                                                        int groups, float* __restrict__ partials) {
  __shared__ float Qs[32][HD];
  __shared__ float Ls[32];
  const int b = blockIdx.z, g = blockIdx.y;
  const int lo = cu[b];
  const int n = cu[b + 1] - lo;
  const int jbase = blockIdx.x * 64;
  if (jbase >= n) return;
  const int j = jbase + threadIdx.x;
  float acc = 0.f;
  for (int h = g; h < H; h += groups) {
    float kv[HD];
#pragma unroll
    for (int c = 0; c < HD; ++c)
      kv[c] = j < n ? to_f32(K[static_cast<int64_t>(lo + j) * rs + (h / kv_group) * HD + c]) * scale : 0.f;
    const int qstart = causal ? jbase : 0;
    for (int i0 = qstart; i0 < n; i0 += 32) {
      __syncthreads();
      for (int e = threadIdx.x; e < 32 * HD; e += 64) {
        const int r = e / HD, c = e % HD;
        const int i = i0 + r;
        Qs[r][c] = i < n ? to_f32(Q[static_cast<int64_t>(lo + i) * rs + h * HD + c]) : 0.f;
      }
      if (threadIdx.x < 32) {
        const int i = i0 + threadIdx.x;
        Ls[threadIdx.x] = i < n ? lse[static_cast<int64_t>(h) * Tn + lo + i] : 0.f;
      }
      __syncthreads();
      if (j < n) {
        for (int ii = 0; ii < 32; ++ii) {
          const int i = i0 + ii;
          if (i >= n || (causal && j > i)) continue;
          float sc = 0.f;
#pragma unroll
          for (int c = 0; c < HD; ++c) sc += Qs[ii][c] * kv[c];
          acc += expf(sc - Ls[ii]);
        }
      }
    }
  }
  if (j < n) partials[static_cast<int64_t>(g) * Tn + lo + j] = acc;
}

template <typename T>
hipError_t valu_dispatch(hipStream_t s, const void* q, const void* k, int64_t rs,
                         const float* lse, int H, int kvg, int hd, int causal, float scale, int B,
                         int max_len, int Trows, const int32_t* cu, float* partials,
                         int groups) {
  const dim3 grid((max_len + 63) / 64, groups, B), block(64);
  const T* qp = static_cast<const T*>(q);
  const T* kp = static_cast<const T*>(k);
  switch (hd) {
    case 16: return launch(K_SCORE, score_valu_kernel<T, 16>, grid, block, 0, s, qp, kp, rs, lse, H, kvg, causal, scale, cu, Trows, groups, partials);
    case 32: return launch(K_SCORE, score_valu_kernel<T, 32>, grid, block, 0, s, qp, kp, rs, lse, H, kvg, causal, scale, cu, Trows, groups, partials);
    case 64: return launch(K_SCORE, score_valu_kernel<T, 64>, grid, block, 0, s, qp, kp, rs, lse, H, kvg, causal, scale, cu, Trows, groups, partials);
    case 128: return launch(K_SCORE, score_valu_kernel<T, 128>, grid, block, 0, s, qp, kp, rs, lse, H, kvg, causal, scale, cu, Trows, groups, partials);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

// Head groups: the smallest divisor G of H that gives the grid at least
// ~1024 workgroups (H when none does); the MFMA path only.
int score_groups(int dtype, int H, int hd, int T) {
  if (!(dtype == 1 && (hd == 64 || hd == 128))) return 1;
  const int kblocks = (T + kScoreKeys - 1) / kScoreKeys;
  for (int g = 1; g <= H; ++g)
    if (H % g == 0 && kblocks * g >= 1024) return g;
  return H;
}

hipError_t launch_score(hipStream_t s, int dtype, const void* q, const void* k,
                        int64_t row_stride, const float* lse, int H, int kv_group, int hd, int causal,
                        float scale, int B, int max_len, int T, const int32_t* cu_dev,
                        float* partials, int groups) {
  if (B == 0 || max_len == 0) return hipSuccess;
  if (dtype == 1 && (hd == 64 || hd == 128)) {
    const dim3 grid((max_len + kScoreKeys - 1) / kScoreKeys, groups, B), block(256);
    const bf16_t* qp = static_cast<const bf16_t*>(q);
    const bf16_t* kp = static_cast<const bf16_t*>(k);
    const float sl = scale * kLog2e;
    if (hd == 64)
      return launch(K_SCORE, score_mfma_kernel<64, kScoreKeys>, grid, block, 0, s, qp, kp, row_stride,
                    lse, H, kv_group, causal, sl, cu_dev, T, groups, partials);
    return launch(K_SCORE, score_mfma_kernel<128, kScoreKeys>, grid, block, 0, s, qp, kp, row_stride,
                  lse, H, kv_group, causal, sl, cu_dev, T, groups, partials);
  }
  if (dtype == 1)
    return valu_dispatch<bf16_t>(s, q, k, row_stride, lse, H, kv_group, hd, causal, scale, B,
                                 max_len, T, cu_dev, partials, groups);
  return valu_dispatch<float>(s, q, k, row_stride, lse, H, kv_group, hd, causal, scale, B, max_len,
                              T, cu_dev, partials, groups);
}

}  // namespace zsa
