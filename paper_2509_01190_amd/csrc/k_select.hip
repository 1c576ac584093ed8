// Per-sequence top-k of the contribution scores (keep the k highest, ties to
// the lower row, output in ascending row order; optionally the last row of
// every sequence is always kept and the other k - 1 are chosen by score).
//
// One 1024-thread workgroup (16 waves) per sequence. The score of a row is
// first finalised as the fixed-order sum of the per-head-group partial sums
// (deterministic), then mapped to an order-preserving 32-bit key and held in
// LDS (up to 16384 rows; longer sequences re-read the partials).
// The k-th largest key is found by an MSB-first radix select (4 passes of
// 8-bit digits over a 256-bin LDS histogram; one wave scans the histogram
// with a 64-lane prefix sum). Rows above the threshold key are kept, plus
// the first (k - #above) rows equal to it in row order; a stable block-wide
// ballot/popcount prefix sum writes them in ascending order, so no sort is
// needed.
#include "zsa_internal.h"

namespace zsa {
namespace {

constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / 64;
constexpr int kSelLdsCap = 16384;

// order-preserving map float -> uint32 (-0 folded onto +0)
__device__ __forceinline__ uint32_t order_key(float s) {
  uint32_t u = __float_as_uint(s);
  if (u == 0x80000000u) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float finalise(const float* __restrict__ partials, int groups, int T,
                                          int row) {
  float s = 0.f;
  for (int g = 0; g < groups; ++g) s += partials[static_cast<int64_t>(g) * T + row];
  return s;
}

__global__ __launch_bounds__(kSelThreads) void select_kernel(
    const float* __restrict__ partials, int groups, int T, const int32_t* __restrict__ cu_in,
    const int32_t* __restrict__ cu_out, int32_t* __restrict__ kept,
    float* __restrict__ scores_out, int lds_cap, int keep_last) {
  extern __shared__ uint32_t keys[];
  __shared__ uint32_t hist[256];
  __shared__ uint32_t wave_cnt[kSelWaves];
  __shared__ uint32_t sh_digit, sh_krem;

  const int b = blockIdx.x;
  const int lo = cu_in[b];
  const int n = cu_in[b + 1] - lo;
  const int out0 = cu_out[b];
  const int k = cu_out[b + 1] - out0;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const bool staged = n <= lds_cap;

  // with keep_last the sequence's last row takes the largest key, above
  // every finite or infinite score, so it is always among the k kept
  for (int i = tid; i < n; i += kSelThreads) {
    const float s = finalise(partials, groups, T, lo + i);
    if (scores_out != nullptr) scores_out[lo + i] = s;
    if (staged) keys[i] = (keep_last && i == n - 1) ? 0xffffffffu : order_key(s);
  }
  if (k <= 0 || n <= 0) return;
  if (k >= n) {
    for (int i = tid; i < n; i += kSelThreads) kept[out0 + i] = lo + i;
    return;
  }
  __syncthreads();

  auto key_at = [&](int i) -> uint32_t {
    if (staged) return keys[i];
    return (keep_last && i == n - 1) ? 0xffffffffu : order_key(finalise(partials, groups, T, lo + i));
  };

  uint32_t prefix = 0u;
  uint32_t krem = static_cast<uint32_t>(k);
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    const uint32_t hi_mask = pass == 0 ? 0u : (0xffffffffu << (shift + 8));
    if (tid < 256) hist[tid] = 0u;
    __syncthreads();
    for (int i = tid; i < n; i += kSelThreads) {
      const uint32_t key = key_at(i);
      if (((key ^ prefix) & hi_mask) == 0u) atomicAdd(&hist[(key >> shift) & 255u], 1u);
    }
    __syncthreads();
    if (wave == 0) {
      // lane l owns digits 255-4l, 254-4l, 253-4l, 252-4l (descending)
      uint32_t c[4];
      uint32_t lsum = 0u;
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        c[t] = hist[255 - 4 * lane - t];
        lsum += c[t];
      }
      uint32_t incl = lsum;
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        const uint32_t v = __shfl_up(incl, off, 64);
        if (lane >= off) incl += v;
      }
      const uint32_t excl = incl - lsum;
      if (excl < krem && krem <= incl) {  // exactly one lane
        uint32_t acc = excl;
        bool done = false;
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          if (!done && acc + c[t] >= krem) {
            sh_digit = static_cast<uint32_t>(255 - 4 * lane - t);
            sh_krem = krem - acc;
            done = true;
          }
          acc += c[t];
        }
      }
    }
    __syncthreads();
    prefix |= sh_digit << shift;
    krem = sh_krem;
    __syncthreads();
  }
  const uint32_t thresh = prefix;

  const uint64_t lt_mask = (1ull << lane) - 1ull;
  uint32_t run_eq = 0u, run_sel = 0u;
  for (int base = 0; base < n; base += kSelThreads) {
    const int i = base + tid;
    const bool valid = i < n;
    const uint32_t key = valid ? key_at(i) : 0u;
    const bool eq = valid && key == thresh;
    const bool gt = valid && key > thresh;

    const uint64_t m_eq = __ballot(eq);
    if (lane == 0) wave_cnt[wave] = static_cast<uint32_t>(__popcll(m_eq));
    __syncthreads();
    uint32_t woff = 0u, tot = 0u;
#pragma unroll
    for (int w = 0; w < kSelWaves; ++w) {
      const uint32_t c = wave_cnt[w];
      woff += w < wave ? c : 0u;
      tot += c;
    }
    const uint32_t eq_rank = run_eq + woff + static_cast<uint32_t>(__popcll(m_eq & lt_mask));
    run_eq += tot;
    const bool sel = gt || (eq && eq_rank < krem);
    __syncthreads();

    const uint64_t m_sel = __ballot(sel);
    if (lane == 0) wave_cnt[wave] = static_cast<uint32_t>(__popcll(m_sel));
    __syncthreads();
    woff = 0u;
    tot = 0u;
#pragma unroll
    for (int w = 0; w < kSelWaves; ++w) {
      const uint32_t c = wave_cnt[w];
      woff += w < wave ? c : 0u;
      tot += c;
    }
    const uint32_t slot = run_sel + woff + static_cast<uint32_t>(__popcll(m_sel & lt_mask));
    if (sel && slot < static_cast<uint32_t>(k)) kept[out0 + slot] = lo + i;
    run_sel += tot;
    __syncthreads();
  }
}

__global__ void finalize_kernel(const float* __restrict__ partials, int groups, int T,
                                float* __restrict__ scores) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < T) scores[i] = finalise(partials, groups, T, i);
}

}  // namespace

hipError_t launch_select(hipStream_t s, const float* partials, int groups, int T, int B,
                         int max_len, const int32_t* cu_in_dev, const int32_t* cu_out_dev,
                         int32_t* kept_rows, float* scores_out, int keep_last) {
  if (B == 0) return hipSuccess;
  const int cap = max_len < kSelLdsCap ? max_len : kSelLdsCap;
  const size_t shmem = static_cast<size_t>(cap > 0 ? cap : 1) * sizeof(uint32_t);
  return launch(K_SELECT, select_kernel, dim3(B), dim3(kSelThreads), shmem, s, partials, groups,
                T, cu_in_dev, cu_out_dev, kept_rows, scores_out, cap, keep_last);
}

hipError_t launch_score_finalize(hipStream_t s, const float* partials, int groups, int T,
                                 float* scores) {
  if (T == 0) return hipSuccess;
  return launch(K_SCORE, finalize_kernel, dim3((T + 255) / 256), dim3(256), 0, s, partials,
                groups, T, scores);
}

}  // namespace zsa
