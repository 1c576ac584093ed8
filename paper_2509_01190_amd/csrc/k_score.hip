// Contribution score of every row at a pruning layer: the column sums of
// the normalised soft-score matrices, summed over heads,
//     s[j] = sum_h sum_i exp(q_i . k_j * scale - lse_h[i]),
// over the rows i the mask lets see row j. The normalised probability needs
// each query row's final log-sum-exp, which the attention pass has already
// written, so this is a second sweep over Q K^T that never stores P.
//
// bf16, head_dim 64/128 (MFMA): one workgroup of 8 waves per (key block of
// KB = 128 or 256 keys, query head, sequence). Its K tile is staged in
// LDS; the waves stride over 32-query tiles, keep the tile's Q fragments in
// registers and compute S = Q K^T with v_mfma_f32_32x32x16_bf16 in the
// *non*-transposed layout, where a lane owns one key column and 16 query
// rows, so the column sum is in-lane adds. Every workgroup reads the query
// rows of its head once, so the bytes moved per score fall as the key block
// grows; the block is the wider one that still gives the grid two
// workgroups per CU. Lane halves
// and waves are combined in a fixed order and the workgroup writes one
// partial vector per head ([H][T]); the top-k kernel adds the H partials in
// a fixed order. No atomics: the result is bitwise reproducible. Causal
// workgroups start at the first query that can see their keys and skip the
// 32-key columns no query of a tile can see.
//
// fp32 / other head dims: one thread per key, vector ALU.
#include <math.h>

#include "zsa_internal.h"

namespace zsa {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr int kScoreWaves = 8;

template <int HD, int KB>
__global__ __launch_bounds__(64 * kScoreWaves) __attribute__((amdgpu_waves_per_eu(HD == 64 ? 4 : 2))) void score_mfma_kernel(
    const bf16_t* __restrict__ Q, const bf16_t* __restrict__ K, int64_t rs,
    const float* __restrict__ lse, int H, int kv_group, int causal, float scale_log2,
    const int32_t* __restrict__ cu, int T, float* __restrict__ partials) {
  constexpr int NW = kScoreWaves, NT = 64 * NW;
  constexpr int KLD = HD + 8;  // K tile row stride (bf16): conflict-free fragment reads
  constexpr int KK = HD / 16;
  constexpr int KS = KB / 32;  // 32-key columns
  constexpr int LPR = HD / 8;   // lanes per 16-byte-chunked Q row
  constexpr int RPI = 64 / LPR;  // Q rows per load
  constexpr int NQI = 32 / RPI;  // loads per 32-row tile
  static_assert(KB * KLD * 2 >= NW * KB * 4, "the reduction fits the K tile");
  __shared__ __align__(16) unsigned char smem[KB * KLD * 2];
  __shared__ __align__(16) unsigned char qbuf[NW][32 * HD * 2];  // each wave's Q tile
  bf16_t* Ks = reinterpret_cast<bf16_t*>(smem);

  const int b = blockIdx.z, h = blockIdx.y;
  const int lo = cu[b];
  const int n = cu[b + 1] - lo;
  const int j0 = blockIdx.x * KB;
  if (j0 >= n) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int hf = lane >> 5, l32 = lane & 31;

  for (int c = tid; c < KB * HD / 8; c += NT) {
    const int r = c / (HD / 8), ch = (c % (HD / 8)) * 8;
    // keys past the sequence repeat the last row; their columns are not written
    *reinterpret_cast<uint4*>(Ks + r * KLD + ch) =
        *reinterpret_cast<const uint4*>(K + static_cast<int64_t>(lo + min(j0 + r, n - 1)) * rs +
                                        (h / kv_group) * HD + ch);
  }
  __syncthreads();

  float colsum[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) colsum[ks] = 0.f;
  // this head's log-sum-exp of the sequence's rows, in exp2 units; rows past
  // the sequence read as zeros (their scores are masked)
  const __amdgpu_buffer_rsrc_t lres = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<float*>(lse + static_cast<int64_t>(h) * T + lo), 0, static_cast<uint32_t>(n) * 4u,
      0x00020000);
  // Query tiles of 32 rows, strided over the waves; the next tile's Q is
  // loaded while this tile's products and exps run. Rows past the sequence
  // are clamped and masked. The loads cover whole cache lines (HD / 8 lanes
  // per row); the wave passes each tile through its LDS buffer (chunk c of
  // row r at r * 2 HD + (c ^ (r % 8)) * 16) into the MFMA fragments (lane
  // l: row l % 32, chunk 2 kk + l / 32). Fragments loaded straight from
  // memory would touch 32 lines per load, a quarter of each.
  const bf16_t* qh = Q + static_cast<int64_t>(lo) * rs + h * HD + (lane % LPR) * 8;
  unsigned char* const qw = qbuf[wave];
  int i0 = (causal ? (j0 & ~31) : 0) + wave * 32;
  u32x4 qn[NQI];
  if (i0 < n) {
#pragma unroll
    for (int i = 0; i < NQI; ++i)
      qn[i] = *reinterpret_cast<const u32x4*>(qh + static_cast<int64_t>(min(i0 + RPI * i + lane / LPR, n - 1)) * rs);
  }
  for (; i0 < n; i0 += 32 * NW) {
    // LDS operations of a wave run in order: these stores follow the last
    // tile's fragment reads
#pragma unroll
    for (int i = 0; i < NQI; ++i) {
      const int r = RPI * i + lane / LPR;
      *reinterpret_cast<u32x4*>(qw + r * (HD * 2) + (((lane % LPR) ^ (r & 7)) << 4)) = qn[i];
    }
    bf16x8_t qa[KK];
#pragma unroll
    for (int kk = 0; kk < KK; ++kk)
      qa[kk] = __builtin_bit_cast(
          bf16x8_t, *reinterpret_cast<const u32x4*>(qw + l32 * (HD * 2) + (((2 * kk + hf) ^ (l32 & 7)) << 4)));
    const int inext = i0 + 32 * NW;
    if (inext < n) {
#pragma unroll
      for (int i = 0; i < NQI; ++i)
        qn[i] = *reinterpret_cast<const u32x4*>(qh + static_cast<int64_t>(min(inext + RPI * i + lane / LPR, n - 1)) * rs);
    }
    // this lane's 16 query rows: i0 + 8 (r/4) + 4 hf + r%4
    float L[16];
#pragma unroll
    for (int r = 0; r < 16; ++r)
      L[r] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                                           lres, static_cast<uint32_t>(i0 + 8 * (r >> 2) + 4 * hf + (r & 3)) * 4u, 0, 0)) *
             kLog2e;
    // S for the tile and key column ks: acc[r] = query i0 + 8 (r/4) + 4 hf + r%4,
    // key j0 + 32 ks + l32
    auto block = [&](int ks) {
      f32x16_t acc;
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[r] = 0.f;
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) {
        const bf16x8_t kf = __builtin_bit_cast(
            bf16x8_t, *reinterpret_cast<const u32x4*>(Ks + (ks * 32 + l32) * KLD + kk * 16 + hf * 8));
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qa[kk], kf, acc, 0, 0, 0);
      }
      return acc;
    };
    if (i0 + 32 <= n && (!causal || i0 >= j0 + KB)) {
      // every query of the tile sees every key of the block: no masks, and
      // column ks + 1's products are issued before column ks's exps
      f32x16_t a0 = block(0);
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        f32x16_t a1;
        if (ks + 1 < KS) a1 = block(ks + 1);
        float tsum = 0.f;
#pragma unroll
        for (int r = 0; r < 16; ++r) tsum += __builtin_amdgcn_exp2f(fmaf(a0[r], scale_log2, -L[r]));
        colsum[ks] += tsum;
        if (ks + 1 < KS) a0 = a1;
      }
    } else {
      // the tile crosses the sequence end or the diagonal
      const bool tail = i0 + 32 > n;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        // under the causal mask no query of the tile sees this or any later
        // column once its first key is past the tile's last query
        if (causal && j0 + 32 * ks > i0 + 31) break;
        const f32x16_t acc = block(ks);
        float tsum = 0.f;
        if (!tail && (!causal || j0 + 32 * ks + 31 <= i0)) {
#pragma unroll
          for (int r = 0; r < 16; ++r) tsum += __builtin_amdgcn_exp2f(fmaf(acc[r], scale_log2, -L[r]));
        } else {
          const int j = j0 + ks * 32 + l32;
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int i = i0 + 8 * (r >> 2) + 4 * hf + (r & 3);
            const bool ok = i < n && (!causal || j <= i);
            tsum += ok ? __builtin_amdgcn_exp2f(fmaf(acc[r], scale_log2, -L[r])) : 0.f;
          }
        }
        colsum[ks] += tsum;
      }
    }
  }
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) colsum[ks] = half_swap_sum(colsum[ks]);
  __syncthreads();  // every wave is done with the K tile
  float* red = reinterpret_cast<float*>(smem);  // [NW][KB]
  if (hf == 0) {
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) red[wave * KB + 32 * ks + l32] = colsum[ks];
  }
  __syncthreads();
  for (int c = tid; c < KB; c += NT) {
    const int j = j0 + c;
    float v = red[c];
#pragma unroll
    for (int w = 1; w < NW; ++w) v += red[w * KB + c];
    if (j < n) partials[static_cast<int64_t>(h) * T + lo + j] = v;
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

// Partial vectors per row: one per query head on the MFMA path.
int score_groups(int dtype, int H, int hd, int T) {
  (void)T;
  return dtype == 1 && (hd == 64 || hd == 128) ? H : 1;
}

hipError_t launch_score(hipStream_t s, int dtype, const void* q, const void* k,
                        int64_t row_stride, const float* lse, int H, int kv_group, int hd, int causal,
                        float scale, int B, int max_len, int T, const int32_t* cu_dev,
                        float* partials, int groups) {
  if (B == 0 || max_len == 0) return hipSuccess;
  if (dtype == 1 && (hd == 64 || hd == 128)) {
    if (groups != H) return hipErrorInvalidValue;
    const bf16_t* qp = static_cast<const bf16_t*>(q);
    const bf16_t* kp = static_cast<const bf16_t*>(k);
    const float sl = scale * kLog2e;
    // 256-key blocks where the grid still holds two workgroups per CU, else
    // 128 (measured, us, 8 x 2048 causal rows, 32 heads, hd 64: 128-key
    // blocks 104.5, 256 94.0, 512 105.9 (its 16 column sums and query
    // fragments spill at four waves per SIMD); 4 x 4096 rows, hd 128: 395
    // at 128 keys, 305 at 256)
    const long slots = 2L * device_cu_count();
    auto wgs = [&](int kb) { return static_cast<long>((max_len + kb - 1) / kb) * H * B; };
    const int kb = wgs(256) >= slots ? 256 : 128;
    const dim3 block(64 * kScoreWaves);
    const dim3 grid((max_len + kb - 1) / kb, H, B);
#define ZSA_SCORE(HD_, KB_)                                                                      \
  return launch(K_SCORE, score_mfma_kernel<HD_, KB_>, grid, block, 0, s, qp, kp, row_stride, lse, H, \
                kv_group, causal, sl, cu_dev, T, partials)
    if (hd == 64) {
      if (kb == 256) ZSA_SCORE(64, 256);
      ZSA_SCORE(64, 128);
    }
    if (kb == 256) ZSA_SCORE(128, 256);
    ZSA_SCORE(128, 128);
#undef ZSA_SCORE
  }
  if (dtype == 1)
    return valu_dispatch<bf16_t>(s, q, k, row_stride, lse, H, kv_group, hd, causal, scale, B,
                                 max_len, T, cu_dev, partials, groups);
  return valu_dispatch<float>(s, q, k, row_stride, lse, H, kv_group, hd, causal, scale, B, max_len,
                              T, cu_dev, partials, groups);
}

}  // namespace zsa
