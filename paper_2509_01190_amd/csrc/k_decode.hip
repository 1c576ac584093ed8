// Generation after a pruned prefill: the key/value cache and the attention
// of one new row per sequence over it.
//
// Cache layout: [layer][batch][capacity][k | v], kvd = kv_heads * head_dim
// elements each for k and v (k after the rotary embedding), storage dtype.
// A layer's cache holds the rows that entered that layer in the prefill
// (fewer after every pruning point) followed by the generated rows.
//
// kv_store: copies the k | v columns of the fused projection output into the
// cache (prefill: every row of a layer). 16-byte chunks, coalesced.
//
// decode_attn: one new query row per sequence over its len cached rows (its
// own k / v appended first), split over the cache; decode_combine merges
// the splits. The work is HBM-bound on the cache rows: 2 * kvd * size bytes
// per cached row and layer.
#include <math.h>

#include <algorithm>

#include "zsa_internal.h"

namespace zsa {
namespace {

constexpr float kLog2e = 1.4426950408889634f;

__global__ __launch_bounds__(256) void kv_store_kernel(
    const uint4* __restrict__ src, int64_t src_stride, int src_col, int cpr,
    const int32_t* __restrict__ cu, const int32_t* __restrict__ start, uint4* __restrict__ cache,
    int cap, int rows_per_block) {
  const int b = blockIdx.y;
  const int lo = cu[b];
  const int n = cu[b + 1] - lo;
  const int st = start != nullptr ? start[b] : 0;
  const int r0 = blockIdx.x * rows_per_block;
  for (int i = threadIdx.x; i < rows_per_block * cpr; i += blockDim.x) {
    const int r = r0 + i / cpr, c = i % cpr;
    if (r >= n) break;
    cache[(static_cast<int64_t>(b) * cap + st + r) * cpr + c] =
        src[static_cast<int64_t>(lo + r) * src_stride + src_col + c];
  }
}

// decode_attn: grid (split, key/value head g, sequence b); a workgroup of
// kDecWaves waves takes `rounds` blocks of kDecRows consecutive cache rows,
// kDecRowsW rows per wave per block, for all G query heads that read head g
// (grouped-query attention reads each cache row once per group).
//  * scores: v_mfma_f32_16x16x32_bf16 with A = the G query rows (lane l:
//    head l % 16, zero past G) and B = 16 cache rows of K (lane l: row
//    l % 16), so lane l gets the scores of cache row l % 16 for heads
//    4 (l / 16) .. + 3; K goes from memory straight into the operands.
//  * online softmax per wave (running max per head, rescaled sums);
//    probabilities go through a per-wave LDS strip [kDecRowsW rows][G];
//  * P V on the vector ALU: each lane holds 16 bytes (8 columns) of V rows
//    in registers, loaded row-contiguously together with K;
//  * the waves' (max, sum, o) merge in wave order into the split's partial.
// decode_combine then merges the splits of each (sequence, head group) in
// split order (fixed, so the result is reproducible).
// The new row's k / v (head g) are copied into cache row len - 1 by the
// workgroup whose rows include it, before that workgroup reads the cache.
constexpr int kDecWaves = 4;                     // waves per workgroup
constexpr int kDecRowsW = 32;                    // cache rows per wave and block
constexpr int kDecTiles = kDecRowsW / 16;         // 16-row score tiles per wave
constexpr int kDecRows = kDecWaves * kDecRowsW;  // cache rows per workgroup and block

typedef __bf16 dec_bf16x8_t __attribute__((ext_vector_type(8)));
typedef float dec_f32x4_t __attribute__((ext_vector_type(4)));

// qkv: the projection rows [B, q_stride] (query head h at columns h*HD, the
// new row's k at kv_col, its v at kv_col + kvd); cache of this layer
// [B][cap][2 kvd]; len [B] rows attended, the new one included. Partials:
// m, l [B][H][S], o [B][H][S][HD].
template <int HD, int G>
__global__ __launch_bounds__(kDecWaves * 64) void decode_attn_kernel(
    const bf16_t* __restrict__ qkv, int64_t q_stride, int kv_col, bf16_t* __restrict__ cache,
    int cap, int kvd, const int32_t* __restrict__ len, int H, float scale_log2, int S, int rounds,
    float* __restrict__ m_part, float* __restrict__ l_part, float* __restrict__ o_part) {
  constexpr int KS = HD / 32;             // 32-wide K steps of a score tile
  constexpr int LPR = HD / 8;             // lanes per V row (16 bytes each)
  constexpr int RPI = 64 / LPR;           // V rows per load instruction
  constexpr int NVI = kDecRowsW / RPI;    // V loads per lane and block
  __shared__ float ps[kDecWaves][kDecRowsW * G];
  __shared__ float wm[kDecWaves][G], wl[kDecWaves][G];
  __shared__ __align__(16) float wo[kDecWaves][G * HD];
  const int s = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int l16 = lane & 15, kg = lane >> 4;
  const int n = len[b];
  const int row0 = s * rounds * kDecRows;
  const int row_end = min(n, row0 + rounds * kDecRows);
  const int rowe = 2 * kvd;  // cache row, elements
  bf16_t* seq = cache + static_cast<int64_t>(b) * cap * rowe;
  const bf16_t* qrow = qkv + static_cast<int64_t>(b) * q_stride;
  const int hbase = g * G;
  if (n - 1 >= row0 && n - 1 < row_end) {  // uniform over the workgroup
    if (tid < 2 * LPR) {
      const int kv = tid / LPR, c = (tid % LPR) * 8;  // kv 0: k, 1: v
      *reinterpret_cast<uint4*>(seq + static_cast<int64_t>(n - 1) * rowe + kv * kvd + g * HD + c) =
          *reinterpret_cast<const uint4*>(qrow + kv_col + kv * kvd + g * HD + c);
    }
    __syncthreads();
  }
  dec_bf16x8_t qf[KS];
#pragma unroll
  for (int j = 0; j < KS; ++j) {
    uint4 v = make_uint4(0u, 0u, 0u, 0u);
    if (l16 < G) v = *reinterpret_cast<const uint4*>(qrow + (hbase + l16) * HD + 32 * j + 8 * kg);
    qf[j] = __builtin_bit_cast(dec_bf16x8_t, v);
  }
  // cache rows past len read as zeros (their scores are masked)
  const uint32_t rowb = static_cast<uint32_t>(rowe) * 2u;
  const __amdgpu_buffer_rsrc_t res =
      __builtin_amdgcn_make_buffer_rsrc(seq, 0, static_cast<uint32_t>(n) * rowb, 0x00020000);
  const uint32_t koff = l16 * rowb + static_cast<uint32_t>(g * HD + 8 * kg) * 2u;
  const int vr = lane / LPR, vc = lane % LPR;
  const uint32_t voff = vr * rowb + static_cast<uint32_t>(kvd + g * HD + 8 * vc) * 2u;
  float m_run[4], l_run[4];  // heads 4 kg + r of this lane's 16-lane group
  float o[G][8];             // every head, this lane's 8 V columns
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    m_run[r] = -INFINITY;
    l_run[r] = 0.f;
  }
#pragma unroll
  for (int h = 0; h < G; ++h)
#pragma unroll
    for (int e = 0; e < 8; ++e) o[h][e] = 0.f;
  float* pw = ps[wave];
  for (int rd = 0; rd < rounds; ++rd) {
    const int r0 = row0 + rd * kDecRows + wave * kDecRowsW;
    if (r0 >= row_end) break;
    u32x4 kr[kDecTiles][KS], vreg[NVI];
#pragma unroll
    for (int i = 0; i < kDecTiles; ++i)
#pragma unroll
      for (int j = 0; j < KS; ++j)
        kr[i][j] = __builtin_bit_cast(
            u32x4, __builtin_amdgcn_raw_buffer_load_b128(res, koff + (r0 + 16 * i) * rowb + 64u * j, 0, 0));
#pragma unroll
    for (int jj = 0; jj < NVI; ++jj)
      vreg[jj] = __builtin_bit_cast(
          u32x4, __builtin_amdgcn_raw_buffer_load_b128(res, voff + (r0 + RPI * jj) * rowb, 0, 0));
    __builtin_amdgcn_sched_barrier(0);
    dec_f32x4_t sc[kDecTiles];
#pragma unroll
    for (int i = 0; i < kDecTiles; ++i) {
      sc[i] = dec_f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int j = 0; j < KS; ++j)
        sc[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
            qf[j], __builtin_bit_cast(dec_bf16x8_t, kr[i][j]), sc[i], 0, 0, 0);
    }
    float alpha[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      float mx = -INFINITY;
#pragma unroll
      for (int i = 0; i < kDecTiles; ++i) {
        const float v = r0 + 16 * i + l16 < n ? sc[i][r] * scale_log2 : -INFINITY;
        sc[i][r] = v;
        mx = fmaxf(mx, v);
      }
#pragma unroll
      for (int off = 1; off < 16; off <<= 1) mx = fmaxf(mx, __shfl_xor(mx, off, 64));
      const float mnew = fmaxf(m_run[r], mx);  // finite: row r0 is below len
      alpha[r] = __builtin_amdgcn_exp2f(m_run[r] - mnew);
      m_run[r] = mnew;
      float ls = 0.f;
#pragma unroll
      for (int i = 0; i < kDecTiles; ++i) {
        const float p = __builtin_amdgcn_exp2f(sc[i][r] - mnew);
        ls += p;
        if (4 * kg + r < G) pw[(16 * i + l16) * G + 4 * kg + r] = p;
      }
      l_run[r] = l_run[r] * alpha[r] + ls;
    }
    if (rd > 0) {
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const float a = __builtin_bit_cast(
            float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, alpha[h % 4]), 16 * (h / 4)));
#pragma unroll
        for (int e = 0; e < 8; ++e) o[h][e] *= a;
      }
    }
#pragma unroll
    for (int jj = 0; jj < NVI; ++jj) {
      const float* prow = pw + (RPI * jj + vr) * G;
      float vf[8];
      unpack16(make_uint4(vreg[jj][0], vreg[jj][1], vreg[jj][2], vreg[jj][3]), vf, bf16_t());
#pragma unroll
      for (int h = 0; h < G; ++h) {
        const float p = prow[h];
#pragma unroll
        for (int e = 0; e < 8; ++e) o[h][e] = fmaf(p, vf[e], o[h][e]);
      }
    }
  }
  // the wave's sums: l over its 16-lane group, o over the lanes that hold
  // the same V columns
#pragma unroll
  for (int r = 0; r < 4; ++r)
#pragma unroll
    for (int off = 1; off < 16; off <<= 1) l_run[r] += __shfl_xor(l_run[r], off, 64);
#pragma unroll
  for (int h = 0; h < G; ++h)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
#pragma unroll
      for (int off = LPR; off < 32; off <<= 1) o[h][e] += __shfl_xor(o[h][e], off, 64);
      o[h][e] = half_swap_sum(o[h][e]);
    }
  if (lane < LPR) {
#pragma unroll
    for (int h = 0; h < G; ++h)
#pragma unroll
      for (int e = 0; e < 8; ++e) wo[wave][h * HD + 8 * lane + e] = o[h][e];
  }
  if (l16 == 0) {
#pragma unroll
    for (int r = 0; r < 4; ++r)
      if (4 * kg + r < G) {
        wm[wave][4 * kg + r] = m_run[r];
        wl[wave][4 * kg + r] = l_run[r];
      }
  }
  __syncthreads();
  const int64_t pbase = (static_cast<int64_t>(b) * H + hbase) * S + s;  // head h adds h * S
  for (int it = tid; it < G * HD; it += kDecWaves * 64) {
    const int h = it / HD, c = it % HD;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < kDecWaves; ++w) M = fmaxf(M, wm[w][h]);
    float L = 0.f, Ov = 0.f;
    if (M != -INFINITY) {
#pragma unroll
      for (int w = 0; w < kDecWaves; ++w) {
        const float f = __builtin_amdgcn_exp2f(wm[w][h] - M);
        L = fmaf(wl[w][h], f, L);
        Ov = fmaf(wo[w][h * HD + c], f, Ov);
      }
    }
    if (c == 0) {
      m_part[pbase + static_cast<int64_t>(h) * S] = M;
      l_part[pbase + static_cast<int64_t>(h) * S] = L;
    }
    o_part[(pbase + static_cast<int64_t>(h) * S) * HD + c] = Ov;
  }
}

// grid (query head h, sequence b), one thread per channel: the S (at most
// kDecMaxSplits) split partials of (b, h) merged in split order, loaded 16
// at a time; splits without rows hold (-inf, 0, 0) and weigh 0
constexpr int kDecMaxSplits = 64;

template <int HD>
__global__ __launch_bounds__(HD) void decode_combine_kernel(
    const float* __restrict__ m_part, const float* __restrict__ l_part,
    const float* __restrict__ o_part, int S, int H, bf16_t* __restrict__ out, int64_t out_stride) {
  constexpr int U = 16;
  const int h = blockIdx.x, b = blockIdx.y, c = threadIdx.x;
  const int64_t hb = (static_cast<int64_t>(b) * H + h) * S;
  float M = -INFINITY;
  for (int y0 = 0; y0 < S; y0 += U) {
    float mv[U];
#pragma unroll
    for (int u = 0; u < U; ++u) mv[u] = y0 + u < S ? m_part[hb + y0 + u] : -INFINITY;
#pragma unroll
    for (int u = 0; u < U; ++u) M = fmaxf(M, mv[u]);
  }
  float L = 0.f, Ov = 0.f;
  for (int y0 = 0; y0 < S; y0 += U) {
    float mv[U], lv[U], ov[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      mv[u] = -INFINITY;
      lv[u] = 0.f;
      ov[u] = 0.f;
      if (y0 + u < S) {
        mv[u] = m_part[hb + y0 + u];
        lv[u] = l_part[hb + y0 + u];
        ov[u] = o_part[(hb + y0 + u) * HD + c];
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const float f = __builtin_amdgcn_exp2f(mv[u] - M);
      L = fmaf(lv[u], f, L);
      Ov = fmaf(ov[u], f, Ov);
    }
  }
  out[static_cast<int64_t>(b) * out_stride + h * HD + c] = f32_to_bf16(Ov / L);
}

template <int HD, int G>
hipError_t launch_dec(hipStream_t s, const bf16_t* qkv, int64_t q_stride, int kv_col,
                      bf16_t* cache, int cap, int kvd, const int32_t* len, int B, int H, int Hkv,
                      float sl, int S, int rounds, float* m, float* l, float* o, bf16_t* out,
                      int64_t out_stride) {
  hipError_t e = launch(K_ATTENTION, decode_attn_kernel<HD, G>, dim3(S, Hkv, B),
                        dim3(kDecWaves * 64), 0, s, qkv, q_stride, kv_col, cache, cap, kvd, len, H,
                        sl, S, rounds, m, l, o);
  if (e != hipSuccess) return e;
  return launch(K_ATTENTION, decode_combine_kernel<HD>, dim3(H, B), dim3(HD), 0, s, m, l, o, S, H,
                out, out_stride);
}

// Blocks of kDecRows rows per workgroup: one block per split up to
// kDecMaxSplits splits, fewer when the batch's (sequence, head group) pairs
// alone give about eight workgroups per CU; longer caches take several
// blocks per workgroup.
void decode_plan(int max_len, int B, int Hkv, int* S, int* rounds) {
  const int blocks = (max_len + kDecRows - 1) / kDecRows;
  const int pairs = B * Hkv;
  const int want = std::max(
      1, std::min({blocks, kDecMaxSplits, (8 * device_cu_count() + pairs - 1) / pairs}));
  *rounds = (blocks + want - 1) / want;
  *S = (blocks + *rounds - 1) / *rounds;
}

}  // namespace

int decode_splits_bound(int cap) { return std::min((cap + kDecRows - 1) / kDecRows, kDecMaxSplits); }

bool decode_supported(int dtype, int hd, int group) {
  return dtype == 1 && (hd == 64 || hd == 128) &&
         (group == 1 || group == 2 || group == 4 || group == 8);
}

hipError_t launch_kv_store(hipStream_t s, int dtype, const void* src, int64_t src_stride,
                           int src_col, int kvd, int B, int max_rows, const int32_t* cu_dev,
                           const int32_t* start_dev, void* cache_layer, int cap) {
  if (B == 0 || max_rows == 0) return hipSuccess;
  const int esz = dtype == 1 ? 2 : 4;
  const int cpr = 2 * kvd * esz / 16;
  const int rpb = cpr >= 256 ? 1 : 256 / cpr;
  const dim3 grid((max_rows + rpb - 1) / rpb, B);
  return launch(K_MISC, kv_store_kernel, grid, dim3(256), 0, s, static_cast<const uint4*>(src),
                src_stride * esz / 16, src_col * esz / 16, cpr, cu_dev, start_dev,
                static_cast<uint4*>(cache_layer), cap, rpb);
}

hipError_t launch_decode_attention(hipStream_t s, const void* qkv, int64_t q_stride, int kv_col,
                                   void* cache_layer, int cap, int hd, int H, int Hkv,
                                   const int32_t* len_dev, int B, int max_len, float scale,
                                   float* m_part, float* l_part, float* o_part, void* out,
                                   int64_t out_stride) {
  if (B == 0) return hipSuccess;
  const int kvd = Hkv * hd, group = H / Hkv;
  const float sl = scale * kLog2e;
  int S, rounds;
  decode_plan(max_len, B, Hkv, &S, &rounds);
  const bf16_t* qp = static_cast<const bf16_t*>(qkv);
  bf16_t* cp = static_cast<bf16_t*>(cache_layer);
  bf16_t* op = static_cast<bf16_t*>(out);
#define ZSA_DEC(HD_, G_)                                                                    \
  if (hd == HD_ && group == G_)                                                             \
    return launch_dec<HD_, G_>(s, qp, q_stride, kv_col, cp, cap, kvd, len_dev, B, H, Hkv, sl, \
                               S, rounds, m_part, l_part, o_part, op, out_stride);
  ZSA_DEC(64, 1) ZSA_DEC(64, 2) ZSA_DEC(64, 4) ZSA_DEC(64, 8)
  ZSA_DEC(128, 1) ZSA_DEC(128, 2) ZSA_DEC(128, 4) ZSA_DEC(128, 8)
#undef ZSA_DEC
  return hipErrorInvalidValue;
}

}  // namespace zsa
