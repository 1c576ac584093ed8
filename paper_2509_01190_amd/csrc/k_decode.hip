// Generation after a pruned prefill: the key/value cache and the attention
// of one new row per sequence over it.
//
// Cache layout: [layer][batch][capacity][k | v], kvd = kv_heads * head_dim
// elements each for k and v (k after the rotary embedding), storage dtype.
// A layer's cache holds the rows that entered that layer in the prefill
// (fewer after every pruning point) followed by the generated rows.
//
// kv_store: copies the k | v columns of the fused projection output into the
// cache (prefill: every row of a layer; decode: the one new row per
// sequence, at its current cache length). 16-byte chunks, coalesced.
//
// decode_attn: one new query row per sequence over its len cached rows (the
// new row's own k / v already stored). Split over the cache: workgroup
// (split, kv head, sequence) takes up to kDecKeys rows of one key/value
// head and every query head that reads it (grouped-query attention shares
// the cache reads), computes scores, a softmax local to the split and the
// split's share of P V, and writes (max, sum, o) partials in fp32.
// decode_combine merges the splits of each (sequence, query head) in split
// order (fixed, so the result is reproducible). The work is HBM-bound on
// the cache rows: 2 * kvd * size bytes per cached row and layer.
#include <math.h>

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

constexpr int kDecKeys = 128;  // cache rows per split and workgroup (one per thread)

// q: new rows [B, q_stride] (query head h at columns h*HD); cache of this
// layer [B][cap][2 kvd]; len [B] rows in the cache (the new one included).
// Partials: m, l [B][H][S], o [B][H][S][HD].
template <int HD, int G>
__global__ __launch_bounds__(kDecKeys) void decode_attn_kernel(
    const bf16_t* __restrict__ q, int64_t q_stride, const bf16_t* __restrict__ cache, int cap,
    int kvd, const int32_t* __restrict__ len, int H, float scale_log2, int S,
    float* __restrict__ m_part, float* __restrict__ l_part, float* __restrict__ o_part) {
  static_assert(HD <= kDecKeys && kDecKeys % HD == 0, "row phases");
  __shared__ float qs[G][HD];
  __shared__ float ps[G][kDecKeys];
  __shared__ float red[2][G];
  __shared__ bf16_t vs[kDecKeys][HD + 8];
  const int s = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n = len[b];
  const int j0 = s * kDecKeys;
  const int nk = min(kDecKeys, n - j0);  // rows of this split (may be <= 0)
  const int h0 = g * G;
  const int64_t part = (static_cast<int64_t>(b) * H + h0) * S + s;  // (b, h0, s)
  if (nk <= 0) {
    for (int e = tid; e < G; e += kDecKeys) {
      m_part[part + static_cast<int64_t>(e) * S] = -INFINITY;
      l_part[part + static_cast<int64_t>(e) * S] = 0.f;
    }
    for (int e = tid; e < G * HD; e += kDecKeys)
      o_part[(part + static_cast<int64_t>(e / HD) * S) * HD + e % HD] = 0.f;
    return;
  }
  for (int e = tid; e < G * HD; e += kDecKeys)
    qs[e / HD][e % HD] =
        to_f32(q[static_cast<int64_t>(b) * q_stride + (h0 + e / HD) * HD + e % HD]);
  // this split's V rows of head g into LDS (16-byte chunks)
  const bf16_t* rows = cache + (static_cast<int64_t>(b) * cap + j0) * 2 * kvd;
  for (int e = tid; e < nk * (HD / 8); e += kDecKeys) {
    const int r = e / (HD / 8), c = (e % (HD / 8)) * 8;
    *reinterpret_cast<uint4*>(&vs[r][c]) =
        *reinterpret_cast<const uint4*>(rows + static_cast<int64_t>(r) * 2 * kvd + kvd + g * HD + c);
  }
  __syncthreads();
  // scores: thread t takes cache row j0 + t against every query head of the group
  float sc[G];
  const bool valid = tid < nk;
#pragma unroll
  for (int e = 0; e < G; ++e) sc[e] = 0.f;
  if (valid) {
    const bf16_t* krow = rows + static_cast<int64_t>(tid) * 2 * kvd + g * HD;
#pragma unroll 4
    for (int c = 0; c < HD; c += 8) {
      float kf[8];
      unpack16(*reinterpret_cast<const uint4*>(krow + c), kf, bf16_t());
#pragma unroll
      for (int e = 0; e < G; ++e)
#pragma unroll
        for (int u = 0; u < 8; ++u) sc[e] = fmaf(qs[e][c + u], kf[u], sc[e]);
    }
  }
  // split-local softmax per query head: max, then exp and sum
#pragma unroll
  for (int e = 0; e < G; ++e) {
    float v = valid ? sc[e] * scale_log2 : -INFINITY;
    sc[e] = v;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
    if (lane == 0) red[wave][e] = v;
  }
  __syncthreads();
  float mx[G];
#pragma unroll
  for (int e = 0; e < G; ++e) mx[e] = fmaxf(red[0][e], red[1][e]);
  __syncthreads();
#pragma unroll
  for (int e = 0; e < G; ++e) {
    const float p = valid ? __builtin_amdgcn_exp2f(sc[e] - mx[e]) : 0.f;
    ps[e][tid] = p;
    float v = p;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    if (lane == 0) red[wave][e] = v;
  }
  __syncthreads();
  if (tid == 0) {
#pragma unroll
    for (int e = 0; e < G; ++e) {
      m_part[part + static_cast<int64_t>(e) * S] = mx[e];
      l_part[part + static_cast<int64_t>(e) * S] = red[0][e] + red[1][e];
    }
  }
  // o[e][c] = sum_t p[e][t] v[t][c]: thread column c = tid % HD; the
  // kDecKeys / HD row phases (rows t = ph, ph + PH, ...) are added in phase
  // order through LDS
  constexpr int PH = kDecKeys / HD;
  const int c = tid % HD, ph = tid / HD;
  float acc[G];
#pragma unroll
  for (int e = 0; e < G; ++e) acc[e] = 0.f;
  for (int t = ph; t < nk; t += PH) {
    const float v = to_f32(vs[t][c]);
#pragma unroll
    for (int e = 0; e < G; ++e) acc[e] = fmaf(ps[e][t], v, acc[e]);
  }
  __syncthreads();               // every thread is done reading ps
  float* stage = &ps[0][0];      // [PH][G][HD] floats = G * kDecKeys
#pragma unroll
  for (int e = 0; e < G; ++e) stage[(ph * G + e) * HD + c] = acc[e];
  __syncthreads();
  if (ph == 0) {
#pragma unroll
    for (int e = 0; e < G; ++e) {
      float v = stage[e * HD + c];
#pragma unroll
      for (int k = 1; k < PH; ++k) v += stage[(k * G + e) * HD + c];
      o_part[(part + static_cast<int64_t>(e) * S) * HD + c] = v;
    }
  }
}

// one workgroup of HD threads per (query head, sequence): merge the splits
__global__ void decode_combine_kernel(const float* __restrict__ m_part,
                                      const float* __restrict__ l_part,
                                      const float* __restrict__ o_part, int S, int H, int HD,
                                      bf16_t* __restrict__ out, int64_t out_stride) {
  const int h = blockIdx.x, b = blockIdx.y, c = threadIdx.x;
  const int64_t base = (static_cast<int64_t>(b) * H + h) * S;
  float M = -INFINITY;
  for (int s = 0; s < S; ++s) M = fmaxf(M, m_part[base + s]);
  float L = 0.f, acc = 0.f;
  for (int s = 0; s < S; ++s) {
    const float w = l_part[base + s] > 0.f ? __builtin_amdgcn_exp2f(m_part[base + s] - M) : 0.f;
    L = fmaf(l_part[base + s], w, L);
    acc = fmaf(o_part[(base + s) * HD + c], w, acc);
  }
  out[static_cast<int64_t>(b) * out_stride + h * HD + c] = f32_to_bf16(acc / L);
}

template <int HD, int G>
hipError_t launch_dec(hipStream_t s, const bf16_t* q, int64_t q_stride, const bf16_t* cache,
                      int cap, int kvd, const int32_t* len, int B, int H, int Hkv, float sl,
                      int S, float* m, float* l, float* o) {
  return launch(K_ATTENTION, decode_attn_kernel<HD, G>, dim3(S, Hkv, B), dim3(kDecKeys), 0, s, q,
                q_stride, cache, cap, kvd, len, H, sl, S, m, l, o);
}

}  // namespace

int decode_splits(int max_len) { return (max_len + kDecKeys - 1) / kDecKeys; }

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

hipError_t launch_decode_attention(hipStream_t s, const void* q, int64_t q_stride,
                                   const void* cache_layer, int cap, int hd, int H, int Hkv,
                                   const int32_t* len_dev, int B, int S, float scale,
                                   float* m_part, float* l_part, float* o_part, void* out,
                                   int64_t out_stride) {
  if (B == 0) return hipSuccess;
  const int kvd = Hkv * hd, group = H / Hkv;
  const float sl = scale * kLog2e;
  const bf16_t* qp = static_cast<const bf16_t*>(q);
  const bf16_t* cp = static_cast<const bf16_t*>(cache_layer);
  hipError_t e = hipErrorInvalidValue;
#define ZSA_DEC(HD_, G_)                                                                      \
  if (hd == HD_ && group == G_)                                                               \
    e = launch_dec<HD_, G_>(s, qp, q_stride, cp, cap, kvd, len_dev, B, H, Hkv, sl, S, m_part, \
                            l_part, o_part);
  ZSA_DEC(64, 1) ZSA_DEC(64, 2) ZSA_DEC(64, 4) ZSA_DEC(64, 8)
  ZSA_DEC(128, 1) ZSA_DEC(128, 2) ZSA_DEC(128, 4) ZSA_DEC(128, 8)
#undef ZSA_DEC
  if (e != hipSuccess) return e;
  return launch(K_ATTENTION, decode_combine_kernel, dim3(H, B), dim3(hd), 0, s, m_part, l_part,
                o_part, S, H, hd, static_cast<bf16_t*>(out), out_stride);
}

}  // namespace zsa
