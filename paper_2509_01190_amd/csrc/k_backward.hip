// Backward pass through the pruned block (the fine-tuning step of Eq. 3
// trains through the pruned forward; the kept rows are constants).
//
// Row-wise pieces: transposes (so both products of a projection's backward
// run on the forward's NT GEMM), column sums (bias / gain gradients, in a
// fixed order), LayerNorm / RMSNorm backward, GELU / SwiGLU backward, the
// scatter that undoes compaction (dropped rows get zero gradient), the
// per-row dot D_i = dO_i . O_i, and the inverse rotary rotation.
//
// Attention backward (bf16, head_dim 64 / 128, MFMA), with P recomputed
// from the forward's log-sum-exp:
//     dV = P^T dO,  dP = dO V^T,  dS = P o (dP - D),  dK = scale dS^T Q,
//     dQ = scale dS K.
// attn_bwd_dkdv: one workgroup per (128-key block, key/value head,
// sequence), 32 keys per wave; the waves walk the 32-query tiles together
// from one double-buffered LDS stage (Q and dO in rows and transposed),
// compute S = Q K^T and dP = dO V^T in the layout where a lane owns one key,
// and multiply P and dS, packed as MFMA A operands, with the transposed
// tiles. Each key's dK / dV is summed by one wave in query order (no
// atomics). For grouped-query attention the workgroup also loops over the
// query heads that read its key/value head.
// attn_bwd_dq: one workgroup per (128-query block, head, sequence), laid out
// like the forward attention: S^T and dP^T with a lane owning one query, dS
// packed as the B operand of dQ^T += K^T dS^T, K^T staged in LDS.
#include <math.h>

#include "zsa_internal.h"

namespace zsa {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
constexpr float kLog2e = 1.4426950408889634f;

template <typename T>
__device__ __forceinline__ void load8(const T* p, float* v);
template <>
__device__ __forceinline__ void load8<bf16_t>(const bf16_t* p, float* v) {
  unpack16(*reinterpret_cast<const uint4*>(p), v, bf16_t());
}
template <>
__device__ __forceinline__ void load8<float>(const float* p, float* v) {
  unpack16(reinterpret_cast<const uint4*>(p)[0], v, 0.f);
  unpack16(reinterpret_cast<const uint4*>(p)[1], v + 4, 0.f);
}
template <typename T>
__device__ __forceinline__ void store8(T* p, const float* v);
template <>
__device__ __forceinline__ void store8<bf16_t>(bf16_t* p, const float* v) {
  *reinterpret_cast<uint4*>(p) = pack16(v, bf16_t());
}
template <>
__device__ __forceinline__ void store8<float>(float* p, const float* v) {
  reinterpret_cast<uint4*>(p)[0] = pack16(v, 0.f);
  reinterpret_cast<uint4*>(p)[1] = pack16(v + 4, 0.f);
}

// ---------------------------------------------------------------------------
// transpose: out[c][r] = in[r][c] for r < R, 0 for R <= r < Rpad
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void transpose_kernel(const T* __restrict__ in, int R, int C,
                                                        int64_t ldi, T* __restrict__ out,
                                                        int Rpad) {
  __shared__ T tile[32][33];
  const int r0 = blockIdx.y * 32, c0 = blockIdx.x * 32;
  const int tx = threadIdx.x & 31, ty = threadIdx.x >> 5;  // 8 rows per pass
  for (int k = ty; k < 32; k += 8) {
    const int r = r0 + k, c = c0 + tx;
    tile[k][tx] = (r < R && c < C) ? in[static_cast<int64_t>(r) * ldi + c] : T(0.f);
  }
  __syncthreads();
  for (int k = ty; k < 32; k += 8) {
    const int c = c0 + k, r = r0 + tx;
    if (c < C && r < Rpad) out[static_cast<int64_t>(c) * Rpad + r] = tile[tx][k];
  }
}

// bf16, 64 x 64 tiles with 16-byte loads and stores (C, R multiples of 8 for
// the vector paths; edges fall back to element accesses)
__global__ __launch_bounds__(256) void transpose64_kernel(const bf16_t* __restrict__ in, int R,
                                                          int C, int64_t ldi,
                                                          bf16_t* __restrict__ out, int Rpad) {
  __shared__ bf16_t tile[64][64 + 2];
  const int r0 = blockIdx.y * 64, c0 = blockIdx.x * 64;
  const int t = threadIdx.x;
  for (int k = t; k < 64 * 8; k += 256) {
    const int r = k / 8, ch = (k % 8) * 8;
    const int gr = r0 + r, gc = c0 + ch;
    if (gr < R && gc + 8 <= C) {
      const uint4 v = *reinterpret_cast<const uint4*>(in + static_cast<int64_t>(gr) * ldi + gc);
      const bf16_t* e = reinterpret_cast<const bf16_t*>(&v);
#pragma unroll
      for (int j = 0; j < 8; ++j) tile[r][ch + j] = e[j];
    } else {
#pragma unroll
      for (int j = 0; j < 8; ++j)
        tile[r][ch + j] = (gr < R && gc + j < C) ? in[static_cast<int64_t>(gr) * ldi + gc + j]
                                                 : bf16_t(0.f);
    }
  }
  __syncthreads();
  for (int k = t; k < 64 * 8; k += 256) {
    const int c = k / 8, rh = (k % 8) * 8;   // output row c0 + c, columns r0 + rh ..
    const int gc = c0 + c, gr = r0 + rh;
    if (gc >= C) continue;
    if (gr + 8 <= Rpad) {
      uint4 v;
      bf16_t* e = reinterpret_cast<bf16_t*>(&v);
#pragma unroll
      for (int j = 0; j < 8; ++j) e[j] = tile[rh + j][c];
      *reinterpret_cast<uint4*>(out + static_cast<int64_t>(gc) * Rpad + gr) = v;
    } else {
      for (int j = 0; j < 8 && gr + j < Rpad; ++j)
        out[static_cast<int64_t>(gc) * Rpad + gr + j] = tile[rh + j][c];
    }
  }
}

// ---------------------------------------------------------------------------
// column sums in a fixed order: stage 1 sums chunks of kColRows rows (each
// thread 8 consecutive columns with 16-byte loads, 8 row lanes per block
// added in lane order), stage 2 adds the chunks in chunk order
// ---------------------------------------------------------------------------
constexpr int kColRows = 64;   // rows per stage-1 chunk
constexpr int kColLanes = 8;   // row lanes per block

// sum over rows of a[r][c] (or of a[r][c] * xhat[r][c] when x is given, with
// xhat = (x - mean_r) * rstd_r from stats [R][2]); C a multiple of 8
template <typename T>
__global__ __launch_bounds__(256) void colsum_stage1(const T* __restrict__ a, int64_t lda,
                                                     const T* __restrict__ x, int64_t ldx,
                                                     const float* __restrict__ stats, int R,
                                                     int C, float* __restrict__ part) {
  __shared__ float red[kColLanes][32 * 8 + 4];
  const int cg = threadIdx.x & 31, lane_r = threadIdx.x >> 5;
  const int c0 = (blockIdx.x * 32 + cg) * 8;
  const int r0 = blockIdx.y * kColRows;
  float s[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) s[e] = 0.f;
  if (c0 < C) {
    const int r1 = min(R, r0 + kColRows);
    for (int r = r0 + lane_r; r < r1; r += kColLanes) {
      float v[8];
      load8<T>(a + static_cast<int64_t>(r) * lda + c0, v);
      if (x != nullptr) {
        float xv[8];
        load8<T>(x + static_cast<int64_t>(r) * ldx + c0, xv);
        const float mu = stats[2 * r], rs = stats[2 * r + 1];
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] *= (xv[e] - mu) * rs;
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) s[e] += v[e];
    }
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) red[lane_r][cg * 8 + e] = s[e];
  __syncthreads();
  if (lane_r == 0 && c0 < C) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      float v = red[0][cg * 8 + e];
#pragma unroll
      for (int k = 1; k < kColLanes; ++k) v += red[k][cg * 8 + e];
      part[static_cast<int64_t>(blockIdx.y) * C + c0 + e] = v;
    }
  }
}

__global__ void zero_f32_kernel(float* __restrict__ p, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0.f;
}

// ---------------------------------------------------------------------------
// norm backward: one wave per row.
//   LN:  dx = rstd (g dh - mean(g dh) - xhat mean(g dh xhat))
//   RMS: dx = rstd (g dh - xhat mean(g dh xhat))
// out = res + dx (res may alias out, or be NULL); stats[r] = (mean, rstd)
// (mean 0 for RMS) for the gain / shift gradients.
// ---------------------------------------------------------------------------
template <typename T, int RMS, int NC>
__global__ __launch_bounds__(256) void norm_bwd_kernel(const T* __restrict__ x,
                                                       const T* __restrict__ g,
                                                       const T* __restrict__ dh, const T* res,
                                                       T* out, int R, int d, float eps,
                                                       float* __restrict__ stats) {
  // one wave per row; lane owns the 8-column chunks lane, lane + 64, ...
  // (NC of them, d <= NC * 512), held in registers across the passes
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= R) return;
  const int64_t base = static_cast<int64_t>(row) * d;
  float xv[NC][8], gd[NC][8];
  float s = 0.f;
#pragma unroll
  for (int k = 0; k < NC; ++k) {
    const int c = (k * 64 + lane) * 8;
    if (c < d) {
      float gv[8];
      load8<T>(x + base + c, xv[k]);
      load8<T>(g + c, gv);
      load8<T>(dh + base + c, gd[k]);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        gd[k][e] *= gv[e];
        s += xv[k][e];
      }
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) xv[k][e] = gd[k][e] = 0.f;
    }
  }
  float mean = 0.f;
  if (!RMS) {
    for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o, 64);
    mean = s / d;
  }
  float ss = 0.f;
#pragma unroll
  for (int k = 0; k < NC; ++k) {
    if ((k * 64 + lane) * 8 < d) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float v = xv[k][e] - mean;
        ss += v * v;
      }
    }
  }
  for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o, 64);
  const float rstd = 1.0f / sqrtf(ss / d + eps);
  float s1 = 0.f, s2 = 0.f;  // sum(g dh), sum(g dh xhat)
#pragma unroll
  for (int k = 0; k < NC; ++k) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      s1 += gd[k][e];
      s2 += gd[k][e] * (xv[k][e] - mean) * rstd;  // zero on chunks past d
    }
  }
  for (int o = 32; o > 0; o >>= 1) {
    s1 += __shfl_xor(s1, o, 64);
    s2 += __shfl_xor(s2, o, 64);
  }
  const float m1 = RMS ? 0.f : s1 / d, m2 = s2 / d;
#pragma unroll
  for (int k = 0; k < NC; ++k) {
    const int c = (k * 64 + lane) * 8;
    if (c < d) {
      float o[8], rv[8];
      if (res != nullptr) load8<T>(res + base + c, rv);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float xh = (xv[k][e] - mean) * rstd;
        o[e] = rstd * (gd[k][e] - m1 - xh * m2) + (res != nullptr ? rv[e] : 0.f);
      }
      store8<T>(out + base + c, o);
    }
  }
  if (lane == 0) {
    stats[2 * row] = mean;
    stats[2 * row + 1] = rstd;
  }
}

// ---------------------------------------------------------------------------
// activation backward. GELU: du = dF (Phi(u) + u phi(u)). SwiGLU on
// interleaved columns (2f gate, 2f+1 up): dgate = dF up silu'(gate),
// dup = dF silu(gate), silu'(z) = s (1 + z (1 - s)), s = sigmoid(z).
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void act_bwd_kernel(const T* __restrict__ dF,
                                                      const T* __restrict__ u, T* __restrict__ du,
                                                      int64_t rows, int F, int swiglu) {
  // 8 consecutive outputs f..f+7 of one row per thread
  const int64_t i = (static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x) * 8;
  if (i >= rows * F) return;
  const int64_t r = i / F;
  const int f = static_cast<int>(i - r * F);
  float g[8];
  load8<T>(dF + i, g);
  if (swiglu) {
    float u0[8], u1[8], o0[8], o1[8];
    load8<T>(u + r * 2 * F + 2 * f, u0);       // gate, up of outputs f .. f+3
    load8<T>(u + r * 2 * F + 2 * f + 8, u1);   // ... of f+4 .. f+7
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float z0 = u0[2 * e], up0 = u0[2 * e + 1], s0 = 1.0f / (1.0f + expf(-z0));
      const float z1 = u1[2 * e], up1 = u1[2 * e + 1], s1 = 1.0f / (1.0f + expf(-z1));
      o0[2 * e] = g[e] * up0 * s0 * (1.0f + z0 * (1.0f - s0));
      o0[2 * e + 1] = g[e] * z0 * s0;
      o1[2 * e] = g[4 + e] * up1 * s1 * (1.0f + z1 * (1.0f - s1));
      o1[2 * e + 1] = g[4 + e] * z1 * s1;
    }
    store8<T>(du + r * 2 * F + 2 * f, o0);
    store8<T>(du + r * 2 * F + 2 * f + 8, o1);
  } else {
    float z[8], o[8];
    load8<T>(u + i, z);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float cdf = 0.5f * (1.0f + erff(z[e] * 0.70710678118654752f));
      const float pdf = 0.39894228040143268f * __expf(-0.5f * z[e] * z[e]);
      o[e] = g[e] * (cdf + z[e] * pdf);
    }
    store8<T>(du + i, o);
  }
}

// the activation itself from the pre-activation u (GELU, or SwiGLU on
// interleaved gate / up columns): the backward's recomputed forward
template <typename T>
__global__ __launch_bounds__(256) void act_fwd_kernel(const T* __restrict__ u, T* __restrict__ f,
                                                      int64_t rows, int F, int swiglu) {
  const int64_t i = (static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x) * 8;
  if (i >= rows * F) return;
  const int64_t r = i / F;
  const int c = static_cast<int>(i - r * F);
  float o[8];
  if (swiglu) {
    float u0[8], u1[8];
    load8<T>(u + r * 2 * F + 2 * c, u0);
    load8<T>(u + r * 2 * F + 2 * c + 8, u1);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      o[e] = u0[2 * e] / (1.0f + expf(-u0[2 * e])) * u0[2 * e + 1];
      o[4 + e] = u1[2 * e] / (1.0f + expf(-u1[2 * e])) * u1[2 * e + 1];
    }
  } else {
    float z[8];
    load8<T>(u + i, z);
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] = 0.5f * z[e] * (1.0f + erff(z[e] * 0.70710678118654752f));
  }
  store8<T>(f + i, o);
}

// ---------------------------------------------------------------------------
// undo compaction: dst[r] = src[inv[r]] for kept rows, 0 for dropped ones
// ---------------------------------------------------------------------------
__global__ void inverse_index_kernel(const int32_t* __restrict__ kept, int t_out, int t_in,
                                     int32_t* __restrict__ inv) {
  // one pass per row of the input: rows not found stay -1 (filled first)
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < t_out) {
    const int r = kept[i];
    if (r >= 0 && r < t_in) inv[r] = i;
  }
}

__global__ void fill_i32_kernel(int32_t* __restrict__ p, int n, int v) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

__global__ __launch_bounds__(256) void scatter_rows_kernel(const uint4* __restrict__ src,
                                                           const int32_t* __restrict__ inv,
                                                           int t_in, int cpr,
                                                           uint4* __restrict__ dst) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i >= static_cast<int64_t>(t_in) * cpr) return;
  const int r = static_cast<int>(i / cpr), c = static_cast<int>(i % cpr);
  const int s = inv[r];
  dst[i] = s >= 0 ? src[static_cast<int64_t>(s) * cpr + c] : make_uint4(0u, 0u, 0u, 0u);
}

// D[h][r] = sum_c dO[r][h hd + c] O[r][h hd + c]: each thread takes 8
// consecutive columns, the L = hd / 8 threads of one head (L a power of two
// up to 64, adjacent lanes of one wave) add theirs in a fixed butterfly
template <typename T>
__global__ __launch_bounds__(256) void rowdot_kernel(const T* __restrict__ dO,
                                                     const T* __restrict__ O, int64_t ld, int T_,
                                                     int H, int hd, float* __restrict__ D) {
  const int L = hd / 8, per_row = H * L;
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  const bool live = i < static_cast<int64_t>(T_) * per_row;
  const int r = live ? static_cast<int>(i / per_row) : 0;
  const int c8 = live ? static_cast<int>(i - static_cast<int64_t>(r) * per_row) : 0;
  float s = 0.f;
  if (live) {
    float va[8], vb[8];
    load8<T>(dO + static_cast<int64_t>(r) * ld + c8 * 8, va);
    load8<T>(O + static_cast<int64_t>(r) * ld + c8 * 8, vb);
#pragma unroll
    for (int e = 0; e < 8; ++e) s = fmaf(va[e], vb[e], s);
  }
  // groups of L lanes start at multiples of L within the wave (64 % L == 0
  // and each block is 256 threads), so the butterfly stays inside one head
  for (int o = 1; o < L; o <<= 1) s += __shfl_xor(s, o, 64);
  if (live && (c8 & (L - 1)) == 0) D[static_cast<int64_t>(c8 / L) * T_ + r] = s;
}

// inverse rotary rotation of the gradient, in place, on the first `cols`
// columns (whole heads) of rows of a [rows, ld] array
template <typename T>
__global__ __launch_bounds__(256) void rope_bwd_kernel(T* __restrict__ g, int64_t ld, int rows,
                                                       int cols, int hd,
                                                       const int32_t* __restrict__ pos,
                                                       EpiParams ep) {
  const int half = hd / 2;
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  const int pairs = cols / 2;
  if (i >= static_cast<int64_t>(rows) * pairs) return;
  const int r = static_cast<int>(i / pairs);
  const int pr = static_cast<int>(i % pairs);
  const int head = pr / half, k = pr % half;
  const int64_t a = static_cast<int64_t>(r) * ld + head * hd + k;
  float sn, cs;
  rope_angle(pos[r], ep.inv_freq[k], &sn, &cs);
  const float x = to_f32(g[a]), y = to_f32(g[a + half]);
  g[a] = from_f32<T>(x * cs + y * sn);
  g[a + half] = from_f32<T>(y * cs - x * sn);
}

// ---------------------------------------------------------------------------
// attention backward, dK and dV
// ---------------------------------------------------------------------------
__device__ __forceinline__ float pick4(const float4& v, int i) {
  return i == 0 ? v.x : i == 1 ? v.y : i == 2 ? v.z : v.w;
}

// Each workgroup owns 128 consecutive keys of one kv head, 32 per wave. The
// waves sweep the query tiles of 32 together: each tile of Q and dO (with
// the rows' log-sum-exp and D) is staged once per workgroup into LDS, in
// rows (the A operands of S = Q K^T and dP = dO V^T) and transposed (the B
// operands of dV += P^T dO and dK += dS^T Q), double-buffered so the next
// tile's global loads overlap this tile's MFMAs. P and dS leave the
// accumulators with the keys on the lanes and the queries in the registers,
// so they are the A operands of the dV and dK products as they are; each
// wave keeps its keys' dK and dV and writes them once.
template <int HD>
__global__ __launch_bounds__(256) void attn_bwd_dkdv_kernel(
    const bf16_t* __restrict__ Q, const bf16_t* __restrict__ K, const bf16_t* __restrict__ V,
    int64_t rs, const bf16_t* __restrict__ dO, int64_t ors, const float* __restrict__ lse,
    const float* __restrict__ Dv, int T, int kv_group, int causal, float scale,
    float scale_log2, const int32_t* __restrict__ cu, bf16_t* __restrict__ dK,
    bf16_t* __restrict__ dV, int64_t grs) {
  constexpr int KW = 128, QT = 32;
  constexpr int KK = HD / 16, CT = HD / 32;
  constexpr int RLD = HD + 8;            // row tile stride (bf16)
  constexpr int TLD = QT + 4;            // transposed tile stride (bf16), 18 dwords
  constexpr int ROW_E = QT * RLD, TR_E = HD * TLD;
  constexpr int BUF = 4 * ROW_E + 4 * TR_E + 2 * QT * 4;  // bytes of one stage
  constexpr int TASKS = 2 * (QT / 2) * (HD / 8);          // (tensor, query pair, chunk)
  constexpr int NT = TASKS / 256;
  static_assert(NT >= 1 && NT * 256 == TASKS, "staging tasks must fill the block");
  static_assert(BUF % 16 == 0, "stage size");
  static_assert(8 * 32 * RLD * 2 <= 2 * BUF, "output staging fits the stages");
  __shared__ __align__(16) unsigned char smem[2 * BUF];

  const int b = blockIdx.z, g = blockIdx.y;
  const int lo = cu[b];
  const int n = cu[b + 1] - lo;
  const int j0 = blockIdx.x * KW;
  if (j0 >= n) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5, l32 = lane & 31;
  const int jw = j0 + wave * 32;  // the wave's first key
  const bool wave_live = jw < n;

  bf16x8_t kf[KK], vf[KK];
  {
    const int jr = lo + min(jw + l32, n - 1);
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      kf[kk] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const u32x4*>(
                                                K + static_cast<int64_t>(jr) * rs + g * HD + kk * 16 + half * 8));
      vf[kk] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const u32x4*>(
                                                V + static_cast<int64_t>(jr) * rs + g * HD + kk * 16 + half * 8));
    }
  }
  f32x16_t dk[CT], dv[CT];
#pragma unroll
  for (int ct = 0; ct < CT; ++ct)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      dk[ct][r] = 0.f;
      dv[ct][r] = 0.f;
    }

  // queries before the first key see none of the keys (causal)
  const int qs = causal ? j0 : 0;
  const int ntile = (n - qs + QT - 1) / QT;
  const int rounds = ntile * kv_group;

  u32x4 st[NT][2];
  float stl = 0.f;
  auto fetch = [&](int t) {
    const int e = t / ntile, i0 = qs + (t - e * ntile) * QT, h = g * kv_group + e;
#pragma unroll
    for (int k = 0; k < NT; ++k) {
      const int task = tid + 256 * k;
      const int tensor = task / (TASKS / 2), rem = task % (TASKS / 2);
      const int rp = rem / (HD / 8), ch = (rem % (HD / 8)) * 8;
      const int r0 = lo + min(i0 + 2 * rp, n - 1), r1 = lo + min(i0 + 2 * rp + 1, n - 1);
      const bf16_t* src = tensor ? dO : Q;
      const int64_t ld = tensor ? ors : rs;
      st[k][0] = *reinterpret_cast<const u32x4*>(src + static_cast<int64_t>(r0) * ld + h * HD + ch);
      st[k][1] = *reinterpret_cast<const u32x4*>(src + static_cast<int64_t>(r1) * ld + h * HD + ch);
    }
    if (tid < 2 * QT) {
      const int64_t i = static_cast<int64_t>(h) * T + lo + min(i0 + (tid & (QT - 1)), n - 1);
      stl = tid < QT ? lse[i] * kLog2e : Dv[i];
    }
  };
  auto stash = [&](int buf) {
    bf16_t* rowQ = reinterpret_cast<bf16_t*>(smem + buf * BUF);
    bf16_t* trQ = rowQ + 2 * ROW_E;
    float* LD = reinterpret_cast<float*>(trQ + 2 * TR_E);
#pragma unroll
    for (int k = 0; k < NT; ++k) {
      const int task = tid + 256 * k;
      const int tensor = task / (TASKS / 2), rem = task % (TASKS / 2);
      const int rp = rem / (HD / 8), ch = (rem % (HD / 8)) * 8;
      bf16_t* rw = rowQ + tensor * ROW_E;
      bf16_t* tr = trQ + tensor * TR_E;
      *reinterpret_cast<u32x4*>(rw + (2 * rp) * RLD + ch) = st[k][0];
      *reinterpret_cast<u32x4*>(rw + (2 * rp + 1) * RLD + ch) = st[k][1];
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        const uint32_t a0 = st[k][0][c >> 1], a1 = st[k][1][c >> 1];
        const uint32_t lo16 = (c & 1) ? (a0 >> 16) : (a0 & 0xffffu);
        const uint32_t hi16 = (c & 1) ? (a1 & 0xffff0000u) : (a1 << 16);
        *reinterpret_cast<uint32_t*>(tr + (ch + c) * TLD + 2 * rp) = lo16 | hi16;
      }
    }
    if (tid < 2 * QT) LD[tid] = stl;
  };

  fetch(0);
  stash(0);
  __syncthreads();
  for (int t = 0; t < rounds; ++t) {
    if (t + 1 < rounds) fetch(t + 1);
    const int e = t / ntile, i0 = qs + (t - e * ntile) * QT;
    // a wave whose keys all lie past this tile's last query sees none of it
    if (wave_live && !(causal && jw > i0 + QT - 1)) {
      const bf16_t* rowQ = reinterpret_cast<const bf16_t*>(smem + (t & 1) * BUF);
      const bf16_t* rowD = rowQ + ROW_E;
      const bf16_t* trQ = rowQ + 2 * ROW_E;
      const bf16_t* trD = trQ + TR_E;
      const float* LD = reinterpret_cast<const float*>(trQ + 2 * TR_E);
      f32x16_t s, dp;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        s[r] = 0.f;
        dp[r] = 0.f;
      }
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) {
        const bf16x8_t qa = __builtin_bit_cast(
            bf16x8_t, *reinterpret_cast<const u32x4*>(rowQ + l32 * RLD + kk * 16 + half * 8));
        const bf16x8_t da = __builtin_bit_cast(
            bf16x8_t, *reinterpret_cast<const u32x4*>(rowD + l32 * RLD + kk * 16 + half * 8));
        s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qa, kf[kk], s, 0, 0, 0);
        dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(da, vf[kk], dp, 0, 0, 0);
      }
      // s[r], dp[r]: query i0 + 8 (r/4) + 4 half + r%4, key jw + l32. Keys
      // past the sequence only feed accumulator rows that are not written.
      const int j = jw + l32;
      const bool edge = i0 + QT > n || (causal && jw + 31 > i0);
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        const float4 L4 = *reinterpret_cast<const float4*>(LD + 8 * a + 4 * half);
        const float4 D4 = *reinterpret_cast<const float4*>(LD + QT + 8 * a + 4 * half);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int r = 4 * a + q;
          float p = __builtin_amdgcn_exp2f(fmaf(s[r], scale_log2, -pick4(L4, q)));
          if (edge) {
            const int i = i0 + 8 * a + 4 * half + q;
            if (i >= n || (causal && j > i)) p = 0.f;
          }
          s[r] = p;
          dp[r] = p * (dp[r] - pick4(D4, q));
        }
      }
#pragma unroll
      for (int g4 = 0; g4 < 2; ++g4) {
        const int rb = 8 * g4;
        const u32x4 pw = {pack_bf16x2(s[rb], s[rb + 1]), pack_bf16x2(s[rb + 2], s[rb + 3]),
                          pack_bf16x2(s[rb + 4], s[rb + 5]), pack_bf16x2(s[rb + 6], s[rb + 7])};
        const u32x4 sw = {pack_bf16x2(dp[rb], dp[rb + 1]), pack_bf16x2(dp[rb + 2], dp[rb + 3]),
                          pack_bf16x2(dp[rb + 4], dp[rb + 5]), pack_bf16x2(dp[rb + 6], dp[rb + 7])};
        const bf16x8_t pa = __builtin_bit_cast(bf16x8_t, pw);
        const bf16x8_t sa = __builtin_bit_cast(bf16x8_t, sw);
        const int base = 16 * g4 + 4 * half;  // queries base..+3, base+8..+11
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) {
          const bf16_t* dr = trD + (ct * 32 + l32) * TLD + base;
          const bf16_t* qrw = trQ + (ct * 32 + l32) * TLD + base;
          const uint2 d_lo = *reinterpret_cast<const uint2*>(dr);
          const uint2 d_hi = *reinterpret_cast<const uint2*>(dr + 8);
          const uint2 q_lo = *reinterpret_cast<const uint2*>(qrw);
          const uint2 q_hi = *reinterpret_cast<const uint2*>(qrw + 8);
          const u32x4 bd = {d_lo.x, d_lo.y, d_hi.x, d_hi.y};
          const u32x4 bq = {q_lo.x, q_lo.y, q_hi.x, q_hi.y};
          dv[ct] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(pa, __builtin_bit_cast(bf16x8_t, bd),
                                                           dv[ct], 0, 0, 0);
          dk[ct] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(sa, __builtin_bit_cast(bf16x8_t, bq),
                                                           dk[ct], 0, 0, 0);
        }
      }
    }
    if (t + 1 < rounds) stash((t + 1) & 1);
    __syncthreads();
  }
  // acc[ct][r]: key jw + 8 (r/4) + 4 half + r%4, channel ct*32 + l32; staged
  // as bf16 rows in LDS (the wave's own region), then written 16 bytes a lane
  bf16_t* ov = reinterpret_cast<bf16_t*>(smem) + wave * 2 * 32 * RLD;
  bf16_t* okk = ov + 32 * RLD;
#pragma unroll
  for (int ct = 0; ct < CT; ++ct)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int key = 8 * (r >> 2) + 4 * half + (r & 3);
      ov[key * RLD + ct * 32 + l32] = f32_to_bf16(dv[ct][r]);
      okk[key * RLD + ct * 32 + l32] = f32_to_bf16(dk[ct][r] * scale);
    }
  __syncthreads();
  for (int c = lane; c < 32 * (HD / 8); c += 64) {
    const int key = c / (HD / 8), ch = (c % (HD / 8)) * 8;
    if (jw + key >= n) continue;
    const int64_t o = static_cast<int64_t>(lo + jw + key) * grs + g * HD + ch;
    *reinterpret_cast<u32x4*>(dV + o) = *reinterpret_cast<const u32x4*>(ov + key * RLD + ch);
    *reinterpret_cast<u32x4*>(dK + o) = *reinterpret_cast<const u32x4*>(okk + key * RLD + ch);
  }
}

// ---------------------------------------------------------------------------
// attention backward, dQ
// ---------------------------------------------------------------------------
template <int HD>
__global__ __launch_bounds__(256) void attn_bwd_dq_kernel(
    const bf16_t* __restrict__ Q, const bf16_t* __restrict__ K, const bf16_t* __restrict__ V,
    int64_t rs, const bf16_t* __restrict__ dO, int64_t ors, const float* __restrict__ lse,
    const float* __restrict__ Dv, int T, int kv_group, int causal, float scale, float scale_log2,
    const int32_t* __restrict__ cu, bf16_t* __restrict__ dQ, int64_t grs) {
  constexpr int BQ = 128, BKEY = 64;
  constexpr int KLD = HD + 8, TLD = BKEY + 8, OLD = HD + 8;
  constexpr int KK = HD / 16, CT = HD / 32;
  constexpr int KB = BKEY * KLD * 2, TB = HD * TLD * 2;
  constexpr int SMEM = 2 * KB + TB > 4 * 32 * OLD * 2 ? 2 * KB + TB : 4 * 32 * OLD * 2;
  __shared__ __align__(16) unsigned char smem[SMEM];
  bf16_t* Ks = reinterpret_cast<bf16_t*>(smem);
  bf16_t* Vs = reinterpret_cast<bf16_t*>(smem + KB);
  bf16_t* Kt = reinterpret_cast<bf16_t*>(smem + 2 * KB);

  const int b = blockIdx.z, h = blockIdx.y;
  const int lo = cu[b];
  const int n = cu[b + 1] - lo;
  const int q0 = blockIdx.x * BQ;
  if (q0 >= n) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5, l32 = lane & 31;
  const int qrow = q0 + wave * 32 + l32;
  const int qr = lo + min(qrow, n - 1);
  const int hk = h / kv_group;
  bf16x8_t qf[KK], df[KK];
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) {
    qf[kk] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const u32x4*>(
                                              Q + static_cast<int64_t>(qr) * rs + h * HD + kk * 16 + half * 8));
    df[kk] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const u32x4*>(
                                              dO + static_cast<int64_t>(qr) * ors + h * HD + kk * 16 + half * 8));
  }
  const float Lq = lse[static_cast<int64_t>(h) * T + qr] * kLog2e;
  const float Dq = Dv[static_cast<int64_t>(h) * T + qr];
  f32x16_t acc[CT];
#pragma unroll
  for (int ct = 0; ct < CT; ++ct)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[ct][r] = 0.f;

  const int kend = causal ? min(n, q0 + BQ) : n;
  const int wave_q0 = q0 + wave * 32;
  for (int j0 = 0; j0 < kend; j0 += BKEY) {
    __syncthreads();
    for (int c = tid; c < BKEY * HD / 8; c += 256) {
      const int r = c / (HD / 8), ch = (c % (HD / 8)) * 8;
      const int64_t row = lo + min(j0 + r, n - 1);
      *reinterpret_cast<u32x4*>(Ks + r * KLD + ch) =
          *reinterpret_cast<const u32x4*>(K + row * rs + hk * HD + ch);
      *reinterpret_cast<u32x4*>(Vs + r * KLD + ch) =
          *reinterpret_cast<const u32x4*>(V + row * rs + hk * HD + ch);
    }
    // K^T with key pairs packed
    for (int c = tid; c < (BKEY / 2) * (HD / 8); c += 256) {
      const int rp = c / (HD / 8), ch = (c % (HD / 8)) * 8;
      const int64_t r0 = lo + min(j0 + 2 * rp, n - 1), r1 = lo + min(j0 + 2 * rp + 1, n - 1);
      const u32x4 k0 = *reinterpret_cast<const u32x4*>(K + r0 * rs + hk * HD + ch);
      const u32x4 k1 = *reinterpret_cast<const u32x4*>(K + r1 * rs + hk * HD + ch);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const uint32_t w0 = k0[e >> 1], w1 = k1[e >> 1];
        const uint32_t x0 = (e & 1) ? (w0 >> 16) : (w0 & 0xffffu);
        const uint32_t x1 = (e & 1) ? (w1 & 0xffff0000u) : (w1 << 16);
        *reinterpret_cast<uint32_t*>(Kt + (ch + e) * TLD + 2 * rp) = x0 | x1;
      }
    }
    __syncthreads();
    if (causal && j0 > wave_q0 + 31) continue;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      f32x16_t s, dp;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        s[r] = 0.f;
        dp[r] = 0.f;
      }
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) {
        const bf16x8_t ka = __builtin_bit_cast(
            bf16x8_t, *reinterpret_cast<const u32x4*>(Ks + (ks * 32 + l32) * KLD + kk * 16 + half * 8));
        const bf16x8_t va = __builtin_bit_cast(
            bf16x8_t, *reinterpret_cast<const u32x4*>(Vs + (ks * 32 + l32) * KLD + kk * 16 + half * 8));
        s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qf[kk], s, 0, 0, 0);
        dp = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, df[kk], dp, 0, 0, 0);
      }
      // s[r], dp[r]: key j0 + 32 ks + 8 (r/4) + 4 half + r%4, query qrow
      const bool edge = j0 + BKEY > n || (causal && j0 + BKEY - 1 > wave_q0);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float p = __builtin_amdgcn_exp2f(fmaf(s[r], scale_log2, -Lq));
        if (edge) {
          const int j = j0 + ks * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
          if (j >= n || qrow >= n || (causal && j > qrow)) p = 0.f;
        }
        s[r] = p * (dp[r] - Dq);  // dS
      }
#pragma unroll
      for (int g4 = 0; g4 < 2; ++g4) {
        const int rb = 8 * g4;
        const u32x4 sw = {pack_bf16x2(s[rb], s[rb + 1]), pack_bf16x2(s[rb + 2], s[rb + 3]),
                          pack_bf16x2(s[rb + 4], s[rb + 5]), pack_bf16x2(s[rb + 6], s[rb + 7])};
        const bf16x8_t sb = __builtin_bit_cast(bf16x8_t, sw);
        const int base = ks * 32 + 16 * g4 + 4 * half;
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) {
          const bf16_t* kr = Kt + (ct * 32 + l32) * TLD + base;
          const uint2 a_lo = *reinterpret_cast<const uint2*>(kr);
          const uint2 a_hi = *reinterpret_cast<const uint2*>(kr + 8);
          const u32x4 av = {a_lo.x, a_lo.y, a_hi.x, a_hi.y};
          acc[ct] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, av), sb,
                                                             acc[ct], 0, 0, 0);
        }
      }
    }
  }
  // acc[ct][r] = dQ^T[channel ct*32 + 8 (r/4) + 4 half + r%4][query qrow] / scale
  __syncthreads();
  bf16_t* Os = reinterpret_cast<bf16_t*>(smem) + wave * 32 * OLD;
#pragma unroll
  for (int ct = 0; ct < CT; ++ct)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int c = ct * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
      Os[l32 * OLD + c] = f32_to_bf16(acc[ct][r] * scale);
    }
  __syncthreads();
  for (int c = lane; c < 32 * HD / 8; c += 64) {
    const int r = c / (HD / 8), ch = (c % (HD / 8)) * 8;
    const int q = q0 + wave * 32 + r;
    if (q < n)
      *reinterpret_cast<u32x4*>(dQ + static_cast<int64_t>(lo + q) * grs + h * HD + ch) =
          *reinterpret_cast<const u32x4*>(Os + r * OLD + ch);
  }
}

template <typename T>
hipError_t transpose_t(hipStream_t s, const void* in, int R, int C, int64_t ldi, void* out,
                       int Rpad) {
  const dim3 grid((C + 31) / 32, (Rpad + 31) / 32);
  return launch(K_MISC, transpose_kernel<T>, grid, dim3(256), 0, s, static_cast<const T*>(in), R,
                C, ldi, static_cast<T*>(out), Rpad);
}

}  // namespace

bool backward_supported(int dtype, int hd) { return dtype == 1 && (hd == 64 || hd == 128); }

hipError_t launch_transpose(hipStream_t s, int dtype, const void* in, int R, int C, int64_t ldi,
                            void* out, int Rpad) {
  if (C == 0 || Rpad == 0) return hipSuccess;
  if (dtype == 1 && ldi % 8 == 0 && Rpad % 8 == 0)
    return launch(K_MISC, transpose64_kernel, dim3((C + 63) / 64, (Rpad + 63) / 64), dim3(256), 0,
                  s, static_cast<const bf16_t*>(in), R, C, ldi, static_cast<bf16_t*>(out), Rpad);
  return dtype == 1 ? transpose_t<bf16_t>(s, in, R, C, ldi, out, Rpad)
                    : transpose_t<float>(s, in, R, C, ldi, out, Rpad);
}

size_t colsum_scratch_floats(int R, int C) {
  size_t f = 0;
  for (int rows = R; rows > kColRows;) {
    rows = (rows + kColRows - 1) / kColRows;
    f += static_cast<size_t>(rows) * C;
  }
  return f + C;
}

// passes of 64x row reduction (fixed order) until one row is left; the
// first pass reads the input (times xhat when x is given), the others the
// fp32 partial rows of the previous pass
hipError_t launch_colsum(hipStream_t s, int dtype, const void* a, int64_t lda, const void* x,
                         int64_t ldx, const float* stats, int R, int C, float* scratch,
                         float* out) {
  if (C == 0) return hipSuccess;
  if (R == 0)
    return launch(K_MISC, zero_f32_kernel, dim3((C + 255) / 256), dim3(256), 0, s, out, C);
  const dim3 block(256);
  int rows = R;
  bool first = true;
  const float* src = nullptr;
  float* dst = scratch;
  while (true) {
    const int chunks = (rows + kColRows - 1) / kColRows;
    float* target = chunks == 1 ? out : dst;
    const dim3 grid((C + 255) / 256, chunks);  // 32 column groups of 8 per block
    hipError_t e;
    if (first && dtype == 1)
      e = launch(K_MISC, colsum_stage1<bf16_t>, grid, block, 0, s, static_cast<const bf16_t*>(a),
                 lda, static_cast<const bf16_t*>(x), ldx, stats, rows, C, target);
    else if (first)
      e = launch(K_MISC, colsum_stage1<float>, grid, block, 0, s, static_cast<const float*>(a),
                 lda, static_cast<const float*>(x), ldx, stats, rows, C, target);
    else
      e = launch(K_MISC, colsum_stage1<float>, grid, block, 0, s, src, static_cast<int64_t>(C),
                 static_cast<const float*>(nullptr), static_cast<int64_t>(0), nullptr, rows, C,
                 target);
    if (e != hipSuccess || chunks == 1) return e;
    first = false;
    src = dst;
    dst += static_cast<size_t>(chunks) * C;
    rows = chunks;
  }
}

template <typename T, int RMS>
static hipError_t norm_bwd_nc(hipStream_t s, const void* x, const void* g, const void* dh,
                              const void* res, void* out, int R, int d, float eps, float* stats) {
  const dim3 grid((R + 3) / 4), block(256);
  auto* xp = static_cast<const T*>(x);
  auto* gp = static_cast<const T*>(g);
  auto* dp = static_cast<const T*>(dh);
  auto* rp = static_cast<const T*>(res);
  auto* op = static_cast<T*>(out);
  const int nc = (d + 511) / 512;
  if (nc <= 1) return launch(K_NORM, norm_bwd_kernel<T, RMS, 1>, grid, block, 0, s, xp, gp, dp, rp, op, R, d, eps, stats);
  if (nc <= 2) return launch(K_NORM, norm_bwd_kernel<T, RMS, 2>, grid, block, 0, s, xp, gp, dp, rp, op, R, d, eps, stats);
  if (nc <= 4) return launch(K_NORM, norm_bwd_kernel<T, RMS, 4>, grid, block, 0, s, xp, gp, dp, rp, op, R, d, eps, stats);
  if (nc <= 8) return launch(K_NORM, norm_bwd_kernel<T, RMS, 8>, grid, block, 0, s, xp, gp, dp, rp, op, R, d, eps, stats);
  return launch(K_NORM, norm_bwd_kernel<T, RMS, 16>, grid, block, 0, s, xp, gp, dp, rp, op, R, d, eps, stats);
}

hipError_t launch_norm_bwd(hipStream_t s, int dtype, int kind, const void* x, const void* g,
                           const void* dh, const void* res, void* out, int R, int d, float eps,
                           float* stats) {
  if (R == 0) return hipSuccess;
  if (d % 8 != 0 || d > 16 * 512) return hipErrorInvalidValue;
  if (dtype == 1)
    return kind == 1 ? norm_bwd_nc<bf16_t, 1>(s, x, g, dh, res, out, R, d, eps, stats)
                     : norm_bwd_nc<bf16_t, 0>(s, x, g, dh, res, out, R, d, eps, stats);
  return kind == 1 ? norm_bwd_nc<float, 1>(s, x, g, dh, res, out, R, d, eps, stats)
                   : norm_bwd_nc<float, 0>(s, x, g, dh, res, out, R, d, eps, stats);
}

hipError_t launch_act_bwd(hipStream_t s, int dtype, const void* dF, const void* u, void* du,
                          int rows, int F, int swiglu) {
  const int64_t total = static_cast<int64_t>(rows) * F;
  if (total == 0) return hipSuccess;
  const dim3 grid(static_cast<unsigned>((total / 8 + 255) / 256));  // F % 8 == 0
  if (dtype == 1)
    return launch(K_MISC, act_bwd_kernel<bf16_t>, grid, dim3(256), 0, s,
                  static_cast<const bf16_t*>(dF), static_cast<const bf16_t*>(u),
                  static_cast<bf16_t*>(du), static_cast<int64_t>(rows), F, swiglu);
  return launch(K_MISC, act_bwd_kernel<float>, grid, dim3(256), 0, s,
                static_cast<const float*>(dF), static_cast<const float*>(u),
                static_cast<float*>(du), static_cast<int64_t>(rows), F, swiglu);
}

hipError_t launch_act_fwd(hipStream_t s, int dtype, const void* u, void* f, int rows, int F,
                          int swiglu) {
  const int64_t total = static_cast<int64_t>(rows) * F;
  if (total == 0) return hipSuccess;
  const dim3 grid(static_cast<unsigned>((total / 8 + 255) / 256));  // F % 8 == 0
  if (dtype == 1)
    return launch(K_MISC, act_fwd_kernel<bf16_t>, grid, dim3(256), 0, s,
                  static_cast<const bf16_t*>(u), static_cast<bf16_t*>(f),
                  static_cast<int64_t>(rows), F, swiglu);
  return launch(K_MISC, act_fwd_kernel<float>, grid, dim3(256), 0, s, static_cast<const float*>(u),
                static_cast<float*>(f), static_cast<int64_t>(rows), F, swiglu);
}

hipError_t launch_scatter_rows(hipStream_t s, int dtype, int d, const void* src,
                               const int32_t* kept, int t_out, int t_in, int32_t* inv,
                               void* dst) {
  if (t_in == 0) return hipSuccess;
  hipError_t e = launch(K_MISC, fill_i32_kernel, dim3((t_in + 255) / 256), dim3(256), 0, s, inv,
                        t_in, -1);
  if (e != hipSuccess) return e;
  if (t_out > 0) {
    e = launch(K_MISC, inverse_index_kernel, dim3((t_out + 255) / 256), dim3(256), 0, s, kept,
               t_out, t_in, inv);
    if (e != hipSuccess) return e;
  }
  const int cpr = d * (dtype == 1 ? 2 : 4) / 16;
  const int64_t total = static_cast<int64_t>(t_in) * cpr;
  return launch(K_MISC, scatter_rows_kernel, dim3(static_cast<unsigned>((total + 255) / 256)),
                dim3(256), 0, s, static_cast<const uint4*>(src), inv, t_in, cpr,
                static_cast<uint4*>(dst));
}

hipError_t launch_rowdot(hipStream_t s, int dtype, const void* dO, const void* O, int64_t ld,
                         int T, int H, int hd, float* D) {
  const int L = hd / 8;
  if (hd % 8 != 0 || L > 64 || (L & (L - 1)) != 0) return hipErrorInvalidValue;
  const int64_t total = static_cast<int64_t>(T) * H * L;
  if (total == 0) return hipSuccess;
  const dim3 grid(static_cast<unsigned>((total + 255) / 256));
  if (dtype == 1)
    return launch(K_MISC, rowdot_kernel<bf16_t>, grid, dim3(256), 0, s,
                  static_cast<const bf16_t*>(dO), static_cast<const bf16_t*>(O), ld, T, H, hd, D);
  return launch(K_MISC, rowdot_kernel<float>, grid, dim3(256), 0, s, static_cast<const float*>(dO),
                static_cast<const float*>(O), ld, T, H, hd, D);
}

hipError_t launch_rope_bwd(hipStream_t s, int dtype, void* g, int64_t ld, int rows, int cols,
                           int hd, const int32_t* pos, const EpiParams& ep) {
  const int64_t total = static_cast<int64_t>(rows) * (cols / 2);
  if (total == 0) return hipSuccess;
  const dim3 grid(static_cast<unsigned>((total + 255) / 256));
  if (dtype == 1)
    return launch(K_MISC, rope_bwd_kernel<bf16_t>, grid, dim3(256), 0, s, static_cast<bf16_t*>(g),
                  ld, rows, cols, hd, pos, ep);
  return launch(K_MISC, rope_bwd_kernel<float>, grid, dim3(256), 0, s, static_cast<float*>(g), ld,
                rows, cols, hd, pos, ep);
}

hipError_t launch_attention_bwd(hipStream_t s, const void* q, const void* k, const void* v,
                                int64_t rs, const void* dO, int64_t ors, const float* lse,
                                const float* D, int H, int kv_group, int hd, int causal,
                                float scale, int B, int max_len, int T, const int32_t* cu_dev,
                                void* dq, void* dk, void* dv, int64_t grs) {
  if (B == 0 || max_len == 0) return hipSuccess;
  const float sl = scale * kLog2e;
  auto* qp = static_cast<const bf16_t*>(q);
  auto* kp = static_cast<const bf16_t*>(k);
  auto* vp = static_cast<const bf16_t*>(v);
  auto* dp = static_cast<const bf16_t*>(dO);
  const int Hkv = H / kv_group;
  hipError_t e;
  if (hd == 64) {
    e = launch(K_ATTENTION, attn_bwd_dkdv_kernel<64>, dim3((max_len + 127) / 128, Hkv, B),
               dim3(256), 0, s, qp, kp, vp, rs, dp, ors, lse, D, T, kv_group, causal, scale, sl,
               cu_dev, static_cast<bf16_t*>(dk), static_cast<bf16_t*>(dv), grs);
    if (e != hipSuccess) return e;
    return launch(K_ATTENTION, attn_bwd_dq_kernel<64>, dim3((max_len + 127) / 128, H, B),
                  dim3(256), 0, s, qp, kp, vp, rs, dp, ors, lse, D, T, kv_group, causal, scale, sl,
                  cu_dev, static_cast<bf16_t*>(dq), grs);
  }
  e = launch(K_ATTENTION, attn_bwd_dkdv_kernel<128>, dim3((max_len + 127) / 128, Hkv, B),
             dim3(256), 0, s, qp, kp, vp, rs, dp, ors, lse, D, T, kv_group, causal, scale, sl,
             cu_dev, static_cast<bf16_t*>(dk), static_cast<bf16_t*>(dv), grs);
  if (e != hipSuccess) return e;
  return launch(K_ATTENTION, attn_bwd_dq_kernel<128>, dim3((max_len + 127) / 128, H, B),
                dim3(256), 0, s, qp, kp, vp, rs, dp, ors, lse, D, T, kv_group, causal, scale, sl,
                cu_dev, static_cast<bf16_t*>(dq), grs);
}

}  // namespace zsa
