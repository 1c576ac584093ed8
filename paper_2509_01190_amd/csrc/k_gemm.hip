// Projections of the pre-norm block: y = epilogue(x W^T + bias).
//
// x [M, K] and W [N, K] are both K-contiguous ("NT" GEMM, PyTorch Linear
// layout), so every MFMA operand fragment is one 16-byte run of 8
// consecutive K values from a row of x or of W.
//
// bf16 kernels, fp32 accumulation, chosen by shape in launch_gemm:
//  * gemm_bf16_dma_kernel: 128x128 tiles on 4 waves or 256x256 on 8, K
//    slices loaded straight into swizzled LDS stages; split K for short
//    grids, the slices summed in slice order by splitk_reduce_kernel;
//  * gemm_bf16_persist_kernel: 128x128 tiles, two workgroups per CU walking
//    their XCD's range of tiles, the epilogue from registers;
//  * gemm_bf16_w4p_kernel: 256x256 or 256x192 tiles on four waves (one per
//    SIMD), one workgroup per CU streaming the K slices of its tiles as one
//    sequence (products whose tiles fill their rounds on the CUs,
//    w4p_width); the GELU and SwiGLU epilogues store from registers, the
//    others whole lines through a per-wave LDS staging buffer;
//  * gemm_bf16_w4_kernel: its slice loop with one tile per workgroup (a
//    tuning baseline, ZSA_GEMM_TILE);
//  * gemm_skinny_kernel: products of at most 16 rows, and of up to 1024
//    rows whose 128x128 tiles would number under 64 (generation and short
//    pruned layers): no shared tiles, operands loaded in whole cache lines
//    and passed through a per-wave LDS buffer into
//    v_mfma_f32_16x16x32_bf16 fragments;
//  * gemm_bf16_mfma_kernel: the register-staged 128x128 original, kept as a
//    tuning baseline (ZSA_GEMM_TILE).
// The others use v_mfma_f32_32x32x16_bf16. fp32 storage: a 64x128
// vector-ALU tile (4x8 outputs per thread).
//
// Epilogues (same order and precision in every kernel that takes them):
// bias, exact GELU, SwiGLU on interleaved gate/up columns, residual add, or
// the rotary rotation of head channel pairs (i, i+hd/2) -- the last in the
// direct-to-LDS, register-staged and few-row kernels, and (angles from a
// per-row table) in the persistent four-wave kernel.
#include <math.h>
#include <stdlib.h>

#include <algorithm>
#include <type_traits>

#include "zsa_internal.h"

namespace zsa {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

// the persistent four-wave kernel's rotary epilogue for head_dim 128 (its
// EPI_ROPE instance serves head_dim 64)
constexpr int kEpiRope128 = 5;

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

// Exact (erf-based) GELU, z Phi(z) = z (1 + erf(z / sqrt 2)) / 2, with erf by
// Abramowitz & Stegun, Handbook of Mathematical Functions, 7.1.26:
// erf(x) = 1 - P(t) exp(-x^2), P(t) = a1 t + a2 t^2 + a3 t^3 + a4 t^4 + a5 t^5,
// t = 1 / (1 + p x), x >= 0, |error| <= 1.5e-7, and erf odd. Oddness gives
// z Phi(z) = max(z, 0) - |z| P(t) exp(-z^2 / 2) / 2 for either sign of z
// (t formed from |z| / sqrt 2): one fma instead of a sign transfer and the
// (1 + erf) / 2 scaling, with the 1/2 folded into the coefficients and the
// 1/sqrt 2 into p.
__device__ __forceinline__ float gelu_erf(float z) {
  const float a = fabsf(z);
  const float t = __builtin_amdgcn_rcpf(fmaf(0.3275911f * 0.70710678118654752f, a, 1.0f));
  const float hp =
      t * (0.5f * 0.254829592f +
           t * (0.5f * -0.284496736f +
                t * (0.5f * 1.421413741f + t * (0.5f * -1.453152027f + t * (0.5f * 1.061405429f)))));
  return fmaf(-a * hp, __expf(-0.5f * z * z), fmaxf(z, 0.0f));
}
// z sigmoid(z) = z / (1 + 2^(-z log2 e)) from the hardware exp2 and
// reciprocal, made as accurate as the library exp with an IEEE division:
// the exponent is formed with its rounding error (one fma) and the error of
// log2 e's fp32 value, which then scale the exp2 result to first order
// (2^(p + dp) = 2^p (1 + dp ln 2)), and one Newton step refines the
// reciprocal's quotient. Against float64 over 2^20 inputs in [-100, 100]
// (measured on gfx950): at most 3.0 ulp (mean 0.37) and 6 bf16 roundings in
// 10^6 different from the exact value's, as for the library form (2.3 ulp,
// 0.35, 6); the plain hardware pair reached 60 ulp and 30. About 10 vector
// instructions instead of about 30 (the SwiGLU epilogue was a fifth of a
// 2048-deep tile's time). Below z = -88.7 (2^p overflows) the result is -0,
// as z / (1 + inf) is.
__device__ __forceinline__ float silu(float z) {
  constexpr float kL2e = 1.44269502f;         // fp32(log2 e)
  constexpr float kL2eLo = 1.925963033e-08f;  // log2 e - kL2e
  constexpr float kLn2f = 0.693147182f;
  const float p = -z * kL2e;
  const float dp = fmaf(-z, kL2e, -p) - z * kL2eLo;  // p + dp = -z log2 e
  float e = __builtin_amdgcn_exp2f(p);
  e = fmaf(e, dp * kLn2f, e);
  const float d = 1.0f + e;
  const float r = __builtin_amdgcn_rcpf(d);
  float q = z * r;
  q = fmaf(r, fmaf(-d, q, z), q);
  return p >= 128.0f ? z * 0.0f : q;
}

// tile: fp32 [BM][ldt] in LDS holding (x W^T) for rows m0.., columns n0..
template <typename T, int BM, int BN, int NT>
__device__ void epilogue_tile(const float* tile, int ldt, int m0, int n0, int M, int N,
                              const EpiParams& ep) {
  const T* bias = static_cast<const T*>(ep.bias);
  T* y = static_cast<T*>(ep.y);
  const int tid = threadIdx.x;
  if (ep.epi == EPI_SWIGLU) {
    constexpr int OPR = BN / 2 / 8;  // 8-wide output items per row
    for (int it = tid; it < BM * OPR; it += NT) {
      const int r = it / OPR;
      const int cv = it - r * OPR;
      const int m = m0 + r;
      const int oc = n0 / 2 + cv * 8;
      if (m >= M || oc >= N / 2) continue;
      float out[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int zc = 2 * (cv * 8 + e);
        float g = tile[r * ldt + zc];
        float u = tile[r * ldt + zc + 1];
        if (bias != nullptr) {
          g += to_f32(bias[n0 + zc]);
          u += to_f32(bias[n0 + zc + 1]);
        }
        out[e] = silu(g) * u;
      }
      store8<T>(y + static_cast<int64_t>(m) * ep.ldy + oc, out);
    }
    return;
  }
  constexpr int IPR = BN / 8;
  const int hd = ep.head_dim;
  const int half = hd >> 1;
  for (int it = tid; it < BM * IPR; it += NT) {
    const int r = it / IPR;
    const int cv = it - r * IPR;
    const int m = m0 + r;
    const int n = n0 + cv * 8;
    if (m >= M || n >= N) continue;
    float z[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) z[e] = tile[r * ldt + cv * 8 + e];
    if (bias != nullptr) {
      float bv[8];
      load8<T>(bias + n, bv);
#pragma unroll
      for (int e = 0; e < 8; ++e) z[e] += bv[e];
    }
    if (ep.epi == EPI_GELU) {
#pragma unroll
      for (int e = 0; e < 8; ++e) z[e] = gelu_erf(z[e]);
    } else if (ep.epi == EPI_RESIDUAL) {
      float rv[8];
      load8<T>(static_cast<const T*>(ep.residual) + static_cast<int64_t>(m) * ep.ldy + n, rv);
#pragma unroll
      for (int e = 0; e < 8; ++e) z[e] += rv[e];
    } else if (ep.epi == EPI_ROPE && n < ep.rope_cols) {
      const int p = ep.pos[m];
      const int c0 = n % hd;  // head-local channel of the first of the 8 outputs
      const bool lower = c0 < half;
      const int pcol = cv * 8 + (lower ? half : -half);  // partner columns in the tile
      float pb[8];
      if (bias != nullptr) {
        load8<T>(bias + n + (lower ? half : -half), pb);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) pb[e] = 0.f;
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float zp = tile[r * ldt + pcol + e] + pb[e];
        const int i = (c0 + e) - (lower ? 0 : half);
        float sn, cs;
        if (ep.rope_cs != nullptr) {
          const float2 t = reinterpret_cast<const float2*>(ep.rope_cs)[static_cast<int64_t>(m) * half + i];
          cs = t.x;
          sn = t.y;
        } else {
          rope_angle(p, ep.inv_freq[i], &sn, &cs);
        }
        z[e] = lower ? (z[e] * cs - zp * sn) : (z[e] * cs + zp * sn);
      }
    }
    store8<T>(y + static_cast<int64_t>(m) * ep.ldy + n, z);
  }
}

// ---------------------------------------------------------------------------
// bf16 MFMA GEMM
// ---------------------------------------------------------------------------
constexpr int kBK = 64, kLDK = kBK + 8;  // K step; padded LDS row (bf16)
constexpr int kMinSplitSteps = 4;          // K steps per split-K slice, at least
constexpr int kMinSplitK = 1024;           // shortest K that is split

// fp32 epilogue tile: 128 rows of BN columns, row stride BN + 4
template <int BM, int BN>
constexpr int mfma_lds_bytes() {
  return 2 * (BM + BN) * kLDK * 2 > 128 * (BN + 4) * 4 ? 2 * (BM + BN) * kLDK * 2
                                                        : 128 * (BN + 4) * 4;
}

// BM x BN output tile, WM x WN waves, each wave (BM/WM) x (BN/WN) made of
// 32x32 MFMA tiles. The operand staging arrays are indexed only by
// unrolled constants so they stay in VGPRs, and the next K step's global
// loads are issued before this step's MFMAs so their latency is hidden.
template <int BM, int BN, int WM, int WN>
__global__ __launch_bounds__(WM * WN * 64) void gemm_bf16_mfma_kernel(
    const bf16_t* __restrict__ X, const bf16_t* __restrict__ W, int M, int N, int K,
    EpiParams ep) {
  static_assert(BM % 128 == 0 && (BN == 128 || BN == 256), "tile shape");
  constexpr int NT = WM * WN * 64;
  constexpr int kTileLd = BN + 4;
  constexpr int WTM = BM / WM, WTN = BN / WN;
  constexpr int TM = WTM / 32, TN = WTN / 32;
  constexpr int RPP = NT / 8;                 // rows covered by one pass of 16-byte chunks
  constexpr int ACH = BM / RPP, BCH = BN / RPP;
  extern __shared__ __align__(16) unsigned char smem[];
  bf16_t* As = reinterpret_cast<bf16_t*>(smem);  // [2][BM][kLDK]
  bf16_t* Bs = As + 2 * BM * kLDK;               // [2][BN][kLDK]
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int m0 = blockIdx.x * BM;
  const int n0 = blockIdx.y * BN;
  const int lrow = tid >> 3, lkc = (tid & 7) * 8;

  // Rows past M (or N) are clamped to the last row instead of zeroed: they
  // only feed output rows (columns) that are never stored, and a mask
  // applied at load time would make the loads wait before the MFMAs.
  const bf16_t* xp[ACH];
#pragma unroll
  for (int i = 0; i < ACH; ++i)
    xp[i] = X + static_cast<int64_t>(min(m0 + lrow + i * RPP, M - 1)) * K + lkc;
  const bf16_t* wp[BCH];
#pragma unroll
  for (int i = 0; i < BCH; ++i)
    wp[i] = W + static_cast<int64_t>(min(n0 + lrow + i * RPP, N - 1)) * K + lkc;
  u32x4 ra[ACH], rb[BCH];

#define ZSA_GLOAD(k0)                                                              \
  _Pragma("unroll") for (int i = 0; i < ACH; ++i) {                                \
    ra[i] = *reinterpret_cast<const u32x4*>(xp[i] + (k0));                         \
  }                                                                                \
  _Pragma("unroll") for (int i = 0; i < BCH; ++i) {                                \
    rb[i] = *reinterpret_cast<const u32x4*>(wp[i] + (k0));                         \
  }
#define ZSA_SSTORE(buf)                                                            \
  _Pragma("unroll") for (int i = 0; i < ACH; ++i)                                  \
    *reinterpret_cast<u32x4*>(As + ((buf) * BM + lrow + i * RPP) * kLDK + lkc) = ra[i]; \
  _Pragma("unroll") for (int i = 0; i < BCH; ++i)                                  \
    *reinterpret_cast<u32x4*>(Bs + ((buf) * BN + lrow + i * RPP) * kLDK + lkc) = rb[i];

  f32x16_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  const int KT = K / kBK;
  ZSA_GLOAD(0)
  ZSA_SSTORE(0)
  __syncthreads();
  for (int kt = 0; kt < KT; ++kt) {
    const int buf = kt & 1;
    const bool more = kt + 1 < KT;
    if (more) {
      ZSA_GLOAD((kt + 1) * kBK)
    }
    const bf16_t* Ab = As + (buf * BM + wm * WTM + (lane & 31)) * kLDK + (lane >> 5) * 8;
    const bf16_t* Bb = Bs + (buf * BN + wn * WTN + (lane & 31)) * kLDK + (lane >> 5) * 8;
#pragma unroll
    for (int kk = 0; kk < kBK / 16; ++kk) {
      bf16x8_t a[TM], b[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i)
        a[i] = __builtin_bit_cast(bf16x8_t,
                                  *reinterpret_cast<const u32x4*>(Ab + i * 32 * kLDK + kk * 16));
#pragma unroll
      for (int j = 0; j < TN; ++j)
        b[j] = __builtin_bit_cast(bf16x8_t,
                                  *reinterpret_cast<const u32x4*>(Bb + j * 32 * kLDK + kk * 16));
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
    if (more) {
      ZSA_SSTORE(buf ^ 1)
    }
    __syncthreads();
  }
#undef ZSA_GLOAD
#undef ZSA_SSTORE

  // accumulator layout of a 32x32 MFMA tile: lane l, register r holds
  // row 8*(r/4) + 4*(l/32) + r%4, column l%32. The fp32 tile is staged
  // through LDS 128 rows at a time.
  float* tile = reinterpret_cast<float*>(smem);
#pragma unroll
  for (int pass = 0; pass < BM / 128; ++pass) {
    if (pass > 0) __syncthreads();
    if ((wm * WTM) / 128 == pass) {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int row = wm * WTM - pass * 128 + i * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
            const int col = wn * WTN + j * 32 + (lane & 31);
            tile[row * kTileLd + col] = acc[i][j][r];
          }
    }
    __syncthreads();
    epilogue_tile<bf16_t, 128, BN, NT>(tile, kTileLd, m0 + pass * 128, n0, M, N, ep);
  }
}

// ---------------------------------------------------------------------------
// XCD-aware tile order
// ---------------------------------------------------------------------------
// Workgroups are handed to the 8 XCDs round-robin by linear id, and every XCD
// has its own L2. Workgroup L therefore runs on XCD k = L % 8 as that XCD's
// j-th workgroup (j = L / 8). The output tiles are put in a grouped order --
// groups of kXcdGroup M-tiles, and within a group every N-tile with the
// group's M-tiles inner -- and XCD k takes a contiguous, balanced range of
// that order. Neighbouring tiles of the order share A rows or W columns, so
// a range's operands are fetched from memory about once into its XCD's L2;
// and since the ranges split the tiles, not the M-tiles, all 8 XCDs work
// even when there is a single M-tile (short inputs, decoding). The grid is
// 8 x (largest range) one-dimensional workgroups; the ones past their range
// exit.
constexpr int kXcds = 8;
constexpr int kXcdGroup = 8;

template <int BM, int BN>
__device__ __forceinline__ bool xcd_tile(int M, int N, int* mt, int* nt) {
  const int nM = (M + BM - 1) / BM, nN = (N + BN - 1) / BN;
  const int k = blockIdx.x % kXcds, j = blockIdx.x / kXcds;
  const int tiles = nM * nN;
  const int per = tiles / kXcds, extra = tiles % kXcds;
  if (j >= per + (k < extra ? 1 : 0)) return false;
  const int t = k * per + min(k, extra) + j;  // position in the grouped order
  const int g = t / (kXcdGroup * nN);
  const int gm0 = g * kXcdGroup;
  const int gsz = min(kXcdGroup, nM - gm0);
  const int r = t - g * kXcdGroup * nN;
  *nt = r / gsz;
  *mt = gm0 + r % gsz;
  return true;
}

inline dim3 xcd_grid(int M, int N, int BM, int BN) {
  const int tiles = ((M + BM - 1) / BM) * ((N + BN - 1) / BN);
  return dim3(static_cast<unsigned>(kXcds * ((tiles + kXcds - 1) / kXcds)));
}

// Stores from the accumulators. The operand-swapped 32x32 MFMA leaves lane l
// (half h = l / 32) with four consecutive columns 8g + 4h .. 8g + 4h + 3 of
// row l % 32 of its 32 x 32 block in register group g, 8 bytes. A
// v_permlane32_swap of each dword of groups g and g + 1 (g even) exchanges
// the upper lanes' group-g words with the lower lanes' group-(g + 1) words:
// the lower lanes then hold all eight columns of group g and the upper lanes
// those of group g + 1, so each lane stores 16 contiguous bytes and one store
// instruction covers 32 bytes of each of 32 rows (half as many stores as
// 8-byte ones). A residual is read the same way and swapped back.
__device__ __forceinline__ void lane_swap(uint32_t& lo, uint32_t& hi) {
  const auto r = __builtin_amdgcn_permlane32_swap(lo, hi, false, false);
  lo = r[0];
  hi = r[1];
}

// residual of columns nc .. nc + 31 of row m: r[p] = the 16 bytes at column
// nc + (2p + half) * 8, as loaded (res_epilogue32 swaps them)
__device__ __forceinline__ void res_load32(__amdgpu_buffer_rsrc_t rres, uint32_t m, int nc, int half,
                                           int ldy, uint32_t (&r)[2][4]) {
#pragma unroll
  for (int p = 0; p < 2; ++p) {
    const auto v = __builtin_amdgcn_raw_buffer_load_b128(
        rres, (m * static_cast<uint32_t>(ldy) + static_cast<uint32_t>(nc + (2 * p + half) * 8)) * 2u, 0, 0);
    r[p][0] = v[0];
    r[p][1] = v[1];
    r[p][2] = v[2];
    r[p][3] = v[3];
  }
}

// finished bf16 values of one 32 x 32 accumulator block (this lane's row,
// columns nc .. nc + 31; bw[g] = the bias of the lane's four columns of group
// g): v[p] = the 16 bytes of columns nc + (2p + half) * 8 .. + 7; for SwiGLU
// v[p].x, .y = the 8 bytes of output columns nc / 2 + 8p + 4 half .. + 3
template <int EPI>
__device__ __forceinline__ void epi_pack32(const f32x16_t& a, const uint2 (&bw)[4], uint32_t (&r)[2][4],
                                           u32x4 (&v)[2]) {
  if (EPI == EPI_SWIGLU) {
    // gate and up on columns 2c, 2c + 1: a lane's four columns of group g
    // give outputs nc / 2 + 4g + 2 half (+1); after the swap of groups 2p
    // and 2p + 1 the lower lanes hold outputs nc / 2 + 8p .. + 3 and the
    // upper lanes the next four, 8 bytes each (ldy is the output width)
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      uint32_t pk[2];
#pragma unroll
      for (int gg = 0; gg < 2; ++gg) {
        const int g = 2 * p + gg;
        const float z0 = a[4 * g + 0] + __uint_as_float(bw[g].x << 16);
        const float z1 = a[4 * g + 1] + __uint_as_float(bw[g].x & 0xffff0000u);
        const float z2 = a[4 * g + 2] + __uint_as_float(bw[g].y << 16);
        const float z3 = a[4 * g + 3] + __uint_as_float(bw[g].y & 0xffff0000u);
        pk[gg] = pack_bf16x2(silu(z0) * z1, silu(z2) * z3);
      }
      lane_swap(pk[0], pk[1]);
      v[p] = u32x4{pk[0], pk[1], 0u, 0u};
    }
    return;
  }
#pragma unroll
  for (int p = 0; p < 2; ++p) {
    if (EPI == EPI_RESIDUAL) {
      lane_swap(r[p][0], r[p][2]);
      lane_swap(r[p][1], r[p][3]);
    }
    uint32_t pk[2][2];
#pragma unroll
    for (int gg = 0; gg < 2; ++gg) {
      const int g = 2 * p + gg;
      float z[4];
      z[0] = a[4 * g + 0] + __uint_as_float(bw[g].x << 16);
      z[1] = a[4 * g + 1] + __uint_as_float(bw[g].x & 0xffff0000u);
      z[2] = a[4 * g + 2] + __uint_as_float(bw[g].y << 16);
      z[3] = a[4 * g + 3] + __uint_as_float(bw[g].y & 0xffff0000u);
      if (EPI == EPI_GELU) {
#pragma unroll
        for (int e = 0; e < 4; ++e) z[e] = gelu_erf(z[e]);
      } else if (EPI == EPI_RESIDUAL) {
        z[0] += __uint_as_float(r[p][2 * gg] << 16);
        z[1] += __uint_as_float(r[p][2 * gg] & 0xffff0000u);
        z[2] += __uint_as_float(r[p][2 * gg + 1] << 16);
        z[3] += __uint_as_float(r[p][2 * gg + 1] & 0xffff0000u);
      }
      pk[gg][0] = pack_bf16x2(z[0], z[1]);
      pk[gg][1] = pack_bf16x2(z[2], z[3]);
    }
    lane_swap(pk[0][0], pk[1][0]);
    lane_swap(pk[0][1], pk[1][1]);
    v[p] = u32x4{pk[0][0], pk[0][1], pk[1][0], pk[1][1]};
  }
}

// epilogue of one 32 x 32 accumulator block stored straight from the
// registers: rows m (this lane's), columns nc .. nc + 31
template <int EPI>
__device__ __forceinline__ void epi_store32(const f32x16_t& a, const uint2 (&bw)[4], uint32_t (&r)[2][4],
                                            __amdgpu_buffer_rsrc_t yres, uint32_t m, int nc, int half,
                                            int ldy) {
  u32x4 v[2];
  epi_pack32<EPI>(a, bw, r, v);
#pragma unroll
  for (int p = 0; p < 2; ++p) {
    if (EPI == EPI_SWIGLU) {
      typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
      const u32x2 w = {v[p][0], v[p][1]};
      __builtin_amdgcn_raw_buffer_store_b64(
          w, yres, (m * static_cast<uint32_t>(ldy) + static_cast<uint32_t>(nc / 2 + 8 * p + 4 * half)) * 2u,
          0, 0);
    } else {
      __builtin_amdgcn_raw_buffer_store_b128(
          v[p], yres, (m * static_cast<uint32_t>(ldy) + static_cast<uint32_t>(nc + (2 * p + half) * 8)) * 2u,
          0, 0);
    }
  }
}

// Epilogue from the accumulators of a wave whose block starts at row mb,
// column nb: acc[i][j][4g + e] = C[m][n + e], m = mb + 32 i + l32,
// n = nb + 32 j + 8 g + 4 half (the operand-swapped MFMA holds C^T); bias,
// GELU or residual, then raw buffer stores, whose range check drops rows
// past M. N is a multiple of the wave's column block.
template <int TM, int TN, int EPI>
__device__ __forceinline__ void reg_epilogue(const f32x16_t (&acc)[TM][TN], int mb, int nb, int M,
                                             int l32, int half, const EpiParams& ep) {
  const int ybytes = M * ep.ldy * 2;
  const __amdgpu_buffer_rsrc_t yres = __builtin_amdgcn_make_buffer_rsrc(ep.y, 0, ybytes, 0x00020000);
  const __amdgpu_buffer_rsrc_t rres = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<void*>(EPI == EPI_RESIDUAL ? ep.residual : ep.y), 0, ybytes, 0x00020000);
  const bf16_t* bias = static_cast<const bf16_t*>(ep.bias);
  // Loads go ahead of stores -- every bias word first, each block's
  // residual before the previous block's stores: vector memory operations
  // are counted in issue order, so a load issued after a store could only
  // be waited for together with that store. One 32 x 32 block at a time
  // keeps the residual registers few.
  uint2 bw[TN][4];
#pragma unroll
  for (int j = 0; j < TN; ++j)
#pragma unroll
    for (int g = 0; g < 4; ++g)
      bw[j][g] = bias != nullptr
                     ? *reinterpret_cast<const uint2*>(bias + nb + j * 32 + g * 8 + half * 4)
                     : make_uint2(0u, 0u);
  uint32_t r[2][2][4];
  if (EPI == EPI_RESIDUAL) res_load32(rres, static_cast<uint32_t>(mb + l32), nb, half, ep.ldy, r[0]);
#pragma unroll
  for (int j = 0; j < TN; ++j) {
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int st = j * TM + i;
      if (EPI == EPI_RESIDUAL && st + 1 < TM * TN) {
        const int j1 = (st + 1) / TM, i1 = (st + 1) % TM;
        res_load32(rres, static_cast<uint32_t>(mb + i1 * 32 + l32), nb + j1 * 32, half, ep.ldy,
                   r[(st + 1) & 1]);
      }
      const uint32_t m = static_cast<uint32_t>(mb + i * 32 + l32);
      epi_store32<EPI>(acc[i][j], bw[j], r[st & 1], yres, m, nb + j * 32, half, ep.ldy);
    }
  }
}

// ---------------------------------------------------------------------------
// bf16 MFMA GEMM with direct-to-LDS operand loads
// ---------------------------------------------------------------------------
// global_load_lds_dwordx4 writes each lane's 16 bytes to LDS at
// (wave-uniform base) + 16 * lane, so one instruction fills 1 KiB of a tile
// whose rows are one K slice of KB bf16 (RB = 2 KB bytes): 1024 / RB rows.
// Tiles are stored unpadded with the 16-byte chunk c of row r at position
// c ^ ((r / RPP) & (CPR - 1)), where CPR = RB / 16 chunks make a row and
// RPP = 256 / RB rows share one 256-byte span of the 64 banks. The DMA
// writes stay contiguous, and the 16 lanes of an MFMA fragment read phase
// (16 consecutive rows, one logical chunk) land on 16 distinct 4-bank
// groups. Operands never pass through VGPRs.
//
// NS stages form a ring: the loads of K slice t + NS - 1 are issued at the
// top of step t, so NS - 1 slices are in flight while the MFMAs of slice t
// run. Each wave waits only for its own loads of slice t (vmcnt counts the
// later slices' loads as still outstanding), one barrier publishes the
// slice to the workgroup and also retires the stage the new loads reuse.
// The fp32 output tile is staged through LDS in passes of ER rows.
template <int KB>
struct Slice {
  static constexpr int RB = KB * 2;      // bytes per tile row
  static constexpr int CPR = RB / 16;    // 16-byte chunks per row
  static constexpr int RPD = 1024 / RB;  // rows per 1 KiB load instruction
  static constexpr int RPP = 256 / RB;   // rows per 256-byte bank span
};

template <int KB>
__device__ __forceinline__ int swz(int r, int c) {
  return c ^ ((r / Slice<KB>::RPP) & (Slice<KB>::CPR - 1));
}

template <int BM, int BN, int KB, int NS, int ER>
constexpr int dma_lds_bytes() {
  return NS * (BM + BN) * Slice<KB>::RB > ER * (BN + 4) * 4 ? NS * (BM + BN) * Slice<KB>::RB
                                                             : ER * (BN + 4) * 4;
}

// waves per SIMD the tile's LDS footprint allows (160 KiB per CU)
template <int BM, int BN, int WM, int WN, int KB, int NS, int ER>
constexpr int dma_waves_per_simd() {
  return (163840 / dma_lds_bytes<BM, BN, KB, NS, ER>()) * WM * WN / 4;
}

// s_waitcnt immediate: vector-memory count <= n, LDS/scalar and export counts 0
__device__ __forceinline__ constexpr int vmcnt_imm(int n) { return (n & 15) | ((n >> 4) << 14); }

// Workgroup barrier for the K pipeline. __syncthreads() carries a
// workgroup-scope release fence, for which the compiler waits on every
// outstanding global operation -- including the K slices meant to stay in
// flight. Here the DMA writes a wave depends on are covered by its explicit
// vmcnt wait before the barrier, its own LDS reads by the lgkmcnt wait, the
// asm memory clobber keeps the compiler from moving memory operations
// across it, and the scheduling barriers keep every other instruction
// (MFMAs included) on its side of it.
__device__ __forceinline__ void barrier_lds() {
  __builtin_amdgcn_sched_barrier(0);
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
}

template <int BM, int BN, int WM, int WN, int KB, int NS, int ER>
__global__ __launch_bounds__(WM * WN * 64)
__attribute__((amdgpu_waves_per_eu(dma_waves_per_simd<BM, BN, WM, WN, KB, NS, ER>(),
                                   dma_waves_per_simd<BM, BN, WM, WN, KB, NS, ER>()))) void
gemm_bf16_dma_kernel(
    const bf16_t* __restrict__ X, const bf16_t* __restrict__ W, int M, int N, int K,
    EpiParams ep, int kchunk, float* __restrict__ part) {
  static_assert(BM % 128 == 0 && (BN == 128 || BN == 256), "tile shape");
  static_assert((KB == 32 || KB == 64) && NS >= 2 && ER % 32 == 0 && BM % ER == 0, "pipeline");
  using SL = Slice<KB>;
  constexpr int NW = WM * WN;
  constexpr int NT = NW * 64;
  constexpr int kTileLd = BN + 4;
  constexpr int WTM = BM / WM, WTN = BN / WN;
  constexpr int TM = WTM / 32, TN = WTN / 32;
  constexpr int AI = BM / SL::RPD / NW, BI = BN / SL::RPD / NW;  // 1 KiB loads per wave
  static_assert(AI * NW * SL::RPD == BM && BI * NW * SL::RPD == BN, "loads per wave");
  constexpr int SB = (BM + BN) * SL::RB;  // bytes per stage: A rows, then B rows
  constexpr int KS = KB / 16;              // MFMA k-substeps per slice
  extern __shared__ __align__(16) unsigned char smem[];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  // wave index as a scalar: the DMA destinations derived from it are then
  // wave-uniform scalars (M0) instead of per-lane values read back each time
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WN, wn = wave % WN;
  int mt, nt;
  if (!xcd_tile<BM, BN>(M, N, &mt, &nt)) return;
  const int m0 = mt * BM;
  const int n0 = nt * BN;

  // split K: workgroup row y covers K columns [y * kchunk, y * kchunk + kchunk)
  const int kbeg = blockIdx.y * kchunk;
  const int KTOT = min(kchunk, K - kbeg) / KB;

  // per-lane global sources of this wave's loads (row clamped; the logical
  // chunk is the position un-swizzled for the destination row)
  const int lr = lane / SL::CPR, lp = lane % SL::CPR;
  const bf16_t* asrc[AI];
#pragma unroll
  for (int i = 0; i < AI; ++i) {
    const int r = (i * NW + wave) * SL::RPD + lr;
    asrc[i] = X + static_cast<int64_t>(min(m0 + r, M - 1)) * K + kbeg + swz<KB>(r, lp) * 8;
  }
  const bf16_t* bsrc[BI];
#pragma unroll
  for (int i = 0; i < BI; ++i) {
    const int r = (i * NW + wave) * SL::RPD + lr;
    bsrc[i] = W + static_cast<int64_t>(min(n0 + r, N - 1)) * K + kbeg + swz<KB>(r, lp) * 8;
  }
// the LDS-DMA builtin exists only in the device pass; the host pass only
// needs the kernel's launch stub
#if defined(__HIP_DEVICE_COMPILE__)
  typedef __attribute__((address_space(3))) void lds_void;
#define ZSA_DMA1(src, dst) __builtin_amdgcn_global_load_lds((src), (lds_void*)(dst), 16, 0, 0)
#else
#define ZSA_DMA1(src, dst) ((void)(src), (void)(dst))
#endif
#define ZSA_DMA(s, k0)                                                                   \
  _Pragma("unroll") for (int i = 0; i < AI; ++i)                                         \
    ZSA_DMA1(asrc[i] + (k0), smem + (s) * SB + (i * NW + wave) * 1024);                  \
  _Pragma("unroll") for (int i = 0; i < BI; ++i)                                         \
    ZSA_DMA1(bsrc[i] + (k0), smem + (s) * SB + BM * SL::RB + (i * NW + wave) * 1024);

  f32x16_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

  // byte offsets (within a stage) of this lane's fragments for each k-substep
  const int l32 = lane & 31, half = lane >> 5;
  int aoff[TM][KS], boff[TN][KS];
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int r = wm * WTM + i * 32 + l32;
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) aoff[i][kk] = r * SL::RB + swz<KB>(r, kk * 2 + half) * 16;
  }
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const int r = wn * WTN + j * 32 + l32;
#pragma unroll
    for (int kk = 0; kk < KS; ++kk)
      boff[j][kk] = BM * SL::RB + r * SL::RB + swz<KB>(r, kk * 2 + half) * 16;
  }

  // one K step on stage S (a compile-time constant, so every LDS address is
  // a register plus an immediate): wait for this wave's loads of slice T,
  // publish it with one barrier, start the loads of slice T + NS - 1 into the
  // stage slice T - 1 used, then run the MFMAs, reading the next k-substep's
  // fragments ahead. Near the end fewer later slices are in flight, so the
  // wait there is for all of them.
#define ZSA_STEP(S, T)                                                                   \
  {                                                                                      \
    if (KTOT - 1 - (T) >= NS - 2)                                                        \
      __builtin_amdgcn_s_waitcnt(vmcnt_imm((NS - 2) * (AI + BI)));                       \
    else                                                                                 \
      __builtin_amdgcn_s_waitcnt(0);                                                     \
    barrier_lds();                                                                       \
    if ((T) + NS - 1 < KTOT) {                                                           \
      ZSA_DMA(((S) + NS - 1) % NS, ((T) + NS - 1) * KB)                                  \
    }                                                                                    \
    const unsigned char* st = smem + (S) * SB;                                           \
    bf16x8_t a[2][TM], b[2][TN];                                                         \
    _Pragma("unroll") for (int i = 0; i < TM; ++i)                                       \
      a[0][i] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const u32x4*>(st + aoff[i][0])); \
    _Pragma("unroll") for (int j = 0; j < TN; ++j)                                       \
      b[0][j] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const u32x4*>(st + boff[j][0])); \
    _Pragma("unroll") for (int kk = 0; kk < KS; ++kk) {                                  \
      const int cur = kk & 1, nxt = cur ^ 1;                                             \
      if (kk + 1 < KS) {                                                                 \
        _Pragma("unroll") for (int i = 0; i < TM; ++i)                                   \
          a[nxt][i] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const u32x4*>(st + aoff[i][kk + 1])); \
        _Pragma("unroll") for (int j = 0; j < TN; ++j)                                   \
          b[nxt][j] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const u32x4*>(st + boff[j][kk + 1])); \
      }                                                                                  \
      __builtin_amdgcn_sched_barrier(0);                                                 \
      _Pragma("unroll") for (int i = 0; i < TM; ++i)                                     \
        _Pragma("unroll") for (int j = 0; j < TN; ++j)                                   \
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b[cur][j], a[cur][i], acc[i][j], 0, 0, 0); \
      __builtin_amdgcn_sched_barrier(0);                                                 \
    }                                                                                    \
  }

  // operands swapped in the MFMA: the accumulator holds C^T, so lane l owns
  // output row l%32 of an m-block and 4 consecutive columns per register group
#pragma unroll
  for (int s = 0; s < NS - 1; ++s)
    if (s < KTOT) {
      ZSA_DMA(s, s * KB)
    }
  int kt = 0;
  for (; kt + NS <= KTOT; kt += NS) {
#pragma unroll
    for (int s = 0; s < NS; ++s) ZSA_STEP(s, kt + s)
  }
  // kt is a multiple of NS here, so slice kt + s sits in stage s
#pragma unroll
  for (int s = 0; s < NS - 1; ++s)
    if (kt + s < KTOT) ZSA_STEP(s, kt + s)
#undef ZSA_STEP
#undef ZSA_DMA
#undef ZSA_DMA1
  // acc[i][j][4g + e] = C[m][n + e] with m = wm*WTM + 32 i + l%32 and
  // n = wn*WTN + 32 j + 8 g + 4 (l/32) inside the tile: every register group
  // is 4 consecutive columns of one row, staged with one 16-byte LDS write
  // (rows BN + 4 floats apart, so 16 lanes cover the 64 banks once). The
  // 32-row blocks are aligned, so each lies in one pass of ER rows.
  if (part != nullptr) {
    // split K: the raw fp32 partial tile goes to slice y of part [S][M][N]
    // (N is a multiple of 8, so a 4-column group is inside or outside whole)
    float* dst = part + static_cast<int64_t>(blockIdx.y) * M * N;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int m = m0 + wm * WTM + i * 32 + l32;
          const int n = n0 + wn * WTN + j * 32 + g * 8 + half * 4;
          if (m < M && n < N)
            *reinterpret_cast<float4*>(dst + static_cast<int64_t>(m) * N + n) =
                make_float4(acc[i][j][4 * g], acc[i][j][4 * g + 1], acc[i][j][4 * g + 2],
                            acc[i][j][4 * g + 3]);
        }
    return;
  }
  float* tile = reinterpret_cast<float*>(smem);
#pragma unroll
  for (int pass = 0; pass < BM / ER; ++pass) {
    __syncthreads();  // operand stages (pass 0) or the previous pass's tile are free
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      if ((wm * WTM + i * 32) / ER != pass) continue;
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int row = wm * WTM + i * 32 - pass * ER + l32;
          const int col = wn * WTN + j * 32 + g * 8 + half * 4;
          const float4 v = make_float4(acc[i][j][4 * g], acc[i][j][4 * g + 1],
                                       acc[i][j][4 * g + 2], acc[i][j][4 * g + 3]);
          *reinterpret_cast<float4*>(tile + row * kTileLd + col) = v;
        }
    }
    __syncthreads();
    epilogue_tile<bf16_t, ER, BN, NT>(tile, kTileLd, m0 + pass * ER, n0, M, N, ep);
  }
}

// Split-K finish: sums the S partial tiles of an 8 x 128 output block in
// slice order (fixed, so the result is reproducible), then applies the
// epilogue exactly as the unsplit kernel does. One float4 per thread; the
// slice loads are issued in groups of four before their (ordered) adds.
constexpr int kRedRows = 8, kRedCols = 128;

__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float* __restrict__ part,
                                                            int S, int M, int N, EpiParams ep) {
  __shared__ __align__(16) float tile[kRedRows * (kRedCols + 4)];
  const int m0 = blockIdx.x * kRedRows, n0 = blockIdx.y * kRedCols;
  const int64_t slice = static_cast<int64_t>(M) * N;
  const int r = threadIdx.x / (kRedCols / 4), c = (threadIdx.x % (kRedCols / 4)) * 4;
  const int m = m0 + r, n = n0 + c;
  float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
  if (m < M && n < N) {
    const float* src = part + static_cast<int64_t>(m) * N + n;
    int y = 0;
    for (; y + 4 <= S; y += 4) {
      float4 t[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) t[u] = *reinterpret_cast<const float4*>(src + (y + u) * slice);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        v.x += t[u].x;
        v.y += t[u].y;
        v.z += t[u].z;
        v.w += t[u].w;
      }
    }
    for (; y < S; ++y) {
      const float4 t = *reinterpret_cast<const float4*>(src + y * slice);
      v.x += t.x;
      v.y += t.y;
      v.z += t.z;
      v.w += t.w;
    }
  }
  *reinterpret_cast<float4*>(tile + r * (kRedCols + 4) + c) = v;
  __syncthreads();
  epilogue_tile<bf16_t, kRedRows, kRedCols, 256>(tile, kRedCols + 4, m0, n0, M, N, ep);
}

// fp32 sum of the S slices [S][total4] (float4 units), in slice order
__global__ __launch_bounds__(256) void splitk_sum_f32_kernel(const float4* __restrict__ part,
                                                             int S, int64_t total4,
                                                             float4* __restrict__ out) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i >= total4) return;
  float4 v = part[i];
  for (int y = 1; y < S; ++y) {
    const float4 t = part[y * total4 + i];
    v.x += t.x;
    v.y += t.y;
    v.z += t.z;
    v.w += t.w;
  }
  out[i] = v;
}

// ---------------------------------------------------------------------------
// Few-row products (generation, and the short layers of deep pruning)
// ---------------------------------------------------------------------------
// y = epi(x W^T) for few rows of x: with M <= 16 the whole cost is one read
// of W (M multiply-adds per weight), and for narrow outputs up to about a
// thousand rows the tiled kernels' output tiles are too few to fill the
// GPU or mostly multiply padding. The kernel has no
// shared tiles: v_mfma_f32_16x16x32_bf16 takes A = 16 rows of W (lane l:
// row l % 16, the 8 K values 8 (l / 16) .. + 7 of a 32-wide step) and B =
// 16 x rows (lane l: row l % 16, zero past M); lane l then holds outputs
// (row l % 16 of x, W rows 4 (l / 16) .. + 3).
//
// A workgroup owns 16 CB output columns and 16 MB rows over the whole of
// K: its 8 waves take consecutive K ranges and their partial sums are added
// in wave order through LDS, so no other workgroup is involved and the
// result is reproducible. Loads go through buffer resources: W rows past N,
// x rows past M and offsets set past the end read as zeros.
// For the rotary epilogue each 16 columns are 8 channels of a head and
// their partners hd / 2 further on, so each rotation pair is local.
constexpr int kSkCols = 16;   // output columns (W rows) per column block
constexpr int kSkWaves = 8;   // K ranges per workgroup
constexpr int kSkMaxM = 16;   // rows of x per row block
constexpr int kSkMaxRows = 4096;  // rows of x per launch (a grid of 16-row blocks)

// output column of column j of 16-column block t (rope_half = hd / 2 for
// the rotary epilogue, else 0)
__device__ __forceinline__ int skinny_col(int t, int j, int rope_half) {
  if (rope_half == 0) return t * kSkCols + j;
  const int per_head = rope_half / 8;  // column blocks per head
  const int h = t / per_head, i0 = (t % per_head) * 8;
  return h * 2 * rope_half + i0 + (j & 7) + (j >> 3) * rope_half;
}

// CPL > 0: x is first normalised as the block's pre-norm does (LayerNorm,
// or RMSNorm with mean 0): wave w takes row w (M <= 8), CPL 16-byte
// chunks of it per lane, for the exact two-pass mean and
// centred sum of squares in fp32; the gain (and shift) go to LDS; each x
// fragment then becomes bf16((x - mean) * rstd * gain + shift) before its
// MFMAs, the values the separate normalisation would have stored.
//
// MB > 1: a workgroup takes MB blocks of 16 rows (the same W fragments feed
// MB MFMAs), so W is re-read once per 16 MB rows instead of once per 16.
// CB > 1: it takes CB blocks of 16 columns (the same x fragments feed CB
// MFMAs), so x is re-read once per 16 CB columns. A wave moves its K range
// in groups of 64 K values (128 bytes of each W and x row); a round holds
// NG groups. DB: two rounds of registers, the next round's loads in flight
// while a round is multiplied (for K ranges longer than one round).
constexpr int sk_groups(int MB, int CB, bool DB) {
  return (DB ? 4 : 8) / (CB + MB) >= 4 ? 4 : (DB ? 4 : 8) / (CB + MB) >= 2 ? 2 : 1;
}

template <int CPL, int MB, int CB, bool DB>
__global__ __launch_bounds__(kSkWaves * 64) void gemm_skinny_kernel(
    const bf16_t* __restrict__ X, const bf16_t* __restrict__ W, int M, int N, int K, int kc,
    EpiParams ep, PreNorm pn) {
  static_assert(CPL == 0 || (MB == 1 && CB == 1), "the folded norm takes one block");
  constexpr int RM = kSkMaxM * MB;  // rows per workgroup
  constexpr int CN = kSkCols * CB;  // columns per workgroup
  constexpr int NT = kSkWaves * 64;
  constexpr int GR = CN + RM;                          // W and x rows of a group
  constexpr int LPG = GR / 8;                          // 1 KiB loads per group
  constexpr int NG = sk_groups(MB, CB, DB);            // groups per round
  constexpr int RK = 64 * NG;                          // K values per round
  constexpr int kTrBytes = kSkWaves * GR * 128;        // one group per wave
  constexpr int kRedBytes = kSkWaves * RM * (CN + 1) * 4;
  extern __shared__ __align__(16) uint4 gain_shift[];  // CPL > 0: gain [K / 8], shift [K / 8]
  // the waves' transposition buffers, then (after the K loop) the partial sums
  __shared__ __align__(16) unsigned char lds[kTrBytes > kRedBytes ? kTrBytes : kRedBytes];
  __shared__ float tile[RM][CN + 1];
  __shared__ float row_stat[2][RM];  // mean, rstd of each x row
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int l16 = lane & 15, kg = lane >> 4;
  const int t = blockIdx.x;  // the workgroup's column blocks are CB t .. CB t + CB - 1
  // blockIdx.y picks a block of RM rows of x (M is then this block's rows)
  const int mrow0 = blockIdx.y * RM;
  X += static_cast<int64_t>(mrow0) * K;
  M = min(RM, M - mrow0);
  const int rope_half = ep.epi == EPI_ROPE ? ep.head_dim / 2 : 0;
  const int k0 = wave * kc, k1 = min(K, k0 + kc);
  const __amdgpu_buffer_rsrc_t xres = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<bf16_t*>(X), 0, static_cast<uint32_t>(M) * K * 2u, 0x00020000);
  const __amdgpu_buffer_rsrc_t wres = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<bf16_t*>(W), 0, static_cast<uint32_t>(N) * K * 2u, 0x00020000);
  constexpr uint32_t kPast = 0x80000000u;  // beyond both buffers: reads zeros
  const int C8 = K / 8;                    // 16-byte chunks of a row
  // Loads cover whole 128-byte lines: load i of a group moves group rows
  // 8 i .. 8 i + 7 (W rows first, then x rows), lane l the 16-byte chunk
  // l % 8 of row 8 i + l / 8. The wave then stores them to its LDS buffer
  // (chunk c of group row r at r * 128 + (c ^ (r % 8)) * 16) and reads back
  // MFMA fragments: lane l of step s takes chunk 4 s + l / 16 of row l % 16
  // of a block. (Fragments loaded straight from memory would touch 16 lines
  // per load, half of each: about a third of the throughput.)
  const int lc = lane & 7, lr = lane >> 3;
  uint32_t roff[LPG];  // byte offset of this lane's chunk at K step 0 (kPast: none)
#pragma unroll
  for (int i = 0; i < LPG; ++i) {
    const int r = 8 * i + lr;
    if (r < CN) {
      roff[i] = static_cast<uint32_t>(skinny_col(t * CB + r / kSkCols, r % kSkCols, rope_half)) * K * 2u +
                lc * 16u;
    } else {
      roff[i] = static_cast<uint32_t>(r - CN) * K * 2u + lc * 16u;
    }
  }
  unsigned char* const trb = lds + wave * GR * 128;  // this wave's buffer
  // The epilogue's operands of this thread's output items (item it = tid +
  // q NT: row it / CN, workgroup column it % CN) are requested before
  // anything else, so the epilogue waits for no global load after the
  // reduction.
  constexpr int IPT = (RM * CN + NT - 1) / NT;  // items per thread
  float pre_b[IPT], pre_r[IPT];
#pragma unroll
  for (int q = 0; q < IPT; ++q) {
    const int it = tid + q * NT;
    const int m = it / CN, jj = it % CN;
    const int c = skinny_col(t * CB + jj / kSkCols, jj % kSkCols, rope_half);
    const bool live = m < M && c < N;
    pre_b[q] = live && ep.bias != nullptr ? to_f32(static_cast<const bf16_t*>(ep.bias)[c]) : 0.f;
    pre_r[q] = live && ep.epi == EPI_RESIDUAL
                   ? to_f32(static_cast<const bf16_t*>(
                         ep.residual)[(mrow0 + m) * static_cast<int64_t>(ep.ldy) + c])
                   : 0.f;
  }
  // the normalisation's inputs are requested next, so waiting for them
  // leaves the first round in flight
  uint4 gs[2], rowc[CPL > 0 ? CPL : 1];  // gain / shift chunks: 2 K / 8 <= 2 x 512
  if constexpr (CPL > 0) {
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int c = tid + q * NT;
      gs[q] = make_uint4(0u, 0u, 0u, 0u);
      if (c < 2 * C8) {
        const bf16_t* src = c < C8 ? pn.g + 8 * c : (pn.b != nullptr ? pn.b + 8 * (c - C8) : nullptr);
        if (src != nullptr) gs[q] = *reinterpret_cast<const uint4*>(src);
      }
    }
#pragma unroll
    for (int i = 0; i < CPL; ++i) {
      const int c = lane + 64 * i;
      rowc[i] = __builtin_bit_cast(
          uint4, __builtin_amdgcn_raw_buffer_load_b128(
                     xres, wave < M && c < C8 ? (static_cast<uint32_t>(wave) * K + 8 * c) * 2u : kPast,
                     0, 0));
    }
    __builtin_amdgcn_sched_barrier(0);
  }
  uint4 v[DB ? 2 : 1][NG][LPG];
  // the loads of the round at k into buffer BUF (chunks past the wave's K
  // range read zeros)
  auto issue = [&](auto BUF, int k) {
    constexpr int u = decltype(BUF)::value;
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      const int kk = k + 64 * g;
      const bool in = kk + 8 * lc < k1;
#pragma unroll
      for (int i = 0; i < LPG; ++i)
        v[u][g][i] = __builtin_bit_cast(
            uint4, __builtin_amdgcn_raw_buffer_load_b128(8 * i < CN ? wres : xres,
                                                         in ? roff[i] + kk * 2u : kPast, 0, 0));
    }
  };
  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  const int rounds = k0 < k1 ? (k1 - k0 + RK - 1) / RK : 0;
  if (rounds > 0) issue(I0{}, k0);
  __builtin_amdgcn_sched_barrier(0);
  float mean[MB], rstd[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) mean[mb] = rstd[mb] = 0.f;
  if constexpr (CPL > 0) {
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int c = tid + q * NT;
      if (c < 2 * C8) gain_shift[c] = gs[q];
    }
    const float inv_d = 1.0f / static_cast<float>(K);
    float sum = 0.f, sq = 0.f, mu = 0.f;
    if (!pn.rms) {
#pragma unroll
      for (int i = 0; i < CPL; ++i) {
        float f[8];
        unpack16(rowc[i], f, bf16_t());
#pragma unroll
        for (int e = 0; e < 8; ++e) sum += f[e];
      }
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) sum += __shfl_xor(sum, off, 64);
      mu = sum * inv_d;
    }
#pragma unroll
    for (int i = 0; i < CPL; ++i) {
      if (lane + 64 * i < C8) {
        float f[8];
        unpack16(rowc[i], f, bf16_t());
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float d = f[e] - mu;
          sq += d * d;
        }
      }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) sq += __shfl_xor(sq, off, 64);
    if (lane == 0) {
      row_stat[0][wave] = mu;
      row_stat[1][wave] = 1.0f / sqrtf(sq * inv_d + pn.eps);
    }
    barrier_lds();
    if (l16 < M) {
      mean[0] = row_stat[0][l16];
      rstd[0] = row_stat[1][l16];
    }
  }
  f32x4_t acc[CB][MB];
#pragma unroll
  for (int cb = 0; cb < CB; ++cb)
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) acc[cb][mb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  // the MFMAs of the round at k, from buffer BUF: each group goes through
  // the wave's LDS buffer (LDS operations of a wave run in order, so a
  // group's stores follow the previous group's fragment reads)
  auto compute = [&](auto BUF, int k) {
    constexpr int u = decltype(BUF)::value;
#pragma unroll
    for (int g = 0; g < NG; ++g) {
#pragma unroll
      for (int i = 0; i < LPG; ++i) {
        const int r = 8 * i + lr;
        *reinterpret_cast<uint4*>(trb + r * 128 + ((lc ^ (r & 7)) << 4)) = v[u][g][i];
      }
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        const int ch = 4 * s + kg;
        bf16x8_t af[CB], bj[MB];
#pragma unroll
        for (int cb = 0; cb < CB; ++cb) {
          const int r = 16 * cb + l16;
          af[cb] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const uint4*>(trb + r * 128 + ((ch ^ (r & 7)) << 4)));
        }
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
          const int r = CN + 16 * mb + l16;
          bj[mb] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const uint4*>(trb + r * 128 + ((ch ^ (r & 7)) << 4)));
        }
        if constexpr (CPL > 0) {
          const int c = min(k + 64 * g + 8 * ch, K - 8) / 8;
          float gg[8], sh[8];
          unpack16(gain_shift[c], gg, bf16_t());
          unpack16(gain_shift[C8 + c], sh, bf16_t());
#pragma unroll
          for (int mb = 0; mb < MB; ++mb) {
            float f[8], o[8];
            unpack16(__builtin_bit_cast(uint4, bj[mb]), f, bf16_t());
#pragma unroll
            for (int e = 0; e < 8; ++e) o[e] = (f[e] - mean[mb]) * rstd[mb] * gg[e] + sh[e];
            bj[mb] = __builtin_bit_cast(bf16x8_t, pack16(o, bf16_t()));
          }
        }
#pragma unroll
        for (int cb = 0; cb < CB; ++cb)
#pragma unroll
          for (int mb = 0; mb < MB; ++mb)
            acc[cb][mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[cb], bj[mb], acc[cb][mb], 0, 0, 0);
      }
    }
  };
  if constexpr (!DB) {
    for (int r = 0; r < rounds; ++r) {
      if (r > 0) issue(I0{}, k0 + r * RK);
      __builtin_amdgcn_sched_barrier(0);
      compute(I0{}, k0 + r * RK);
    }
  } else {
    // the round after the one multiplied is always in flight (a round past
    // the range reads zeros, so the issue is unconditional and every wait
    // is for the older buffer only)
    for (int r = 0; r < rounds; r += 2) {
      issue(I1{}, k0 + (r + 1) * RK);
      __builtin_amdgcn_sched_barrier(0);
      compute(I0{}, k0 + r * RK);
      if (r + 1 >= rounds) break;
      issue(I0{}, k0 + (r + 2) * RK);
      __builtin_amdgcn_sched_barrier(0);
      compute(I1{}, k0 + (r + 1) * RK);
    }
  }
  // every wave is past its transposition buffer before the partial sums
  // take that space
  __syncthreads();
  float (*red)[RM][CN + 1] = reinterpret_cast<float (*)[RM][CN + 1]>(lds);
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    if (16 * mb + l16 < M) {
#pragma unroll
      for (int cb = 0; cb < CB; ++cb)
#pragma unroll
        for (int r = 0; r < 4; ++r) red[wave][16 * mb + l16][16 * cb + 4 * kg + r] = acc[cb][mb][r];
    }
  }
  __syncthreads();
  const int items = M * CN;
  // elementwise epilogues finish each item where its partial sums meet;
  // SwiGLU and the rotary one pair columns, through a tile in LDS
  const bool paired = ep.epi == EPI_SWIGLU || ep.epi == EPI_ROPE;
#pragma unroll
  for (int q = 0; q < IPT; ++q) {
    const int it = tid + q * NT;
    if (it >= items) break;
    const int m = it / CN, jj = it % CN;
    float z = 0.f;
#pragma unroll
    for (int w = 0; w < kSkWaves; ++w) z += red[w][m][jj];
    z += pre_b[q];
    if (paired) {
      tile[m][jj] = z;
      continue;
    }
    const int c = skinny_col(t * CB + jj / kSkCols, jj % kSkCols, rope_half);
    if (c >= N) continue;
    if (ep.epi == EPI_GELU) z = gelu_erf(z);
    else if (ep.epi == EPI_RESIDUAL) z += pre_r[q];
    static_cast<bf16_t*>(ep.y)[(mrow0 + m) * static_cast<int64_t>(ep.ldy) + c] = f32_to_bf16(z);
  }
  if (!paired) return;
  __syncthreads();
#pragma unroll
  for (int q = 0; q < IPT; ++q) {
    const int it = tid + q * NT;
    if (it >= items) break;
    const int m = it / CN, jj = it % CN, j = jj % kSkCols;
    const int c = skinny_col(t * CB + jj / kSkCols, j, rope_half);
    if (c >= N) continue;
    const int64_t row = mrow0 + m;  // row of x and of the output
    bf16_t* y = static_cast<bf16_t*>(ep.y) + row * ep.ldy;
    const float z = tile[m][jj];
    float v = z;
    if (ep.epi == EPI_SWIGLU) {  // gate, up on columns 2f, 2f + 1
      if (j & 1) continue;
      y[c / 2] = f32_to_bf16(silu(z) * tile[m][jj + 1]);
      continue;
    } else if (c < ep.rope_cols) {
      const float zp = tile[m][jj ^ 8];
      const int i = (c % ep.head_dim) % rope_half;
      float sn, cs;
      if (ep.rope_cs != nullptr) {
        const float2 tc = reinterpret_cast<const float2*>(ep.rope_cs)[row * rope_half + i];
        cs = tc.x;
        sn = tc.y;
      } else {
        rope_angle(ep.pos[row], ep.inv_freq[i], &sn, &cs);
      }
      v = j < 8 ? z * cs - zp * sn : z * cs + zp * sn;
    }
    y[c] = f32_to_bf16(v);
  }
}

// ---------------------------------------------------------------------------
// vector-ALU GEMM (fp32 storage, and any shape)
// ---------------------------------------------------------------------------
constexpr int vBM = 64, vBN = 128, vBK = 16;

template <typename T>
__global__ __launch_bounds__(256) void gemm_valu_kernel(const T* __restrict__ X,
                                                        const T* __restrict__ W, int M, int N,
                                                        int K, EpiParams ep) {
  __shared__ float As[vBK][vBM + 4];
  __shared__ float Bs[vBK][vBN + 4];
  __shared__ float tile[vBM * (vBN + 4)];
  const int tid = threadIdx.x;
  const int tx = tid & 15, ty = tid >> 4;
  const int m0 = blockIdx.x * vBM, n0 = blockIdx.y * vBN;
  float acc[4][8];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[i][j] = 0.f;
  for (int k0 = 0; k0 < K; k0 += vBK) {
#pragma unroll
    for (int i = 0; i < vBM * vBK / 256; ++i) {
      const int e = tid + i * 256;
      const int mm = e / vBK, kk = e % vBK;
      const int gm = m0 + mm, gk = k0 + kk;
      As[kk][mm] = (gm < M && gk < K) ? to_f32(X[static_cast<int64_t>(gm) * K + gk]) : 0.f;
    }
#pragma unroll
    for (int i = 0; i < vBN * vBK / 256; ++i) {
      const int e = tid + i * 256;
      const int nn = e / vBK, kk = e % vBK;
      const int gn = n0 + nn, gk = k0 + kk;
      Bs[kk][nn] = (gn < N && gk < K) ? to_f32(W[static_cast<int64_t>(gn) * K + gk]) : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < vBK; ++kk) {
      float a[4], b[8];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = As[kk][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 8; ++j) b[j] = Bs[kk][tx * 8 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[i][j] += a[i] * b[j];
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) tile[(ty * 4 + i) * (vBN + 4) + tx * 8 + j] = acc[i][j];
  __syncthreads();
  epilogue_tile<T, vBM, vBN, 256>(tile, vBN + 4, m0, n0, M, N, ep);
}


// ---------------------------------------------------------------------------
// persistent bf16 GEMM, epilogue in registers (bias, GELU, residual)
// ---------------------------------------------------------------------------
// Two workgroups per CU stay resident and each walks a strided share of its
// XCD's range of 128 x 128 output tiles (the grouped order above). Between
// two tiles nothing drains: once the last K slice of a tile has been read,
// the first slice of the next tile is put in flight, and only then is the
// finished tile's epilogue done -- in registers, from the accumulators
// (which hold C^T: lane l owns row l%32 of a 32-row block and 4 consecutive
// columns per register group), with raw buffer stores whose range check
// drops the rows past M. The stores are not waited for; the next tile's
// first wait counts them as the youngest operations in flight (vector
// memory operations complete in issue order), so it waits for its slice
// only. The bias is read with scalar loads; a residual is fetched during
// the tile's last K step.
//
// Operand staging and the K pipeline are those of gemm_bf16_dma_kernel
// (KB-wide slices, 2 stages, swizzled direct-to-LDS loads; used with
// 64-wide slices at two workgroups per CU). N must be a multiple of 128;
// outputs and residual of fewer than 2^31 bytes.
// The plain and residual epilogues store whole lines through 4 KiB of LDS
// per wave past the two stages, where WPC workgroups still fit a CU's 160
// KiB (64-wide slices at two per CU: exactly). Same box, us per launch
// with the kernel pinned: 8192 x 2304 x 768 37.9 -> 36.0, 4096 x 2304 x 768
// 22.4 -> 21.5, 2048 x 6144 x 2048 53.6 -> 52.5; the residual products
// within run-to-run noise, also with their residual read as whole lines
// through the same buffer (kept as 16-byte reads, fetched during the last K
// step, where their latency is hidden).
template <int EPI, int KB, int WPC>
constexpr bool persist_stages_epilogue() {
  return (EPI == EPI_NONE || EPI == EPI_RESIDUAL) && WPC * (2 * (128 + 128) * KB * 2 + 4 * 4096) <= 163840;
}

template <int EPI, int KB, int WPC>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(WPC, WPC))) void
gemm_bf16_persist_kernel(const bf16_t* __restrict__ X, const bf16_t* __restrict__ W, int M, int N,
                         int K, EpiParams ep) {
  constexpr int BM = 128, BN = 128, NW = 4, WN = 2;
  constexpr int WTM = 64, WTN = 64, TM = 2, TN = 2;
  using SL = Slice<KB>;
  constexpr int AI = BM / SL::RPD / NW, BI = BN / SL::RPD / NW;
  constexpr int SB = (BM + BN) * SL::RB;
  constexpr int KS = KB / 16;
  extern __shared__ __align__(16) unsigned char smem[];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WN, wn = wave % WN;
  const int l32 = lane & 31, half = lane >> 5;

  const int nM = (M + BM - 1) / BM, nN = N / BN;
  const int tiles = nM * nN;
  const int xcd = blockIdx.x % kXcds, slot = blockIdx.x / kXcds;
  const int slots = gridDim.x / kXcds;
  const int per = tiles / kXcds, extra = tiles % kXcds;
  const int tbeg = xcd * per + min(xcd, extra);
  const int tcount = per + (xcd < extra ? 1 : 0);
  int k = slot;
  if (k >= tcount) return;
  auto tile_at = [&](int t, int* m0, int* n0) {
    const int g = t / (kXcdGroup * nN);
    const int gm0 = g * kXcdGroup;
    const int gsz = min(kXcdGroup, nM - gm0);
    const int r = t - g * kXcdGroup * nN;
    *n0 = (r / gsz) * BN;
    *m0 = (gm0 + r % gsz) * BM;
  };
  const int KTOT = K / KB;

  const int lr = lane / SL::CPR, lp = lane % SL::CPR;
  const bf16_t* asrc[AI];
  const bf16_t* bsrc[BI];
  auto set_sources = [&](int m0, int n0) {
#pragma unroll
    for (int i = 0; i < AI; ++i) {
      const int r = (i * NW + wave) * SL::RPD + lr;
      asrc[i] = X + static_cast<int64_t>(min(m0 + r, M - 1)) * K + swz<KB>(r, lp) * 8;
    }
#pragma unroll
    for (int i = 0; i < BI; ++i) {
      const int r = (i * NW + wave) * SL::RPD + lr;
      bsrc[i] = W + static_cast<int64_t>(n0 + r) * K + swz<KB>(r, lp) * 8;
    }
  };
#if defined(__HIP_DEVICE_COMPILE__)
  typedef __attribute__((address_space(3))) void lds_void;
#define ZSA_DMA1(src, dst) __builtin_amdgcn_global_load_lds((src), (lds_void*)(dst), 16, 0, 0)
#else
#define ZSA_DMA1(src, dst) ((void)(src), (void)(dst))
#endif
#define ZSA_DMA(s, k0)                                                                   \
  _Pragma("unroll") for (int i = 0; i < AI; ++i)                                         \
    ZSA_DMA1(asrc[i] + (k0), smem + (s) * SB + (i * NW + wave) * 1024);                  \
  _Pragma("unroll") for (int i = 0; i < BI; ++i)                                         \
    ZSA_DMA1(bsrc[i] + (k0), smem + (s) * SB + BM * SL::RB + (i * NW + wave) * 1024);

  int aoff[TM][KS], boff[TN][KS];
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int r = wm * WTM + i * 32 + l32;
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) aoff[i][kk] = r * SL::RB + swz<KB>(r, kk * 2 + half) * 16;
  }
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const int r = wn * WTN + j * 32 + l32;
#pragma unroll
    for (int kk = 0; kk < KS; ++kk)
      boff[j][kk] = BM * SL::RB + r * SL::RB + swz<KB>(r, kk * 2 + half) * 16;
  }

  const int ybytes = M * ep.ldy * 2;
  const __amdgpu_buffer_rsrc_t yres = __builtin_amdgcn_make_buffer_rsrc(ep.y, 0, ybytes, 0x00020000);
  const __amdgpu_buffer_rsrc_t rres = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<void*>(EPI == EPI_RESIDUAL ? ep.residual : ep.y), 0, ybytes, 0x00020000);
  const bf16_t* bias = static_cast<const bf16_t*>(ep.bias);

  int m0, n0;
  tile_at(tbeg + k, &m0, &n0);
  set_sources(m0, n0);
  ZSA_DMA(0, 0)
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
  barrier_lds();
  // Every wait below is straight-line code with a fixed count of younger
  // vector memory operations, so the compiler's own waits agree with it:
  // at the top of a tile slice 0 is in LDS and published.
  while (true) {
    f32x16_t acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
    uint32_t res[TM][TN][2][4];
    uint2 bw[TN][4];
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int g = 0; g < 4; ++g) bw[j][g] = make_uint2(0u, 0u);

    // the work of K step T on stage S once slice T is published: start slice
    // T + 1 into the other stage; one step before the last (in the only step
    // when K is one slice) fetch the epilogue's bias and residual, which the
    // last step's wait then covers; then the MFMAs
#define ZSA_PBODY(S, T)                                                                  \
  {                                                                                      \
    if ((T) + 1 < KTOT) {                                                                \
      ZSA_DMA(((S) + 1) & 1, ((T) + 1) * KB)                                             \
    }                                                                                    \
    if ((T) + 2 == KTOT || KTOT == 1) {                                                  \
      if (bias != nullptr) {                                                             \
        _Pragma("unroll") for (int j = 0; j < TN; ++j)                                   \
          _Pragma("unroll") for (int g = 0; g < 4; ++g)                                  \
            bw[j][g] = *reinterpret_cast<const uint2*>(                                  \
                bias + n0 + wn * WTN + j * 32 + g * 8 + half * 4);                       \
      }                                                                                  \
      if (EPI == EPI_RESIDUAL) {                                                         \
        _Pragma("unroll") for (int i = 0; i < TM; ++i)                                   \
          _Pragma("unroll") for (int j = 0; j < TN; ++j)                                 \
            res_load32(rres, static_cast<uint32_t>(m0 + wm * WTM + i * 32 + l32),        \
                       n0 + wn * WTN + j * 32, half, ep.ldy, res[i][j]);                 \
      }                                                                                  \
    }                                                                                    \
    const unsigned char* st = smem + (S) * SB;                                           \
    bf16x8_t a[2][TM], b[2][TN];                                                         \
    _Pragma("unroll") for (int i = 0; i < TM; ++i)                                       \
      a[0][i] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const u32x4*>(st + aoff[i][0])); \
    _Pragma("unroll") for (int j = 0; j < TN; ++j)                                       \
      b[0][j] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const u32x4*>(st + boff[j][0])); \
    _Pragma("unroll") for (int kk = 0; kk < KS; ++kk) {                                  \
      const int cur = kk & 1, nxt = cur ^ 1;                                             \
      if (kk + 1 < KS) {                                                                 \
        _Pragma("unroll") for (int i = 0; i < TM; ++i)                                   \
          a[nxt][i] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const u32x4*>(st + aoff[i][kk + 1])); \
        _Pragma("unroll") for (int j = 0; j < TN; ++j)                                   \
          b[nxt][j] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const u32x4*>(st + boff[j][kk + 1])); \
      }                                                                                  \
      __builtin_amdgcn_sched_barrier(0);                                                 \
      _Pragma("unroll") for (int i = 0; i < TM; ++i)                                     \
        _Pragma("unroll") for (int j = 0; j < TN; ++j)                                   \
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b[cur][j], a[cur][i], acc[i][j], 0, 0, 0); \
      __builtin_amdgcn_sched_barrier(0);                                                 \
    }                                                                                    \
  }
    // K steps after the first: slice T is the only operation in flight
#define ZSA_PSTEP(S, T)                                                                  \
  {                                                                                      \
    asm volatile("" ::: "memory");                                                       \
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));                                            \
    barrier_lds();                                                                       \
    ZSA_PBODY(S, T)                                                                      \
  }

    ZSA_PBODY(0, 0)
    int kt = 1;
    for (; kt + 2 <= KTOT; kt += 2) {
      ZSA_PSTEP(1, kt)
      ZSA_PSTEP(0, kt + 1)
    }
    if (kt < KTOT) ZSA_PSTEP(1, kt)
#undef ZSA_PSTEP
#undef ZSA_PBODY

    // every wave is done reading the stages and nothing is in flight: put
    // the next tile's first slice in flight before this tile's epilogue
    const int knext = k + slots;
    const bool more = knext < tcount;
    int m0n = m0, n0n = n0;
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
    barrier_lds();
    if (more) {
      tile_at(tbeg + knext, &m0n, &n0n);
      set_sources(m0n, n0n);
      ZSA_DMA(0, 0)
    }
    if constexpr (persist_stages_epilogue<EPI, KB, WPC>()) {
      // whole-line stores through the wave's 4 KiB staging buffer past the
      // two stages (the layout of reg_epilogue_lds): row block i is one
      // 32 x 64 chunk, whose values go in while chunk i - 1's line reads are
      // in flight
      unsigned char* const stg = smem + 2 * SB + wave * 4096;
      const int lr8 = lane >> 3, lc8 = lane & 7;
      unsigned char* const sline = stg + lr8 * 128 + ((lc8 ^ lr8) << 4);
      auto goff = [&](int i, int q) {
        return (static_cast<uint32_t>(m0 + wm * WTM + 32 * i + lr8 + 8 * q) * static_cast<uint32_t>(ep.ldy) +
                static_cast<uint32_t>(n0 + wn * WTN + 8 * lc8)) * 2u;
      };
      u32x4 wv[4];
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        u32x4 v[TN][2];
#pragma unroll
        for (int j = 0; j < TN; ++j) epi_pack32<EPI>(acc[i][j], bw[j], res[i][j], v[j]);
        if (i > 0) {
#pragma unroll
          for (int q = 0; q < 4; ++q) __builtin_amdgcn_raw_buffer_store_b128(wv[q], yres, goff(i - 1, q), 0, 0);
        }
        asm volatile("" ::: "memory");
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int p = 0; p < 2; ++p)
            *reinterpret_cast<u32x4*>(stg + l32 * 128 + (((4 * j + 2 * p + half) ^ (l32 & 7)) << 4)) = v[j][p];
        asm volatile("" ::: "memory");
#pragma unroll
        for (int q = 0; q < 4; ++q) wv[q] = *reinterpret_cast<const u32x4*>(sline + q * 1024);
        asm volatile("" ::: "memory");
      }
#pragma unroll
      for (int q = 0; q < 4; ++q) __builtin_amdgcn_raw_buffer_store_b128(wv[q], yres, goff(TM - 1, q), 0, 0);
    } else {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          epi_store32<EPI>(acc[i][j], bw[j], res[i][j], yres,
                           static_cast<uint32_t>(m0 + wm * WTM + i * 32 + l32), n0 + wn * WTN + j * 32,
                           half, ep.ldy);
    }
    if (!more) break;
    k = knext;
    m0 = m0n;
    n0 = n0n;
    // the next tile's slice 0 (and this tile's stores) have completed
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
    barrier_lds();
  }
#undef ZSA_DMA
#undef ZSA_DMA1
}


// CUs of the current device (cached per device)
int device_cus() {
  static int cus[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cus[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
      n = 256;
    cus[dev] = n;
  }
  return cus[dev];
}

// the persistent kernels take bf16 products with N a multiple of 128, K a
// multiple of 64, no rotary epilogue, buffers below 2^31 bytes, and output
// (and residual) rows of whole 16-byte units on 16-byte boundaries
bool persist_ok(int M, int N, int K, const EpiParams& ep) {
  if (N % 128 != 0 || K % 64 != 0 || K < 64 || M <= 0) return false;
  if (reinterpret_cast<uintptr_t>(ep.bias) % 8 != 0 || ep.ldy % 8 != 0) return false;
  if (reinterpret_cast<uintptr_t>(ep.y) % 16 != 0 || reinterpret_cast<uintptr_t>(ep.residual) % 16 != 0)
    return false;
  if (ep.epi != EPI_NONE && ep.epi != EPI_GELU && ep.epi != EPI_RESIDUAL && ep.epi != EPI_SWIGLU)
    return false;
  if (ep.epi == EPI_SWIGLU && N % 16 != 0) return false;
  return static_cast<int64_t>(M + 128) * ep.ldy * 2 < (int64_t{1} << 31);
}

template <int EPI, int KB, int WPC>
hipError_t launch_persist(hipStream_t s, const void* x, int M, int K, const void* w, int N,
                          const EpiParams& ep) {
  constexpr int lds = 2 * (128 + 128) * KB * 2 + (persist_stages_epilogue<EPI, KB, WPC>() ? 4 * 4096 : 0);
  static bool lds_raised = false;
  if (!lds_raised) {
    const hipError_t e = hipFuncSetAttribute(
        reinterpret_cast<const void*>(gemm_bf16_persist_kernel<EPI, KB, WPC>),
        hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    if (e != hipSuccess) return e;
    lds_raised = true;
  }
  const int tiles = ((M + 127) / 128) * (N / 128);
  const int wgs = std::min(tiles, device_cus() * WPC);
  const int grid = kXcds * ((wgs + kXcds - 1) / kXcds);
  return launch(K_GEMM, gemm_bf16_persist_kernel<EPI, KB, WPC>, dim3(grid), dim3(256), lds, s,
                static_cast<const bf16_t*>(x), static_cast<const bf16_t*>(w), M, N, K, ep);
}

// ---------------------------------------------------------------------------
// bf16 GEMM, 256x256 tiles on four waves of 128x128 (one wave per SIMD)
// ---------------------------------------------------------------------------
// Per 64-wide K slice a wave reads 32 fragments (32 KiB) for 64 MFMAs: two
// thirds of the LDS reads per FLOP of four waves of 128x64. K slices of 64
// (a stage row is one 128-byte line of a W or x row, so every 1 KiB load
// fills 8 whole lines) live in two stages filled by buffer loads straight
// into LDS, in the swizzled layout of gemm_bf16_dma_kernel (the buffer range
// check turns rows past M into zeros, whose outputs are dropped). With one
// wave per SIMD nothing else hides LDS latency or a barrier, so each slice
// runs as two MFMA blocks and the work that would stall sits between their
// MFMAs (the order is pinned with scheduling barriers):
//   block A: MFMAs of the slice's first 32 K values, interleaved with the
//            reads of its last 32 K values' fragments;
//   wait for this wave's share of slice t + 1; barrier (publishes it, and
//            every wave is done with the stage of slice t);
//   block B: MFMAs of the last 32 K values, interleaved with the reads of
//            slice t + 1's first fragments and the loads of slice t + 2 into
//            the stage of slice t.
// Loads past the last slice go to an offset past the buffers (they read
// zeros into a stage that is not read again), so the loop body has no
// branches and every wait count is fixed.
template <int EPI>
__global__ __launch_bounds__(256) void gemm_bf16_w4_kernel(const bf16_t* __restrict__ X,
                                                          const bf16_t* __restrict__ W, int M,
                                                          int N, int K, EpiParams ep) {
  constexpr int BM = 256, BN = 256, KB = 64;
  using SL = Slice<KB>;
  constexpr int SB = (BM + BN) * SL::RB;        // bytes per stage
  constexpr int LPW = (BM + BN) / SL::RPD / 4;  // 1 KiB loads per wave per stage
  constexpr int ALD = BM / SL::RPD / 4;         // of which A rows
  static_assert(LPW == 16 && ALD == 8, "stage layout");
  extern __shared__ __align__(16) unsigned char smem[];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;  // 2 x 2 waves of 128 x 128
  const int l32 = lane & 31, half = lane >> 5;
  int mt, nt;
  if (!xcd_tile<BM, BN>(M, N, &mt, &nt)) return;
  const int m0 = mt * BM, n0 = nt * BN;
  const int KT = K / KB;
  const __amdgpu_buffer_rsrc_t xres =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16_t*>(X), 0, M * K * 2, 0x00020000);
  const __amdgpu_buffer_rsrc_t wres =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16_t*>(W), 0, N * K * 2, 0x00020000);
  // wave w moves row blocks i * 4 + w (8 rows each; A rows, then B rows);
  // stage row r = 8 blk + lr has swizzle (r / RPP) & (CPR - 1) =
  // (4 blk + lr / 2) & 7, which depends on blk only through the wave's parity
  const int lr = lane / SL::CPR, lp = lane % SL::CPR;
  const uint32_t lane_off =
      static_cast<uint32_t>(lr * K * 2 + swz<KB>((wave & 1) * SL::RPD + lr, lp) * 16);
  typedef __attribute__((address_space(3))) void lds_void;
  auto dma1 = [&](int st, int t, int i) {
    const int blk = i * 4 + wave;
    const uint32_t row0 = i < ALD ? static_cast<uint32_t>(m0 + blk * SL::RPD)
                                  : static_cast<uint32_t>(n0 + blk * SL::RPD - BM);
    const uint32_t off = t < KT ? (row0 * K + t * KB) * 2u + lane_off : 0x80000000u;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(i < ALD ? xres : wres,
                                             (lds_void*)(smem + st * SB + blk * 1024), 16, off, 0,
                                             0, 0);
  };
  // fragment q of k-substep kk: A block q (q < 4) or B block q - 4; row r of
  // a 32-row block sits at r * RB, its chunk c at (c ^ ((r / RPP) & 7)) * 16
  const int sw = (l32 / SL::RPP) & (SL::CPR - 1);
  int ab[4], bb[4];
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) {
    ab[kk] = (wm * 128 + l32) * SL::RB + ((kk * 2 + half) ^ sw) * 16;
    bb[kk] = BM * SL::RB + (wn * 128 + l32) * SL::RB + ((kk * 2 + half) ^ sw) * 16;
  }
  f32x16_t acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
  // f0: fragments of k-substeps 0, 1 of a slice; f1: of k-substeps 2, 3
  bf16x8_t f0[2][8], f1[2][8];
  auto rd1 = [&](const unsigned char* st, int kk, bf16x8_t (&f)[8], int q) {
    const int off = q < 4 ? ab[kk] + q * 32 * SL::RB : bb[kk] + (q - 4) * 32 * SL::RB;
    f[q] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const u32x4*>(st + off));
  };
  // MFMA p of a k-substep: output block (p / 4, p % 4), operands swapped so
  // the accumulator holds C^T (four consecutive columns per register group)
  auto mma1 = [&](bf16x8_t (&f)[8], int p) {
    acc[p / 4][p % 4] =
        __builtin_amdgcn_mfma_f32_32x32x16_bf16(f[4 + p % 4], f[p / 4], acc[p / 4][p % 4], 0, 0, 0);
  };
  // prologue: slices 0 and 1 in flight, slice 0 published, its first
  // fragments read
#pragma unroll
  for (int i = 0; i < LPW; ++i) dma1(0, 0, i);
#pragma unroll
  for (int i = 0; i < LPW; ++i) dma1(1, 1, i);
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(vmcnt_imm(LPW));
  barrier_lds();
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    rd1(smem, 0, f0[0], q);
    rd1(smem, 1, f0[1], q);
  }
  int s = 0;
  for (int t = 0; t < KT; ++t) {
    const unsigned char* cur = smem + s * SB;
    const unsigned char* nxt = smem + (s ^ 1) * SB;
    // block A
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      __builtin_amdgcn_sched_barrier(0);
      mma1(f0[q / 8], 2 * (q % 8));
      rd1(cur, 2 + q / 8, f1[q / 8], q % 8);
      mma1(f0[q / 8], 2 * (q % 8) + 1);
    }
    __builtin_amdgcn_sched_barrier(0);
    // slice t + 1 (the only loads in flight) has landed
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
    barrier_lds();
    // block B
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      __builtin_amdgcn_sched_barrier(0);
      mma1(f1[q / 8], 2 * (q % 8));
      rd1(nxt, q / 8, f0[q / 8], q % 8);
      mma1(f1[q / 8], 2 * (q % 8) + 1);
      dma1(s, t + 2, q);
    }
    __builtin_amdgcn_sched_barrier(0);
    s ^= 1;
  }
  reg_epilogue<4, 4, EPI>(acc, m0 + wm * 128, n0 + wn * 128, M, l32, half, ep);
}

template <int EPI>
hipError_t launch_w4_1(hipStream_t s, const void* x, int M, int K, const void* w, int N,
                       const EpiParams& ep) {
  constexpr int lds = 2 * 512 * 64 * 2;
  static bool lds_raised = false;
  if (!lds_raised) {
    const hipError_t e = hipFuncSetAttribute(
        reinterpret_cast<const void*>(gemm_bf16_w4_kernel<EPI>),
        hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    if (e != hipSuccess) return e;
    lds_raised = true;
  }
  return launch(K_GEMM, gemm_bf16_w4_kernel<EPI>, xcd_grid(M, N, 256, 256), dim3(256), lds, s,
                static_cast<const bf16_t*>(x), static_cast<const bf16_t*>(w), M, N, K, ep);
}

// Epilogue of gemm_bf16_w4p_kernel: reg_epilogue with the bias read from
// LDS (blds holds the bf16 bias of columns nb, nb + 1, ...; zeros when the
// product has none), one 32 x 32 block at a time in a pinned order (the
// scheduler would otherwise read every accumulator out at once).
template <int TM, int TN, int EPI>
__device__ __forceinline__ void reg_epilogue_lb(const f32x16_t (&acc)[TM][TN], int mb, int nb, int M,
                                                int l32, int half, const EpiParams& ep,
                                                const unsigned char* blds) {
  const int ybytes = M * ep.ldy * 2;
  const __amdgpu_buffer_rsrc_t yres = __builtin_amdgcn_make_buffer_rsrc(ep.y, 0, ybytes, 0x00020000);
  const __amdgpu_buffer_rsrc_t rres = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<void*>(EPI == EPI_RESIDUAL ? ep.residual : ep.y), 0, ybytes, 0x00020000);
  // block (i, j) = step j * TM + i. The next step's residual is loaded
  // before this step's stores: vector memory operations are counted in issue
  // order, so a load issued after a store could only be waited for together
  // with that store.
  uint32_t r[2][2][4];
  if (EPI == EPI_RESIDUAL) res_load32(rres, static_cast<uint32_t>(mb + l32), nb, half, ep.ldy, r[0]);
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    uint2 bw[4];
#pragma unroll
    for (int g = 0; g < 4; ++g)
      bw[g] = *reinterpret_cast<const uint2*>(blds + (j * 32 + g * 8 + half * 4) * 2);
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      __builtin_amdgcn_sched_barrier(0);
      const int st = j * TM + i;
      if (EPI == EPI_RESIDUAL && st + 1 < TM * TN) {
        const int j1 = (st + 1) / TM, i1 = (st + 1) % TM;
        res_load32(rres, static_cast<uint32_t>(mb + i1 * 32 + l32), nb + j1 * 32, half, ep.ldy,
                   r[(st + 1) & 1]);
      }
      __builtin_amdgcn_sched_barrier(0);
      const uint32_t m = static_cast<uint32_t>(mb + i * 32 + l32);
      epi_store32<EPI>(acc[i][j], bw, r[st & 1], yres, m, nb + j * 32, half, ep.ldy);
    }
  }
}

// Epilogue of gemm_bf16_w4p_kernel through a per-wave LDS staging buffer
// (stg, 4 KiB), for the plain and residual epilogues. A store straight from
// the accumulators covers 32 bytes of each of 32 rows, a quarter of a
// 128-byte line each; here the wave takes chunks of 32 rows x 64 columns (two
// 32 x 32 accumulator blocks), writes the finished bf16 values of a chunk to
// stg in the accumulator layout and reads them back as 16 bytes of one row
// per lane, so that each store instruction covers 8 rows x 128 bytes. A
// residual goes the other way: whole-line loads, issued one chunk ahead,
// turned into the accumulator layout through stg. Row r of stg holds its
// 16-byte chunk c at r * 128 + ((c ^ (r & 7)) << 4), so the rows a line read
// or write covers hit distinct banks. No barrier: a wave's LDS operations run
// in issue order, and compiler fences keep each cross-lane read after the
// writes it depends on. A 256 x 192 tile leaves each wave a third 32-column
// block per row block, which is stored straight from the registers. Measured
// (us per launch, 256 x 256 tiles): 16384 x 16384 x 2048 902.8 -> 854.9,
// 16384 x 768 x 3072 with a residual 78.0 -> 76.2, 8192 x 2048 x 8192 with a
// residual 205.3 -> 201.0; 256 x 192 tiles: 16384 x 2304 x 768 60.3 -> 56.9.
// The GELU and SwiGLU epilogues keep the direct stores: their arithmetic,
// not the store pattern, bounds them (16384 x 3072 x 768 with GELU took 91.1
// us direct, 95.5 staged, and 92.0 with line-shaped stores and no staging;
// SwiGLU staged and software-pipelined like the plain path: 0.3-1.2 %
// slower at K = 2048, 1.4-2.2 % faster at K = 4096).
template <int TM, int TN, int EPI>
__device__ __forceinline__ void reg_epilogue_lds(const f32x16_t (&acc)[TM][TN], int mb, int nb, int M,
                                                 int l32, int half, const EpiParams& ep,
                                                 const unsigned char* blds, unsigned char* stg) {
  constexpr int BPC = 2;            // accumulator blocks per chunk
  constexpr int NCH = TN / BPC;     // staged chunks per row block
  if constexpr (EPI == EPI_GELU || EPI == EPI_SWIGLU) {
    reg_epilogue_lb<TM, TN, EPI>(acc, mb, nb, M, l32, half, ep, blds);
  } else {
    const int ybytes = M * ep.ldy * 2;
    const uint32_t ldy = static_cast<uint32_t>(ep.ldy);
    const __amdgpu_buffer_rsrc_t yres = __builtin_amdgcn_make_buffer_rsrc(ep.y, 0, ybytes, 0x00020000);
    const __amdgpu_buffer_rsrc_t rres = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<void*>(EPI == EPI_RESIDUAL ? ep.residual : ep.y), 0, ybytes, 0x00020000);
    const int lane = l32 + 32 * half;
    const int lr = lane >> 3, lc = lane & 7;  // line layout: rows lr + 8q, chunk lc
    unsigned char* const sline = stg + lr * 128 + ((lc ^ lr) << 4);
    auto sacc = [&](int c) { return stg + l32 * 128 + ((c ^ (l32 & 7)) << 4); };
    // chunk step t = i * NCH + k: rows mb + 32 i .., columns nb + 64 k ..
    constexpr int T = TM * NCH;
    auto goff = [&](int t, int q) {
      return ((static_cast<uint32_t>(mb + 32 * (t / NCH) + lr + 8 * q)) * ldy +
              static_cast<uint32_t>(nb + 64 * (t % NCH) + 8 * lc)) * 2u;
    };
    u32x4 rq[4];              // a chunk's residual as loaded (line layout)
    uint32_t r[BPC][2][4];    // the residual of the chunk computed next
    u32x4 w[4];               // the previous chunk's values, line layout
    auto rload = [&](int t) {
#pragma unroll
      for (int q = 0; q < 4; ++q)
        rq[q] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rres, goff(t, q), 0, 0));
    };
    // rq -> stg (line layout) -> r (accumulator layout, as res_load32 gives)
    auto stage_res = [&]() {
#pragma unroll
      for (int q = 0; q < 4; ++q) *reinterpret_cast<u32x4*>(sline + q * 1024) = rq[q];
      asm volatile("" ::: "memory");
#pragma unroll
      for (int jj = 0; jj < BPC; ++jj)
#pragma unroll
        for (int p = 0; p < 2; ++p) {
          const u32x4 v = *reinterpret_cast<const u32x4*>(sacc(4 * jj + 2 * p + half));
          r[jj][p][0] = v[0];
          r[jj][p][1] = v[1];
          r[jj][p][2] = v[2];
          r[jj][p][3] = v[3];
        }
      asm volatile("" ::: "memory");
    };
    // Software-pipelined: chunk t's arithmetic runs while the line reads of
    // chunk t - 1 are in flight, and its stores follow. Vector memory
    // operations are counted in issue order, so each residual load is
    // issued before the stores it must not wait for: chunk t + 2's after
    // chunk t's stores, waited for after chunk t + 1's.
    if (EPI == EPI_RESIDUAL) {
      rload(0);
      stage_res();
      if (T > 1) rload(1);
    }
#pragma unroll
    for (int t = 0; t < T; ++t) {
      const int i = t / NCH, k = t % NCH;
      __builtin_amdgcn_sched_barrier(0);
      u32x4 v[BPC][2];
#pragma unroll
      for (int jj = 0; jj < BPC; ++jj) {
        const int j = k * BPC + jj;
        uint2 bw[4];
#pragma unroll
        for (int g = 0; g < 4; ++g)
          bw[g] = *reinterpret_cast<const uint2*>(blds + (j * 32 + g * 8 + half * 4) * 2);
        epi_pack32<EPI>(acc[i][j], bw, r[jj], v[jj]);
      }
      if (t > 0) {
#pragma unroll
        for (int q = 0; q < 4; ++q) __builtin_amdgcn_raw_buffer_store_b128(w[q], yres, goff(t - 1, q), 0, 0);
      }
      asm volatile("" ::: "memory");
#pragma unroll
      for (int jj = 0; jj < BPC; ++jj)
#pragma unroll
        for (int p = 0; p < 2; ++p) *reinterpret_cast<u32x4*>(sacc(4 * jj + 2 * p + half)) = v[jj][p];
      asm volatile("" ::: "memory");
#pragma unroll
      for (int q = 0; q < 4; ++q) w[q] = *reinterpret_cast<const u32x4*>(sline + q * 1024);
      asm volatile("" ::: "memory");
      if (EPI == EPI_RESIDUAL && t + 1 < T) {
        stage_res();
        if (t + 2 < T) rload(t + 2);
      }
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) __builtin_amdgcn_raw_buffer_store_b128(w[q], yres, goff(T - 1, q), 0, 0);
    // the third 32-column block of a 256 x 192 tile's waves
    if constexpr (TN % BPC != 0) {
      constexpr int j = TN - 1;
      uint2 bw[4];
#pragma unroll
      for (int g = 0; g < 4; ++g)
        bw[g] = *reinterpret_cast<const uint2*>(blds + (j * 32 + g * 8 + half * 4) * 2);
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        __builtin_amdgcn_sched_barrier(0);
        uint32_t r[2][4];
        const uint32_t m = static_cast<uint32_t>(mb + i * 32 + l32);
        if (EPI == EPI_RESIDUAL) res_load32(rres, m, nb + j * 32, half, ep.ldy, r);
        epi_store32<EPI>(acc[i][j], bw, r, yres, m, nb + j * 32, half, ep.ldy);
      }
    }
  }
}

// Rotary epilogue of gemm_bf16_w4p_kernel: 256-wide tiles and head_dim 64
// or 128, so a wave's 128 columns hold whole heads and the partner c + hd/2
// of a channel c sits in the same lane, in another 32 x 32 block (the next
// one for head_dim 64, two further for 128). z = acc + bias; for each head
// below rope_cols and each channel pair (i, i + hd/2): lower = z_l cos -
// z_u sin, upper = z_u cos + z_l sin, the (cos, sin) of the row's position
// read from the per-row table (the values rope_angle gives); heads at or
// past rope_cols are stored as they are. Table rows past M read zeros
// through the buffer range check (and their stores are dropped).
template <int TM, int TN, int HD>
__device__ __forceinline__ void rope_epilogue_lb(const f32x16_t (&acc)[TM][TN], int mb, int nb, int M,
                                                 int l32, int half, const EpiParams& ep,
                                                 const unsigned char* blds) {
  static_assert(TN == 4 && (HD == 64 || HD == 128), "128-column wave blocks of whole heads");
  constexpr int HH = HD / 2;
  // Channel sets: head_dim 64 has one (channels 0..31, shared by the wave's
  // two heads), 128 two (0..31 and 32..63 of its one head); a step is one
  // set on one 32-row block
  constexpr int NSTEP = (HD / 64) * TM;
  const int ybytes = M * ep.ldy * 2;
  const __amdgpu_buffer_rsrc_t yres = __builtin_amdgcn_make_buffer_rsrc(ep.y, 0, ybytes, 0x00020000);
  const __amdgpu_buffer_rsrc_t tres = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<float*>(ep.rope_cs), 0, M * HH * 8, 0x00020000);
  uint32_t unused[2][4];
  const uint2 zb[4] = {make_uint2(0u, 0u), make_uint2(0u, 0u), make_uint2(0u, 0u), make_uint2(0u, 0u)};
  // table values of step it into buffer b: (cos, sin) of channels
  // 32 set + 8 g + 4 half .. + 3 of the lane's row, 32 bytes per g
  uint32_t tv[2][4][2][4];
  auto load_step = [&](int it, int b) {
    const int cset = it / TM, i = it % TM;
    const uint32_t m = static_cast<uint32_t>(mb + i * 32 + l32);
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const uint32_t toff =
          (m * static_cast<uint32_t>(HH) + static_cast<uint32_t>(32 * cset + 8 * g + 4 * half)) * 8u;
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        const auto t = __builtin_amdgcn_raw_buffer_load_b128(tres, toff + 16u * q, 0, 0);
#pragma unroll
        for (int w = 0; w < 4; ++w) tv[b][g][q][w] = t[w];
      }
    }
  };
  // The next step's table loads are issued before this step's stores:
  // vector memory operations are counted in issue order, so a load issued
  // after a store could only be waited for together with that store.
  load_step(0, 0);
#pragma unroll
  for (int it = 0; it < NSTEP; ++it) {
    __builtin_amdgcn_sched_barrier(0);
    if (it + 1 < NSTEP) load_step(it + 1, (it + 1) & 1);
    __builtin_amdgcn_sched_barrier(0);
    const int cset = it / TM, i = it % TM;
    const uint32_t m = static_cast<uint32_t>(mb + i * 32 + l32);
#pragma unroll
    for (int pr = 0; pr < 2; ++pr) {
      if (HD == 128 && pr != cset) continue;
      // blocks jl (lower channels) and ju (their partners) of one pair
      const int jl = HD == 64 ? 2 * pr : pr;
      const int ju = HD == 64 ? jl + 1 : jl + 2;
      const bool rot = nb + (HD == 64 ? 64 * pr : 0) < ep.rope_cols;
      f32x16_t lo, up;
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const uint2 bl = *reinterpret_cast<const uint2*>(blds + (jl * 32 + g * 8 + half * 4) * 2);
        const uint2 bu = *reinterpret_cast<const uint2*>(blds + (ju * 32 + g * 8 + half * 4) * 2);
        const float b[2][4] = {{__uint_as_float(bl.x << 16), __uint_as_float(bl.x & 0xffff0000u),
                                __uint_as_float(bl.y << 16), __uint_as_float(bl.y & 0xffff0000u)},
                               {__uint_as_float(bu.x << 16), __uint_as_float(bu.x & 0xffff0000u),
                                __uint_as_float(bu.y << 16), __uint_as_float(bu.y & 0xffff0000u)}};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float zl = acc[i][jl][4 * g + e] + b[0][e];
          const float zu = acc[i][ju][4 * g + e] + b[1][e];
          const float cs = __uint_as_float(tv[it & 1][g][e >> 1][(e & 1) * 2]);
          const float sn = __uint_as_float(tv[it & 1][g][e >> 1][(e & 1) * 2 + 1]);
          lo[4 * g + e] = rot ? zl * cs - zu * sn : zl;
          up[4 * g + e] = rot ? zu * cs + zl * sn : zu;
        }
      }
      epi_store32<EPI_NONE>(lo, zb, unused, yres, m, nb + jl * 32, half, ep.ldy);
      epi_store32<EPI_NONE>(up, zb, unused, yres, m, nb + ju * 32, half, ep.ldy);
    }
  }
}

// Rotary epilogue with head_dim 64 through the per-wave staging buffer of
// reg_epilogue_lds: a step (32 rows, one channel pair of blocks 2 pr and
// 2 pr + 1) is exactly one 32 x 64 chunk, written in the accumulator layout
// and stored as whole lines, the step's arithmetic overlapping the previous
// step's line reads. The table loads of the next row block are issued before
// the stores that follow them. Same box, us per projection (rotary table
// included): 16384 x 6144 x 2048 344.7 -> 341.4, 4096 x 6144 x 2048 105.3 ->
// 103.4. Head dim 128 pairs blocks 0 and 2, which are not adjacent, and
// keeps rope_epilogue_lb.
template <int TM, int TN, int HD>
__device__ __forceinline__ void rope_epilogue_lds(const f32x16_t (&acc)[TM][TN], int mb, int nb, int M,
                                                  int l32, int half, const EpiParams& ep,
                                                  const unsigned char* blds, unsigned char* stg) {
  if constexpr (HD != 64) {
    rope_epilogue_lb<TM, TN, HD>(acc, mb, nb, M, l32, half, ep, blds);
  } else {
    static_assert(TN == 4, "128-column wave blocks of whole heads");
    constexpr int HH = HD / 2;
    const int ybytes = M * ep.ldy * 2;
    const uint32_t ldy = static_cast<uint32_t>(ep.ldy);
    const __amdgpu_buffer_rsrc_t yres = __builtin_amdgcn_make_buffer_rsrc(ep.y, 0, ybytes, 0x00020000);
    const __amdgpu_buffer_rsrc_t tres = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(ep.rope_cs), 0, M * HH * 8, 0x00020000);
    uint32_t unused[2][4];
    const uint2 zb[4] = {make_uint2(0u, 0u), make_uint2(0u, 0u), make_uint2(0u, 0u), make_uint2(0u, 0u)};
    const int lane = l32 + 32 * half;
    const int lr = lane >> 3, lc = lane & 7;
    unsigned char* const sline = stg + lr * 128 + ((lc ^ lr) << 4);
    auto sacc = [&](int c) { return stg + l32 * 128 + ((c ^ (l32 & 7)) << 4); };
    // chunk t = 2 i + pr: rows mb + 32 i .., columns nb + 64 pr ..
    auto goff = [&](int t, int q) {
      return ((static_cast<uint32_t>(mb + 32 * (t >> 1) + lr + 8 * q)) * ldy +
              static_cast<uint32_t>(nb + 64 * (t & 1) + 8 * lc)) * 2u;
    };
    // (cos, sin) of channels 8 g + 4 half .. + 3 of the lane's row in row
    // block i, into buffer b
    uint32_t tv[2][4][2][4];
    auto load_step = [&](int i, int b) {
      const uint32_t m = static_cast<uint32_t>(mb + i * 32 + l32);
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const uint32_t toff = (m * static_cast<uint32_t>(HH) + static_cast<uint32_t>(8 * g + 4 * half)) * 8u;
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          const auto t = __builtin_amdgcn_raw_buffer_load_b128(tres, toff + 16u * q, 0, 0);
#pragma unroll
          for (int w = 0; w < 4; ++w) tv[b][g][q][w] = t[w];
        }
      }
    };
    u32x4 w[4];
    load_step(0, 0);
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      __builtin_amdgcn_sched_barrier(0);
      if (i + 1 < TM) load_step(i + 1, (i + 1) & 1);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int pr = 0; pr < 2; ++pr) {
        const int t = 2 * i + pr;
        const int jl = 2 * pr, ju = jl + 1;
        const bool rot = nb + 64 * pr < ep.rope_cols;
        f32x16_t lo, up;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const uint2 bl = *reinterpret_cast<const uint2*>(blds + (jl * 32 + g * 8 + half * 4) * 2);
          const uint2 bu = *reinterpret_cast<const uint2*>(blds + (ju * 32 + g * 8 + half * 4) * 2);
          const float b[2][4] = {{__uint_as_float(bl.x << 16), __uint_as_float(bl.x & 0xffff0000u),
                                  __uint_as_float(bl.y << 16), __uint_as_float(bl.y & 0xffff0000u)},
                                 {__uint_as_float(bu.x << 16), __uint_as_float(bu.x & 0xffff0000u),
                                  __uint_as_float(bu.y << 16), __uint_as_float(bu.y & 0xffff0000u)}};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float zl = acc[i][jl][4 * g + e] + b[0][e];
            const float zu = acc[i][ju][4 * g + e] + b[1][e];
            const float cs = __uint_as_float(tv[i & 1][g][e >> 1][(e & 1) * 2]);
            const float sn = __uint_as_float(tv[i & 1][g][e >> 1][(e & 1) * 2 + 1]);
            lo[4 * g + e] = rot ? zl * cs - zu * sn : zl;
            up[4 * g + e] = rot ? zu * cs + zl * sn : zu;
          }
        }
        u32x4 vl[2], vu[2];
        epi_pack32<EPI_NONE>(lo, zb, unused, vl);
        epi_pack32<EPI_NONE>(up, zb, unused, vu);
        if (t > 0) {
#pragma unroll
          for (int q = 0; q < 4; ++q) __builtin_amdgcn_raw_buffer_store_b128(w[q], yres, goff(t - 1, q), 0, 0);
        }
        asm volatile("" ::: "memory");
#pragma unroll
        for (int p = 0; p < 2; ++p) {
          *reinterpret_cast<u32x4*>(sacc(2 * p + half)) = vl[p];
          *reinterpret_cast<u32x4*>(sacc(4 + 2 * p + half)) = vu[p];
        }
        asm volatile("" ::: "memory");
#pragma unroll
        for (int q = 0; q < 4; ++q) w[q] = *reinterpret_cast<const u32x4*>(sline + q * 1024);
        asm volatile("" ::: "memory");
      }
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) __builtin_amdgcn_raw_buffer_store_b128(w[q], yres, goff(2 * TM - 1, q), 0, 0);
  }
}

// ---------------------------------------------------------------------------
// bf16 GEMM, persistent form of the four-wave kernel
// ---------------------------------------------------------------------------
// One workgroup per CU walks a strided share of its XCD's range of 256 x BN
// tiles (the grouped order above) and streams their K slices as one
// sequence: the loads of slice g + 2 run on into the next tile, so when the
// last slice of a tile has been multiplied, the first slices of the next are
// in flight or landed and the finished tile's epilogue overlaps them (a
// workgroup per tile would instead start each tile by waiting for its first
// slice). The slice loop is that of gemm_bf16_w4_kernel, generalised to
// BN = 256 (waves of 128 x 128) and BN = 192 (waves of 128 x 96, for N = 768
// and 2304, whose 256-wide tiles leave a round part-filled): each block
// spreads its fragment reads (and, in block B, its loads) evenly over its
// MFMAs. The bias of a tile travels with its first slice, as a
// direct-to-LDS load into one of two 1 KiB buffers (by tile parity), so the
// epilogue waits for no global load: such a wait would also wait for the
// slice loads issued before it, since vector memory operations complete in
// issue order. A tile's accumulators restart from MFMAs whose C operand is
// zero. K is at least two slices, so a bias buffer is refilled only after
// every wave has passed the epilogue that read it (the refill is issued
// after a barrier of the next tile).
template <int EPI, int BN>
__global__ __launch_bounds__(256) void gemm_bf16_w4p_kernel(const bf16_t* __restrict__ X,
                                                           const bf16_t* __restrict__ W, int M,
                                                           int N, int K, EpiParams ep) {
  constexpr int BM = 256, KB = 64;
  constexpr int TM = 4, TN = BN / 64;           // 32 x 32 blocks per wave (rows, columns)
  constexpr int NF = TM + TN;                   // fragments per 16-wide k-substep
  constexpr int NP = TM * TN;                   // MFMAs per k-substep
  constexpr int NMB = 2 * NP, NRB = 2 * NF;     // MFMAs and fragment reads per block
  using SL = Slice<KB>;
  constexpr int SB = (BM + BN) * SL::RB;        // bytes per stage
  constexpr int LPW = (BM + BN) / SL::RPD / 4;  // 1 KiB loads per wave per stage
  constexpr int ALD = BM / SL::RPD / 4;         // of which A rows
  static_assert(BN == 256 || BN == 192, "tile width");
  static_assert(NMB >= NRB && NMB >= LPW, "interleave");
  extern __shared__ __align__(16) unsigned char smem[];
  unsigned char* const blds = smem + 2 * SB;  // bias buffers, 1 KiB each, then 4 KiB of staging per wave
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;  // 2 x 2 waves of 128 x BN / 2
  const int l32 = lane & 31, half = lane >> 5;

  const int nM = (M + BM - 1) / BM, nN = N / BN;
  const int tiles = nM * nN;
  const int xcd = blockIdx.x % kXcds, slot = blockIdx.x / kXcds;
  const int slots = gridDim.x / kXcds;
  // XCD k's tiles: when the tile grid splits into 8 equal blocks (ra x rb
  // of them), the block (k / rb, k % rb) whose A rows and W columns add up
  // to the fewest panels (each XCD then fetches fewer operand bytes into its
  // L2 than a band of the whole grid would need); otherwise a contiguous,
  // balanced range of the grouped order. Inside either, groups of
  // kXcdGroup M-tiles with every N-tile of the range.
  int ra = 0, rb = 0, best = 0;
  for (int a = 1; a <= kXcds; a *= 2) {
    const int b = kXcds / a;
    if (nM % a != 0 || nN % b != 0) continue;
    const int cost = nM / a + nN / b;
    if (ra == 0 || cost < best) {
      ra = a;
      rb = b;
      best = cost;
    }
  }
  const int rm = ra > 0 ? nM / ra : nM, rn = ra > 0 ? nN / rb : nN;  // the range's grid
  const int rm0 = ra > 0 ? (xcd / rb) * rm : 0, rn0 = ra > 0 ? (xcd % rb) * rn : 0;
  const int per = tiles / kXcds, extra = tiles % kXcds;
  const int tbeg = ra > 0 ? 0 : xcd * per + min(xcd, extra);
  const int tcount = ra > 0 ? rm * rn : per + (xcd < extra ? 1 : 0);
  if (slot >= tcount) return;
  const int count = (tcount - slot + slots - 1) / slots;  // tiles of this workgroup
  const int KT = K / KB;
  auto tile_at = [&](int p, int* m0, int* n0) {
    const int t = tbeg + slot + p * slots;
    const int g = t / (kXcdGroup * rn);
    const int gm0 = g * kXcdGroup;
    const int gsz = min(kXcdGroup, rm - gm0);
    const int r = t - g * kXcdGroup * rn;
    *n0 = (rn0 + r / gsz) * BN;
    *m0 = (rm0 + gm0 + r % gsz) * BM;
  };
  const __amdgpu_buffer_rsrc_t xres =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16_t*>(X), 0, M * K * 2, 0x00020000);
  const __amdgpu_buffer_rsrc_t wres =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16_t*>(W), 0, N * K * 2, 0x00020000);
  // no bias: an empty range, whose loads read zeros
  const __amdgpu_buffer_rsrc_t bres = __builtin_amdgcn_make_buffer_rsrc(
      ep.bias != nullptr ? const_cast<void*>(ep.bias) : const_cast<bf16_t*>(X), 0,
      ep.bias != nullptr ? N * 2 : 0, 0x00020000);
  // wave w moves row blocks i * 4 + w of a stage (8 rows each; A rows, then
  // B rows); stage row r = 8 blk + lr has swizzle (4 blk + lr / 2) & 7,
  // which depends on blk only through the wave's parity
  const int lr = lane / SL::CPR, lp = lane % SL::CPR;
  const uint32_t lane_off =
      static_cast<uint32_t>(lr * K * 2 + swz<KB>((wave & 1) * SL::RPD + lr, lp) * 16);
  typedef __attribute__((address_space(3))) void lds_void;
  // abase / bbase: byte offsets of the slice's first A and B rows (its K
  // step included); 0x80000000 past the stream
  auto dma1 = [&](int st, uint32_t abase, uint32_t bbase, bool live, int i) {
    const int blk = i * 4 + wave;
    const uint32_t off =
        live ? (i < ALD ? abase + static_cast<uint32_t>(blk * SL::RPD) * K * 2u
                        : bbase + static_cast<uint32_t>((blk - 4 * ALD) * SL::RPD) * K * 2u) +
                   lane_off
             : 0x80000000u;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(i < ALD ? xres : wres,
                                             (lds_void*)(smem + st * SB + blk * 1024), 16, off, 0,
                                             0, 0);
  };
  // the bias of the tile at n0 into buffer p & 1 (lanes past the BN columns
  // fill the buffer's unused rest)
  auto bias_dma = [&](int p, int n0) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(bres, (lds_void*)(blds + (p & 1) * 1024), 16,
                                             static_cast<uint32_t>(n0 * 2 + lane * 16), 0, 0, 0);
  };
  // fragment q of k-substep kk: A block q (q < TM) or B block q - TM; row r
  // of a 32-row block sits at r * RB, its chunk c at (c ^ ((r / RPP) & 7)) * 16
  const int sw = (l32 / SL::RPP) & (SL::CPR - 1);
  int ab[4], bb[4];
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) {
    ab[kk] = (wm * 128 + l32) * SL::RB + ((kk * 2 + half) ^ sw) * 16;
    bb[kk] = BM * SL::RB + (wn * (BN / 2) + l32) * SL::RB + ((kk * 2 + half) ^ sw) * 16;
  }
  f32x16_t acc[TM][TN];
  // f0: fragments of k-substeps 0, 1 of a slice; f1: of k-substeps 2, 3
  bf16x8_t f0[2][NF], f1[2][NF];
  auto rd1 = [&](const unsigned char* st, int kk, bf16x8_t (&f)[NF], int q) {
    const int off = q < TM ? ab[kk] + q * 32 * SL::RB : bb[kk] + (q - TM) * 32 * SL::RB;
    f[q] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const u32x4*>(st + off));
  };
  // MFMA p of a k-substep: output block (p / TN, p % TN), operands swapped
  // so the accumulator holds C^T (four consecutive columns per register group)
  auto mma1 = [&](bf16x8_t (&f)[NF], int p) {
    acc[p / TN][p % TN] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f[TM + p % TN], f[p / TN],
                                                                  acc[p / TN][p % TN], 0, 0, 0);
  };
  auto mma0 = [&](bf16x8_t (&f)[NF], int p) {
    const f32x16_t zero = {};
    acc[p / TN][p % TN] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f[TM + p % TN], f[p / TN], zero, 0, 0, 0);
  };
  // prologue: the first tile's bias and slices 0 and 1 in flight, slice 0
  // (and the bias) published, its first fragments read
  int m0, n0;
  tile_at(0, &m0, &n0);
  {
    const uint32_t abase = static_cast<uint32_t>(m0) * K * 2u;
    const uint32_t bbase = static_cast<uint32_t>(n0) * K * 2u;
    if (wave == 0) bias_dma(0, n0);
#pragma unroll
    for (int i = 0; i < LPW; ++i) dma1(0, abase, bbase, true, i);
#pragma unroll
    for (int i = 0; i < LPW; ++i) dma1(1, abase + KB * 2, bbase + KB * 2, true, i);
  }
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(vmcnt_imm(LPW));
  barrier_lds();
#pragma unroll
  for (int q = 0; q < NF; ++q) {
    rd1(smem, 0, f0[0], q);
    rd1(smem, 1, f0[1], q);
  }
  // the load stream runs two slices ahead: tile dp, K step dt
  int dp = KT > 2 ? 0 : 1, dt = KT > 2 ? 2 : 0;
  int dm0 = m0, dn0 = n0;
  if (dp == 1 && count > 1) tile_at(1, &dm0, &dn0);
  int s = 0;
  // fragment read r of a block follows MFMA r * NMB / NRB; load d of block B
  // follows MFMA d * NMB / LPW + 1 (the order is pinned by the scheduling
  // barriers)
  // block A: the MFMAs of the slice's first 32 K values with the reads of
  // its last 32 K values' fragments (the first slice of a tile starts its
  // sums from zero)
  auto block_a = [&](auto first) {
    const unsigned char* cur = smem + s * SB;
#pragma unroll
    for (int mi = 0; mi < NMB; ++mi) {
      __builtin_amdgcn_sched_barrier(0);
      if (decltype(first)::value && mi < NP) mma0(f0[0], mi); else mma1(f0[mi / NP], mi % NP);
#pragma unroll
      for (int r = 0; r < NRB; ++r)
        if (r * NMB / NRB == mi) rd1(cur, 2 + r / NF, f1[r / NF], r % NF);
    }
    __builtin_amdgcn_sched_barrier(0);
    // the next slice (and any earlier epilogue's stores) have landed
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
    barrier_lds();
  };
  // block B: the MFMAs of the last 32 K values with the loads of the stream's
  // next slice into this slice's stage and (but in a tile's last slice) the
  // reads of the next slice's first fragments
  auto block_b = [&](auto last) {
    const unsigned char* nxt = smem + (s ^ 1) * SB;
    const bool live = dp < count;
    const uint32_t abase = static_cast<uint32_t>(dm0) * K * 2u + static_cast<uint32_t>(dt * KB * 2);
    const uint32_t bbase = static_cast<uint32_t>(dn0) * K * 2u + static_cast<uint32_t>(dt * KB * 2);
#pragma unroll
    for (int mi = 0; mi < NMB; ++mi) {
      __builtin_amdgcn_sched_barrier(0);
      mma1(f1[mi / NP], mi % NP);
#pragma unroll
      for (int r = 0; r < NRB; ++r)
        if (!decltype(last)::value && r * NMB / NRB == mi) rd1(nxt, r / NF, f0[r / NF], r % NF);
#pragma unroll
      for (int d = 0; d < LPW; ++d)
        if (d * NMB / LPW + 1 == mi) dma1(s, abase, bbase, live, d);
    }
    __builtin_amdgcn_sched_barrier(0);
    if (live && dt == 0 && wave == 0) bias_dma(dp, dn0);
    if (++dt == KT) {
      dt = 0;
      if (++dp < count) tile_at(dp, &dm0, &dn0);
    }
    s ^= 1;
  };
  using yes = std::integral_constant<bool, true>;
  using no = std::integral_constant<bool, false>;
  for (int p = 0; p < count; ++p) {
    block_a(yes{});
    block_b(no{});
    for (int t = 1; t + 1 < KT; ++t) {
      block_a(no{});
      block_b(no{});
    }
    block_a(no{});
    block_b(yes{});
    if constexpr (EPI == EPI_ROPE || EPI == kEpiRope128)
      rope_epilogue_lds<TM, TN, EPI == EPI_ROPE ? 64 : 128>(acc, m0 + wm * 128, n0 + wn * (BN / 2), M,
                                                            l32, half, ep, blds + (p & 1) * 1024 + wn * BN,
                                                            blds + 2048 + wave * 4096);
    else
      reg_epilogue_lds<TM, TN, EPI>(acc, m0 + wm * 128, n0 + wn * (BN / 2), M, l32, half, ep,
                                    blds + (p & 1) * 1024 + wn * BN, blds + 2048 + wave * 4096);
    if (p + 1 < count) {
      tile_at(p + 1, &m0, &n0);
      // the next tile's first fragments (its slice 0 was published by the
      // barrier of this tile's last slice)
#pragma unroll
      for (int q = 0; q < NF; ++q) {
        rd1(smem + s * SB, 0, f0[0], q);
        rd1(smem + s * SB, 1, f0[1], q);
      }
    }
  }
}

template <int EPI, int BN>
hipError_t launch_w4p_1(hipStream_t s, const void* x, int M, int K, const void* w, int N,
                        const EpiParams& ep) {
  // stages, bias buffers and (plain, residual and head-dim-64 rotary
  // epilogues) 4 KiB of epilogue staging per wave
  constexpr int lds = 2 * (256 + BN) * 64 * 2 + 2 * 1024 +
                      (EPI == EPI_NONE || EPI == EPI_RESIDUAL || EPI == EPI_ROPE ? 4 * 4096 : 0);
  static bool lds_raised = false;
  if (!lds_raised) {
    const hipError_t e = hipFuncSetAttribute(
        reinterpret_cast<const void*>(gemm_bf16_w4p_kernel<EPI, BN>),
        hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    if (e != hipSuccess) return e;
    lds_raised = true;
  }
  const int tiles = ((M + 255) / 256) * (N / BN);
  const int wgs = std::min(tiles, device_cus());
  const int grid = kXcds * ((wgs + kXcds - 1) / kXcds);
  return launch(K_GEMM, gemm_bf16_w4p_kernel<EPI, BN>, dim3(grid), dim3(256), lds, s,
                static_cast<const bf16_t*>(x), static_cast<const bf16_t*>(w), M, N, K, ep);
}

// the four-wave kernel takes the products the persistent one takes, with N a
// multiple of 256 and both operands below 2^31 bytes (buffer range checks)
bool w4_ok(int M, int N, int K, const EpiParams& ep) {
  return persist_ok(M, N, K, ep) && N % 256 == 0 &&
         static_cast<int64_t>(M + 256) * K * 2 < (int64_t{1} << 31) &&
         static_cast<int64_t>(N) * K * 2 < (int64_t{1} << 31);
}

hipError_t launch_w4(hipStream_t s, const void* x, int M, int K, const void* w, int N,
                     const EpiParams& ep) {
  if (ep.epi == EPI_GELU) return launch_w4_1<EPI_GELU>(s, x, M, K, w, N, ep);
  if (ep.epi == EPI_RESIDUAL) return launch_w4_1<EPI_RESIDUAL>(s, x, M, K, w, N, ep);
  if (ep.epi == EPI_SWIGLU) return launch_w4_1<EPI_SWIGLU>(s, x, M, K, w, N, ep);
  return launch_w4_1<EPI_NONE>(s, x, M, K, w, N, ep);
}

// the persistent four-wave kernel: the four-wave kernel's products with K of
// at least two slices (bn: the tile width, 256 or 192, which N is a multiple of)
bool w4p_ok(int M, int N, int K, const EpiParams& ep, int bn = 256) {
  if (ep.epi == EPI_ROPE) {
    // the rotary epilogue: 256-wide tiles (whole heads per wave) and a table
    if (bn != 256 || ep.rope_cs == nullptr || (ep.head_dim != 64 && ep.head_dim != 128) ||
        ep.rope_cols % ep.head_dim != 0 || N % ep.head_dim != 0 ||
        static_cast<int64_t>(M) * (ep.head_dim / 2) * 8 >= (int64_t{1} << 31))
      return false;
    EpiParams plain = ep;
    plain.epi = EPI_NONE;
    return w4p_ok(M, N, K, plain, bn);
  }
  return persist_ok(M, N, K, ep) && N % bn == 0 && K >= 128 &&
         static_cast<int64_t>(M + 256) * K * 2 < (int64_t{1} << 31) &&
         static_cast<int64_t>(N) * K * 2 < (int64_t{1} << 31);
}

// Tile width (256 or 192) of the persistent four-wave kernel for a product,
// or 0 where it does not pay. Measured on M = 2048 .. 16384, N = 768 ..
// 3072, K = 768 and 3072 against the persistent 128x128 kernel (which needs
// twice the operand bytes per FLOP): a width pays when its tiles fill their
// last round on the CUs at least half (three-quarters with the GELU
// epilogue, which one wave per SIMD leaves exposed), or number at least
// 0.68 of one round (16384 x 768 x 3072, 256 wide, 192 tiles: 69.2 against
// 78.0 us; 11456 x 768 x 3072, 192 wide, 180 tiles: 58.3 against 77.9;
// 2748 x 3072 x 768 with GELU, 192 wide, 176 tiles: 22.6 against 25.8;
// 11456 x 2304 x 768, 256 wide, 1.58 rounds: 47.6 against 51.6; the
// rotary 4096 x 6144 x 2048, 1.5 rounds: the 16-layer decoder at keep rate
// 0.5 15.64 -> 15.54 ms); rounds filled less lose (16384 x 2304 x 768, 256
// wide, 2.25 rounds: 68.0 against 67.4 us; 8192 x 768 x 3072, 192 wide, half
// a round: 52.3 against 47.8 us; 10485 x 768 x 768, 0.64 of a round: 22.8
// against 20.4; 6710 x 3072 x 768 with GELU, 1.69 rounds: 45.8 against
// 41.3). Of the widths that pay, the better-filled
// one is taken, 256 on a tie (more FLOPs per operand byte): 192 for
// 16384 x 2304 x 768 (three whole rounds: 57.9 us) and 16384 x 768 x K (one:
// 25.8 and 65.2 us for K = 768 and 3072), 256 for 16384 x 3072 x 768 (85.9
// us; persistent 128x128 95.2). For K > 3072 (the 4096-wide decoder) a
// width pays from one whole round of tiles on.
int w4p_width(int M, int N, int K, const EpiParams& ep) {
  const long cus = device_cus();
  int best = 0;
  long best_fill = 0, best_slots = 1;  // the fill best_fill / best_slots
  for (const int bn : {256, 192}) {
    if (!w4p_ok(M, N, K, ep, bn)) continue;
    const long tiles = static_cast<long>((M + 255) / 256) * (N / bn);
    const long rem = tiles % cus;
    bool pays;
    if (K > 3072) pays = tiles >= cus;
    else if (tiles >= cus) pays = rem == 0 || (ep.epi == EPI_GELU ? 4 * rem >= 3 * cus : 2 * rem >= cus);
    else pays = 100 * tiles >= 68 * cus;
    if (!pays) continue;
    const long slots = (tiles + cus - 1) / cus * cus;
    if (best == 0 || tiles * best_slots > best_fill * slots) {
      best = bn;
      best_fill = tiles;
      best_slots = slots;
    }
  }
  return best;
}

template <int BN>
hipError_t launch_w4p(hipStream_t s, const void* x, int M, int K, const void* w, int N,
                      const EpiParams& ep) {
  if (ep.epi == EPI_ROPE) {
    if constexpr (BN == 256) {
      if (ep.head_dim == 64) return launch_w4p_1<EPI_ROPE, 256>(s, x, M, K, w, N, ep);
      if (ep.head_dim == 128) return launch_w4p_1<kEpiRope128, 256>(s, x, M, K, w, N, ep);
    }
    return hipErrorInvalidValue;
  }
  if (ep.epi == EPI_GELU) return launch_w4p_1<EPI_GELU, BN>(s, x, M, K, w, N, ep);
  if (ep.epi == EPI_RESIDUAL) return launch_w4p_1<EPI_RESIDUAL, BN>(s, x, M, K, w, N, ep);
  if (ep.epi == EPI_SWIGLU) return launch_w4p_1<EPI_SWIGLU, BN>(s, x, M, K, w, N, ep);
  return launch_w4p_1<EPI_NONE, BN>(s, x, M, K, w, N, ep);
}

template <int KB, int WPC>
hipError_t launch_persist_any(hipStream_t s, const void* x, int M, int K, const void* w, int N,
                              const EpiParams& ep) {
  if (ep.epi == EPI_GELU) return launch_persist<EPI_GELU, KB, WPC>(s, x, M, K, w, N, ep);
  if (ep.epi == EPI_RESIDUAL) return launch_persist<EPI_RESIDUAL, KB, WPC>(s, x, M, K, w, N, ep);
  if (ep.epi == EPI_SWIGLU) return launch_persist<EPI_SWIGLU, KB, WPC>(s, x, M, K, w, N, ep);
  return launch_persist<EPI_NONE, KB, WPC>(s, x, M, K, w, N, ep);
}

template <int BM, int BN, int WM, int WN>
hipError_t launch_mfma(hipStream_t s, const void* x, int M, int K, const void* w, int N,
                       const EpiParams& ep) {
  constexpr int lds = mfma_lds_bytes<BM, BN>();
  static bool lds_raised = false;  // more than 64 KiB of dynamic LDS per workgroup
  if (!lds_raised) {
    const hipError_t e = hipFuncSetAttribute(
        reinterpret_cast<const void*>(gemm_bf16_mfma_kernel<BM, BN, WM, WN>),
        hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    if (e != hipSuccess) return e;
    lds_raised = true;
  }
  const dim3 grid((M + BM - 1) / BM, (N + BN - 1) / BN);
  return launch(K_GEMM, gemm_bf16_mfma_kernel<BM, BN, WM, WN>, grid, dim3(WM * WN * 64), lds, s,
                static_cast<const bf16_t*>(x), static_cast<const bf16_t*>(w), M, N, K, ep);
}

template <int BM, int BN, int WM, int WN, int KB, int NS, int ER>
hipError_t launch_dma(hipStream_t s, const void* x, int M, int K, const void* w, int N,
                      const EpiParams& ep, int S = 1, int kchunk = 0, float* part = nullptr) {
  constexpr int lds = dma_lds_bytes<BM, BN, KB, NS, ER>();
  static bool lds_raised = false;
  if (!lds_raised) {
    const hipError_t e = hipFuncSetAttribute(
        reinterpret_cast<const void*>(gemm_bf16_dma_kernel<BM, BN, WM, WN, KB, NS, ER>),
        hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    if (e != hipSuccess) return e;
    lds_raised = true;
  }
  dim3 grid = xcd_grid(M, N, BM, BN);
  grid.y = S;
  return launch(K_GEMM, gemm_bf16_dma_kernel<BM, BN, WM, WN, KB, NS, ER>, grid,
                dim3(WM * WN * 64), lds, s, static_cast<const bf16_t*>(x),
                static_cast<const bf16_t*>(w), M, N, K, ep, S > 1 ? kchunk : K, part);
}

// ZSA_GEMM_TILE pins one kernel variant (a tuning aid; 0 or unset = by shape):
// 128 / 256 / 2564 / 2568: register-staged 128x128, 256x128, 256x256 on 4 and
// on 8 waves; 1281 / 2563 / 2562 / 2561: direct-to-LDS 128x128, 256x128,
// 256x256 on 4 and on 8 waves (64-wide K slices, 2 stages); 3241: 128x128
// with 32-wide slices in 4 stages; 6431: 128x128 with 3 stages; 2542:
// 256x256 on 4 waves (128x128 per wave) with 64-row epilogue passes; 1289:
// the persistent 128x128 kernel; 2544: the 256x256 four-wave kernel with
// pinned MFMA / fragment-read interleaving and the epilogue in registers;
// 2545: its persistent form; 1925: that with 256x192 tiles.
int gemm_tile_override() {
  static const int v = [] {
    const char* e = getenv("ZSA_GEMM_TILE");
    return e == nullptr ? 0 : atoi(e);
  }();
  return v;
}

}  // namespace

// Split K when the 128 x 128 output tiles fill under 0.7 of the CUs once
// and K is long (at least kMinSplitK): S slices of at least
// kMinSplitSteps K steps, S x tiles <= 512 workgroups (one round, no tail).
// Every slice is non-empty and all but the last have kchunk columns. Per
// projection (both launches), M x 768 x 3072 with a residual: 256 rows 26.6
// -> 15.9 us, 2048 rows 31.7 -> 27.1, 3584 rows (168 tiles) 34.0 -> 32.5,
// 3904 rows (186 tiles) 34.9 -> 39.6 (not split), 4096 rows (192 tiles)
// 32.1 -> 35.5 (not split); 1024 x 2048 x 8192 71.5
// (persistent 128 x 128) -> 53.4. Up to K = 2048 launch_gemm leaves the
// products the persistent 128x128 kernel takes unsplit (1024 x 2048 x 2048
// with a residual: split 27.7 against 22.8 us on that kernel), but the
// rotary products of the same grids, which it does not take, need the
// split (the 1B-shaped decoder at keep rate 0.1 9.66 -> 9.73 ms without).
void splitk_plan(int M, int N, int K, int* S, int* kchunk) {
  *S = 1;
  *kchunk = K;
  if (K % kBK != 0 || K < kMinSplitK) return;
  const long tiles = static_cast<long>((M + 127) / 128) * ((N + 127) / 128);
  const int steps = K / kBK;
  if (10 * tiles >= 7 * device_cus()) return;
  const int want = std::min(static_cast<int>(512 / tiles), steps / kMinSplitSteps);
  if (want < 2) return;
  const int per = (steps + want - 1) / want;
  *S = (steps + per - 1) / per;
  *kchunk = per * kBK;
}

int device_cu_count() { return device_cus(); }

// Few-row products: one workgroup per 16 output columns; each of its waves
// takes a K range of whole 32-wide steps.
bool skinny_ok(int dtype, int M, int N, int K, const EpiParams& ep) {
  if (dtype != 1 || M < 1 || M > kSkMaxRows || K % 32 != 0 || K < 32) return false;
  if (static_cast<int64_t>(N + 4 * kSkCols) * K * 2 >= (int64_t{1} << 31)) return false;
  if (ep.epi == EPI_SWIGLU && N % 2 != 0) return false;
  if (ep.epi == EPI_ROPE && (ep.head_dim < 16 || ep.head_dim % 16 != 0 || N % ep.head_dim != 0))
    return false;
  return true;
}

// The few-row kernel replaces the tiled ones for short products: its loads
// go straight to the matrix cores with no tile rounding of M, but each
// block of 16 (32) rows re-reads W (from L2) and each block of 16 (32)
// columns re-reads x. Measured (us per call, W of each call not in L2;
// few-row with one / two 16-column blocks per workgroup against the tiled
// kernels chosen by shape):
//   M x N x K                 few-row 1 / 2   tiled
//   4 x 4096 x 14336          24.1 / 31.3     28.6   (every M <= 16: few-row)
//   40 x 6144 x 2048          11.2 / 10.5     14.1
//   40 x 16384 x 2048         26.7 / 23.2     20.8   (128 tiles of 128 x 128)
//   160 x 3072 x 768 (GELU)    7.2 /  6.0     10.7
//   160 x 768 x 3072           6.4 /  7.9     12.9
//   163 x 6144 x 2048         27.4 / 21.8     21.9   (96 tiles)
//   163 x 2048 x 8192         30.6 / 26.6     24.1
//   256 x 3072 x 768 (GELU)   10.2 /  8.7     10.8
//   512 x 2304 x 768          13.6 / 11.4      9.9   (72 tiles)
//   512 x 768 x 3072          14.3 / 13.4     18.8
//   640 x 768 x 3072               /  14.0     19.4   (policy's choice)
//   1024 x 768 x 768               /   8.5     10.3
//   1024 x 768 x 3072              /  20.2     22.8
// so it takes M <= 16, and up to 1024 rows while the 128 x 128 output
// tiles are fewer than 64 (past 512 rows: 768-column outputs).
bool skinny_pays(int M, int N, int K) {
  (void)K;
  const long tiles128 = static_cast<long>((M + 127) / 128) * ((N + 127) / 128);
  return M <= kSkMaxM || (M <= 1024 && tiles128 < 64);
}

// The folded pre-norm: every workgroup normalises the x fragments it
// reads (its statistics from one more read of its rows), which pays only
// while the rows are one per wave and the workgroups few: at most two per
// CU (a q|k|v projection in generation; not a wide up-projection, where a
// separate normalisation is cheaper than re-doing it in each of thousands
// of workgroups). Folded into the 160-row projections of the every-layer
// GPT-2-shaped stack it made the step at keep rate 0.02 0.705 -> 0.872 ms.
bool skinny_norm_ok(int M, int N, int K) {
  return M >= 1 && M <= kSkWaves && K % 32 == 0 && K <= 4096 &&
         (N + kSkCols - 1) / kSkCols <= 2 * device_cus();
}

// 16-row blocks per workgroup of the few-row kernel: two past 16 rows
int skinny_mb(int M, int N, int K) {
  (void)N;
  (void)K;
  return M <= kSkMaxM ? 1 : 2;
}

// 16-column blocks per workgroup: two for grids of two-row-block
// workgroups of at least 512, or 384 when K >= 1024 (the x re-reads they
// save outweigh the workgroups lost; table above); one up to 16 rows
// (generation streams W, which the x rows barely add to).
int skinny_cb(int M, int N, int K) {
  if (skinny_mb(M, N, K) < 2) return 1;
  const long wgs =
      static_cast<long>((N + kSkCols - 1) / kSkCols) * ((M + 2 * kSkMaxM - 1) / (2 * kSkMaxM));
  return wgs >= 512 || (wgs >= 384 && K >= 1024) ? 2 : 1;
}

hipError_t launch_gemm_skinny(hipStream_t s, const void* x, int M, int K, const void* w, int N,
                              const EpiParams& ep, const PreNorm* pn) {
  if (M == 0 || N == 0) return hipSuccess;
  const int kc = ((K + kSkWaves * 64 - 1) / (kSkWaves * 64)) * 64;  // whole 64-wide groups
  const bf16_t* xp = static_cast<const bf16_t*>(x);
  const bf16_t* wp = static_cast<const bf16_t*>(w);
  const dim3 block(kSkWaves * 64);
  const int nblk = (N + kSkCols - 1) / kSkCols;
  const bool norm = pn != nullptr && pn->g != nullptr;
  const int mb = norm ? 1 : skinny_mb(M, N, K);
  const int cb = norm ? 1 : skinny_cb(M, N, K);
  const dim3 grid((nblk + cb - 1) / cb, (M + kSkMaxM * mb - 1) / (kSkMaxM * mb));
#define ZSA_SK_LAUNCH(CPL_, MB_, CB_, DB_, LDS_, PN_)                                            \
  return launch(K_GEMM, gemm_skinny_kernel<CPL_, MB_, CB_, DB_>, grid, block, LDS_, s, xp, wp, M, \
                N, K, kc, ep, PN_)
  // two buffers when a wave's K range is longer than one full round
  const bool db = kc > 64 * sk_groups(mb, cb, false);
  if (!norm) {
    if (mb >= 2) {
      if (cb >= 2) {
        if (db) ZSA_SK_LAUNCH(0, 2, 2, true, 0, PreNorm{});
        ZSA_SK_LAUNCH(0, 2, 2, false, 0, PreNorm{});
      }
      if (db) ZSA_SK_LAUNCH(0, 2, 1, true, 0, PreNorm{});
      ZSA_SK_LAUNCH(0, 2, 1, false, 0, PreNorm{});
    }
    if (db) ZSA_SK_LAUNCH(0, 1, 1, true, 0, PreNorm{});
    ZSA_SK_LAUNCH(0, 1, 1, false, 0, PreNorm{});
  }
  if (!skinny_norm_ok(M, N, K)) return hipErrorInvalidValue;
  const size_t lds = static_cast<size_t>(K) / 8 * 2 * sizeof(uint4);
  const int cpl = (K / 8 + 63) / 64;
  if (db) {
    if (cpl <= 2) ZSA_SK_LAUNCH(2, 1, 1, true, lds, *pn);
    if (cpl <= 4) ZSA_SK_LAUNCH(4, 1, 1, true, lds, *pn);
    ZSA_SK_LAUNCH(8, 1, 1, true, lds, *pn);
  }
  if (cpl <= 2) ZSA_SK_LAUNCH(2, 1, 1, false, lds, *pn);
  if (cpl <= 4) ZSA_SK_LAUNCH(4, 1, 1, false, lds, *pn);
  ZSA_SK_LAUNCH(8, 1, 1, false, lds, *pn);
#undef ZSA_SK_LAUNCH
}

size_t splitk_bytes(int S, int M, int N) {
  return S > 1 ? static_cast<size_t>(S) * M * N * sizeof(float) : 0;
}

size_t gemm_workspace_bytes(int dtype, int M, int N, int K) {
  if (dtype != 1) return 0;
  int S, kchunk;
  splitk_plan(M, N, K, &S, &kchunk);
  return splitk_bytes(S, M, N);
}

size_t gemm_workspace_bound(int dtype, int max_rows, int N, int K) {
  size_t b = 0;
  // within a 128-row bucket the plan is fixed and the need grows with M, so
  // the largest M of each bucket bounds it
  for (int mt = 1; (mt - 1) * 128 < max_rows; ++mt) {
    const int m = std::min(mt * 128, max_rows);
    b = std::max(b, gemm_workspace_bytes(dtype, m, N, K));
  }
  return b;
}

namespace {
__global__ __launch_bounds__(256) void rope_table_kernel(const int32_t* __restrict__ pos, int M,
                                                         int hh, EpiParams ep,
                                                         float2* __restrict__ out) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (idx >= static_cast<int64_t>(M) * hh) return;
  const int m = static_cast<int>(idx / hh), i = static_cast<int>(idx % hh);
  float sn, cs;
  rope_angle(pos[m], ep.inv_freq[i], &sn, &cs);
  out[idx] = make_float2(cs, sn);
}
}  // namespace

hipError_t launch_rope_table(hipStream_t s, const int32_t* pos, int M, const EpiParams& ep,
                             float* out) {
  const int hh = ep.head_dim / 2;
  const int64_t n = static_cast<int64_t>(M) * hh;
  if (n == 0) return hipSuccess;
  return launch(K_GEMM, rope_table_kernel, dim3(static_cast<unsigned>((n + 255) / 256)),
                dim3(256), 0, s, pos, M, hh, ep, reinterpret_cast<float2*>(out));
}

// out[M][N] = x W^T in fp32 (no epilogue): the weight gradients of the
// backward pass (few output tiles, K = the rows of the batch); bf16
// operands with K a multiple of 64. Small grids split K as the forward
// does, and the slices are added in slice order.
hipError_t launch_gemm_f32(hipStream_t s, const void* x, int M, int K, const void* w, int N,
                           float* out, void* ws, size_t ws_bytes) {
  if (M == 0 || N == 0) return hipSuccess;
  if (K % kBK != 0) return hipErrorInvalidValue;
  EpiParams ep{};
  int S = 1, kchunk = K;
  splitk_plan(M, N, K, &S, &kchunk);
  if (S > 1 && ws != nullptr && ws_bytes >= splitk_bytes(S, M, N)) {
    float* part = static_cast<float*>(ws);
    const hipError_t e = launch_dma<128, 128, 2, 2, 64, 2, 128>(s, x, M, K, w, N, ep, S, kchunk, part);
    if (e != hipSuccess) return e;
    const int64_t total4 = static_cast<int64_t>(M) * N / 4;
    return launch(K_GEMM, splitk_sum_f32_kernel, dim3(static_cast<unsigned>((total4 + 255) / 256)),
                  dim3(256), 0, s, static_cast<const float4*>(ws), S, total4,
                  reinterpret_cast<float4*>(out));
  }
  return launch_dma<128, 128, 2, 2, 64, 2, 128>(s, x, M, K, w, N, ep, 1, K, out);
}

size_t gemm_f32_workspace_bound(int M, int N, int K) {
  int S, kchunk;
  splitk_plan(M, N, K, &S, &kchunk);
  return splitk_bytes(S, M, N);
}

bool gemm_takes_skinny(int dtype, int M, int N, int K, const EpiParams& ep) {
  return gemm_tile_override() == 0 && skinny_ok(dtype, M, N, K, ep) && skinny_pays(M, N, K);
}

hipError_t launch_gemm(hipStream_t s, int dtype, const void* x, int M, int K, const void* w,
                       int N, const EpiParams& ep, void* ws, size_t ws_bytes) {
  if (M == 0 || N == 0) return hipSuccess;
  if (gemm_takes_skinny(dtype, M, N, K, ep)) return launch_gemm_skinny(s, x, M, K, w, N, ep);
  if (dtype == 1 && K % kBK == 0) {
    int S = 1, kchunk = K;
    splitk_plan(M, N, K, &S, &kchunk);
    // (K <= 2048: the persistent 128x128 kernel beats the split where it
    // takes the epilogue; see splitk_plan)
    if (S > 1 && ws != nullptr && ws_bytes >= splitk_bytes(S, M, N) &&
        !(K <= 2048 && persist_ok(M, N, K, ep))) {
      float* part = static_cast<float*>(ws);
      const hipError_t e =
          launch_dma<128, 128, 2, 2, 64, 2, 128>(s, x, M, K, w, N, ep, S, kchunk, part);
      if (e != hipSuccess) return e;
      return launch(K_GEMM, splitk_reduce_kernel,
                    dim3((M + kRedRows - 1) / kRedRows, (N + kRedCols - 1) / kRedCols), dim3(256),
                    0, s, static_cast<const float*>(part), S, M, N, ep);
    }
    switch (gemm_tile_override()) {
      case 128: return launch_mfma<128, 128, 2, 2>(s, x, M, K, w, N, ep);
      case 256: return launch_mfma<256, 128, 2, 2>(s, x, M, K, w, N, ep);
      case 2564: return launch_mfma<256, 256, 2, 2>(s, x, M, K, w, N, ep);
      case 2568: return launch_mfma<256, 256, 2, 4>(s, x, M, K, w, N, ep);
      case 1281: return launch_dma<128, 128, 2, 2, 64, 2, 128>(s, x, M, K, w, N, ep);
      case 2563: return launch_dma<256, 128, 2, 2, 64, 2, 128>(s, x, M, K, w, N, ep);
      case 2562: return launch_dma<256, 256, 2, 2, 64, 2, 128>(s, x, M, K, w, N, ep);
      case 2561: return launch_dma<256, 256, 2, 4, 64, 2, 128>(s, x, M, K, w, N, ep);
      case 3241: return launch_dma<128, 128, 2, 2, 32, 4, 64>(s, x, M, K, w, N, ep);
      case 6431: return launch_dma<128, 128, 2, 2, 64, 3, 64>(s, x, M, K, w, N, ep);
      case 2542: return launch_dma<256, 256, 2, 2, 64, 2, 64>(s, x, M, K, w, N, ep);
      case 1289:
        if (persist_ok(M, N, K, ep)) return launch_persist_any<64, 2>(s, x, M, K, w, N, ep);
        break;
      case 2544:
        if (w4_ok(M, N, K, ep)) return launch_w4(s, x, M, K, w, N, ep);
        break;
      case 2545:
        if (w4p_ok(M, N, K, ep)) return launch_w4p<256>(s, x, M, K, w, N, ep);
        break;
      case 1925:
        if (w4p_ok(M, N, K, ep, 192)) return launch_w4p<192>(s, x, M, K, w, N, ep);
        break;
      default: break;
    }
    // Measured on the projection shapes of the 768-wide stacks (N = 768,
    // 2304, 3072; K = 768, 3072; M = 2048 .. 16384): the persistent
    // four-wave kernel where w4p_width finds a tile width that pays, the
    // persistent 128x128 kernel otherwise. For longer K (the decoders, K =
    // 4096 .. 14336): the persistent four-wave kernel from one round of its
    // tiles on (8192 x 4096 x 14336: 754 against 994 us for the 8-wave
    // kernel below; 4096 x 6144 x 4096: 173 against 210 us), else -- and for
    // the rotary and SwiGLU epilogues -- direct-to-LDS 256x256 tiles over 8
    // waves (128x64 per wave) once the grid holds at least four rounds of
    // them, else the persistent 128x128 kernel (1632 x 2048 x 8192: 74.5
    // against 81.3 us direct-to-LDS 128x128; 1472 x 4096 x 4096 61.8 against
    // 65.7; 3276 x 4096 x 14336 432 against 430), or direct-to-LDS 128x128
    // tiles for the epilogues it lacks.
    const int bn = w4p_width(M, N, K, ep);
    if (bn == 256) return launch_w4p<256>(s, x, M, K, w, N, ep);
    if (bn == 192) return launch_w4p<192>(s, x, M, K, w, N, ep);
    if (K <= 3072 && persist_ok(M, N, K, ep)) return launch_persist_any<64, 2>(s, x, M, K, w, N, ep);
    const long tiles256 = static_cast<long>((M + 255) / 256) * ((N + 255) / 256);
    if (tiles256 >= 1024) return launch_dma<256, 256, 2, 4, 64, 2, 128>(s, x, M, K, w, N, ep);
    if (persist_ok(M, N, K, ep)) return launch_persist_any<64, 2>(s, x, M, K, w, N, ep);
    return launch_dma<128, 128, 2, 2, 64, 2, 128>(s, x, M, K, w, N, ep);
  }
  const dim3 grid((M + vBM - 1) / vBM, (N + vBN - 1) / vBN);
  if (dtype == 1)
    return launch(K_GEMM, gemm_valu_kernel<bf16_t>, grid, dim3(256), 0, s,
                  static_cast<const bf16_t*>(x), static_cast<const bf16_t*>(w), M, N, K, ep);
  return launch(K_GEMM, gemm_valu_kernel<float>, grid, dim3(256), 0, s,
                static_cast<const float*>(x), static_cast<const float*>(w), M, N, K, ep);
}

}  // namespace zsa
