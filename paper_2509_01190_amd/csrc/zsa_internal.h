// Internal declarations shared by the HIP kernels and the C-ABI layer.
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>
#include <stddef.h>
#include <stdint.h>

#include <utility>

namespace zsa {

typedef uint16_t bf16_t;

// ---------------------------------------------------------------------------
// storage conversions (fp32 compute, f32 or bf16 storage)
// ---------------------------------------------------------------------------
__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16_t h) {
  return __uint_as_float(static_cast<uint32_t>(h) << 16);
}

// fp32 -> bf16 by v_cvt_pk_bf16_f32: round to nearest even, bit-identical
// to the integer rounding (u + 0x7fff + lsb) >> 16 for every normal and
// infinite input (checked exhaustively on gfx950; only subnormal inputs,
// |x| < 2^-126, differ); NaN stays NaN.
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const f32x2_t v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}
// the pair {x[l], x[l ^ 32]} of lane l in one VALU op (v_permlane32_swap:
// the first result is x[l & 31], the second x[(l & 31) + 32] on every
// lane), so combining the two gives the same value, in the same operand
// order, on both halves of the wave -- without an LDS round trip
__device__ __forceinline__ float half_swap_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float half_swap_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
  return static_cast<bf16_t>(pack_bf16x2(f, 0.f) & 0xffffu);
}

template <typename T>
__device__ __forceinline__ T from_f32(float x);
template <>
__device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <>
__device__ __forceinline__ bf16_t from_f32<bf16_t>(float x) { return f32_to_bf16(x); }

// 16-byte vector of storage elements
template <typename T>
struct Vec16 {
  static constexpr int N = 16 / sizeof(T);
};

__device__ __forceinline__ void unpack16(const uint4& v, float* out, float) {
  out[0] = __uint_as_float(v.x); out[1] = __uint_as_float(v.y);
  out[2] = __uint_as_float(v.z); out[3] = __uint_as_float(v.w);
}
__device__ __forceinline__ void unpack16(const uint4& v, float* out, bf16_t) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    out[2 * i] = __uint_as_float(w[i] << 16);
    out[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}
__device__ __forceinline__ uint4 pack16(const float* in, float) {
  return make_uint4(__float_as_uint(in[0]), __float_as_uint(in[1]), __float_as_uint(in[2]),
                    __float_as_uint(in[3]));
}
__device__ __forceinline__ uint4 pack16(const float* in, bf16_t) {
  return make_uint4(pack_bf16x2(in[0], in[1]), pack_bf16x2(in[2], in[3]),
                    pack_bf16x2(in[4], in[5]), pack_bf16x2(in[6], in[7]));
}

// native 16-byte vector (first-class in LLVM, so arrays of it stay in
// registers; HIP's uint4 is a struct whose copies can end up on the stack)
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// keep a 16-byte value or zero it, without a select between two uint4 objects
// (which the compiler lowers through a stack slot)
__device__ __forceinline__ uint4 keep16(const uint4& v, bool keep) {
  const uint32_t m = keep ? 0xffffffffu : 0u;
  return make_uint4(v.x & m, v.y & m, v.z & m, v.w & m);
}

// ---------------------------------------------------------------------------
// launch helper with the optional per-class timing hook
// ---------------------------------------------------------------------------
enum KClass { K_GEMM = 0, K_ATTENTION = 1, K_SCORE = 2, K_SELECT = 3, K_GATHER = 4,
              K_NORM = 5, K_MISC = 6, K_NCLASS = 7 };

// returns true and a (start, stop) pair if the next launch of this class is timed
bool timing_take(int kclass, hipEvent_t* start, hipEvent_t* stop);
// records the thread's last error text (zsa_last_error) and returns code
int set_error(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));

template <typename... KArgs, typename... Args>
inline hipError_t launch(int kclass, void (*kernel)(KArgs...), dim3 grid, dim3 block,
                         size_t shmem, hipStream_t stream, Args... args) {
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (timing_take(kclass, &e0, &e1)) {
    hipExtLaunchKernelGGL(kernel, grid, block, static_cast<uint32_t>(shmem), stream, e0, e1, 0,
                          static_cast<KArgs>(args)...);
  } else {
    hipLaunchKernelGGL(kernel, grid, block, static_cast<uint32_t>(shmem), stream,
                       static_cast<KArgs>(args)...);
  }
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// GEMM epilogue parameters (shared by the MFMA and the vector-ALU GEMMs)
// ---------------------------------------------------------------------------
enum Epi { EPI_NONE = 0, EPI_GELU = 1, EPI_SWIGLU = 2, EPI_RESIDUAL = 3, EPI_ROPE = 4 };

constexpr int kMaxHalfHead = 64;  // head_dim <= 128 for the rotary epilogue

// sine and cosine of the rotary angle pos * inv_freq: the angle is formed in
// double and reduced to [-pi, pi] with a two-constant (Cody-Waite)
// subtraction of multiples of 2*pi before the fp32 sincos
__device__ __forceinline__ void rope_angle(int p, double inv_freq, float* s, float* c) {
  const double two_pi_hi = 6.283185307179586;       // nearest double to 2*pi
  const double two_pi_lo = 2.4492935982947064e-16;  // 2*pi - two_pi_hi
  const double a = static_cast<double>(p) * inv_freq;
  const double q = rint(a * 0.15915494309189535);   // a / (2*pi)
  double r = fma(-q, two_pi_hi, a);
  r = fma(-q, two_pi_lo, r);
  sincosf(static_cast<float>(r), s, c);
}

struct EpiParams {
  int epi;
  const void* bias;      // [N] or null
  const void* residual;  // [M, ldy] or null
  void* y;               // output
  int ldy;               // output row stride (elements)
  const int32_t* pos;    // [M] rotary positions
  int head_dim;
  int rope_cols;
  // per-row rotary table [M][head_dim / 2] of (cos, sin) pairs (fp32), the
  // values rope_angle gives for that row's position; null: each kernel forms
  // the angles itself
  const float* rope_cs;
  double inv_freq[kMaxHalfHead];  // theta^(-2i/hd), computed on the host in double
};

// bytes of a rotary table for M rows (launch_rope_table)
inline size_t rope_table_bytes(int M, int head_dim) {
  return static_cast<size_t>(M) * (head_dim / 2) * 2 * sizeof(float);
}
// out[m][i] = (cos, sin) of pos[m] * inv_freq[i] for i < head_dim / 2
hipError_t launch_rope_table(hipStream_t s, const int32_t* pos, int M, const EpiParams& ep,
                             float* out);

// ---------------------------------------------------------------------------
// kernel launchers (one translation unit each)
// ---------------------------------------------------------------------------
hipError_t launch_norm(hipStream_t s, int dtype, int kind, const void* x, const void* g,
                       const void* b, int rows, int d, float eps, void* y);

// y = epi(x W^T + bias); x [M, K], W [N, K]. ws (may be NULL) holds split-K
// partials; the bf16 path splits K for small grids when ws_bytes covers it.
hipError_t launch_gemm(hipStream_t s, int dtype, const void* x, int M, int K, const void* w,
                       int N, const EpiParams& ep, void* ws, size_t ws_bytes);
// split-K plan of the bf16 path and its workspace (0 when K is not split)
void splitk_plan(int M, int N, int K, int* S, int* kchunk);
size_t splitk_bytes(int S, int M, int N);
size_t gemm_workspace_bytes(int dtype, int M, int N, int K);
// the most any M <= max_rows needs
size_t gemm_workspace_bound(int dtype, int max_rows, int N, int K);

int device_cu_count();  // compute units of the current device

// Few-row product (bf16, up to 4096 rows of x in blocks of 16): W streamed
// into MFMA operands, one workgroup per 16 output columns and 16 rows over
// the whole of K (no workspace).
// With pn (gain non-null; skinny_norm_ok: M <= 8, K <= 4096, few output
// tiles) x is first normalised as launch_norm would (LayerNorm with shift,
// or RMSNorm).
struct PreNorm {
  const bf16_t* g;  // gain [K], or null: x is used as it is
  const bf16_t* b;  // LayerNorm shift [K] or null
  int rms;          // 1: RMSNorm, 0: LayerNorm
  float eps;
};
bool skinny_ok(int dtype, int M, int N, int K, const EpiParams& ep);
bool skinny_pays(int M, int N, int K);  // launch_gemm takes it for such shapes
bool skinny_norm_ok(int M, int N, int K);
// launch_gemm runs this product on the few-row kernel
bool gemm_takes_skinny(int dtype, int M, int N, int K, const EpiParams& ep);
hipError_t launch_gemm_skinny(hipStream_t s, const void* x, int M, int K, const void* w, int N,
                              const EpiParams& ep, const PreNorm* pn = nullptr);

// query head h reads key/value head h / kv_group (kv_group = H / H_kv)
hipError_t launch_attention(hipStream_t s, int dtype, const void* q, const void* k,
                            const void* v, int64_t row_stride, int H, int kv_group, int hd,
                            int causal, float scale, int B, int max_len, int T,
                            const int32_t* cu_dev, void* out, int64_t out_stride, float* lse);

// writes G partial score vectors [G][T] (G = head groups); returns G via *groups
hipError_t launch_score(hipStream_t s, int dtype, const void* q, const void* k,
                        int64_t row_stride, const float* lse, int H, int kv_group, int hd,
                        int causal, float scale, int B, int max_len, int T,
                        const int32_t* cu_dev, float* partials, int groups);
int score_groups(int dtype, int H, int hd, int T);

hipError_t launch_score_finalize(hipStream_t s, const float* partials, int groups, int T,
                                 float* scores);

// per-sequence top-k over sum_g partials[g*T + row]; cu_out gives output
// offsets; keep_last always keeps each sequence's last row
hipError_t launch_select(hipStream_t s, const float* partials, int groups, int T, int B,
                         int max_len, const int32_t* cu_in_dev, const int32_t* cu_out_dev,
                         int32_t* kept_rows, float* scores_out, int keep_last);

// generation: key/value cache rows and the attention of one new row per
// sequence (cache layout [batch][cap][k | v] per layer, kvd = H_kv * hd)
hipError_t launch_kv_store(hipStream_t s, int dtype, const void* src, int64_t src_stride,
                           int src_col, int kvd, int B, int max_rows, const int32_t* cu_dev,
                           const int32_t* start_dev, void* cache_layer, int cap);
// qkv [B, q_stride]: query heads at column 0, the new row's k | v at kv_col;
// appends them at cache row len - 1, then attends over len rows. Partials:
// m, l [B][H][decode_splits_bound(cap)], o [...][hd]
hipError_t launch_decode_attention(hipStream_t s, const void* qkv, int64_t q_stride, int kv_col,
                                   void* cache_layer, int cap, int hd, int H, int Hkv,
                                   const int32_t* len_dev, int B, int max_len, float scale,
                                   float* m_part, float* l_part, float* o_part, void* out,
                                   int64_t out_stride);
int decode_splits_bound(int cap);
bool decode_supported(int dtype, int hd, int group);

// backward pass (bf16, head_dim 64 / 128 for the attention part)
bool backward_supported(int dtype, int hd);
hipError_t launch_gemm_f32(hipStream_t s, const void* x, int M, int K, const void* w, int N,
                           float* out, void* ws, size_t ws_bytes);
size_t gemm_f32_workspace_bound(int M, int N, int K);
hipError_t launch_transpose(hipStream_t s, int dtype, const void* in, int R, int C, int64_t ldi,
                            void* out, int Rpad);
size_t colsum_scratch_floats(int R, int C);
hipError_t launch_colsum(hipStream_t s, int dtype, const void* a, int64_t lda, const void* x,
                         int64_t ldx, const float* stats, int R, int C, float* scratch,
                         float* out);
hipError_t launch_norm_bwd(hipStream_t s, int dtype, int kind, const void* x, const void* g,
                           const void* dh, const void* res, void* out, int R, int d, float eps,
                           float* stats);
hipError_t launch_act_fwd(hipStream_t s, int dtype, const void* u, void* f, int rows, int F,
                          int swiglu);
hipError_t launch_act_bwd(hipStream_t s, int dtype, const void* dF, const void* u, void* du,
                          int rows, int F, int swiglu);
hipError_t launch_scatter_rows(hipStream_t s, int dtype, int d, const void* src,
                               const int32_t* kept, int t_out, int t_in, int32_t* inv,
                               void* dst);
hipError_t launch_rowdot(hipStream_t s, int dtype, const void* dO, const void* O, int64_t ld,
                         int T, int H, int hd, float* D);
hipError_t launch_rope_bwd(hipStream_t s, int dtype, void* g, int64_t ld, int rows, int cols,
                           int hd, const int32_t* pos, const EpiParams& ep);
hipError_t launch_attention_bwd(hipStream_t s, const void* q, const void* k, const void* v,
                                int64_t rs, const void* dO, int64_t ors, const float* lse,
                                const float* D, int H, int kv_group, int hd, int causal,
                                float scale, int B, int max_len, int T, const int32_t* cu_dev,
                                void* dq, void* dk, void* dv, int64_t grs);

// row gather of up to two [*, d] arrays plus pos
hipError_t launch_gather(hipStream_t s, int dtype, int d, int t_in, const int32_t* kept,
                         int t_out, const void* src0, void* dst0, const void* src1, void* dst1,
                         const int32_t* pos, int32_t* pos_out);

hipError_t launch_upload_i32(hipStream_t s, int32_t* dst, const int32_t* host_vals, int n);
hipError_t launch_copy_i32(hipStream_t s, int32_t* dst, const int32_t* src, int n);

}  // namespace zsa
