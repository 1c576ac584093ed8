// Attention of Eq. 1, softmax(Q K^T * scale + M) V, per sequence and head
// (query head h reads key/value head h / kv_group: grouped-query attention),
// over packed variable-length rows; also writes the natural-log
// log-sum-exp of every score row (used by the contribution scores).
//
// bf16, head_dim 64/128 (MFMA): one workgroup of NW waves per (32 NW-query
// block, head, sequence); each wave owns 32 queries and walks 64-key tiles
// staged in LDS (K row-major; V transposed at head_dim 64, row-major at 128
// and read through transposing LDS reads). The wave computes the
// *transposed* score tile S^T = K Q^T with v_mfma_f32_32x32x16_bf16, so a
// lane holds 32 key scores of one query: the online-softmax max and sum are
// in-lane plus one swap with lane l^32, and the probabilities already sit in
// the B-operand layout of O^T += V^T P^T (P rounded to bf16), with no trip
// through LDS. The k-slot order of P^T is whatever the accumulator gives; V^T
// is read from LDS in that same order, which leaves the contraction unchanged.
// Causal blocks skip key tiles above the diagonal and are scheduled
// heaviest-first.
//
// fp32 (and any other head_dim): one thread per query with the row in
// registers, 32-key LDS tiles, the same online softmax.
#include <math.h>

#include "zsa_internal.h"

namespace zsa {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// Head dim 64 fits four waves per SIMD (128 registers), 128 two. A workgroup
// reads every K and V row of its sequence and head once, so the bytes moved
// per query fall as the query block grows: the loads, not the MFMAs or the
// exponentials, bound the kernel at these lengths (a copy without any of
// the compute takes 35 of the 48.5 us of 32 sequences x 12 heads x 512 rows
// with 4 waves). 8 waves (256 queries, two workgroups per CU) halve them.
template <int HD, int NW>
__global__ __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(HD == 64 ? 4 : 2))) void attn_mfma_kernel(
    const bf16_t* __restrict__ Q, const bf16_t* __restrict__ K, const bf16_t* __restrict__ V,
    int64_t rs, int kv_group, int causal, float scale_log2, const int32_t* __restrict__ cu,
    bf16_t* __restrict__ O, int64_t os, float* __restrict__ lse, int T) {
  constexpr int NT = 64 * NW, BQ = 32 * NW, BKEY = 64;
  constexpr int KLD = HD + 8;    // K tile row stride (bf16)
  // V^T tile row stride (bf16): 34 dwords. The fragment reads (32
  // consecutive rows, 8 bytes each) hit distinct bank pairs and stay 8-byte
  // aligned, so they are ds_read_b64 with immediate offsets. In row r the
  // 8-byte chunk of keys 4c .. 4c + 3 sits at chunk c ^ (VSW * (r / 32)):
  // the transposing writes of a wave (rows 8j + e of 8 channel blocks j, 8
  // key pairs) then cover all 64 banks once, where rows j and j + 4
  // otherwise met in one bank (2-way), while the 32 rows of a fragment read
  // share one XOR and stay conflict-free (head_dim 64: 292.8 against
  // 296.1 us on 8 x 2048 causal rows, 32 heads). Head dim 128 keeps the
  // plain layout: the swizzle there measured 2 % slower.
  constexpr int VLD = BKEY + 4;
  constexpr int VSW = HD == 64 ? 4 : 0;
  // Head dim 128 stores V as it comes (key rows, the K tile's row stride)
  // and reads the V^T fragments with gfx950's transposing LDS reads
  // (ds_read_b64_tr_b16): 4 x 4096 causal rows, 32 heads, 986 -> 929 us.
  // At head dim 64 the same reads took 296 -> 296 us on 8 x 2048 causal
  // rows and 40.6 -> 42.2 us on 32 x 512, so it keeps the transposed tile.
  constexpr bool VTR = HD == 128;
  constexpr int OLD = HD + 8;    // output staging row stride
  constexpr int KBYTES = BKEY * KLD * 2, VBYTES = VTR ? KBYTES : HD * VLD * 2;
  constexpr int BUF = KBYTES + VBYTES;
  // K/V tile buffers: eight-wave blocks keep four (tiles stored two ahead,
  // a barrier after every second tile: 297.0 -> 292.2 us on 8 x 2048 causal
  // rows, 83.7 -> 80.8 on 8 x 1024, 11.2 -> 10.2 on 8 x 256, head dim 128
  // on 4 x 4096 rows 1017 -> 994); four-wave blocks two (one ahead, a
  // barrier per tile), which keeps four of them on a CU
  constexpr int NB = NW == 8 ? 4 : 2, LA = NB / 2;
  constexpr int SBYTES = NB * BUF > NW * 32 * OLD * 2 ? NB * BUF : NW * 32 * OLD * 2;
  constexpr int KITEMS = BKEY * HD / 8;        // 16-byte K chunks per tile
  constexpr int VITEMS = (BKEY / 2) * (HD / 8);  // V row-pair chunks per tile
  static_assert(KITEMS % NT == 0 && (VITEMS % NT == 0 || VITEMS < NT), "tile split");
  constexpr int KCH = KITEMS / NT;                   // per thread
  constexpr int VPR = VITEMS < NT ? 1 : VITEMS / NT;  // per thread (some idle if fewer)
  __shared__ __align__(16) unsigned char smem[SBYTES];

  const int b = blockIdx.z, h = blockIdx.y;
  const int lo = cu[b];
  const int n = cu[b + 1] - lo;
  const int nqb = (n + BQ - 1) / BQ;
  if (static_cast<int>(blockIdx.x) >= nqb) return;
  const int qb = causal ? nqb - 1 - static_cast<int>(blockIdx.x) : static_cast<int>(blockIdx.x);
  const int q0 = qb * BQ;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5, l32 = lane & 31;
  const int qrow = q0 + wave * 32 + l32;
  bf16x8_t qf[HD / 16];
#pragma unroll
  for (int kk = 0; kk < HD / 16; ++kk) {
    // rows past the sequence are clamped, not zeroed: their outputs are not stored
    const int qr = min(qrow, n - 1);
    qf[kk] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const u32x4*>(
                                              Q + static_cast<int64_t>(lo + qr) * rs + h * HD + kk * 16 + half * 8));
  }

  // K/V tiles of a later key block are prefetched into registers while the
  // current block is computed, and stored LA blocks ahead into NB LDS
  // buffers; a barrier follows every LA blocks.
  // The loads go through a buffer resource spanning this sequence's rows,
  // so keys past the sequence read as zeros (they are masked to probability
  // 0); a thread's offsets within a tile are fixed, plus the tile's start.
  // grouped-query attention: query head h reads key/value head h / kv_group
  const int hk = h / kv_group;
  const uint32_t seq_bytes = static_cast<uint32_t>(static_cast<int64_t>(n) * rs * 2);
  const __amdgpu_buffer_rsrc_t kres = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<bf16_t*>(K + static_cast<int64_t>(lo) * rs + hk * HD), 0, seq_bytes, 0x00020000);
  const __amdgpu_buffer_rsrc_t vres = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<bf16_t*>(V + static_cast<int64_t>(lo) * rs + hk * HD), 0, seq_bytes, 0x00020000);
  uint32_t koff[KCH], voff[VPR];
#pragma unroll
  for (int i = 0; i < KCH; ++i) {
    const int c = tid + i * NT;
    koff[i] = static_cast<uint32_t>((c / (HD / 8)) * rs + (c % (HD / 8)) * 8) * 2u;
  }
  // threads past the tile's V chunks (when there are fewer than threads)
  // load from past the buffer range (zeros) and store nothing
  const bool vth = VITEMS >= NT || tid < VITEMS;
#pragma unroll
  for (int i = 0; i < VPR; ++i) {
    const int c = tid + i * NT;
    voff[i] = vth ? static_cast<uint32_t>((2 * (c / (HD / 8))) * rs + (c % (HD / 8)) * 8) * 2u
                  : 0x80000000u;
  }
  const uint32_t row_bytes = static_cast<uint32_t>(rs * 2);
  u32x4 kreg[KCH], vreg[VPR][2], vrow[KCH];
  auto load_tile = [&](int j0) {
    const uint32_t t0 = static_cast<uint32_t>(j0) * row_bytes;
    // the whole offset goes in the vector operand, which the range check covers
#pragma unroll
    for (int i = 0; i < KCH; ++i)
      kreg[i] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(kres, koff[i] + t0, 0, 0));
    if constexpr (VTR) {
      // V rows at the K offsets (one row stride)
#pragma unroll
      for (int i = 0; i < KCH; ++i)
        vrow[i] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(vres, koff[i] + t0, 0, 0));
      return;
    }
#pragma unroll
    for (int i = 0; i < VPR; ++i) {
      vreg[i][0] = __builtin_bit_cast(
          u32x4, __builtin_amdgcn_raw_buffer_load_b128(vres, voff[i] + t0, 0, 0));
      vreg[i][1] = __builtin_bit_cast(
          u32x4, __builtin_amdgcn_raw_buffer_load_b128(vres, voff[i] + t0 + row_bytes, 0, 0));
    }
  };
  auto store_tile = [&](int buf) {
    bf16_t* Ks = reinterpret_cast<bf16_t*>(smem + buf * BUF);
    bf16_t* Vt = reinterpret_cast<bf16_t*>(smem + buf * BUF + KBYTES);
#pragma unroll
    for (int i = 0; i < KCH; ++i) {
      const int c = tid + i * NT;
      const int r = c / (HD / 8), ch = (c % (HD / 8)) * 8;
      *reinterpret_cast<u32x4*>(Ks + r * KLD + ch) = kreg[i];
      if constexpr (VTR) *reinterpret_cast<u32x4*>(Vt + r * KLD + ch) = vrow[i];
    }
    if (VTR || !vth) return;
#pragma unroll
    for (int i = 0; i < VPR; ++i) {
      const int c = tid + i * NT;
      const int rp = c / (HD / 8), ch = (c % (HD / 8)) * 8;
      // rows ch .. ch + 7 share one 32-row group, hence one swizzle
      bf16_t* vt = Vt + ch * VLD + 4 * ((rp >> 1) ^ (VSW * (ch >> 5))) + 2 * (rp & 1);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const uint32_t w0 = vreg[i][0][e >> 1], w1 = vreg[i][1][e >> 1];
        const uint32_t x0 = (e & 1) ? (w0 >> 16) : (w0 & 0xffffu);
        const uint32_t x1 = (e & 1) ? (w1 & 0xffff0000u) : (w1 << 16);
        *reinterpret_cast<uint32_t*>(vt + e * VLD) = x0 | x1;
      }
    }
  };

  float m_run = -INFINITY, l_run = 0.f;  // running max in raw score units
  f32x16_t o[HD / 32];
#pragma unroll
  for (int ct = 0; ct < HD / 32; ++ct)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[ct][r] = 0.f;

  const int kend = causal ? min(n, q0 + BQ) : n;
  const int wave_q0 = q0 + wave * 32;
  load_tile(0);
  store_tile(0);
  if (LA == 2 && BKEY < kend) {
    load_tile(BKEY);
    store_tile(1);
  }
  if (LA * BKEY < kend) load_tile(LA * BKEY);
  __syncthreads();
  int t = 0;
  for (int j0 = 0; j0 < kend; j0 += BKEY, ++t) {
    const int buf = t % NB;
    if (j0 + LA * BKEY < kend) {
      // the buffer of block t + LA was last read by block t + LA - NB, before
      // the last barrier; the barrier after block t + LA - 1 publishes it
      store_tile((t + LA) % NB);
      if (j0 + (LA + 1) * BKEY < kend) load_tile(j0 + (LA + 1) * BKEY);
    }
    const bf16_t* Ks = reinterpret_cast<const bf16_t*>(smem + buf * BUF);
    const bf16_t* Vt = reinterpret_cast<const bf16_t*>(smem + buf * BUF + KBYTES);
    if (!causal || j0 <= wave_q0 + 31) {
      f32x16_t s[2];
      const f32x16_t zero = {};
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
#pragma unroll
        for (int kk = 0; kk < HD / 16; ++kk) {
          const bf16x8_t a = __builtin_bit_cast(
              bf16x8_t, *reinterpret_cast<const u32x4*>(Ks + (ks * 32 + l32) * KLD + kk * 16 + half * 8));
          s[ks] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[kk], kk == 0 ? zero : s[ks], 0, 0, 0);
        }
      }
      // s[ks][r]: query qrow, key j0 + 32 ks + 8 (r/4) + 4 half + r%4 (raw q.k)
      // masks only on the tiles that cross the sequence end or the diagonal
      if (j0 + BKEY > n || (causal && j0 + BKEY - 1 > wave_q0)) {
#pragma unroll
        for (int ks = 0; ks < 2; ++ks)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int j = j0 + ks * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
            if (j >= n || (causal && j > qrow)) s[ks][r] = -INFINITY;
          }
      }
      float mloc = -INFINITY;
#pragma unroll
      for (int ks = 0; ks < 2; ++ks)
#pragma unroll
        for (int r = 0; r < 16; ++r) mloc = fmaxf(mloc, s[ks][r]);
      mloc = half_swap_max(mloc);
      const float m_new = fmaxf(m_run, mloc);
      // The reference max moves (and the sums and accumulators are rescaled)
      // only when some query's max has grown by more than 2^8 in exp2 units
      // since the reference was set: probabilities stay below 256 (exact in
      // fp32, full relative precision in bf16), and since the output and the
      // log-sum-exp are both taken relative to the reference, the result is
      // the same for any reference. A row's first valid scores always move
      // it (from -inf). scale > 0, so the max of the scaled scores is the
      // scaled max.
      if (__builtin_amdgcn_ballot_w64(m_new == -INFINITY ? false
                                                         : !((m_new - m_run) * scale_log2 <= 8.0f)) != 0) {
        const float alpha = m_new == -INFINITY ? 1.0f : __builtin_amdgcn_exp2f((m_run - m_new) * scale_log2);
        l_run *= alpha;
#pragma unroll
        for (int ct = 0; ct < HD / 32; ++ct)
#pragma unroll
          for (int r = 0; r < 16; ++r) o[ct][r] *= alpha;
        m_run = m_new;
      }
      const float m_use = m_run == -INFINITY ? 0.f : m_run * scale_log2;
      float rsum = 0.f;
#pragma unroll
      for (int ks = 0; ks < 2; ++ks)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float p = __builtin_amdgcn_exp2f(fmaf(s[ks][r], scale_log2, -m_use));
          s[ks][r] = p;
          rsum += p;
        }
      rsum = half_swap_sum(rsum);
      l_run += rsum;
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int ks = g >> 1, rb = (g & 1) * 8;
        const u32x4 pw = {pack_bf16x2(s[ks][rb], s[ks][rb + 1]), pack_bf16x2(s[ks][rb + 2], s[ks][rb + 3]),
                          pack_bf16x2(s[ks][rb + 4], s[ks][rb + 5]), pack_bf16x2(s[ks][rb + 6], s[ks][rb + 7])};
        const bf16x8_t pb = __builtin_bit_cast(bf16x8_t, pw);
        if constexpr (VTR) {
          // pb's slots 0..3 hold keys kb + 4 half + 0..3 and slots 4..7 keys
          // kb + 8 + 4 half + 0..3 (kb = 32 ks + 16 (g & 1)); the V^T
          // fragment gives channel ct * 32 + l32 the same keys in the same
          // slots. A transposing read gives each lane of a 16-lane group
          // element c (its lane number in the group) of four 16-element
          // rows, row r pieced together from the 4-element runs at the
          // addresses of the group's lanes 4r .. 4r + 3: so the group's
          // lanes point at key rows kb + 4 half + r and channel runs
          // 16 ((lane / 16) & 1) + 4 (lane & 3).
          typedef short s16x4 __attribute__((ext_vector_type(4)));
          typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
          typedef __attribute__((address_space(3))) const char lds_char;
          const bf16_t* tr0 = Vt + (ks * 32 + (g & 1) * 16 + 4 * half + ((lane & 15) >> 2)) * KLD +
                              16 * ((lane >> 4) & 1) + 4 * (lane & 3);
#pragma unroll
          for (int ct = 0; ct < HD / 32; ++ct) {
            const bf16_t* vr = tr0 + ct * 32;
            const s16x4 lo4 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)((lds_char*)vr));
            const s16x4 hi4 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)((lds_char*)(vr + 8 * KLD)));
            const uint2 l2 = __builtin_bit_cast(uint2, lo4), h2 = __builtin_bit_cast(uint2, hi4);
            const u32x4 av = {l2.x, l2.y, h2.x, h2.y};
            o[ct] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, av), pb, o[ct], 0, 0, 0);
          }
          continue;
        }
        // key chunks 8 ks + 4 (g & 1) + half and that + 2; the swizzle is even,
        // so it leaves half (the only lane-dependent part) alone and the
        // offsets stay immediates on one base address
        const bf16_t* vr0 = Vt + l32 * VLD + 4 * half;
#pragma unroll
        for (int ct = 0; ct < HD / 32; ++ct) {
          const bf16_t* vr = vr0 + ct * 32 * VLD;
          const int c0 = ks * 8 + (g & 1) * 4;
          const uint2 lo4 = *reinterpret_cast<const uint2*>(vr + 4 * (c0 ^ (VSW * ct)));
          const uint2 hi4 = *reinterpret_cast<const uint2*>(vr + 4 * ((c0 + 2) ^ (VSW * ct)));
          const u32x4 av = {lo4.x, lo4.y, hi4.x, hi4.y};
          o[ct] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, av), pb, o[ct], 0, 0, 0);
        }
      }
    }
    if (t % LA == LA - 1) __syncthreads();
  }
  if (LA > 1) __syncthreads();  // every wave is past the tiles before the output staging reuses them

  // o[ct][r] = O^T[channel ct*32 + 8 (r/4) + 4 half + r%4][query qrow]
  const float inv_l = l_run > 0.f ? 1.0f / l_run : 0.f;
  bf16_t* Os = reinterpret_cast<bf16_t*>(smem) + wave * 32 * OLD;
#pragma unroll
  for (int ct = 0; ct < HD / 32; ++ct)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int c = ct * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
      Os[l32 * OLD + c] = f32_to_bf16(o[ct][r] * inv_l);
    }
  __syncthreads();
  for (int c = lane; c < 32 * HD / 8; c += 64) {
    const int r = c / (HD / 8), ch = (c % (HD / 8)) * 8;
    const int qr = q0 + wave * 32 + r;
    if (qr < n)
      *reinterpret_cast<u32x4*>(O + static_cast<int64_t>(lo + qr) * os + h * HD + ch) =
          *reinterpret_cast<const u32x4*>(Os + r * OLD + ch);
  }
  if (lse != nullptr && half == 0 && qrow < n)
    lse[static_cast<int64_t>(h) * T + lo + qrow] = (m_run * scale_log2 + log2f(l_run)) * kLn2;
}

template <typename T, int HD>
__global__ __launch_bounds__(64) void attn_valu_kernel(const T* __restrict__ Q,
                                                       const T* __restrict__ K,
                                                       const T* __restrict__ V, int64_t rs,
                                                       int kv_group, int causal, float scale,
                                                       const int32_t* __restrict__ cu,
                                                       T* __restrict__ O, int64_t os,
                                                       float* __restrict__ lse, int Tn) {
  constexpr int BKEY = 32;
  __shared__ float Ks[BKEY][HD];
  __shared__ float Vs[BKEY][HD];
  const int b = blockIdx.z, h = blockIdx.y;
  const int lo = cu[b];
  const int n = cu[b + 1] - lo;
  const int qbase = blockIdx.x * 64;
  if (qbase >= n) return;
  const int q = qbase + threadIdx.x;
  const bool active = q < n;
  float qv[HD], o[HD];
#pragma unroll
  for (int c = 0; c < HD; ++c) {
    qv[c] = active ? to_f32(Q[static_cast<int64_t>(lo + q) * rs + h * HD + c]) * scale : 0.f;
    o[c] = 0.f;
  }
  float m = -INFINITY, l = 0.f;
  const int kend = causal ? min(n, qbase + 64) : n;
  for (int j0 = 0; j0 < kend; j0 += BKEY) {
    for (int e = threadIdx.x; e < BKEY * HD; e += 64) {
      const int r = e / HD, c = e % HD;
      const int j = j0 + r;
      Ks[r][c] = j < n ? to_f32(K[static_cast<int64_t>(lo + j) * rs + (h / kv_group) * HD + c]) : 0.f;
      Vs[r][c] = j < n ? to_f32(V[static_cast<int64_t>(lo + j) * rs + (h / kv_group) * HD + c]) : 0.f;
    }
    __syncthreads();
    if (active) {
      for (int jj = 0; jj < BKEY; ++jj) {
        const int j = j0 + jj;
        if (j >= n || (causal && j > q)) continue;
        float sc = 0.f;
#pragma unroll
        for (int c = 0; c < HD; ++c) sc += qv[c] * Ks[jj][c];
        if (sc > m) {
          const float corr = expf(m - sc);
          l *= corr;
#pragma unroll
          for (int c = 0; c < HD; ++c) o[c] *= corr;
          m = sc;
        }
        const float p = expf(sc - m);
        l += p;
#pragma unroll
        for (int c = 0; c < HD; ++c) o[c] += p * Vs[jj][c];
      }
    }
    __syncthreads();
  }
  if (active) {
    const float inv = 1.0f / l;
#pragma unroll
    for (int c = 0; c < HD; ++c)
      O[static_cast<int64_t>(lo + q) * os + h * HD + c] = from_f32<T>(o[c] * inv);
    if (lse != nullptr) lse[static_cast<int64_t>(h) * Tn + lo + q] = m + logf(l);
  }
}

template <typename T>
hipError_t valu_dispatch(hipStream_t s, const void* q, const void* k, const void* v, int64_t rs,
                         int H, int kvg, int hd, int causal, float scale, int B, int max_len, int Trows,
                         const int32_t* cu, void* out, int64_t os, float* lse) {
  const dim3 grid((max_len + 63) / 64, H, B), block(64);
  const T* qp = static_cast<const T*>(q);
  const T* kp = static_cast<const T*>(k);
  const T* vp = static_cast<const T*>(v);
  T* op = static_cast<T*>(out);
  switch (hd) {
    case 16: return launch(K_ATTENTION, attn_valu_kernel<T, 16>, grid, block, 0, s, qp, kp, vp, rs, kvg, causal, scale, cu, op, os, lse, Trows);
    case 32: return launch(K_ATTENTION, attn_valu_kernel<T, 32>, grid, block, 0, s, qp, kp, vp, rs, kvg, causal, scale, cu, op, os, lse, Trows);
    case 64: return launch(K_ATTENTION, attn_valu_kernel<T, 64>, grid, block, 0, s, qp, kp, vp, rs, kvg, causal, scale, cu, op, os, lse, Trows);
    case 128: return launch(K_ATTENTION, attn_valu_kernel<T, 128>, grid, block, 0, s, qp, kp, vp, rs, kvg, causal, scale, cu, op, os, lse, Trows);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_attention(hipStream_t s, int dtype, const void* q, const void* k,
                            const void* v, int64_t row_stride, int H, int kv_group, int hd,
                            int causal, float scale, int B, int max_len, int T,
                            const int32_t* cu_dev, void* out, int64_t out_stride, float* lse) {
  if (B == 0 || max_len == 0) return hipSuccess;
  if (dtype == 1 && (hd == 64 || hd == 128)) {
    const bf16_t* qp = static_cast<const bf16_t*>(q);
    const bf16_t* kp = static_cast<const bf16_t*>(k);
    const bf16_t* vp = static_cast<const bf16_t*>(v);
    bf16_t* op = static_cast<bf16_t*>(out);
    const float sl = scale * kLog2e;
    // 256-query blocks for the longer sequences (measured: head dim 64, 32
    // sequences x 12 heads x 512 rows 48.5 -> 45.9 us; head dim 128, 4 x 32
    // heads x 4096 rows, causal, 1212 -> 1168 us, x 2048 rows 327 -> 309 us,
    // x 368 rows even)
    if (hd == 64 && max_len > 128)
      return launch(K_ATTENTION, attn_mfma_kernel<64, 8>, dim3((max_len + 255) / 256, H, B),
                    dim3(512), 0, s, qp, kp, vp, row_stride, kv_group, causal, sl, cu_dev, op,
                    out_stride, lse, T);
    if (hd == 128 && max_len > 512)
      return launch(K_ATTENTION, attn_mfma_kernel<128, 8>, dim3((max_len + 255) / 256, H, B),
                    dim3(512), 0, s, qp, kp, vp, row_stride, kv_group, causal, sl, cu_dev, op,
                    out_stride, lse, T);
    const dim3 grid((max_len + 127) / 128, H, B), block(256);
    if (hd == 64)
      return launch(K_ATTENTION, attn_mfma_kernel<64, 4>, grid, block, 0, s, qp, kp, vp, row_stride,
                    kv_group, causal, sl, cu_dev, op, out_stride, lse, T);
    return launch(K_ATTENTION, attn_mfma_kernel<128, 4>, grid, block, 0, s, qp, kp, vp, row_stride,
                  kv_group, causal, sl, cu_dev, op, out_stride, lse, T);
  }
  if (dtype == 1)
    return valu_dispatch<bf16_t>(s, q, k, v, row_stride, H, kv_group, hd, causal, scale, B,
                                 max_len, T, cu_dev, out, out_stride, lse);
  return valu_dispatch<float>(s, q, k, v, row_stride, H, kv_group, hd, causal, scale, B, max_len,
                              T, cu_dev, out, out_stride, lse);
}

}  // namespace zsa
