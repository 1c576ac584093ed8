// Host-only driver of the C-ABI under AddressSanitizer and
// UndefinedBehaviorSanitizer: the Eq. 2 keep-count schedule (Sec. 3.3) and
// every argument-validation path of every entry point. It is linked with
// stand-ins for the device side that abort if reached, so each rejected call
// also shows that validation finishes before the first launch.
//
// Golden keep counts arrive on stdin, one "n keep_rate tau expected" per
// line. Prints "ok <cases>" and exits 0 when every check holds.
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <vector>

#include "../../include/zsa.h"

namespace {

int g_checks = 0;

void check(bool ok, const char* what, int line) {
  ++g_checks;
  if (!ok) {
    fprintf(stderr, "check failed (line %d): %s; last error: %s\n", line, what, zsa_last_error());
    exit(1);
  }
}
#define CHECK_TRUE(cond) check((cond), #cond, __LINE__)
// a rejected call: the status, and a non-empty message
#define EXPECT_RC(call, code)                                                  \
  do {                                                                         \
    const int rc_ = (call);                                                    \
    check(rc_ == (code), #call " returned the wrong status", __LINE__);        \
    check(zsa_last_error()[0] != '\0', "empty error text after " #call, __LINE__); \
  } while (0)

// fake device addresses: validation only inspects their alignment
void* A(uintptr_t v) { return reinterpret_cast<void*>(v); }
const void* C(uintptr_t v) { return reinterpret_cast<const void*>(v); }
float* F(uintptr_t v) { return reinterpret_cast<float*>(v); }
int32_t* I(uintptr_t v) { return reinterpret_cast<int32_t*>(v); }

zsa_layer_cfg cfg_of(int kind, int d, int H, int F, int causal, int dtype) {
  zsa_layer_cfg c;
  memset(&c, 0, sizeof(c));
  c.kind = kind;
  c.d_model = d;
  c.n_heads = H;
  c.head_dim = d / H;
  c.d_ff = F;
  c.causal = causal;
  c.dtype = dtype;
  c.tau = 5;
  c.norm_eps = 1e-5f;
  c.rope_theta = 1e4f;
  return c;
}

zsa_layer_weights weights_at(uintptr_t base) {
  zsa_layer_weights w;
  const void** p = reinterpret_cast<const void**>(&w);
  for (int i = 0; i < 12; ++i) p[i] = C(base + 0x1000 * i);
  return w;
}

void keep_count_checks() {
  // golden values (Eq. 2 worked cases) from stdin
  int n, tau, expect;
  double a;
  int golden = 0;
  while (scanf("%d %lf %d %d", &n, &a, &tau, &expect) == 4) {
    int32_t k = -1;
    CHECK_TRUE(zsa_keep_count(n, a, tau, &k) == ZSA_OK);
    if (k != expect) fprintf(stderr, "n %d rate %.17g tau %d: %d != %d\n", n, a, tau, k, expect);
    CHECK_TRUE(k == expect);
    ++golden;
  }
  CHECK_TRUE(golden >= 10);
  // invariants over a grid of lengths, rates and floors
  for (int tau_i : {1, 5, 17}) {
    for (int len = 0; len <= 3000; len += (len < 64 ? 1 : 37)) {
      int32_t prev = -1;
      for (int i = 0; i <= 1000; ++i) {
        const double rate = i / 1000.0;
        int32_t k = -1;
        CHECK_TRUE(zsa_keep_count(len, rate, tau_i, &k) == ZSA_OK);
        CHECK_TRUE(k >= 0 && k <= len);
        CHECK_TRUE(k >= (len < tau_i ? len : tau_i));
        CHECK_TRUE(k >= prev);  // monotone in the keep rate
        prev = k;
        const double fl = floor(rate * len + 1e-9);
        if (fl > tau_i && fl < len) CHECK_TRUE(k == static_cast<int32_t>(fl));
      }
      int32_t k1 = -1, k0 = -1;
      CHECK_TRUE(zsa_keep_count(len, 1.0, tau_i, &k1) == ZSA_OK && k1 == len);
      CHECK_TRUE(zsa_keep_count(len, 0.0, tau_i, &k0) == ZSA_OK &&
                 k0 == (len < tau_i ? len : tau_i));
    }
  }
  int32_t k;
  EXPECT_RC(zsa_keep_count(10, NAN, 5, &k), ZSA_EINVAL);
  EXPECT_RC(zsa_keep_count(10, -1e-12, 5, &k), ZSA_EINVAL);
  EXPECT_RC(zsa_keep_count(10, 1.0000001, 5, &k), ZSA_EINVAL);
  EXPECT_RC(zsa_keep_count(10, INFINITY, 5, &k), ZSA_EINVAL);
  EXPECT_RC(zsa_keep_count(10, -INFINITY, 5, &k), ZSA_EINVAL);
  EXPECT_RC(zsa_keep_count(10, 0.5, 0, &k), ZSA_EINVAL);
  EXPECT_RC(zsa_keep_count(-1, 0.5, 5, &k), ZSA_EINVAL);
  EXPECT_RC(zsa_keep_count(10, 0.5, 5, nullptr), ZSA_EINVAL);
}

void keep_schedule_checks() {
  const int32_t lens[4] = {512, 2048, 3, 100};
  const double rates[4] = {0.5, 0.1, 0.9, 0.3};
  int32_t out[4 * 3];
  CHECK_TRUE(zsa_keep_schedule(4, lens, rates, 5, 3, out) == ZSA_OK);
  for (int b = 0; b < 4; ++b) {
    int32_t cur = lens[b];
    for (int p = 0; p < 3; ++p) {
      int32_t k;
      CHECK_TRUE(zsa_keep_count(cur, rates[b], 5, &k) == ZSA_OK);
      CHECK_TRUE(out[p * 4 + b] == k);  // compounded on the previous count
      cur = k;
    }
  }
  CHECK_TRUE(out[0] == 256 && out[4] == 128 && out[8] == 64);
  CHECK_TRUE(out[1] == 204 && out[5] == 20 && out[9] == 5);
  CHECK_TRUE(out[2] == 3 && out[6] == 3);  // shorter than tau: kept whole
  CHECK_TRUE(zsa_keep_schedule(0, nullptr, nullptr, 5, 3, nullptr) == ZSA_OK);
  EXPECT_RC(zsa_keep_schedule(-1, lens, rates, 5, 1, out), ZSA_EINVAL);
  EXPECT_RC(zsa_keep_schedule(4, lens, rates, 5, -1, out), ZSA_EINVAL);
  EXPECT_RC(zsa_keep_schedule(4, nullptr, rates, 5, 1, out), ZSA_EINVAL);
  EXPECT_RC(zsa_keep_schedule(4, lens, nullptr, 5, 1, out), ZSA_EINVAL);
  EXPECT_RC(zsa_keep_schedule(4, lens, rates, 5, 1, nullptr), ZSA_EINVAL);
  EXPECT_RC(zsa_keep_schedule(4, lens, rates, 0, 1, out), ZSA_EINVAL);
  const double bad_rates[4] = {0.5, NAN, 0.5, 0.5};
  EXPECT_RC(zsa_keep_schedule(4, lens, bad_rates, 5, 1, out), ZSA_EINVAL);
  const int32_t bad_lens[4] = {5, -1, 5, 5};
  EXPECT_RC(zsa_keep_schedule(4, bad_lens, rates, 5, 1, out), ZSA_EINVAL);
}

void norm_checks() {
  EXPECT_RC(zsa_norm(nullptr, 7, 0, C(0x1000), C(0x2000), nullptr, 4, 64, 1e-5f, A(0x3000)),
            ZSA_EINVAL);
  EXPECT_RC(zsa_norm(nullptr, ZSA_F32, 2, C(0x1000), C(0x2000), nullptr, 4, 64, 1e-5f, A(0x3000)),
            ZSA_EINVAL);
  EXPECT_RC(zsa_norm(nullptr, ZSA_F32, 0, C(0x1000), C(0x2000), nullptr, -1, 64, 1e-5f, A(0x3000)),
            ZSA_EINVAL);
  EXPECT_RC(zsa_norm(nullptr, ZSA_BF16, 0, C(0x1000), C(0x2000), nullptr, 4, 12, 1e-5f, A(0x3000)),
            ZSA_EALIGN);
  EXPECT_RC(zsa_norm(nullptr, ZSA_BF16, 0, C(0x1000), C(0x2000), nullptr, 4, 8200, 1e-5f,
                     A(0x3000)),
            ZSA_EUNSUPPORTED);
  EXPECT_RC(zsa_norm(nullptr, ZSA_F32, 0, nullptr, C(0x2000), nullptr, 4, 64, 1e-5f, A(0x3000)),
            ZSA_EINVAL);
  EXPECT_RC(zsa_norm(nullptr, ZSA_F32, 0, C(0x1004), C(0x2000), nullptr, 4, 64, 1e-5f, A(0x3000)),
            ZSA_EALIGN);
  EXPECT_RC(zsa_norm(nullptr, ZSA_F32, 0, C(0x1000), nullptr, nullptr, 4, 64, 1e-5f, A(0x3000)),
            ZSA_EINVAL);
  EXPECT_RC(zsa_norm(nullptr, ZSA_F32, 0, C(0x1000), C(0x2000), nullptr, 4, 64, 1e-5f, nullptr),
            ZSA_EINVAL);
  EXPECT_RC(zsa_norm(nullptr, ZSA_F32, 0, C(0x1000), C(0x2000), C(0x2008), 4, 64, 1e-5f,
                     A(0x3000)),
            ZSA_EALIGN);
  // no rows: x and y may be NULL and nothing is launched
  EXPECT_RC(zsa_norm(nullptr, ZSA_BF16, 0, nullptr, C(0x2000), nullptr, 0, 64, 1e-5f, nullptr),
            ZSA_OK);
  EXPECT_RC(zsa_norm(nullptr, ZSA_BF16, 0, nullptr, nullptr, nullptr, 0, 64, 1e-5f, nullptr),
            ZSA_EINVAL);
}

void linear_checks() {
  auto lin = [](int dtype, const void* x, int m, int k, const void* w, int n, const void* bias,
                int epi, const void* res, const int32_t* pos, int hd, int rope_cols, float theta,
                void* y, void* ws, size_t ws_bytes) {
    return zsa_linear(nullptr, dtype, x, m, k, w, n, bias, epi, res, pos, hd, rope_cols, theta, y,
                      ws, ws_bytes);
  };
  const void* x = C(0x1000);
  const void* w = C(0x2000);
  void* y = A(0x3000);
  EXPECT_RC(lin(5, x, 4, 64, w, 64, nullptr, 0, nullptr, nullptr, 0, 0, 1e4f, y, nullptr, 0),
            ZSA_EINVAL);
  EXPECT_RC(lin(ZSA_BF16, x, -1, 64, w, 64, nullptr, 0, nullptr, nullptr, 0, 0, 1e4f, y, nullptr, 0),
            ZSA_EINVAL);
  EXPECT_RC(lin(ZSA_BF16, x, 4, 4, w, 64, nullptr, 0, nullptr, nullptr, 0, 0, 1e4f, y, nullptr, 0),
            ZSA_EALIGN);
  EXPECT_RC(lin(ZSA_BF16, x, 4, 64, w, 60, nullptr, 0, nullptr, nullptr, 0, 0, 1e4f, y, nullptr, 0),
            ZSA_ESHAPE);
  EXPECT_RC(lin(ZSA_BF16, x, 4, 64, w, 64, nullptr, 5, nullptr, nullptr, 0, 0, 1e4f, y, nullptr, 0),
            ZSA_EINVAL);
  EXPECT_RC(lin(ZSA_BF16, x, 4, 64, w, 72, nullptr, ZSA_EPI_SWIGLU, nullptr, nullptr, 0, 0, 1e4f, y,
                nullptr, 0),
            ZSA_ESHAPE);
  EXPECT_RC(lin(ZSA_BF16, nullptr, 4, 64, w, 64, nullptr, 0, nullptr, nullptr, 0, 0, 1e4f, y,
                nullptr, 0),
            ZSA_EINVAL);
  // no rows: the row operands may be NULL and nothing is launched
  EXPECT_RC(lin(ZSA_BF16, nullptr, 0, 64, w, 64, nullptr, ZSA_EPI_RESIDUAL, nullptr, nullptr, 0, 0,
                1e4f, nullptr, nullptr, 0),
            ZSA_OK);
  EXPECT_RC(lin(ZSA_BF16, nullptr, 0, 64, w, 64, nullptr, ZSA_EPI_ROPE, nullptr, nullptr, 64, 64,
                1e4f, nullptr, nullptr, 0),
            ZSA_OK);
  EXPECT_RC(lin(ZSA_BF16, nullptr, 0, 64, nullptr, 64, nullptr, 0, nullptr, nullptr, 0, 0, 1e4f,
                nullptr, nullptr, 0),
            ZSA_EINVAL);
  EXPECT_RC(lin(ZSA_BF16, x, 4, 64, C(0x2002), 64, nullptr, 0, nullptr, nullptr, 0, 0, 1e4f, y,
                nullptr, 0),
            ZSA_EALIGN);
  EXPECT_RC(lin(ZSA_BF16, x, 4, 64, w, 64, C(0x4004), 0, nullptr, nullptr, 0, 0, 1e4f, y, nullptr,
                0),
            ZSA_EALIGN);
  EXPECT_RC(lin(ZSA_BF16, x, 4, 64, w, 64, nullptr, ZSA_EPI_RESIDUAL, nullptr, nullptr, 0, 0, 1e4f,
                y, nullptr, 0),
            ZSA_EINVAL);
  const int32_t* pos = I(0x5000);
  EXPECT_RC(lin(ZSA_BF16, x, 4, 64, w, 192, nullptr, ZSA_EPI_ROPE, nullptr, pos, 48, 96, 1e4f, y,
                nullptr, 0),
            ZSA_EUNSUPPORTED);
  EXPECT_RC(lin(ZSA_BF16, x, 4, 64, w, 192, nullptr, ZSA_EPI_ROPE, nullptr, pos, 64, 96, 1e4f, y,
                nullptr, 0),
            ZSA_ESHAPE);
  EXPECT_RC(lin(ZSA_BF16, x, 4, 64, w, 192, nullptr, ZSA_EPI_ROPE, nullptr, pos, 64, 256, 1e4f, y,
                nullptr, 0),
            ZSA_ESHAPE);
  EXPECT_RC(lin(ZSA_BF16, x, 4, 64, w, 192, nullptr, ZSA_EPI_ROPE, nullptr, nullptr, 64, 128, 1e4f,
                y, nullptr, 0),
            ZSA_EINVAL);
  EXPECT_RC(lin(ZSA_BF16, x, 4, 64, w, 192, nullptr, ZSA_EPI_ROPE, nullptr, pos, 64, 128, 0.f, y,
                nullptr, 0),
            ZSA_EINVAL);
  EXPECT_RC(lin(ZSA_BF16, x, 4, 64, w, 64, nullptr, 0, nullptr, nullptr, 0, 0, 1e4f, y, A(0x6008),
                64),
            ZSA_EALIGN);
  CHECK_TRUE(zsa_linear_workspace_size(ZSA_BF16, 0, 64, 64) == 0);
  CHECK_TRUE(zsa_linear_workspace_size(ZSA_BF16, 4, -1, 64) == 0);
}

void attention_checks() {
  const int32_t cu[2] = {0, 8};
  const int32_t cu_bad0[2] = {1, 8};
  const int32_t cu_down[3] = {0, 8, 4};
  const void* q = C(0x1000);
  auto att = [&](int dtype, const void* qq, int64_t rs, int H, int Hkv, int hd, float scale,
                 int batch, const int32_t* cuh, const int32_t* cud, void* out, int64_t os,
                 float* lse, float* scores, void* ws, size_t wsb) {
    return zsa_attention_with_scores(nullptr, dtype, qq, q, q, rs, H, Hkv, hd, 0, scale, batch, cuh,
                                     cud, out, os, lse, scores, ws, wsb);
  };
  const int32_t* cud = I(0x2000);
  void* out = A(0x3000);
  EXPECT_RC(att(3, q, 128, 2, 0, 64, 0.1f, 1, cu, cud, out, 128, F(0x4000), nullptr, nullptr, 0),
            ZSA_EINVAL);
  EXPECT_RC(att(ZSA_BF16, q, 96, 2, 0, 48, 0.1f, 1, cu, cud, out, 96, F(0x4000), nullptr, nullptr, 0),
            ZSA_EUNSUPPORTED);
  EXPECT_RC(att(ZSA_BF16, q, 384, 6, 4, 64, 0.1f, 1, cu, cud, out, 384, F(0x4000), nullptr, nullptr,
                0),
            ZSA_ESHAPE);
  EXPECT_RC(att(ZSA_BF16, q, 128, 0, 0, 64, 0.1f, 1, cu, cud, out, 128, F(0x4000), nullptr, nullptr,
                0),
            ZSA_EINVAL);
  EXPECT_RC(att(ZSA_BF16, q, 128, 2, 0, 64, 0.1f, -1, cu, cud, out, 128, F(0x4000), nullptr, nullptr,
                0),
            ZSA_EINVAL);
  EXPECT_RC(att(ZSA_BF16, q, 128, 2, 0, 64, 0.1f, 1, nullptr, cud, out, 128, F(0x4000), nullptr,
                nullptr, 0),
            ZSA_EINVAL);
  EXPECT_RC(att(ZSA_BF16, q, 128, 2, 0, 64, 0.1f, 1, cu, nullptr, out, 128, F(0x4000), nullptr,
                nullptr, 0),
            ZSA_EINVAL);
  EXPECT_RC(att(ZSA_BF16, q, 128, 2, 0, 64, 0.1f, 1, cu_bad0, cud, out, 128, F(0x4000), nullptr,
                nullptr, 0),
            ZSA_ESHAPE);
  EXPECT_RC(att(ZSA_BF16, q, 128, 2, 0, 64, 0.1f, 2, cu_down, cud, out, 128, F(0x4000), nullptr,
                nullptr, 0),
            ZSA_ESHAPE);
  EXPECT_RC(att(ZSA_BF16, C(0x1002), 128, 2, 0, 64, 0.1f, 1, cu, cud, out, 128, F(0x4000), nullptr,
                nullptr, 0),
            ZSA_EALIGN);
  EXPECT_RC(att(ZSA_BF16, q, 128, 2, 0, 64, 0.1f, 1, cu, cud, nullptr, 128, F(0x4000), nullptr,
                nullptr, 0),
            ZSA_EINVAL);
  EXPECT_RC(att(ZSA_BF16, q, 124, 2, 0, 64, 0.1f, 1, cu, cud, out, 128, F(0x4000), nullptr, nullptr,
                0),
            ZSA_EALIGN);
  EXPECT_RC(att(ZSA_BF16, q, 64, 2, 0, 64, 0.1f, 1, cu, cud, out, 128, F(0x4000), nullptr, nullptr,
                0),
            ZSA_ESHAPE);
  EXPECT_RC(att(ZSA_BF16, q, 128, 2, 0, 64, 0.f, 1, cu, cud, out, 128, F(0x4000), nullptr, nullptr,
                0),
            ZSA_EINVAL);
  EXPECT_RC(att(ZSA_BF16, q, 128, 2, 0, 64, NAN, 1, cu, cud, out, 128, F(0x4000), nullptr, nullptr,
                0),
            ZSA_EINVAL);
  EXPECT_RC(att(ZSA_BF16, q, 128, 2, 0, 64, 0.1f, 1, cu, cud, out, 128, nullptr, F(0x5000), nullptr,
                0),
            ZSA_EWORKSPACE);
  const int32_t cu_long[2] = {0, 200000};
  EXPECT_RC(att(ZSA_BF16, q, 12288, 32, 0, 128, 0.1f, 1, cu_long, cud, out, 4096, F(0x4000),
                nullptr, nullptr, 0),
            ZSA_EUNSUPPORTED);
  // every sequence empty: the row operands may be NULL and nothing is launched
  const int32_t cu_empty[3] = {0, 0, 0};
  EXPECT_RC(zsa_attention_with_scores(nullptr, ZSA_BF16, nullptr, nullptr, nullptr, 128, 2, 0, 64,
                                      1, 0.1f, 2, cu_empty, cud, nullptr, 128, nullptr, nullptr,
                                      nullptr, 0),
            ZSA_OK);
  EXPECT_RC(zsa_score_positions(nullptr, ZSA_BF16, nullptr, nullptr, 128, nullptr, 2, 0, 64, 1,
                                0.1f, 2, cu_empty, cud, nullptr, nullptr, 0),
            ZSA_OK);
  EXPECT_RC(zsa_attention_with_scores(nullptr, ZSA_BF16, nullptr, nullptr, nullptr, 128, 2, 0, 64,
                                      1, 0.1f, 1, cu, cud, out, 128, F(0x4000), nullptr, nullptr,
                                      0),
            ZSA_EINVAL);
  CHECK_TRUE(zsa_attention_workspace_size(0, 8, 1) == 0);
  CHECK_TRUE(zsa_attention_workspace_size(2, 8, 1) > zsa_attention_workspace_size(2, 8, 0));

  // scores alone
  EXPECT_RC(zsa_score_positions(nullptr, ZSA_BF16, q, q, 128, nullptr, 2, 0, 64, 1, 0.1f, 1, cu,
                                cud, F(0x5000), A(0x6000), 1 << 20),
            ZSA_EINVAL);
  EXPECT_RC(zsa_score_positions(nullptr, ZSA_BF16, q, q, 128, F(0x4000), 2, 0, 64, 1, 0.1f, 1, cu,
                                cud, nullptr, A(0x6000), 1 << 20),
            ZSA_EINVAL);
  EXPECT_RC(zsa_score_positions(nullptr, ZSA_BF16, q, q, 128, F(0x4000), 2, 0, 64, 1, 0.1f, 1, cu,
                                cud, F(0x5000), nullptr, 0),
            ZSA_EWORKSPACE);
  EXPECT_RC(zsa_score_positions(nullptr, ZSA_BF16, q, q, 128, F(0x4000), 2, 0, 64, 1, -1.f, 1, cu,
                                cud, F(0x5000), A(0x6000), 1 << 20),
            ZSA_EINVAL);
  CHECK_TRUE(zsa_score_workspace_size(-1, 8) == 0);
}

void select_gather_checks() {
  const int32_t cu[3] = {0, 8, 20};
  const int32_t k_ok[2] = {4, 6};
  const int32_t k_big[2] = {9, 6};
  const int32_t k_neg[2] = {-1, 6};
  const int32_t cu_down[3] = {0, 8, 4};
  const float* s = F(0x1000);
  const int32_t* cud = I(0x2000);
  EXPECT_RC(zsa_select_topk(nullptr, s, 2, cu_down, cud, k_ok, 0, I(0x3000), A(0x4000), 1024),
            ZSA_ESHAPE);
  EXPECT_RC(zsa_select_topk(nullptr, s, 2, cu, cud, nullptr, 0, I(0x3000), A(0x4000), 1024),
            ZSA_EINVAL);
  EXPECT_RC(zsa_select_topk(nullptr, s, 2, cu, cud, k_big, 0, I(0x3000), A(0x4000), 1024),
            ZSA_ESHAPE);
  EXPECT_RC(zsa_select_topk(nullptr, s, 2, cu, cud, k_neg, 0, I(0x3000), A(0x4000), 1024),
            ZSA_ESHAPE);
  EXPECT_RC(zsa_select_topk(nullptr, nullptr, 2, cu, cud, k_ok, 0, I(0x3000), A(0x4000), 1024),
            ZSA_EINVAL);
  EXPECT_RC(zsa_select_topk(nullptr, s, 2, cu, cud, k_ok, 0, nullptr, A(0x4000), 1024), ZSA_EINVAL);
  EXPECT_RC(zsa_select_topk(nullptr, s, 2, cu, cud, k_ok, 1, I(0x3000), A(0x4000), 4),
            ZSA_EWORKSPACE);
  EXPECT_RC(zsa_select_topk(nullptr, s, 2, cu, cud, k_ok, 1, I(0x3000), nullptr, 1024),
            ZSA_EWORKSPACE);
  CHECK_TRUE(zsa_select_workspace_size(-1) == 0);
  CHECK_TRUE(zsa_select_workspace_size(31) >= 32 * 4);

  EXPECT_RC(zsa_compact_gather(nullptr, 9, C(0x1000), 64, nullptr, 8, I(0x2000), 4, A(0x3000),
                               nullptr),
            ZSA_EINVAL);
  EXPECT_RC(zsa_compact_gather(nullptr, ZSA_BF16, C(0x1000), 12, nullptr, 8, I(0x2000), 4,
                               A(0x3000), nullptr),
            ZSA_EALIGN);
  EXPECT_RC(zsa_compact_gather(nullptr, ZSA_BF16, C(0x1000), 64, nullptr, -1, I(0x2000), 4,
                               A(0x3000), nullptr),
            ZSA_EINVAL);
  EXPECT_RC(zsa_compact_gather(nullptr, ZSA_BF16, C(0x1000), 64, I(0x5000), 8, I(0x2000), 4,
                               A(0x3000), nullptr),
            ZSA_EINVAL);
  EXPECT_RC(zsa_compact_gather(nullptr, ZSA_BF16, nullptr, 64, nullptr, 8, I(0x2000), 4, A(0x3000),
                               nullptr),
            ZSA_EINVAL);
  EXPECT_RC(zsa_compact_gather(nullptr, ZSA_BF16, C(0x1000), 64, nullptr, 8, I(0x2000), 4,
                               A(0x3008), nullptr),
            ZSA_EALIGN);
  EXPECT_RC(zsa_compact_gather(nullptr, ZSA_BF16, C(0x1000), 64, nullptr, 8, nullptr, 4, A(0x3000),
                               nullptr),
            ZSA_EINVAL);
}

// one bad field of an otherwise valid layer configuration at a time
void cfg_checks() {
  const int32_t cu[2] = {0, 16};
  int32_t cu_out[2];
  const zsa_layer_weights w = weights_at(0x100000);
  auto layer = [&](const zsa_layer_cfg* c) {
    return zsa_layer_forward(nullptr, c, &w, C(0x1000), I(0x2000), 1, cu, I(0x3000), nullptr,
                             A(0x4000), I(0x5000), cu_out, I(0x6000), nullptr, nullptr, A(0x7000),
                             size_t{1} << 40);
  };
  const zsa_layer_cfg good = cfg_of(ZSA_DECODER, 256, 4, 512, 1, ZSA_BF16);
  EXPECT_RC(layer(nullptr), ZSA_EINVAL);
  zsa_layer_cfg c = good;
  c.kind = 2;
  EXPECT_RC(layer(&c), ZSA_EINVAL);
  c = good;
  c.dtype = 4;
  EXPECT_RC(layer(&c), ZSA_EINVAL);
  c = good;
  c.n_heads = 3;
  EXPECT_RC(layer(&c), ZSA_ESHAPE);
  c = good;
  c.n_heads = 1;
  c.head_dim = 256;
  EXPECT_RC(layer(&c), ZSA_EUNSUPPORTED);
  c = good;
  c.d_ff = 4;
  EXPECT_RC(layer(&c), ZSA_EALIGN);
  c = good;
  c.d_model = 8704;
  c.n_heads = 68;
  c.head_dim = 128;
  EXPECT_RC(layer(&c), ZSA_EUNSUPPORTED);
  c = good;
  c.tau = 0;
  EXPECT_RC(layer(&c), ZSA_EINVAL);
  c = good;
  c.norm_eps = NAN;
  EXPECT_RC(layer(&c), ZSA_EINVAL);
  c = good;
  c.rope_theta = 0.f;
  EXPECT_RC(layer(&c), ZSA_EINVAL);
  c = good;
  c.n_kv_heads = 3;
  EXPECT_RC(layer(&c), ZSA_ESHAPE);
  c = good;
  c.n_kv_heads = -1;
  EXPECT_RC(layer(&c), ZSA_ESHAPE);
  // the encoder ignores rope_theta
  c = cfg_of(ZSA_ENCODER, 256, 4, 512, 0, ZSA_BF16);
  c.rope_theta = 0.f;
  c.tau = 0;
  EXPECT_RC(layer(&c), ZSA_EINVAL);  // still the tau check, not the rotary base
}

void layer_checks() {
  const int32_t cu[3] = {0, 16, 40};
  int32_t cu_out[3];
  const zsa_layer_cfg c = cfg_of(ZSA_ENCODER, 256, 4, 512, 0, ZSA_BF16);
  const zsa_layer_weights w = weights_at(0x100000);
  const double rates[2] = {0.5, 0.5};
  const double bad_rates[2] = {0.5, 1.5};
  auto layer = [&](const zsa_layer_weights* ww, const void* x, const int32_t* pos,
                   const int32_t* cuh, const double* kr, int32_t* cuo, void* ws, size_t wsb) {
    return zsa_layer_forward(nullptr, &c, ww, x, pos, 2, cuh, I(0x3000), kr, A(0x4000), I(0x5000),
                             cuo, I(0x6000), nullptr, nullptr, ws, wsb);
  };
  const size_t big = size_t{1} << 40;
  EXPECT_RC(layer(nullptr, C(0x1000), I(0x2000), cu, rates, cu_out, A(0x7000), big), ZSA_EINVAL);
  zsa_layer_weights bad = w;
  bad.w_o = nullptr;
  EXPECT_RC(layer(&bad, C(0x1000), I(0x2000), cu, rates, cu_out, A(0x7000), big), ZSA_EINVAL);
  bad = w;
  bad.b_up = C(0x100008);
  EXPECT_RC(layer(&bad, C(0x1000), I(0x2000), cu, rates, cu_out, A(0x7000), big), ZSA_EALIGN);
  bad = w;
  bad.norm2_b = C(0x100004);
  EXPECT_RC(layer(&bad, C(0x1000), I(0x2000), cu, rates, cu_out, A(0x7000), big), ZSA_EALIGN);
  const int32_t cu_down[3] = {0, 16, 8};
  EXPECT_RC(layer(&w, C(0x1000), I(0x2000), cu_down, rates, cu_out, A(0x7000), big), ZSA_ESHAPE);
  EXPECT_RC(layer(&w, nullptr, I(0x2000), cu, rates, cu_out, A(0x7000), big), ZSA_EINVAL);
  EXPECT_RC(layer(&w, C(0x1000), nullptr, cu, rates, cu_out, A(0x7000), big), ZSA_EINVAL);
  EXPECT_RC(layer(&w, C(0x1000), I(0x2000), cu, rates, nullptr, A(0x7000), big), ZSA_EINVAL);
  EXPECT_RC(layer(&w, C(0x1000), I(0x2000), cu, bad_rates, cu_out, A(0x7000), big), ZSA_EINVAL);
  EXPECT_RC(layer(&w, C(0x1000), I(0x2000), cu, rates, cu_out, A(0x7000), 16), ZSA_EWORKSPACE);
  EXPECT_RC(layer(&w, C(0x1000), I(0x2000), cu, rates, cu_out, nullptr, big), ZSA_EWORKSPACE);
  CHECK_TRUE(zsa_layer_workspace_size(nullptr, 16, 1) == 0);
  CHECK_TRUE(zsa_layer_workspace_size(&c, -1, 1) == 0);
  CHECK_TRUE(zsa_layer_workspace_size(&c, 4096, 2) > zsa_layer_workspace_size(&c, 16, 2));
}

void stack_checks() {
  const int32_t cu[3] = {0, 16, 40};
  int32_t cu_out[3], counts[6];
  zsa_layer_cfg c = cfg_of(ZSA_DECODER, 256, 4, 512, 1, ZSA_BF16);
  zsa_layer_weights w[3] = {weights_at(0x100000), weights_at(0x200000), weights_at(0x300000)};
  const double rates[2] = {0.5, 0.25};
  const int32_t pa[2] = {1, 3};
  const size_t big = size_t{1} << 40;
  auto stack = [&](const zsa_layer_cfg* cc, const zsa_layer_weights* ww, int L, const int32_t* p,
                   int np, const double* kr, const void* x, int32_t* cuo, void* kv, int kv_cap,
                   size_t wsb) {
    return zsa_stack_forward(nullptr, cc, ww, L, p, np, kr, x, I(0x2000), 2, cu, I(0x3000),
                             A(0x4000), I(0x5000), cuo, I(0x6000), counts, nullptr, nullptr,
                             nullptr, kv, kv_cap, A(0x7000), wsb);
  };
  EXPECT_RC(stack(&c, w, 0, pa, 2, rates, C(0x1000), cu_out, nullptr, 0, big), ZSA_EINVAL);
  EXPECT_RC(stack(&c, nullptr, 3, pa, 2, rates, C(0x1000), cu_out, nullptr, 0, big), ZSA_EINVAL);
  zsa_layer_weights keep = w[1];
  w[1].w_down = C(0x200002);
  EXPECT_RC(stack(&c, w, 3, pa, 2, rates, C(0x1000), cu_out, nullptr, 0, big), ZSA_EALIGN);
  CHECK_TRUE(strstr(zsa_last_error(), "layer 2") != nullptr);
  w[1] = keep;
  EXPECT_RC(stack(&c, w, 3, nullptr, 2, rates, C(0x1000), cu_out, nullptr, 0, big), ZSA_EINVAL);
  const int32_t pa_high[2] = {1, 4};
  EXPECT_RC(stack(&c, w, 3, pa_high, 2, rates, C(0x1000), cu_out, nullptr, 0, big), ZSA_EINVAL);
  const int32_t pa_flat[2] = {2, 2};
  EXPECT_RC(stack(&c, w, 3, pa_flat, 2, rates, C(0x1000), cu_out, nullptr, 0, big), ZSA_EINVAL);
  EXPECT_RC(stack(&c, w, 3, pa, -1, rates, C(0x1000), cu_out, nullptr, 0, big), ZSA_EINVAL);
  EXPECT_RC(stack(&c, w, 3, pa, 2, nullptr, C(0x1000), cu_out, nullptr, 0, big), ZSA_EINVAL);
  const double nan_rates[2] = {NAN, 0.5};
  EXPECT_RC(stack(&c, w, 3, pa, 2, nan_rates, C(0x1000), cu_out, nullptr, 0, big), ZSA_EINVAL);
  EXPECT_RC(stack(&c, w, 3, pa, 2, rates, C(0x1008), cu_out, nullptr, 0, big), ZSA_EALIGN);
  EXPECT_RC(stack(&c, w, 3, pa, 2, rates, C(0x1000), nullptr, nullptr, 0, big), ZSA_EINVAL);
  EXPECT_RC(stack(&c, w, 3, pa, 2, rates, C(0x1000), cu_out, A(0x8008), 64, big), ZSA_EALIGN);
  EXPECT_RC(stack(&c, w, 3, pa, 2, rates, C(0x1000), cu_out, A(0x8000), 20, big), ZSA_ESHAPE);
  EXPECT_RC(stack(&c, w, 3, pa, 2, rates, C(0x1000), cu_out, nullptr, 0, 64), ZSA_EWORKSPACE);
  zsa_layer_cfg enc = cfg_of(ZSA_ENCODER, 256, 4, 512, 0, ZSA_BF16);
  EXPECT_RC(stack(&enc, w, 3, pa, 2, rates, C(0x1000), cu_out, A(0x8000), 64, big), ZSA_EINVAL);
  CHECK_TRUE(zsa_stack_workspace_size(&c, 40, 2, -1) == 0);
  CHECK_TRUE(zsa_stack_workspace_size(&c, 40, 2, 2) > zsa_layer_workspace_size(&c, 40, 2));

  // backward
  float* g = F(0x900000);
  zsa_layer_grads gr[3];
  for (auto& x : gr) {
    float** p = reinterpret_cast<float**>(&x);
    for (int i = 0; i < 12; ++i) p[i] = g;
  }
  auto bwd = [&](const zsa_layer_cfg* cc, const zsa_layer_grads* gg, const int32_t* p,
                 const double* kr, const void* dy, size_t wsb) {
    return zsa_stack_backward(nullptr, cc, w, gg, 3, p, 2, kr, C(0x1000), I(0x2000), 2, cu,
                              I(0x3000), dy, A(0xa000), A(0x7000), wsb);
  };
  zsa_layer_cfg f32 = cfg_of(ZSA_DECODER, 256, 4, 512, 1, ZSA_F32);
  EXPECT_RC(bwd(&f32, gr, pa, rates, C(0xb000), big), ZSA_EUNSUPPORTED);
  zsa_layer_cfg mark = c;
  mark.mark_only = 1;
  EXPECT_RC(bwd(&mark, gr, pa, rates, C(0xb000), big), ZSA_EUNSUPPORTED);
  EXPECT_RC(bwd(&c, nullptr, pa, rates, C(0xb000), big), ZSA_EINVAL);
  gr[2].w_up = nullptr;
  EXPECT_RC(bwd(&c, gr, pa, rates, C(0xb000), big), ZSA_EINVAL);
  gr[2].w_up = g;
  EXPECT_RC(bwd(&c, gr, pa_flat, rates, C(0xb000), big), ZSA_EINVAL);
  EXPECT_RC(bwd(&c, gr, pa, nan_rates, C(0xb000), big), ZSA_EINVAL);
  EXPECT_RC(bwd(&c, gr, pa, rates, C(0xb004), big), ZSA_EALIGN);
  EXPECT_RC(bwd(&c, gr, pa, rates, C(0xb000), 64), ZSA_EWORKSPACE);
}

void decode_checks() {
  zsa_layer_cfg c = cfg_of(ZSA_DECODER, 256, 4, 512, 1, ZSA_BF16);
  const zsa_layer_weights w[2] = {weights_at(0x100000), weights_at(0x200000)};
  const int32_t pos[2] = {10, 20};
  const int32_t kvl[4] = {10, 20, 5, 9};
  const int32_t kvl_full[4] = {10, 64, 5, 9};
  const size_t big = size_t{1} << 40;
  auto dec = [&](const zsa_layer_cfg* cc, int L, int B, const void* x, const int32_t* p, void* kv,
                 int cap, const int32_t* kl, size_t wsb) {
    return zsa_decode_step(nullptr, cc, w, L, B, x, p, kv, cap, kl, A(0x3000), A(0x7000), wsb);
  };
  zsa_layer_cfg enc = cfg_of(ZSA_ENCODER, 256, 4, 512, 0, ZSA_BF16);
  EXPECT_RC(dec(&enc, 2, 2, C(0x1000), pos, A(0x8000), 64, kvl, big), ZSA_EINVAL);
  zsa_layer_cfg narrow = cfg_of(ZSA_DECODER, 256, 8, 512, 1, ZSA_BF16);  // head_dim 32
  EXPECT_RC(dec(&narrow, 2, 2, C(0x1000), pos, A(0x8000), 64, kvl, big), ZSA_EUNSUPPORTED);
  EXPECT_RC(dec(&c, 0, 2, C(0x1000), pos, A(0x8000), 64, kvl, big), ZSA_EINVAL);
  EXPECT_RC(dec(&c, 2, -1, C(0x1000), pos, A(0x8000), 64, kvl, big), ZSA_EINVAL);
  EXPECT_RC(dec(&c, 2, 2, C(0x1000), pos, A(0x8000), 0, kvl, big), ZSA_EINVAL);
  EXPECT_RC(dec(&c, 2, 2, C(0x1004), pos, A(0x8000), 64, kvl, big), ZSA_EALIGN);
  EXPECT_RC(dec(&c, 2, 2, C(0x1000), pos, A(0x8010), 64, kvl, big), ZSA_EINVAL);
  EXPECT_RC(dec(&c, 2, 2, C(0x1000), nullptr, A(0x8000), 64, kvl, big), ZSA_EINVAL);
  EXPECT_RC(dec(&c, 2, 2, C(0x1000), pos, A(0x8000), 64, kvl_full, big), ZSA_ESHAPE);
  EXPECT_RC(dec(&c, 2, 2, C(0x1000), pos, A(0x8000), 64, kvl, 64), ZSA_EWORKSPACE);
  EXPECT_RC(dec(&c, 2, 2, C(0x1000), pos, A(0x8000), 1 << 24, kvl, big), ZSA_EUNSUPPORTED);
  CHECK_TRUE(dec(&c, 2, 0, nullptr, nullptr, nullptr, 0, nullptr, 0) == ZSA_OK);  // no rows
}

void timing_checks() {
  EXPECT_RC(zsa_timing_arm(-1, 4), ZSA_EINVAL);
  EXPECT_RC(zsa_timing_arm(ZSA_K_NCLASS, 4), ZSA_EINVAL);
  EXPECT_RC(zsa_timing_arm(ZSA_K_GEMM, 0), ZSA_EINVAL);
  int32_t n = -1;
  double ms = -1.0;
  EXPECT_RC(zsa_timing_read(ZSA_K_NCLASS, &n, &ms), ZSA_EINVAL);
  EXPECT_RC(zsa_timing_read(ZSA_K_GEMM, nullptr, &ms), ZSA_EINVAL);
  // never armed: nothing timed, no event touched
  CHECK_TRUE(zsa_timing_read(ZSA_K_GEMM, &n, &ms) == ZSA_OK && n == 0 && ms == 0.0);
}

}  // namespace

int main() {
  CHECK_TRUE(strstr(zsa_version(), "gfx950") != nullptr);
  keep_count_checks();
  keep_schedule_checks();
  norm_checks();
  linear_checks();
  attention_checks();
  select_gather_checks();
  cfg_checks();
  layer_checks();
  stack_checks();
  decode_checks();
  timing_checks();
  printf("ok %d\n", g_checks);
  return 0;
}
