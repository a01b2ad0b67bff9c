// Host-side check of the C ABI's argument validation under AddressSanitizer
// and UndefinedBehaviorSanitizer (host code only; the device code is built
// as usual and never launched).  Every call below is rejected before any HIP
// call, so the fake device addresses are never dereferenced and no GPU is
// needed.  Also drives the pure host helpers (status strings, the
// thread-local message, workspace and attention sizes) with degenerate and
// very large sizes.  Exit status 0 when every expectation holds.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <limits>

#include "catq.h"

static int failures = 0;

static void expect(const char* what, int got, int want) {
  const char* msg = catq_last_error_message();
  if (got != want) {
    std::printf("FAIL %s: status %d, expected %d (%s)\n", what, got, want, msg);
    ++failures;
  } else if (want != CATQ_OK && (msg == nullptr || std::strlen(msg) == 0)) {
    std::printf("FAIL %s: status %d without a message\n", what, got);
    ++failures;
  }
}

#define EXPECT(call, want) expect(#call, (int)(call), (want))

static void* const F = reinterpret_cast<void*>(0x100000);   // aligned, never dereferenced
static void* const F2 = reinterpret_cast<void*>(0x100002);  // misaligned

static catq_lmst_params params(int mode, float s = 15.f, int g = 128, float delta0 = 0.5f,
                               float s_bwd = 30.f) {
  catq_lmst_params p;
  std::memset(&p, 0, sizeof(p));
  p.group_size = g;
  p.mode = mode;
  p.delta0 = delta0;
  p.s = s;
  p.s_bwd = s_bwd;
  p.factor_stride[0] = p.factor_stride[1] = p.factor_stride[2] = 1;
  return p;
}

static catq_attn_desc attn(int b, int s, int hq, int hkv, int d, int aq = 0) {
  catq_attn_desc a;
  std::memset(&a, 0, sizeof(a));
  a.batch = b;
  a.seq = s;
  a.n_q = hq;
  a.n_kv = hkv;
  a.head_dim = d;
  a.qk_norm = 1;
  a.rope_theta = 1e6f;
  a.eps = 1e-6f;
  a.act_quant = aq;
  return a;
}

int main() {
  const float* ff = static_cast<const float*>(F);
  float* fw = static_cast<float*>(F);
  const float nan = std::numeric_limits<float>::quiet_NaN();
  const float inf = std::numeric_limits<float>::infinity();

  // status strings, including values outside the enum
  for (int c = -3; c < 12; ++c) {
    const char* s = catq_status_string((catq_status)c);
    if (!s || std::strncmp(s, "CATQ_", 5) != 0) {
      std::printf("FAIL status string %d\n", c);
      ++failures;
    }
  }

  // catq_modulate_ternarize
  catq_lmst_params ok = params(CATQ_SOFT);
  auto mt = [&](const catq_lmst_params* p, const void* W, int64_t d_out, int64_t d_in,
                int wdt, int sm, void* wf, int8_t* codes) {
    return catq_modulate_ternarize(W, (catq_dtype)wdt, d_out, d_in, ff, ff, ff, p, fw, sm, wf,
                                   CATQ_BF16, codes, nullptr, nullptr);
  };
  EXPECT(mt(&ok, nullptr, 4, 128, 1, 0, F, nullptr), CATQ_ERR_NULL);
  EXPECT(mt(nullptr, F, 4, 128, 1, 0, F, nullptr), CATQ_ERR_NULL);
  EXPECT(mt(&ok, F, 0, 128, 1, 0, F, nullptr), CATQ_ERR_SHAPE);
  EXPECT(mt(&ok, F, -5, 128, 1, 0, F, nullptr), CATQ_ERR_SHAPE);
  EXPECT(mt(&ok, F, 4, 96, 1, 0, F, nullptr), CATQ_ERR_SHAPE);
  EXPECT(mt(&ok, F, INT64_MAX, 128, 1, 0, F, nullptr), CATQ_ERR_SHAPE);
  EXPECT(mt(&ok, F, 4, INT64_MAX - 127, 1, 0, F, nullptr), CATQ_ERR_SHAPE);
  catq_lmst_params g96 = params(CATQ_SOFT, 15.f, 96), g0 = params(CATQ_SOFT, 15.f, 0),
                   gneg = params(CATQ_SOFT, 15.f, -128), g1024 = params(CATQ_SOFT, 15.f, 1024);
  EXPECT(mt(&g96, F, 4, 384, 1, 0, F, nullptr), CATQ_ERR_VALUE);
  EXPECT(mt(&g0, F, 4, 128, 1, 0, F, nullptr), CATQ_ERR_VALUE);
  EXPECT(mt(&gneg, F, 4, 128, 1, 0, F, nullptr), CATQ_ERR_VALUE);
  EXPECT(mt(&g1024, F, 4, 1024, 1, 0, F, nullptr), CATQ_ERR_VALUE);
  catq_lmst_params s0 = params(CATQ_SOFT, 0.f), snan = params(CATQ_SOFT, nan),
                   sinf = params(CATQ_SOFT, inf), d0 = params(CATQ_SOFT, 15.f, 128, 0.f),
                   dnan = params(CATQ_SOFT, 15.f, 128, nan),
                   sb = params(CATQ_SOFT, 15.f, 128, 0.5f, -1.f), m7 = params(7),
                   mneg = params(-1);
  EXPECT(mt(&s0, F, 4, 128, 1, 0, F, nullptr), CATQ_ERR_VALUE);
  EXPECT(mt(&snan, F, 4, 128, 1, 0, F, nullptr), CATQ_ERR_VALUE);
  EXPECT(mt(&sinf, F, 4, 128, 1, 0, F, nullptr), CATQ_ERR_VALUE);
  EXPECT(mt(&d0, F, 4, 128, 1, 0, F, nullptr), CATQ_ERR_VALUE);
  EXPECT(mt(&dnan, F, 4, 128, 1, 0, F, nullptr), CATQ_ERR_VALUE);
  EXPECT(mt(&sb, F, 4, 128, 1, 0, F, nullptr), CATQ_ERR_VALUE);
  EXPECT(mt(&m7, F, 4, 128, 1, 0, F, nullptr), CATQ_ERR_VALUE);
  EXPECT(mt(&mneg, F, 4, 128, 1, 0, F, nullptr), CATQ_ERR_VALUE);
  catq_lmst_params st2 = ok;
  st2.factor_stride[1] = 2;
  EXPECT(mt(&st2, F, 4, 128, 1, 0, F, nullptr), CATQ_ERR_VALUE);
  st2.factor_stride[1] = -1;
  EXPECT(mt(&st2, F, 4, 128, 1, 0, F, nullptr), CATQ_ERR_VALUE);
  EXPECT(mt(&ok, F, 4, 128, 5, 0, F, nullptr), CATQ_ERR_DTYPE);
  EXPECT(mt(&ok, F, 4, 128, -1, 0, F, nullptr), CATQ_ERR_DTYPE);
  EXPECT(mt(&ok, F, 4, 128, 1, 2, F, nullptr), CATQ_ERR_VALUE);
  EXPECT(mt(&ok, F, 4, 128, 1, 0, nullptr, nullptr), CATQ_ERR_NULL);
  EXPECT(mt(&ok, F, 4, 128, 1, 0, F, static_cast<int8_t*>(F)), CATQ_ERR_VALUE);
  EXPECT(mt(&ok, F2, 4, 128, 1, 0, F, nullptr), CATQ_ERR_ALIGN);

  // catq_ternarize_pack
  catq_lmst_params hard = params(CATQ_HARD);
  auto tp = [&](const catq_lmst_params* p, const void* W, int64_t d_out, int64_t d_in,
                void* packed) {
    return catq_ternarize_pack(W, CATQ_BF16, d_out, d_in, ff, ff, ff, p, fw, 1,
                               static_cast<uint8_t*>(packed), nullptr, nullptr);
  };
  EXPECT(tp(&hard, nullptr, 4, 256, F), CATQ_ERR_NULL);
  EXPECT(tp(&hard, F, 4, 256, nullptr), CATQ_ERR_NULL);
  EXPECT(tp(&ok, F, 4, 256, F), CATQ_ERR_VALUE);
  EXPECT(tp(&hard, F, 0, 256, F), CATQ_ERR_SHAPE);
  EXPECT(tp(&hard, F, 4, 96, F), CATQ_ERR_SHAPE);
  EXPECT(tp(&hard, F, 4, 256, F2), CATQ_ERR_ALIGN);

  // catq_fakeq_linear_fwd
  auto fwd = [&](const void* X, int dt, int64_t M, int64_t N, int64_t K, int E,
                 const int64_t* offs, const void* res, int ydt, int rdt) {
    return catq_fakeq_linear_fwd(X, F, (catq_dtype)dt, F, (catq_dtype)ydt, M, N, K, E, offs, res,
                                 (catq_dtype)rdt, nullptr);
  };
  const int64_t* fo = static_cast<const int64_t*>(F);
  EXPECT(fwd(F, 1, 0, 8, 8, 1, nullptr, nullptr, 1, 1), CATQ_ERR_SHAPE);
  EXPECT(fwd(F, 1, 8, 8, 12, 1, nullptr, nullptr, 1, 1), CATQ_ERR_SHAPE);
  EXPECT(fwd(F, 1, INT64_MAX, INT64_MAX, 8, 1, nullptr, nullptr, 1, 1), CATQ_ERR_SHAPE);
  EXPECT(fwd(nullptr, 1, 8, 8, 8, 1, nullptr, nullptr, 1, 1), CATQ_ERR_NULL);
  EXPECT(fwd(F, 1, 8, 8, 8, 4, nullptr, nullptr, 1, 1), CATQ_ERR_NULL);
  EXPECT(fwd(F, 9, 8, 8, 8, 1, nullptr, nullptr, 1, 1), CATQ_ERR_DTYPE);
  EXPECT(fwd(F, 1, 8, 8, 8, 4, fo, F, 1, 1), CATQ_ERR_VALUE);
  EXPECT(fwd(F, 0, 8, 8, 8, 1, nullptr, nullptr, 1, 0), CATQ_ERR_DTYPE);
  EXPECT(fwd(F2, 1, 8, 8, 8, 1, nullptr, nullptr, 1, 1), CATQ_ERR_ALIGN);
  EXPECT(fwd(F, 1, 8, 8, 8, 0, nullptr, nullptr, 1, 1), CATQ_ERR_SHAPE);

  // catq_fakeq_linear_bwd
  auto bwd = [&](int64_t M, int64_t N, int64_t K, void* dX, float* gm, float* ga, float* gd,
                 const float* dmu, size_t ws_bytes) {
    return catq_fakeq_linear_bwd(F, F, F, CATQ_BF16, M, N, K, 1, nullptr, F, CATQ_BF16, ff, dmu,
                                 ff, ff, &ok, dX, gm, ga, gd, nullptr, F, ws_bytes, nullptr);
  };
  EXPECT(bwd(64, 256, 128, F, fw, fw, fw, ff, 16), CATQ_ERR_WORKSPACE);
  EXPECT(bwd(64, 256, 128, F, fw, fw, fw, nullptr, 1u << 30), CATQ_ERR_NULL);
  EXPECT(bwd(64, 252, 128, F, fw, fw, fw, ff, 1u << 30), CATQ_ERR_SHAPE);
  EXPECT(bwd(64, 256, 128, F, fw, nullptr, fw, ff, 1u << 30), CATQ_ERR_NULL);
  EXPECT(bwd(64, 256, 128, nullptr, nullptr, nullptr, nullptr, ff, 1u << 30), CATQ_ERR_NULL);
  EXPECT(bwd(64, 256, 128, F2, nullptr, nullptr, nullptr, ff, 1u << 30), CATQ_ERR_ALIGN);
  EXPECT(bwd(INT64_MAX / 2, 256, 128, F, fw, fw, fw, ff, 1u << 30), CATQ_ERR_SHAPE);

  // catq_block_recon_loss and its allocation-free variant
  EXPECT(catq_block_recon_loss(F, F, CATQ_BF16, 12, fw, nullptr, CATQ_BF16, F, 1 << 20, nullptr),
         CATQ_ERR_SHAPE);
  EXPECT(catq_block_recon_loss(F, F, CATQ_BF16, 16, fw, nullptr, CATQ_BF16, F, 8, nullptr),
         CATQ_ERR_WORKSPACE);
  EXPECT(catq_block_recon_loss(F, nullptr, CATQ_BF16, 16, fw, nullptr, CATQ_BF16, F, 1 << 20,
                               nullptr),
         CATQ_ERR_NULL);
  EXPECT(catq_block_recon_loss_noalloc(F, F, CATQ_BF16, -8, fw, nullptr, CATQ_BF16, nullptr),
         CATQ_ERR_SHAPE);
  EXPECT(catq_block_recon_loss_noalloc(F, F, (catq_dtype)7, 16, fw, F, CATQ_BF16, nullptr),
         CATQ_ERR_DTYPE);
  EXPECT(catq_block_recon_loss_noalloc(F2, F, CATQ_BF16, 16, fw, nullptr, CATQ_BF16, nullptr),
         CATQ_ERR_ALIGN);

  // catq_pack_ternary
  EXPECT(catq_pack_ternary(static_cast<int8_t*>(F), 4, 6, static_cast<uint8_t*>(F), nullptr),
         CATQ_ERR_SHAPE);
  EXPECT(catq_pack_ternary(nullptr, 4, 8, static_cast<uint8_t*>(F), nullptr), CATQ_ERR_NULL);

  // catq_ternary_linear
  auto tl = [&](int64_t M, int64_t ldx, int64_t d_out, int64_t d_in, int g, int dt) {
    return catq_ternary_linear(F, M, ldx, static_cast<uint8_t*>(F), ff, d_out, d_in, g, F,
                               (catq_dtype)dt, d_out, nullptr);
  };
  EXPECT(tl(0, 256, 32, 256, 128, 0), CATQ_OK);  // M = 0: no-op, nothing launched
  EXPECT(tl(-1, 256, 32, 256, 128, 0), CATQ_ERR_SHAPE);
  EXPECT(tl(4, 256, 32, 192, 128, 0), CATQ_ERR_SHAPE);
  EXPECT(tl(4, 256, 32, 256, 64, 0), CATQ_ERR_VALUE);
  EXPECT(tl(4, 256, 32, 256, 0, 0), CATQ_ERR_VALUE);
  EXPECT(tl(4, 256, 32, 256, 128, 3), CATQ_ERR_DTYPE);
  EXPECT(tl(4, INT64_MAX, 32, 256, 128, 0), CATQ_ERR_SHAPE);

  // glue entry points
  EXPECT(catq_aux_rmsnorm_fwd(F, CATQ_BF16, 4, 12, 1e-6f, F, fw, nullptr), CATQ_ERR_SHAPE);
  EXPECT(catq_aux_swiglu_fwd(F, 4, 12, F, nullptr), CATQ_ERR_SHAPE);
  EXPECT(catq_fakeq_gateup_swiglu_fwd(F, nullptr, 4, 16, 64, F, F, nullptr), CATQ_ERR_NULL);
  EXPECT(catq_fakeq_down_swiglu_bwd(F, F, 4, 64, 12, F, F, F, nullptr), CATQ_ERR_SHAPE);
  EXPECT(catq_aux_act_quant(F, CATQ_BF16, 4, 64, 24, F, nullptr), CATQ_ERR_SHAPE);
  EXPECT(catq_aux_adamw(fw, ff, fw, fw, 4, 0, 1e-3f, 0.9, 0.999, 1e-8, -1.f, 1.f, nullptr),
         CATQ_ERR_SHAPE);
  EXPECT(catq_aux_adamw(fw, ff, fw, fw, 4, 1, 1e-3f, 1.5, 0.999, 1e-8, -1.f, 1.f, nullptr),
         CATQ_ERR_VALUE);
  EXPECT(catq_aux_adamw(fw, ff, fw, fw, 4, INT64_MAX, 1e-3f, 0.9, 0.999, 0.0, -1.f, 1.f, nullptr),
         CATQ_ERR_VALUE);
  catq_attn_desc a1 = attn(1, 16, 3, 2, 64), a2 = attn(1, 16, 2, 1, 96), a3 = attn(1, 16, 2, 1, 64),
                 a4 = attn(1, 16, 2, 0, 64), a5 = attn(-1, 16, 2, 1, 64),
                 a6 = attn(1, 16, 2, 1, 256, 1);
  EXPECT(catq_aux_attention_fwd(&a1, F, F, F, 1u << 30, nullptr), CATQ_ERR_SHAPE);
  EXPECT(catq_aux_attention_fwd(&a2, F, F, F, 1u << 30, nullptr), CATQ_ERR_SHAPE);
  EXPECT(catq_aux_attention_fwd(&a3, F, F, F, 16, nullptr), CATQ_ERR_WORKSPACE);
  EXPECT(catq_aux_attention_fwd(&a4, F, F, F, 1u << 30, nullptr), CATQ_ERR_SHAPE);
  EXPECT(catq_aux_attention_fwd(&a5, F, F, F, 1u << 30, nullptr), CATQ_ERR_SHAPE);
  EXPECT(catq_aux_attention_fwd(&a6, F, F, F, 1u << 30, nullptr), CATQ_ERR_VALUE);
  EXPECT(catq_aux_attention_fwd(nullptr, F, F, F, 1u << 30, nullptr), CATQ_ERR_NULL);
  EXPECT(catq_aux_moe_route(ff, 8, 4, 5, static_cast<int32_t*>(F), fw, static_cast<int32_t*>(F),
                            static_cast<int64_t*>(F), F, 4096, nullptr),
         CATQ_ERR_SHAPE);

  // size helpers: degenerate and very large arguments must not overflow
  volatile size_t sink = 0;
  const int64_t big[] = {0, 1, 8, 8192, int64_t(1) << 31, int64_t(1) << 40, INT64_MAX};
  for (int64_t m : big)
    for (int64_t n : big) {
      sink += catq_workspace_size(CATQ_WS_LINEAR_BWD, m, n, 4096, 1);
      sink += catq_workspace_size(CATQ_WS_LINEAR_BWD, 8192, m, n, 128);
      sink += catq_workspace_size(CATQ_WS_LOSS, m, 1, 1, 1);
      sink += catq_aux_moe_route_workspace_bytes(m, 128, 8);
    }
  sink += catq_workspace_size(CATQ_WS_LINEAR_BWD, -1, 8, 8, 1);
  sink += catq_workspace_size(7, 8, 8, 8, 1);
  const int dims[] = {0, 1, 16, 4096, 1 << 20, INT32_MAX};
  for (int b : dims)
    for (int s : dims) {
      catq_attn_desc d = attn(b, s, 64, 4, 128);
      sink += catq_attn_saved_bytes(&d);
      sink += catq_attn_bwd_workspace_bytes(&d);
    }
  catq_attn_desc dz = attn(1, 16, 2, 0, 64);
  sink += catq_attn_saved_bytes(&dz) + catq_attn_bwd_workspace_bytes(&dz);
  (void)sink;

  // tracing without a GPU: everything but enable/get on a live trace
  EXPECT(catq_trace_enable(0), CATQ_ERR_VALUE);
  EXPECT(catq_trace_enable(-4), CATQ_ERR_VALUE);
  catq_trace_pause(0);
  catq_trace_reset();
  if (catq_trace_count() != 0) {
    std::printf("FAIL trace count\n");
    ++failures;
  }
  catq_trace_rec rec;
  EXPECT(catq_trace_get(0, &rec), CATQ_ERR_VALUE);
  EXPECT(catq_trace_get(-1, &rec), CATQ_ERR_VALUE);
  EXPECT(catq_trace_get(0, nullptr), CATQ_ERR_NULL);
  catq_trace_disable();

  std::printf("%s: %d failure(s)\n", failures ? "FAILED" : "ok", failures);
  return failures ? 1 : 0;
}
