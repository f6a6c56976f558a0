// Host-side checks of the C ABI under AddressSanitizer and UBSan (built with
// the sanitizers on the host code only; no GPU is needed): configuration
// validation, per-sequence layouts, workspace plans, argument checks of every
// entry point, and the error paths that reach the HIP runtime (which fails
// cleanly without a device). Exits non-zero on the first failed expectation;
// the sanitizers abort on any memory error or undefined behaviour.
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "ldr.h"

static int g_fail = 0;
#define EXPECT(c)                                                     \
  do {                                                                \
    if (!(c)) {                                                       \
      std::fprintf(stderr, "%s:%d: expectation failed: %s\n", __FILE__, __LINE__, #c); \
      ++g_fail;                                                       \
    }                                                                 \
  } while (0)

static ldr_config qwen3_8b() {
  ldr_config c;
  std::memset(&c, 0, sizeof(c));
  c.hidden = 4096; c.n_q_heads = 32; c.n_kv_heads = 8; c.head_dim = 128; c.mlp = 12288;
  c.vocab = 151936; c.n_layers = 5; c.n_feat_layers = 5; c.block = 16; c.window = 256;
  c.summary = 16; c.dtype = LDR_BF16; c.rope_theta = 1e6f; c.ntk_alpha = 1.f; c.rms_eps = 1e-6f;
  return c;
}

static ldr_config tiny() {
  ldr_config c = qwen3_8b();
  c.hidden = 256; c.n_q_heads = 4; c.n_kv_heads = 4; c.head_dim = 64; c.mlp = 1024;
  c.vocab = 4096; c.n_layers = 1; c.n_feat_layers = 3; c.block = 8; c.window = 64;
  c.dtype = LDR_F32;
  return c;
}

static void configs() {
  const ldr_config good[] = {qwen3_8b(), tiny()};
  for (const ldr_config& c : good) {
    EXPECT(ldr_config_check(&c) == LDR_OK);
    const size_t st = ldr_views_state_bytes(&c);
    EXPECT(st > 0 && ldr_views_stride_bytes(&c) >= st && ldr_views_stride_bytes(&c) % 256 == 0);
    size_t off[5];
    EXPECT(ldr_views_layout(&c, off) == LDR_OK);
    for (int i = 0; i < 5; ++i) EXPECT(off[i] <= st && off[i] % 256 == 0);
    for (int i = 1; i < 5; ++i) EXPECT(off[i] >= off[i - 1]);
    EXPECT(ldr_views_layout(&c, nullptr) == LDR_EINVAL);
    size_t prev = 0;
    for (int b = 1; b <= 64; b *= 2) {
      const size_t ws = ldr_workspace_bytes(&c, b);
      EXPECT(ws > prev);
      prev = ws;
      EXPECT(ldr_draft_step_sample_workspace_bytes(&c, b) >= ws);
    }
    EXPECT(ldr_workspace_bytes(&c, 0) == 0 && ldr_workspace_bytes(&c, -3) == 0);
    const int32_t n = ldr_draft_step_launches(&c, nullptr, 0);
    EXPECT(n > 0);
    // a short buffer takes only its capacity (ASan checks the bound)
    std::vector<int32_t> kinds(2);
    EXPECT(ldr_draft_step_launches(&c, kinds.data(), 2) == n);
    std::vector<int32_t> all(n);
    EXPECT(ldr_draft_step_launches(&c, all.data(), n) == n);
  }
  EXPECT(ldr_views_state_bytes(nullptr) == 0 && ldr_config_check(nullptr) == LDR_EINVAL);
  struct Bad { const char* what; void (*edit)(ldr_config&); };
  const Bad bad[] = {
      {"hidden 0", [](ldr_config& c) { c.hidden = 0; }},
      {"hidden not /64", [](ldr_config& c) { c.hidden = 4100; }},
      {"heads", [](ldr_config& c) { c.n_q_heads = 30; }},
      {"head_dim", [](ldr_config& c) { c.head_dim = 96; }},
      {"block 0", [](ldr_config& c) { c.block = 0; }},
      {"block 17", [](ldr_config& c) { c.block = 17; }},
      {"window", [](ldr_config& c) { c.window = 0; }},
      {"summary", [](ldr_config& c) { c.summary = 0; }},
      {"vocab", [](ldr_config& c) { c.vocab = -1; }},
      {"layers", [](ldr_config& c) { c.n_layers = 0; }},
      {"dtype", [](ldr_config& c) { c.dtype = (ldr_dtype)7; }},
      {"eps", [](ldr_config& c) { c.rms_eps = 0.f; }},
      {"theta nan", [](ldr_config& c) { c.rope_theta = std::strtof("nan", nullptr); }},
      {"all views dropped", [](ldr_config& c) { c.drop_views = 7; }},
      {"unknown drop bit", [](ldr_config& c) { c.drop_views = 8; }},
      {"pool slots", [](ldr_config& c) { c.pool_slots = 31; c.pool_stride[0] = 4; c.pool_stride[1] = 64; }},
      {"pool stride", [](ldr_config& c) { c.pool_slots = 32; c.pool_stride[0] = 0; c.pool_stride[1] = 64; }},
  };
  for (const Bad& b : bad) {
    ldr_config c = qwen3_8b();
    b.edit(c);
    if (ldr_config_check(&c) != LDR_EINVAL || ldr_views_state_bytes(&c) != 0 ||
        ldr_workspace_bytes(&c, 16) != 0 || ldr_draft_step_launches(&c, nullptr, 0) >= 0) {
      std::fprintf(stderr, "config not rejected: %s\n", b.what);
      ++g_fail;
    }
  }
}

static void entry_points() {
  const ldr_config c = qwen3_8b();
  alignas(256) static uint8_t host_buf[4096];
  void* fake = host_buf;                   // never dereferenced: every call below fails early
  void* mis = host_buf + 4;                // misaligned
  ldr_views* v = nullptr;
  int64_t* pos = reinterpret_cast<int64_t*>(host_buf + 256);
  // views
  EXPECT(ldr_views_init(nullptr, &c, 16, fake, pos, fake, nullptr, 0, nullptr, nullptr, nullptr,
                        nullptr) == LDR_EINVAL);
  EXPECT(ldr_views_init(&v, &c, 0, fake, pos, fake, nullptr, 0, nullptr, nullptr, nullptr,
                        nullptr) == LDR_EINVAL && v == nullptr);
  EXPECT(ldr_views_init(&v, &c, 16, nullptr, pos, fake, nullptr, 0, nullptr, nullptr, nullptr,
                        nullptr) == LDR_EINVAL);
  EXPECT(ldr_views_init(&v, &c, 16, mis, pos, fake, nullptr, 0, nullptr, nullptr, nullptr,
                        nullptr) == LDR_EINVAL);
  EXPECT(ldr_views_init(&v, &c, 16, fake, pos, nullptr, nullptr, 0, nullptr, nullptr, nullptr,
                        nullptr) == LDR_EINVAL);       // the learned summary needs G
  EXPECT(ldr_views_init(&v, &c, 16, fake, pos, fake, nullptr, -1, nullptr, nullptr, nullptr,
                        nullptr) == LDR_EINVAL);
  EXPECT(ldr_views_init(&v, &c, 16, fake, pos, fake, nullptr, 8, fake, fake, fake,
                        nullptr) == LDR_EINVAL);       // a prefix needs its row counts
  // valid arguments reach the runtime: without a device the bookkeeping
  // allocation fails and the handle is released (LeakSanitizer checks it)
  const int rc = ldr_views_init(&v, &c, 16, fake, pos, fake, nullptr, 0, nullptr, nullptr,
                                nullptr, nullptr);
  EXPECT(rc == LDR_ENOMEM || rc == LDR_EHIP || rc == LDR_OK);
  if (rc == LDR_OK) ldr_views_destroy(v);
  EXPECT(ldr_views_update(nullptr, reinterpret_cast<const int32_t*>(fake), 17, fake, fake, fake,
                          nullptr) == LDR_EINVAL);
  EXPECT(ldr_views_status(nullptr, 0, nullptr) == LDR_EINVAL);
  ldr_views_destroy(nullptr);
  // draft step
  EXPECT(ldr_draft_step(nullptr, nullptr, nullptr, nullptr, fake, 0, nullptr) == LDR_EINVAL);
  EXPECT(ldr_draft_step_sample(nullptr, nullptr, nullptr, nullptr, 1.f, 0, 0, nullptr, nullptr,
                               nullptr, fake, 0, nullptr) == LDR_EINVAL);
  EXPECT(ldr_draft_step_events(nullptr, nullptr, nullptr, nullptr, fake, 0, nullptr, 0,
                               nullptr) == LDR_EINVAL);
  // tiling
  EXPECT(ldr_tiled_bytes(0, 32) == 0 && ldr_tiled_bytes(10, 33) == 0);
  EXPECT(ldr_tiled_bytes(300, 64) == (size_t)512 * 64 * 2);
  EXPECT(ldr_tile_matrix(nullptr, 10, 64, 64, fake, 1 << 20, nullptr) == LDR_EINVAL);
  EXPECT(ldr_tile_matrix(fake, 10, 64, 32, fake, 1 << 20, nullptr) == LDR_EINVAL);  // ld < cols
  EXPECT(ldr_tile_matrix(fake, 10, 64, 64, fake, 16, nullptr) == LDR_EINVAL);        // short dst
  // sampling
  float* f = reinterpret_cast<float*>(host_buf);
  int32_t* t = reinterpret_cast<int32_t*>(host_buf + 1024);
  const size_t sws = ldr_sample_workspace_bytes(256, 151936);
  EXPECT(sws > 0 && ldr_sample_workspace_bytes(0, 5) == 0);
  EXPECT(ldr_sample(nullptr, 256, 151936, 1.f, 0, 0, 0, t, f, f, fake, sws, nullptr) == LDR_EINVAL);
  EXPECT(ldr_sample(f, 256, 151936, -1.f, 0, 0, 0, t, f, f, fake, sws, nullptr) == LDR_EINVAL);
  EXPECT(ldr_sample(f, 256, 151936, 1.f, -1, 0, 0, t, f, f, fake, sws, nullptr) == LDR_EINVAL);
  EXPECT(ldr_sample(f, 256, 151936, 1.f, 0, 0, 0, t, f, f, fake, sws - 1, nullptr) == LDR_EINVAL);
  EXPECT(ldr_sample_noalloc(f, 600000, 16, 1.f, 0, 0, 0, t, f, f, nullptr) == LDR_ESCRATCH);
  EXPECT(ldr_sample_noalloc(nullptr, 4, 16, 1.f, 0, 0, 0, t, f, f, nullptr) == LDR_EINVAL);
  const int nr = ldr_sample_noalloc(f, 4, 16, 1.f, 0, 0, 0, t, f, f, nullptr);
  EXPECT(nr == LDR_EHIP || nr == LDR_OK);           // no device: the scratch lookup fails
  EXPECT(ldr_sample_markov(f, 2, 3, 64, t, fake, fake, 7, LDR_BF16, 1.f, 0, 0, 0, t, f, f, fake,
                           1 << 20, nullptr) == LDR_EINVAL);   // rank not a multiple of 8
  EXPECT(ldr_sample_markov(f, 2, 3, 64, t, fake, fake, 8, 5, 1.f, 0, 0, 0, t, f, f, fake, 1 << 20,
                           nullptr) == LDR_EINVAL);            // dtype
  // verification
  const size_t vws = ldr_verify_workspace_bytes(16, 16, 151936);
  EXPECT(vws > 0 && ldr_verify_workspace_bytes(16, 0, 10) == 0);
  EXPECT(ldr_verify(f, f, f, t, 16, 16, 151936, 1.f, -1, 0, 0, t, t, t, fake, vws,
                    nullptr) == LDR_EINVAL);
  EXPECT(ldr_verify(f, nullptr, f, t, 16, 16, 151936, 1.f, 0, 0, 0, t, t, t, fake, vws,
                    nullptr) == LDR_EINVAL);
  EXPECT(ldr_verify(f, f, f, t, 16, 16, 151936, 1.f, 0, 0, 0, t, t, t, fake, vws - 1,
                    nullptr) == LDR_EINVAL);
  EXPECT(ldr_gumbel_fill(0, 0, 0, 0, 10, f, nullptr) == LDR_EINVAL);
  EXPECT(ldr_gumbel_fill(0, 0, 4, 1, 10, f, nullptr) == LDR_EINVAL);
  for (int code = -10; code <= 5; ++code) EXPECT(ldr_strerror(code) != nullptr);
}

int main() {
  configs();
  entry_points();
  if (g_fail) {
    std::fprintf(stderr, "%d expectation(s) failed\n", g_fail);
    return 1;
  }
  std::printf("abi checks ok\n");
  return 0;
}
