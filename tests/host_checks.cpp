// Host-only checks of the WINO library's C ABI, built with AddressSanitizer
// and UndefinedBehaviorSanitizer on the host code (tests/test_abi_cpu.py
// builds and runs it): every path here returns before any HIP call, so it
// runs without a GPU.  Exits non-zero on the first failed check.
#include <cmath>
#include <cstdio>
#include <cstring>
#include <cstdlib>
#include <vector>

#include "wino.h"

static int g_checks = 0;
#define CHECK(cond)                                                        \
  do {                                                                     \
    ++g_checks;                                                            \
    if (!(cond)) {                                                         \
      std::fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #cond); \
      std::exit(1);                                                        \
    }                                                                      \
  } while (0)

static wino_model_config tiny_cfg() {
  wino_model_config c{};
  c.n_layers = 2; c.d_model = 256; c.n_heads = 4; c.head_dim = 64; c.d_ff = 704; c.vocab = 4096;
  c.rope_theta = 10000.f; c.rms_eps = 1e-5f;
  return c;
}

static wino_params params(int B, int P, int G, int Lb, int mask, float t1 = 0.7f, float t2 = 0.9f) {
  wino_params p{};
  p.batch = B; p.prompt_len = P; p.gen_len = G; p.block_len = Lb; p.mask_id = mask;
  p.tau1 = t1; p.tau2 = t2;
  return p;
}

int main() {
  // sizes
  wino_model_config cfg = tiny_cfg();
  const size_t w1 = wino_workspace_bytes(&cfg, 1, 112), w2 = wino_workspace_bytes(&cfg, 2, 112);
  CHECK(w1 > 0 && w2 > w1);
  CHECK(wino_workspace_bytes(nullptr, 1, 112) == 0 && wino_workspace_bytes(&cfg, 0, 112) == 0);
  wino_model_config big = cfg;
  big.n_layers = 32; big.d_model = 4096; big.n_heads = 32; big.head_dim = 128; big.d_ff = 12288;
  big.vocab = 126464;
  CHECK(wino_workspace_bytes(&big, 16, 544) > wino_workspace_bytes(&big, 1, 544));
  CHECK(wino_epilogue_workspace_bytes(8, 32, 126464) >= (size_t)8 * 32 * 8 * 20);
  CHECK(wino_epilogue_workspace_bytes(0, 32, 126464) == 0);

  // wino_create: arguments rejected before any device work
  wino_ctx* ctx = nullptr;
  wino_weights w{};
  CHECK(wino_create(nullptr, &w, 1, 112, &ctx) == WINO_ERR_INVALID_ARG);
  CHECK(wino_create(&cfg, &w, 0, 112, &ctx) == WINO_ERR_SHAPE);
  CHECK(std::strcmp(wino_last_error(nullptr), "max_batch or max_seq") == 0);
  wino_model_config bad = cfg;
  bad.head_dim = 96; bad.d_model = 384;
  CHECK(wino_create(&bad, &w, 1, 112, &ctx) == WINO_ERR_UNSUPPORTED);
  bad = cfg; bad.vocab = 4000;
  CHECK(wino_create(&bad, &w, 1, 112, &ctx) == WINO_ERR_UNSUPPORTED);
  bad = cfg; bad.rms_eps = NAN;
  CHECK(wino_create(&bad, &w, 1, 112, &ctx) == WINO_ERR_UNSUPPORTED);
  bad = cfg; bad.act_precision = 2;
  CHECK(wino_create(&bad, &w, 1, 112, &ctx) == WINO_ERR_UNSUPPORTED);
  CHECK(wino_create(&cfg, &w, 1, 112, &ctx) == WINO_ERR_INVALID_ARG);  // null weights
  CHECK(ctx == nullptr);

  // the workspace limit, with placeholder (never dereferenced) weight pointers
  std::vector<const void*> layer(cfg.n_layers, reinterpret_cast<const void*>(0x1000));
  const void* ph = reinterpret_cast<const void*>(0x1000);
  wino_weights fake{ph, layer.data(), layer.data(), layer.data(), layer.data(), layer.data(), layer.data(),
                    ph, ph, nullptr};
  char lim[64];
  std::snprintf(lim, sizeof lim, "%zu", w2 - 1);
  setenv("WINO_WORKSPACE_LIMIT", lim, 1);
  CHECK(wino_create(&cfg, &fake, 2, 112, &ctx) == WINO_ERR_NO_MEMORY && ctx == nullptr);
  setenv("WINO_WORKSPACE_LIMIT", "0", 1);
  CHECK(wino_create(&cfg, &fake, 1, 112, &ctx) == WINO_ERR_NO_MEMORY && ctx == nullptr);
  unsetenv("WINO_WORKSPACE_LIMIT");

  // entry points without a context
  wino_params p = params(1, 32, 64, 16, 4095);
  CHECK(wino_step(nullptr, &p, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr) ==
        WINO_ERR_INVALID_ARG);
  CHECK(wino_decode(nullptr, &p, nullptr, nullptr, nullptr, nullptr, 0, nullptr, nullptr, nullptr) ==
        WINO_ERR_INVALID_ARG);
  CHECK(wino_decode_block(nullptr, &p, nullptr, nullptr, nullptr, nullptr, nullptr) == WINO_ERR_INVALID_ARG);
  CHECK(wino_row_losses(nullptr, &p, nullptr, nullptr, nullptr, nullptr) == WINO_ERR_INVALID_ARG);
  CHECK(wino_debug_logits(nullptr, &p, nullptr, nullptr, nullptr, nullptr) == WINO_ERR_INVALID_ARG);
  CHECK(wino_debug_forward(nullptr, &p, nullptr, nullptr, 0, nullptr, nullptr) == WINO_ERR_INVALID_ARG);
  CHECK(wino_destroy(nullptr) == WINO_ERR_INVALID_ARG);
  CHECK(wino_profile(nullptr, 1) == WINO_ERR_INVALID_ARG);
  CHECK(wino_profile_read(nullptr, nullptr, nullptr, nullptr, nullptr) == WINO_ERR_INVALID_ARG);

  // standalone epilogue: host-side validation (placeholder device pointers)
  void* d = reinterpret_cast<void*>(0x1000);
  int32_t* di = reinterpret_cast<int32_t*>(0x1000);
  uint8_t* du = reinterpret_cast<uint8_t*>(0x1000);
  wino_params e = params(1, 0, 16, 16, 4095, NAN, 0.9f);
  CHECK(wino_epilogue(&e, 4096, d, di, du, nullptr, nullptr, d, 1 << 20, nullptr) == WINO_ERR_INVALID_ARG);
  e = params(1, 0, 16, 16, 5000);
  CHECK(wino_epilogue(&e, 4096, d, di, du, nullptr, nullptr, d, 1 << 20, nullptr) == WINO_ERR_INVALID_ARG);
  e = params(1, 0, 16, 16, 4095);
  CHECK(wino_epilogue(&e, 4100, d, di, du, nullptr, nullptr, d, 1 << 20, nullptr) == WINO_ERR_SHAPE);
  CHECK(wino_epilogue(&e, 4096, d, di, du, nullptr, nullptr, d, 16, nullptr) == WINO_ERR_SHAPE);
  CHECK(wino_epilogue(&e, 4096, nullptr, di, du, nullptr, nullptr, d, 1 << 20, nullptr) == WINO_ERR_INVALID_ARG);
  CHECK(wino_epilogue(&e, 4096, d, di, du, nullptr, nullptr, nullptr, 1 << 20, nullptr) == WINO_ERR_INVALID_ARG);
  e.tokens_per_step = -1;
  CHECK(wino_epilogue_noalloc(&e, 4096, d, di, du, nullptr, nullptr, nullptr) == WINO_ERR_INVALID_ARG);
  e = params(128, 0, 128, 128, 126463);
  CHECK(wino_epilogue_workspace_bytes(128, 128, 126464) > WINO_EPILOGUE_NOALLOC_MAX_BYTES);
  CHECK(wino_epilogue_noalloc(&e, 126464, d, di, du, nullptr, nullptr, nullptr) == WINO_ERR_SHAPE);

  // GEMM test entry point: the tile planner rejects shapes without a kernel
  CHECK(wino_debug_gemm(nullptr, d, 64, 128, 64, nullptr, nullptr) == WINO_ERR_INVALID_ARG);
  CHECK(wino_debug_gemm(d, d, 0, 128, 64, reinterpret_cast<float*>(d), nullptr) == WINO_ERR_SHAPE);
  CHECK(wino_debug_gemm(d, d, 64, 128, 40, reinterpret_cast<float*>(d), nullptr) == WINO_ERR_UNSUPPORTED);
  CHECK(wino_debug_gemm(d, d, 64, 100, 64, reinterpret_cast<float*>(d), nullptr) == WINO_ERR_UNSUPPORTED);

  // strings
  for (int s = -7; s <= 0; ++s) CHECK(wino_status_string(static_cast<wino_status>(s)) != nullptr);
  CHECK(wino_kernel_class_name(-1)[0] == 0 && wino_kernel_class_name(WINO_N_KERNEL_CLASSES)[0] == 0);
  for (int k = 0; k < WINO_N_KERNEL_CLASSES; ++k) CHECK(wino_kernel_class_name(k)[0] != 0);
  // the last failed wino_create on this thread (the workspace-limit case above)
  CHECK(std::strcmp(wino_last_error(nullptr), "workspace larger than WINO_WORKSPACE_LIMIT") == 0);

  std::printf("host checks ok: %d\n", g_checks);
  return 0;
}
