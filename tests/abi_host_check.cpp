// Host-side check of the C ABI's argument validation and failure paths,
// built with AddressSanitizer and UndefinedBehaviorSanitizer on the host code
// (tests/test_abi_sanitized.py).  On a machine without a GPU the create call
// fails in its first HIP call, which exercises the clean-up of a partial
// handle; every other call here must reject its arguments without touching
// device memory.
#include <cstdio>
#include <cstring>
#include "hieravg.h"
int main() {
  int fails = 0;
  auto expect = [&](bool ok, const char* what) { if (!ok) { std::printf("FAIL %s\n", what); ++fails; } };
  expect(hieravg_create(0, 1, 1, 1, 1, 0.1f, 8, 0) == nullptr, "P=0");
  expect(std::strstr(hieravg_last_error(), "P must be") != nullptr, "P msg");
  expect(hieravg_create(4, 3, 1, 1, 1, 0.1f, 8, 0) == nullptr, "S");
  expect(hieravg_create_config(nullptr) == nullptr, "null cfg");
  hieravg_config c{};
  c.P = 4; c.S = 2; c.K1 = 2; c.K2 = 2; c.B = 8; c.kind = HIERAVG_KIND_MLP; c.in_dim = 10; c.hidden = 5;
  c.classes = 3; c.n_samples = 10; c.lr = 0.1f; c.momentum = 1.5f;
  expect(hieravg_create_config(&c) == nullptr, "momentum");
  c.momentum = 0.0f;
  hieravg_t h = hieravg_create_config(&c);  // no GPU here: the create fails cleanly
  std::printf("create without device: %p (%s)\n", (void*)h, hieravg_last_error());
  if (h) hieravg_destroy(h);
  expect(hieravg_round(nullptr) == HIERAVG_EINVAL, "round null");
  expect(hieravg_params(nullptr, nullptr, 0) == HIERAVG_EINVAL, "params null");
  expect(hieravg_check_finite(nullptr) == HIERAVG_EINVAL, "finite null");
  expect(hieravg_set_step_count(nullptr, 1) == HIERAVG_EINVAL, "step null");
  double loss = 0.0;
  int64_t hits = 0;
  expect(hieravg_evaluate_noalloc(nullptr, 0, 0, 1, &loss, &hits) == HIERAVG_EINVAL, "evaluate_noalloc null");
  expect(std::strcmp(hieravg_kernel_class_name(-1), "") == 0, "class -1");
  expect(std::strcmp(hieravg_kernel_class_name(hieravg_kernel_classes()), "") == 0, "class n");
  hieravg_destroy(nullptr);
  std::printf("%s\n", fails ? "host checks FAILED" : "host checks ok");
  return fails != 0;
}
