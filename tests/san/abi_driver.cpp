// Host-side paths of the C ABI under AddressSanitizer and UndefinedBehavior-
// Sanitizer: every workspace-size function over a sweep of shapes (including
// the largest accepted ones, whose byte counts near 2^63 must not overflow),
// and every entry point's argument checks, which return before any HIP call
// (so this runs without a GPU).  Prints one line per failed expectation and
// exits non-zero if there is any.
#include <math.h>
#include <stdint.h>
#include <stdio.h>

#include "triattn.h"

static int failures = 0;
#define EXPECT(cond)                                                  \
  do {                                                                \
    if (!(cond)) {                                                    \
      ++failures;                                                     \
      printf("FAIL %s:%d: %s\n", __FILE__, __LINE__, #cond);          \
    }                                                                 \
  } while (0)

// fake, 16-byte aligned, non-null addresses: every call below is invalid
// (or only sizes), so the library must return before touching them
static void* const P = (void*)0x10000;
static void* const U = (void*)0x10008;  // misaligned

int main() {
  const int64_t ns[] = {1, 2, 31, 32, 33, 255, 256, 257, 768, 1536, 4097, 8192};
  const int64_t hs[] = {1, 4, 64};
  const int64_t ds[] = {16, 32, 64};
  for (int node = 0; node < 2; ++node)
    for (int dt = 0; dt < 2; ++dt)
      for (int64_t n : ns)
        for (int64_t h : hs)
          for (int64_t d : ds) {
            size_t f = 0, b = 0, fb = 0, bb = 0;
            EXPECT(tri_attn_fwd_workspace_bytes(node, dt, n, h, d, &f) == TRIATTN_OK);
            EXPECT(tri_attn_bwd_workspace_bytes(node, dt, n, h, d, &b) == TRIATTN_OK);
            EXPECT(b >= f && f > 0);
            EXPECT(tri_attn_fwd_batched_workspace_bytes(node, dt, 3, n, h, d, &fb) ==
                   TRIATTN_OK);
            EXPECT(tri_attn_bwd_batched_workspace_bytes(node, dt, 3, n, h, d, &bb) ==
                   TRIATTN_OK);
            EXPECT(fb >= f && bb >= b);
          }
  for (int64_t n : ns) {
    size_t rf = 0, rb = 0;
    EXPECT(tri_attn_rows_fwd_workspace_bytes(TRIATTN_BF16, n, 1, 4, 32, &rf) == TRIATTN_OK);
    EXPECT(tri_attn_rows_bwd_workspace_bytes(TRIATTN_BF16, n, n, 4, 32, &rb) == TRIATTN_OK);
    EXPECT(tri_attn_rows_fwd_workspace_bytes(TRIATTN_BF16, n, n + 1, 4, 32, &rf) ==
           TRIATTN_ERR_INVALID_ARG);
  }
  size_t x = 0;
  EXPECT(tri_attn_fwd_workspace_bytes(0, TRIATTN_BF16, 8193, 4, 32, &x) ==
         TRIATTN_ERR_INVALID_ARG);
  EXPECT(tri_attn_fwd_workspace_bytes(0, TRIATTN_BF16, 8, 65, 32, &x) ==
         TRIATTN_ERR_INVALID_ARG);
  EXPECT(tri_attn_fwd_workspace_bytes(0, TRIATTN_BF16, 8, 4, 128, &x) ==
         TRIATTN_ERR_UNSUPPORTED);
  EXPECT(tri_attn_fwd_workspace_bytes(0, TRIATTN_BF16, 8, 4, 32, nullptr) ==
         TRIATTN_ERR_INVALID_ARG);
  EXPECT(tri_attn_fwd_batched_workspace_bytes(0, TRIATTN_BF16, 0, 8, 4, 32, &x) ==
         TRIATTN_ERR_INVALID_ARG);
  EXPECT(tri_attn_fwd_batched_workspace_bytes(0, TRIATTN_BF16, (int64_t)1 << 21, 8, 4, 32,
                                              &x) == TRIATTN_ERR_INVALID_ARG);

  // attention entry points: argument errors
  const float sc = 0.17677669f;
  EXPECT(tri_attn_fwd(2, 1, 16, 2, 32, sc, P, P, P, P, P, nullptr, P, (float*)P, P, 1 << 30,
                      nullptr) == TRIATTN_ERR_INVALID_ARG);
  EXPECT(tri_attn_fwd(0, 1, 16, 2, 32, NAN, P, P, P, P, P, nullptr, P, (float*)P, P, 1 << 30,
                      nullptr) == TRIATTN_ERR_INVALID_ARG);
  EXPECT(tri_attn_fwd(0, 1, 16, 2, 32, sc, U, P, P, P, P, nullptr, P, (float*)P, P, 1 << 30,
                      nullptr) == TRIATTN_ERR_INVALID_ARG);
  EXPECT(tri_attn_fwd(0, 1, 16, 2, 32, sc, P, P, P, P, P, nullptr, P, (float*)P, P, 16,
                      nullptr) == TRIATTN_ERR_WORKSPACE);
  EXPECT(tri_attn_fwd_noalloc(0, 1, 2048, 4, 32, sc, P, P, P, P, P, nullptr, P, (float*)P,
                              nullptr) == TRIATTN_ERR_TOO_LARGE);
  EXPECT(tri_attn_bwd(0, 1, 16, 2, 32, sc, P, P, P, P, P, nullptr, P, (float*)P, P, P, P, P,
                      nullptr, P, P, 1 << 30, nullptr) == TRIATTN_ERR_INVALID_ARG);
  EXPECT(tri_attn_bwd(0, 1, 16, 2, 32, sc, P, P, P, P, P, nullptr, P, (float*)P, P, P, P, P,
                      P, P, P, 16, nullptr) == TRIATTN_ERR_WORKSPACE);
  EXPECT(tri_attn_fwd_batched(0, 1, 0, 16, 2, 32, sc, P, P, P, P, P, nullptr, P, (float*)P, P,
                              1 << 30, nullptr) == TRIATTN_ERR_INVALID_ARG);
  EXPECT(tri_attn_bwd_batched(0, 1, 2, 16, 2, 32, sc, P, P, P, P, P, nullptr, P, (float*)P, P,
                              P, P, P, P, P, P, 16, nullptr) == TRIATTN_ERR_WORKSPACE);
  EXPECT(tri_attn_rows_fwd(1, 16, 0, 2, 32, sc, P, P, P, P, P, nullptr, P, (float*)P, P,
                           1 << 30, nullptr) == TRIATTN_ERR_INVALID_ARG);
  EXPECT(tri_attn_rows_bwd(1, 16, 4, 2, 32, sc, P, P, P, P, P, nullptr, P, (float*)P, P, P,
                           P, P, P, (float*)P, P, 16, nullptr) == TRIATTN_ERR_WORKSPACE);

  // fused layer-norm + linear and transition layer: sizes and argument errors
  const int64_t cols[] = {128, 128, 128, 128, 4};
  void* outs[5] = {P, P, P, P, P};
  const void* douts[5] = {P, P, P, P, P};
  for (int64_t m : {(int64_t)1, (int64_t)37, (int64_t)589824}) {
    EXPECT(tri_ln_linear_bwd_workspace_bytes(TRIATTN_BF16, m, 128, 5, cols, &x) == TRIATTN_OK);
    EXPECT(tri_transition_fwd_workspace_bytes(TRIATTN_BF16, m, 128, 512, &x) == TRIATTN_OK);
    EXPECT(tri_transition_bwd_workspace_bytes(TRIATTN_BF16, m, 128, 512, &x) == TRIATTN_OK);
  }
  const int64_t bad_cols[] = {128, 3};
  EXPECT(tri_ln_linear_fwd(TRIATTN_BF16, 10, 128, 2, bad_cols, 1e-5f, P, P, P, P, outs,
                           (float*)P, (float*)P, nullptr) != TRIATTN_OK);
  EXPECT(tri_ln_linear_fwd(TRIATTN_BF16, 10, 64, 5, cols, 1e-5f, P, P, P, P, outs, (float*)P,
                           (float*)P, nullptr) != TRIATTN_OK);
  EXPECT(tri_ln_linear_bwd(TRIATTN_BF16, 10, 128, 5, cols, P, P, P, P, (float*)P, (float*)P,
                           douts, P, (float*)P, (float*)P, (float*)P, P, 16, nullptr) ==
         TRIATTN_ERR_WORKSPACE);
  EXPECT(tri_transition_fwd(TRIATTN_BF16, 10, 128, 100, 1e-5f, P, P, P, P, P, P, (float*)P,
                            (float*)P, P, 1 << 30, nullptr) != TRIATTN_OK);
  EXPECT(tri_transition_bwd(TRIATTN_F32, 10, 128, 512, P, P, P, P, P, (float*)P, (float*)P, P,
                            P, (float*)P, (float*)P, (float*)P, (float*)P, P, 1 << 30,
                            nullptr) == TRIATTN_ERR_UNSUPPORTED);
  EXPECT(tri_attn_mfma_probe(0, 1, (float*)P, nullptr) == TRIATTN_ERR_INVALID_ARG);
  for (int s = -1; s < 7; ++s) EXPECT(tri_attn_status_string(s) != nullptr);

  printf("abi driver: %d failures\n", failures);
  return failures == 0 ? 0 : 1;
}
