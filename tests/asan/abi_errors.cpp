// The C ABI's host-side paths under the address and undefined-behaviour
// sanitizers: every entry point with invalid arguments (each must return its
// error code and a message, touching no device memory), the host-only helpers
// with valid and edge-case arguments, and the launch-failure path (the
// launchers are stubs that fail).  Fake device pointers are never
// dereferenced.  Exit status 0 when every check holds.
#include <math.h>
#include <stdio.h>
#include <string.h>

#include "../../include/sparstar.h"
#include "../../paper_2608_10519_amd/csrc/host_internal.h"

static int failures = 0, passes = 0;

#define EXPECT(call, code, substr)                                                                      \
  do {                                                                                                  \
    const long long rc_ = (long long)(call);                                                            \
    const char* m_ = sparstar_last_error();                                                             \
    if (rc_ != (long long)(code) || strstr(m_, substr) == nullptr) {                                    \
      fprintf(stderr, "FAIL line %d: rc %lld (want %d), message '%s' (want '%s')\n", __LINE__, rc_,     \
              (int)(code), m_, substr);                                                                 \
      ++failures;                                                                                       \
    } else {                                                                                            \
      ++passes;                                                                                         \
    }                                                                                                   \
  } while (0)

#define CHECK(cond)                                                   \
  do {                                                                \
    if (!(cond)) {                                                    \
      fprintf(stderr, "FAIL line %d: %s\n", __LINE__, #cond);         \
      ++failures;                                                     \
    } else {                                                          \
      ++passes;                                                       \
    }                                                                 \
  } while (0)

static void* const F = (void*)0x10000;  // 256-byte aligned, never dereferenced
static int32_t* const FI = (int32_t*)0x20000;
static float* const FF = (float*)0x30000;

static int score(const void* q, int B, int H, int64_t Lq, int64_t Lk, int D, int b, const double* bud, int nb,
                 const sparstar_range* keep, int nkeep, int stride, void* ws, size_t ws_bytes) {
  return sparstar_score_blocks(q, F, B, H, Lq, Lk, D, b, bud, nb, keep, nkeep, FI, FI, stride, nullptr, ws,
                               ws_bytes, nullptr);
}

int main() {
  const double r25[1] = {0.25}, r15[1] = {1.5}, rneg[1] = {-0.1}, rnan[1] = {NAN}, r3[3] = {0.1, 0.2, 0.3};
  const sparstar_range text[1] = {{128, 256}}, bad[1] = {{600, 500}}, past[1] = {{0, 2000}};
  sparstar_range nine[9];
  for (int i = 0; i < 9; ++i) nine[i] = sparstar_range{0, 1};
  const size_t big = size_t(1) << 40;

  // selector
  EXPECT(score(F, 1, 2, 512, 1152, 96, 64, r25, 1, text, 1, 6, F, big), SPARSTAR_ERR_UNSUPPORTED, "head dim");
  EXPECT(score(F, 1, 2, 512, 1152, 64, 96, r25, 1, text, 1, 6, F, big), SPARSTAR_ERR_UNSUPPORTED, "block size");
  EXPECT(score(F, 0, 2, 512, 1152, 64, 64, r25, 1, text, 1, 6, F, big), SPARSTAR_ERR_INVALID_ARG, "B and H");
  EXPECT(score(F, 1, 300, 512, 1152, 64, 64, r25, 1, text, 1, 6, F, big), SPARSTAR_ERR_UNSUPPORTED, "H must");
  EXPECT(score(F, 1, 2, -1, 1152, 64, 64, r25, 1, text, 1, 6, F, big), SPARSTAR_ERR_INVALID_ARG, "Lq");
  EXPECT(score(F, 1, 2, 512, 0, 64, 64, r25, 1, text, 1, 6, F, big), SPARSTAR_ERR_INVALID_ARG, "Lk");
  EXPECT(score(F, 1, 2, int64_t(1) << 31, 1152, 64, 64, r25, 1, text, 1, 6, F, big), SPARSTAR_ERR_INVALID_ARG,
         "2^30");
  EXPECT(score(F, 1, 2, 512, 1152, 64, 64, r15, 1, text, 1, 6, F, big), SPARSTAR_ERR_INVALID_ARG, "outside [0, 1]");
  EXPECT(score(F, 1, 2, 512, 1152, 64, 64, rneg, 1, text, 1, 6, F, big), SPARSTAR_ERR_INVALID_ARG, "outside");
  EXPECT(score(F, 1, 2, 512, 1152, 64, 64, rnan, 1, text, 1, 6, F, big), SPARSTAR_ERR_INVALID_ARG, "outside");
  EXPECT(score(F, 1, 2, 512, 1152, 64, 64, nullptr, 1, text, 1, 6, F, big), SPARSTAR_ERR_INVALID_ARG, "budget");
  EXPECT(score(F, 1, 2, 512, 1152, 64, 64, r3, 3, text, 1, 6, F, big), SPARSTAR_ERR_INVALID_ARG, "n_budget");
  EXPECT(score(F, 1, 2, 512, 1152, 64, 64, r25, 1, bad, 1, 6, F, big), SPARSTAR_ERR_INVALID_ARG, "keep[0]");
  EXPECT(score(F, 1, 2, 512, 1152, 64, 64, r25, 1, past, 1, 6, F, big), SPARSTAR_ERR_INVALID_ARG, "keep[0]");
  EXPECT(score(F, 1, 2, 512, 1152, 64, 64, r25, 1, nine, 9, 6, F, big), SPARSTAR_ERR_INVALID_ARG, "n_keep");
  EXPECT(score(F, 1, 2, 512, 1152, 64, 64, r25, 1, nullptr, 2, 6, F, big), SPARSTAR_ERR_INVALID_ARG, "keep is null");
  EXPECT(score(F, 1, 2, 512, 1152, 64, 64, r25, 1, text, 1, 5, F, big), SPARSTAR_ERR_INVALID_ARG, "kv_stride");
  EXPECT(score(F, 1, 2, 512, 1152, 64, 64, r25, 1, text, 1, 6, nullptr, big), SPARSTAR_ERR_WORKSPACE, "null");
  EXPECT(score(F, 1, 2, 512, 1152, 64, 64, r25, 1, text, 1, 6, (char*)F + 16, big), SPARSTAR_ERR_WORKSPACE,
         "256-byte");
  EXPECT(score(F, 1, 2, 512, 1152, 64, 64, r25, 1, text, 1, 6, F, 100), SPARSTAR_ERR_WORKSPACE, "required");
  EXPECT(score((char*)F + 2, 1, 2, 512, 1152, 64, 64, r25, 1, text, 1, 6, F, big), SPARSTAR_ERR_INVALID_ARG,
         "16-byte");
  // valid arguments reach the (failing) launcher
  EXPECT(score(F, 1, 2, 512, 1152, 64, 64, r25, 1, text, 1, 6, F, big), SPARSTAR_ERR_HIP, "pool launch");
  // an empty query side is a no-op
  EXPECT(score(F, 1, 2, 0, 1152, 64, 64, r25, 1, text, 1, 6, F, big), SPARSTAR_OK, "");
  EXPECT(sparstar_score_blocks_fused(F, F, 1, 2, 512, 64 * SPARSTAR_FUSED_MAX_BLOCKS + 1, 64, 64, r25, 1, text, 1,
                                     FI, FI, 1000, F, big, nullptr),
         SPARSTAR_ERR_UNSUPPORTED, "at most");
  // the static-scratch selector's checks, validate-only (no HIP call)
  const sparstar_range t720[1] = {{72000, 72512}};
  EXPECT(sparstar::score_blocks_internal(F, F, 1, 24, 72000, 144512, 128, 64, r25, 1, t720, 1, FI, FI, 571, FF,
                                         nullptr, SPARSTAR_STATIC_SCRATCH_BYTES, nullptr, true),
         SPARSTAR_OK, "");
  EXPECT(sparstar::score_blocks_internal(F, F, 1, 24, 72000, 144512, 128, 64, r25, 1, t720, 1, FI, FI, 571, nullptr,
                                         nullptr, SPARSTAR_STATIC_SCRATCH_BYTES, nullptr, true),
         SPARSTAR_ERR_WORKSPACE, "required");

  // attention
  EXPECT(sparstar_sparse_attn_fwd(F, F, F, 1, 2, 512, 1152, 96, 64, FI, FI, 6, 0.f, F, FF, nullptr, 0, nullptr),
         SPARSTAR_ERR_UNSUPPORTED, "head dim");
  EXPECT(sparstar_sparse_attn_fwd(nullptr, F, F, 1, 2, 512, 1152, 64, 64, FI, FI, 6, 0.f, F, FF, nullptr, 0,
                                  nullptr),
         SPARSTAR_ERR_INVALID_ARG, "non-null");
  EXPECT(sparstar_sparse_attn_fwd(F, F, F, 1, 2, 512, 1152, 64, 64, nullptr, FI, 6, 0.f, F, FF, nullptr, 0, nullptr),
         SPARSTAR_ERR_INVALID_ARG, "kv_num_blocks");
  EXPECT(sparstar_sparse_attn_fwd(F, F, F, 1, 2, 512, 1152, 64, 64, FI, FI, 0, 0.f, F, FF, nullptr, 0, nullptr),
         SPARSTAR_ERR_INVALID_ARG, "kv_stride");
  EXPECT(sparstar_sparse_attn_fwd(F, F, F, 1, 2, 512, 1152, 64, 64, FI, FI, 6, NAN, F, FF, nullptr, 0, nullptr),
         SPARSTAR_ERR_INVALID_ARG, "finite");
  EXPECT(sparstar_dense_attn_fwd(F, F, F, 1, 2, 512, 1152, 64, 64, INFINITY, F, FF, nullptr, 0, nullptr),
         SPARSTAR_ERR_INVALID_ARG, "finite");
  EXPECT(sparstar_sparse_attn_fwd(F, F, F, 1, 2, 512, 1152, 64, 64, FI, FI, 6, 0.f, F, (float*)((char*)FF + 2),
                                  nullptr, 0, nullptr),
         SPARSTAR_ERR_INVALID_ARG, "4-byte");
  EXPECT(sparstar_dense_attn_fwd(F, F, F, 1, 2, 512, 1152, 64, 64, 0.f, F, FF, (char*)F + 16, big, nullptr),
         SPARSTAR_ERR_WORKSPACE, "256-byte");
  EXPECT(sparstar_dense_attn_fwd(F, F, F, 1, 2, 512, 1152, 64, 64, 0.f, F, FF, F, 100, nullptr),
         SPARSTAR_ERR_WORKSPACE, "required");
  EXPECT(sparstar_sparse_attn_fwd(F, F, F, 1, 2, 512, 1152, 64, 64, FI, FI, 6, 0.f, F, FF, nullptr, 0, nullptr),
         SPARSTAR_ERR_HIP, "attention launch");
  EXPECT(sparstar_dense_attn_fwd(F, F, F, 1, 2, 0, 1152, 64, 64, 0.f, F, FF, nullptr, 0, nullptr), SPARSTAR_OK, "");

  // retained mass and the token-wise bound
  EXPECT(sparstar_retained_mass(FF, FF, -1, FF, nullptr), SPARSTAR_ERR_INVALID_ARG, "n must");
  EXPECT(sparstar_retained_mass(nullptr, FF, 4, FF, nullptr), SPARSTAR_ERR_INVALID_ARG, "non-null");
  EXPECT(sparstar_retained_mass(FF, FF, 0, FF, nullptr), SPARSTAR_ERR_HIP, "retained-mass launch");
  const int64_t rows[2] = {0, 700};
  EXPECT(sparstar_token_topk_mass(F, F, 1, 2, 512, 1152, 64, rows, 2, FI, FF, 0.f, FF, F, big, nullptr),
         SPARSTAR_ERR_INVALID_ARG, "outside [0, Lq");
  EXPECT(sparstar_token_topk_mass(F, F, 1, 2, 512, 1152, 64, rows, 0, FI, FF, 0.f, FF, F, big, nullptr),
         SPARSTAR_ERR_INVALID_ARG, "n_rows");
  EXPECT(sparstar_token_topk_mass(F, F, 1, 2, 512, 1152, 64, rows, 1, FI, FF, 0.f, FF, F, 10, nullptr),
         SPARSTAR_ERR_WORKSPACE, "required");
  EXPECT(sparstar_token_topk_mass(F, F, 1, 2, 512, 1152, 64, rows, 1, FI, FF, 0.f, FF, F, big, nullptr),
         SPARSTAR_ERR_HIP, "top-n mass launch");

  // host-only helpers
  CHECK(sparstar_kv_stride(24, 144512, 64, r25, 1, t720, 1) == 8 + 563);
  EXPECT(sparstar_kv_stride(24, 0, 64, r25, 1, t720, 1), SPARSTAR_ERR_INVALID_ARG, "Lk");
  EXPECT(sparstar_kv_stride(24, 144512, 96, r25, 1, t720, 1), SPARSTAR_ERR_UNSUPPORTED, "block size");
  sparstar_range out[2];
  CHECK(sparstar_clip_keep_ranges(1, sparstar_range{72000, 72512}, sparstar_range{0, 72000}, out, 2) == 2);
  CHECK(out[0].begin == 72000 && out[1].end == 72000);
  CHECK(sparstar_clip_keep_ranges(3, sparstar_range{72000, 72512}, sparstar_range{0, 72000}, out, 2) == 1);
  EXPECT(sparstar_clip_keep_ranges(0, sparstar_range{0, 1}, sparstar_range{1, 2}, out, 2), SPARSTAR_ERR_INVALID_ARG,
         "clip");
  EXPECT(sparstar_clip_keep_ranges(1, sparstar_range{0, 1}, sparstar_range{1, 2}, out, 1), SPARSTAR_ERR_INVALID_ARG,
         "room");
  const int64_t lqs[5] = {2880, 11520, 25920, 46080, 72000};
  const double fin[4] = {0.625, 0.1875, 0.1875, 0.09375};
  double rho[5];
  EXPECT(sparstar_scale_densities(lqs, 5, fin, 4, rho), SPARSTAR_OK, "");
  CHECK(rho[0] == -1.0 && rho[1] == 0.625 && rho[4] == 0.09375);
  EXPECT(sparstar_scale_densities(lqs, 3, fin, 4, rho), SPARSTAR_ERR_INVALID_ARG, "n_finest");
  const int64_t dup[2] = {100, 100};
  const double two[2] = {0.5, 0.25};
  EXPECT(sparstar_scale_densities(dup, 2, two, 2, rho), SPARSTAR_ERR_INVALID_ARG, "densities");
  EXPECT(sparstar_scale_densities(nullptr, 2, two, 2, rho), SPARSTAR_ERR_INVALID_ARG, "null");
  CHECK(sparstar_score_workspace_bytes(1, 24, 72000, 144512, 96, 64) == 0);
  CHECK(sparstar_attn_workspace_bytes(1, 2, 512, 960, 64, 64) == 0);
  CHECK(sparstar_attn_workspace_bytes(1, 24, 72000, 144512, 128, 64) > 0);
  CHECK(sparstar::score_pooled_bytes(1, 24, 72000, 144512, 128, 64) < SPARSTAR_STATIC_SCRATCH_BYTES);
  CHECK(sparstar_token_topk_workspace_bytes(1, 2, 1152, 17) == 0);

  printf("%d checks passed, %d failed\n", passes, failures);
  return failures == 0 ? 0 : 1;
}
