// Host-only driver for the C-ABI argument validation (tv_abi.cpp), built with
// AddressSanitizer and UndefinedBehaviorSanitizer by tests/test_abi_sanitize.py.
// The launchers are replaced by stubs that record the call, so no GPU is
// touched: every entry point is called with valid and invalid arguments and
// its return code and launch decision are checked.
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include "tv.h"
#include "tv_launch.h"

static int g_launches = 0;

namespace tv {
int launch(const VerifyArgs&, Algo, void*, hipStream_t) { ++g_launches; return TV_OK; }
int launch_sample(const SampleArgs&, hipStream_t) { ++g_launches; return TV_OK; }
int launch_commit(const CommitArgs&, hipStream_t) { ++g_launches; return TV_OK; }
int launch_lmhead(const LmheadArgs&, void*, hipStream_t) { ++g_launches; return TV_OK; }
int static_scratch(void** ptr, size_t* bytes) {
  static unsigned char fake[256] __attribute__((aligned(256)));
  *ptr = fake;
  *bytes = kStaticScratchBytes;
  return TV_OK;
}
}  // namespace tv

static int failures = 0;
#define EXPECT(cond)                                                      \
  do {                                                                    \
    if (!(cond)) {                                                        \
      fprintf(stderr, "%s:%d: expected %s\n", __FILE__, __LINE__, #cond); \
      ++failures;                                                         \
    }                                                                     \
  } while (0)

int main() {
  // fake, never dereferenced device addresses (aligned as the ABI requires)
  const uintptr_t A = 0x10000, WS = 0x40000000;
  int32_t* ip = reinterpret_cast<int32_t*>(A);
  float* fp = reinterpret_cast<float*>(A);
  const void* tgt = reinterpret_cast<const void*>(A);
  const void* drf = reinterpret_cast<const void*>(A + 0x1000);
  void* ws = reinterpret_cast<void*>(WS);
  const size_t wsb = tv_workspace_size(2, 5, 100);
  EXPECT(wsb > 0 && wsb % 256 == 0);
  EXPECT(tv_workspace_size(0, 5, 100) == 0);
  EXPECT(tv_workspace_size(TV_MAX_BATCH + 1, 5, 100) == 0);
  EXPECT(tv_workspace_size(TV_MAX_BATCH, TV_MAX_NODES, TV_MAX_VOCAB) <= tv::kStaticScratchBytes);

  auto verify = [&](int32_t batch, int32_t n1, int32_t V, int32_t dtype, float T, int32_t mode,
                    const void* t, const void* d, void* w, size_t wb, int32_t* parents) {
    return tv_verify(batch, n1, V, parents, ip, t, d, dtype, T, fp, mode, ip, ip, ip, ip,
                     nullptr, nullptr, nullptr, nullptr, w, wb, nullptr);
  };
  int before = g_launches;
  EXPECT(verify(2, 5, 100, TV_DTYPE_BF16, 1.0f, 0, tgt, drf, ws, wsb, ip) == TV_OK);
  EXPECT(g_launches == before + 1);
  before = g_launches;
  EXPECT(verify(-1, 5, 100, TV_DTYPE_BF16, 1.0f, 0, tgt, drf, ws, wsb, ip) == TV_ERR_INVALID_ARG);
  EXPECT(verify(2, 0, 100, TV_DTYPE_BF16, 1.0f, 0, tgt, drf, ws, wsb, ip) == TV_ERR_INVALID_ARG);
  EXPECT(verify(2, 5, 1, TV_DTYPE_BF16, 1.0f, 0, tgt, drf, ws, wsb, ip) == TV_ERR_INVALID_ARG);
  EXPECT(verify(2, 5, 100, 9, 1.0f, 0, tgt, drf, ws, wsb, ip) == TV_ERR_INVALID_ARG);
  EXPECT(verify(2, 5, 100, TV_DTYPE_BF16, 1.0f, 5, tgt, drf, ws, wsb, ip) == TV_ERR_INVALID_ARG);
  EXPECT(verify(2, 5, 100, TV_DTYPE_BF16, NAN, 0, tgt, drf, ws, wsb, ip) == TV_ERR_INVALID_ARG);
  EXPECT(verify(2, 5, 100, TV_DTYPE_BF16, INFINITY, 0, tgt, drf, ws, wsb, ip) == TV_ERR_INVALID_ARG);
  EXPECT(verify(2, 5, 100, TV_DTYPE_BF16, 1e-5f, 0, tgt, drf, ws, wsb, ip) == TV_ERR_UNSUPPORTED);
  EXPECT(verify(TV_MAX_BATCH + 1, 5, 100, TV_DTYPE_BF16, 1.0f, 0, tgt, drf, ws, wsb, ip) ==
         TV_ERR_UNSUPPORTED);
  EXPECT(verify(2, TV_MAX_NODES + 1, 100, TV_DTYPE_BF16, 1.0f, 0, tgt, drf, ws, wsb, ip) ==
         TV_ERR_UNSUPPORTED);
  EXPECT(verify(2, 5, TV_MAX_VOCAB_F32 + 1, TV_DTYPE_F32, 1.0f, 0, tgt, drf, ws, wsb, ip) ==
         TV_ERR_UNSUPPORTED);
  EXPECT(verify(2, 5, 100, TV_DTYPE_BF16, 1.0f, 0, nullptr, drf, ws, wsb, ip) == TV_ERR_INVALID_ARG);
  EXPECT(verify(2, 5, 100, TV_DTYPE_BF16, 1.0f, 0, tgt, drf, ws, wsb, nullptr) == TV_ERR_INVALID_ARG);
  EXPECT(verify(2, 5, 100, TV_DTYPE_BF16, 1.0f, 0, reinterpret_cast<const void*>(A + 1),
                reinterpret_cast<const void*>(A + 1), ws, wsb, ip) == TV_ERR_INVALID_ARG);
  EXPECT(verify(2, 5, 100, TV_DTYPE_BF16, 1.0f, 0, reinterpret_cast<const void*>(A + 2),
                reinterpret_cast<const void*>(A + 4), ws, wsb, ip) == TV_ERR_UNSUPPORTED);
  EXPECT(verify(2, 5, 100, TV_DTYPE_BF16, 1.0f, 0, tgt, drf, nullptr, wsb, ip) == TV_ERR_WORKSPACE);
  EXPECT(verify(2, 5, 100, TV_DTYPE_BF16, 1.0f, 0, tgt, drf,
                reinterpret_cast<void*>(WS + 128), wsb, ip) == TV_ERR_WORKSPACE);
  EXPECT(verify(2, 5, 100, TV_DTYPE_BF16, 1.0f, 0, tgt, drf, ws, 256, ip) == TV_ERR_WORKSPACE);
  EXPECT(g_launches == before);           // no argument error reaches a launcher
  EXPECT(verify(0, 5, 100, TV_DTYPE_BF16, 1.0f, 0, nullptr, nullptr, nullptr, 0, nullptr) == TV_OK);
  EXPECT(g_launches == before);           // an empty batch launches nothing

  before = g_launches;
  EXPECT(tv_verify_noalloc(2, 5, 100, ip, ip, tgt, drf, TV_DTYPE_BF16, 1.0f, fp, 0, ip, ip, ip, ip,
                           nullptr, nullptr, nullptr, nullptr, nullptr) == TV_OK);
  EXPECT(tv_verify_noalloc(2, 5, 100, nullptr, ip, tgt, drf, TV_DTYPE_BF16, 1.0f, fp, 0, ip, ip, ip,
                           ip, nullptr, nullptr, nullptr, nullptr, nullptr) == TV_ERR_INVALID_ARG);
  EXPECT(g_launches == before + 1);

  before = g_launches;
  EXPECT(tv_draft_tokens(2, 5, 100, ip, drf, TV_DTYPE_BF16, 1.0f, fp, 0, ip, ip, nullptr) == TV_OK);
  EXPECT(tv_draft_tokens(2, 5, 100, ip, reinterpret_cast<const void*>(A + 1), TV_DTYPE_BF16, 1.0f,
                         fp, 0, ip, ip, nullptr) == TV_ERR_INVALID_ARG);
  EXPECT(tv_draft_tokens(2, 5, 100, ip, drf, TV_DTYPE_BF16, 0.0f, fp, 0, ip, ip, nullptr) ==
         TV_ERR_INVALID_ARG);
  EXPECT(g_launches == before + 1);

  before = g_launches;
  EXPECT(tv_commit_paths(2, 5, ip, ip, ip, ip, ip, 4, ip, ip, ip, nullptr) == TV_OK);
  EXPECT(tv_commit_paths(2, 5, ip, ip, ip, ip, ip, -1, ip, ip, ip, nullptr) == TV_ERR_INVALID_ARG);
  EXPECT(tv_commit_paths(2, 5, ip, ip, ip, ip, ip, 4, nullptr, ip, ip, nullptr) == TV_ERR_INVALID_ARG);
  EXPECT(tv_commit_paths(2, 5, ip, ip, ip, ip, ip, 0, nullptr, ip, ip, nullptr) == TV_OK);
  EXPECT(g_launches == before + 2);

  before = g_launches;
  const float* fm = reinterpret_cast<const float*>(A);
  const double* dm = reinterpret_cast<const double*>(A);
  EXPECT(tv_verify_stats(2, 5, 100, ip, ip, tgt, drf, TV_DTYPE_BF16, 1.0f, fp, 0, fm, dm, fm, dm,
                         ip, ip, ip, ip, nullptr, nullptr, nullptr, nullptr, ws, wsb, nullptr) ==
         TV_OK);
  EXPECT(tv_verify_stats(2, 5, 100, ip, ip, tgt, drf, TV_DTYPE_BF16, 1.0f, fp, 0, nullptr, dm, fm,
                         dm, ip, ip, ip, ip, nullptr, nullptr, nullptr, nullptr, ws, wsb,
                         nullptr) == TV_ERR_INVALID_ARG);
  EXPECT(g_launches == before + 1);
  before = g_launches;
  const size_t lwb = tv_lmhead_workspace_size(4, 1000);
  EXPECT(lwb > 0 && lwb % 256 == 0);
  double* dp = reinterpret_cast<double*>(A);
  EXPECT(tv_lmhead_stats(4, 64, 1000, tgt, drf, 1.0f, reinterpret_cast<void*>(A), fp, dp, ws, lwb,
                         nullptr) == TV_OK);
  EXPECT(tv_lmhead_stats(4, 60, 1000, tgt, drf, 1.0f, reinterpret_cast<void*>(A), fp, dp, ws, lwb,
                         nullptr) == TV_ERR_UNSUPPORTED);
  EXPECT(tv_lmhead_stats(4, 64, 1000, tgt, drf, 1.0f, reinterpret_cast<void*>(A), fp, dp, ws, 16,
                         nullptr) == TV_ERR_WORKSPACE);
  EXPECT(g_launches == before + 1);

  for (int c = -3; c < 8; ++c) EXPECT(tv_status_string(c) != nullptr);
  if (failures) {
    fprintf(stderr, "%d failures\n", failures);
    return 1;
  }
  printf("abi validation: all checks passed\n");
  return 0;
}
