// Host-side driver for the AddressSanitizer check of the C ABI (no GPU needed).
//
// It exercises every host path of the library that runs before device work:
// descriptor validation, the shape set, workspace sizing (frequency groups,
// padded groups, value-width padding, segment and sub-segment heuristics) and
// the argument checks of every entry point.  Each entry-point call is given at
// least one invalid argument, so no call reaches a kernel launch.  Built with
// -fsanitize=address on the host side only; prints "ok" and exits 0 when every
// status is as expected.
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <initializer_list>

#include "flex.h"

namespace {

int fails = 0;

void expect(int got, int want, const char* what, int line) {
  if (got != want) {
    std::printf("FAIL line %d %s: status %d, expected %d\n", line, what, got, want);
    ++fails;
  }
}
#define EXPECT(call, want) expect((call), (want), #call, __LINE__)

flex_desc make(int B, int H, int N, int d, int dv, int m, int variant, int causal, int io) {
  flex_desc x;
  std::memset(&x, 0, sizeof(x));
  x.B = B; x.H = H; x.N = N; x.d = d; x.dv = dv; x.m = m;
  x.variant = variant; x.causal = causal; x.chunk = 0; x.segments = 0;
  x.io_dtype = io; x.grad_dtype = FLEX_F32; x.sigma = 1.0f;
  return x;
}

}  // namespace

int main() {
  size_t bytes = 0;
  // the shape set: every d, dv, m a multiple of 16 up to 256, both variants,
  // causal or not, several N (ragged, one chunk, many segments)
  const int widths[] = {32, 64, 128};
  const int lengths[] = {1, 17, 64, 65, 1000, 70000};
  for (int d : widths)
    for (int dv : widths)
      for (int m = 16; m <= 256; m += 16)
        for (int variant = 0; variant < 2; ++variant)
          for (int causal = 0; causal < 2; ++causal)
            for (int N : lengths) {
              flex_desc x = make(2, 3, N, d, dv, m, variant, causal, FLEX_BF16);
              EXPECT(flex_workspace_size(&x, FLEX_PASS_FWD, &bytes), FLEX_OK);
              EXPECT(flex_workspace_size(&x, FLEX_PASS_BWD, &bytes), FLEX_OK);
              EXPECT(flex_workspace_size(&x, FLEX_PASS_FEATURE_MAP, &bytes), FLEX_OK);
              for (int seg : {1, 3, 256, 5000}) {
                x.segments = seg;
                EXPECT(flex_workspace_size(&x, FLEX_PASS_BWD, &bytes), FLEX_OK);
              }
              for (int chunk : {16, 32, 64}) {
                x.segments = 0;
                x.chunk = chunk;
                EXPECT(flex_workspace_size(&x, FLEX_PASS_FWD, &bytes), FLEX_OK);
              }
            }
  // fp32 shapes
  for (int m = 16; m <= 256; m += 16) {
    flex_desc x = make(1, 2, 300, 32, 32, m, FLEX_NONSTATIONARY, 1, FLEX_F32);
    EXPECT(flex_workspace_size(&x, FLEX_PASS_BWD, &bytes), FLEX_OK);
    x.dv = 64;
    EXPECT(flex_workspace_size(&x, FLEX_PASS_FWD, &bytes), FLEX_ERR_UNSUPPORTED);
  }
  // invalid and unsupported descriptors
  {
    flex_desc x = make(1, 2, 100, 64, 64, 128, FLEX_NONSTATIONARY, 1, FLEX_BF16);
    flex_desc y;
    y = x; y.B = 0;            EXPECT(flex_workspace_size(&y, FLEX_PASS_FWD, &bytes), FLEX_ERR_INVALID_ARG);
    y = x; y.N = -5;           EXPECT(flex_workspace_size(&y, FLEX_PASS_FWD, &bytes), FLEX_ERR_INVALID_ARG);
    y = x; y.m = 0;            EXPECT(flex_workspace_size(&y, FLEX_PASS_FWD, &bytes), FLEX_ERR_INVALID_ARG);
    y = x; y.m = 272;          EXPECT(flex_workspace_size(&y, FLEX_PASS_FWD, &bytes), FLEX_ERR_UNSUPPORTED);
    y = x; y.m = 100;          EXPECT(flex_workspace_size(&y, FLEX_PASS_FWD, &bytes), FLEX_ERR_UNSUPPORTED);
    y = x; y.d = 48;           EXPECT(flex_workspace_size(&y, FLEX_PASS_FWD, &bytes), FLEX_ERR_UNSUPPORTED);
    y = x; y.dv = 96;          EXPECT(flex_workspace_size(&y, FLEX_PASS_FWD, &bytes), FLEX_ERR_UNSUPPORTED);
    y = x; y.chunk = 48;       EXPECT(flex_workspace_size(&y, FLEX_PASS_FWD, &bytes), FLEX_ERR_UNSUPPORTED);
    y = x; y.chunk = -16;      EXPECT(flex_workspace_size(&y, FLEX_PASS_FWD, &bytes), FLEX_ERR_INVALID_ARG);
    y = x; y.segments = -1;    EXPECT(flex_workspace_size(&y, FLEX_PASS_FWD, &bytes), FLEX_ERR_INVALID_ARG);
    y = x; y.variant = 7;      EXPECT(flex_workspace_size(&y, FLEX_PASS_FWD, &bytes), FLEX_ERR_INVALID_ARG);
    y = x; y.causal = 2;       EXPECT(flex_workspace_size(&y, FLEX_PASS_FWD, &bytes), FLEX_ERR_INVALID_ARG);
    y = x; y.io_dtype = 9;     EXPECT(flex_workspace_size(&y, FLEX_PASS_FWD, &bytes), FLEX_ERR_INVALID_ARG);
    y = x; y.grad_dtype = 1;   EXPECT(flex_workspace_size(&y, FLEX_PASS_BWD, &bytes), FLEX_ERR_UNSUPPORTED);
    y = x; y.sigma = 0.0f;     EXPECT(flex_workspace_size(&y, FLEX_PASS_FWD, &bytes), FLEX_ERR_INVALID_ARG);
    y = x; y.B = 1 << 20; y.H = 1 << 20;
    EXPECT(flex_workspace_size(&y, FLEX_PASS_FWD, &bytes), FLEX_ERR_INVALID_ARG);
    EXPECT(flex_workspace_size(nullptr, FLEX_PASS_FWD, &bytes), FLEX_ERR_INVALID_ARG);
    EXPECT(flex_workspace_size(&x, 17, &bytes), FLEX_ERR_INVALID_ARG);
    EXPECT(flex_workspace_size(&x, FLEX_PASS_FWD, nullptr), FLEX_ERR_INVALID_ARG);
    // the distillation loss: non-causal, its own shapes
    y = x; y.causal = 0;       EXPECT(flex_workspace_size(&y, FLEX_PASS_AWD, &bytes), FLEX_OK);
    y = x;                     EXPECT(flex_workspace_size(&y, FLEX_PASS_AWD, &bytes), FLEX_ERR_UNSUPPORTED);
  }
  // entry points: each call has at least one invalid argument (NULL, misaligned,
  // variant mismatch or a workspace too small), so none reaches the device
  {
    flex_desc x = make(1, 2, 100, 64, 32, 128, FLEX_NONSTATIONARY, 1, FLEX_BF16);
    flex_desc s = x; s.variant = FLEX_STATIONARY;
    void* P = reinterpret_cast<void*>(uintptr_t(0x10000));
    float* Pf = static_cast<float*>(P);
    void* mis = reinterpret_cast<void*>(uintptr_t(0x10002));
    const size_t big = size_t(1) << 40;
    EXPECT(flex_linattn_fwd(nullptr, P, P, P, Pf, Pf, Pf, P, Pf, P, big, nullptr), FLEX_ERR_INVALID_ARG);
    EXPECT(flex_linattn_fwd(&x, nullptr, P, P, Pf, Pf, Pf, P, Pf, P, big, nullptr), FLEX_ERR_INVALID_ARG);
    EXPECT(flex_linattn_fwd(&x, P, P, P, Pf, nullptr, Pf, P, Pf, P, big, nullptr), FLEX_ERR_INVALID_ARG);
    EXPECT(flex_linattn_fwd(&s, P, P, P, Pf, Pf, Pf, P, Pf, P, big, nullptr), FLEX_ERR_INVALID_ARG);
    EXPECT(flex_linattn_fwd(&x, mis, P, P, Pf, Pf, Pf, P, Pf, P, big, nullptr), FLEX_ERR_INVALID_ARG);
    EXPECT(flex_linattn_fwd(&x, P, P, P, Pf, Pf, Pf, P, Pf, nullptr, big, nullptr), FLEX_ERR_WORKSPACE);
    EXPECT(flex_linattn_fwd(&x, P, P, P, Pf, Pf, Pf, P, Pf, P, 16, nullptr), FLEX_ERR_WORKSPACE);
    EXPECT(flex_linattn_prefill(&x, P, P, P, Pf, Pf, Pf, P, Pf, nullptr, P, big, nullptr), FLEX_ERR_INVALID_ARG);
    EXPECT(flex_linattn_prefill(&x, P, P, P, Pf, Pf, Pf, P, Pf, Pf, P, 16, nullptr), FLEX_ERR_WORKSPACE);
    flex_desc nc = x; nc.causal = 0;
    EXPECT(flex_linattn_prefill(&nc, P, P, P, Pf, Pf, Pf, P, Pf, Pf, P, big, nullptr), FLEX_ERR_UNSUPPORTED);
    EXPECT(flex_linattn_fwd_noalloc(&x, nullptr, P, P, Pf, Pf, Pf, P, Pf, nullptr), FLEX_ERR_INVALID_ARG);
    flex_desc huge = make(2, 16, 8192, 128, 128, 256, FLEX_NONSTATIONARY, 1, FLEX_BF16);
    EXPECT(flex_linattn_fwd_noalloc(&huge, P, P, P, Pf, Pf, Pf, P, Pf, nullptr), FLEX_ERR_WORKSPACE);
    EXPECT(flex_linattn_bwd(&x, P, P, P, Pf, Pf, Pf, P, Pf, P, P, P, P, Pf, Pf, Pf, nullptr, 0, P, 16, nullptr),
           FLEX_ERR_WORKSPACE);
    EXPECT(flex_linattn_bwd(&x, P, P, P, Pf, Pf, Pf, P, nullptr, P, P, P, P, Pf, Pf, Pf, nullptr, 0, P, big,
                            nullptr), FLEX_ERR_INVALID_ARG);
    EXPECT(flex_linattn_bwd(&x, P, P, P, Pf, Pf, Pf, P, Pf, P, P, P, P, Pf, nullptr, Pf, nullptr, 0, P, big,
                            nullptr), FLEX_ERR_INVALID_ARG);
    EXPECT(flex_linattn_bwd(&x, P, P, P, Pf, Pf, Pf, P, Pf, P, P, P, P, Pf, Pf, Pf, P, 16, P, big, nullptr),
           FLEX_ERR_WORKSPACE);
    EXPECT(flex_feature_map(&x, nullptr, Pf, Pf, Pf, P, nullptr, 0, nullptr), FLEX_ERR_INVALID_ARG);
    EXPECT(flex_feature_map(&x, P, Pf, nullptr, Pf, P, nullptr, 0, nullptr), FLEX_ERR_INVALID_ARG);
    flex_desc dd = make(2, 3, 1, 64, 32, 128, FLEX_NONSTATIONARY, 1, FLEX_BF16);
    EXPECT(flex_decode_step(&dd, P, P, P, Pf, Pf, Pf, nullptr, P, Pf, nullptr), FLEX_ERR_INVALID_ARG);
    dd.d = 66;
    EXPECT(flex_decode_step(&dd, P, P, P, Pf, Pf, Pf, Pf, P, Pf, nullptr), FLEX_ERR_UNSUPPORTED);
    flex_desc aw = make(2, 2, 64, 64, 64, 64, FLEX_NONSTATIONARY, 0, FLEX_BF16);
    EXPECT(flex_awd_loss(&aw, P, P, Pf, Pf, Pf, Pf, Pf, Pf, Pf, P, 16, nullptr), FLEX_ERR_WORKSPACE);
    EXPECT(flex_awd_loss(&aw, P, P, Pf, nullptr, Pf, Pf, Pf, Pf, Pf, P, big, nullptr), FLEX_ERR_INVALID_ARG);
  }
  for (int st = -1; st <= 6; ++st)
    if (!flex_status_string(st)) {
      std::printf("FAIL status string %d\n", st);
      ++fails;
    }
  EXPECT(flex_abi_version(), FLEX_ABI_VERSION);
  std::printf(fails ? "FAILED %d\n" : "ok\n", fails);
  return fails ? 1 : 0;
}
