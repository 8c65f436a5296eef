// Host-side paths of the C ABI under AddressSanitizer and
// UndefinedBehaviorSanitizer: argument validation, the workspace layout of
// every supported size, operation and approximation, the float64
// transfer-function tables (the upload that follows them fails without a
// GPU), range checks of overlapping buffers and the no-allocation limit.
// Linked against host-only objects of the library; nothing is launched.
// Prints "ALL OK" when every expectation holds.
#include <hip/hip_runtime.h>

#include <climits>
#include <cstdint>
#include <cstdio>
#include <vector>

#include "../../include/lr.h"

static int g_fail = 0;
#define EXPECT(c)                                           \
  do {                                                      \
    if (!(c)) {                                             \
      std::printf("FAIL line %d: %s\n", __LINE__, #c);      \
      ++g_fail;                                             \
    }                                                       \
  } while (0)

static void* fake(uintptr_t a) { return reinterpret_cast<void*>(a); }

int main() {
  const int sizes[] = {64, 100, 128, 200, 256, 350, 400, 500, 512, 1000, 1024};
  int32_t y0[10] = {50, 50, 50, 50, 90, 90, 90, 130, 130, 130};
  int32_t x0[10] = {30, 70, 110, 150, 50, 90, 130, 50, 90, 130};
  // workspace and saved-state sizes: every size, padding, approximation, operation and a few batches
  for (int N : sizes) {
    const int half = (N - N / 2) % 2 ? N / 2 + 1 : N / 2;  // a padded layer, N - n even
    for (int n : {N, N - 2, half}) {
      for (int approx = 0; approx <= 4; ++approx) {
        lr_detector det{n >= 170 ? 10 : 0, 20, y0, x0};
        lr_donn net{532e-9, 36e-6, 0.3, approx, n, N, 5, 1.0f, det, static_cast<const lr_c64*>(fake(0x1000)), 0,
                    nullptr};
        for (int op = 0; op <= 2; ++op) {
          for (int b : {0, 1, 7, 500}) {
            const int64_t w = lr_workspace_size(&net, b, op);
            if (approx == LR_FRAUNHOFER && op != LR_OP_PROPAGATE) {
              EXPECT(w == -LR_E_APPROX);
            } else if (approx == LR_FRAUNHOFER && (N % 2)) {
              EXPECT(w == -LR_E_SIZE);
            } else {
              EXPECT(w >= 0);
            }
          }
          EXPECT(lr_workspace_size(&net, -1, op) < 0);
        }
        if (approx != LR_FRAUNHOFER) EXPECT(lr_saved_size(&net, 500) == 6LL * 500 * n * n * 8);
        EXPECT(lr_workspace_size(&net, 4, 7) == -LR_E_ARG);
        EXPECT(lr_workspace_size(&net, INT32_MAX, LR_OP_FORWARD) > 0 || approx == LR_FRAUNHOFER);
      }
    }
  }
  // detector origins near INT32_MAX and negative ones
  {
    int32_t big[1] = {INT32_MAX - 5};
    int32_t zero[1] = {0};
    int32_t neg[1] = {INT32_MIN};
    for (auto* ys : {big, zero, neg}) {
      for (auto* xs : {big, zero, neg}) {
        lr_detector det{1, 20, ys, xs};
        lr_donn net{532e-9, 36e-6, 0.3, 0, 200, 200, 5, 1.0f, det, static_cast<const lr_c64*>(fake(0x1000)), 0,
                    nullptr};
        const bool ok = ys == zero && xs == zero;
        EXPECT((lr_workspace_size(&net, 4, LR_OP_FORWARD) > 0) == ok);
        if (!ok) {
          float* sums = static_cast<float*>(fake(0x90000000));
          EXPECT(lr_detector_readout(static_cast<const lr_c64*>(fake(0x1000)), 2, 200, &det, sums, nullptr) ==
                 LR_E_ARG);
        }
      }
    }
    lr_detector huge{1, INT32_MAX, zero, zero};
    lr_donn net{532e-9, 36e-6, 0.3, 0, 200, 200, 5, 1.0f, huge, static_cast<const lr_c64*>(fake(0x1000)), 0,
                nullptr};
    EXPECT(lr_workspace_size(&net, 4, LR_OP_FORWARD) == -LR_E_ARG);
  }
  // overlapping ranges are rejected before anything is enqueued
  {
    lr_detector det{0, 1, nullptr, nullptr};
    lr_donn net{532e-9, 36e-6, 0.3, 0, 200, 200, 5, 1.0f, det, static_cast<const lr_c64*>(fake(0x1000)), 0, nullptr};
    const size_t field = 2ull * 200 * 200 * 8;
    const int64_t ws = lr_workspace_size(&net, 2, LR_OP_PROPAGATE);
    EXPECT(ws > 0);
    auto* in = static_cast<const lr_c64*>(fake(0x10000000));
    EXPECT(lr_propagate(&net, 2, in, static_cast<lr_c64*>(fake(0x10000000 + field - 8)), 0, fake(0x40000000),
                        static_cast<size_t>(ws), nullptr) == LR_E_ALIAS);
    EXPECT(lr_propagate(&net, 2, in, static_cast<lr_c64*>(fake(0x20000000)), 0, fake(0x20000000 + 8),
                        static_cast<size_t>(ws), nullptr) == LR_E_ALIAS);
    float* phi = static_cast<float*>(fake(0x30000000));
    float* g = static_cast<float*>(fake(0x30000000 + 64));
    EXPECT(lr_adam_update(phi, static_cast<const float*>(fake(0x50000000)), g, static_cast<float*>(fake(0x60000000)),
                          100, 1, 0.5f, 0.9f, 0.999f, 1e-8f, nullptr) == LR_E_ALIAS);
    EXPECT(lr_loss(0, static_cast<const float*>(fake(0x1000)), static_cast<const int32_t*>(fake(0x9000)), 4, 10,
                   nullptr, static_cast<float*>(fake(0x1000 + 4)), nullptr) == LR_E_ALIAS);
  }
  // no-allocation propagate: limit and rejection of larger workspaces
  {
    lr_detector det{0, 1, nullptr, nullptr};
    lr_donn net{532e-9, 36e-6, 0.3, 1, 512, 1024, 1, 1.0f, det, static_cast<const lr_c64*>(fake(0x1000)), 0,
                nullptr};
    EXPECT(lr_propagate_noalloc_limit() == static_cast<int64_t>(LR_NOALLOC_SCRATCH_BYTES));
    EXPECT(lr_workspace_size(&net, 64, LR_OP_PROPAGATE) > lr_propagate_noalloc_limit());
    EXPECT(lr_propagate_noalloc(&net, 64, static_cast<const lr_c64*>(fake(0x10000000)),
                                static_cast<lr_c64*>(fake(0x80000000)), 0, nullptr) == LR_E_WORKSPACE);
  }
  // float64 transfer-function tables of every approximation (host arithmetic);
  // only where no GPU is visible, since the destination is not device memory
  int devices = 0;
  if (hipGetDeviceCount(&devices) != hipSuccess) devices = 0;
  if (devices == 0) {
    std::vector<lr_c64> host(1024 * 1024);
    for (int N : {64, 100, 200, 350, 1000, 1024}) {
      for (int approx = 0; approx <= 4; ++approx) {
        const int r = lr_tf_build(532e-9, 36e-6, 0.3, approx, N, host.data(), nullptr);
        const bool shape_ok = !((approx == LR_FRESNEL_IR || approx == LR_RS_IR) && N == 350);
        EXPECT(r == (shape_ok ? LR_E_HIP : LR_E_SIZE));
      }
    }
    EXPECT(lr_tf_build(532e-9, 36e-6, -0.3, LR_FRESNEL, 200, host.data(), nullptr) == LR_E_HIP);  // back-propagation
  } else {
    std::printf("(GPU present: transfer-function tables skipped)\n");
  }
  for (int s = -1; s <= 8; ++s) EXPECT(lr_status_string(s) != nullptr);
  if (g_fail) {
    std::printf("%d failures\n", g_fail);
    return 1;
  }
  std::printf("ALL OK\n");
  return 0;
}
