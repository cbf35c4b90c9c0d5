// Host sanitizer run of the C ABI (test infrastructure): libsa's sources are
// built with AddressSanitizer and UndefinedBehaviorSanitizer on the host side
// (device code unchanged) and linked into this driver, which calls every entry
// point of include/sa.h with every kind of invalid argument and checks the
// documented status and message. With no GPU present it also passes
// well-formed arguments (fake device addresses that no kernel ever reads),
// which run the host-side dispatch up to the launch and must come back as
// SA_ERR_HIP. Exits non-zero on a wrong status; the sanitizers abort on any
// out-of-bounds access or undefined behaviour in the host code.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>
#include <cstring>

#include "sa.h"

namespace {

int failures = 0;

void expect(const char* what, int rc, int want) {
  if (rc != want) {
    std::printf("FAIL %s: status %d, expected %d (%s)\n", what, rc, want, sa_last_error());
    ++failures;
  } else if (want != SA_OK && std::strlen(sa_last_error()) == 0) {
    std::printf("FAIL %s: status %d without a message\n", what, rc);
    ++failures;
  }
}

void* const F = reinterpret_cast<void*>(0x100000);        // aligned fake device address
void* const G = reinterpret_cast<void*>(0x200000);
void* const ODD = reinterpret_cast<void*>(0x100008);      // not 16-byte aligned
int32_t* const W = reinterpret_cast<int32_t*>(0x300000);  // int32 array
int32_t* const WODD = reinterpret_cast<int32_t*>(0x300002);
float* const L = reinterpret_cast<float*>(0x400000);

int fwd(void* q = F, void* out = F, float* lse = nullptr, int B = 2, int T = 8, int H = 2, int d = 64, int Lb = 2,
        int La = 1, int32_t* len = nullptr, int dt = SA_BF16) {
  return sa_forward(q, F, F, out, lse, B, T, H, d, Lb, La, len, dt, nullptr);
}

int bwd(float* lse = L, void* dq = F, int B = 2, int T = 8, int d = 64, int Lb = 2, int La = 1, int dt = SA_BF16) {
  return sa_backward(F, F, F, F, lse, F, dq, F, F, B, T, 2, d, Lb, La, nullptr, dt, nullptr);
}

}  // namespace

int main() {
  int ndev = 0;
  const bool gpu = hipGetDeviceCount(&ndev) == hipSuccess && ndev > 0;
  (void)hipGetLastError();

  if (sa_abi_version() != 1) {
    std::printf("FAIL abi version %d\n", sa_abi_version());
    ++failures;
  }

  // sa_forward
  expect("fwd empty batch", fwd(F, F, nullptr, 0), SA_OK);
  expect("fwd empty T, NULL q", fwd(nullptr, F, nullptr, 2, 0), SA_OK);
  expect("fwd negative B", fwd(F, F, nullptr, -1), SA_ERR_INVALID);
  expect("fwd negative H", fwd(F, F, nullptr, 2, 8, -2), SA_ERR_INVALID);
  expect("fwd negative Lb", fwd(F, F, nullptr, 2, 8, 2, 64, -1), SA_ERR_INVALID);
  expect("fwd negative La", fwd(F, F, nullptr, 2, 8, 2, 64, 2, -3), SA_ERR_INVALID);
  expect("fwd d = 48", fwd(F, F, nullptr, 2, 8, 2, 48), SA_ERR_UNSUPPORTED);
  expect("fwd dtype 7", fwd(F, F, nullptr, 2, 8, 2, 64, 2, 1, nullptr, 7), SA_ERR_UNSUPPORTED);
  expect("fwd NULL q", fwd(nullptr), SA_ERR_NULL);
  expect("fwd NULL out", fwd(F, nullptr), SA_ERR_NULL);
  expect("fwd misaligned q", fwd(ODD), SA_ERR_INVALID);
  expect("fwd misaligned lengths", fwd(F, F, nullptr, 2, 8, 2, 64, 2, 1, WODD), SA_ERR_INVALID);
  expect("fwd B*T*H overflow", fwd(F, F, nullptr, 1 << 16, 1 << 12, 1 << 4), SA_ERR_INVALID);
  expect("fwd T too long", fwd(F, F, nullptr, 1, (1 << 30) + 1, 1), SA_ERR_INVALID);
  expect("fwd T*H*d overflow", fwd(F, F, nullptr, 1, 1 << 20, 1 << 10, 64), SA_ERR_INVALID);

  // sa_backward
  expect("bwd empty", bwd(L, F, 0), SA_OK);
  expect("bwd NULL lse", bwd(nullptr), SA_ERR_NULL);
  expect("bwd NULL dq", bwd(L, nullptr), SA_ERR_NULL);
  expect("bwd d = 16", bwd(L, F, 2, 8, 16), SA_ERR_UNSUPPORTED);
  expect("bwd misaligned dq", bwd(L, ODD), SA_ERR_INVALID);
  expect("bwd misaligned lse", bwd(reinterpret_cast<float*>(0x400002)), SA_ERR_INVALID);
  expect("bwd negative La", bwd(L, F, 2, 8, 64, 2, -1), SA_ERR_INVALID);

  // llsa_forward, llsa_backward
  expect("llsa fwd NULL q", llsa_forward(nullptr, F, F, F, nullptr, 2, 8, 2, 32, 2, 1, nullptr, SA_F32, nullptr),
         SA_ERR_NULL);
  expect("llsa fwd negative La",
         llsa_forward(F, F, F, F, nullptr, 2, 8, 2, 32, 2, -1, nullptr, SA_F32, nullptr), SA_ERR_INVALID);
  expect("llsa fwd empty", llsa_forward(F, F, F, F, nullptr, 0, 8, 2, 32, 2, 1, nullptr, SA_F32, nullptr), SA_OK);
  expect("llsa bwd NULL lse",
         llsa_backward(F, F, F, F, nullptr, F, F, F, F, 2, 8, 2, 64, 2, 1, nullptr, SA_BF16, nullptr), SA_ERR_NULL);
  expect("llsa bwd misaligned dv",
         llsa_backward(F, F, F, F, L, F, F, F, ODD, 2, 8, 2, 64, 2, 1, nullptr, SA_BF16, nullptr), SA_ERR_INVALID);
  expect("llsa bwd d = 128",
         llsa_backward(F, F, F, F, L, F, F, F, F, 2, 8, 2, 128, 2, 1, nullptr, SA_BF16, nullptr), SA_ERR_UNSUPPORTED);

  // llsa_paper_forward, llsa_paper_backward
  expect("paper fwd La too large",
         llsa_paper_forward(F, F, F, F, L, 2, 8, 2, 64, 2, SA_LLSA_PAPER_MAX_LA + 1, nullptr, SA_BF16, nullptr),
         SA_ERR_INVALID);
  expect("paper fwd NULL lse", llsa_paper_forward(F, F, F, F, nullptr, 2, 8, 2, 64, 2, 3, nullptr, SA_BF16, nullptr),
         SA_ERR_NULL);
  expect("paper bwd dtype 5",
         llsa_paper_backward(F, F, F, F, L, F, F, F, F, 2, 8, 2, 64, 2, 3, nullptr, 5, nullptr),
         SA_ERR_UNSUPPORTED);
  expect("paper bwd NULL dk",
         llsa_paper_backward(F, F, F, F, L, F, F, nullptr, F, 2, 8, 2, 64, 2, 3, nullptr, SA_BF16, nullptr),
         SA_ERR_NULL);

  // sa_stream_step
  expect("stream NULL step",
         sa_stream_step(F, F, F, F, F, F, F, 10, nullptr, nullptr, 4, 2, 64, 6, 3, nullptr, SA_BF16, nullptr),
         SA_ERR_NULL);
  expect("stream ring too small",
         sa_stream_step(F, F, F, F, F, F, F, 9, W, nullptr, 4, 2, 64, 6, 3, nullptr, SA_BF16, nullptr),
         SA_ERR_INVALID);
  expect("stream window too wide",
         sa_stream_step(F, F, F, F, F, F, F, 2000, W, nullptr, 4, 2, 64, 1500, 3, nullptr, SA_BF16, nullptr),
         SA_ERR_INVALID);
  expect("stream negative S",
         sa_stream_step(F, F, F, F, F, F, F, 10, W, nullptr, -1, 2, 64, 6, 3, nullptr, SA_BF16, nullptr),
         SA_ERR_INVALID);
  expect("stream misaligned step",
         sa_stream_step(F, F, F, F, F, F, F, 10, WODD, nullptr, 4, 2, 64, 6, 3, nullptr, SA_BF16, nullptr),
         SA_ERR_INVALID);
  expect("stream empty", sa_stream_step(F, F, F, F, F, F, F, 10, W, nullptr, 0, 2, 64, 6, 3, nullptr, SA_BF16, nullptr),
         SA_OK);
  expect("llsa stream NULL ring",
         llsa_stream_step(F, F, F, F, F, F, F, F, F, nullptr, F, F, 10, W, nullptr, nullptr, 4, 2, 64, 6, 3, nullptr,
                          SA_BF16, nullptr),
         SA_ERR_NULL);
  expect("llsa stream ring too small",
         llsa_stream_step(F, F, F, F, F, F, F, F, F, F, F, F, 9, W, nullptr, nullptr, 4, 2, 64, 6, 3, nullptr,
                          SA_BF16, nullptr),
         SA_ERR_INVALID);

  // sa_copy_reference
  expect("copy odd size", sa_copy_reference(F, G, 24, 0, nullptr), SA_ERR_INVALID);
  expect("copy negative size", sa_copy_reference(F, G, -16, 0, nullptr), SA_ERR_INVALID);
  expect("copy mode 2", sa_copy_reference(F, G, 64, 2, nullptr), SA_ERR_INVALID);
  expect("copy NULL src", sa_copy_reference(nullptr, G, 64, 0, nullptr), SA_ERR_NULL);
  expect("copy overlap", sa_copy_reference(F, reinterpret_cast<char*>(F) + 16, 64, 0, nullptr), SA_ERR_INVALID);
  expect("copy empty", sa_copy_reference(F, G, 0, 1, nullptr), SA_OK);

  // well-formed arguments run the host-side dispatch (band plans, window
  // segments, kernel choice) up to the launch, which fails without a device.
  // Skipped when a GPU is present: the fake addresses must never reach one.
  if (!gpu) {
    const int wd[][3] = {{64, 64, 8}, {32, 200, 200}, {64, 100, 20}, {64, 0, 0}, {64, 30, 15}};
    for (const auto& c : wd) {
      const int d = c[0], Lb = c[1], La = c[2];
      expect("fwd dispatch", fwd(F, F, L, 3, 300, 2, d, Lb, La, W), SA_ERR_HIP);
      expect("fwd dispatch f32", fwd(F, F, L, 3, 300, 2, d, Lb, La, W, SA_F32), SA_ERR_HIP);
      expect("bwd dispatch", bwd(L, F, 3, 300, d, Lb, La), SA_ERR_HIP);
      expect("llsa fwd dispatch",
             llsa_forward(F, F, F, F, L, 3, 300, 2, d, Lb, La, W, SA_BF16, nullptr), SA_ERR_HIP);
      expect("paper fwd dispatch",
             llsa_paper_forward(F, F, F, F, L, 3, 300, 2, d, Lb, La, W, SA_BF16, nullptr),
             La > SA_LLSA_PAPER_MAX_LA ? SA_ERR_INVALID : SA_ERR_HIP);
      expect("stream dispatch", sa_stream_step(F, F, F, F, F, F, F, Lb + La + 1, W, nullptr, 4, 2, d, Lb, La, W,
                                               SA_BF16, nullptr),
             SA_ERR_HIP);
    }
    for (const auto& c : wd) {
      for (int dt : {SA_BF16, SA_F32}) {
        expect("llsa bwd dispatch",
               llsa_backward(F, F, F, F, L, F, F, F, F, 3, 300, 2, c[0], c[1], c[2], W, dt, nullptr), SA_ERR_HIP);
        expect("paper bwd dispatch",
               llsa_paper_backward(F, F, F, F, L, F, F, F, F, 3, 300, 2, c[0], c[1], c[2], W, dt, nullptr),
               c[2] > SA_LLSA_PAPER_MAX_LA ? SA_ERR_INVALID : SA_ERR_HIP);
      }
    }
    expect("copy dispatch", sa_copy_reference(F, G, 4096, 1, nullptr), SA_ERR_HIP);
  }

  if (failures) {
    std::printf("%d failures\n", failures);
    return 1;
  }
  std::printf("sanitized ABI run ok (%s)\n", gpu ? "GPU present: dispatch calls skipped" : "no GPU");
  return 0;
}
