// Host-side helpers for the C ABI implementation.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "fastcoder.h"

namespace fc {

// Workspace carving: hands out 256-byte aligned slices of a caller buffer.
struct Carver {
  char* base;
  size_t used;
  explicit Carver(void* p) : base((char*)p), used(0) {}
  template <typename T>
  T* take(size_t count) {
    used = (used + 255) & ~(size_t)255;
    T* r = base ? (T*)(base + used) : nullptr;
    used += count * sizeof(T);
    return r;
  }
};

inline fc_status launch_status() {
  hipError_t e = hipGetLastError();
  return e == hipSuccess ? FC_OK : FC_ERR_DEVICE;
}

}  // namespace fc

#define FC_CHECK_HIP(expr)                 \
  do {                                     \
    if ((expr) != hipSuccess) {            \
      (void)hipGetLastError();             \
      return FC_ERR_DEVICE;                \
    }                                      \
  } while (0)

#define FC_CHECK_LAUNCH()                  \
  do {                                     \
    if (hipGetLastError() != hipSuccess) { \
      return FC_ERR_DEVICE;                \
    }                                      \
  } while (0)
