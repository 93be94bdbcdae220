// host.hpp -- host-side plumbing shared by the launchers: error reporting, workspace carving,
// launch checks.
#pragma once
#include <hip/hip_runtime.h>
#include <stdarg.h>
#include <stddef.h>
#include <stdint.h>
#include <stdio.h>

#include "hmoe.h"

namespace hmoe {

// Thread-local message behind hmoe_last_error().
void set_error(const char* fmt, ...);
void clear_error();

// Carves 256-byte aligned pieces out of a caller workspace.  With base == nullptr it only
// measures, so the same code sizes and carves.
struct Workspace {
  char* base;
  size_t cap;
  size_t off = 0;
  Workspace(void* b, size_t c) : base(static_cast<char*>(b)), cap(c) {}
  template <typename T>
  T* take(size_t count) {
    off = (off + 255) & ~size_t(255);
    T* p = base ? reinterpret_cast<T*>(base + off) : nullptr;
    off += count * sizeof(T);
    return p;
  }
  bool fits() const { return base == nullptr || off <= cap; }
};

inline int hip_check(hipError_t e, const char* what) {
  if (e != hipSuccess) {
    set_error("%s: %s", what, hipGetErrorString(e));
    return HMOE_EHIP;
  }
  return HMOE_OK;
}

// Call after a launch: reports a launch-configuration failure as HMOE_EHIP.
inline int launch_check(const char* what) { return hip_check(hipGetLastError(), what); }

inline size_t dtype_size(hmoe_dtype_t dt) { return dt == HMOE_BF16 ? 2 : 4; }

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Compute units of the current device; cached per device.
inline int device_cus() {
  static int cache[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cache[dev] == 0) {
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0) cus = 256;
    cache[dev] = cus;
  }
  return cache[dev];
}

// Optional per-launch HIP-event timing (off unless hmoe_timer_enable(1) was called).
void timer_pre(const char* label, hipStream_t st);
void timer_post(hipStream_t st);

// Launch a kernel through the timer hooks and report launch failures as HMOE_EHIP.
#define HMOE_LAUNCH(label, kernel, grid, block, lds, st, ...)          \
  do {                                                                 \
    ::hmoe::timer_pre(label, st);                                      \
    hipLaunchKernelGGL(kernel, grid, block, lds, st, __VA_ARGS__);     \
    ::hmoe::timer_post(st);                                            \
    int _lrc = ::hmoe::launch_check(label);                            \
    if (_lrc != HMOE_OK) return _lrc;                                  \
  } while (0)

#define HMOE_TRY(...)                 \
  do {                                \
    int _rc = (__VA_ARGS__);          \
    if (_rc != HMOE_OK) return _rc;   \
  } while (0)

}  // namespace hmoe
