// Internal helpers shared by the PARK HIP kernels and the host API.
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/park.h"

namespace park {

typedef uint16_t bf16_t;

// ------------------------------------------------------------ bf16 <-> f32
__device__ __forceinline__ float bf2f(bf16_t x) { return __uint_as_float(((uint32_t)x) << 16); }

// round-to-nearest-even float -> bf16 (NaN stays NaN)
__device__ __forceinline__ bf16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (bf16_t)((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (bf16_t)(u >> 16);
}

template <typename T>
__device__ __forceinline__ float to_f(T x);
template <>
__device__ __forceinline__ float to_f<float>(float x) { return x; }
template <>
__device__ __forceinline__ float to_f<bf16_t>(bf16_t x) { return bf2f(x); }

// ------------------------------------------------------------ status bits
// The sticky device status word lives in the first 4 bytes of a workspace.
enum : int {
  ST_NOT_SPD = 1,      // stabilised metric not positive definite
  ST_NONFINITE = 2,    // non-finite value in an input or a reduction
};

__device__ __forceinline__ void raise_status(int* status, int bit) {
  if (status) atomicOr(status, bit);
}

// ------------------------------------------------------------ host helpers
struct Carver {
  char* base;
  size_t off = 0;
  explicit Carver(void* b) : base((char*)b) {}
  template <class T>
  T* take(size_t n) {
    off = (off + 255) & ~(size_t)255;
    T* p = base ? (T*)(base + off) : nullptr;
    off += n * sizeof(T);
    return p;
  }
};

// Per-kernel profiler (park_profile_*).  When enabled, a launch takes two
// events and is issued with hipExtLaunchKernelGGL, which timestamps the
// dispatch itself; prof_commit files the pair under the kernel's name.
bool prof_take(hipEvent_t* a, hipEvent_t* b);
void prof_commit(const char* name, hipEvent_t a, hipEvent_t b);

// Records the message of a failed call (park_last_error).
park_status fail(park_status st, const char* fmt, ...);

#define PARK_LAUNCH(name, kernel, grid, block, shmem, stream, ...)                    \
  do {                                                                                \
    hipEvent_t pa_ = nullptr, pb_ = nullptr;                                          \
    if (::park::prof_take(&pa_, &pb_)) {                                              \
      hipExtLaunchKernelGGL(kernel, grid, block, shmem, stream, pa_, pb_, 0, __VA_ARGS__); \
      ::park::prof_commit(name, pa_, pb_);                                            \
    } else {                                                                          \
      hipLaunchKernelGGL(kernel, grid, block, shmem, stream, __VA_ARGS__);            \
    }                                                                                 \
    hipError_t e_ = hipGetLastError();                                                \
    if (e_ != hipSuccess)                                                             \
      return ::park::fail(PARK_ERR_HIP, "%s: %s", name, hipGetErrorString(e_));       \
  } while (0)

#define PARK_TRY(expr)                 \
  do {                                 \
    park_status s_ = (expr);           \
    if (s_ != PARK_OK) return s_;      \
  } while (0)

inline size_t elem_size(int dtype) { return dtype == PARK_BF16 ? 2 : 4; }

}  // namespace park
