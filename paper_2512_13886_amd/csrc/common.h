// Shared helpers of the OPTIMA gfx950 library: vector types, error macros,
// workspace carving and block reductions.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <algorithm>
#include <utility>

#include "optima.h"

namespace optima {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x16 __attribute__((ext_vector_type(16)));

// Output tile of the MFMA GEMM core and the padding unit of every matrix the
// core reads (rows and the contraction dimension are padded to it).
constexpr int kTile = 128;
constexpr int kThreads = 256;

#define OPTIMA_HIP_TRY(expr)                  \
  do {                                        \
    hipError_t e_ = (expr);                   \
    if (e_ != hipSuccess) return OPTIMA_E_HIP; \
  } while (0)

#define OPTIMA_LAUNCH_CHECK()                              \
  do {                                                     \
    if (hipPeekAtLastError() != hipSuccess) {              \
      (void)hipGetLastError();                             \
      return OPTIMA_E_HIP;                                 \
    }                                                      \
  } while (0)

inline int64_t round_up(int64_t a, int64_t b) { return (a + b - 1) / b * b; }
inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Sequential carving of a caller workspace into 256-byte aligned pieces. The
// same sequence of take() calls sizes the workspace (base == nullptr) and
// hands out the pointers.
struct Carver {
  char* base;
  size_t off = 0;
  explicit Carver(void* b) : base(static_cast<char*>(b)) {}
  template <typename T>
  T* take(size_t count) {
    off = (off + 255) & ~size_t(255);
    T* p = base ? reinterpret_cast<T*>(base + off) : nullptr;
    off += count * sizeof(T);
    return p;
  }
  size_t bytes() const { return (off + 255) & ~size_t(255); }
};

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Sum of one double per thread over a block of kThreads threads; every thread
// gets the total. `smem` needs kThreads / 64 doubles.
__device__ inline double block_sum(double v, double* smem) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) smem[wave] = v;
  __syncthreads();
  double t = 0.0;
  for (int w = 0; w < kThreads / 64; ++w) t += smem[w];
  return t;
}

}  // namespace optima
