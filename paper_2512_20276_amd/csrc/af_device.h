// Device-side building blocks shared by the kernel sources: element types and conversions, the
// MFMA instruction per element type, 16-byte chunks, compile-time loops, XCD-aware tile order.
#pragma once

#include <hip/hip_runtime.h>

#include <algorithm>
#include <type_traits>

#include "af_internal.h"

namespace af {

typedef __bf16 bf16;
typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(__bf16)))) __bf16 bf16x4;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef __attribute__((__vector_size__(8 * sizeof(float)))) float f32x8;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;
typedef __attribute__((__vector_size__(4 * sizeof(unsigned)))) unsigned u32x4;  // raw 16 bytes

__device__ __forceinline__ float to_f(bf16 x) { return (float)x; }
__device__ __forceinline__ float to_f(float x) { return x; }
template <typename T>
__device__ __forceinline__ T from_f(float x);
template <>
__device__ __forceinline__ bf16 from_f<bf16>(float x) { return (bf16)x; }
template <>
__device__ __forceinline__ float from_f<float>(float x) { return x; }

// ------------------------------------------------------------------ MFMA per element type
template <typename T>
struct Mma;
template <>
struct Mma<bf16> {
  typedef bf16x8 frag;  // 8 consecutive k, 16 bytes
  __device__ __forceinline__ static f32x4 mma(frag a, frag b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
};
template <>
struct Mma<float> {
  typedef f32x8 frag;  // 8 consecutive k, 32 bytes
  __device__ __forceinline__ static f32x4 mma(frag a, frag b, f32x4 c) {
#pragma unroll
    for (int j = 0; j < 8; ++j) c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[j], b[j], c, 0, 0, 0);
    return c;
  }
};

// 16-byte global/LDS chunk
template <typename T>
struct Chunk {
  static constexpr int N = 16 / sizeof(T);
};

__device__ __forceinline__ uint4 zero4() { return make_uint4(0, 0, 0, 0); }

// Compile-time loop: f(std::integral_constant<int, I>) for I in [B, E).  Register arrays indexed
// by such constants are promoted to registers before any loop transformation runs.
template <int B, int E, class F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

// ------------------------------------------------------------------ XCD-aware tile order
// Workgroups are dispatched round-robin over the 8 XCDs (each with its own L2).  Give each
// XCD a contiguous run of logical tiles so the M tiles that share a weight panel run on one
// XCD and the panel is fetched from HBM once.
#ifndef AF_XCD_REMAP
#define AF_XCD_REMAP 1
#endif
__device__ __forceinline__ int xcd_remap(int bid, int total) {
  if (!AF_XCD_REMAP) return bid;
  const int q = total / 8, r = total % 8;
  const int x = bid % 8, j = bid / 8;
  return x * q + (x < r ? x : r) + j;
}


// 8 consecutive elements with 16-byte (bf16) or 32-byte (fp32) accesses.
template <typename T>
__device__ __forceinline__ void load8(const T* p, T* r) {
  if constexpr (sizeof(T) == 2) {
    *(uint4*)r = *(const uint4*)p;
  } else {
    *(uint4*)r = *(const uint4*)p;
    *(uint4*)(r + 4) = *(const uint4*)(p + 4);
  }
}
template <typename T>
__device__ __forceinline__ void store8(T* p, const T* r) {
  if constexpr (sizeof(T) == 2) {
    *(uint4*)p = *(const uint4*)r;
  } else {
    *(uint4*)p = *(const uint4*)r;
    *(uint4*)(p + 4) = *(const uint4*)(r + 4);
  }
}

}  // namespace af
