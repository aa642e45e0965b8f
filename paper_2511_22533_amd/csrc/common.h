// Shared device-side definitions for the gfx950 kernels: element types, MFMA
// fragment traits for the 32x32 matrix-core family, and small helpers.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace f3c {

// Timing of one profiled library call. While it is set on this thread, every
// kernel launch goes through AMD's extended launch, which stamps the events
// with the kernels' own start and end: the first kernel of the call stamps
// start, each kernel re-stamps stop. The pair then spans the call's kernels
// without the host's dispatch gap in front of them.
struct LaunchTimer {
  hipEvent_t start = nullptr, stop = nullptr;
  bool used = false;
};

inline LaunchTimer& launch_timer() {
  static thread_local LaunchTimer t;
  return t;
}

// Kernel launch used by every kernel of the library (same arguments as
// hipLaunchKernelGGL).
template <typename F, typename... Args>
inline void launch(F kernel, dim3 grid, dim3 block, uint32_t shmem, hipStream_t s, Args... args) {
  LaunchTimer& t = launch_timer();
  if (!t.stop) {
    hipLaunchKernelGGL(kernel, grid, block, shmem, s, args...);
    return;
  }
  hipExtLaunchKernelGGL(kernel, grid, block, shmem, s, t.used ? nullptr : t.start, t.stop, 0u, args...);
  t.used = true;
}

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// 32x32 MFMA family. One instruction multiplies a 32xK by a Kx32 tile. Each
// lane l feeds E consecutive K-elements of row (A) / column (B) l % 32 for the
// K-group l / 32; the 16 accumulators of lane l hold column l % 32 and rows
// 8*(i/4) + 4*(l/32) + i%4, i = 0..15.
template <typename T> struct Mfma;

template <> struct Mfma<bf16> {
  static constexpr int E = 8;          // elements per lane per instruction (K = 16)
  typedef bf16x8 frag;
  static __device__ __forceinline__ f32x16 mma(const frag& a, const frag& b, const f32x16& c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
};

template <> struct Mfma<float> {
  static constexpr int E = 1;          // K = 2
  typedef float frag;
  static __device__ __forceinline__ f32x16 mma(const frag& a, const frag& b, const f32x16& c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
};

__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(bf16 x) { return static_cast<float>(x); }

template <typename T> __device__ __forceinline__ T from_f32(float x);
template <> __device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <> __device__ __forceinline__ bf16 from_f32<bf16>(float x) { return static_cast<bf16>(x); }

// GELU in its tanh form, 0.5 x (1 + tanh(u)) with u = sqrt(2/pi) (x + 0.044715 x^3),
// evaluated as the identical x / (1 + e^(-2u)): one exponential and one
// reciprocal instead of the library tanhf (measured on MI355X: the MLP's first
// projection at 32768 rows, 485 -> 447 us; a plain store takes 440 us). For
// u far below zero e^(-2u) overflows to +inf and the result is -0.
__device__ __forceinline__ float gelu_tanh(float x) {
  const float k0 = 0.7978845608028654f;   // sqrt(2/pi)
  const float k1 = 0.044715f;
  const float u = k0 * (x + k1 * x * x * x);
  const float e = __builtin_amdgcn_exp2f(u * -2.8853900817779268f);   // 2^(-2u log2(e)) = e^(-2u)
  return x * __builtin_amdgcn_rcpf(1.0f + e);
}

__device__ __forceinline__ float silu(float x) { return x / (1.0f + expf(-x)); }

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// Workgroups are dispatched round-robin over the 8 XCDs (each with its own
// L2). Map the hardware workgroup id to a logical id so that each XCD receives
// one contiguous range of logical ids (sizes differ by at most one).
__device__ __forceinline__ int xcd_logical_id(int hw, int total) {
  constexpr int kXcd = 8;
  const int x = hw % kXcd, i = hw / kXcd;
  const int q = total / kXcd, r = total % kXcd;
  return x * q + (x < r ? x : r) + i;
}

// 16 bytes per lane from global memory straight into LDS at lds_block + 16 *
// lane (gfx950 global_load_lds_dwordx4; the block base is wave-uniform and
// goes through M0). Written as inline assembly so that the compiler does not
// track it: it would otherwise wait for every outstanding LDS load of this
// kind before any LDS read. A kernel using it orders these loads itself (an
// s_waitcnt on the vector-memory counter and a barrier before a tile is
// read); waits the compiler places for its own loads only grow more
// conservative, since the counter retires in issue order.
__device__ __forceinline__ void dma16(const char* gptr, char* lds_block) {
  const uint32_t base = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)lds_block;
  asm volatile("global_load_lds_dwordx4 %0, off" : : "v"(gptr), "{m0}"(__builtin_amdgcn_readfirstlane(base))
               : "memory");
}

// Wait until at most N vector-memory operations are outstanding (gfx9
// s_waitcnt encoding; expcnt and lgkmcnt left at their maxima).
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// Sample lookup in a segment table off[0..B] (off[B] = total rows).
__device__ __forceinline__ int find_segment(const int* off, int B, int row) {
  int b = 0;
  while (b + 1 < B && off[b + 1] <= row) ++b;
  return b;
}

}  // namespace f3c
