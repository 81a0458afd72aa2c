// Shared device helpers for the gfx950 kernels: bf16 storage conversions,
// MFMA operand types, wave64 reductions.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace spec {

// Kernel-level timing: a timer arms a start / stop event pair for the next
// launch made through launch_kernel, which then records the kernel's own
// start and end (the interval a profiler reports), not the dispatch around
// it.  Unarmed, launch_kernel is a plain launch (the only form used under
// graph capture).
struct LaunchEvents {
  hipEvent_t start = nullptr, stop = nullptr;
};
inline LaunchEvents& launch_events() {
  static thread_local LaunchEvents e;
  return e;
}
template <typename F, typename... Args>
inline void launch_kernel(F kernel, dim3 grid, dim3 block, size_t lds, hipStream_t st, Args... args) {
  LaunchEvents& le = launch_events();
  if (le.start) {
    const LaunchEvents ev = le;
    le = LaunchEvents{};
    hipExtLaunchKernelGGL(kernel, grid, block, static_cast<uint32_t>(lds), st, ev.start, ev.stop, 0u, args...);
  } else {
    kernel<<<grid, block, lds, st>>>(args...);
  }
}

typedef uint16_t bf16_t;  // storage type: bf16 bit pattern
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;
constexpr int kPage = 16;

__device__ __forceinline__ float bf16_to_f32(bf16_t x) {
  return __uint_as_float(static_cast<uint32_t>(x) << 16);
}

// fp32 -> bf16, round to nearest, ties to even (inputs are finite).
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return static_cast<bf16_t>(u >> 16);
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return static_cast<uint32_t>(f32_to_bf16(lo)) | (static_cast<uint32_t>(f32_to_bf16(hi)) << 16);
}

// Element-type traits: storage type T in {float, bf16_t}; loads widen to fp32.
template <typename T> struct Elem;
template <> struct Elem<float> {
  __device__ __forceinline__ static float load(const float* p) { return *p; }
  __device__ __forceinline__ static float to_f32(float x) { return x; }
  __device__ __forceinline__ static float from_f32(float x) { return x; }
};
template <> struct Elem<bf16_t> {
  __device__ __forceinline__ static float load(const bf16_t* p) { return bf16_to_f32(*p); }
  __device__ __forceinline__ static float to_f32(bf16_t x) { return bf16_to_f32(x); }
  __device__ __forceinline__ static bf16_t from_f32(float x) { return f32_to_bf16(x); }
};

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Streaming 16-byte loads (nontemporal hint: data read once stays out of the way
// of reused operands in the caches).
__device__ __forceinline__ uint4 ld_stream(const uint4* p) {
  const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ float4 ld_stream(const float4* p) {
  const f32x4 v = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p));
  return make_float4(v.x, v.y, v.z, v.w);
}

__device__ __forceinline__ f32x4 mfma16x16x32(const uint4& a, const uint4& b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

__device__ __forceinline__ f32x4 mfma16x16x32v(const u32x4& a, const u32x4& b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// ---------------------------------------------------------------------------
// Direct-to-LDS loads (global -> LDS with no register staging) and the
// explicit waits their users issue.

typedef __attribute__((address_space(3))) void* lptr_t;

// One global_load_lds_dwordx4: lane i's 16 bytes at base + off_bytes land in
// LDS at byte lds + 16 i (M0 holds the LDS address; one wait state separates
// the M0 write from the load).  Issued as inline asm so that the compiler's
// own wait insertion (which cannot tell the LDS stages apart and would wait
// for every load in flight before each LDS read) leaves these loads to the
// explicit per-stage waits of the kernel.
__device__ __forceinline__ void load_lds16(const void* base, uint32_t off_bytes, uint32_t lds) {
  asm volatile(
      "s_mov_b32 m0, %2\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %0, %1" ::"v"(off_bytes),
      "s"(base), "s"(__builtin_amdgcn_readfirstlane(lds))
      : "memory", "m0");
}
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return static_cast<uint32_t>(reinterpret_cast<uintptr_t>((lptr_t)(p)));
}

// s_waitcnt for at most n outstanding vector-memory operations (vmcnt bits
// [3:0] and [15:14]) and no outstanding LDS operation (lgkmcnt 0); expcnt is
// left at its maximum.
#define SPEC_WAIT_VM_LDS(n) __builtin_amdgcn_s_waitcnt(((n) & 15) | (((n) >> 4) << 14) | (7 << 4))

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, kWave));
  return v;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

// (value, index) max with ties to the lower index.
__device__ __forceinline__ void argmax_merge(float& v, int& i, float v2, int i2) {
  if (v2 > v || (v2 == v && i2 < i)) { v = v2; i = i2; }
}

__device__ __forceinline__ void wave_argmax(float& v, int& i) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    float v2 = __shfl_xor(v, o, kWave);
    int i2 = __shfl_xor(i, o, kWave);
    argmax_merge(v, i, v2, i2);
  }
}

}  // namespace spec
