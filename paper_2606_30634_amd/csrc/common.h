// Internal helpers shared by the gfx950 kernels and the host code of the stage library.
#pragma once
#include <hip/hip_runtime.h>
#include <cstdint>
#include <cstddef>

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

#define WAVE 64

// fp32 <-> storage conversions; the bf16 cast is round-to-nearest-even on gfx950.
__device__ __forceinline__ float to_f32(float v) { return v; }
__device__ __forceinline__ float to_f32(bf16 v) { return (float)v; }
template <typename T> __device__ __forceinline__ T from_f32(float v);
template <> __device__ __forceinline__ float from_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16 from_f32<bf16>(float v) { return (bf16)v; }

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, WAVE);
  return v;
}
__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, WAVE);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, WAVE));
  return v;
}

// Block-wide sum for blockDim.x a multiple of 64 (<= 1024); result valid in every thread.
template <typename T>
__device__ __forceinline__ T block_sum(T v, T* smem /* >= 16 entries */) {
  v = wave_sum(v);
  const int w = threadIdx.x / WAVE, l = threadIdx.x % WAVE, nw = blockDim.x / WAVE;
  __syncthreads();
  if (l == 0) smem[w] = v;
  __syncthreads();
  T r = 0;
  for (int i = 0; i < nw; ++i) r += smem[i];  // fixed order: deterministic
  return r;
}

static inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

// MFMA fragment (v_mfma_f32_32x32x16_bf16 operand) whose row index runs along the columns of a
// [k][row] LDS tile of pitch P elements: row r0 + lane mod 32, k = k0 + 8 (lane / 32) .. +7.
// ds_read_b64_tr_b16 lets each 16-lane group read a 4 x 16 block (lanes 4r..4r+3 supply row r,
// 4 consecutive elements each) and hands column j to lane j; two such reads give 8 k.
// Addresses must be 8-byte aligned (r0 and P multiples of 4).
typedef short v4i16_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ bf16x8 frag_tr(const bf16* T, int P, int r0, int k0) {
  const int l = threadIdx.x % 64, g = l / 16, i = l % 16;
  const int r = r0 + 16 * (g & 1) + 4 * (i & 3);
  const int k = k0 + 8 * (g >> 1) + (i >> 2);
  typedef __attribute__((address_space(3))) v4i16_t lds_v4i16;
  const v4i16_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(T + k * P + r));
  const v4i16_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)(T + (k + 4) * P + r));
  bf16x8 f;
  __builtin_memcpy(&f, &lo, 8);
  __builtin_memcpy(reinterpret_cast<char*>(&f) + 8, &hi, 8);
  return f;
}

// Compile-time loop: f(std::integral_constant<int, 0>) ... f(<N-1>).  Keeps register-array indices
// constant even where a loop body holds a barrier (which can stop the unroller).
#include <utility>
template <typename F, int... Is>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, Is...>) {
  (f(std::integral_constant<int, Is>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// ------------------------------------------------------------------ direct-to-LDS loads (gfx950)
// s_waitcnt: at most N vector-memory operations and no LDS operation outstanding
template <int N>
__device__ __forceinline__ void wait_vm_lds() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (0 << 8));
}

// One 16-byte global -> LDS load per lane from base + voff bytes (base wave-uniform; lane l
// writes lds + 16 l).  Issued as inline assembly so that the compiler neither counts it in its own
// waits nor orders LDS reads after it: a kernel waits for these loads itself (wait_vm_lds)
// before the barrier that publishes the LDS they fill.
__device__ __forceinline__ void dma16(const void* base, uint32_t voff, uint32_t lds) {
  asm volatile("global_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(base), "{m0}"(lds) : "memory");
}
// The same with 4 bytes per lane (lane l writes lds + 4 l).
__device__ __forceinline__ void dma4(const void* base, uint32_t voff, uint32_t lds) {
  asm volatile("global_load_lds_dword %0, %1" ::"v"(voff), "s"(base), "{m0}"(lds) : "memory");
}

__device__ __forceinline__ void block_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// LDS byte address of a pointer into __shared__ memory (the m0 operand of dma16 / dma4)
template <typename T>
__device__ __forceinline__ uint32_t lds_addr(const T* p) {
  typedef __attribute__((address_space(3))) const T lds_t;
  return (uint32_t)(uintptr_t)(lds_t*)p;
}
