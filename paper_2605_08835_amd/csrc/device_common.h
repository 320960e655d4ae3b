// Device-side helpers shared by the kernels: element types, 8-wide vector
// loads/stores with conversion to fp32, and wavefront reductions (wave64).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sd {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// 8 consecutive elements <-> 8 floats.
__device__ inline void load8f(const float* p, float v[8]) {
  float4 a = *reinterpret_cast<const float4*>(p);
  float4 b = *reinterpret_cast<const float4*>(p + 4);
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
  v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}
__device__ inline void load8f(const bf16* p, float v[8]) {
  bf16x8 a = *reinterpret_cast<const bf16x8*>(p);
#pragma unroll
  for (int i = 0; i < 8; ++i) v[i] = (float)a[i];
}
__device__ inline void store8f(float* p, const float v[8]) {
  *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
  *reinterpret_cast<float4*>(p + 4) = make_float4(v[4], v[5], v[6], v[7]);
}
__device__ inline void store8f(bf16* p, const float v[8]) {
  bf16x8 a;
#pragma unroll
  for (int i = 0; i < 8; ++i) a[i] = (bf16)v[i];
  *reinterpret_cast<bf16x8*>(p) = a;
}

template <typename T> __device__ inline float to_f(T x) { return (float)x; }
template <typename T> __device__ inline T from_f(float x) { return (T)x; }

// x sigmoid(x) with the hardware reciprocal (1 ulp) instead of a division.
__device__ inline float silu_f(float x) { return x * __builtin_amdgcn_rcpf(1.0f + __expf(-x)); }

// GELU(x) = x Phi(x), Phi(x) = (1 + erf(x / sqrt 2)) / 2, with erf from
// Abramowitz & Stegun 7.1.26 (absolute error below 1.5e-7, far under a
// bf16 rounding): for u >= 0, 1 - erf(u) = t (a1 + t (a2 + t (a3 + t (a4 +
// t a5)))) exp(-u^2), t = 1 / (1 + p u).  A reciprocal and an exp2 are its
// only transcendental instructions, against a library erff's piecewise
// polynomials; the bf16 GEGLU epilogues use it.  The 1/sqrt(2) of u and
// the 1/2 of h are folded into the constants (p / sqrt 2, a_i / 2).
__device__ inline float gelu_as(float x) {
  const float t = __builtin_amdgcn_rcpf(fmaf(0.23164193223f, fabsf(x), 1.0f));  // 1 / (1 + p u)
  float p = fmaf(t, 0.5307027145f, -0.7265760135f);
  p = fmaf(t, p, 0.7107068705f);
  p = fmaf(t, p, -0.142248368f);
  p = fmaf(t, p, 0.127414796f);
  // h = (1 - erf(u)) / 2 = t p exp(-u^2) with the halved a_i; exp(-u^2) = exp2(-x^2 log2(e) / 2)
  const float h = t * p * __builtin_amdgcn_exp2f(x * x * -0.72134752044448170f);
  return x * (x >= 0.f ? 1.0f - h : h);
}

__device__ inline float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ inline double wave_sum_d(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Buffer-resource loads: an offset at or past the resource's size reads as
// zero, so a masked-off element takes the offset OOB and no branch.
constexpr int OOB = (int)0x80000000u;

__device__ inline __amdgpu_buffer_rsrc_t make_rsrc(const void* base, long bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}
__device__ inline bf16x8 buf_load16(__amdgpu_buffer_rsrc_t r, int off) {
  return __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}

// One 16-byte-per-lane direct-to-LDS load (64 lanes -> 1 KB at `lds`).
// The builtin exists only for the device pass; the host pass of this file
// compiles the kernels' launch stubs and never runs this body.
__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t r, bf16* lds, int off) {
#if defined(__HIP_DEVICE_COMPILE__)
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, lds, 16, off, 0, 0, 0);
#endif
}

// Workgroup barrier for the direct-to-LDS pipelines.  __syncthreads()
// carries a workgroup release fence, for which the compiler waits for every
// outstanding load that writes LDS (vmcnt(0)), including the prefetches of
// later K stages, so each stage would have only one compute phase to land.
// The kernels instead wait with an explicit vmcnt for the loads of the stage
// they are about to read, then meet here: every wave's loads of that stage
// have landed once all waves have passed.  The empty asm statements keep
// the compiler from moving LDS accesses across the barrier.
__device__ __forceinline__ void stage_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

template <int WAITN>
__device__ __forceinline__ void wait_vmcnt() {
  // s_waitcnt with only the vector-memory counter limited to WAITN
  static_assert(WAITN >= 0 && WAITN < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((WAITN & 15) | (7 << 4) | (15 << 8) | ((WAITN >> 4) << 14));
}

// s_waitcnt with only the LDS / scalar-memory counter limited to 0
__device__ __forceinline__ void wait_lgkm0() {
  __builtin_amdgcn_s_waitcnt(15 | (7 << 4) | (0 << 8) | (3 << 14));
}

}  // namespace sd
