// Device-side types and helpers for gfx950 (CDNA4, 64-lane wavefronts).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace llmcad {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;

// D = A(16x32) * B(32x16) + C on the matrix cores, bf16 inputs, fp32 accumulate.
// Operand lanes: lane l holds row/column (l % 16) and the 8 k-slots of group
// (l / 16); A and B use the same k-slot assignment, so which physical k each
// slot carries is free as long as both operands agree.  Result: lane l holds
// D[4 * (l / 16) + i][l % 16], i = 0..3.
__device__ __forceinline__ f32x4 mfma16x16x32(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// Index of this thread's wavefront as a wave-uniform (scalar) value.  Every
// guard of a matrix-core instruction must be uniform in this sense: a guard
// the compiler sees as lane-divergent becomes an EXEC mask, the compiler may
// drop the skip branch around a short masked block, and a matrix instruction
// issued with EXEC all zero still updates its accumulator.
__device__ __forceinline__ int wave_index() {
  return __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
}
// A value the caller knows is the same in every lane of the wave, made
// scalar so that branches on it are scalar branches.
__device__ __forceinline__ int wave_uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }

// Global-memory access.  Pointers that reach a device function through a
// structure or a reference are generic to the compiler, and a generic access
// is a FLAT instruction, which counts on both the vector-memory and the
// out-of-order LDS/scalar counters: every wait for one of them then drains all
// loads in flight.  These casts make the access a global one (in-order vector
// counter only, so a pipeline can wait for its oldest stage alone).
// (The host pass of a HIP compile only type-checks device code; address
// spaces mean nothing there.)
#if defined(__HIP_DEVICE_COMPILE__)
#define LLMCAD_GLOBAL __attribute__((address_space(1)))
#define LLMCAD_CONSTANT __attribute__((address_space(4)))
#define LLMCAD_LDS __attribute__((address_space(3)))
#else
#define LLMCAD_GLOBAL
#define LLMCAD_CONSTANT
#define LLMCAD_LDS
#endif
template <class T>
__device__ __forceinline__ T ldg(const T* p) {
  return *(const LLMCAD_GLOBAL T*)p;
}
template <class T>
__device__ __forceinline__ void stg(T* p, const T& v) {
  *(LLMCAD_GLOBAL T*)p = v;
}
// LDS access through a pointer the compiler cannot trace to a __shared__
// object (a generic access would be FLAT, counted with global loads).
template <class T>
__device__ __forceinline__ T lds_ld(const void* p) {
  return *(const LLMCAD_LDS T*)p;
}
template <class T>
__device__ __forceinline__ void lds_st(void* p, const T& v) {
  *(LLMCAD_LDS T*)p = v;
}

__device__ __forceinline__ float bf2f(bf16 x) { return (float)x; }
__device__ __forceinline__ bf16 f2bf(float x) { return (bf16)x; }  // round to nearest even

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, kWave);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, kWave));
  return v;
}

// Max with the lowest index among equal values, across the wave.
__device__ __forceinline__ void wave_argmax(float& v, int& idx) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    float ov = __shfl_xor(v, off, kWave);
    int oi = __shfl_xor(idx, off, kWave);
    if (ov > v || (ov == v && oi < idx)) {
      v = ov;
      idx = oi;
    }
  }
}

// Lane moves inside each row of 16 lanes, on the vector ALU (DPP), for the
// epilogues' reductions and neighbour exchanges: a __shfl is a ds_bpermute,
// an LDS round trip, and a chain of dependent ones serialises.
constexpr int kDppQuadXor1 = 0xB1;       // quad_perm [1,0,3,2]: reads lane ^ 1
constexpr int kDppQuadXor2 = 0x4E;       // quad_perm [2,3,0,1]: reads lane ^ 2
constexpr int kDppRowShl1 = 0x101;       // row_shl:1: lane i of a row reads lane i + 1 (lane 15 gets 0)
constexpr int kDppRowRor8 = 0x128;       // row_ror:8: reads lane (i + 8) mod 16, i.e. lane ^ 8
constexpr int kDppRowMirror = 0x140;     // reads lane 15 - i of the row
constexpr int kDppRowHalfMirror = 0x141; // reads lane 7 - i of the half row
template <int CTRL>
__device__ __forceinline__ int dpp_i(int v) {
  return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xF, 0xF, false);
}
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __int_as_float(dpp_i<CTRL>(__float_as_int(v)));
}
// Sum over the 16 lanes of each row (quads first, then half rows, then the
// row); every lane gets the same bits (each step adds a pair in both orders).
__device__ __forceinline__ float row16_sum(float v) {
  v += dpp_f<kDppQuadXor1>(v);
  v += dpp_f<kDppQuadXor2>(v);
  v += dpp_f<kDppRowHalfMirror>(v);
  v += dpp_f<kDppRowMirror>(v);
  return v;
}
// Across rows: the values of lanes l and l ^ 16 (l ^ 32) of the wave, from
// one gfx950 permlane swap of the value with itself (lane l gets both of its
// pair, in an order that depends on l), on the vector ALU.
__device__ __forceinline__ void pair_xor16(float v, float& a, float& b) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  a = __uint_as_float(r[0]);
  b = __uint_as_float(r[1]);
}
__device__ __forceinline__ void pair_xor32(float v, float& a, float& b) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  a = __uint_as_float(r[0]);
  b = __uint_as_float(r[1]);
}
// Max / sum over lanes l, l ^ 16, l ^ 32, l ^ 48 (a column of the wave's four
// rows), xor 16 first: the same bits as v op shfl_xor(v, 16), then 32.
__device__ __forceinline__ float col4_max(float v) {
  float a, b;
  pair_xor16(v, a, b);
  v = fmaxf(a, b);
  pair_xor32(v, a, b);
  return fmaxf(a, b);
}
__device__ __forceinline__ float col4_sum(float v) {
  float a, b;
  pair_xor16(v, a, b);
  v = a + b;
  pair_xor32(v, a, b);
  return a + b;
}
// Max with the lowest index among equal values, over the 16 lanes of each row.
template <int CTRL>
__device__ __forceinline__ void argmax_step(float& v, int& idx) {
  const float ov = dpp_f<CTRL>(v);
  const int oi = dpp_i<CTRL>(idx);
  if (ov > v || (ov == v && oi < idx)) {
    v = ov;
    idx = oi;
  }
}
__device__ __forceinline__ void row16_argmax(float& v, int& idx) {
  argmax_step<kDppQuadXor1>(v, idx);
  argmax_step<kDppQuadXor2>(v, idx);
  argmax_step<kDppRowHalfMirror>(v, idx);
  argmax_step<kDppRowMirror>(v, idx);
}

// Workgroup barrier for LDS hand-offs only: waits for this wave's LDS
// accesses, not for its global loads (__syncthreads also drains every global
// load in flight, which would defeat a prefetch issued before it).
__device__ __forceinline__ void lds_barrier() {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0); vmcnt and expcnt left alone
  __builtin_amdgcn_s_barrier();
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// Hand-off between workgroups of one launch without L2 maintenance.
//
// A full device-scope fence on this GPU writes back and invalidates the
// XCD's L2, which costs far more than the data it protects.  Instead, data
// read by another workgroup of the same launch is written with
// device-coherent stores and read with device-coherent loads (relaxed
// device-scope atomics: they bypass non-coherent L2 state), and
// arrive_last only has to wait until this workgroup's stores have completed
// before counting its arrival with a device-scope atomic.
__device__ __forceinline__ void st_coherent(float* p, float v) {
  __hip_atomic_store((LLMCAD_GLOBAL float*)p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_coherent(int* p, int v) {
  __hip_atomic_store((LLMCAD_GLOBAL int*)p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_coherent2(float* p, float a, float b) {  // p 8-byte aligned
  const uint64_t bits = (uint64_t)__float_as_uint(a) | ((uint64_t)__float_as_uint(b) << 32);
  __hip_atomic_store((LLMCAD_GLOBAL uint64_t*)p, bits, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_coherent_bf2(bf16* p, float a, float b) {  // p 4-byte aligned
  const uint32_t lo = (uint32_t)__builtin_bit_cast(uint16_t, f2bf(a));
  const uint32_t hi = (uint32_t)__builtin_bit_cast(uint16_t, f2bf(b));
  __hip_atomic_store((LLMCAD_GLOBAL uint32_t*)p, lo | (hi << 16), __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_coherent_bf(bf16* p, float a) {  // p 2-byte aligned
  __hip_atomic_store((LLMCAD_GLOBAL uint16_t*)p, __builtin_bit_cast(uint16_t, f2bf(a)), __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float ld_coherent(const float* p) {
  return __hip_atomic_load((const LLMCAD_GLOBAL float*)p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ int ld_coherent(const int* p) {
  return __hip_atomic_load((const LLMCAD_GLOBAL int*)p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float2 ld_coherent2(const float* p) {  // p 8-byte aligned
  const uint64_t bits =
      __hip_atomic_load((const LLMCAD_GLOBAL uint64_t*)p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return make_float2(__uint_as_float((uint32_t)bits), __uint_as_float((uint32_t)(bits >> 32)));
}
// Device-scope counter updates.
__device__ __forceinline__ int atomic_add_dev(int* p, int v) {
  return __hip_atomic_fetch_add((LLMCAD_GLOBAL int*)p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Counts this workgroup's arrival on `counter`; returns true (to every
// thread) in the last of `expected` arriving workgroups, which also resets
// the counter.  The caller's cross-workgroup data must have been written
// with st_coherent*; the last workgroup reads it with ld_coherent*.  Must be
// called by all threads of the workgroup.
__device__ __forceinline__ bool arrive_last(int* counter, int expected, int* lds_flag) {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);  // keep the stores above in program order
  __builtin_amdgcn_s_waitcnt(0);            // and wait until they have completed
  __syncthreads();
  if (threadIdx.x == 0) {
    const int old = atomic_add_dev(counter, 1);
    const int last = (old == expected - 1);
    if (last) st_coherent(counter, 0);
    *lds_flag = last;
  }
  __syncthreads();
  return *lds_flag != 0;
}

}  // namespace llmcad
