// Device-side helpers shared by the lstmloop kernels (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ll {

typedef uint16_t bf16_t;   // raw bfloat16 bits
typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8_t;
typedef __attribute__((ext_vector_type(4))) float f32x4;

// ---------------------------------------------------------------- bf16
__device__ __forceinline__ float bf16_to_f32(bf16_t v) {
  return __uint_as_float(((uint32_t)v) << 16);
}

// float -> bfloat16, round to nearest even (NaN kept quiet).
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (bf16_t)((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (bf16_t)(u >> 16);
}

// Element-type traits: storage of matrix-core operands.
template <typename T> struct Op;
template <> struct Op<float> {
  static constexpr int kPerChunk = 4;            // elements per 16-byte chunk
  __device__ static __forceinline__ float load(const float* p) { return *p; }
  __device__ static __forceinline__ float to_f32(float v) { return v; }
  __device__ static __forceinline__ float from_f32(float v) { return v; }
};
template <> struct Op<bf16_t> {
  static constexpr int kPerChunk = 8;
  __device__ static __forceinline__ float to_f32(bf16_t v) { return bf16_to_f32(v); }
  __device__ static __forceinline__ bf16_t from_f32(float v) { return f32_to_bf16(v); }
};

// One "k-step": every lane supplies one 16-byte chunk of A and of B.
// bf16: one 16x16x32 MFMA.  f32: four 16x16x4 MFMAs; element j of the lane's
// chunk is the lane's k-slot in the j-th instruction (A and B use the same
// assignment, so the sum over k is unchanged).
template <typename T> struct Mfma;
template <> struct Mfma<bf16_t> {
  __device__ static __forceinline__ f32x4 step(uint4 a, uint4 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(
        __builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
  }
};
template <> struct Mfma<float> {
  __device__ static __forceinline__ f32x4 step(uint4 a, uint4 b, f32x4 c) {
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), c, 0, 0, 0);
    return c;
  }
};

// ----------------------------------------------------- activations
// sigmoid(u) = 1 / (1 + e^-u) on the hardware exponential and reciprocal:
// relative error about (|u| / 2 + 4) float ulps (the rounding of the
// exponent's argument grows with |u|); saturates correctly (e^x -> inf or 0).
__device__ __forceinline__ float sigmoidf_(float u) {
  return __builtin_amdgcn_rcpf(1.0f + __expf(-u));
}
// tanh(u) = 1 - 2 / (1 + e^{2u}) for |u| >= 1/8, which saturates correctly
// but near 0 keeps only an absolute error of about one ulp of 1; below 1/8
// the odd Taylor series of tanh to the u^7 term (u - u^3/3 + 2u^5/15 -
// 17u^7/315, truncation below 2e-9 relative there), so the relative error
// stays a few ulps down to the smallest normal inputs.  Both forms are
// evaluated and one is selected: no branch.
__device__ __forceinline__ float tanhf_(float u) {
  const float big = 1.0f - 2.0f * __builtin_amdgcn_rcpf(1.0f + __expf(2.0f * u));
  const float u2 = u * u;
  const float small = u + u * u2 * (-0.333333343f + u2 * (0.133333340f + u2 * -0.0539682545f));
  return __builtin_fabsf(u) < 0.125f ? small : big;
}

__device__ __forceinline__ uint4 zero4() { return make_uint4(0u, 0u, 0u, 0u); }

__device__ __forceinline__ uint4 ld16(const void* p) {
  return *reinterpret_cast<const uint4*>(p);
}

// ------------------------------------------------------ grid barrier
// All work-groups of a cooperative launch arrive on a monotonically growing
// counter; barrier number k (0-based) completes when the counter reaches
// (k + 1) * nwg.  The arrival is an agent-scope release; the waiter polls
// with relaxed agent-scope loads and then issues an agent-scope acquire
// fence.  A wait longer than `limit` wall-clock ticks sets LL_DEVERR_BARRIER
// in *err and raises *abort_flag (cleared before every launch sequence);
// every later wait then returns at once, so the grid always drains.
struct GridBarrier {
  unsigned* ctr;
  int* abort_flag;
  int* err;
  unsigned nwg;
  unsigned count;   // barriers passed so far by this work-group
  uint64_t limit;   // wall_clock64() ticks
};

__device__ __forceinline__ void grid_sync(GridBarrier& gb) {
  gb.count += 1;
  __syncthreads();
  if (threadIdx.x == 0) {
    const unsigned target = gb.count * gb.nwg;
    __hip_atomic_fetch_add(gb.ctr, 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
    if (__hip_atomic_load(gb.abort_flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0) {
      const uint64_t t0 = wall_clock64();
      unsigned polls = 0;
      while (__hip_atomic_load(gb.ctr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target) {
        __builtin_amdgcn_s_sleep(1);
        if ((++polls & 1023u) == 0) {
          if (__hip_atomic_load(gb.abort_flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0) break;
          if (wall_clock64() - t0 > gb.limit) {
            __hip_atomic_fetch_or(gb.err, 2, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(gb.abort_flag, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            break;
          }
        }
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
  }
  __syncthreads();
}

}  // namespace ll
