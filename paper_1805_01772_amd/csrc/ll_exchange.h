// Device helpers of the exchange loops (XCD-local and chip-wide): work-group
// identity from the XCC_ID register, buffer loads with explicit cache policy,
// flag publication and bounded flag waits.
#pragma once

#include "ll_kernels.h"

namespace ll {

constexpr int kXccIdReg = (3 << 11) | 20;    // s_getreg: HW_REG_XCC_ID, bits [3:0]

// Wave-uniform copy of a value every lane holds (keeps it in a scalar
// register, so buffer descriptors built from it stay scalar).
__device__ __forceinline__ int uni(int v) { return __builtin_amdgcn_readfirstlane(v); }

// Raw buffer resource over `bytes` bytes from `base` (stride 0; reads past
// the end return zeros).  Both arguments must be the same on every lane; they
// are read from the first lane so that the descriptor lives in scalar
// registers.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, unsigned bytes) {
  const unsigned long long p = reinterpret_cast<unsigned long long>(base);
  const unsigned lo = __builtin_amdgcn_readfirstlane((unsigned)p);
  const unsigned hi = __builtin_amdgcn_readfirstlane((unsigned)(p >> 32));
  void* pb = reinterpret_cast<void*>(((unsigned long long)hi << 32) | lo);
  return __builtin_amdgcn_make_buffer_rsrc(pb, (short)0, (int)__builtin_amdgcn_readfirstlane(bytes),
                                           0x00020000);
}
// 16-byte read with cache policy sc1 (device scope): it bypasses the CU's L1
// and sees what other CUs of the same XCD stored in the L2, and what CUs of
// other XCDs stored with device-scope stores (st_dev); data that nobody
// rewrites is still served at L2 bandwidth (measured).
constexpr int kCpolSc1 = 16;
__device__ __forceinline__ uint4 ld_chunk_l2(__amdgpu_buffer_rsrc_t r, unsigned off) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kCpolSc1));
}
// 4-byte read with cache policy sc1 (served by the L2, like ld_chunk_l2).
__device__ __forceinline__ float ld_f32_l2(__amdgpu_buffer_rsrc_t r, unsigned off) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, kCpolSc1));
}
// Plain 4-byte read through a buffer descriptor.
__device__ __forceinline__ float ld_f32(__amdgpu_buffer_rsrc_t r, unsigned off) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
}
// Plain 16-byte read of four floats through a buffer descriptor.
__device__ __forceinline__ float4 ld_f32x4(__amdgpu_buffer_rsrc_t r, unsigned off) {
  return __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}
// Offset past every buffer range used here: a lane with nothing to read
// loads from it and gets zeros, so no load needs a per-lane branch.
constexpr unsigned kOOB = 0x80000000u;

// Every vector memory operation of the wave done (vmcnt(0)), through the
// builtin: the compiler's own wait tracking then knows that every earlier
// load has landed.  (An inline-asm wait is opaque to it: after one, it waited
// again for loads issued before it, at a point where that also meant waiting
// for every store issued since.)  The empty asm statements keep the
// compiler from moving memory operations across the wait.
__device__ __forceinline__ void wait_all_vm() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xF70);   // vmcnt(0); expcnt, lgkmcnt: no wait
  asm volatile("" ::: "memory");
}

// Group of this work-group: (XCD, rank within the XCD).
__device__ __forceinline__ void join_group(unsigned* rank_ctr, int* s_info) {
  if (threadIdx.x == 0) {
    const int x = __builtin_amdgcn_s_getreg(kXccIdReg) & 15;
    s_info[0] = x;
    s_info[1] = (int)atomicAdd(rank_ctr + (x & 7), 1u);
  }
  __syncthreads();
}

// Publish: every wave waits until its stores are acknowledged by the L2, the
// work-group meets, and thread 0 stores `value` into the flag.  The flag
// store has work-group scope (cache policy sc0): the CU's vector L1 is
// write-through, so the store reaches the XCD's L2, where the consumers
// (CUs of the same XCD) poll with sc1 loads.  An agent-scope store (sc1) is
// written through past the L2 and was measured to slow the loops down
// (forward 0.58 -> 0.75 ms, gradient 0.75 -> 1.47 ms at the H = 1024
// workload); consumers on other XCDs use publish_dev.
__device__ __forceinline__ void publish(unsigned* flag, unsigned value) {
  wait_all_vm();
  __syncthreads();
  if (threadIdx.x == 0) __hip_atomic_store(flag, value, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

// Publish to every XCD: as publish, with a device-scope flag store (the
// data must have been stored with st_dev).
__device__ __forceinline__ void publish_dev(unsigned* flag, unsigned value) {
  wait_all_vm();
  __syncthreads();
  if (threadIdx.x == 0) __hip_atomic_store(flag, value, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Wait until flags[p(l)] >= need for the lanes l < n (p(l) = (p0 + l) % P),
// with the loop's wall-clock limit and abort flag.
template <typename Args>
__device__ __forceinline__ void wait_flags(const Args& a, const unsigned* flags, int p0, int n,
                                           int P, unsigned need) {
  const int lane = threadIdx.x & 63;
  const unsigned* fp = flags + (p0 + (lane < n ? lane : 0)) % P;
  unsigned long long t0 = 0;
  unsigned polls = 0;
  while (true) {
    const unsigned f = __hip_atomic_load(fp, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (__builtin_amdgcn_ballot_w64(lane < n && f < need) == 0) return;
    if (polls == 0) t0 = wall_clock64();
    __builtin_amdgcn_s_sleep(1);
    if ((++polls & 255u) == 0) {
      if (__hip_atomic_load(a.abort_flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) return;
      if (wall_clock64() - t0 > a.limit) {
        __hip_atomic_fetch_or(a.err, LL_DEVERR_BARRIER_BIT, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(a.abort_flag, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        return;
      }
    }
  }
}


// Wait until flags[idx] >= need for every lane with `mine` set (each lane
// names its own flag), with the loop's wall-clock limit and abort flag.
template <typename Args>
__device__ __forceinline__ void wait_each(const Args& a, const unsigned* flags, int idx, bool mine,
                                          unsigned need) {
  const unsigned* fp = flags + (mine ? idx : 0);
  unsigned long long t0 = 0;
  unsigned polls = 0;
  while (true) {
    const unsigned f = __hip_atomic_load(fp, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (__builtin_amdgcn_ballot_w64(mine && f < need) == 0) return;
    if (polls == 0) t0 = wall_clock64();
    __builtin_amdgcn_s_sleep(1);
    if ((++polls & 255u) == 0) {
      if (__hip_atomic_load(a.abort_flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) return;
      if (wall_clock64() - t0 > a.limit) {
        __hip_atomic_fetch_or(a.err, LL_DEVERR_BARRIER_BIT, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(a.abort_flag, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        return;
      }
    }
  }
}

// Stores with cache policy sc1 (device scope): written through to the point
// where loads of every XCD see them.
constexpr int kCpolStoreDev = 16;
__device__ __forceinline__ void st_dev(__amdgpu_buffer_rsrc_t r, unsigned off, float v) {
  __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), r, off, 0, kCpolStoreDev);
}
__device__ __forceinline__ void st_dev(__amdgpu_buffer_rsrc_t r, unsigned off, bf16_t v) {
  __builtin_amdgcn_raw_buffer_store_b16(v, r, off, 0, kCpolStoreDev);
}

}  // namespace ll
