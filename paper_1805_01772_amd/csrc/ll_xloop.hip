// XCD-local variants of the two device-side loops.
//
// MI355X has 8 XCDs of 32 CUs; each XCD has its own L2, shared by its CUs.
// Here the 32 work-groups resident on one XCD form a group that runs the
// recurrence of its own batch rows (row tiles x, x+8, ... for XCD x) and
// splits the hidden units 32 ways, so every value exchanged inside the loop
// (h_t forward, dz_t backward) moves only through that XCD's L2:
//   * producers write it with plain stores (the vector L1 writes through to
//     the L2);
//   * the arrays it lands in are filled with an all-ones pattern (a NaN
//     payload no arithmetic result carries: produced NaNs are stored in
//     canonical form) before the loop starts, and every element is written
//     exactly once per call;
//   * consumers read it with agent-scope atomic loads, which bypass the
//     CU's L1, and re-read any element that still holds the fill pattern.
// There is no grid barrier and no L2 writeback or invalidate in the loop:
// the data itself carries the readiness.  A work-group learns its XCD from
// the XCC_ID hardware register and its rank from a per-XCD counter, so the
// mapping does not depend on the dispatch order.
//
// Each work-group keeps its recurrent weight slice on chip for the whole
// loop, in registers (the first KSR k-steps of each wave's share; any rest in
// LDS).
#include "ll_kernels.h"

namespace ll {

namespace {

constexpr int kXccIdReg = (3 << 11) | 20;    // s_getreg: HW_REG_XCC_ID, bits [3:0]

__device__ __forceinline__ unsigned long long ld_u64_agent(const void* p) {
  return __hip_atomic_load(reinterpret_cast<const unsigned long long*>(p), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
}

// True if any element of the 8-byte word still holds the fill pattern.
template <typename T> __device__ __forceinline__ bool pending(unsigned long long v);
template <> __device__ __forceinline__ bool pending<bf16_t>(unsigned long long v) {
  const unsigned long long m = v & (v >> 1) & 0x7fff7fff7fff7fffull;   // low 15 bits all ones
  const unsigned long long t = m & (m >> 2);
  const unsigned long long t2 = t & (t >> 4);
  const unsigned long long t3 = t2 & (t2 >> 8);
  // element e is all-ones iff bit 0 of t3 (in its 16-bit lane) and bit 15 are set
  const unsigned long long full = t3 & (v >> 15) & 0x0001000100010001ull;
  return full != 0;
}
template <> __device__ __forceinline__ bool pending<float>(unsigned long long v) {
  return ((unsigned)v == 0xffffffffu) || ((unsigned)(v >> 32) == 0xffffffffu);
}

// Store forms of an exchanged value: NaN in canonical form (never all ones).
template <typename T> __device__ __forceinline__ T to_exchange(float v);
template <> __device__ __forceinline__ float to_exchange<float>(float v) {
  return v != v ? __uint_as_float(0x7fc00000u) : v;
}
template <> __device__ __forceinline__ bf16_t to_exchange<bf16_t>(float v) {
  return v != v ? (bf16_t)0x7fc0 : f32_to_bf16(v);
}

// 16-byte operand chunk from float data (h0 at step 0), converted.
template <typename T> __device__ __forceinline__ uint4 xchunk_from_f32(const float* p);
template <> __device__ __forceinline__ uint4 xchunk_from_f32<float>(const float* p) {
  return ld16(p);
}
template <> __device__ __forceinline__ uint4 xchunk_from_f32<bf16_t>(const float* p) {
  const float4 a = *reinterpret_cast<const float4*>(p);
  const float4 b = *reinterpret_cast<const float4*>(p + 4);
  uint4 r;
  r.x = (uint32_t)f32_to_bf16(a.x) | ((uint32_t)f32_to_bf16(a.y) << 16);
  r.y = (uint32_t)f32_to_bf16(a.z) | ((uint32_t)f32_to_bf16(a.w) << 16);
  r.z = (uint32_t)f32_to_bf16(b.x) | ((uint32_t)f32_to_bf16(b.y) << 16);
  r.w = (uint32_t)f32_to_bf16(b.z) | ((uint32_t)f32_to_bf16(b.w) << 16);
  return r;
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

}  // namespace

size_t xfwd_lds(int KSW, int KSR, int NCT) {
  const int KSL = KSW > KSR ? KSW - KSR : 0;
  return (size_t)4 * KSL * NCT * 64 * 16 + (size_t)3 * NCT * 256 * sizeof(float);
}
size_t xbwd_lds(int KSW, int KSR, int NCT) {
  const int KSL = KSW > KSR ? KSW - KSR : 0;
  size_t red = (size_t)4 * NCT * 256 * sizeof(float);
  const size_t dbr = (size_t)16 * 4 * 16 * NCT * sizeof(float);
  if (red < dbr) red = dbr;
  return (size_t)4 * KSL * NCT * 64 * 16 + red;
}

// ---------------------------------------------------------------------------
// Forward loop, XCD-local.  Member `rank` of XCD x owns hidden units
// j0 .. j0+HJ-1 (HJ = 4 NCT: all four gates of each unit, NCT column tiles of
// 16 gate columns) of the rows in tiles x, x+8, ...  Step t for a row tile:
//   poll h_{t-1} rows (K split across the 4 waves) while the next step's
//   input projections are prefetched, z = Zx + h W_h (MFMA), add the other
//   waves' partial products in LDS (one round), cell update in the waves that
//   own complete units (all four gates of 16 units each, lane-local), push
//   the stack, write h_t (history = exchange) and y_t.
// ---------------------------------------------------------------------------
template <typename T, int NCT, int KSW, int KSR, int MRT_MAX>
__global__ __launch_bounds__(256, 1) void xfwd_kernel(XLoopArgs a) {
  extern __shared__ uint4 lds[];
  __shared__ int s_info[2];
  constexpr int KPC = Op<T>::kPerChunk;
  constexpr int HJ = 4 * NCT;
  constexpr int NCW = NCT / 4;                 // waves that own complete units
  constexpr int KSL = KSW > KSR ? KSW - KSR : 0;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int q = lane >> 4, l16 = lane & 15;

  join_group(a.rank_ctr, s_info);
  const int grp = s_info[0], rank = s_info[1];
  if (grp >= 8 || rank >= 32) {
    if (tid == 0) {
      __hip_atomic_fetch_or(a.err, LL_DEVERR_BARRIER_BIT, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(a.abort_flag, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    return;
  }
  if (rank >= a.P) return;
  const int H = a.H, B = a.B;
  const long G4 = 4L * H;
  const int j0 = rank * HJ;
  const int KS = H / (4 * KPC);
  const int ks0 = min(KS, wave * KSW), ks1 = min(KS, ks0 + KSW);
  const T* WT = reinterpret_cast<const T*>(a.W);
  T* HH = reinterpret_cast<T*>(a.X);

  // Weight slice: column tile ct, lane column l16 <-> local gate column
  // ct*16 + l16 = gate * HJ + u.
  uint4 wr[NCT][KSR];
#pragma unroll
  for (int ct = 0; ct < NCT; ++ct) {
    const int c = ct * 16 + l16;
    const int gate = c / HJ, u = c - gate * HJ;
    const T* wcol = WT + ((long)gate * H + j0 + u) * a.ldw + a.woff;
#pragma unroll
    for (int i = 0; i < KSR; ++i) {
      const int ks = ks0 + i;
      wr[ct][i] = ks < ks1 ? ld16(wcol + (ks * 4 + q) * KPC) : zero4();
    }
#pragma unroll
    for (int i = 0; i < KSL; ++i) {
      const int ks = ks0 + KSR + i;
      lds[((wave * KSL + i) * NCT + ct) * 64 + lane] = ks < ks1 ? ld16(wcol + (ks * 4 + q) * KPC) : zero4();
    }
  }
  // partial products of the non-owning waves: slot (ct, s), s < 3
  float* red = reinterpret_cast<float*>(lds + 4 * KSL * NCT * 64);

  // Cell waves: lane (l16, q) owns unit ju and rows 4q + i of every tile.
  const bool cellw = wave < NCW;
  const int ju = j0 + 16 * wave + l16;
  int pr[MRT_MAX][4];
  float hs[MRT_MAX][4], cs[MRT_MAX][4];
#pragma unroll
  for (int mt = 0; mt < MRT_MAX; ++mt)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = (grp + 8 * mt) * 16 + 4 * q + i;
      pr[mt][i] = (mt < a.MRT && r < B) ? a.perm[r] : -1;
      hs[mt][i] = 0.f;
      cs[mt][i] = 0.f;
      if (cellw && pr[mt][i] >= 0) {
        if (a.h0) hs[mt][i] = a.h0[(long)pr[mt][i] * H + ju];
        if (a.c0) cs[mt][i] = a.c0[(long)pr[mt][i] * H + ju];
      }
    }
  __syncthreads();

  const int T_eff = a.meta[0];
  int A_t = a.active[0], off_t = a.off[0], off_p = 0;
  float zx[MRT_MAX][4][4];
#pragma unroll
  for (int mt = 0; mt < MRT_MAX; ++mt)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = (grp + 8 * mt) * 16 + 4 * q + i;
#pragma unroll
      for (int g = 0; g < 4; ++g)
        zx[mt][i][g] = (cellw && mt < a.MRT && r < A_t && T_eff > 0)
                           ? a.Zx[(off_t + r) * G4 + (long)g * H + ju] : 0.f;
    }

  for (int t = 0; t < T_eff; ++t) {
    const int A_n = a.active[t + 1];
    const int off_n = a.off[t + 1];
    float zn[MRT_MAX][4][4];
#pragma unroll
    for (int mt = 0; mt < MRT_MAX; ++mt)
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int g = 0; g < 4; ++g) zn[mt][i][g] = 0.f;
    bool fetched = false;
#pragma unroll
    for (int mt = 0; mt < MRT_MAX; ++mt) {
      if (mt >= a.MRT) continue;
      const int r0 = (grp + 8 * mt) * 16;
      if (r0 >= A_t) {
        if (cellw && a.y) {
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (pr[mt][i] >= 0) a.y[((long)t * B + pr[mt][i]) * H + ju] = 0.f;
        }
        continue;
      }
      // 1. issue the loads of h_{t-1} (this wave's k-steps)
      const int ar = r0 + l16;
      const bool aok = ar < A_t;
      const T* src[KSW];
      unsigned long long lo[KSW], hi[KSW];
#pragma unroll
      for (int i = 0; i < KSW; ++i) {
        const int ks = ks0 + i;
        src[i] = (t > 0 && aok && ks < ks1) ? HH + (long)(off_p + ar) * H + (ks * 4 + q) * KPC : nullptr;
        lo[i] = src[i] ? ld_u64_agent(src[i]) : 0ull;
        hi[i] = src[i] ? ld_u64_agent(src[i] + 8 / sizeof(T)) : 0ull;
      }
      // 2. prefetch the next step's input projections (issued after step 1)
      if (!fetched) {
        fetched = true;
#pragma unroll
        for (int m2 = 0; m2 < MRT_MAX; ++m2)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int r = (grp + 8 * m2) * 16 + 4 * q + i;
            if (cellw && m2 < a.MRT && r < A_n) {
#pragma unroll
              for (int g = 0; g < 4; ++g) zn[m2][i][g] = a.Zx[(off_n + r) * G4 + (long)g * H + ju];
            }
          }
      }
      // 3. complete h_{t-1}: re-read anything that still holds the fill pattern
      uint4 av[KSW];
      unsigned todo = 0;
#pragma unroll
      for (int i = 0; i < KSW; ++i) {
        av[i] = make_uint4((unsigned)lo[i], (unsigned)(lo[i] >> 32), (unsigned)hi[i], (unsigned)(hi[i] >> 32));
        if (src[i] && (pending<T>(lo[i]) || pending<T>(hi[i]))) todo |= 1u << i;
      }
      if (t == 0) {
#pragma unroll
        for (int i = 0; i < KSW; ++i) {
          const int ks = ks0 + i;
          av[i] = (aok && ks < ks1 && a.h0)
                      ? xchunk_from_f32<T>(a.h0 + (long)a.perm[ar] * H + (ks * 4 + q) * KPC)
                      : zero4();
        }
      }
      if (todo) {
        const unsigned long long t0 = wall_clock64();
        unsigned polls = 0;
        while (todo) {
          __builtin_amdgcn_s_sleep(1);
#pragma unroll
          for (int i = 0; i < KSW; ++i) {
            if (todo & (1u << i)) {
              const unsigned long long l2 = ld_u64_agent(src[i]);
              const unsigned long long h2 = ld_u64_agent(src[i] + 8 / sizeof(T));
              av[i] = make_uint4((unsigned)l2, (unsigned)(l2 >> 32), (unsigned)h2, (unsigned)(h2 >> 32));
              if (!pending<T>(l2) && !pending<T>(h2)) todo &= ~(1u << i);
            }
          }
          if ((++polls & 255u) == 0) {
            if (__hip_atomic_load(a.abort_flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) break;
            if (wall_clock64() - t0 > a.limit) {
              __hip_atomic_fetch_or(a.err, LL_DEVERR_BARRIER_BIT, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
              __hip_atomic_store(a.abort_flag, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
              break;
            }
          }
        }
      }
      // 4. partial product over this wave's k-steps
      f32x4 acc[NCT];
#pragma unroll
      for (int ct = 0; ct < NCT; ++ct) acc[ct] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int i = 0; i < KSW; ++i) {
        if (ks0 + i < ks1) {
#pragma unroll
          for (int ct = 0; ct < NCT; ++ct) {
            const uint4 bv = i < KSR ? wr[ct][i < KSR ? i : 0]
                                     : lds[((wave * KSL + (i - KSR)) * NCT + ct) * 64 + lane];
            acc[ct] = Mfma<T>::step(av[i], bv, acc[ct]);
          }
        }
      }
      // 5. partial products of non-owners -> LDS; owners add them
#pragma unroll
      for (int ct = 0; ct < NCT; ++ct) {
        const int owner = ct % NCW;
        if (wave != owner) {
          const int slot = ct * 3 + (wave - (wave > owner ? 1 : 0));
#pragma unroll
          for (int e = 0; e < 4; ++e) red[(slot * 4 + e) * 64 + lane] = acc[ct][e];
        }
      }
      __syncthreads();
      if (cellw) {
        float z[4][4];    // [gate][row slot]
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int ct = g * NCW + (NCW == 2 ? (wave & 1) : 0);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            float v = acc[ct][e];
            v += red[((ct * 3 + 0) * 4 + e) * 64 + lane];
            v += red[((ct * 3 + 1) * 4 + e) * 64 + lane];
            v += red[((ct * 3 + 2) * 4 + e) * 64 + lane];
            z[g][e] = v;
          }
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int r = r0 + 4 * q + i;
          if (pr[mt][i] < 0) continue;
          float* yrow = a.y ? a.y + ((long)t * B + pr[mt][i]) * H : nullptr;
          if (r < A_t) {
            const long krow = off_t + r;
            const float ig = sigmoidf_(z[0][i] + zx[mt][i][0]);
            const float fg = sigmoidf_(z[1][i] + zx[mt][i][1]);
            const float gg = tanhf_(z[2][i] + zx[mt][i][2]);
            const float og = sigmoidf_(z[3][i] + zx[mt][i][3]);
            const float cn = fg * cs[mt][i] + ig * gg;
            const float hn = og * tanhf_(cn);
            HH[krow * H + ju] = to_exchange<T>(hn);
            if (a.stack) {
              float* st = a.stack + krow * 5 * H;
              st[ju] = ig;
              st[H + ju] = fg;
              st[2 * H + ju] = gg;
              st[3 * H + ju] = og;
              st[4 * H + ju] = cn;
            }
            cs[mt][i] = cn;
            hs[mt][i] = hn;
            if (yrow) yrow[ju] = hn;
          } else if (yrow) {
            yrow[ju] = 0.f;
          }
        }
      }
      __syncthreads();
    }
    off_p = off_t;
    off_t = off_n;
    A_t = A_n;
#pragma unroll
    for (int mt = 0; mt < MRT_MAX; ++mt)
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int g = 0; g < 4; ++g) zx[mt][i][g] = zn[mt][i][g];
  }

  if (cellw) {
#pragma unroll
    for (int mt = 0; mt < MRT_MAX; ++mt)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if (pr[mt][i] < 0) continue;
        const long b = pr[mt][i];
        a.hT[b * H + ju] = hs[mt][i];
        a.cT[b * H + ju] = cs[mt][i];
        if (a.y)
          for (int t = T_eff; t < a.T_max; ++t) a.y[((long)t * B + b) * H + ju] = 0.f;
      }
  }
}

// ---------------------------------------------------------------------------
// Gradient loop, XCD-local.  Member `rank` owns hidden units j0 .. j0+HJ-1
// (HJ = 16 NCT).  Step t (descending) for a row tile:
//   phase 1 (own units, from values prefetched during step t+1): dz and dc,
//     write dz (the exchange array), accumulate db;
//   phase 2: poll the dz rows of the tile (all 4H gate columns, K split
//     across the 4 waves, two batches) while the stack rows of step t-1 are
//     prefetched; dh <- dz W_h^T for the own units (MFMA); one LDS round adds
//     the 4 partial products.
// ---------------------------------------------------------------------------
template <typename T, int NCT, int KSW, int KSR, int MRT_MAX>
__global__ __launch_bounds__(256, 1) void xbwd_kernel(XLoopArgs a) {
  extern __shared__ uint4 lds[];
  __shared__ int s_info[2];
  constexpr int KPC = Op<T>::kPerChunk;
  constexpr int HJ = 16 * NCT;                 // units per work-group
  constexpr int EPT = HJ / 16;                 // elements per thread per tile
  constexpr int KSL = KSW > KSR ? KSW - KSR : 0;
  constexpr int KB = KSW < 16 ? KSW : 16;      // k-steps per load batch
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int q = lane >> 4, l16 = lane & 15;

  join_group(a.rank_ctr, s_info);
  const int grp = s_info[0], rank = s_info[1];
  if (grp >= 8 || rank >= 32) {
    if (tid == 0) {
      __hip_atomic_fetch_or(a.err, LL_DEVERR_BARRIER_BIT, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(a.abort_flag, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    return;
  }
  if (rank >= a.P) return;
  const int H = a.H, B = a.B;
  const long G4 = 4L * H;
  const long H5 = 5L * H;
  const int j0 = rank * HJ;
  const int KS = (int)(G4 / (4 * KPC));
  const int ks0 = min(KS, wave * KSW), ks1 = min(KS, ks0 + KSW);
  const T* W = reinterpret_cast<const T*>(a.W);
  T* DZ = reinterpret_cast<T*>(a.X);

  // W_h row of output column ct*16 + l16 (a hidden unit of this member)
  uint4 wr[NCT][KSR];
#pragma unroll
  for (int ct = 0; ct < NCT; ++ct) {
    const T* wrow = W + (long)(a.woff + j0 + ct * 16 + l16) * G4;
#pragma unroll
    for (int i = 0; i < KSR; ++i) {
      const int ks = ks0 + i;
      wr[ct][i] = ks < ks1 ? ld16(wrow + (ks * 4 + q) * KPC) : zero4();
    }
#pragma unroll
    for (int i = 0; i < KSL; ++i) {
      const int ks = ks0 + KSR + i;
      lds[((wave * KSL + i) * NCT + ct) * 64 + lane] = ks < ks1 ? ld16(wrow + (ks * 4 + q) * KPC) : zero4();
    }
  }
  float* red = reinterpret_cast<float*>(lds + 4 * KSL * NCT * 64);   // [4 waves][NCT][4][64]

  // element k of a tile for this thread: e = tid + 256 k -> (row e / HJ, unit e % HJ)
  int pr[MRT_MAX][EPT];
  float dh[MRT_MAX][EPT], dc[MRT_MAX][EPT];
#pragma unroll
  for (int mt = 0; mt < MRT_MAX; ++mt)
#pragma unroll
    for (int k = 0; k < EPT; ++k) {
      const int e = tid + 256 * k;
      const int r = (grp + 8 * mt) * 16 + e / HJ;
      const int j = j0 + e % HJ;
      pr[mt][k] = (mt < a.MRT && r < B) ? a.perm[r] : -1;
      dh[mt][k] = 0.f;
      dc[mt][k] = 0.f;
      if (pr[mt][k] >= 0) {
        if (a.dhT) dh[mt][k] = a.dhT[(long)pr[mt][k] * H + j];
        if (a.dcT) dc[mt][k] = a.dcT[(long)pr[mt][k] * H + j];
      }
    }
  float dbacc[EPT][4];
#pragma unroll
  for (int k = 0; k < EPT; ++k)
#pragma unroll
    for (int g = 0; g < 4; ++g) dbacc[k][g] = 0.f;

  // popped values of a (step, tile): i, f, g, o, c_t, c_{t-1}, dy
  auto fetch = [&](float (&v)[EPT][7], int tt, int mt, int A, int off, int offp) {
#pragma unroll
    for (int k = 0; k < EPT; ++k) {
      const int e = tid + 256 * k;
      const int r = (grp + 8 * mt) * 16 + e / HJ;
      const int j = j0 + e % HJ;
#pragma unroll
      for (int c = 0; c < 7; ++c) v[k][c] = 0.f;
      if (tt >= 0 && r < A) {
        const float* st = a.stack + (off + r) * H5;
        v[k][0] = st[j];
        v[k][1] = st[H + j];
        v[k][2] = st[2 * H + j];
        v[k][3] = st[3 * H + j];
        v[k][4] = st[4 * H + j];
        if (tt > 0) v[k][5] = a.stack[(long)(offp + r) * H5 + 4 * H + j];
        else if (a.c0) v[k][5] = a.c0[(long)pr[mt][k] * H + j];
        if (a.dy)
          v[k][6] = a.dy_compact ? a.dy[(long)(off + r) * H + j]
                                 : a.dy[((long)tt * B + pr[mt][k]) * H + j];
      }
    }
  };

  const int T_eff = a.meta[0];
  int t = T_eff - 1;
  int A_t = t >= 0 ? a.active[t] : 0;
  int off_t = t >= 0 ? a.off[t] : 0;
  int off_p = t >= 1 ? a.off[t - 1] : 0;
  float pv[MRT_MAX][EPT][7];
#pragma unroll
  for (int mt = 0; mt < MRT_MAX; ++mt)
    if (mt < a.MRT) fetch(pv[mt], t, mt, A_t, off_t, off_p);
  __syncthreads();

  for (; t >= 0; --t) {
    const int A_n = t >= 1 ? a.active[t - 1] : 0;
    const int off_n = off_p;
    const int off_pn = t >= 2 ? a.off[t - 2] : 0;
#pragma unroll
    for (int mt = 0; mt < MRT_MAX; ++mt) {
      if (mt >= a.MRT) continue;
      const int r0 = (grp + 8 * mt) * 16;
      if (r0 >= A_t) {
        // rows of this tile may start running at step t-1 (lengths >= t)
        fetch(pv[mt], t - 1, mt, A_n, off_n, off_pn);
        continue;
      }
      // phase 1
#pragma unroll
      for (int k = 0; k < EPT; ++k) {
        const int e = tid + 256 * k;
        const int r = r0 + e / HJ;
        if (r >= A_t) continue;
        const int j = j0 + e % HJ;
        const long krow = off_t + r;
        const float dht = dh[mt][k] + pv[mt][k][6];
        const float ig = pv[mt][k][0], fg = pv[mt][k][1], gg = pv[mt][k][2], og = pv[mt][k][3];
        const float c = pv[mt][k][4], cp = pv[mt][k][5];
        const float tc = tanhf_(c);
        const float d_o = dht * tc;
        const float dct = dc[mt][k] + dht * og * (1.f - tc * tc);
        const float dz0 = dct * gg * (ig * (1.f - ig));
        const float dz1 = dct * cp * (fg * (1.f - fg));
        const float dz2 = dct * ig * (1.f - gg * gg);
        const float dz3 = d_o * (og * (1.f - og));
        T* dzr = DZ + krow * G4;
        dzr[j] = to_exchange<T>(dz0);
        dzr[H + j] = to_exchange<T>(dz1);
        dzr[2 * H + j] = to_exchange<T>(dz2);
        dzr[3 * H + j] = to_exchange<T>(dz3);
        dbacc[k][0] += dz0;
        dbacc[k][1] += dz1;
        dbacc[k][2] += dz2;
        dbacc[k][3] += dz3;
        dc[mt][k] = dct * fg;
      }
      // phase 2
      const int ar = r0 + l16;
      const T* arow = ar < A_t ? DZ + (long)(off_t + ar) * G4 : nullptr;
      f32x4 acc[NCT];
#pragma unroll
      for (int ct = 0; ct < NCT; ++ct) acc[ct] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int b0 = 0; b0 < KSW; b0 += KB) {
        const T* src[KB];
        unsigned long long lo[KB], hi[KB];
#pragma unroll
        for (int i = 0; i < KB; ++i) {
          const int ks = ks0 + b0 + i;
          src[i] = (arow && b0 + i < KSW && ks < ks1) ? arow + (ks * 4 + q) * KPC : nullptr;
          lo[i] = src[i] ? ld_u64_agent(src[i]) : 0ull;
          hi[i] = src[i] ? ld_u64_agent(src[i] + 8 / sizeof(T)) : 0ull;
        }
        if (b0 == 0) fetch(pv[mt], t - 1, mt, A_n, off_n, off_pn);   // next step's pops
        uint4 av[KB];
        unsigned todo = 0;
#pragma unroll
        for (int i = 0; i < KB; ++i) {
          av[i] = make_uint4((unsigned)lo[i], (unsigned)(lo[i] >> 32), (unsigned)hi[i], (unsigned)(hi[i] >> 32));
          if (src[i] && (pending<T>(lo[i]) || pending<T>(hi[i]))) todo |= 1u << i;
        }
        if (todo) {
          const unsigned long long t0 = wall_clock64();
          unsigned polls = 0;
          while (todo) {
            __builtin_amdgcn_s_sleep(1);
#pragma unroll
            for (int i = 0; i < KB; ++i) {
              if (todo & (1u << i)) {
                const unsigned long long l2 = ld_u64_agent(src[i]);
                const unsigned long long h2 = ld_u64_agent(src[i] + 8 / sizeof(T));
                av[i] = make_uint4((unsigned)l2, (unsigned)(l2 >> 32), (unsigned)h2, (unsigned)(h2 >> 32));
                if (!pending<T>(l2) && !pending<T>(h2)) todo &= ~(1u << i);
              }
            }
            if ((++polls & 255u) == 0) {
              if (__hip_atomic_load(a.abort_flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) break;
              if (wall_clock64() - t0 > a.limit) {
                __hip_atomic_fetch_or(a.err, LL_DEVERR_BARRIER_BIT, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                __hip_atomic_store(a.abort_flag, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                break;
              }
            }
          }
        }
#pragma unroll
        for (int i = 0; i < KB; ++i) {
          const int ii = b0 + i;
          if (ii < KSW && ks0 + ii < ks1) {
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct) {
              const uint4 bv = ii < KSR ? wr[ct][ii < KSR ? ii : 0]
                                        : lds[((wave * KSL + (ii - KSR)) * NCT + ct) * 64 + lane];
              acc[ct] = Mfma<T>::step(av[i], bv, acc[ct]);
            }
          }
        }
      }
#pragma unroll
      for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
        for (int e = 0; e < 4; ++e) red[((wave * NCT + ct) * 4 + e) * 64 + lane] = acc[ct][e];
      __syncthreads();
#pragma unroll
      for (int k = 0; k < EPT; ++k) {
        const int e = tid + 256 * k;
        const int row = e / HJ, u = e - (e / HJ) * HJ;
        if (r0 + row >= A_t) continue;
        // element (row, u): column tile u/16, lane (row/4)*16 + u%16, slot row%4
        const int ct = u >> 4, ln = (row >> 2) * 16 + (u & 15), ee = row & 3;
        float s = red[((0 * NCT + ct) * 4 + ee) * 64 + ln];
        s += red[((1 * NCT + ct) * 4 + ee) * 64 + ln];
        s += red[((2 * NCT + ct) * 4 + ee) * 64 + ln];
        s += red[((3 * NCT + ct) * 4 + ee) * 64 + ln];
        dh[mt][k] = s;
      }
      __syncthreads();
    }
    A_t = A_n;
    off_t = off_n;
    off_p = off_pn;
  }

#pragma unroll
  for (int mt = 0; mt < MRT_MAX; ++mt)
#pragma unroll
    for (int k = 0; k < EPT; ++k) {
      if (pr[mt][k] < 0) continue;
      const long b = pr[mt][k];
      const int j = j0 + (tid + 256 * k) % HJ;
      if (a.dh0) a.dh0[b * H + j] = dh[mt][k];
      if (a.dc0) a.dc0[b * H + j] = dc[mt][k];
    }
  // db partial of this work-group (its rows of this XCD), fixed order
  __syncthreads();
#pragma unroll
  for (int k = 0; k < EPT; ++k) {
    const int e = tid + 256 * k;
#pragma unroll
    for (int g = 0; g < 4; ++g) red[(e / HJ) * 4 * HJ + g * HJ + e % HJ] = dbacc[k][g];
  }
  __syncthreads();
  for (int c = tid; c < 4 * HJ; c += 256) {
    float s = 0.f;
    for (int m = 0; m < 16; ++m) s += red[m * 4 * HJ + c];
    const int g = c / HJ, u = c - (c / HJ) * HJ;
    a.db_part[(long)grp * G4 + (long)g * H + j0 + u] = s;
  }
}

// Fill rows [0, total) of a compact array of `row_bytes`-byte rows with the
// all-ones pattern.  row_bytes % 16 == 0.
__global__ __launch_bounds__(256) void fill_pending_kernel(uint4* base, long row_chunks,
                                                           const int* meta) {
  const long n = (long)meta[1] * row_chunks;
  const uint4 ones = make_uint4(~0u, ~0u, ~0u, ~0u);
  for (long i = blockIdx.x * 256L + threadIdx.x; i < n; i += gridDim.x * 256L) base[i] = ones;
}

// ------------------------------------------------------------ launchers
namespace {

}  // namespace

// Kernel for a (dtype, H class, row tiles per XCD) combination.
//   bf16: HJ = 32 units, forward NCT 8, KSW = H/128; backward NCT 2, KSW = H/32.
//   f32:  HJ = 16 units, forward NCT 4, KSW = H/64;  backward NCT 1, KSW = H/16.
// hc in {1, 2, 4, 8} is the forward KSW; mrt <= 4 row tiles per XCD.  The
// register-resident share of the weight slice (KSR of KSW k-steps per wave)
// is chosen per instantiation so that nothing spills to scratch.
namespace {
template <typename T, int NF, int NB, int HC, int RF, int RB, int MRT>
XKernels x_make() {
  XKernels k{};
  k.fwd = reinterpret_cast<const void*>(&xfwd_kernel<T, NF, HC, RF, MRT>);
  k.bwd = reinterpret_cast<const void*>(&xbwd_kernel<T, NB, 4 * HC, RB, MRT>);
  k.lds_fwd = xfwd_lds(HC, RF, NF);
  k.lds_bwd = xbwd_lds(4 * HC, RB, NB);
  return k;
}
}  // namespace

template <typename T>
XKernels x_kernels(int hc, int mrt) {
  constexpr bool bf = sizeof(T) == 2;
  constexpr int NF = bf ? 8 : 4;
  constexpr int NB = bf ? 2 : 1;
  const bool one = mrt <= 1;
  if (mrt > 4) return XKernels{};
  if constexpr (bf) {
    switch (hc) {
      case 1: return one ? x_make<T, NF, NB, 1, 1, 4, 1>() : x_make<T, NF, NB, 1, 1, 4, 4>();
      case 2: return one ? x_make<T, NF, NB, 2, 2, 8, 1>() : x_make<T, NF, NB, 2, 2, 8, 4>();
      case 4: return one ? x_make<T, NF, NB, 4, 4, 16, 1>() : x_make<T, NF, NB, 4, 2, 16, 4>();
      case 8: return one ? x_make<T, NF, NB, 8, 8, 24, 1>() : x_make<T, NF, NB, 8, 4, 16, 4>();
      default: return XKernels{};
    }
  } else {
  switch (hc) {
    case 1: return one ? x_make<T, NF, NB, 1, 1, 4, 1>() : x_make<T, NF, NB, 1, 1, 4, 4>();
    case 2: return one ? x_make<T, NF, NB, 2, 2, 8, 1>() : x_make<T, NF, NB, 2, 2, 8, 4>();
    case 4: return one ? x_make<T, NF, NB, 4, 4, 16, 1>() : x_make<T, NF, NB, 4, 4, 16, 4>();
    case 8: return one ? x_make<T, NF, NB, 8, 8, 32, 1>() : x_make<T, NF, NB, 8, 8, 24, 4>();
    default: return XKernels{};
  }
  }
}

template XKernels x_kernels<float>(int, int);
template XKernels x_kernels<bf16_t>(int, int);

hipError_t x_setup(const XKernels& k, int* occ_fwd, int* occ_bwd) {
  // a variant that spills registers to scratch memory is not used
  hipFuncAttributes fa{}, fb{};
  hipError_t e = hipFuncGetAttributes(&fa, k.fwd);
  if (e != hipSuccess) return e;
  e = hipFuncGetAttributes(&fb, k.bwd);
  if (e != hipSuccess) return e;
  if (fa.localSizeBytes > 0 || fb.localSizeBytes > 0) {
    *occ_fwd = 0;
    *occ_bwd = 0;
    return hipSuccess;
  }
  e = hipFuncSetAttribute(k.fwd, hipFuncAttributeMaxDynamicSharedMemorySize, (int)k.lds_fwd);
  if (e != hipSuccess) return e;
  e = hipFuncSetAttribute(k.bwd, hipFuncAttributeMaxDynamicSharedMemorySize, (int)k.lds_bwd);
  if (e != hipSuccess) return e;
  e = hipOccupancyMaxActiveBlocksPerMultiprocessor(occ_fwd, k.fwd, 256, k.lds_fwd);
  if (e != hipSuccess) return e;
  return hipOccupancyMaxActiveBlocksPerMultiprocessor(occ_bwd, k.bwd, 256, k.lds_bwd);
}

hipError_t x_launch(const void* fn, const XLoopArgs& a, int nwg, size_t lds, hipStream_t s) {
  XLoopArgs copy = a;
  void* kargs[] = {&copy};
  return hipLaunchCooperativeKernel(fn, dim3(nwg), dim3(256), kargs, (unsigned)lds, s);
}

hipError_t launch_fill_pending(void* base, long row_bytes, const int* meta, long cap_rows,
                               hipStream_t s) {
  const long chunks = cap_rows * (row_bytes / 16);
  long blocks = (chunks + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(fill_pending_kernel, dim3((unsigned)blocks), dim3(256), 0, s,
                     reinterpret_cast<uint4*>(base), row_bytes / 16, meta);
  return hipGetLastError();
}

}  // namespace ll
