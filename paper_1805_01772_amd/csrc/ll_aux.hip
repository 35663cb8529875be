// Small kernels around the loops: trip count and length ordering, operand
// transposes, zero fill of finished rows, deterministic reductions.
#include <algorithm>

#include "ll_kernels.h"

namespace ll {

// ---------------------------------------------------------------------------
// Loop preparation (one work-group; any size up to 1024 threads).
//   * range check of seq_len; a bad length sets LL_DEVERR_SEQ_LEN and makes
//     the loops run zero iterations (every length treated as 0);
//   * T_eff = max_b seq_len[b]: the loop predicate is t < T_eff, decided here
//     on the device, and it is also the iteration count the gradient loop
//     replays (the forward loop counter of the loop gradient);
//   * perm: batch rows ordered by decreasing length (ties by index), so the
//     rows still running at step t are the prefix r < active[t];
//   * off[t] = sum_{t' < t} active[t']: rows of step t occupy compact rows
//     off[t] .. off[t] + active[t] - 1 of every per-step array (stack,
//     history, pre-activations, dz);  meta[1] = off[T_max] = sum of lengths;
//   * rowmap[k] = t * B + perm[r] for compact row k = off[t] + r.
//   * clears the barrier counters and the abort flag of this launch sequence.
// ---------------------------------------------------------------------------
__device__ void prep_body(const PrepArgs& a, int* smem) {
  const int* __restrict__ seq_len = a.seq_len;
  const int B = a.B, T_max = a.T_max, t_in_lds = a.t_in_lds, n_pow2 = a.n_pow2;
  int* __restrict__ perm = a.perm;
  int* __restrict__ active = a.active;
  int* __restrict__ off = a.off;
  int* __restrict__ rowmap = a.rowmap;
  int* __restrict__ meta = a.meta;
  int* __restrict__ trip_out = a.trip_out;
  // sort keys: (T_max - length) << 32 | row, ascending = decreasing length,
  // ties by row index; entries n_pow2 > B pad with the largest key
  unsigned long long* s_key = reinterpret_cast<unsigned long long*>(smem);   // [n_pow2]
  int* s_act = smem + 2 * n_pow2; // [T_max + 1] when t_in_lds
  int* s_off = s_act + T_max + 1; // [T_max + 1] when t_in_lds
  __shared__ int s_bad;
  __shared__ int s_wsum[16];
  __shared__ int s_carry;
  const int tid = threadIdx.x, nt = blockDim.x;
  const int lane = tid & 63, wave = tid >> 6, nwaves = nt >> 6;
  if (tid == 0) { s_bad = 0; s_carry = 0; }
  __syncthreads();
  for (int b = tid; b < B; b += nt) {
    const int L = seq_len[b];
    if (L < 0 || L > T_max) s_bad = 1;
    s_key[b] = ((unsigned long long)(unsigned)(T_max - (L < 0 || L > T_max ? 0 : L)) << 32) | (unsigned)b;
  }
  for (int b = B + tid; b < n_pow2; b += nt) s_key[b] = ~0ull;
  __syncthreads();
  const int bad = s_bad;
  // bitonic sort of the n_pow2 keys (O(B log^2 B) compare-exchanges, all in LDS)
  for (int k = 2; k <= n_pow2; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int i = tid; i < n_pow2; i += nt) {
        const int ixj = i ^ j;
        if (ixj > i) {
          const unsigned long long u = s_key[i], v = s_key[ixj];
          const bool up = (i & k) == 0;
          if ((u > v) == up) {
            s_key[i] = v;
            s_key[ixj] = u;
          }
        }
      }
      __syncthreads();
    }
  }
  // sorted row r: perm[r] = row index, length T_max - (key >> 32) (0 for
  // every row when some length is out of range)
  auto s_perm = [&](int r) { return (int)(unsigned)(s_key[r] & 0xffffffffu); };
  auto s_sorted = [&](int r) { return bad ? 0 : T_max - (int)(unsigned)(s_key[r] >> 32); };
  for (int r = tid; r < B; r += nt) perm[r] = s_perm(r);
  const int T_eff = B > 0 ? s_sorted(0) : 0;
  // active[t] = #{r : sorted length > t}; lengths are non-increasing in r
  for (int t = tid; t <= T_max; t += nt) {
    int lo = 0, hi = B;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (s_sorted(mid) > t) lo = mid + 1; else hi = mid;
    }
    active[t] = lo;
    if (t_in_lds) s_act[t] = lo;
  }
  __syncthreads();
  // exclusive prefix sum of active[0..T_max) into off[0..T_max]
  for (int base = 0; base <= T_max; base += nt) {
    const int t = base + tid;
    const int v = (t < T_max) ? (t_in_lds ? s_act[t] : active[t]) : 0;
    int incl = v;
    for (int d = 1; d < 64; d <<= 1) {
      const int u = __shfl_up(incl, d, 64);
      if (lane >= d) incl += u;
    }
    if (lane == 63) s_wsum[wave] = incl;
    __syncthreads();
    int wpre = 0, tot = 0;
    for (int w = 0; w < nwaves; ++w) {
      const int s = s_wsum[w];
      if (w < wave) wpre += s;
      tot += s;
    }
    const int carry = s_carry;
    if (t <= T_max) {
      off[t] = carry + wpre + incl - v;
      if (t_in_lds) s_off[t] = carry + wpre + incl - v;
    }
    __syncthreads();
    if (tid == 0) s_carry = carry + tot;
    __syncthreads();
  }
  const int total = s_carry;
  // rowmap: compact row off[t] + r -> t * B + perm[r]; one wave per step
  for (int t = wave; t < T_eff; t += nwaves) {
    const int n = t_in_lds ? s_act[t] : active[t];
    const int o = t_in_lds ? s_off[t] : off[t];
    for (int r = lane; r < n; r += 64) rowmap[o + r] = t * B + s_perm(r);
  }
  if (tid == 0) {
    meta[0] = T_eff;
    meta[1] = total;
    meta[3] = 0;                       // abort flag
    for (int i = 4; i < META_INTS; ++i) meta[i] = 0;   // barrier and rank counters
    if (bad) atomicOr(&meta[2], LL_DEVERR_SEQ_LEN_BIT);
    if (trip_out) *trip_out = T_eff;
  }
}

// out[c * ldo + r] = in[r * ldi + c], r < R, c < C.
template <typename T>
__global__ __launch_bounds__(256) void transpose_kernel(const T* __restrict__ in, int R, int C,
                                                        int ldi, T* __restrict__ out, int ldo) {
  __shared__ T tile[64][65];
  const int r0 = blockIdx.y * 64, c0 = blockIdx.x * 64;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  for (int i = ty; i < 64; i += 4) {
    const int r = r0 + i, c = c0 + tx;
    if (r < R && c < C) tile[i][tx] = in[(long)r * ldi + c];
  }
  __syncthreads();
  for (int i = ty; i < 64; i += 4) {
    const int c = c0 + i, r = r0 + tx;
    if (c < C && r < R) out[(long)c * ldo + r] = tile[tx][i];
  }
}

// Gather compact rows and transpose: out[c * ldo + k] = src_k[c] for
// k < meta[1] (sum of lengths), c < C.  Source row of compact row k:
//   mode 0: in + rowmap[k] * C         (time-major input, original batch order)
//   mode 1: in + k * C                 (already compact)
//   mode 2: h_{t-1} of that row: t = rowmap[k] / B, r = k - off[t];
//           t > 0: in + (off[t-1] + r) * C (compact history of h);
//           t = 0: bf/fp conversion of h0f[perm[r] * C] (float, NULL = 0).
// A 64 x 64 tile per work-group, moved in 16-byte chunks both ways: thread
// (row k, chunk) loads KPC consecutive columns of one source row, the tile
// goes through LDS (row pitch padded by one chunk), and thread (column c,
// chunk) stores KPC consecutive k of one output row.  C is a multiple of KPC
// (the plan checks I and H), so no chunk straddles the end of a row; chunks
// of k past the sum of lengths are written as zeros.
template <typename T>
__global__ __launch_bounds__(256) void gather_transpose_kernel(GatherTArgs g) {
  constexpr int KPC = Op<T>::kPerChunk;
  constexpr int CPR = 64 / KPC;              // chunks per 64-element tile row
  __shared__ T tile[64][64 + KPC];
  const int total = g.meta[1];
  const int k0 = blockIdx.x * 64, c0 = blockIdx.y * 64;
  if (k0 >= total) return;
  const int tid = threadIdx.x;
  const T* in = reinterpret_cast<const T*>(g.in);
  for (int i = tid; i < 64 * CPR; i += 256) {
    const int kr = i / CPR, ch = i % CPR;
    const int k = k0 + kr, c = c0 + ch * KPC;
    uint4 v = zero4();
    if (k < total && c < g.C) {
      if (g.mode == 0) {
        v = ld16(in + (long)g.rowmap[k] * g.C + c);
      } else if (g.mode == 1) {
        v = ld16(in + (long)k * g.C + c);
      } else {
        const int t = g.rowmap[k] / g.B;
        const int r = k - g.off[t];
        if (t > 0) {
          v = ld16(in + (long)(g.off[t - 1] + r) * g.C + c);
        } else if (g.h0f) {
          const float* f = g.h0f + (long)g.perm[r] * g.C + c;
          T tmp[KPC];
#pragma unroll
          for (int e = 0; e < KPC; ++e) tmp[e] = Op<T>::from_f32(f[e]);
          __builtin_memcpy(&v, tmp, 16);
        }
      }
    }
    __builtin_memcpy(&tile[kr][ch * KPC], &v, 16);
  }
  __syncthreads();
  T* out = reinterpret_cast<T*>(g.out);
  for (int i = tid; i < 64 * CPR; i += 256) {
    const int cr = i / CPR, ch = i % CPR;
    const int c = c0 + cr, k = k0 + ch * KPC;
    if (c >= g.C) continue;
    T tmp[KPC];
#pragma unroll
    for (int e = 0; e < KPC; ++e) tmp[e] = tile[ch * KPC + e][cr];
    uint4 v;
    __builtin_memcpy(&v, tmp, 16);
    *reinterpret_cast<uint4*>(out + (long)c * g.ldo + k) = v;
  }
}

// Zero the rows (t, b) of a [T_max, B, C] float array with t >= seq_len[b]
// (all rows if the lengths failed the range check).  C % 4 == 0.
// (The bodies of the small kernels take their work-group index and count,
// so that one launch can run several of them side by side.)
__device__ void zero_finished_rows_body(float* __restrict__ dst, int T_max, int B, int C,
                                        const int* __restrict__ seq_len, const int* __restrict__ meta,
                                        int bid, int nb) {
  const int bad = meta[2] & LL_DEVERR_SEQ_LEN_BIT;
  const long rows = (long)T_max * B;
  const int c4 = C >> 2;
  for (long row = bid * 4L + (threadIdx.x >> 6); row < rows; row += nb * 4L) {
    const int t = (int)(row / B), b = (int)(row % B);
    if (!bad && t < seq_len[b]) continue;
    float4* p = reinterpret_cast<float4*>(dst + row * C);
    for (int i = threadIdx.x & 63; i < c4; i += 64) p[i] = make_float4(0.f, 0.f, 0.f, 0.f);
  }
}
__global__ __launch_bounds__(256) void zero_finished_rows_kernel(float* __restrict__ dst, int T_max,
                                                                 int B, int C,
                                                                 const int* __restrict__ seq_len,
                                                                 const int* __restrict__ meta) {
  zero_finished_rows_body(dst, T_max, B, C, seq_len, meta, blockIdx.x, gridDim.x);
}

// Row maps of the gate recomputation (one thread per padded row (t, r)).
__global__ __launch_bounds__(256) void rc_maps_kernel(const int* __restrict__ active,
                                                      const int* __restrict__ off,
                                                      const int* __restrict__ perm, int B, int T_max,
                                                      long cap, int* __restrict__ xmap,
                                                      int* __restrict__ cmap, int* __restrict__ prevmap) {
  const long n = (long)T_max * B;
  for (long i = blockIdx.x * 256L + threadIdx.x; i < n; i += gridDim.x * 256L) {
    const int t = (int)(i / B), r = (int)(i % B);
    const bool run = r < active[t];
    xmap[i] = run ? t * B + perm[r] : 0;
    cmap[i] = run ? off[t] + r : 0;
    prevmap[i] = run ? (t > 0 ? (int)(off[t - 1] + r) : (int)(cap + r)) : (int)cap;
  }
}

__global__ __launch_bounds__(256) void prev_rows_kernel(const int* __restrict__ active,
                                                        const int* __restrict__ off, int B, int T_max,
                                                        long cap, int* __restrict__ prev) {
  prev_rows_body(active, off, B, T_max, cap, prev, blockIdx.x, gridDim.x, 256);
}

template <typename T>
__global__ __launch_bounds__(256) void h0_rows_kernel(const float* __restrict__ h0,
                                                      const int* __restrict__ perm, int B, int H,
                                                      T* __restrict__ dst) {
  h0_rows_body<T>(h0, perm, B, H, dst, blockIdx.x, gridDim.x, 256);
}

__global__ __launch_bounds__(256) void sum_slices_kernel(const float* __restrict__ ws, int S,
                                                         long stride, long n, long cols, long ldo,
                                                         float* __restrict__ out) {
  sum_slices_body(ws, S, stride, n, cols, ldo, out, blockIdx.x, gridDim.x, 256);
}

// out[r] = sum_k A[row(r)][k] * op(w[k]) for the compact rows r < meta[1]
// (row(r) = rowmap[r], or r without a map; op = rounding to the operand
// type): the input part of the cond body's predicate.  One wave per row;
// fixed summation order (lane partials, then a butterfly over the wave).
template <typename T>
__global__ __launch_bounds__(256) void row_dot_kernel(const T* __restrict__ A, int lda,
                                                      const int* __restrict__ rowmap,
                                                      const int* __restrict__ meta,
                                                      const float* __restrict__ w, int K,
                                                      float* __restrict__ out) {
  const int rows = meta[1];
  const int lane = threadIdx.x & 63;
  for (long r = blockIdx.x * 4L + (threadIdx.x >> 6); r < rows; r += gridDim.x * 4L) {
    const T* a = A + (long)(rowmap ? rowmap[r] : r) * lda;
    float p = 0.f;
    for (int k = lane; k < K; k += 64) p += Op<T>::to_f32(a[k]) * Op<T>::to_f32(Op<T>::from_f32(w[k]));
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) p += __shfl_xor(p, m, 64);
    if (lane == 0) out[r] = p;
  }
}

// dst[j][4 u + g] = W[row0 + j][g H + u] for j, u < H, g < 4: W_h in the
// unit-major reduction order of the single-layer LSTM gradient loop.
// One thread per (j, u): four coalesced reads (consecutive threads take
// consecutive u) and one 4-element store.
template <typename T>
__global__ __launch_bounds__(256) void permute_um_kernel(const T* __restrict__ W, int row0, int H,
                                                         T* __restrict__ dst) {
  permute_um_body<T>(W, row0, H, dst, blockIdx.x, gridDim.x, 256);
}

// float -> operand type copy (used for bf16(h0) and similar small arrays).
template <typename T>
__global__ __launch_bounds__(256) void convert_kernel(const float* __restrict__ in, long n,
                                                      T* __restrict__ out) {
  for (long i = blockIdx.x * 256L + threadIdx.x; i < n; i += gridDim.x * 256L)
    out[i] = Op<T>::from_f32(in[i]);
}

// Tile (r0, c0) of the transpose out[c * ldo + r] = in[r * ldi + c], r < R,
// c < C, 64 x 64 elements in 16-byte chunks both ways: thread (row, chunk)
// loads KPC consecutive columns of one input row into LDS (row pitch padded
// by one chunk), thread (column, chunk) stores KPC consecutive rows of one
// output row.  R, C, ldi and ldo are multiples of KPC and both arrays
// 16-byte aligned (the plan checks I and H; W and W^T are 16-byte aligned).
template <typename T>
__device__ void transpose_tile(const T* __restrict__ in, int R, int C, int ldi, T* __restrict__ out,
                               int ldo, int r0, int c0, T (*tile)[64 + Op<T>::kPerChunk]) {
  constexpr int KPC = Op<T>::kPerChunk;
  constexpr int CPR = 64 / KPC;
  for (int idx = threadIdx.x; idx < 64 * CPR; idx += blockDim.x) {
    const int i = idx / CPR, j = idx - i * CPR;
    const int r = r0 + i, c = c0 + j * KPC;
    uint4 v = zero4();
    if (r < R && c < C) v = *reinterpret_cast<const uint4*>(in + (long)r * ldi + c);
    T tmp[KPC];
    __builtin_memcpy(tmp, &v, 16);
#pragma unroll
    for (int e = 0; e < KPC; ++e) tile[i][j * KPC + e] = tmp[e];
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < 64 * CPR; idx += blockDim.x) {
    const int cl = idx / CPR, j = idx - cl * CPR;
    const int c = c0 + cl, r = r0 + j * KPC;
    if (c < C && r < R) {
      T tmp[KPC];
#pragma unroll
      for (int e = 0; e < KPC; ++e) tmp[e] = tile[j * KPC + e][cl];
      uint4 v;
      __builtin_memcpy(&v, tmp, 16);
      *reinterpret_cast<uint4*>(out + (long)c * ldo + r) = v;
    }
  }
  __syncthreads();   // the tile is free for the next one
}

// The forward's set-up in one launch: work-group 0 runs prep; the others
// transpose W of every layer into W^T (row n = gate column n), tile by tile.
template <typename T>
__global__ __launch_bounds__(512) void fwd_setup_kernel(FwdSetupArgs a) {
  extern __shared__ int smem[];
  if (blockIdx.x == 0) {
    prep_body(a.prep, smem);
    return;
  }
  __shared__ T tile[64][64 + Op<T>::kPerChunk];
  const int tiles = a.job[0].tiles + (a.njobs > 1 ? a.job[1].tiles : 0);
  for (int k = blockIdx.x - 1; k < tiles; k += gridDim.x - 1) {
    const int j = k < a.job[0].tiles ? 0 : 1;
    const TransposeJob& q = a.job[j];
    const int kk = k - (j ? a.job[0].tiles : 0);
    const int tr = kk / q.tiles_c, tc = kk - tr * q.tiles_c;
    transpose_tile<T>(static_cast<const T*>(q.in), q.R, q.C, q.ldi, static_cast<T*>(q.out), q.ldo, tr * 64,
                      tc * 64, tile);
  }
}

// Several independent small tasks in one launch, each on its own range of
// work-groups (a grid-stride loop over its range).
template <typename T>
__global__ __launch_bounds__(256) void small_tasks_kernel(SmallTasks ts) {
  int b = blockIdx.x, i = 0;
  while (i + 1 < ts.n && b >= ts.t[i].blocks) {
    b -= ts.t[i].blocks;
    ++i;
  }
  const SmallTask& k = ts.t[i];
  switch (k.kind) {
    case kTaskZeroU32: {
      unsigned* p = static_cast<unsigned*>(k.out);
      for (long j = b * 256L + threadIdx.x; j < k.l0; j += k.blocks * 256L) p[j] = 0u;
      break;
    }
    case kTaskZeroFinishedRows:
      zero_finished_rows_body(static_cast<float*>(k.out), k.i0, k.i1, k.i2, static_cast<const int*>(k.a),
                              static_cast<const int*>(k.b), b, k.blocks);
      break;
    case kTaskPermuteUm:
      permute_um_body<T>(static_cast<const T*>(k.a), k.i0, k.i1, static_cast<T*>(k.out), b, k.blocks, 256);
      break;
    case kTaskSumSlices:
      sum_slices_body(static_cast<const float*>(k.a), k.i0, k.l0, k.l1, k.l2, k.l3, static_cast<float*>(k.out), b,
                      k.blocks, 256);
      break;
    case kTaskPrevRows:
      prev_rows_body(static_cast<const int*>(k.a), static_cast<const int*>(k.b), k.i0, k.i1, k.l0,
                     static_cast<int*>(k.out), b, k.blocks, 256);
      break;
    case kTaskH0Rows:
      h0_rows_body<T>(static_cast<const float*>(k.a), static_cast<const int*>(k.b), k.i0, k.i1,
                      static_cast<T*>(k.out), b, k.blocks, 256);
      break;
    default:
      break;
  }
}

// ------------------------------------------------------------ launchers
template <typename T>
hipError_t launch_fwd_setup(const int* seq_len, int B, int T_max, int* perm, int* active, int* off,
                            int* rowmap, int* meta, int* trip_out, int nw, const T* const* W, const int* R,
                            int C, T* const* WT, hipStream_t s) {
  if (nw < 0 || nw > 2) return hipErrorInvalidValue;
  FwdSetupArgs a{};
  int n_pow2 = 1;
  while (n_pow2 < B) n_pow2 <<= 1;
  // sort keys (8 bytes per row, B <= 4096: at most 32 KB), and the per-step
  // counts and offsets when all fits in 64 KB
  const size_t keys = (size_t)n_pow2 * 8;
  const int t_in_lds = keys + 2 * ((size_t)T_max + 1) * sizeof(int) <= 64 * 1024;
  const size_t smem = keys + (t_in_lds ? 2 * ((size_t)T_max + 1) * sizeof(int) : 0);
  a.prep = PrepArgs{seq_len, B, T_max, perm, active, off, rowmap, meta, trip_out, t_in_lds, n_pow2};
  a.njobs = nw;
  long tiles = 0;
  for (int l = 0; l < nw; ++l) {
    TransposeJob& q = a.job[l];
    q.in = W[l];
    q.out = WT[l];
    q.R = R[l];
    q.C = C;
    q.ldi = C;
    q.ldo = R[l];
    q.tiles_c = (C + 63) / 64;
    q.tiles = ((R[l] + 63) / 64) * q.tiles_c;
    tiles += q.tiles;
  }
  // (four work-groups of 512 per compute unit fit the LDS of small shapes)
  const long nblk = 1 + std::min(tiles, 1024L);
  hipLaunchKernelGGL(fwd_setup_kernel<T>, dim3((unsigned)nblk), dim3(512), smem, s, a);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_small_tasks(const SmallTasks& ts, hipStream_t s) {
  if (ts.n <= 0) return hipSuccess;
  long nblk = 0;
  for (int i = 0; i < ts.n; ++i) nblk += ts.t[i].blocks;
  hipLaunchKernelGGL(small_tasks_kernel<T>, dim3((unsigned)nblk), dim3(256), 0, s, ts);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_transpose(const T* in, int R, int C, int ldi, T* out, int ldo, hipStream_t s) {
  dim3 grid((C + 63) / 64, (R + 63) / 64);
  hipLaunchKernelGGL(transpose_kernel<T>, grid, dim3(256), 0, s, in, R, C, ldi, out, ldo);
  return hipGetLastError();
}

// Sustained matrix-core rate: every wave runs 8 independent accumulator
// chains for `iters` rounds, of the 16x16 k-step the loops use
// (SHAPE32 = false: 16x16x32 bf16 / four 16x16x4 f32) or of the 32x32 shape
// (true: 32x32x16 bf16 / 32x32x2 f32).
template <typename T, bool SHAPE32>
__global__ __launch_bounds__(256) void mfma_peak_kernel(int iters, float* sink) {
  const uint4 a = make_uint4(0x3f803f80u + threadIdx.x, 0x3f803f80u, 0x3c003c00u, 0x3f803f80u);
  const uint4 b = make_uint4(0x3f803f80u, 0x3f803f80u + blockIdx.x, 0x3f803f80u, 0x3c003c00u);
  float s = 0.f;
  if constexpr (SHAPE32) {
    typedef __attribute__((ext_vector_type(16))) float f32x16;
    f32x16 acc[8];
#pragma unroll
    for (int c = 0; c < 8; ++c)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[c][e] = 0.f;
    for (int i = 0; i < iters; ++i) {
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        if constexpr (sizeof(T) == 2)
          acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                          __builtin_bit_cast(bf16x8_t, b), acc[c], 0, 0, 0);
        else
          acc[c] = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.x), __uint_as_float(b.y), acc[c], 0, 0, 0);
      }
    }
#pragma unroll
    for (int c = 0; c < 8; ++c) s += acc[c][0] + acc[c][15];
  } else {
    f32x4 acc[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) acc[c] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int i = 0; i < iters; ++i) {
#pragma unroll
      for (int c = 0; c < 8; ++c) acc[c] = Mfma<T>::step(a, b, acc[c]);
    }
#pragma unroll
    for (int c = 0; c < 8; ++c) s += acc[c][0] + acc[c][1] + acc[c][2] + acc[c][3];
  }
  if (s == 1234.5f) sink[threadIdx.x] = s;
}

// The cell's activation functions applied element-wise (fn 0: sigmoid,
// 1: tanh), for checking them against a float64 reference.
__global__ __launch_bounds__(256) void eval_activations_kernel(const float* __restrict__ in,
                                                               float* __restrict__ out, long n, int fn) {
  for (long i = blockIdx.x * 256L + threadIdx.x; i < n; i += (long)gridDim.x * 256) {
    const float u = in[i];
    out[i] = fn == 0 ? sigmoidf_(u) : tanhf_(u);
  }
}

hipError_t eval_activations(const float* in, float* out, long n, int fn, hipStream_t s) {
  long blocks = (n + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(eval_activations_kernel, dim3((unsigned)blocks), dim3(256), 0, s, in, out, n, fn);
  return hipGetLastError();
}

template <typename T>
hipError_t measure_mfma_peak(int n_cu, bool shape32, double* tflops) {
  // flops of one chain round: 16x16x32 bf16, four 16x16x4 f32, 32x32x16 bf16, one 32x32x2 f32
  const double flop_per_step = shape32 ? (sizeof(T) == 2 ? 32.0 * 32 * 16 * 2 : 32.0 * 32 * 2 * 2)
                                       : (sizeof(T) == 2 ? 16.0 * 16 * 32 * 2 : 4.0 * 16 * 16 * 4 * 2);
  const int iters = sizeof(T) == 2 ? 20000 : 2000;
  const int blocks = n_cu * 8;
  float* sink = nullptr;
  hipStream_t st = nullptr;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  hipError_t e = hipMalloc(&sink, 256 * sizeof(float));
  if (e == hipSuccess) e = hipStreamCreateWithFlags(&st, hipStreamNonBlocking);
  if (e == hipSuccess) e = hipEventCreate(&e0);
  if (e == hipSuccess) e = hipEventCreate(&e1);
  const void* fn = shape32 ? reinterpret_cast<const void*>(&mfma_peak_kernel<T, true>)
                           : reinterpret_cast<const void*>(&mfma_peak_kernel<T, false>);
  float ms = 0.f;
  int it = iters;
  float* sk = sink;
  void* kargs[] = {&it, &sk};
  for (int rep = 0; rep < 2 && e == hipSuccess; ++rep) {   // the first launch warms up
    e = hipLaunchKernel(fn, dim3(blocks), dim3(256), kargs, 0, st);
    if (e == hipSuccess) e = hipEventRecord(e0, st);
    if (e == hipSuccess) e = hipLaunchKernel(fn, dim3(blocks), dim3(256), kargs, 0, st);
    if (e == hipSuccess) e = hipEventRecord(e1, st);
    if (e == hipSuccess) e = hipEventSynchronize(e1);
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, e0, e1);
  }
  if (e == hipSuccess && ms > 0.f)
    *tflops = (double)blocks * 4 * 8 * iters * flop_per_step / (ms * 1e-3) / 1e12;
  if (e0) (void)hipEventDestroy(e0);
  if (e1) (void)hipEventDestroy(e1);
  if (st) (void)hipStreamDestroy(st);
  if (sink) (void)hipFree(sink);
  return e;
}
template hipError_t measure_mfma_peak<float>(int, bool, double*);
template hipError_t measure_mfma_peak<bf16_t>(int, bool, double*);

template <typename T>
hipError_t launch_gather_transpose(const GatherTArgs& g, int cap_rows, hipStream_t s) {
  dim3 grid((cap_rows + 63) / 64, (g.C + 63) / 64);
  hipLaunchKernelGGL(gather_transpose_kernel<T>, grid, dim3(256), 0, s, g);
  return hipGetLastError();
}

// out[rowmap[r] * C + c] = sum_k ws[k * stride + r * C + c] for the compact
// rows r < meta[1] (the sum over ponder slots of the nested-loop body's dx).
__global__ __launch_bounds__(256) void sum_scatter_rows_kernel(const float* __restrict__ ws, int nsl, long stride,
                                                               const int* __restrict__ meta,
                                                               const int* __restrict__ rowmap, int C,
                                                               float* __restrict__ out) {
  const long N = meta[1];
  const long total = N * C;
  for (long i = blockIdx.x * 256L + threadIdx.x; i < total; i += (long)gridDim.x * 256) {
    const long r = i / C, c = i - r * C;
    float v = 0.f;
    for (int k = 0; k < nsl; ++k) v += ws[k * stride + i];
    out[(long)rowmap[r] * C + c] = v;
  }
}

hipError_t launch_sum_scatter_rows(const float* ws, int nsl, long stride, const int* meta, const int* rowmap,
                                   int C, float* out, long cap_rows, hipStream_t s) {
  long blocks = (cap_rows * C + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(sum_scatter_rows_kernel, dim3((unsigned)blocks), dim3(256), 0, s, ws, nsl, stride, meta,
                     rowmap, C, out);
  return hipGetLastError();
}

hipError_t launch_zero_finished_rows(float* dst, int T_max, int B, int C, const int* seq_len,
                                     const int* meta, hipStream_t s) {
  const long rows = (long)T_max * B;
  int blocks = (int)((rows + 3) / 4);
  if (blocks > 8192) blocks = 8192;
  hipLaunchKernelGGL(zero_finished_rows_kernel, dim3(blocks), dim3(256), 0, s, dst, T_max, B, C,
                     seq_len, meta);
  return hipGetLastError();
}

hipError_t launch_rc_maps(const int* active, const int* off, const int* perm, int B, int T_max,
                          long cap, int* xmap, int* cmap, int* prevmap, hipStream_t s) {
  long blocks = ((long)T_max * B + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(rc_maps_kernel, dim3((unsigned)blocks), dim3(256), 0, s, active, off, perm, B,
                     T_max, cap, xmap, cmap, prevmap);
  return hipGetLastError();
}

hipError_t launch_prev_rows(const int* active, const int* off, int B, int T_max, long cap, int* prev,
                            hipStream_t s) {
  long blocks = ((long)T_max * B + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(prev_rows_kernel, dim3((unsigned)blocks), dim3(256), 0, s, active, off, B, T_max, cap,
                     prev);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_h0_rows(const float* h0, const int* perm, int B, int H, T* dst, hipStream_t s) {
  long blocks = ((long)B * H + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(h0_rows_kernel<T>, dim3((unsigned)blocks), dim3(256), 0, s, h0, perm, B, H, dst);
  return hipGetLastError();
}

hipError_t launch_sum_slices(const float* ws, int S, long stride, long n, float* out,
                             hipStream_t s) {
  return launch_sum_slices_2d(ws, S, stride, 1, n, out, n, s);
}

hipError_t launch_sum_slices_2d(const float* ws, int S, long stride, long rows, long cols, float* out,
                                long ldo, hipStream_t s) {
  const long n = rows * cols;
  if (cols < 1 || ldo < cols) return hipErrorInvalidValue;
  long blocks = (n + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(sum_slices_kernel, dim3((unsigned)blocks), dim3(256), 0, s, ws, S, stride, n,
                     cols, ldo, out);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_convert(const float* in, long n, T* out, hipStream_t s) {
  long blocks = (n + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(convert_kernel<T>, dim3((unsigned)blocks), dim3(256), 0, s, in, n, out);
  return hipGetLastError();
}

template hipError_t launch_fwd_setup<float>(const int*, int, int, int*, int*, int*, int*, int*, int*, int,
                                             const float* const*, const int*, int, float* const*, hipStream_t);
template hipError_t launch_fwd_setup<bf16_t>(const int*, int, int, int*, int*, int*, int*, int*, int*, int,
                                              const bf16_t* const*, const int*, int, bf16_t* const*, hipStream_t);
template <typename T>
__global__ __launch_bounds__(256) void pre_jobs_kernel(PreJobs j) {
  pre_jobs_body<T>(j, blockIdx.x, gridDim.x, 256);
}
template <typename T>
hipError_t launch_pre_jobs(const PreJobs& j, hipStream_t s) {
  hipLaunchKernelGGL(pre_jobs_kernel<T>, dim3(64), dim3(256), 0, s, j);
  return hipGetLastError();
}
template hipError_t launch_pre_jobs<float>(const PreJobs&, hipStream_t);
template hipError_t launch_pre_jobs<bf16_t>(const PreJobs&, hipStream_t);
template hipError_t launch_small_tasks<float>(const SmallTasks&, hipStream_t);
template hipError_t launch_small_tasks<bf16_t>(const SmallTasks&, hipStream_t);
template hipError_t launch_transpose<float>(const float*, int, int, int, float*, int, hipStream_t);
template hipError_t launch_transpose<bf16_t>(const bf16_t*, int, int, int, bf16_t*, int,
                                             hipStream_t);
template hipError_t launch_gather_transpose<float>(const GatherTArgs&, int, hipStream_t);
template hipError_t launch_gather_transpose<bf16_t>(const GatherTArgs&, int, hipStream_t);
template hipError_t launch_h0_rows<float>(const float*, const int*, int, int, float*, hipStream_t);
template hipError_t launch_h0_rows<bf16_t>(const float*, const int*, int, int, bf16_t*, hipStream_t);
template <typename T>
hipError_t launch_row_dot(const T* A, int lda, const int* rowmap, const int* meta, long cap, const float* w,
                          int K, float* out, hipStream_t s) {
  long blocks = (cap + 3) / 4;
  if (blocks > 4096) blocks = 4096;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(row_dot_kernel<T>, dim3((unsigned)blocks), dim3(256), 0, s, A, lda, rowmap, meta, w, K,
                     out);
  return hipGetLastError();
}
template hipError_t launch_row_dot<float>(const float*, int, const int*, const int*, long, const float*, int,
                                          float*, hipStream_t);
template hipError_t launch_row_dot<bf16_t>(const bf16_t*, int, const int*, const int*, long, const float*, int,
                                           float*, hipStream_t);
template <typename T>
hipError_t launch_permute_um(const T* W, int row0, int H, T* dst, hipStream_t s) {
  long blocks = ((long)H * H + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(permute_um_kernel<T>, dim3((unsigned)blocks), dim3(256), 0, s, W, row0, H, dst);
  return hipGetLastError();
}
template hipError_t launch_permute_um<float>(const float*, int, int, float*, hipStream_t);
template hipError_t launch_permute_um<bf16_t>(const bf16_t*, int, int, bf16_t*, hipStream_t);
template hipError_t launch_convert<float>(const float*, long, float*, hipStream_t);
template hipError_t launch_convert<bf16_t>(const float*, long, bf16_t*, hipStream_t);

}  // namespace ll
