// XCD-local variants of the two device-side loops.
//
// MI355X has 8 XCDs of 32 CUs; each XCD has its own L2, shared by its CUs.
// Here the 32 work-groups resident on one XCD form a group that runs the
// recurrence of its own batch rows (row tiles x, x+8, ... for XCD x) and
// splits the hidden units 32 ways, so every value exchanged inside the loop
// (h_t forward, dz_t backward) moves only through that XCD's L2.
//
// The exchange goes through a ring of two slots per row tile, laid out in the
// order the consumers' matrix-core operands need it: block ks of a slot holds
// k-step ks (32 bf16 or 16 fp32 columns) of the tile's 16 rows, lane l's 16
// bytes being row l % 16, k-chunk l / 16.  Every block has exactly one
// producer (its columns are the producer's own hidden units), and a consumer
// wave reads each of its k-steps as one contiguous 1 KB load.
//   * A producer stores its blocks with plain stores (the vector L1 writes
//     through to the L2), waits until they are acknowledged
//     (s_waitcnt vmcnt(0)), meets its work-group at a barrier, and one thread
//     stores the step number into the producer's flag.
//   * A consumer wave polls, one lane per producer, the flags of the blocks it
//     needs with L1-bypassing loads, then reads the blocks with L1-bypassing
//     (cache policy sc1) loads: they are in the shared L2 by then.
// Slot t % 2 is rewritten at step t + 2 (t - 2 in the gradient loop) only
// after every member has published step t + 1, which each does after reading
// slot t % 2, so two slots suffice.  There is no grid barrier and no L2
// writeback or invalidate in the loop.  A work-group learns its XCD from the
// XCC_ID hardware register and its rank from a per-XCD counter, so the
// mapping does not depend on the dispatch order.
//
// Each work-group keeps its recurrent weight slice on chip for the whole
// loop, in registers (the first KSR k-steps of each wave's share; any rest in
// LDS).
#include "ll_kernels.h"
#include "ll_exchange.h"

namespace ll {


// 8 waves per work-group, two per SIMD: the weight slice of a work-group is
// split over 8 waves' registers (the reduction dimension is split 8 ways).
constexpr int XNW = 8;
constexpr int XNT = 64 * XNW;
// Per-step loop metadata (active rows, compact offsets) for steps
// lo .. lo+WIN, kept in LDS so that no step waits on a global load for it.
constexpr int WIN = 256;

// Partial products in LDS: [wave][element i of the MFMA result][column
// tile][lane], one slice of NCT*64 + 16 floats per (wave, i).  The pad of 16
// floats puts the four rows a 16-lane group of the cell reads in distinct
// LDS banks.
constexpr int xfwd_is(int NCT) { return NCT * 64 + 16; }
__host__ __device__ constexpr int xbwd_is(int NCT) { return NCT * 64 + 16; }
__host__ __device__ constexpr int xbwd_red_floats(int NCT) {
  return XNW * 4 * xbwd_is(NCT) > 16 * 4 * 16 * NCT ? XNW * 4 * xbwd_is(NCT) : 16 * 4 * 16 * NCT;
}

// LDS of the forward kernel: weight k-steps not in registers, partial
// products, metadata window, perm rows.
// (cond body: the waves' partial predicate sums, skip_floats more)
size_t xfwd_lds(int KSW, int KSR, int NCT, int mrt_max, int skip_floats = 0) {
  const int KSL = KSW > KSR ? KSW - KSR : 0;
  return (size_t)XNW * KSL * NCT * 64 * 16 + (size_t)XNW * 4 * xfwd_is(NCT) * 4 +
         (size_t)2 * (WIN + 1) * 4 + (size_t)mrt_max * 16 * 4 + (size_t)skip_floats * 4;
}
// floats of the cond body's LDS: XNW x 16 partial sums
constexpr int xfwd_skip_floats() { return XNW * 16; }
// LDS of the gradient kernel: weight k-steps not in registers, partial
// products (reused for the db rows at the end), metadata window, perm rows.
__host__ __device__ constexpr int xbwd_tail_chunks(int NCT, int mrt_max) {
  return (xbwd_red_floats(NCT) * 4 + 2 * (WIN + 1) * 4 + mrt_max * 16 * 4 + 15) / 16;
}
size_t xbwd_lds(int KSW, int KSR, int NCT, int mrt_max) {
  const int KSL = KSW > KSR ? KSW - KSR : 0;
  return (size_t)XNW * KSL * NCT * 64 * 16 + (size_t)xbwd_tail_chunks(NCT, mrt_max) * 16;
}

__device__ __forceinline__ void load_window(const XLoopArgs& a, int* win, int lo) {
  __syncthreads();
  for (int i = threadIdx.x; i <= WIN; i += blockDim.x) {
    const int t = lo + i;
    win[i] = t <= a.T_max ? a.active[t] : 0;
    win[WIN + 1 + i] = t <= a.T_max ? a.off[t] : 0;
  }
  __syncthreads();
}

// Stack row of (step t, compact index r) in the stack ring.
__device__ __forceinline__ long stack_row(const XLoopArgs& a, int t, int r) {
  const int k = t / a.chunk_steps;
  return ((long)((k % a.nslots) * a.chunk_steps + (t - k * a.chunk_steps)) * a.B + r);
}
// Row of (step t, compact index r) where the gates i, f, g, o are popped.
__device__ __forceinline__ long gate_row(const XLoopArgs& a, int t, int r) {
  if (!a.gstk) return stack_row(a, t, r);
  const int k = t / a.gchunk;
  return ((long)((k % a.gslots) * a.gchunk + (t - k * a.gchunk)) * a.B + r);
}

// Ring slot of row tile mt: ring_ks blocks of 1 KB.
__device__ __forceinline__ char* ring_tile(const XLoopArgs& a, int slot, int grp, int mt) {
  return reinterpret_cast<char*>(a.ring) + ((long)((slot * 8 + grp) * a.MRT + mt) * a.ring_ks << 10);
}

// ---------------------------------------------------------------------------
// Forward loop, XCD-local.  Member `rank` of XCD x owns hidden units
// j0 .. j0+HJ-1 (HJ = 4 NCT: all four gates of each unit, NCT column tiles of
// 16 gate columns) of the rows in tiles x, x+8, ...; HJ units are one k-step
// of the recurrent product, ring block `rank`.  Step t for a row tile:
//   1. every wave waits for the producers of its k-steps of h_{t-1} (K split
//      over the 8 waves) and reads them from the ring; the cell threads also
//      fetch the next step's input projections;
//   2. z = h W_h over the wave's k-steps (MFMA), partial products -> LDS;
//   3. cell: thread (row, unit) of the first 16*HJ threads adds the 8
//      partial products of its four gates and the input projection, runs the
//      cell, stores h_t into the ring and publishes it; then the h history,
//      the stack row and y_t.
// ---------------------------------------------------------------------------
// TOP: the upper layer of the two-layer wavefront.  Its recurrent product
// runs over K = I_l + H = 2H: the first in_ks k-steps are y1_t, read from the
// lower layer's ring for step t (bf16(y1_t) in the bf16 contract: the ring
// holds the operand-type h_t), the rest h_{t-1} from its own ring; the bias
// replaces the hoisted input projection.
// G: gate blocks of the cell (4: LSTM i, f, g, o; 1: Elman RNN, h = tanh(z);
// 3: GRU r, u, n with the reset gate applied after the recurrent product).
// SKIP (LSTM only): the body is cond(s > 0, LSTM step, keep the state) with
// s = (x_t . w_px + h_{t-1} . w_ph) + b_p per row.  The x part comes
// precomputed per compact row (a.sx); the h part is one more matrix-core
// column of the recurrent product (w_ph as column 0 of an extra 16-column
// tile, over the h_{t-1} chunks each wave already holds; every member of an
// XCD computes it identically, so all take the same branch); the guard of
// every (step, row) is pushed for the gradient loop.
// ACT (LSTM only): the body is a nested while-loop (Adaptive Computation
// Time's halting rule): the LSTM step applied to (x_t, h, c) up to
// a.ponder_max times; after ponder step k a row's halting probability
// p = sigmoid(h^k . w_p + b_p) (h part by the same extra matrix-core column
// as the cond body's) is summed into P, and the row stops pondering once
// P >= 1 - eps.  The row tile runs a ponder iteration while any of its rows
// still ponders (every member computes the same sums, so all agree), and
// each iteration is one exchange round; rows that stopped keep their state.
// The forward pushes, per (step, ponder step k, row), the step's values at
// stack slot k (rows k * slot_rows + compact row), the guard (1 = the row
// pondered) and the state h^{k+1} (into HI); per (step, row tile) the inner
// trip count (ntrip).  The exchange counts ponder iterations, not steps.
template <typename T, int NCT, int KSW, int KSR, int MRT_MAX, bool TOP, int G = 4, bool SKIP = false,
          bool ACT = false>
__device__ __forceinline__ void xfwd_body(const XLoopArgs& a, int grp, int rank, uint4* lds) {
  constexpr bool PRED = SKIP || ACT;   // the extra predicate column of the recurrent product
  constexpr int KPC = Op<T>::kPerChunk;
  constexpr int HJ = 16 * NCT / G;
  constexpr int KSL = KSW > KSR ? KSW - KSR : 0;
  constexpr int IS = xfwd_is(NCT);
  static_assert(16 * HJ <= XNT, "one cell thread per (row, unit) of a tile");
  static_assert(HJ == 4 * KPC, "a member's units are one k-step");
  const int tid = threadIdx.x, lane = tid & 63, wave = uni(tid >> 6);
  const int q = lane >> 4, l16 = lane & 15;
  const int H = a.H, B = a.B;
  const long G4 = (long)G * H;                           // gate columns
  const int j0 = rank * HJ;
  const int KX = TOP ? a.in_ks : 0;                      // k-steps from the lower layer
  const int KS = KX + H / (4 * KPC);
  const int ks0 = min(KS, wave * KSW), ks1 = min(KS, ks0 + KSW);
  const int nks = ks1 - ks0;                             // k-steps of this wave
  const T* WT = reinterpret_cast<const T*>(a.W);
  T* HH = reinterpret_cast<T*>(a.X);

  // weight slice: column tile ct, lane column l16 <-> local gate column
  // ct*16 + l16 = gate * HJ + u
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
  float* red = reinterpret_cast<float*>(lds + XNW * KSL * NCT * 64);   // [XNW][4][IS]
  int* win = reinterpret_cast<int*>(red + XNW * 4 * IS);               // [2][WIN+1]
  int* sperm = win + 2 * (WIN + 1);                                   // [MRT][16]
  float* sred = reinterpret_cast<float*>(sperm + MRT_MAX * 16);       // SKIP: [XNW][16]
  static_assert(!(PRED && (TOP || G != 4)), "the cond and nested-loop bodies are built on the single-layer LSTM loop");
  static_assert(!(SKIP && ACT), "one body");
  // SKIP / ACT: the predicate's (halting unit's) h weights as the B operand
  // of a 16-column tile whose column 0 is w_p (operand-rounded), the rest zero
  uint4 wpr[PRED ? KSW : 1];
  if constexpr (PRED) {
#pragma unroll
    for (int i = 0; i < KSW; ++i) {
      const int ks = ks0 + i;
      alignas(16) T v[KPC];
#pragma unroll
      for (int e = 0; e < KPC; ++e)
        v[e] = Op<T>::from_f32(l16 == 0 && ks < ks1 ? a.wp[(ks * 4 + q) * KPC + e] : 0.f);
      wpr[i] = *reinterpret_cast<const uint4*>(v);
    }
  }
  const float bp = PRED ? a.bp[0] : 0.f;
  // ACT: halting threshold 1 - eps (eps = 0.01) and the ponder counters of
  // each row tile (exchange rounds so far)
  const float act_thr = 1.0f - 0.01f;
  int itc[MRT_MAX];
#pragma unroll
  for (int mt = 0; mt < MRT_MAX; ++mt) itc[mt] = 0;

  // cell thread: 16 lanes take 16 consecutive units of one row, a wave four
  // rows (the four MFMA result elements of one lane group)
  const bool cellt = tid < 16 * HJ;
  const int cu = (tid >> 8) * 16 + (tid & 15);    // local unit
  const int crow = (tid >> 4) & 15;               // row within the tile
  const int ju = j0 + cu;
  // LDS slot of this thread's gate-0 partial product of wave 0
  const float* rp = red + (crow & 3) * IS + (cu >> 4) * 64 + (crow >> 2) * 16 + (cu & 15);
  // byte offset of (crow, cu) in a ring block
  const int rbo = ((crow + 16 * (cu / KPC)) * KPC + cu % KPC) * (int)sizeof(T);
  // GRU: recurrent bias of the candidate block, added before the reset gate
  const float bhn = (G == 3 && cellt) ? a.bhn[ju] : 0.f;
  float hs[MRT_MAX], cs[MRT_MAX];
  if (tid < MRT_MAX * 16) {
    const int r = (grp + 8 * (tid >> 4)) * 16 + (tid & 15);
    sperm[tid] = ((tid >> 4) < a.MRT && r < B) ? a.perm[r] : -1;
  }
  __syncthreads();
#pragma unroll
  for (int mt = 0; mt < MRT_MAX; ++mt) {
    const int b = sperm[mt * 16 + crow];
    hs[mt] = 0.f;
    cs[mt] = 0.f;
    if (cellt && b >= 0) {
      if (a.h0) hs[mt] = a.h0[(long)b * H + ju];
      if (a.c0) cs[mt] = a.c0[(long)b * H + ju];
    }
  }

  const int T_eff = uni(a.meta[0]);
  const int t0 = a.t_begin, t1 = min(a.t_end, T_eff);
  int wlo = t0 > 0 ? t0 - 1 : 0;
  load_window(a, win, wlo);
  // input projections of the cell thread's (row, unit), one step ahead (the
  // upper wavefront layer: its bias)
  float zf[MRT_MAX][G];
  float sxf[MRT_MAX];   // SKIP: x part of the predicate, one step ahead
  if constexpr (TOP) {
#pragma unroll
    for (int mt = 0; mt < MRT_MAX; ++mt)
#pragma unroll
      for (int g = 0; g < G; ++g) zf[mt][g] = cellt ? a.zbias[(long)g * H + ju] : 0.f;
  } else {
    const int A0 = t0 < t1 ? win[t0 - wlo] : 0, off0 = win[WIN + 1 + t0 - wlo];
#pragma unroll
    for (int mt = 0; mt < MRT_MAX; ++mt) {
      const int r = (grp + 8 * mt) * 16 + crow;
#pragma unroll
      for (int g = 0; g < G; ++g)
        zf[mt][g] = (cellt && mt < a.MRT && r < A0) ? a.Zx[(long)(off0 + r) * G4 + (long)g * H + ju] : 0.f;
      sxf[mt] = (SKIP && cellt && mt < a.MRT && r < A0) ? a.sx[off0 + r] : 0.f;
    }
  }

  for (int t = t0; t < t1; ++t) {
    if (t + 1 > wlo + WIN) {   // the window keeps step t-1 as well
      wlo = t - 1;
      load_window(a, win, wlo);
    }
    const int A_t = uni(win[t - wlo]), A_n = uni(win[t + 1 - wlo]);
    const int off_t = uni(win[WIN + 1 + t - wlo]), off_n = uni(win[WIN + 1 + t + 1 - wlo]);
#pragma unroll
    for (int mt = 0; mt < MRT_MAX; ++mt) {
      if (mt >= a.MRT) continue;
      const int r0 = (grp + 8 * mt) * 16;
      if (r0 >= A_t) {
        if (a.y && cellt) {   // finished tile: y_t = 0 for its rows
          const int b = sperm[mt * 16 + crow];
          if (b >= 0) a.y[((long)t * B + b) * H + ju] = 0.f;
        }
        continue;
      }
      unsigned* flags = a.flags + (grp * a.MRT + mt) * 32;
      const int r = r0 + crow;
      const bool act = cellt && r < A_t;
      float zc[G];
      float sxc = 0.f;
      // ACT: this thread's row still ponders; the row's summed halting
      // probability
      bool prow = act;
      float Psum = 0.f;
      const int nk = ACT ? a.ponder_max : 1;
      int k = 0;
      for (; k < nk; ++k) {
      // exchange round of this iteration: the step (one round per step), or
      // the tile's ponder counter
      const int cnt = ACT ? itc[mt] : t;
      // 1. h_{t-1} of this wave's k-steps (for the launch's first step the
      //    ring holds the entering state); the upper wavefront layer first
      //    takes y1_t from the lower layer's ring
      const int kx1 = min(ks1, KX);                        // [ks0, kx1): lower layer's k-steps
      if (TOP && ks0 < kx1)
        wait_flags(a, a.in_flags + (grp * a.MRT + mt) * 32, ks0, kx1 - ks0, a.in_ks, (unsigned)(t + 2));
      if ((ACT ? cnt > 0 : t > t0) && max(ks0, KX) < ks1)
        wait_flags(a, flags, max(ks0, KX) - KX, ks1 - max(ks0, KX), a.P, (unsigned)(cnt + 1));
      const __amdgpu_buffer_rsrc_t rs = make_rsrc(ring_tile(a, (cnt + 1) & 1, grp, mt), (unsigned)(a.ring_ks << 10));
      __amdgpu_buffer_rsrc_t rsx = rs;
      if constexpr (TOP)
        rsx = make_rsrc(reinterpret_cast<const char*>(a.in_ring) +
                            ((long)(((t & 1) * 8 + grp) * a.MRT + mt) * a.in_ks << 10),
                        (unsigned)(a.in_ks << 10));
      uint4 av[KSW];
#pragma unroll
      for (int i = 0; i < KSW; ++i) {
        const int ks = ks0 + i;
        av[i] = ks < KX ? ld_chunk_l2(rsx, i < nks ? (unsigned)((ks << 10) + lane * 16) : kOOB)
                        : ld_chunk_l2(rs, i < nks ? (unsigned)(((ks - KX) << 10) + lane * 16) : kOOB);
      }
      if (k == 0) {
#pragma unroll
      for (int g = 0; g < G; ++g) zc[g] = zf[mt][g];
      sxc = sxf[mt];
      if constexpr (!TOP) {  // input projections of step t+1 (rows past A_n read zeros)
        const int nr = max(0, min(16, A_n - r0));
        const __amdgpu_buffer_rsrc_t rz = make_rsrc(a.Zx + (long)(off_n + r0) * G4, (unsigned)(nr * G4 * 4));
        const unsigned zo = cellt ? (unsigned)((crow * G4 + ju) * 4) : kOOB;
#pragma unroll
        for (int g = 0; g < G; ++g) zf[mt][g] = ld_f32(rz, zo + g * H * 4);
        if constexpr (SKIP) {
          const __amdgpu_buffer_rsrc_t rx = make_rsrc(a.sx + off_n + r0, (unsigned)(nr * 4));
          sxf[mt] = ld_f32(rx, cellt ? (unsigned)(crow * 4) : kOOB);
        }
      }
      }
      // 2. partial products over this wave's k-steps, column tiles in two
      //    halves, into red[wave][i][ct][lane] (the previous tile's cell has
      //    read them: it ended at a barrier)
      constexpr int NHALF = NCT % 2 == 0 ? 2 : 1;
#pragma unroll
      for (int hf = 0; hf < NHALF; ++hf) {
        constexpr int NH = NCT / NHALF;
        f32x4 acc[NH];
#pragma unroll
        for (int c = 0; c < NH; ++c) acc[c] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int i = 0; i < KSW; ++i) {
          if (i < nks) {
#pragma unroll
            for (int c = 0; c < NH; ++c) {
              const int ct = hf * NH + c;
              const uint4 bv = i < KSR ? wr[ct][i < KSR ? i : 0]
                                       : lds[((wave * KSL + (i - KSR)) * NCT + ct) * 64 + lane];
              acc[c] = Mfma<T>::step(av[i], bv, acc[c]);
            }
          }
        }
#pragma unroll
        for (int c = 0; c < NH; ++c)
#pragma unroll
          for (int i = 0; i < 4; ++i) red[(wave * 4 + i) * IS + (hf * NH + c) * 64 + lane] = acc[c][i];
      }
      if constexpr (PRED) {
        // h part of the predicate (halting unit) over this wave's k-steps:
        // column 0 of the extra tile; result element i of lane 16 q is row 4 q + i
        f32x4 accp = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int i = 0; i < KSW; ++i)
          if (i < nks) accp = Mfma<T>::step(av[i], wpr[i], accp);
        if (l16 == 0) {
#pragma unroll
          for (int i = 0; i < 4; ++i) sred[wave * 16 + q * 4 + i] = accp[i];
        }
      }
      __syncthreads();
      // the lower wavefront layer rewrites ring slot t % 2 only after the
      // upper layer has published step t - 2, its last read of that slot
      if (a.out_flags && t >= 2)
        wait_flags(a, a.out_flags + (grp * a.MRT + mt) * 32, 0, a.P, a.P, (unsigned)t);
      // 3. cell of (crow, cu): gate g is local column g*HJ + cu
      float ig = 0.f, fg = 0.f, gg = 0.f, og = 0.f, cn = 0.f, hn = 0.f;
      bool run = true;   // SKIP: the branch this row takes; ACT: the row ponders
      if constexpr (SKIP) {
        float sh = sred[crow];
#pragma unroll
        for (int w2 = 1; w2 < XNW; ++w2) sh += sred[w2 * 16 + crow];
        run = (sxc + sh) + bp > 0.f;
      }
      if constexpr (ACT) {
        // halting after ponder step k (its state h^k is this iteration's
        // operand): p = sigmoid(h^k . w_p + b_p), summed in float32
        if (k > 0 && prow) {
          float sh = sred[crow];
#pragma unroll
          for (int w2 = 1; w2 < XNW; ++w2) sh += sred[w2 * 16 + crow];
          Psum += sigmoidf_(sh + bp);
          if (Psum >= act_thr) prow = false;
        }
        run = prow;
        // no row of the tile ponders any more: the nested loop ends (every
        // member takes the same decision from the same sums)
        if (__syncthreads_or(prow ? 1 : 0) == 0) break;
      }
      if (cellt) {
        float z[G], zh[G];
#pragma unroll
        for (int g = 0; g < G; ++g) {
          const float* p = rp + g * (HJ / 16) * 64;
          float v = p[0];
#pragma unroll
          for (int w2 = 1; w2 < XNW; ++w2) v += p[w2 * 4 * IS];
          zh[g] = v;
          z[g] = v + zc[g];
        }
        if constexpr (G == 4) {
          ig = sigmoidf_(z[0]);
          fg = sigmoidf_(z[1]);
          gg = tanhf_(z[2]);
          og = sigmoidf_(z[3]);
          cn = fg * cs[mt] + ig * gg;
          hn = og * tanhf_(cn);
          if ((SKIP || ACT) && !run) {   // the false branch / a halted row keeps the state
            cn = cs[mt];
            hn = hs[mt];
          }
        } else if constexpr (G == 3) {
          // GRU: r, u, n, zh_n + b_hn and h_{t-1} take the places of the
          // LSTM's i, f, g, o and c_t in the stack row
          ig = sigmoidf_(z[0]);
          fg = sigmoidf_(z[1]);
          og = zh[2] + bhn;
          gg = tanhf_(zc[2] + ig * og);
          cn = hs[mt];
          hn = (1.f - fg) * gg + fg * cn;
        } else {
          hn = tanhf_(z[0]);
        }
        if (act) {
          *reinterpret_cast<T*>(ring_tile(a, cnt & 1, grp, mt) + (rank << 10) + rbo) = Op<T>::from_f32(hn);
          if constexpr (G == 4) cs[mt] = cn;
          hs[mt] = hn;
        }
      }
      publish(flags + rank, (unsigned)(cnt + 2));
      if constexpr (ACT) {
        itc[mt] = cnt + 1;
        // ponder step k's values at stack slot k, its guard, and h^{k+1}
        if (act && a.stack) {
          const long vr = (long)k * a.slot_rows + off_t + r;
          float* srow = a.stack + vr * a.sld;
          *reinterpret_cast<float4*>(srow + 4 * ju) = make_float4(ig, fg, gg, og);
          srow[a.scoff + ju] = cn;
          reinterpret_cast<T*>(a.HI)[vr * H + ju] = Op<T>::from_f32(hn);
          if (rank == 0 && cu == 0) a.guard[vr] = run ? 1.f : 0.f;
        }
        continue;
      }
      if (act) {
        const long cr = off_t + r;
        HH[cr * H + ju] = Op<T>::from_f32(hn);
        if (a.stack) {
          float* srow = a.stack + stack_row(a, t, r) * a.sld;
          if constexpr (G == 4 || G == 3) {
            // the unit's four gate values side by side (stack row: 4H gate
            // values unit by unit, then c): one 16-byte store
            if (a.sgates) *reinterpret_cast<float4*>(srow + 4 * ju) = make_float4(ig, fg, gg, og);
            srow[a.scoff + ju] = cn;
            if (SKIP && rank == 0 && cu == 0) a.guard[cr] = run ? 1.f : 0.f;
          } else {
            srow[a.scoff + ju] = hn;   // the RNN's gradient needs only h_t
          }
        }
      }
      if (a.y && cellt) {
        const int b = sperm[mt * 16 + crow];
        if (b >= 0) a.y[((long)t * B + b) * H + ju] = act ? hn : 0.f;
      }
      }   // ponder iterations
      if constexpr (ACT) {
        // the step's result: the last ponder state; the tile's inner trip count
        if (act) HH[(long)(off_t + r) * H + ju] = Op<T>::from_f32(hs[mt]);
        if (a.y && cellt) {
          const int b = sperm[mt * 16 + crow];
          if (b >= 0) a.y[((long)t * B + b) * H + ju] = act ? hs[mt] : 0.f;
        }
        if (a.stack && rank == 0 && threadIdx.x == 0) a.ntrip[(long)t * 8 * a.MRT + grp * a.MRT + mt] = k;
      }
    }
  }

  if (cellt) {
#pragma unroll
    for (int mt = 0; mt < MRT_MAX; ++mt) {
      const int b = sperm[mt * 16 + crow];
      if (b < 0) continue;
      a.hT[(long)b * H + ju] = hs[mt];
      if (a.cT) a.cT[(long)b * H + ju] = cs[mt];
      if (a.y)
        for (int t = max(T_eff, t0); t < a.t_end; ++t) a.y[((long)t * B + b) * H + ju] = 0.f;
    }
  }
}

template <typename T, int NCT, int KSW, int KSR, int MRT_MAX, int G, bool SKIP, bool ACT = false>
__global__ __launch_bounds__(XNT, 1) void xfwd_kernel(XLoopArgs a) {
  extern __shared__ uint4 lds[];
  __shared__ int s_info[2];
  join_group(a.rank_ctr, s_info);
  const int grp = uni(s_info[0]), rank = uni(s_info[1]);
  if (grp >= 8 || rank >= 32) {
    if (threadIdx.x == 0) {
      __hip_atomic_fetch_or(a.err, LL_DEVERR_BARRIER_BIT, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(a.abort_flag, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    return;
  }
  if (rank >= a.P) return;
  xfwd_body<T, NCT, KSW, KSR, MRT_MAX, false, G, SKIP, ACT>(a, grp, rank, lds);
}

// Two-layer wavefront, forward: members 0 .. P-1 of every XCD run the lower
// layer (a0), members P .. 2P-1 the upper layer (a1), one step behind.
template <typename T, int NCT, int KSWB, int KSRB, int KSWT, int KSRT, int MRT_MAX>
__global__ __launch_bounds__(XNT, 1) void xfwd2_kernel(XLoopArgs a0, XLoopArgs a1) {
  extern __shared__ uint4 lds[];
  __shared__ int s_info[2];
  join_group(a0.rank_ctr, s_info);
  const int grp = uni(s_info[0]), rank = uni(s_info[1]);
  if (grp >= 8 || rank >= 32) {
    if (threadIdx.x == 0) {
      __hip_atomic_fetch_or(a0.err, LL_DEVERR_BARRIER_BIT, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(a0.abort_flag, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    return;
  }
  if (rank < a0.P)
    xfwd_body<T, NCT, KSWB, KSRB, MRT_MAX, false>(a0, grp, rank, lds);
  else if (rank < a0.P + a1.P)
    xfwd_body<T, NCT, KSWT, KSRT, MRT_MAX, true>(a1, grp, rank - a0.P, lds);
}

// ---------------------------------------------------------------------------
// Gradient loop, XCD-local.  Member `rank` owns hidden units j0 .. j0+HJ-1
// (HJ = 16 NCT); thread (row, unit) of the first 16*HJ threads keeps dh, dc
// of that row and unit.  The dz columns of gate g of the member's units are
// k-step g*P + rank of the product dz W_h^T (the single-layer LSTM loop
// orders the reduction unit-major instead: its k-steps 4 rank .. 4 rank + 3
// hold the member's units, four gates each).  Step t (descending), per row
// tile:
//   phase 1: from the values popped during step t+1: dh_tot, dz, dc; store
//     dz into the ring and publish it; then the dz rows for the dW and dx
//     products; accumulate db;
//   phase 2: wait for the producers of the wave's k-steps (all 4H gate
//     columns, K split over the 8 waves), read them in two batches (the pops
//     of step t-1 are issued after the last batch), dh <- dz W_h^T for the
//     own units (MFMA); the thread of (row, unit) adds the 8 partial
//     products.
// ---------------------------------------------------------------------------
// ROLE 0: a single layer; 1: the lower layer of the two-layer wavefront
// (its dy comes from the upper layer's dyx ring, one step later); 2: the upper
// layer, which also computes dy_{lower} = dz W_x^T for its units (NCO = 2 NCT
// output column tiles: W_h rows, then W_x rows) and publishes it per step.
// SKIP: the LSTM body with a cond (see xfwd_body); the popped guard picks
// each row's branch gradient: the LSTM step's, or the identity (dz = 0,
// dh_{t-1} = dh_tot, dc_{t-1} = dc_t).
// ACT: the body holds a nested loop (see xfwd_body).  Step t pops the tile's
// inner trip count n and runs a nested gradient loop of n iterations, ponder
// step n-1 down to 0, each one exchange round: the ponder step's values and
// guard are popped from its stack slot (the guard picks the LSTM step's
// gradient or the identity); dy_t enters at the last ponder step; c of the
// step before ponder step 0 is the previous step's last ponder state.  dz of
// ponder step k goes to dz slot k (slots the tile did not run get zeros).
template <typename T, int NCT, int KSW, int KSR, int MRT_MAX, int ROLE, int G = 4, bool SKIP = false,
          bool ACT = false>
__device__ __forceinline__ void xbwd_body(const XLoopArgs& a, int grp, int rank, uint4* lds) {
  constexpr int KPC = Op<T>::kPerChunk;
  constexpr int HJ = 16 * NCT;                 // units per work-group
  constexpr int NCO = ROLE == 2 ? 2 * NCT : NCT;   // output column tiles
  constexpr int KSL = KSW > KSR ? KSW - KSR : 0;
  constexpr int KB = KSW < 4 ? KSW : 4;        // k-steps per load batch
  constexpr int IS = xbwd_is(NCO);
  static_assert(16 * HJ <= XNT, "one thread per (row, unit) of a tile");
  static_assert(HJ == 4 * KPC, "a member's units of one gate are one k-step");
  const int tid = threadIdx.x, lane = tid & 63, wave = uni(tid >> 6);
  const int q = lane >> 4, l16 = lane & 15;
  const int H = a.H, B = a.B, P = a.P;
  const long G4 = (long)G * H;                          // gate columns (ring blocks, W_h row width)
  // dz rows for the products after the loop: the gate blocks, and for the GRU
  // a fourth, the candidate block's recurrent-side value da_n * r
  constexpr int GB = G == 3 ? 4 : G;
  const long GBH = (long)GB * H;
  const int j0 = rank * HJ;
  const int KS = (int)(G4 / (4 * KPC));
  // pops per (step, tile) and thread: LSTM i, f, g, o, c_t, c_{t-1}, dy;
  // GRU r, u, n, zh_n + b_hn, h_{t-1}, dy; RNN h_t, dy
  constexpr bool GUARDED = SKIP || ACT;   // a popped guard picks each row's gradient
  constexpr int NPOP = (G == 4 ? 7 : G == 3 ? 6 : 2) + (GUARDED ? 1 : 0);
  constexpr int NPV = GUARDED ? 8 : 7;   // popped values kept per (tile, thread); [7] = guard
  // Unit-major reduction order (single-layer LSTM loop): k = 4 u + g over
  // units u and gates g, so a member's dz values of one unit are adjacent in
  // the ring and k-steps 4 r .. 4 r + 3 are member r's; the weights come
  // from W_h permuted to that order (a.W = [H, 4H], a.woff = 0).  Otherwise
  // k = g H + u and k-step g P + r is member r's gate g.
  constexpr bool UM = G == 4 && ROLE == 0;
  static_assert(!(GUARDED && (ROLE != 0 || G != 4)), "the cond and nested-loop bodies are built on the single-layer LSTM loop");
  const int ks0 = min(KS, wave * KSW), ks1 = min(KS, ks0 + KSW);
  const int nks = ks1 - ks0;                            // k-steps of this wave
  const T* W = reinterpret_cast<const T*>(a.W);
  T* DZ = reinterpret_cast<T*>(a.X);

  uint4 wr[NCO][KSR];
#pragma unroll
  for (int ct = 0; ct < NCO; ++ct) {
    const T* wrow = ct < NCT ? W + (long)(a.woff + j0 + ct * 16 + l16) * G4
                             : reinterpret_cast<const T*>(a.Wx) + (long)(j0 + (ct - NCT) * 16 + l16) * G4;
#pragma unroll
    for (int i = 0; i < KSR; ++i) {
      const int ks = ks0 + i;
      wr[ct][i] = ks < ks1 ? ld16(wrow + (ks * 4 + q) * KPC) : zero4();
    }
#pragma unroll
    for (int i = 0; i < KSL; ++i) {
      const int ks = ks0 + KSR + i;
      lds[((wave * KSL + i) * NCO + ct) * 64 + lane] = ks < ks1 ? ld16(wrow + (ks * 4 + q) * KPC) : zero4();
    }
  }
  float* red = reinterpret_cast<float*>(lds + XNW * KSL * NCO * 64);   // [XNW][4][IS]
  int* win = reinterpret_cast<int*>(red + xbwd_red_floats(NCO));       // [2][WIN+1]
  int* sperm = win + 2 * (WIN + 1);                                   // [MRT][16]

  // (row, unit) of this thread: 16 lanes take 16 consecutive units of one
  // row, a wave four rows (the four MFMA result elements of a lane group)
  const bool cellt = tid < 16 * HJ;
  const int cu = (tid >> 8) * 16 + (tid & 15);
  const int crow = (tid >> 4) & 15;
  const int ju = j0 + cu;
  const float* rp = red + (crow & 3) * IS + (cu >> 4) * 64 + (crow >> 2) * 16 + (cu & 15);
  const int rbo = ((crow + 16 * (cu / KPC)) * KPC + cu % KPC) * (int)sizeof(T);
  if (tid < MRT_MAX * 16) {
    const int r = (grp + 8 * (tid >> 4)) * 16 + (tid & 15);
    sperm[tid] = ((tid >> 4) < a.MRT && r < B) ? a.perm[r] : -1;
  }
  __syncthreads();
  float dh[MRT_MAX], dc[MRT_MAX];
#pragma unroll
  for (int mt = 0; mt < MRT_MAX; ++mt) {
    dh[mt] = 0.f;
    dc[mt] = 0.f;
    const int b = cellt ? sperm[mt * 16 + crow] : -1;
    if (b >= 0) {
      if (a.dhT) dh[mt] = a.dhT[(long)b * H + ju];
      if (a.dcT) dc[mt] = a.dcT[(long)b * H + ju];
    }
  }
  float dbacc[GB];
#pragma unroll
  for (int g = 0; g < GB; ++g) dbacc[g] = 0.f;
  float* dbst = a.db_state ? a.db_state + ((long)(grp * 32 + rank) * XNT + tid) * 4 : nullptr;
  if (dbst && a.db_resume) {
#pragma unroll
    for (int g = 0; g < GB; ++g) dbacc[g] = dbst[g];
  }

  // pops of (step tt, tile mt) for this thread: i, f, g, o, c_t, c_{t-1}, dy;
  // zeros for rows not running at tt (every read is issued, out of range)
  auto fetch = [&](float (&v)[NPV], int tt, int mt, int A, int off, int offp) {
    const int r0 = (grp + 8 * mt) * 16;
    const int nr = tt >= 0 ? max(0, min(16, A - r0)) : 0;
    const bool ok = cellt && crow < nr;
    const int b = sperm[mt * 16 + crow];
    const int ts = max(tt, 0);
    const long SL = a.sld, GL = a.gstk ? a.gld : a.sld;
    const unsigned so = ok ? (unsigned)((crow * SL + ju) * 4) : kOOB;
    const __amdgpu_buffer_rsrc_t rs =
        make_rsrc(a.stack + stack_row(a, ts, r0) * SL + a.scoff, (unsigned)(nr * SL * 4));
    if constexpr (G == 1) {   // RNN: h_t and dy
      v[0] = ld_f32(rs, so);
      v[1] = v[2] = v[3] = v[4] = v[5] = 0.f;
      (void)b;
    } else {
    const float* gbase = a.gstk ? a.gstk : a.stack;
    const __amdgpu_buffer_rsrc_t rg = make_rsrc(gbase + gate_row(a, ts, r0) * GL, (unsigned)(nr * GL * 4));
    if (a.gstk) {   // recomputed gates: gate-major rows
      const unsigned go = ok ? (unsigned)((crow * GL + ju) * 4) : kOOB;
#pragma unroll
      for (int c = 0; c < 4; ++c) v[c] = ld_f32(rg, go + c * H * 4);
    } else {        // the stack's gate values, unit by unit: one 16-byte read
      const float4 g4 = ld_f32x4(rg, ok ? (unsigned)((crow * GL + 4 * ju) * 4) : kOOB);
      v[0] = g4.x;
      v[1] = g4.y;
      v[2] = g4.z;
      v[3] = g4.w;
    }
    v[4] = ld_f32(rs, so);
    if constexpr (G == 3) {   // GRU: h_{t-1} was pushed with the step
      v[5] = 0.f;
    } else if (tt > 0) {
      const __amdgpu_buffer_rsrc_t rp2 =
          make_rsrc(a.stack + stack_row(a, tt - 1, r0) * SL + a.scoff, (unsigned)(nr * SL * 4));
      v[5] = ld_f32(rp2, so);
    } else {
      const __amdgpu_buffer_rsrc_t rc = make_rsrc(a.c0, a.c0 ? (unsigned)(B * H * 4) : 0u);
      v[5] = ld_f32(rc, ok ? (unsigned)((b * H + ju) * 4) : kOOB);
    }
    }
    if (a.dy_compact) {
      const __amdgpu_buffer_rsrc_t rd = make_rsrc(a.dy + (long)(off + r0) * H, (unsigned)(nr * H * 4));
      v[6] = ld_f32(rd, ok ? (unsigned)((crow * H + ju) * 4) : kOOB);
    } else {
      const __amdgpu_buffer_rsrc_t rd =
          make_rsrc(a.dy ? a.dy + (long)ts * B * H : nullptr, a.dy ? (unsigned)(B * H * 4) : 0u);
      v[6] = ld_f32(rd, ok ? (unsigned)((b * H + ju) * 4) : kOOB);
    }
    if constexpr (SKIP) {
      const __amdgpu_buffer_rsrc_t rgd = make_rsrc(a.guard + off + r0, (unsigned)(nr * 4));
      v[NPV - 1] = ld_f32(rgd, ok ? (unsigned)(crow * 4) : kOOB);
    }
    (void)offp;
  };
  // ACT: pops of ponder step kk of step tt for this thread (zeros for rows
  // not running at tt): the step's i, f, g, o, c at slot kk, the c before it
  // (slot kk-1, or the last ponder slot np_prev - 1 of step tt-1 at compact
  // offset offp, or c0), dy_t only at the last ponder step (kk = n_tt - 1),
  // and the guard
  auto fetch_act = [&](float (&v)[NPV], int tt, int kk, int n_tt, int mt, int A, int off, int offp,
                       int np_prev) {
    const int r0 = (grp + 8 * mt) * 16;
    const int nr = tt >= 0 ? max(0, min(16, A - r0)) : 0;
    const bool ok = cellt && crow < nr;
    const int b = sperm[mt * 16 + crow];
    const long SL = a.sld;
    const long vr = (long)max(kk, 0) * a.slot_rows + off + r0;     // first row of the tile's slot
    const __amdgpu_buffer_rsrc_t rg = make_rsrc(a.stack + vr * SL, (unsigned)(nr * SL * 4));
    const unsigned go = ok ? (unsigned)((crow * SL + ju) * 4) : kOOB;
    const float4 g4 = ld_f32x4(rg, ok ? (unsigned)((crow * SL + 4 * ju) * 4) : kOOB);
    v[0] = g4.x;
    v[1] = g4.y;
    v[2] = g4.z;
    v[3] = g4.w;
    v[4] = ld_f32(rg, go + a.scoff * 4);
    if (kk > 0) {
      const __amdgpu_buffer_rsrc_t rp2 =
          make_rsrc(a.stack + (vr - a.slot_rows) * SL, (unsigned)(nr * SL * 4));
      v[5] = ld_f32(rp2, go + a.scoff * 4);
    } else if (tt > 0) {
      const long pr = (long)(np_prev - 1) * a.slot_rows + offp + r0;
      const __amdgpu_buffer_rsrc_t rp2 = make_rsrc(a.stack + pr * SL, (unsigned)(nr * SL * 4));
      v[5] = ld_f32(rp2, go + a.scoff * 4);
    } else {
      const __amdgpu_buffer_rsrc_t rc = make_rsrc(a.c0, a.c0 ? (unsigned)(B * H * 4) : 0u);
      v[5] = ld_f32(rc, ok ? (unsigned)((b * H + ju) * 4) : kOOB);
    }
    const bool last = kk == n_tt - 1;
    const __amdgpu_buffer_rsrc_t rd =
        make_rsrc(a.dy && last ? a.dy + (long)max(tt, 0) * B * H : nullptr, a.dy && last ? (unsigned)(B * H * 4) : 0u);
    v[6] = ld_f32(rd, ok ? (unsigned)((b * H + ju) * 4) : kOOB);
    const __amdgpu_buffer_rsrc_t rgd = make_rsrc(a.guard + vr, (unsigned)(nr * 4));
    v[NPV - 1] = ld_f32(rgd, ok ? (unsigned)(crow * 4) : kOOB);
  };
  // ACT: the inner trip count of (step tt, tile mt), within [1, ponder_max]
  auto ntrip_of = [&](int tt, int mt) -> int {
    if (!ACT || tt < 0) return 1;
    const int n = uni(a.ntrip[(long)tt * 8 * a.MRT + grp * a.MRT + mt]);
    return min(max(n, 1), a.ponder_max);
  };
  // ACT: pops of the first ponder iteration of step tt (its last ponder step)
  auto fetch_step = [&](float (&v)[NPV], int tt, int mt, int A, int off, int offp) {
    const int n = ntrip_of(tt, mt);
    fetch_act(v, tt, n - 1, n, mt, A, off, offp, ntrip_of(tt - 1, mt));
  };

  const int T_eff = uni(a.meta[0]);
  const int t0 = a.t_begin, t1 = min(a.t_end, T_eff);
  // the window covers steps t-2 .. t+2 of every step t of the loop
  int wlo = t1 + 1 - WIN > 0 ? t1 + 1 - WIN : 0;
  load_window(a, win, wlo);
  float pv[MRT_MAX][NPV];
  {
    const int t = t1 - 1;
    const int A_t = t >= 0 ? win[t - wlo] : 0;
    const int off_t = t >= 0 ? win[WIN + 1 + t - wlo] : 0;
    const int off_p = t >= 1 ? win[WIN + 1 + t - 1 - wlo] : 0;
#pragma unroll
    for (int mt = 0; mt < MRT_MAX; ++mt) {
      if (mt >= a.MRT) continue;
      if constexpr (ACT) fetch_step(pv[mt], t, mt, A_t, off_t, off_p);
      else fetch(pv[mt], t, mt, A_t, off_t, off_p);
    }
  }
  // ACT: exchange rounds per row tile so far (the flags count them)
  int itb[MRT_MAX];
#pragma unroll
  for (int mt = 0; mt < MRT_MAX; ++mt) itb[mt] = 1;

  for (int t = t1 - 1; t >= t0; --t) {
    if (t - 2 < wlo && wlo > 0) {
      wlo = t + 2 - WIN > 0 ? t + 2 - WIN : 0;
      load_window(a, win, wlo);
    }
    const int A_t = uni(win[t - wlo]);
    const int off_t = uni(win[WIN + 1 + t - wlo]);
    const int A_n = uni(t >= 1 ? win[t - 1 - wlo] : 0);
    const int off_n = uni(t >= 1 ? win[WIN + 1 + t - 1 - wlo] : 0);
    const int off_pn = uni(t >= 2 ? win[WIN + 1 + t - 2 - wlo] : 0);
#pragma unroll
    for (int mt = 0; mt < MRT_MAX; ++mt) {
      if (mt >= a.MRT) continue;
      const int r0 = (grp + 8 * mt) * 16;
      if (r0 >= A_t) {
        // rows of this tile may start running at step t-1 (lengths >= t)
        if constexpr (ACT) fetch_step(pv[mt], t - 1, mt, A_n, off_n, off_pn);
        else fetch(pv[mt], t - 1, mt, A_n, off_n, off_pn);
        continue;
      }
      unsigned* flags = a.flags + (grp * a.MRT + mt) * 32;
      const bool act = cellt && r0 + crow < A_t;
      // ACT: the nested gradient loop over ponder steps n-1 .. 0 of step t;
      // one iteration otherwise
      const int n_t = ntrip_of(t, mt);
      for (int kk = ACT ? n_t - 1 : 0; kk >= 0; --kk) {
      const int cnt = ACT ? itb[mt] : T_eff - t;   // flag value of this exchange round
      char* slot = ring_tile(a, ACT ? cnt & 1 : t & 1, grp, mt);
      // dyx ring slot of this tile for step t: [16 rows][H] floats
      const long dyx_off = ((long)(((t & 1) * 8 + grp) * a.MRT + mt) * 16) * H;
      float dyl = 0.f;   // lower wavefront layer: dy of its output from the upper layer
      if constexpr (ROLE == 1) {
        wait_flags(a, a.dyx_flags + (grp * a.MRT + mt) * 32, rank, 1, 32, (unsigned)(T_eff - t));
        const __amdgpu_buffer_rsrc_t ry =
            make_rsrc(reinterpret_cast<const float*>(a.dyx_ring) + dyx_off, (unsigned)(16 * H * 4));
        dyl = ld_f32_l2(ry, act ? (unsigned)((crow * H + ju) * 4) : kOOB);
      }
      // phase 1 (dz: the ring's values, the recurrent side; GRU: dzx_n is
      // the input side's candidate value, dhu the direct term of dh_{t-1})
      float dz[G], dzx_n = 0.f, dhu = 0.f;
#pragma unroll
      for (int g = 0; g < G; ++g) dz[g] = 0.f;
      if (act) {
        const float dht = dh[mt] + pv[mt][6] + dyl;
        if constexpr (G == 4) {
          const float ig = pv[mt][0], fg = pv[mt][1], gg = pv[mt][2], og = pv[mt][3];
          const float c = pv[mt][4], cp = pv[mt][5];
          const float tc = tanhf_(c);
          const float d_o = dht * tc;
          const float dct = dc[mt] + dht * og * (1.f - tc * tc);
          dz[0] = dct * gg * (ig * (1.f - ig));
          dz[1] = dct * cp * (fg * (1.f - fg));
          dz[2] = dct * ig * (1.f - gg * gg);
          dz[3] = d_o * (og * (1.f - og));
          if (GUARDED && pv[mt][NPV - 1] == 0.f) {   // the row kept its state at step t (ponder step kk)
            dz[0] = dz[1] = dz[2] = dz[3] = 0.f;
            dhu = dht;
          } else {
            dc[mt] = dct * fg;
          }
        } else if constexpr (G == 3) {
          const float rg = pv[mt][0], ug = pv[mt][1], ng = pv[mt][2], hnv = pv[mt][3];
          const float hp = pv[mt][4];
          const float dan = dht * (1.f - ug) * (1.f - ng * ng);
          dz[0] = dan * hnv * (rg * (1.f - rg));
          dz[1] = dht * (hp - ng) * (ug * (1.f - ug));
          dz[2] = dan * rg;
          dzx_n = dan;
          dhu = dht * ug;
        } else {
          const float hv = pv[mt][0];
          dz[0] = dht * (1.f - hv * hv);
        }
        if constexpr (UM) {
          // the unit's four gate values are adjacent in the unit-major order:
          // one 8-byte (bf16) / 16-byte (f32) store
          const int u = j0 + cu, ku = (u % KPC) * 4;
          char* dst = slot + ((u / KPC) << 10) + ((crow + 16 * (ku / KPC)) * KPC + ku % KPC) * (int)sizeof(T);
          if constexpr (sizeof(T) == 2) {
            const unsigned lo = (unsigned)Op<T>::from_f32(dz[0]) | ((unsigned)Op<T>::from_f32(dz[1]) << 16);
            const unsigned hi = (unsigned)Op<T>::from_f32(dz[2]) | ((unsigned)Op<T>::from_f32(dz[3]) << 16);
            *reinterpret_cast<uint2*>(dst) = make_uint2(lo, hi);
          } else {
            *reinterpret_cast<float4*>(dst) = make_float4(dz[0], dz[1], dz[2], dz[3]);
          }
        } else {
#pragma unroll
          for (int g = 0; g < G; ++g)
            *reinterpret_cast<T*>(slot + ((g * P + rank) << 10) + rbo) = Op<T>::from_f32(dz[g]);
        }
      }
      publish(flags + rank, (unsigned)cnt);
      if (ACT && act && kk == n_t - 1) {
        // dz slots of ponder steps the tile did not run at step t: zeros
        for (int k2 = n_t; k2 < a.ponder_max; ++k2) {
          T* dzz = DZ + ((long)k2 * a.slot_rows + off_t + r0 + crow) * GBH + ju;
#pragma unroll
          for (int g = 0; g < G; ++g) dzz[(long)g * H] = Op<T>::from_f32(0.f);
        }
      }
      if (act) {
        T* dzr = DZ + ((long)(ACT ? kk : 0) * a.slot_rows + off_t + r0 + crow) * GBH + ju;
        if constexpr (G == 3) {   // [da_r, da_u, da_n, da_n * r]
          dzr[0] = Op<T>::from_f32(dz[0]);
          dzr[H] = Op<T>::from_f32(dz[1]);
          dzr[2L * H] = Op<T>::from_f32(dzx_n);
          dzr[3L * H] = Op<T>::from_f32(dz[2]);
          dbacc[0] += dz[0];
          dbacc[1] += dz[1];
          dbacc[2] += dzx_n;
          dbacc[3] += dz[2];
        } else {
#pragma unroll
          for (int g = 0; g < G; ++g) {
            dzr[(long)g * H] = Op<T>::from_f32(dz[g]);
            dbacc[g] += dz[g];
          }
        }
      }
      // phase 2
      if constexpr (UM)   // k-steps 4 r .. 4 r + 3 come from member r
        wait_flags(a, flags, ks0 / 4, (nks + 3) / 4, P, (unsigned)cnt);
      else
        wait_flags(a, flags, ks0, nks < 64 ? nks : 64, P, (unsigned)cnt);
      // the pops of the next iteration: ponder step kk-1 of this step, or the
      // previous step's last ponder step (ACT); the previous step otherwise
      auto fetch_next = [&]() {
        if constexpr (ACT) {
          if (kk > 0) fetch_act(pv[mt], t, kk - 1, n_t, mt, A_t, off_t, off_n, ntrip_of(t - 1, mt));
          else fetch_step(pv[mt], t - 1, mt, A_n, off_n, off_pn);
        } else {
          fetch(pv[mt], t - 1, mt, A_n, off_n, off_pn);
        }
      };
      const __amdgpu_buffer_rsrc_t rs = make_rsrc(slot, (unsigned)(a.ring_ks << 10));
      f32x4 acc[NCO];
#pragma unroll
      for (int ct = 0; ct < NCO; ++ct) acc[ct] = f32x4{0.f, 0.f, 0.f, 0.f};
      // the wave's k-steps of the dz tile straight into registers, KB at a
      // time (measured faster than loading them all into LDS at once); the
      // next iteration's pops behind the last batch
#pragma unroll
      for (int b0 = 0; b0 < KSW; b0 += KB) {
        uint4 av[KB];
#pragma unroll
        for (int i = 0; i < KB; ++i)
          av[i] = ld_chunk_l2(rs, b0 + i < nks ? (unsigned)(((ks0 + b0 + i) << 10) + lane * 16) : kOOB);
        if (b0 + KB >= KSW) fetch_next();
#pragma unroll
        for (int i = 0; i < KB; ++i) {
          const int ii = b0 + i;
          if (ii < KSW && ii < nks) {
#pragma unroll
            for (int ct = 0; ct < NCO; ++ct) {
              const uint4 bv = ii < KSR ? wr[ct][ii < KSR ? ii : 0]
                                        : lds[((wave * KSL + (ii - KSR)) * NCO + ct) * 64 + lane];
              acc[ct] = Mfma<T>::step(av[i], bv, acc[ct]);
            }
          }
        }
      }
      // partial products -> red (the previous tile's sums were read before
      // this step's publish barrier)
#pragma unroll
      for (int ct = 0; ct < NCO; ++ct)
#pragma unroll
        for (int e = 0; e < 4; ++e) red[(wave * 4 + e) * IS + ct * 64 + lane] = acc[ct][e];
      __syncthreads();
      if (act) {
        float s = rp[0];
#pragma unroll
        for (int w2 = 1; w2 < XNW; ++w2) s += rp[w2 * 4 * IS];
        dh[mt] = (G == 3 || GUARDED) ? s + dhu : s;
      }
      if constexpr (ACT) itb[mt] = cnt + 1;
      if constexpr (ROLE == 2) {
        // dy of the lower layer's output at step t for the own units; the
        // slot held step t+2, which the lower partner has read once it has
        // published that step (if the tile ran at t+2)
        if (r0 < win[t + 2 - wlo])
          wait_flags(a, a.peer_flags + (grp * a.MRT + mt) * 32, rank, 1, 32, (unsigned)(T_eff - (t + 2)));
        if (act) {
          const float* rx = rp + NCT * 64;
          float s = rx[0];
#pragma unroll
          for (int w2 = 1; w2 < XNW; ++w2) s += rx[w2 * 4 * IS];
          reinterpret_cast<float*>(a.dyx_ring)[dyx_off + crow * H + ju] = s;
        }
        publish(a.dyx_flags + (grp * a.MRT + mt) * 32 + rank, (unsigned)(T_eff - t));
      }
      }   // ponder iterations
    }
  }

#pragma unroll
  for (int mt = 0; mt < MRT_MAX; ++mt) {
    const int b = cellt ? sperm[mt * 16 + crow] : -1;
    if (b < 0) continue;
    if (a.dh0) a.dh0[(long)b * H + ju] = dh[mt];
    if (a.dc0) a.dc0[(long)b * H + ju] = dc[mt];
  }
  if (dbst) {
#pragma unroll
    for (int g = 0; g < GB; ++g) dbst[g] = dbacc[g];
  }
  // db partial of this work-group (its rows of this XCD), fixed order
  __syncthreads();
  if (cellt) {
#pragma unroll
    for (int g = 0; g < GB; ++g) red[(crow * GB + g) * HJ + cu] = dbacc[g];
  }
  __syncthreads();
  for (int c = tid; c < GB * HJ; c += XNT) {
    float s = 0.f;
    for (int m = 0; m < 16; ++m) s += red[m * GB * HJ + c];
    const int g = c / HJ, u = c - (c / HJ) * HJ;
    a.db_part[(long)grp * GBH + (long)g * H + j0 + u] = s;
  }
  // dx at the finished steps of every row: zeros, written by XCDs 1 .. 7
  // once their own steps are done (XCD 0 holds the longest rows, tile 0, so
  // the others end first): XCD x takes the batch rows b = x - 1 (mod 7), its
  // waves the rows, its members the steps
  if (a.dx_zero && t0 == 0 && grp > 0) {
    const bool bad = (a.err[0] & LL_DEVERR_SEQ_LEN_BIT) != 0;
    const int I4 = a.I >> 2;
    for (int b = grp - 1 + 7 * wave; b < B; b += 7 * XNW) {
      const int len = bad ? 0 : a.seq_len[b];
      for (int t = len + rank; t < a.T_max; t += P) {
        float4* row = reinterpret_cast<float4*>(a.dx_zero + ((long)t * B + b) * a.I);
        for (int i = lane; i < I4; i += 64) row[i] = make_float4(0.f, 0.f, 0.f, 0.f);
      }
    }
  }
}

template <typename T, int NCT, int KSW, int KSR, int MRT_MAX, int G, bool SKIP, bool ACT = false>
__global__ __launch_bounds__(XNT, 1) void xbwd_kernel(XLoopArgs a) {
  extern __shared__ uint4 lds[];
  __shared__ int s_info[2];
  join_group(a.rank_ctr, s_info);
  const int grp = uni(s_info[0]), rank = uni(s_info[1]);
  if (grp >= 8 || rank >= 32) {
    if (threadIdx.x == 0) {
      __hip_atomic_fetch_or(a.err, LL_DEVERR_BARRIER_BIT, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(a.abort_flag, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    return;
  }
  if (rank >= a.P) return;
  xbwd_body<T, NCT, KSW, KSR, MRT_MAX, 0, G, SKIP, ACT>(a, grp, rank, lds);
}

// Two-layer wavefront, gradient: members 0 .. P-1 of every XCD run the lower
// layer (a0) one step behind the upper layer (a1, members P .. 2P-1).
template <typename T, int NCT, int KSW, int KSRB, int KSRT, int MRT_MAX>
__global__ __launch_bounds__(XNT, 1) void xbwd2_kernel(XLoopArgs a0, XLoopArgs a1) {
  extern __shared__ uint4 lds[];
  __shared__ int s_info[2];
  join_group(a0.rank_ctr, s_info);
  const int grp = uni(s_info[0]), rank = uni(s_info[1]);
  if (grp >= 8 || rank >= 32) {
    if (threadIdx.x == 0) {
      __hip_atomic_fetch_or(a0.err, LL_DEVERR_BARRIER_BIT, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(a0.abort_flag, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    return;
  }
  if (rank < a0.P)
    xbwd_body<T, NCT, KSW, KSRB, MRT_MAX, 1>(a0, grp, rank, lds);
  else if (rank < a0.P + a1.P)
    xbwd_body<T, NCT, KSW, KSRT, MRT_MAX, 2>(a1, grp, rank - a0.P, lds);
}

// Forward loop set-up: the entering h rows (length order, operand type) into
// ring slot `slot` of every row tile in the consumers' lane order (the
// launch's first step t0 reads it as h_{t0-1}: slot (t0 + 1) % 2), and the
// launch's flags to zero.  One element per thread:
//   f = (((x * MRT + mt) * KS + ks) * 64 + l) * KPC + e
//   row r = (x + 8 mt) * 16 + l % 16, unit u = ks * 4 KPC + (l / 16) * KPC + e.
template <typename T>
__global__ __launch_bounds__(256) void x_prepare_fwd_kernel(XPrepArgs a) {
  x_prepare_body<T>(a, blockIdx.x, gridDim.x, 256);
}

__global__ __launch_bounds__(256) void zero_u32_kernel(unsigned* p, int n) {
  for (int i = blockIdx.x * 256 + threadIdx.x; i < n; i += gridDim.x * 256) p[i] = 0u;
}

template <typename T>
hipError_t launch_x_prepare_fwd(const float* h0, const int* perm, int B, int H, int mrt, int ring_ks,
                                int slot, void* ring, unsigned* flags, int nflags, hipStream_t s) {
  constexpr int KPC = Op<T>::kPerChunk;
  const long n = 8L * mrt * (H / (4 * KPC)) * 64 * KPC;
  long blocks = (n + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(x_prepare_fwd_kernel<T>, dim3((unsigned)blocks), dim3(256), 0, s,
                     XPrepArgs{h0, perm, B, H, mrt, ring_ks, slot, ring, flags, nflags});
  return hipGetLastError();
}
template hipError_t launch_x_prepare_fwd<float>(const float*, const int*, int, int, int, int, int, void*,
                                                unsigned*, int, hipStream_t);
template hipError_t launch_x_prepare_fwd<bf16_t>(const float*, const int*, int, int, int, int, int, void*,
                                                 unsigned*, int, hipStream_t);

__global__ __launch_bounds__(64) void copy_i32_kernel(const int* __restrict__ src, int* __restrict__ dst, int n) {
  for (int i = threadIdx.x; i < n; i += 64) dst[i] = src[i];
}

hipError_t launch_copy_i32(const int* src, int* dst, int n, hipStream_t s) {
  hipLaunchKernelGGL(copy_i32_kernel, dim3(1), dim3(64), 0, s, src, dst, n);
  return hipGetLastError();
}

hipError_t launch_zero_u32(unsigned* p, int n, hipStream_t s) {
  int blocks = (n + 255) / 256;
  if (blocks > 1024) blocks = 1024;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(zero_u32_kernel, dim3(blocks), dim3(256), 0, s, p, n);
  return hipGetLastError();
}

// ------------------------------------------------------------ launchers

// Kernel for a (dtype, H class, row tiles per XCD) combination.
//   bf16: HJ = 32 units, forward NCT 8, KSW = H/256; backward NCT 2, KSW = H/64.
//   f32:  HJ = 16 units, forward NCT 4, KSW = H/128; backward NCT 1, KSW = H/32.
// hc in {1, 2, 4} is the forward KSW (k-steps per wave, 8 waves); mrt <= 4
// row tiles per XCD.
namespace {
template <typename T, int NF, int NB, int HC, int RF, int RB, int MRT, int G = 4, bool SKIP = false,
          bool ACT = false>
XKernels x_make() {
  XKernels k{};
  k.fwd = reinterpret_cast<const void*>(&xfwd_kernel<T, NF, HC, RF, MRT, G, SKIP, ACT>);
  k.lds_fwd = xfwd_lds(HC, RF, NF, MRT, (SKIP || ACT) ? xfwd_skip_floats() : 0);
  k.bwd = reinterpret_cast<const void*>(&xbwd_kernel<T, NB, G * HC, RB, MRT, G, SKIP, ACT>);
  k.lds_bwd = xbwd_lds(G * HC, RB, NB, MRT);
  return k;
}
}  // namespace

// RF / RB: k-steps per wave whose weights stay in registers (the rest in LDS),
// chosen so that no instantiation spills.
//   bf16: HJ = 32 units, forward NCT 8, KSW = H/256; backward NCT 2, KSW = H/64.
//   f32:  HJ = 16 units, forward NCT 4, KSW = H/128; backward NCT 1, KSW = H/32.
// (LSTM; the Elman RNN has one gate block: forward NCT 2 / 1, backward KSW
// = H/256 / H/128, every weight in registers; the GRU three: forward NCT
// 6 / 3, backward KSW = 3H/256 / 3H/128.)
// hc in {1, 2, 4} is the forward KSW (k-steps per wave, 8 waves); mrt <= 4
template <typename T>
XKernels x_kernels(int hc, int mrt, int gates, bool skip, bool act) {
  constexpr bool bf = sizeof(T) == 2;
  constexpr int NF = bf ? 8 : 4;
  constexpr int NB = bf ? 2 : 1;
  const bool one = mrt <= 1;
  if (mrt > 4) return XKernels{};
  if (act) {   // the LSTM tiling with the nested-loop body
    if (gates != 4 || skip) return XKernels{};
    switch (hc) {
      case 1: return one ? x_make<T, NF, NB, 1, 1, 4, 1, 4, false, true>() : x_make<T, NF, NB, 1, 1, 4, 4, 4, false, true>();
      case 2: return one ? x_make<T, NF, NB, 2, 2, 8, 1, 4, false, true>() : x_make<T, NF, NB, 2, 2, 6, 4, 4, false, true>();
      case 4: return one ? x_make<T, NF, NB, 4, 4, 16, 1, 4, false, true>() : x_make<T, NF, NB, 4, 3, 8, 4, 4, false, true>();
      default: return XKernels{};
    }
  }
  if (skip) {   // the LSTM tiling with the cond body
    if (gates != 4) return XKernels{};
    switch (hc) {
      case 1: return one ? x_make<T, NF, NB, 1, 1, 4, 1, 4, true>() : x_make<T, NF, NB, 1, 1, 4, 4, 4, true>();
      case 2: return one ? x_make<T, NF, NB, 2, 2, 8, 1, 4, true>() : x_make<T, NF, NB, 2, 2, 6, 4, 4, true>();
      case 4: return one ? x_make<T, NF, NB, 4, 4, 16, 1, 4, true>() : x_make<T, NF, NB, 4, 3, 8, 4, 4, true>();
      default: return XKernels{};
    }
  }
  if (gates == 1) {
    constexpr int NR = bf ? 2 : 1;
    switch (hc) {
      case 1: return one ? x_make<T, NR, NB, 1, 1, 1, 1, 1>() : x_make<T, NR, NB, 1, 1, 1, 4, 1>();
      case 2: return one ? x_make<T, NR, NB, 2, 2, 2, 1, 1>() : x_make<T, NR, NB, 2, 2, 2, 4, 1>();
      case 4: return one ? x_make<T, NR, NB, 4, 4, 4, 1, 1>() : x_make<T, NR, NB, 4, 4, 4, 4, 1>();
      default: return XKernels{};
    }
  }
  if (gates == 3) {
    constexpr int NG = bf ? 6 : 3;
    switch (hc) {
      case 1: return one ? x_make<T, NG, NB, 1, 1, 3, 1, 3>() : x_make<T, NG, NB, 1, 1, 3, 4, 3>();
      case 2: return one ? x_make<T, NG, NB, 2, 2, 6, 1, 3>() : x_make<T, NG, NB, 2, 2, 6, 4, 3>();
      case 4: return one ? x_make<T, NG, NB, 4, 4, 12, 1, 3>() : x_make<T, NG, NB, 4, 4, 8, 4, 3>();
      default: return XKernels{};
    }
  }
  if (gates != 4) return XKernels{};
  switch (hc) {
    case 1: return one ? x_make<T, NF, NB, 1, 1, 4, 1>() : x_make<T, NF, NB, 1, 1, 4, 4>();
    case 2: return one ? x_make<T, NF, NB, 2, 2, 8, 1>() : x_make<T, NF, NB, 2, 2, 6, 4>();
    case 4: return one ? x_make<T, NF, NB, 4, 4, 16, 1>() : x_make<T, NF, NB, 4, 3, 8, 4>();
    default: return XKernels{};
  }
}

template XKernels x_kernels<float>(int, int, int, bool, bool);
template XKernels x_kernels<bf16_t>(int, int, int, bool, bool);

// Two-layer wavefront kernels: the lower layer as in x_kernels, the upper one
// with twice the forward k-steps (K = I_l + H = 2H) and, in the gradient, twice
// the output column tiles (W_h and W_x rows).  RFT / RBT: register k-steps of
// the upper layer's role.
namespace {
template <typename T, int NF, int NB, int HC, int RFB, int RFT, int RBB, int RBT, int MRT>
XKernels x_make2() {
  XKernels k{};
  k.fwd = reinterpret_cast<const void*>(&xfwd2_kernel<T, NF, HC, RFB, 2 * HC, RFT, MRT>);
  k.bwd = reinterpret_cast<const void*>(&xbwd2_kernel<T, NB, 4 * HC, RBB, RBT, MRT>);
  const size_t fb = xfwd_lds(HC, RFB, NF, MRT), ft = xfwd_lds(2 * HC, RFT, NF, MRT);
  const size_t bb = xbwd_lds(4 * HC, RBB, NB, MRT), bt = xbwd_lds(4 * HC, RBT, 2 * NB, MRT);
  k.lds_fwd = fb > ft ? fb : ft;
  k.lds_bwd = bb > bt ? bb : bt;
  return k;
}
}  // namespace

template <typename T>
XKernels x_kernels2(int hc, int mrt) {
  constexpr bool bf = sizeof(T) == 2;
  constexpr int NF = bf ? 8 : 4;
  constexpr int NB = bf ? 2 : 1;
  const bool one = mrt <= 1;
  if (mrt > 4) return XKernels{};
  switch (hc) {
    case 1: return one ? x_make2<T, NF, NB, 1, 1, 2, 4, 4, 1>() : x_make2<T, NF, NB, 1, 1, 2, 4, 4, 4>();
    case 2: return one ? x_make2<T, NF, NB, 2, 2, 4, 8, 6, 1>() : x_make2<T, NF, NB, 2, 2, 3, 6, 5, 4>();
    default: return XKernels{};
  }
}

template XKernels x_kernels2<float>(int, int);
template XKernels x_kernels2<bf16_t>(int, int);

hipError_t x_setup(const XKernels& k, int* occ_fwd, int* occ_bwd) {
  // a variant that spills more than a few registers to scratch is not used
  hipFuncAttributes fa{}, fb{};
  hipError_t e = hipFuncGetAttributes(&fa, k.fwd);
  if (e != hipSuccess) return e;
  e = hipFuncGetAttributes(&fb, k.bwd);
  if (e != hipSuccess) return e;
  if (fa.localSizeBytes > 32 || fb.localSizeBytes > 32) {
    *occ_fwd = 0;
    *occ_bwd = 0;
    return hipSuccess;
  }
  e = hipFuncSetAttribute(k.fwd, hipFuncAttributeMaxDynamicSharedMemorySize, (int)k.lds_fwd);
  if (e != hipSuccess) return e;
  e = hipFuncSetAttribute(k.bwd, hipFuncAttributeMaxDynamicSharedMemorySize, (int)k.lds_bwd);
  if (e != hipSuccess) return e;
  e = hipOccupancyMaxActiveBlocksPerMultiprocessor(occ_fwd, k.fwd, XNT, k.lds_fwd);
  if (e != hipSuccess) return e;
  return hipOccupancyMaxActiveBlocksPerMultiprocessor(occ_bwd, k.bwd, XNT, k.lds_bwd);
}

hipError_t x_launch(const void* fn, const XLoopArgs& a, int nwg, size_t lds, hipStream_t s) {
  XLoopArgs copy = a;
  void* kargs[] = {&copy};
  return hipLaunchKernel(fn, dim3(nwg), dim3(XNT), kargs, lds, s);
}

hipError_t x_launch2(const void* fn, const XLoopArgs& a0, const XLoopArgs& a1, int nwg, size_t lds,
                     hipStream_t s) {
  XLoopArgs c0 = a0, c1 = a1;
  void* kargs[] = {&c0, &c1};
  return hipLaunchKernel(fn, dim3(nwg), dim3(XNT), kargs, lds, s);
}

}  // namespace ll
