// Chip-wide variants of the two device-side loops, for shapes whose
// recurrent weights need more than one XCD (bf16 H = 2048: W_h is 32 MB; f32
// H = 1024: 16 MB).  The weights stay in registers for the whole loop, split
// over all 256 work-groups, and the loop state crosses XCDs every step.
//
// Work split.  XCD x owns hidden units [x UX, (x+1) UX), UX = H / 8.  Its 32
// work-groups form a KG x NG grid (rank = kq NG + nq): work-group (kq, nq)
// holds the weights of reduction slice kq (KC = H / 2 rows of the product's
// reduction dimension) for the output columns of N-group nq, and runs the
// cell of CW units of that N-group (the N-group's units split KG ways).
//   forward:  z = h_{t-1} W_h, K = H, KG = 2, NG = 16; N-group columns are
//             the 4 gates of UN = 4 NCT units.
//   gradient: dh_{t-1} = dz_t W_h^T, K = 4H, KG = 8, NG = 4; N-group
//             columns are UN = 16 NCT units.
// Both give every work-group KC x 16 NCT weights (KSW k-steps per wave, the
// K slice split over 8 waves) and CW = 2 NCT cell units.  Every row tile of
// the batch runs on every work-group.
//
// One step (forward; the gradient loop is the same with its cell first):
//   phase A: for every running row tile, wait until the producers of the
//     wave's k-steps of h_{t-1} have published them, load them from the
//     exchange ring (device-scope loads, two tiles ahead), multiply, reduce
//     the 8 waves' partials in LDS (two buffers, one barrier per tile) and
//     store the work-group's partial product (16 rows x 16 NCT columns);
//     then publish all tiles' partials at once.
//   phase B: wait for the KG partial products of the own N-group, sum them,
//     add the input projection, run the cell for CW units of every row, store
//     h_t into the ring with device-scope stores (written through to where
//     every XCD's loads see it), publish; then the h history, stack and y.
// Ring slots (two per row tile) and partial slots (two) are reused two steps
// later; every writer of a slot has, through the chain of flags it waited
// for, seen every reader of the slot's previous contents finish.  Every wait
// has the loop's wall-clock limit and abort flag.
#include "ll_kernels.h"
#include "ll_exchange.h"

namespace ll {

constexpr int CNW = 8;
constexpr int CNT = 64 * CNW;
constexpr int CWIN = 256;    // steps of loop metadata kept in LDS

template <typename T, int KSW, int NCT>
struct CShape {
  static constexpr int KPC = Op<T>::kPerChunk;
  static constexpr int H = 64 * KSW * KPC;
  static constexpr int UX = H / 8;         // units per XCD
  static constexpr int KC = H / 2;         // reduction slice per work-group (both loops)
  static constexpr int CW = 2 * NCT;       // cell units per work-group
  static constexpr int CT = 16 * CW;       // cell threads per row tile
  static constexpr int TPP = CNT / CT;     // row tiles per cell pass
  static constexpr int PW = 16 * 16 * NCT; // partial floats per (work-group, row tile)
  static constexpr int RB = CNW * NCT * 256;  // floats of one LDS partial buffer
  static constexpr int EPT = NCT / 2;          // partial floats each thread reduces
  static_assert(EPT == 1 || EPT == 2, "reduction split");
  static constexpr int NPROD = KSW * 4 * KPC / CW;   // producers of one wave's k-steps
  static_assert(KSW * KPC == 8 * NCT, "H = 64 KSW KPC = 512 NCT");
  static_assert(CW % KPC == 0 && CT % 64 == 0 && TPP * CT == CNT, "cell layout");
  static_assert(NPROD <= 64, "one lane per producer");
};

namespace {

__device__ __forceinline__ void c_window(const CLoopArgs& a, int* win, int lo) {
  __syncthreads();
  for (int i = threadIdx.x; i <= CWIN; i += blockDim.x) {
    const int t = lo + i;
    win[i] = (t >= 0 && t <= a.T_max) ? a.active[t] : 0;
    win[CWIN + 1 + i] = (t >= 0 && t <= a.T_max) ? a.off[t] : 0;
  }
  __syncthreads();
}

__device__ __forceinline__ void c_fail(const CLoopArgs& a) {
  if (threadIdx.x == 0) {
    __hip_atomic_fetch_or(a.err, LL_DEVERR_BARRIER_BIT, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(a.abort_flag, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// Work-group (0..255 over the chip) of the cell that produces unit j, for a
// KG x NG split with NG-group width UN and cell width CW.
template <int UX, int UN, int CW, int NG>
__device__ __forceinline__ int producer_of(int j) {
  const int v = j % UX;
  return (j / UX) * 32 + ((v % UN) / CW) * NG + v / UN;
}

// Wait until every flag this lane names is >= need: flag (tile m, producer
// pr) for the pairs i = lane + 64 j < n_pairs, m = i / NPROD, pr = i % NPROD;
// flag index m * 256 + prod[pr] where prod is the lane's producer table.
template <int NPROD, int NJ>
__device__ __forceinline__ void wait_tiles(const CLoopArgs& a, const unsigned* flags, int nt, int my_prod,
                                           unsigned need) {
  const int lane = threadIdx.x & 63;
  const unsigned* fp[NJ];
  bool mine[NJ];
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const int i = lane + 64 * j;
    const int m = i / NPROD, pr = i % NPROD;
    // the producer of pair i is the one lane pr names
    const int id = __shfl(my_prod, pr, 64);
    mine[j] = m < nt;
    fp[j] = flags + (mine[j] ? m * 256 + id : 0);
  }
  unsigned long long t0 = 0;
  unsigned polls = 0;
  while (true) {
    bool pend = false;
#pragma unroll
    for (int j = 0; j < NJ; ++j)
      pend |= mine[j] && __hip_atomic_load(fp[j], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < need;
    if (__builtin_amdgcn_ballot_w64(pend) == 0) return;
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

// The 8 waves' partial products of one row tile, summed: thread tid takes
// EPT of the 4 rows of item (column tile, lane) it = tid / (4 / EPT), the
// LDS buffer being [wave][item] float4.  out(c, rq, e, v) receives column
// c = ct*16 + lane % 16, row 4 rq + e.
template <int NCT, int EPT, typename Out>
__device__ __forceinline__ void reduce_waves(const float4* rb, Out out) {
  const int tid = threadIdx.x;
  const int it = tid / (4 / EPT), e0 = (tid % (4 / EPT)) * EPT;
  const float* rf = reinterpret_cast<const float*>(rb) + it * 4 + e0;
  float v[EPT];
#pragma unroll
  for (int i = 0; i < EPT; ++i) v[i] = rf[i];
#pragma unroll
  for (int w2 = 1; w2 < CNW; ++w2)
#pragma unroll
    for (int i = 0; i < EPT; ++i) v[i] += rf[w2 * NCT * 256 + i];
  const int c = (it >> 6) * 16 + (it & 15), rq = (it >> 4) & 3;
#pragma unroll
  for (int i = 0; i < EPT; ++i) out(c, rq, e0 + i, v[i]);
}

// Byte offset of element (row, column n) of row tile m in ring slot sl:
// blocks of 4 KPC columns, lane l of a block holding row l % 16, columns
// (l / 16) KPC .. + KPC.
template <typename T>
__device__ __forceinline__ unsigned ring_off(int sl, int mrt, int ks_tile, int m, int row, int n) {
  constexpr int KPC = Op<T>::kPerChunk;
  const int ks = n / (4 * KPC), cq = (n % (4 * KPC)) / KPC, e = n % KPC;
  return (unsigned)(((((sl * mrt + m) * ks_tile + ks) * 64 + cq * 16 + row) * 16) + e * (int)sizeof(T));
}

}  // namespace

// ---------------------------------------------------------------------------
// Forward loop, chip-wide.
// ---------------------------------------------------------------------------
template <typename T, int KSW, int NCT, int MRT_MAX>
__global__ __launch_bounds__(CNT, 1) void cfwd_kernel(CLoopArgs a) {
  using S = CShape<T, KSW, NCT>;
  constexpr int KPC = S::KPC, H = S::H, UX = S::UX, KC = S::KC, CW = S::CW, CT = S::CT;
  constexpr int TPP = S::TPP, PW = S::PW, RB = S::RB, NPROD = S::NPROD, EPT = S::EPT;
  constexpr int KG = 2, NG = 16, UN = 4 * NCT;
  constexpr int KS = H / (4 * KPC);
  constexpr int NPASS = (MRT_MAX + TPP - 1) / TPP;
  static_assert(NPASS * KG <= 64, "one lane per partial flag");
  constexpr long G4 = 4L * H, H5 = 5L * H;
  __shared__ float4 red[2 * RB / 4];
  __shared__ int win[2 * (CWIN + 1)];
  __shared__ int sperm[MRT_MAX * 16];
  __shared__ int s_info[2];

  join_group(a.rank_ctr, s_info);
  const int x = uni(s_info[0]), rank = uni(s_info[1]);
  if (x >= 8 || rank >= 32 || a.H != H || a.MRT > MRT_MAX) {
    c_fail(a);
    return;
  }
  const int kq = rank / NG, nq = rank % NG;
  const int tid = threadIdx.x, lane = tid & 63, wave = uni(tid >> 6);
  const int q = lane >> 4, l16 = lane & 15;
  const int B = a.B, MRT = a.MRT;
  const T* WT = reinterpret_cast<const T*>(a.W);
  T* HH = reinterpret_cast<T*>(a.X);
  const int kb0 = kq * (KC / (4 * KPC)) + wave * KSW;   // first k-step of this wave

  // weight slice: lane column l16 of column tile ct is local column
  // ct*16 + l16 = gate * UN + u
  uint4 wr[NCT][KSW];
#pragma unroll
  for (int ct = 0; ct < NCT; ++ct) {
    const int c = ct * 16 + l16;
    const int g = c / UN, u = c - g * UN;
    const T* wcol = WT + ((long)g * H + x * UX + nq * UN + u) * a.ldw + a.woff;
#pragma unroll
    for (int i = 0; i < KSW; ++i) wr[ct][i] = ld16(wcol + ((kb0 + i) * 4 + q) * KPC);
  }
  for (int i = tid; i < MRT_MAX * 16; i += CNT) sperm[i] = i < B ? a.perm[i] : -1;

  // cell thread: tile slot tp of a pass, row crow, unit jc
  const int tp = uni(tid / CT), crow = (tid / CW) & 15, uu = tid % CW;
  const int jc = x * UX + nq * UN + kq * CW + uu;
  __syncthreads();
  float hs[NPASS], cs[NPASS];
#pragma unroll
  for (int p = 0; p < NPASS; ++p) {
    const int m = p * TPP + tp;
    const int b = m < MRT ? sperm[m * 16 + crow] : -1;
    hs[p] = (b >= 0 && a.h0) ? a.h0[(long)b * H + jc] : 0.f;
    cs[p] = (b >= 0 && a.c0) ? a.c0[(long)b * H + jc] : 0.f;
  }

  const int T_eff = uni(a.meta[0]);
  const int t1 = min(a.T_max, T_eff);
  int wlo = 0;
  c_window(a, win, 0);
  const __amdgpu_buffer_rsrc_t rring = make_rsrc(a.ring, (unsigned)(2 * MRT * KS) << 10);
  const __amdgpu_buffer_rsrc_t rpart = make_rsrc(a.part, (unsigned)(2L * 8 * MRT * 32 * PW * 4));

  // input projections of the cell thread's rows at step t
  float zx[NPASS][4];
  auto load_zx = [&](int t) {
    const int A = uni(win[t - wlo]), off = uni(win[CWIN + 1 + t - wlo]);
    const __amdgpu_buffer_rsrc_t rz = make_rsrc(a.Zx + (long)off * G4, (unsigned)(A * G4 * 4));
#pragma unroll
    for (int p = 0; p < NPASS; ++p) {
      const int r = (p * TPP + tp) * 16 + crow;
      const unsigned zo = r < A ? (unsigned)((r * G4 + jc) * 4) : kOOB;
#pragma unroll
      for (int g = 0; g < 4; ++g) zx[p][g] = ld_f32(rz, zo + g * H * 4);
    }
  };
  // h history, stack row and y of step tt (A rows running from compact
  // offset off), from the cell registers, after h_tt is published
  float gv[NPASS][5];
  auto flush = [&](int tt, int A, int off) {
#pragma unroll
    for (int p = 0; p < NPASS; ++p) {
      const int m = p * TPP + tp, r = m * 16 + crow;
      const bool act = r < A;
      if (act) {
        const long cr = off + r;
        HH[cr * H + jc] = Op<T>::from_f32(hs[p]);
        if (a.stack) {
          float* st = a.stack + cr * H5 + jc;
#pragma unroll
          for (int c = 0; c < 5; ++c) st[(long)c * H] = gv[p][c];
        }
      }
      if (a.y && m < MRT) {
        const int b = sperm[r];
        if (b >= 0) a.y[((long)tt * B + b) * H + jc] = act ? hs[p] : 0.f;
      }
    }
  };

  for (int t = 0; t < t1; ++t) {
    if (t + 1 > wlo + CWIN) {
      wlo = t;
      c_window(a, win, wlo);
    }
    const int A_t = uni(win[t - wlo]), off_t = uni(win[CWIN + 1 + t - wlo]);
    const int nt = (A_t + 15) >> 4;
    const int sl = t & 1;

    // ---- phase A: partial products of every running tile
    // every producer of this wave's k-steps has published h_{t-1} of every
    // running tile (one wait for all tiles: they are published together)
    if (t > 0)
      wait_tiles<NPROD, (MRT_MAX * NPROD + 63) / 64>(
          a, a.xflags, nt, producer_of<UX, UN, CW, NG>(kb0 * 4 * KPC + (lane % NPROD) * CW), (unsigned)(t + 1));
    auto load_a = [&](int m, uint4 (&v)[KSW]) {
      const __amdgpu_buffer_rsrc_t rs =
          make_rsrc(reinterpret_cast<char*>(a.ring) + ((long)((sl ^ 1) * MRT + m) * KS << 10), (unsigned)KS << 10);
#pragma unroll
      for (int i = 0; i < KSW; ++i) v[i] = ld_chunk_l2(rs, (unsigned)(((kb0 + i) << 10) + lane * 16));
    };
    // tile m: operands in cur; the operands of tile m+2 go to nxt2
    auto tile = [&](int m, uint4 (&cur)[KSW], uint4 (&nxt2)[KSW]) {
      if (m + 2 < nt) load_a(m + 2, nxt2);
      // the input projections of this step, issued after the next tiles'
      // operands so that the first products do not wait for them
      if (m == 0) load_zx(t);
      f32x4 acc[NCT];
#pragma unroll
      for (int ct = 0; ct < NCT; ++ct) acc[ct] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int i = 0; i < KSW; ++i)
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct) acc[ct] = Mfma<T>::step(cur[i], wr[ct][i], acc[ct]);
      // LDS buffer m % 2: [wave][ct][lane] float4 (the lane's 4 result rows)
      float4* rb = red + (m & 1) * (RB / 4);
#pragma unroll
      for (int ct = 0; ct < NCT; ++ct)
        rb[(wave * NCT + ct) * 64 + lane] = make_float4(acc[ct][0], acc[ct][1], acc[ct][2], acc[ct][3]);
      __syncthreads();
      // column c = gate * UN + kc * CW + uu; partial layout
      // [kc][row / 4][uu][row % 4][gate], so that a cell reads its 4 gates
      // as one 16-byte load
      float* pd = a.part + ((long)((sl * 8 + x) * MRT + m) * 32 + rank) * PW;
      reduce_waves<NCT, EPT>(rb, [&](int c, int rq, int e, float v) {
        const int g = c / UN, u = c - g * UN, kc = u / CW, ou = u - kc * CW;
        pd[(((kc * 4 + rq) * CW + ou) * 4 + e) * 4 + g] = v;
      });
    };
    // three operand buffers with fixed roles per unrolled tile, so that no
    // register copy waits for a load in flight
    uint4 a0[KSW], a1[KSW], a2[KSW];
    load_a(0, a0);
    if (nt > 1) load_a(1, a1);
    for (int m = 0; m < nt; m += 3) {
      tile(m, a0, a2);
      if (m + 1 < nt) tile(m + 1, a1, a0);
      if (m + 2 < nt) tile(m + 2, a2, a1);
    }
    wait_all_vm();
    __syncthreads();
    if (tid < nt)
      __hip_atomic_store(a.pflags + (x * MRT + tid) * 32 + rank, (unsigned)(t + 2), __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);

    // ---- phase B: the KG partial products of this N-group, cells
    {
      const int p = lane / KG, k = lane % KG;
      const int m = p * TPP + tp;
      wait_each(a, a.pflags, (x * MRT + m) * 32 + k * NG + nq, lane < NPASS * KG && m < nt, (unsigned)(t + 2));
    }
    float zs[NPASS][4];
#pragma unroll
    for (int p = 0; p < NPASS; ++p) {
      const int m = p * TPP + tp;
#pragma unroll
      for (int g = 0; g < 4; ++g) zs[p][g] = zx[p][g];
      if (m < nt) {
        const long base = (long)((sl * 8 + x) * MRT + m) * 32 * PW;
#pragma unroll
        for (int k = 0; k < KG; ++k) {
          const uint4 v = ld_chunk_l2(rpart, (unsigned)((base + (long)(k * NG + nq) * PW +
                                                         (((kq * 4 + (crow >> 2)) * CW + uu) * 4 + (crow & 3)) * 4) *
                                                        4));
          zs[p][0] += __uint_as_float(v.x);
          zs[p][1] += __uint_as_float(v.y);
          zs[p][2] += __uint_as_float(v.z);
          zs[p][3] += __uint_as_float(v.w);
        }
      }
    }
#pragma unroll
    for (int p = 0; p < NPASS; ++p) {
      const int m = p * TPP + tp, r = m * 16 + crow;
      gv[p][0] = sigmoidf_(zs[p][0]);
      gv[p][1] = sigmoidf_(zs[p][1]);
      gv[p][2] = tanhf_(zs[p][2]);
      gv[p][3] = sigmoidf_(zs[p][3]);
      gv[p][4] = gv[p][1] * cs[p] + gv[p][0] * gv[p][2];
      if (m < nt && r < A_t) {
        cs[p] = gv[p][4];
        hs[p] = gv[p][3] * tanhf_(gv[p][4]);
        st_dev(rring, ring_off<T>(sl, MRT, KS, m, crow, jc), Op<T>::from_f32(hs[p]));
      }
    }
    wait_all_vm();
    __syncthreads();
    if (tid < nt)
      __hip_atomic_store(a.xflags + tid * 256 + x * 32 + rank, (unsigned)(t + 2), __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
    flush(t, A_t, off_t);
  }

#pragma unroll
  for (int p = 0; p < NPASS; ++p) {
    const int m = p * TPP + tp;
    const int b = m < MRT ? sperm[m * 16 + crow] : -1;
    if (b < 0) continue;
    a.hT[(long)b * H + jc] = hs[p];
    a.cT[(long)b * H + jc] = cs[p];
    if (a.y)
      for (int t = max(T_eff, 0); t < a.T_max; ++t) a.y[((long)t * B + b) * H + jc] = 0.f;
  }
}

// ---------------------------------------------------------------------------
// Gradient loop, chip-wide.  Step t (descending):
//   phase B': dh_t of the rows that ran at step t+1 is the sum of the KG
//     partial products of step t+1 (other rows keep dhT); with the values
//     popped for step t: dh_tot, dc, dz; dz into the ring, publish; then the
//     dz rows for the dW and dx products and db; pops of step t-1 issued;
//   phase A': partial products of dh_{t-1} = dz_t W_h^T for every running
//     tile, published at once.
// After the last step, dh0 of the rows that ran at step 0 is the sum of the
// partial products of step 0.
// ---------------------------------------------------------------------------
template <typename T, int KSW, int NCT, int MRT_MAX>
__global__ __launch_bounds__(CNT, 1) void cbwd_kernel(CLoopArgs a) {
  using S = CShape<T, KSW, NCT>;
  constexpr int KPC = S::KPC, H = S::H, UX = S::UX, KC = S::KC, CW = S::CW, CT = S::CT;
  constexpr int TPP = S::TPP, PW = S::PW, RB = S::RB, NPROD = S::NPROD, EPT = S::EPT;
  constexpr int KG = 8, NG = 4, UN = 16 * NCT;
  constexpr int KS = 4 * H / (4 * KPC);
  constexpr int NPASS = (MRT_MAX + TPP - 1) / TPP;
  static_assert(NPASS * KG <= 64, "one lane per partial flag");
  constexpr long G4 = 4L * H, H5 = 5L * H;
  __shared__ float4 red[2 * RB / 4];
  __shared__ int win[2 * (CWIN + 1)];
  __shared__ int sperm[MRT_MAX * 16];
  __shared__ int s_info[2];

  join_group(a.rank_ctr, s_info);
  const int x = uni(s_info[0]), rank = uni(s_info[1]);
  if (x >= 8 || rank >= 32 || a.H != H || a.MRT > MRT_MAX) {
    c_fail(a);
    return;
  }
  const int kq = rank / NG, nq = rank % NG;
  const int tid = threadIdx.x, lane = tid & 63, wave = uni(tid >> 6);
  const int q = lane >> 4, l16 = lane & 15;
  const int B = a.B, MRT = a.MRT;
  const T* W = reinterpret_cast<const T*>(a.W);
  T* DZ = reinterpret_cast<T*>(a.X);
  const int kb0 = kq * (KC / (4 * KPC)) + wave * KSW;   // first dz k-step of this wave

  // weight slice: output column ct*16 + l16 is unit x UX + nq UN + ct*16 + l16;
  // the product's reduction runs over the 4H columns of W
  uint4 wr[NCT][KSW];
#pragma unroll
  for (int ct = 0; ct < NCT; ++ct) {
    const T* wrow = W + (long)(a.woff + x * UX + nq * UN + ct * 16 + l16) * G4;
#pragma unroll
    for (int i = 0; i < KSW; ++i) wr[ct][i] = ld16(wrow + ((kb0 + i) * 4 + q) * KPC);
  }
  for (int i = tid; i < MRT_MAX * 16; i += CNT) sperm[i] = i < B ? a.perm[i] : -1;

  const int tp = uni(tid / CT), crow = (tid / CW) & 15, uu = tid % CW;
  const int jc = x * UX + nq * UN + kq * CW + uu;
  __syncthreads();
  float dh[NPASS], dc[NPASS];
#pragma unroll
  for (int p = 0; p < NPASS; ++p) {
    const int m = p * TPP + tp;
    const int b = m < MRT ? sperm[m * 16 + crow] : -1;
    dh[p] = (b >= 0 && a.dhT) ? a.dhT[(long)b * H + jc] : 0.f;
    dc[p] = (b >= 0 && a.dcT) ? a.dcT[(long)b * H + jc] : 0.f;
  }
  float dbacc[4] = {0.f, 0.f, 0.f, 0.f};

  const int T_eff = uni(a.meta[0]);
  const int t1 = min(a.T_max, T_eff);
  // the window covers steps t-2 .. t+1 of every step t
  int wlo = t1 + 1 - CWIN > 0 ? t1 + 1 - CWIN : 0;
  c_window(a, win, wlo);
  const __amdgpu_buffer_rsrc_t rring = make_rsrc(a.ring, (unsigned)(2 * MRT * KS) << 10);
  const __amdgpu_buffer_rsrc_t rpart = make_rsrc(a.part, (unsigned)(2L * 8 * MRT * 32 * PW * 4));

  // pops of step tt for the cell thread's rows: i, f, g, o, c_t, c_{t-1}, dy
  float pv[NPASS][7];
  auto fetch = [&](int tt) {
    const int A = uni(win[tt - wlo]), off = uni(win[CWIN + 1 + tt - wlo]);
    const int offp = tt > 0 ? uni(win[CWIN + 1 + tt - 1 - wlo]) : 0;
    const __amdgpu_buffer_rsrc_t rs = make_rsrc(a.stack + (long)off * H5, (unsigned)(A * H5 * 4));
    const __amdgpu_buffer_rsrc_t rp2 =
        make_rsrc(a.stack + (long)offp * H5 + 4L * H, tt > 0 ? (unsigned)(A * H5 * 4) : 0u);
    const __amdgpu_buffer_rsrc_t rc = make_rsrc(a.c0, (tt == 0 && a.c0) ? (unsigned)(B * H * 4) : 0u);
    const __amdgpu_buffer_rsrc_t rd =
        a.dy_compact ? make_rsrc(a.dy + (long)off * H, (unsigned)(A * H * 4))
                     : make_rsrc(a.dy ? a.dy + (long)tt * B * H : nullptr, a.dy ? (unsigned)(B * H * 4) : 0u);
#pragma unroll
    for (int p = 0; p < NPASS; ++p) {
      const int m = p * TPP + tp, r = m * 16 + crow;
      const bool ok = r < A;
      const int b = m < MRT ? sperm[r] : 0;
      const unsigned so = ok ? (unsigned)((r * H5 + jc) * 4) : kOOB;
#pragma unroll
      for (int c = 0; c < 5; ++c) pv[p][c] = ld_f32(rs, so + c * H * 4);
      pv[p][5] = tt > 0 ? ld_f32(rp2, so) : ld_f32(rc, ok ? (unsigned)((b * H + jc) * 4) : kOOB);
      pv[p][6] = ld_f32(rd, ok ? (unsigned)((a.dy_compact ? r * H + jc : b * H + jc) * 4) : kOOB);
    }
  };
  // dh of the rows that ran at step tt from the partial products of that
  // step (slot tt % 2); A_tt rows, value T_eff - tt
  auto gather_dh = [&](int tt, int A_tt) {
    const int ntt = (A_tt + 15) >> 4;
    {
      const int p = lane / KG, k = lane % KG;
      const int m = p * TPP + tp;
      wait_each(a, a.pflags, (x * MRT + m) * 32 + k * NG + nq, lane < NPASS * KG && m < ntt,
                (unsigned)(T_eff - tt));
    }
#pragma unroll
    for (int p = 0; p < NPASS; ++p) {
      const int m = p * TPP + tp, r = m * 16 + crow;
      if (m < ntt) {
        const long base = (long)(((tt & 1) * 8 + x) * MRT + m) * 32 * PW;
        float s = 0.f;
#pragma unroll
        for (int k = 0; k < KG; ++k)
          s += ld_f32_l2(rpart, (unsigned)((base + (long)(k * NG + nq) * PW +
                                            ((kq * 4 + (crow >> 2)) * CW + uu) * 4 + (crow & 3)) * 4));
        if (r < A_tt) dh[p] = s;
      }
    }
  };

  if (t1 > 0) fetch(t1 - 1);
  for (int t = t1 - 1; t >= 0; --t) {
    if (t - 2 < wlo && wlo > 0) {
      wlo = t + 1 - CWIN > 0 ? t + 1 - CWIN : 0;
      c_window(a, win, wlo);
    }
    const int A_t = uni(win[t - wlo]), off_t = uni(win[CWIN + 1 + t - wlo]);
    const int nt = (A_t + 15) >> 4;
    const int sl = t & 1;

    // ---- phase B'
    if (t + 1 < t1) gather_dh(t + 1, uni(win[t + 1 - wlo]));
    float dz[NPASS][4];
#pragma unroll
    for (int p = 0; p < NPASS; ++p) {
      const int m = p * TPP + tp, r = m * 16 + crow;
#pragma unroll
      for (int g = 0; g < 4; ++g) dz[p][g] = 0.f;
      if (m < nt && r < A_t) {
        const float dht = dh[p] + pv[p][6];
        const float ig = pv[p][0], fg = pv[p][1], gg = pv[p][2], og = pv[p][3];
        const float c = pv[p][4], cp = pv[p][5];
        const float tc = tanhf_(c);
        const float d_o = dht * tc;
        const float dct = dc[p] + dht * og * (1.f - tc * tc);
        dz[p][0] = dct * gg * (ig * (1.f - ig));
        dz[p][1] = dct * cp * (fg * (1.f - fg));
        dz[p][2] = dct * ig * (1.f - gg * gg);
        dz[p][3] = d_o * (og * (1.f - og));
        dc[p] = dct * fg;
#pragma unroll
        for (int g = 0; g < 4; ++g)
          st_dev(rring, ring_off<T>(sl, MRT, KS, m, crow, g * H + jc), Op<T>::from_f32(dz[p][g]));
      }
    }
    wait_all_vm();
    __syncthreads();
    if (tid < nt)
      __hip_atomic_store(a.xflags + tid * 256 + x * 32 + rank, (unsigned)(T_eff - t), __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
#pragma unroll
    for (int p = 0; p < NPASS; ++p) {
      const int m = p * TPP + tp, r = m * 16 + crow;
      if (m < nt && r < A_t) {
        T* dzr = DZ + (long)(off_t + r) * G4 + jc;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          dzr[(long)g * H] = Op<T>::from_f32(dz[p][g]);
          dbacc[g] += dz[p][g];
        }
      }
    }

    // ---- phase A': partial products of dh_{t-1}
    // every producer of this wave's dz columns has published dz_t of every
    // running tile (the wave's columns lie in one gate block)
    wait_tiles<NPROD, (MRT_MAX * NPROD + 63) / 64>(
        a, a.xflags, nt, producer_of<UX, UN, CW, NG>((kb0 * 4 * KPC + (lane % NPROD) * CW) % H),
        (unsigned)(T_eff - t));
    auto load_a = [&](int m, uint4 (&v)[KSW]) {
      const __amdgpu_buffer_rsrc_t rs =
          make_rsrc(reinterpret_cast<char*>(a.ring) + ((long)(sl * MRT + m) * KS << 10), (unsigned)KS << 10);
#pragma unroll
      for (int i = 0; i < KSW; ++i) v[i] = ld_chunk_l2(rs, (unsigned)(((kb0 + i) << 10) + lane * 16));
    };
    auto tile = [&](int m, uint4 (&cur)[KSW], uint4 (&nxt2)[KSW]) {
      if (m + 2 < nt) load_a(m + 2, nxt2);
      // pops of step t-1, issued after the next tiles' operands
      if (m == 0 && t >= 1) fetch(t - 1);
      f32x4 acc[NCT];
#pragma unroll
      for (int ct = 0; ct < NCT; ++ct) acc[ct] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int i = 0; i < KSW; ++i)
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct) acc[ct] = Mfma<T>::step(cur[i], wr[ct][i], acc[ct]);
      float4* rb = red + (m & 1) * (RB / 4);
#pragma unroll
      for (int ct = 0; ct < NCT; ++ct)
        rb[(wave * NCT + ct) * 64 + lane] = make_float4(acc[ct][0], acc[ct][1], acc[ct][2], acc[ct][3]);
      __syncthreads();
      // local unit c = kc * CW + uu; partial layout [kc][row / 4][uu][row % 4]
      float* pd = a.part + ((long)((sl * 8 + x) * MRT + m) * 32 + rank) * PW;
      reduce_waves<NCT, EPT>(rb, [&](int c, int rq, int e, float v) {
        const int kc = c / CW, ou = c - kc * CW;
        pd[((kc * 4 + rq) * CW + ou) * 4 + e] = v;
      });
    };
    uint4 a0[KSW], a1[KSW], a2[KSW];
    load_a(0, a0);
    if (nt > 1) load_a(1, a1);
    for (int m = 0; m < nt; m += 3) {
      tile(m, a0, a2);
      if (m + 1 < nt) tile(m + 1, a1, a0);
      if (m + 2 < nt) tile(m + 2, a2, a1);
    }
    wait_all_vm();
    __syncthreads();
    if (tid < nt)
      __hip_atomic_store(a.pflags + (x * MRT + tid) * 32 + rank, (unsigned)(T_eff - t), __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
  }
  if (t1 > 0) gather_dh(0, uni(win[0 - wlo]));

#pragma unroll
  for (int p = 0; p < NPASS; ++p) {
    const int m = p * TPP + tp;
    const int b = m < MRT ? sperm[m * 16 + crow] : -1;
    if (b < 0) continue;
    if (a.dh0) a.dh0[(long)b * H + jc] = dh[p];
    if (a.dc0) a.dc0[(long)b * H + jc] = dc[p];
  }
  // db of the work-group's CW units (each unit's cell runs on exactly one
  // work-group): sum over the cell threads of the unit, fixed order
  __syncthreads();
  float* rf = reinterpret_cast<float*>(red);
#pragma unroll
  for (int g = 0; g < 4; ++g) rf[g * CNT + tid] = dbacc[g];
  __syncthreads();
  if (tid < 4 * CW) {
    const int g = tid / CW, u = tid % CW;
    float s = 0.f;
    for (int i = u; i < CNT; i += CW) s += rf[g * CNT + i];
    a.db[(long)g * H + x * UX + nq * UN + kq * CW + u] = s;
  }
}

// Set-up: h0 rows into ring slot 1 in the consumers' order, flags to zero.
//   f = ((m * KS + ks) * 64 + l) * KPC + e: row m*16 + l % 16,
//   unit ks * 4 KPC + (l / 16) * KPC + e.
template <typename T>
__global__ __launch_bounds__(256) void c_prepare_kernel(const float* __restrict__ h0,
                                                        const int* __restrict__ perm, int B, int H, int MRT,
                                                        void* ring, unsigned* flags, int nflags) {
  constexpr int KPC = Op<T>::kPerChunk;
  const int KS = H / (4 * KPC);
  const long n = (long)MRT * KS * 64 * KPC;
  T* slot1 = reinterpret_cast<T*>(ring) + n;
  for (long f = blockIdx.x * 256L + threadIdx.x; f < n; f += gridDim.x * 256L) {
    const int e = (int)(f % KPC);
    const int l = (int)((f / KPC) % 64);
    const int ks = (int)((f / (64 * KPC)) % KS);
    const int m = (int)(f / (64L * KPC * KS));
    const int r = m * 16 + (l & 15);
    const int u = ks * 4 * KPC + (l >> 4) * KPC + e;
    slot1[f] = Op<T>::from_f32((h0 && r < B) ? h0[(long)perm[r] * H + u] : 0.f);
  }
  for (long i = blockIdx.x * 256L + threadIdx.x; i < nflags; i += gridDim.x * 256L) flags[i] = 0u;
}

template <typename T>
hipError_t launch_c_prepare(const float* h0, const int* perm, int B, int H, int mrt, void* ring,
                            unsigned* flags, int nflags, hipStream_t s) {
  constexpr int KPC = Op<T>::kPerChunk;
  const long n = (long)mrt * (H / (4 * KPC)) * 64 * KPC;
  long blocks = (std::max(n, (long)nflags) + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(c_prepare_kernel<T>, dim3((unsigned)blocks), dim3(256), 0, s, h0, perm, B, H, mrt, ring,
                     flags, nflags);
  return hipGetLastError();
}
template hipError_t launch_c_prepare<float>(const float*, const int*, int, int, int, void*, unsigned*, int,
                                            hipStream_t);
template hipError_t launch_c_prepare<bf16_t>(const float*, const int*, int, int, int, void*, unsigned*, int,
                                             hipStream_t);

// Kernels for a (dtype, H): bf16 H = 2048 (KSW 4, NCT 4), f32 H = 1024 (KSW 4,
// NCT 2); up to 16 row tiles (B <= 256).
template <typename T>
CKernels c_kernels(int H, int mrt) {
  constexpr bool bf = sizeof(T) == 2;
  constexpr int NCT = bf ? 4 : 2;
  using S = CShape<T, 4, NCT>;
  CKernels k{};
  if (H != S::H || mrt < 1 || mrt > 16) return k;
  k.fwd = reinterpret_cast<const void*>(&cfwd_kernel<T, 4, NCT, 16>);
  k.bwd = reinterpret_cast<const void*>(&cbwd_kernel<T, 4, NCT, 16>);
  k.lds_fwd = 0;
  k.lds_bwd = 0;
  k.pw = S::PW;
  return k;
}
template CKernels c_kernels<float>(int, int);
template CKernels c_kernels<bf16_t>(int, int);

hipError_t c_setup(const CKernels& k, int* occ_fwd, int* occ_bwd) {
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
  e = hipOccupancyMaxActiveBlocksPerMultiprocessor(occ_fwd, k.fwd, CNT, 0);
  if (e != hipSuccess) return e;
  return hipOccupancyMaxActiveBlocksPerMultiprocessor(occ_bwd, k.bwd, CNT, 0);
}

hipError_t c_launch(const void* fn, const CLoopArgs& a, size_t lds, hipStream_t s) {
  CLoopArgs copy = a;
  void* kargs[] = {&copy};
  return hipLaunchKernel(fn, dim3(256), dim3(CNT), kargs, lds, s);
}

}  // namespace ll
