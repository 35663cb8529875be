// Kernel argument blocks and launchers of the lstmloop library (internal).
#pragma once

#include "ll_device.h"

namespace ll {

constexpr int LL_DEVERR_SEQ_LEN_BIT = 1;
constexpr int LL_DEVERR_BARRIER_BIT = 2;

// meta[] layout (device int array owned by a plan)
//   0: T_eff   1: total rows (sum of lengths)   2: error word   3: abort flag
//   4..7: grid-barrier counters
//   16 + 8 * launch + xcd: per-XCD rank counters of the XCD-local loops
//   (launch 0/1: forward layer 0/1, launch 2/3: backward layer 0/1)
constexpr int META_INTS = 64;
constexpr int META_RANK0 = 16;

struct GatherTArgs {
  const void* in;
  void* out;
  int C;
  int ldo;
  int mode;             // 0 rowmap gather, 1 compact, 2 previous-h history
  int B;
  const int* meta;
  const int* rowmap;
  const int* off;
  const int* perm;
  const float* h0f;     // mode 2, t = 0
};

// C[crow(m), n] = sum_k A[arow(m), k] * Bm[n, k] (+ bias[n]), both operands
// K-contiguous ("NT").  M, K may come from device memory (sum of lengths).
// The forward loop's entering state in its ring (slot `slot`, the operand
// layout: row r = (x + 8 mt) * 16 + l % 16 of XCD x, unit u = ks * 4 KPC +
// (l / 16) * KPC + e for lane l, element e of k-step ks; rows in length order
// through perm, zeros past B or without h0) and its flags cleared.
struct XPrepArgs {
  const float* h0;
  const int* perm;
  int B, H, MRT, ring_ks, slot;
  void* ring;
  unsigned* flags;
  int nflags;
};
template <typename T>
__device__ inline void x_prepare_body(const XPrepArgs& a, long bid, long nb, int nthreads) {
  constexpr int KPC = Op<T>::kPerChunk;
  const int KS = a.H / (4 * KPC);
  const long n = 8L * a.MRT * KS * 64 * KPC;
  T* slot1 = reinterpret_cast<T*>(reinterpret_cast<char*>(a.ring) + ((long)a.slot * 8 * a.MRT * a.ring_ks << 10));
  for (long f = bid * nthreads + threadIdx.x; f < n; f += nb * nthreads) {
    const int e = (int)(f % KPC);
    const int l = (int)((f / KPC) % 64);
    const int ks = (int)((f / (64 * KPC)) % KS);
    const int tile = (int)(f / (64L * KPC * KS));
    const int x = tile / a.MRT, mt = tile - x * a.MRT;
    const int r = (x + 8 * mt) * 16 + (l & 15);
    const int u = ks * 4 * KPC + (l >> 4) * KPC + e;
    const float v = (a.h0 && r < a.B) ? a.h0[(long)a.perm[r] * a.H + u] : 0.f;
    // block ks of tile `tile` in the slot (tiles are ring_ks blocks apart)
    slot1[(((long)tile * a.ring_ks + ks) * 64 + l) * KPC + e] = Op<T>::from_f32(v);
  }
  for (long i = bid * nthreads + threadIdx.x; i < a.nflags; i += nb * nthreads) a.flags[i] = 0u;
}

// Row map of the h_{t-1} operand of dW over rows: prev[off[t] + r] = the
// history row of the same sequence one step earlier (rows cap + r hold h0).
__device__ inline void prev_rows_body(const int* __restrict__ active, const int* __restrict__ off, int B,
                                      int T_max, long cap, int* __restrict__ prev, long bid, long nb,
                                      int nthreads) {
  const long n = (long)T_max * B;
  for (long i = bid * nthreads + threadIdx.x; i < n; i += nb * nthreads) {
    const int t = (int)(i / B), r = (int)(i % B);
    if (r < active[t]) prev[off[t] + r] = t > 0 ? off[t - 1] + r : (int)(cap + r);
  }
}
// h0 rows in length order, operand type.
template <typename T>
__device__ inline void h0_rows_body(const float* __restrict__ h0, const int* __restrict__ perm, int B, int H,
                                    T* __restrict__ dst, long bid, long nb, int nthreads) {
  const long n = (long)B * H;
  for (long i = bid * nthreads + threadIdx.x; i < n; i += nb * nthreads) {
    const int r = (int)(i / H), j = (int)(i % H);
    dst[i] = Op<T>::from_f32(h0 ? h0[(long)perm[r] * H + j] : 0.f);
  }
}
// out[r * ldo + c] = sum_{s < S} ws[s * stride + r * cols + c], fixed order.
__device__ inline void sum_slices_body(const float* __restrict__ ws, int S, long stride, long n, long cols,
                                       long ldo, float* __restrict__ out, long bid, long nb, int nthreads) {
  for (long i = bid * nthreads + threadIdx.x; i < n; i += nb * nthreads) {
    float acc = 0.0f;
    for (int s = 0; s < S; ++s) acc += ws[s * stride + i];
    const long r = i / cols;
    out[r * ldo + (i - r * cols)] = acc;
  }
}

// W_h (rows row0 .. row0 + H - 1 of W [rows, 4H]) in unit-major column
// order: dst[j][4u + g] = W[row0 + j][g H + u].
template <typename T>
__device__ inline void permute_um_body(const T* __restrict__ W, int row0, int H, T* __restrict__ dst, long bid,
                                       long nb, int nthreads) {
  const long n = (long)H * H;
  for (long i = bid * nthreads + threadIdx.x; i < n; i += nb * nthreads) {
    const long j = i / H;
    const int u = (int)(i - j * H);
    const T* src = W + (row0 + j) * 4L * H + u;
    struct alignas(4 * sizeof(T)) Quad { T v[4]; } q;
#pragma unroll
    for (int g = 0; g < 4; ++g) q.v[g] = src[(long)g * H];
    *reinterpret_cast<Quad*>(dst + 4 * i) = q;
  }
}

// Small jobs a product's launch can carry in work-groups of its own
// (pre_blocks of them, ahead of the product's): each is skipped when its
// output is NULL.
struct PreJobs {
  XPrepArgs xp;                          // the forward loop's entering state (xp.ring)
  const int* active;                     // the h_{t-1} row map of dW over rows (prev)
  const int* off;
  int B, T_max;
  long cap;
  int* prev;
  const float* h0;                       // h0 rows in length order (h0dst, operand type)
  const int* perm;
  int H;
  void* h0dst;
  const float* ws;                       // a sum of S slices (sum_out)
  int S;
  long stride, n, cols, ldo;
  float* sum_out;
  const void* pw;                        // W_h in unit-major order (pdst, operand type)
  int prow0, pH;
  void* pdst;
  unsigned* zero;                        // nzero words to zero
  int nzero;
};
template <typename T>
__device__ inline void pre_jobs_body(const PreJobs& j, long bid, long nb, int nthreads) {
  if (j.xp.ring) x_prepare_body<T>(j.xp, bid, nb, nthreads);
  if (j.prev) prev_rows_body(j.active, j.off, j.B, j.T_max, j.cap, j.prev, bid, nb, nthreads);
  if (j.h0dst) h0_rows_body<T>(j.h0, j.perm, j.B, j.H, static_cast<T*>(j.h0dst), bid, nb, nthreads);
  if (j.sum_out) sum_slices_body(j.ws, j.S, j.stride, j.n, j.cols, j.ldo, j.sum_out, bid, nb, nthreads);
  if (j.pdst)
    permute_um_body<T>(static_cast<const T*>(j.pw), j.prow0, j.pH, static_cast<T*>(j.pdst), bid, nb, nthreads);
  for (long i = bid * nthreads + threadIdx.x; i < j.nzero; i += nb * nthreads) j.zero[i] = 0u;
}

struct GemmArgs {
  const void* A;
  long lda;
  const int* a_rowmap;   // NULL: arow(m) = m
  const void* Bm;
  long ldb;
  float* C;
  long ldc;
  const int* c_rowmap;   // NULL: crow(m) = m
  const float* bias;     // NULL: none
  int M;                 // rows (capacity when M_dev is set)
  const int* M_dev;      // NULL or device scalar: rows actually present
  int N;
  int K;
  const int* K_dev;      // NULL or device scalar: reduction length
  int splits;            // > 1: split-K; slice z written to C + z * split_stride
  long split_stride;
  int a_rows;            // rows of A the row map addresses (0: M)
  int k_zero_tail;       // 1: both operands hold zeros from K up to the next multiple of 8
  // > 0: LSTM gate epilogue with H = act_h: C = act(Z + A B^T), Z = C
  // (addend NULL) or addend[add_rowmap[m] * ld_add + n], act the logistic
  // function on columns [0, 2H) and [3H, 4H), tanh on [2H, 3H) (needs
  // splits == 1 and no bias)
  int act_h;
  const float* addend;
  const int* add_rowmap;
  long ld_add;
  // pre_blocks > 0: the launch also runs the jobs of `pre` (the forward
  // loop's entering state and flags, dW's row maps, a slice sum), in
  // pre_blocks work-groups of its own
  int pre_blocks;
  PreJobs pre;
};
template <typename T>
hipError_t launch_pre_jobs(const PreJobs& j, hipStream_t s);

struct LoopGeom {
  int HJ;       // hidden units per work-group (multiple of 4)
  int RG;       // work-groups per unit block (row groups)
  int NRT;      // 16-row tiles covering the batch
  int MRT;      // row tiles per work-group = ceil(NRT / RG)
  int nwg;      // (H / HJ) * RG
  size_t lds_fwd;
  size_t lds_bwd;
};

struct FwdLoopArgs {
  int B, H, T_max;
  int HJ, RG, MRT;
  const int* meta;
  const int* active;
  const int* off;
  const int* perm;
  const float* Zx;        // [cap, 4H] float: x_t W_x + b for every compact row
  const void* WT;         // [4H, ldw] operand type: row n = gate column n of W
  int ldw;
  int woff;               // column of WT where the h rows of W start (= I_l)
  const float* h0;        // [B, H] original order, or NULL
  const float* c0;
  void* HH;               // [cap, H] operand type: h_t history (compact rows)
  float* stack;           // [cap, 5H] float: i, f, g, o, c_t (NULL = inference)
  float* y;               // [T_max, B, H] or NULL
  float* hT;
  float* cT;
  unsigned* bar;
  int* abort_flag;
  int* err;
  unsigned long long limit;
};

struct BwdLoopArgs {
  int B, H, T_max;
  int HJ, RG, MRT;
  const int* meta;
  const int* active;
  const int* off;
  const int* perm;
  const void* W;          // [rows, 4H] operand type, natural layout
  int wrow0;              // first row of the h part of W (= I_l)
  const float* stack;     // [cap, 5H]
  const float* c0;        // [B, H] original order, or NULL
  const float* dy;        // NULL, [T_max, B, H] (dy_compact = 0) or [cap, H] (= 1)
  int dy_compact;
  const float* dhT;
  const float* dcT;
  void* DZ;               // [cap, 4H] operand type (output)
  float* db_part;         // [RG, 4H]
  float* dh0;
  float* dc0;
  unsigned* bar;
  int* abort_flag;
  int* err;
  unsigned long long limit;
};

// XCD-local loops (ll_xloop.hip).  One argument block serves both directions.
struct XLoopArgs {
  int B, H, T_max;
  int P;                  // members per XCD that own a unit block (H / HJ)
  int MRT;                // row tiles per XCD = ceil(ceil(B/16) / 8)
  const int* meta;
  const int* active;
  const int* off;
  const int* perm;
  // (G gate blocks: LSTM 4, GRU 3, RNN 1; GB = 4 for the GRU, else G)
  const void* W;          // forward: W^T [G H, ldw]; backward: W [rows, G H]
  int ldw;
  int woff;               // forward: column of the h part in W^T; backward: row of W_h
  void* X;                // forward: h history [cap, H]; backward: dz [cap, GB H] (operand type)
  void* ring;             // exchange ring [2][8][MRT][ring_ks][1 KB] (forward: slot 1 holds h0)
  int ring_ks;            // k-step blocks per row tile: H / (4 KPC) forward, 4H / (4 KPC) backward
  unsigned* flags;        // [8][MRT][32] per-member step flags, zero before the launch
  const float* Zx;        // forward: [cap, 4H]
  const float* h0;
  const float* c0;
  float* stack;           // forward: push (NULL = inference); backward: pop
  float* y;
  float* hT;
  float* cT;
  const float* dy;
  int dy_compact;
  const float* dhT;
  const float* dcT;
  float* db_part;         // backward: [8, GB H]
  const float* bhn;       // GRU, forward: the candidate block's recurrent bias [H]
  // LSTM with a cond body: predicate s = (x_t . w_px + h_{t-1} . w_ph) + b_p
  const float* wp;        // forward: w_ph [H] (float, rounded to the operand type)
  const float* bp;        // forward: b_p (device scalar)
  const float* sx;        // forward: x_t . w_px per compact row [cap]
  float* guard;           // guard per compact row [cap] (1 = the LSTM step ran):
                          // pushed by the forward, popped by the gradient
  float* dh0;
  float* dc0;
  unsigned* rank_ctr;     // [8], zero before the launch
  int* abort_flag;
  int* err;
  unsigned long long limit;
  // steps of this launch: [t_begin, min(t_end, T_eff)) (the gradient loop runs
  // them in descending order); the loop state enters through h0/c0 (dhT/dcT)
  // and leaves through hT/cT (dh0/dc0)
  int t_begin, t_end;
  // stack ring: row of (step t, compact index r) is
  //   (((t / chunk_steps) % nslots) * chunk_steps + t % chunk_steps) * B + r
  int chunk_steps, nslots;
  float* db_state;        // backward: per-thread db sums carried between launches (NULL: none)
  int db_resume;          // backward: 1 = start from db_state
  // two-layer wavefront (one launch runs both layers, the upper one a step
  // behind in the forward direction, ahead in the gradient direction):
  const void* in_ring;    // upper layer, forward: the lower layer's ring (its h_t is y1_t)
  const unsigned* in_flags;
  int in_ks;              // k-steps of the recurrent product taken from in_ring
  const float* zbias;     // upper layer, forward: bias (there is no hoisted input projection)
  const unsigned* out_flags;  // lower layer, forward: the upper layer's flags (ring reuse)
  void* dyx_ring;         // gradient: dy of the lower layer's output, [2][8][MRT][16][H] float
  unsigned* dyx_flags;    // gradient: per-member flags of dyx_ring ([8][MRT][32])
  const unsigned* peer_flags;  // gradient: the other layer's step flags
  const void* Wx;         // upper layer, gradient: W rows of the input part [I_l, 4H]
  // saved values: the c field of row (t, r) at stack + stack_row(t, r) * sld
  // + scoff; i, f, g, o at gstk + grow(t, r) * gld + {0, H, 2H, 3H}, where
  // grow maps like stack_row with gchunk / gslots (gstk NULL: the gates sit
  // in the stack rows, those of unit u at 4u .. 4u+3)
  int sld, scoff;
  int sgates;             // forward: 1 = push i, f, g, o with c (0: c only); the
                          // GRU pushes r, u, n, zh_n + b_hn and h_{t-1} in their places
  const float* gstk;
  int gld, gchunk, gslots;
  // LSTM with a nested loop (ACT): at most ponder_max ponder steps per step;
  // ponder step k of compact row cr sits at row k * slot_rows + cr of the
  // stack, the guards, HI (forward: h^{k+1}, operand type) and dz (backward)
  int ponder_max;
  long slot_rows;
  int* ntrip;             // [T_max][8 * MRT] inner trip count per (step, row tile)
  void* HI;
  // gradient: dx [T_max, B, I] floats to zero at every row's finished steps
  // (t >= seq_len[b]; all steps if the lengths failed the range check), or
  // NULL; XCDs 1 .. 7 zero them after their last step
  float* dx_zero;
  const int* seq_len;
  int I;
};

// Chip-wide loops (ll_cloop.hip), for shapes whose recurrent weights need
// more than one XCD: XCD x owns hidden units [x H/8, (x+1) H/8); its 32
// work-groups split the reduction (K) and the units (N) of the recurrent
// product.  Every row tile of the batch runs on every work-group.
struct CLoopArgs {
  int B, H, T_max;
  int MRT;                // row tiles of the batch = ceil(B / 16)
  const int* meta;
  const int* active;
  const int* off;
  const int* perm;
  const void* W;          // forward: W^T [4H, ldw]; backward: W [rows, 4H]
  int ldw;
  int woff;               // forward: column of the h part in W^T; backward: row of W_h
  void* X;                // forward: h history [cap, H]; backward: dz [cap, 4H] (operand type)
  void* ring;             // exchange ring [2][MRT][ring_ks][1 KB] (forward: slot 1 holds h0)
  int ring_ks;            // blocks per row tile: H / (4 KPC) forward, 4H / (4 KPC) backward
  float* part;            // partial products [2][8][MRT][32][pw]
  unsigned* xflags;       // exchange flags [MRT][256] (one per work-group and row tile)
  unsigned* pflags;       // partial-product flags [8][MRT][32]
  unsigned* rank_ctr;     // [8]
  const float* Zx;        // forward: [cap, 4H]
  const float* h0;
  const float* c0;
  float* stack;           // [cap, 5H] compact rows: forward push (NULL = inference), backward pop
  float* y;
  float* hT;
  float* cT;
  const float* dy;
  int dy_compact;
  const float* dhT;
  const float* dcT;
  float* db;              // backward: [4H]
  float* dh0;
  float* dc0;
  int* abort_flag;
  int* err;
  unsigned long long limit;
};

struct CKernels {
  const void* fwd;
  const void* bwd;
  size_t lds_fwd;
  size_t lds_bwd;
  int pw;                 // partial floats per (work-group, row tile)
};
template <typename T>
CKernels c_kernels(int H, int mrt);
hipError_t c_setup(const CKernels& k, int* occ_fwd, int* occ_bwd);
hipError_t c_launch(const void* fn, const CLoopArgs& a, size_t lds, hipStream_t s);
// h0 rows (length order, operand type) into ring slot 1 and every flag and
// rank counter of the launch to zero.
template <typename T>
hipError_t launch_c_prepare(const float* h0, const int* perm, int B, int H, int mrt, void* ring,
                            unsigned* flags, int nflags, hipStream_t s);

struct XKernels {
  const void* fwd;
  const void* bwd;
  size_t lds_fwd;
  size_t lds_bwd;
};

// gates: 4 (LSTM), 3 (GRU) or 1 (Elman RNN); skip: the LSTM body with a
// cond; act: the LSTM body with a nested loop (ACT's halting rule)
template <typename T>
XKernels x_kernels(int hc, int mrt, int gates = 4, bool skip = false, bool act = false);
hipError_t x_setup(const XKernels& k, int* occ_fwd, int* occ_bwd);
hipError_t x_launch(const void* fn, const XLoopArgs& a, int nwg, size_t lds, hipStream_t s);
// Two-layer wavefront: one launch runs both layers (a0 lower, a1 upper);
// needs 2 H / HJ <= 32 members per XCD.
template <typename T>
XKernels x_kernels2(int hc, int mrt);
hipError_t x_launch2(const void* fn, const XLoopArgs& a0, const XLoopArgs& a1, int nwg, size_t lds,
                     hipStream_t s);
// h0 rows into ring slot 1 (consumer lane order) and the launch's flags to zero.
template <typename T>
hipError_t launch_x_prepare_fwd(const float* h0, const int* perm, int B, int H, int mrt, int ring_ks,
                                int slot, void* ring, unsigned* flags, int nflags, hipStream_t s);
// dst[0 .. n) = src[0 .. n) (one wave; n small)
hipError_t launch_copy_i32(const int* src, int* dst, int n, hipStream_t s);
// out[rowmap[r]] = sum of nsl slices (stride floats apart) of compact row r, r < meta[1]
hipError_t launch_sum_scatter_rows(const float* ws, int nsl, long stride, const int* meta, const int* rowmap,
                                   int C, float* out, long cap_rows, hipStream_t s);
hipError_t launch_zero_u32(unsigned* p, int n, hipStream_t s);

// Sustained matrix-core rate of the device (TFLOP/s), for reports: the 16x16
// k-step the loops use, or the 32x32 shape.
template <typename T>
hipError_t measure_mfma_peak(int n_cu, bool shape32, double* tflops);
// sigmoid (fn 0) or tanh (fn 1) of n floats, as the loop kernels compute them
hipError_t eval_activations(const float* in, float* out, long n, int fn, hipStream_t s);

// The forward's set-up in one launch: prep (length order, active rows and
// compact offsets per step, row map, T_eff into meta[0] and *trip_out, the
// range check, the cleared barrier counters) on one work-group, beside the
// transposes W[l] [R[l], C] -> WT[l] [C, R[l]] of nw <= 2 layers.
struct PrepArgs {
  const int* seq_len;
  int B, T_max;
  int* perm;
  int* active;
  int* off;
  int* rowmap;
  int* meta;
  int* trip_out;
  int t_in_lds, n_pow2;
};
struct TransposeJob {
  const void* in;
  void* out;
  int R, C, ldi, ldo, tiles_c, tiles;
};
struct FwdSetupArgs {
  PrepArgs prep;
  int njobs;
  TransposeJob job[2];
};
template <typename T>
hipError_t launch_fwd_setup(const int* seq_len, int B, int T_max, int* perm, int* active, int* off,
                            int* rowmap, int* meta, int* trip_out, int nw, const T* const* W, const int* R,
                            int C, T* const* WT, hipStream_t s);

// Several independent small kernels in one launch (kernel launches cost a few
// microseconds each on this GPU, small ones mostly that): each task runs on
// its own range of work-groups.
enum SmallTaskKind : int {
  kTaskZeroU32,            // out[0 .. l0) = 0 (unsigned)
  kTaskZeroFinishedRows,   // zero rows t >= seq_len[b] of out [i0 = T_max, i1 = B, i2 = C] (a = seq_len, b = meta)
  kTaskPermuteUm,          // W_h (a, rows i0 ..) in unit-major order into out (i1 = H)
  kTaskSumSlices,          // out = sum of i0 slices of a (l0 = stride, l1 = n, l2 = cols, l3 = ldo)
  kTaskPrevRows,           // out[k] = history row of h_{t-1} of compact row k (a = active, b = off, i0 = B, i1 = T_max, l0 = cap)
  kTaskH0Rows,             // out = h0 rows (a, float) in length order (b = perm, i0 = B, i1 = H), operand type
};
struct SmallTask {
  int kind, blocks;
  const void* a;
  const void* b;
  void* out;
  long l0, l1, l2, l3;
  int i0, i1, i2;
};
constexpr int kMaxSmallTasks = 6;
struct SmallTasks {
  int n;
  SmallTask t[kMaxSmallTasks];
};
template <typename T>
hipError_t launch_small_tasks(const SmallTasks& ts, hipStream_t s);

template <typename T>
struct SmallBatch {
  SmallTasks ts{};
  static int blocks_for(long n, long per, long cap) {
    const long b = (n + per - 1) / per;
    return (int)(b < 1 ? 1 : b > cap ? cap : b);
  }
  hipError_t add(SmallTask t) {
    if (ts.n >= kMaxSmallTasks) return hipErrorInvalidValue;
    ts.t[ts.n++] = t;
    return hipSuccess;
  }
  hipError_t zero_u32(unsigned* p, long n) {
    SmallTask t{};
    t.kind = kTaskZeroU32;
    t.out = p;
    t.l0 = n;
    t.blocks = blocks_for(n, 256, 1024);
    return add(t);
  }
  hipError_t zero_finished_rows(float* dst, int T_max, int B, int C, const int* seq_len, const int* meta) {
    SmallTask t{};
    t.kind = kTaskZeroFinishedRows;
    t.out = dst;
    t.a = seq_len;
    t.b = meta;
    t.i0 = T_max;
    t.i1 = B;
    t.i2 = C;
    t.blocks = blocks_for((long)T_max * B, 4, 4096);
    return add(t);
  }
  hipError_t permute_um(const T* W, int row0, int H, T* dst) {
    SmallTask t{};
    t.kind = kTaskPermuteUm;
    t.a = W;
    t.out = dst;
    t.i0 = row0;
    t.i1 = H;
    t.blocks = blocks_for((long)H * H, 256, 4096);
    return add(t);
  }
  hipError_t sum_slices(const float* ws, int S, long stride, long rows, long cols, float* out, long ldo) {
    if (cols < 1 || ldo < cols) return hipErrorInvalidValue;
    SmallTask t{};
    t.kind = kTaskSumSlices;
    t.a = ws;
    t.out = out;
    t.i0 = S;
    t.l0 = stride;
    t.l1 = rows * cols;
    t.l2 = cols;
    t.l3 = ldo;
    t.blocks = blocks_for(rows * cols, 256, 4096);
    return add(t);
  }
  hipError_t prev_rows(const int* active, const int* off, int B, int T_max, long cap, int* prev) {
    SmallTask t{};
    t.kind = kTaskPrevRows;
    t.a = active;
    t.b = off;
    t.out = prev;
    t.i0 = B;
    t.i1 = T_max;
    t.l0 = cap;
    t.blocks = blocks_for((long)T_max * B, 256, 4096);
    return add(t);
  }
  hipError_t h0_rows(const float* h0, const int* perm, int B, int H, T* dst) {
    SmallTask t{};
    t.kind = kTaskH0Rows;
    t.a = h0;
    t.b = perm;
    t.out = dst;
    t.i0 = B;
    t.i1 = H;
    t.blocks = blocks_for((long)B * H, 256, 4096);
    return add(t);
  }
  // one launch of every task added since the last one (none: nothing)
  hipError_t launch(hipStream_t s) {
    const hipError_t e = launch_small_tasks<T>(ts, s);
    ts.n = 0;
    return e;
  }
};
template <typename T>
hipError_t launch_transpose(const T* in, int R, int C, int ldi, T* out, int ldo, hipStream_t s);
template <typename T>
hipError_t launch_gather_transpose(const GatherTArgs& g, int cap_rows, hipStream_t s);
hipError_t launch_zero_finished_rows(float* dst, int T_max, int B, int C, const int* seq_len,
                                     const int* meta, hipStream_t s);
// Row maps of the gate recomputation over padded rows (t, r), r < B:
//   xmap[t B + r] = t B + perm[r] (time-major input row),
//   cmap[t B + r] = off[t] + r (compact row), prevmap[t B + r] = off[t-1] + r
//   for t > 0 and cap + r for t = 0 (where the h0 rows follow the history);
// rows not running at t map to row 0 (x, compact) and cap (h_{t-1}).
hipError_t launch_rc_maps(const int* active, const int* off, const int* perm, int B, int T_max,
                          long cap, int* xmap, int* cmap, int* prevmap, hipStream_t s);
// dst[r * H + j] = h0[perm[r] * H + j] in the operand type (0 if h0 is NULL).
template <typename T>
hipError_t launch_h0_rows(const float* h0, const int* perm, int B, int H, T* dst, hipStream_t s);
hipError_t launch_sum_slices(const float* ws, int S, long stride, long n, float* out,
                             hipStream_t s);
// out[r * ldo + c] = sum over s < S of ws[s * stride + r * cols + c], for
// r < rows, c < cols.
hipError_t launch_sum_slices_2d(const float* ws, int S, long stride, long rows, long cols, float* out,
                                long ldo, hipStream_t s);
template <typename T>
hipError_t launch_convert(const float* in, long n, T* out, hipStream_t s);
// prev[off[t] + r] = off[t-1] + r (t > 0) or cap + r (t = 0) for r <
// active[t]: the h history row of each compact row's h_{t-1} (rows cap ..
// cap + B - 1 hold h0 in length order).
hipError_t launch_prev_rows(const int* active, const int* off, int B, int T_max, long cap, int* prev,
                            hipStream_t s);
// dst[j][4 u + g] = W[row0 + j][g H + u] (j, u < H, g < 4): the recurrent
// weights in the unit-major reduction order of the single-layer LSTM
// gradient loop.
template <typename T>
hipError_t launch_permute_um(const T* W, int row0, int H, T* dst, hipStream_t s);
// out[r] = sum_k A[rowmap ? rowmap[r] : r][k] * op(w[k]) for r < meta[1]
// (at most cap rows); the input part of the cond body's predicate.
template <typename T>
hipError_t launch_row_dot(const T* A, int lda, const int* rowmap, const int* meta, long cap, const float* w,
                          int K, float* out, hipStream_t s);

template <typename T>
hipError_t launch_gemm_nt(const GemmArgs& g, hipStream_t s);

// C[m][n] = sum over k < K of A[arow(k)][m] B[k][n] (bf16 operands, fp32
// result): the product over the rows of two row-major operands, as dW =
// [X; Hprev]^T DZ needs, with no transposed copies.  arow(k) = a_rowmap[k]
// (NULL: k).  Needs M and N multiples of 8 and 16-byte aligned rows.
struct GemmTnArgs {
  const void* A;
  long lda;
  const int* a_rowmap;
  int a_rows;            // rows of A the row map addresses
  const void* Bm;
  long ldb;
  int b_rows;            // rows of B (>= K)
  float* C;
  long ldc;
  int M, N, K;
  const int* K_dev;      // NULL or device scalar: rows actually present (<= K)
  int splits;            // > 1: split-K; slice z written to C + z * split_stride
  long split_stride;
  // optional second operand for the C rows from M1 on (M1 a multiple of the
  // 256-row tile): C[m][n] for m >= M1 reads A2[a2row(k)][m - M1]
  const void* A2;
  long lda2;
  const int* a2_rowmap;
  int a2_rows;
  int M1;
  // two splits summed in place (splits == 2, tile_flags non-NULL): per output
  // tile two words (zero between launches; each launch leaves them zero); the
  // split that finishes first writes its slice of C (device-scope stores),
  // the second adds it to its own sums and writes out[m * ldo + n]
  unsigned* tile_flags;
  float* out;
  long ldo;
};
bool gemm_tn_applies(const GemmTnArgs& g);
hipError_t launch_gemm_tn(const GemmTnArgs& g, hipStream_t s);
// Whether launch_gemm_nt takes the large-tile bf16 kernel for g, and how
// many times the launch fills n_cu compute units (row capacity g.M).
bool gemm_big_applies(const GemmArgs& g, int elem_bytes);
long gemm_rounds(const GemmArgs& g, int elem_bytes, int n_cu);
constexpr int kGemmBigTile = 256;

// Recurrent loops (cooperative launches).
template <typename T>
hipError_t loop_kernel_setup(int mrt, size_t lds_fwd, size_t lds_bwd, int* max_wg_per_cu_fwd,
                             int* max_wg_per_cu_bwd);
template <typename T>
hipError_t launch_fwd_loop(const FwdLoopArgs& a, int nwg, size_t lds, hipStream_t s);
template <typename T>
hipError_t launch_bwd_loop(const BwdLoopArgs& a, int nwg, size_t lds, hipStream_t s);

// LDS bytes the loops need for a geometry (see ll_loop.hip).
size_t fwd_loop_lds(int H, int HJ, int elem_bytes);
size_t bwd_loop_lds(int H, int HJ, int elem_bytes);

}  // namespace ll
