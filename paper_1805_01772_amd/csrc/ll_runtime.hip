// Host runtime of lstmloop: plan (stack and scratch allocation, launch
// geometry), argument validation, the enqueue order of the forward and
// gradient loops, and the C ABI declared in include/lstmloop.h.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "lstmloop.h"
#include "ll_kernels.h"

using ll::bf16_t;

namespace {

thread_local std::string g_last_error;

ll_status fail(ll_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return s;
}

#define LL_HIP(call)                                                              \
  do {                                                                            \
    hipError_t e_ = (call);                                                       \
    if (e_ != hipSuccess)                                                         \
      return fail(LL_EHIP, "%s failed: %s", #call, hipGetErrorString(e_));        \
  } while (0)

#define LL_STATUS(call)         \
  do {                          \
    ll_status st_ = (call);     \
    if (st_ != LL_OK) return st_; \
  } while (0)

enum PlanState { ST_EMPTY = 0, ST_FWD_DONE = 1 };

class DeviceGuard {
 public:
  explicit DeviceGuard(int dev) {
    if (hipGetDevice(&prev_) != hipSuccess) prev_ = -1;
    if (prev_ != dev) hipSetDevice(dev);
  }
  ~DeviceGuard() {
    int cur = -1;
    if (prev_ >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev_) hipSetDevice(prev_);
  }

 private:
  int prev_ = -1;
};

long round_up(long v, long m) { return (v + m - 1) / m * m; }

// Events that only order work on this device (streams of one device, the
// host waiting for completion): no system-scope fences (measured: each such
// fence left the GPU idle for several microseconds).
constexpr unsigned kOrderEventFlags = hipEventDisableTiming | hipEventDisableSystemFence;

// Loop launches of every plan on one device form one chain: each starts
// after the previous one (whatever plan or stream enqueued it) has
// completed.  The loops need all compute units co-resident, so two of them
// must never run at once.  While every loop launch on the device has come
// from one stream, stream order alone keeps them apart and nothing is
// recorded (each event record cost the GPU several microseconds of idle
// time); the first launch from another stream waits for the device to
// finish its work (a host-side synchronisation, once per device), and from
// then on every launch records an event that the next one, on another
// stream, waits for.  (Skipped on a stream that is being captured into a
// graph: an event recorded outside the capture cannot be waited on there.)
struct LoopChain {
  std::mutex mu;
  hipEvent_t last = nullptr;
  bool recorded = false;
  bool any = false;                    // a loop launch has happened
  bool multi = false;                  // loop launches have come from more than one stream
  hipStream_t last_stream = nullptr;   // the stream of the last loop launch
};
LoopChain g_loop_chain[64];

template <typename Launch>
hipError_t chained_loop_launch(int device, hipStream_t s, Launch&& launch) {
  hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(s, &cap) != hipSuccess) cap = hipStreamCaptureStatusNone;
  if (cap != hipStreamCaptureStatusNone || device < 0 || device >= 64) return launch();
  LoopChain& c = g_loop_chain[device];
  std::lock_guard<std::mutex> lock(c.mu);
  if (!c.multi) {
    if (!c.any || c.last_stream == s) {
      const hipError_t e = launch();
      if (e == hipSuccess) {
        c.any = true;
        c.last_stream = s;
      }
      return e;
    }
    // a second stream: the loops enqueued so far (on the first one) end first
    hipError_t e = hipDeviceSynchronize();
    if (e != hipSuccess) return e;
    c.multi = true;
  }
  if (!c.last) {
    hipError_t e = hipEventCreateWithFlags(&c.last, kOrderEventFlags);
    if (e != hipSuccess) {
      c.last = nullptr;
      return e;
    }
  }
  if (c.recorded && c.last_stream != s) {   // (on the same stream, stream order suffices)
    hipError_t e = hipStreamWaitEvent(s, c.last, 0);
    if (e != hipSuccess) return e;
  }
  hipError_t e = launch();
  if (e != hipSuccess) return e;
  e = hipEventRecord(c.last, s);
  if (e == hipSuccess) c.recorded = true;
  c.last_stream = s;
  return e;
}

}  // namespace

struct ll_plan {
  ll_desc d{};
  int device = 0;
  int es = 4;            // operand element bytes
  bool bf16 = false;
  int G = 4;             // gate blocks of the cell: 4 (LSTM), 3 (GRU), 1 (Elman RNN)
  int GB = 4;            // dz row and bias blocks: the GRU's 4 (r, u, n, and the
                         // candidate's recurrent side), else G
  long cap = 0;          // compact-row capacity = T_max * B
  long ldT = 0;          // leading dimension of transposed per-row arrays
  ll::LoopGeom geom{};
  int n_cu = 0;
  unsigned long long barrier_ticks = 0;
  int dw_splits[2][3] = {{1, 1, 1}, {1, 1, 1}};   // split-K of each dW product (layer, part)
  bool xmode = false;          // XCD-local loops (ll_xloop.hip)
  ll::XKernels xk{};
  int xP = 0;                  // unit blocks per XCD
  int xMRT = 0;                // row tiles per XCD
  int xhc = 0;                 // forward k-steps per wave
  // chip-wide loops (ll_cloop.hip): weights split over all XCDs
  bool cmode = false;
  ll::CKernels ck{};
  int cMRT = 0;
  void* cring = nullptr;
  float* cpart = nullptr;
  unsigned* cflags = nullptr;  // [8] rank counters, exchange flags [MRT][256], partial flags [8][MRT][32]
  int cflag_words = 0;
  // two-layer wavefront: one launch per direction runs both layers
  bool wave = false;
  ll::XKernels xk2{};
  // device memory
  int* perm = nullptr;
  int* active = nullptr;
  int* off = nullptr;
  int* rowmap = nullptr;
  int* meta = nullptr;
  void* WT[2] = {nullptr, nullptr};
  float* Zx = nullptr;
  float* stack[2] = {nullptr, nullptr};
  void* HH[2] = {nullptr, nullptr};
  void* DZ = nullptr;
  void* DZT = nullptr;
  void* XT = nullptr;           // [I_l + H, ldT]: x (or y of the layer below) transposed, then h_prev
                                //   transposed (rows I_l ..), the A operand of one dW product
  float* dyc = nullptr;
  void* xring = nullptr;       // XCD-local loops: exchange ring
  // XCD-local loops: [8] rank counters, then step flags [8][MRT][32] (the
  // wavefront: lower layer, upper layer, dy exchange)
  unsigned* xflags = nullptr;
  int xflag_words = 0;
  // single-layer plans whose gradient loop is one launch: its flags, of
  // their own, cleared by the forward's input-projection launch
  unsigned* xflags_b = nullptr;
  void* xring2 = nullptr;      // wavefront: the upper layer's exchange ring
  void* DZ2 = nullptr;         // wavefront: dz of the upper layer
  float* dyx = nullptr;        // wavefront: dy exchange [2][8][MRT][16][H]
  float* db_part2 = nullptr;   // wavefront: db partials of the upper layer
  // stack spill (XCD-local loops only): device ring of nslots chunks of
  // chunk_steps steps per layer, pinned host copy of every chunk
  bool spill = false;
  int chunk_steps = 0, nslots = 1, nchunks = 1;
  long slot_floats = 0;
  float* host_stack[2] = {nullptr, nullptr};
  hipStream_t cstream = nullptr;
  hipStream_t cstream2 = nullptr;   // chunks alternate between the two copy streams
  // recomputation instead of saved gates (XCD-local loops only): the forward
  // pushes only c_t ([T_max*B, H] per layer); the gradient pass recomputes
  // i, f, g, o of each chunk of rc_steps steps into gslot just before the
  // chunk's launch, from x_t (or y_t of the layer below), the h history and W
  bool recompute = false;
  int rc_steps = 0, rc_chunks = 1;
  float* gslot = nullptr;       // [rc_steps * B, 4H]
  int* rc_inmap = nullptr;      // [2][T_max * B]: input row of (t, r): x (time-major), compact
  int* rc_prevmap = nullptr;    // [T_max * B]: h history row of h_{t-1} (rows cap.. hold h0)
  float* rc_bias = nullptr;     // [layers, 4H]: the forward's bias, kept for the recomputation
  // side stream for the dx product, which runs beside the dW products after
  // the gradient loop (forked from and joined back into the call's stream)
  hipStream_t gstream = nullptr;
  hipEvent_t ev_fork = nullptr, ev_join = nullptr;
  hipEvent_t ev_compute = nullptr;
  hipEvent_t ev_done = nullptr;   // recorded on the call's stream at the end of every call
  bool done_recorded = false;
  // the saved forward's input-projection launches also wrote dW's h_{t-1}
  // row map and h0 rows (the gradient pass then skips those tasks)
  bool rows_prepared = false;
  // ... and W_h in unit-major order and, with xflags_b, the gradient loop's flags
  bool bwd_prepared = false;
  std::vector<hipEvent_t> ev_d2h, ev_h2d;   // per (layer, slot)
  float* carry = nullptr;      // [4][B, H]: h, c (forward) / dh, dc (backward) between chunks
  float* db_state = nullptr;   // per-thread db sums between backward chunks
  float* db_part = nullptr;
  float* ws = nullptr;
  long ws_floats = 0;
  // LSTM body with a cond: the predicate's input part per compact row, and
  // the guard stack of each layer ([layers][cap], 1 = the LSTM step ran)
  bool skip = false;
  float* sx = nullptr;
  float* guards = nullptr;
  // LSTM body with a nested loop: at most M ponder steps; per ponder slot k
  // the stack, guards, dz rows and (forward) h^{k+1} in HI; inner trip counts
  bool act = false;
  int M = 1;
  void* HI = nullptr;
  int* ntrip = nullptr;
  // XCD-local LSTM gradient loops: W_h of each layer in the unit-major
  // reduction order ([H, 4H], operand type)
  void* Wum[2] = {nullptr, nullptr};
  // bf16 dW from the row-major operands: h history row of each compact row's
  // h_{t-1} (h0 rows after the history), and the split-K of each product
  int* prevc = nullptr;
  int tn_splits[2][3] = {{1, 1, 1}, {1, 1, 1}};
  // products over rows split in two sum in place: two words per output tile
  unsigned* tn_flags = nullptr;
  long tn_flag_words = 0;
  bool dw_rows[2] = {false, false};   // layer's dW from the row-major operands
  int64_t stack_device_bytes = 0;
  int64_t stack_host_bytes = 0;
  // saved forward
  int state = ST_EMPTY;
  const void* x = nullptr;
  const int32_t* seq_len = nullptr;
  const void* W[2] = {nullptr, nullptr};
  const float* h0 = nullptr;
  const float* c0 = nullptr;
  hipStream_t last_stream = nullptr;
  // stage timing: bit s set = stage s recorded
  uint32_t timing_mask = 0;
  struct Rec {
    int stage;
    hipEvent_t a, b;
  };
  std::vector<Rec> recs;
  std::vector<hipEvent_t> ev_pool;
  double t_ms[LL_STAGE_COUNT] = {};
  int64_t t_n[LL_STAGE_COUNT] = {};
};

namespace {

int in_width(const ll_plan* p, int l) { return l == 0 ? p->d.I : p->d.H; }

// The dW products of layer l: dW[a_row .. a_row+m, c_col .. c_col+n] =
// XT[a_row .. a_row+m]  DZT[b_row .. b_row+n]^T, XT = [X^T; Hprev^T] and DZT
// the transposed dz rows.  One product over the stacked operand; the GRU's
// two sides differ in the candidate block (dz_n on the input side, da_n * r
// on the recurrent side, dz columns 2H and 3H), so its r, u blocks take one
// product over the stacked operand and the candidate block one per side.
struct DwPart {
  int a_row, m, b_row, n, c_col;
};
int dw_parts(const ll_plan* p, int l, DwPart* out) {
  const int H = p->d.H, Il = in_width(p, l);
  if (p->G == 3) {
    out[0] = DwPart{0, Il + H, 0, 2 * H, 0};
    out[1] = DwPart{0, Il, 2 * H, H, 2 * H};
    out[2] = DwPart{Il, H, 3 * H, H, 2 * H};
    return 3;
  }
  out[0] = DwPart{0, Il + H, 0, p->G * H, 0};
  return 1;
}

// The same products taken straight from the row-major operands (bf16): the
// input part (rows 0 .. Il - 1 of dW, A = the layer's input rows) and the
// recurrent part (rows Il .., A = the h history rows of h_{t-1}) read
// different arrays, so each is a product of its own; b_row is the dz column.
// When the input width is a multiple of the 256-row tile the two parts of
// one dz column range are one launch (m = Il + H; rows from Il on read the
// h history).
int dw_parts_rows(const ll_plan* p, int l, DwPart* out) {
  const int H = p->d.H, Il = in_width(p, l);
  if (p->G == 3) {
    out[0] = DwPart{0, Il, 0, 3 * H, 0};
    out[1] = DwPart{Il, H, 0, 2 * H, 0};
    out[2] = DwPart{Il, H, 3 * H, H, 2 * H};
    return 3;
  }
  if (Il % ll::kGemmBigTile == 0) {
    out[0] = DwPart{0, Il + H, 0, p->G * H, 0};
    return 1;
  }
  out[0] = DwPart{0, Il, 0, p->G * H, 0};
  out[1] = DwPart{Il, H, 0, p->G * H, 0};
  return 2;
}

hipEvent_t take_event(ll_plan* p) {
  if (!p->ev_pool.empty()) {
    hipEvent_t e = p->ev_pool.back();
    p->ev_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  // (timing only: no system-scope fence, which would idle the GPU for
  // several microseconds at every bracket)
  if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) return nullptr;
  return e;
}

// Stage bracket: tbeg records the opening event, tend the closing one (only
// for the stages the plan times).
hipEvent_t tbeg(ll_plan* p, hipStream_t s, int stage) {
  if (!(p->timing_mask & (1u << stage))) return nullptr;
  hipEvent_t a = take_event(p);
  if (a && hipEventRecord(a, s) != hipSuccess) {
    p->ev_pool.push_back(a);
    return nullptr;
  }
  return a;
}

void tend(ll_plan* p, hipStream_t s, int stage, hipEvent_t a) {
  if (!a) return;
  hipEvent_t b = take_event(p);
  if (!b || hipEventRecord(b, s) != hipSuccess) {
    p->ev_pool.push_back(a);
    if (b) p->ev_pool.push_back(b);
    return;
  }
  p->recs.push_back(ll_plan::Rec{stage, a, b});
}

void drain_timing(ll_plan* p) {
  for (auto& r : p->recs) {
    float ms = 0.f;
    if (hipEventSynchronize(r.b) == hipSuccess && hipEventElapsedTime(&ms, r.a, r.b) == hipSuccess) {
      p->t_ms[r.stage] += ms;
      p->t_n[r.stage] += 1;
    }
    p->ev_pool.push_back(r.a);
    p->ev_pool.push_back(r.b);
  }
  p->recs.clear();
}

void free_plan_memory(ll_plan* p) {
  void* ptrs[] = {p->perm, p->active, p->off, p->rowmap, p->meta, p->WT[0], p->WT[1], p->Zx,
                  p->stack[0], p->stack[1], p->HH[0], p->HH[1], p->DZ, p->DZT, p->XT,
                  p->dyc, p->xring, p->xflags, p->db_part, p->ws, p->carry, p->db_state,
                  p->xring2, p->DZ2, p->dyx, p->db_part2, p->cring, p->cpart, p->cflags,
                  p->gslot, p->rc_inmap, p->rc_prevmap, p->rc_bias, p->sx, p->guards, p->Wum[0],
                  p->Wum[1], p->prevc, p->HI, p->ntrip, p->tn_flags, p->xflags_b};
  for (void* q : ptrs)
    if (q) (void)hipFree(q);
  for (float* h : p->host_stack)
    if (h) (void)hipHostFree(h);
  for (hipEvent_t e : p->ev_d2h)
    if (e) (void)hipEventDestroy(e);
  for (hipEvent_t e : p->ev_h2d)
    if (e) (void)hipEventDestroy(e);
  if (p->ev_compute) (void)hipEventDestroy(p->ev_compute);
  if (p->cstream) (void)hipStreamDestroy(p->cstream);
  if (p->cstream2) (void)hipStreamDestroy(p->cstream2);
  if (p->ev_fork) (void)hipEventDestroy(p->ev_fork);
  if (p->ev_join) (void)hipEventDestroy(p->ev_join);
  if (p->ev_done) (void)hipEventDestroy(p->ev_done);
  if (p->gstream) (void)hipStreamDestroy(p->gstream);
}

ll_status dalloc(void** out, size_t bytes, const char* what) {
  *out = nullptr;
  if (bytes == 0) bytes = 16;
  hipError_t e = hipMalloc(out, bytes);
  if (e != hipSuccess) {
    *out = nullptr;
    (void)hipGetLastError();
    return fail(LL_ENOMEM, "device allocation of %zu bytes for %s failed: %s", bytes, what,
                hipGetErrorString(e));
  }
  return LL_OK;
}

// Choose the loop work split: hidden units per work-group HJ in {16, 8, 4},
// row groups RG; as many work-groups as compute units allow (one per CU,
// the weight slice fills most of the LDS), then the widest HJ.
bool choose_geometry(int B, int H, int es, int n_cu, size_t lds_max, ll::LoopGeom* out) {
  const int NRT = (B + 15) / 16;
  bool found = false;
  ll::LoopGeom best{};
  for (int HJ : {16, 8, 4}) {
    if (H % HJ) continue;
    const int NCB = H / HJ;
    if (NCB > n_cu) continue;
    const size_t lf = ll::fwd_loop_lds(H, HJ, es), lb = ll::bwd_loop_lds(H, HJ, es);
    if (lf > lds_max || lb > lds_max) continue;
    int RG = std::min(NRT, n_cu / NCB);
    if (RG < 1) RG = 1;
    const int MRT = (NRT + RG - 1) / RG;
    if (MRT > 16) continue;
    const int nwg = NCB * RG;
    if (!found || nwg > best.nwg) {
      best = ll::LoopGeom{HJ, RG, NRT, MRT, nwg, lf, lb};
      found = true;
    }
  }
  if (found) *out = best;
  return found;
}

ll_status validate_desc(const ll_desc* d) {
  if (!d) return fail(LL_EINVAL, "desc is NULL");
  if (d->T_max < 1 || d->B < 1 || d->I < 1 || d->H < 1)
    return fail(LL_EINVAL, "T_max, B, I, H must be >= 1 (got %d, %d, %d, %d)", d->T_max, d->B,
                d->I, d->H);
  if (d->layers != 1 && d->layers != 2)
    return fail(LL_EINVAL, "layers must be 1 or 2 (got %d)", d->layers);
  if (d->dtype != LL_F32 && d->dtype != LL_BF16)
    return fail(LL_EINVAL, "dtype must be LL_F32 or LL_BF16 (got %d)", d->dtype);
  if (d->spill != 0 && d->spill != 1) return fail(LL_EINVAL, "spill must be 0 or 1");
  if (d->spill_chunk_steps < 0 || d->device_stack_budget_bytes < 0)
    return fail(LL_EINVAL, "spill_chunk_steps and device_stack_budget_bytes must be >= 0");
  if (d->recompute != 0 && d->recompute != 1) return fail(LL_EINVAL, "recompute must be 0 or 1");
  if (d->recompute && d->spill)
    return fail(LL_EUNSUPPORTED, "recompute and spill are alternatives; choose one");
  if (d->cell != LL_CELL_LSTM && d->cell != LL_CELL_RNN && d->cell != LL_CELL_GRU &&
      d->cell != LL_CELL_LSTM_SKIP && d->cell != LL_CELL_LSTM_ACT)
    return fail(LL_EINVAL,
                "cell must be LL_CELL_LSTM, LL_CELL_RNN, LL_CELL_GRU, LL_CELL_LSTM_SKIP or LL_CELL_LSTM_ACT (got %d)",
                d->cell);
  if (d->cell == LL_CELL_LSTM_ACT) {
    if (d->ponder_max < 1 || d->ponder_max > LL_ACT_PONDER_MAX)
      return fail(LL_EINVAL, "ponder_max must be in 1 .. %d for LL_CELL_LSTM_ACT (got %d)", LL_ACT_PONDER_MAX,
                  d->ponder_max);
    if (d->layers != 1) return fail(LL_EUNSUPPORTED, "the nested-loop body is built for one layer");
  } else if (d->ponder_max != 0) {
    return fail(LL_EINVAL, "ponder_max must be 0 for cells other than LL_CELL_LSTM_ACT (got %d)", d->ponder_max);
  }
  if (d->cell != LL_CELL_LSTM && (d->spill || d->recompute))
    return fail(LL_EUNSUPPORTED, "spill and recompute are built for the LSTM cell only");
  if ((long)d->T_max * d->B > (1L << 30))
    return fail(LL_EUNSUPPORTED, "T_max * B = %ld exceeds 2^30 rows", (long)d->T_max * d->B);
  if (d->H % 32) return fail(LL_EUNSUPPORTED, "H = %d must be a multiple of 32", d->H);
  const int ialign = d->dtype == LL_BF16 ? 8 : 4;
  if (d->I % ialign)
    return fail(LL_EUNSUPPORTED, "I = %d must be a multiple of %d for this dtype", d->I, ialign);
  if (d->B > 4096) return fail(LL_EUNSUPPORTED, "B = %d exceeds 4096", d->B);
  if (d->reserved != 0) return fail(LL_EINVAL, "desc.reserved must be 0 (got %d)", d->reserved);
  return LL_OK;
}

// Every decision of a plan that needs no device memory: problem, launch
// forms (XCD-local, chip-wide or grid-barrier loops; wavefront), memory
// policy, dW paths and their split-K.  Used by ll_plan_create and by the
// forward that allocates nothing.  `prop` is the device's properties, the
// device current.
ll_status plan_configure(ll_plan* p, const ll_desc* desc, int device, const hipDeviceProp_t& prop) {
  p->d = *desc;
  p->device = device;
  p->bf16 = desc->dtype == LL_BF16;
  p->es = p->bf16 ? 2 : 4;
  p->G = desc->cell == LL_CELL_RNN ? 1 : desc->cell == LL_CELL_GRU ? 3 : 4;
  p->skip = desc->cell == LL_CELL_LSTM_SKIP;
  p->act = desc->cell == LL_CELL_LSTM_ACT;
  p->M = p->act ? desc->ponder_max : 1;
  p->GB = desc->cell == LL_CELL_GRU ? 4 : p->G;
  p->n_cu = prop.multiProcessorCount;
  p->cap = (long)desc->T_max * desc->B;
  p->ldT = round_up(p->cap, 64);
  int wall_khz = 0;
  if (hipDeviceGetAttribute(&wall_khz, hipDeviceAttributeWallClockRate, device) != hipSuccess ||
      wall_khz <= 0)
    wall_khz = 100000;
  p->barrier_ticks = (unsigned long long)wall_khz * 5000ull;   // 5 s

  const size_t lds_max = prop.sharedMemPerBlock > 0 ? (size_t)prop.sharedMemPerBlock : 65536;
  size_t lds_limit = lds_max;
  {
    int optin = 0;
    if (hipDeviceGetAttribute(&optin, hipDeviceAttributeSharedMemPerBlockOptin, device) ==
            hipSuccess &&
        optin > 0)
      lds_limit = std::max(lds_limit, (size_t)optin);
  }
  const int H = desc->H, B = desc->B, L = desc->layers;
  if (!choose_geometry(B, H, p->es, p->n_cu, lds_limit, &p->geom)) {
    return fail(LL_EUNSUPPORTED,
                "no loop geometry fits: H = %d, B = %d, %d CUs, %zu bytes of LDS per group", H,
                B, prop.multiProcessorCount, lds_limit);
  }
  int occ_f = 0, occ_b = 0;
  hipError_t he = p->bf16 ? ll::loop_kernel_setup<bf16_t>(p->geom.MRT, p->geom.lds_fwd,
                                                          p->geom.lds_bwd, &occ_f, &occ_b)
                          : ll::loop_kernel_setup<float>(p->geom.MRT, p->geom.lds_fwd,
                                                         p->geom.lds_bwd, &occ_f, &occ_b);
  if (he != hipSuccess) {
    return fail(LL_EHIP, "loop kernel setup failed: %s", hipGetErrorString(he));
  }
  if ((long)occ_f * p->n_cu < p->geom.nwg || (long)occ_b * p->n_cu < p->geom.nwg) {
    return fail(LL_EUNSUPPORTED,
                "loops need %d co-resident work-groups; occupancy allows %d/%d per CU x %d CUs",
                p->geom.nwg, occ_f, occ_b, p->n_cu);
  }

  // XCD-local loops: 8 XCDs x 32 CUs, every exchanged row 128-byte aligned,
  // H split 32 ways (bf16: 32 units per work-group, f32: 16).
  const char* loops_env = getenv("LSTMLOOP_LOOPS");
  const bool allow = !(loops_env && strcmp(loops_env, "grid") == 0);
  {
    const int HJx = p->bf16 ? 32 : 16;
    const int P = H / HJx;
    if (allow && p->n_cu == 256 && H % HJx == 0 && P >= 1 && P <= 32 &&
        ((long)H * p->es) % 128 == 0) {
      const int KS = p->bf16 ? H / 32 : H / 16;      // forward k-steps, 8 waves share them
      const int need = (KS + 7) / 8;
      const int hc = need <= 1 ? 1 : need <= 2 ? 2 : need <= 4 ? 4 : 0;
      const int mrt = ((B + 15) / 16 + 7) / 8;
      if (hc && mrt <= 16) {
        ll::XKernels xk = p->bf16 ? ll::x_kernels<bf16_t>(hc, mrt, p->G, p->skip, p->act)
                                  : ll::x_kernels<float>(hc, mrt, p->G, p->skip, p->act);
        if (xk.fwd && xk.bwd && xk.lds_fwd <= lds_limit && xk.lds_bwd <= lds_limit) {
          int of = 0, ob = 0;
          if (ll::x_setup(xk, &of, &ob) == hipSuccess && of >= 1 && ob >= 1) {
            p->xmode = true;
            p->xk = xk;
            p->xP = P;
            p->xMRT = mrt;
            p->xhc = hc;
          } else {
            (void)hipGetLastError();
          }
        }
      }
    }
  }

  // The Elman RNN, GRU and cond-body cells run on the XCD-local loops only.
  if ((p->G != 4 || p->skip || p->act) && !p->xmode) {
    return fail(LL_EUNSUPPORTED, "the %s cell needs the XCD-local loops (H = %d, B = %d do not fit them)",
                p->G == 1 ? "RNN" : p->G == 3 ? "GRU" : p->act ? "nested-loop LSTM" : "cond-body LSTM", H, B);
  }

  // Chip-wide loops where one XCD cannot hold the recurrent weights (bf16
  // H = 2048, f32 H = 1024, B <= 256).
  if (!p->xmode && allow && p->n_cu == 256) {
    const int mrt = (B + 15) / 16;
    ll::CKernels ck = p->bf16 ? ll::c_kernels<bf16_t>(H, mrt) : ll::c_kernels<float>(H, mrt);
    if (ck.fwd && ck.bwd) {
      int of = 0, ob = 0;
      if (ll::c_setup(ck, &of, &ob) == hipSuccess && of >= 1 && ob >= 1) {
        p->cmode = true;
        p->ck = ck;
        p->cMRT = mrt;
      } else {
        (void)hipGetLastError();
      }
    }
  }

  // Stack spill (swapping of the saved values to host memory while the loop
  // runs): the XCD-local loops run one launch per chunk of steps, and the
  // stack becomes a device ring of nslots chunks.
  if (desc->spill) {
    if (!p->xmode) {
      return fail(LL_EUNSUPPORTED, "spill needs the XCD-local loops (H = %d, B = %d do not fit them)",
                  H, B);
    }
    p->spill = true;
    p->chunk_steps = std::min(desc->T_max, desc->spill_chunk_steps > 0 ? desc->spill_chunk_steps : 32);
    p->nchunks = (desc->T_max + p->chunk_steps - 1) / p->chunk_steps;
    p->slot_floats = (long)p->chunk_steps * B * 5 * H;
    const long slot_bytes = p->slot_floats * (long)sizeof(float);
    long r = desc->device_stack_budget_bytes > 0 ? desc->device_stack_budget_bytes / slot_bytes : 4;
    p->nslots = (int)std::max(3L, std::min(r, (long)p->nchunks));
  }
  if (desc->recompute) {
    if (!p->xmode) {
      return fail(LL_EUNSUPPORTED,
                  "recompute needs the XCD-local loops (H = %d, B = %d do not fit them)", H, B);
    }
    p->recompute = true;
    p->rc_steps = std::min(desc->T_max, desc->spill_chunk_steps > 0 ? desc->spill_chunk_steps : 32);
    p->rc_chunks = (desc->T_max + p->rc_steps - 1) / p->rc_steps;
  }

  // Two-layer wavefront: on every XCD, members 0..P-1 run the lower layer
  // and P..2P-1 the upper one, so both layers' steps overlap in one launch.
  // LSTMLOOP_WAVEFRONT=off at plan creation runs the layers one after the
  // other.
  if (L == 2 && p->G == 4 && !p->skip && p->xmode && !p->spill && !p->recompute && 2 * p->xP <= 32 &&
      p->xhc <= 2) {
    const char* wf = getenv("LSTMLOOP_WAVEFRONT");
    if (!(wf && strcmp(wf, "off") == 0)) {
      ll::XKernels xk2 = p->bf16 ? ll::x_kernels2<bf16_t>(p->xhc, p->xMRT)
                                 : ll::x_kernels2<float>(p->xhc, p->xMRT);
      if (xk2.fwd && xk2.bwd && xk2.lds_fwd <= lds_limit && xk2.lds_bwd <= lds_limit) {
        int of = 0, ob = 0;
        if (ll::x_setup(xk2, &of, &ob) == hipSuccess && of >= 1 && ob >= 1) {
          p->wave = true;
          p->xk2 = xk2;
        } else {
          (void)hipGetLastError();
        }
      }
    }
  }

  // dW split-K, per product: enough work-groups to cover the chip (one
  // 256x256 tile per compute unit for the large-tile bf16 kernel, two 128x128
  // tiles else).  The products run one after the other and share the
  // workspace of the partial sums.
  // bf16 dW: the product over rows (no transposed copies, but its operand
  // reads run it at ~0.72 of the rate of the product on transposed copies,
  // measured ~0.72 vs ~1.0 PFLOP/s) or the transposes (~2.2 TB/s) plus that
  // product, whichever the model says is shorter: rows win while
  // flops / transposed bytes < ~1170 (H = I = 1024: ~683; H = I = 2048: ~1365)
  p->ws_floats = 0;
  // The product over rows addresses each operand (x or the layer below's
  // h history, this layer's h history with the h0 rows, dz) through 32-bit
  // buffer offsets: a layer whose operand reaches 2^31 bytes takes the
  // transposes instead, whatever the model says.
  for (int l = 0; l < L; ++l) {
    const double Il = in_width(p, l);
    const double flops = 2.0 * (Il + H) * p->G * H, bytes = (Il + H + p->GB * H) * 2.0 * p->es;
    const long lim = 1L << 31;
    const bool fits = p->cap * (long)Il * 2 < lim && (p->cap + B) * (long)H * 2 < lim &&
                      p->cap * (long)p->GB * H * 2 < lim;
    p->dw_rows[l] = p->bf16 && fits && flops / bytes < 1170.0;
  }
  for (int l = 0; l < L; ++l) {   // the products over rows
    if (!p->dw_rows[l]) continue;
    DwPart parts[3];
    const int np = dw_parts_rows(p, l, parts);
    for (int k = 0; k < np; ++k) {
      const long tiles = (long)((parts[k].m + ll::kGemmBigTile - 1) / ll::kGemmBigTile) *
                         ((parts[k].n + ll::kGemmBigTile - 1) / ll::kGemmBigTile);
      long sp = (p->n_cu + tiles - 1) / tiles;
      sp = std::max(1L, std::min(16L, std::min(sp, std::max(1L, p->cap / 256))));
      p->tn_splits[l][k] = (int)sp;
      if (sp > 1) p->ws_floats = std::max(p->ws_floats, sp * parts[k].m * parts[k].n);
      if (sp == 2) p->tn_flag_words = std::max(p->tn_flag_words, 2 * tiles);
    }
  }
  for (int l = 0; l < L; ++l) {
    if (p->dw_rows[l]) continue;
    DwPart parts[3];
    const int np = dw_parts(p, l, parts);
    for (int k = 0; k < np; ++k) {
      ll::GemmArgs g{};
      g.lda = g.ldb = p->ldT;
      g.M = parts[k].m;
      g.N = parts[k].n;
      g.K = (int)p->cap;
      g.splits = 1;
      g.k_zero_tail = 1;
      const bool big = ll::gemm_big_applies(g, (int)p->es);
      const long tile = big ? ll::kGemmBigTile : 128;
      const long tiles = (long)((g.M + tile - 1) / tile) * ((g.N + tile - 1) / tile);
      const long want = big ? p->n_cu : 2L * p->n_cu;
      long s = (want + tiles - 1) / tiles;
      s = std::max(1L, std::min(16L, s));
      const long max_by_k = std::max(1L, p->cap / 256);
      p->dw_splits[l][k] = (int)std::min(s, max_by_k);
      if (p->dw_splits[l][k] > 1)
        p->ws_floats = std::max(p->ws_floats, (long)p->dw_splits[l][k] * g.M * g.N);
    }
  }
  // nested-loop body: the dW products of the M ponder slots all go to the
  // workspace before one sum, and so do the M dx products (compact rows)
  if (p->act) {
    long need = (long)p->M * p->cap * desc->I;
    for (int k = 0; k < 3; ++k) {
      DwPart parts[3];
      const int np = p->dw_rows[0] ? dw_parts_rows(p, 0, parts) : dw_parts(p, 0, parts);
      if (k >= np) break;
      const long sp = p->dw_rows[0] ? p->tn_splits[0][k] : p->dw_splits[0][k];
      need = std::max(need, (long)p->M * sp * parts[k].m * parts[k].n);
    }
    p->ws_floats = std::max(p->ws_floats, need);
  }
  return LL_OK;
}

// The plan's device buffers in one place: `take(slot, bytes, what)` gives
// each its memory (ll_plan_create: a device allocation; the forward that
// allocates nothing: a piece of the library's scratch array).  fwd_only:
// only what an inference forward touches (no stack, no gradient buffers).
template <typename Take>
ll_status plan_layout(ll_plan* p, bool fwd_only, Take&& take) {
  const ll_desc* desc = &p->d;
  const int H = desc->H, B = desc->B, L = desc->layers;
  const int maxI = std::max(desc->I, H);

  const size_t es = p->es;
  const long cap = p->cap;
#define ALLOC(ptr, bytes, what)                                      \
  do {                                                               \
    void* tmp_ = nullptr;                                            \
    ll_status s_ = take(&tmp_, (size_t)(bytes), what);               \
    if (s_ != LL_OK) return s_;                                      \
    ptr = reinterpret_cast<decltype(ptr)>(tmp_);                     \
  } while (0)
  ALLOC(p->perm, sizeof(int) * B, "perm");
  ALLOC(p->active, sizeof(int) * (desc->T_max + 1), "active");
  ALLOC(p->off, sizeof(int) * (desc->T_max + 1), "off");
  ALLOC(p->rowmap, sizeof(int) * cap, "rowmap");
  ALLOC(p->meta, sizeof(int) * ll::META_INTS, "meta");
  for (int l = 0; l < L; ++l) {
    ALLOC(p->WT[l], es * p->G * H * (in_width(p, l) + H), "transposed W");
    if (!fwd_only)
      ALLOC(p->stack[l],
            sizeof(float) * (p->spill ? p->nslots * p->slot_floats
                                      : (long)p->M * cap * (p->recompute || p->G == 1 ? 1 : 5) * H),
            "stack");
    // (B more rows hold h0 in the operand type, the h_{t-1} of step 0)
    ALLOC(p->HH[l], es * (cap + B) * H, "h history");
  }
  ALLOC(p->Zx, sizeof(float) * cap * p->G * H, "input projection");
  if (!fwd_only) ALLOC(p->DZ, es * p->M * cap * p->GB * H, "dz");
  if (p->act && !fwd_only) {
    ALLOC(p->HI, es * p->M * cap * H, "ponder states");
    ALLOC(p->ntrip, sizeof(int) * (long)desc->T_max * 8 * std::max(p->xMRT, 1), "inner trip counts");
  }
  if (!fwd_only && (!p->dw_rows[0] || (L == 2 && !p->dw_rows[1]))) {   // (transposed copies for the NT products)
    ALLOC(p->DZT, es * p->GB * H * p->ldT, "dz transposed");
    ALLOC(p->XT, es * (maxI + H) * p->ldT, "x and h_prev transposed");
  }
  if (L == 2 && !fwd_only) ALLOC(p->dyc, sizeof(float) * cap * H, "inter-layer gradient");
  if (p->xmode) {
    // two slots x 8 XCDs x row tiles x (G H / k-step) blocks of 1 KB
    const long ks_b = (long)p->G * H * (long)es / 64;
    ALLOC(p->xring, 2L * 8 * p->xMRT * ks_b * 1024, "exchange ring");
    p->xflag_words = 8 + (p->wave ? 3 : 1) * 8 * p->xMRT * 32;
    ALLOC(p->xflags, sizeof(unsigned) * p->xflag_words, "exchange flags");
    if (!fwd_only && L == 1 && !p->spill && !p->recompute)
      ALLOC(p->xflags_b, sizeof(unsigned) * p->xflag_words, "gradient loop flags");
    if (p->wave) {
      ALLOC(p->xring2, 2L * 8 * p->xMRT * ks_b * 1024, "exchange ring");
      if (!fwd_only) {
        ALLOC(p->DZ2, es * cap * 4 * H, "dz");
        ALLOC(p->dyx, sizeof(float) * 2L * 8 * p->xMRT * 16 * H, "dy exchange");
        ALLOC(p->db_part2, sizeof(float) * 8 * 4 * H, "db partials");
      }
    }
  }
  if (p->cmode) {
    // two slots x row tiles x (4H / k-step) blocks of 1 KB; partial products
    ALLOC(p->cring, 2L * p->cMRT * (4L * H * (long)es / 64) * 1024, "exchange ring");
    ALLOC(p->cpart, sizeof(float) * 2L * 8 * p->cMRT * 32 * p->ck.pw, "partial products");
    p->cflag_words = 8 + p->cMRT * 256 + 8 * p->cMRT * 32;
    ALLOC(p->cflags, sizeof(unsigned) * p->cflag_words, "exchange flags");
  }
  if (p->skip) ALLOC(p->sx, sizeof(float) * cap, "predicate input part");
  if (fwd_only) return LL_OK;   // the rest serves the saved stack and the gradient pass
  if (p->recompute) {
    ALLOC(p->gslot, sizeof(float) * (long)p->rc_steps * B * 4 * H, "recomputed gates");
    ALLOC(p->rc_inmap, sizeof(int) * 2 * cap, "recomputation row maps");
    ALLOC(p->rc_prevmap, sizeof(int) * cap, "recomputation row maps");
    ALLOC(p->rc_bias, sizeof(float) * L * 4 * H, "saved bias");
  }
  if (p->spill || p->recompute) {
    ALLOC(p->carry, sizeof(float) * 4 * B * H, "chunk carry");
    ALLOC(p->db_state, sizeof(float) * 8 * 32 * 512 * 4, "db state");
  }
  ALLOC(p->db_part, sizeof(float) * std::max(p->geom.RG, 8) * p->GB * H, "db partials");
  if (p->xmode && p->G == 4)
    for (int l = 0; l < L; ++l) ALLOC(p->Wum[l], es * 4L * H * H, "permuted recurrent weights");
  if (p->dw_rows[0] || p->dw_rows[1]) ALLOC(p->prevc, sizeof(int) * cap, "previous-row map");
  if (p->skip || p->act) ALLOC(p->guards, sizeof(float) * L * p->M * cap, "guard stack");
  if (p->ws_floats > 0) ALLOC(p->ws, sizeof(float) * p->ws_floats, "split-K workspace");
  if (p->tn_flag_words > 0) ALLOC(p->tn_flags, sizeof(unsigned) * p->tn_flag_words, "split-K tile counters");
#undef ALLOC
  return LL_OK;
}

// A copy between device memory and pinned host memory on the DMA engines.
// The runtime runs one-dimensional such copies as blit kernels on the compute
// units, which the persistent loops need whole (measured on the spill
// workload: a loop chunk beside such a copy took 0.49 ms against 0.13 ms
// alone); two-dimensional copies with rows of 1 MiB go to the copy engines
// (same ~52 GB/s, no kernel).
hipError_t copy_on_dma_engine(void* dst, const void* src, size_t bytes, hipMemcpyKind kind, hipStream_t s) {
  constexpr size_t kRow = 1u << 20;
  const size_t rows = bytes / kRow, rem = bytes - rows * kRow;
  if (rows > 0) {
    hipError_t e = hipMemcpy2DAsync(dst, kRow, src, kRow, kRow, rows, kind, s);
    if (e != hipSuccess) return e;
  }
  if (rem > 0)
    return hipMemcpy2DAsync(static_cast<char*>(dst) + rows * kRow, rem,
                            static_cast<const char*>(src) + rows * kRow, rem, rem, 1, kind, s);
  return hipSuccess;
}

}  // namespace

extern "C" {

const char* ll_last_error(void) { return g_last_error.c_str(); }

const char* ll_version(void) { return "lstmloop 0.1 (gfx950)"; }

ll_status ll_measure_mfma_peak(int32_t device, int32_t dtype, int32_t shape, double* tflops) {
  if (!tflops) return fail(LL_EINVAL, "tflops is NULL");
  if (dtype != LL_F32 && dtype != LL_BF16) return fail(LL_EINVAL, "dtype must be LL_F32 or LL_BF16");
  if (shape != 16 && shape != 32) return fail(LL_EINVAL, "shape must be 16 or 32 (got %d)", shape);
  int ndev = 0;
  LL_HIP(hipGetDeviceCount(&ndev));
  if (device < 0 || device >= ndev) return fail(LL_EINVAL, "device %d out of range (%d devices)", device, ndev);
  DeviceGuard guard(device);
  hipDeviceProp_t prop;
  LL_HIP(hipGetDeviceProperties(&prop, device));
  *tflops = 0.0;
  LL_HIP(dtype == LL_BF16 ? ll::measure_mfma_peak<bf16_t>(prop.multiProcessorCount, shape == 32, tflops)
                          : ll::measure_mfma_peak<float>(prop.multiProcessorCount, shape == 32, tflops));
  return LL_OK;
}

ll_status ll_eval_activations(int32_t device, const float* in, float* out, int64_t n, int32_t fn) {
  if (fn != 0 && fn != 1) return fail(LL_EINVAL, "fn must be 0 (sigmoid) or 1 (tanh), got %d", fn);
  if (n < 0) return fail(LL_EINVAL, "n = %lld is negative", (long long)n);
  if (n > 0 && (!in || !out)) return fail(LL_EINVAL, "in and out are required");
  int ndev = 0;
  LL_HIP(hipGetDeviceCount(&ndev));
  if (device < 0 || device >= ndev) return fail(LL_EINVAL, "device %d out of range (%d devices)", device, ndev);
  if (n == 0) return LL_OK;
  DeviceGuard guard(device);
  LL_HIP(ll::eval_activations(in, out, (long)n, fn, nullptr));
  LL_HIP(hipStreamSynchronize(nullptr));
  return LL_OK;
}

ll_status ll_plan_create(const ll_desc* desc, int device, ll_plan** out) {
  if (!out) return fail(LL_EINVAL, "out is NULL");
  *out = nullptr;
  ll_status st = validate_desc(desc);
  if (st != LL_OK) return st;
  int ndev = 0;
  LL_HIP(hipGetDeviceCount(&ndev));
  if (device < 0 || device >= ndev)
    return fail(LL_EINVAL, "device %d out of range (%d devices)", device, ndev);
  DeviceGuard guard(device);
  hipDeviceProp_t prop;
  LL_HIP(hipGetDeviceProperties(&prop, device));
  if (!prop.cooperativeLaunch)
    return fail(LL_EUNSUPPORTED, "device %d does not support cooperative launches", device);

  ll_plan* p = new (std::nothrow) ll_plan();
  if (!p) return fail(LL_ENOMEM, "host allocation of the plan failed");
  st = plan_configure(p, desc, device, prop);
  if (st != LL_OK) {
    delete p;
    return st;
  }
  const int H = desc->H, B = desc->B, L = desc->layers;
  const long cap = p->cap;
  const size_t es = p->es;
  {
    auto take = [](void** slot, size_t bytes, const char* what) { return dalloc(slot, bytes, what); };
    st = plan_layout(p, false, take);
    if (st != LL_OK) {
      free_plan_memory(p);
      delete p;
      return st;
    }
  }
  if (p->HI && hipMemset(p->HI, 0, es * p->M * cap * H) != hipSuccess) {
    free_plan_memory(p);
    delete p;
    return fail(LL_EHIP, "hipMemset of the ponder states failed");
  }
  if (hipMemset(p->meta, 0, sizeof(int) * ll::META_INTS) != hipSuccess ||
      (p->tn_flags && hipMemset(p->tn_flags, 0, sizeof(unsigned) * p->tn_flag_words) != hipSuccess)) {
    free_plan_memory(p);
    delete p;
    return fail(LL_EHIP, "hipMemset of the plan's meta words or tile counters failed");
  }
  if (hipStreamCreateWithFlags(&p->gstream, hipStreamNonBlocking) != hipSuccess ||
      hipEventCreateWithFlags(&p->ev_fork, kOrderEventFlags) != hipSuccess ||
      hipEventCreateWithFlags(&p->ev_join, kOrderEventFlags) != hipSuccess ||
      hipEventCreateWithFlags(&p->ev_done, kOrderEventFlags) != hipSuccess) {
    free_plan_memory(p);
    delete p;
    return fail(LL_EHIP, "creating the plan's side stream failed");
  }
  if (p->spill) {
    // only the chunks a later chunk evicts from the ring are swapped out (and
    // back in); the last nslots chunks stay on the device
    const size_t hbytes = sizeof(float) * (size_t)std::max(0, p->nchunks - p->nslots) * (size_t)p->slot_floats;
    for (int l = 0; l < L && hbytes > 0; ++l) {
      if (hipHostMalloc(reinterpret_cast<void**>(&p->host_stack[l]), hbytes, hipHostMallocDefault) !=
          hipSuccess) {
        free_plan_memory(p);
        delete p;
        return fail(LL_ENOMEM, "pinned host allocation of %zu bytes for the spilled stack failed", hbytes);
      }
    }
    bool ok = hipStreamCreateWithFlags(&p->cstream, hipStreamNonBlocking) == hipSuccess &&
              hipStreamCreateWithFlags(&p->cstream2, hipStreamNonBlocking) == hipSuccess &&
              hipEventCreateWithFlags(&p->ev_compute, hipEventDisableTiming) == hipSuccess;
    p->ev_d2h.assign((size_t)L * p->nslots, nullptr);
    p->ev_h2d.assign((size_t)L * p->nslots, nullptr);
    for (size_t i = 0; ok && i < p->ev_d2h.size(); ++i)
      ok = hipEventCreateWithFlags(&p->ev_d2h[i], hipEventDisableTiming) == hipSuccess &&
           hipEventCreateWithFlags(&p->ev_h2d[i], hipEventDisableTiming) == hipSuccess;
    if (!ok) {
      free_plan_memory(p);
      delete p;
      return fail(LL_EHIP, "creating the spill copy stream and events failed");
    }
  }
  const int64_t stack_dev = p->spill ? (int64_t)sizeof(float) * p->nslots * p->slot_floats
                                     : (int64_t)sizeof(float) * p->M * cap * (p->recompute || p->G == 1 ? 1 : 5) * H;
  p->stack_device_bytes = (int64_t)L * (stack_dev + (int64_t)es * (cap + (p->recompute ? B : 0)) * H);
  if (p->recompute) p->stack_device_bytes += (int64_t)sizeof(float) * p->rc_steps * B * 4 * H;
  p->stack_host_bytes =
      p->spill ? (int64_t)L * (int64_t)sizeof(float) * std::max(0, p->nchunks - p->nslots) * p->slot_floats : 0;
  *out = p;
  return LL_OK;
}

ll_status ll_plan_destroy(ll_plan* p) {
  if (!p) return LL_OK;
  DeviceGuard guard(p->device);
  // the plan's own work only: the last call's work (its closing event, which
  // stays valid even if the caller has destroyed that stream), the side
  // stream and the copy stream
  if (p->ev_done && p->done_recorded) (void)hipEventSynchronize(p->ev_done);
  if (p->gstream) (void)hipStreamSynchronize(p->gstream);
  if (p->cstream) (void)hipStreamSynchronize(p->cstream);
  if (p->cstream2) (void)hipStreamSynchronize(p->cstream2);
  drain_timing(p);
  for (hipEvent_t e : p->ev_pool) hipEventDestroy(e);
  free_plan_memory(p);
  delete p;
  return LL_OK;
}

ll_status ll_plan_set_timing_stages(ll_plan* p, uint32_t stage_mask) {
  if (!p) return fail(LL_EINVAL, "plan is NULL");
  if (stage_mask >> LL_STAGE_COUNT) return fail(LL_EINVAL, "stage mask 0x%x names no stage", stage_mask);
  DeviceGuard guard(p->device);
  drain_timing(p);
  for (int i = 0; i < LL_STAGE_COUNT; ++i) {
    p->t_ms[i] = 0.0;
    p->t_n[i] = 0;
  }
  p->timing_mask = stage_mask;
  return LL_OK;
}

ll_status ll_plan_set_timing(ll_plan* p, int32_t enable) {
  return ll_plan_set_timing_stages(p, enable ? (1u << LL_STAGE_COUNT) - 1u : 0u);
}

ll_status ll_plan_read_timing(ll_plan* p, int32_t stage, double* total_ms, int64_t* n) {
  if (!p) return fail(LL_EINVAL, "plan is NULL");
  if (stage < 0 || stage >= LL_STAGE_COUNT) return fail(LL_EINVAL, "stage %d out of range", stage);
  DeviceGuard guard(p->device);
  drain_timing(p);
  if (total_ms) *total_ms = p->t_ms[stage];
  if (n) *n = p->t_n[stage];
  return LL_OK;
}

ll_status ll_plan_stack_bytes(const ll_plan* p, int64_t* dev, int64_t* host) {
  if (!p) return fail(LL_EINVAL, "plan is NULL");
  if (dev) *dev = p->stack_device_bytes;
  if (host) *host = p->stack_host_bytes;
  return LL_OK;
}

ll_status ll_plan_geometry(const ll_plan* p, int32_t* nwg, int32_t* hj, int32_t* rg,
                           int32_t* loop_form, int32_t* wavefront, int32_t* dw_in_place) {
  if (!p) return fail(LL_EINVAL, "plan is NULL");
  if (dw_in_place) *dw_in_place = (p->dw_rows[0] ? 1 : 0) | (p->dw_rows[1] ? 2 : 0);
  if (nwg) *nwg = (p->xmode || p->cmode) ? 256 : p->geom.nwg;
  if (hj) *hj = p->xmode ? (p->bf16 ? 32 : 16) : p->cmode ? p->d.H / 256 : p->geom.HJ;
  if (rg) *rg = p->xmode ? 8 : p->cmode ? 1 : p->geom.RG;
  if (loop_form) *loop_form = p->xmode ? LL_LOOPS_XCD : p->cmode ? LL_LOOPS_CHIP : LL_LOOPS_GRID;
  if (wavefront) *wavefront = p->wave ? 1 : 0;
  return LL_OK;
}

}  // extern "C"

namespace {

// Fields shared by every argument block of a chip-wide launch.
ll::CLoopArgs c_common(const ll_plan* p) {
  ll::CLoopArgs a{};
  a.B = p->d.B;
  a.H = p->d.H;
  a.T_max = p->d.T_max;
  a.MRT = p->cMRT;
  a.meta = p->meta;
  a.active = p->active;
  a.off = p->off;
  a.perm = p->perm;
  a.ring = p->cring;
  a.part = p->cpart;
  a.rank_ctr = p->cflags;
  a.xflags = p->cflags + 8;
  a.pflags = p->cflags + 8 + p->cMRT * 256;
  a.abort_flag = p->meta + 3;
  a.err = p->meta + 2;
  a.limit = p->barrier_ticks;
  return a;
}

// Fields shared by both layers' argument blocks of an XCD-local launch.
ll::XLoopArgs x_common(const ll_plan* p) {
  ll::XLoopArgs a{};
  a.B = p->d.B;
  a.H = p->d.H;
  a.T_max = p->d.T_max;
  a.P = p->xP;
  a.MRT = p->xMRT;
  a.meta = p->meta;
  a.active = p->active;
  a.off = p->off;
  a.perm = p->perm;
  a.rank_ctr = p->xflags;
  a.abort_flag = p->meta + 3;
  a.err = p->meta + 2;
  a.limit = p->barrier_ticks;
  a.t_begin = 0;
  a.t_end = p->d.T_max;
  a.chunk_steps = p->d.T_max;
  a.nslots = 1;
  // stack rows: LSTM i, f, g, o, c_t (5H: the four gate values of unit u at
  // 4u .. 4u+3, then c_t); GRU r, u, n, zh_n + b_hn, h_{t-1} (the same
  // layout); the RNN pushes h_t only
  const bool five = p->G == 4 || p->G == 3;
  a.sld = five ? 5 * p->d.H : p->d.H;
  a.scoff = five ? 4 * p->d.H : 0;
  a.sgates = five ? 1 : 0;
  return a;
}

// Two-layer wavefront, forward: the input projection of layer 0 only (the
// upper layer multiplies y1_t inside the loop), then one launch in which the
// upper layer's step t follows the lower layer's step t on every XCD.
template <typename T>
ll_status enqueue_fwd_wave(ll_plan* p, hipStream_t s, const void* x, const void* const* W,
                           const float* const* bias, const float* h0, const float* c0, float* y,
                           float* hT, float* cT, bool save) {
  const ll_desc& d = p->d;
  const int H = d.H, B = d.B, I = d.I;
  const long BH = (long)B * H;
  hipEvent_t ev = tbeg(p, s, LL_STAGE_INPUT_PROJ);
  (void)W;   // (transposed by the set-up launch)
  ll::GemmArgs g{};
  g.A = x;
  g.lda = I;
  g.a_rowmap = p->rowmap;
  g.Bm = p->WT[0];
  g.ldb = I + H;
  g.C = p->Zx;
  g.ldc = 4L * H;
  g.bias = bias[0];
  g.M = (int)p->cap;
  g.M_dev = p->meta + 1;
  g.N = 4 * H;
  g.K = I;
  g.splits = 1;
  LL_HIP(ll::launch_gemm_nt<T>(g, s));
  tend(p, s, LL_STAGE_INPUT_PROJ, ev);

  const int ring_ks = (int)((long)H * p->es / 64);
  unsigned* F0 = p->xflags + 8;
  unsigned* F1 = F0 + 8L * p->xMRT * 32;
  ev = tbeg(p, s, LL_STAGE_LOOP_SETUP);
  LL_HIP(ll::launch_x_prepare_fwd<T>(h0, p->perm, B, H, p->xMRT, ring_ks, 1, p->xring, p->xflags,
                                     p->xflag_words, s));
  LL_HIP(ll::launch_x_prepare_fwd<T>(h0 ? h0 + BH : nullptr, p->perm, B, H, p->xMRT, ring_ks, 1,
                                     p->xring2, nullptr, 0, s));
  tend(p, s, LL_STAGE_LOOP_SETUP, ev);

  ll::XLoopArgs a0 = x_common(p), a1 = x_common(p);
  a0.ring = p->xring;
  a0.ring_ks = ring_ks;
  a0.flags = F0;
  a0.W = p->WT[0];
  a0.ldw = I + H;
  a0.woff = I;
  a0.X = p->HH[0];
  a0.Zx = p->Zx;
  a0.stack = save ? p->stack[0] : nullptr;
  a0.h0 = h0;
  a0.c0 = c0;
  a0.hT = hT;
  a0.cT = cT;
  a0.out_flags = F1;

  a1.ring = p->xring2;
  a1.ring_ks = ring_ks;
  a1.flags = F1;
  a1.W = p->WT[1];
  a1.ldw = 2 * H;
  a1.woff = 0;
  a1.X = p->HH[1];
  a1.zbias = bias[1];
  a1.stack = save ? p->stack[1] : nullptr;
  a1.y = y;
  a1.h0 = h0 ? h0 + BH : nullptr;
  a1.c0 = c0 ? c0 + BH : nullptr;
  a1.hT = hT + BH;
  a1.cT = cT + BH;
  a1.in_ring = p->xring;
  a1.in_flags = F0;
  a1.in_ks = ring_ks;
  ev = tbeg(p, s, LL_STAGE_FWD_LOOP);
  LL_HIP(chained_loop_launch(p->device, s, [&] { return ll::x_launch2(p->xk2.fwd, a0, a1, 256, p->xk2.lds_fwd, s); }));
  tend(p, s, LL_STAGE_FWD_LOOP, ev);
  return LL_OK;
}

template <typename T>
ll_status enqueue_fwd(ll_plan* p, hipStream_t s, const void* x, const int32_t* seq_len,
                      const void* const* W, const float* const* bias, const float* h0,
                      const float* c0, float* y, float* hT, float* cT, int32_t* trip,
                      bool save) {
  const ll_desc& d = p->d;
  const int H = d.H, B = d.B, L = d.layers;
  // prep (one work-group) beside the transposes W^T of every layer (row n =
  // gate column n, the K-contiguous operand of the input projection and the
  // loop), in one launch
  hipEvent_t ev = tbeg(p, s, LL_STAGE_PREP);
  {
    const T* Wl[2] = {nullptr, nullptr};
    T* WTl[2] = {nullptr, nullptr};
    int R[2] = {0, 0};
    for (int l = 0; l < L; ++l) {
      Wl[l] = reinterpret_cast<const T*>(W[l]);
      WTl[l] = reinterpret_cast<T*>(p->WT[l]);
      R[l] = in_width(p, l) + H;
    }
    LL_HIP(ll::launch_fwd_setup<T>(seq_len, B, d.T_max, p->perm, p->active, p->off, p->rowmap, p->meta,
                                   trip, L, Wl, R, p->G * H, WTl, s));
  }
  tend(p, s, LL_STAGE_PREP, ev);
  p->rows_prepared = false;
  p->bwd_prepared = false;
  if (p->wave) return enqueue_fwd_wave<T>(p, s, x, W, bias, h0, c0, y, hT, cT, save);
  p->rows_prepared = save;   // (the input projections below carry them)
  p->bwd_prepared = save && p->xmode && p->G == 4;
  for (int l = 0; l < L; ++l) {
    const int Il = in_width(p, l);
    ev = tbeg(p, s, LL_STAGE_INPUT_PROJ);
    // Zx = x_t W_x + b for every compact row (layer 0 gathers time-major x)
    ll::GemmArgs g{};
    g.A = l == 0 ? x : p->HH[0];
    g.lda = Il;
    g.a_rowmap = l == 0 ? p->rowmap : nullptr;
    g.Bm = p->WT[l];
    g.ldb = Il + H;
    g.C = p->Zx;
    g.ldc = (long)p->G * H;
    g.bias = bias[l];
    g.M = (int)p->cap;
    g.M_dev = p->meta + 1;
    g.N = p->G * H;
    g.K = Il;
    g.splits = 1;
    // the XCD-local loop's entering state (ring slot 1, read at step 0) and
    // flags, and for a gradient pass with dW over rows the h_{t-1} row map
    // and this layer's h0 rows, prepared in work-groups of this launch beside
    // the product's (they depend only on prep and h0)
    if (p->xmode) {
      g.pre_blocks = 16;
      g.pre.xp = ll::XPrepArgs{h0 ? h0 + (long)l * B * H : nullptr, p->perm, B, H, p->xMRT,
                               (int)((long)H * p->es / 64), 1, p->xring, p->xflags, p->xflag_words};
    }
    // (and for the gradient pass: W_h in unit-major order, its flags)
    if (save && p->xmode && p->G == 4) {
      g.pre_blocks = 32;
      g.pre.pw = W[l];
      g.pre.prow0 = Il;
      g.pre.pH = H;
      g.pre.pdst = p->Wum[l];
      if (p->xflags_b) {
        g.pre.zero = p->xflags_b;
        g.pre.nzero = p->xflag_words;
      }
    }
    if (save && p->dw_rows[l]) {
      g.pre_blocks = std::max(g.pre_blocks, 16);
      g.pre.active = p->active;
      g.pre.off = p->off;
      g.pre.B = B;
      g.pre.T_max = d.T_max;
      g.pre.cap = p->cap;
      g.pre.prev = p->prevc;
      g.pre.h0 = h0 ? h0 + (long)l * B * H : nullptr;
      g.pre.perm = p->perm;
      g.pre.H = H;
      g.pre.h0dst = reinterpret_cast<T*>(p->HH[l]) + p->cap * H;
    }
    LL_HIP(ll::launch_gemm_nt<T>(g, s));
    // cond body: the input part of the predicate, x_t . w_px per compact row
    if (p->skip)
      LL_HIP(ll::launch_row_dot<T>(static_cast<const T*>(g.A), Il, g.a_rowmap, p->meta, p->cap, bias[l] + 4L * H,
                                   Il, p->sx, s));
    tend(p, s, LL_STAGE_INPUT_PROJ, ev);
    if (p->xmode) {
      const int ring_ks = (int)((long)H * p->es / 64);
      ll::XLoopArgs xa = x_common(p);
      if (p->recompute) {   // push c_t only; keep the bias for the gate recomputation
        xa.sld = H;
        xa.scoff = 0;
        xa.sgates = 0;
        if (save)
          LL_HIP(hipMemcpyAsync(p->rc_bias + (long)l * 4 * H, bias[l], sizeof(float) * 4 * H,
                                hipMemcpyDeviceToDevice, s));
      }
      xa.ring = p->xring;
      xa.ring_ks = ring_ks;
      xa.rank_ctr = p->xflags;
      xa.flags = p->xflags + 8;
      xa.B = B;
      xa.H = H;
      xa.T_max = d.T_max;
      xa.P = p->xP;
      xa.MRT = p->xMRT;
      xa.meta = p->meta;
      xa.active = p->active;
      xa.off = p->off;
      xa.perm = p->perm;
      xa.W = p->WT[l];
      xa.ldw = Il + H;
      xa.woff = Il;
      xa.X = p->HH[l];
      xa.Zx = p->Zx;
      xa.bhn = p->G == 3 ? bias[l] + 3L * H : nullptr;
      if (p->skip) {   // bias[l] = [b (4H), w_px (I_l), w_ph (H), b_p]
        xa.wp = bias[l] + 4L * H + Il;
        xa.bp = bias[l] + 4L * H + Il + H;
        xa.sx = p->sx;
        xa.guard = p->guards ? p->guards + (long)l * p->cap : nullptr;
      }
      if (p->act) {    // bias = [b (4H), w_p (H), b_p]
        xa.wp = bias[l] + 4L * H;
        xa.bp = bias[l] + 5L * H;
        xa.guard = p->guards;
        xa.ponder_max = p->M;
        xa.slot_rows = p->cap;
        xa.ntrip = p->ntrip;
        xa.HI = p->HI;
      }
      xa.stack = save ? p->stack[l] : nullptr;
      xa.y = (l == L - 1) ? y : nullptr;
      xa.abort_flag = p->meta + 3;
      xa.err = p->meta + 2;
      xa.limit = p->barrier_ticks;
      const float* hin = h0 ? h0 + (long)l * B * H : nullptr;
      // (the RNN and GRU have no cell state: c0 is ignored, cT written as
      // zeros if given)
      const float* cin = c0 && p->G == 4 ? c0 + (long)l * B * H : nullptr;
      float* hout = hT + (long)l * B * H;
      float* cout = cT ? cT + (long)l * B * H : nullptr;
      // one launch per chunk of steps when the stack spills, else one launch
      const int C = p->spill ? p->chunk_steps : d.T_max;
      const int nch = p->spill ? p->nchunks : 1;
      xa.chunk_steps = C;
      xa.nslots = p->spill ? p->nslots : 1;
      for (int k = 0; k < nch; ++k) {
        const int t0 = k * C, t1 = std::min(d.T_max, t0 + C);
        const int slot = k % xa.nslots;
        const bool last = k == nch - 1;
        // (the first launch's entering state: prepared by the input projection's launch)
        if (k > 0) {
          ev = tbeg(p, s, LL_STAGE_LOOP_SETUP);
          // the chunk that used this ring slot before has reached host memory
          if (p->spill && save && k >= p->nslots)
            LL_HIP(hipStreamWaitEvent(s, p->ev_d2h[l * p->nslots + slot], 0));
          LL_HIP(ll::launch_x_prepare_fwd<T>(hin, p->perm, B, H, p->xMRT, ring_ks, (t0 + 1) & 1, p->xring,
                                             p->xflags, p->xflag_words, s));
          tend(p, s, LL_STAGE_LOOP_SETUP, ev);
        }
        ev = tbeg(p, s, LL_STAGE_FWD_LOOP);
        xa.t_begin = t0;
        xa.t_end = t1;
        xa.h0 = hin;
        xa.c0 = cin;
        xa.hT = last ? hout : p->carry;
        xa.cT = last ? cout : p->carry + (long)B * H;
        LL_HIP(chained_loop_launch(p->device, s, [&] { return ll::x_launch(p->xk.fwd, xa, 256, p->xk.lds_fwd, s); }));
        tend(p, s, LL_STAGE_FWD_LOOP, ev);
        if (p->spill && save && k < nch - p->nslots) {   // evicted later: swap it out on the copy stream
          LL_HIP(hipEventRecord(p->ev_compute, s));
          // (two copy streams: the next chunk's copy is queued while this one runs)
          hipStream_t cs = (k & 1) ? p->cstream2 : p->cstream;
          LL_HIP(hipStreamWaitEvent(cs, p->ev_compute, 0));
          LL_HIP(copy_on_dma_engine(p->host_stack[l] + (long)k * p->slot_floats,
                                    p->stack[l] + (long)slot * p->slot_floats, sizeof(float) * p->slot_floats,
                                    hipMemcpyDeviceToHost, cs));
          LL_HIP(hipEventRecord(p->ev_d2h[l * p->nslots + slot], cs));
        }
        hin = p->carry;
        cin = p->carry + (long)B * H;
      }
      continue;
    }
    if (p->cmode) {
      const float* hin = h0 ? h0 + (long)l * B * H : nullptr;
      ev = tbeg(p, s, LL_STAGE_LOOP_SETUP);
      LL_HIP(ll::launch_c_prepare<T>(hin, p->perm, B, H, p->cMRT, p->cring, p->cflags, p->cflag_words, s));
      tend(p, s, LL_STAGE_LOOP_SETUP, ev);
      ll::CLoopArgs ca = c_common(p);
      ca.W = p->WT[l];
      ca.ldw = Il + H;
      ca.woff = Il;
      ca.X = p->HH[l];
      ca.ring_ks = (int)((long)H * p->es / 64);
      ca.Zx = p->Zx;
      ca.h0 = hin;
      ca.c0 = c0 ? c0 + (long)l * B * H : nullptr;
      ca.stack = save ? p->stack[l] : nullptr;
      ca.y = (l == L - 1) ? y : nullptr;
      ca.hT = hT + (long)l * B * H;
      ca.cT = cT + (long)l * B * H;
      ev = tbeg(p, s, LL_STAGE_FWD_LOOP);
      LL_HIP(chained_loop_launch(p->device, s, [&] { return ll::c_launch(p->ck.fwd, ca, p->ck.lds_fwd, s); }));
      tend(p, s, LL_STAGE_FWD_LOOP, ev);
      continue;
    }
    ll::FwdLoopArgs a{};
    a.B = B;
    a.H = H;
    a.T_max = d.T_max;
    a.HJ = p->geom.HJ;
    a.RG = p->geom.RG;
    a.MRT = p->geom.MRT;
    a.meta = p->meta;
    a.active = p->active;
    a.off = p->off;
    a.perm = p->perm;
    a.Zx = p->Zx;
    a.WT = p->WT[l];
    a.ldw = Il + H;
    a.woff = Il;
    a.h0 = h0 ? h0 + (long)l * B * H : nullptr;
    a.c0 = c0 ? c0 + (long)l * B * H : nullptr;
    a.HH = p->HH[l];
    a.stack = save ? p->stack[l] : nullptr;
    a.y = (l == L - 1) ? y : nullptr;
    a.hT = hT + (long)l * B * H;
    a.cT = cT + (long)l * B * H;
    a.bar = reinterpret_cast<unsigned*>(p->meta + 4 + l);   // one counter per launch
    a.abort_flag = p->meta + 3;
    a.err = p->meta + 2;
    a.limit = p->barrier_ticks;
    ev = tbeg(p, s, LL_STAGE_FWD_LOOP);
    LL_HIP(chained_loop_launch(p->device, s, [&] { return ll::launch_fwd_loop<T>(a, p->geom.nwg, p->geom.lds_fwd, s); }));
    tend(p, s, LL_STAGE_FWD_LOOP, ev);
  }
  return LL_OK;
}

// Products after the gradient loop of layer l: db from the loop's row-group
// partials, dW = [x_t, h_{t-1}]^T dz_t summed over steps, and, if dx is not
// NULL, dx_t = dz_t W_x^T (layer 0: time-major [T_max, B, I]; layer 1:
// compact rows, the gradient of the layer below).  dz: [cap, 4H] compact rows.
template <typename T>
ll_status bwd_products(ll_plan* p, hipStream_t s, int l, const void* dz, const float* db_part,
                       float* dx, float* const* dW, float* const* dbias) {
  const ll_desc& d = p->d;
  const int H = d.H, B = d.B;
  const int Il = in_width(p, l);
  hipEvent_t ev = nullptr;
  // dx_t = dz_t W_x^T: scattered to time-major dx (layer 0) or kept compact
  // as the gradient of the layer below (layer 1).  A product whose grid fills
  // the chip at most a few times runs on the side stream beside the dW
  // products (both only read dz) and is joined back before returning; a
  // larger one runs after them on the call's stream (measured: two large
  // products side by side only slow each other).
  ll::GemmArgs gx{};
  const int GH = p->G * H;     // gate columns of W
  const int GBH = p->GB * H;   // dz row width, bias length
  gx.A = dz;
  gx.lda = GBH;
  gx.Bm = p->W[l];
  gx.ldb = GH;
  gx.M = (int)p->cap;
  gx.M_dev = p->meta + 1;
  gx.N = Il;
  gx.K = GH;
  gx.splits = 1;
  gx.C = dx;
  if (l == 0) {
    gx.ldc = d.I;
    gx.c_rowmap = p->rowmap;
  } else {
    gx.ldc = H;
  }
  // db = the sum of the gradient loop's row-group partials, carried by the
  // dx product's launch when there is one
  const int db_slices = p->xmode ? 8 : p->cmode ? 1 : p->geom.RG;
  const bool db_in_dx = dx != nullptr;
  if (db_in_dx) {
    gx.pre_blocks = 4;
    gx.pre.ws = db_part;
    gx.pre.S = db_slices;
    gx.pre.stride = GBH;
    gx.pre.n = GBH;
    gx.pre.cols = GBH;
    gx.pre.ldo = GBH;
    gx.pre.sum_out = dbias[l];
  }
  auto dx_product = [&](hipStream_t st) -> ll_status {
    hipEvent_t evx = tbeg(p, st, LL_STAGE_DX);
    LL_HIP(ll::launch_gemm_nt<T>(gx, st));
    tend(p, st, LL_STAGE_DX, evx);
    return LL_OK;
  };
  // (the grid covers the row capacity T_max * B; groups past the running
  // rows return at once)
  const bool side = dx && ll::gemm_rounds(gx, (int)sizeof(T), p->n_cu) <= 2;
  if (side) {
    LL_HIP(hipEventRecord(p->ev_fork, s));
    LL_HIP(hipStreamWaitEvent(p->gstream, p->ev_fork, 0));
    LL_STATUS(dx_product(p->gstream));
    LL_HIP(hipEventRecord(p->ev_join, p->gstream));
  }
  // one launch: db = sum of the row-group partials; (cond body) no gradient
  // for the predicate's parameters (a step function); for dW straight from
  // the row-major operands, the h history row of every compact row's
  // h_{t-1}, and h0 (length order) after the history
  ev = tbeg(p, s, LL_STAGE_BWD_OPERANDS);
  {
    ll::SmallBatch<T> ops;
    if (!db_in_dx)
      LL_HIP(ops.sum_slices(db_part, db_slices, GBH, 1, GBH, dbias[l], GBH));
    if (p->skip) LL_HIP(ops.zero_u32(reinterpret_cast<unsigned*>(dbias[l] + GBH), Il + H + 1));
    if (p->dw_rows[l] && !p->rows_prepared) {
      LL_HIP(ops.prev_rows(p->active, p->off, B, d.T_max, p->cap, p->prevc));
      LL_HIP(ops.h0_rows(p->h0 ? p->h0 + (long)l * B * H : nullptr, p->perm, B, H,
                         reinterpret_cast<T*>(p->HH[l]) + p->cap * H));
    }
    LL_HIP(ops.launch(s));   // (nothing left: no launch)
  }
  tend(p, s, LL_STAGE_BWD_OPERANDS, ev);
  if (p->dw_rows[l]) {
    ev = tbeg(p, s, LL_STAGE_DW);
    DwPart parts[3];
    const int np = dw_parts_rows(p, l, parts);
    for (int k = 0; k < np; ++k) {
      const DwPart& q = parts[k];
      const bool in_part = q.a_row == 0;
      ll::GemmTnArgs g{};
      if (in_part) {
        g.A = l == 0 ? p->x : p->HH[0];
        g.a_rowmap = l == 0 ? p->rowmap : nullptr;
        g.a_rows = (int)p->cap;
        if (q.m > Il) {   // both parts in one launch
          g.A2 = p->HH[l];
          g.lda2 = H;
          g.a2_rowmap = p->prevc;
          g.a2_rows = (int)(p->cap + B);
          g.M1 = Il;
        }
      } else {
        g.A = p->HH[l];
        g.a_rowmap = p->prevc;
        g.a_rows = (int)(p->cap + B);
      }
      g.lda = in_part ? Il : H;
      g.Bm = static_cast<const T*>(dz) + q.b_row;
      g.ldb = GBH;
      g.b_rows = (int)p->cap;
      g.M = q.m;
      g.N = q.n;
      g.K = (int)p->cap;
      g.K_dev = p->meta + 1;
      g.splits = p->tn_splits[l][k];
      // (the plan chose this path only for operands below 2^31 bytes, and
      // lstm_loop_fwd accepted only a 16-byte aligned x)
      if (!ll::gemm_tn_applies(g))
        return fail(LL_EHIP, "internal: the dW product over rows does not apply to layer %d", l);
      float* out = dW[l] + (long)q.a_row * GH + q.c_col;
      if (g.splits == 2 && p->tn_flags) {   // the two splits sum in place
        g.C = p->ws;
        g.ldc = q.n;
        g.split_stride = (long)q.m * q.n;
        g.tile_flags = p->tn_flags;
        g.out = out;
        g.ldo = GH;
        LL_HIP(ll::launch_gemm_tn(g, s));
      } else if (g.splits > 1) {
        g.C = p->ws;
        g.ldc = q.n;
        g.split_stride = (long)q.m * q.n;
        LL_HIP(ll::launch_gemm_tn(g, s));
        LL_HIP(ll::launch_sum_slices_2d(p->ws, g.splits, g.split_stride, q.m, q.n, out, GH, s));
      } else {
        g.C = out;
        g.ldc = GH;
        LL_HIP(ll::launch_gemm_tn(g, s));
      }
    }
  } else {
    ev = tbeg(p, s, LL_STAGE_BWD_OPERANDS);
    // transposed operands of the dW products (reduction over compact rows)
    ll::GatherTArgs gt{};
    gt.B = B;
    gt.meta = p->meta;
    gt.rowmap = p->rowmap;
    gt.off = p->off;
    gt.perm = p->perm;
    gt.ldo = (int)p->ldT;
    gt.in = dz;
    gt.out = p->DZT;
    gt.C = GBH;
    gt.mode = 1;
    LL_HIP(ll::launch_gather_transpose<T>(gt, (int)p->cap, s));
    gt.in = l == 0 ? p->x : p->HH[0];
    gt.out = p->XT;
    gt.C = Il;
    gt.mode = l == 0 ? 0 : 1;
    LL_HIP(ll::launch_gather_transpose<T>(gt, (int)p->cap, s));
    gt.in = p->HH[l];
    gt.out = static_cast<char*>(p->XT) + p->es * Il * p->ldT;
    gt.C = H;
    gt.mode = 2;
    gt.h0f = p->h0 ? p->h0 + (long)l * B * H : nullptr;
    LL_HIP(ll::launch_gather_transpose<T>(gt, (int)p->cap, s));
    tend(p, s, LL_STAGE_BWD_OPERANDS, ev);
    // dW = [X^T; Hprev^T] DZ (the parts of dw_parts)
    ev = tbeg(p, s, LL_STAGE_DW);
    {
      DwPart parts[3];
      const int np = dw_parts(p, l, parts);
      const long rowb = p->es * p->ldT;   // bytes per transposed row
      for (int k = 0; k < np; ++k) {
        const DwPart& q = parts[k];
        float* out = dW[l] + (long)q.a_row * GH + q.c_col;
        ll::GemmArgs g{};
        g.A = static_cast<const char*>(p->XT) + q.a_row * rowb;
        g.lda = p->ldT;
        g.Bm = static_cast<const char*>(p->DZT) + q.b_row * rowb;
        g.ldb = p->ldT;
        g.M = q.m;
        g.N = q.n;
        g.K = (int)p->cap;
        g.K_dev = p->meta + 1;
        g.k_zero_tail = 1;   // the transposes write zeros past the last row, up to a multiple of 64
        g.splits = p->dw_splits[l][k];
        if (g.splits > 1) {
          g.C = p->ws;
          g.ldc = q.n;
          g.split_stride = (long)q.m * q.n;
          LL_HIP(ll::launch_gemm_nt<T>(g, s));
          LL_HIP(ll::launch_sum_slices_2d(p->ws, g.splits, g.split_stride, q.m, q.n, out, GH, s));
        } else {
          g.C = out;
          g.ldc = GH;
          LL_HIP(ll::launch_gemm_nt<T>(g, s));
        }
      }
    }
  }
  tend(p, s, LL_STAGE_DW, ev);
  if (side) LL_HIP(hipStreamWaitEvent(s, p->ev_join, 0));
  else if (dx) LL_STATUS(dx_product(s));
  return LL_OK;
}

// Products after the gradient loop of the nested-loop body (one layer):
// dW = sum over ponder slots k of [x_t, h^k_prev]^T dz_k, where the h part of
// slot 0 is h_{t-1} (the h history's previous row, h0 after it) and that of
// slot k > 0 is h^k (HI slot k-1, the same compact row); db from the loop's
// partials, zero in the halting part; dx_t = sum_k dz_k W_x^T.  Every slot's
// product goes to the workspace and one sum follows (dz rows of slots a row
// tile did not run are zero).
template <typename T>
ll_status act_products(ll_plan* p, hipStream_t s, float* dx, float* const* dW, float* const* dbias) {
  const ll_desc& d = p->d;
  const int H = d.H, B = d.B, I = d.I, M = p->M;
  const long cap = p->cap;
  const int GH = 4 * H;
  const T* DZ = static_cast<const T*>(p->DZ);
  const T* HI = static_cast<const T*>(p->HI);
  // one launch: db, zero in the halting part, the dW operand maps
  hipEvent_t ev = tbeg(p, s, LL_STAGE_BWD_OPERANDS);
  {
    ll::SmallBatch<T> ops;
    LL_HIP(ops.sum_slices(p->db_part, 8, GH, 1, GH, dbias[0], GH));
    LL_HIP(ops.zero_u32(reinterpret_cast<unsigned*>(dbias[0] + GH), H + 1));
    if (p->dw_rows[0]) {
      LL_HIP(ops.prev_rows(p->active, p->off, B, d.T_max, cap, p->prevc));
      LL_HIP(ops.h0_rows(p->h0, p->perm, B, H, reinterpret_cast<T*>(p->HH[0]) + cap * H));
    }
    LL_HIP(ops.launch(s));
  }
  tend(p, s, LL_STAGE_BWD_OPERANDS, ev);
  if (p->dw_rows[0]) {
    ev = tbeg(p, s, LL_STAGE_DW);
    DwPart parts[3];
    const int np = dw_parts_rows(p, 0, parts);
    for (int q = 0; q < np; ++q) {
      const DwPart& pt = parts[q];
      const bool in_part = pt.a_row == 0;
      const int sp = p->tn_splits[0][q];
      for (int k = 0; k < M; ++k) {
        // the h rows of slot k: h_{t-1} through the previous-row map, or h^k
        const void* hsrc = k == 0 ? p->HH[0] : static_cast<const void*>(HI + (long)(k - 1) * cap * H);
        const int* hmap = k == 0 ? p->prevc : nullptr;
        const int hrows = k == 0 ? (int)(cap + B) : (int)cap;
        ll::GemmTnArgs g{};
        if (in_part) {
          g.A = p->x;
          g.a_rowmap = p->rowmap;
          g.a_rows = (int)cap;
          g.lda = I;
          if (pt.m > I) {
            g.A2 = hsrc;
            g.lda2 = H;
            g.a2_rowmap = hmap;
            g.a2_rows = hrows;
            g.M1 = I;
          }
        } else {
          g.A = hsrc;
          g.a_rowmap = hmap;
          g.a_rows = hrows;
          g.lda = H;
        }
        g.Bm = DZ + (long)k * cap * GH + pt.b_row;
        g.ldb = GH;
        g.b_rows = (int)cap;
        g.M = pt.m;
        g.N = pt.n;
        g.K = (int)cap;
        g.K_dev = p->meta + 1;
        g.splits = sp;
        g.C = p->ws + (long)k * sp * pt.m * pt.n;
        g.ldc = pt.n;
        g.split_stride = (long)pt.m * pt.n;
        if (!ll::gemm_tn_applies(g))
          return fail(LL_EHIP, "internal: the dW product over rows does not apply (ponder slot %d)", k);
        LL_HIP(ll::launch_gemm_tn(g, s));
      }
      LL_HIP(ll::launch_sum_slices_2d(p->ws, M * sp, (long)pt.m * pt.n, pt.m, pt.n,
                                      dW[0] + (long)pt.a_row * GH + pt.c_col, GH, s));
    }
    tend(p, s, LL_STAGE_DW, ev);
  } else {
    DwPart parts[3];
    const int np = dw_parts(p, 0, parts);
    const DwPart& pt = parts[0];   // (one product over the stacked [X^T; Hprev^T] for the LSTM)
    const int sp = p->dw_splits[0][0];
    const long rowb = p->es * p->ldT;
    (void)np;
    for (int k = 0; k < M; ++k) {
      ev = tbeg(p, s, LL_STAGE_BWD_OPERANDS);
      ll::GatherTArgs gt{};
      gt.B = B;
      gt.meta = p->meta;
      gt.rowmap = p->rowmap;
      gt.off = p->off;
      gt.perm = p->perm;
      gt.ldo = (int)p->ldT;
      gt.in = DZ + (long)k * cap * GH;
      gt.out = p->DZT;
      gt.C = GH;
      gt.mode = 1;
      LL_HIP(ll::launch_gather_transpose<T>(gt, (int)cap, s));
      if (k == 0) {   // x rows: the same for every slot
        gt.in = p->x;
        gt.out = p->XT;
        gt.C = I;
        gt.mode = 0;
        LL_HIP(ll::launch_gather_transpose<T>(gt, (int)cap, s));
      }
      gt.out = static_cast<char*>(p->XT) + p->es * I * p->ldT;
      gt.C = H;
      if (k == 0) {
        gt.in = p->HH[0];
        gt.mode = 2;
        gt.h0f = p->h0;
      } else {
        gt.in = HI + (long)(k - 1) * cap * H;
        gt.mode = 1;
        gt.h0f = nullptr;
      }
      LL_HIP(ll::launch_gather_transpose<T>(gt, (int)cap, s));
      tend(p, s, LL_STAGE_BWD_OPERANDS, ev);
      ev = tbeg(p, s, LL_STAGE_DW);
      ll::GemmArgs g{};
      g.A = p->XT;
      g.lda = p->ldT;
      g.Bm = static_cast<const char*>(p->DZT) + pt.b_row * rowb;
      g.ldb = p->ldT;
      g.M = pt.m;
      g.N = pt.n;
      g.K = (int)cap;
      g.K_dev = p->meta + 1;
      g.k_zero_tail = 1;
      g.splits = sp;
      g.C = p->ws + (long)k * sp * pt.m * pt.n;
      g.ldc = pt.n;
      g.split_stride = (long)pt.m * pt.n;
      LL_HIP(ll::launch_gemm_nt<T>(g, s));
      tend(p, s, LL_STAGE_DW, ev);
    }
    ev = tbeg(p, s, LL_STAGE_DW);
    LL_HIP(ll::launch_sum_slices_2d(p->ws, M * sp, (long)pt.m * pt.n, pt.m, pt.n, dW[0], GH, s));
    tend(p, s, LL_STAGE_DW, ev);
  }
  if (!dx) return LL_OK;
  // dx: one product per slot into compact rows of the workspace, then the
  // sum over slots scattered to time-major rows
  ev = tbeg(p, s, LL_STAGE_DX);
  for (int k = 0; k < M; ++k) {
    ll::GemmArgs gx{};
    gx.A = DZ + (long)k * cap * GH;
    gx.lda = GH;
    gx.Bm = p->W[0];
    gx.ldb = GH;
    gx.M = (int)cap;
    gx.M_dev = p->meta + 1;
    gx.N = I;
    gx.K = GH;
    gx.splits = 1;
    gx.C = p->ws + (long)k * cap * I;
    gx.ldc = I;
    LL_HIP(ll::launch_gemm_nt<T>(gx, s));
  }
  LL_HIP(ll::launch_sum_scatter_rows(p->ws, M, cap * I, p->meta, p->rowmap, I, dx, cap, s));
  tend(p, s, LL_STAGE_DX, ev);
  return LL_OK;
}

// Two-layer wavefront, gradient: one launch in which the upper layer's step t
// runs beside the lower layer's step t+1 on every XCD; the upper layer hands
// dy of the lower layer's output over per step (dz W_x^T of its own units),
// so no dx product of layer 1 is needed.  Then the dW and db products of both
// layers and dx of layer 0.
template <typename T>
ll_status enqueue_bwd_wave(ll_plan* p, hipStream_t s, const float* dy, const float* dhT,
                           const float* dcT, float* dx, float* const* dW, float* const* dbias,
                           float* dh0, float* dc0) {
  const ll_desc& d = p->d;
  const int H = d.H, B = d.B;
  const long BH = (long)B * H;
  const long fw = 8L * p->xMRT * 32;
  unsigned* F0 = p->xflags + 8;
  unsigned* F1 = F0 + fw;
  unsigned* FY = F1 + fw;
  // one launch: the dx rows of finished steps to zero, the flags
  hipEvent_t ev = tbeg(p, s, LL_STAGE_LOOP_SETUP);
  {
    ll::SmallBatch<T> setup;
    if (dx) LL_HIP(setup.zero_finished_rows(dx, d.T_max, B, d.I, p->seq_len, p->meta));
    LL_HIP(setup.zero_u32(p->xflags, p->xflag_words));
    LL_HIP(setup.launch(s));
  }
  tend(p, s, LL_STAGE_LOOP_SETUP, ev);
  const int ring_ks = (int)(4L * H * p->es / 64);
  ll::XLoopArgs a0 = x_common(p), a1 = x_common(p);
  a0.ring = p->xring;
  a0.ring_ks = ring_ks;
  a0.flags = F0;
  a0.W = p->W[0];
  a0.woff = d.I;
  a0.X = p->DZ;
  a0.c0 = p->c0;
  a0.stack = p->stack[0];
  a0.dhT = dhT;
  a0.dcT = dcT;
  a0.db_part = p->db_part;
  a0.dh0 = dh0;
  a0.dc0 = dc0;
  a0.dyx_ring = p->dyx;
  a0.dyx_flags = FY;

  a1.ring = p->xring2;
  a1.ring_ks = ring_ks;
  a1.flags = F1;
  a1.W = p->W[1];
  a1.woff = H;
  a1.Wx = p->W[1];
  a1.X = p->DZ2;
  a1.c0 = p->c0 ? p->c0 + BH : nullptr;
  a1.stack = p->stack[1];
  a1.dy = dy;
  a1.dy_compact = 0;
  a1.dhT = dhT ? dhT + BH : nullptr;
  a1.dcT = dcT ? dcT + BH : nullptr;
  a1.db_part = p->db_part2;
  a1.dh0 = dh0 ? dh0 + BH : nullptr;
  a1.dc0 = dc0 ? dc0 + BH : nullptr;
  a1.dyx_ring = p->dyx;
  a1.dyx_flags = FY;
  a1.peer_flags = F0;
  ev = tbeg(p, s, LL_STAGE_BWD_LOOP);
  LL_HIP(chained_loop_launch(p->device, s, [&] { return ll::x_launch2(p->xk2.bwd, a0, a1, 256, p->xk2.lds_bwd, s); }));
  tend(p, s, LL_STAGE_BWD_LOOP, ev);
  LL_STATUS(bwd_products<T>(p, s, 1, p->DZ2, p->db_part2, nullptr, dW, dbias));
  return bwd_products<T>(p, s, 0, p->DZ, p->db_part, dx, dW, dbias);
}

// Gate recomputation (recompute = 1): row maps over padded rows (t, r) and
// the h0 rows after every layer's h history, once per gradient pass.
template <typename T>
ll_status recompute_setup(ll_plan* p, hipStream_t s) {
  const ll_desc& d = p->d;
  const int H = d.H, B = d.B;
  hipEvent_t ev = tbeg(p, s, LL_STAGE_LOOP_SETUP);
  LL_HIP(ll::launch_rc_maps(p->active, p->off, p->perm, B, d.T_max, p->cap, p->rc_inmap,
                            p->rc_inmap + p->cap, p->rc_prevmap, s));
  for (int l = 0; l < d.layers; ++l)
    LL_HIP(ll::launch_h0_rows<T>(p->h0 ? p->h0 + (long)l * B * H : nullptr, p->perm, B, H,
                                 reinterpret_cast<T*>(p->HH[l]) + p->cap * H, s));
  tend(p, s, LL_STAGE_LOOP_SETUP, ev);
  return LL_OK;
}

// i, f, g, o of steps [t0, t1) of layer l into gslot (row (t - t0) B + r):
// z = x_t W_x + b (the top layer reuses its input projection, still in Zx),
// then act(z + h_{t-1} W_h) in the second product's epilogue.
template <typename T>
ll_status recompute_gates(ll_plan* p, hipStream_t s, int l, int t0, int t1) {
  const ll_desc& d = p->d;
  const int H = d.H, B = d.B, Il = in_width(p, l);
  const long M = (long)(t1 - t0) * B;
  const int* xmap = p->rc_inmap;
  const int* cmap = p->rc_inmap + p->cap;
  hipEvent_t ev = tbeg(p, s, LL_STAGE_RECOMPUTE);
  const bool zx_live = l == d.layers - 1;   // Zx holds this layer's projections
  if (!zx_live) {
    ll::GemmArgs g{};
    g.A = l == 0 ? p->x : p->HH[0];
    g.lda = Il;
    g.a_rowmap = (l == 0 ? xmap : cmap) + (long)t0 * B;
    g.a_rows = (int)p->cap;
    g.Bm = p->WT[l];
    g.ldb = Il + H;
    g.K = Il;
    g.N = 4 * H;
    g.M = (int)M;
    g.bias = p->rc_bias + (long)l * 4 * H;
    g.C = p->gslot;
    g.ldc = 4L * H;
    g.splits = 1;
    LL_HIP(ll::launch_gemm_nt<T>(g, s));
  }
  ll::GemmArgs h{};
  h.A = p->HH[l];
  h.lda = H;
  h.a_rowmap = p->rc_prevmap + (long)t0 * B;
  h.a_rows = (int)(p->cap + B);
  h.Bm = reinterpret_cast<const T*>(p->WT[l]) + Il;
  h.ldb = Il + H;
  h.K = H;
  h.N = 4 * H;
  h.M = (int)M;
  h.C = p->gslot;
  h.ldc = 4L * H;
  h.splits = 1;
  h.act_h = H;
  if (zx_live) {
    h.addend = p->Zx;
    h.add_rowmap = cmap + (long)t0 * B;
    h.ld_add = 4L * H;
  }
  LL_HIP(ll::launch_gemm_nt<T>(h, s));
  tend(p, s, LL_STAGE_RECOMPUTE, ev);
  return LL_OK;
}

template <typename T>
ll_status enqueue_bwd(ll_plan* p, hipStream_t s, const float* dy, const float* dhT,
                      const float* dcT, float* dx, float* const* dW, float* const* dbias,
                      float* dh0, float* dc0) {
  const ll_desc& d = p->d;
  const int H = d.H, B = d.B, L = d.layers;
  hipEvent_t ev = nullptr;
  if (p->wave) return enqueue_bwd_wave<T>(p, s, dy, dhT, dcT, dx, dW, dbias, dh0, dc0);
  // the set-up before each loop launch, in one launch: the dx rows of
  // finished steps to zero (once; the XCD-local gradient loop of layer 0
  // zeroes them itself), W_h in unit-major order, the flags
  ll::SmallBatch<T> setup;
  if (dx && !p->xmode) LL_HIP(setup.zero_finished_rows(dx, d.T_max, B, d.I, p->seq_len, p->meta));
  for (int l = L - 1; l >= 0; --l) {
    const int Il = in_width(p, l);
    if (p->xmode) {
      ll::XLoopArgs xa = x_common(p);
      xa.ring = p->xring;
      xa.ring_ks = (int)((long)p->G * H * p->es / 64);
      // flags cleared by the saved forward's input projection, or here
      unsigned* fl = p->bwd_prepared && p->xflags_b ? p->xflags_b : p->xflags;
      xa.rank_ctr = fl;
      xa.flags = fl + 8;
      xa.B = B;
      xa.H = H;
      xa.T_max = d.T_max;
      xa.P = p->xP;
      xa.MRT = p->xMRT;
      xa.meta = p->meta;
      xa.active = p->active;
      xa.off = p->off;
      xa.perm = p->perm;
      xa.W = p->W[l];
      xa.woff = Il;
      if (p->G == 4) {   // the LSTM loop reduces in unit-major order (permuted by the forward)
        if (!p->bwd_prepared)
          LL_HIP(setup.permute_um(static_cast<const T*>(p->W[l]), Il, H, static_cast<T*>(p->Wum[l])));
        xa.W = p->Wum[l];
        xa.woff = 0;
      }
      xa.X = p->DZ;
      if (l == 0 && dx) {   // dx at finished steps, zeroed by XCDs 1 .. 7 after their last step
        xa.dx_zero = dx;
        xa.seq_len = p->seq_len;
        xa.I = d.I;
      }
      xa.c0 = p->c0 && p->G == 4 ? p->c0 + (long)l * B * H : nullptr;
      xa.stack = p->stack[l];
      xa.guard = p->skip ? p->guards + (long)l * p->cap : p->act ? p->guards : nullptr;
      if (p->act) {
        xa.ponder_max = p->M;
        xa.slot_rows = p->cap;
        xa.ntrip = p->ntrip;
      }
      if (l == L - 1) {
        xa.dy = dy;
        xa.dy_compact = 0;
      } else {
        xa.dy = p->dyc;
        xa.dy_compact = 1;
      }
      xa.db_part = p->db_part;
      xa.abort_flag = p->meta + 3;
      xa.err = p->meta + 2;
      xa.limit = p->barrier_ticks;
      const float* dhin = dhT ? dhT + (long)l * B * H : nullptr;
      const float* dcin = dcT && p->G == 4 ? dcT + (long)l * B * H : nullptr;
      float* dhout = dh0 ? dh0 + (long)l * B * H : nullptr;
      float* dcout = dc0 ? dc0 + (long)l * B * H : nullptr;
      const int C = p->spill ? p->chunk_steps : p->recompute ? p->rc_steps : d.T_max;
      const int nch = p->spill ? p->nchunks : p->recompute ? p->rc_chunks : 1;
      const int R = p->spill ? p->nslots : 1;
      xa.chunk_steps = p->spill ? C : d.T_max;
      xa.nslots = R;
      xa.db_state = (p->spill || p->recompute) ? p->db_state : nullptr;
      if (p->recompute) {   // c_t from the c-only stack, the gates from the chunk buffer
        xa.sld = H;
        xa.scoff = 0;
        xa.gstk = p->gslot;
        xa.gld = 4 * H;
        xa.gchunk = C;
        xa.gslots = 1;
        if (l == L - 1) LL_STATUS(recompute_setup<T>(p, s));
      }
      // chunks at or above nch - R are still in the ring after the forward; a
      // chunk j below is swapped in after the launch of chunk j + R (the last
      // use of its slot) and waited for before the launches of j + 1 (which
      // reads c_{t-1} from it) and j
      auto wait_loaded = [&](int j) -> hipError_t {
        if (!p->spill || j < 0 || j >= nch - R) return hipSuccess;
        return hipStreamWaitEvent(s, p->ev_h2d[l * R + j % R], 0);
      };
      for (int k = nch - 1; k >= 0; --k) {
        const int t0 = k * C, t1 = std::min(d.T_max, t0 + C);
        const bool first = k == nch - 1, last = k == 0;
        ev = tbeg(p, s, LL_STAGE_LOOP_SETUP);
        LL_HIP(wait_loaded(k));
        LL_HIP(wait_loaded(k - 1));
        if (fl == p->xflags) LL_HIP(setup.zero_u32(p->xflags, p->xflag_words));
        LL_HIP(setup.launch(s));   // (nothing left: no launch)
        tend(p, s, LL_STAGE_LOOP_SETUP, ev);
        if (p->recompute) LL_STATUS(recompute_gates<T>(p, s, l, t0, t1));
        ev = tbeg(p, s, LL_STAGE_BWD_LOOP);
        xa.t_begin = t0;
        xa.t_end = t1;
        xa.db_resume = first ? 0 : 1;
        xa.dhT = first ? dhin : p->carry + 2L * B * H;
        xa.dcT = first ? dcin : p->carry + 3L * B * H;
        xa.dh0 = last ? dhout : p->carry + 2L * B * H;
        xa.dc0 = last ? dcout : p->carry + 3L * B * H;
        LL_HIP(chained_loop_launch(p->device, s, [&] { return ll::x_launch(p->xk.bwd, xa, 256, p->xk.lds_bwd, s); }));
        tend(p, s, LL_STAGE_BWD_LOOP, ev);
        const int j = k - R;   // swap chunk j into the slot chunk k leaves
        if (p->spill && j >= 0) {
          LL_HIP(hipEventRecord(p->ev_compute, s));
          hipStream_t cs = (j & 1) ? p->cstream2 : p->cstream;
          LL_HIP(hipStreamWaitEvent(cs, p->ev_compute, 0));
          LL_HIP(copy_on_dma_engine(p->stack[l] + (long)(j % R) * p->slot_floats,
                                    p->host_stack[l] + (long)j * p->slot_floats, sizeof(float) * p->slot_floats,
                                    hipMemcpyHostToDevice, cs));
          LL_HIP(hipEventRecord(p->ev_h2d[l * R + j % R], cs));
        }
      }
    }
    if (p->cmode) {
      ev = tbeg(p, s, LL_STAGE_LOOP_SETUP);
      LL_HIP(setup.zero_u32(p->cflags, p->cflag_words));
      LL_HIP(setup.launch(s));
      tend(p, s, LL_STAGE_LOOP_SETUP, ev);
      ll::CLoopArgs ca = c_common(p);
      ca.W = p->W[l];
      ca.woff = Il;
      ca.X = p->DZ;
      ca.ring_ks = (int)(4L * H * p->es / 64);
      ca.c0 = p->c0 ? p->c0 + (long)l * B * H : nullptr;
      ca.stack = p->stack[l];
      ca.dy = l == L - 1 ? dy : p->dyc;
      ca.dy_compact = l == L - 1 ? 0 : 1;
      ca.dhT = dhT ? dhT + (long)l * B * H : nullptr;
      ca.dcT = dcT ? dcT + (long)l * B * H : nullptr;
      ca.db = p->db_part;
      ca.dh0 = dh0 ? dh0 + (long)l * B * H : nullptr;
      ca.dc0 = dc0 ? dc0 + (long)l * B * H : nullptr;
      ev = tbeg(p, s, LL_STAGE_BWD_LOOP);
      LL_HIP(chained_loop_launch(p->device, s, [&] { return ll::c_launch(p->ck.bwd, ca, p->ck.lds_bwd, s); }));
      tend(p, s, LL_STAGE_BWD_LOOP, ev);
    }
    ll::BwdLoopArgs a{};
    a.B = B;
    a.H = H;
    a.T_max = d.T_max;
    a.HJ = p->geom.HJ;
    a.RG = p->geom.RG;
    a.MRT = p->geom.MRT;
    a.meta = p->meta;
    a.active = p->active;
    a.off = p->off;
    a.perm = p->perm;
    a.W = p->W[l];
    a.wrow0 = Il;
    a.stack = p->stack[l];
    a.c0 = p->c0 ? p->c0 + (long)l * B * H : nullptr;
    if (l == L - 1) {
      a.dy = dy;
      a.dy_compact = 0;
    } else {
      a.dy = p->dyc;
      a.dy_compact = 1;
    }
    a.dhT = dhT ? dhT + (long)l * B * H : nullptr;
    a.dcT = dcT ? dcT + (long)l * B * H : nullptr;
    a.DZ = p->DZ;
    a.db_part = p->db_part;
    a.dh0 = dh0 ? dh0 + (long)l * B * H : nullptr;
    a.dc0 = dc0 ? dc0 + (long)l * B * H : nullptr;
    a.bar = reinterpret_cast<unsigned*>(p->meta + 6 + l);   // one counter per launch
    a.abort_flag = p->meta + 3;
    a.err = p->meta + 2;
    a.limit = p->barrier_ticks;
    if (!p->xmode && !p->cmode) {
      LL_HIP(setup.launch(s));
      ev = tbeg(p, s, LL_STAGE_BWD_LOOP);
      LL_HIP(chained_loop_launch(p->device, s, [&] { return ll::launch_bwd_loop<T>(a, p->geom.nwg, p->geom.lds_bwd, s); }));
      tend(p, s, LL_STAGE_BWD_LOOP, ev);
    }
    if (p->act) {
      LL_STATUS(act_products<T>(p, s, dx, dW, dbias));
      continue;
    }
    LL_STATUS(bwd_products<T>(p, s, l, p->DZ, p->db_part, l == 0 ? dx : p->dyc, dW, dbias));
  }
  return LL_OK;
}

}  // namespace

extern "C" {

ll_status lstm_loop_fwd(ll_plan* p, void* stream, const void* x, const int32_t* seq_len,
                        const void* const* W, const float* const* bias, const float* h0,
                        const float* c0, float* y, float* hT, float* cT, int32_t* trip_count,
                        int32_t save_for_backward) {
  if (!p) return fail(LL_EINVAL, "plan is NULL");
  if (!x || !seq_len || !W || !bias || !hT || (!cT && p->G == 4))
    return fail(LL_EINVAL, "x, seq_len, W, bias, hT and (LSTM) cT are required");
  for (int l = 0; l < p->d.layers; ++l)
    if (!W[l] || !bias[l]) return fail(LL_EINVAL, "W[%d] or bias[%d] is NULL", l, l);
  // the kernels read and write every array in 16-byte chunks
  {
    const void* ptrs[] = {x, seq_len, h0, c0, y, hT, cT, trip_count};
    const char* names[] = {"x", "seq_len", "h0", "c0", "y", "hT", "cT", "trip_count"};
    for (int i = 0; i < 8; ++i)
      if (reinterpret_cast<uintptr_t>(ptrs[i]) & 15)
        return fail(LL_EINVAL, "%s = %p is not 16-byte aligned", names[i], ptrs[i]);
    for (int l = 0; l < p->d.layers; ++l)
      if ((reinterpret_cast<uintptr_t>(W[l]) | reinterpret_cast<uintptr_t>(bias[l])) & 15)
        return fail(LL_EINVAL, "W[%d] = %p or bias[%d] = %p is not 16-byte aligned", l, W[l], l,
                    (const void*)bias[l]);
  }
  DeviceGuard guard(p->device);
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  p->state = ST_EMPTY;
  ll_status st = p->bf16 ? enqueue_fwd<bf16_t>(p, s, x, seq_len, W, bias, h0, c0, y, hT, cT,
                                               trip_count, save_for_backward != 0)
                         : enqueue_fwd<float>(p, s, x, seq_len, W, bias, h0, c0, y, hT, cT,
                                              trip_count, save_for_backward != 0);
  p->last_stream = s;
  if (hipEventRecord(p->ev_done, s) == hipSuccess) p->done_recorded = true;
  if (st != LL_OK) return st;
  if (save_for_backward) {
    p->state = ST_FWD_DONE;
    p->x = x;
    p->seq_len = seq_len;
    for (int l = 0; l < p->d.layers; ++l) p->W[l] = W[l];
    p->h0 = h0;
    p->c0 = c0;
  }
  return LL_OK;
}

ll_status lstm_loop_bwd(ll_plan* p, void* stream, const void* x, const int32_t* seq_len,
                        const void* const* W, const float* dy, const float* dhT,
                        const float* dcT, float* dx, float* const* dW, float* const* dbias,
                        float* dh0, float* dc0) {
  if (!p) return fail(LL_EINVAL, "plan is NULL");
  if (p->state != ST_FWD_DONE)
    return fail(LL_ESTATE, "no saved forward on this plan (call lstm_loop_fwd with "
                           "save_for_backward=1 first)");
  if (!x || !seq_len || !W) return fail(LL_EINVAL, "x, seq_len and W are required");
  if (x != p->x || seq_len != p->seq_len)
    return fail(LL_EINVAL, "x or seq_len differs from the saved forward's (%p, %p saved; %p, %p given)",
                p->x, (const void*)p->seq_len, x, (const void*)seq_len);
  for (int l = 0; l < p->d.layers; ++l)
    if (W[l] != p->W[l])
      return fail(LL_EINVAL, "W[%d] = %p differs from the saved forward's %p", l, W[l], p->W[l]);
  if (!dW || !dbias) return fail(LL_EINVAL, "dW and dbias are required");
  for (int l = 0; l < p->d.layers; ++l)
    if (!dW[l] || !dbias[l]) return fail(LL_EINVAL, "dW[%d] or dbias[%d] is NULL", l, l);
  {
    const void* ptrs[] = {dy, dhT, dcT, dx, dh0, dc0};
    const char* names[] = {"dy", "dhT", "dcT", "dx", "dh0", "dc0"};
    for (int i = 0; i < 6; ++i)
      if (reinterpret_cast<uintptr_t>(ptrs[i]) & 15)
        return fail(LL_EINVAL, "%s = %p is not 16-byte aligned", names[i], ptrs[i]);
    for (int l = 0; l < p->d.layers; ++l)
      if ((reinterpret_cast<uintptr_t>(dW[l]) | reinterpret_cast<uintptr_t>(dbias[l])) & 15)
        return fail(LL_EINVAL, "dW[%d] = %p or dbias[%d] = %p is not 16-byte aligned", l, (void*)dW[l], l,
                    (void*)dbias[l]);
  }
  DeviceGuard guard(p->device);
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  ll_status st = p->bf16 ? enqueue_bwd<bf16_t>(p, s, dy, dhT, dcT, dx, dW, dbias, dh0, dc0)
                         : enqueue_bwd<float>(p, s, dy, dhT, dcT, dx, dW, dbias, dh0, dc0);
  p->last_stream = s;
  if (hipEventRecord(p->ev_done, s) == hipSuccess) p->done_recorded = true;
  p->state = ST_EMPTY;
  return st;
}

// ---------------------------------------------------------------------------
// The inference forward that allocates nothing: every buffer of an inference
// plan comes from this file-scope device array.  Host code never passes the
// array's name to a kernel or a copy (in host code it is only a stand-in
// symbol): it uses the device address hipGetSymbolAddress returns, looked up
// once per device with that device current.
// ---------------------------------------------------------------------------
}  // extern "C"

namespace {

static __device__ __align__(256) unsigned char scratch[LL_NOALLOC_SCRATCH_BYTES];

std::mutex g_scratch_mu;
void* g_scratch_ptr[64] = {};

ll_status scratch_address(int device, unsigned char** out) {
  if (device < 0 || device >= 64) return fail(LL_EUNSUPPORTED, "device %d: at most 64 devices", device);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[device]) {
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr)
      return fail(LL_EHIP, "hipGetSymbolAddress of the scratch array on device %d failed: %s", device,
                  hipGetErrorString(e));
    g_scratch_ptr[device] = ptr;
  }
  *out = static_cast<unsigned char*>(g_scratch_ptr[device]);
  return LL_OK;
}

}  // namespace

extern "C" {

ll_status lstm_loop_fwd_noalloc(const ll_desc* desc, void* stream, const void* x,
                                const int32_t* seq_len, const void* const* W,
                                const float* const* bias, const float* h0, const float* c0,
                                float* y, float* hT, float* cT, int32_t* trip_count,
                                int32_t* device_error) {
  ll_status st = validate_desc(desc);
  if (st != LL_OK) return st;
  if (desc->spill || desc->recompute)
    return fail(LL_EUNSUPPORTED, "the forward without allocation saves no stack: spill and recompute "
                                 "(memory policies of the saved stack) must be 0");
  const bool two_state = desc->cell == LL_CELL_LSTM || desc->cell == LL_CELL_LSTM_SKIP;
  if (!x || !seq_len || !W || !bias || !hT || (!cT && two_state))
    return fail(LL_EINVAL, "x, seq_len, W, bias, hT and (LSTM) cT are required");
  for (int l = 0; l < desc->layers; ++l)
    if (!W[l] || !bias[l]) return fail(LL_EINVAL, "W[%d] or bias[%d] is NULL", l, l);
  {
    const void* ptrs[] = {x, seq_len, h0, c0, y, hT, cT, trip_count, device_error};
    const char* names[] = {"x", "seq_len", "h0", "c0", "y", "hT", "cT", "trip_count", "device_error"};
    for (int i = 0; i < 9; ++i)
      if (reinterpret_cast<uintptr_t>(ptrs[i]) & 15)
        return fail(LL_EINVAL, "%s = %p is not 16-byte aligned", names[i], ptrs[i]);
    for (int l = 0; l < desc->layers; ++l)
      if ((reinterpret_cast<uintptr_t>(W[l]) | reinterpret_cast<uintptr_t>(bias[l])) & 15)
        return fail(LL_EINVAL, "W[%d] = %p or bias[%d] = %p is not 16-byte aligned", l, W[l], l,
                    (const void*)bias[l]);
  }
  int device = 0;
  LL_HIP(hipGetDevice(&device));
  hipDeviceProp_t prop;
  LL_HIP(hipGetDeviceProperties(&prop, device));
  ll_plan p;   // decisions only: no stream, no event, no device allocation
  st = plan_configure(&p, desc, device, prop);
  if (st != LL_OK) return st;
  unsigned char* base = nullptr;
  st = scratch_address(device, &base);
  if (st != LL_OK) return st;
  size_t used = 0;
  auto take = [&](void** slot, size_t bytes, const char* what) -> ll_status {
    const size_t at = (used + 255) & ~(size_t)255;
    if (bytes > LL_NOALLOC_SCRATCH_BYTES || at + bytes > LL_NOALLOC_SCRATCH_BYTES)
      return fail(LL_EUNSUPPORTED,
                  "T_max = %d, B = %d, I = %d, H = %d, layers = %d need more than the %llu bytes of "
                  "scratch of the forward without allocation (%s: %zu bytes at offset %zu); use a plan",
                  desc->T_max, desc->B, desc->I, desc->H, desc->layers,
                  (unsigned long long)LL_NOALLOC_SCRATCH_BYTES, what, bytes, at);
    *slot = base + at;
    used = at + bytes;
    return LL_OK;
  };
  st = plan_layout(&p, true, take);
  if (st != LL_OK) return st;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  // the device error word must start at zero (prep only ORs into it); the
  // exchange flags are cleared by each loop's set-up kernel
  LL_HIP(ll::launch_zero_u32(reinterpret_cast<unsigned*>(p.meta), ll::META_INTS, s));
  st = p.bf16 ? enqueue_fwd<bf16_t>(&p, s, x, seq_len, W, bias, h0, c0, y, hT, cT, trip_count, false)
              : enqueue_fwd<float>(&p, s, x, seq_len, W, bias, h0, c0, y, hT, cT, trip_count, false);
  if (st != LL_OK) return st;
  if (device_error) LL_HIP(ll::launch_copy_i32(p.meta + 2, device_error, 1, s));
  return LL_OK;
}

ll_status ll_status_sync(ll_plan* p, int32_t* device_error) {
  if (!p) return fail(LL_EINVAL, "plan is NULL");
  DeviceGuard guard(p->device);
  if (p->done_recorded) LL_HIP(hipEventSynchronize(p->ev_done));
  int32_t e = 0;
  LL_HIP(hipMemcpy(&e, p->meta + 2, sizeof(int32_t), hipMemcpyDeviceToHost));
  const int32_t zero = 0;
  LL_HIP(hipMemcpy(p->meta + 2, &zero, sizeof(int32_t), hipMemcpyHostToDevice));
  if (device_error) *device_error = e;
  return LL_OK;
}

}  // extern "C"
