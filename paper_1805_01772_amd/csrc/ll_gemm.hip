// Matrix-core GEMM with both operands K-contiguous:
//   C[crow(m), n] = sum_k A[arow(m), k] * Bm[n, k] (+ bias[n])
// Used for the products of the loop that do not sit on the recurrence:
//   * the input projection x_t W_x + b of every compact row (hoisted out of
//     the forward loop: it does not depend on h, so it can run ahead of the
//     loop the way independent work of later iterations may);
//   * dx_t = dz_t W_x^T of every compact row (the write of dx_t that is the
//     gradient of reading x_t);
//   * dW = sum over iterations of [x_t, h_{t-1}]^T dz_t (the loop-constant
//     gradient, a sum over iterations), with the reduction running over the
//     compact rows of all steps.
// Two kernels:
//   * gemm_nt_kernel (any element type, any shape): 256 threads = 4 waves in
//     a 2x2 arrangement, 128x128 output tile; each wave owns 64x64 = 4x4 MFMA
//     tiles of 16x16.  A k-tile is 128 bytes of every row (8 chunks of 16
//     bytes), staged through LDS with a 16-byte row pad; the next k-tile is
//     fetched into registers while the current one is multiplied.
//   * gemm_nt_bf16_lds_kernel (bf16 operands with 16-byte aligned rows): a
//     256x256 output tile on 8 waves, operands loaded straight into LDS
//     (buffer loads with the LDS-destination form), two LDS stages, 32x32x16
//     MFMAs.  Per k-tile of 64 a work-group moves 64 KB into LDS for 8.4
//     MFLOP, half the bytes per flop of the 128x128 tile.
// Epilogues read everything they need (bias, row maps, gate addends) into
// registers before their stores.  A load placed after a store that the
// compiler cannot prove disjoint from it waits for every store in flight
// (s_waitcnt vmcnt(0)), which serialised the 1024 stores of a 256x256 fp32
// tile: 93 of the input projection's 215 us at I = H = 1024, B = 128.
#include "ll_exchange.h"

namespace ll {

namespace {

template <typename T>
__device__ __forceinline__ uint4 load_chunk(const T* row, int kk, int kend) {
  constexpr int KPC = Op<T>::kPerChunk;
  if (kk + KPC <= kend) return ld16(row + kk);
  uint4 v = zero4();
  if (kk >= kend) return v;
  T tmp[KPC];
#pragma unroll
  for (int e = 0; e < KPC; ++e) tmp[e] = (kk + e < kend) ? row[kk + e] : T(0);
  __builtin_memcpy(&v, tmp, 16);
  return v;
}

// Gate activation of column block blk (i, f, g, o): tanh for g, the
// logistic function for the others (the recomputation of saved gates).
__device__ __forceinline__ float lstm_gate_act(float u, int blk) {
  return blk == 2 ? tanhf_(u) : sigmoidf_(u);
}

}  // namespace

template <typename T>
__global__ __launch_bounds__(256, 2) void gemm_nt_kernel(GemmArgs g) {
  constexpr int KPC = Op<T>::kPerChunk;
  constexpr int BM = 128, BN = 128;
  constexpr int CH = 8;              // 16-byte chunks per row in a k-tile
  constexpr int KT = CH * KPC;       // elements per k-tile
  constexpr int PITCH = CH + 1;      // row pitch in chunks
  __shared__ uint4 sA[BM * PITCH];
  __shared__ uint4 sB[BN * PITCH];

  const int M = g.M_dev ? min(*g.M_dev, g.M) : g.M;
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;
  if (m0 >= M) return;
  const int K = g.K_dev ? *g.K_dev : g.K;
  const int z = blockIdx.z;
  const int kper = ((K + g.splits - 1) / g.splits + KT - 1) / KT * KT;
  const int kb = min(K, z * kper);
  const int ke = min(K, kb + kper);
  const int nkt = (ke - kb + KT - 1) / KT;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int q = lane >> 4, l16 = lane & 15;

  const T* A = reinterpret_cast<const T*>(g.A);
  const T* Bm = reinterpret_cast<const T*>(g.Bm);
  const T* arow[4];
  const T* brow[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int c = tid + 256 * i;
    const int row = c >> 3;
    const int m = m0 + row, n = n0 + row;
    arow[i] = nullptr;
    brow[i] = nullptr;
    if (m < M) arow[i] = A + (long)(g.a_rowmap ? g.a_rowmap[m] : m) * g.lda;
    if (n < g.N) brow[i] = Bm + (long)n * g.ldb;
  }
  uint4 ra[4], rb[4];
  auto fetch = [&](int kt) {
    const int kbase = kb + kt * KT;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int c = tid + 256 * i;
      const int kk = kbase + (c & 7) * KPC;
      ra[i] = arow[i] ? load_chunk<T>(arow[i], kk, ke) : zero4();
      rb[i] = brow[i] ? load_chunk<T>(brow[i], kk, ke) : zero4();
    }
  };
  auto stash = [&]() {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int c = tid + 256 * i;
      const int row = c >> 3, ch = c & 7;
      sA[row * PITCH + ch] = ra[i];
      sB[row * PITCH + ch] = rb[i];
    }
  };

  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  if (nkt > 0) {
    fetch(0);
    stash();
    __syncthreads();
  }
  for (int kt = 0; kt < nkt; ++kt) {
    if (kt + 1 < nkt) fetch(kt + 1);
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      uint4 a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) a[i] = sA[(wm * 64 + i * 16 + l16) * PITCH + s * 4 + q];
#pragma unroll
      for (int j = 0; j < 4; ++j) b[j] = sB[(wn * 64 + j * 16 + l16) * PITCH + s * 4 + q];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = Mfma<T>::step(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
    if (kt + 1 < nkt) {
      stash();
      __syncthreads();
    }
  }

  // epilogue: loads first, then stores (file header)
  const bool split = g.splits > 1;
  float* __restrict__ Cb = g.C + (split ? (long)z * g.split_stride : 0L);
  const float* __restrict__ bias = (g.bias && (!split || z == 0)) ? g.bias : nullptr;
  const int* __restrict__ crm = split ? nullptr : g.c_rowmap;
  const int N = g.N, act_h = g.act_h;
  const long ldc = g.ldc;
  float bn[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int n = n0 + wn * 64 + j * 16 + l16;
    bn[j] = bias && n < N ? bias[n] : 0.f;
  }
  int crows[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int m = m0 + wm * 64 + i * 16 + q * 4 + e;
      crows[i][e] = m < M ? (crm ? crm[m] : m) : -1;
    }
  __builtin_amdgcn_s_waitcnt(0xF70);   // vmcnt(0): those loads, ahead of any store
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int* crow = crows[i];
    int mrow[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) mrow[e] = m0 + wm * 64 + i * 16 + q * 4 + e;
    float zin[4][4];
    if (act_h) {
#pragma unroll
      for (int e = 0; e < 4; ++e)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int n = n0 + wn * 64 + j * 16 + l16;
          zin[e][j] = crow[e] < 0 || n >= N ? 0.f
                      : g.addend ? g.addend[(long)g.add_rowmap[mrow[e]] * g.ld_add + n]
                                 : Cb[(long)crow[e] * ldc + n];
        }
      __builtin_amdgcn_s_waitcnt(0xF70);
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      if (crow[e] < 0) continue;
      float* cr = Cb + (long)crow[e] * ldc;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int n = n0 + wn * 64 + j * 16 + l16;
        if (n < N) {
          float v = acc[i][j][e] + bn[j];
          if (act_h) v = lstm_gate_act(v + zin[e][j], n / act_h);
          cr[n] = v;
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Large-tile bf16 kernel.
//
// Work-groups: 512 threads = 8 waves, 4 (rows) x 2 (columns); a wave owns a
// 64x128 block of the 256x256 tile = 2x4 MFMA tiles of 32x32 (128
// accumulator registers, so two waves share each SIMD).
//
// LDS: per stage, the A and B k-tiles (256 rows x 64 elements, 32 KB each) as
// 8 chunks of 16 bytes per row.  Chunk c of row r sits in slot c ^ swz(r),
// swz(r) = (r & 7) ^ ((r >> 3) & 1): the 16 rows read by 16 consecutive
// lanes hit 16 different 16-byte bank groups, and so do 8 consecutive rows.
// A load instruction (64 lanes x 16 bytes) fills 8 rows: lane l writes slot
// l % 8 of row l / 8 (the hardware places lane l's data at base + 16 l), so it
// reads k-chunk (l % 8) ^ swz(row) of that row.
//
// Pipeline: the loads of k-tile kt + 1 go into the other stage while k-tile
// kt is multiplied; one barrier per k-tile.  The stage being read and the
// stage being filled are different arrays, so the compiler does not wait for
// the fills before each LDS read.
//
// Rows past M or N and k-chunks past the end of the reduction read as zero
// (buffer loads past the descriptor's range return zero); a chunk that
// straddles the end of K is read whole, which needs K % 8 == 0 or zeros in
// the operands up to the next multiple of 8 (GemmArgs::k_zero_tail).
//
// Tile order: work-group id L runs on XCD L % 8 (round-robin dispatch); XCD x
// takes a contiguous share of the tiles that exist for the M rows actually
// present, ordered in groups of 4 row tiles, so the work-groups running
// together on one XCD read 4 A panels and about 8 B panels through its L2.
// ---------------------------------------------------------------------------
namespace {

typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((address_space(3))) void lds_void_t;

constexpr int kBigTile = 256;
constexpr int kBigThreads = 512;
constexpr int kBigGroupRows = 4;

__device__ __forceinline__ int big_swz(int r) { return (r & 7) ^ ((r >> 3) & 1); }

}  // namespace

__global__ __launch_bounds__(kBigThreads, 1) void gemm_nt_bf16_lds_kernel(GemmArgs g, unsigned a_bytes,
                                                                         unsigned b_bytes) {
  constexpr int BM = kBigTile, BN = kBigTile;
  constexpr int NW = kBigThreads / 64;       // 8 waves
  constexpr int WGN = 2;                     // waves across the columns
  constexpr int WM = BM / (NW / WGN), WN = BN / WGN;   // 64 x 128 per wave
  constexpr int MI = WM / 32, NI = WN / 32;  // 2 x 4 MFMA tiles
  constexpr int KT = 64;                     // elements per k-tile
  constexpr int CH = BM * 8;                 // chunks per operand and stage
  constexpr int LI = BM / 8 / NW;            // load instructions per wave and operand
  __shared__ uint4 sA0[CH], sA1[CH], sB0[CH], sB1[CH];

  if ((int)blockIdx.x < g.pre_blocks) {   // the jobs carried by this launch
    pre_jobs_body<bf16_t>(g.pre, blockIdx.x, g.pre_blocks, kBigThreads);
    return;
  }
  const int M = g.M_dev ? min(*g.M_dev, g.M) : g.M;
  const int K = g.K_dev ? *g.K_dev : g.K;
  const int nmt = (M + BM - 1) / BM, nnt = (g.N + BN - 1) / BN;
  const int per_split = nmt * nnt;
  const int ntiles = per_split * g.splits;
  const int share = (ntiles + 7) / 8;
  const int L = blockIdx.x - g.pre_blocks;
  const int t = (L & 7) * share + (L >> 3);
  if ((L >> 3) >= share || t >= ntiles) return;
  const int z = t / per_split;
  const int tt = t - z * per_split;
  const int grp = tt / (kBigGroupRows * nnt);
  const int fm = grp * kBigGroupRows;
  const int gsz = min(nmt - fm, kBigGroupRows);
  const int within = tt - grp * kBigGroupRows * nnt;
  const int m0 = (fm + within % gsz) * BM, n0 = (within / gsz) * BN;

  const int kper = ((K + g.splits - 1) / g.splits + KT - 1) / KT * KT;
  const int kb = min(K, z * kper);
  const int ke = min(K, kb + kper);
  const int nkt = (ke - kb + KT - 1) / KT;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WGN, wn = wave % WGN;
  const int l32 = lane & 31, kc = lane >> 5;

  const __amdgpu_buffer_rsrc_t ra = make_rsrc(g.A, a_bytes);
  const __amdgpu_buffer_rsrc_t rb = make_rsrc(g.Bm, b_bytes);
  // this lane's source in load instruction i: row (i NW + wave) 8 + lane / 8,
  // k-chunk ach / bch of the k-tile (byte offset without the k-tile base)
  unsigned aoff[LI], boff[LI];
  int ach[LI], bch[LI];
#pragma unroll
  for (int i = 0; i < LI; ++i) {
    const int row = (i * NW + wave) * 8 + (lane >> 3);
    const int m = m0 + row, n = n0 + row;
    ach[i] = bch[i] = (lane & 7) ^ big_swz(row);
    aoff[i] = m < M ? (unsigned)((g.a_rowmap ? g.a_rowmap[m] : m) * (long)g.lda * 2 + ach[i] * 16) : kOOB;
    boff[i] = n < g.N ? (unsigned)(n * (long)g.ldb * 2 + bch[i] * 16) : kOOB;
  }
  auto fill = [&](int kt, uint4* a_dst, uint4* b_dst) {
    const int k0 = kb + kt * KT;
    const bool full = k0 + KT <= ke;
    const unsigned kbytes = (unsigned)k0 * 2u;
#pragma unroll
    for (int i = 0; i < LI; ++i) {
      const bool past = !full & (k0 + ach[i] * 8 >= ke);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (lds_void_t*)(a_dst + (i * NW + wave) * 64), 16,
                                               past ? kOOB : aoff[i] + kbytes, 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < LI; ++i) {
      const bool past = !full & (k0 + bch[i] * 8 >= ke);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, (lds_void_t*)(b_dst + (i * NW + wave) * 64), 16,
                                               past ? kOOB : boff[i] + kbytes, 0, 0, 0);
    }
  };

  f32x16 acc[MI][NI];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < NI; ++j) acc[i][j] = f32x16{};

  // MFMA operand lanes: lane l supplies row (A) / column (B) l % 32 and the
  // 8 consecutive k of chunk 2 ks + l / 32 of k-step ks
  const int sw = big_swz(l32);
  const int arow = (wm * WM + l32) * 8, brow = (wn * WN + l32) * 8;
  auto step = [&](int kt, const uint4* a, const uint4* b, uint4* a_next, uint4* b_next) {
    // this wave's fills of k-tile kt have landed; the barrier makes every
    // wave's visible and ends every wave's reads of the other stage
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (kt + 1 < nkt) fill(kt + 1, a_next, b_next);
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const int c = (2 * ks + kc) ^ sw;
      uint4 av[MI], bv[NI];
#pragma unroll
      for (int i = 0; i < MI; ++i) av[i] = a[arow + i * 256 + c];
#pragma unroll
      for (int j = 0; j < NI; ++j) bv[j] = b[brow + j * 256 + c];
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NI; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              __builtin_bit_cast(bf16x8_t, av[i]), __builtin_bit_cast(bf16x8_t, bv[j]), acc[i][j], 0, 0, 0);
    }
  };
  if (nkt > 0) fill(0, sA0, sB0);
  for (int kt = 0; kt < nkt; kt += 2) {
    step(kt, sA0, sB0, sA1, sB1);
    if (kt + 1 < nkt) step(kt + 1, sA1, sB1, sA0, sB0);
  }

  // result register r of lane l: row (r % 4) + 8 (r / 4) + 4 (l / 32), column
  // l % 32.  Loads first, then stores (file header).
  const bool split = g.splits > 1;
  float* __restrict__ Cb = g.C + (split ? (long)z * g.split_stride : 0L);
  const float* __restrict__ bias = (g.bias && (!split || z == 0)) ? g.bias : nullptr;
  const int* __restrict__ crm = split ? nullptr : g.c_rowmap;
  const int N = g.N, act_h = g.act_h;
  const long ldc = g.ldc;
  float bn[NI];
#pragma unroll
  for (int j = 0; j < NI; ++j) {
    const int n = n0 + wn * WN + j * 32 + l32;
    bn[j] = bias && n < N ? bias[n] : 0.f;
  }
  int crows[MI][16];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int m = m0 + wm * WM + i * 32 + (r & 3) + 8 * (r >> 2) + 4 * kc;
      crows[i][r] = m < M ? (crm ? crm[m] : m) : -1;
    }
  __builtin_amdgcn_s_waitcnt(0xF70);   // vmcnt(0): those loads, ahead of any store
#pragma unroll
  for (int i = 0; i < MI; ++i) {
    const int* crow = crows[i];
    if (act_h) {
      int mrow[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) mrow[r] = m0 + wm * WM + i * 32 + (r & 3) + 8 * (r >> 2) + 4 * kc;
      // gate recomputation: four rows' addends at a time, then their stores
#pragma unroll
      for (int r0 = 0; r0 < 16; r0 += 4) {
        float zin[4][NI];
#pragma unroll
        for (int e = 0; e < 4; ++e)
#pragma unroll
          for (int j = 0; j < NI; ++j) {
            const int n = n0 + wn * WN + j * 32 + l32;
            const int r = r0 + e;
            zin[e][j] = crow[r] < 0 || n >= N ? 0.f
                        : g.addend ? g.addend[(long)g.add_rowmap[mrow[r]] * g.ld_add + n]
                                   : Cb[(long)crow[r] * ldc + n];
          }
        __builtin_amdgcn_s_waitcnt(0xF70);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int r = r0 + e;
          if (crow[r] < 0) continue;
          float* cr = Cb + (long)crow[r] * ldc;
#pragma unroll
          for (int j = 0; j < NI; ++j) {
            const int n = n0 + wn * WN + j * 32 + l32;
            if (n < N) cr[n] = lstm_gate_act(acc[i][j][r] + bn[j] + zin[e][j], n / act_h);
          }
        }
      }
    } else {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        if (crow[r] < 0) continue;
        float* cr = Cb + (long)crow[r] * ldc;
#pragma unroll
        for (int j = 0; j < NI; ++j) {
          const int n = n0 + wn * WN + j * 32 + l32;
          if (n < N) cr[n] = acc[i][j][r] + bn[j];
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Product over rows, bf16: C[m][n] = sum_k A[arow(k)][m] B[k][n] (dW = [X;
// Hprev]^T DZ straight from the row-major operands).  The same work-group
// shape, tile order and epilogue as the kernel above; what differs is the
// operand layout and the pipeline depth (four LDS stages).  A k-tile of
// either operand is 32 rows (k) x 256 columns, loaded row by row (a row's 512 bytes are contiguous
// in memory): LDS holds [k][32 chunks of 16 bytes], chunk c of row k in
// slot c ^ tn_swz(k).  The matrix-core operands need 8 consecutive k per
// lane; gfx950's transposing LDS read (ds_read_b64_tr_b16) gives them: in
// each 16-lane group, lane i's j-th element is the (i % 4)-th element of the
// 8 bytes that lane 4 j + i / 4 addressed.  Lane s of the group therefore
// addresses row k0 + s / 4, columns c0 + 4 (s % 4) .. + 3, and lane i
// receives column c0 + i at rows k0 .. k0 + 3; two such reads (k0, k0 + 4)
// make the 8 k of a 32x32x16 operand.  The swizzle (slot XOR 0, 6, 10, 12
// for rows k % 4 = 0 .. 3) puts the four rows a 16-lane group reads at
// distinct 32-byte bank groups within 128 bytes, and the eight row pieces of
// two neighbouring groups at distinct ones within 256 bytes (measured on
// the dW shape: 0.81 PFLOP/s against 0.70 without a swizzle).  The row map
// of a k-tile is loaded four k-tiles ahead, so no fill waits on it.
// ---------------------------------------------------------------------------
namespace {

__device__ __forceinline__ int tn_swz(int k) { return (0x0c0a0600u >> ((k & 3) * 8)) & 31; }

typedef short tn_v4s __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint2 ds_read_tr16(const uint4* base, unsigned byte_off) {
  const tn_v4s v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) tn_v4s*)((__attribute__((address_space(3))) char*)base + byte_off));
  return __builtin_bit_cast(uint2, v);
}

}  // namespace

__global__ __launch_bounds__(kBigThreads, 1) void gemm_tn_bf16_lds_kernel(GemmTnArgs g, unsigned a_bytes,
                                                                         unsigned b_bytes, unsigned a2_bytes) {
  constexpr int BM = kBigTile, BN = kBigTile;
  constexpr int NW = kBigThreads / 64;       // 8 waves
  constexpr int WGN = 2;
  constexpr int WM = BM / (NW / WGN), WN = BN / WGN;   // 64 x 128 per wave
  constexpr int MI = WM / 32, NI = WN / 32;
  constexpr int KT = 32;                     // rows (k) per k-tile
  constexpr int RC = BM * 2 / 16;            // 16-byte chunks per row of a k-tile (32)
  constexpr int CH = KT * RC;                // chunks per operand and stage
  constexpr int LI = CH / 64 / NW;           // load instructions per wave and operand (2)
  // four stages: the fills run three k-tiles ahead.  Every fill, map read
  // and step is issued unconditionally (k-tiles past the end load zeros and
  // add nothing), so each wave's memory operations follow one fixed pattern
  // and the compiler's wait counts across the loop stay exact
  __shared__ uint4 sA0[CH], sA1[CH], sA2[CH], sA3[CH], sB0[CH], sB1[CH], sB2[CH], sB3[CH];

  const int M = g.M;
  const int K = g.K_dev ? min(*g.K_dev, g.K) : g.K;
  const int nmt = (M + BM - 1) / BM, nnt = (g.N + BN - 1) / BN;
  const int per_split = nmt * nnt;
  const int ntiles = per_split * g.splits;
  const int share = (ntiles + 7) / 8;
  const int L = blockIdx.x;
  const int t = (L & 7) * share + (L >> 3);
  if ((L >> 3) >= share || t >= ntiles) return;
  const int z = t / per_split;
  const int tt = t - z * per_split;
  const int grp = tt / (kBigGroupRows * nnt);
  const int fm = grp * kBigGroupRows;
  const int gsz = min(nmt - fm, kBigGroupRows);
  const int within = tt - grp * kBigGroupRows * nnt;
  const int m0 = (fm + within % gsz) * BM, n0 = (within / gsz) * BN;

  const int kper = ((K + g.splits - 1) / g.splits + KT - 1) / KT * KT;
  const int kb = min(K, z * kper);
  const int ke = min(K, kb + kper);
  const int nkt = (ke - kb + KT - 1) / KT;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WGN, wn = wave % WGN;

  // the operand this tile's rows come from
  const bool second = g.A2 && m0 >= g.M1;
  const __amdgpu_buffer_rsrc_t ra = second ? make_rsrc(g.A2, a2_bytes) : make_rsrc(g.A, a_bytes);
  const __amdgpu_buffer_rsrc_t rb = make_rsrc(g.Bm, b_bytes);
  const long lda = second ? g.lda2 : g.lda;
  const int* a_rowmap = second ? g.a2_rowmap : g.a_rowmap;
  const int am0 = second ? m0 - g.M1 : m0, aM = second ? M - g.M1 : (g.A2 ? g.M1 : M);
  // load instruction i of this wave: k-tile rows (i NW + wave) 2 + lane / 32,
  // LDS slot lane % 32 of that row, which holds column chunk slot ^ tn_swz(row)
  int lrow[LI];
  unsigned acol[LI], bcol[LI];   // byte offset of the chunk within a row (kOOB: past M / N)
#pragma unroll
  for (int i = 0; i < LI; ++i) {
    lrow[i] = (i * NW + wave) * 2 + (lane >> 5);
    const int c = (lane & 31) ^ tn_swz(lrow[i]);
    acol[i] = am0 + c * 8 < aM ? (unsigned)((am0 + c * 8) * 2) : kOOB;
    bcol[i] = n0 + c * 8 < g.N ? (unsigned)((n0 + c * 8) * 2) : kOOB;
  }
  // row-map entries, read with no branch (past the map's end: zero) four
  // k-tiles ahead of the fill that uses them (buffer kt % 4)
  const bool has_map = a_rowmap != nullptr;
  const __amdgpu_buffer_rsrc_t rmap = make_rsrc(a_rowmap, has_map ? (unsigned)ke * 4u : 0u);
  unsigned amap[4][LI];
  auto load_map = [&](int kt, unsigned (&dst)[LI]) {
    const int k0 = kb + kt * KT;
#pragma unroll
    for (int i = 0; i < LI; ++i)
      dst[i] = __builtin_amdgcn_raw_buffer_load_b32(rmap, (unsigned)(k0 + lrow[i]) * 4u, 0, 0);
  };
  auto fill = [&](int kt, uint4* a_dst, uint4* b_dst, unsigned (&am)[LI]) {
    const int k0 = kb + kt * KT;
#pragma unroll
    for (int i = 0; i < LI; ++i) {
      const int k = k0 + lrow[i];
      const bool ok = k < ke;
      const long ar = has_map ? (long)am[i] : (long)k;
      const unsigned ao = ok && acol[i] != kOOB ? (unsigned)(ar * lda * 2) + acol[i] : kOOB;
      const unsigned bo = ok && bcol[i] != kOOB ? (unsigned)((long)k * g.ldb * 2) + bcol[i] : kOOB;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (lds_void_t*)(a_dst + (i * NW + wave) * 64), 16, ao, 0, 0, 0);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, (lds_void_t*)(b_dst + (i * NW + wave) * 64), 16, bo, 0, 0, 0);
    }
    load_map(kt + 4, am);
  };

  f32x16 acc[MI][NI];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < NI; ++j) acc[i][j] = f32x16{};

  // transposing reads: group G = lane / 16 takes k-half G / 2 and column half
  // G % 2 of a 32-wide operand block; lane s of the group addresses row
  // s / 4 (+ 4 for the second read), columns 4 (s % 4) .. + 3
  const int G = lane >> 4, s16 = lane & 15;
  const int rk = (G >> 1) * 8 + (s16 >> 2);          // row within a 16-row k-step
  const int cc = (G & 1) * 16 + 4 * (s16 & 3);       // column within a 32-column block
  auto rd = [&](const uint4* base, int k_local, int col) -> uint2 {
    const unsigned off = (unsigned)((k_local * RC + ((col >> 3) ^ tn_swz(k_local))) * 16 + (col & 7) * 2);
    return ds_read_tr16(base, off);
  };
  auto step = [&](int kt, const uint4* a, const uint4* b, uint4* a_fill, uint4* b_fill, unsigned (&am)[LI]) {
    // k-tile kt's loads have landed (in flight still: the map reads its fill
    // issued after them, 3 LI operations for each of the fills of kt + 1 and
    // kt + 2); the barrier makes every wave's visible and ends every wave's
    // reads of the stage refilled next (k-tile kt - 1's)
    static_assert(7 * LI <= 15, "vmcnt field");
    __builtin_amdgcn_s_waitcnt(0xF70 | (7 * LI));
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    fill(kt + 3, a_fill, b_fill, am);
#pragma unroll
    for (int ks = 0; ks < KT / 16; ++ks) {
      const int k_local = ks * 16 + rk;
      uint4 av[MI], bv[NI];
#pragma unroll
      for (int i = 0; i < MI; ++i) {
        const int col = wm * WM + i * 32 + cc;
        const uint2 lo = rd(a, k_local, col), hi = rd(a, k_local + 4, col);
        av[i] = make_uint4(lo.x, lo.y, hi.x, hi.y);
      }
#pragma unroll
      for (int j = 0; j < NI; ++j) {
        const int col = wn * WN + j * 32 + cc;
        const uint2 lo = rd(b, k_local, col), hi = rd(b, k_local + 4, col);
        bv[j] = make_uint4(lo.x, lo.y, hi.x, hi.y);
      }
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NI; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              __builtin_bit_cast(bf16x8_t, av[i]), __builtin_bit_cast(bf16x8_t, bv[j]), acc[i][j], 0, 0, 0);
    }
  };
  // prologue: the maps of k-tiles 0 .. 3, the fills of 0 .. 2 (each fill
  // then reads the map four k-tiles ahead into the buffer it just used)
  load_map(0, amap[0]);
  load_map(1, amap[1]);
  load_map(2, amap[2]);
  load_map(3, amap[3]);
  fill(0, sA0, sB0, amap[0]);
  fill(1, sA1, sB1, amap[1]);
  fill(2, sA2, sB2, amap[2]);
  for (int kt = 0; kt < nkt; kt += 4) {
    step(kt, sA0, sB0, sA3, sB3, amap[3]);
    step(kt + 1, sA1, sB1, sA0, sB0, amap[0]);
    step(kt + 2, sA2, sB2, sA1, sB1, amap[1]);
    step(kt + 3, sA3, sB3, sA2, sB2, amap[2]);
  }
  // the fills issued past the last k-tile write this work-group's LDS:
  // they land before the work-group (and its LDS) ends
  __builtin_amdgcn_s_waitcnt(0xF70);

  // result register r of lane l: row (r % 4) + 8 (r / 4) + 4 (l / 32), column l % 32
  const int l32 = lane & 31, kc = lane >> 5;
  if (g.tile_flags && g.splits == 2) {
    // The two splits of this tile meet on its counter: the first to arrive
    // stores its sums to its slice of C and then sets the tile's ready word;
    // the second waits for that word (the first is already running, so the
    // wait ends), adds the slice to its own sums and writes the result.  The
    // sum of two terms does not depend on which came first.
    __shared__ int s_first;
    unsigned* arrive = g.tile_flags + 2L * tt;
    unsigned* ready = arrive + 1;
    if (tid == 0)
      s_first = __hip_atomic_fetch_add(arrive, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0u;
    __syncthreads();
    const bool first = s_first != 0;
    const unsigned slice_bytes = (unsigned)((long)M * g.ldc * 4);
    if (first) {
      const __amdgpu_buffer_rsrc_t rc = make_rsrc(g.C + (long)z * g.split_stride, slice_bytes);
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int m = m0 + wm * WM + i * 32 + (r & 3) + 8 * (r >> 2) + 4 * kc;
#pragma unroll
          for (int j = 0; j < NI; ++j) {
            const int n = n0 + wn * WN + j * 32 + l32;
            st_dev(rc, m < M && n < g.N ? (unsigned)(((long)m * g.ldc + n) * 4) : kOOB, acc[i][j][r]);
          }
        }
      wait_all_vm();
      __syncthreads();
      if (tid == 0) __hip_atomic_store(ready, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      return;
    }
    if (tid == 0) {   // (bounded: about a second of polls, far past any store burst)
      for (unsigned polls = 0; polls < (1u << 24); ++polls) {
        if (__hip_atomic_load(ready, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0u) break;
        __builtin_amdgcn_s_sleep(1);
      }
    }
    __syncthreads();
    const __amdgpu_buffer_rsrc_t ro = make_rsrc(g.C + (long)(1 - z) * g.split_stride, slice_bytes);
#pragma unroll
    for (int i = 0; i < MI; ++i) {
      float other[16][NI];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int m = m0 + wm * WM + i * 32 + (r & 3) + 8 * (r >> 2) + 4 * kc;
#pragma unroll
        for (int j = 0; j < NI; ++j) {
          const int n = n0 + wn * WN + j * 32 + l32;
          other[r][j] = ld_f32_l2(ro, m < M && n < g.N ? (unsigned)(((long)m * g.ldc + n) * 4) : kOOB);
        }
      }
      __builtin_amdgcn_s_waitcnt(0xF70);   // vmcnt(0): those loads, ahead of the stores
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int m = m0 + wm * WM + i * 32 + (r & 3) + 8 * (r >> 2) + 4 * kc;
        if (m >= M) continue;
        float* orow = g.out + (long)m * g.ldo;
#pragma unroll
        for (int j = 0; j < NI; ++j) {
          const int n = n0 + wn * WN + j * 32 + l32;
          if (n < g.N) orow[n] = z == 0 ? acc[i][j][r] + other[r][j] : other[r][j] + acc[i][j][r];
        }
      }
    }
    if (tid == 0) {   // both splits are past the counter: clear it for the next launch
      __hip_atomic_store(arrive, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(ready, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    return;
  }
  float* Cb = g.C + (g.splits > 1 ? (long)z * g.split_stride : 0L);
#pragma unroll
  for (int i = 0; i < MI; ++i) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int m = m0 + wm * WM + i * 32 + (r & 3) + 8 * (r >> 2) + 4 * kc;
      if (m >= M) continue;
      float* cr = Cb + (long)m * g.ldc;
#pragma unroll
      for (int j = 0; j < NI; ++j) {
        const int n = n0 + wn * WN + j * 32 + l32;
        if (n < g.N) cr[n] = acc[i][j][r];
      }
    }
  }
}

bool gemm_tn_applies(const GemmTnArgs& g) {
  if (g.M % 8 || g.N % 8 || g.lda % 8 || g.ldb % 8 || g.splits < 1) return false;
  if ((reinterpret_cast<uintptr_t>(g.A) | reinterpret_cast<uintptr_t>(g.Bm) |
       reinterpret_cast<uintptr_t>(g.A2)) & 15)
    return false;
  if (g.A2 && (g.M1 % kBigTile || g.M1 <= 0 || g.M1 >= g.M || g.lda2 % 8)) return false;
  const long ab = (long)(g.a_rows > 0 ? g.a_rows : g.K) * g.lda * 2, bb = (long)g.b_rows * g.ldb * 2;
  const long a2b = g.A2 ? (long)g.a2_rows * g.lda2 * 2 : 0;
  return ab < (long)kOOB && bb < (long)kOOB && a2b < (long)kOOB;
}

hipError_t launch_gemm_tn(const GemmTnArgs& g, hipStream_t s) {
  if (!gemm_tn_applies(g)) return hipErrorInvalidValue;
  const long ab = (long)(g.a_rows > 0 ? g.a_rows : g.K) * g.lda * 2, bb = (long)g.b_rows * g.ldb * 2;
  const long a2b = g.A2 ? (long)g.a2_rows * g.lda2 * 2 : 0;
  const long tiles = (long)((g.M + kBigTile - 1) / kBigTile) * ((g.N + kBigTile - 1) / kBigTile) * g.splits;
  const long grid = (tiles + 7) / 8 * 8;
  hipLaunchKernelGGL(gemm_tn_bf16_lds_kernel, dim3((unsigned)grid), dim3(kBigThreads), 0, s, g, (unsigned)ab,
                     (unsigned)bb, (unsigned)a2b);
  return hipGetLastError();
}

namespace {

// Bytes of A and B the products of g may address (0 if past a 31-bit range).
void big_ranges(const GemmArgs& g, long* a_bytes, long* b_bytes) {
  *a_bytes = (long)(g.a_rows > 0 ? g.a_rows : g.M) * g.lda * 2;
  *b_bytes = (long)g.N * g.ldb * 2;
}

}  // namespace

bool gemm_big_applies(const GemmArgs& g, int elem_bytes) {
  if (elem_bytes != 2 || g.splits < 1) return false;
  if (g.lda % 8 != 0 || g.ldb % 8 != 0) return false;
  if ((reinterpret_cast<uintptr_t>(g.A) | reinterpret_cast<uintptr_t>(g.Bm)) & 15) return false;
  if (!g.k_zero_tail && (g.K_dev || g.K % 8 != 0)) return false;
  long ab, bb;
  big_ranges(g, &ab, &bb);
  return ab < (long)kOOB && bb < (long)kOOB;
}

long gemm_rounds(const GemmArgs& g, int elem_bytes, int n_cu) {
  if (gemm_big_applies(g, elem_bytes)) {
    const long tiles = (long)((g.M + kBigTile - 1) / kBigTile) * ((g.N + kBigTile - 1) / kBigTile) * g.splits;
    return (tiles + n_cu - 1) / n_cu;
  }
  const long groups = (long)((g.M + 127) / 128) * ((g.N + 127) / 128) * g.splits;
  return (groups + 2L * n_cu - 1) / (2L * n_cu);
}

template <typename T>
hipError_t launch_gemm_nt(const GemmArgs& g, hipStream_t s) {
  if (g.act_h > 0 && (g.splits != 1 || g.bias)) return hipErrorInvalidValue;
  if (g.pre_blocks < 0) return hipErrorInvalidValue;
  if (gemm_big_applies(g, (int)sizeof(T)) && sizeof(T) == 2) {
    long ab, bb;
    big_ranges(g, &ab, &bb);
    const long tiles = (long)((g.M + kBigTile - 1) / kBigTile) * ((g.N + kBigTile - 1) / kBigTile) * g.splits;
    const long share = (tiles + 7) / 8;
    hipLaunchKernelGGL(gemm_nt_bf16_lds_kernel, dim3((unsigned)(share * 8 + g.pre_blocks)), dim3(kBigThreads), 0,
                       s, g, (unsigned)ab, (unsigned)bb);
    return hipGetLastError();
  }
  if (g.pre_blocks > 0) {   // (the other kernels take no extra work-groups)
    const hipError_t e = launch_pre_jobs<T>(g.pre, s);
    if (e != hipSuccess) return e;
  }
  dim3 grid((g.N + 127) / 128, (g.M + 127) / 128, g.splits);
  hipLaunchKernelGGL(gemm_nt_kernel<T>, grid, dim3(256), 0, s, g);
  return hipGetLastError();
}

template hipError_t launch_gemm_nt<float>(const GemmArgs&, hipStream_t);
template hipError_t launch_gemm_nt<bf16_t>(const GemmArgs&, hipStream_t);

}  // namespace ll
