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
// 256 threads = 4 waves in a 2x2 arrangement, 128x128 output tile; each wave
// owns 64x64 = 4x4 MFMA tiles of 16x16.  A k-tile is 128 bytes of every row
// (8 chunks of 16 bytes), staged through LDS with a 16-byte row pad; the next
// k-tile is fetched into registers while the current one is multiplied.
#include "ll_kernels.h"

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

  const bool split = g.splits > 1;
  float* Cb = g.C + (split ? (long)z * g.split_stride : 0L);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int m = m0 + wm * 64 + i * 16 + q * 4 + e;
      if (m >= M) continue;
      const long crow = (!split && g.c_rowmap) ? (long)g.c_rowmap[m] : (long)m;
      float* cr = Cb + crow * g.ldc;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int n = n0 + wn * 64 + j * 16 + l16;
        if (n < g.N) {
          float v = acc[i][j][e];
          if (g.bias && (!split || z == 0)) v += g.bias[n];
          cr[n] = v;
        }
      }
    }
  }
}

long gemm_groups(long M, long N) { return ((N + 127) / 128) * ((M + 127) / 128); }

template <typename T>
hipError_t launch_gemm_nt(const GemmArgs& g, hipStream_t s) {
  dim3 grid((g.N + 127) / 128, (g.M + 127) / 128, g.splits);
  hipLaunchKernelGGL(gemm_nt_kernel<T>, grid, dim3(256), 0, s, g);
  return hipGetLastError();
}

template hipError_t launch_gemm_nt<float>(const GemmArgs&, hipStream_t);
template hipError_t launch_gemm_nt<bf16_t>(const GemmArgs&, hipStream_t);

}  // namespace ll
