// The two device-side while-loops: the forward LSTM recurrence and its
// gradient loop.  Each is one persistent cooperative launch whose work-groups
// run the loop themselves: the trip count T_eff is read from device memory
// (written by the prep kernel), so no step needs the host.
//
// Work split (both loops).  The batch, in length order, is cut into 16-row
// tiles; the hidden units into blocks of HJ.  Work-group (cb, rg) owns unit
// block cb and the row tiles rg, rg + RG, rg + 2RG, ...  Because rows are in
// decreasing length order, the rows still running at step t are a prefix, so
// finished tiles drop out of the work evenly across the RG groups.  The
// work-group keeps its slice of the recurrent weights in LDS for the whole
// loop (the weights are loop constants, entered once), and its share of the
// loop state (c, h forward; dh, dc backward) in registers.  The 4 waves split
// the reduction dimension; partial products meet in LDS.  One grid barrier per
// step publishes the exchanged operand (h_t forward, dz_t backward).
#include "ll_kernels.h"

namespace ll {

namespace {

constexpr int RPB = 20;   // LDS row pitch (floats) of the backward partials

// 16-byte operand chunk from float data (h0 at step 0), converted.
template <typename T> __device__ __forceinline__ uint4 chunk_from_f32(const float* p);
template <> __device__ __forceinline__ uint4 chunk_from_f32<float>(const float* p) {
  return ld16(p);
}
template <> __device__ __forceinline__ uint4 chunk_from_f32<bf16_t>(const float* p) {
  const float4 a = *reinterpret_cast<const float4*>(p);
  const float4 b = *reinterpret_cast<const float4*>(p + 4);
  uint4 r;
  r.x = (uint32_t)f32_to_bf16(a.x) | ((uint32_t)f32_to_bf16(a.y) << 16);
  r.y = (uint32_t)f32_to_bf16(a.z) | ((uint32_t)f32_to_bf16(a.w) << 16);
  r.z = (uint32_t)f32_to_bf16(b.x) | ((uint32_t)f32_to_bf16(b.y) << 16);
  r.w = (uint32_t)f32_to_bf16(b.z) | ((uint32_t)f32_to_bf16(b.w) << 16);
  return r;
}

}  // namespace

size_t fwd_loop_lds(int H, int HJ, int elem_bytes) {
  return (size_t)H * 4 * HJ * elem_bytes + (size_t)4 * 16 * (4 * HJ + 4) * sizeof(float);
}

size_t bwd_loop_lds(int H, int HJ, int elem_bytes) {
  size_t red = (size_t)4 * 16 * RPB * sizeof(float);
  const size_t dbr = (size_t)16 * 4 * HJ * sizeof(float);
  if (dbr > red) red = dbr;
  return (size_t)H * 4 * HJ * elem_bytes + red;
}

// ---------------------------------------------------------------------------
// Forward loop.  Step t (for t < T_eff, rows r < active[t]):
//   z = Zx[row] + h_{t-1} W_h            (MFMA; Zx = x_t W_x + b, hoisted)
//   i, f, o = sigmoid, g = tanh; c_t = f c + i g; h_t = o tanh(c_t)
//   push i, f, g, o, c_t onto the stack row; h_t into the history (operand
//   type), which is also what step t+1 multiplies; y_t = h_t.
// Rows whose sequence has ended keep c, h and get y_t = 0.
// ---------------------------------------------------------------------------
template <typename T, int MRT_MAX>
__global__ __launch_bounds__(256, 1) void fwd_loop_kernel(FwdLoopArgs a) {
  extern __shared__ uint4 lds[];
  constexpr int KPC = Op<T>::kPerChunk;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int q = lane >> 4, l16 = lane & 15;
  const int H = a.H, HJ = a.HJ, B = a.B, RG = a.RG;
  const int NCT = HJ >> 2;
  const int rg = blockIdx.x % RG, cb = blockIdx.x / RG;
  const int j0 = cb * HJ;
  const int KS = H / (4 * KPC);
  const int kspw = (KS + 3) >> 2;
  const int ks0 = min(KS, wave * kspw), ks1 = min(KS, ks0 + kspw);
  const long G4 = 4L * H;
  const T* WT = reinterpret_cast<const T*>(a.WT);
  T* HH = reinterpret_cast<T*>(a.HH);

  // Recurrent weight slice -> LDS, in fragment order: chunk (ks, ct, lane')
  // holds W_h[(4 ks + q') KPC .. +KPC, column(ct, lane' % 16)].
  const int nchunks = KS * NCT * 64;
  for (int idx = tid; idx < nchunks; idx += 256) {
    const int ks = idx / (NCT * 64);
    const int rem = idx - ks * NCT * 64;
    const int ct = rem >> 6, lp = rem & 63;
    const int c = ct * 16 + (lp & 15);
    const int gate = c / HJ, u = c - gate * HJ;
    const long n = (long)gate * H + j0 + u;
    const int k = (ks * 4 + (lp >> 4)) * KPC;
    lds[idx] = ld16(WT + n * a.ldw + a.woff + k);
  }
  float* red = reinterpret_cast<float*>(lds + nchunks);
  const int RP = 4 * HJ + 4;

  const bool has_elem = tid < 16 * HJ;
  const int em = tid / HJ, eu = tid - (tid / HJ) * HJ;
  const int j = j0 + eu;
  float hs[MRT_MAX], cs[MRT_MAX];
#pragma unroll
  for (int mt = 0; mt < MRT_MAX; ++mt) {
    hs[mt] = 0.f;
    cs[mt] = 0.f;
    if (mt < a.MRT && has_elem) {
      const int r = (rg + mt * RG) * 16 + em;
      if (r < B) {
        const long b = a.perm[r];
        if (a.h0) hs[mt] = a.h0[b * H + j];
        if (a.c0) cs[mt] = a.c0[b * H + j];
      }
    }
  }
  __syncthreads();

  GridBarrier gb{a.bar, a.abort_flag, a.err, gridDim.x, 0u, a.limit};
  const int T_eff = a.meta[0];
  for (int t = 0; t < T_eff; ++t) {
    const int A_t = a.active[t];
    const int off_t = a.off[t];
    const int off_p = t > 0 ? a.off[t - 1] : 0;
#pragma unroll
    for (int mt = 0; mt < MRT_MAX; ++mt) {
      if (mt >= a.MRT) continue;
      const int r0 = (rg + mt * RG) * 16;
      if (r0 >= A_t) {
        if (a.y && has_elem) {
          const int r = r0 + em;
          if (r < B) a.y[((long)t * B + a.perm[r]) * H + j] = 0.f;
        }
        continue;
      }
      f32x4 acc[4];
#pragma unroll
      for (int ct = 0; ct < 4; ++ct) acc[ct] = f32x4{0.f, 0.f, 0.f, 0.f};
      const int ar = r0 + l16;
      const bool aok = ar < A_t;
      const T* arow = nullptr;
      const float* arow0 = nullptr;
      if (aok) {
        if (t > 0) arow = HH + (long)(off_p + ar) * H;
        else if (a.h0) arow0 = a.h0 + (long)a.perm[ar] * H;
      }
      for (int kc = ks0; kc < ks1; kc += 8) {
        uint4 av[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const int ks = kc + i;
          const int k = (ks * 4 + q) * KPC;
          av[i] = zero4();
          if (ks < ks1) {
            if (arow) av[i] = ld16(arow + k);
            else if (arow0) av[i] = chunk_from_f32<T>(arow0 + k);
          }
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const int ks = kc + i;
          if (ks < ks1) {
#pragma unroll
            for (int ct = 0; ct < 4; ++ct)
              if (ct < NCT) acc[ct] = Mfma<T>::step(av[i], lds[(ks * NCT + ct) * 64 + lane], acc[ct]);
          }
        }
      }
#pragma unroll
      for (int ct = 0; ct < 4; ++ct) {
        if (ct < NCT) {
#pragma unroll
          for (int e = 0; e < 4; ++e) red[(wave * 16 + q * 4 + e) * RP + ct * 16 + l16] = acc[ct][e];
        }
      }
      __syncthreads();
      if (has_elem) {
        const int r = r0 + em;
        if (r < B) {
          const long b = a.perm[r];
          float* yrow = a.y ? a.y + ((long)t * B + b) * H : nullptr;
          if (r < A_t) {
            const long krow = off_t + r;
            const float* zx = a.Zx + krow * G4;
            float z[4];
#pragma unroll
            for (int gi = 0; gi < 4; ++gi) {
              const int col = gi * HJ + eu;
              float s = red[(0 * 16 + em) * RP + col];
              s += red[(1 * 16 + em) * RP + col];
              s += red[(2 * 16 + em) * RP + col];
              s += red[(3 * 16 + em) * RP + col];
              z[gi] = s + zx[(long)gi * H + j];
            }
            const float ig = sigmoidf_(z[0]);
            const float fg = sigmoidf_(z[1]);
            const float gg = tanhf_(z[2]);
            const float og = sigmoidf_(z[3]);
            const float cn = fg * cs[mt] + ig * gg;
            const float hn = og * tanhf_(cn);
            if (a.stack) {
              float* st = a.stack + krow * 5 * H;
              st[j] = ig;
              st[H + j] = fg;
              st[2 * H + j] = gg;
              st[3 * H + j] = og;
              st[4 * H + j] = cn;
            }
            HH[krow * H + j] = Op<T>::from_f32(hn);
            cs[mt] = cn;
            hs[mt] = hn;
            if (yrow) yrow[j] = hn;
          } else if (yrow) {
            yrow[j] = 0.f;
          }
        }
      }
      __syncthreads();
    }
    grid_sync(gb);
  }

#pragma unroll
  for (int mt = 0; mt < MRT_MAX; ++mt) {
    if (mt < a.MRT && has_elem) {
      const int r = (rg + mt * RG) * 16 + em;
      if (r < B) {
        const long b = a.perm[r];
        a.hT[b * H + j] = hs[mt];
        a.cT[b * H + j] = cs[mt];
        if (a.y)
          for (int t = T_eff; t < a.T_max; ++t) a.y[((long)t * B + b) * H + j] = 0.f;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Gradient loop.  Step t = T_eff-1 .. 0 (rows r < active[t]):
//   phase 1 (own units): pop i, f, g, o, c_t (and c_{t-1}) of the row;
//     dh_tot = dh + dy_t; do = dh_tot tanh(c_t);
//     dc_tot = dc + dh_tot o (1 - tanh^2 c_t);
//     dz = [dc_tot g i(1-i), dc_tot c_{t-1} f(1-f), dc_tot i (1-g^2), do o(1-o)];
//     dc <- dc_tot f; db += dz; publish dz (operand type)
//   grid barrier
//   phase 2 (own units): dh <- dz W_h^T over all 4H gate columns (MFMA).
// Rows whose sequence had ended at step t pass dh and dc through unchanged.
// ---------------------------------------------------------------------------
template <typename T, int MRT_MAX>
__global__ __launch_bounds__(256, 1) void bwd_loop_kernel(BwdLoopArgs a) {
  extern __shared__ uint4 lds[];
  constexpr int KPC = Op<T>::kPerChunk;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int q = lane >> 4, l16 = lane & 15;
  const int H = a.H, HJ = a.HJ, B = a.B, RG = a.RG;
  const int rg = blockIdx.x % RG, cb = blockIdx.x / RG;
  const int j0 = cb * HJ;
  const long G4 = 4L * H;
  const int KS = (int)(G4 / (4 * KPC));
  const int kspw = (KS + 3) >> 2;
  const int ks0 = min(KS, wave * kspw), ks1 = min(KS, ks0 + kspw);
  const T* W = reinterpret_cast<const T*>(a.W);
  T* DZ = reinterpret_cast<T*>(a.DZ);

  // W_h rows j0 .. j0+HJ-1 (all 4H columns) -> LDS: chunk (ks, q', n') holds
  // W_h[j0 + n', (4 ks + q') KPC .. +KPC].
  const int nchunks = KS * 4 * HJ;
  for (int idx = tid; idx < nchunks; idx += 256) {
    const int ks = idx / (4 * HJ);
    const int rem = idx - ks * 4 * HJ;
    const int qq = rem / HJ, n = rem - (rem / HJ) * HJ;
    lds[idx] = ld16(W + (long)(a.wrow0 + j0 + n) * G4 + (ks * 4 + qq) * KPC);
  }
  float* red = reinterpret_cast<float*>(lds + nchunks);

  const bool has_elem = tid < 16 * HJ;
  const int em = tid / HJ, eu = tid - (tid / HJ) * HJ;
  const int j = j0 + eu;
  float dh[MRT_MAX], dc[MRT_MAX];
#pragma unroll
  for (int mt = 0; mt < MRT_MAX; ++mt) {
    dh[mt] = 0.f;
    dc[mt] = 0.f;
    if (mt < a.MRT && has_elem) {
      const int r = (rg + mt * RG) * 16 + em;
      if (r < B) {
        const long b = a.perm[r];
        if (a.dhT) dh[mt] = a.dhT[b * H + j];
        if (a.dcT) dc[mt] = a.dcT[b * H + j];
      }
    }
  }
  float dbacc[4] = {0.f, 0.f, 0.f, 0.f};
  __syncthreads();

  GridBarrier gb{a.bar, a.abort_flag, a.err, gridDim.x, 0u, a.limit};
  const int T_eff = a.meta[0];
  for (int t = T_eff - 1; t >= 0; --t) {
    const int A_t = a.active[t];
    const int off_t = a.off[t];
    const int off_p = t > 0 ? a.off[t - 1] : 0;
    // phase 1
#pragma unroll
    for (int mt = 0; mt < MRT_MAX; ++mt) {
      if (mt >= a.MRT || !has_elem) continue;
      const int r = (rg + mt * RG) * 16 + em;
      if (r >= A_t) continue;
      const long krow = off_t + r;
      float dht = dh[mt];
      if (a.dy)
        dht += a.dy_compact ? a.dy[krow * H + j]
                            : a.dy[((long)t * B + a.perm[r]) * H + j];
      const float* st = a.stack + krow * 5 * H;
      const float ig = st[j], fg = st[H + j], gg = st[2 * H + j], og = st[3 * H + j];
      const float c = st[4 * H + j];
      float cp;
      if (t > 0) cp = a.stack[(long)(off_p + r) * 5 * H + 4 * H + j];
      else cp = a.c0 ? a.c0[(long)a.perm[r] * H + j] : 0.f;
      const float tc = tanhf_(c);
      const float d_o = dht * tc;
      const float dct = dc[mt] + dht * og * (1.f - tc * tc);
      const float dz0 = dct * gg * (ig * (1.f - ig));
      const float dz1 = dct * cp * (fg * (1.f - fg));
      const float dz2 = dct * ig * (1.f - gg * gg);
      const float dz3 = d_o * (og * (1.f - og));
      T* dzr = DZ + krow * G4;
      dzr[j] = Op<T>::from_f32(dz0);
      dzr[H + j] = Op<T>::from_f32(dz1);
      dzr[2 * H + j] = Op<T>::from_f32(dz2);
      dzr[3 * H + j] = Op<T>::from_f32(dz3);
      dbacc[0] += dz0;
      dbacc[1] += dz1;
      dbacc[2] += dz2;
      dbacc[3] += dz3;
      dc[mt] = dct * fg;
    }
    grid_sync(gb);
    // phase 2
#pragma unroll
    for (int mt = 0; mt < MRT_MAX; ++mt) {
      if (mt >= a.MRT) continue;
      const int r0 = (rg + mt * RG) * 16;
      if (r0 >= A_t) continue;
      f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
      const int ar = r0 + l16;
      const T* arow = ar < A_t ? DZ + (long)(off_t + ar) * G4 : nullptr;
      const bool bok = l16 < HJ;
      for (int kc = ks0; kc < ks1; kc += 8) {
        uint4 av[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const int ks = kc + i;
          av[i] = (arow && ks < ks1) ? ld16(arow + (ks * 4 + q) * KPC) : zero4();
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const int ks = kc + i;
          if (ks < ks1) {
            const uint4 bv = bok ? lds[(ks * 4 + q) * HJ + l16] : zero4();
            acc = Mfma<T>::step(av[i], bv, acc);
          }
        }
      }
#pragma unroll
      for (int e = 0; e < 4; ++e) red[(wave * 16 + q * 4 + e) * RPB + l16] = acc[e];
      __syncthreads();
      if (has_elem) {
        const int r = r0 + em;
        if (r < A_t) {
          float s = red[(0 * 16 + em) * RPB + eu];
          s += red[(1 * 16 + em) * RPB + eu];
          s += red[(2 * 16 + em) * RPB + eu];
          s += red[(3 * 16 + em) * RPB + eu];
          dh[mt] = s;
        }
      }
      __syncthreads();
    }
  }

#pragma unroll
  for (int mt = 0; mt < MRT_MAX; ++mt) {
    if (mt < a.MRT && has_elem) {
      const int r = (rg + mt * RG) * 16 + em;
      if (r < B) {
        const long b = a.perm[r];
        if (a.dh0) a.dh0[b * H + j] = dh[mt];
        if (a.dc0) a.dc0[b * H + j] = dc[mt];
      }
    }
  }
  // db partial of this work-group: sum of its rows, fixed order
  __syncthreads();
  if (has_elem) {
#pragma unroll
    for (int g = 0; g < 4; ++g) red[em * 4 * HJ + g * HJ + eu] = dbacc[g];
  }
  __syncthreads();
  for (int c = tid; c < 4 * HJ; c += 256) {
    float s = 0.f;
    for (int m = 0; m < 16; ++m) s += red[m * 4 * HJ + c];
    const int g = c / HJ, u = c - (c / HJ) * HJ;
    a.db_part[(long)rg * G4 + (long)g * H + j0 + u] = s;
  }
}

// ------------------------------------------------------------ launchers
namespace {

template <typename T>
const void* fwd_fn(int mrt) {
  if (mrt <= 1) return reinterpret_cast<const void*>(&fwd_loop_kernel<T, 1>);
  if (mrt <= 2) return reinterpret_cast<const void*>(&fwd_loop_kernel<T, 2>);
  if (mrt <= 4) return reinterpret_cast<const void*>(&fwd_loop_kernel<T, 4>);
  if (mrt <= 8) return reinterpret_cast<const void*>(&fwd_loop_kernel<T, 8>);
  return reinterpret_cast<const void*>(&fwd_loop_kernel<T, 16>);
}
template <typename T>
const void* bwd_fn(int mrt) {
  if (mrt <= 1) return reinterpret_cast<const void*>(&bwd_loop_kernel<T, 1>);
  if (mrt <= 2) return reinterpret_cast<const void*>(&bwd_loop_kernel<T, 2>);
  if (mrt <= 4) return reinterpret_cast<const void*>(&bwd_loop_kernel<T, 4>);
  if (mrt <= 8) return reinterpret_cast<const void*>(&bwd_loop_kernel<T, 8>);
  return reinterpret_cast<const void*>(&bwd_loop_kernel<T, 16>);
}

}  // namespace

template <typename T>
hipError_t loop_kernel_setup(int mrt, size_t lds_fwd, size_t lds_bwd, int* max_fwd,
                             int* max_bwd) {
  const void* f = fwd_fn<T>(mrt);
  const void* b = bwd_fn<T>(mrt);
  hipError_t e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds_fwd);
  if (e != hipSuccess) return e;
  e = hipFuncSetAttribute(b, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds_bwd);
  if (e != hipSuccess) return e;
  e = hipOccupancyMaxActiveBlocksPerMultiprocessor(max_fwd, f, 256, lds_fwd);
  if (e != hipSuccess) return e;
  return hipOccupancyMaxActiveBlocksPerMultiprocessor(max_bwd, b, 256, lds_bwd);
}

template <typename T>
hipError_t launch_fwd_loop(const FwdLoopArgs& a, int nwg, size_t lds, hipStream_t s) {
  FwdLoopArgs copy = a;
  void* kargs[] = {&copy};
  return hipLaunchCooperativeKernel(fwd_fn<T>(a.MRT), dim3(nwg), dim3(256), kargs,
                                    (unsigned)lds, s);
}

template <typename T>
hipError_t launch_bwd_loop(const BwdLoopArgs& a, int nwg, size_t lds, hipStream_t s) {
  BwdLoopArgs copy = a;
  void* kargs[] = {&copy};
  return hipLaunchCooperativeKernel(bwd_fn<T>(a.MRT), dim3(nwg), dim3(256), kargs,
                                    (unsigned)lds, s);
}

template hipError_t loop_kernel_setup<float>(int, size_t, size_t, int*, int*);
template hipError_t loop_kernel_setup<bf16_t>(int, size_t, size_t, int*, int*);
template hipError_t launch_fwd_loop<float>(const FwdLoopArgs&, int, size_t, hipStream_t);
template hipError_t launch_fwd_loop<bf16_t>(const FwdLoopArgs&, int, size_t, hipStream_t);
template hipError_t launch_bwd_loop<float>(const BwdLoopArgs&, int, size_t, hipStream_t);
template hipError_t launch_bwd_loop<bf16_t>(const BwdLoopArgs&, int, size_t, hipStream_t);

}  // namespace ll
