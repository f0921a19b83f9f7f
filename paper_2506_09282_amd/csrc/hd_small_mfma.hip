// Small-batch matrix-core kernels on B as given or column-tiled.
#include "hd_small.hpp"

namespace hd {
namespace sp {

namespace {

// ---------------------------------------------------------------------------
// Matrix-core kernel (fp32, 8 < N <= 64): NTI sample tiles of 16, MS 4-row
// steps per wave. Wave w accumulates V^T[16 d x 16 n] per sample tile over
// its quarter of the F rows; the waves' partials are summed through LDS.
//   A operand (16x16x4 f32): lane l holds B[f0 + l/16][d0 + l%16]
//   B operand: lane l holds X[16t + l%16][f0 + l/16]; these values do not
//     depend on the column block, so each wave loads them once into registers
//   result: lane l, reg r holds V^T[d0 + 4(l/16) + r][16t + l%16]
// LDS: red[4][NTI][16][16] | hs[16*NTI][17] | sl[16*NTI*K]
// ---------------------------------------------------------------------------
template <int MS>
struct MfmaBuf {
  float a[MS];
  float c[kW];
};

template <int NTI, int MS, int LAY>
__global__ __launch_bounds__(kThreads, 1) void small_mfma_kernel(
    const float* __restrict__ X, const float* __restrict__ B, const float* __restrict__ C,
    int32_t* __restrict__ labels, float* __restrict__ scores, int N, int F, int D, int K, int act,
    int nblocks, int lds_floats, void* __restrict__ workspace) {
  constexpr int NB = 16 * NTI;
  constexpr int FQ = 4 * MS;                  // rows per wave
  extern __shared__ __attribute__((aligned(16))) float smem[];
  float* sl = smem;                                // [NB*K]
  float* red = sl + (NB * K + 3) / 4 * 4;          // [4][NTI][256]
  float* hs = red + kWaves * NTI * 256;            // [NB][17]
  float* xs = red;  // [nb][F]: X rows, only until the operands are in registers
  const SmallWs ws = small_ws(workspace);
  const ColView<float, LAY> bv{B, D, F}, cv{C, D, K};
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int G = gridDim.x;
  const BlockWalk walk = block_walk(blockIdx.x, G, nblocks);
  const bool det = (act & kActDet) != 0;
  act &= 1;
  const int R = det ? G : replicas(G, N * K);
  const int nb = min(NB, N);
  const int npairs = nb * K;
  const int arow = wave * FQ + (lane >> 4);  // A-operand row of step 0
  const int acol = lane & 15;
  const int nmine = walk.count();

  auto load = [&](MfmaBuf<MS>& x, int i) {
    const int blk = walk.block_of(i);
#pragma unroll
    for (int s = 0; s < MS; ++s) {
      // rows past F are clamped and meet zero X values; columns past D give
      // garbage that is zeroed after encoding
      const int f = arow + 4 * s;
      x.a[s] = bv.get(blk, f < F ? f : F - 1, acol);
    }
    load_c_pair(cv, K, blk, npairs, x.c);
  };

  // B is in flight while X (rows 0..nb-1, one contiguous range) is copied to
  // LDS and each wave's operand values are read back into registers.
  MfmaBuf<MS> b0, b1, b2;
  ring3_start(nmine, b0, b1, load);
  for (int p = tid; p < NB * K; p += kThreads) sl[p] = 0.0f;
  copy_flat_to_lds(X, xs, nb * F);
  __syncthreads();
  float xr[MS][NTI];
#pragma unroll
  for (int s = 0; s < MS; ++s)
#pragma unroll
    for (int t = 0; t < NTI; ++t) {
      const int n = 16 * t + (lane & 15), f = arow + 4 * s;
      const float v = xs[(n < nb ? n : 0) * F + (f < F ? f : 0)];
      xr[s][t] = (n < nb && f < F) ? v : 0.0f;
    }

  auto process = [&](const MfmaBuf<MS>& x, int i) {
    const int blk = walk.block_of(i);
    const int64_t d0 = (int64_t)blk * kW;
    f32x4 acc[NTI];
#pragma unroll
    for (int t = 0; t < NTI; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < MS; ++s)
#pragma unroll
      for (int t = 0; t < NTI; ++t)
        acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(x.a[s], xr[s][t], acc[t], 0, 0, 0);
    __syncthreads();  // previous block's readers of red / hs are done
#pragma unroll
    for (int t = 0; t < NTI; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        red[(wave * NTI + t) * 256 + (4 * (lane >> 4) + r) * 16 + (lane & 15)] = acc[t][r];
    __syncthreads();
    for (int e = tid; e < NB * kW; e += kThreads) {
      const int n = e / kW, c = e % kW;
      const int t = n / 16, j = n % 16;
      float v = 0.0f;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) v += red[(w * NTI + t) * 256 + c * 16 + j];
      hs[n * (kW + 1) + c] = (d0 + c < D && n < nb) ? activate(v, act) : 0.0f;
    }
    __syncthreads();
    block_scores(cv, hs, sl, npairs, K, blk, x.c);
  };

  ring3_run(nmine, b0, b1, b2, load, process);
  __syncthreads();
  publish_and_finish(sl, 0, nb, N, K, R, ws, labels, scores, smem, lds_floats, true, det);
}


// ---------------------------------------------------------------------------
// Block matrix-core kernel (fp32, 8 < N <= 32, one column block per
// workgroup). Same operand mapping as small_mfma_kernel; X (all nb rows, one
// contiguous range) is loaded first, since it is shared by every workgroup
// and hits L2, then the block's B rows and C values, so the X wait does not
// wait for B. X passes through LDS into registers; the LDS then holds the
// wave partials.
// LDS: xs[nb][F] during staging, then red[4][NTI][256] | hs[16*NTI][17]
// ---------------------------------------------------------------------------
template <int NTI, int MS, int LAY>
__global__ __launch_bounds__(kThreads) void small_block_mfma_kernel(
    const float* __restrict__ X, const float* __restrict__ B, const float* __restrict__ C,
    int32_t* __restrict__ labels, float* __restrict__ scores, int N, int F, int D, int K, int act,
    int lds_floats, void* __restrict__ workspace) {
  constexpr int NB = 16 * NTI;
  constexpr int FQ = 4 * MS;  // rows per wave
  constexpr int XV = NTI * MS / 4;  // float4 of X per thread: 16 NTI rows of up to 16 MS
  extern __shared__ __attribute__((aligned(16))) float smem[];
  float* xs = smem;
  float* red = smem;
  float* hs = red + kWaves * NTI * 256;
  const SmallWs ws = small_ws(workspace);
  const ColView<float, LAY> bv{B, D, F}, cv{C, D, K};
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int G = gridDim.x;
  const int blk = xcd_block(blockIdx.x, G);
  const bool det = (act & kActDet) != 0;
  act &= 1;
  const int R = det ? G : replicas(G, N * K);
  const int nb = min(NB, N);
  const int npairs = nb * K;
  const int arow = wave * FQ + (lane >> 4);
  const int acol = lane & 15;
  const int64_t d0 = (int64_t)blk * kW;

  // 1. X: XV float4 per thread, addresses clamped
  const int n4 = nb * F / 4;
  const int rot = x_rotation(n4);
  const float4* x4 = reinterpret_cast<const float4*>(X);
  float4 xv[XV];
  int at[XV];
#pragma unroll
  for (int j = 0; j < XV; ++j) {
    const int i = j * kThreads + tid;
    const int r = i + rot >= n4 ? i + rot - n4 : i + rot;
    at[j] = i < n4 ? r : n4;
    xv[j] = x4[i < n4 ? r : 0];
  }
  // keep the X loads ahead of the B loads (the wait for X must not wait for B)
  __builtin_amdgcn_sched_barrier(0);
  // 2. B rows (A operand) and the pair's C values
  float a[MS];
#pragma unroll
  for (int s = 0; s < MS; ++s) {
    // rows past F are clamped and meet zero X values; columns past D give
    // garbage that is zeroed after encoding
    const int f = arow + 4 * s;
    a[s] = bv.get(blk, f < F ? f : F - 1, acol);
  }
  float cpair[kW];
  load_c_pair(cv, K, blk, npairs, cpair);

  // 3. X to LDS, then the wave's operand values to registers. Stores are
  // unconditional (a branch per store lets the compiler sink each load to its
  // store); threads past the end write the spare slot after X.
#pragma unroll
  for (int j = 0; j < XV; ++j) reinterpret_cast<float4*>(xs)[at[j]] = xv[j];
  for (int i = 4 * n4 + tid; i < nb * F; i += kThreads) xs[i] = X[i];
  __syncthreads();
  float xr[MS][NTI];
#pragma unroll
  for (int s = 0; s < MS; ++s)
#pragma unroll
    for (int t = 0; t < NTI; ++t) {
      const int n = 16 * t + (lane & 15), f = arow + 4 * s;
      const float v = xs[(n < nb ? n : 0) * F + (f < F ? f : 0)];
      xr[s][t] = (n < nb && f < F) ? v : 0.0f;
    }

  // 4. V^T tiles over the wave's rows, summed over the waves through LDS
  f32x4 acc[NTI];
#pragma unroll
  for (int t = 0; t < NTI; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < MS; ++s)
#pragma unroll
    for (int t = 0; t < NTI; ++t)
      acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[s], xr[s][t], acc[t], 0, 0, 0);
  __syncthreads();  // every wave has read its X values: xs becomes red
#pragma unroll
  for (int t = 0; t < NTI; ++t)
#pragma unroll
    for (int r = 0; r < 4; ++r)
      red[(wave * NTI + t) * 256 + (4 * (lane >> 4) + r) * 16 + (lane & 15)] = acc[t][r];
  __syncthreads();
  for (int e = tid; e < NB * kW; e += kThreads) {
    const int n = e / kW, c = e % kW;
    const int t = n / 16, j = n % 16;
    float v = 0.0f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) v += red[(w * NTI + t) * 256 + c * 16 + j];
    hs[n * (kW + 1) + c] = (d0 + c < D && n < nb) ? activate(v, act) : 0.0f;
  }
  __syncthreads();

  // 5. partial scores of this block straight to the replica
  float* my = ws.sacc + (int64_t)(blockIdx.x % R) * N * K;
  for (int p = tid; p < npairs; p += kThreads) {
    const int n = p / K, k = p - n * K;
    float sc = 0.0f;
    if (p == tid) {
#pragma unroll
      for (int j = 0; j < kW; ++j) sc = fmaf(hs[n * (kW + 1) + j], cpair[j], sc);
    } else {
#pragma unroll
      for (int j = 0; j < kW; ++j) sc = fmaf(hs[n * (kW + 1) + j], cv.get(blk, k, j), sc);
    }
    publish_add(my + p, sc);
  }
  float none[1] = {0.0f};
  publish_and_finish(none, 0, 0, N, K, R, ws, labels, scores, smem, lds_floats, true, det);
}


template <int NTI, int MS, int LAY>
hipError_t launch_mfma(const SmallPlan& p, const Args& a) {
  const hipError_t attr = allow_lds<&small_mfma_kernel<NTI, MS, LAY>>();
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL((small_mfma_kernel<NTI, MS, LAY>), dim3(p.grid), dim3(kThreads), p.lds,
                     a.stream, (const float*)a.X, (const float*)a.B, (const float*)a.C, a.labels,
                     a.scores, a.N, a.F, a.D, a.K, a.act, p.nblocks, (int)(p.lds / sizeof(float)),
                     a.ws);
  return hipGetLastError();
}

template <int NTI, int LAY>
hipError_t launch_mfma_ms(const SmallPlan& p, const Args& a) {
  switch (p.ms) {
    case 12: return launch_mfma<NTI, 12, LAY>(p, a);
    case 24: return launch_mfma<NTI, 24, LAY>(p, a);
    case 36: return launch_mfma<NTI, 36, LAY>(p, a);
    default: return launch_mfma<NTI, 48, LAY>(p, a);
  }
}

template <int LAY>
hipError_t launch_mfma_nti(const SmallPlan& p, const Args& a) {
  switch (p.nb) {
    case 1: return launch_mfma_ms<1, LAY>(p, a);
    case 2: return launch_mfma_ms<2, LAY>(p, a);
    case 3: return launch_mfma_ms<3, LAY>(p, a);
    default: return launch_mfma_ms<4, LAY>(p, a);
  }
}

template <int NTI, int MS, int LAY>
hipError_t launch_bmfma(const SmallPlan& p, const Args& a) {
  const hipError_t attr = allow_lds<&small_block_mfma_kernel<NTI, MS, LAY>>();
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL((small_block_mfma_kernel<NTI, MS, LAY>), dim3(p.grid), dim3(kThreads), p.lds,
                     a.stream, (const float*)a.X, (const float*)a.B, (const float*)a.C, a.labels,
                     a.scores, a.N, a.F, a.D, a.K, a.act, (int)(p.lds / sizeof(float)), a.ws);
  return hipGetLastError();
}

template <int NTI, int LAY>
hipError_t launch_bmfma_ms(const SmallPlan& p, const Args& a) {
  switch (p.ms) {
    case 12: return launch_bmfma<NTI, 12, LAY>(p, a);
    case 24: return launch_bmfma<NTI, 24, LAY>(p, a);
    case 36: return launch_bmfma<NTI, 36, LAY>(p, a);
    default: return launch_bmfma<NTI, 48, LAY>(p, a);
  }
}

}  // namespace

hipError_t launch_mfma_family(SmallPlan& p, const Args& a, int lay) {
  widen_for_final(p, a.N, a.K);
  return lay == kTiled ? launch_mfma_nti<kTiled>(p, a) : launch_mfma_nti<kRawVec>(p, a);
}

hipError_t launch_bmfma_family(SmallPlan& p, const Args& a, int lay) {
  widen_for_final(p, a.N, a.K);
  if (lay == kTiled)
    return p.nb == 1 ? launch_bmfma_ms<1, kTiled>(p, a) : launch_bmfma_ms<2, kTiled>(p, a);
  return p.nb == 1 ? launch_bmfma_ms<1, kRawVec>(p, a) : launch_bmfma_ms<2, kRawVec>(p, a);
}

}  // namespace sp
}  // namespace hd
