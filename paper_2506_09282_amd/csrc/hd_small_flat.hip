// Small-batch flat kernel (N <= 8): one column block per workgroup.
#include "hd_small.hpp"

namespace hd {
namespace sp {

namespace {

// ---------------------------------------------------------------------------
// Flat kernel (N <= 8, one column block per workgroup). Every load a
// workgroup needs (its block of B, its rows of X, its pairs' C values) is
// issued at entry; several workgroups share a CU, so the hardware overlaps
// them. Thread (cg, rg) handles columns 4cg..4cg+3 and rows rg + 64u of
// each f-chunk of 64*RPT rows.
// LDS: red[16][NB][16] | hs[NB][17]
// ---------------------------------------------------------------------------
template <typename T, int NB, int RPT, int LAY>
__global__ __launch_bounds__(kThreads) void small_flat_kernel(
    const T* __restrict__ X, const T* __restrict__ B, const T* __restrict__ C,
    int32_t* __restrict__ labels, float* __restrict__ scores, int N, int F, int D, int K, int act,
    void* __restrict__ workspace) {
  constexpr int kChunk = kRG * RPT;
  __shared__ float red[kWaves * 4 * NB * kW];
  __shared__ float hs[NB * (kW + 1)];
  const SmallWs ws = small_ws(workspace);
  const ColView<T, LAY> bv{B, D, F}, cv{C, D, K};
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int cg = tid % kCG, rg = tid / kCG;
  const int G = gridDim.x;
  const int blk = xcd_block(blockIdx.x, G);
  const bool det = (act & kActDet) != 0;
  act &= 1;
  const int R = det ? G : replicas(G, N * K);
  const int64_t d0 = (int64_t)blk * kW;
  const int npairs = N * K;

  float cpair[kW];
  load_c_pair(cv, K, blk, npairs, cpair);
  float acc[NB][4];
#pragma unroll
  for (int n = 0; n < NB; ++n) acc[n][0] = acc[n][1] = acc[n][2] = acc[n][3] = 0.0f;
  for (int f0 = 0; f0 < F; f0 += kChunk) {
    float4 b[RPT];
    float x[RPT][NB];
#pragma unroll
    for (int u = 0; u < RPT; ++u) {
      // rows past F are clamped and get a zero X factor; columns past D
      // give garbage that is zeroed after encoding
      const int f = f0 + rg + kRG * u;
      const int fc = f < F ? f : F - 1;
      b[u] = bv.get4(blk, fc, cg * 4);
    }
#pragma unroll
    for (int u = 0; u < RPT; ++u) {
      const int f = f0 + rg + kRG * u;
#pragma unroll
      for (int n = 0; n < NB; ++n) {
        const float v = load_elem(X, (int64_t)(n < N ? n : 0) * F + (f < F ? f : 0));
        x[u][n] = (f < F && n < N) ? v : 0.0f;
      }
    }
#pragma unroll
    for (int u = 0; u < RPT; ++u)
#pragma unroll
      for (int n = 0; n < NB; ++n) {
        acc[n][0] = fmaf(x[u][n], b[u].x, acc[n][0]);
        acc[n][1] = fmaf(x[u][n], b[u].y, acc[n][1]);
        acc[n][2] = fmaf(x[u][n], b[u].z, acc[n][2]);
        acc[n][3] = fmaf(x[u][n], b[u].w, acc[n][3]);
      }
  }
  // lanes 16r..16r+15 hold 4 row groups x 4 column groups: DPP sums the row
  // groups, then the 16 (wave, row) partials are summed through LDS
#pragma unroll
  for (int n = 0; n < NB; ++n)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float v = row_sum4(acc[n][q]);
      if ((lane & 15) < kCG) red[((wave * 4 + (lane >> 4)) * NB + n) * kW + (lane & 3) * 4 + q] = v;
    }
  __syncthreads();
  if (tid < NB * kW) {
    const int n = tid / kW, c = tid % kW;
    float v = 0.0f;
#pragma unroll
    for (int w = 0; w < kWaves * 4; ++w) v += red[(w * NB + n) * kW + c];
    hs[n * (kW + 1) + c] = (d0 + c < D && n < N) ? activate(v, act) : 0.0f;
  }
  __syncthreads();
  float* my = ws.sacc + (int64_t)(blockIdx.x % R) * N * K;
  if (tid < npairs) {
    const int n = tid / K;
    float sc = 0.0f;
#pragma unroll
    for (int j = 0; j < kW; ++j) sc = fmaf(hs[n * (kW + 1) + j], cpair[j], sc);
    publish_add(my + tid, sc);
  }
  for (int p = tid + kThreads; p < npairs; p += kThreads) {
    const int n = p / K, k = p - n * K;
    float sc = 0.0f;
#pragma unroll
    for (int j = 0; j < kW; ++j) sc = fmaf(hs[n * (kW + 1) + j], cv.get(blk, k, j), sc);
    publish_add(my + p, sc);
  }
  float none[1] = {0.0f};
  publish_and_finish(none, 0, 0, N, K, R, ws, labels, scores, red, kWaves * 4 * NB * kW, true,
                     det);
}


template <typename T, int NB, int RPT, int LAY>
hipError_t launch_flat(const SmallPlan& p, const Args& a) {
  hipLaunchKernelGGL((small_flat_kernel<T, NB, RPT, LAY>), dim3(p.grid), dim3(kThreads), 0,
                     a.stream, (const T*)a.X, (const T*)a.B, (const T*)a.C, a.labels, a.scores,
                     a.N, a.F, a.D, a.K, a.act, a.ws);
  return hipGetLastError();
}

template <typename T, int NB, int LAY>
hipError_t launch_flat_rpt(const SmallPlan& p, const Args& a) {
  switch (p.rpt) {
    case 4: return launch_flat<T, NB, 4, LAY>(p, a);
    case 9: return launch_flat<T, NB, 9, LAY>(p, a);
    default: return launch_flat<T, NB, 16, LAY>(p, a);
  }
}

template <typename T, int LAY>
hipError_t launch_flat_nb(const SmallPlan& p, const Args& a) {
  switch (p.nb) {
    case 1: return launch_flat_rpt<T, 1, LAY>(p, a);
    case 2: return launch_flat_rpt<T, 2, LAY>(p, a);
    case 4: return launch_flat_rpt<T, 4, LAY>(p, a);
    default: return launch_flat_rpt<T, 8, LAY>(p, a);
  }
}

}  // namespace

hipError_t launch_flat_family(const SmallPlan& p, const Args& a, int dt, int lay) {
  if (dt == 0)
    return lay == kTiled ? launch_flat_nb<float, kTiled>(p, a) : launch_flat_nb<float, kRawVec>(p, a);
  return lay == kTiled ? launch_flat_nb<bf16raw, kTiled>(p, a) : launch_flat_nb<bf16raw, kRawVec>(p, a);
}

}  // namespace sp
}  // namespace hd
