// Small-batch VALU kernel: the fallback for every layout and type.
#include "hd_small.hpp"

namespace hd {
namespace sp {

namespace {

// ---------------------------------------------------------------------------
// VALU kernel: NB samples per pass; 4 float4 column groups x 64 row groups.
// Thread (cg, rg) handles columns 4cg..4cg+3 of a block and rows rg + 64u.
// The thread's X values (rows rg + 64u of its NB samples) are the same for
// every block; when F fits one chunk they are loaded once into registers.
// LDS: xs[NB][FC] (only when F needs several chunks) | red[4][4][NB][16] |
//      hs[NB][17] | sl[NB*K]
// ---------------------------------------------------------------------------
template <typename T, int NB>
struct ValuBuf {
  float4 b[kRpt];
  float c[kW];
};

template <typename T, int NB, int LAY>
__global__ __launch_bounds__(kThreads, 1) void small_valu_kernel(
    const T* __restrict__ X, const T* __restrict__ B, const T* __restrict__ C,
    int32_t* __restrict__ labels, float* __restrict__ scores, int N, int F, int D, int K, int act,
    int FC, int nblocks, int lds_floats, void* __restrict__ workspace) {
  extern __shared__ __attribute__((aligned(16))) float smem[];
  const int nchunks = (F + FC - 1) / FC;
  const bool xcached = nchunks == 1;
  float* xs = smem;
  float* red = xs + (xcached ? 0 : NB * FC);  // [wave][row][NB][16]
  float* hs = red + kWaves * 4 * NB * kW;
  float* sl = hs + NB * (kW + 1);
  const SmallWs ws = small_ws(workspace);
  const ColView<T, LAY> bv{B, D, F}, cv{C, D, K};
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int cg = tid % kCG, rg = tid / kCG;
  const int G = gridDim.x;
  const BlockWalk walk = block_walk(blockIdx.x, G, nblocks);
  const bool det = (act & kActDet) != 0;
  act &= 1;
  const int R = det ? G : replicas(G, N * K);
  const int nmine = walk.count();
  const int nitems = nmine * nchunks;

  for (int nb0 = 0; nb0 < N; nb0 += NB) {
    const int nb = min(NB, N - nb0);
    const int npairs = nb * K;
    for (int p = tid; p < NB * K; p += kThreads) sl[p] = 0.0f;

    // Items are (block, chunk) pairs in this workgroup's order.
    auto load = [&](ValuBuf<T, NB>& x, int it) {
      const int blk = walk.block_of(it / nchunks), ch = it % nchunks;
      const int f0 = ch * FC, fcn = min(FC, F - f0);
#pragma unroll
      for (int u = 0; u < kRpt; ++u) {
        // rows past the chunk are clamped (their X factor is zero or the row
        // is skipped); columns past D give garbage zeroed after encoding
        const int f = rg + kRG * u;
        const int fc = f < fcn ? f : fcn - 1;
        x.b[u] = bv.get4(blk, f0 + fc, cg * 4);
      }
      load_c_pair(cv, K, blk, npairs, x.c);
    };

    ValuBuf<T, NB> b0, b1, b2;
    ring3_start(nitems, b0, b1, load);  // B is in flight while X is fetched
    float xr[kRpt][NB];
    if (xcached) {
#pragma unroll
      for (int u = 0; u < kRpt; ++u) {
        const int f = rg + kRG * u;
#pragma unroll
        for (int n = 0; n < NB; ++n) {
          const float v = load_elem(X, (int64_t)(nb0 + (n < nb ? n : 0)) * F + (f < F ? f : 0));
          xr[u][n] = (f < F && n < nb) ? v : 0.0f;
        }
      }
    }

    float acc[NB][4];
    auto process = [&](const ValuBuf<T, NB>& x, int it) {
      const int blk = walk.block_of(it / nchunks), ch = it % nchunks;
      const int f0 = ch * FC, fcn = min(FC, F - f0);
      const int64_t d0 = (int64_t)blk * kW;
      if (ch == 0) {
#pragma unroll
        for (int n = 0; n < NB; ++n) acc[n][0] = acc[n][1] = acc[n][2] = acc[n][3] = 0.0f;
      }
      if (xcached) {
#pragma unroll
        for (int u = 0; u < kRpt; ++u)
#pragma unroll
          for (int n = 0; n < NB; ++n) {
            const float xv = xr[u][n];
            acc[n][0] = fmaf(xv, x.b[u].x, acc[n][0]);
            acc[n][1] = fmaf(xv, x.b[u].y, acc[n][1]);
            acc[n][2] = fmaf(xv, x.b[u].z, acc[n][2]);
            acc[n][3] = fmaf(xv, x.b[u].w, acc[n][3]);
          }
      } else {
        __syncthreads();
        stage_rows_chunk(X, xs, FC, nb0, NB, F, N, f0, fcn);
        __syncthreads();
#pragma unroll
        for (int u = 0; u < kRpt; ++u) {
          const int f = rg + kRG * u;
          if (f < fcn) {
#pragma unroll
            for (int n = 0; n < NB; ++n) {
              const float xv = xs[n * FC + f];
              acc[n][0] = fmaf(xv, x.b[u].x, acc[n][0]);
              acc[n][1] = fmaf(xv, x.b[u].y, acc[n][1]);
              acc[n][2] = fmaf(xv, x.b[u].z, acc[n][2]);
              acc[n][3] = fmaf(xv, x.b[u].w, acc[n][3]);
            }
          }
        }
      }
      if (ch != nchunks - 1) return;
      // Lane l of a wave is (cg = l%4, row group = l/4). DPP sums the 4 row
      // groups of each 16-lane row; lanes 0..3 of each row then hold the
      // row's partial for their columns.
      __syncthreads();  // previous block's readers of red / hs are done
#pragma unroll
      for (int n = 0; n < NB; ++n)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const float v = row_sum4(acc[n][q]);
          if ((lane & 15) < kCG)
            red[((wave * 4 + (lane >> 4)) * NB + n) * kW + (lane & 3) * 4 + q] = v;
        }
      __syncthreads();
      for (int i = tid; i < NB * kW; i += kThreads) {
        const int n = i / kW, c = i % kW;
        float v = 0.0f;
#pragma unroll
        for (int w = 0; w < kWaves * 4; ++w) v += red[(w * NB + n) * kW + c];
        hs[n * (kW + 1) + c] = (d0 + c < D && n < nb) ? activate(v, act) : 0.0f;
      }
      __syncthreads();
      block_scores(cv, hs, sl, npairs, K, blk, x.c);
    };

    ring3_run(nitems, b0, b1, b2, load, process);
    __syncthreads();
    publish_and_finish(sl, nb0, nb, N, K, R, ws, labels, scores, smem, lds_floats,
                       nb0 + NB >= N, det);
  }
}


template <typename T, int NB, int LAY>
hipError_t launch_valu(const SmallPlan& p, const Args& a) {
  const hipError_t attr = allow_lds<&small_valu_kernel<T, NB, LAY>>();
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL((small_valu_kernel<T, NB, LAY>), dim3(p.grid), dim3(kThreads), p.lds,
                     a.stream, (const T*)a.X, (const T*)a.B, (const T*)a.C, a.labels, a.scores,
                     a.N, a.F, a.D, a.K, a.act, p.FC, p.nblocks, (int)(p.lds / sizeof(float)),
                     a.ws);
  return hipGetLastError();
}

template <typename T, int LAY>
hipError_t launch_valu_nb(const SmallPlan& p, const Args& a) {
  if constexpr (LAY == kRawScalar) {  // at most 2 samples per pass (register budget)
    return p.nb == 1 ? launch_valu<T, 1, LAY>(p, a) : launch_valu<T, 2, LAY>(p, a);
  } else {
    switch (p.nb) {
      case 1: return launch_valu<T, 1, LAY>(p, a);
      case 2: return launch_valu<T, 2, LAY>(p, a);
      case 4: return launch_valu<T, 4, LAY>(p, a);
      default: return launch_valu<T, 8, LAY>(p, a);
    }
  }
}

}  // namespace

hipError_t launch_valu_family(SmallPlan& p, const Args& a, int dt, int lay) {
  widen_for_final(p, a.N, a.K);
  if (dt == 0) {
    switch (lay) {
      case kTiled: return launch_valu_nb<float, kTiled>(p, a);
      case kRawVec: return launch_valu_nb<float, kRawVec>(p, a);
      default: return launch_valu_nb<float, kRawScalar>(p, a);
    }
  }
  switch (lay) {
    case kTiled: return launch_valu_nb<bf16raw, kTiled>(p, a);
    case kRawVec: return launch_valu_nb<bf16raw, kRawVec>(p, a);
    default: return launch_valu_nb<bf16raw, kRawScalar>(p, a);
  }
}

}  // namespace sp
}  // namespace hd
