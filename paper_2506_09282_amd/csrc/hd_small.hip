// Small-batch fused inference (N <= 64): the GPU form of the paper's
// small-batch variant (Sec. III-C, Alg. 3), which splits the hypervector
// dimension D across workers and sums their partial score matrices.
//
// One workgroup owns 32 consecutive columns of B (a "column block" of the
// encoded matrix, Alg. 2) and all F rows of it, so its encoding sums are
// complete and HardSign (Eq. 1) is applied in registers: H never leaves the
// chip. B is read exactly once, as coalesced 128-byte row segments (fp32).
// Each workgroup then forms its partial S over its 32 columns and adds it,
// with fp32 atomics, into one of R replicated accumulators (R spreads the
// atomic traffic over many cache lines). The last workgroup to finish (an
// atomic ticket) sums the replicas, takes the row argmax (Eq. 9), writes
// labels/scores and re-zeroes the accumulators and the ticket.
#include "hd_common.hpp"
#include "hd_internal.hpp"

namespace hd {

namespace {

constexpr int kThreads = 256;
constexpr int kColGroups = kSmallCols / 4;         // 8 groups of 4 columns
constexpr int kRowGroups = kThreads / kColGroups;  // 32 row groups
constexpr int kRowsPerBatch = 8;                   // B rows per thread per load batch
constexpr int kXsFloats = 16384;                   // LDS budget for the staged X^T chunk

template <int NB>
constexpr int xs_pitch() {
  return NB >= 4 ? NB + 4 : NB;
}

struct SmallWs {
  unsigned* counter;
  float* sacc;  // [R][N][K]
};

__host__ __device__ inline SmallWs small_ws(void* ws) {
  SmallWs w;
  w.counter = reinterpret_cast<unsigned*>(ws);
  w.sacc = reinterpret_cast<float*>(reinterpret_cast<char*>(ws) + 256);
  return w;
}

template <typename T, bool VEC>
__device__ __forceinline__ float4 load_b4(const T* __restrict__ B, int64_t row, int64_t col,
                                          int64_t D) {
  if (VEC) {
    if (col < D) return load4(B, row * D + col);
    return make_float4(0.f, 0.f, 0.f, 0.f);
  }
  float v[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) v[q] = (col + q < D) ? load_elem(B, row * D + col + q) : 0.0f;
  return make_float4(v[0], v[1], v[2], v[3]);
}

template <typename T, int NB, bool VEC>
__global__ __launch_bounds__(kThreads) void small_fused_kernel(
    const T* __restrict__ X, const T* __restrict__ B, const T* __restrict__ C,
    int32_t* __restrict__ labels, float* __restrict__ scores, int N, int F, int D, int K, int act,
    int FC, void* __restrict__ workspace) {
  constexpr int P = xs_pitch<NB>();
  extern __shared__ float smem[];
  float* xs = smem;                              // [FC][P]   X^T chunk
  float* red = xs + FC * P;                      // [4][NB][32] per-wave column sums
  float* hs = red + 4 * NB * kSmallCols;         // [NB][33]  encoded block
  __shared__ int s_last;

  const SmallWs ws = small_ws(workspace);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int cg = tid % kColGroups, rg = tid / kColGroups;
  const int g = blockIdx.x;
  const int64_t d0 = (int64_t)g * kSmallCols;
  const int64_t dcol = d0 + cg * 4;
  const int R = gridDim.x < kSmallReplicas ? (int)gridDim.x : kSmallReplicas;
  float* my_sacc = ws.sacc + (int64_t)(g % R) * N * K;

  for (int nb0 = 0; nb0 < N; nb0 += NB) {
    float acc[NB][4];
#pragma unroll
    for (int n = 0; n < NB; ++n) acc[n][0] = acc[n][1] = acc[n][2] = acc[n][3] = 0.0f;

    for (int fc0 = 0; fc0 < F; fc0 += FC) {
      const int fcn = min(FC, F - fc0);
      const int jmax = (fcn + kRowGroups - 1) / kRowGroups;  // row batches are uniform
      float4 b0[kRowsPerBatch], b1[kRowsPerBatch];
      auto load_batch = [&](float4(&dst)[kRowsPerBatch], int j0) {
#pragma unroll
        for (int u = 0; u < kRowsPerBatch; ++u) {
          const int f = rg + kRowGroups * (j0 + u);
          dst[u] = (f < fcn) ? load_b4<T, VEC>(B, fc0 + f, dcol, D) : make_float4(0.f, 0.f, 0.f, 0.f);
        }
      };
      auto compute_batch = [&](const float4(&src)[kRowsPerBatch], int j0) {
#pragma unroll
        for (int u = 0; u < kRowsPerBatch; ++u) {
          const int f = rg + kRowGroups * (j0 + u);
          if (f < fcn) {
            const float* xrow = xs + f * P;
#pragma unroll
            for (int n = 0; n < NB; ++n) {
              const float x = xrow[n];
              acc[n][0] = fmaf(x, src[u].x, acc[n][0]);
              acc[n][1] = fmaf(x, src[u].y, acc[n][1]);
              acc[n][2] = fmaf(x, src[u].z, acc[n][2]);
              acc[n][3] = fmaf(x, src[u].w, acc[n][3]);
            }
          }
        }
      };

      // Issue the first B batch before staging X so both latencies overlap.
      load_batch(b0, 0);
      __syncthreads();  // previous readers of xs are done
      for (int i = tid; i < NB * fcn; i += kThreads) {
        const int n = i / fcn, f = i - n * fcn;
        xs[f * P + n] = (nb0 + n < N) ? load_elem(X, (int64_t)(nb0 + n) * F + fc0 + f) : 0.0f;
      }
      __syncthreads();
      for (int j0 = 0; j0 < jmax; j0 += 2 * kRowsPerBatch) {
        const bool more1 = j0 + kRowsPerBatch < jmax;
        if (more1) load_batch(b1, j0 + kRowsPerBatch);
        compute_batch(b0, j0);
        if (more1) {
          if (j0 + 2 * kRowsPerBatch < jmax) load_batch(b0, j0 + 2 * kRowsPerBatch);
          compute_batch(b1, j0 + kRowsPerBatch);
        }
      }
    }

    // Sum the 8 row groups of this wave (lanes differing in bits 3..5).
#pragma unroll
    for (int n = 0; n < NB; ++n)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        float v = acc[n][q];
        v += __shfl_xor(v, 8, kWave);
        v += __shfl_xor(v, 16, kWave);
        v += __shfl_xor(v, 32, kWave);
        acc[n][q] = v;
      }
    if (lane < kColGroups) {
#pragma unroll
      for (int n = 0; n < NB; ++n)
#pragma unroll
        for (int q = 0; q < 4; ++q) red[(wave * NB + n) * kSmallCols + lane * 4 + q] = acc[n][q];
    }
    __syncthreads();
    for (int i = tid; i < NB * kSmallCols; i += kThreads) {
      const int n = i / kSmallCols, c = i % kSmallCols;
      const float v = (red[(0 * NB + n) * kSmallCols + c] + red[(1 * NB + n) * kSmallCols + c]) +
                      (red[(2 * NB + n) * kSmallCols + c] + red[(3 * NB + n) * kSmallCols + c]);
      const bool valid = (d0 + c < D) && (nb0 + n < N);
      hs[n * 33 + c] = valid ? activate(v, act) : 0.0f;
    }
    __syncthreads();
    // Partial similarity of this column block (Eq. 8 restricted to 32 dims).
    const int ncols = (int)min((int64_t)kSmallCols, (int64_t)D - d0);
    for (int p = tid; p < NB * K; p += kThreads) {
      const int n = p / K, k = p - n * K;
      if (nb0 + n >= N) continue;
      const T* crow = C + (int64_t)k * D + d0;
      const float* hrow = hs + n * 33;
      float s = 0.0f;
      for (int c = 0; c < ncols; ++c) s = fmaf(hrow[c], load_elem(crow, c), s);
      unsafeAtomicAdd(my_sacc + (int64_t)(nb0 + n) * K + k, s);
    }
  }

  // Ticket: the last workgroup to arrive finishes the reduction.
  __threadfence();
  __syncthreads();
  if (tid == 0) s_last = (atomicAdd(ws.counter, 1u) == gridDim.x - 1) ? 1 : 0;
  __syncthreads();
  if (!s_last) return;
  __threadfence();

  const int64_t NK = (int64_t)N * K;
  for (int n = wave; n < N; n += kThreads / kWave) {
    float best = -__builtin_huge_valf();
    int best_k = 0x7fffffff;
    for (int k = lane; k < K; k += kWave) {
      float s = 0.0f;
      for (int r = 0; r < R; ++r) s += load_coherent(ws.sacc + r * NK + (int64_t)n * K + k);
      if (scores) scores[(int64_t)n * K + k] = s;
      if (k == lane || s > best) {
        best = s;
        best_k = k;
      }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      const float ob = __shfl_xor(best, off, kWave);
      const int ok = __shfl_xor(best_k, off, kWave);
      if (ob > best || (ob == best && ok < best_k)) {
        best = ob;
        best_k = ok;
      }
    }
    if (lane == 0) labels[n] = best_k;
  }
  __syncthreads();
  for (int64_t i = tid; i < (int64_t)R * NK; i += kThreads) store_coherent(ws.sacc + i, 0.0f);
  if (tid == 0) __hip_atomic_store(ws.counter, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

template <typename T, int NB, bool VEC>
hipError_t launch_nb(const void* X, const void* B, const void* C, int32_t* labels, float* scores,
                     int N, int F, int D, int K, int act, void* ws, hipStream_t stream) {
  constexpr int P = xs_pitch<NB>();
  int FC = kXsFloats / P;
  if (FC > F) FC = F;
  const size_t lds = sizeof(float) * ((size_t)FC * P + 4 * NB * kSmallCols + NB * 33);
  const int G = (int)cdiv(D, kSmallCols);
  static const hipError_t attr = hipFuncSetAttribute(
      reinterpret_cast<const void*>(&small_fused_kernel<T, NB, VEC>),
      hipFuncAttributeMaxDynamicSharedMemorySize, 96 * 1024);
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL((small_fused_kernel<T, NB, VEC>), dim3(G), dim3(kThreads), lds, stream,
                     (const T*)X, (const T*)B, (const T*)C, labels, scores, N, F, D, K, act, FC,
                     ws);
  return hipGetLastError();
}

template <typename T, bool VEC>
hipError_t launch_t(const void* X, const void* B, const void* C, int32_t* labels, float* scores,
                    int N, int F, int D, int K, int act, void* ws, hipStream_t stream) {
  if (N <= 1) return launch_nb<T, 1, VEC>(X, B, C, labels, scores, N, F, D, K, act, ws, stream);
  if (N <= 2) return launch_nb<T, 2, VEC>(X, B, C, labels, scores, N, F, D, K, act, ws, stream);
  if (N <= 4) return launch_nb<T, 4, VEC>(X, B, C, labels, scores, N, F, D, K, act, ws, stream);
  if (N <= 8) return launch_nb<T, 8, VEC>(X, B, C, labels, scores, N, F, D, K, act, ws, stream);
  if (N <= 16) return launch_nb<T, 16, VEC>(X, B, C, labels, scores, N, F, D, K, act, ws, stream);
  return launch_nb<T, 32, VEC>(X, B, C, labels, scores, N, F, D, K, act, ws, stream);
}

}  // namespace

size_t small_workspace_bytes(int64_t N, int64_t F, int64_t D, int64_t K) {
  (void)F;
  const int64_t G = cdiv(D, kSmallCols);
  const int64_t R = G < kSmallReplicas ? G : kSmallReplicas;
  return 256 + sizeof(float) * (size_t)(R * N * K);
}

hipError_t launch_small(const void* X, const void* B, const void* C, int32_t* labels,
                        float* scores, int64_t N, int64_t F, int64_t D, int64_t K, int dt,
                        int act, void* workspace, hipStream_t stream) {
  const size_t align = dt == 0 ? 16 : 8;
  const bool vec = (D % 4 == 0) && ((uintptr_t)B % align == 0);
  const int n = (int)N, f = (int)F, d = (int)D, k = (int)K;
  if (dt == 0)
    return vec ? launch_t<float, true>(X, B, C, labels, scores, n, f, d, k, act, workspace, stream)
               : launch_t<float, false>(X, B, C, labels, scores, n, f, d, k, act, workspace, stream);
  return vec ? launch_t<bf16raw, true>(X, B, C, labels, scores, n, f, d, k, act, workspace, stream)
             : launch_t<bf16raw, false>(X, B, C, labels, scores, n, f, d, k, act, workspace, stream);
}

}  // namespace hd
