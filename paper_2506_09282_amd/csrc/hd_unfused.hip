// Unfused stages: Stage I writes H to device memory (hd_encode), Stage II
// reads it back (hd_similarity). Used for tests and hand composition; the
// fused kernels never materialise H.
#include "hd_common.hpp"
#include "hd_internal.hpp"

namespace hd {

// ---------------------------------------------------------------------------
// Stage I (Eq. 7 with Eq. 1): H[n,d] = act(sum_f X[n,f] B[f,d]).
// 64x64 output tile per workgroup, 256 threads with a 4x4 register tile each,
// F streamed through LDS in steps of 16. Grid-stride over tiles.
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void encode_kernel(const T* __restrict__ X,
                                                     const T* __restrict__ B,
                                                     float* __restrict__ H, int64_t N, int64_t F,
                                                     int64_t D, int act, int64_t tiles_d,
                                                     int64_t total_tiles) {
  constexpr int BM = 64, BN = 64, BK = 16;
  __shared__ float xs[BK][BM + 4];
  __shared__ float bs[BK][BN + 4];
  const int tid = threadIdx.x;
  const int tx = tid & 15, ty = tid >> 4;
  for (int64_t tile = blockIdx.x; tile < total_tiles; tile += gridDim.x) {
    const int64_t n0 = (tile / tiles_d) * BM;
    const int64_t d0 = (tile % tiles_d) * BN;
    float acc[4][4] = {};
    for (int64_t f0 = 0; f0 < F; f0 += BK) {
      __syncthreads();
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int idx = tid + 256 * i;
        {
          const int n = idx / BK, f = idx % BK;
          const int64_t gn = n0 + n, gf = f0 + f;
          xs[f][n] = (gn < N && gf < F) ? load_elem(X, gn * F + gf) : 0.0f;
        }
        {
          const int f = idx / BN, d = idx % BN;
          const int64_t gf = f0 + f, gd = d0 + d;
          bs[f][d] = (gf < F && gd < D) ? load_elem(B, gf * D + gd) : 0.0f;
        }
      }
      __syncthreads();
#pragma unroll
      for (int kk = 0; kk < BK; ++kk) {
        float a[4], b[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) a[i] = xs[kk][ty * 4 + i];
#pragma unroll
        for (int j = 0; j < 4; ++j) b[j] = bs[kk][tx * 4 + j];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t gn = n0 + ty * 4 + i;
      if (gn >= N) continue;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int64_t gd = d0 + tx * 4 + j;
        if (gd < D) H[gn * D + gd] = activate(acc[i][j], act);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Stage II (Eq. 8, Eq. 9) on a given H: one workgroup per sample row
// (grid-stride), classes in chunks of 8, block reduction, first-max argmax.
// ---------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void similarity_kernel(const float* __restrict__ H,
                                                         const T* __restrict__ C,
                                                         int32_t* __restrict__ labels,
                                                         float* __restrict__ scores, int64_t N,
                                                         int64_t D, int64_t K) {
  constexpr int KC = 8;
  __shared__ float red[4][KC];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  for (int64_t n = blockIdx.x; n < N; n += gridDim.x) {
    const float* h = H + n * D;
    float best = 0.0f;
    int32_t best_k = 0;
    for (int64_t k0 = 0; k0 < K; k0 += KC) {
      const int kc = (int)((K - k0) < KC ? (K - k0) : KC);
      float acc[KC] = {};
      for (int64_t d = tid; d < D; d += 256) {
        const float hv = h[d];
#pragma unroll
        for (int j = 0; j < KC; ++j)
          if (j < kc) acc[j] = fmaf(hv, load_elem(C, (k0 + j) * D + d), acc[j]);
      }
#pragma unroll
      for (int j = 0; j < KC; ++j) {
        const float s = wave_sum(acc[j]);
        if (lane == 0) red[wave][j] = s;
      }
      __syncthreads();
      if (tid == 0) {
        for (int j = 0; j < kc; ++j) {
          const float s = (red[0][j] + red[1][j]) + (red[2][j] + red[3][j]);
          if (scores) scores[n * K + k0 + j] = s;
          if ((k0 + j) == 0 || s > best) {
            best = s;
            best_k = (int32_t)(k0 + j);
          }
        }
      }
      __syncthreads();
    }
    if (tid == 0) labels[n] = best_k;
  }
}

// Zero-fill of [p, p + bytes): 16-byte stores over the aligned body, bytes at
// the ragged end one by one. p is 256-byte aligned (workspace rule).
__global__ __launch_bounds__(256) void zero_kernel(uint4* __restrict__ p, int64_t n16,
                                                   unsigned char* __restrict__ tail, int ntail) {
  const uint4 z = make_uint4(0u, 0u, 0u, 0u);
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n16;
       i += (int64_t)gridDim.x * 256)
    p[i] = z;
  if (blockIdx.x == 0 && (int)threadIdx.x < ntail) tail[threadIdx.x] = 0;
}

hipError_t launch_zero(void* p, size_t bytes, hipStream_t stream) {
  if (bytes == 0) return hipSuccess;
  const int64_t n16 = (int64_t)(bytes / 16);
  const int ntail = (int)(bytes % 16);
  const int64_t g = cdiv(n16 > 0 ? n16 : 1, 256);
  hipLaunchKernelGGL(zero_kernel, dim3((unsigned)(g < 4096 ? g : 4096)), dim3(256), 0, stream,
                     static_cast<uint4*>(p), n16, static_cast<unsigned char*>(p) + n16 * 16,
                     ntail);
  return hipGetLastError();
}

static int grid_for(int64_t work) {
  const int64_t cap = 1 << 20;
  return (int)(work < cap ? (work > 0 ? work : 1) : cap);
}

hipError_t launch_encode(const void* X, const void* B, float* H, int64_t N, int64_t F, int64_t D,
                         int dt, int act, hipStream_t stream) {
  const int64_t tiles_d = cdiv(D, 64), tiles = cdiv(N, 64) * tiles_d;
  const dim3 grid(grid_for(tiles)), block(256);
  if (dt == 0)
    hipLaunchKernelGGL(encode_kernel<float>, grid, block, 0, stream, (const float*)X,
                       (const float*)B, H, N, F, D, act, tiles_d, tiles);
  else
    hipLaunchKernelGGL(encode_kernel<bf16raw>, grid, block, 0, stream, (const bf16raw*)X,
                       (const bf16raw*)B, H, N, F, D, act, tiles_d, tiles);
  return hipGetLastError();
}

hipError_t launch_similarity(const float* H, const void* C, int32_t* labels, float* scores,
                             int64_t N, int64_t D, int64_t K, int c_dt, hipStream_t stream) {
  const dim3 grid(grid_for(N)), block(256);
  if (c_dt == 0)
    hipLaunchKernelGGL(similarity_kernel<float>, grid, block, 0, stream, H, (const float*)C,
                       labels, scores, N, D, K);
  else
    hipLaunchKernelGGL(similarity_kernel<bf16raw>, grid, block, 0, stream, H,
                       (const bf16raw*)C, labels, scores, N, D, K);
  return hipGetLastError();
}

}  // namespace hd
