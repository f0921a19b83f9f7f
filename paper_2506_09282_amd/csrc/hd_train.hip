// Single-pass class-hypervector construction (Sec. II-C): the codebook row
// of class k is the normalised bundle of the encoded hypervectors of the
// samples labelled k,
//   counts[k,d] += sum over n with y[n] == k of HardSign(sum_f X[n,f] B[f,d])
//   M[k,d]       = HardSign(counts[k,d])          (Eq. 1: ties and empty classes to +1)
// (encoding Eq. 2-3, bundling Sec. II-A). The sums are exact integers.
//
// bundle_valu_kernel: one workgroup per (64-column block of D, share of the
// samples). It encodes 64-sample x 64-column tiles (F streamed through LDS in
// steps of 16, a 4x4 register tile per thread, fp32 accumulation), applies
// HardSign, adds each +1/-1 into its class's counter in LDS (integer atomics),
// and after its last tile adds its nonzero counters into the caller's sums
// with one device atomic each. Splitting the samples over workgroups keeps
// the grid large while the device atomics stay few (K * 64 per workgroup).
#include "hd_common.hpp"
#include "hd_internal.hpp"

namespace hd {

namespace {

constexpr int kTile = 64;     // samples and columns per tile
constexpr int kFStep = 16;    // features per LDS step

template <typename T>
__global__ __launch_bounds__(256) void bundle_valu_kernel(const T* __restrict__ X,
                                                     const T* __restrict__ B,
                                                     const int32_t* __restrict__ y,
                                                     int32_t* __restrict__ counts, int64_t N,
                                                     int64_t F, int64_t D, int K, int nsplit) {
  __shared__ float xs[kFStep][kTile + 4];
  __shared__ float bs[kFStep][kTile + 4];
  __shared__ int ys[kTile];
  extern __shared__ int cnt[];  // [K][64]
  const int tid = threadIdx.x;
  const int tx = tid & 15, ty = tid >> 4;
  const int64_t db = blockIdx.x / nsplit;
  const int split = (int)(blockIdx.x % nsplit);
  const int64_t d0 = db * kTile;
  for (int i = tid; i < K * kTile; i += 256) cnt[i] = 0;
  const int64_t ntiles = cdiv(N, kTile);
  for (int64_t t = split; t < ntiles; t += nsplit) {
    const int64_t n0 = t * kTile;
    __syncthreads();  // the previous tile's labels are no longer read
    if (tid < kTile) {
      const int64_t n = n0 + tid;
      const int k = n < N ? y[n] : -1;
      ys[tid] = (k >= 0 && k < K) ? k : -1;  // labels outside [0, K) are skipped
    }
    float acc[4][4] = {};
    for (int64_t f0 = 0; f0 < F; f0 += kFStep) {
      __syncthreads();
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int idx = tid + 256 * i;
        {
          const int n = idx / kFStep, f = idx % kFStep;
          const int64_t gn = n0 + n, gf = f0 + f;
          xs[f][n] = (gn < N && gf < F) ? load_elem(X, gn * F + gf) : 0.0f;
        }
        {
          const int f = idx / kTile, d = idx % kTile;
          const int64_t gf = f0 + f, gd = d0 + d;
          bs[f][d] = (gf < F && gd < D) ? load_elem(B, gf * D + gd) : 0.0f;
        }
      }
      __syncthreads();
#pragma unroll
      for (int kk = 0; kk < kFStep; ++kk) {
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
    // HardSign of the tile and its class sums (rows past N and columns past
    // D are skipped: they carry label -1 or are never flushed)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int k = ys[ty * 4 + i];
      if (k < 0) continue;
#pragma unroll
      for (int j = 0; j < 4; ++j)
        atomicAdd(&cnt[k * kTile + tx * 4 + j], hardsign(acc[i][j]) > 0.0f ? 1 : -1);
    }
  }
  __syncthreads();
  for (int i = tid; i < K * kTile; i += 256) {
    const int k = i / kTile, c = i % kTile;
    const int v = cnt[i];
    if (v != 0 && d0 + c < D) atomicAdd(&counts[(int64_t)k * D + d0 + c], v);
  }
}

// M = HardSign(counts), elementwise.
__global__ __launch_bounds__(256) void class_hardsign_kernel(const int32_t* __restrict__ counts,
                                                             float* __restrict__ M,
                                                             int64_t total) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * 256)
    M[i] = hardsign((float)counts[i]);
}

// Counters of up to kBundleMaxK classes take up to 128 KiB of LDS, above the
// default dynamic limit: raise it once per device and kernel.
template <typename T>
hipError_t allow_counter_lds() {
  static PerDeviceOnce once;
  return once_per_device(once, [] {
    return hipFuncSetAttribute(reinterpret_cast<const void*>(&bundle_valu_kernel<T>),
                               hipFuncAttributeMaxDynamicSharedMemorySize,
                               (int)(sizeof(int) * kBundleMaxK * kTile));
  });
}

}  // namespace

bool bundle_supported(int64_t K) { return K >= 1 && K <= kBundleMaxK; }

hipError_t launch_bundle(const void* X, const void* B, const int32_t* y, int32_t* counts,
                         int64_t N, int64_t F, int64_t D, int64_t K, int dt,
                         hipStream_t stream) {
  const int64_t dblocks = cdiv(D, kTile), ntiles = cdiv(N, kTile);
  // enough workgroups to fill the chip (several per compute unit), each
  // taking at least a few sample tiles
  int64_t nsplit = cdiv(4 * (int64_t)num_cus(), dblocks);
  if (nsplit > ntiles) nsplit = ntiles;
  if (nsplit < 1) nsplit = 1;
  const dim3 grid((unsigned)(dblocks * nsplit)), block(256);
  const size_t lds = sizeof(int) * (size_t)K * kTile;
  const hipError_t attr = dt == 0 ? allow_counter_lds<float>() : allow_counter_lds<bf16raw>();
  if (attr != hipSuccess) return attr;
  if (dt == 0)
    hipLaunchKernelGGL(bundle_valu_kernel<float>, grid, block, lds, stream, (const float*)X,
                       (const float*)B, y, counts, N, F, D, (int)K, (int)nsplit);
  else
    hipLaunchKernelGGL(bundle_valu_kernel<bf16raw>, grid, block, lds, stream, (const bf16raw*)X,
                       (const bf16raw*)B, y, counts, N, F, D, (int)K, (int)nsplit);
  return hipGetLastError();
}

hipError_t launch_class_hardsign(const int32_t* counts, float* M, int64_t K, int64_t D,
                                 hipStream_t stream) {
  const int64_t total = K * D;
  const int64_t g = cdiv(total, 256);
  hipLaunchKernelGGL(class_hardsign_kernel, dim3((unsigned)(g < 65536 ? g : 65536)), dim3(256), 0,
                     stream, counts, M, total);
  return hipGetLastError();
}

}  // namespace hd
