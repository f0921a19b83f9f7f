// Small-batch fused inference (N <= 64): the GPU form of the paper's
// small-batch variant (Sec. III-C, Alg. 3), which splits the hypervector
// dimension D across workers and sums their partial score matrices.
//
// Work unit. A "column block" is 16 consecutive columns of B with all F rows
// (a column block of the encoded matrix, Alg. 2): its encoding sums are
// complete inside one workgroup, so HardSign (Eq. 1) is applied on chip and H
// never reaches device memory. B is read exactly once.
//
// Grid. One persistent workgroup per compute unit walks its share of column
// blocks; the next block's B rows are in flight while the current block is
// computed. Blocks are ordered so that each XCD (with its own L2) walks a
// contiguous range of columns, so blocks sharing 128-byte L2 lines are read
// through the same L2.
//
// Compute. N <= 8 (and bf16 inputs): plain fp32 FMAs. 8 < N <= 64 with fp32
// inputs: the 16x16x4 fp32 matrix instruction (twice the unpacked vector FMA
// rate), with X^T staged in LDS as the B operand and B's row segments as the
// A operand.
//
// Reduction. Each workgroup sums its blocks' partial scores locally, adds
// them with fp32 atomics into one of R replicated accumulators, and takes a
// ticket; the last workgroup reads-and-clears the replicas, takes the row
// argmax (Eq. 9) and writes labels/scores. hd_common.hpp explains why the
// hand-off uses atomics and no device-scope fence.
//
// Wait counters. Global loads are issued unconditionally (addresses clamped
// into the buffers, results selected afterwards) so the compiler can track
// how many are outstanding across loop iterations; a block's C rows are loaded
// before the next block's B rows, so waiting for them does not drain the
// prefetch.
#include "hd_common.hpp"
#include "hd_internal.hpp"

namespace hd {

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;
constexpr int kW = 16;                // columns per block
constexpr int kCG = kW / 4;           // float4 column groups per block
constexpr int kRG = kThreads / kCG;   // row groups (VALU kernel)
constexpr int kRpt = 12;              // B rows per thread per chunk (VALU kernel)
constexpr int kLdsBudget = 159 * 1024;

// Workspace: the final ticket counter, kGroups group counters (each on its
// own 256-byte line), then the R score replicas [R][N][K].
constexpr int kGroups = 32;
constexpr int kLine = 256;

struct SmallWs {
  unsigned* counter;
  unsigned* group;  // group g's counter at group + g * kLine / 4
  float* sacc;      // [R][N][K]
};

__host__ __device__ inline SmallWs small_ws(void* ws) {
  SmallWs w;
  char* b = reinterpret_cast<char*>(ws);
  w.counter = reinterpret_cast<unsigned*>(b);
  w.group = reinterpret_cast<unsigned*>(b + kLine);
  w.sacc = reinterpret_cast<float*>(b + kLine * (1 + kGroups));
  return w;
}

// Score replicas: enough that few workgroups add into each address (atomics
// on one address are serialised), few enough that the finishing workgroup
// reads all of them in one batch (R*N*K <= 16 per thread).
__host__ __device__ inline int replicas(int G, int NK) {
  int r = (16 * 256) / (NK > 0 ? NK : 1);
  r = r < 4 ? 4 : r > kSmallReplicas ? kSmallReplicas : r;
  return G < r ? G : r;
}

// Block order. Workgroups are dispatched round-robin over the 8 XCDs, so
// workgroup b runs on XCD b % 8. The blocks are split evenly between XCDs
// into contiguous ranges (neighbouring blocks share 128-byte L2 lines), and
// each XCD's workgroups take its range round-robin. A workgroup's k-th block
// is block_of(k); it owns blocks while block_of(k) < its XCD's range end.
struct BlockWalk {
  int start, stride, end;
  __device__ int block_of(int k) const { return start + k * stride; }
  __device__ int count() const { return start < end ? (end - start + stride - 1) / stride : 0; }
};

__device__ __forceinline__ BlockWalk block_walk(int b, int G, int nblocks) {
  const int x = b % 8, j = b / 8;
  const int per = G / 8, rem = G % 8;
  const int gx = per + (x < rem ? 1 : 0);  // workgroups on this XCD
  const int nx = G < 8 ? G : 8;            // XCDs that have workgroups
  BlockWalk w;
  if (x >= nx) {
    w.start = w.end = 0;
    w.stride = 1;
    return w;
  }
  const int r0 = (int)((int64_t)nblocks * x / nx), r1 = (int)((int64_t)nblocks * (x + 1) / nx);
  w.start = r0 + j;
  w.stride = gx;
  w.end = r1;
  return w;
}

// Where a column block's values live. Block blk covers columns 16 blk ..
// 16 blk + 15 of a matrix with `rows` rows (B: F rows, C: K rows).
//   kRawScalar / kRawVec: the caller's row-major matrix [rows][D]; columns
//     past D are clamped into the row (their values are garbage and only meet
//     zeroed encodings). kRawVec needs D % 4 == 0 and aligned bases, so a
//     4-column group is either wholly inside the row or wholly past it.
//   kTiled: the packed model's column-block layout [nblk][rows][16], zero past
//     column D: one block is a single contiguous run, which keeps the DRAM
//     access stream sequential (64-byte pieces of many rows are not).
constexpr int kRawScalar = 0, kRawVec = 1, kTiled = 2;

template <typename T, int LAY>
struct ColView {
  const T* __restrict__ p;
  int64_t D;
  int rows;
  // B[r][16 blk + c .. +3]; c is a multiple of 4
  __device__ __forceinline__ float4 get4(int blk, int r, int c) const {
    if (LAY == kTiled) return load4(p, ((int64_t)blk * rows + r) * kW + c);
    const int64_t col = (int64_t)blk * kW + c;
    if (LAY == kRawVec) return load4(p, (int64_t)r * D + (col < D ? col : 0));
    float v[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) v[q] = load_elem(p, (int64_t)r * D + (col + q < D ? col + q : D - 1));
    return make_float4(v[0], v[1], v[2], v[3]);
  }
  __device__ __forceinline__ float get(int blk, int r, int c) const {
    if (LAY == kTiled) return load_elem(p, ((int64_t)blk * rows + r) * kW + c);
    const int64_t col = (int64_t)blk * kW + c;
    return load_elem(p, (int64_t)r * D + (col < D ? col : D - 1));
  }
};

// Copy the first n floats of X into LDS: 16-byte loads and stores, all of a
// thread's loads in flight at once. X is 16-byte aligned. Stores are
// unconditional (a branch per store lets the compiler sink each load to its
// store, serialising them); threads past the end write the spare float4 slot
// after the n floats, which the caller provides.
__device__ __forceinline__ int x_rotation(int n4) {
  // Every workgroup reads all of X. Starting each at a different 1 KiB
  // offset spreads the simultaneous reads over the L2 channels instead of
  // sending all of them to the channel holding the first bytes.
  return n4 > 0 ? (int)(((int64_t)blockIdx.x * 37 * 64) % n4) : 0;
}

__device__ void copy_flat_to_lds(const float* __restrict__ X, float* xs, int n) {
  const int tid = threadIdx.x;
  const int n4 = n / 4;
  const int rot = x_rotation(n4);
  const float4* src = reinterpret_cast<const float4*>(X);
  float4* dst = reinterpret_cast<float4*>(xs);
  constexpr int kBatch = 24;
  for (int base = 0; base < n4; base += kThreads * kBatch) {
    float4 v[kBatch];
    int at[kBatch];
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const int i = base + j * kThreads + tid;
      const int r = i + rot >= n4 ? i + rot - n4 : i + rot;
      at[j] = i < n4 ? r : n4;
      v[j] = src[i < n4 ? r : 0];
    }
#pragma unroll
    for (int j = 0; j < kBatch; ++j) dst[at[j]] = v[j];
  }
  for (int i = 4 * n4 + tid; i < n; i += kThreads) xs[i] = X[i];
}

// Generic staging of an f-chunk [fc0, fc0+fcn) of rows [n0, n0+NB) (zero past
// N) into xs[n*Pf + f - fc0].
template <typename T>
__device__ void stage_rows_chunk(const T* __restrict__ X, float* xs, int Pf, int n0, int NB, int F,
                                 int N, int fc0, int fcn) {
  for (int i = threadIdx.x; i < NB * fcn; i += kThreads) {
    const int n = i / fcn, f = i - n * fcn;
    xs[n * Pf + f] = (n0 + n < N) ? load_elem(X, (int64_t)(n0 + n) * F + fc0 + f) : 0.0f;
  }
}

// The 16 C values C[k][16 blk .. 16 blk + 15] of (sample, class) pair
// p = threadIdx.x, loaded unconditionally with clamped addresses so the load
// count per thread is fixed. No select is applied to the loaded values (that
// would force a wait right here): pairs past N*K are never used and columns
// past D meet zeroed encoded values.
template <typename T, int LAY>
__device__ __forceinline__ void load_c_pair(const ColView<T, LAY>& cv, int K, int blk, int npairs,
                                            float (&c)[kW]) {
  const int p = threadIdx.x;
  const int k = p < npairs ? p % K : 0;
#pragma unroll
  for (int j = 0; j < kW; j += 4) {
    const float4 v = cv.get4(blk, k, j);
    c[j] = v.x;
    c[j + 1] = v.y;
    c[j + 2] = v.z;
    c[j + 3] = v.w;
  }
}

// Partial similarity of one finished block: sl[n*K + k] += sum_c hs[n][c] C[k][d0+c]
// (Eq. 8 restricted to the block's columns). hs is [NB][kW+1]; pair
// threadIdx.x uses the preloaded cpair, further pairs read C directly.
template <typename T, int LAY>
__device__ void block_scores(const ColView<T, LAY>& cv, const float* hs, float* sl, int npairs,
                             int K, int blk, const float (&cpair)[kW]) {
  const int tid = threadIdx.x;
  if (tid < npairs) {
    const int n = tid / K;
    float s = 0.0f;
#pragma unroll
    for (int j = 0; j < kW; ++j) s = fmaf(hs[n * (kW + 1) + j], cpair[j], s);
    sl[tid] += s;
  }
  for (int p = tid + kThreads; p < npairs; p += kThreads) {
    const int n = p / K, k = p - n * K;
    float s = 0.0f;
#pragma unroll
    for (int j = 0; j < kW; ++j) s = fmaf(hs[n * (kW + 1) + j], cv.get(blk, k, j), s);
    sl[p] += s;
  }
}

// Publish this workgroup's partial scores (samples [nb0, nb0+nb)); after the
// last sample block, take a ticket and, in the last workgroup, finish: sum
// the replicas, write scores and labels, and re-zero the ticket.
//
// Tickets are drawn in two levels. Atomics on one address are performed one
// after another (about 10 ns each), so a single counter drawn by hundreds of
// workgroups would serialise for microseconds. Workgroup b draws from group
// counter b % kGroups; the group's last drawer (which then knows that every
// member's partials are performed) resets it and draws from the final
// counter; the last of those finishes.
__device__ void publish_and_finish(const float* sl, int nb0, int nb, int N, int K, int R,
                                   const SmallWs& ws, int32_t* __restrict__ labels,
                                   float* __restrict__ scores, float* buf, int buf_floats,
                                   bool finish) {
  const int tid = threadIdx.x;
  float* my = ws.sacc + (int64_t)(blockIdx.x % R) * N * K;
  for (int p = tid; p < nb * K; p += kThreads) publish_add(my + (int64_t)nb0 * K + p, sl[p]);
  if (!finish) return;
  __shared__ int s_last;
  wait_own_memory_ops();
  __syncthreads();
  if (tid == 0) {
    const unsigned G = gridDim.x, ng = G < kGroups ? G : kGroups, g = blockIdx.x % ng;
    const unsigned gsize = G / ng + (g < G % ng ? 1u : 0u);
    unsigned* gc = ws.group + g * (kLine / 4);
    int last = 0;
    if (take_ticket(gc) == gsize - 1) {
      reset_counter(gc);
      last = take_ticket(ws.counter) == ng - 1 ? 1 : 0;
    }
    s_last = last;
  }
  __syncthreads();
  if (!s_last) return;
  const int64_t NK = (int64_t)N * K;
  const int64_t total = (int64_t)R * NK;
  if (total <= buf_floats) {
    constexpr int kBatch = 16;
    for (int64_t base = 0; base < total; base += (int64_t)kThreads * kBatch) {
      float v[kBatch];
#pragma unroll
      for (int j = 0; j < kBatch; ++j) {
        const int64_t i = base + (int64_t)j * kThreads + tid;
        v[j] = i < total ? take_and_clear(ws.sacc + i) : 0.0f;
      }
#pragma unroll
      for (int j = 0; j < kBatch; ++j) {
        const int64_t i = base + (int64_t)j * kThreads + tid;
        if (i < total) buf[i] = v[j];
      }
    }
    __syncthreads();
    for (int64_t o = tid; o < NK; o += kThreads) {
      float s = 0.0f;
      for (int r = 0; r < R; ++r) s += buf[r * NK + o];
      buf[o] = s;  // replica 0's slot now holds the total
      if (scores) scores[o] = s;
    }
    __syncthreads();
    for (int n = tid; n < N; n += kThreads) {
      float best = buf[(int64_t)n * K];
      int best_k = 0;
      for (int k = 1; k < K; ++k) {
        const float s = buf[(int64_t)n * K + k];
        if (s > best) {
          best = s;
          best_k = k;
        }
      }
      labels[n] = best_k;
    }
  } else {
    const int lane = tid & 63, wave = tid >> 6;
    for (int n = wave; n < N; n += kWaves) {
      float best = -__builtin_huge_valf();
      int best_k = 0x7fffffff;
      for (int k = lane; k < K; k += kWave) {
        float t[kSmallReplicas];
#pragma unroll
        for (int r = 0; r < kSmallReplicas; ++r)
          t[r] = r < R ? take_and_clear(ws.sacc + r * NK + (int64_t)n * K + k) : 0.0f;
        float s = 0.0f;
#pragma unroll
        for (int r = 0; r < kSmallReplicas; ++r) s += t[r];
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
  }
  if (tid == 0) reset_counter(ws.counter);
}

// Sum of v over lanes {l, l+4, l+8, l+12} of each 16-lane row (DPP row
// rotations, no LDS traffic).
__device__ __forceinline__ float row_sum4(float v) {
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v),
                                                              0x128, 0xf, 0xf, false));  // row_ror:8
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v),
                                                              0x124, 0xf, 0xf, false));  // row_ror:4
  return v;
}

// Three-deep prefetch ring over a workgroup's items: while item i is
// processed, items i+1 and i+2 are in flight. Buffers are named (no register
// copies, which would wait on the loads). ring3_start issues the first two
// items; the caller can do independent work before ring3_run.
template <class Buf, class LoadF>
__device__ __forceinline__ void ring3_start(int nitems, Buf& b0, Buf& b1, LoadF&& load) {
  if (nitems <= 0) return;
  load(b0, 0);
  load(b1, nitems > 1 ? 1 : 0);
}

template <class Buf, class LoadF, class ProcF>
__device__ __forceinline__ void ring3_run(int nitems, Buf& b0, Buf& b1, Buf& b2, LoadF&& load,
                                          ProcF&& process) {
  auto cl = [&](int i) { return i < nitems ? i : nitems - 1; };
  for (int it = 0; it < nitems; it += 3) {
    load(b2, cl(it + 2));
    __builtin_amdgcn_sched_barrier(0);
    process(b0, it);
    if (it + 1 >= nitems) break;
    load(b0, cl(it + 3));
    __builtin_amdgcn_sched_barrier(0);
    process(b1, it + 1);
    if (it + 2 >= nitems) break;
    load(b1, cl(it + 4));
    __builtin_amdgcn_sched_barrier(0);
    process(b2, it + 2);
  }
}

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
  const int R = replicas(G, N * K);
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
                       nb0 + NB >= N);
  }
}

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
  const int R = replicas(G, N * K);
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
  publish_and_finish(sl, 0, nb, N, K, R, ws, labels, scores, smem, lds_floats, true);
}

// ---------------------------------------------------------------------------
// Flat kernel (N <= 8, one column block per workgroup). Every load a
// workgroup needs (its block of B, its rows of X, its pairs' C values) is
// issued at entry; several workgroups share a CU, so the hardware overlaps
// them. Thread (cg, rg) handles columns 4cg..4cg+3 and rows rg + 64u of
// each f-chunk of 64*RPT rows.
// LDS: red[16][NB][16] | hs[NB][17]
// ---------------------------------------------------------------------------
__device__ __forceinline__ int xcd_block(int b, int G) {
  // contiguous column ranges per XCD (blocks sharing L2 lines meet in one L2)
  const int per = G / 8, rem = G % 8, x = b % 8, j = b / 8;
  return x * per + min(x, rem) + j;
}

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
  const int R = replicas(G, N * K);
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
  publish_and_finish(none, 0, 0, N, K, R, ws, labels, scores, red, kWaves * 4 * NB * kW, true);
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
  const int R = replicas(G, N * K);
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
  publish_and_finish(none, 0, 0, N, K, R, ws, labels, scores, smem, lds_floats, true);
}

// ---------------------------------------------------------------------------
// Fragment matrix-core kernel (fp32, 8 < N <= 64, packed model). The packed
// model holds, per 16-column block, the 16x16x4 A operands in the order the
// waves consume them (see pack_frag_kernel): wave w's lane l = (d, q) with
// d = l % 16, q = l / 16 covers the MS consecutive rows
// f = 4*MS*w + MS*q + 0..MS-1 of column 16 blk + d, four rows per float4, so
// a block costs each lane MS/4 16-byte loads and each wave-wide load is one
// contiguous 1 KiB run. Matrix step s of the wave multiplies row
// 4*MS*w + MS*q + s (lane group q) with the same rows of X^T, read from a
// verbatim copy of X in LDS.
//
// Persistent: one workgroup per CU walks its column blocks with two blocks of
// B in flight (ring3), X stays in LDS, and the workgroup's partial scores
// accumulate in LDS and are published once.
// LDS: sl[NB*K] | red[4][NTI][256] | hs[NB][17] | xs[NB*F + 16*MS] (+ 4 spare)
// ---------------------------------------------------------------------------
template <int MS>
struct FragBuf {
  float4 a[MS / 4];
  float c[kW];
};

template <int NTI, int MS>
__global__ __launch_bounds__(kThreads, 1) void small_frag_mfma_kernel(
    const float* __restrict__ X, const float4* __restrict__ Bf, const float* __restrict__ C,
    int32_t* __restrict__ labels, float* __restrict__ scores, int N, int F, int D, int K, int act,
    int nblocks, int lds_floats, void* __restrict__ workspace) {
  constexpr int NB = 16 * NTI;
  constexpr int G4 = MS / 4;
  extern __shared__ __attribute__((aligned(16))) float smem[];
  float* sl = smem;                           // [NB*K]
  float* red = sl + (NB * K + 3) / 4 * 4;     // [4][NTI][256]
  float* hs = red + kWaves * NTI * 256;       // [NB][17]
  float* xs = hs + (NB * (kW + 1) + 3) / 4 * 4;  // [NB*F + 16*MS] + 4 spare
  const SmallWs ws = small_ws(workspace);
  const ColView<float, kTiled> cv{C, D, K};
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int G = gridDim.x;
  const BlockWalk walk = block_walk(blockIdx.x, G, nblocks);
  const int R = replicas(G, N * K);
  const int nb = min(NB, N);
  const int npairs = nb * K;
  const int nmine = walk.count();

  auto load = [&](FragBuf<MS>& x, int i) {
    const int blk = walk.block_of(i);
    const float4* p = Bf + ((int64_t)blk * kWaves + wave) * G4 * kWave + lane;
#pragma unroll
    for (int g = 0; g < G4; ++g) x.a[g] = p[g * kWave];
    load_c_pair(cv, K, blk, npairs, x.c);
  };
  // X is copied verbatim into LDS (xs[n*F + f]), before any B load is
  // issued: a wait for a load also waits for every load issued before it,
  // and X (shared by all workgroups, in L2) would otherwise wait for HBM.
  // Each workgroup starts at a different offset so that they do not all read
  // the same L2 lines at once. Stores are unconditional (past the end they go
  // to the spare slot) so that no load is sunk to its store. Steps past F
  // read the next row (finite values times zero B) or, after the last row,
  // the zeroed run of 16*MS floats.
  const int n4 = nb * F / 4;
  {
    const int rot = (int)(((int64_t)blockIdx.x * 37 * 64) % n4);
    const float4* x4 = reinterpret_cast<const float4*>(X);
    float4* xs4 = reinterpret_cast<float4*>(xs);
    const int spare4 = (NB * F + 16 * MS + 3) / 4;
    constexpr int kXB = NTI * MS / 4 < 40 ? NTI * MS / 4 : 40;
    for (int base = 0; base < n4; base += kThreads * kXB) {
      float4 v[kXB];
      int at[kXB];
#pragma unroll
      for (int j = 0; j < kXB; ++j) {
        const int i = base + j * kThreads + tid;
        const int r = i + rot >= n4 ? i + rot - n4 : i + rot;
        at[j] = i < n4 ? r : spare4;
        v[j] = x4[i < n4 ? r : rot];
      }
#pragma unroll
      for (int j = 0; j < kXB; ++j) xs4[at[j]] = v[j];
    }
    for (int e = 4 * n4 + tid; e < nb * F; e += kThreads) xs[e] = X[e];
    for (int e = tid; e < 16 * MS; e += kThreads) xs[nb * F + e] = 0.0f;
  }
  // B for the first two blocks goes out once X is on chip
  FragBuf<MS> b0, b1, b2;
  ring3_start(nmine, b0, b1, load);
  for (int p = tid; p < NB * K; p += kThreads) sl[p] = 0.0f;
  __syncthreads();

  const int xoff = (lane & 15) * F + 4 * MS * wave + MS * (lane >> 4);
  auto process = [&](const FragBuf<MS>& x, int i) {
    const int blk = walk.block_of(i);
    const int64_t d0 = (int64_t)blk * kW;
    // two independent accumulator chains per sample tile (steps 4g, 4g+2
    // and 4g+1, 4g+3), interleaved over the tiles, so consecutive matrix
    // instructions do not wait on each other's results
    f32x4 acc[NTI][2];
#pragma unroll
    for (int t = 0; t < NTI; ++t) acc[t][0] = acc[t][1] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int g = 0; g < G4; ++g) {
      float4 xg[NTI];
#pragma unroll
      for (int t = 0; t < NTI; ++t) {
        const float* q = xs + xoff + 16 * t * F + 4 * g;
        xg[t] = make_float4(q[0], q[1], q[2], q[3]);
      }
#pragma unroll
      for (int t = 0; t < NTI; ++t)
        acc[t][0] = __builtin_amdgcn_mfma_f32_16x16x4f32(x.a[g].x, xg[t].x, acc[t][0], 0, 0, 0);
#pragma unroll
      for (int t = 0; t < NTI; ++t)
        acc[t][1] = __builtin_amdgcn_mfma_f32_16x16x4f32(x.a[g].y, xg[t].y, acc[t][1], 0, 0, 0);
#pragma unroll
      for (int t = 0; t < NTI; ++t)
        acc[t][0] = __builtin_amdgcn_mfma_f32_16x16x4f32(x.a[g].z, xg[t].z, acc[t][0], 0, 0, 0);
#pragma unroll
      for (int t = 0; t < NTI; ++t)
        acc[t][1] = __builtin_amdgcn_mfma_f32_16x16x4f32(x.a[g].w, xg[t].w, acc[t][1], 0, 0, 0);
    }
    __syncthreads();  // previous block's readers of red / hs are done
#pragma unroll
    for (int t = 0; t < NTI; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        red[(wave * NTI + t) * 256 + (4 * (lane >> 4) + r) * 16 + (lane & 15)] =
            acc[t][0][r] + acc[t][1][r];
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
  publish_and_finish(sl, 0, nb, N, K, R, ws, labels, scores, smem, lds_floats, true);
}

// Writes the fragment section: out[((blk*4 + w)*(MS/4) + g)*64 + l][e] =
// B[4*MS*w + MS*(l/16) + 4g + e][16 blk + l%16], zero past F or D.
__global__ __launch_bounds__(256) void pack_frag_kernel(const float* __restrict__ B,
                                                        float* __restrict__ out, int64_t F,
                                                        int64_t D, int64_t nblk, int MS) {
  const int64_t per_blk = (int64_t)256 * MS;  // 16 columns x 16*MS rows
  const int64_t total = nblk * per_blk;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * 256) {
    const int64_t e = i % 4, l = (i / 4) % 64, g = (i / 256) % (MS / 4),
                  w = (i / (64 * MS)) % 4, blk = i / per_blk;
    const int64_t f = 4 * MS * w + MS * (l / 16) + 4 * g + e;
    const int64_t col = blk * kW + l % 16;
    out[i] = (f < F && col < D) ? B[f * D + col] : 0.0f;
  }
}

int num_cus() {
  static const int cus = [] {
    int dev = 0, v = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 256;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        v <= 0)
      return 256;
    return v;
  }();
  return cus;
}

constexpr int kMfmaSteps[] = {12, 24, 36, 48};  // 4-row steps per wave: F <= 16 * MS

struct SmallPlan {
  bool flat;  // one block per workgroup (N <= 8)
  int rpt;    // flat kernel: rows per thread per chunk
  bool bmfma;  // block matrix-core kernel (one block per workgroup, N <= 32)
  bool frag;   // fragment matrix-core kernel (packed model)
  bool mfma;
  int nb;    // VALU samples per pass, or MFMA sample tiles
  int ms;    // MFMA steps per wave
  int FC;    // VALU f-chunk
  size_t lds;
  int grid;
  int nblocks;
};

// The VALU kernel serves every layout and alignment; it is the support
// criterion. Returns nb == 0 when nb * K does not fit in LDS.
SmallPlan plan_valu(int64_t N, int64_t F, int64_t D, int64_t K) {
  SmallPlan p{};
  p.nblocks = (int)cdiv(D, kW);
  p.grid = p.nblocks < num_cus() ? p.nblocks : num_cus();
  const int nb = N <= 1 ? 1 : N <= 2 ? 2 : N <= 4 ? 4 : N <= 8 ? 8 : N <= 16 ? 16 : 32;
  const int64_t fixed =
      (int64_t)sizeof(float) * (kWaves * 4 * nb * kW + nb * (kW + 1) + nb * K);
  if (fixed > kLdsBudget) return p;
  if (F <= kRG * kRpt) {
    p.FC = (int)F;  // one chunk: X lives in registers, no staging area
    p.lds = (size_t)fixed;
  } else {
    int64_t fc = (kLdsBudget - fixed) / (int64_t)(sizeof(float) * nb);
    if (fc > kRG * kRpt) fc = kRG * kRpt;  // one chunk holds at most kRG*kRpt rows
    if (fc < 1) return p;
    p.FC = (int)fc;
    p.lds = (size_t)fixed + sizeof(float) * (size_t)fc * nb;
  }
  p.nb = nb;
  return p;
}

// Fragment section: rows per lane (MS) for F, or 0 when F is outside
// [4, 16 * 64] (the section is then absent).
constexpr int kFragMS[] = {12, 24, 36, 48, 64};
int frag_ms(int64_t F) {
  if (F < 4) return 0;
  for (int ms : kFragMS)
    if (16 * (int64_t)ms >= F) return ms;
  return 0;
}

size_t frag_bytes(int64_t F, int64_t D, int dt) {
  const int ms = dt == 0 ? frag_ms(F) : 0;
  return (size_t)cdiv(D, kW) * 256 * ms * sizeof(float);
}

// Kernel choice: N <= 8 takes the flat kernel; fp32 with 8 < N <= 64 a
// matrix-core kernel (the fragment kernel on a packed model, else the block
// kernel for N <= 32 or the persistent one) when its LDS fits; raw matrices
// with unaligned bases or D % 4 != 0 (kRawScalar) and everything else take
// the VALU kernel.
SmallPlan plan_small(int64_t N, int64_t F, int64_t D, int64_t K, int dt, int lay, bool x_aligned) {
  SmallPlan v = plan_valu(N, F, D, K);
  if (v.nb == 0 || lay == kRawScalar) return v;
  SmallPlan p{};
  p.nblocks = v.nblocks;
  if (lay == kTiled && dt == 0 && x_aligned && N > 8 && frag_ms(F) > 0) {
    const int nti = (int)cdiv(N, 16), ms = frag_ms(F);
    const int64_t nbk = 16 * nti;
    const int64_t floats = (nbk * K + 3) / 4 * 4 + kWaves * nti * 256 +
                           (nbk * (kW + 1) + 3) / 4 * 4 + (nbk * F + 16 * ms + 3) / 4 * 4 + 4;
    if ((int64_t)sizeof(float) * floats <= kLdsBudget) {
      p.frag = true;
      p.nb = nti;
      p.ms = ms;
      p.lds = sizeof(float) * (size_t)floats;
      p.grid = v.grid;
      return p;
    }
  }
  if (N <= 8) {
    p.flat = true;
    p.nb = N <= 1 ? 1 : N <= 2 ? 2 : N <= 4 ? 4 : 8;
    p.rpt = F <= kRG * 4 ? 4 : F <= kRG * 9 ? 9 : 16;
    p.grid = p.nblocks;
    return p;
  }
  if (dt == 0 && x_aligned && N <= 32) {
    const int nti = (int)cdiv(N, 16);
    for (int ms : kMfmaSteps) {
      if ((int64_t)16 * ms < F) continue;
      const int64_t red = kWaves * nti * 256 + 16 * nti * (kW + 1);
      const int64_t xs = N * F + 4;  // X and one spare float4
      const int64_t lds = (int64_t)sizeof(float) * (red > xs ? red : xs);
      if (lds > kLdsBudget) break;
      p.bmfma = true;
      p.nb = nti;
      p.ms = ms;
      p.lds = (size_t)lds;
      p.grid = p.nblocks;
      return p;
    }
  }
  if (dt == 0 && x_aligned) {
    const int nti = (int)cdiv(N, 16);
    for (int ms : kMfmaSteps) {
      if ((int64_t)16 * ms < F) continue;
      const int64_t scratch = kWaves * nti * 256 + 16 * nti * (kW + 1);
      const int64_t xs = N * F + 4;  // X and one spare float4
      const int64_t lds = (int64_t)sizeof(float) *
                          ((16 * nti * K + 3) / 4 * 4 + (scratch > xs ? scratch : xs));
      if (lds <= kLdsBudget) {
        p.mfma = true;
        p.nb = nti;
        p.ms = ms;
        p.lds = (size_t)lds;
        p.grid = v.grid;
        return p;
      }
      break;
    }
  }
  return v;
}

// The last workgroup reuses all of LDS to sum the R score replicas, so give
// the launch at least R*N*K floats when that fits.
void widen_for_final(SmallPlan& p, int64_t N, int64_t K) {
  const size_t want = sizeof(float) * (size_t)replicas(p.grid, (int)(N * K)) * N * K;
  if (p.lds < want && want <= (size_t)kLdsBudget) p.lds = want;
}

template <typename KernelT>
hipError_t allow_lds(KernelT* k) {
  return hipFuncSetAttribute(reinterpret_cast<const void*>(k),
                             hipFuncAttributeMaxDynamicSharedMemorySize, kLdsBudget);
}

struct Args {
  const void *X, *B, *C;
  int32_t* labels;
  float* scores;
  int N, F, D, K, act;
  void* ws;
  hipStream_t stream;
};

template <typename T, int NB, int LAY>
hipError_t launch_valu(const SmallPlan& p, const Args& a) {
  static const hipError_t attr = allow_lds(&small_valu_kernel<T, NB, LAY>);
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL((small_valu_kernel<T, NB, LAY>), dim3(p.grid), dim3(kThreads), p.lds,
                     a.stream, (const T*)a.X, (const T*)a.B, (const T*)a.C, a.labels, a.scores,
                     a.N, a.F, a.D, a.K, a.act, p.FC, p.nblocks, (int)(p.lds / sizeof(float)),
                     a.ws);
  return hipGetLastError();
}

template <typename T, int LAY>
hipError_t launch_valu_nb(const SmallPlan& p, const Args& a) {
  switch (p.nb) {
    case 1: return launch_valu<T, 1, LAY>(p, a);
    case 2: return launch_valu<T, 2, LAY>(p, a);
    case 4: return launch_valu<T, 4, LAY>(p, a);
    case 8: return launch_valu<T, 8, LAY>(p, a);
    case 16: return launch_valu<T, 16, LAY>(p, a);
    default: return launch_valu<T, 32, LAY>(p, a);
  }
}

template <int NTI, int MS, int LAY>
hipError_t launch_mfma(const SmallPlan& p, const Args& a) {
  static const hipError_t attr = allow_lds(&small_mfma_kernel<NTI, MS, LAY>);
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

template <int NTI, int MS, int LAY>
hipError_t launch_bmfma(const SmallPlan& p, const Args& a) {
  static const hipError_t attr = allow_lds(&small_block_mfma_kernel<NTI, MS, LAY>);
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

template <int NTI, int MS>
hipError_t launch_frag(const SmallPlan& p, const Args& a, const void* frag) {
  static const hipError_t attr = allow_lds(&small_frag_mfma_kernel<NTI, MS>);
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL((small_frag_mfma_kernel<NTI, MS>), dim3(p.grid), dim3(kThreads), p.lds,
                     a.stream, (const float*)a.X, (const float4*)frag, (const float*)a.C,
                     a.labels, a.scores, a.N, a.F, a.D, a.K, a.act, p.nblocks,
                     (int)(p.lds / sizeof(float)), a.ws);
  return hipGetLastError();
}

template <int NTI>
hipError_t launch_frag_ms(const SmallPlan& p, const Args& a, const void* frag) {
  switch (p.ms) {
    case 12: return launch_frag<NTI, 12>(p, a, frag);
    case 24: return launch_frag<NTI, 24>(p, a, frag);
    case 36: return launch_frag<NTI, 36>(p, a, frag);
    case 48: return launch_frag<NTI, 48>(p, a, frag);
    default: return launch_frag<NTI, 64>(p, a, frag);
  }
}

hipError_t launch_frag_nti(const SmallPlan& p, const Args& a, const void* frag) {
  switch (p.nb) {
    case 1: return launch_frag_ms<1>(p, a, frag);
    case 2: return launch_frag_ms<2>(p, a, frag);
    case 3: return launch_frag_ms<3>(p, a, frag);
    default: return launch_frag_ms<4>(p, a, frag);
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

template <typename T, int LAY>
hipError_t launch_plan(SmallPlan& p, const Args& a) {
  if constexpr (LAY != kRawScalar) {
    if (p.flat) return launch_flat_nb<T, LAY>(p, a);
    if constexpr (sizeof(T) == 4) {
      if (p.bmfma) {
        widen_for_final(p, a.N, a.K);
        return p.nb == 1 ? launch_bmfma_ms<1, LAY>(p, a) : launch_bmfma_ms<2, LAY>(p, a);
      }
      if (p.mfma) {
        widen_for_final(p, a.N, a.K);
        return launch_mfma_nti<LAY>(p, a);
      }
    }
  }
  widen_for_final(p, a.N, a.K);
  return launch_valu_nb<T, LAY>(p, a);
}

template <typename T>
hipError_t launch_t(SmallPlan& p, int lay, const Args& a) {
  switch (lay) {
    case kTiled: return launch_plan<T, kTiled>(p, a);
    case kRawVec: return launch_plan<T, kRawVec>(p, a);
    default: return launch_plan<T, kRawScalar>(p, a);
  }
}

// Small-batch column-tiled model image: B as [nblk][F][16], then C as
// [nblk][K][16] (each section starting on a 256-byte boundary), zero past
// column D.
template <typename T>
__global__ __launch_bounds__(256) void pack_small_kernel(const T* __restrict__ src,
                                                         T* __restrict__ dst, int64_t rows,
                                                         int64_t D, int64_t nblk) {
  const int64_t total = nblk * rows * kW;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * 256) {
    const int64_t c = i % kW, r = (i / kW) % rows, blk = i / (kW * rows);
    const int64_t col = blk * kW + c;
    dst[i] = col < D ? src[r * D + col] : T(0);
  }
}

template <typename T>
hipError_t pack_small_t(const void* B, const void* C, int64_t F, int64_t D, int64_t K,
                        void* out, hipStream_t stream) {
  const int64_t nblk = cdiv(D, kW);
  T* b = static_cast<T*>(out);
  T* c = reinterpret_cast<T*>(static_cast<char*>(out) + (nblk * F * kW * sizeof(T) + 255) / 256 * 256);
  const int64_t gb = cdiv(nblk * F * kW, 256), gc = cdiv(nblk * K * kW, 256);
  hipLaunchKernelGGL(pack_small_kernel<T>, dim3((unsigned)(gb < 65536 ? gb : 65536)), dim3(256), 0,
                     stream, (const T*)B, b, F, D, nblk);
  hipLaunchKernelGGL(pack_small_kernel<T>, dim3((unsigned)(gc < 65536 ? gc : 65536)), dim3(256), 0,
                     stream, (const T*)C, c, K, D, nblk);
  return hipGetLastError();
}

}  // namespace

bool small_supported(int64_t N, int64_t F, int64_t D, int64_t K, int dt) {
  return plan_valu(N, F, D, K).nb > 0;
}

size_t small_workspace_bytes(int64_t N, int64_t F, int64_t D, int64_t K, int dt) {
  return (size_t)kLine * (1 + kGroups) + sizeof(float) * (size_t)kSmallReplicas * N * K;
}

const char* small_kernel_name(int64_t N, int64_t F, int64_t D, int64_t K, int dt, bool tiled) {
  const SmallPlan p = plan_small(N, F, D, K, dt, tiled ? kTiled : kRawVec, true);
  if (p.nb == 0) return "";
  return p.flat ? "small_flat_kernel" : p.frag ? "small_frag_mfma_kernel"
                                      : p.bmfma ? "small_block_mfma_kernel"
                                      : p.mfma  ? "small_mfma_kernel" : "small_valu_kernel";
}

// Small-batch section of a packed model: column tiles of B, column tiles of
// C, then (fp32, 4 <= F <= 1024) the fragment copy of B, each on a 256-byte
// boundary.
size_t small_tiles_bytes(int64_t F, int64_t D, int64_t K, int dt) {
  const size_t es = dt == 0 ? 4 : 2;
  const size_t nblk = (size_t)cdiv(D, kW);
  return (nblk * F * kW * es + 255) / 256 * 256 + (nblk * K * kW * es + 255) / 256 * 256;
}

size_t small_packed_bytes(int64_t F, int64_t D, int64_t K, int dt) {
  return small_tiles_bytes(F, D, K, dt) + (frag_bytes(F, D, dt) + 255) / 256 * 256;
}

hipError_t launch_pack_small(const void* B, const void* C, int64_t F, int64_t D, int64_t K, int dt,
                             void* out, hipStream_t stream) {
  const hipError_t e = dt == 0 ? pack_small_t<float>(B, C, F, D, K, out, stream)
                               : pack_small_t<bf16raw>(B, C, F, D, K, out, stream);
  if (e != hipSuccess || frag_bytes(F, D, dt) == 0) return e;
  const int64_t nblk = cdiv(D, kW);
  const int ms = frag_ms(F);
  const int64_t g = cdiv(nblk * 256 * ms, 256);
  hipLaunchKernelGGL(pack_frag_kernel, dim3((unsigned)(g < 65536 ? g : 65536)), dim3(256), 0,
                     stream, (const float*)B,
                     reinterpret_cast<float*>(static_cast<char*>(out) + small_tiles_bytes(F, D, K, dt)),
                     F, D, nblk, ms);
  return hipGetLastError();
}

hipError_t launch_small(const void* X, const void* B, const void* C, bool tiled, int32_t* labels,
                        float* scores, int64_t N, int64_t F, int64_t D, int64_t K, int dt,
                        int act, void* workspace, hipStream_t stream) {
  const size_t align = dt == 0 ? 16 : 8;
  int lay = kTiled;
  const void* frag = nullptr;
  if (tiled) {
    // the packed image's small-batch section
    const size_t es = dt == 0 ? 4 : 2;
    C = static_cast<const char*>(B) + (cdiv(D, kW) * F * kW * es + 255) / 256 * 256;
    if (frag_bytes(F, D, dt) > 0) frag = static_cast<const char*>(B) + small_tiles_bytes(F, D, K, dt);
  } else {
    const bool vec = (D % 4 == 0) && ((uintptr_t)B % align == 0) && ((uintptr_t)C % align == 0);
    lay = vec ? kRawVec : kRawScalar;
  }
  SmallPlan p = plan_small(N, F, D, K, dt, lay, (uintptr_t)X % 16 == 0);
  if (p.nb == 0) return hipErrorInvalidValue;
  const Args a{X, B, C, labels, scores, (int)N, (int)F, (int)D, (int)K, act, workspace, stream};
  if (p.frag) {
    if (!frag) return hipErrorInvalidValue;
    widen_for_final(p, N, K);
    return launch_frag_nti(p, a, frag);
  }
  return dt == 0 ? launch_t<float>(p, lay, a) : launch_t<bf16raw>(p, lay, a);
}

}  // namespace hd
