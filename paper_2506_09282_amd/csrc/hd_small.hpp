// Internal header of the small-batch path (N <= 64): shared constants,
// device helpers, the launch plan and the per-kernel-family launchers.
#pragma once

#include "hd_common.hpp"
#include "hd_internal.hpp"

namespace hd {
namespace sp {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;
constexpr int kW = 16;                // columns per block
constexpr int kCG = kW / 4;           // float4 column groups per block
constexpr int kRG = kThreads / kCG;   // row groups (VALU kernel)
constexpr int kRpt = 12;              // B rows per thread per chunk (VALU kernel)
constexpr int kLdsBudget = 159 * 1024;

// Workspace: the final ticket counter, kGroups group counters (each on its
// own 256-byte line), then the R score replicas [R][N][K]. Eight groups
// (measured at the activity shape against 16 and 32: fp32 N = 32 12.3 us
// against 12.5 and 12.5 us, N = 1 9.1 against 9.2 and 9.2 us).
constexpr int kGroups = 8;
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
// on one address are serialised), few enough that the finishing workgroup's
// exchanges stay cheap: about 256 replica values in all, 8 to 32 replicas
// (measured at the activity shape: N = 1 9.2 us with 32 replicas, 11.4 us
// with 8; N = 8 10.6 us with 8, 10.9 us with 21).
__host__ __device__ inline int replicas(int G, int NK) {
  int r = 256 / (NK > 0 ? NK : 1);
  r = r < 8 ? 8 : r > kSmallReplicas ? kSmallReplicas : r;
  return G < r ? G : r;
}

// Block order. Workgroups are dispatched round-robin over the 8 XCDs, so
// workgroup b runs on XCD b % 8. The blocks are split evenly between XCDs
// into contiguous ranges (neighbouring blocks share 128-byte L2 lines), and
// each XCD's workgroups take its range round-robin. A workgroup's k-th block
// is block_of(k); it owns blocks while block_of(k) < its XCD's range end.
struct BlockWalk {
  int start, stride, end;
  __host__ __device__ int block_of(int k) const { return start + k * stride; }
  __host__ __device__ int count() const {
    return start < end ? (end - start + stride - 1) / stride : 0;
  }
};

__host__ __device__ __forceinline__ BlockWalk block_walk(int b, int G, int nblocks) {
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

__device__ inline void copy_flat_to_lds(const float* __restrict__ X, float* xs, int n) {
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
//
// Deterministic mode (det, with R == G: one replica per workgroup): every
// replica slot receives exactly one add onto zero, so it holds that
// workgroup's partial exactly, and the sums are taken in a fixed order: the
// group's last drawer sums its members' slots in member order into the
// group's slot (after the G replicas), and the final workgroup sums the group
// slots in group order. Scores and labels are then identical from run to run.
template <int NT>
__device__ void finish_deterministic(int N, int K, const SmallWs& ws,
                                     int32_t* __restrict__ labels, float* __restrict__ scores,
                                     float* buf, int buf_floats, int* s_last) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  constexpr int kB = 32;  // slots read per batch (independent atomics in flight)
  const unsigned G = gridDim.x, ng = G < kGroups ? G : kGroups, g = blockIdx.x % ng;
  const unsigned gsize = G / ng + (g < G % ng ? 1u : 0u);
  const int64_t NK = (int64_t)N * K;
  float* gacc = ws.sacc + (int64_t)G * NK;
  // sum of `count` slots base[j * stride + o] in order j = 0, 1, ...
  auto ordered_sum = [&](const float* base, int64_t stride, unsigned count, int64_t o) {
    float s = 0.0f;
    for (unsigned j0 = 0; j0 < count; j0 += kB) {
      float t[kB];
#pragma unroll
      for (int j = 0; j < kB; ++j)
        t[j] = j0 + j < count ? take_and_clear(const_cast<float*>(base) + (j0 + j) * stride + o)
                              : 0.0f;
#pragma unroll
      for (int j = 0; j < kB; ++j)
        if (j0 + j < count) s += t[j];
    }
    return s;
  };
  if (tid == 0) {
    unsigned* gc = ws.group + g * (kLine / 4);
    const int last = take_ticket(gc) == gsize - 1 ? 1 : 0;
    if (last) reset_counter(gc);
    *s_last = last;
  }
  __syncthreads();
  if (!*s_last) return;
  // group g's members are workgroups g, g + ng, g + 2 ng, ...
  for (int64_t o = tid; o < NK; o += NT)
    publish_store(gacc + (int64_t)g * NK + o,
                  ordered_sum(ws.sacc + (int64_t)g * NK, (int64_t)ng * NK, gsize, o));
  wait_own_memory_ops();
  __syncthreads();
  if (tid == 0) *s_last = take_ticket(ws.counter) == ng - 1 ? 1 : 0;
  __syncthreads();
  if (!*s_last) return;
  if (NK <= buf_floats) {
    for (int64_t o = tid; o < NK; o += NT) {
      const float s = ordered_sum(gacc, NK, ng, o);
      buf[o] = s;
      if (scores) scores[o] = s;
    }
    __syncthreads();
    for (int n = tid; n < N; n += NT) {
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
    for (int n = wave; n < N; n += NT / kWave) {
      float best = -__builtin_huge_valf();
      int best_k = 0x7fffffff;
      for (int k = lane; k < K; k += kWave) {
        const float s = ordered_sum(gacc, NK, ng, (int64_t)n * K + k);
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

template <int NT = kThreads>
__device__ void publish_and_finish(const float* sl, int nb0, int nb, int N, int K, int R,
                                   const SmallWs& ws, int32_t* __restrict__ labels,
                                   float* __restrict__ scores, float* buf, int buf_floats,
                                   bool finish, bool det) {
  const int tid = threadIdx.x;
  float* my = ws.sacc + (int64_t)(blockIdx.x % R) * N * K;
  for (int p = tid; p < nb * K; p += NT) publish_add(my + (int64_t)nb0 * K + p, sl[p]);
  if (!finish) return;
  __shared__ int s_last;
  wait_own_memory_ops();
  __syncthreads();
  if (det) {
    finish_deterministic<NT>(N, K, ws, labels, scores, buf, buf_floats, &s_last);
    return;
  }
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
    for (int64_t base = 0; base < total; base += (int64_t)NT * kBatch) {
      float v[kBatch];
#pragma unroll
      for (int j = 0; j < kBatch; ++j) {
        const int64_t i = base + (int64_t)j * NT + tid;
        v[j] = i < total ? take_and_clear(ws.sacc + i) : 0.0f;
      }
#pragma unroll
      for (int j = 0; j < kBatch; ++j) {
        const int64_t i = base + (int64_t)j * NT + tid;
        if (i < total) buf[i] = v[j];
      }
    }
    __syncthreads();
    for (int64_t o = tid; o < NK; o += NT) {
      float s = 0.0f;
      for (int r = 0; r < R; ++r) s += buf[r * NK + o];
      buf[o] = s;  // replica 0's slot now holds the total
      if (scores) scores[o] = s;
    }
    __syncthreads();
    for (int n = tid; n < N; n += NT) {
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
    for (int n = wave; n < N; n += (NT / kWave)) {
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


constexpr int kMfmaSteps[] = {12, 24, 36, 48};  // 4-row steps per wave: F <= 16 * MS

struct SmallPlan {
  bool flat;  // one block per workgroup (N <= 8)
  int rpt;    // flat kernel: rows per thread per chunk
  bool bmfma;  // block matrix-core kernel (one block per workgroup, N <= 32)
  bool frag;   // fragment matrix-core kernel (packed model)
  int cslots;  // fragment kernel: C slots (blocks per workgroup)
  int npass;   // fragment kernel: sample passes (2: two passes of 32, B kept in registers)
  bool mfma;
  int nb;    // VALU samples per pass, or MFMA sample tiles
  int ms;    // MFMA steps per wave
  int FC;    // VALU f-chunk
  size_t lds;
  int grid;
  int nblocks;
};

// The last workgroup reuses all of LDS to sum the R score replicas, so give
// the launch at least R*N*K floats when that fits.
inline void widen_for_final(SmallPlan& p, int64_t N, int64_t K) {
  const size_t want = sizeof(float) * (size_t)replicas(p.grid, (int)(N * K)) * N * K;
  if (p.lds < want && want <= (size_t)kLdsBudget) p.lds = want;
}

// Lets a kernel use up to kLdsBudget bytes of dynamic LDS on the current
// device (set once per device and kernel).
template <auto Kernel>
hipError_t allow_lds() {
  static PerDeviceOnce once;  // one per kernel: the template argument is its address
  return once_per_device(once, [] {
    return hipFuncSetAttribute(reinterpret_cast<const void*>(Kernel),
                               hipFuncAttributeMaxDynamicSharedMemorySize, kLdsBudget);
  });
}

// Kernel argument `act` of the small-batch kernels: bit 0 the activation
// (1 = identity), bit 1 the deterministic reduction.
constexpr int kActDet = kSmallActDet;

struct Args {
  const void *X, *B, *C;
  int32_t* labels;
  float* scores;
  int N, F, D, K, act;
  void* ws;
  hipStream_t stream;
};

__device__ __forceinline__ int xcd_block(int b, int G) {
  // contiguous column ranges per XCD (blocks sharing L2 lines meet in one L2)
  const int per = G / 8, rem = G % 8, x = b % 8, j = b / 8;
  return x * per + min(x, rem) + j;
}

constexpr int kFragThreads = 512;
constexpr int kFragMaxK = 16;

// LDS floats of the streaming kernel's C and X regions (the same column
// split as the fragment kernel). C is filled in 1 KiB (256-float) pieces by
// buffer-to-LDS loads, so both are rounded up to whole pieces; the X region
// also holds a zeroed run of 16*MS floats after the X rows and 4 spare
// floats.
__host__ __device__ inline int frag_cs_floats(int cslots, int K) {
  return (cslots * K * kW + 255) / 256 * 256;
}
__host__ __device__ inline int frag_xs_floats(int NB, int F, int MS) {
  const int chunks = (NB * F / 4 + 63) / 64 * 256;
  const int run = NB * F + 16 * MS;
  return (chunks > run ? chunks : run) + 4;
}

// Streaming kernel (hd_stream.hip).
struct StreamArgs {
  const void *X, *frag, *C;
  const unsigned* ready;
  int32_t* labels;
  float* scores;
  unsigned* done;
  int nbatch, N, F, K, act;
  void* ws;
  hipStream_t stream;
};
size_t stream_workspace_bytes(int64_t nbatch, int64_t N, int64_t K);
hipError_t launch_stream_family(const SmallPlan& p, const StreamArgs& a);

// Launchers, one translation unit per kernel family. Each applies the
// plan (tile counts, steps, LDS bytes) to its kernel template.
hipError_t launch_valu_family(SmallPlan& p, const Args& a, int dt, int lay);
hipError_t launch_flat_family(const SmallPlan& p, const Args& a, int dt, int lay);
hipError_t launch_mfma_family(SmallPlan& p, const Args& a, int lay);
hipError_t launch_bmfma_family(SmallPlan& p, const Args& a, int lay);
hipError_t launch_frag_family(SmallPlan& p, const Args& a, const void* frag, int dt);
hipError_t launch_pack_frag(const void* B, void* out, int64_t F, int64_t D, int64_t nblk, int ms,
                            int dt, hipStream_t stream);

}  // namespace sp
}  // namespace hd
