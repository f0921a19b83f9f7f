// Streaming inference: one persistent launch consumes a queue of small batches
// against a model whose share of B stays in registers for the whole stream.
//
// This is the GPU form of the paper's producer-consumer pipeline for a
// continuous stream of small batches (Sec. I: real-time streams; Sec. III-A:
// producer and consumer thread pools joined by queues; Sec. III-C Alg. 3: the
// small-batch variant that splits the hypervector dimension D). Each
// workgroup owns up to three 16-column blocks of the packed fragment model
// (the same column split as the single-batch fragment kernel), loads them
// into registers once, and then, batch after batch:
//   - its compute waves run Stage I (Eq. 7) on the matrix cores,
//   - its finish waves apply HardSign (Eq. 1) and form the block's partial
//     scores (Eq. 8) on the fp32 matrix instruction,
//   - one wave prefetches the next batch's X into LDS (the queue, Sec. III-A),
//   - one wave publishes the previous batch's partial scores (fp32 atomics
//     into one of a few replicas) and then counts itself into that batch's
//     "published" counter,
// and one extra workgroup, the reducer, sums each batch's replicas once all
// compute workgroups have published it, takes the argmax (Eq. 9) and writes
// the labels; compute workgroups never wait for it. B is read from memory
// once per launch instead of once per batch.
//
// Roles in a compute workgroup (512 threads, 8 waves, one per compute unit):
//   wave 0       publisher of batch i-1,
//   waves 0..3   loaders of batch i+1's X (through registers); wave 1 also
//                waits on the queue,
//   waves 2, 3   per-block finish (two of the four column phases each),
//   waves 4..7   matrix instructions, each over a quarter of F.
// All waves take part in every barrier; the publisher issues its atomics at
// the start of a batch and waits for them at its end. The reducer (the last
// workgroup, on the compute unit the others leave free) runs its eight waves
// over the batches b = w, w + 8, ...
//
// The queue: batch b may be read once *ready > b (ready NULL: every batch is
// present at launch). The loader polls with a relaxed system-scope load and
// an acquire fence, so the batch's X written by the host or another device
// queue is seen. A batch that does not become ready within kSpinLimit polls
// (about half a second), or a ready value with bit 31 set, ends the stream
// after the batches already taken; *done counts the batches whose labels
// were written.
#include "hd_small.hpp"

namespace hd {
namespace sp {

namespace {

constexpr int kStreamThreads = 512;
constexpr int kStreamReplicas = 8;   // score replicas per batch
constexpr unsigned kStopBit = 0x80000000u;
constexpr int kSpinLimit = 1 << 21;  // polls of s_sleep(10): about half a second

// Workspace region of one batch: the published counter on its own line,
// then the score replicas [R][N][K].
__host__ __device__ inline size_t stream_batch_bytes(int N, int K) {
  return (size_t)kLine + ((size_t)kStreamReplicas * N * K * sizeof(float) + 255) / 256 * 256;
}

template <int MS>
struct SBuf {
  float4 a[MS / 4];
};

// Queue state of batch b: 1 ready, 0 not yet, -1 the stream has ended
// before it. With `block`, waits (polling with s_sleep) until the answer is
// not 0, giving up after kSpinLimit polls (-1).
__device__ inline int batch_state(const unsigned* ready, unsigned b, bool block) {
  if (!ready) return 1;
  for (int spin = 0; spin < kSpinLimit; ++spin) {
    const unsigned v = __hip_atomic_load(ready, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    if ((v & ~kStopBit) > b) {
      __atomic_thread_fence(__ATOMIC_ACQUIRE);  // the batch's X is visible after this
      return 1;
    }
    if (v & kStopBit) return -1;
    if (!block) return 0;
    __builtin_amdgcn_s_sleep(10);
  }
  return -1;
}

__device__ __forceinline__ void raw_barrier() {
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): this wave's LDS stores are done
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_barrier();
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

template <int NTI, int MS>
__global__ __launch_bounds__(kStreamThreads, 1) void stream_frag_kernel(
    const float* __restrict__ X, const float4* __restrict__ Bf, const float* __restrict__ C,
    const unsigned* ready, int32_t* __restrict__ labels, float* __restrict__ scores,
    unsigned* done, int nbatch, int N, int F, int K, int act, int nblocks, int cslots,
    void* __restrict__ workspace) {
  constexpr int NB = 16 * NTI;
  constexpr int G4 = MS / 4;
  extern __shared__ __attribute__((aligned(16))) float smem[];
  float* sl = smem;                              // [2][NB*K] scores of the last batch
  float* red = sl + (2 * NB * K + 3) / 4 * 4;    // [2][4][NTI][4][64]
  float* cs = red + 2 * kWaves * NTI * 256;      // C of block i at slot i
  float* xs = cs + frag_cs_floats(cslots, K);    // X, 1 KiB chunks, then a zeroed run
  __shared__ int s_stop;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const bool compute = wave >= kWaves;
  const int cw = wave - kWaves;
  const int G = gridDim.x - 1;  // compute workgroups; the last one is the reducer
  char* const wsb = static_cast<char*>(workspace);
  const size_t bbytes = stream_batch_bytes(N, K);
  const int R = G < kStreamReplicas ? G : kStreamReplicas;
  const int64_t NK = (int64_t)N * K;
  if ((int)blockIdx.x == G) {
    // Reducer: wave w takes batches w, w + 8, ...; a batch is reduced once
    // all G compute workgroups have counted themselves into it (their
    // partial scores are performed by then). It stops when the queue shows
    // the batch will never come, or after kSpinLimit polls.
    float* fin = smem + wave * NB * K;
    for (int b = wave; b < nbatch; b += kStreamThreads / kWave) {
      char* reg = wsb + kLine + (size_t)b * bbytes;
      unsigned* counter = reinterpret_cast<unsigned*>(reg);
      float* rep = reinterpret_cast<float*>(reg + kLine);
      bool ok = false;
      for (int spin = 0; spin < kSpinLimit; ++spin) {
        if (__hip_atomic_load(counter, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >= (unsigned)G) {
          ok = true;
          break;
        }
        if (ready) {
          const unsigned v = __hip_atomic_load(ready, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
          if ((v & kStopBit) && (v & ~kStopBit) <= (unsigned)b) break;
        }
        __builtin_amdgcn_s_sleep(10);
      }
      if (!ok) return;
      for (int64_t p = lane; p < NK; p += kWave) {
        float t[kStreamReplicas];
#pragma unroll
        for (int r = 0; r < kStreamReplicas; ++r)
          t[r] = r < R ? take_and_clear(rep + r * NK + p) : 0.0f;
        float sum = 0.0f;
#pragma unroll
        for (int r = 0; r < kStreamReplicas; ++r) sum += t[r];
        fin[p] = sum;
        if (scores) scores[(int64_t)b * NK + p] = sum;
      }
      __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0): fin is written (one wave)
      for (int n = lane; n < N; n += kWave) {
        float best = fin[n * K];
        int best_k = 0;
        for (int k = 1; k < K; ++k) {
          const float v = fin[n * K + k];
          if (v > best) {
            best = v;
            best_k = k;
          }
        }
        labels[(int64_t)b * N + n] = best_k;
      }
      if (lane == 0) {
        reset_counter(counter);
        if (done) __hip_atomic_fetch_add(done, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
    return;
  }
  const BlockWalk walk = block_walk(blockIdx.x, G, nblocks);
  const int nmine = walk.count();  // 0 to 3 (at most 3 is checked on the host)
  const int nb = min(NB, N);
  const int npairs = nb * K;
  const int n4 = nb * F / 4;
  const int kc4 = K * kW / 4;
  const int64_t xstride = (int64_t)N * F;

  // Batches start on 16-byte boundaries when X does and N*F % 4 == 0; then X
  // moves in 16-byte pieces, otherwise in 4-byte pieces (N*F % 4 == 0 makes
  // nb * F = 4 * n4: there is no partial piece).
  const bool x16 = ((uintptr_t)X % 16 == 0) && (xstride % 4 == 0);
  const int n1 = nb * F;  // floats of X per batch
  // X moves through the registers of waves 0..3 (256 threads): thread t
  // loads pieces t + 256 j by buffer loads (offsets past the batch read as
  // zero), all in flight at once, as soon as the batch is known to be in the
  // queue, and stores them into LDS at the end of the batch, by which time
  // they have arrived. (Buffer-to-LDS loads were measured to issue at only
  // about one 1 KiB load per 40 ns per compute unit, which held up the
  // block steps.)
  constexpr int kXL = (NB * 576 / 4 + 255) / 256;  // float4 registers per thread
  float4 xv[kXL];
  auto x_load = [&](int b, int t) {
    const float* xb = X + (int64_t)b * xstride;
    const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(xb), 0, x16 ? n4 * 16 : n1 * 4, 0x00020000);
    if (x16) {
#pragma unroll
      for (int j = 0; j < kXL; ++j)  // pieces past the batch read as zero
        xv[j] = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(
                                               xr, (unsigned)(t + 256 * j) * 16u, 0, 0));
    } else {
      // component c of xv[j] holds float t + 256 (4 j + c)
#pragma unroll
      for (int j = 0; j < kXL; ++j) {
        if (1024 * j >= n1) break;  // uniform
        float v[4];
#pragma unroll
        for (int c = 0; c < 4; ++c)
          v[c] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                                               xr, (unsigned)(t + 256 * (4 * j + c)) * 4u, 0, 0));
        xv[j] = make_float4(v[0], v[1], v[2], v[3]);
      }
    }
  };
  auto x_store = [&](int t) {
    if (x16) {
      float4* xs4 = reinterpret_cast<float4*>(xs);
#pragma unroll
      for (int j = 0; j < kXL; ++j)
        if (t + 256 * j < n4) xs4[t + 256 * j] = xv[j];
    } else {
#pragma unroll
      for (int j = 0; j < kXL; ++j) {
        const int e = t + 1024 * j;
        if (e < n1) xs[e] = xv[j].x;
        if (e + 256 < n1) xs[e + 256] = xv[j].y;
        if (e + 512 < n1) xs[e + 512] = xv[j].z;
        if (e + 768 < n1) xs[e + 768] = xv[j].w;
      }
    }
  };

  // ---- prologue: X of batch 0 and the blocks' C values first, then B ----
  __shared__ int s_next;
  if (tid == 0) s_stop = 0;
  if (tid == 64) s_next = batch_state(ready, 0u, true);
  raw_barrier();  // batch 0 is in the queue (or the stream has ended)
  const bool have0 = *(volatile int*)&s_next == 1;
  if (!compute && have0) x_load(0, tid);
  if (wave == 1) {
    const __amdgpu_buffer_rsrc_t cr4 = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(C), 0, nblocks * kc4 * 16, 0x00020000);
    const int ncc = (nmine * kc4 + kWave - 1) / kWave;
    for (int c = 0; c < ncc; ++c) {
      const int e = c * kWave + lane;
      const int bk = e / kc4;
      const unsigned off = e < nmine * kc4
          ? (unsigned)(((int64_t)walk.block_of(bk) * kc4 + (e - bk * kc4)) * 16) : 0x80000000u;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          cr4, (__attribute__((address_space(3))) void*)(cs + c * kWave * 4), 16, off, 0, 0, 0);
    }
  }
  raw_barrier();  // X and C are requested (s_stop is initialised)
  // compute waves: the workgroup's (at most three) blocks of B, resident for
  // the whole stream; blocks past the last one read a broadcast address
  SBuf<MS> b0, b1, b2;
  auto load_b = [&](SBuf<MS>& x, int i) {
    const float4* p = i < nmine
        ? Bf + ((int64_t)walk.block_of(i) * kWaves + cw) * G4 * kWave + lane : Bf;
    const int stride = i < nmine ? kWave : 0;
#pragma unroll
    for (int g = 0; g < G4; ++g) x.a[g] = p[g * stride];
  };
  if (compute) {
    load_b(b0, 0);
    load_b(b1, 1);
    load_b(b2, 2);
  } else {
    if (have0) x_store(tid);
    if (wave == 1) __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): C is in LDS
    if (!have0 && tid == 0) s_stop = 1;
    for (int e = tid; e < 16 * MS; e += 256) xs[nb * F + e] = 0.0f;
    // queue state of batch 1, read by the loaders at the top of batch 0
    if (tid == 64) s_next = 1 < nbatch ? batch_state(ready, 1u, false) : -1;
  }
  raw_barrier();

  // ---- per batch ----
  const int xoff = (lane & 15) * F + 4 * MS * cw + MS * (lane >> 4);
  float4 xr[G4][NTI];
  auto multiply = [&](const SBuf<MS>& x, int i) {
    f32x4 acc[NTI][2];
#pragma unroll
    for (int t = 0; t < NTI; ++t) acc[t][0] = acc[t][1] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int g = 0; g < G4; ++g) {
#pragma unroll
      for (int t = 0; t < NTI; ++t)
        acc[t][0] = __builtin_amdgcn_mfma_f32_16x16x4f32(x.a[g].x, xr[g][t].x, acc[t][0], 0, 0, 0);
#pragma unroll
      for (int t = 0; t < NTI; ++t)
        acc[t][1] = __builtin_amdgcn_mfma_f32_16x16x4f32(x.a[g].y, xr[g][t].y, acc[t][1], 0, 0, 0);
#pragma unroll
      for (int t = 0; t < NTI; ++t)
        acc[t][0] = __builtin_amdgcn_mfma_f32_16x16x4f32(x.a[g].z, xr[g][t].z, acc[t][0], 0, 0, 0);
#pragma unroll
      for (int t = 0; t < NTI; ++t)
        acc[t][1] = __builtin_amdgcn_mfma_f32_16x16x4f32(x.a[g].w, xr[g][t].w, acc[t][1], 0, 0, 0);
    }
    // lane l holds V^T[d = 4(l/16) + q][n = l%16], q = 0..3; value q goes
    // to plane q of red[i % 2][cw][t], at position l (conflict-free)
    float* r = red + ((i & 1) * kWaves + cw) * NTI * 256 + lane;
#pragma unroll
    for (int t = 0; t < NTI; ++t)
#pragma unroll
      for (int q = 0; q < 4; ++q) r[t * 256 + q * 64] = acc[t][0][q] + acc[t][1][q];
  };
  // Finish waves 2, 3 (fw = 0, 1): Stage II on the fp32 matrix instruction
  // (as in the single-batch fragment kernel). Wave fw takes the column
  // phases q = 2 fw, 2 fw + 1 of every sample tile: lane l sums the four
  // wave partials of V^T[4(l/16) + q][l%16] (plane q of red), applies
  // HardSign and feeds it as the B operand of S^T += C_blk · H^T, whose A
  // operand is C[k = l%16][4(l/16) + q] (rows past K repeat class K-1 and are
  // never stored). sacc[t] holds S^T[4(l/16) + r][16 t + l%16] over the
  // workgroup's blocks; the two waves' sums go to their own halves of sl and
  // are added when they are published.
  const bool finisher = wave == 2 || wave == 3;
  const int fw = wave - 2;
  const float* cl = cs + min(lane & 15, K - 1) * kW + 4 * (lane >> 4);
  f32x4 sacc[NTI];
#pragma unroll
  for (int t = 0; t < NTI; ++t) sacc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  auto finish = [&](int i) {
    if (!finisher) return;  // uniform per wave
    const float* r = red + (i & 1) * kWaves * NTI * 256 + lane;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int q = 2 * fw + h;
      const float cv = cl[i * K * kW + q];
#pragma unroll
      for (int t = 0; t < NTI; ++t) {
        const float* p = r + t * 256 + q * 64;
        const float v = (p[0] + p[NTI * 256]) + (p[2 * NTI * 256] + p[3 * NTI * 256]);
        sacc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(cv, activate(v, act), sacc[t], 0, 0, 0);
      }
    }
  };
  // Publisher (wave 0): batch b's partial scores (in sl) into replica
  // blockIdx % R of the batch's region (issued at the start of the next
  // batch), then, once they are performed (at the end of that batch), one
  // count into the batch's published counter for the reducer.
  auto publish_issue = [&](int b) {
    float* rep = reinterpret_cast<float*>(wsb + kLine + (size_t)b * bbytes + kLine);
    float* my = rep + (int64_t)(blockIdx.x % R) * NK;
    for (int p = lane; p < npairs; p += kWave) publish_add(my + p, sl[p] + sl[NB * K + p]);
  };
  auto publish_done = [&](int b) {
    unsigned* counter = reinterpret_cast<unsigned*>(wsb + kLine + (size_t)b * bbytes);
    wait_own_memory_ops();
    if (lane == 0) (void)take_ticket(counter);
  };

  // The roles run separate loops with the same barriers (so that the
  // registers holding the resident B and the X operands are live only in the
  // compute waves' loop). Each batch: B (X in registers), then one barrier
  // per block step, then the end of the batch.
  int b = 0;
  if (compute) {
    for (; b < nbatch; ++b) {
      if (*(volatile int*)&s_stop) break;  // uniform: read after a barrier
#pragma unroll
      for (int g = 0; g < G4; ++g)
#pragma unroll
        for (int t = 0; t < NTI; ++t) {
          const float* q = xs + xoff + 16 * t * F + 4 * g;
          xr[g][t] = make_float4(q[0], q[1], q[2], q[3]);
        }
      raw_barrier();  // X of batch b is in registers: the LDS buffer is free
      multiply(b0, 0);
      raw_barrier();
      if (nmine > 1) {
        multiply(b1, 1);
        raw_barrier();
      }
      if (nmine > 2) {
        multiply(b2, 2);
        raw_barrier();
      }
      raw_barrier();  // end of batch b
    }
    return;
  }
  for (; b < nbatch; ++b) {
    if (*(volatile int*)&s_stop) break;
    // Was the next batch in the queue at the end of the previous one? Then
    // waves 0..3 request its X first thing; otherwise wave 1 waits for it at
    // the end of this batch (which is not held up) and moves it alone.
    const int next0 = *(volatile int*)&s_next;
    if (next0 == 1) x_load(b + 1, tid);
    if (wave == 0 && b > 0) publish_issue(b - 1);  // sl holds batch b-1's scores
    raw_barrier();
    raw_barrier();
    if (nmine > 1) {
      finish(0);
      raw_barrier();
    }
    if (nmine > 2) {
      finish(1);
      raw_barrier();
    }
    if (nmine > 0) finish(nmine - 1);  // a workgroup may own no block (it publishes zeros)
    if (finisher) {
      float* slw = sl + fw * (NB * K);
#pragma unroll
      for (int t = 0; t < NTI; ++t) {
        const int n = 16 * t + (lane & 15);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int k = 4 * (lane >> 4) + r;
          if (k < K && n < nb) slw[n * K + k] = sacc[t][r];
        }
        sacc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
      }
    }
    if (wave == 0 && b > 0) publish_done(b - 1);
    if (next0 == 1) x_store(tid);  // X of batch b+1 (the compute waves hold b's)
    if (wave == 1 && next0 == 0) {
      if (batch_state(ready, (unsigned)(b + 1), true) == 1) {
        for (int q = 0; q < 4; ++q) {
          x_load(b + 1, lane + 64 * q);
          x_store(lane + 64 * q);
        }
      } else if (lane == 0) {
        s_stop = 1;  // read by every wave after the barrier below
      }
    }
    if (wave == 1 && next0 == -1 && b + 1 < nbatch && lane == 0) s_stop = 1;
    // queue state of batch b+2, read by the loaders at the top of batch b+1
    if (tid == 64)
      s_next = b + 2 < nbatch ? batch_state(ready, (unsigned)(b + 2), false) : -1;
    raw_barrier();  // end of batch b: its scores in sl, X of batch b+1 in LDS
  }
  if (wave == 0 && b > 0) {
    publish_issue(b - 1);
    publish_done(b - 1);
  }
}

template <int NTI, int MS>
hipError_t launch_stream_t(const SmallPlan& p, const StreamArgs& a) {
  const hipError_t attr = allow_lds<&stream_frag_kernel<NTI, MS>>();
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL((stream_frag_kernel<NTI, MS>), dim3(p.grid + 1), dim3(kStreamThreads), p.lds,
                     a.stream, (const float*)a.X, (const float4*)a.frag, (const float*)a.C,
                     a.ready, a.labels, a.scores, a.done, a.nbatch, a.N, a.F, a.K, a.act,
                     p.nblocks, p.cslots, a.ws);
  return hipGetLastError();
}

template <int NTI>
hipError_t launch_stream_ms(const SmallPlan& p, const StreamArgs& a) {
  switch (p.ms) {
    case 12: return launch_stream_t<NTI, 12>(p, a);
    case 24: return launch_stream_t<NTI, 24>(p, a);
    default: return launch_stream_t<NTI, 36>(p, a);
  }
}

}  // namespace

size_t stream_workspace_bytes(int64_t nbatch, int64_t N, int64_t K) {
  return (size_t)kLine + (size_t)nbatch * stream_batch_bytes((int)N, (int)K);
}

hipError_t launch_stream_family(const SmallPlan& p, const StreamArgs& a) {
  return p.nb == 1 ? launch_stream_ms<1>(p, a) : launch_stream_ms<2>(p, a);
}

}  // namespace sp
}  // namespace hd
