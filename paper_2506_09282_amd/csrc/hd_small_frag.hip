// Small-batch matrix-core kernel on the packed fragment layout.
#include <type_traits>

#include "hd_small.hpp"

namespace hd {
namespace sp {

namespace {

// ---------------------------------------------------------------------------
// Fragment matrix-core kernel (8 < N <= 64, packed model). Compute wave w
// owns the 4*MS rows f = 4*MS*w .. 4*MS*w + 4*MS - 1 of F.
//   fp32: the packed model holds, per 16-column block, the 16x16x4 A operands
//     in the order the waves consume them (see pack_frag_kernel): lane
//     l = (d, q), d = l % 16, q = l / 16, covers the MS consecutive rows
//     f = 4*MS*w + MS*q + 0..MS-1 of column 16 blk + d, four rows per float4,
//     so a block costs each lane MS/4 16-byte loads and each wave-wide load
//     is one contiguous 1 KiB run. Matrix step s multiplies row
//     4*MS*w + MS*q + s (lane group q) with the same rows of X^T, read from a
//     verbatim copy of X in LDS.
//   bf16: the A operands of v_mfma_f32_16x16x32_bf16 (see pack_frag16_kernel):
//     step s of wave w, lane (d, q) holds the eight bf16 of rows
//     f = 4*MS*w + 32*s + 8*q + 0..7 of column 16 blk + d (zero past the
//     wave's rows or F), S16 = ceil(MS/8) steps, one 16-byte load each; X is
//     staged in LDS as bf16 and each lane's eight X values are assembled
//     from aligned dwords. The matrix instruction's k index is the same
//     row of both operands, and its 16x16 result has the fp32 instruction's
//     layout, so everything after the matrix steps is shared.
//   int8: the same steps on v_mfma_i32_16x16x32_i8, eight int8 rows per lane
//     and step in an 8-byte word (see pack_frag8_kernel); X is staged as
//     int8. The int32 results are exact and convert exactly to fp32 while
//     |V| <= 2^24 (F <= 1024 rows of products of at most 2^14), and the
//     finish work then adds integers below 2^24, so the int8 path is exact.
//
// Persistent, one 512-thread workgroup per CU walking its column blocks,
// with the waves split by role so that memory, matrix and reduction work
// overlap:
//   waves 4..7 (compute): hold three blocks of B in flight and run the
//     matrix instructions of block i, leaving their partial V (each over a
//     quarter of F) in red[i % 2];
//   waves 0..3 (finish): first stage X and the C values of every block of
//     the workgroup into LDS (their loads do not queue behind B, since load
//     counters are per wave), then, while block i is multiplied, turn block
//     i-1's partials into HardSign values (Eq. 1) and multiply them with
//     the block's C on the fp32 matrix instruction (Eq. 8).
// One barrier per block hands red from one role to the other.
// LDS: red[2][4 waves][NTI][4 q][64 lanes] | cs[cslots][K*16] |
//      xs: fp32 [NB*F + 16*MS] (+ 4 spare), bf16 [NB*F + 32*MS] (+ 8 spare),
//      int8 [NB*F + 32*MS] (+ 16 spare); cslots >= blocks per workgroup
// ---------------------------------------------------------------------------

// One block's A operands per lane: MS/4 float4 (fp32), or ceil(MS/8) words
// of eight elements (uint4 of bf16, uint2 of int8).
template <int MS, int ESZ>
struct FragBuf {
  using Word = std::conditional_t<ESZ == 4, float4, std::conditional_t<ESZ == 2, uint4, uint2>>;
  Word a[ESZ == 4 ? MS / 4 : (MS + 7) / 8];
};

// Four consecutive elements starting at element 4*i (16-byte or 8-byte aligned), as fp32.
__device__ __forceinline__ float4 load4w(const float* p, int64_t i) {
  return reinterpret_cast<const float4*>(p)[i];
}
__device__ __forceinline__ float4 load4w(const bf16raw* p, int64_t i) {
  const uint2 u = reinterpret_cast<const uint2*>(p)[i];
  return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u),
                     __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xffff0000u));
}
__device__ __forceinline__ float4 load4w(const int8_t* p, int64_t i) {
  const uint32_t u = reinterpret_cast<const uint32_t*>(p)[i];
  return make_float4((float)(int8_t)(u & 0xff), (float)(int8_t)((u >> 8) & 0xff),
                     (float)(int8_t)((u >> 16) & 0xff), (float)(int8_t)(u >> 24));
}

template <typename T, int NTI, int MS, bool RING, int NPASS>
__global__ __launch_bounds__(kFragThreads, 1) void small_frag_mfma_kernel(
    const T* __restrict__ X, const float4* __restrict__ Bf, const T* __restrict__ C,
    int32_t* __restrict__ labels, float* __restrict__ scores, int N, int F, int D, int K, int act,
    int nblocks, int cslots, int lds_floats, void* __restrict__ workspace) {
  static_assert(NPASS == 1 || !RING, "two sample passes keep every block of B in registers");
  constexpr int ESZ = (int)sizeof(T);
  constexpr bool N16 = ESZ == 2;  // bf16 operands
  constexpr bool N8 = ESZ == 1;   // int8 operands
  constexpr bool NARROW = ESZ < 4;  // 32-row steps of eight elements per lane
  constexpr int NB = 16 * NTI;  // samples per pass
  constexpr int G4 = MS / 4;
  constexpr int S16 = (MS + 7) / 8;
  constexpr int NW = NARROW ? S16 : G4;  // A operand words per lane per block
  // X operands: they do not depend on the block, so when the registers allow
  // they are read from LDS once per pass into registers (no LDS latency
  // between matrix instructions)
  // (registers: three B buffers and NTI X words of NW words each)
  constexpr int kWordRegs = ESZ == 1 ? 2 : 4;
  constexpr bool kXReg = (3 + NTI) * NW * kWordRegs <= 180;
  extern __shared__ __attribute__((aligned(16))) float smem[];
  float* red = smem;                         // [2][4][NTI][4][64]
  float* cs = red + 2 * kWaves * NTI * 256;  // [cslots][K*16]: C of block i at slot i
  float* xs = cs + cslots * K * kW;          // X of one pass (fp32 or bf16)
  const SmallWs ws = small_ws(workspace);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const bool compute = wave >= kWaves;
  const int cw = wave - kWaves;  // compute wave index
  const int G = gridDim.x;
  const BlockWalk walk = block_walk(blockIdx.x, G, nblocks);
  const bool det = (act & kActDet) != 0;
  act &= 1;
  const int R = det ? G : replicas(G, N * K);
  const int nmine = walk.count();
  // A workgroup may own no block (when the blocks of an XCD are fewer than
  // its workgroups). The two roles' barrier counts below assume at least one
  // block, so such a workgroup only takes its ticket: it has nothing to add.
  if (nmine == 0) {
    publish_and_finish<kFragThreads>(smem, 0, 0, N, K, R, ws, labels, scores, smem, lds_floats,
                                     true, det);
    return;
  }

  // The two roles run separate code paths from the first instruction, with
  // the same barrier count (nmine + 2), so that the compiler's load-counter
  // bookkeeping for one role's loads never merges with the other's: each
  // matrix step then waits only for its own block's B, not for loads issued
  // after it.
  if (compute) {
    // B fragments of blocks 0, 1, 2. Blocks past the workgroup's last one
    // are "loaded" from a single broadcast address (one 16-byte request per
    // wave instruction), so the load count per step never depends on a branch.
    using Buf = FragBuf<MS, ESZ>;
    using Word = typename Buf::Word;
    const Word* Bw = reinterpret_cast<const Word*>(Bf);
    Buf b0, b1, b2;
    auto load_b = [&](Buf& x, int i) {
      const Word* p = i < nmine
          ? Bw + ((int64_t)walk.block_of(i) * kWaves + cw) * NW * kWave + lane : Bw;
      const int stride = i < nmine ? kWave : 0;
#pragma unroll
      for (int g = 0; g < NW; ++g) x.a[g] = p[g * stride];
    };
    load_b(b0, 0);  // blocks 1 and 2 go out after the barrier, so that X
    __syncthreads();  // competes with one block of B only; X and C are in LDS
    load_b(b1, 1);

    // fp32: this lane's X^T rows start at xoff; bf16, int8: its eight X
    // values of step s, tile t start at element xoff + 16*t*F + 32*s
    const int xoff = NARROW ? (lane & 15) * F + 4 * MS * cw + 8 * (lane >> 4)
                            : (lane & 15) * F + 4 * MS * cw + MS * (lane >> 4);
    // eight consecutive bf16 X values from element e: the five dwords that
    // hold elements e - e % 2 .. e + 9, realigned by 0 or 2 bytes
    auto x16 = [&](int e) {
      const uint32_t* q = reinterpret_cast<const uint32_t*>(xs) + (e >> 1);
      const uint32_t w0 = q[0], w1 = q[1], w2 = q[2], w3 = q[3], w4 = q[4];
      const uint32_t sh = (uint32_t)(e & 1) * 2;
      return make_uint4(__builtin_amdgcn_alignbyte(w1, w0, sh), __builtin_amdgcn_alignbyte(w2, w1, sh),
                        __builtin_amdgcn_alignbyte(w3, w2, sh), __builtin_amdgcn_alignbyte(w4, w3, sh));
    };
    // eight consecutive int8 X values from element e: three aligned dwords
    // realigned by 0..3 bytes
    auto x8 = [&](int e) {
      const uint32_t* q = reinterpret_cast<const uint32_t*>(xs) + (e >> 2);
      const uint32_t w0 = q[0], w1 = q[1], w2 = q[2];
      const uint32_t sh = (uint32_t)(e & 3);
      return make_uint2(__builtin_amdgcn_alignbyte(w1, w0, sh), __builtin_amdgcn_alignbyte(w2, w1, sh));
    };
    using XWord = typename Buf::Word;
    XWord xr[kXReg ? NW : 1][kXReg ? NTI : 1];
    auto x_word = [&](int g, int t) -> XWord {
      if constexpr (N16) {
        return x16(xoff + 16 * t * F + 32 * g);
      } else if constexpr (N8) {
        return x8(xoff + 16 * t * F + 32 * g);
      } else {
        const float* q = xs + xoff + 16 * t * F + 4 * g;
        return make_float4(q[0], q[1], q[2], q[3]);
      }
    };
    auto read_x = [&] {
      if constexpr (kXReg) {
#pragma unroll
        for (int g = 0; g < NW; ++g)
#pragma unroll
          for (int t = 0; t < NTI; ++t) xr[g][t] = x_word(g, t);
      }
    };
    read_x();
    load_b(b2, 2);
    auto multiply = [&](const Buf& x, int i) {
      // two independent accumulator chains per sample tile, interleaved over
      // the tiles (fp32: steps 4g, 4g+2 and 4g+1, 4g+3; bf16, int8: even and
      // odd 32-row steps)
      using Acc = std::conditional_t<N8, i32x4, f32x4>;
      Acc acc[NTI][2];
#pragma unroll
      for (int t = 0; t < NTI; ++t) acc[t][0] = acc[t][1] = Acc{0, 0, 0, 0};
#pragma unroll
      for (int g = 0; g < NW; ++g) {
        XWord xg[NTI];
#pragma unroll
        for (int t = 0; t < NTI; ++t) {
          if constexpr (kXReg) {
            xg[t] = xr[g][t];
          } else {
            xg[t] = x_word(g, t);
          }
        }
        if constexpr (N16) {
#pragma unroll
          for (int t = 0; t < NTI; ++t)
            acc[t][g & 1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(bf16x8, x.a[g]), __builtin_bit_cast(bf16x8, xg[t]),
                acc[t][g & 1], 0, 0, 0);
        } else if constexpr (N8) {
#pragma unroll
          for (int t = 0; t < NTI; ++t)
            acc[t][g & 1] = __builtin_amdgcn_mfma_i32_16x16x32_i8(
                __builtin_bit_cast(long, x.a[g]), __builtin_bit_cast(long, xg[t]),
                acc[t][g & 1], 0, 0, 0);
        } else {
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
      }
      // lane l holds V^T[d = 4(l/16) + q][n = l%16], q = 0..3; value q goes
      // to plane q of red[i % 2][cw][t], at position l (conflict-free)
      float* r = red + ((i & 1) * kWaves + cw) * NTI * 256 + lane;
#pragma unroll
      for (int t = 0; t < NTI; ++t)
#pragma unroll
        for (int q = 0; q < 4; ++q) r[t * 256 + q * 64] = (float)(acc[t][0][q] + acc[t][1][q]);
    };
    // Step i (one barrier each): multiply block i and reload its buffer with
    // block i+3. B buffers are named per step (no register copies, which
    // would wait on the loads).
    if constexpr (!RING) {
      // At most three blocks per workgroup: straight-line steps, no reloads.
      // Without a loop the compiler counts the outstanding loads exactly, so
      // step i waits only for block i (the ring's loop makes it wait for
      // loads issued after block i as well). A second pass of samples reuses
      // the three blocks held in registers.
#pragma unroll
      for (int pass = 0; pass < NPASS; ++pass) {
        if (pass > 0) {
          __syncthreads();  // the finish waves' last step of the previous pass
          __syncthreads();  // this pass's X is in LDS
          read_x();
        }
        // Barriers: the finish waves take one for the first X, nmine + 1 per
        // pass (their step loop) and one for each further pass's X; these
        // waves take the first X's, nmine per pass, two between passes (the
        // finish waves' last step, the next X) and one at the end.
        multiply(b0, 0);
        __syncthreads();
        if (nmine > 1) {
          multiply(b1, 1);
          __syncthreads();
        }
        if (nmine > 2) {
          multiply(b2, 2);
          __syncthreads();
        }
      }
    } else {
      auto stepc = [&](Buf& b, int i) {
        multiply(b, i);
        load_b(b, i + 3);
        __syncthreads();
      };
      for (int it = 0; it < nmine; it += 3) {
        stepc(b0, it);
        if (it + 1 >= nmine) break;
        stepc(b1, it + 1);
        if (it + 2 >= nmine) break;
        stepc(b2, it + 2);
      }
    }
    __syncthreads();  // the finish waves' last step
  } else {
    // X copied verbatim into LDS (xs[n*F + f], the pass's rows). Each
    // workgroup starts at a different offset so that they do not all read the
    // same L2 lines at once; stores are unconditional (past the end they go
    // to the spare slot) so that no load is sunk to its store. Steps past F
    // read the next row (finite values times zero B) or, after the last row,
    // the zeroed run of 16*MS floats. Rows of a pass start 16-byte aligned
    // (NB*F floats per pass, NB a multiple of 16).
    // X moves in 16-byte words of 16 / ESZ elements, staged as it is
    // (a native vector type: HIP's uint4 copied as a whole goes through the stack)
    using SWord = std::conditional_t<NARROW, i32x4, float4>;
    constexpr int EPW = 16 / ESZ;  // elements per word
    constexpr int ZRUN = NARROW ? 32 * MS : 16 * MS;  // zeroed elements after the rows
    // words per thread for NB rows of up to 16*MS elements: NB*16*MS / (EPW * 256)
    constexpr int kXBw = (NTI * MS + EPW - 1) / EPW;
    constexpr int kXB = kXBw < 40 ? kXBw : 40;
    SWord* xsw = reinterpret_cast<SWord*>(xs);
    const int spare = (NB * F + ZRUN + EPW - 1) / EPW;
    struct XBatch {
      SWord v[kXB];
      int at[kXB];
    };
    auto x_rows = [&](int pass) { return min(NB, N - NB * pass); };
    // loads of one batch of the pass's words (base: first word index). A
    // pass has at least one word: the first has more than 8 rows of F >= 4,
    // and a second pass is planned only for rows too long for one pass.
    auto x_load = [&](XBatch& xb, int pass, int base) {
      const T* Xp = X + (int64_t)NB * pass * F;
      const int nw = x_rows(pass) * F / EPW;
      const int rot = (int)(((int64_t)blockIdx.x * 37 * 64) % nw);
#pragma unroll
      for (int j = 0; j < kXB; ++j) {
        const int i = base + j * kThreads + tid;
        const int r = i + rot >= nw ? i + rot - nw : i + rot;
        xb.at[j] = i < nw ? r : spare;
        if constexpr (NARROW)
          xb.v[j] = reinterpret_cast<const i32x4*>(Xp)[i < nw ? r : rot];
        else
          xb.v[j] = load4w(Xp, i < nw ? r : rot);
      }
    };
    auto x_store = [&](const XBatch& xb) {
#pragma unroll
      for (int j = 0; j < kXB; ++j) xsw[xb.at[j]] = xb.v[j];
    };
    // the rest of the pass after its first batch: further batches, the
    // elements past the last whole word, and the zeroed run
    auto x_finish = [&](int pass) {
      const T* Xp = X + (int64_t)NB * pass * F;
      const int rows = x_rows(pass), nw = rows * F / EPW;
      for (int base = kThreads * kXB; base < nw; base += kThreads * kXB) {
        XBatch xb;
        x_load(xb, pass, base);
        x_store(xb);
      }
      if constexpr (NARROW) {
        using E = std::conditional_t<N16, unsigned short, unsigned char>;
        E* xh = reinterpret_cast<E*>(xs);
        const E* Xh = reinterpret_cast<const E*>(Xp);
        for (int e = EPW * nw + tid; e < rows * F; e += kThreads) xh[e] = Xh[e];
        for (int e = tid; e < ZRUN; e += kThreads) xh[rows * F + e] = 0;
      } else {
        for (int e = EPW * nw + tid; e < rows * F; e += kThreads) xs[e] = load_elem(Xp, e);
        for (int e = tid; e < ZRUN; e += kThreads) xs[rows * F + e] = 0.0f;
      }
    };
    {
      XBatch xb;
      x_load(xb, 0, 0);
      x_store(xb);
    }
    x_finish(0);
    // block i's K*16 C values are one contiguous run of the column tiles
    const int kc4 = K * kW / 4;
    for (int e = tid; e < nmine * kc4; e += kThreads) {
      const int b = e / kc4, r = e - b * kc4;
      reinterpret_cast<float4*>(cs)[e] = load4w(C + (int64_t)walk.block_of(b) * K * kW, r);
    }
    __syncthreads();

    // Block i's partial scores (Eq. 1, Eq. 8) on the fp32 matrix
    // instruction. On this chip fp32 VALU instructions do not overlap the
    // fp32 matrix instructions of their SIMD, so every finish instruction
    // adds to the matrix time of its SIMD; one matrix instruction per tile
    // replaces the per-class multiply-adds. Finish wave fw takes the
    // columns d = 4j + fw (j = 0..3) of every tile: lane l sums the four
    // wave partials of V^T[d = 4(l/16) + fw][n = l%16] (plane fw of red),
    // applies HardSign, and feeds it as the B operand (k = l/16, column n)
    // of S^T += C_blk · H^T, whose A operand is C[k = l%16][4(l/16) + fw]
    // (rows past K repeat class K-1 and are never read). The result,
    // S^T[4(l/16) + r][l%16], accumulates over the blocks; the four waves'
    // sums are added once, at publication. Columns past D need no mask:
    // the packed C is zero there.
    const int fw = wave;
    const float* cl = cs + min(lane & 15, K - 1) * kW + 4 * (lane >> 4) + fw;
    f32x4 sacc[NPASS][NTI];
#pragma unroll
    for (int p = 0; p < NPASS; ++p)
#pragma unroll
      for (int t = 0; t < NTI; ++t) sacc[p][t] = f32x4{0, 0, 0, 0};
    auto finish = [&](int i, f32x4 (&sa)[NTI]) {
      const float cv = cl[i * K * kW];
      const float* r = red + (i & 1) * kWaves * NTI * 256 + fw * 64 + lane;
#pragma unroll
      for (int t = 0; t < NTI; ++t) {
        const float* q = r + t * 256;
        const float v = (q[0] + q[NTI * 256]) + (q[2 * NTI * 256] + q[3 * NTI * 256]);
        sa[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(cv, activate(v, act), sa[t], 0, 0, 0);
      }
    };
    // Step i (one barrier each, nmine + 1 steps per pass): finish block i-1
    // while the compute waves multiply block i. With a second pass, its X is
    // requested at the start of the first pass and stored once the compute
    // waves no longer read the first pass's X: after step 0 when they hold X
    // in registers, else after the pass.
#pragma unroll
    for (int pass = 0; pass < NPASS; ++pass) {
      XBatch next;
      const bool more = pass + 1 < NPASS;
      if (more) x_load(next, pass + 1, 0);
      const bool early = more && kXReg;
      for (int i = 0; i <= nmine; ++i) {
        if (i > 0) finish(i - 1, sacc[pass]);
        if (early && i == 1) x_store(next);
        __syncthreads();
      }
      if (more) {
        if (!early) x_store(next);
        x_finish(pass + 1);
        __syncthreads();  // the next pass's X is in LDS
      }
    }
    // Each wave's sums, [fw][pass][t][lane][4], into red (no longer read by
    // the compute waves after the last step's barrier).
    f32x4* part = reinterpret_cast<f32x4*>(red) + fw * NPASS * NTI * 64 + lane;
#pragma unroll
    for (int p = 0; p < NPASS; ++p)
#pragma unroll
      for (int t = 0; t < NTI; ++t) part[(p * NTI + t) * 64] = sacc[p][t];
  }
  __syncthreads();
  // The workgroup's partial scores: sample n = NB*p + 16t + j, class k is
  // element k % 4 of lane 16(k/4) + j of each finish wave's tile (p, t),
  // summed over the four waves in a fixed order.
  {
    float* my = ws.sacc + (int64_t)(blockIdx.x % R) * N * K;
    const int rows = min(NPASS * NB, N);
    const float* part = red;
    for (int e = tid; e < rows * K; e += kFragThreads) {
      const int n = e / K, k = e - n * K;
      const int pt = n >> 4;  // pass * NTI + tile
      const int o = (pt * 64 + (k >> 2) * 16 + (n & 15)) * 4 + (k & 3);
      constexpr int WS = NPASS * NTI * 256;  // one wave's sums
      publish_add(my + e, (part[o] + part[o + WS]) + (part[o + 2 * WS] + part[o + 3 * WS]));
    }
  }
  publish_and_finish<kFragThreads>(smem, 0, 0, N, K, R, ws, labels, scores, smem, lds_floats,
                                   true, det);
}

// Writes the fragment section: out[((blk*4 + w)*(MS/4) + g)*64 + l][e] =
// B[4*MS*w + MS*(l/16) + 4g + e][16 blk + l%16], zero past F or D (fp32).
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
    out[i] = (f < F && col < D) ? load_elem(B, f * D + col) : 0.0f;
  }
}

// Writes the bf16 fragment section: word ((blk*4 + w)*S16 + s)*64 + l holds
// the eight bf16 B[f][16 blk + l%16], f = 4*MS*w + 32*s + 8*(l/16) + 0..7,
// zero where that row is past the wave's 4*MS rows, past F or past D.
__global__ __launch_bounds__(256) void pack_frag16_kernel(const bf16raw* __restrict__ B,
                                                          uint4* __restrict__ out, int64_t F,
                                                          int64_t D, int64_t nblk, int MS) {
  const int S16 = (MS + 7) / 8;
  const int64_t per_blk = (int64_t)4 * S16 * 64;  // words per 16-column block
  const int64_t total = nblk * per_blk;
  const unsigned short* Bh = reinterpret_cast<const unsigned short*>(B);
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * 256) {
    const int64_t l = i % 64, s = (i / 64) % S16, w = (i / (64 * S16)) % 4, blk = i / per_blk;
    const int64_t col = blk * kW + l % 16;
    uint32_t h[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int64_t r = 32 * s + 8 * (l / 16) + j;  // row within the wave's share
      const int64_t f = 4 * MS * w + r;
      h[j] = (r < 4 * MS && f < F && col < D) ? Bh[f * D + col] : 0u;
    }
    out[i] = make_uint4(h[0] | h[1] << 16, h[2] | h[3] << 16, h[4] | h[5] << 16, h[6] | h[7] << 16);
  }
}

// Writes the int8 fragment section: word ((blk*4 + w)*S16 + s)*64 + l holds
// the eight int8 B[f][16 blk + l%16], f = 4*MS*w + 32*s + 8*(l/16) + 0..7,
// zero where that row is past the wave's 4*MS rows, past F or past D.
__global__ __launch_bounds__(256) void pack_frag8_kernel(const int8_t* __restrict__ B,
                                                         uint2* __restrict__ out, int64_t F,
                                                         int64_t D, int64_t nblk, int MS) {
  const int S16 = (MS + 7) / 8;
  const int64_t per_blk = (int64_t)4 * S16 * 64;  // words per 16-column block
  const int64_t total = nblk * per_blk;
  const uint8_t* Bb = reinterpret_cast<const uint8_t*>(B);
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * 256) {
    const int64_t l = i % 64, s = (i / 64) % S16, w = (i / (64 * S16)) % 4, blk = i / per_blk;
    const int64_t col = blk * kW + l % 16;
    uint32_t b[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int64_t r = 32 * s + 8 * (l / 16) + j;  // row within the wave's share
      const int64_t f = 4 * MS * w + r;
      b[j] = (r < 4 * MS && f < F && col < D) ? Bb[f * D + col] : 0u;
    }
    out[i] = make_uint2(b[0] | b[1] << 8 | b[2] << 16 | b[3] << 24,
                        b[4] | b[5] << 8 | b[6] << 16 | b[7] << 24);
  }
}


template <typename T, int NTI, int MS, bool RING, int NPASS>
hipError_t launch_frag_t(const SmallPlan& p, const Args& a, const void* frag) {
  const hipError_t attr = allow_lds<&small_frag_mfma_kernel<T, NTI, MS, RING, NPASS>>();
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL((small_frag_mfma_kernel<T, NTI, MS, RING, NPASS>), dim3(p.grid),
                     dim3(kFragThreads), p.lds, a.stream, (const T*)a.X, (const float4*)frag,
                     (const T*)a.C, a.labels, a.scores, a.N, a.F, a.D, a.K, a.act, p.nblocks,
                     p.cslots, (int)(p.lds / sizeof(float)), a.ws);
  return hipGetLastError();
}

// The ring (reloads inside a loop) only where some workgroup walks more than
// three blocks; the first workgroup of each XCD walks the most. Two sample
// passes (planned only without the ring) for 32 < N <= 64 when X of all the
// samples does not fit LDS.
template <typename T, int NTI, int MS>
hipError_t launch_frag(const SmallPlan& p, const Args& a, const void* frag) {
  if constexpr (NTI == 2) {
    if (p.npass == 2) return launch_frag_t<T, 2, MS, false, 2>(p, a, frag);
  }
  if (p.npass != 1) return hipErrorInvalidValue;
  int most = 0;
  for (int x = 0; x < 8; ++x) {
    const int c = block_walk(x, p.grid, p.nblocks).count();
    most = c > most ? c : most;
  }
  return most > 3 ? launch_frag_t<T, NTI, MS, true, 1>(p, a, frag)
                  : launch_frag_t<T, NTI, MS, false, 1>(p, a, frag);
}

template <typename T, int NTI>
hipError_t launch_frag_ms(const SmallPlan& p, const Args& a, const void* frag) {
  switch (p.ms) {
    case 12: return launch_frag<T, NTI, 12>(p, a, frag);
    case 24: return launch_frag<T, NTI, 24>(p, a, frag);
    case 36: return launch_frag<T, NTI, 36>(p, a, frag);
    case 48: return launch_frag<T, NTI, 48>(p, a, frag);
    default: return launch_frag<T, NTI, 64>(p, a, frag);
  }
}

template <typename T>
hipError_t launch_frag_nti(const SmallPlan& p, const Args& a, const void* frag) {
  switch (p.nb) {
    case 1: return launch_frag_ms<T, 1>(p, a, frag);
    case 2: return launch_frag_ms<T, 2>(p, a, frag);
    case 3: return launch_frag_ms<T, 3>(p, a, frag);
    default: return launch_frag_ms<T, 4>(p, a, frag);
  }
}

}  // namespace

hipError_t launch_frag_family(SmallPlan& p, const Args& a, const void* frag, int dt) {
  widen_for_final(p, a.N, a.K);
  if (dt == 2) return launch_frag_nti<int8_t>(p, a, frag);
  return dt == 0 ? launch_frag_nti<float>(p, a, frag) : launch_frag_nti<bf16raw>(p, a, frag);
}

hipError_t launch_pack_frag(const void* B, void* out, int64_t F, int64_t D, int64_t nblk, int ms,
                            int dt, hipStream_t stream) {
  if (dt >= 1) {
    const int64_t gn = cdiv(nblk * 4 * ((ms + 7) / 8) * 64, 256);
    const dim3 g((unsigned)(gn < 65536 ? gn : 65536));
    if (dt == 1)
      hipLaunchKernelGGL(pack_frag16_kernel, g, dim3(256), 0, stream, (const bf16raw*)B,
                         static_cast<uint4*>(out), F, D, nblk, ms);
    else
      hipLaunchKernelGGL(pack_frag8_kernel, g, dim3(256), 0, stream, (const int8_t*)B,
                         static_cast<uint2*>(out), F, D, nblk, ms);
    return hipGetLastError();
  }
  const int64_t g = cdiv(nblk * 256 * ms, 256);
  const dim3 grid((unsigned)(g < 65536 ? g : 65536));
  hipLaunchKernelGGL(pack_frag_kernel, grid, dim3(256), 0, stream, (const float*)B,
                     static_cast<float*>(out), F, D, nblk, ms);
  return hipGetLastError();
}

}  // namespace sp
}  // namespace hd
