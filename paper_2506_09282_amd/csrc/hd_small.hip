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
#include "hd_small.hpp"

namespace hd {

using namespace sp;

namespace {

// The VALU kernel serves every layout and alignment; it is the support
// criterion. Returns nb == 0 when nb * K does not fit in LDS.
// Samples per pass of the VALU kernel: its X values and accumulators live in
// registers (kRpt*NB + 4*NB floats per thread), so larger batches take several
// passes. Beyond 8 (2 with scalar raw loads) the kernel spills to scratch and
// runs up to two orders of magnitude slower.
SmallPlan plan_valu(int64_t N, int64_t F, int64_t D, int64_t K, int max_nb) {
  SmallPlan p{};
  p.nblocks = (int)cdiv(D, kW);
  p.grid = p.nblocks < num_cus() ? p.nblocks : num_cus();
  int nb = N <= 1 ? 1 : N <= 2 ? 2 : N <= 4 ? 4 : 8;
  nb = nb < max_nb ? nb : max_nb;
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
  // fp32: MS/4 float4 per lane, wave and block; bf16 and int8: ceil(MS/8)
  // words of eight elements (16 or 8 bytes, the narrow matrix instructions'
  // operands)
  const int ms = frag_ms(F);
  if (dt >= 1) return (size_t)cdiv(D, kW) * 4 * ((ms + 7) / 8) * 64 * (dt == 1 ? 16 : 8);
  return (size_t)cdiv(D, kW) * 256 * ms * sizeof(float);
}

// Kernel choice: on a packed model the fragment kernel for N > 4 (every N
// for int8) when its LDS fits (at N = 8: fp32 10.8 us, bf16 9.0 us, against
// 11.6 and 10.8 us on the flat kernel); otherwise N <= 8 takes the flat
// kernel; fp32 with 8 < N <= 64 a matrix-core kernel (the block kernel for
// N <= 32 or the persistent one) when its LDS fits; raw matrices with
// unaligned bases or D % 4 != 0 (kRawScalar) and everything else take the
// VALU kernel.
SmallPlan plan_small(int64_t N, int64_t F, int64_t D, int64_t K, int dt, int lay, bool x_aligned) {
  if (lay == kRawScalar) return plan_valu(N, F, D, K, 2);
  SmallPlan v = plan_valu(N, F, D, K, 8);
  if (v.nb == 0) return v;
  SmallPlan p{};
  p.nblocks = v.nblocks;
  // int8 runs only on the fragment kernel, for every N
  if (lay == kTiled && x_aligned && (N > 4 || dt == 2) && frag_ms(F) > 0) {
    const int ms = frag_ms(F);
    int64_t cslots = 1;  // the most blocks any workgroup walks
    for (int b = 0; b < v.grid; ++b) {
      const int c = block_walk(b, v.grid, v.nblocks).count();
      cslots = c > cslots ? c : cslots;
    }
    // LDS: the partials (later each finish wave's scores), the blocks' C,
    // one pass's X (fp32: NB*F + 16*MS floats and a spare float4; bf16,
    // int8: NB*F + 32*MS elements and a spare 16-byte word)
    auto frag_floats = [&](int64_t nti) {
      const int64_t nbk = 16 * nti;
      const int64_t epw = dt == 1 ? 8 : 16;
      const int64_t xf = dt >= 1 ? ((nbk * F + 32 * ms + epw - 1) / epw + 1) * 4
                                 : (nbk * F + 16 * ms + 3) / 4 * 4 + 4;
      return 2 * kWaves * nti * 256 + cslots * K * kW + xf;
    };
    // all samples in one pass; else, when X of all of them does not fit and
    // no workgroup walks more than three blocks (B stays in registers), two
    // passes of 32
    int64_t nti = cdiv(N, 16), npass = 1;
    int64_t floats = frag_floats(nti);
    if ((int64_t)sizeof(float) * floats > kLdsBudget && N > 32 && cslots <= 3) {
      nti = 2;
      npass = 2;
      floats = frag_floats(2);
    }
    if (K <= kFragMaxK && (int64_t)sizeof(float) * floats <= kLdsBudget) {
      p.frag = true;
      p.npass = (int)npass;
      p.cslots = (int)cslots;
      p.nb = (int)nti;
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

hipError_t launch_plan(SmallPlan& p, const Args& a, int dt, int lay) {
  if (lay != kRawScalar) {
    if (p.flat) return launch_flat_family(p, a, dt, lay);
    if (dt == 0 && p.bmfma) return launch_bmfma_family(p, a, lay);
    if (dt == 0 && p.mfma) return launch_mfma_family(p, a, lay);
  }
  return launch_valu_family(p, a, dt, lay);
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

// WITH_B: the column tiles of B as well (not for int8)
template <typename T, bool WITH_B>
hipError_t pack_small_t(const void* B, const void* C, int64_t F, int64_t D, int64_t K,
                        void* out, hipStream_t stream) {
  const int64_t nblk = cdiv(D, kW);
  T* b = static_cast<T*>(out);
  T* c = reinterpret_cast<T*>(static_cast<char*>(out) +
                              (WITH_B ? (nblk * F * kW * sizeof(T) + 255) / 256 * 256 : 0));
  const int64_t gb = cdiv(nblk * F * kW, 256), gc = cdiv(nblk * K * kW, 256);
  if constexpr (WITH_B)
    hipLaunchKernelGGL(pack_small_kernel<T>, dim3((unsigned)(gb < 65536 ? gb : 65536)), dim3(256),
                       0, stream, (const T*)B, b, F, D, nblk);
  if (!C) {
    // no codebook yet (a model packed for training): class tiles are zero
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_zero(c, (size_t)nblk * K * kW * sizeof(T), stream);
  }
  hipLaunchKernelGGL(pack_small_kernel<T>, dim3((unsigned)(gc < 65536 ? gc : 65536)), dim3(256), 0,
                     stream, (const T*)C, c, K, D, nblk);
  return hipGetLastError();
}

}  // namespace

// Streaming plan: fp32, N <= 32, K <= 16, rows per lane at most 36 (F <= 576)
// and at most three blocks per workgroup, so that a compute wave's share of
// B (three blocks) and its X operands fit its registers. p.grid counts the
// compute workgroups; the launch adds the reducer workgroup.
static SmallPlan plan_stream(int64_t N, int64_t F, int64_t D, int64_t K, int dt) {
  SmallPlan p{};
  const int ms = frag_ms(F);
  if (dt != 0 || N < 1 || N > 32 || K > kFragMaxK || ms < 1 || ms > 36) return p;
  p.nblocks = (int)cdiv(D, kW);
  // one compute unit is left to the reducer workgroup
  const int cus = num_cus() > 1 ? num_cus() - 1 : 1;
  p.grid = p.nblocks < cus ? p.nblocks : cus;
  int64_t cslots = 1;
  for (int b = 0; b < p.grid; ++b) {
    const int c = block_walk(b, p.grid, p.nblocks).count();
    cslots = c > cslots ? c : cslots;
  }
  if (cslots > 3) return p;
  if ((int64_t)p.nblocks * K * kW * 4 >= ((int64_t)1 << 31)) return p;
  const int nti = N <= 16 ? 1 : 2;
  const int64_t nbk = 16 * nti;
  const int64_t floats = (2 * nbk * K + 3) / 4 * 4 + 2 * kWaves * nti * 256 +
                         frag_cs_floats((int)cslots, (int)K) +
                         frag_xs_floats((int)nbk, (int)F, ms);
  // the reducer workgroup's eight per-wave sums use the same allocation
  if (floats < 8 * nbk * K || (int64_t)sizeof(float) * floats > kLdsBudget) return p;
  p.frag = true;
  p.npass = 1;
  p.cslots = (int)cslots;
  p.nb = nti;
  p.ms = ms;
  p.lds = sizeof(float) * (size_t)floats;
  return p;
}

bool small_supported(int64_t N, int64_t F, int64_t D, int64_t K, int dt) {
  if (dt == 2) return plan_small(N, F, D, K, dt, kTiled, true).frag;  // packed int8 only
  return plan_valu(N, F, D, K, 8).nb > 0;
}

size_t small_workspace_bytes(int64_t N, int64_t F, int64_t D, int64_t K, int dt, bool det) {
  // every plan's grid is at most one workgroup per column block
  const int64_t slots = det ? cdiv(D, kW) + kGroups : kSmallReplicas;
  return (size_t)kLine * (1 + kGroups) + sizeof(float) * (size_t)slots * N * K;
}

bool small_matrix_core(int64_t N, int64_t F, int64_t D, int64_t K, int dt, bool tiled) {
  const SmallPlan p = plan_small(N, F, D, K, dt, tiled ? kTiled : kRawVec, true);
  return p.nb > 0 && (p.frag || p.bmfma || p.mfma);
}

const char* small_kernel_name(int64_t N, int64_t F, int64_t D, int64_t K, int dt, bool tiled) {
  const SmallPlan p = plan_small(N, F, D, K, dt, tiled ? kTiled : kRawVec, true);
  if (p.nb == 0) return "";
  return p.flat ? "small_flat_kernel" : p.frag ? "small_frag_mfma_kernel"
                                      : p.bmfma ? "small_block_mfma_kernel"
                                      : p.mfma  ? "small_mfma_kernel" : "small_valu_kernel";
}

// Small-batch section of a packed model: column tiles of B (not for int8,
// which only the fragment kernel serves), column tiles of C, then
// (4 <= F <= 1024) the fragment copy of B, each on a 256-byte boundary.
size_t small_btiles_bytes(int64_t F, int64_t D, int dt) {
  const size_t es = dt == 0 ? 4 : 2;
  return dt == 2 ? 0 : ((size_t)cdiv(D, kW) * F * kW * es + 255) / 256 * 256;
}
size_t small_tiles_bytes(int64_t F, int64_t D, int64_t K, int dt) {
  const size_t es = dt == 0 ? 4 : dt == 1 ? 2 : 1;
  const size_t nblk = (size_t)cdiv(D, kW);
  return small_btiles_bytes(F, D, dt) + (nblk * K * kW * es + 255) / 256 * 256;
}

size_t small_packed_bytes(int64_t F, int64_t D, int64_t K, int dt) {
  return small_tiles_bytes(F, D, K, dt) + (frag_bytes(F, D, dt) + 255) / 256 * 256;
}

hipError_t launch_pack_small(const void* B, const void* C, int64_t F, int64_t D, int64_t K, int dt,
                             void* out, hipStream_t stream) {
  const hipError_t e = dt == 0   ? pack_small_t<float, true>(B, C, F, D, K, out, stream)
                       : dt == 1 ? pack_small_t<bf16raw, true>(B, C, F, D, K, out, stream)
                                 : pack_small_t<int8_t, false>(B, C, F, D, K, out, stream);
  if (e != hipSuccess || frag_bytes(F, D, dt) == 0) return e;
  return launch_pack_frag(B, static_cast<char*>(out) + small_tiles_bytes(F, D, K, dt), F, D,
                          cdiv(D, kW), frag_ms(F), dt, stream);
}

bool stream_supported(int64_t N, int64_t F, int64_t D, int64_t K, int dt) {
  return plan_stream(N, F, D, K, dt).frag;
}

size_t stream_ws_bytes(int64_t nbatch, int64_t N, int64_t K) {
  return stream_workspace_bytes(nbatch, N, K);
}

hipError_t launch_stream(const void* X, const void* packed_small, const unsigned* ready,
                         int32_t* labels, float* scores, unsigned* done, int64_t nbatch,
                         int64_t N, int64_t F, int64_t D, int64_t K, int act, void* workspace,
                         hipStream_t stream) {
  const SmallPlan p = plan_stream(N, F, D, K, 0);
  if (!p.frag || frag_bytes(F, D, 0) == 0) return hipErrorInvalidValue;
  const char* base = static_cast<const char*>(packed_small);
  const void* C = base + (cdiv(D, kW) * F * kW * 4 + 255) / 256 * 256;
  const void* frag = base + small_tiles_bytes(F, D, K, 0);
  const StreamArgs a{X, frag, C, ready, labels, scores, done, (int)nbatch, (int)N, (int)F,
                     (int)K, act, workspace, stream};
  return launch_stream_family(p, a);
}

hipError_t launch_small(const void* X, const void* B, const void* C, bool tiled, int32_t* labels,
                        float* scores, int64_t N, int64_t F, int64_t D, int64_t K, int dt,
                        int act, void* workspace, hipStream_t stream) {
  const size_t align = dt == 0 ? 16 : 8;
  int lay = kTiled;
  const void* frag = nullptr;
  if (tiled) {
    // the packed image's small-batch section
    C = static_cast<const char*>(B) + small_btiles_bytes(F, D, dt);
    if (frag_bytes(F, D, dt) > 0) frag = static_cast<const char*>(B) + small_tiles_bytes(F, D, K, dt);
  } else {
    const bool vec = (D % 4 == 0) && ((uintptr_t)B % align == 0) && ((uintptr_t)C % align == 0);
    lay = vec ? kRawVec : kRawScalar;
  }
  SmallPlan p = plan_small(N, F, D, K, dt, lay, (uintptr_t)X % 16 == 0);
  if (p.nb == 0) return hipErrorInvalidValue;
  if ((act & kActDet) && p.grid > cdiv(D, kW)) return hipErrorInvalidValue;  // workspace bound
  const Args a{X, B, C, labels, scores, (int)N, (int)F, (int)D, (int)K, act, workspace, stream};
  if (p.frag) {
    if (!frag) return hipErrorInvalidValue;
    return launch_frag_family(p, a, frag, dt);
  }
  if (dt == 2) return hipErrorInvalidValue;  // int8: the fragment kernel only
  return launch_plan(p, a, dt, lay);
}

}  // namespace hd
