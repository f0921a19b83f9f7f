// Large-batch fused inference on the matrix cores: the GPU form of the
// paper's large-batch variant (Sec. III-C, Alg. 4), which splits the batch N
// across workers, each accumulating its rows of S over every column block of
// the encoded matrix.
//
// Formulation. Stage I is computed transposed, V^T[d,n] = sum_f B^T[d,f] X[n,f],
// so that the hypervector dimension d is the MFMA row index and the sample n
// the column index. With the 32x32 MFMA accumulator layout each lane then
// holds 16 d-values of one sample, which after HardSign (Eq. 1) are exactly a
// B-operand fragment of the Stage II MFMA S^T[k,n] += C[k,d] H^T[d,n] (Eq. 8)
// up to a fixed permutation of d. The permutation is absorbed into the tiled
// copy of C, so the encoded block goes from accumulators to the next MFMA
// without touching LDS or device memory: H is never materialised.
//
// Data layout. A workgroup owns NT = 32*NTILES samples; their rows of X are
// copied once into LDS (zero padded) and stay resident while the workgroup
// sweeps its slice of D. B and C are read from a tiled copy made once per
// model (the parameter tiling of Sec. III-D): every MFMA A-fragment is one
// contiguous, fully coalesced 1 KiB block, so B streams straight from L2 into
// registers with a software-pipelined prefetch ring. When even 32 rows of X do
// not fit LDS (wide F), the F-chunked kernels below stream the tile through
// LDS in chunks of f-steps instead and keep V in registers across the chunks.
//
// Work split. Each of the 4 waves owns "units" of 64 hypervector dimensions
// (two 32-row MFMA tiles) round-robin within the workgroup's D slice and keeps
// its own partial S; the waves' partials are summed through LDS at the end.
// When there are too few sample tiles to fill the GPU, D is also split into
// DS slices whose partial scores are combined by the last-arriving workgroup
// of each sample tile (ticket counter, self-cleaning).
#include <type_traits>

#include "hd_common.hpp"
#include "hd_internal.hpp"

namespace hd {

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = 4;
// f-steps of B fragments in flight per wave: deeper while registers allow
constexpr int prefetch_of(int ntiles, int kb) { return ntiles * kb <= 4 ? 8 : 4; }
// Ring depth of the int8 resident-X kernel where 8 would be used: a unit's
// f-steps run in groups of the depth, the last group padded with zero X, and
// int8's 32-row f-steps leave few steps per unit, so take 10 when it pads
// fewer steps. The depth must be even: the X fragments are double-buffered by
// the step's index within its group.
constexpr int fused_prefetch(int nfs) {
  const int pad8 = (nfs + 7) / 8 * 8 - nfs, pad10 = (nfs + 9) / 10 * 10 - nfs;
  return pad10 < pad8 ? 10 : 8;
}
constexpr int kMaxSlices = 64;  // D slices per sample tile (split-D)
constexpr int kLdsBytes = 160 * 1024 - 256;  // leave room for static LDS

template <typename U, typename V>
__device__ __forceinline__ U bitcast(const V& v) {
  static_assert(sizeof(U) == sizeof(V), "size");
  U u;
  __builtin_memcpy(&u, &v, sizeof(U));
  return u;
}

// ---------------------------------------------------------------------------
// Element-type traits. One "f-step" consumes one 16-byte fragment per lane of
// both operands: 16 features for bf16 (one 32x32x16 MFMA), 8 features for
// fp32 (four 32x32x2 MFMAs).
// ---------------------------------------------------------------------------
struct TrBF16 {
  typedef bf16raw elem;
  static constexpr int kFStep = 16;
  static constexpr int kVec = 8;  // elements per 16-byte group
  static constexpr int kEsz = 2;
  // element e of a 16-byte group held as four dwords: set, read, clear
  __device__ static void put(uint32_t (&t)[4], int e, elem x) {
    t[e >> 1] |= (uint32_t)x << (16 * (e & 1));
  }
  __device__ static elem get(const uint32_t (&t)[4], int e) {
    return (uint16_t)(t[e >> 1] >> (16 * (e & 1)));
  }
  __device__ static void clear(uint32_t (&t)[4], int e) { t[e >> 1] &= ~(0xffffu << (16 * (e & 1))); }
  // Stage I accumulator value v is >= 0 (the HardSign test, Eq. 1)
  __device__ static bool nonneg(float v) { return v >= 0.0f; }
  static constexpr int kStage1Mfma = 1;  // matrix instructions per stage1 call
  static constexpr int kCFrags = 2;  // 1 KiB C fragments per (d-block, class block)
  // LDS position of feature column c inside a sample row.
  __device__ static int lds_pos(int c) { return c; }
  __device__ static void stage1(f32x16& acc, const uint4& a, const uint4& b) {
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bitcast<bf16x8>(a), bitcast<bf16x8>(b), acc,
                                                  0, 0, 0);
  }
  // first step of a sum: the instruction's accumulator input is the constant 0
  __device__ static void stage1_init(f32x16& acc, const uint4& a, const uint4& b) {
    acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bitcast<bf16x8>(a), bitcast<bf16x8>(b),
                                                  f32x16{}, 0, 0, 0);
  }
};

struct TrF32 {
  typedef float elem;
  static constexpr int kFStep = 8;
  static constexpr int kVec = 4;
  static constexpr int kEsz = 4;
  __device__ static void put(uint32_t (&t)[4], int e, elem x) { t[e] = __float_as_uint(x); }
  __device__ static elem get(const uint32_t (&t)[4], int e) { return __uint_as_float(t[e]); }
  __device__ static void clear(uint32_t (&t)[4], int e) { t[e] = 0u; }
  __device__ static bool nonneg(float v) { return v >= 0.0f; }
  static constexpr int kStage1Mfma = 4;
  static constexpr int kCFrags = 4;
  // Within each group of 8 features the even ones are stored first, so a
  // lane of MFMA k-half g reads its four features (g, g+2, g+4, g+6) as one
  // 16-byte word.
  __device__ static int lds_pos(int c) {
    const int r = c & 7;
    return (c & ~7) + 4 * (r & 1) + (r >> 1);
  }
  __device__ static void stage1(f32x16& acc, const uint4& a, const uint4& b) {
    const float4 af = bitcast<float4>(a), bf = bitcast<float4>(b);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(af.x, bf.x, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(af.y, bf.y, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(af.z, bf.z, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(af.w, bf.w, acc, 0, 0, 0);
  }
  __device__ static void stage1_init(f32x16& acc, const uint4& a, const uint4& b) {
    const float4 af = bitcast<float4>(a), bf = bitcast<float4>(b);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(af.x, bf.x, f32x16{}, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(af.y, bf.y, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(af.z, bf.z, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(af.w, bf.w, acc, 0, 0, 0);
  }
};

// int8 model variant: X and B int8, Stage I on the int8 matrix instruction
// with exact int32 accumulation (the accumulator registers hold the int32
// bits), HardSign on the exact integer; Stage II takes C widened to bf16
// (exact for |c| <= 128) through the bf16 path. One f-step is 32 features.
struct TrI8 {
  typedef int8_t elem;
  static constexpr int kFStep = 32;
  static constexpr int kVec = 16;
  static constexpr int kEsz = 1;
  static constexpr int kStage1Mfma = 1;
  static constexpr int kCFrags = 2;  // C tiles are the bf16 ones
  __device__ static void put(uint32_t (&t)[4], int e, elem x) {
    t[e >> 2] |= (uint32_t)(uint8_t)x << (8 * (e & 3));
  }
  __device__ static elem get(const uint32_t (&t)[4], int e) {
    return (int8_t)(uint8_t)(t[e >> 2] >> (8 * (e & 3)));
  }
  __device__ static void clear(uint32_t (&t)[4], int e) { t[e >> 2] &= ~(0xffu << (8 * (e & 3))); }
  __device__ static bool nonneg(float v) { return __float_as_int(v) >= 0; }
  __device__ static int lds_pos(int c) { return c; }
  __device__ static void stage1(f32x16& acc, const uint4& a, const uint4& b) {
    acc = bitcast<f32x16>(__builtin_amdgcn_mfma_i32_32x32x32_i8(
        bitcast<i32x4>(a), bitcast<i32x4>(b), bitcast<i32x16>(acc), 0, 0, 0));
  }
  __device__ static void stage1_init(f32x16& acc, const uint4& a, const uint4& b) {
    acc = bitcast<f32x16>(
        __builtin_amdgcn_mfma_i32_32x32x32_i8(bitcast<i32x4>(a), bitcast<i32x4>(b), i32x16{}, 0, 0, 0));
  }
};

// Largest sizes of the int8 variant for which every sum is exact: |V| <=
// 128 * 128 * F < 2^31 in int32, and |S| <= 128 * D <= 2^24 in fp32.
constexpr int64_t kI8MaxF = (int64_t(1) << 17) - 1;
constexpr int64_t kI8MaxD = int64_t(1) << 17;

// LDS row padding of an X tile: one 16-byte group (keeps the 32 rows read by
// one fragment load on distinct LDS banks).
template <class Tr>
constexpr int pad_of() {
  return 16 / Tr::kEsz;
}

// Number of f-steps and padded row pitch (elements) of the LDS X tile.
template <class Tr>
__host__ __device__ inline int nfs_of(int F) {
  return (F + Tr::kFStep - 1) / Tr::kFStep;
}
template <class Tr>
__host__ __device__ inline int pitch_of(int F) {
  // Padding by half a 16-byte group (bf16) / one group (fp32) keeps the
  // 32 rows read by one fragment load on distinct LDS banks.
  return nfs_of<Tr>(F) * Tr::kFStep + pad_of<Tr>();
}

// ---------------------------------------------------------------------------
// Tiled model image.
//   B tile (db, fs): 64 lanes x 16 bytes; lane l holds
//     bf16: B[16fs + 8(l/32) + e][32db + l%32], e = 0..7
//     fp32: B[8fs + 2j + l/32][32db + l%32],   j = 0..3
//   C tile, bf16 (db, h, kb): lane l holds C[32kb + l%32][32db + 16h + 4(l/32) + e]
//     for e = 0..3 and C[..][32db + 16h + 8 + 4(l/32) + e - 4] for e = 4..7
//   C tile, fp32 (db, kb, q): lane l holds C[32kb + l%32][32db + 8q + 4(l/32) + j]
// Out-of-range entries are zero. NDB is rounded up to even (64-dim units).
// ---------------------------------------------------------------------------
struct PackGeom {
  int ndb, nfs, kb;
  size_t b_bytes, c_bytes;
};

// Class blocks of 32 handled per launch: 1, 2 or 4.
inline int kb_of(int64_t K) {
  const int kb = (int)cdiv(K, 32);
  return kb == 3 ? 4 : kb;
}

// Sample tiles per workgroup of the F-chunked kernel: 4 when the accumulators
// fit in registers, fewer as class blocks grow.
template <class Tr>
constexpr int chunk_ntiles(int kb) {
  return kb > 2 ? (Tr::kEsz <= 2 ? 2 : 1) : kb == 2 ? 2 : 4;
}

template <class Tr>
PackGeom pack_geom(int64_t F, int64_t D, int64_t K) {
  PackGeom g;
  g.ndb = (int)(cdiv(D, 64) * 2);
  g.nfs = nfs_of<Tr>((int)F);
  g.kb = kb_of(K);
  g.b_bytes = (size_t)g.ndb * g.nfs * 1024;
  g.c_bytes = (size_t)g.ndb * g.kb * Tr::kCFrags * 1024;
  return g;
}

__global__ void pack_b_bf16(const bf16raw* __restrict__ B, uint4* __restrict__ Bp, int F, int D,
                            int ndb, int nfs) {
  const int64_t frag = blockIdx.x;
  const int l = threadIdx.x;
  if (frag >= (int64_t)ndb * nfs) return;
  const int db = (int)(frag / nfs), fs = (int)(frag % nfs);
  const int d = 32 * db + (l & 31);
  uint16_t v[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int f = 16 * fs + 8 * (l >> 5) + e;
    v[e] = (f < F && d < D) ? B[(int64_t)f * D + d] : (uint16_t)0;
  }
  Bp[frag * 64 + l] = make_uint4(v[0] | (uint32_t)v[1] << 16, v[2] | (uint32_t)v[3] << 16,
                                 v[4] | (uint32_t)v[5] << 16, v[6] | (uint32_t)v[7] << 16);
}

__global__ void pack_b_f32(const float* __restrict__ B, uint4* __restrict__ Bp, int F, int D,
                           int ndb, int nfs) {
  const int64_t frag = blockIdx.x;
  const int l = threadIdx.x;
  if (frag >= (int64_t)ndb * nfs) return;
  const int db = (int)(frag / nfs), fs = (int)(frag % nfs);
  const int d = 32 * db + (l & 31);
  float v[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int f = 8 * fs + 2 * j + (l >> 5);
    v[j] = (f < F && d < D) ? B[(int64_t)f * D + d] : 0.0f;
  }
  Bp[frag * 64 + l] = make_uint4(__float_as_uint(v[0]), __float_as_uint(v[1]),
                                 __float_as_uint(v[2]), __float_as_uint(v[3]));
}

__global__ void pack_b_i8(const int8_t* __restrict__ B, uint4* __restrict__ Bp, int F, int D,
                          int ndb, int nfs) {
  const int64_t frag = blockIdx.x;
  const int l = threadIdx.x;
  if (frag >= (int64_t)ndb * nfs) return;
  const int db = (int)(frag / nfs), fs = (int)(frag % nfs);
  const int d = 32 * db + (l & 31);
  uint32_t t[4] = {0u, 0u, 0u, 0u};
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    const int f = 32 * fs + 16 * (l >> 5) + e;
    if (f < F && d < D) TrI8::put(t, e, B[(int64_t)f * D + d]);
  }
  Bp[frag * 64 + l] = make_uint4(t[0], t[1], t[2], t[3]);
}

// int8 C into the bf16 C tiles (an int8 value is exact in bf16).
__global__ void pack_c_i8(const int8_t* __restrict__ C, uint4* __restrict__ Cp, int D, int K,
                          int ndb, int kb) {
  const int64_t frag = blockIdx.x;
  const int l = threadIdx.x;
  if (frag >= (int64_t)ndb * 2 * kb) return;
  const int kbi = (int)(frag % kb);
  const int h = (int)((frag / kb) % 2);
  const int db = (int)(frag / (2 * kb));
  const int k = 32 * kbi + (l & 31);
  uint32_t v[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int d = 32 * db + 16 * h + 4 * (l >> 5) + (e < 4 ? e : 8 + e - 4);
    const float c = (k < K && d < D) ? (float)C[(int64_t)k * D + d] : 0.0f;
    v[e] = __float_as_uint(c) >> 16;
  }
  Cp[frag * 64 + l] = make_uint4(v[0] | v[1] << 16, v[2] | v[3] << 16, v[4] | v[5] << 16,
                                 v[6] | v[7] << 16);
}

// grid: ndb * 2 * kb fragments of 64 lanes.
__global__ void pack_c_bf16(const bf16raw* __restrict__ C, uint4* __restrict__ Cp, int D, int K,
                            int ndb, int kb) {
  const int64_t frag = blockIdx.x;
  const int l = threadIdx.x;
  if (frag >= (int64_t)ndb * 2 * kb) return;
  const int kbi = (int)(frag % kb);
  const int h = (int)((frag / kb) % 2);
  const int db = (int)(frag / (2 * kb));
  const int k = 32 * kbi + (l & 31);
  uint16_t v[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int d = 32 * db + 16 * h + 4 * (l >> 5) + (e < 4 ? e : 8 + e - 4);
    v[e] = (k < K && d < D) ? C[(int64_t)k * D + d] : (uint16_t)0;
  }
  Cp[frag * 64 + l] = make_uint4(v[0] | (uint32_t)v[1] << 16, v[2] | (uint32_t)v[3] << 16,
                                 v[4] | (uint32_t)v[5] << 16, v[6] | (uint32_t)v[7] << 16);
}

// grid: ndb * kb * 4 fragments of 64 lanes.
__global__ void pack_c_f32(const float* __restrict__ C, uint4* __restrict__ Cp, int D, int K,
                           int ndb, int kb) {
  const int64_t frag = blockIdx.x;
  const int l = threadIdx.x;
  if (frag >= (int64_t)ndb * kb * 4) return;
  const int q = (int)(frag % 4);
  const int kbi = (int)((frag / 4) % kb);
  const int db = (int)(frag / (4 * kb));
  const int k = 32 * kbi + (l & 31);
  float v[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int d = 32 * db + 8 * q + 4 * (l >> 5) + j;
    v[j] = (k < K && d < D) ? C[(int64_t)k * D + d] : 0.0f;
  }
  Cp[frag * 64 + l] = make_uint4(__float_as_uint(v[0]), __float_as_uint(v[1]),
                                 __float_as_uint(v[2]), __float_as_uint(v[3]));
}

// ---------------------------------------------------------------------------
// Stage II on one finished 32x32 V^T tile (rows d of block db, columns n of
// one sample tile): activation, then accumulate S^T for every class block.
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t pack2_bf16(float a, float b) {
  // round-to-nearest-even fp32 -> bf16 for finite values
  uint32_t ua = __float_as_uint(a), ub = __float_as_uint(b);
  ua = (ua + 0x7fffu + ((ua >> 16) & 1u)) >> 16;
  ub = (ub + 0x7fffu + ((ub >> 16) & 1u)) >> 16;
  return ua | (ub << 16);
}

__device__ __forceinline__ uint32_t sign_pair(float a, float b) {
  const uint32_t lo = a >= 0.0f ? 0x3F80u : 0xBF80u;
  const uint32_t hi = b >= 0.0f ? 0x3F80u : 0xBF80u;
  return lo | (hi << 16);
}

template <int KB, int ACT>
__device__ __forceinline__ void stage2_bf16(const f32x16& v, const uint4 (&cfr)[2][KB],
                                            f32x16 (&s)[KB]) {
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    if constexpr (ACT == 0) {
      uint4 hb;
      hb.x = sign_pair(v[8 * h + 0], v[8 * h + 1]);
      hb.y = sign_pair(v[8 * h + 2], v[8 * h + 3]);
      hb.z = sign_pair(v[8 * h + 4], v[8 * h + 5]);
      hb.w = sign_pair(v[8 * h + 6], v[8 * h + 7]);
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
        s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bitcast<bf16x8>(cfr[h][kb]),
                                                        bitcast<bf16x8>(hb), s[kb], 0, 0, 0);
    } else {
      // Identity test mode: split v into three bf16 terms (about 24 bits).
      float r[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) r[e] = v[8 * h + e];
#pragma unroll
      for (int t = 0; t < 3; ++t) {
        uint4 hb;
        hb.x = pack2_bf16(r[0], r[1]);
        hb.y = pack2_bf16(r[2], r[3]);
        hb.z = pack2_bf16(r[4], r[5]);
        hb.w = pack2_bf16(r[6], r[7]);
        const uint32_t w[4] = {hb.x, hb.y, hb.z, hb.w};
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const uint32_t bits = (w[e >> 1] >> (16 * (e & 1))) & 0xffffu;
          r[e] -= __uint_as_float(bits << 16);
        }
#pragma unroll
        for (int kb = 0; kb < KB; ++kb)
          s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bitcast<bf16x8>(cfr[h][kb]),
                                                          bitcast<bf16x8>(hb), s[kb], 0, 0, 0);
      }
    }
  }
}

template <int KB, int ACT>
__device__ __forceinline__ void stage2_f32(const f32x16& v, const uint4 (&cfr)[KB][4],
                                           f32x16 (&s)[KB]) {
#pragma unroll
  for (int q = 0; q < 4; ++q) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float h = ACT ? v[4 * q + j] : hardsign(v[4 * q + j]);
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) {
        const float c = __uint_as_float(j == 0 ? cfr[kb][q].x
                                         : j == 1 ? cfr[kb][q].y
                                         : j == 2 ? cfr[kb][q].z
                                                  : cfr[kb][q].w);
        s[kb] = __builtin_amdgcn_mfma_f32_32x32x2f32(c, h, s[kb], 0, 0, 0);
      }
    }
  }
}

// C fragments of one 64-dim unit (two d-blocks).
template <class Tr, int KB>
struct CFrags;
template <int KB>
struct CFrags<TrBF16, KB> {
  uint4 f[2][2][KB];  // [db2][h][kb]
  __device__ void load(const uint4* __restrict__ Cp, int db0, int lane) {
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int kb = 0; kb < KB; ++kb)
          f[b][h][kb] = Cp[((int64_t)((db0 + b) * 2 + h) * KB + kb) * 64 + lane];
  }
  template <int ACT>
  __device__ void apply(const f32x16& v, int b, f32x16 (&s)[KB]) const {
    stage2_bf16<KB, ACT>(v, f[b], s);
  }
};
template <int KB>
struct CFrags<TrF32, KB> {
  uint4 f[2][KB][4];  // [db2][kb][q]
  __device__ void load(const uint4* __restrict__ Cp, int db0, int lane) {
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
#pragma unroll
        for (int q = 0; q < 4; ++q)
          f[b][kb][q] = Cp[(((int64_t)(db0 + b) * KB + kb) * 4 + q) * 64 + lane];
  }
  template <int ACT>
  __device__ void apply(const f32x16& v, int b, f32x16 (&s)[KB]) const {
    stage2_f32<KB, ACT>(v, f[b], s);
  }
};

template <int KB>
struct CFrags<TrI8, KB> : CFrags<TrBF16, KB> {
  template <int ACT>
  __device__ void apply(const f32x16& v, int b, f32x16 (&s)[KB]) const {
    f32x16 vf;  // the exact int32 sums as floats (sign and zero preserved)
#pragma unroll
    for (int r = 0; r < 16; ++r) vf[r] = (float)__float_as_int(v[r]);
    stage2_bf16<KB, ACT>(vf, this->f[b], s);
  }
};

struct LargeWs {
  unsigned* counters;  // [ntiles]
  float* part;         // [DS][N][K]
};

__host__ __device__ inline LargeWs large_ws(void* ws, int64_t ntiles) {
  LargeWs w;
  w.counters = reinterpret_cast<unsigned*>(ws);
  const size_t cbytes = ((size_t)ntiles * sizeof(unsigned) + 255) / 256 * 256;
  w.part = reinterpret_cast<float*>(reinterpret_cast<char*>(ws) + cbytes);
  return w;
}

// Combine the waves' partial scores through LDS, then argmax (Eq. 9) and
// write; with a split of D, publish this slice's partial scores and let the
// tile's last slice finish (fixed slice order, so results are deterministic).
template <int NTILES, int KB>
__device__ void finish_tile(f32x16 (&sacc)[NTILES][KB], unsigned char* lds, int* s_last_p,
                            int32_t* __restrict__ labels, float* __restrict__ scores, int N, int K,
                            int DS, int ntiles, int slice, int tile, int n0,
                            void* __restrict__ workspace) {
  constexpr int NT = 32 * NTILES;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int& s_last = *s_last_p;
  __syncthreads();  // X tile no longer needed
  float* sred = reinterpret_cast<float*>(lds);  // [kWaves][NT][32*KB]
  constexpr int KP = 32 * KB;
#pragma unroll
  for (int t = 0; t < NTILES; ++t)
#pragma unroll
    for (int kb = 0; kb < KB; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int k = 32 * kb + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        const int n = 32 * t + (lane & 31);
        sred[((int64_t)wave * NT + n) * KP + k] = sacc[t][kb][r];
      }
  __syncthreads();
  const int rows = min(NT, N - n0);
  if (DS == 1) {
    for (int n = tid; n < rows; n += kThreads) {
      float best = 0.0f;
      int best_k = 0;
      for (int k = 0; k < K; ++k) {
        float s = 0.0f;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) s += sred[((int64_t)w * NT + n) * KP + k];
        if (scores) scores[(int64_t)(n0 + n) * K + k] = s;
        if (k == 0 || s > best) {
          best = s;
          best_k = k;
        }
      }
      labels[n0 + n] = best_k;
    }
    return;
  }
  // Split-D: publish this slice's partial, the last slice of the tile finishes
  // (summing the slices in a fixed order, so results are deterministic).
  const LargeWs ws = large_ws(workspace, ntiles);
  float* mypart = ws.part + (int64_t)slice * N * K;
  for (int i = tid; i < rows * K; i += kThreads) {
    const int n = i / K, k = i - n * K;
    float s = 0.0f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) s += sred[((int64_t)w * NT + n) * KP + k];
    publish_store(mypart + (int64_t)(n0 + n) * K + k, s);
  }
  wait_own_memory_ops();
  __syncthreads();
  if (tid == 0) s_last = (take_ticket(ws.counters + tile) == (unsigned)DS - 1) ? 1 : 0;
  __syncthreads();
  if (!s_last) return;
  for (int i = tid; i < rows * K; i += kThreads) {
    const int n = i / K, k = i - n * K;
    float s = 0.0f;
    // slices in groups of 16 whose reads are all in flight together
    for (int sl0 = 0; sl0 < DS; sl0 += 16) {
      float t[16];
#pragma unroll
      for (int j = 0; j < 16; ++j)
        t[j] = sl0 + j < DS ? take_and_clear(ws.part + ((int64_t)(sl0 + j) * N + n0 + n) * K + k)
                            : 0.0f;
#pragma unroll
      for (int j = 0; j < 16; ++j) s += t[j];
    }
    sred[i] = s;  // the per-wave partials are no longer needed
  }
  __syncthreads();
  for (int n = tid; n < rows; n += kThreads) {
    float best = 0.0f;
    int best_k = 0;
    for (int k = 0; k < K; ++k) {
      const float s = sred[n * K + k];
      if (scores) scores[(int64_t)(n0 + n) * K + k] = s;
      if (k == 0 || s > best) {
        best = s;
        best_k = k;
      }
    }
    labels[n0 + n] = best_k;
  }
  if (tid == 0) reset_counter(ws.counters + tile);
}

// ---------------------------------------------------------------------------
// The fused kernel.
// ---------------------------------------------------------------------------
template <class Tr, int NTILES, int KB, int ACT, int PF>
__global__ __launch_bounds__(kThreads, 1) void large_fused_kernel(
    const typename Tr::elem* __restrict__ X, const uint4* __restrict__ Bp,
    const uint4* __restrict__ Cp, int32_t* __restrict__ labels, float* __restrict__ scores,
    int N, int F, int K, int ndb, int DS, void* __restrict__ workspace) {
  typedef typename Tr::elem T;
  constexpr int NT = 32 * NTILES;
  static_assert(PF % 2 == 0, "X fragments are double-buffered by step parity");
  constexpr int kPrefetch = PF;  // B ring depth in f-steps
  extern __shared__ __attribute__((aligned(16))) unsigned char lds[];
  __shared__ int s_last;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nfs = nfs_of<Tr>(F);
  const int pitch = pitch_of<Tr>(F);  // elements
  const int ntiles = (int)cdiv(N, NT);
  // Consecutive workgroups take different D slices, so with round-robin
  // dispatch over the XCDs each XCD's L2 serves one slice of B.
  const int slice = blockIdx.x % DS;
  const int tile = blockIdx.x / DS;
  const int n0 = tile * NT;
  const int units = ndb / 2;
  const int u_begin = (int)((int64_t)units * slice / DS);
  const int u_end = (int)((int64_t)units * (slice + 1) / DS);

  // ---- X tile -> LDS (rows n0..n0+NT, zero padded) -------------------------
  // A 16-byte zero slot follows the tile: padding f-steps past nfs read it.
  T* xt = reinterpret_cast<T*>(lds);
  const T* xzero = xt + NT * pitch;
  if (tid == 0) *reinterpret_cast<uint4*>(xt + NT * pitch) = make_uint4(0u, 0u, 0u, 0u);
  {
    // zero the padding columns F..nfs*kFStep and whole rows past N
    const int fpad = nfs * Tr::kFStep;
    for (int i = tid; i < NT * (fpad - F); i += kThreads) {
      const int r = i / (fpad - F), c = F + i % (fpad - F);
      xt[r * pitch + Tr::lds_pos(c)] = T(0);
    }
    const int rows = min(NT, N - n0);
    for (int i = tid; i < (NT - rows) * fpad; i += kThreads) {
      const int r = rows + i / fpad, c = i % fpad;
      xt[r * pitch + Tr::lds_pos(c)] = T(0);
    }
    // The tile's rows are one contiguous range of X: read it with aligned
    // 16-byte buffer loads (out-of-range dwords read as zero) and scatter.
    const int64_t e0 = (int64_t)n0 * F, e1 = (int64_t)(n0 + rows) * F;
    const int64_t g0 = e0 / Tr::kVec, g1 = cdiv(e1, Tr::kVec);
    const T* base = X + g0 * Tr::kVec;
    const int64_t total_bytes = ((int64_t)N * F - g0 * Tr::kVec) * Tr::kEsz;
    const int nrec = (int)(total_bytes < 0x7fffffff ? total_bytes : 0x7fffffff);
    const __amdgpu_buffer_rsrc_t rsrc =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<T*>(base), 0, nrec, 0x00020000);
    const int ng = (int)(g1 - g0);
    const int64_t nx_total = (int64_t)N * F;
    for (int g = tid; g < ng; g += kThreads) {
      uint4 w;
      if ((g0 + g + 1) * Tr::kVec <= nx_total) {
        w = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rsrc, g * 16, 0, 0));
      } else {
        // last, partial group of X: element loads inside the allocation only
        uint32_t t[4] = {0u, 0u, 0u, 0u};
        const int64_t first = (g0 + g) * Tr::kVec;
        for (int j = 0; j < Tr::kVec; ++j) {
          if (first + j >= nx_total) break;
          Tr::put(t, j, X[first + j]);
        }
        w = make_uint4(t[0], t[1], t[2], t[3]);
      }
      int64_t e = (g0 + g) * Tr::kVec - e0;  // element offset inside the tile
      int r = (int)(e >= 0 ? e / F : -1);
      int c = (int)(e - (int64_t)r * F);
      const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
      for (int j = 0; j < Tr::kVec; ++j) {
        if (e >= 0 && r < rows) xt[r * pitch + Tr::lds_pos(c)] = Tr::get(ws, j);
        ++e;
        if (e == 0) {
          r = 0;
          c = 0;
        } else if (e > 0) {
          if (++c == F) {
            c = 0;
            ++r;
          }
        }
      }
    }
  }
  __syncthreads();

  // ---- main sweep over this wave's 64-dim units ---------------------------
  f32x16 sacc[NTILES][KB];
#pragma unroll
  for (int t = 0; t < NTILES; ++t)
#pragma unroll
    for (int kb = 0; kb < KB; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) sacc[t][kb][r] = 0.0f;

  // byte offset of this lane's 16-byte X fragment word for f-step 0, tile 0
  const int xrow = lane & 31, xhalf = lane >> 5;
  const T* xlane = xt + xrow * pitch + xhalf * (Tr::kFStep / 2);
  const int nfsl = (nfs + kPrefetch - 1) / kPrefetch * kPrefetch;

  int u = u_begin + wave;
  uint4 afr[kPrefetch][2];
  // B fragments through a buffer resource: 32-bit byte offsets, no 64-bit
  // address arithmetic per load (the packed B is below 2 GiB)
  const __amdgpu_buffer_rsrc_t brsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint4*>(Bp), 0, ndb * nfs * 1024, 0x00020000);
  auto bfrag = [&](int uu, int fs, int b) -> uint4 {
    return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(
                                         brsrc, ((2 * uu + b) * nfs + fs) * 1024 + lane * 16, 0, 0));
  };
  if (u < u_end) {
    // slots past nfs hold a valid fragment too: padding steps multiply them
    // by the zero slot, so they must be finite
#pragma unroll
    for (int i = 0; i < kPrefetch; ++i) {
      afr[i][0] = bfrag(u, i < nfs ? i : nfs - 1, 0);
      afr[i][1] = bfrag(u, i < nfs ? i : nfs - 1, 1);
    }
  }
  for (; u < u_end; u += kWaves) {
    const int un = u + kWaves;
    const bool has_next = un < u_end;
    CFrags<Tr, KB> cf;
    cf.load(Cp, 2 * u, lane);
    // With 64-sample tiles the unit's first step starts the accumulators from
    // the matrix instruction's constant-zero input (measured faster there);
    // with 128-sample tiles they are zeroed here (measured faster there).
    constexpr bool kZeroInput = NTILES <= 2;
    f32x16 vacc[2][NTILES];
    if constexpr (!kZeroInput) {
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int t = 0; t < NTILES; ++t)
#pragma unroll
          for (int r = 0; r < 16; ++r) vacc[b][t][r] = 0.0f;
    }

    uint4 xfr[2][NTILES];
#pragma unroll
    for (int t = 0; t < NTILES; ++t)
      xfr[0][t] = *reinterpret_cast<const uint4*>(xlane + t * 32 * pitch);

    // Every step issues the same loads and matrix instructions
    // unconditionally, with no branch in the loop body, so the compiler can
    // interleave the refill arithmetic with the matrix instructions and track
    // the wait counters across the loop. Padding steps past nfs (up to
    // kPrefetch-1 of them) multiply a valid, finite B fragment by the zero
    // slot. The unit's first group of kPrefetch steps always runs and issues
    // ring loads after the C fragment loads above, so Stage II never waits
    // for the ring in flight before using them (with a zero-trip path the
    // compiler would make it wait for every ring load).
    auto steps = [&](int fs0, auto first) __attribute__((always_inline)) {
#pragma unroll
      for (int i = 0; i < kPrefetch; ++i) {
        const int fs = fs0 + i;
        const int fsn = fs + 1;
#pragma unroll
        for (int t = 0; t < NTILES; ++t)
          xfr[(i + 1) & 1][t] = *reinterpret_cast<const uint4*>(
              fsn < nfs ? xlane + t * 32 * pitch + fsn * Tr::kFStep : xzero);
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
          for (int t = 0; t < NTILES; ++t) {
            if (kZeroInput && decltype(first)::value && i == 0)
              Tr::stage1_init(vacc[b][t], afr[i][b], xfr[i & 1][t]);
            else
              Tr::stage1(vacc[b][t], afr[i][b], xfr[i & 1][t]);
          }
        // instruction order per step: the next step's X reads (LDS) first, so
        // they complete under this step's matrix instructions, then the
        // matrix instructions, then the ring refill loads
        __builtin_amdgcn_sched_group_barrier(0x100, NTILES, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 2 * NTILES * Tr::kStage1Mfma, 0);
        __builtin_amdgcn_sched_group_barrier(0x020, 2, 0);
        // ring refill: step fs + kPrefetch of this unit, else the first steps
        // of the wave's next unit, else a harmless reload of a valid fragment
        const int nx = fs + kPrefetch;
        const int j = nx - nfsl;
        const bool cur = nx < nfs;
        const bool nxt = !cur && has_next && j >= 0 && j < nfs;
        const int tu = nxt ? un : u;
        const int tf = cur ? nx : (nxt ? j : nfs - 1);
        afr[i][0] = bfrag(tu, tf, 0);
        afr[i][1] = bfrag(tu, tf, 1);
      }
    };
    if constexpr (kZeroInput) {
      steps(0, std::true_type{});
      for (int fs0 = kPrefetch; fs0 < nfsl; fs0 += kPrefetch) steps(fs0, std::false_type{});
    } else {
      int fs0 = 0;
      do {  // always runs at least once (nfsl >= kPrefetch)
        steps(fs0, std::false_type{});
        fs0 += kPrefetch;
      } while (fs0 < nfsl);
    }
    // Stage II on the finished unit.
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int t = 0; t < NTILES; ++t) cf.template apply<ACT>(vacc[b][t], b, sacc[t]);
  }

  finish_tile<NTILES, KB>(sacc, lds, &s_last, labels, scores, N, K, DS, ntiles, slice, tile, n0,
                          workspace);
}

// ---------------------------------------------------------------------------
// F-chunked variant, for feature counts whose X tile does not fit in LDS
// (e.g. F = 3072). The workgroup walks its units in lockstep iterations, one
// unit per wave each; an iteration streams the tile's X through LDS in chunks
// of fsc f-steps and accumulates each wave's V^T over every chunk in
// registers before Stage II, so H still never leaves the chip. X is read
// again (from L2 or the last-level cache) once per iteration.
// ---------------------------------------------------------------------------
template <class Tr, int NTILES, int KB, int ACT>
__global__ __launch_bounds__(kThreads, 1) void large_chunked_kernel(
    const typename Tr::elem* __restrict__ X, const uint4* __restrict__ Bp,
    const uint4* __restrict__ Cp, int32_t* __restrict__ labels, float* __restrict__ scores,
    int N, int F, int K, int ndb, int DS, int fsc, void* __restrict__ workspace) {
  typedef typename Tr::elem T;
  constexpr int NT = 32 * NTILES;
  constexpr int kPrefetch = prefetch_of(NTILES, KB);
  constexpr int kSB = 8;  // staging items per thread per batch
  extern __shared__ __attribute__((aligned(16))) unsigned char lds[];
  __shared__ int s_last;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nfs = nfs_of<Tr>(F);
  const int nchunks = (nfs + fsc - 1) / fsc;
  const int pitch = fsc * Tr::kFStep + pad_of<Tr>();  // elements
  const int ntiles = (int)cdiv(N, NT);
  const int slice = blockIdx.x % DS;
  const int tile = blockIdx.x / DS;
  const int n0 = tile * NT;
  const int rows = min(NT, N - n0);
  const int units = ndb / 2;
  const int u_begin = (int)((int64_t)units * slice / DS);
  const int u_end = (int)((int64_t)units * (slice + 1) / DS);

  T* xt = reinterpret_cast<T*>(lds);
  const T* xzero = xt + NT * pitch;  // 16-byte zero slot after the chunk tile

  // Stage f-steps [fs0, fs0 + fsc) of the tile's rows into LDS, zero past F
  // and past the last sample. A work item is one f-step of one row: two
  // 16-byte groups of X in, two 16-byte LDS words out (fp32 interleaves the
  // two groups into the even/odd order of lds_pos). Loads are issued in
  // unconditional batches with addresses clamped into X and masked after.
  const bool vec = (F % Tr::kVec) == 0 && ((uintptr_t)X % 16) == 0;
  auto stage = [&](int fs0) {
    const int fsn = min(fsc, nfs - fs0);
    const int items = NT * fsn;
    for (int base = 0; base < items; base += kThreads * kSB) {
      uint4 w[kSB][2];
#pragma unroll
      for (int j = 0; j < kSB; ++j) {
        const int i = base + j * kThreads + tid;
        const int r = i / fsn, s = i - r * fsn;
        const int rr = r < rows ? r : rows - 1;
        const T* xr = X + (int64_t)(n0 + rr) * F;
#pragma unroll
        for (int g = 0; g < 2; ++g) {
          const int c = (fs0 + s) * Tr::kFStep + g * Tr::kVec;
          if (vec) {
            const int cc = c < F ? c : F - Tr::kVec;
            w[j][g] = *reinterpret_cast<const uint4*>(xr + cc);
          } else {
            uint32_t t[4] = {0u, 0u, 0u, 0u};
#pragma unroll
            for (int e = 0; e < Tr::kVec; ++e) {
              const int ce = c + e < F ? c + e : F - 1;
              Tr::put(t, e, xr[ce]);
            }
            w[j][g] = make_uint4(t[0], t[1], t[2], t[3]);
          }
        }
      }
#pragma unroll
      for (int j = 0; j < kSB; ++j) {
        const int i = base + j * kThreads + tid;
        if (i >= items) break;
        const int r = i / fsn, s = i - r * fsn;
#pragma unroll
        for (int g = 0; g < 2; ++g) {
          const int c = (fs0 + s) * Tr::kFStep + g * Tr::kVec;
          if (r >= rows || c >= F) {
            w[j][g] = make_uint4(0u, 0u, 0u, 0u);
          } else if (c + Tr::kVec > F) {  // ragged last group (F % kVec != 0)
            uint32_t t[4] = {w[j][g].x, w[j][g].y, w[j][g].z, w[j][g].w};
#pragma unroll
            for (int e = 0; e < Tr::kVec; ++e)
              if (c + e >= F) Tr::clear(t, e);
            w[j][g] = make_uint4(t[0], t[1], t[2], t[3]);
          }
        }
        uint4* dst = reinterpret_cast<uint4*>(xt + r * pitch + s * Tr::kFStep);
        if constexpr (Tr::kEsz != 4) {
          dst[0] = w[j][0];
          dst[1] = w[j][1];
        } else {  // fp32: even features of the step first (lds_pos)
          dst[0] = make_uint4(w[j][0].x, w[j][0].z, w[j][1].x, w[j][1].z);
          dst[1] = make_uint4(w[j][0].y, w[j][0].w, w[j][1].y, w[j][1].w);
        }
      }
    }
  };

  f32x16 sacc[NTILES][KB];
#pragma unroll
  for (int t = 0; t < NTILES; ++t)
#pragma unroll
    for (int kb = 0; kb < KB; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) sacc[t][kb][r] = 0.0f;

  const int xrow = lane & 31, xhalf = lane >> 5;
  const T* xlane = xt + xrow * pitch + xhalf * (Tr::kFStep / 2);
  const __amdgpu_buffer_rsrc_t brsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint4*>(Bp), 0, ndb * nfs * 1024, 0x00020000);
  auto bfrag = [&](int uu, int fs, int b) -> uint4 {
    return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(
                                         brsrc, ((2 * uu + b) * nfs + fs) * 1024 + lane * 16, 0, 0));
  };

  const int n_it = (u_end - u_begin + kWaves - 1) / kWaves;
  for (int it = 0; it < n_it; ++it) {
    const int u = u_begin + wave + it * kWaves;
    const bool valid = u < u_end;
    const int uu = valid ? u : u_begin;  // waves without a unit compute and discard
    CFrags<Tr, KB> cf;
    cf.load(Cp, 2 * uu, lane);
    f32x16 vacc[2][NTILES];
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int t = 0; t < NTILES; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) vacc[b][t][r] = 0.0f;

    for (int ch = 0; ch < nchunks; ++ch) {
      const int fs0 = ch * fsc;
      const int fsn = min(fsc, nfs - fs0);  // f-steps of this chunk
      __syncthreads();  // the previous chunk's readers are done
      if (tid == 0) *reinterpret_cast<uint4*>(xt + NT * pitch) = make_uint4(0u, 0u, 0u, 0u);
      stage(fs0);
      __syncthreads();
      uint4 afr[kPrefetch][2];
#pragma unroll
      for (int i = 0; i < kPrefetch; ++i) {
        afr[i][0] = bfrag(uu, fs0 + (i < fsn ? i : fsn - 1), 0);
        afr[i][1] = bfrag(uu, fs0 + (i < fsn ? i : fsn - 1), 1);
      }
      uint4 xfr[2][NTILES];
#pragma unroll
      for (int t = 0; t < NTILES; ++t)
        xfr[0][t] = *reinterpret_cast<const uint4*>(xlane + t * 32 * pitch);
      const int fsl = (fsn + kPrefetch - 1) / kPrefetch * kPrefetch;
      // Same branch-free step as the resident kernel: padding steps past fsn
      // multiply a valid B fragment by the zero slot.
      for (int s0 = 0; s0 < fsl; s0 += kPrefetch) {
#pragma unroll
        for (int i = 0; i < kPrefetch; ++i) {
          const int fs = s0 + i;
          const int fsx = fs + 1;
#pragma unroll
          for (int t = 0; t < NTILES; ++t)
            xfr[(i + 1) & 1][t] = *reinterpret_cast<const uint4*>(
                fsx < fsn ? xlane + t * 32 * pitch + fsx * Tr::kFStep : xzero);
#pragma unroll
          for (int b = 0; b < 2; ++b)
#pragma unroll
            for (int t = 0; t < NTILES; ++t) Tr::stage1(vacc[b][t], afr[i][b], xfr[i & 1][t]);
          __builtin_amdgcn_sched_group_barrier(0x100, NTILES, 0);
          __builtin_amdgcn_sched_group_barrier(0x008, 2 * NTILES * Tr::kStage1Mfma, 0);
          __builtin_amdgcn_sched_group_barrier(0x020, 2, 0);
          const int nx = fs + kPrefetch;
          afr[i][0] = bfrag(uu, fs0 + (nx < fsn ? nx : fsn - 1), 0);
          afr[i][1] = bfrag(uu, fs0 + (nx < fsn ? nx : fsn - 1), 1);
        }
      }
    }
    if (valid) {
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int t = 0; t < NTILES; ++t) cf.template apply<ACT>(vacc[b][t], b, sacc[t]);
    }
  }
  __syncthreads();  // the last chunk's readers are done before LDS is reused
  finish_tile<NTILES, KB>(sacc, lds, &s_last, labels, scores, N, K, DS, ntiles, slice, tile, n0,
                          workspace);
}

// LDS fragment reads of the double-buffered kernel. With buffer-to-LDS loads
// in flight the compiler would put a full vmcnt(0) wait before every LDS
// read it cannot prove disjoint from them; these reads are issued directly
// and completed by an explicit lgkmcnt(0) tied to the destination registers.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}
typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 lds_read16_issue(uint32_t addr) {
  u32x4_t v;
  asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"(addr));
  return __builtin_bit_cast(uint4, v);
}
template <int NT>
__device__ __forceinline__ void lds_reads_complete(uint4 (&v)[NT]) {
  u32x4_t a = __builtin_bit_cast(u32x4_t, v[0]);
  u32x4_t b = __builtin_bit_cast(u32x4_t, v[NT > 1 ? 1 : 0]);
  u32x4_t c = __builtin_bit_cast(u32x4_t, v[NT > 2 ? 2 : 0]);
  u32x4_t d = __builtin_bit_cast(u32x4_t, v[NT > 3 ? 3 : 0]);
  if constexpr (NT == 1)
    asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(a));
  else if constexpr (NT == 2)
    asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(a), "+v"(b));
  else
    asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(a), "+v"(b), "+v"(c), "+v"(d));
  v[0] = __builtin_bit_cast(uint4, a);
  if constexpr (NT > 1) v[1] = __builtin_bit_cast(uint4, b);
  if constexpr (NT > 2) v[2] = __builtin_bit_cast(uint4, c);
  if constexpr (NT > 3) v[3] = __builtin_bit_cast(uint4, d);
}

// ---------------------------------------------------------------------------
// bf16 / int8 F-chunked variant with the X chunks double-buffered in LDS and
// filled by direct buffer-to-LDS loads (lane l of a 16-byte load lands at the wave's
// LDS base + 16 l; out-of-range offsets deliver zeros). The loads of the next
// chunk are issued two per f-step at the start of the current one, so they
// overlap the matrix instructions. Chunks are a fixed kDmaFsc f-steps (the
// last one of a unit padded with zero X), which keeps the B fragment ring
// running across chunk and unit boundaries, and lets the barrier that
// publishes a chunk wait only for the LDS loads, not for the ring behind them.
// An LDS row is W = 2 kDmaFsc + 1 slots of 16 bytes: two per f-step plus one
// padding slot that keeps the 32 rows of a fragment read on distinct banks.
// Requires F to be a whole number of 16-byte groups and a 16-byte aligned X.
// ---------------------------------------------------------------------------
constexpr int kDmaFsc = 16;

// The double-buffered kernel works on 64-sample workgroup tiles. With one
// class block each wave takes two units per pass over the X chunks: the same
// accumulator registers as 128 samples times one unit, with the X chunks
// re-read half as often.
constexpr int kDmaNtiles = 2;
__host__ __device__ constexpr int dma_units_per_wave(int ntiles, int kb) {
  return ntiles == 2 && kb == 1 ? 2 : 1;
}

__host__ __device__ constexpr int dma_loads_per_wave(int ntiles) {
  return (32 * ntiles * (2 * kDmaFsc + 1) + kThreads - 1) / kThreads;
}

template <class Tr, int NTILES, int KB, int ACT>
__global__ __launch_bounds__(kThreads, 1) void large_chunked_dma_kernel(
    const typename Tr::elem* __restrict__ X, const uint4* __restrict__ Bp,
    const uint4* __restrict__ Cp, int32_t* __restrict__ labels, float* __restrict__ scores, int N,
    int F, int K, int ndb, int DS, void* __restrict__ workspace) {
  typedef typename Tr::elem T;
  static_assert(Tr::kEsz <= 2, "16-byte slots of bf16 or int8");
  constexpr int NT = 32 * NTILES;
  constexpr int UPW = dma_units_per_wave(NTILES, KB);  // units per wave per X pass
  constexpr int kPF = UPW > 1 ? 4 : prefetch_of(NTILES, KB);
  constexpr int FSC = kDmaFsc;
  constexpr int W = 2 * FSC + 1;                 // slots per LDS row
  constexpr int pitch = Tr::kVec * W;            // elements
  constexpr int P = dma_loads_per_wave(NTILES);  // LDS loads per wave per chunk
  constexpr int kDmaSteps = (P + 1) / 2;         // the first steps issue them, two each
  constexpr int kAfter = 2 * UPW * (FSC - kDmaSteps);  // ring loads issued after the last one
  constexpr int kWait = kAfter < 2 * UPW * kPF ? kAfter : 2 * UPW * kPF;
  constexpr int buf_elems = P * kThreads * Tr::kVec;
  constexpr int kTileBytes = 32 * pitch * Tr::kEsz;  // 32 rows of a buffer
  constexpr int kStepBytes = Tr::kFStep * Tr::kEsz;  // one f-step of a row
  static_assert(FSC % kPF == 0 && kDmaSteps <= FSC && kWait <= 63, "chunk schedule");
  // s_waitcnt immediate: vmcnt(kWait), expcnt and lgkmcnt not waited on
  constexpr int kWaitImm = 0x0F70 | (kWait & 15) | ((kWait >> 4) << 14);
  extern __shared__ __attribute__((aligned(16))) unsigned char lds[];
  __shared__ int s_last;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nfs = nfs_of<Tr>(F);
  const int nchunks = (nfs + FSC - 1) / FSC;
  const int nfl = nchunks * FSC;  // f-steps per unit, padded to whole chunks
  const int ntiles = (int)cdiv(N, NT);
  const int slice = blockIdx.x % DS;
  const int tile = blockIdx.x / DS;
  const int n0 = tile * NT;
  const int rows = min(NT, N - n0);
  const int units = ndb / 2;
  const int u_begin = (int)((int64_t)units * slice / DS);
  const int u_end = (int)((int64_t)units * (slice + 1) / DS);

  T* xb = reinterpret_cast<T*>(lds);        // two buffers of buf_elems
  const T* xzero = xb + 2 * buf_elems;      // 16-byte zero slot
  if (tid == 0) *reinterpret_cast<uint4*>(xb + 2 * buf_elems) = make_uint4(0u, 0u, 0u, 0u);

  // The tile's rows of X as one buffer resource; rows past N are out of range.
  const __amdgpu_buffer_rsrc_t xrsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<T*>(X + (int64_t)n0 * F), 0, rows * F * Tr::kEsz, 0x00020000);
  // Load p of this wave for chunk ch into buffer `buf`: slot q of the buffer.
  auto dma = [&](int ch, int p, int buf) {
    int q = (p * kWaves + wave) * 64 + lane;
    // recomputed at each use: hoisting the per-load slot arithmetic out of
    // the chunk loop would hold dozens of registers for the whole unit
    asm volatile("" : "+v"(q));
    const int r = q / W, rem = q - r * W;
    const int col = (ch * FSC + (rem >> 1)) * Tr::kFStep + (rem & 1) * Tr::kVec;
    const bool ok = r < rows && rem < 2 * FSC && col < F;
    const unsigned off = ok ? (unsigned)((r * F + col) * Tr::kEsz) : 0x80000000u;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        xrsrc,
        (__attribute__((address_space(3))) void*)(xb + buf * buf_elems +
                                                  (p * kWaves + wave) * 64 * Tr::kVec),
        16, off, 0, 0, 0);
  };

  f32x16 sacc[NTILES][KB];
#pragma unroll
  for (int t = 0; t < NTILES; ++t)
#pragma unroll
    for (int kb = 0; kb < KB; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) sacc[t][kb][r] = 0.0f;

  const int xrow = lane & 31, xhalf = lane >> 5;
  const int xlane = xrow * pitch + xhalf * (Tr::kFStep / 2);  // element offset in a buffer
  const __amdgpu_buffer_rsrc_t brsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint4*>(Bp), 0, ndb * nfs * 1024, 0x00020000);
  auto bfrag = [&](int uu, int fs, int b) -> uint4 {
    return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(
                                         brsrc, ((2 * uu + b) * nfs + fs) * 1024 + lane * 16, 0, 0));
  };
  // this wave's j-th unit in iteration it (a valid unit when it has none: computed, discarded)
  auto unit_idx = [&](int it, int j) { return u_begin + wave + (it * UPW + j) * kWaves; };
  auto unit_of = [&](int it, int j) {
    const int u = unit_idx(it, j);
    return u < u_end ? u : u_begin;
  };

  for (int p = 0; p < P; ++p) dma(0, p, 0);
  // ring slot g % kPF of unit j holds f-step g of the current unit j
  uint4 afr[UPW][kPF][2];
#pragma unroll
  for (int j = 0; j < UPW; ++j) {
    const int u0 = unit_of(0, j);
#pragma unroll
    for (int i = 0; i < kPF; ++i) {
      afr[j][i][0] = bfrag(u0, i < nfs ? i : nfs - 1, 0);
      afr[j][i][1] = bfrag(u0, i < nfs ? i : nfs - 1, 1);
    }
  }
  int cur = 0;
  const int n_it = (u_end - u_begin + kWaves * UPW - 1) / (kWaves * UPW);
  for (int it = 0; it < n_it; ++it) {
    int uu[UPW], un[UPW];
    CFrags<Tr, KB> cf[UPW];
    f32x16 vacc[UPW][2][NTILES];
#pragma unroll
    for (int j = 0; j < UPW; ++j) {
      uu[j] = unit_of(it, j);
      un[j] = unit_of(it + 1, j);
      cf[j].load(Cp, 2 * uu[j], lane);
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int t = 0; t < NTILES; ++t)
#pragma unroll
          for (int r = 0; r < 16; ++r) vacc[j][b][t][r] = 0.0f;
    }

    for (int ch = 0; ch < nchunks; ++ch) {
      const int fs0 = ch * FSC;
      const int fsn = min(FSC, nfs - fs0);
      const int nch = ch + 1 < nchunks ? ch + 1 : 0;  // the next chunk to fill
      // This wave's loads of chunk ch are done (only ring loads were issued
      // after them); after the barrier every wave's are, and nobody still
      // reads the other buffer.
      __builtin_amdgcn_s_waitcnt(kWaitImm);
      __syncthreads();
      const uint32_t xc = lds_addr(xb + cur * buf_elems + xlane);
      const uint32_t xz = lds_addr(xzero);
      const int nbuf = cur ^ 1;
      uint4 xfr[2][NTILES];
#pragma unroll
      for (int t = 0; t < NTILES; ++t) xfr[0][t] = lds_read16_issue(xc + t * kTileBytes);
#pragma unroll
      for (int s = 0; s < FSC; ++s) {
        const int i = s % kPF;
        lds_reads_complete<NTILES>(xfr[s & 1]);
#pragma unroll
        for (int t = 0; t < NTILES; ++t)
          xfr[(s + 1) & 1][t] =
              lds_read16_issue(s + 1 < fsn ? xc + t * kTileBytes + (s + 1) * kStepBytes : xz);
#pragma unroll
        for (int j = 0; j < UPW; ++j)
#pragma unroll
          for (int b = 0; b < 2; ++b)
#pragma unroll
            for (int t = 0; t < NTILES; ++t)
              Tr::stage1(vacc[j][b][t], afr[j][i][b], xfr[s & 1][t]);
        __builtin_amdgcn_sched_group_barrier(0x008, 2 * NTILES * UPW, 0);
        if (s < kDmaSteps)
          __builtin_amdgcn_sched_group_barrier(0x020, 2 * UPW + 2, 0);
        else
          __builtin_amdgcn_sched_group_barrier(0x020, 2 * UPW, 0);
        // refill: f-step g of this unit, else the next unit's first steps
        const int g = fs0 + s + kPF;
        const int rg0 = g < nfl ? g : g - nfl;
        const int rg = rg0 < nfs ? rg0 : nfs - 1;
#pragma unroll
        for (int j = 0; j < UPW; ++j) {
          const int ru = g < nfl ? uu[j] : un[j];
          afr[j][i][0] = bfrag(ru, rg, 0);
          afr[j][i][1] = bfrag(ru, rg, 1);
        }
        if (s < kDmaSteps) {
          dma(nch, 2 * s < P ? 2 * s : P - 1, nbuf);  // a repeated load is harmless
          dma(nch, 2 * s + 1 < P ? 2 * s + 1 : P - 1, nbuf);
        }
      }
      lds_reads_complete<NTILES>(xfr[FSC & 1]);  // the padding read of the last step
      cur = nbuf;
    }
#pragma unroll
    for (int j = 0; j < UPW; ++j) {
      if (unit_idx(it, j) < u_end) {
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
          for (int t = 0; t < NTILES; ++t) cf[j].template apply<ACT>(vacc[j][b][t], b, sacc[t]);
      }
    }
  }
  __builtin_amdgcn_s_waitcnt(0x0F70);  // no load into LDS is still in flight
  __syncthreads();
  finish_tile<NTILES, KB>(sacc, lds, &s_last, labels, scores, N, K, DS, ntiles, slice, tile, n0,
                          workspace);
}

// ---------------------------------------------------------------------------
// Single-pass training on the matrix cores (Sec. II-C): the class sums
// counts[k][d] += sum over samples n of class k of HardSign(X_n B)[d], from
// the tiled B of a packed model.
//
// Stage I is computed here as V = X B, not transposed: the same fragments as
// inference with the two operands exchanged, so the sample n is the MFMA row
// index and the hypervector dimension d the column index. Each lane then ends
// with 16 samples of one column, and the 32 lanes of a half-wave hold 32
// consecutive columns of one sample: the class-counter adds in LDS touch 32
// consecutive words of one class row per instruction, free of bank and
// address conflicts.
//
// A work item is (sample tile of NT samples, column group of 256 = one
// 64-column unit per wave). A workgroup takes one column group and a
// contiguous range of sample tiles; each tile's X streams through LDS in
// chunks of fsc f-steps while V stays in registers across the chunks, and the
// workgroup's class counters [K][256] stay in LDS until its last tile, then
// are added into the caller's counts with one device atomic per nonzero
// counter.
// ---------------------------------------------------------------------------
constexpr int kBundleCols = 64 * kWaves;
constexpr int kBundleStageBatch = 4;  // staging items per thread per batch

// Stage f-steps [fs0, fs0 + fsn) of rows n0 .. n0 + rows - 1 of X into the
// LDS tile (row pitch `pitch` elements), zero past F; rows past `rows` are
// not written (their labels are invalid, so their V is never used).
template <class Tr, int NT>
__device__ __forceinline__ void bundle_stage(typename Tr::elem* xt, const typename Tr::elem* X,
                                             int F, int64_t n0, int rows, int fs0, int fsn,
                                             int pitch, bool vec, int tid) {
  typedef typename Tr::elem T;
  constexpr int kSB = kBundleStageBatch;
  const int items = NT * fsn;
  for (int base = 0; base < items; base += kThreads * kSB) {
    uint4 w[kSB][2];
#pragma unroll
    for (int j = 0; j < kSB; ++j) {
      const int i = base + j * kThreads + tid;
      const int r = i / fsn, s = i - r * fsn;
      const int rr = r < rows ? r : rows - 1;  // clamped into X, masked below
      const T* xr = X + (n0 + rr) * (int64_t)F;
#pragma unroll
      for (int g = 0; g < 2; ++g) {
        const int c = (fs0 + s) * Tr::kFStep + g * Tr::kVec;
        if (vec) {
          const int cc = c < F ? c : F - Tr::kVec;
          w[j][g] = *reinterpret_cast<const uint4*>(xr + cc);
        } else {
          uint32_t t[4] = {0u, 0u, 0u, 0u};
#pragma unroll
          for (int e = 0; e < Tr::kVec; ++e) {
            const int ce = c + e < F ? c + e : F - 1;
            Tr::put(t, e, xr[ce]);
          }
          w[j][g] = make_uint4(t[0], t[1], t[2], t[3]);
        }
      }
    }
#pragma unroll
    for (int j = 0; j < kSB; ++j) {
      const int i = base + j * kThreads + tid;
      if (i >= items) break;
      const int r = i / fsn, s = i - r * fsn;
      if (r >= rows) continue;
#pragma unroll
      for (int g = 0; g < 2; ++g) {
        const int c = (fs0 + s) * Tr::kFStep + g * Tr::kVec;
        if (c >= F) {
          w[j][g] = make_uint4(0u, 0u, 0u, 0u);
        } else if (c + Tr::kVec > F) {  // ragged last group (F % kVec != 0)
          uint32_t t[4] = {w[j][g].x, w[j][g].y, w[j][g].z, w[j][g].w};
#pragma unroll
          for (int e = 0; e < Tr::kVec; ++e)
            if (c + e >= F) Tr::clear(t, e);
          w[j][g] = make_uint4(t[0], t[1], t[2], t[3]);
        }
      }
      uint4* dst = reinterpret_cast<uint4*>(xt + r * pitch + s * Tr::kFStep);
      if constexpr (Tr::kEsz != 4) {
        dst[0] = w[j][0];
        dst[1] = w[j][1];
      } else {  // fp32: even features of the step first (lds_pos)
        dst[0] = make_uint4(w[j][0].x, w[j][0].z, w[j][1].x, w[j][1].z);
        dst[1] = make_uint4(w[j][0].y, w[j][0].w, w[j][1].y, w[j][1].w);
      }
    }
  }
}

template <class Tr, int NTILES, int OCC>
__global__ __launch_bounds__(kThreads, OCC) void bundle_mfma_kernel(
    const typename Tr::elem* __restrict__ X, const uint4* __restrict__ Bp,
    const int32_t* __restrict__ y, int32_t* __restrict__ counts, int N, int F, int D, int K,
    int ndb, int ngroups, int fsc) {
  typedef typename Tr::elem T;
  constexpr int NT = 32 * NTILES;
  constexpr int kPrefetch = prefetch_of(NTILES, 1);
  extern __shared__ __attribute__((aligned(16))) unsigned char lds[];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nfs = nfs_of<Tr>(F);
  const int nchunks = (nfs + fsc - 1) / fsc;
  const int pitch = fsc * Tr::kFStep + pad_of<Tr>();  // elements
  const int units = ndb / 2;
  const int ncg = (units + kWaves - 1) / kWaves;
  const int cg = blockIdx.x % ncg;
  const int sg = blockIdx.x / ncg;
  const int ntiles = (N + NT - 1) / NT;
  const int t_begin = (int)((int64_t)ntiles * sg / ngroups);
  const int t_end = (int)((int64_t)ntiles * (sg + 1) / ngroups);

  // LDS: [X chunk tile NT x pitch | 16-byte zero slot | labels NT | counters K x 256]
  T* xt = reinterpret_cast<T*>(lds);
  const size_t xbytes = (size_t)NT * pitch * sizeof(T) + 16;
  const T* xzero = xt + NT * pitch;
  int* ys = reinterpret_cast<int*>(lds + xbytes);
  int* cnt = ys + NT;
  for (int i = tid; i < K * kBundleCols; i += kThreads) cnt[i] = 0;
  if (tid == 0) *reinterpret_cast<uint4*>(xt + NT * pitch) = make_uint4(0u, 0u, 0u, 0u);

  const int u = cg * kWaves + wave;
  const bool valid = u < units;
  const int uu = valid ? u : cg * kWaves;  // waves without a unit compute and discard
  const int xrow = lane & 31, xhalf = lane >> 5;
  const T* xlane = xt + xrow * pitch + xhalf * (Tr::kFStep / 2);
  const __amdgpu_buffer_rsrc_t brsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint4*>(Bp), 0, ndb * nfs * 1024, 0x00020000);
  auto bfrag = [&](int fs, int b) -> uint4 {
    return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(
                                         brsrc, ((2 * uu + b) * nfs + fs) * 1024 + lane * 16, 0, 0));
  };
  const bool vec = (F % Tr::kVec) == 0 && ((uintptr_t)X % 16) == 0;

  for (int tile = t_begin; tile < t_end; ++tile) {
    const int64_t n0 = (int64_t)tile * NT;
    const int rows = (int)min((int64_t)NT, (int64_t)N - n0);
    f32x16 vacc[2][NTILES];
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int t = 0; t < NTILES; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) vacc[b][t][r] = 0.0f;

    for (int ch = 0; ch < nchunks; ++ch) {
      const int fs0 = ch * fsc;
      const int fsn = min(fsc, nfs - fs0);
      __syncthreads();  // the previous chunk's (and tile's) readers are done
      if (ch == 0 && tid < NT) {
        int k = -1;
        if (tid < rows) {
          k = y[n0 + tid];
          if (k < 0 || k >= K) k = -1;  // labels outside [0, K) are skipped
        }
        ys[tid] = k;
      }
      bundle_stage<Tr, NT>(xt, X, F, n0, rows, fs0, fsn, pitch, vec, tid);
      __syncthreads();
      uint4 afr[kPrefetch][2];
#pragma unroll
      for (int i = 0; i < kPrefetch; ++i) {
        afr[i][0] = bfrag(fs0 + (i < fsn ? i : fsn - 1), 0);
        afr[i][1] = bfrag(fs0 + (i < fsn ? i : fsn - 1), 1);
      }
      uint4 xfr[2][NTILES];
#pragma unroll
      for (int t = 0; t < NTILES; ++t)
        xfr[0][t] = *reinterpret_cast<const uint4*>(xlane + t * 32 * pitch);
      const int fsl = (fsn + kPrefetch - 1) / kPrefetch * kPrefetch;
      // Branch-free steps as in inference: padding steps past fsn multiply a
      // valid B fragment by the zero slot.
      for (int s0 = 0; s0 < fsl; s0 += kPrefetch) {
#pragma unroll
        for (int i = 0; i < kPrefetch; ++i) {
          const int fs = s0 + i;
          const int fsx = fs + 1;
#pragma unroll
          for (int t = 0; t < NTILES; ++t)
            xfr[(i + 1) & 1][t] = *reinterpret_cast<const uint4*>(
                fsx < fsn ? xlane + t * 32 * pitch + fsx * Tr::kFStep : xzero);
#pragma unroll
          for (int b = 0; b < 2; ++b)
#pragma unroll
            for (int t = 0; t < NTILES; ++t) Tr::stage1(vacc[b][t], xfr[i & 1][t], afr[i][b]);
          __builtin_amdgcn_sched_group_barrier(0x100, NTILES, 0);
          __builtin_amdgcn_sched_group_barrier(0x008, 2 * NTILES * Tr::kStage1Mfma, 0);
          __builtin_amdgcn_sched_group_barrier(0x020, 2, 0);
          const int nx = fs + kPrefetch;
          afr[i][0] = bfrag(fs0 + (nx < fsn ? nx : fsn - 1), 0);
          afr[i][1] = bfrag(fs0 + (nx < fsn ? nx : fsn - 1), 1);
        }
      }
    }
    // HardSign (Eq. 1) and the class sums. Accumulator r of lane l is row
    // 8(r/4) + 4(l/32) + r%4 (a sample) of column l%32 (a dimension).
    if (valid) {
#pragma unroll
      for (int t = 0; t < NTILES; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int k = ys[32 * t + 8 * (r >> 2) + 4 * xhalf + (r & 3)];
          if (k >= 0) {
#pragma unroll
            for (int b = 0; b < 2; ++b)
              atomicAdd(&cnt[k * kBundleCols + wave * 64 + 32 * b + xrow],
                        Tr::nonneg(vacc[b][t][r]) ? 1 : -1);
          }
        }
    }
  }
  __syncthreads();
  const int64_t d0 = (int64_t)cg * kBundleCols;
  for (int i = tid; i < K * kBundleCols; i += kThreads) {
    const int k = i / kBundleCols, c = i % kBundleCols;
    const int v = cnt[i];
    if (v != 0 && d0 + c < D) atomicAdd(&counts[(int64_t)k * D + d0 + c], v);
  }
}

// bf16 and int8 training with the X chunks double-buffered in LDS and filled
// by buffer-to-LDS loads, on the schedule of large_chunked_dma_kernel: 64-sample
// tiles, chunks of kDmaFsc f-steps, the next chunk's loads issued two per
// f-step at the start of the current one, the B fragment ring running on
// across chunks and tiles (a wave keeps its units for every tile). The
// labels of the tile a chunk belongs to travel with it: one 4-byte
// buffer-to-LDS load per wave at the chunk's first step (every wave writes the
// same values) into a label buffer selected by tile parity.
// Requires F to be a whole number of 16-byte groups and a 16-byte aligned X.
template <class Tr, int UPW>
__global__ __launch_bounds__(kThreads, 1) void bundle_dma_kernel(
    const typename Tr::elem* __restrict__ X, const uint4* __restrict__ Bp,
    const int32_t* __restrict__ y, int32_t* __restrict__ counts, int N, int F, int D, int K,
    int ndb, int ngroups) {
  typedef typename Tr::elem T;
  static_assert(Tr::kEsz <= 2, "16-byte slots of bf16 or int8");
  constexpr int NTILES = kDmaNtiles;
  constexpr int NT = 32 * NTILES;
  constexpr int kPF = UPW > 1 ? 4 : prefetch_of(NTILES, 1);
  constexpr int FSC = kDmaFsc;
  constexpr int W = 2 * FSC + 1;                 // 16-byte slots per LDS row
  constexpr int pitch = Tr::kVec * W;            // elements
  constexpr int P = dma_loads_per_wave(NTILES);  // X loads per wave per chunk
  constexpr int kDmaSteps = (P + 1) / 2;
  constexpr int kAfter = 2 * UPW * (FSC - kDmaSteps);
  constexpr int kWait = kAfter < 2 * UPW * kPF ? kAfter : 2 * UPW * kPF;
  constexpr int buf_elems = P * kThreads * Tr::kVec;
  constexpr int kCols = kWaves * UPW * 64;  // columns per workgroup
  constexpr int kTileBytes = 32 * pitch * Tr::kEsz;     // 32 rows of a buffer
  constexpr int kStepBytes = Tr::kFStep * Tr::kEsz;     // one f-step of a row
  static_assert(NT == 64 && FSC % kPF == 0 && kDmaSteps <= FSC && kWait <= 63, "schedule");
  constexpr int kWaitImm = 0x0F70 | (kWait & 15) | ((kWait >> 4) << 14);
  extern __shared__ __attribute__((aligned(16))) unsigned char lds[];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nfs = nfs_of<Tr>(F);
  const int nchunks = (nfs + FSC - 1) / FSC;
  const int nfl = nchunks * FSC;
  const int units = ndb / 2;
  const int ncg = (units + kWaves * UPW - 1) / (kWaves * UPW);
  const int cg = blockIdx.x % ncg;
  const int sg = blockIdx.x / ncg;
  const int ntiles = (N + NT - 1) / NT;
  const int t_begin = (int)((int64_t)ntiles * sg / ngroups);
  const int t_end = (int)((int64_t)ntiles * (sg + 1) / ngroups);

  // LDS: [two X buffers | zero slot | labels 2 x NT | counters K x kCols]
  T* xb = reinterpret_cast<T*>(lds);
  const T* xzero = xb + 2 * buf_elems;
  int* ys = reinterpret_cast<int*>(lds + 2 * buf_elems * sizeof(T) + 16);
  int* cnt = ys + 2 * NT;
  if (tid == 0) *reinterpret_cast<uint4*>(xb + 2 * buf_elems) = make_uint4(0u, 0u, 0u, 0u);
  for (int i = tid; i < K * kCols; i += kThreads) cnt[i] = 0;

  // Load p of this wave for chunk ch of tile tl into buffer buf (rows past N
  // and columns past F are out of the resource's range and read as zero).
  auto dma = [&](int tl, int ch, int p, int buf) {
    const int64_t n0 = (int64_t)tl * NT;
    const int rows = (int)min((int64_t)NT, (int64_t)N - n0);
    const __amdgpu_buffer_rsrc_t xr = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<T*>(X + n0 * F), 0, rows * F * Tr::kEsz, 0x00020000);
    int q = (p * kWaves + wave) * 64 + lane;
    asm volatile("" : "+v"(q));
    const int r = q / W, rem = q - r * W;
    const int col = (ch * FSC + (rem >> 1)) * Tr::kFStep + (rem & 1) * Tr::kVec;
    const bool ok = r < rows && rem < 2 * FSC && col < F;
    const unsigned off = ok ? (unsigned)((r * F + col) * Tr::kEsz) : 0x80000000u;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        xr,
        (__attribute__((address_space(3))) void*)(xb + buf * buf_elems +
                                                  (p * kWaves + wave) * 64 * Tr::kVec),
        16, off, 0, 0, 0);
  };
  // The labels of tile tl into label buffer tl & 1 (lane l: row l).
  auto label_dma = [&](int tl) {
    const int64_t n0 = (int64_t)tl * NT;
    const int rows = (int)min((int64_t)NT, (int64_t)N - n0);
    const __amdgpu_buffer_rsrc_t yr = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<int32_t*>(y + n0), 0, rows * 4, 0x00020000);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        yr, (__attribute__((address_space(3))) void*)(ys + (tl & 1) * NT), 4,
        (unsigned)lane * 4u, 0, 0, 0);
  };

  const int xrow = lane & 31, xhalf = lane >> 5;
  const int xlane = xrow * pitch + xhalf * (Tr::kFStep / 2);
  const __amdgpu_buffer_rsrc_t brsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint4*>(Bp), 0, ndb * nfs * 1024, 0x00020000);
  auto bfrag = [&](int uu, int fs, int b) -> uint4 {
    return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(
                                         brsrc, ((2 * uu + b) * nfs + fs) * 1024 + lane * 16, 0, 0));
  };
  // this wave's j-th unit (a valid unit of the group when it has none:
  // computed and discarded)
  int uu[UPW];
  bool uvalid[UPW];
#pragma unroll
  for (int j = 0; j < UPW; ++j) {
    const int u = cg * kWaves * UPW + j * kWaves + wave;
    uvalid[j] = u < units;
    uu[j] = uvalid[j] ? u : cg * kWaves * UPW;
  }

  if (t_begin < t_end) {
    label_dma(t_begin);
    for (int p = 0; p < P; ++p) dma(t_begin, 0, p, 0);
  }
  uint4 afr[UPW][kPF][2];
#pragma unroll
  for (int j = 0; j < UPW; ++j)
#pragma unroll
    for (int i = 0; i < kPF; ++i) {
      afr[j][i][0] = bfrag(uu[j], i < nfs ? i : nfs - 1, 0);
      afr[j][i][1] = bfrag(uu[j], i < nfs ? i : nfs - 1, 1);
    }
  int cur = 0;
  for (int tile = t_begin; tile < t_end; ++tile) {
    const int rows = min(NT, N - tile * NT);
    f32x16 vacc[UPW][2][NTILES];
#pragma unroll
    for (int j = 0; j < UPW; ++j)
#pragma unroll
      for (int b = 0; b < 2; ++b)
#pragma unroll
        for (int t = 0; t < NTILES; ++t)
#pragma unroll
          for (int r = 0; r < 16; ++r) vacc[j][b][t][r] = 0.0f;

    for (int ch = 0; ch < nchunks; ++ch) {
      const int fs0 = ch * FSC;
      const int fsn = min(FSC, nfs - fs0);
      // the chunk to fill next: the next one of this tile, else the first of
      // the next tile (the last tile reloads its own first chunk, unread)
      const bool last = ch + 1 == nchunks;
      const int ntl = last ? (tile + 1 < t_end ? tile + 1 : tile) : tile;
      const int nch = last ? 0 : ch + 1;
      __builtin_amdgcn_s_waitcnt(kWaitImm);
      __syncthreads();
      const uint32_t xc = lds_addr(xb + cur * buf_elems + xlane);
      const uint32_t xz = lds_addr(xzero);
      const int nbuf = cur ^ 1;
      uint4 xfr[2][NTILES];
#pragma unroll
      for (int t = 0; t < NTILES; ++t) xfr[0][t] = lds_read16_issue(xc + t * kTileBytes);
#pragma unroll
      for (int s = 0; s < FSC; ++s) {
        const int i = s % kPF;
        lds_reads_complete<NTILES>(xfr[s & 1]);
#pragma unroll
        for (int t = 0; t < NTILES; ++t)
          xfr[(s + 1) & 1][t] =
              lds_read16_issue(s + 1 < fsn ? xc + t * kTileBytes + (s + 1) * kStepBytes : xz);
#pragma unroll
        for (int j = 0; j < UPW; ++j)
#pragma unroll
          for (int b = 0; b < 2; ++b)
#pragma unroll
            for (int t = 0; t < NTILES; ++t)
              Tr::stage1(vacc[j][b][t], xfr[s & 1][t], afr[j][i][b]);
        __builtin_amdgcn_sched_group_barrier(0x008, 2 * NTILES * UPW, 0);
        if (s == 0)
          __builtin_amdgcn_sched_group_barrier(0x020, 2 * UPW + 3, 0);
        else if (s < kDmaSteps)
          __builtin_amdgcn_sched_group_barrier(0x020, 2 * UPW + 2, 0);
        else
          __builtin_amdgcn_sched_group_barrier(0x020, 2 * UPW, 0);
        // refill: f-step g of the units (past the padded end: the next tile's
        // first steps of the same units)
        const int g = fs0 + s + kPF;
        const int rg0 = g < nfl ? g : g - nfl;
        const int rg = rg0 < nfs ? rg0 : nfs - 1;
#pragma unroll
        for (int j = 0; j < UPW; ++j) {
          afr[j][i][0] = bfrag(uu[j], rg, 0);
          afr[j][i][1] = bfrag(uu[j], rg, 1);
        }
        if (s == 0) label_dma(ntl);  // before this chunk's last X load
        if (s < kDmaSteps) {
          dma(ntl, nch, 2 * s < P ? 2 * s : P - 1, nbuf);
          dma(ntl, nch, 2 * s + 1 < P ? 2 * s + 1 : P - 1, nbuf);
        }
      }
      lds_reads_complete<NTILES>(xfr[FSC & 1]);
      cur = nbuf;
    }
    // HardSign (Eq. 1) and the class sums of this tile.
    const int* yt = ys + (tile & 1) * NT;
#pragma unroll
    for (int j = 0; j < UPW; ++j) {
      if (!uvalid[j]) continue;
#pragma unroll
      for (int t = 0; t < NTILES; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = 32 * t + 8 * (r >> 2) + 4 * xhalf + (r & 3);
          const int k = row < rows ? yt[row] : -1;
          if (k >= 0 && k < K) {
#pragma unroll
            for (int b = 0; b < 2; ++b)
              atomicAdd(&cnt[k * kCols + (j * kWaves + wave) * 64 + 32 * b + xrow],
                        Tr::nonneg(vacc[j][b][t][r]) ? 1 : -1);
          }
        }
    }
  }
  __builtin_amdgcn_s_waitcnt(0x0F70);  // no load into LDS is still in flight
  __syncthreads();
  const int64_t d0 = (int64_t)cg * kCols;
  for (int i = tid; i < K * kCols; i += kThreads) {
    const int k = i / kCols, c = i % kCols;
    const int v = cnt[i];
    if (v != 0 && d0 + c < D) atomicAdd(&counts[(int64_t)k * D + d0 + c], v);
  }
}

// ---------------------------------------------------------------------------
// Host-side configuration.
// ---------------------------------------------------------------------------
struct LargeCfg {
  int ntiles_per_wg;  // NTILES
  int kb;
  int fsc;            // f-steps per X chunk; 0 = the whole X tile stays in LDS
  bool dma;           // chunks double-buffered by buffer-to-LDS loads (bf16)
  int ds;
  int64_t ntiles;      // sample tiles
  size_t lds;
  bool ok;
};

// Calls f with the element traits of dt (0 fp32, 1 bf16, 2 int8).
template <class Fn>
auto with_traits(int dt, Fn&& f) {
  if (dt == 0) return f(TrF32{});
  if (dt == 2) return f(TrI8{});
  return f(TrBF16{});
}

template <class Tr>
LargeCfg large_cfg(int64_t N, int64_t F, int64_t D, int64_t K, bool x16 = true) {
  LargeCfg c{};
  if (cdiv(K, 32) > 4 || F > (1 << 20) || N > (1 << 30)) return c;
  if (Tr::kEsz == 1 && (F > kI8MaxF || D > kI8MaxD)) return c;
  // B fragments are addressed with 32-bit byte offsets
  if (cdiv(D, 64) * 2 * nfs_of<Tr>((int)F) * 1024 >= ((int64_t)1 << 31)) return c;
  const int pitch = pitch_of<Tr>((int)F);
  const int kbr = kb_of(K);
  for (int nt : {4, 2, 1}) {
    if (nt == 4 && kbr > 2) continue;
    const size_t xbytes = (size_t)32 * nt * pitch * Tr::kEsz + 16;  // + zero slot
    const size_t rbytes = (size_t)kWaves * 32 * nt * 32 * kbr * 4;
    const size_t need = xbytes > rbytes ? xbytes : rbytes;
    if (need <= (size_t)kLdsBytes) {
      c.ntiles_per_wg = nt;
      c.lds = need;
      break;
    }
  }
  // The double-buffered kernel: 64-sample tiles, X chunks by buffer-to-LDS
  // loads (16-byte groups of bf16 or int8).
  auto try_dma = [&]() {
    if (!(Tr::kEsz <= 2 && F % Tr::kVec == 0 && x16)) return false;
    // two buffers of P * kThreads slots of 16 bytes, plus the zero slot
    const int dnt = kDmaNtiles;
    const size_t drbytes = (size_t)kWaves * 32 * dnt * 32 * kbr * 4;
    const size_t dbytes = (size_t)2 * dma_loads_per_wave(dnt) * kThreads * 16 + 16;
    if (dbytes > (size_t)kLdsBytes || drbytes > (size_t)kLdsBytes) return false;
    c.dma = true;
    c.ntiles_per_wg = dnt;
    c.fsc = kDmaFsc;
    c.lds = dbytes > drbytes ? dbytes : drbytes;
    return true;
  };
  // int8 rows are short enough that a wide F still fits LDS as a 32-sample
  // tile; the double-buffered kernel uses each B fragment for 64 samples.
  if (Tr::kEsz == 1 && c.ntiles_per_wg == 1) try_dma();
  if (!c.ntiles_per_wg) {
    // X tile too large for LDS: stream it in chunks of f-steps
    const int nt = chunk_ntiles<Tr>(kbr);
    const size_t rbytes = (size_t)kWaves * 32 * nt * 32 * kbr * 4;
    const int pad = pad_of<Tr>();
    const int64_t cols = ((int64_t)kLdsBytes - 16) / (32 * nt * Tr::kEsz) - pad;
    const int fsc = (int)(cols / Tr::kFStep);
    if (fsc < 8 || rbytes > (size_t)kLdsBytes) return c;
    c.ntiles_per_wg = nt;
    c.fsc = fsc;
    const size_t xbytes = (size_t)32 * nt * (fsc * Tr::kFStep + pad) * Tr::kEsz + 16;
    c.lds = xbytes > rbytes ? xbytes : rbytes;
    try_dma();
  }
  c.kb = kbr;
  c.ntiles = cdiv(N, 32 * c.ntiles_per_wg);
  // Split D when there are too few sample tiles to give every CU a workgroup,
  // down to slices of 4 units (one per wave): with one sample tile, 64 slices
  // ran bf16 N = 32 at the activity shape in 35 us against 46 us with 16.
  const int64_t units = cdiv(D, 64);
  const int cus = num_cus();
  int ds = 1;
  while (c.ntiles * ds < cus && ds < kMaxSlices && units / (ds * 2) >= kWaves / 2) ds *= 2;
  c.ds = ds;
  c.ok = true;
  return c;
}

// Lets a kernel use kLdsBytes of dynamic LDS on the current device (set once
// per device and kernel).
template <auto Kernel>
hipError_t allow_large_lds() {
  static PerDeviceOnce once;  // one per kernel: the template argument is its address
  return once_per_device(once, [] {
    return hipFuncSetAttribute(reinterpret_cast<const void*>(Kernel),
                               hipFuncAttributeMaxDynamicSharedMemorySize, kLdsBytes);
  });
}

template <class Tr, int NTILES, int KB, int ACT, int PF>
hipError_t launch_fused(const LargeCfg& c, const void* X, const uint4* Bp, const uint4* Cp,
                        int32_t* labels, float* scores, int64_t N, int64_t F, int64_t K, int ndb,
                        void* ws, hipStream_t stream) {
  const dim3 grid((unsigned)(c.ntiles * c.ds)), block(kThreads);
  const hipError_t attr = allow_large_lds<&large_fused_kernel<Tr, NTILES, KB, ACT, PF>>();
  if (attr != hipSuccess) return attr;
  hipLaunchKernelGGL((large_fused_kernel<Tr, NTILES, KB, ACT, PF>), grid, block, c.lds, stream,
                     (const typename Tr::elem*)X, Bp, Cp, labels, scores, (int)N, (int)F, (int)K,
                     ndb, c.ds, ws);
  return hipGetLastError();
}

template <class Tr, int NTILES, int KB, int ACT>
hipError_t launch_act(const LargeCfg& c, const void* X, const uint4* Bp, const uint4* Cp,
                      int32_t* labels, float* scores, int64_t N, int64_t F, int64_t K, int ndb,
                      void* ws, hipStream_t stream) {
  const dim3 grid((unsigned)(c.ntiles * c.ds)), block(kThreads);
  if (c.fsc > 0) {
    if (c.dma) {
      if constexpr (Tr::kEsz <= 2 && NTILES == kDmaNtiles) {
        const hipError_t dattr =
            allow_large_lds<&large_chunked_dma_kernel<Tr, NTILES, KB, ACT>>();
        if (dattr != hipSuccess) return dattr;
        hipLaunchKernelGGL((large_chunked_dma_kernel<Tr, NTILES, KB, ACT>), grid, block, c.lds,
                           stream, (const typename Tr::elem*)X, Bp, Cp, labels, scores, (int)N,
                           (int)F, (int)K, ndb, c.ds, ws);
        return hipGetLastError();
      }
      return hipErrorInvalidValue;
    }
    if constexpr (NTILES == chunk_ntiles<Tr>(KB)) {
      const hipError_t cattr = allow_large_lds<&large_chunked_kernel<Tr, NTILES, KB, ACT>>();
      if (cattr != hipSuccess) return cattr;
      hipLaunchKernelGGL((large_chunked_kernel<Tr, NTILES, KB, ACT>), grid, block, c.lds, stream,
                         (const typename Tr::elem*)X, Bp, Cp, labels, scores, (int)N, (int)F,
                         (int)K, ndb, c.ds, c.fsc, ws);
      return hipGetLastError();
    }
    return hipErrorInvalidValue;
  }
  constexpr int kPF = prefetch_of(NTILES, KB);
  if constexpr (kPF == 8 && ACT == 0 && Tr::kEsz == 1) {
    if (fused_prefetch(nfs_of<Tr>((int)F)) == 10)
      return launch_fused<Tr, NTILES, KB, ACT, 10>(c, X, Bp, Cp, labels, scores, N, F, K, ndb,
                                                   ws, stream);
  }
  return launch_fused<Tr, NTILES, KB, ACT, kPF>(c, X, Bp, Cp, labels, scores, N, F, K, ndb, ws,
                                                stream);
}

template <class Tr, int NTILES, int KB>
hipError_t launch_cfg(const LargeCfg& c, const void* X, const uint4* Bp, const uint4* Cp,
                      int32_t* labels, float* scores, int64_t N, int64_t F, int64_t K, int ndb,
                      int act, void* ws, hipStream_t stream) {
  if (act)
    return launch_act<Tr, NTILES, KB, 1>(c, X, Bp, Cp, labels, scores, N, F, K, ndb, ws, stream);
  return launch_act<Tr, NTILES, KB, 0>(c, X, Bp, Cp, labels, scores, N, F, K, ndb, ws, stream);
}

template <class Tr>
hipError_t launch_tr(const void* X, const void* packed, int32_t* labels, float* scores,
                     int64_t N, int64_t F, int64_t D, int64_t K, int act, void* ws,
                     hipStream_t stream) {
  const LargeCfg c = large_cfg<Tr>(N, F, D, K, ((uintptr_t)X % 16) == 0);
  if (!c.ok) return hipErrorInvalidValue;
  const PackGeom g = pack_geom<Tr>(F, D, K);
  const uint4* Bp = (const uint4*)packed;
  const uint4* Cp = (const uint4*)((const char*)packed + g.b_bytes);
  const int nt = c.ntiles_per_wg, kb = c.kb;
#define HD_LAUNCH(NTV, KBV)                                                                       \
  if (nt == NTV && kb == KBV)                                                                     \
    return launch_cfg<Tr, NTV, KBV>(c, X, Bp, Cp, labels, scores, N, F, K, g.ndb, act, ws, stream);
  HD_LAUNCH(4, 1)
  HD_LAUNCH(4, 2)
  HD_LAUNCH(2, 1)
  HD_LAUNCH(2, 2)
  HD_LAUNCH(2, 4)
  HD_LAUNCH(1, 1)
  HD_LAUNCH(1, 2)
  HD_LAUNCH(1, 4)
#undef HD_LAUNCH
  return hipErrorInvalidValue;
}

// Training plan: NTILES sample tiles of 32 per workgroup, f-steps per X
// chunk, workgroups per compute unit (from LDS and registers), and the
// number of sample-tile groups.
struct BundleCfg {
  int nt, occ, fsc, ngroups, ncg;
  int dma_upw;  // > 0: the double-buffered bf16 kernel with this many units per wave
  size_t lds;
  bool ok;
};

template <class Tr>
BundleCfg bundle_cfg(int64_t N, int64_t F, int64_t D, int64_t K, bool x16 = true) {
  BundleCfg c{};
  if (K < 1 || K > kBundleMfmaMaxK || F > (1 << 20) || N > (1 << 30) || N < 1) return c;
  if (Tr::kEsz == 1 && F > kI8MaxF) return c;
  if (cdiv(D, 64) * 2 * nfs_of<Tr>((int)F) * 1024 >= ((int64_t)1 << 31)) return c;
  if (Tr::kEsz <= 2 && F % Tr::kVec == 0 && x16) {
    // double-buffered kernel: two units per wave while the class counters fit
    const size_t base = (size_t)2 * dma_loads_per_wave(kDmaNtiles) * kThreads * 16 + 16 +
                        sizeof(int) * 2 * 32 * kDmaNtiles;
    for (int upw : {2, 1}) {
      const size_t need = base + sizeof(int) * (size_t)K * kWaves * upw * 64;
      if (need <= (size_t)kLdsBytes) {
        c.dma_upw = upw;
        c.nt = kDmaNtiles;
        c.occ = 1;
        c.fsc = kDmaFsc;
        c.lds = need;
        c.ncg = (int)cdiv(cdiv(D, 64), kWaves * upw);
        const int64_t ntiles = cdiv(N, 32 * c.nt);
        int64_t g = (int64_t)num_cus() / c.ncg;
        if (g < 1) g = 1;
        if (g > ntiles) g = ntiles;
        c.ngroups = (int)g;
        c.ok = true;
        return c;
      }
    }
  }
  c.nt = Tr::kEsz == 1 ? 4 : 2;
  c.occ = Tr::kEsz == 1 ? 1 : 2;
  const int nfs = nfs_of<Tr>((int)F);
  const int pad = pad_of<Tr>();
  const size_t fixed = 16 + sizeof(int) * (32 * c.nt + (size_t)K * kBundleCols);
  const size_t per_row = (size_t)32 * c.nt * Tr::kEsz;  // bytes per LDS column of the tile
  // Two workgroups per compute unit (fp32) while the class counters leave
  // room for a chunk of at least 4 f-steps in half the LDS, else one.
  if (c.occ > 1 && fixed + per_row * (4 * Tr::kFStep + pad) > (size_t)kLdsBytes / c.occ) c.occ = 1;
  const size_t budget = (size_t)kLdsBytes / c.occ;
  if (fixed + per_row * (Tr::kFStep + pad) > budget) return c;
  int64_t fsc = (int64_t)((budget - fixed) / per_row - pad) / Tr::kFStep;
  if (fsc > nfs) fsc = nfs;
  if (fsc < 1) return c;
  c.fsc = (int)fsc;
  c.lds = fixed + per_row * (c.fsc * Tr::kFStep + pad);
  c.ncg = (int)cdiv(cdiv(D, 64), kWaves);
  const int64_t ntiles = cdiv(N, 32 * c.nt);
  int64_t g = (int64_t)num_cus() * c.occ / c.ncg;
  if (g < 1) g = 1;
  if (g > ntiles) g = ntiles;
  c.ngroups = (int)g;
  c.ok = true;
  return c;
}

template <class Tr>
hipError_t launch_bundle_dma(const BundleCfg& c, const void* X, const void* packed,
                             const int32_t* y, int32_t* counts, int64_t N, int64_t F, int64_t D,
                             int64_t K, int ndb, hipStream_t stream) {
  typedef typename Tr::elem T;
  const dim3 grid((unsigned)(c.ncg * c.ngroups)), block(kThreads);
  if (c.dma_upw == 2) {
    const hipError_t a = allow_large_lds<&bundle_dma_kernel<Tr, 2>>();
    if (a != hipSuccess) return a;
    hipLaunchKernelGGL((bundle_dma_kernel<Tr, 2>), grid, block, c.lds, stream, (const T*)X,
                       (const uint4*)packed, y, counts, (int)N, (int)F, (int)D, (int)K, ndb,
                       c.ngroups);
  } else {
    const hipError_t a = allow_large_lds<&bundle_dma_kernel<Tr, 1>>();
    if (a != hipSuccess) return a;
    hipLaunchKernelGGL((bundle_dma_kernel<Tr, 1>), grid, block, c.lds, stream, (const T*)X,
                       (const uint4*)packed, y, counts, (int)N, (int)F, (int)D, (int)K, ndb,
                       c.ngroups);
  }
  return hipGetLastError();
}

}  // namespace

bool bundle_packed_supported(int64_t N, int64_t F, int64_t D, int64_t K, int dt) {
  return with_traits(dt, [&](auto tr) { return bundle_cfg<decltype(tr)>(N, F, D, K).ok; });
}

const char* bundle_packed_kernel_name(int64_t N, int64_t F, int64_t D, int64_t K, int dt) {
  if (dt == 0) return bundle_cfg<TrF32>(N, F, D, K).ok ? "bundle_mfma_kernel" : "";
  if (dt == 2) {
    const BundleCfg c = bundle_cfg<TrI8>(N, F, D, K);
    if (!c.ok) return "";
    return c.dma_upw > 0 ? "bundle_dma_kernel" : "bundle_mfma_kernel";
  }
  const BundleCfg c = bundle_cfg<TrBF16>(N, F, D, K);
  if (!c.ok) return "";
  return c.dma_upw > 0 ? "bundle_dma_kernel" : "bundle_mfma_kernel";
}

hipError_t launch_bundle_packed(const void* X, const void* packed, const int32_t* y,
                                int32_t* counts, int64_t N, int64_t F, int64_t D, int64_t K,
                                int dt, hipStream_t stream) {
  const dim3 block(kThreads);
  if (dt == 0) {
    const BundleCfg c = bundle_cfg<TrF32>(N, F, D, K);
    if (!c.ok) return hipErrorInvalidValue;
    const PackGeom g = pack_geom<TrF32>(F, D, 1);
    auto* k = &bundle_mfma_kernel<TrF32, 2, 2>;
    const hipError_t a = allow_large_lds<&bundle_mfma_kernel<TrF32, 2, 2>>();
    if (a != hipSuccess) return a;
    hipLaunchKernelGGL(k, dim3((unsigned)(c.ncg * c.ngroups)), block, c.lds, stream,
                       (const float*)X, (const uint4*)packed, y, counts, (int)N, (int)F, (int)D,
                       (int)K, g.ndb, c.ngroups, c.fsc);
  } else if (dt == 2) {
    const BundleCfg c = bundle_cfg<TrI8>(N, F, D, K, ((uintptr_t)X % 16) == 0);
    if (!c.ok) return hipErrorInvalidValue;
    const PackGeom g = pack_geom<TrI8>(F, D, 1);
    if (c.dma_upw > 0)
      return launch_bundle_dma<TrI8>(c, X, packed, y, counts, N, F, D, K, g.ndb, stream);
    auto* k = &bundle_mfma_kernel<TrI8, 4, 1>;
    const hipError_t a = allow_large_lds<&bundle_mfma_kernel<TrI8, 4, 1>>();
    if (a != hipSuccess) return a;
    hipLaunchKernelGGL(k, dim3((unsigned)(c.ncg * c.ngroups)), block, c.lds, stream,
                       (const int8_t*)X, (const uint4*)packed, y, counts, (int)N, (int)F,
                       (int)D, (int)K, g.ndb, c.ngroups, c.fsc);
  } else {
    const BundleCfg c = bundle_cfg<TrBF16>(N, F, D, K, ((uintptr_t)X % 16) == 0);
    if (!c.ok) return hipErrorInvalidValue;
    const PackGeom g = pack_geom<TrBF16>(F, D, 1);
    if (c.dma_upw > 0)
      return launch_bundle_dma<TrBF16>(c, X, packed, y, counts, N, F, D, K, g.ndb, stream);
    auto* k = &bundle_mfma_kernel<TrBF16, 2, 2>;
    const hipError_t a = allow_large_lds<&bundle_mfma_kernel<TrBF16, 2, 2>>();
    if (a != hipSuccess) return a;
    hipLaunchKernelGGL(k, dim3((unsigned)(c.ncg * c.ngroups)), block, c.lds, stream,
                       (const bf16raw*)X, (const uint4*)packed, y, counts, (int)N, (int)F,
                       (int)D, (int)K, g.ndb, c.ngroups, c.fsc);
  }
  return hipGetLastError();
}

bool large_supported(int64_t N, int64_t F, int64_t D, int64_t K, int dt) {
  return with_traits(dt, [&](auto tr) { return large_cfg<decltype(tr)>(N, F, D, K).ok; });
}

const char* large_kernel_name(int64_t N, int64_t F, int64_t D, int64_t K, int dt) {
  const LargeCfg c =
      with_traits(dt, [&](auto tr) { return large_cfg<decltype(tr)>(N, F, D, K); });
  if (!c.ok) return "";
  if (c.fsc > 0) return c.dma ? "large_chunked_dma_kernel" : "large_chunked_kernel";
  return "large_fused_kernel";
}

size_t large_packed_bytes(int64_t F, int64_t D, int64_t K, int dt) {
  const PackGeom g = with_traits(dt, [&](auto tr) { return pack_geom<decltype(tr)>(F, D, K); });
  return g.b_bytes + g.c_bytes;
}

size_t large_workspace_bytes_for(int64_t N, int64_t F, int64_t D, int64_t K, int dt,
                                 bool x16) {
  const LargeCfg c =
      with_traits(dt, [&](auto tr) { return large_cfg<decltype(tr)>(N, F, D, K, x16); });
  if (!c.ok || c.ds == 1) return 0;
  const size_t cbytes = ((size_t)c.ntiles * sizeof(unsigned) + 255) / 256 * 256;
  return cbytes + sizeof(float) * (size_t)c.ds * N * K;
}

// The plan (tile size, D slices) depends on whether X is 16-byte aligned, which
// the size query does not know: size for the larger of the two plans.
size_t large_workspace_bytes(int64_t N, int64_t F, int64_t D, int64_t K, int dt) {
  const size_t a = large_workspace_bytes_for(N, F, D, K, dt, true);
  const size_t b = large_workspace_bytes_for(N, F, D, K, dt, false);
  return a > b ? a : b;
}

hipError_t launch_pack(const void* B, const void* C, int64_t F, int64_t D, int64_t K, int dt,
                       void* packed, hipStream_t stream) {
  if (dt == 0) {
    const PackGeom g = pack_geom<TrF32>(F, D, K);
    uint4* Bp = (uint4*)packed;
    uint4* Cp = (uint4*)((char*)packed + g.b_bytes);
    hipLaunchKernelGGL(pack_b_f32, dim3((unsigned)((int64_t)g.ndb * g.nfs)), dim3(64), 0, stream,
                       (const float*)B, Bp, (int)F, (int)D, g.ndb, g.nfs);
    hipLaunchKernelGGL(pack_c_f32, dim3((unsigned)((int64_t)g.ndb * g.kb * 4)), dim3(64), 0,
                       stream, (const float*)C, Cp, (int)D, C ? (int)K : 0, g.ndb, g.kb);
  } else if (dt == 2) {
    const PackGeom g = pack_geom<TrI8>(F, D, K);
    uint4* Bp = (uint4*)packed;
    uint4* Cp = (uint4*)((char*)packed + g.b_bytes);
    hipLaunchKernelGGL(pack_b_i8, dim3((unsigned)((int64_t)g.ndb * g.nfs)), dim3(64), 0, stream,
                       (const int8_t*)B, Bp, (int)F, (int)D, g.ndb, g.nfs);
    hipLaunchKernelGGL(pack_c_i8, dim3((unsigned)((int64_t)g.ndb * 2 * g.kb)), dim3(64), 0,
                       stream, (const int8_t*)C, Cp, (int)D, C ? (int)K : 0, g.ndb, g.kb);
  } else {
    const PackGeom g = pack_geom<TrBF16>(F, D, K);
    uint4* Bp = (uint4*)packed;
    uint4* Cp = (uint4*)((char*)packed + g.b_bytes);
    hipLaunchKernelGGL(pack_b_bf16, dim3((unsigned)((int64_t)g.ndb * g.nfs)), dim3(64), 0,
                       stream, (const bf16raw*)B, Bp, (int)F, (int)D, g.ndb, g.nfs);
    hipLaunchKernelGGL(pack_c_bf16, dim3((unsigned)((int64_t)g.ndb * 2 * g.kb)), dim3(64), 0,
                       stream, (const bf16raw*)C, Cp, (int)D, C ? (int)K : 0, g.ndb, g.kb);
  }
  return hipGetLastError();
}

hipError_t launch_large(const void* X, const void* packed, int32_t* labels, float* scores,
                        int64_t N, int64_t F, int64_t D, int64_t K, int dt, int act,
                        void* workspace, hipStream_t stream) {
  if (dt == 0)
    return launch_tr<TrF32>(X, packed, labels, scores, N, F, D, K, act, workspace, stream);
  if (dt == 2)
    return launch_tr<TrI8>(X, packed, labels, scores, N, F, D, K, act, workspace, stream);
  return launch_tr<TrBF16>(X, packed, labels, scores, N, F, D, K, act, workspace, stream);
}

}  // namespace hd
