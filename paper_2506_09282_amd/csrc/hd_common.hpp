// Internal device helpers shared by the HDC inference kernels (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hd {

typedef uint16_t bf16raw;  // raw bfloat16 bit pattern
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef int i32x16 __attribute__((ext_vector_type(16)));
typedef short i16x8 __attribute__((ext_vector_type(8)));

constexpr int kWave = 64;

__device__ __forceinline__ float bf16_to_f32(uint32_t bits16) {
  return __uint_as_float(bits16 << 16);
}

// Element loads widened to fp32 (exact for every storage type).
__device__ __forceinline__ float load_elem(const float* p, int64_t i) { return p[i]; }
__device__ __forceinline__ float load_elem(const bf16raw* p, int64_t i) {
  return bf16_to_f32(p[i]);
}
__device__ __forceinline__ float load_elem(const int8_t* p, int64_t i) { return (float)p[i]; }

// Four consecutive elements starting at p[i]; i must be a multiple of 4 and
// the base 16-byte (fp32) / 8-byte (bf16) aligned.
__device__ __forceinline__ float4 load4(const float* p, int64_t i) {
  return *reinterpret_cast<const float4*>(p + i);
}
__device__ __forceinline__ float4 load4(const bf16raw* p, int64_t i) {
  const uint2 u = *reinterpret_cast<const uint2*>(p + i);
  return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u),
                     __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xffff0000u));
}

// Eq. 1 of the paper: +1 for v >= 0 (so -0.0 gives +1), -1 otherwise
// (NaN compares false and gives -1). A literal comparison, not a sign-bit test.
__device__ __forceinline__ float hardsign(float v) { return v >= 0.0f ? 1.0f : -1.0f; }

__device__ __forceinline__ float activate(float v, int act) { return act ? v : hardsign(v); }

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, kWave);
  return v;
}

// Cross-workgroup hand-off without cache write-back.
//
// Data that one workgroup passes to another moves only through device-scope
// atomic read-modify-writes, which are performed at a single coherence point
// for each address. A workgroup publishes with no-return atomics, waits until
// they are performed (s_waitcnt, all counters to zero) and only then takes a
// ticket with a relaxed device-scope fetch-add; the workgroup that draws the
// last ticket reads every published value with an atomic exchange against 0,
// which both observes all performed atomics and leaves the slot zeroed for
// the next call. A device-scope release fence would also work, but on gfx950
// it writes back the whole L2 (buffer_wbl2) in every workgroup, which costs
// tens of microseconds per launch.
__device__ __forceinline__ void wait_own_memory_ops() { __builtin_amdgcn_s_waitcnt(0); }
__device__ __forceinline__ unsigned take_ticket(unsigned* counter) {
  return __hip_atomic_fetch_add(counter, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float take_and_clear(float* p) {
  return __hip_atomic_exchange(p, 0.0f, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void publish_add(float* p, float v) {
  unsafeAtomicAdd(p, v);  // native no-return fp32 atomic add (device memory)
}
__device__ __forceinline__ void publish_store(float* p, float v) {
  // an exchange (not a plain store) so the value lands where atomics are performed
  (void)__hip_atomic_exchange(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void reset_counter(unsigned* counter) {
  (void)__hip_atomic_exchange(counter, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__host__ __device__ constexpr int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

}  // namespace hd
