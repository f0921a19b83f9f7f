// Host-side declarations shared between the C-ABI layer and the launchers.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <mutex>

namespace hd {

// Launch settings the library takes once per device (kernel attributes, the
// compute-unit count). They are kept per device id, because a process may
// drive several GPUs and each call uses whichever device is current; apart
// from these write-once values the library holds no state between calls.
constexpr int kMaxDevices = 64;

struct PerDeviceOnce {
  std::once_flag flag[kMaxDevices];
  hipError_t err[kMaxDevices] = {};
};

// Runs f() once for the current device and returns its (remembered) result.
template <class Fn>
hipError_t once_per_device(PerDeviceOnce& o, Fn&& f) {
  int dev = 0;
  const hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return f();
  std::call_once(o.flag[dev], [&] { o.err[dev] = f(); });
  return o.err[dev];
}

// Compute units of the current device (256 on MI355X), read once per device.
int num_cus();

// Small-batch fused path (split-D across workgroups).
constexpr int kSmallMaxN = 64;
constexpr int kSmallReplicas = 32;  // replicated score accumulators

bool small_supported(int64_t N, int64_t F, int64_t D, int64_t K, int dt);
// `act` of launch_small: bit 0 the activation, bit 1 the deterministic reduction.
constexpr int kSmallActDet = 2;
// Workspace of the small-batch kernels; det: the deterministic reduction (one
// score replica per workgroup plus one per ticket group).
size_t small_workspace_bytes(int64_t N, int64_t F, int64_t D, int64_t K, int dt, bool det);
// Name of the kernel launch_small would use for 16-byte aligned operands.
// Whether the small-batch plan for these sizes (16-byte aligned operands)
// runs on the matrix cores rather than the VALU fallback.
bool small_matrix_core(int64_t N, int64_t F, int64_t D, int64_t K, int dt, bool tiled);
const char* small_kernel_name(int64_t N, int64_t F, int64_t D, int64_t K, int dt, bool tiled);

// Bytes of the column-tiled model section the small-batch path reads from a
// packed model, and the kernel that writes it.
size_t small_packed_bytes(int64_t F, int64_t D, int64_t K, int dt);
hipError_t launch_pack_small(const void* B, const void* C, int64_t F, int64_t D, int64_t K, int dt,
                             void* out, hipStream_t stream);
// tiled: B points at that section (C is then ignored); otherwise B and C are
// the caller's row-major matrices.
hipError_t launch_small(const void* X, const void* B, const void* C, bool tiled, int32_t* labels,
                        float* scores, int64_t N, int64_t F, int64_t D, int64_t K, int dt,
                        int act, void* workspace, hipStream_t stream);

// Zero-fill of a device range (a kernel, not hipMemsetAsync, so that callers
// may capture it in a graph).
hipError_t launch_zero(void* p, size_t bytes, hipStream_t stream);

// Streaming inference: nbatch batches of N samples against a packed fp32
// model whose share of B stays in registers (packed_small points at the
// packed image's small-batch section).
bool stream_supported(int64_t N, int64_t F, int64_t D, int64_t K, int dt);
size_t stream_ws_bytes(int64_t nbatch, int64_t N, int64_t K);
hipError_t launch_stream(const void* X, const void* packed_small, const unsigned* ready,
                         int32_t* labels, float* scores, unsigned* done, int64_t nbatch,
                         int64_t N, int64_t F, int64_t D, int64_t K, int act, void* workspace,
                         hipStream_t stream);

// Single-pass training (class sums of HardSign(X B), then their HardSign).
constexpr int64_t kBundleMaxK = 512;
bool bundle_supported(int64_t K);
hipError_t launch_bundle(const void* X, const void* B, const int32_t* y, int32_t* counts,
                         int64_t N, int64_t F, int64_t D, int64_t K, int dt, hipStream_t stream);
hipError_t launch_class_hardsign(const int32_t* counts, float* M, int64_t K, int64_t D,
                                 hipStream_t stream);
// The same class sums on the matrix cores, from the tiled B of a packed model
// (the large-batch section at the start of the image).
constexpr int64_t kBundleMfmaMaxK = 128;
bool bundle_packed_supported(int64_t N, int64_t F, int64_t D, int64_t K, int dt);
// Name of the kernel launch_bundle_packed uses for 16-byte aligned X ("" if unsupported).
const char* bundle_packed_kernel_name(int64_t N, int64_t F, int64_t D, int64_t K, int dt);
hipError_t launch_bundle_packed(const void* X, const void* packed, const int32_t* y,
                                int32_t* counts, int64_t N, int64_t F, int64_t D, int64_t K,
                                int dt, hipStream_t stream);

// Unfused stages.
hipError_t launch_encode(const void* X, const void* B, float* H, int64_t N, int64_t F, int64_t D,
                         int dt, int act, hipStream_t stream);
hipError_t launch_similarity(const float* H, const void* C, int32_t* labels, float* scores,
                             int64_t N, int64_t D, int64_t K, int c_dt, hipStream_t stream);

// Large-batch fused path (MFMA, packed model).
bool large_supported(int64_t N, int64_t F, int64_t D, int64_t K, int dt);
// Name of the kernel launch_large uses for these sizes ("" if unsupported).
const char* large_kernel_name(int64_t N, int64_t F, int64_t D, int64_t K, int dt);
size_t large_packed_bytes(int64_t F, int64_t D, int64_t K, int dt);
// Workspace of the large-batch kernels: for the plan taken with X 16-byte
// aligned (x16) or not, and the larger of the two (what the size query gives).
size_t large_workspace_bytes_for(int64_t N, int64_t F, int64_t D, int64_t K, int dt, bool x16);
size_t large_workspace_bytes(int64_t N, int64_t F, int64_t D, int64_t K, int dt);
hipError_t launch_pack(const void* B, const void* C, int64_t F, int64_t D, int64_t K, int dt,
                       void* packed, hipStream_t stream);
hipError_t launch_large(const void* X, const void* packed, int32_t* labels, float* scores,
                        int64_t N, int64_t F, int64_t D, int64_t K, int dt, int act,
                        void* workspace, hipStream_t stream);

}  // namespace hd
