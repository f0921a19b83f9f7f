// Host-side declarations shared between the C-ABI layer and the launchers.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace hd {

// Small-batch fused path (split-D across workgroups).
constexpr int kSmallMaxN = 64;
constexpr int kSmallReplicas = 32;  // replicated score accumulators

bool small_supported(int64_t N, int64_t F, int64_t D, int64_t K, int dt);
size_t small_workspace_bytes(int64_t N, int64_t F, int64_t D, int64_t K, int dt);
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
size_t large_workspace_bytes(int64_t N, int64_t F, int64_t D, int64_t K, int dt);
hipError_t launch_pack(const void* B, const void* C, int64_t F, int64_t D, int64_t K, int dt,
                       void* packed, hipStream_t stream);
hipError_t launch_large(const void* X, const void* packed, int32_t* labels, float* scores,
                        int64_t N, int64_t F, int64_t D, int64_t K, int dt, int act,
                        void* workspace, hipStream_t stream);

}  // namespace hd
