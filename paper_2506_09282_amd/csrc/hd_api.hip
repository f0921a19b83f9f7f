// C ABI entry points: argument validation on the host (before anything is
// enqueued), path selection, and kernel launch on the caller's stream.
#include <atomic>

#include "../../include/hd.h"
#include "hd_internal.hpp"

namespace {

constexpr int64_t kMaxDim = int64_t(1) << 30;

bool dims_ok(int64_t N, int64_t F, int64_t D, int64_t K) {
  return N <= kMaxDim && F <= kMaxDim && D <= kMaxDim && K <= kMaxDim;
}

bool enums_ok(int dt, int act) {
  return (dt == HD_F32 || dt == HD_BF16 || dt == HD_I8) && (act == 0 || act == 1);
}

// The int8 model variant runs on the large-batch matrix-core kernels only,
// with the HardSign activation.
bool i8_ok(int dt, int act) { return dt != HD_I8 || act == 0; }

// The act argument of the inference calls: an hd_act, optionally OR-ed with
// HD_DETERMINISTIC.
int act_base(int act) { return act & ~HD_DETERMINISTIC; }
bool det_of(int act) { return (act & HD_DETERMINISTIC) != 0; }

size_t align256(size_t x) { return (x + 255) / 256 * 256; }

// Path choice. The split-D small-batch path serves small batches whenever its
// scratch fits, everything else the batch-split matrix-core path, with these
// exceptions taken from the measured samples/s curves (F = 561, D = 10240):
// * bf16 above 8 samples with B as given: the small-batch VALU kernel makes
//   several passes over B (40 us at N = 16, 72 us at N = 32), the matrix-core
//   path takes 34 us at N = 16..32; a packed bf16 model carries bf16
//   fragments and takes the fragment kernel (9-11 us for N = 16..64);
// * int8 runs on the fragment kernel only with a packed model (8-10 us for
//   N <= 64), else on the matrix-core path;
// * 64 < N <= 256 in fp32 and on a packed bf16 or int8 model: the
//   matrix-core path has only a few sample tiles (fp32: 138 us for
//   N = 65..256; bf16: 39-47 us; int8: 33-39 us), while the small path takes
//   18 us (fp32) or about 10 us (bf16, int8) per 64 samples, so it runs in
//   64-sample chunks, one after another on the stream, when its 64-sample
//   plan runs on the matrix cores (not the VALU fallback).
enum class Route { kSmall, kSmallChunked, kLarge, kNone };
constexpr int64_t kSmallMaxNBf16 = 8;
constexpr int64_t kChunkedMaxN = 256;

Route route(int64_t N, int64_t F, int64_t D, int64_t K, int dt, bool tiled) {
  if (dt == HD_I8) {
    // int8 on a packed model: the fragment kernel for small batches (it takes
    // 16-byte aligned X; others fall back to the large-batch kernels, which
    // the workspace query covers as well). The large-batch bounds on F and D
    // keep every sum exact, on either path.
    if (!hd::large_supported(N, F, D, K, dt)) return Route::kNone;
    if (tiled && N <= hd::kSmallMaxN && hd::small_supported(N, F, D, K, dt)) return Route::kSmall;
    if (tiled && N > hd::kSmallMaxN && N <= kChunkedMaxN &&
        hd::small_supported(hd::kSmallMaxN, F, D, K, dt))
      return Route::kSmallChunked;
    return Route::kLarge;
  }
  const bool small_ok = N <= hd::kSmallMaxN && hd::small_supported(N, F, D, K, dt);
  if (small_ok && (dt == HD_F32 || N <= kSmallMaxNBf16)) return Route::kSmall;
  // a packed bf16 model carries bf16 fragments: the fragment kernel serves it
  if (small_ok && dt == HD_BF16 && tiled && hd::small_matrix_core(N, F, D, K, dt, tiled))
    return Route::kSmall;
  if (dt == HD_F32 && N > hd::kSmallMaxN && N <= kChunkedMaxN &&
      hd::small_matrix_core(hd::kSmallMaxN, F, D, K, dt, tiled))
    return Route::kSmallChunked;
  if (dt == HD_BF16 && tiled && N > hd::kSmallMaxN && N <= kChunkedMaxN &&
      hd::small_matrix_core(hd::kSmallMaxN, F, D, K, dt, tiled))
    return Route::kSmallChunked;
  if (hd::large_supported(N, F, D, K, dt)) return Route::kLarge;
  return small_ok ? Route::kSmall : Route::kNone;
}

// Batch size of each small-path launch for a route.
int64_t small_n(Route r, int64_t N) { return r == Route::kSmallChunked ? hd::kSmallMaxN : N; }

hd_status from_hip(hipError_t e) { return e == hipSuccess ? HD_OK : HD_ERR_HIP; }

size_t esize(int dt) { return dt == HD_F32 ? 4 : dt == HD_I8 ? 1 : 2; }

// Packed model image: [fragment-tiled B and C for the matrix-core path |
// column-tiled B and C for the small-batch path]. Both sections start on a
// 256-byte boundary of the (256-byte aligned) image.
struct Image {
  size_t large, small, total;
};

Image image_layout(int64_t F, int64_t D, int64_t K, int dt) {
  Image im;
  im.large = align256(hd::large_packed_bytes(F, D, K, dt));
  im.small = align256(hd::small_packed_bytes(F, D, K, dt));
  im.total = im.large + im.small;
  return im;
}

// Every element pointer must be aligned to its element size; packed images
// and workspaces to 256 bytes (what hipMalloc returns).
bool aligned(const void* p, size_t a) { return (uintptr_t)p % a == 0; }

}  // namespace

namespace hd {

int num_cus() {
  static std::atomic<int> cus[kMaxDevices];  // 0 until read for that device
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 256;
  const bool cached = dev >= 0 && dev < kMaxDevices;
  if (cached) {
    const int v = cus[dev].load(std::memory_order_relaxed);
    if (v > 0) return v;
  }
  int v = 0;
  if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      v <= 0)
    v = 256;
  if (cached) cus[dev].store(v, std::memory_order_relaxed);
  return v;
}

}  // namespace hd

extern "C" {

const char* hd_status_str(hd_status s) {
  switch (s) {
    case HD_OK:
      return "HD_OK";
    case HD_ERR_ARG:
      return "HD_ERR_ARG: invalid argument";
    case HD_ERR_UNSUPPORTED:
      return "HD_ERR_UNSUPPORTED: size or type combination not supported";
    case HD_ERR_WORKSPACE:
      return "HD_ERR_WORKSPACE: workspace or packed buffer too small";
    case HD_ERR_HIP:
      return "HD_ERR_HIP: HIP launch failed";
  }
  return "HD_ERR_UNKNOWN";
}

hd_status hd_encode(const void* X, const void* B, float* H, int64_t N, int64_t F, int64_t D,
                    hd_dtype dt, hd_act act, hipStream_t stream) {
  if (N < 0 || F < 1 || D < 1 || !enums_ok(dt, act)) return HD_ERR_ARG;
  if (!dims_ok(N, F, D, 1) || dt == HD_I8) return HD_ERR_UNSUPPORTED;
  if (N == 0) return HD_OK;
  if (!X || !B || !H) return HD_ERR_ARG;
  if (!aligned(X, esize(dt)) || !aligned(B, esize(dt)) || !aligned(H, 4)) return HD_ERR_ARG;
  return from_hip(hd::launch_encode(X, B, H, N, F, D, dt, act, stream));
}

hd_status hd_similarity(const float* H, const void* C, int32_t* labels, float* scores, int64_t N,
                        int64_t D, int64_t K, hd_dtype c_dt, hipStream_t stream) {
  if (N < 0 || D < 1 || K < 1 || !enums_ok(c_dt, 0)) return HD_ERR_ARG;
  if (!dims_ok(N, 1, D, K) || c_dt == HD_I8) return HD_ERR_UNSUPPORTED;
  if (N == 0) return HD_OK;
  if (!H || !C || !labels) return HD_ERR_ARG;
  if (!aligned(H, 4) || !aligned(C, esize(c_dt)) || !aligned(labels, 4) || !aligned(scores, 4))
    return HD_ERR_ARG;
  return from_hip(hd::launch_similarity(H, C, labels, scores, N, D, K, c_dt, stream));
}

size_t hd_model_packed_bytes(int64_t F, int64_t D, int64_t K, hd_dtype dt) {
  if (F < 1 || D < 1 || K < 1 || !enums_ok(dt, 0) || !dims_ok(0, F, D, K)) return 0;
  return image_layout(F, D, K, dt).total;
}

// Workspace one call needs: with a packed model or raw matrices, in the
// default or the deterministic mode (the size queries cover both modes).
static size_t workspace_need(int64_t N, int64_t F, int64_t D, int64_t K, int dt, bool packed,
                             bool det) {
  const Route r = route(N, F, D, K, dt, packed);
  if ((r == Route::kSmall || r == Route::kSmallChunked) && dt == HD_I8) {
    // an unaligned X takes the large-batch kernels instead
    const size_t s = hd::small_workspace_bytes(small_n(r, N), F, D, K, dt, det);
    const size_t l = hd::large_workspace_bytes(N, F, D, K, dt);
    return s > l ? s : l;
  }
  if (r == Route::kSmall || r == Route::kSmallChunked)
    return hd::small_workspace_bytes(small_n(r, N), F, D, K, dt, det);
  if (packed) return hd::large_workspace_bytes(N, F, D, K, dt);
  return align256(hd::large_workspace_bytes(N, F, D, K, dt)) +
         align256(hd::large_packed_bytes(F, D, K, dt));
}

static size_t workspace_query(int64_t N, int64_t F, int64_t D, int64_t K, int dt, bool packed) {
  if (N < 1 || F < 1 || D < 1 || K < 1 || !enums_ok(dt, 0) || !dims_ok(N, F, D, K)) return 0;
  const size_t a = workspace_need(N, F, D, K, dt, packed, false);
  const size_t b = workspace_need(N, F, D, K, dt, packed, true);
  return a > b ? a : b;
}

size_t hd_infer_packed_workspace_bytes(int64_t N, int64_t F, int64_t D, int64_t K, hd_dtype dt) {
  return workspace_query(N, F, D, K, dt, true);
}

size_t hd_infer_workspace_bytes(int64_t N, int64_t F, int64_t D, int64_t K, hd_dtype dt) {
  return workspace_query(N, F, D, K, dt, false);
}

hd_status hd_pack_model(const void* B, const void* C, int64_t F, int64_t D, int64_t K, hd_dtype dt,
                        void* packed, size_t packed_bytes, hipStream_t stream) {
  if (F < 1 || D < 1 || K < 1 || !enums_ok(dt, 0)) return HD_ERR_ARG;
  if (!dims_ok(0, F, D, K)) return HD_ERR_UNSUPPORTED;
  if (!B || !packed) return HD_ERR_ARG;  // C may be NULL: a model packed for training
  if (!aligned(B, esize(dt)) || !aligned(C, esize(dt)) || !aligned(packed, 256)) return HD_ERR_ARG;
  const Image im = image_layout(F, D, K, dt);
  if (packed_bytes < im.total) return HD_ERR_WORKSPACE;
  char* p = static_cast<char*>(packed);
  if (hd::launch_pack(B, C, F, D, K, dt, p, stream) != hipSuccess) return HD_ERR_HIP;
  if (im.small > 0 && hd::launch_pack_small(B, C, F, D, K, dt, p + im.large, stream) != hipSuccess)
    return HD_ERR_HIP;
  return HD_OK;
}

// dry: run every host-side check and return the status the call would have,
// enqueueing nothing.
static hd_status infer_common(const void* X, const void* B, const void* C, const void* packed,
                              int32_t* labels, float* scores, int64_t N, int64_t F, int64_t D,
                              int64_t K, hd_dtype dt, int act, void* workspace,
                              size_t workspace_bytes, hipStream_t stream, bool dry = false) {
  if (N < 0 || F < 1 || D < 1 || K < 1 || !enums_ok(dt, act_base(act))) return HD_ERR_ARG;
  if (!dims_ok(N, F, D, K) || !i8_ok(dt, act_base(act))) return HD_ERR_UNSUPPORTED;
  if (N == 0) return HD_OK;
  if (!X || !labels || (packed ? false : (!B || !C))) return HD_ERR_ARG;
  const bool det = det_of(act);
  act = act_base(act);
  const size_t es = esize(dt);
  if (!aligned(X, es) || !aligned(labels, 4) || !aligned(scores, 4) || !aligned(workspace, 256) ||
      (packed ? !aligned(packed, 256) : (!aligned(B, es) || !aligned(C, es))))
    return HD_ERR_ARG;
  Route r = route(N, F, D, K, dt, packed != nullptr);
  if (r == Route::kNone) return HD_ERR_UNSUPPORTED;
  if ((r == Route::kSmall || r == Route::kSmallChunked) && dt == HD_I8 && (uintptr_t)X % 16 != 0)
    r = Route::kLarge;
  const size_t need = workspace_need(N, F, D, K, dt, packed != nullptr, det);
  if (need > 0 && !workspace) return HD_ERR_ARG;
  if (workspace_bytes < need) return HD_ERR_WORKSPACE;

  if (r == Route::kSmall || r == Route::kSmallChunked) {
    if (dry) return HD_OK;
    if (packed) B = static_cast<const char*>(packed) + image_layout(F, D, K, dt).large;
    const int64_t step = small_n(r, N);
    for (int64_t n0 = 0; n0 < N; n0 += step) {
      const int64_t n = N - n0 < step ? N - n0 : step;
      const hipError_t e = hd::launch_small(
          static_cast<const char*>(X) + n0 * F * (int64_t)es, B, C, packed != nullptr,
          labels + n0, scores ? scores + n0 * K : nullptr, n, F, D, K, dt,
          act | (det ? hd::kSmallActDet : 0), workspace, stream);
      if (e != hipSuccess) return HD_ERR_HIP;
    }
    return HD_OK;
  }
  // The plan taken for this X (its alignment can change the tile size and the
  // D split) must fit the workspace the caller sized with the query.
  const size_t plan_ws = hd::large_workspace_bytes_for(N, F, D, K, dt, (uintptr_t)X % 16 == 0);
  if (packed) {
    if (workspace_bytes < plan_ws) return HD_ERR_WORKSPACE;
    if (dry) return HD_OK;
    return from_hip(
        hd::launch_large(X, packed, labels, scores, N, F, D, K, dt, act, workspace, stream));
  }
  // Raw matrices: the scratch that must start at zero (tile counters, split-D
  // partial scores) stays at offset 0, the same place every route keeps it, and
  // the packed copy of B and C goes after it. The copy is cleared again once
  // the kernel has read it, so the whole workspace is zero after the call and
  // can be reused by a call of any shape.
  const size_t zone = align256(hd::large_workspace_bytes(N, F, D, K, dt));
  const size_t pb = hd::large_packed_bytes(F, D, K, dt);
  if (plan_ws > zone || workspace_bytes < zone + pb) return HD_ERR_WORKSPACE;
  if (dry) return HD_OK;
  char* copy = static_cast<char*>(workspace) + zone;
  if (hd::launch_pack(B, C, F, D, K, dt, copy, stream) != hipSuccess) return HD_ERR_HIP;
  const hipError_t e =
      hd::launch_large(X, copy, labels, scores, N, F, D, K, dt, act, workspace, stream);
  if (e != hipSuccess) return HD_ERR_HIP;
  return from_hip(hd::launch_zero(copy, pb, stream));
}

hd_status hd_infer(const void* X, const void* B, const void* C, int32_t* labels, float* scores,
                   int64_t N, int64_t F, int64_t D, int64_t K, hd_dtype dt, hd_act act,
                   void* workspace, size_t workspace_bytes, hipStream_t stream) {
  return infer_common(X, B, C, nullptr, labels, scores, N, F, D, K, dt, act, workspace,
                      workspace_bytes, stream);
}

const char* hd_infer_kernel(int64_t N, int64_t F, int64_t D, int64_t K, hd_dtype dt, int packed) {
  if (N < 1 || F < 1 || D < 1 || K < 1 || !enums_ok(dt, 0) || !dims_ok(N, F, D, K)) return "";
  const Route r = route(N, F, D, K, dt, packed != 0);
  if (r == Route::kSmall || r == Route::kSmallChunked)
    return hd::small_kernel_name(small_n(r, N), F, D, K, dt, packed != 0);
  return r == Route::kLarge ? hd::large_kernel_name(N, F, D, K, dt) : "";
}

hd_status hd_infer_packed(const void* X, const void* packed, int32_t* labels, float* scores,
                          int64_t N, int64_t F, int64_t D, int64_t K, hd_dtype dt, hd_act act,
                          void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (N > 0 && !packed) return HD_ERR_ARG;
  return infer_common(X, nullptr, nullptr, packed, labels, scores, N, F, D, K, dt, act, workspace,
                      workspace_bytes, stream);
}

size_t hd_infer_stream_workspace_bytes(int64_t nbatch, int64_t N, int64_t F, int64_t D,
                                       int64_t K, hd_dtype dt) {
  if (nbatch < 1 || N < 1 || F < 1 || D < 1 || K < 1 || !enums_ok(dt, 0) ||
      !dims_ok(N, F, D, K) || nbatch > kMaxDim)
    return 0;
  if (dt == HD_I8 || !hd::stream_supported(N, F, D, K, dt)) return 0;
  return hd::stream_ws_bytes(nbatch, N, K);
}

hd_status hd_infer_stream(const void* X, const void* packed, const uint32_t* ready,
                          int32_t* labels, float* scores, uint32_t* done, int64_t nbatch,
                          int64_t N, int64_t F, int64_t D, int64_t K, hd_dtype dt, hd_act act,
                          void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (nbatch < 0 || N < 1 || F < 1 || D < 1 || K < 1 || !enums_ok(dt, act_base(act)))
    return HD_ERR_ARG;
  if (det_of(act)) return HD_ERR_UNSUPPORTED;
  if (!dims_ok(N, F, D, K) || nbatch > kMaxDim || nbatch * N > kMaxDim)
    return HD_ERR_UNSUPPORTED;
  if (nbatch == 0) return HD_OK;
  if (!X || !packed || !labels || !workspace) return HD_ERR_ARG;
  if (!aligned(X, 4) || !aligned(packed, 256) || !aligned(labels, 4) || !aligned(scores, 4) ||
      !aligned(ready, 4) || !aligned(done, 4) || !aligned(workspace, 256))
    return HD_ERR_ARG;
  if (dt == HD_I8 || !hd::stream_supported(N, F, D, K, dt)) return HD_ERR_UNSUPPORTED;
  if (workspace_bytes < hd::stream_ws_bytes(nbatch, N, K)) return HD_ERR_WORKSPACE;
  const char* small = static_cast<const char*>(packed) + image_layout(F, D, K, dt).large;
  return from_hip(hd::launch_stream(X, small, ready, labels, scores, done, nbatch, N, F, D, K,
                                    act, workspace, stream));
}

hd_status hd_bundle_classes(const void* X, const void* B, const int32_t* y, int32_t* counts,
                            int64_t N, int64_t F, int64_t D, int64_t K, hd_dtype dt,
                            hipStream_t stream) {
  if (N < 0 || F < 1 || D < 1 || K < 1 || !enums_ok(dt, 0)) return HD_ERR_ARG;
  if (!dims_ok(N, F, D, K) || !hd::bundle_supported(K) || dt == HD_I8) return HD_ERR_UNSUPPORTED;
  if (N == 0) return HD_OK;
  if (!X || !B || !y || !counts) return HD_ERR_ARG;
  if (!aligned(X, esize(dt)) || !aligned(B, esize(dt)) || !aligned(y, 4) || !aligned(counts, 4))
    return HD_ERR_ARG;
  return from_hip(hd::launch_bundle(X, B, y, counts, N, F, D, K, dt, stream));
}

hd_status hd_bundle_classes_packed(const void* X, const void* packed, const int32_t* y,
                                   int32_t* counts, int64_t N, int64_t F, int64_t D, int64_t K,
                                   hd_dtype dt, hipStream_t stream) {
  if (N < 0 || F < 1 || D < 1 || K < 1 || !enums_ok(dt, 0)) return HD_ERR_ARG;
  if (!dims_ok(N, F, D, K)) return HD_ERR_UNSUPPORTED;
  if (N > 0 && !hd::bundle_packed_supported(N, F, D, K, dt)) return HD_ERR_UNSUPPORTED;
  if (N == 0) return HD_OK;
  if (!X || !packed || !y || !counts) return HD_ERR_ARG;
  if (!aligned(X, esize(dt)) || !aligned(packed, 256) || !aligned(y, 4) || !aligned(counts, 4))
    return HD_ERR_ARG;
  return from_hip(hd::launch_bundle_packed(X, packed, y, counts, N, F, D, K, dt, stream));
}

const char* hd_bundle_kernel(int64_t N, int64_t F, int64_t D, int64_t K, hd_dtype dt, int packed) {
  if (N < 1 || F < 1 || D < 1 || K < 1 || !enums_ok(dt, 0) || !dims_ok(N, F, D, K)) return "";
  if (packed) return hd::bundle_packed_kernel_name(N, F, D, K, dt);
  return hd::bundle_supported(K) && dt != HD_I8 ? "bundle_valu_kernel" : "";
}

hd_status hd_class_hardsign(const int32_t* counts, float* M, int64_t K, int64_t D,
                            hipStream_t stream) {
  if (K < 1 || D < 1) return HD_ERR_ARG;
  if (!dims_ok(0, 1, D, K)) return HD_ERR_UNSUPPORTED;
  if (!counts || !M || !aligned(counts, 4) || !aligned(M, 4)) return HD_ERR_ARG;
  return from_hip(hd::launch_class_hardsign(counts, M, K, D, stream));
}

// ---------------------------------------------------------------------------
// hd_infer_packed_noalloc: hd_infer_packed with the library's own scratch.
// The scratch is a file-scope device array: each GPU the library runs on
// holds one copy for the life of the process. Host code never passes the
// array's name to a kernel (in host code it is a stand-in, not a device
// address); it takes the device address once per device with
// hipGetSymbolAddress and uses that.
// ---------------------------------------------------------------------------
namespace {

constexpr size_t kScratchBytes = size_t(4) << 20;
__device__ __align__(256) unsigned char scratch[kScratchBytes];

hd::PerDeviceOnce g_scratch_once;
void* g_scratch_ptr[hd::kMaxDevices];

hd_status scratch_ptr(void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= hd::kMaxDevices) return HD_ERR_HIP;
  const hipError_t e = hd::once_per_device(g_scratch_once, [dev] {
    void* p = nullptr;
    const hipError_t r = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (r == hipSuccess) g_scratch_ptr[dev] = p;
    return r;
  });
  if (e != hipSuccess || !g_scratch_ptr[dev]) return HD_ERR_HIP;
  *out = g_scratch_ptr[dev];
  return HD_OK;
}

}  // namespace

size_t hd_noalloc_scratch_bytes(void) { return kScratchBytes; }

hd_status hd_infer_packed_noalloc(const void* X, const void* packed, int32_t* labels,
                                  float* scores, int64_t N, int64_t F, int64_t D, int64_t K,
                                  hd_dtype dt, hd_act act, hipStream_t stream) {
  if (N > 0 && !packed) return HD_ERR_ARG;
  if (N < 0 || F < 1 || D < 1 || K < 1 || !enums_ok(dt, act_base(act))) return HD_ERR_ARG;
  if (!dims_ok(N, F, D, K) || !i8_ok(dt, act_base(act))) return HD_ERR_UNSUPPORTED;
  if (N == 0) return HD_OK;
  const size_t need = workspace_need(N, F, D, K, dt, true, det_of(act));
  if (need > kScratchBytes) return HD_ERR_WORKSPACE;
  void* ws = nullptr;
  // every check of the allocating entry point, before anything is enqueued
  // (the scratch's alignment and size stand in for a caller's workspace)
  hd_status st = infer_common(X, nullptr, nullptr, packed, labels, scores, N, F, D, K, dt, act,
                              reinterpret_cast<void*>(uintptr_t(256)), kScratchBytes, stream,
                              true);
  if (st != HD_OK) return st;
  st = scratch_ptr(&ws);
  if (st != HD_OK) return st;
  // The kernels leave their scratch zeroed, but a call that never finished
  // (or a caller that wrote the memory) would leave it otherwise: clear the
  // part this call uses with a fill kernel (not a memset node, so the call
  // can be captured in a graph).
  if (need > 0 && hd::launch_zero(ws, need, stream) != hipSuccess) return HD_ERR_HIP;
  return infer_common(X, nullptr, nullptr, packed, labels, scores, N, F, D, K, dt, act, ws,
                      kScratchBytes, stream);
}

}  // extern "C"
