/*
 * hd.h — C ABI of the MI355X (gfx950) batched hyperdimensional-computing
 * inference library (with single-pass training and an int8 model variant).
 *
 * The operation is the two-stage HDC inference of ScalableHD (Sec. II-D,
 * Alg. 1): with raw features X[N,F], base hypervectors B[F,D] and class
 * hypervectors C[K,D] (the paper's M),
 *   Stage I  (Eq. 7, Eq. 2-3):  H = HardSign(X B),  HardSign(x) = +1 if x >= 0 else -1 (Eq. 1)
 *   Stage II (Eq. 8, Eq. 9):    S = H C^T,  labels[n] = argmax_k S[n,k]
 *
 * Conventions shared by every entry point:
 *   - Layout: dense, contiguous, row-major. X[N,F], B[F,D], C[K,D], H[N,D],
 *     scores[N,K]. The paper's J = M^T is C read column-major.
 *   - Types: hd_dtype names the element type of X, B and C (HD_BF16 buffers
 *     hold raw bfloat16 bit patterns). Accumulation is fp32 (int32 for
 *     HD_I8 Stage I). H and scores are fp32; labels are int32 in [0, K).
 *   - Pointers: X, B, C, H, labels, scores, workspace and packed models are
 *     DEVICE pointers owned by the caller. The library allocates nothing,
 *     frees nothing and keeps no pointer after a call returns. Outputs must
 *     not alias inputs.
 *   - Streams: work is enqueued on `stream` (0 = the null stream) and the call
 *     returns without synchronising; results are valid once the stream has
 *     reached that point.
 *   - Errors: arguments are validated on the host before anything is
 *     enqueued; a failing call enqueues nothing. N == 0 is a no-op returning
 *     HD_OK. HD_ERR_HIP reports a launch failure (hipGetLastError).
 *   - Ties: HardSign(0) = +1 (Eq. 1: ties broken toward +1, so -0.0 -> +1);
 *     argmax ties go to the lowest class index (the paper is silent; this is
 *     the first-maximum convention).
 *   - Limits: 1 <= F, D, K <= 2^30 and 0 <= N <= 2^30; anything larger
 *     returns HD_ERR_UNSUPPORTED. The fused calls on the large-batch path
 *     (bf16 with N > 8; fp32 with N > 256, or N > 64 where the small-batch
 *     kernels would not use the matrix cores) further need K <= 128,
 *     F <= 2^20 and a tiled B below 2 GiB (2 * ceil(D/64) * ceil(F/s) KiB,
 *     s = 16 features for bf16, 8 for fp32). Otherwise a call with N <= 64
 *     falls back to the small-batch kernels and a larger one returns
 *     HD_ERR_UNSUPPORTED.
 *   - Thread safety: besides write-once launch settings kept per device
 *     (kernel LDS attributes, the compute-unit count), the library holds no
 *     state between calls; concurrent calls are safe when each uses its own
 *     workspace.
 */
#ifndef HD_H_
#define HD_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ihipStream_t *hipStream_t;

typedef enum {
  HD_OK = 0,
  HD_ERR_ARG = 1,         /* null pointer, negative/zero size, bad enum */
  HD_ERR_UNSUPPORTED = 2, /* size or dtype/act combination beyond what is built */
  HD_ERR_WORKSPACE = 3,   /* workspace or packed buffer too small */
  HD_ERR_HIP = 4          /* a HIP launch failed */
} hd_status;

/*
 * HD_I8: the int8 model variant (the quantised models of Sec. II-C, which the
 * paper mentions and does not use): X, B and C hold int8 values; Stage I sums
 * exactly in int32 on the int8 matrix instructions, HardSign is taken on the
 * exact sum, and Stage II is exact in fp32 (C widened exactly to bf16 or
 * fp32). Every result is therefore exact: scores are integers, and labels and
 * scores equal the mathematical definition bit for bit. Scales of a
 * quantised model do not enter: a positive scale of X or B leaves every
 * HardSign unchanged, and a per-class scale of C is the caller's to apply to
 * the returned scores. Supported by hd_pack_model, hd_infer, hd_infer_packed,
 * hd_infer_packed_noalloc, hd_bundle_classes_packed and the size and kernel
 * queries, with HD_ACT_HARDSIGN, K <= 128, F <= 131071 (|sum| < 2^31) and
 * D <= 131072 (|score| <= 2^24). Small batches on a packed model (N <= 256,
 * K <= 16, F <= 1024, X 16-byte aligned) run on the small-batch fragment
 * kernel (int8 matrix instructions, exact int32 sums converted exactly to
 * fp32), everything else on the large-batch kernels; the workspace queries
 * cover both. Elsewhere HD_ERR_UNSUPPORTED.
 */
typedef enum { HD_F32 = 0, HD_BF16 = 1, HD_I8 = 2 } hd_dtype;

/* HD_ACT_HARDSIGN is the paper's encoding activation (Sec. II-B, Eq. 3).
 * HD_ACT_IDENTITY skips it (H = X B): a linear test mode, S = X B C^T. */
typedef enum { HD_ACT_HARDSIGN = 0, HD_ACT_IDENTITY = 1 } hd_act;

/*
 * Flag OR-ed into the act argument of hd_infer, hd_infer_packed and
 * hd_infer_packed_noalloc: scores and labels identical bit for bit from call
 * to call for the same inputs (the split of D of Sec. III-C Alg. 3 otherwise
 * sums partial scores with fp32 atomics in arrival order, which can change
 * their low bits, and so a near-tie label, between calls). The small-batch
 * path then gives each workgroup its own partial-score slot and sums the
 * slots in a fixed order; the large-batch path already sums in a fixed
 * order. The workspace size queries cover this mode. Not supported by
 * hd_infer_stream (HD_ERR_UNSUPPORTED).
 */
#define HD_DETERMINISTIC 0x100

/* Human-readable name of a status code (static string, never NULL). */
const char *hd_status_str(hd_status s);

/*
 * Stage I alone (Alg. 1 Stage I; Eq. 7 with the activation of Eq. 1):
 *   H[n,d] = act( sum_f X[n,f] * B[f,d] )      written as fp32 to H[N,D].
 * This entry point materialises H in device memory; it exists for tests and
 * for composing the stages by hand. hd_infer never materialises H.
 */
hd_status hd_encode(const void *X, const void *B, float *H, int64_t N, int64_t F, int64_t D,
                    hd_dtype dt, hd_act act, hipStream_t stream);

/*
 * Stage II alone (Alg. 1 Stage II; Eq. 8 and Eq. 9) on a real matrix H[N,D]:
 *   S[n,k] = sum_d H[n,d] * C[k,d];  labels[n] = lowest k maximising S[n,k].
 * C has element type c_dt. scores may be NULL (then only labels are written).
 */
hd_status hd_similarity(const float *H, const void *C, int32_t *labels, float *scores, int64_t N,
                        int64_t D, int64_t K, hd_dtype c_dt, hipStream_t stream);

/* Bytes of device workspace hd_infer needs for these sizes (0 is possible). */
size_t hd_infer_workspace_bytes(int64_t N, int64_t F, int64_t D, int64_t K, hd_dtype dt);

/*
 * Alg. 1 end to end, fused: labels[N] (and scores[N,K] when non-NULL) from
 * X, B, C, with the encoded matrix H never written to device memory.
 * workspace: caller-owned device buffer (256-byte aligned) of at least
 *   hd_infer_workspace_bytes(N, F, D, K, dt) bytes, ZEROED BY THE CALLER
 *   BEFORE ITS FIRST USE. Every call leaves every byte it used at zero again,
 *   so one workspace can serve consecutive calls of any shape on one stream
 *   without clearing, as long as it is large enough for each. Calls that
 *   overlap in time must not share a workspace. May be NULL only when the
 *   required size is 0. A call whose launch plan needs more than
 *   workspace_bytes returns HD_ERR_WORKSPACE and enqueues nothing.
 * The small-batch path splits the hypervector dimension D across workgroups
 * (the paper's small-batch variant, Sec. III-C Alg. 3) and reduces partial
 * scores with fp32 atomics, so score low bits can vary from run to run; the
 * large-batch path splits the batch (the large-batch variant, Alg. 4) and
 * repacks B and C into the workspace first (the parameter tiling of
 * Sec. III-D; the copy is cleared again after use) unless a packed model is
 * supplied through hd_infer_packed.
 */
hd_status hd_infer(const void *X, const void *B, const void *C, int32_t *labels, float *scores,
                   int64_t N, int64_t F, int64_t D, int64_t K, hd_dtype dt, hd_act act,
                   void *workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * One-time model tiling (Sec. III-D: B and J = M^T stored in the block order
 * the consumer reads them). The packed image is opaque; its size depends only
 * on (F, D, K, dt). packed must be a device buffer of at least
 * hd_model_packed_bytes(F, D, K, dt) bytes. C may be NULL before the class
 * hypervectors exist (a model packed for hd_bundle_classes_packed): the class
 * part of the image is then zero.
 */
size_t hd_model_packed_bytes(int64_t F, int64_t D, int64_t K, hd_dtype dt);
hd_status hd_pack_model(const void *B, const void *C, int64_t F, int64_t D, int64_t K, hd_dtype dt,
                        void *packed, size_t packed_bytes, hipStream_t stream);

/* Bytes of workspace hd_infer_packed needs (no room for a packed model). */
size_t hd_infer_packed_workspace_bytes(int64_t N, int64_t F, int64_t D, int64_t K, hd_dtype dt);

/*
 * Alg. 1 end to end from a model packed by hd_pack_model with the same
 * (F, D, K, dt). X is read as given (row-major, never pre-packed). Same
 * workspace and output rules as hd_infer.
 */
hd_status hd_infer_packed(const void *X, const void *packed, int32_t *labels, float *scores,
                          int64_t N, int64_t F, int64_t D, int64_t K, hd_dtype dt, hd_act act,
                          void *workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Streaming inference over a queue of small batches (the producer-consumer
 * pipeline of Sec. III-A for the real-time streams of Sec. I, with the
 * small-batch split of D of Sec. III-C Alg. 3): ONE persistent launch runs
 * Alg. 1 on nbatch batches of N samples each, keeping the model's share of B
 * in registers for the whole stream, so B is read once per launch rather
 * than once per batch; while batch b is multiplied, batch b+1's X is loaded
 * and batch b-1's partial scores are reduced.
 *   X       [nbatch][N][F] fp32, batch b at X + b*N*F (4-byte aligned; 16-byte
 *           aligned with N*F % 4 == 0 is faster).
 *   packed  a model packed by hd_pack_model (fp32).
 *   ready   NULL (every batch is present when the launch starts) or a 32-bit
 *           counter in device memory or in mapped pinned host memory: batch b
 *           is read only once *ready > b, with acquire ordering (write batch
 *           b's X, then publish b+1 with release ordering). Setting bit 31
 *           ends the stream after the batches already published. A batch not
 *           published within about half a second also ends the stream.
 *   labels  [nbatch][N] int32; scores [nbatch][N][K] fp32 or NULL.
 *   done    NULL or a device/host-mapped counter that is incremented once
 *           per batch whose labels (and scores) have been written.
 *   workspace  hd_infer_stream_workspace_bytes(nbatch, ...) bytes, zeroed
 *           before first use and left zeroed (one region per batch).
 * Supported: fp32, 1 <= N <= 32, K <= 16, F <= 576, D <= 48 * (compute
 * units - 1); otherwise HD_ERR_UNSUPPORTED (the workspace size query returns
 * 0). The launch holds every compute unit but one with one workgroup each,
 * plus one workgroup that reduces each batch's partial scores.
 * Scores are summed with fp32 atomics (low bits may vary between runs).
 * Results for batch b are complete once the launch finishes (or, with a
 * queue, once *done > b as seen after a system-scope acquire).
 */
size_t hd_infer_stream_workspace_bytes(int64_t nbatch, int64_t N, int64_t F, int64_t D,
                                       int64_t K, hd_dtype dt);
hd_status hd_infer_stream(const void *X, const void *packed, const uint32_t *ready,
                          int32_t *labels, float *scores, uint32_t *done, int64_t nbatch,
                          int64_t N, int64_t F, int64_t D, int64_t K, hd_dtype dt, hd_act act,
                          void *workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * hd_infer_packed without a caller workspace, for callers that cannot
 * allocate device memory or pass one in: code under HIP graph capture,
 * tight serving loops, harnesses that forbid allocation. It allocates
 * nothing (no hipMalloc, hipFree or allocating library routine); the
 * scratch its kernels need (tickets, replicated partial scores, split-D
 * partials) is a fixed device array of hd_noalloc_scratch_bytes() bytes
 * (4 MiB) inside the library, one per GPU, held until the process ends.
 * Calls whose scratch need in their mode (default or HD_DETERMINISTIC; at
 * most hd_infer_packed_workspace_bytes) exceeds that return HD_ERR_WORKSPACE
 * before anything is enqueued. Each call first
 * clears the part it uses (a fill kernel on `stream`), so the array's
 * contents from an earlier call do not matter. All calls on one GPU share
 * the array: calls that overlap in time on one GPU (other streams, other
 * host threads) race and must be serialised by the caller. Otherwise the
 * arguments, checks and results are those of hd_infer_packed.
 */
size_t hd_noalloc_scratch_bytes(void);
hd_status hd_infer_packed_noalloc(const void *X, const void *packed, int32_t *labels,
                                  float *scores, int64_t N, int64_t F, int64_t D, int64_t K,
                                  hd_dtype dt, hd_act act, hipStream_t stream);

/*
 * Single-pass training (Sec. II-C): the class hypervector of class k is the
 * bundle (elementwise sum, Sec. II-A) of the encoded hypervectors
 * H_n = HardSign(X_n B) (Eq. 2-3) of the samples with label k, normalised
 * by HardSign (Eq. 1). The sums are exact integers, so training over many
 * chunks of samples is two calls:
 *
 * hd_bundle_classes ADDS, for every sample n with 0 <= y[n] < K,
 * HardSign(X_n B) (+1 or -1 per dimension, +1 for a zero product) into
 * counts[y[n]][:]. Samples whose label lies outside [0, K) are skipped.
 *   X       [N][F] row-major, dt; B [F][D] row-major, dt (element-aligned).
 *   y       [N] int32 labels (device memory).
 *   counts  [K][D] int32, device memory, caller-owned and caller-initialised
 *           (zero it before the first chunk); calls on one stream
 *           accumulate. |counts| never exceeds the number of samples seen,
 *           so up to 2^31 - 1 samples per class are exact.
 * The product is accumulated in fp32 (bf16 inputs are widened exactly), so
 * a sample whose X_n B column lies within fp32 rounding of zero can take
 * either sign, as in inference. Counters are added with integer atomics:
 * the result is independent of their order.
 * Supported: 1 <= K <= 512; N == 0 enqueues nothing.
 *
 * hd_class_hardsign writes M[k][d] = +1.0f if counts[k][d] >= 0, else
 * -1.0f (Eq. 1; a tie or an empty class gives +1): the model C = M that
 * hd_infer and hd_pack_model take, as [K][D] fp32.
 * Both return HD_ERR_ARG for negative or zero sizes (N may be 0), NULL or
 * misaligned pointers, HD_ERR_UNSUPPORTED outside the supported sizes,
 * HD_ERR_HIP when a launch fails; nothing is enqueued on an error.
 */
hd_status hd_bundle_classes(const void *X, const void *B, const int32_t *y, int32_t *counts,
                            int64_t N, int64_t F, int64_t D, int64_t K, hd_dtype dt,
                            hipStream_t stream);
hd_status hd_class_hardsign(const int32_t *counts, float *M, int64_t K, int64_t D,
                            hipStream_t stream);

/*
 * hd_bundle_classes on the matrix cores, reading B from a model packed by
 * hd_pack_model with the same (F, D, dt) (the tiled B of Sec. III-D; the
 * image's class part is not read, so it may have been packed with C == NULL
 * and any K). Same arguments, semantics and errors as hd_bundle_classes, and
 * bit-identical counts wherever no product lies within rounding of zero
 * (both accumulate in fp32, in different orders).
 * Supported: 1 <= K <= 128, N <= 2^30.
 */
hd_status hd_bundle_classes_packed(const void *X, const void *packed, const int32_t *y,
                                   int32_t *counts, int64_t N, int64_t F, int64_t D, int64_t K,
                                   hd_dtype dt, hipStream_t stream);

/*
 * Introspection: the name of the kernel that hd_bundle_classes (packed == 0)
 * or hd_bundle_classes_packed (packed != 0) launches for these sizes,
 * assuming a 16-byte aligned X; "" when the call would be rejected. Static
 * string.
 */
const char *hd_bundle_kernel(int64_t N, int64_t F, int64_t D, int64_t K, hd_dtype dt, int packed);

/*
 * Introspection: the name of the main kernel that hd_infer (packed == 0) or
 * hd_infer_packed (packed != 0) launches for these sizes, assuming 16-byte
 * aligned operands; "" when the call would be rejected. The returned string
 * is static. Used by benchmarks and profilers to find the kernel's dispatches.
 */
const char *hd_infer_kernel(int64_t N, int64_t F, int64_t D, int64_t K, hd_dtype dt, int packed);

#ifdef __cplusplus
}
#endif

#endif /* HD_H_ */
