"""C-ABI checks that need no GPU: the library loads, exports every function
``include/hd.h`` declares, and rejects bad arguments on the host before any
HIP call (these calls return before anything is enqueued)."""
import ctypes
import os
import re

import pytest

import paper_2506_09282_amd as hd

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "hd.h")
FAKE = 0x10000  # never dereferenced: validation fails first


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(hd_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(hd.LIB_PATH):
        from paper_2506_09282_amd import build
        build.build()
    return hd.lib()


def test_header_symbols_exported(L):
    names = declared_functions()
    assert set(names) == set(hd.SYMBOLS), names
    raw = ctypes.CDLL(hd.LIB_PATH)
    for n in names:
        assert hasattr(raw, n), n


def test_status_strings(L):
    for s in range(5):
        assert L.hd_status_str(s).startswith(b"HD_")
    assert L.hd_status_str(99) == b"HD_ERR_UNKNOWN"


def test_workspace_sizes(L):
    # small batch: 256-byte ticket header + replicated accumulators
    small = L.hd_infer_workspace_bytes(32, 561, 10240, 6, hd.HD_F32)
    # counters (the final one and 8 group counters, 256 bytes each), then the
    # score replicas: 32 (default mode) or one per workgroup (at most one per
    # 16-column block) plus one per ticket group (deterministic mode); the
    # query covers both
    assert small == 256 * 9 + 4 * max(32, 10240 // 16 + 8) * 32 * 6
    assert L.hd_infer_workspace_bytes(0, 561, 10240, 6, hd.HD_F32) == 0
    assert L.hd_infer_workspace_bytes(5, 0, 10, 6, hd.HD_F32) == 0
    # large batch, raw entry: holds the tiled model
    big = L.hd_infer_workspace_bytes(65536, 617, 10240, 26, hd.HD_BF16)
    tiled_b = 320 * 39 * 1024
    assert big >= tiled_b
    assert L.hd_infer_packed_workspace_bytes(65536, 617, 10240, 26, hd.HD_BF16) < tiled_b
    img = L.hd_model_packed_bytes(617, 10240, 26, hd.HD_BF16)
    assert img >= tiled_b + 617 * 10240 * 2 + 26 * 10240 * 2


def _infer(L, X=FAKE, B=FAKE, C=FAKE, labels=FAKE, scores=None, N=4, F=8, D=64, K=3,
           dt=hd.HD_F32, act=0, ws=FAKE, wsb=1 << 20):
    return L.hd_infer(X, B, C, labels, scores, N, F, D, K, dt, act, ws, wsb, None)


def test_infer_argument_errors(L):
    assert _infer(L, X=None) == hd.HD_ERR_ARG
    assert _infer(L, B=None) == hd.HD_ERR_ARG
    assert _infer(L, C=None) == hd.HD_ERR_ARG
    assert _infer(L, labels=None) == hd.HD_ERR_ARG
    assert _infer(L, N=-1) == hd.HD_ERR_ARG
    assert _infer(L, F=0) == hd.HD_ERR_ARG
    assert _infer(L, D=0) == hd.HD_ERR_ARG
    assert _infer(L, K=0) == hd.HD_ERR_ARG
    assert _infer(L, dt=7) == hd.HD_ERR_ARG
    assert _infer(L, act=5) == hd.HD_ERR_ARG
    assert _infer(L, ws=None) == hd.HD_ERR_ARG
    assert _infer(L, wsb=16) == hd.HD_ERR_WORKSPACE
    assert _infer(L, F=1 << 31) == hd.HD_ERR_UNSUPPORTED
    # N == 0 is a no-op, even with null buffers
    assert _infer(L, N=0, X=None, labels=None, ws=None, wsb=0) == hd.HD_OK


def test_large_batch_limits(L):
    """N > 256 (fp32) or N > 64 (bf16) takes the large-batch path: K <= 128, F <= 2^20,
    tiled B below 2 GiB. These are rejected on the host before any device call."""
    assert _infer(L, N=300, K=129) == hd.HD_ERR_UNSUPPORTED
    assert _infer(L, N=100, K=129, dt=hd.HD_BF16) == hd.HD_ERR_UNSUPPORTED
    assert _infer(L, N=300, F=(1 << 20) + 1, D=64) == hd.HD_ERR_UNSUPPORTED
    # fp32: 2 * ceil(D/64) * ceil(F/8) KiB >= 2 GiB
    assert _infer(L, N=300, F=8192, D=64 * 1024) == hd.HD_ERR_UNSUPPORTED


def test_other_entry_argument_errors(L):
    assert L.hd_encode(None, FAKE, FAKE, 4, 8, 16, 0, 0, None) == hd.HD_ERR_ARG
    assert L.hd_encode(FAKE, FAKE, FAKE, 4, 0, 16, 0, 0, None) == hd.HD_ERR_ARG
    assert L.hd_encode(FAKE, FAKE, FAKE, 0, 8, 16, 0, 0, None) == hd.HD_OK
    assert L.hd_similarity(FAKE, None, FAKE, None, 4, 16, 3, 0, None) == hd.HD_ERR_ARG
    assert L.hd_similarity(FAKE, FAKE, FAKE, None, 4, 16, 0, 0, None) == hd.HD_ERR_ARG
    assert L.hd_pack_model(FAKE, FAKE, 8, 16, 3, 0, FAKE, 8, None) == hd.HD_ERR_WORKSPACE
    assert L.hd_pack_model(None, FAKE, 8, 16, 3, 0, FAKE, 1 << 30, None) == hd.HD_ERR_ARG
    assert L.hd_infer_packed(FAKE, None, FAKE, None, 100, 8, 16, 3, 0, 0, FAKE, 1 << 20,
                             None) == hd.HD_ERR_ARG


def test_product_path_does_not_touch_oracle():
    """The binding and the HIP sources never import, link or load the oracle."""
    pkg = os.path.join(ROOT, "paper_2506_09282_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".hpp", ".cpp", ".h")):
                text = open(os.path.join(dirpath, f)).read()
                assert "oracle" not in text.lower(), f


def test_workspace_query_covers_unaligned_x_plan(L):
    """The large-batch plan depends on X's alignment: bf16 X that is not
    16-byte aligned takes the register-staged chunked kernel (128-sample
    tiles, so fewer tiles and a deeper split of D to fill 256 compute units).
    The size query must cover that plan's tile counters and split-D partial
    scores, not only the aligned plan's."""
    F, D, K = 3072, 10240, 10
    for N in (8192, 16384):
        tiles = N // 128
        ds = 1
        while tiles * ds < 256:
            ds *= 2
        counters = (tiles * 4 + 255) // 256 * 256
        need = counters + 4 * ds * N * K
        assert L.hd_infer_packed_workspace_bytes(N, F, D, K, hd.HD_BF16) >= need, N
        raw = L.hd_infer_workspace_bytes(N, F, D, K, hd.HD_BF16)
        assert raw >= need + L.hd_model_packed_bytes(F, D, K, hd.HD_BF16) // 2, N


def test_noalloc_argument_errors(L):
    """The allocation-free entry point validates like hd_infer_packed and
    rejects a scratch need above its fixed size, all before any device call."""
    sb = L.hd_noalloc_scratch_bytes()
    assert sb == 4 << 20
    f = L.hd_infer_packed_noalloc
    assert f(FAKE, None, FAKE, None, 100, 8, 16, 3, 0, 0, None) == hd.HD_ERR_ARG
    assert f(None, FAKE, FAKE, None, 100, 8, 16, 3, 0, 0, None) == hd.HD_ERR_ARG
    assert f(FAKE, FAKE, FAKE, None, 4, 0, 16, 3, 0, 0, None) == hd.HD_ERR_ARG
    assert f(FAKE, FAKE, FAKE, None, 4, 8, 16, 3, 9, 0, None) == hd.HD_ERR_ARG
    assert f(FAKE, FAKE, FAKE, None, 0, 8, 16, 3, 0, 0, None) == hd.HD_OK
    N, F, D, K = 2000, 3072, 10240, 128
    assert L.hd_infer_packed_workspace_bytes(N, F, D, K, hd.HD_BF16) > sb
    assert f(FAKE, FAKE, FAKE, None, N, F, D, K, hd.HD_BF16, 0, None) == hd.HD_ERR_WORKSPACE


def test_training_argument_errors(L):
    """hd_bundle_classes / hd_class_hardsign reject bad arguments before any
    device call; N == 0 is a no-op."""
    f = L.hd_bundle_classes
    assert f(FAKE, FAKE, FAKE, FAKE, 0, 8, 64, 3, 0, None) == hd.HD_OK
    assert f(None, None, None, None, 0, 8, 64, 3, 0, None) == hd.HD_OK
    assert f(None, FAKE, FAKE, FAKE, 4, 8, 64, 3, 0, None) == hd.HD_ERR_ARG
    assert f(FAKE, FAKE, None, FAKE, 4, 8, 64, 3, 0, None) == hd.HD_ERR_ARG
    assert f(FAKE, FAKE, FAKE, None, 4, 8, 64, 3, 0, None) == hd.HD_ERR_ARG
    assert f(FAKE, FAKE, FAKE, FAKE, -1, 8, 64, 3, 0, None) == hd.HD_ERR_ARG
    assert f(FAKE, FAKE, FAKE, FAKE, 4, 0, 64, 3, 0, None) == hd.HD_ERR_ARG
    assert f(FAKE, FAKE, FAKE, FAKE, 4, 8, 0, 3, 0, None) == hd.HD_ERR_ARG
    assert f(FAKE, FAKE, FAKE, FAKE, 4, 8, 64, 0, 0, None) == hd.HD_ERR_ARG
    assert f(FAKE, FAKE, FAKE, FAKE, 4, 8, 64, 3, 7, None) == hd.HD_ERR_ARG
    assert f(FAKE + 2, FAKE, FAKE, FAKE, 4, 8, 64, 3, 0, None) == hd.HD_ERR_ARG
    assert f(FAKE, FAKE, FAKE + 2, FAKE, 4, 8, 64, 3, 1, None) == hd.HD_ERR_ARG
    assert f(FAKE, FAKE, FAKE, FAKE, 4, 8, 64, 513, 0, None) == hd.HD_ERR_UNSUPPORTED
    g = L.hd_class_hardsign
    assert g(None, FAKE, 3, 64, None) == hd.HD_ERR_ARG
    assert g(FAKE, None, 3, 64, None) == hd.HD_ERR_ARG
    assert g(FAKE, FAKE, 0, 64, None) == hd.HD_ERR_ARG
    assert g(FAKE, FAKE, 3, 0, None) == hd.HD_ERR_ARG
    assert g(FAKE + 1, FAKE, 3, 64, None) == hd.HD_ERR_ARG


def test_packed_training_argument_errors(L):
    f = L.hd_bundle_classes_packed
    assert f(FAKE, FAKE, FAKE, FAKE, 0, 8, 64, 3, 0, None) == hd.HD_OK
    assert f(None, FAKE, FAKE, FAKE, 4, 8, 64, 3, 0, None) == hd.HD_ERR_ARG
    assert f(FAKE, None, FAKE, FAKE, 4, 8, 64, 3, 0, None) == hd.HD_ERR_ARG
    assert f(FAKE, FAKE + 16, FAKE, FAKE, 4, 8, 64, 3, 0, None) == hd.HD_ERR_ARG  # image alignment
    assert f(FAKE, FAKE, FAKE, FAKE, 4, 8, 64, 129, 0, None) == hd.HD_ERR_UNSUPPORTED
    assert f(FAKE, FAKE, FAKE, FAKE, 4, 8, 64, 3, 5, None) == hd.HD_ERR_ARG
    # a model packed without a codebook: C may be NULL, B may not
    assert L.hd_pack_model(None, None, 8, 16, 3, 0, FAKE, 1 << 30, None) == hd.HD_ERR_ARG


def test_int8_limits(L):
    """The int8 variant: HardSign only, exactness bounds on F and D, the
    fragment kernel for small batches on a packed model and the large-batch
    kernels otherwise, no stage-alone or streaming call."""
    I8 = hd.HD_I8
    assert _infer(L, dt=I8, act=1) == hd.HD_ERR_UNSUPPORTED
    assert _infer(L, dt=I8, F=131072) == hd.HD_ERR_UNSUPPORTED
    assert _infer(L, dt=I8, D=131073) == hd.HD_ERR_UNSUPPORTED
    assert _infer(L, dt=I8, K=129) == hd.HD_ERR_UNSUPPORTED
    for n in (1, 9, 32, 64):
        assert L.hd_infer_kernel(n, 561, 10240, 6, I8, 1) == b"small_frag_mfma_kernel"
    # 64 < N <= 256: 64-sample calls of the fragment kernel; above, the large kernels
    assert L.hd_infer_kernel(65, 561, 10240, 6, I8, 1) == b"small_frag_mfma_kernel"
    assert L.hd_infer_kernel(256, 561, 10240, 6, I8, 1) == b"small_frag_mfma_kernel"
    assert L.hd_infer_kernel(257, 561, 10240, 6, I8, 1) == b"large_fused_kernel"
    assert L.hd_infer_kernel(32, 561, 10240, 6, I8, 0) == b"large_fused_kernel"  # raw B, C
    assert L.hd_infer_kernel(32, 1025, 10240, 6, I8, 1) != b"small_frag_mfma_kernel"
    assert L.hd_infer_kernel(32, 561, 10240, 17, I8, 1) == b"large_fused_kernel"
    # (an X that is not 16-byte aligned falls back to the large-batch kernels,
    # and the workspace query covers that route: tests/test_gpu_int8.py)
    assert L.hd_infer_kernel(1, 131071, 64, 2, I8, 1) == b"large_chunked_kernel"
    assert L.hd_encode(FAKE, FAKE, FAKE, 4, 8, 16, I8, 0, None) == hd.HD_ERR_UNSUPPORTED
    assert L.hd_similarity(FAKE, FAKE, FAKE, None, 4, 16, 3, I8, None) == hd.HD_ERR_UNSUPPORTED
    assert L.hd_bundle_classes(FAKE, FAKE, FAKE, FAKE, 4, 8, 64, 3, I8, None) == \
        hd.HD_ERR_UNSUPPORTED
    assert L.hd_infer_stream_workspace_bytes(4, 1, 561, 10240, 6, I8) == 0
    assert L.hd_bundle_kernel(100, 617, 4096, 26, I8, 1) == b"bundle_mfma_kernel"
    assert L.hd_bundle_kernel(100, 617, 4096, 26, I8, 0) == b""
    # the packed image's small-batch section holds C's column tiles and the
    # fragment copy of B (F <= 1024), not B's column tiles
    assert L.hd_model_packed_bytes(617, 4096, 26, I8) < L.hd_model_packed_bytes(617, 4096, 26, 1)
    nblk, s16 = 4096 // 16, (48 + 7) // 8  # F = 617: 48 rows per lane
    frag = nblk * 4 * s16 * 64 * 8
    ctiles = -(-nblk * 26 * 16 // 256) * 256
    assert L.hd_model_packed_bytes(617, 4096, 26, I8) >= frag + ctiles
    # F = 1025 has no fragment copy (1 MB at F = 1024) and one more 32-row
    # step of the large-batch section (128 KB)
    assert L.hd_model_packed_bytes(1025, 4096, 26, I8) < L.hd_model_packed_bytes(1024, 4096, 26, I8)


def test_deterministic_flag(L):
    """HD_DETERMINISTIC combines with either activation on the inference calls
    and is refused by the streaming call; other bits are invalid."""
    DET = hd.HD_DETERMINISTIC
    assert _infer(L, N=0, X=None, labels=None, ws=None, wsb=0, act=DET) == hd.HD_OK
    assert _infer(L, N=0, X=None, labels=None, ws=None, wsb=0, act=DET | 1) == hd.HD_OK
    assert _infer(L, act=0x200) == hd.HD_ERR_ARG
    assert _infer(L, act=DET | 2) == hd.HD_ERR_ARG
    assert L.hd_infer_stream(FAKE, FAKE, None, FAKE, None, None, 1, 4, 8, 64, 3, 0, DET, FAKE,
                             1 << 20, None) == hd.HD_ERR_UNSUPPORTED
    assert L.hd_encode(FAKE, FAKE, FAKE, 4, 8, 16, 0, DET, None) == hd.HD_ERR_ARG


def test_routes_of_new_paths(L):
    """Kernel choice of the bf16 fragment route, the training kernels and the
    int8 variant (host planning only)."""
    k = L.hd_infer_kernel
    # packed bf16 small batches: the fragment kernel (bf16 fragments); raw: large-batch
    assert k(32, 561, 10240, 6, hd.HD_BF16, 1) == b"small_frag_mfma_kernel"
    assert k(32, 561, 10240, 6, hd.HD_BF16, 0) == b"large_fused_kernel"
    assert k(32, 561, 10240, 17, hd.HD_BF16, 1) == b"large_fused_kernel"  # K > 16
    # 64-sample calls of the fragment kernel up to 256 samples of a packed bf16 model
    assert k(256, 561, 10240, 6, hd.HD_BF16, 1) == b"small_frag_mfma_kernel"
    assert k(257, 561, 10240, 6, hd.HD_BF16, 1) == b"large_fused_kernel"
    assert k(100, 561, 10240, 6, hd.HD_BF16, 0) == b"large_fused_kernel"
    b = L.hd_bundle_kernel
    assert b(16384, 3072, 10240, 10, hd.HD_BF16, 1) == b"bundle_dma_kernel"
    assert b(16384, 3072, 10240, 10, hd.HD_I8, 1) == b"bundle_dma_kernel"
    assert b(16384, 3071, 10240, 10, hd.HD_BF16, 1) == b"bundle_mfma_kernel"  # F % 8 != 0
    assert b(4096, 784, 10240, 10, hd.HD_F32, 1) == b"bundle_mfma_kernel"
    assert b(4096, 784, 10240, 129, hd.HD_F32, 1) == b""      # packed path: K <= 128
    assert b(4096, 784, 10240, 512, hd.HD_F32, 0) == b"bundle_valu_kernel"
    assert b(4096, 784, 10240, 513, hd.HD_F32, 0) == b""
    # a packed image holds the large-batch fragments, the small-batch column
    # tiles and the small-batch fragments: fp32 ones (MS = 36 rows per lane,
    # 16*MS rows per column) for an fp32 model, bf16 ones (5 steps of 32 rows
    # per wave) for a bf16 model
    f32 = L.hd_model_packed_bytes(561, 10240, 6, hd.HD_F32)
    b16 = L.hd_model_packed_bytes(561, 10240, 6, hd.HD_BF16)
    assert f32 >= 2 * 561 * 10240 * 4 + 576 * 10240 * 4
    assert b16 >= 2 * 561 * 10240 * 2 + 4 * 5 * 32 * 10240 * 2
    assert b16 < f32 // 2 + 4 * 5 * 32 * 10240 * 2
