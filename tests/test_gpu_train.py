"""GPU parity of single-pass training (Sec. II-C): hd_bundle_classes and
hd_class_hardsign (through the C ABI) against the oracle's bundle.

On small-integer inputs the encoding sums are exact in any order, so the
class counts and the codebook must be bit-identical. On real-valued inputs a
sample whose encoding sum lies within fp32 rounding distance of zero (the
fragile set of tolerance.py) may take either sign: the count of class k at
dimension d may then differ from the oracle's by 2 per such sample of class
k, and nowhere else; the codebook must be HardSign of the GPU's own counts,
and equal to the oracle's wherever the oracle's count is farther from zero
than those flips could move it.
"""
import numpy as np
import pytest

import hd_inputs
import oracle
from gpu_util import announce, dev, torch_or_skip
from tolerance import gamma

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def hd():
    torch_or_skip()
    import paper_2506_09282_amd as hd
    hd.lib()
    return hd


def labels_for(N, K, seed, spill=0):
    """Labels in [0, K); ``spill`` of them replaced by values outside it."""
    g = np.random.default_rng(seed + 17)
    y = g.integers(0, K, N).astype(np.int32)
    if spill:
        idx = g.choice(N, size=min(spill, N), replace=False)
        y[idx] = g.choice(np.array([-1, K, K + 5, -(1 << 30), (1 << 30)], np.int32), len(idx))
    return y


PATHS = ["raw", "packed"]


def gpu_train(hd, X, B, y, K, dtype, chunks=1, path="raw"):
    """Class counts and codebook from the GPU: ``raw`` is hd_bundle_classes
    (B as given), ``packed`` hd_bundle_classes_packed (B tiled once by
    hd_pack_model with no codebook)."""
    torch = torch_or_skip()
    Xd, Bd = dev(X, dtype), dev(B, dtype)
    yd = torch.from_numpy(np.ascontiguousarray(y, np.int32)).cuda()
    model = hd.pack_model(Bd) if path == "packed" else None
    counts = torch.zeros((K, B.shape[1]), dtype=torch.int32, device="cuda")
    N = X.shape[0]
    cuts = np.linspace(0, N, chunks + 1).astype(int)
    for a, b in zip(cuts[:-1], cuts[1:]):
        if model is not None:
            hd.bundle_classes_packed(Xd[a:b], model, yd[a:b], K, counts=counts)
        else:
            hd.bundle_classes(Xd[a:b], Bd, yd[a:b], K, counts=counts)
    M = hd.class_hardsign(counts)
    torch.cuda.synchronize()
    return counts.cpu().numpy().astype(np.int64), M.cpu().numpy().astype(np.float64)


def check_exact(counts, M, ref):
    assert np.array_equal(counts, ref["counts"]), np.abs(counts - ref["counts"]).max()
    assert np.array_equal(M, ref["M"])


def check_fragile(counts, M, X, B, y, K, ref):
    """The rule of the module docstring; returns the number of differing
    counts (for the log)."""
    enc = oracle.encode(X, B, want_va=True)
    fragile = np.abs(enc["V"]) <= gamma(X.shape[1]) * enc["A"]
    nf = np.zeros(counts.shape, np.int64)
    for k in range(K):
        sel = y == k
        if sel.any():
            nf[k] = fragile[sel].sum(axis=0)
    diff = counts - ref["counts"]
    assert np.all(diff % 2 == 0)
    assert np.all(np.abs(diff) <= 2 * nf), int((np.abs(diff) - 2 * nf).max())
    assert np.array_equal(M, np.where(counts >= 0, 1.0, -1.0))
    sure = np.abs(ref["counts"]) > 2 * nf
    assert np.array_equal(M[sure], ref["M"][sure])
    return int((diff != 0).sum())


# (N, F, D, K, spill): ragged sample tiles and column blocks, one class,
# more classes than samples (empty classes), the largest supported K, and
# labels outside [0, K).
INTEGER = [
    (1, 5, 64, 1, 0),
    (63, 7, 100, 3, 0),
    (64, 561, 10240, 6, 0),
    (1000, 561, 10240, 6, 25),
    (777, 617, 4999, 26, 10),
    (130, 3072, 1024, 100, 3),
    (50, 40, 300, 80, 0),
    (2100, 33, 640, 512, 40),
    (3000, 100, 2100, 128, 40),
    (4100, 2999, 1000, 7, 0),
]


@pytest.mark.parametrize("path", PATHS)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("N,F,D,K,spill", INTEGER)
def test_integer_counts_bit_exact(hd, N, F, D, K, spill, dtype, path):
    if path == "packed" and K > 128:
        pytest.skip("the packed (matrix-core) path takes K <= 128")
    announce(f"train integer {path} {dtype} N={N} F={F} D={D} K={K} spill={spill}")
    X, B, _ = hd_inputs.make_integer_inputs(N, F, D, 1, seed=N + F + K)
    y = labels_for(N, K, N + K, spill)
    ref = oracle.bundle(X, B, y, K)
    counts, M = gpu_train(hd, X, B, y, K, dtype, path=path)
    check_exact(counts, M, ref)


# Every training kernel on integer inputs, asserting which one ran:
# (N, F, D, K, dtype, path, kernel).
KERNELS = [
    (700, 100, 1000, 9, "f32", "raw", "bundle_valu_kernel"),
    (700, 100, 1000, 9, "bf16", "raw", "bundle_valu_kernel"),
    (700, 100, 1000, 9, "f32", "packed", "bundle_mfma_kernel"),
    (3000, 2999, 700, 100, "f32", "packed", "bundle_mfma_kernel"),
    (700, 101, 1000, 9, "bf16", "packed", "bundle_mfma_kernel"),
    (130, 3072, 1024, 100, "bf16", "packed", "bundle_mfma_kernel"),
    (1000, 3072, 2048, 10, "bf16", "packed", "bundle_dma_kernel"),
    (1, 3072, 2048, 10, "bf16", "packed", "bundle_dma_kernel"),
    (65, 256, 10240, 26, "bf16", "packed", "bundle_dma_kernel"),
    (2047, 616, 1000, 60, "bf16", "packed", "bundle_dma_kernel"),
    (333, 8, 64, 2, "bf16", "packed", "bundle_dma_kernel"),
]


@pytest.mark.parametrize("N,F,D,K,dtype,path,kernel", KERNELS)
def test_every_training_kernel_bit_exact(hd, N, F, D, K, dtype, path, kernel):
    torch = torch_or_skip()
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    assert hd.bundle_kernel(N, F, D, K, tdt, packed=(path == "packed")) == kernel
    announce(f"train kernel {kernel} {dtype} N={N} F={F} D={D} K={K}")
    X, B, _ = hd_inputs.make_integer_inputs(N, F, D, 1, seed=N + 3 * F + K)
    y = labels_for(N, K, N + F, spill=N // 50)
    ref = oracle.bundle(X, B, y, K)
    counts, M = gpu_train(hd, X, B, y, K, dtype, path=path)
    check_exact(counts, M, ref)


@pytest.mark.parametrize("path", PATHS)
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_zero_sums_and_tied_counts(hd, dtype, path):
    """X and B in {-1, 0, 1}: many encoding sums are exactly 0 (HardSign gives
    +1) and many class counts are exactly 0 (the codebook gives +1)."""
    N, F, D, K = 700, 40, 1000, 9
    announce(f"train ties {path} {dtype} N={N} F={F} D={D} K={K}")
    X, B, _ = hd_inputs.make_integer_inputs(N, F, D, 1, seed=5, x_range=1, b_range=1)
    y = labels_for(N, K, 5)
    y[y == 4] = 3  # class 4 is empty: all +1
    ref = oracle.bundle(X, B, y, K)
    assert (ref["counts"] == 0).sum() > 100
    counts, M = gpu_train(hd, X, B, y, K, dtype, path=path)
    check_exact(counts, M, ref)
    assert np.all(M[4] == 1.0) and np.all(counts[4] == 0)


# Real-valued inputs at the workload shapes (features, hypervector width,
# classes), with a few thousand samples.
REAL = [
    ("activity", 2000, 561, 10240, 6, "uniform_pm1", "f32"),
    ("colour_dma", 1200, 3072, 4096, 10, "uniform01", "bf16"),
    ("image", 1500, 617, 10240, 26, "uniform01", "f32"),
    ("image", 1500, 617, 10240, 26, "uniform01", "bf16"),
    ("colour", 600, 3072, 4096, 10, "uniform01", "bf16"),
    ("colour_k100", 600, 3072, 2048, 100, "uniform01_zero20", "f32"),
]


@pytest.mark.parametrize("path", PATHS)
@pytest.mark.parametrize("name,N,F,D,K,dist,dtype", REAL)
def test_real_inputs_within_fragile_flips(hd, name, N, F, D, K, dist, dtype, path):
    announce(f"train real {path} {name} {dtype} N={N} F={F} D={D} K={K}")
    X, B, _ = hd_inputs.make_inputs(N, F, D, 1, dist, seed=3, dtype=dtype)
    y = labels_for(N, K, 3)
    ref = oracle.bundle(X, B, y, K)
    counts, M = gpu_train(hd, X, B, y, K, dtype, path=path)
    ndiff = check_fragile(counts, M, X, B, y, K, ref)
    print(f"[train] {path} {name}: {ndiff} of {counts.size} counts differ (fragile samples)")


@pytest.mark.parametrize("path", PATHS)
@pytest.mark.parametrize("chunks", [2, 7])
def test_chunked_accumulation_equals_one_call(hd, chunks, path):
    """Counts are integers added with atomics: feeding the samples in chunks
    gives the same counts bit for bit, on real-valued inputs too."""
    N, F, D, K = 1300, 561, 2048, 6
    announce(f"train chunks={chunks} {path} N={N}")
    X, B, _ = hd_inputs.make_inputs(N, F, D, 1, "uniform_pm1", seed=9)
    y = labels_for(N, K, 9)
    c1, m1 = gpu_train(hd, X, B, y, K, "f32", chunks=1, path=path)
    ck, mk = gpu_train(hd, X, B, y, K, "f32", chunks=chunks, path=path)
    assert np.array_equal(c1, ck)
    assert np.array_equal(m1, mk)


def test_empty_batch_leaves_counts(hd):
    torch = torch_or_skip()
    counts = torch.full((3, 64), 7, dtype=torch.int32, device="cuda")
    X = torch.empty((0, 5), dtype=torch.float32, device="cuda")
    B = torch.ones((5, 64), dtype=torch.float32, device="cuda")
    y = torch.empty((0,), dtype=torch.int32, device="cuda")
    hd.bundle_classes(X, B, y, 3, counts=counts)
    hd.bundle_classes_packed(X, hd.pack_model(B), y, 3, counts=counts)
    torch.cuda.synchronize()
    assert bool((counts == 7).all())


def test_packed_model_with_codebook_trains_the_same(hd):
    """The packed path reads only the tiled B: a model packed with a codebook
    trains exactly like one packed without."""
    torch = torch_or_skip()
    N, F, D, K = 500, 300, 1000, 5
    X, B, C = hd_inputs.make_inputs(N, F, D, K, "uniform_pm1", seed=12)
    y = labels_for(N, K, 12)
    Xd, Bd, Cd = dev(X, "f32"), dev(B, "f32"), dev(C, "f32")
    yd = torch.from_numpy(y).cuda()
    a = hd.bundle_classes_packed(Xd, hd.pack_model(Bd), yd, K)
    b = hd.bundle_classes_packed(Xd, hd.pack_model(Bd, Cd), yd, K)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


def test_single_sample_classes_round_trip(hd):
    """One sample per class: each codebook row is that sample's encoding, so
    inference on the same samples scores exactly D on the own class and
    returns the sample's label (planted classes; the closed form pinned on
    the oracle)."""
    torch = torch_or_skip()
    K, F, D = 12, 561, 10240
    announce(f"train round trip K={K} F={F} D={D}")
    X, B, _ = hd_inputs.make_integer_inputs(K, F, D, 1, seed=4)
    y = np.arange(K, dtype=np.int32)[::-1].copy()
    H = oracle.encode(X, B)["H"]
    for path in PATHS:
        counts, M = gpu_train(hd, X, B, y, K, "f32", path=path)
        assert np.array_equal(M[y], H)
        Xd, Bd = dev(X, "f32"), dev(B, "f32")
        Md = torch.from_numpy(M.astype(np.float32)).cuda()
        for labels, S in (hd.infer(Xd, Bd, Md, return_scores=True),
                          hd.infer_packed(Xd, hd.pack_model(Bd, Md), return_scores=True)):
            torch.cuda.synchronize()
            S = S.cpu().numpy()
            assert np.array_equal(labels.cpu().numpy(), y)
            assert np.all(S[np.arange(K), y] == D)
