"""GPU parity of the int8 model variant (HD_I8): X, B and C are int8, Stage I
sums exactly in int32 on the int8 matrix instructions, Stage II is exact in
fp32. Every sum is an exact integer, so labels and scores must equal the
oracle's (which sums the same integers exactly in fp64) bit for bit, on
every kernel, with HardSign ties (a zero sum gives +1) and argmax ties (the
lowest class) included, and up to the largest supported F and D.
"""
import numpy as np
import pytest

import hd_inputs
import oracle
from gpu_util import announce, torch_or_skip

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def hd():
    torch_or_skip()
    import paper_2506_09282_amd as hd
    hd.lib()
    return hd


def i8(a):
    torch = torch_or_skip()
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int8)).cuda()


def run(hd, X, B, C, packed):
    torch = torch_or_skip()
    Xd, Bd, Cd = i8(X), i8(B), i8(C)
    if packed:
        y, S = hd.infer_packed(Xd, hd.pack_model(Bd, Cd), return_scores=True)
    else:
        y, S = hd.infer(Xd, Bd, Cd, return_scores=True)
    torch.cuda.synchronize()
    return y.cpu().numpy(), S.cpu().numpy().astype(np.float64)


def check(y, S, ref):
    assert np.array_equal(S, ref["S"]), np.abs(S - ref["S"]).max()
    assert np.array_equal(y, ref["y"])


# (N, F, D, K, packed, kernel): X tile resident (one, two and four 32-sample
# tiles per workgroup, one to four class blocks), X streamed in F-chunks
# (double-buffered by buffer-to-LDS loads when F is a multiple of 16, through
# registers when ragged), one sample (split of D), ragged D.
CASES = [
    (300, 617, 4096, 26, True, "large_fused_kernel"),
    (300, 617, 4096, 26, False, "large_fused_kernel"),
    (1, 561, 10240, 6, False, "large_fused_kernel"),
    (129, 300, 2000, 100, True, "large_fused_kernel"),
    (77, 1000, 999, 40, False, "large_fused_kernel"),
    (200, 3001, 1024, 10, True, "large_fused_kernel"),
    (200, 3072, 1024, 10, True, "large_chunked_dma_kernel"),
    (1000, 4096, 2048, 20, True, "large_chunked_dma_kernel"),
    (200, 6016, 1024, 10, True, "large_chunked_dma_kernel"),
    (33, 8192, 512, 128, False, "large_chunked_dma_kernel"),
    (130, 6001, 700, 70, True, "large_chunked_kernel"),
]


@pytest.mark.parametrize("N,F,D,K,packed,kernel", CASES)
def test_int8_bit_exact(hd, N, F, D, K, packed, kernel):
    torch = torch_or_skip()
    assert hd.infer_kernel(N, F, D, K, torch.int8, packed=packed) == kernel
    announce(f"int8 N={N} F={F} D={D} K={K} packed={packed} ({kernel})")
    X, B, C = hd_inputs.make_int8_inputs(N, F, D, K, seed=N + F + K)
    y, S = run(hd, X, B, C, packed)
    check(y, S, oracle.infer(X, B, C))


# Small batches on a packed model: the fragment kernel on the int8 matrix
# instructions (one to four 16-sample tiles, 12 to 64 rows per lane, the B
# ring when a workgroup walks more than three column blocks, ragged D, the
# smallest F, the most classes it takes).
SMALL_CASES = [
    (1, 561, 10240, 6),
    (9, 617, 4096, 16),
    (16, 33, 1000, 5),
    (32, 561, 10240, 6),
    (48, 700, 2000, 10),
    (64, 1024, 3000, 16),
    (64, 561, 20480, 6),
    (24, 4, 64, 2),
    (40, 1000, 13000, 5),
    (63, 250, 777, 7),
    (65, 561, 10240, 6),  # 64 + 1 samples: two calls
    (128, 617, 4096, 16),  # two 64-sample calls
    (256, 300, 2000, 6),  # four 64-sample calls
]


@pytest.mark.parametrize("N,F,D,K", SMALL_CASES)
@pytest.mark.parametrize("det", [False, True])
def test_int8_small_bit_exact(hd, N, F, D, K, det):
    torch = torch_or_skip()
    assert hd.infer_kernel(N, F, D, K, torch.int8, packed=True) == "small_frag_mfma_kernel"
    announce(f"int8 small N={N} F={F} D={D} K={K} det={det}")
    X, B, C = hd_inputs.make_int8_inputs(N, F, D, K, seed=N + F + K)
    model = hd.pack_model(i8(B), i8(C))
    y, S = hd.infer_packed(i8(X), model, return_scores=True, deterministic=det)
    torch.cuda.synchronize()
    check(y.cpu().numpy(), S.cpu().numpy().astype(np.float64), oracle.infer(X, B, C))


def test_int8_small_extreme_sums_and_ties(hd):
    """F = 1024 with every product at +-128 * 128 (sums reach 2^24, still exact
    in the int32 accumulators and in fp32), then X, B in {-1, 0, 1} with many
    zero sums (HardSign +1) and tied classes (the lowest index wins)."""
    torch = torch_or_skip()
    N, F, D, K = 5, 1024, 256, 3
    announce(f"int8 small extremes N={N} F={F}")
    X = np.full((N, F), -128, np.int8)
    X[1] = 127
    X[2, ::2] = 127
    X[3, 1::4] = 0
    B = np.full((F, D), -128, np.int8)
    B[:, 1::3] = 127
    C = hd_inputs.make_int8_inputs(1, 1, D, K, seed=3)[2]
    assert hd.infer_kernel(N, F, D, K, torch.int8, packed=True) == "small_frag_mfma_kernel"
    ref = oracle.infer(X, B, C, want_va=True)
    assert np.abs(ref["V"]).max() == 2 ** 24
    y, S = run(hd, X, B, C, True)
    check(y, S, ref)
    N, F, D, K = 40, 300, 1000, 6
    X, B, C = hd_inputs.make_int8_inputs(N, F, D, K, seed=9, lo=-1, hi=1)
    C[3] = C[1]
    C[5] = C[1]
    ref = oracle.infer(X, B, C, want_va=True)
    assert (ref["V"] == 0).sum() > 100
    y, S = run(hd, X, B, C, True)
    check(y, S, ref)


def test_int8_small_unaligned_x_and_noalloc(hd):
    """An X that does not start on a 16-byte boundary takes the large-batch
    kernels within the queried workspace; the no-allocation entry point runs
    the fragment kernel on the library's scratch."""
    torch = torch_or_skip()
    N, F, D, K = 32, 561, 10240, 6
    announce(f"int8 small unaligned X and no-alloc N={N}")
    X, B, C = hd_inputs.make_int8_inputs(N, F, D, K, seed=21)
    model = hd.pack_model(i8(B), i8(C))
    ref = oracle.infer(X, B, C)
    buf = torch.zeros(N * F + 64, dtype=torch.int8, device="cuda")
    Xu = buf[1:1 + N * F].view(N, F)
    Xu.copy_(i8(X))
    assert Xu.data_ptr() % 16 != 0
    y, S = hd.infer_packed(Xu, model, return_scores=True)
    torch.cuda.synchronize()
    check(y.cpu().numpy(), S.cpu().numpy().astype(np.float64), ref)
    for n in (N, 9):
        y, S = hd.infer_packed_noalloc(i8(X[:n]), model, return_scores=True)
        torch.cuda.synchronize()
        r = oracle.infer(X[:n], B, C)
        check(y.cpu().numpy(), S.cpu().numpy().astype(np.float64), r)


@pytest.mark.parametrize("N,F,kernel", [(300, 40, "large_fused_kernel"),
                                        (100, 6000, "large_chunked_dma_kernel"),
                                        (100, 6001, "large_chunked_kernel")])
def test_int8_zero_sums_and_argmax_ties(hd, N, F, kernel):
    """X, B in {-1, 0, 1}: many encoding sums are exactly 0 (HardSign +1);
    duplicated class rows tie, and the lowest index must win."""
    torch = torch_or_skip()
    D, K = 512, 6
    assert hd.infer_kernel(N, F, D, K, torch.int8, packed=True) == kernel
    announce(f"int8 ties N={N} F={F}")
    X, B, C = hd_inputs.make_int8_inputs(N, F, D, K, seed=7, lo=-1, hi=1)
    C[3] = C[1]
    C[5] = C[1]
    ref = oracle.infer(X, B, C, want_va=True)
    assert (ref["V"] == 0).sum() > 100
    y, S = run(hd, X, B, C, True)
    check(y, S, ref)


def test_int8_largest_sums(hd):
    """The largest supported F with every product at its extreme (128 * 128):
    the int32 sums come within 2^-14 of their range without wrapping."""
    N, F, D, K = 3, 131071, 64, 2
    announce(f"int8 largest F={F}")
    X = np.full((N, F), -128, np.int8)
    X[1] = 127
    X[2, ::2] = 127
    B = np.full((F, D), -128, np.int8)
    B[:, 1::3] = 127
    C = hd_inputs.make_int8_inputs(1, 1, D, K, seed=3)[2]
    y, S = run(hd, X, B, C, True)
    check(y, S, oracle.infer(X, B, C))


def test_int8_largest_d(hd):
    """D = 131072: the largest score magnitude, 128 * D = 2^24, is still exact."""
    N, F, D, K = 4, 16, 131072, 3
    announce(f"int8 largest D={D}")
    X, B, C = hd_inputs.make_int8_inputs(N, F, D, K, seed=5)
    C[0] = -128
    y, S = run(hd, X, B, C, True)
    check(y, S, oracle.infer(X, B, C))


@pytest.mark.parametrize("N,F,D,K,kernel", [(2000, 617, 4096, 26, "bundle_mfma_kernel"),
                                             (1500, 3072, 2000, 26, "bundle_dma_kernel"),
                                             (130, 4096, 700, 60, "bundle_dma_kernel")])
def test_int8_training_and_round_trip(hd, N, F, D, K, kernel):
    """Single-pass training from int8 samples (exact class sums), then the
    codebook as an int8 model: a class with one sample scores exactly D on
    that sample."""
    torch = torch_or_skip()
    assert hd.bundle_kernel(N, F, D, K, torch.int8, packed=True) == kernel
    announce(f"int8 training N={N} F={F} D={D} K={K} ({kernel})")
    X, B, _ = hd_inputs.make_int8_inputs(N, F, D, 1, seed=11)
    y = np.random.default_rng(11).integers(0, K, N).astype(np.int32)
    y[:K] = np.arange(K)
    y[K:][y[K:] == 4] = 5  # class 4 holds one sample
    model = hd.pack_model(i8(B), K=K)
    counts = hd.bundle_classes_packed(i8(X), model, torch.from_numpy(y).cuda(), K)
    M = hd.class_hardsign(counts)
    torch.cuda.synchronize()
    ref = oracle.bundle(X, B, y, K)
    assert np.array_equal(counts.cpu().numpy(), ref["counts"])
    assert np.array_equal(M.cpu().numpy(), ref["M"])
    Mi8 = M.to(torch.int8)
    labels, S = hd.infer_packed(i8(X[:K]), hd.pack_model(i8(B), Mi8), return_scores=True)
    torch.cuda.synchronize()
    S = S.cpu().numpy()
    assert S[4, 4] == D
    check(labels.cpu().numpy(), S, oracle.infer(X[:K], B, M.cpu().numpy()))


def test_int8_rejects_other_paths(hd):
    torch = torch_or_skip()
    X = torch.zeros((4, 16), dtype=torch.int8, device="cuda")
    B = torch.zeros((16, 64), dtype=torch.int8, device="cuda")
    C = torch.zeros((2, 64), dtype=torch.int8, device="cuda")
    with pytest.raises(hd.HDError):
        hd.infer(X, B, C, act="identity")
    with pytest.raises(hd.HDError):
        hd.encode(X, B)
    with pytest.raises(hd.HDError):
        hd.bundle_classes(X, B, torch.zeros(4, dtype=torch.int32, device="cuda"), 2)
