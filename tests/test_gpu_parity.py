"""GPU parity: the HIP path (called through the C ABI) against the oracle.

Scores agree within 1e-4 of ||c_k||_2 once at most a few HardSign flips on
dimensions whose encoding sum is within rounding distance of zero are undone,
and labels agree with the maximum of those scores (see tolerance.py); on
small-integer inputs every summation order is exact, so there scores and
labels must be bit-identical.
"""
import numpy as np
import pytest

import hd_inputs
import oracle
from gpu_util import (BF16_DRIFT, RTOL, announce, check_against_oracle, check_all_rows, dev,
                      torch_or_skip)
from tolerance import compare, drift_scale, score_scale

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def hd():
    torch_or_skip()
    import paper_2506_09282_amd as hd
    hd.lib()  # raise now if the library is missing
    return hd


def run(hd, X, B, C, dtype, act="hardsign", scores=True, packed=False):
    torch = torch_or_skip()
    Xd, Bd, Cd = dev(X, dtype), dev(B, dtype), dev(C, dtype)
    if packed:
        model = hd.pack_model(Bd, Cd)
        out = hd.infer_packed(Xd, model, act=act, return_scores=scores)
    else:
        out = hd.infer(Xd, Bd, Cd, act=act, return_scores=scores)
    torch.cuda.synchronize()
    if scores:
        y, S = out
        return y.cpu().numpy(), S.cpu().numpy().astype(np.float64)
    return out.cpu().numpy(), None


def inputs(N, F, D, K, dist="uniform_pm1", seed=0, dtype="f32"):
    return hd_inputs.make_inputs(N, F, D, K, dist, seed=seed, dtype=dtype)


# --- the named workloads ----------------------------------------------------

@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_tiny_workload(hd, dtype):
    w = hd_inputs.WORKLOADS["tiny"]
    announce(f"tiny {dtype}")
    X, B, C = inputs(w.N, w.F, w.D, w.K, w.x_dist, dtype=dtype)
    y, S = run(hd, X, B, C, dtype)
    rep, _ = check_against_oracle(X, B, C, y, S)
    assert rep["ok"], rep


@pytest.mark.parametrize("name", ["activity_n1", "activity_n32"])
def test_activity_workloads(hd, name):
    w = hd_inputs.WORKLOADS[name]
    announce(name)
    X, B, C = inputs(w.N, w.F, w.D, w.K, w.x_dist)
    y, S = run(hd, X, B, C, "f32")
    rep, _ = check_against_oracle(X, B, C, y, S)
    assert rep["ok"], rep


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_image_workload_sampled(hd, dtype):
    w = hd_inputs.WORKLOADS["image"]
    announce(f"image {dtype}")
    X, B, C = inputs(w.N, w.F, w.D, w.K, w.x_dist, dtype=dtype)
    y, S = run(hd, X, B, C, dtype)
    rows = np.r_[0:40, w.N - 40:w.N, np.random.default_rng(1).integers(0, w.N, 48)]
    rep, _ = check_against_oracle(X, B, C, y, S, rows=rows)
    assert rep["ok"], rep


def test_speech_workload_all_rows(hd):
    """Speech shape, bf16, every one of the 65536 rows against the oracle."""
    w = hd_inputs.WORKLOADS["speech"]
    announce("speech bf16 N=65536 (all rows)")
    X, B, C = inputs(w.N, w.F, w.D, w.K, w.x_dist, dtype="bf16")
    y, S = run(hd, X, B, C, "bf16", packed=True)
    rep = check_all_rows(X, B, C, y, S)
    announce(f"speech all rows: {rep}")
    assert rep["ok"], rep
    # drift of the bf16 path against the fp32-input oracle, sampled rows
    rows = np.r_[0:32, 4090:4100, w.N - 32:w.N, np.random.default_rng(2).integers(0, w.N, 64)]
    X32, B32, C32 = inputs(w.N, w.F, w.D, w.K, w.x_dist, dtype="f32")
    ref32 = oracle.infer(X32, B32, C32, rows=rows)
    drift = np.abs(S[rows] - ref32["S"]) / drift_scale(C32)[None, :]
    assert drift.max() <= BF16_DRIFT, drift.max()


@pytest.mark.parametrize("name,dtype", [("colour_k10", "bf16"), ("colour_k10", "f32"),
                                        ("colour_k100", "f32")])
def test_colour_workload_sampled(hd, name, dtype):
    torch = torch_or_skip()
    w = hd_inputs.WORKLOADS[name]
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    assert hd.infer_kernel(w.N, w.F, w.D, w.K, tdt).startswith("large_chunked")
    announce(f"{name} {dtype} N={w.N} F={w.F}")
    X, B, C = inputs(w.N, w.F, w.D, w.K, w.x_dist, dtype=dtype)
    y, S = run(hd, X, B, C, dtype, packed=True)
    rows = np.r_[0:24, 8180:8200, w.N - 24:w.N, np.random.default_rng(3).integers(0, w.N, 40)]
    rep, _ = check_against_oracle(X, B, C, y, S, rows=rows)
    assert rep["ok"], rep


def test_colour_k100_all_rows(hd):
    """Colour shape with 100 classes, bf16, every one of the 16384 rows."""
    torch = torch_or_skip()
    w = hd_inputs.WORKLOADS["colour_k100"]
    assert hd.infer_kernel(w.N, w.F, w.D, w.K, torch.bfloat16) == "large_chunked_dma_kernel"
    announce("colour_k100 bf16 N=16384 (all rows)")
    X, B, C = inputs(w.N, w.F, w.D, w.K, w.x_dist, dtype="bf16")
    y, S = run(hd, X, B, C, "bf16", packed=True)
    rep = check_all_rows(X, B, C, y, S)
    announce(f"colour_k100 all rows: {rep}")
    assert rep["ok"], rep


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_activity_shape_largest_batch_sampled(hd, dtype):
    """The largest N of the samples/s curve (activity shape, N = 65536), sampled rows."""
    w = hd_inputs.WORKLOADS["activity_n32"]
    N = hd_inputs.N_SWEEP[-1]
    announce(f"activity shape {dtype} N={N}")
    X, B, C = inputs(N, w.F, w.D, w.K, w.x_dist, seed=5, dtype=dtype)
    y, S = run(hd, X, B, C, dtype, packed=True)
    rows = np.r_[0:16, 32760:32780, N - 16:N, np.random.default_rng(6).integers(0, N, 32)]
    rep, _ = check_against_oracle(X, B, C, y, S, rows=rows)
    assert rep["ok"], rep


@pytest.mark.parametrize("D", [hd_inputs.D_SWEEP[0], hd_inputs.D_SWEEP[-1]])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_colour_single_sample_d_sweep_ends(hd, D, dtype):
    """The single-sample bandwidth sweep (F = 3072, K = 10) at its smallest and largest D."""
    w = hd_inputs.WORKLOADS["colour_n1"]
    announce(f"colour_n1 {dtype} D={D}")
    X, B, C = inputs(w.N, w.F, D, w.K, w.x_dist, dtype=dtype)
    for packed in (False, True):
        y, S = run(hd, X, B, C, dtype, packed=packed)
        rep, _ = check_against_oracle(X, B, C, y, S)
        assert rep["ok"], (packed, rep)


# --- wide features: the X tile streamed through LDS in chunks ---------------

# (N, F, D, K, dtype, kernel): bf16 with F % 8 == 0 double-buffers the chunks
# through buffer-to-LDS loads; ragged F and fp32 stage them through registers.
CHUNKED = [(200, 3000, 300, 10, "bf16", "dma"), (130, 2999, 200, 7, "bf16", ""),
           (70, 2600, 130, 100, "bf16", "dma"), (150, 1300, 256, 5, "f32", ""),
           (90, 1283, 200, 40, "f32", ""), (65, 1500, 100, 70, "f32", ""),
           (257, 5000, 640, 3, "bf16", "dma"), (129, 2560, 64, 33, "bf16", "dma"),
           (300, 2568, 1000, 2, "bf16", "dma"), (66, 2602, 200, 50, "bf16", ""),
           (100, 3000, 200, 128, "bf16", "dma"), (97, 1400, 300, 128, "f32", "")]


@pytest.mark.parametrize("N,F,D,K,dtype,kind", CHUNKED)
def test_wide_features_chunked(hd, N, F, D, K, dtype, kind):
    torch = torch_or_skip()
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    want = "large_chunked_dma_kernel" if kind == "dma" else "large_chunked_kernel"
    assert hd.infer_kernel(N, F, D, K, tdt) == want
    announce(f"chunked {dtype} N={N} F={F} D={D} K={K}")
    X, B, C = inputs(N, F, D, K, "normal", seed=F + K, dtype=dtype)
    for packed in (False, True):
        y, S = run(hd, X, B, C, dtype, packed=packed)
        rep, _ = check_against_oracle(X, B, C, y, S)
        assert rep["ok"], (packed, rep)


@pytest.mark.parametrize("N,F,dtype", [(150, 2600, "bf16"), (150, 2598, "bf16"), (70, 1300, "f32")])
def test_wide_features_identity(hd, N, F, dtype):
    announce(f"chunked identity {dtype} N={N} F={F}")
    X, B, C = inputs(N, F, 500, 6, "normal", seed=9, dtype=dtype)
    y, S = run(hd, X, B, C, dtype, act="identity")
    rep, _ = check_against_oracle(X, B, C, y, S, act="identity")
    assert rep["ok"], rep


def test_wide_features_unaligned_x(hd):
    """X at an offset that is not 16-byte aligned takes the register-staged kernel."""
    torch = torch_or_skip()
    N, F, D, K = 130, 2600, 300, 5
    announce("chunked bf16 unaligned X")
    X, B, C = inputs(N, F, D, K, "normal", seed=11, dtype="bf16")
    Xd = dev(np.concatenate([np.zeros(1, np.float32), X.ravel()]), "bf16")[1:].view(N, F)
    Bd, Cd = dev(B, "bf16"), dev(C, "bf16")
    assert Xd.data_ptr() % 16 != 0
    y, S = hd.infer(Xd, Bd, Cd, return_scores=True)
    torch.cuda.synchronize()
    rep, _ = check_against_oracle(X, B, C, y.cpu().numpy(), S.cpu().numpy().astype(np.float64))
    assert rep["ok"], rep


# --- exactness on small-integer inputs --------------------------------------
# Small integers are exact in bf16 and fp32, and every partial sum stays below
# 2^24, so any summation order is exact: scores and labels must be
# bit-identical to the oracle's. The cases cover every kernel that serves a
# benchmark shape, and each asserts which kernel ran.

INTEGER = [
    # (N, F, D, K, dtype, packed, kernel)
    (1, 561, 10240, 6, "f32", False, "small_flat_kernel"),
    (1, 561, 10240, 6, "f32", True, "small_flat_kernel"),
    (32, 33, 1000, 5, "f32", False, "small_block_mfma_kernel"),
    (16, 561, 10240, 6, "f32", True, "small_frag_mfma_kernel"),
    (32, 561, 10240, 6, "f32", True, "small_frag_mfma_kernel"),
    # more than three column blocks per workgroup: the fragment kernel's B ring
    (32, 561, 20480, 6, "f32", True, "small_frag_mfma_kernel"),
    (24, 1000, 13000, 5, "f32", True, "small_frag_mfma_kernel"),
    (48, 300, 2048, 16, "f32", True, "small_frag_mfma_kernel"),
    (64, 200, 1000, 12, "f32", True, "small_frag_mfma_kernel"),
    (64, 561, 4096, 6, "f32", True, "small_frag_mfma_kernel"),  # two passes of 32 samples
    (50, 1000, 10240, 6, "f32", True, "small_frag_mfma_kernel"),  # two passes, ragged second
    # fewer blocks than workgroups on some XCDs (workgroups that own no block),
    # with two sample passes
    (64, 700, 1500, 6, "f32", True, "small_frag_mfma_kernel"),
    (33, 1000, 1500, 5, "f32", True, "small_frag_mfma_kernel"),
    (64, 561, 20480, 6, "f32", True, "small_mfma_kernel"),
    (64, 100, 2048, 17, "f32", False, "small_mfma_kernel"),
    (65, 100, 2048, 17, "f32", False, None),
    (300, 617, 4096, 26, "f32", False, "large_fused_kernel"),
    (300, 617, 4096, 26, "bf16", True, "large_fused_kernel"),
    (257, 31, 700, 3, "bf16", False, "large_fused_kernel"),
    (300, 784, 2048, 10, "bf16", True, "large_fused_kernel"),
    (32, 561, 2048, 6, "bf16", True, "small_frag_mfma_kernel"),
    (16, 561, 10240, 6, "bf16", True, "small_frag_mfma_kernel"),
    (40, 301, 1000, 16, "bf16", True, "small_frag_mfma_kernel"),
    (60, 1000, 1500, 5, "bf16", True, "small_frag_mfma_kernel"),  # two sample passes
    (32, 561, 2048, 17, "bf16", True, "large_fused_kernel"),
    (128, 561, 2048, 6, "bf16", True, "small_frag_mfma_kernel"),  # two 64-sample calls
    (250, 561, 2048, 6, "bf16", True, "small_frag_mfma_kernel"),  # four calls, the last ragged
    (4, 561, 2048, 6, "bf16", True, "small_flat_kernel"),
    # 4 < N <= 8 on a packed model: the fragment kernel with one partly used tile
    (5, 561, 2048, 6, "bf16", True, "small_frag_mfma_kernel"),
    (8, 561, 10240, 6, "f32", True, "small_frag_mfma_kernel"),
    (200, 3072, 1024, 10, "bf16", True, "large_chunked_dma_kernel"),
    (130, 2600, 512, 100, "bf16", False, "large_chunked_dma_kernel"),
    (200, 3072, 1024, 10, "f32", True, "large_chunked_kernel"),
    (150, 2999, 700, 5, "bf16", True, "large_chunked_kernel"),
]


@pytest.mark.parametrize("N,F,D,K,dtype,packed,kernel", INTEGER)
def test_integer_inputs_bit_exact(hd, N, F, D, K, dtype, packed, kernel):
    torch = torch_or_skip()
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    if kernel is not None:
        assert hd.infer_kernel(N, F, D, K, tdt, packed=packed) == kernel
    announce(f"integer {dtype} N={N} F={F} D={D} K={K} packed={packed} ({kernel})")
    X, B, C = hd_inputs.make_integer_inputs(N, F, D, K, seed=N + F)
    y, S = run(hd, X, B, C, dtype, packed=packed)
    ref = oracle.infer(X, B, C)
    assert np.array_equal(S, ref["S"]), np.abs(S - ref["S"]).max()
    assert np.array_equal(y, ref["y"])


# Inputs in {-1, 0, 1}: many v = 0 (HardSign ties to +1, Eq. 1) and duplicated
# class rows (argmax ties to the lowest index), on every benchmark kernel.
TIES = [
    (5, 40, 512, "f32", False, "small_flat_kernel"),
    (200, 40, 512, "f32", False, "small_mfma_kernel"),
    (300, 40, 512, "f32", False, "large_fused_kernel"),
    (300, 700, 512, "bf16", True, "large_fused_kernel"),
    (250, 700, 512, "bf16", True, "small_frag_mfma_kernel"),  # four 64-sample calls
    (5, 40, 512, "bf16", False, "small_flat_kernel"),
    (200, 40, 512, "bf16", False, "large_fused_kernel"),
    (32, 40, 512, "f32", True, "small_frag_mfma_kernel"),
    (64, 700, 4096, "f32", True, "small_frag_mfma_kernel"),  # two sample passes
    (64, 200, 1024, "f32", True, "small_frag_mfma_kernel"),
    (100, 2560, 512, "bf16", True, "large_chunked_dma_kernel"),
    (32, 40, 512, "bf16", True, "small_frag_mfma_kernel"),
    (100, 2560, 512, "f32", True, "large_chunked_kernel"),
    (100, 2561, 512, "bf16", False, "large_chunked_kernel"),
]


@pytest.mark.parametrize("N,F,D,dtype,packed,kernel", TIES)
def test_hardsign_zero_and_argmax_ties(hd, N, F, D, dtype, packed, kernel):
    torch = torch_or_skip()
    K = 6
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    assert hd.infer_kernel(N, F, D, K, tdt, packed=packed) == kernel
    announce(f"ties {dtype} N={N} F={F} D={D} packed={packed} ({kernel})")
    X, B, C = hd_inputs.make_integer_inputs(N, F, D, 4, seed=3, x_range=1, b_range=1)
    C = np.vstack([C, C[1:2], C[0:1]])
    y, S = run(hd, X, B, C, dtype, packed=packed)
    ref = oracle.infer(X, B, C, want_va=True)
    assert (ref["V"] == 0).any()
    assert (ref["S"][:, 4] == ref["S"][:, 1]).all() and (ref["S"][:, 5] == ref["S"][:, 0]).all()
    assert np.array_equal(S, ref["S"]) and np.array_equal(y, ref["y"])


# --- edge shapes --------------------------------------------------------------

EDGE = [(1, 1, 1, 1), (2, 2, 7, 2), (3, 5, 33, 1), (31, 17, 2047, 2), (33, 64, 10000, 6),
        (63, 1, 96, 3), (64, 561, 2048, 6), (65, 31, 100, 17), (100, 33, 1000, 33),
        (129, 200, 640, 100), (300, 16, 64, 64), (1000, 7, 129, 9), (65, 300, 200, 128)]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("N,F,D,K", EDGE)
def test_edge_shapes(hd, dtype, N, F, D, K):
    announce(f"edge {dtype} N={N} F={F} D={D} K={K}")
    X, B, C = inputs(N, F, D, K, "normal", seed=N * 7 + D, dtype=dtype)
    y, S = run(hd, X, B, C, dtype)
    rep, _ = check_against_oracle(X, B, C, y, S)
    assert rep["ok"], rep


def test_workspace_reused_across_shapes(hd):
    """One workspace, zeroed once, serves a raw large-batch call (which packs
    the model into it) and then small-batch calls: every call leaves it zero."""
    torch = torch_or_skip()
    F, D, K = 99, 2000, 12
    shapes = [(1000, "f32"), (4, "f32"), (40, "f32"), (300, "bf16"), (4, "bf16"), (1000, "f32")]
    need = 0
    for N, dt in shapes:
        tdt = torch.bfloat16 if dt == "bf16" else torch.float32
        need = max(need, hd.infer_workspace_bytes(N, F, D, K, tdt))
    ws = torch.zeros(need, dtype=torch.uint8, device="cuda")
    for i, (N, dt) in enumerate(shapes):
        announce(f"shared workspace N={N} {dt}")
        X, B, C = inputs(N, F, D, K, seed=20 + i, dtype=dt)
        y, S = hd.infer(dev(X, dt), dev(B, dt), dev(C, dt), return_scores=True, workspace=ws)
        torch.cuda.synchronize()
        rep, _ = check_against_oracle(X, B, C, y.cpu().numpy(), S.cpu().numpy())
        assert rep["ok"], (N, dt, rep)
        assert int(ws.count_nonzero()) == 0, (N, dt)


def test_unaligned_x_workspace_covers_plan(hd):
    """bf16 X that is not 16-byte aligned takes the register-staged chunked
    kernel, whose larger tiles split D more: the size query covers that plan
    (the bytes just past the workspace stay untouched) and the result is right."""
    torch = torch_or_skip()
    w = hd_inputs.WORKLOADS["colour_k10"]
    N, F, D, K = 8192, w.F, w.D, w.K
    announce(f"unaligned bf16 X N={N} F={F} K={K}")
    X, B, C = inputs(N, F, D, K, w.x_dist, seed=12, dtype="bf16")
    Xd = dev(np.concatenate([np.zeros(1, np.float32), X.ravel()]), "bf16")[1:].view(N, F)
    assert Xd.data_ptr() % 16 != 0
    model = hd.pack_model(dev(B, "bf16"), dev(C, "bf16"))
    need = int(hd.lib().hd_infer_packed_workspace_bytes(N, F, D, K, hd.HD_BF16))
    assert need > 0
    guard = 1 << 16
    buf = torch.zeros(need + guard, dtype=torch.uint8, device="cuda")
    buf[need:] = 0xA5
    labels = torch.empty(N, dtype=torch.int32, device="cuda")
    scores = torch.empty((N, K), dtype=torch.float32, device="cuda")
    hd.infer_packed(Xd, model, out=(labels, scores), workspace=buf[:need])
    torch.cuda.synchronize()
    assert bool((buf[need:] == 0xA5).all())
    assert int(buf[:need].count_nonzero()) == 0
    rows = np.r_[0:64, N - 64:N, np.random.default_rng(13).integers(0, N, 64)]
    rep, _ = check_against_oracle(X, B, C, labels.cpu().numpy(),
                                  scores.cpu().numpy().astype(np.float64), rows=rows)
    assert rep["ok"], rep


def test_empty_batch(hd):
    torch = torch_or_skip()
    X = torch.empty((0, 10), device="cuda")
    B = torch.randn(10, 64, device="cuda")
    C = torch.randn(3, 64, device="cuda")
    y = hd.infer(X, B, C)
    assert y.shape == (0,)


@pytest.mark.parametrize("N", [16, 500])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_identity_activation(hd, N, dtype):
    announce(f"identity {dtype} N={N}")
    X, B, C = inputs(N, 50, 777, 5, "normal", seed=4, dtype=dtype)
    y, S = run(hd, X, B, C, dtype, act="identity")
    rep, _ = check_against_oracle(X, B, C, y, S, act="identity")
    assert rep["ok"], rep


@pytest.mark.parametrize("N", [8, 300])
def test_labels_without_scores_and_repeat(hd, N):
    """scores = NULL writes labels only; repeated calls on one workspace
    (self-cleaning accumulators and tickets) give the same labels."""
    announce(f"no-scores N={N}")
    X, B, C = inputs(N, 61, 3000, 7, seed=5)
    y0, _ = run(hd, X, B, C, "f32", scores=False)
    ref = oracle.infer(X, B, C, want_va=True)
    rep = compare(None, y0, ref, C, 61, RTOL)
    assert rep["ok"], rep
    for _ in range(5):
        y1, _ = run(hd, X, B, C, "f32", scores=False)
        assert np.array_equal(y0, y1)


@pytest.mark.parametrize("N", [4, 1000])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_packed_model_matches_raw(hd, N, dtype):
    announce(f"packed {dtype} N={N}")
    X, B, C = inputs(N, 99, 2000, 12, seed=6, dtype=dtype)
    y0, S0 = run(hd, X, B, C, dtype)
    y1, S1 = run(hd, X, B, C, dtype, packed=True)
    assert np.array_equal(y0, y1)
    if N > 64:
        assert np.array_equal(S0, S1)  # the large-batch path is deterministic
    else:
        # the small-batch path sums partial scores with fp32 atomics, so the
        # order (and the last bits) can change between calls
        assert np.all(np.abs(S0 - S1) <= RTOL * score_scale(C)[None, :])


# Packed model on the small-batch path against the oracle, covering every
# small kernel: the flat kernel on the column tiles (N <= 8, one and several
# f-chunks), the fragment matrix-core kernel (fp32, N > 8: one to four sample
# tiles, every rows-per-lane size, rows that wrap inside a float4 of X), the
# persistent matrix-core kernel where the fragment kernel's LDS does not fit,
# and the fragment kernel on bf16 models (fp32 fragments, X and C widened).
PACKED_SMALL = [(1, 561, 10240, 6, "f32"), (3, 20, 1000, 4, "f32"), (8, 1100, 777, 9, "f32"),
                (7, 300, 2050, 3, "bf16"), (9, 64, 1000, 5, "f32"), (32, 561, 10240, 6, "f32"),
                (64, 561, 4096, 6, "f32"), (40, 130, 3000, 100, "f32"), (20, 90, 1000, 7, "bf16"),
                (64, 1500, 513, 3, "bf16"), (17, 900, 333, 2, "f32"), (64, 200, 1000, 3, "f32"),
                (12, 5, 64, 3, "f32"), (16, 4, 100, 2, "f32"), (48, 700, 2000, 26, "f32"),
                (24, 300, 1000, 16, "f32"), (10, 100, 500, 13, "f32"),
                (32, 561, 10240, 6, "bf16"), (16, 1023, 999, 16, "bf16"), (9, 5, 64, 2, "bf16"),
                # more than three column blocks per workgroup (the B ring)
                (32, 561, 20480, 6, "f32"), (20, 1000, 16000, 3, "f32"),
                (16, 300, 16384, 10, "bf16"),
                # two passes of 32 samples (X of all samples exceeds LDS)
                (64, 561, 10240, 6, "f32"), (37, 900, 8000, 11, "f32"),
                (64, 561, 10240, 6, "bf16"), (45, 700, 3000, 16, "bf16"),
                # 64-sample calls of a packed bf16 model up to 128 samples
                (100, 561, 4096, 6, "bf16"), (65, 300, 2000, 10, "bf16"),
                # bf16 rows long enough for two sample passes
                (64, 1000, 2000, 6, "bf16")]


@pytest.mark.parametrize("N,F,D,K,dtype", PACKED_SMALL)
def test_packed_small_path(hd, N, F, D, K, dtype):
    announce(f"packed small {dtype} N={N} F={F} D={D} K={K}")
    X, B, C = inputs(N, F, D, K, "uniform_pm1", seed=N + D, dtype=dtype)
    y, S = run(hd, X, B, C, dtype, packed=True)
    rep, _ = check_against_oracle(X, B, C, y, S)
    assert rep["ok"], rep


# --- the stages alone -----------------------------------------------------------

@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_encode_then_similarity(hd, dtype):
    torch = torch_or_skip()
    announce(f"encode/similarity {dtype}")
    X, B, C = inputs(70, 120, 1500, 9, seed=7, dtype=dtype)
    Xd, Bd, Cd = dev(X, dtype), dev(B, dtype), dev(C, dtype)
    H = hd.encode(Xd, Bd)
    y, S = hd.similarity(H, Cd, return_scores=True)
    torch.cuda.synchronize()
    ref = oracle.infer(X, B, C, want_va=True)
    from tolerance import encode_allowed_mismatch
    ok, bad, flips = encode_allowed_mismatch(H.cpu().numpy(), ref, 120)
    assert ok, (bad, flips)
    rep = compare(S.cpu().numpy(), y.cpu().numpy(), ref, C, 120, RTOL)
    assert rep["ok"], rep
    # Stage II alone on the GPU's own H against the oracle's Stage II on it
    Hn = H.cpu().numpy().astype(np.float64)
    r2 = oracle.similarity(Hn, C)
    assert np.all(np.abs(S.cpu().numpy() - r2["S"]) <= RTOL * score_scale(C)[None, :])
    # identity encoding
    Hi = hd.encode(Xd, Bd, act="identity").cpu().numpy()
    ok, bad, _ = encode_allowed_mismatch(Hi, ref, 120, act="identity")
    assert ok, bad
