"""GPU: the deterministic mode (HD_DETERMINISTIC). Repeated calls give
bit-identical scores and labels on every small-batch kernel (whose default
mode sums partial scores with fp32 atomics in arrival order) and on the
large-batch path; the results stay within the oracle rule, are bit-exact on
integer inputs, and leave the workspace reusable by either mode."""
import numpy as np
import pytest

import hd_inputs
import oracle
from gpu_util import RTOL, announce, check_against_oracle, dev, torch_or_skip

pytestmark = pytest.mark.gpu

REPEATS = 20


@pytest.fixture(scope="module")
def hd():
    torch_or_skip()
    import paper_2506_09282_amd as hd
    hd.lib()
    return hd


# (N, F, D, K, dtype, packed, kernel): every small-batch kernel, the chunked
# small route and both large-batch kernels.
CASES = [
    (1, 561, 10240, 6, "f32", False, "small_flat_kernel"),
    (4, 561, 2048, 6, "bf16", True, "small_flat_kernel"),
    (16, 33, 1000, 5, "f32", False, "small_block_mfma_kernel"),
    (16, 3072, 1000, 5, "f32", False, "small_valu_kernel"),
    (64, 33, 1000, 5, "f32", False, "small_mfma_kernel"),
    (32, 561, 10240, 6, "f32", True, "small_frag_mfma_kernel"),
    (64, 617, 10240, 26, "f32", True, "small_valu_kernel"),
    (200, 561, 10240, 6, "f32", True, "small_frag_mfma_kernel"),  # 64-sample calls, two passes
    (32, 561, 10240, 6, "bf16", True, "small_frag_mfma_kernel"),
    (16, 617, 4096, 26, "bf16", True, "large_fused_kernel"),
    (16, 3072, 1000, 5, "bf16", False, "large_chunked_dma_kernel"),
    (32, 561, 20480, 6, "f32", True, "small_frag_mfma_kernel"),  # the fragment kernel's B ring
]
# the small-batch cases (integer inputs are exact for them in any order)
SMALL_CASES = CASES[:9] + CASES[11:]


def run(hd, Xd, Bd, Cd, packed, det, model=None):
    if packed:
        return hd.infer_packed(Xd, model, return_scores=True, deterministic=det)
    return hd.infer(Xd, Bd, Cd, return_scores=True, deterministic=det)


@pytest.mark.parametrize("N,F,D,K,dtype,packed,kernel", CASES)
def test_deterministic_repeats_bit_identical(hd, N, F, D, K, dtype, packed, kernel):
    torch = torch_or_skip()
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    assert hd.infer_kernel(min(N, 64), F, D, K, tdt, packed=packed) == kernel
    announce(f"deterministic {kernel} {dtype} N={N} F={F} D={D} K={K} packed={packed}")
    X, B, C = hd_inputs.make_inputs(N, F, D, K, "uniform_pm1", seed=N + K, dtype=dtype)
    Xd, Bd, Cd = dev(X, dtype), dev(B, dtype), dev(C, dtype)
    model = hd.pack_model(Bd, Cd) if packed else None
    y0, S0 = run(hd, Xd, Bd, Cd, packed, True, model)
    for i in range(REPEATS):
        # interleave default-mode calls on the same cached workspace
        run(hd, Xd, Bd, Cd, packed, False, model)
        y, S = run(hd, Xd, Bd, Cd, packed, True, model)
        torch.cuda.synchronize()
        assert torch.equal(y, y0), i
        assert torch.equal(S, S0), i
    rep, _ = check_against_oracle(X, B, C, y0.cpu().numpy(), S0.cpu().numpy().astype(np.float64),
                                  rtol=RTOL)
    assert rep["ok"], rep


@pytest.mark.parametrize("N,F,D,K,dtype,packed,kernel", SMALL_CASES)
def test_deterministic_integer_bit_exact(hd, N, F, D, K, dtype, packed, kernel):
    """Small integers: every sum is exact in any order, so the fixed-order
    reduction must reproduce the oracle bit for bit."""
    torch = torch_or_skip()
    announce(f"deterministic integer {kernel} N={N}")
    X, B, C = hd_inputs.make_integer_inputs(N, F, D, K, seed=N + F)
    Xd, Bd, Cd = dev(X, dtype), dev(B, dtype), dev(C, dtype)
    model = hd.pack_model(Bd, Cd) if packed else None
    y, S = run(hd, Xd, Bd, Cd, packed, True, model)
    torch.cuda.synchronize()
    ref = oracle.infer(X, B, C)
    assert np.array_equal(S.cpu().numpy().astype(np.float64), ref["S"])
    assert np.array_equal(y.cpu().numpy(), ref["y"])


def test_deterministic_noalloc(hd):
    torch = torch_or_skip()
    N, F, D, K = 32, 561, 10240, 6
    X, B, C = hd_inputs.make_inputs(N, F, D, K, "uniform_pm1", seed=2)
    Xd = dev(X, "f32")
    model = hd.pack_model(dev(B, "f32"), dev(C, "f32"))
    y0, S0 = hd.infer_packed_noalloc(Xd, model, return_scores=True, deterministic=True)
    y1, S1 = hd.infer_packed(Xd, model, return_scores=True, deterministic=True)
    for _ in range(5):
        y2, S2 = hd.infer_packed_noalloc(Xd, model, return_scores=True, deterministic=True)
        torch.cuda.synchronize()
        assert torch.equal(S2, S0) and torch.equal(y2, y0)
    assert torch.equal(S1, S0) and torch.equal(y1, y0)
