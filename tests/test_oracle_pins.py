"""The oracle against its pins (CPU only)."""
import numpy as np
import pytest

import hd_inputs
import oracle
from pins import PINS


@pytest.mark.parametrize("pin", PINS, ids=[p.__name__ for p in PINS])
def test_pin(pin):
    pin(oracle.default())


def test_inputs_deterministic_and_shaped():
    a = hd_inputs.make_inputs(3, 5, 7, 2, seed=1)
    b = hd_inputs.make_inputs(3, 5, 7, 2, seed=1)
    for u, v in zip(a, b):
        assert np.array_equal(u, v) and u.dtype == np.float32
    assert a[0].shape == (3, 5) and a[1].shape == (5, 7) and a[2].shape == (2, 7)
    # B and C do not depend on N
    c = hd_inputs.make_inputs(9, 5, 7, 2, seed=1)
    assert np.array_equal(a[1], c[1]) and np.array_equal(a[2], c[2])


def test_bf16_rounding_matches_torch():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(10000).astype(np.float32) * 1e3,
                        np.array([0.0, -0.0, 1.0, 1.00390625, 1.01171875, 3.4e38, -1e-40],
                                 np.float32)])
    ours = hd_inputs.bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)


def test_image_workload_zero_fraction():
    X = hd_inputs.make_x(512, 784, "uniform01_zero20", seed=0)
    frac = float(np.mean(X == 0.0))
    assert 0.18 < frac < 0.22
    assert X.min() >= 0.0 and X.max() < 1.0


def test_tolerance_rule_self_check():
    """The comparison rule accepts the oracle against itself, accepts a flip
    inside the fragile set and rejects a flip outside it."""
    from tolerance import compare, gamma
    X, B, C = hd_inputs.make_inputs(4, 50, 256, 5, seed=2)
    ref = oracle.infer(X, B, C, want_va=True)
    assert compare(ref["S"], ref["y"], ref, C, 50, 1e-4)["ok"]
    # flip one dimension: outside the fragile set this must be rejected
    n, d = 1, int(np.argmax(np.abs(ref["V"][1])))
    S_bad = ref["S"].copy()
    S_bad[n] -= 2.0 * np.sign(ref["V"][n, d]) * C[:, d]
    rep = compare(S_bad, ref["y"], ref, C, 50, 1e-4)
    assert not rep["score_ok"]
    # a fragile dimension (force it by shrinking v) is allowed to flip
    ref2 = dict(ref)
    ref2["V"] = ref["V"].copy()
    ref2["V"][n, d] = 0.5 * gamma(50) * ref["A"][n, d]
    assert compare(S_bad, ref["y"], ref2, C, 50, 1e-4)["score_ok"]
