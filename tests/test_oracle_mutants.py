"""Plant plausible mistakes in copies of the oracle (on the CPU) and check
that every one of them trips at least one pin. The real oracle is untouched:
each mutant is compiled from a patched copy into a temporary directory."""
import os
import shutil
import subprocess

import pytest

import oracle
from oracle import build as obuild
from pins import PINS

MUTANTS = {
    "hardsign_tie_to_minus": ("return (x >= 0.0) ? 1.0 : -1.0;", "return (x > 0.0) ? 1.0 : -1.0;"),
    "hardsign_zero_level": ("return (x >= 0.0) ? 1.0 : -1.0;", "return (x >= 0.0) ? 1.0 : 0.0;"),
    "dropped_first_feature": ("for (int64_t f = 0; f < F; ++f) {", "for (int64_t f = 1; f < F; ++f) {"),
    "dropped_last_dim_in_score": ("for (int64_t d = 0; d < D; ++d) acc += h[d] * ck[d];",
                                  "for (int64_t d = 0; d < D - 1; ++d) acc += h[d] * ck[d];"),
    "argmax_last_tie": ("if (k > 0 && acc > s[best])", "if (k > 0 && acc >= s[best])"),
    "transposed_base": ("for (int64_t d = 0; d < D; ++d) v[d] += xf * bf[d];",
                        "for (int64_t d = 0; d < D; ++d) v[d] += xf * B[d * F + f];"),
    "wrong_sign_bundle": ("for (int64_t d = 0; d < D; ++d) v[d] += xf * bf[d];",
                          "for (int64_t d = 0; d < D; ++d) v[d] -= xf * bf[d];"),
    "wrong_class_row": ("acc += h[d] * ck[d];", "acc += h[d] * C[d];"),
    "sample_stride": ("encode_sample(X + n * F, B, F, D, v, A ? a : NULL);\n        for (int64_t d = 0; d < D; ++d) h[d]",
                      "encode_sample(X + (n > 0 ? n - 1 : 0) * F, B, F, D, v, A ? a : NULL);\n        for (int64_t d = 0; d < D; ++d) h[d]"),
}


@pytest.fixture(scope="module")
def workdir(tmp_path_factory):
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    return tmp_path_factory.mktemp("mutants")


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, workdir):
    old, new = MUTANTS[name]
    src = open(obuild.SRC).read()
    assert src.count(old) >= 1, f"mutation site for {name} not found"
    msrc = os.path.join(workdir, f"{name}.c")
    mlib = os.path.join(workdir, f"lib{name}.so")
    with open(msrc, "w") as fh:
        fh.write(src.replace(old, new, 1))
    try:
        obuild.build(src=msrc, lib=mlib)
    except subprocess.CalledProcessError:
        pytest.fail(f"mutant {name} did not compile")
    orc = oracle.Oracle(mlib)
    caught = []
    for pin in PINS:
        try:
            pin(orc)
        except (AssertionError, RuntimeError, ValueError, IndexError):
            caught.append(pin.__name__)
    assert caught, f"mutant {name} passed every pin"
