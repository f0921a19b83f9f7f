"""The oracle's single-pass training against its pins, and planted mistakes
in copies of the oracle that the pins must catch."""
import os
import shutil
import subprocess

import pytest

import oracle
from oracle import build as obuild
from pins_train import TRAIN_PINS


@pytest.mark.parametrize("pin", TRAIN_PINS, ids=lambda p: p.__name__)
def test_train_pin(pin):
    pin(oracle.default())


MUTANTS = {
    "codebook_tie_to_minus": ("M[i] = hardsign((double)counts[i]);",
                              "M[i] = counts[i] > 0 ? 1.0 : -1.0;"),
    "bundles_unnormalised_encoding": ("h[(n - n0) * D + d] = hardsign(v[d]);",
                                      "h[(n - n0) * D + d] = v[d];"),
    "label_off_by_one": ("if (k < 0 || k >= K) continue;",
                         "if (k < 0 || k + 1 >= K) continue;"),
    "last_sample_dropped": ("for (int64_t n = n0; n < n1; ++n) {\n      const int32_t k = y[n];",
                            "for (int64_t n = n0; n + 1 < n1; ++n) {\n      const int32_t k = y[n];"),
    "wrong_row": ("counts[k * D + d] +=", "counts[(k * D + d) % (K * D > D ? K * D - D : 1)] +="),
}


@pytest.fixture(scope="module")
def workdir(tmp_path_factory):
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    return tmp_path_factory.mktemp("train_mutants")


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_train_mutant_is_caught(name, workdir):
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
    for pin in TRAIN_PINS:
        try:
            pin(orc)
        except (AssertionError, RuntimeError, ValueError, IndexError):
            caught.append(pin.__name__)
    assert caught, f"mutant {name} passed every pin"
