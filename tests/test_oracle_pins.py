"""The oracle against what the paper and the mathematics fix (CPU only)."""
import os
import shutil
import subprocess
import tempfile

import pytest

import oracle
from tests import pins


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda p: p.__name__)
def test_pin(orc, pin):
    pin(orc)


# Plausible mistakes, each planted into a copy of the oracle's source.  Every
# one must make at least one pin fail, which shows the pins can tell.
MUTANTS = {
    "pseudo_value_drops_beta": ("vt[r] = beta * (v[r] - alpha * Pk);", "vt[r] = (v[r] - alpha * Pk);"),
    "pseudo_value_drops_alpha": ("vt[r] = beta * (v[r] - alpha * Pk);", "vt[r] = beta * (v[r] - Pk);"),
    "erase_sign_flipped": ("alpha * (Pr[c] - beta * Pk * k[c])", "alpha * (Pr[c] + beta * Pk * k[c])"),
    "write_term_dropped": ("+ beta * v[r] * k[c];", ";"),
    "write_term_decayed": ("alpha * (Pr[c] - beta * Pk * k[c]) + beta * v[r] * k[c]",
                           "alpha * (Pr[c] - beta * Pk * k[c] + beta * v[r] * k[c])"),
    "output_from_parent_state": ("acc += Sr[c] * q[c];", "acc += Pr[c] * q[c];"),
    "output_uses_key": ("acc += Sr[c] * q[c];", "acc += Sr[c] * k[c];"),
    "state_transposed_in_matvec": ("Pk += Pr[c] * k[c];", "Pk += P[(size_t)c * dk + r] * k[c];"),
    "parent_taken_as_previous_node": ("const double *P = (p < 0) ? S0u : St + (size_t)p * SS;",
                                      "const double *P = (t == 0) ? S0u : St + (size_t)(t - 1) * SS;"),
    "commit_skips_last_node": ("for (int l = 0; l < path_len[u]; ++l) {",
                               "for (int l = 0; l + 1 < path_len[u]; ++l) {"),
}


@pytest.fixture(scope="module")
def mutant_dir():
    d = tempfile.mkdtemp(prefix="oracle_mutants_")
    yield d
    shutil.rmtree(d, ignore_errors=True)


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_planted_mistake(mutant_dir, name):
    old, new = MUTANTS[name]
    src = open(oracle.SOURCE).read()
    assert src.count(old) >= 1, "mutation site vanished: %s" % name
    path = os.path.join(mutant_dir, name + ".c")
    with open(path, "w") as f:
        f.write(src.replace(old, new))
    lib = oracle.build(src=path, out=os.path.join(mutant_dir, name + ".so"))
    bad = oracle.Oracle(lib)
    caught = []
    for pin in pins.ALL_PINS:
        try:
            pin(bad)
        except (AssertionError, oracle.OracleError, ValueError, IndexError):
            caught.append(pin.__name__)
    assert caught, "no pin catches mutant %s" % name
