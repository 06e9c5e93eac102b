"""CPU tests: the oracle against its pins, and mutants of the oracle against
the same pins (each planted mistake must be caught by at least one pin)."""
import os
import subprocess

import numpy as np
import pytest

import oracle
from tests import oracle_pins

ORACLE_SRC = os.path.join(os.path.dirname(oracle.__file__), "oracle.c")


@pytest.fixture(scope="module")
def lib():
    return oracle._load()


@pytest.mark.parametrize("pin", oracle_pins.ALL_PINS, ids=lambda p: p.__name__)
def test_pin(pin, lib):
    pin(lib)


# (description, exact text in oracle.c, replacement)
MUTANTS = [
    ("dropped last k term", "for (int64_t k = 0; k < K; ++k) {\n            const float a",
     "for (int64_t k = 0; k + 1 < K; ++k) {\n            const float a"),
    ("sign flip in accumulate", "c[j] = c[j] + a * b[j];", "c[j] = c[j] - a * b[j];"),
    ("accumulator not zeroed", "for (int64_t j = 0; j < N; ++j) c[j] = 0.0f;",
     "for (int64_t j = 0; j < N; ++j) c[j] = 1e-3f;"),
    ("transposed B in entries", "B[k * ldb + cols[t]]", "B[cols[t] * ldb + k]"),
    ("wrong row of A in entries", "A[rows[t] * lda + k]", "A[cols[t] * lda + k]"),
    ("slot index used as rank offset", "((int64_t)rank * N_local + j)", "((int64_t)s * N_local + j)"),
    ("own slot skipped", "float* g = G + (int64_t)s * M * ldg;",
     "if (s == rank) continue;\n        float* g = G + (int64_t)s * M * ldg;"),
    ("row stride of gathered taken as N_local", "const int64_t ldg = (int64_t)world * N_local;",
     "const int64_t ldg = N_local + 0 * world;"),
    ("flag index swapped", "(((int64_t)s * world + rank) * tiles_m + m)",
     "(((int64_t)rank * world + s) * tiles_m + m)"),
    ("flag published to one slot only", "for (int s = 0; s < world; ++s)\n        for (int64_t m = 0; m < tiles_m; ++m)",
     "for (int s = rank; s < rank + 1; ++s)\n        for (int64_t m = 0; m < tiles_m; ++m)"),
    ("bf16 decode shift", "((uint32_t)h) << 16", "((uint32_t)h) << 15"),
    ("f16 exponent rebias", "((e + 112u) << 23)", "((e + 111u) << 23)"),
    ("f16 subnormal exponent", "(uint32_t)(113 - shift) << 23", "(uint32_t)(112 - shift) << 23"),
    ("f16 sign dropped", "uint32_t sign = (uint32_t)(h >> 15) & 1u;", "uint32_t sign = 0u * h;"),
    ("copy ring reversed", "((r + shift) % world + world) % world", "((r - shift) % world + world) % world"),
    ("get reads its own slot", "const int src = get ? ((r - shift) % world + world) % world : r;",
     "const int src = r;"),
    ("get writes the peer", "const int dst = get ? r : ((r + shift) % world + world) % world;",
     "const int dst = ((r + shift) % world + world) % world;"),
    ("copy ragged tile edge dropped", "i < rows && i < (tr + 1) * tile_r", "i + 1 < rows && i < (tr + 1) * tile_r"),
    ("copy flag on source slot", "copyflag[(int64_t)dst * tiles_r * tiles_c", "copyflag[(int64_t)r * tiles_r * tiles_c"),
]


def test_mutants_cover_source():
    src = open(ORACLE_SRC).read()
    for desc, old, _ in MUTANTS:
        assert src.count(old) == 1, f"mutation anchor for '{desc}' not unique in oracle.c"


@pytest.mark.parametrize("mutant", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(mutant, tmp_path):
    desc, old, new = mutant
    src = open(ORACLE_SRC).read().replace(old, new)
    c = tmp_path / "mutant.c"
    c.write_text(src)
    so = tmp_path / "libmutant.so"
    oracle.build(str(c), str(so))
    lib = oracle.load_library(str(so))
    caught = []
    for pin in oracle_pins.ALL_PINS:
        try:
            with np.errstate(all="ignore"):
                pin(lib)
        except (AssertionError, ValueError, IndexError):
            caught.append(pin.__name__)
    assert caught, f"no pin catches the mutant '{desc}'"
