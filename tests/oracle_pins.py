"""Pins of the oracle to facts that do not come from the oracle itself.

Each ``pin_*`` takes a loaded oracle library (``oracle.load_library``) and
raises ``AssertionError`` when the oracle disagrees with:

* hand-written values (``tests/golden``: IEEE 16-bit formats, a worked
  gathered-placement example),
* an independent library routine (numpy/torch dtype conversion, numpy
  float64 matmul), or pure-Python float64 brute force on tiny inputs,
* closed forms (identity and one-hot operands, all-ones, small integers whose
  sums are exact in binary32),
* invariants of the gathered layout and of the arrival counters.

The same pins run against deliberately broken copies of ``oracle.c`` in
``test_oracle.py`` to show that each plausible mistake is caught.
"""
from __future__ import annotations

import json
import math
import os
import random

import numpy as np
import torch

import oracle

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
U32 = 2.0 ** -24          # unit roundoff of binary32


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _fp32_sum_bound(A64: np.ndarray, B64: np.ndarray) -> np.ndarray:
    """Forward error bound of a K-term binary32 dot product with exact
    products (16-bit inputs): gamma_{K} * sum |a||b| (Higham, Thm 3.1)."""
    K = A64.shape[1]
    g = K * U32 / (1.0 - K * U32) if K else 0.0
    return g * (np.abs(A64) @ np.abs(B64)) + 1e-30


def _rand_bits(rng: np.random.Generator, shape, dtype: str) -> np.ndarray:
    """Finite random 16-bit patterns of moderate magnitude via torch rounding."""
    x = torch.from_numpy(rng.uniform(-2.0, 2.0, size=shape).astype(np.float32))
    t = x.to(torch.float16 if dtype == "f16" else torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def _to_f64(bits: np.ndarray, dtype: str) -> np.ndarray:
    """Independent widening through torch (a library routine)."""
    t = torch.from_numpy(bits.view(np.int16).copy())
    t = t.view(torch.float16 if dtype == "f16" else torch.bfloat16)
    return t.to(torch.float64).numpy()


# ---------------------------------------------------------------- formats

def pin_decode_golden(lib):
    g = _golden("float16_formats.json")
    for dtype in ("f16", "bf16"):
        pats = np.array([int(h, 16) for h, _ in g[dtype]], dtype=np.uint16)
        want = [float(v) for _, v in g[dtype]]
        got = oracle.decode16(pats, dtype, lib)
        for h, w, x in zip(pats, want, got):
            if math.isnan(w):
                assert math.isnan(x), (dtype, hex(h))
            else:
                assert float(x) == w and math.copysign(1, x) == math.copysign(1, w), \
                    (dtype, hex(h), w, float(x))


def pin_decode_all_patterns(lib):
    pats = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    for dtype in ("f16", "bf16"):
        got = oracle.decode16(pats, dtype, lib)
        ref = _to_f64(pats, dtype).astype(np.float32)
        nan = np.isnan(ref)
        assert np.array_equal(np.isnan(got), nan), dtype
        assert np.array_equal(got[~nan].view(np.uint32), ref[~nan].view(np.uint32)), dtype


# ---------------------------------------------------------------- GEMM

def pin_gemm_bruteforce_tiny(lib):
    rng = np.random.default_rng(11)
    pyr = random.Random(5)
    for trial in range(12):
        M, N, K = pyr.randint(1, 7), pyr.randint(1, 7), pyr.randint(1, 9)
        dtype = "f16" if trial % 2 else "bf16"
        Ab, Bb = _rand_bits(rng, (M, K), dtype), _rand_bits(rng, (K, N), dtype)
        A64, B64 = _to_f64(Ab, dtype), _to_f64(Bb, dtype)
        C = oracle.gemm(oracle.decode16(Ab, dtype, lib), oracle.decode16(Bb, dtype, lib), lib)
        for i in range(M):
            for j in range(N):
                exact = 0.0
                mag = 0.0
                for k in range(K):
                    exact += A64[i, k] * B64[k, j]
                    mag += abs(A64[i, k] * B64[k, j])
                bound = K * U32 / (1 - K * U32) * mag + 1e-30
                assert abs(float(C[i, j]) - exact) <= bound, (trial, i, j, C[i, j], exact)


def pin_gemm_numpy_f64(lib):
    rng = np.random.default_rng(12)
    for (M, N, K, dtype) in ((130, 70, 93, "bf16"), (65, 129, 257, "f16"), (3, 200, 1, "f16")):
        Ab, Bb = _rand_bits(rng, (M, K), dtype), _rand_bits(rng, (K, N), dtype)
        A64, B64 = _to_f64(Ab, dtype), _to_f64(Bb, dtype)
        C = oracle.gemm(oracle.decode16(Ab, dtype, lib), oracle.decode16(Bb, dtype, lib), lib)
        err = np.abs(C.astype(np.float64) - A64 @ B64)
        assert np.all(err <= _fp32_sum_bound(A64, B64)), (M, N, K, float(err.max()))


def pin_gemm_identity(lib):
    rng = np.random.default_rng(13)
    for n in (1, 17, 64):
        B = oracle.decode16(_rand_bits(rng, (n, 33), "bf16"), "bf16", lib)
        C = oracle.gemm(np.eye(n, dtype=np.float32), B, lib)
        assert np.array_equal(C.view(np.uint32), B.view(np.uint32)), n


def pin_gemm_onehot(lib):
    rng = np.random.default_rng(14)
    A = oracle.decode16(_rand_bits(rng, (40, 50), "f16"), "f16", lib)
    sel = rng.integers(0, 50, size=23)
    B = np.zeros((50, 23), dtype=np.float32)
    B[sel, np.arange(23)] = 1.0
    C = oracle.gemm(A, B, lib)
    assert np.array_equal(C, A[:, sel])


def pin_gemm_all_ones(lib):
    ones = np.full((128, 256), 0x3C00, dtype=np.uint16)   # binary16 1.0
    A = oracle.decode16(ones, "f16", lib)
    B = oracle.decode16(np.full((256, 64), 0x3C00, dtype=np.uint16), "f16", lib)
    C = oracle.gemm(A, B, lib)
    assert np.all(C == 256.0)


def pin_gemm_small_integers(lib):
    rng = np.random.default_rng(15)
    A = rng.integers(-4, 5, size=(37, 200))
    B = rng.integers(-4, 5, size=(200, 45))
    C = oracle.gemm(A.astype(np.float32), B.astype(np.float32), lib)
    assert np.array_equal(C.astype(np.int64), A @ B)     # |sums| <= 3200 < 2^24


def pin_gemm_entries(lib):
    rng = np.random.default_rng(16)
    Ab, Bb = _rand_bits(rng, (90, 300), "bf16"), _rand_bits(rng, (300, 77), "bf16")
    A, B = oracle.decode16(Ab, "bf16", lib), oracle.decode16(Bb, "bf16", lib)
    rows = rng.integers(0, 90, size=200)
    cols = rng.integers(0, 77, size=200)
    got = oracle.gemm_entries(A, B, rows, cols, lib)
    A64, B64 = _to_f64(Ab, "bf16"), _to_f64(Bb, "bf16")
    exact = np.einsum("tk,kt->t", A64[rows], B64[:, cols])
    bound = _fp32_sum_bound(A64, B64)[rows, cols]
    assert np.all(np.abs(got - exact) <= bound)
    full = oracle.gemm(A, B, lib)
    assert np.array_equal(got.view(np.uint32), full[rows, cols].view(np.uint32))


# ---------------------------------------------------------------- placement

def _bits_of_ints(x, dtype):
    t = torch.tensor(x, dtype=torch.float32).to(
        torch.float16 if dtype == "f16" else torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def pin_placement_golden(lib):
    g = _golden("gathered_placement.json")
    for case in g["cases"]:
        w, M, N = case["world"], case["M"], case["N_local"]
        st = oracle.GatheredState(w, M, N, case["tile_m"], case["tile_n"])
        A = _bits_of_ints(case["A"], "f16")
        order = [0] if "after_rank0_each_slot" in case else [1]
        partial = case.get("after_rank0_each_slot", case.get("after_rank1_each_slot"))
        for r in order:
            C = oracle.gemm_all_scatter(st, A, _bits_of_ints(case["B_shards"][r], "f16"),
                                        "f16", r, lib)
            assert np.array_equal(C, np.array(case["C_blocks"][r], dtype=np.float32))
        for s in range(w):
            for i in range(M):
                for j in range(w * N):
                    want = partial[i][j]
                    if want == "S":
                        assert st.written[s, i, j] == 0 and np.isnan(st.G[s, i, j]), (s, i, j)
                    else:
                        assert st.written[s, i, j] == 1 and st.G[s, i, j] == want, (s, i, j)
        r0 = order[0]
        expect = np.zeros_like(st.arrived)
        expect[:, r0] = 1
        assert np.array_equal(st.arrived, expect)
        for r in range(w):
            if r not in order:
                oracle.gemm_all_scatter(st, A, _bits_of_ints(case["B_shards"][r], "f16"),
                                        "f16", r, lib)
        full = np.array(case["after_all_ranks_each_slot"], dtype=np.float32)
        for s in range(w):
            assert np.array_equal(st.G[s], full), s
        assert np.all(st.written == 1) and np.all(st.arrived == 1)


def pin_gathered_identity(lib):
    """All ranks in turn: every slot equals A @ [B_0 | ... | B_{w-1}]."""
    rng = np.random.default_rng(17)
    w, M, N, K, dtype = 4, 70, 24, 40, "bf16"
    st = oracle.GatheredState(w, M, N, 32, 16)
    Ab = _rand_bits(rng, (M, K), dtype)
    shards = [_rand_bits(rng, (K, N), dtype) for _ in range(w)]
    for r in (2, 0, 3, 1):
        oracle.gemm_all_scatter(st, Ab, shards[r], dtype, r, lib)
    A64 = _to_f64(Ab, dtype)
    Bcat = np.concatenate([_to_f64(b, dtype) for b in shards], axis=1)
    exact = A64 @ Bcat
    bound = _fp32_sum_bound(A64, Bcat)
    for s in range(w):
        assert np.all(np.abs(st.G[s].astype(np.float64) - exact) <= bound), s
        assert np.array_equal(st.G[s].view(np.uint32), st.G[0].view(np.uint32))
    assert np.all(st.written == 1)
    assert np.all(st.arrived == 1) and st.arrived.shape == (w, w, 3, 2)


def pin_single_rank_footprint(lib):
    """One call writes exactly the rank's column block in every slot and one
    counter per tile per slot; everything else stays untouched."""
    rng = np.random.default_rng(18)
    w, M, N, K, dtype, r = 3, 33, 40, 16, "f16", 1
    st = oracle.GatheredState(w, M, N, 16, 16)
    oracle.gemm_all_scatter(st, _rand_bits(rng, (M, K), dtype),
                            _rand_bits(rng, (K, N), dtype), dtype, r, lib)
    cols = np.zeros(w * N, dtype=bool)
    cols[r * N:(r + 1) * N] = True
    for s in range(w):
        assert np.all(st.written[s][:, cols] == 1) and np.all(st.written[s][:, ~cols] == 0)
        assert np.all(np.isnan(st.G[s][:, ~cols])) and np.all(np.isfinite(st.G[s][:, cols]))
    assert st.arrived.shape == (w, w, 3, 3)
    assert np.all(st.arrived[:, r] == 1)
    assert int(st.arrived.sum()) == w * 3 * 3


# ---------------------------------------------------------------- tile copy

def pin_tile_copy(lib):
    rng = np.random.default_rng(19)
    for (w, rows, cols, tr, tc, shift, dt) in ((8, 40, 24, 16, 16, 1, np.float32),
                                               (5, 17, 9, 8, 4, 3, np.uint16),
                                               (2, 8, 8, 8, 8, 1, np.float32)):
        send = rng.integers(0, 2 ** 16, size=(w, rows, cols)).astype(dt)
        recv = np.zeros_like(send)
        out, flags = oracle.tile_copy(send, recv, tr, tc, shift, lib=lib)
        want = np.roll(send, shift, axis=0)          # slot d receives slot d - shift
        assert np.array_equal(out.view(np.uint8), want.view(np.uint8)), (w, shift)
        ntiles = -(-rows // tr) * -(-cols // tc)
        assert flags.shape == (w, ntiles) and np.all(flags == 1)
        # one source rank alone: only its destination slot changes
        src = w - 1
        out1, flags1 = oracle.tile_copy(send, recv, tr, tc, shift, only_rank=src, lib=lib)
        dst = (src + shift) % w
        assert np.array_equal(out1[dst].view(np.uint8), send[src].view(np.uint8))
        others = [s for s in range(w) if s != dst]
        assert np.all(out1[others].view(np.uint8) == 0)
        assert np.all(flags1[dst] == 1) and np.all(flags1[others] == 0)


def pin_tile_get(lib):
    """Get (Section 3.3.2): rank r pulls slot r - shift into its own slot."""
    rng = np.random.default_rng(23)
    for (w, rows, cols, tr, tc, shift, dt) in ((8, 24, 40, 16, 8, 3, np.float32),
                                               (3, 9, 17, 4, 8, 1, np.uint16)):
        send = rng.integers(0, 2 ** 16, size=(w, rows, cols)).astype(dt)
        recv = np.zeros_like(send)
        out, flags = oracle.tile_copy(send, recv, tr, tc, shift, lib=lib, get=True)
        assert np.array_equal(out.view(np.uint8), np.roll(send, shift, axis=0).view(np.uint8))
        assert np.all(flags == 1)
        me = 1
        out1, flags1 = oracle.tile_copy(send, recv, tr, tc, shift, only_rank=me, lib=lib, get=True)
        assert np.array_equal(out1[me].view(np.uint8), send[(me - shift) % w].view(np.uint8))
        others = [s for s in range(w) if s != me]
        assert np.all(out1[others].view(np.uint8) == 0)
        assert np.all(flags1[me] == 1) and np.all(flags1[others] == 0)


ALL_PINS = [v for k, v in sorted(globals().items()) if k.startswith("pin_")]
