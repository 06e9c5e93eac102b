"""CPU pins of the per-element accumulation bound the GPU parity tests apply
beside the stated tolerance (tests/gpu_util.accumulation_bound_violations).

Correct results built without the GPU pass it: the exact product (float64
library matmul) rounded once to the output format, and an fp32 sum taken in
another order.  A planted mistake of the kind a kernel could make -- one
group of 8 consecutive k dropped from the sum, or one product counted twice
-- fails it.  (The stated max|err| <= tol * max|C| check is a single
threshold for the whole block; this bound follows each element's own
sum of |a||b|.)"""
import numpy as np
import pytest
import torch

import oracle
import workload
from tests.gpu_util import accumulation_bound_violations


def _round(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round float64 values to the 16-bit format (nearest even) and back."""
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(workload.torch_dtype(dtype)).float().numpy()


def _case(dtype, M=96, N=80, K=4096, seed=3):
    dist = "normal_sqrtk" if dtype == "bf16" else "uniform_sqrtk"
    A = workload.gemm_A(M, K, dtype, dist, seed)
    B = workload.gemm_B_shard(K, N, 0, dtype, dist, seed)
    a = oracle.decode16(workload.bits(A), dtype)
    b = oracle.decode16(workload.bits(B), dtype)
    ref = oracle.gemm(a, b)
    abs_ab = oracle.gemm(np.abs(a), np.abs(b))
    exact = a.astype(np.float64) @ b.astype(np.float64)
    return a, b, ref, abs_ab, exact


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
def test_correct_results_pass_the_bound(dtype):
    a, b, ref, abs_ab, exact = _case(dtype)
    K = a.shape[1]
    assert not accumulation_bound_violations(_round(exact, dtype), ref, abs_ab, K, dtype).any()
    # an fp32 sum in another order (k descending, in blocks), then rounded
    other = np.zeros(exact.shape, dtype=np.float32)
    for k0 in range(K - 64, -1, -64):
        other += (a[:, k0:k0 + 64] @ b[k0:k0 + 64, :]).astype(np.float32)
    assert not accumulation_bound_violations(_round(other, dtype), ref, abs_ab, K, dtype).any()
    # zeros of a K = 0 problem are exact
    z = np.zeros((4, 4), dtype=np.float32)
    assert not accumulation_bound_violations(z, z, z, 0, dtype).any()


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
@pytest.mark.parametrize("k0", [0, 2048, 4088])
def test_dropped_k_group_is_caught(dtype, k0):
    a, b, ref, abs_ab, exact = _case(dtype)
    K = a.shape[1]
    dropped = exact - a[:, k0:k0 + 8].astype(np.float64) @ b[k0:k0 + 8, :].astype(np.float64)
    got = _round(dropped, dtype)
    assert accumulation_bound_violations(got, ref, abs_ab, K, dtype).any()


def test_doubled_product_is_caught():
    a, b, ref, abs_ab, exact = _case("bf16", seed=5)
    K = a.shape[1]
    doubled = exact + np.outer(a[:, 17], b[17, :])
    assert accumulation_bound_violations(_round(doubled, "bf16"), ref, abs_ab, K, "bf16").any()
