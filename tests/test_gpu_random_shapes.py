"""Seeded random shapes through the library's own plan choice, against the
CPU oracle: the selection rules (exact-shape table, row-count bands, CU-fill
thresholds, streaming row blocks) meet shapes no other test names, and
whatever they pick must satisfy the operator's tolerance,
|Y - Yref| <= 1e-2 * RMS(Yref) + 2^-7 * |Yref|.  Large outputs are checked
on whole sampled rows and columns.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_17071_amd import workloads as wl
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ka():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_17071_amd import kernelarc
    return kernelarc


def _shapes(seed, count):
    """M spread over the rule bands (1..4, 5..64, 65..1024, above), N and K
    mostly multiples of 8 (the MFMA kernels) with some ragged ones (the
    generic kernel)."""
    rng = np.random.default_rng(seed)
    out = []
    for i in range(count):
        band = i % 4
        M = int(rng.integers(1, 5) if band == 0 else rng.integers(5, 65) if band == 1 else
                rng.integers(65, 1025) if band == 2 else rng.integers(1025, 2561))
        N = int(rng.integers(1, 400)) * 8
        K = int(rng.integers(1, 400)) * 8
        if i % 7 == 6:
            N += int(rng.integers(1, 8))
        if i % 11 == 10:
            K += int(rng.integers(1, 8))
        out.append((M, N, K))
    return out


BF16_SHAPES = _shapes(2024, 24)


@pytest.mark.parametrize("M,N,K", BF16_SHAPES)
def test_random_shape_auto_plan(ka, M, N, K):
    t = wl.make_inputs(wl.custom(M, N, K, seed=M + 3 * N + 7 * K))
    plan = ka.plan_name(ka.select_plan(M, N, K, True))
    gu.note(f"random shape M={M} N={N} K={K} plan={plan}")
    y = gu.run_library(t["X"], t["W"], t["R"])
    if M * N <= 1 << 18:
        gu.check_tolerance(y, gu.oracle_reference(t["X"], t["W"], t["R"]), f"random {plan}")
    else:
        pos = gu.sample_positions(M, N, rows=4, cols=4, seed=M + N)
        gu.check_tolerance(y[pos[0], pos[1]], gu.oracle_reference(t["X"], t["W"], t["R"], pos), f"random {plan}")


I8_SHAPES = [(M, N, (K // 16) * 16 or 16) for (M, N, K) in _shapes(2025, 12)]


@pytest.mark.parametrize("M,N,K", I8_SHAPES)
def test_random_shape_auto_plan_i8(ka, M, N, K):
    t = wl.make_i8_inputs(wl.I8Workload(f"r{M}", M, N, K, False, True, M + N + K))
    plan = ka.plan_name(ka.select_plan_i8(M, N, K, False))
    gu.note(f"random INT8 shape M={M} N={N} K={K} plan={plan}")
    d = {k: (v.cuda() if v is not None else None) for k, v in t.items()}
    y = ka.gemm_i8(d["qX"], d["sx"], d["qW"], d["sw"], d["R"])
    torch.cuda.synchronize()
    got = gu.to_bits(y)
    orc = oracle.default()
    args = (t["qX"].numpy(), t["sx"].numpy(), t["qW"].numpy(), t["sw"].numpy(), wl.bits(t["R"]))
    if M * N <= 1 << 18:
        gu.check_tolerance(got, orc.i8_linear(*args), f"random INT8 {plan}")
    else:
        pos = gu.sample_positions(M, N, rows=4, cols=4, seed=M + N)
        gu.check_tolerance(got[pos[0], pos[1]], orc.i8_linear_at(*args, pos[0], pos[1]), f"random INT8 {plan}")
