"""Whole-output parity at the benchmark's full sizes, through the plan the
library selects (the launch configuration the benchmark times).

For the prefill projection (4096^3 with residual), the plain 8192^3 GEMM and
every sweep shape whose output the sampled checks of test_gpu_parity.py do
not cover whole (more than 2^31 multiply-adds), each call writes into an
output prefilled with NaN, and every element is compared with the oracle:

    |Y - Yref| <= 1e-2 * RMS(Yref) + 2^-7 * |Yref|        (all finite)

for the residual operator and for the plain product on the same X and W
(the residual dominates Y, so the product term is also checked on its own
scale).  The oracle evaluates each k-sum once for both forms.  A rank-1
integer problem of the same size checks every element bit for bit: its exact
result is a_i b_j (u . v) (+ R), every partial sum an integer below 2^24, so a
tile that is skipped, written twice, misplaced or summed over a wrong K range
shows in the exact bits.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle import bf16_bits_to_f64
from paper_2608_17071_amd import workloads as wl
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu

# The configurations whose outputs exceed 2^31 multiply-adds.
FULL_SIZE = [w.name for w in wl.ALL if w.M * w.N * w.K > (1 << 31)]


@pytest.fixture(scope="module")
def ka():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_17071_amd import kernelarc
    return kernelarc


def _nan_call(ka, x, w, r, M, N):
    """One call through the selected plan into a NaN-prefilled output."""
    out = torch.full((M, N), float("nan"), dtype=torch.bfloat16, device="cuda")
    y = ka.gemm_bf16_residual(x, w, r, out=out) if r is not None else ka.gemm_bf16(x, w, out=out)
    torch.cuda.synchronize()
    assert y.data_ptr() == out.data_ptr()
    return gu.to_bits(out)


def _unsigned_zero(bits):
    b = bits.copy()
    b[b == 0x8000] = 0
    return b


def test_full_size_list():
    # configs 3 and 4 and the eight large sweep shapes
    assert {"prefill_m4096_h4096", "square_plain_8192"} <= set(FULL_SIZE)
    assert len(FULL_SIZE) == 10, FULL_SIZE


@pytest.mark.parametrize("name", FULL_SIZE)
def test_whole_output_against_oracle(ka, name):
    w = wl.BY_NAME[name]
    t = wl.make_inputs(w)
    orc = oracle.default()
    xb, wb = wl.bits(t["X"]), wl.bits(t["W"])
    if w.residual:
        ref_plain, ref_res = orc.linear_pair(xb, wb, wl.bits(t["R"]))
    else:
        ref_plain, ref_res = orc.linear(xb, wb), None
    x, wt = t["X"].cuda(), t["W"].cuda()
    for r, ref, form in ((t["R"], ref_res, "residual"), (None, ref_plain, "plain")):
        if ref is None:
            continue
        plan = ka.plan_name_for(w.M, w.N, w.K, r is not None)
        gu.note(f"whole output {name} {form} plan={plan}")
        y = _nan_call(ka, x, wt, r.cuda() if r is not None else None, w.M, w.N)
        ratio = gu.check_tolerance(y, ref, f"{name} {form} ({plan})")
        print(f"{name} {form} {plan}: max err/bound {ratio:.3f}")


@pytest.mark.parametrize("name", FULL_SIZE)
def test_whole_output_rank1_bitwise(ka, name):
    w = wl.BY_NAME[name]
    orc = oracle.default()
    X1, W1, R1, a, b, u, v = wl.rank1_integer(w.M, w.N, w.K, seed=w.seed + 40)
    exact = (np.outer(a, b) * int(np.dot(u, v))).astype(np.float64) + 0.0
    x, wt = X1.cuda(), W1.cuda()
    for r, want, form in ((R1, exact + bf16_bits_to_f64(wl.bits(R1)) + 0.0, "residual"), (None, exact, "plain")):
        plan = ka.plan_name_for(w.M, w.N, w.K, r is not None)
        gu.note(f"rank-1 whole output {name} {form} plan={plan}")
        y = _nan_call(ka, x, wt, r.cuda() if r is not None else None, w.M, w.N)
        np.testing.assert_array_equal(_unsigned_zero(y), orc.round_bf16(want), err_msg=f"{name} {form} ({plan})")
