"""GPU parity: the HIP library against the CPU oracle on the same seeded inputs.

Tolerance (per element, from the stated acceptance bound):
    |Y - Yref| <= 1e-2 * RMS(Yref) + 2^-7 * |Yref|
Bitwise checks where the exact result is fixed independently of summation
order (W = 0, W = I, rank-1 integer inputs), where one plan must reproduce
itself (determinism, row permutation), and for the no-op / K = 0 cases.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle import bf16_bits_to_f64
from paper_2608_17071_amd import workloads as wl
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu

FULL_ORACLE_MACS = 1 << 31   # larger outputs: test_gpu_full_output.py


@pytest.fixture(scope="module")
def ka():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_17071_amd import kernelarc
    return kernelarc


def plan_id(ka, name):
    return ka.plan_names().index(name)


def _parity(ka, w, plain=False):
    t = wl.make_inputs(w)
    X, W, R = t["X"], t["W"], (None if plain else t["R"])
    tag = f"{w.name} {'plain' if plain else ('residual' if R is not None else 'plain')}"
    gu.note(f"{tag} plan={ka.plan_name(ka.select_plan(w.M, w.N, w.K, R is not None))}")
    y = gu.run_library(X, W, R)
    ref = gu.oracle_reference(X, W, R)
    return gu.check_tolerance(y, ref, tag)


# Larger outputs are compared whole in test_gpu_full_output.py.
@pytest.mark.parametrize("name", [w.name for w in wl.ALL if w.M * w.N * w.K <= FULL_ORACLE_MACS])
def test_workload_parity(ka, name):
    w = wl.BY_NAME[name]
    _parity(ka, w)
    if w.residual:
        # the residual dominates Y; check the product term on its own scale too
        _parity(ka, w, plain=True)


def _all_plan_names():
    from paper_2608_17071_amd import kernelarc
    return kernelarc.plan_names()


TILE_SHAPES = [(65, 8, 8), (300, 264, 200), (130, 100, 72), (513, 520, 136)]
PLAN_SHAPES = {
    # plan name: ragged shapes (M, N, K) it supports, K % 8 == 0 for MFMA plans
    "generic_64x64_scalar": [(1, 1, 1), (70, 33, 13), (130, 100, 72)],
    "gemv_valu_w4": [(1, 8, 8), (1, 520, 1000), (3, 100, 4104), (4, 2048, 2048), (2, 77, 136), (1, 9000, 520)],
    "stream_mfma16_k64_splitk": [(2, 24, 8), (31, 520, 1000), (64, 96, 4104), (60, 200, 2056)],
    # 16- and 32-row blocks with X staged through LDS: the rule's split
    # ranges from none (K too shallow) to 16 slices; ragged M, N and K.
    **{n: [(1, 8, 8), (16, 520, 1000), (17, 100, 4104), (64, 96, 2056), (33, 130, 136), (5, 24, 264)]
       for n in ("stream_mfma16_r16_k128s2", "stream_mfma16_r32_k64s4")},
}
PLAN_SHAPES.update({n: TILE_SHAPES for n in _all_plan_names() if n.startswith("tile_")})
assert set(PLAN_SHAPES) == set(_all_plan_names()), "every plan has test shapes"


@pytest.mark.parametrize("plan", sorted(PLAN_SHAPES))
def test_ragged_shapes_every_plan(ka, plan):
    p = plan_id(ka, plan)
    for (M, N, K) in PLAN_SHAPES[plan]:
        assert ka.plan_supports(p, M, N, K), (plan, M, N, K)
        t = wl.make_inputs(wl.custom(M, N, K, seed=M + N + K))
        for R in (t["R"], None):
            gu.note(f"{plan} M={M} N={N} K={K} residual={R is not None}")
            y = gu.run_library(t["X"], t["W"], R, plan=p)
            gu.check_tolerance(y, gu.oracle_reference(t["X"], t["W"], R), f"{plan} {M}x{N}x{K}")


def _unsigned_zero(bits):
    """bf16 patterns with -0 replaced by +0."""
    b = bits.copy()
    b[b == 0x8000] = 0
    return b


def _closed_form_shapes(plan):
    if plan.startswith("gemv"):
        return (4, 200, 200), (3, 136, 1000)
    if plan.startswith("stream"):
        return (23, 200, 200), (40, 136, 1000)
    return (300, 264, 264), (130, 100, 520)


@pytest.mark.parametrize("plan", sorted(PLAN_SHAPES))
def test_closed_forms_bitwise_every_plan(ka, plan):
    p = plan_id(ka, plan)
    orc = oracle.default()
    square, rank1 = _closed_form_shapes(plan)
    M, K = square[0], square[1]          # W = I needs N == K
    M2, N2, K2 = rank1
    t = wl.make_inputs(wl.custom(M, K, K, seed=11))
    X, R = t["X"], t["R"]
    # W = 0  =>  Y = R (values), and the plain product is zero
    gu.note(f"{plan} W=0 M={M} K={K}")
    y = gu.run_library(X, wl.zero_weight(K, K), R, plan=p)
    np.testing.assert_array_equal(bf16_bits_to_f64(y), bf16_bits_to_f64(wl.bits(R)))
    y = gu.run_library(X, wl.zero_weight(K, K), None, plan=p)
    assert not np.any(bf16_bits_to_f64(y))
    # W = I  =>  Y = X exactly (plain), Y = bf16(X + R) wherever X + R is exact in fp32
    gu.note(f"{plan} W=I M={M} K={K}")
    eye = wl.identity_weight(K)
    y = gu.run_library(X, eye, None, plan=p)
    np.testing.assert_array_equal(y, wl.bits(X))
    y = gu.run_library(X, eye, R, plan=p)
    s = bf16_bits_to_f64(wl.bits(X)) + bf16_bits_to_f64(wl.bits(R))
    exact = s.astype(np.float32).astype(np.float64) == s
    assert exact.mean() > 0.99
    np.testing.assert_array_equal(y[exact], orc.round_bf16(s)[exact])
    # rank-1 integer inputs: every partial sum is an exact integer
    gu.note(f"{plan} rank-1 M={M2} N={N2} K={K2}")
    X1, W1, R1, a, b, u, v = wl.rank1_integer(M2, N2, K2, seed=5)
    # (the exact product is an integer; "+ 0.0" makes its zeros +0, and the
    # sign of a zero result is not part of the contract)
    exact1 = (np.outer(a, b) * int(np.dot(u, v))).astype(np.float64) + 0.0
    y = gu.run_library(X1, W1, None, plan=p)
    np.testing.assert_array_equal(_unsigned_zero(y), orc.round_bf16(exact1))
    y = gu.run_library(X1, W1, R1, plan=p)
    np.testing.assert_array_equal(_unsigned_zero(y),
                                  orc.round_bf16(exact1 + bf16_bits_to_f64(wl.bits(R1)) + 0.0))


# Shapes where the tail-split plans split only the tiles of a partial last
# round: (plan, M, N, K).  Each is checked to really take that path.
TAIL_SPLIT_CASES = [("tile_256x256_k64_w8_tailsplit", 2048, 8448, 1024),    # 264 tiles, 256 slots
                    ("tile_256x256_k64_w8_tailsplit", 4096, 5120, 5120),    # 320 tiles: the benchmark shape
                    ("tile_256x256_k64_w8_tailsplit", 2048, 8448, 1040)]    # 264 tiles, K tail


@pytest.mark.parametrize("case", TAIL_SPLIT_CASES, ids=[f"{c[0]}_{c[1]}x{c[2]}x{c[3]}" for c in TAIL_SPLIT_CASES])
def test_tail_split_whole_output(ka, case):
    plan, M, N, K = case
    p = plan_id(ka, plan)
    assert ka.kernelarc_plan_uses_workspace(p, M, N, K) == 1, "the tail tiles must be split"
    orc = oracle.default()
    # every element bitwise, through rank-1 integer inputs
    gu.note(f"{plan} tail split rank-1 M={M} N={N} K={K}")
    X1, W1, R1, a, b, u, v = wl.rank1_integer(M, N, K, seed=7)
    exact1 = (np.outer(a, b) * int(np.dot(u, v))).astype(np.float64) + 0.0
    y = gu.run_library(X1, W1, R1, plan=p)
    np.testing.assert_array_equal(_unsigned_zero(y), orc.round_bf16(exact1 + bf16_bits_to_f64(wl.bits(R1)) + 0.0))
    # random inputs: whole sampled rows and columns against the oracle, and
    # the same bits on a second call
    gu.note(f"{plan} tail split random M={M} N={N} K={K}")
    t = wl.make_inputs(wl.custom(M, N, K, seed=12))
    y1 = gu.run_library(t["X"], t["W"], t["R"], plan=p)
    pos = gu.sample_positions(M, N, seed=12)
    gu.check_tolerance(y1[pos[0], pos[1]], gu.oracle_reference(t["X"], t["W"], t["R"], pos), plan)
    np.testing.assert_array_equal(gu.run_library(t["X"], t["W"], t["R"], plan=p), y1)


# Shapes where the banded plan runs both column bands: (M, N, K, N1), N1 the
# first band's width (whole rounds of 256x256 tiles); ragged M, N and K.
BAND_CASES = [(4000, 4360, 200, 4096), (4096, 4608, 136, 4096), (2048, 8448, 72, 8192)]


@pytest.mark.parametrize("case", BAND_CASES, ids=[f"{c[0]}x{c[1]}x{c[2]}" for c in BAND_CASES])
def test_bands_whole_output(ka, case):
    M, N, K, N1 = case
    p = plan_id(ka, "tile_256x256_k64_w4_m16a_bands")
    assert ka.plan_supports(p, M, N, K)
    orc = oracle.default()
    # every element bitwise, through rank-1 integer inputs, into a NaN-prefilled output
    X1, W1, R1, a, b, u, v = wl.rank1_integer(M, N, K, seed=8)
    exact1 = (np.outer(a, b) * int(np.dot(u, v))).astype(np.float64) + 0.0
    for R, want, form in ((R1, exact1 + bf16_bits_to_f64(wl.bits(R1)) + 0.0, "residual"), (None, exact1, "plain")):
        gu.note(f"bands rank-1 M={M} N={N} K={K} N1={N1} {form}")
        out = torch.full((M, N), float("nan"), dtype=torch.bfloat16, device="cuda")
        y = gu.run_library(X1, W1, R, plan=p, out=out)
        np.testing.assert_array_equal(_unsigned_zero(y), orc.round_bf16(want), err_msg=f"bands {form}")
    # random inputs: the whole output against the oracle
    t = wl.make_inputs(wl.custom(M, N, K, seed=14))
    for R in (t["R"], None):
        gu.note(f"bands random M={M} N={N} K={K} residual={R is not None}")
        out = torch.full((M, N), float("nan"), dtype=torch.bfloat16, device="cuda")
        y = gu.run_library(t["X"], t["W"], R, plan=p, out=out)
        gu.check_tolerance(y, gu.oracle_reference(t["X"], t["W"], R), f"bands {M}x{N}x{K}")


@pytest.mark.parametrize("plan", sorted(PLAN_SHAPES))
def test_deterministic_and_row_permutation(ka, plan):
    p = plan_id(ka, plan)
    M, N, K = PLAN_SHAPES[plan][-1]
    t = wl.make_inputs(wl.custom(M, N, K, seed=3))
    gu.note(f"{plan} determinism M={M} N={N} K={K}")
    y1 = gu.run_library(t["X"], t["W"], t["R"], plan=p)
    y2 = gu.run_library(t["X"], t["W"], t["R"], plan=p)
    np.testing.assert_array_equal(y1, y2)
    perm = torch.from_numpy(np.random.default_rng(0).permutation(M))
    yp = gu.run_library(t["X"][perm].contiguous(), t["W"], t["R"][perm].contiguous(), plan=p)
    np.testing.assert_array_equal(yp, y1[perm.numpy()])


def test_in_place_residual(ka):
    for (M, N, K) in [(16, 4096, 4096), (512, 1024, 512), (77, 300, 136)]:
        t = wl.make_inputs(wl.custom(M, N, K, seed=9))
        gu.note(f"in-place M={M} N={N} K={K}")
        expect = gu.run_library(t["X"], t["W"], t["R"])
        x, w, r = t["X"].cuda(), t["W"].cuda(), t["R"].cuda()
        out = ka.gemm_bf16_residual(x, w, r, out=r)
        torch.cuda.synchronize()
        assert out.data_ptr() == r.data_ptr()
        np.testing.assert_array_equal(gu.to_bits(r), expect)


def test_every_element_written_and_guard_bands(ka):
    for (M, N, K) in [(16, 4096, 4096), (300, 264, 200), (1, 24, 8), (130, 100, 72)]:
        t = wl.make_inputs(wl.custom(M, N, K, seed=4))
        pad = 4096
        buf = torch.full((pad + M * N + pad,), float("nan"), dtype=torch.bfloat16, device="cuda")
        out = buf[pad:pad + M * N].view(M, N)
        gu.note(f"nan-prefill/guard M={M} N={N} K={K}")
        ka.gemm_bf16_residual(t["X"].cuda(), t["W"].cuda(), t["R"].cuda(), out=out)
        torch.cuda.synchronize()
        assert not torch.isnan(out).any()
        assert torch.isnan(buf[:pad]).all() and torch.isnan(buf[pad + M * N:]).all()


def test_edge_sizes(ka):
    x = torch.zeros(0, 64, dtype=torch.bfloat16, device="cuda")
    w = torch.zeros(32, 64, dtype=torch.bfloat16, device="cuda")
    gu.note("M=0")
    assert ka.gemm_bf16(x, w).shape == (0, 32)
    gu.note("N=0")
    assert ka.gemm_bf16(torch.zeros(5, 64, dtype=torch.bfloat16, device="cuda"),
                        torch.zeros(0, 64, dtype=torch.bfloat16, device="cuda")).shape == (5, 0)
    for M in (3, 16, 48, 100):      # GEMV, 16-row streaming (twice), tiles
        r = torch.randn(M, 40, device="cuda").to(torch.bfloat16)
        xe = torch.zeros(M, 0, dtype=torch.bfloat16, device="cuda")
        we = torch.zeros(40, 0, dtype=torch.bfloat16, device="cuda")
        gu.note(f"K=0 M={M}")
        y = ka.gemm_bf16_residual(xe, we, r)
        torch.cuda.synchronize()
        assert torch.equal(y.float(), r.float())
        y = ka.gemm_bf16(xe, we)
        torch.cuda.synchronize()
        assert (y.float() == 0).all()


def test_misaligned_pointers_fall_back(ka):
    M, N, K = 40, 72, 64
    t = wl.make_inputs(wl.custom(M, N, K, seed=2))
    xb = torch.zeros(M * K + 1, dtype=torch.bfloat16, device="cuda")
    x = xb[1:].view(M, K)                    # 2-byte aligned only
    x.copy_(t["X"].cuda())
    gu.note("misaligned X")
    y = ka.gemm_bf16_residual(x, t["W"].cuda(), t["R"].cuda())
    torch.cuda.synchronize()
    gu.check_tolerance(gu.to_bits(y), gu.oracle_reference(t["X"], t["W"], t["R"]), "misaligned")
    tile = plan_id(ka, "tile_128x128_k64_w4")
    with pytest.raises(ka.KernelArcError):
        ka.gemm_bf16_with_plan(tile, x, t["W"].cuda(), t["R"].cuda())


def test_leading_dims_flatten(ka):
    t = wl.make_inputs(wl.custom(6 * 20, 256, 128, seed=8))
    x = t["X"].view(6, 20, 128).cuda()
    r = t["R"].view(6, 20, 256).cuda()
    gu.note("3-d input")
    y = ka.gemm_bf16_residual(x, t["W"].cuda(), r)
    torch.cuda.synchronize()
    assert y.shape == (6, 20, 256)
    gu.check_tolerance(gu.to_bits(y.view(120, 256)), gu.oracle_reference(t["X"], t["W"], t["R"]), "3-d")


def test_graph_replay_matches_eager(ka):
    """Calls captured in a HIP graph give the eager result on every replay
    (the split-K plans' arrival counters must reset themselves)."""
    cases = [("stream_mfma16_r16_k128s2", (16, 1024, 4096)), ("stream_mfma16_r32_k64s4", (16, 4096, 4096)),
             ("gemv_valu_w4", (1, 4096, 4096)),
             ("tile_128x128_k64_w4_splitk", (512, 1024, 2048)), ("tile_256x256_k64_w8", (300, 520, 264)),
             ("tile_64x64_k128s3_w4_splitk", (64, 768, 4096)), ("stream_mfma16_k64_splitk", (64, 1024, 4096)),
             ("tile_256x128_k64s3_w8_lag_splitk", (512, 1024, 4096)),
             ("tile_256x256_k64_w8_tailsplit", (2048, 8448, 1024))]
    for name, (M, N, K) in cases:
        p = plan_id(ka, name)
        t = wl.make_inputs(wl.custom(M, N, K, seed=21))
        gu.note(f"graph {name} M={M} N={N} K={K}")
        eager = gu.run_library(t["X"], t["W"], t["R"], plan=p)
        x, w, r = t["X"].cuda(), t["W"].cuda(), t["R"].cuda()
        y = torch.empty(M, N, dtype=torch.bfloat16, device="cuda")
        ka.gemm_bf16_with_plan(p, x, w, r, out=y)      # any workspace exists before capture
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            ka.gemm_bf16_with_plan(p, x, w, r, out=y)
        y2 = torch.empty_like(y)
        for rep in range(3):
            y.fill_(float("nan"))
            g.replay()
            torch.cuda.synchronize()
            np.testing.assert_array_equal(gu.to_bits(y), eager, err_msg=f"{name} replay {rep}")
            ka.gemm_bf16_with_plan(p, x, w, r, out=y2)   # eager work between replays
            torch.cuda.synchronize()
            np.testing.assert_array_equal(gu.to_bits(y2), eager)


@pytest.mark.parametrize("plan", ["stream_mfma16_r16_k128s2", "stream_mfma16_r32_k64s4"])
def test_stream_many_row_blocks(ka, plan):
    """A wide, shallow decode-like shape forced onto the 16- and 32-row
    streaming plans: thousands of row blocks (several rounds of workgroups,
    no K split), the last block ragged; whole output against the oracle."""
    M, N, K = 16, 65544, 64
    p = plan_id(ka, plan)
    t = wl.make_inputs(wl.custom(M, N, K, seed=14))
    gu.note(f"{plan} many row blocks M={M} N={N} K={K}")
    y = gu.run_library(t["X"], t["W"], t["R"], plan=p)
    gu.check_tolerance(y, gu.oracle_reference(t["X"], t["W"], t["R"]), plan)
