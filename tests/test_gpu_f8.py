"""GPU parity of the FP8 (E4M3) forms against the CPU oracle:
Y = bf16(sx[i] sw[j] S[i,j] (+ R)) and H = bf16(silu(sx swg Sg) (sx swu Su)),
S the sum of products of the decoded E4M3 values.

Tolerance per element, the acceptance bound of the plain operator:
|Y - Yref| <= 1e-2 * RMS(Yref) + 2^-7 * |Yref| (products of E4M3 values are
exact in fp32; the fp32 sums and the scaling add a few 2^-24 relative, the
bf16 rounding of the output dominates).  Bit-exact check: with unit scales
and operands in {-1, 0, 1} every output is a small integer that both the
kernels' fp32 sums and bf16 hold exactly.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle import bf16_bits_to_f64
from paper_2608_17071_amd import workloads as wl
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ka():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_17071_amd import kernelarc
    return kernelarc


def _inputs(M, N, K, seed, swiglu=False, residual=True):
    return wl.make_i8_inputs(wl.I8Workload(f"t{seed}", M, N, K, swiglu, residual, seed, "f8"))


def _u8(t):
    return t.view(torch.uint8).numpy()


def _run(ka, t, swiglu, plan=None, out=None):
    d = {k: (v.cuda() if v is not None else None) for k, v in t.items()}
    if swiglu:
        y = ka.swiglu_f8(d["qX"], d["sx"], d["qW"], d["sw"], d["qWu"], d["swu"], plan=plan, out=out)
    else:
        y = ka.gemm_f8(d["qX"], d["sx"], d["qW"], d["sw"], d["R"], plan=plan, out=out)
    torch.cuda.synchronize()
    return gu.to_bits(y)


def _ref(t, swiglu, positions=None):
    orc = oracle.default()
    R = wl.bits(t["R"]) if t.get("R") is not None else None
    if swiglu:
        args = (_u8(t["qX"]), t["sx"].numpy(), _u8(t["qW"]), t["sw"].numpy(), _u8(t["qWu"]), t["swu"].numpy())
        return orc.f8_swiglu(*args) if positions is None else orc.f8_swiglu_at(*args, *positions)
    args = (_u8(t["qX"]), t["sx"].numpy(), _u8(t["qW"]), t["sw"].numpy(), R)
    return orc.f8_linear(*args) if positions is None else orc.f8_linear_at(*args, *positions)


def _check(ka, M, N, K, seed, swiglu, plan=None, residual=True, what=""):
    t = _inputs(M, N, K, seed, swiglu, residual and not swiglu)
    pname = ka.plan_name(plan) if plan is not None else ka.plan_name(ka.select_plan_f8(M, N, K, swiglu))
    gu.note(f"f8 {'swiglu' if swiglu else 'gemm'} {what} M={M} N={N} K={K} seed={seed} plan={pname}")
    got = _run(ka, t, swiglu, plan)
    gu.check_tolerance(got, _ref(t, swiglu), f"f8 {what} {pname} {M}x{N}x{K}")


def _plans(swiglu):
    from paper_2608_17071_amd import kernelarc
    names = kernelarc.plan_names()
    return [n for i, n in enumerate(names) if kernelarc.plan_supports_f8(i, 200, 264, 1040, swiglu)]


def _shape_for(name):
    if name.endswith("splitk") or name.endswith("tailsplit"):
        return (200, 264, 1040)
    return (77, 136, 528)


@pytest.mark.parametrize("name", _plans(False))
def test_f8_gemm_every_plan(ka, name):
    M, N, K = _shape_for(name)
    _check(ka, M, N, K, 81, False, plan=ka.plan_names().index(name), what="every-plan")


@pytest.mark.parametrize("name", _plans(True))
def test_f8_swiglu_every_plan(ka, name):
    M, N, K = _shape_for(name)
    _check(ka, M, N, K, 82, True, plan=ka.plan_names().index(name), what="every-plan")


@pytest.mark.parametrize("name", ["tile_256x256_k64_w8", "tile_64x64_k128s3_w4_splitk", "tile_128x128_k64s4_w4_lag",
                                  "tile_64x64_k64s4_w4", "tile_256x128_k64s3_w8_lag_splitk",
                                  "tile_64x128_k64s4_w4_splitk", "generic_64x64_scalar"])
def test_f8_small_integer_sums_bit_exact(ka, name):
    plan = ka.plan_names().index(name)
    M, N, K = 150, 200, 256
    rng = np.random.default_rng(5)
    t = {"qX": torch.from_numpy(rng.integers(-1, 2, size=(M, K)).astype(np.float32)).to(torch.float8_e4m3fn),
         "sx": torch.ones(M, dtype=torch.float32),
         "qW": torch.from_numpy(rng.integers(-1, 2, size=(N, K)).astype(np.float32)).to(torch.float8_e4m3fn),
         "sw": torch.ones(N, dtype=torch.float32), "R": None}
    gu.note(f"f8 exact small sums plan={name}")
    got = _run(ka, t, False, plan)
    xd = t["qX"].to(torch.float64).numpy()
    wd = t["qW"].to(torch.float64).numpy()
    np.testing.assert_array_equal(bf16_bits_to_f64(got), xd @ wd.T)


@pytest.mark.parametrize("M,N,K", [(1, 1024, 512), (3, 200, 64), (16, 4096, 1024), (33, 264, 528),
                                   (64, 1000, 1040), (257, 136, 256), (512, 2048, 3072), (130, 100, 144),
                                   (40, 77, 96), (64, 96, 250), (5, 7, 9), (64, 256, 0)])
@pytest.mark.parametrize("swiglu", [False, True])
def test_f8_shapes(ka, M, N, K, swiglu):
    _check(ka, M, N, K, M * 5 + N + K, swiglu, what="shapes")


def test_f8_in_place_and_landmarks(ka):
    """Y == R in place; operands at the format's extremes (+-448, subnormals)."""
    M, N, K = 200, 264, 528
    t = _inputs(M, N, K, 9, False, True)
    gu.note("f8 in place Y == R")
    r = t["R"].cuda()
    d = {k: v.cuda() for k, v in t.items() if k != "R"}
    ka.gemm_f8(d["qX"], d["sx"], d["qW"], d["sw"], r, out=r)
    torch.cuda.synchronize()
    gu.check_tolerance(gu.to_bits(r), _ref(t, False), "f8 in place")
    rng = np.random.default_rng(3)
    vals = np.array([448.0, -448.0, 2.0 ** -6, 2.0 ** -9, -7 * 2.0 ** -9, 1.0, 0.0, 240.0], np.float32)
    t = {"qX": torch.from_numpy(rng.choice(vals, size=(64, 256))).to(torch.float8_e4m3fn),
         "sx": torch.full((64,), 2.0 ** -8, dtype=torch.float32),
         "qW": torch.from_numpy(rng.choice(vals, size=(96, 256))).to(torch.float8_e4m3fn),
         "sw": torch.full((96,), 2.0 ** -8, dtype=torch.float32), "R": None}
    gu.note("f8 landmarks")
    gu.check_tolerance(_run(ka, t, False), _ref(t, False), "f8 landmarks")


def test_f8_rejects(ka):
    gu.note("f8 rejects")
    names = ka.plan_names()
    qx = torch.zeros(64, 128, dtype=torch.float8_e4m3fn, device="cuda")
    qw = torch.zeros(96, 128, dtype=torch.float8_e4m3fn, device="cuda")
    sx = torch.ones(64, dtype=torch.float32, device="cuda")
    sw = torch.ones(96, dtype=torch.float32, device="cuda")
    for n in ("stream_mfma16_k64_splitk", "gemv_valu_w4", "tile_256x256_k64_w4_m16a"):
        with pytest.raises(ka.KernelArcError) as e:
            ka.gemm_f8(qx, sx, qw, sw, plan=names.index(n))
        assert e.value.status == ka.ERR_UNSUPPORTED
    with pytest.raises(ValueError):                     # int8 operands are not FP8
        ka.gemm_f8(qx.view(torch.int8), sx, qw, sw)


@pytest.mark.parametrize("name", [w.name for w in wl.F8])
def test_f8_bench_workloads(ka, name):
    w = wl.F8_BY_NAME[name]
    t = wl.make_i8_inputs(w)
    gu.note(f"f8 bench {name} plan={ka.plan_name(ka.select_plan_f8(w.M, w.N, w.K, w.swiglu))}")
    got = _run(ka, t, w.swiglu)
    pos = gu.sample_positions(w.M, w.N, rows=4, cols=3, seed=w.seed)
    gu.check_tolerance(got[pos[0], pos[1]], _ref(t, w.swiglu, pos), name)
