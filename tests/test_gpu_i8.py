"""GPU parity of the INT8 forms against the CPU oracle:
Y = bf16(sx[i] sw[j] A[i,j] (+ R)) and H = bf16(silu(sx swg Ag) (sx swu Au)),
A = qX qW^T summed exactly in int32.

Tolerance per element, the acceptance bound of the plain operator:
|Y - Yref| <= 1e-2 * RMS(Yref) + 2^-7 * |Yref| (the integer sums are exact;
fp32 conversion and scaling add a few 2^-24 relative, the bf16 rounding of the
output dominates).  Bit-exact checks: with unit scales and |A| <= 256 every
output is an integer that bf16 holds exactly, so the kernels' integer sums
(split-K and K-group hand-offs included) must reproduce the oracle's exact
sums bit for bit.
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
    return wl.make_i8_inputs(wl.I8Workload(f"t{seed}", M, N, K, swiglu, residual, seed))


def _np(t):
    return t.numpy()


def _run(ka, t, swiglu, plan=None, out=None):
    d = {k: (v.cuda() if v is not None else None) for k, v in t.items()}
    if swiglu:
        y = ka.swiglu_i8(d["qX"], d["sx"], d["qW"], d["sw"], d["qWu"], d["swu"], plan=plan, out=out)
    else:
        y = ka.gemm_i8(d["qX"], d["sx"], d["qW"], d["sw"], d["R"], plan=plan, out=out)
    torch.cuda.synchronize()
    return gu.to_bits(y)


def _ref(t, swiglu, positions=None):
    orc = oracle.default()
    R = wl.bits(t["R"]) if t.get("R") is not None else None
    if swiglu:
        args = (_np(t["qX"]), _np(t["sx"]), _np(t["qW"]), _np(t["sw"]), _np(t["qWu"]), _np(t["swu"]))
        return orc.i8_swiglu(*args) if positions is None else orc.i8_swiglu_at(*args, *positions)
    args = (_np(t["qX"]), _np(t["sx"]), _np(t["qW"]), _np(t["sw"]), R)
    return orc.i8_linear(*args) if positions is None else orc.i8_linear_at(*args, *positions)


def _check(ka, M, N, K, seed, swiglu, plan=None, residual=True, what=""):
    t = _inputs(M, N, K, seed, swiglu, residual and not swiglu)
    pname = ka.plan_name(plan) if plan is not None else ka.plan_name(ka.select_plan_i8(M, N, K, swiglu))
    gu.note(f"i8 {'swiglu' if swiglu else 'gemm'} {what} M={M} N={N} K={K} seed={seed} plan={pname}")
    got = _run(ka, t, swiglu, plan)
    gu.check_tolerance(got, _ref(t, swiglu), f"i8 {what} {pname} {M}x{N}x{K}")


def _plans(swiglu):
    from paper_2608_17071_amd import kernelarc
    names = kernelarc.plan_names()
    return [n for i, n in enumerate(names) if kernelarc.plan_supports_i8(i, 200, 264, 1040, swiglu)]


def _shape_for(name):
    if name.endswith("splitk") or name.endswith("tailsplit"):
        return (200, 264, 1040)
    return (77, 136, 528)


@pytest.mark.parametrize("name", _plans(False))
def test_i8_gemm_every_plan(ka, name):
    M, N, K = _shape_for(name)
    _check(ka, M, N, K, 41, False, plan=ka.plan_names().index(name), what="every-plan")


def _stream_plans():
    from paper_2608_17071_amd import kernelarc
    names = kernelarc.plan_names()
    return [n for i, n in enumerate(names) if n.startswith("stream") and kernelarc.plan_supports_i8(i, 33, 264, 1040, False)]


@pytest.mark.parametrize("name", _stream_plans())
@pytest.mark.parametrize("M,N,K", [(1, 8, 16), (16, 520, 1040), (17, 100, 4112), (64, 96, 2064), (33, 130, 144),
                                   (5, 24, 272)])
def test_i8_stream_plans(ka, name, M, N, K):
    """The streaming plans (16- and 32-row blocks) on INT8 operands: one to
    four token blocks, ragged N, K tails inside a stage and K splits from
    none to four slices."""
    _check(ka, M, N, K, 43, False, plan=ka.plan_names().index(name), what="stream")


@pytest.mark.parametrize("name", _plans(True))
def test_i8_swiglu_every_plan(ka, name):
    M, N, K = _shape_for(name)
    _check(ka, M, N, K, 42, True, plan=ka.plan_names().index(name), what="every-plan")


def _unit_case(M, N, K, seed, swiglu):
    """qX, qW in {-1, 0, 1}, unit scales: every |A| <= K <= 256 is exact in bf16."""
    rng = np.random.default_rng(seed)
    t = {"qX": torch.from_numpy(rng.integers(-1, 2, size=(M, K)).astype(np.int8)),
         "sx": torch.ones(M, dtype=torch.float32),
         "qW": torch.from_numpy(rng.integers(-1, 2, size=(N, K)).astype(np.int8)),
         "sw": torch.ones(N, dtype=torch.float32), "R": None}
    if swiglu:
        t["qWu"] = torch.from_numpy(rng.integers(-1, 2, size=(N, K)).astype(np.int8))
        t["swu"] = torch.ones(N, dtype=torch.float32)
    return t


@pytest.mark.parametrize("name", ["tile_256x256_k64_w8", "tile_64x64_k128s3_w4_splitk", "tile_128x128_k64s4_w4_lag",
                                  "tile_64x64_k64s4_w4", "tile_256x128_k64s3_w8_lag_splitk",
                                  "tile_64x128_k64s4_w4_splitk", "generic_64x64_scalar",
                                  "stream_mfma16_r16_k128s2", "stream_mfma16_r32_k64s4"])
def test_i8_integer_sums_bit_exact(ka, name):
    """Unit scales and |A| <= 256: the outputs are the exact integer sums."""
    plan = ka.plan_names().index(name)
    M, N, K = (64 if name.startswith("stream") else 150), 200, 256
    t = _unit_case(M, N, K, 7, False)
    gu.note(f"i8 exact integer sums plan={name}")
    got = _run(ka, t, False, plan)
    A = oracle.default().i8_dot(_np(t["qX"]), _np(t["qW"]))
    np.testing.assert_array_equal(bf16_bits_to_f64(got), A.astype(np.float64))


@pytest.mark.parametrize("M,N,K", [(1, 1024, 512), (3, 200, 64), (16, 4096, 1024), (33, 264, 528),
                                   (64, 1000, 1040), (257, 136, 256), (512, 2048, 3072), (130, 100, 144),
                                   (40, 77, 96), (64, 96, 250), (5, 7, 9), (64, 256, 0)])
@pytest.mark.parametrize("swiglu", [False, True])
def test_i8_shapes(ka, M, N, K, swiglu):
    """Selected plans over skinny and ragged shapes, N not a multiple of 8,
    K not a multiple of 16 (generic kernel) and K = 0."""
    _check(ka, M, N, K, M * 3 + N + K, swiglu, what="shapes")


def test_i8_no_residual_and_in_place(ka):
    M, N, K = 200, 264, 528
    t = _inputs(M, N, K, 9, False, True)
    gu.note("i8 in place Y == R")
    r = t["R"].cuda()
    d = {k: v.cuda() for k, v in t.items() if k != "R"}
    ka.gemm_i8(d["qX"], d["sx"], d["qW"], d["sw"], r, out=r)
    torch.cuda.synchronize()
    gu.check_tolerance(gu.to_bits(r), _ref(t, False), "i8 in place")
    t["R"] = None
    gu.check_tolerance(_run(ka, t, False), _ref(t, False), "i8 no residual")


def test_i8_extremes(ka):
    """-128 everywhere: A = 16384 K, the largest sums the int32 range allows
    per K; K = 4096 gives 2^26 (fp32-exact after conversion)."""
    M, N, K = 64, 128, 4096
    t = {"qX": torch.full((M, K), -128, dtype=torch.int8), "sx": torch.full((M,), 2.0 ** -13, dtype=torch.float32),
         "qW": torch.full((N, K), -128, dtype=torch.int8), "sw": torch.full((N,), 2.0 ** -13, dtype=torch.float32),
         "R": None}
    gu.note("i8 extremes")
    got = _run(ka, t, False)
    assert (bf16_bits_to_f64(got) == 2.0 ** 26 * 2.0 ** -26).all()


def test_i8_rejects(ka):
    gu.note("i8 rejects")
    names = ka.plan_names()
    qx = torch.zeros(64, 128, dtype=torch.int8, device="cuda")
    qw = torch.zeros(96, 128, dtype=torch.int8, device="cuda")
    sx = torch.ones(64, dtype=torch.float32, device="cuda")
    sw = torch.ones(96, dtype=torch.float32, device="cuda")
    for n in ("stream_mfma16_k64_splitk", "gemv_valu_w4"):
        with pytest.raises(ka.KernelArcError) as e:
            ka.gemm_i8(qx, sx, qw, sw, plan=names.index(n))
        assert e.value.status == ka.ERR_UNSUPPORTED
    with pytest.raises(ka.KernelArcError) as e:          # the 16x16 AGPR tile: plain INT8 only
        ka.swiglu_i8(qx, sx, qw, sw, qw, sw, plan=names.index("tile_256x256_k64_w4_m16a"))
    assert e.value.status == ka.ERR_UNSUPPORTED
    with pytest.raises(ka.KernelArcError) as e:          # 64x64 waves cannot pair gate/up blocks
        ka.swiglu_i8(qx, sx, qw, sw, qw, sw, plan=names.index("tile_64x64_k64s4_w4"))
    assert e.value.status == ka.ERR_UNSUPPORTED
    big = torch.zeros(2, 65536 + 16, dtype=torch.int8, device="cuda")
    with pytest.raises(ka.KernelArcError) as e:          # K above 2^16
        ka.gemm_i8(big, sx[:2], big, sx[:2])
    assert e.value.status == ka.ERR_INVALID_ARG
    with pytest.raises(ValueError):
        ka.gemm_i8(qx, sx[:10], qw, sw)


def test_i8_graph_replay(ka):
    M, N, K = 512, 1024, 2048
    t = _inputs(M, N, K, 11, True, False)
    d = {k: v.cuda() for k, v in t.items() if v is not None}
    gu.note("i8 swiglu graph replay")
    eager = ka.swiglu_i8(d["qX"], d["sx"], d["qW"], d["sw"], d["qWu"], d["swu"])
    out = torch.empty_like(eager)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        ka.swiglu_i8(d["qX"], d["sx"], d["qW"], d["sw"], d["qWu"], d["swu"], out=out)
    torch.cuda.current_stream().wait_stream(s)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=s):
        ka.swiglu_i8(d["qX"], d["sx"], d["qW"], d["sw"], d["qWu"], d["swu"], out=out)
    for _ in range(3):
        out.zero_()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int16), eager.view(torch.int16))


@pytest.mark.parametrize("name", [w.name for w in wl.I8])
def test_i8_bench_workloads(ka, name):
    """The benchmark's INT8 shapes at full size with the plan the benchmark
    runs, on whole sampled rows and columns."""
    w = wl.I8_BY_NAME[name]
    t = wl.make_i8_inputs(w)
    gu.note(f"i8 bench {name} plan={ka.plan_name(ka.select_plan_i8(w.M, w.N, w.K, w.swiglu))}")
    got = _run(ka, t, w.swiglu)
    pos = gu.sample_positions(w.M, w.N, rows=4, cols=3, seed=w.seed)
    gu.check_tolerance(got[pos[0], pos[1]], _ref(t, w.swiglu, pos), name)
