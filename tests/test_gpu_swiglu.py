"""GPU parity of SwiGLU, H = silu(X Wg^T) * (X Wu^T), against the CPU oracle.

Tolerance per element, the acceptance bound of the plain operator:
|H - Href| <= 1e-2 * RMS(Href) + 2^-7 * |Href|.  The kernels keep the gate
and up sums in fp32 (their error is far below the absolute term), SiLU is
within a few fp32 ulps and |silu'| <= 1.1, so the single bf16 rounding of H
(at most 2^-8 |H|) dominates.  Bitwise checks: a merged [2N, K] weight gives
the same bits as two separate ones, repeated calls and graph replays give
identical bits.
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


def _inputs(M, N, K, seed, x_scale=1.0):
    g = torch.Generator().manual_seed(seed)
    X = (torch.randn((M, K), generator=g) * x_scale).to(torch.bfloat16)
    s = K ** -0.5 if K > 0 else 1.0
    Wg = (torch.randn((N, K), generator=g) * s).to(torch.bfloat16)
    Wu = (torch.randn((N, K), generator=g) * s).to(torch.bfloat16)
    return X, Wg, Wu


def _check(ka, X, Wg, Wu, what, plan=None, positions=None):
    M, N = X.shape[0], Wg.shape[0]
    pname = ka.plan_name(plan) if plan is not None else ka.plan_name(ka.select_plan_swiglu(M, N, X.shape[1]))
    gu.note(f"swiglu {what} M={M} N={N} K={X.shape[1]} plan={pname}")
    h = ka.swiglu_bf16(X.cuda(), Wg.cuda(), Wu.cuda(), plan=plan)
    torch.cuda.synchronize()
    got = gu.to_bits(h)
    orc = oracle.default()
    if positions is None:
        ref = orc.swiglu(wl.bits(X), wl.bits(Wg), wl.bits(Wu))
        gu.check_tolerance(got, ref, f"swiglu {what} {pname}")
    else:
        ref = orc.swiglu_at(wl.bits(X), wl.bits(Wg), wl.bits(Wu), positions[0], positions[1])
        gu.check_tolerance(got[positions[0], positions[1]], ref, f"swiglu {what} {pname}")
    return got


def _glu_plan_names():
    from paper_2608_17071_amd import kernelarc
    names = kernelarc.plan_names()
    return [n for i, n in enumerate(names) if kernelarc.plan_supports_swiglu(i, 200, 264, 1032)]


def _shape_for(name):
    if name.endswith("splitk") or name.endswith("tailsplit"):
        return (200, 264, 1032)
    return (77, 136, 520)


@pytest.mark.parametrize("name", _glu_plan_names())
def test_swiglu_every_plan(ka, name):
    """Every plan that computes SwiGLU, over several tiles with ragged M, N and K tails."""
    M, N, K = _shape_for(name)
    plan = ka.plan_names().index(name)
    X, Wg, Wu = _inputs(M, N, K, 31)
    _check(ka, X, Wg, Wu, "every-plan", plan=plan)


@pytest.mark.parametrize("M,N,K", [(1, 1024, 512), (3, 200, 64), (16, 4096, 1024), (32, 520, 264),
                                   (33, 264, 520), (64, 1000, 1032), (257, 136, 256), (512, 2048, 3072),
                                   (130, 100, 136), (40, 77, 96), (64, 96, 250), (5, 7, 9), (64, 256, 0)])
def test_swiglu_shapes(ka, M, N, K):
    """Selected plans over skinny and ragged shapes, N not a multiple of 8 (2-byte
    stores), K not a multiple of 8 (generic kernel) and K = 0 (H = 0)."""
    X, Wg, Wu = _inputs(M, N, K, M * 7 + N + K)
    got = _check(ka, X, Wg, Wu, "shapes")
    if K == 0:
        assert (gu.bf16_bits_to_f64(got) == 0).all()


def test_swiglu_saturated_gates(ka):
    """Gate sums far beyond SiLU's curve (|G| up to ~150): H = G U on the
    right, H = 0 (no NaN) on the left, as the oracle has them."""
    X, Wg, Wu = _inputs(256, 512, 256, 5, x_scale=40.0)
    _check(ka, X, Wg, Wu, "saturated")
    X, Wg, Wu = _inputs(256, 512, 256, 6, x_scale=40.0)
    _check(ka, X, Wg, Wu, "saturated-generic", plan=ka.plan_names().index("generic_64x64_scalar"))


def test_swiglu_merged_weight_bitwise(ka):
    """A merged [2N, K] gate_up weight passed as its two halves gives the bits
    of two separate weights."""
    M, N, K = 300, 520, 1032
    X, Wg, Wu = _inputs(M, N, K, 8)
    merged = torch.cat([Wg, Wu], 0).cuda()
    x = X.cuda()
    gu.note("swiglu merged weight")
    a = ka.swiglu_bf16(x, merged[:N], merged[N:])
    b = ka.swiglu_bf16(x, Wg.cuda(), Wu.cuda())
    c = ka.swiglu_bf16(x, Wg.cuda(), Wu.cuda())
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    assert torch.equal(b.view(torch.int16), c.view(torch.int16))


def test_swiglu_same_gate_and_up(ka):
    """Wg == Wu (one buffer for both): H = silu(G) G."""
    X, Wg, _ = _inputs(128, 256, 512, 9)
    _check(ka, X, Wg, Wg, "wg-is-wu")


def test_swiglu_leading_dims(ka):
    """X with leading dimensions [B, T, K] is flattened to M = B*T."""
    B, T, K, N = 3, 37, 264, 136
    g = torch.Generator().manual_seed(10)
    X = torch.randn((B, T, K), generator=g).to(torch.bfloat16)
    Wg = (torch.randn((N, K), generator=g) * K ** -0.5).to(torch.bfloat16)
    Wu = (torch.randn((N, K), generator=g) * K ** -0.5).to(torch.bfloat16)
    gu.note("swiglu leading dims")
    h = ka.swiglu_bf16(X.cuda(), Wg.cuda(), Wu.cuda())
    torch.cuda.synchronize()
    assert tuple(h.shape) == (B, T, N)
    ref = oracle.default().swiglu(wl.bits(X.reshape(B * T, K)), wl.bits(Wg), wl.bits(Wu))
    gu.check_tolerance(gu.to_bits(h.reshape(B * T, N)), ref, "swiglu leading dims")


def test_swiglu_rejects(ka):
    x = torch.zeros(64, 128, dtype=torch.bfloat16, device="cuda")
    w = torch.zeros(96, 128, dtype=torch.bfloat16, device="cuda")
    gu.note("swiglu rejects")
    names = ka.plan_names()
    for n in ("stream_mfma16_k64_splitk", "tile_64x64_k64s4_w4", "gemv_valu_w4"):
        with pytest.raises(ka.KernelArcError) as e:
            ka.swiglu_bf16(x, w, w, plan=names.index(n))
        assert e.value.status == ka.ERR_UNSUPPORTED
    buf = torch.zeros(64 * 128, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(ka.KernelArcError) as e:                  # H overlaps X
        ka.swiglu_bf16(buf.view(64, 128), w, w, out=buf[:64 * 96].view(64, 96))
    assert e.value.status == ka.ERR_INVALID_ARG
    with pytest.raises(ValueError):
        ka.swiglu_bf16(x, w, w[:64])


def test_swiglu_graph_replay(ka):
    M, N, K = 512, 1024, 2048
    X, Wg, Wu = _inputs(M, N, K, 11)
    x, g, u = X.cuda(), Wg.cuda(), Wu.cuda()
    gu.note("swiglu graph replay")
    eager = ka.swiglu_bf16(x, g, u)
    out = torch.empty_like(eager)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        ka.swiglu_bf16(x, g, u, out=out)
    torch.cuda.current_stream().wait_stream(s)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=s):
        ka.swiglu_bf16(x, g, u, out=out)
    for _ in range(3):
        out.zero_()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int16), eager.view(torch.int16))


@pytest.mark.parametrize("name", [w.name for w in wl.GLU])
def test_swiglu_bench_workloads(ka, name):
    """The benchmark's SwiGLU shapes at full size, with the plan the benchmark
    runs, on whole sampled rows and columns."""
    w = wl.GLU_BY_NAME[name]
    t = wl.make_glu_inputs(w)
    pos = gu.sample_positions(w.M, w.N, rows=4, cols=3, seed=w.seed)
    _check(ka, t["X"], t["Wg"], t["Wu"], f"bench {name}", positions=pos)
