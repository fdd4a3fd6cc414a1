"""GPU parity of the grouped (per-expert) forms over an expert-major padded
layout against the CPU oracle: per group g and valid row i < counts[g]
(clamped to [0, M_pad]), Y[g,i] = X[g,i] W[g]^T, or the SwiGLU form.

Tolerance per element as for the plain operator:
|Y - Yref| <= 1e-2 * RMS(Yref) + 2^-7 * |Yref|.  Bitwise checks: gap rows of
the output keep their sentinel bits; NaN in the gap rows of X does not reach
any output (gap rows are never read); each group's rows equal, bit for bit,
the plain entry point run with the same tile plan on that group alone.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_17071_amd import workloads as wl
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu

SENTINEL = 0x5A5A


@pytest.fixture(scope="module")
def ka():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_17071_amd import kernelarc
    return kernelarc


def _inputs(G, Mpad, N, K, counts, seed, glu, gap_nan=True):
    g = torch.Generator().manual_seed(seed)
    X = torch.randn((G, Mpad, K), generator=g).to(torch.bfloat16)
    s = K ** -0.5 if K > 0 else 1.0
    W = (torch.randn((G, N, K), generator=g) * s).to(torch.bfloat16)
    Wu = (torch.randn((G, N, K), generator=g) * s).to(torch.bfloat16) if glu else None
    if counts is not None and gap_nan:
        for e in range(G):
            r = min(max(int(counts[e]), 0), Mpad)
            X[e, r:] = float("nan")          # gap rows must never be read
    return X, W, Wu


def _run(ka, X, W, Wu, counts, plan=None):
    G, Mpad, _ = X.shape
    N = W.shape[1]
    fill = int(np.array(SENTINEL, dtype=np.uint16).view(np.int16))
    out = torch.full((G, Mpad, N), fill, dtype=torch.int16).view(torch.bfloat16).cuda()
    c = torch.from_numpy(np.asarray(counts, dtype=np.int32)).cuda() if counts is not None else None
    if Wu is None:
        ka.gemm_bf16_grouped(X.cuda(), W.cuda(), c, out=out, plan=plan)
    else:
        ka.swiglu_bf16_grouped(X.cuda(), W.cuda(), Wu.cuda(), c, out=out, plan=plan)
    torch.cuda.synchronize()
    return gu.to_bits(out)


def _check(ka, G, Mpad, N, K, counts, seed, glu, plan=None, what=""):
    X, W, Wu = _inputs(G, Mpad, N, K, counts, seed, glu)
    pname = ka.plan_name(plan) if plan is not None else ka.plan_name(ka.select_plan_grouped(G, Mpad, N, K, glu))
    gu.note(f"grouped {'swiglu' if glu else 'gemm'} {what} G={G} Mpad={Mpad} N={N} K={K} counts={counts} plan={pname}")
    got = _run(ka, X, W, Wu, counts, plan)
    orc = oracle.default()
    cnt = np.asarray(counts, dtype=np.int32) if counts is not None else None
    ref = (orc.grouped_swiglu(wl.bits(X), wl.bits(W), wl.bits(Wu), cnt) if glu
           else orc.grouped_linear(wl.bits(X), wl.bits(W), cnt))
    valid = ~np.isnan(ref)
    assert (got[~valid] == SENTINEL).all(), "a gap row of the output was written"
    gu.check_tolerance(got[valid], ref[valid], f"grouped {what} {pname}")
    return X, W, Wu, got


def _plans(glu):
    from paper_2608_17071_amd import kernelarc
    names = kernelarc.plan_names()
    return [n for i, n in enumerate(names) if kernelarc.plan_supports_grouped(i, 5, 130, 264, 520, glu)]


COUNTS = [0, 1, 64, 130, 77]


@pytest.mark.parametrize("name", _plans(False))
def test_grouped_gemm_every_plan(ka, name):
    _check(ka, 5, 130, 136, 520, COUNTS, 61, False, plan=ka.plan_names().index(name), what="every-plan")


@pytest.mark.parametrize("name", _plans(True))
def test_grouped_swiglu_every_plan(ka, name):
    _check(ka, 5, 130, 136, 520, COUNTS, 62, True, plan=ka.plan_names().index(name), what="every-plan")


@pytest.mark.parametrize("glu", [False, True])
@pytest.mark.parametrize("G,Mpad,N,K,counts", [
    (3, 64, 256, 256, None), (4, 96, 520, 264, [-5, 1000, 96, 33]), (7, 33, 100, 136, [33, 0, 0, 5, 17, 32, 1]),
    (2, 300, 1024, 1032, [300, 257]), (6, 40, 77, 96, [40, 39, 1, 0, 8, 20]), (3, 50, 64, 250, [50, 10, 49]),
    (1, 16, 8, 0, [16]), (256, 32, 128, 256, list(range(0, 512, 2)))])
def test_grouped_shapes(ka, G, Mpad, N, K, counts, glu):
    """Selected plans: no counts, clamped counts, empty groups, ragged N and K,
    K not a multiple of 8 (generic), K = 0, 256 experts."""
    _check(ka, G, Mpad, N, K, counts, G + Mpad + N + K, glu, what="shapes")


@pytest.mark.parametrize("name", ["tile_128x128_k64s4_w4_lag", "tile_256x256_k64_w8", "tile_64x128_k64s4_w4"])
def test_grouped_equals_plain_per_group(ka, name):
    """Each group's rows are the plain entry point's bits with the same tile plan."""
    plan = ka.plan_names().index(name)
    counts = [70, 0, 130, 5]
    X, W, _ = _inputs(4, 130, 264, 520, counts, 63, False, gap_nan=False)
    gu.note(f"grouped equals plain {name}")
    got = _run(ka, X, W, None, counts, plan)
    for e, r in enumerate(counts):
        if r == 0:
            continue
        y = ka.gemm_bf16_with_plan(plan, X[e, :r].contiguous().cuda(), W[e].contiguous().cuda())
        torch.cuda.synchronize()
        np.testing.assert_array_equal(got[e, :r], gu.to_bits(y))


def test_grouped_rejects(ka):
    gu.note("grouped rejects")
    names = ka.plan_names()
    x = torch.zeros(4, 64, 128, dtype=torch.bfloat16, device="cuda")
    w = torch.zeros(4, 96, 128, dtype=torch.bfloat16, device="cuda")
    for n in ("tile_128x128_k64_w4_splitk", "tile_256x256_k64_w8_tailsplit", "stream_mfma16_k64_splitk",
              "gemv_valu_w4"):
        with pytest.raises(ka.KernelArcError) as e:
            ka.gemm_bf16_grouped(x, w, plan=names.index(n))
        assert e.value.status == ka.ERR_UNSUPPORTED
    with pytest.raises(ka.KernelArcError) as e:
        ka.swiglu_bf16_grouped(x, w, w, plan=names.index("tile_64x64_k64s4_w4"))
    assert e.value.status == ka.ERR_UNSUPPORTED
    with pytest.raises(ValueError):
        ka.gemm_bf16_grouped(x, w, torch.zeros(3, dtype=torch.int32, device="cuda"))


def test_grouped_counts_from_device_and_graph_replay(ka):
    """counts produced on the device by an earlier kernel of the same stream,
    and HIP-graph replays with counts changed between replays."""
    G, Mpad, N, K = 16, 64, 512, 256
    X, W, _ = _inputs(G, Mpad, N, K, None, 64, False)
    x, w = X.cuda(), W.cuda()
    counts = torch.zeros(G, dtype=torch.int32, device="cuda")
    out = torch.zeros((G, Mpad, N), dtype=torch.bfloat16, device="cuda")
    gu.note("grouped graph replay")
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        ka.gemm_bf16_grouped(x, w, counts, out=out)
    torch.cuda.current_stream().wait_stream(s)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=s):
        ka.gemm_bf16_grouped(x, w, counts, out=out)
    orc = oracle.default()
    for rep in range(3):
        c = (torch.arange(G, dtype=torch.int32, device="cuda") * (rep + 1) * 3) % (Mpad + 1)
        counts.copy_(c)
        out.zero_()
        graph.replay()
        torch.cuda.synchronize()
        cn = c.cpu().numpy()
        ref = orc.grouped_linear(wl.bits(X), wl.bits(W), cn)
        valid = ~np.isnan(ref)
        got = gu.to_bits(out)
        gu.check_tolerance(got[valid], ref[valid], f"grouped replay {rep}")
        assert (got[~valid] == 0).all()


@pytest.mark.parametrize("name", [w.name for w in wl.GROUPED])
def test_grouped_bench_workloads(ka, name):
    """The benchmark's mixture-of-experts shapes at full size with the plan the
    benchmark runs, checked on sampled valid rows of sampled experts."""
    w = wl.GROUPED_BY_NAME[name]
    t = wl.make_grouped_inputs(w, device="cuda")
    plan = ka.select_plan_grouped(w.G, t["Mpad"], w.N, w.K, w.swiglu)
    gu.note(f"grouped bench {name} plan={ka.plan_name(plan)}")
    cnt = t["counts"].cpu().numpy()
    got = _run(ka, t["X"], t["W"], t.get("Wu"), cnt, None)
    rng = np.random.default_rng(w.seed)
    groups = np.sort(rng.choice(w.G, 6, replace=False))
    # the sampled experts' operands, copied to the host as a 6-group problem
    sel = torch.from_numpy(groups).to(t["X"].device)
    sub = {k: wl.bits(t[k].index_select(0, sel).cpu()) for k in ("X", "W", "Wu") if k in t}
    scnt = cnt[groups].copy()
    gi, ri, ci = [], [], []
    for s_, e in enumerate(groups):
        for r in sorted(set([0, int(cnt[e]) - 1] + list(rng.integers(0, cnt[e], 2)))):
            gi += [s_] * w.N
            ri += [r] * w.N
            ci += list(range(w.N))
    gi, ri, ci = np.array(gi), np.array(ri), np.array(ci)
    ref = oracle.default().grouped_at(sub["X"], sub["W"], sub.get("Wu"), scnt, gi, ri, ci)
    gu.check_tolerance(got[groups[gi], ri, ci], ref, name)
    for e in groups:
        assert (got[e, cnt[e]:] == SENTINEL).all()
