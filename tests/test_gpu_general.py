"""GPU parity of the general form D = alpha X W^T + beta C + bias with
row-strided operands, against the CPU oracle's general form.

Tolerance as for the plain operator (per element, from the stated
acceptance bound): |D - Dref| <= 1e-2 * RMS(Dref) + 2^-7 * |Dref|.
Bitwise checks: alpha = beta = 1 without bias reproduces the plain entry
points exactly (same plan), and no element outside the rows' N columns of Y
is written (the padding of every strided Y keeps its sentinel bits).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_17071_amd import workloads as wl
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu

NAN_BITS = 0x7FC0
SENTINEL = 0x5A5A   # an ordinary finite bf16 pattern the kernels never write by chance


@pytest.fixture(scope="module")
def ka():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_17071_amd import kernelarc
    return kernelarc


def _bf16(g, shape, scale):
    return (torch.randn(shape, generator=g) * scale).to(torch.bfloat16)


def _padded_dev(t, pad, fill_bits):
    """t (2-D, CPU) as the leading columns of a wider GPU buffer; returns (buffer, view)."""
    rows, cols = t.shape
    fill = int(np.array(fill_bits, dtype=np.uint16).view(np.int16))
    buf = torch.full((rows, cols + pad), fill, dtype=torch.int16).view(torch.bfloat16)
    buf[:, :cols] = t
    buf = buf.cuda()
    return buf, buf[:, :cols]


def _general_case(ka, M, N, K, seed, alpha, beta, with_c, with_bias, pads=(8, 16, 8, 24), plan=None,
                  positions=None):
    g = torch.Generator().manual_seed(seed)
    X = _bf16(g, (M, K), K ** -0.5)
    W = _bf16(g, (N, K), K ** -0.5)
    C = _bf16(g, (M, N), 1.0)
    b = _bf16(g, (N,), 1.0)
    _, x = _padded_dev(X, pads[0], NAN_BITS)
    _, w = _padded_dev(W, pads[1], NAN_BITS)
    _, c = _padded_dev(C, pads[2], NAN_BITS)
    ybuf, y = _padded_dev(torch.zeros(M, N, dtype=torch.bfloat16), pads[3], SENTINEL)
    bias = b.cuda() if with_bias else None
    pname = ka.plan_name(plan) if plan is not None else "auto"
    gu.note(f"general M={M} N={N} K={K} seed={seed} alpha={alpha} beta={beta} C={with_c} bias={with_bias} "
            f"pads={pads} plan={pname}")
    ka.gemm_bf16_ex(x, w, c if with_c else None, bias, alpha, beta, out=y, plan=plan)
    torch.cuda.synchronize()
    orc = oracle.default()
    args = (wl.bits(X), wl.bits(W), wl.bits(C) if with_c else None, wl.bits(b) if with_bias else None,
            alpha, beta)
    got = gu.to_bits(y)
    if positions is None:
        ref = orc.linear_ex(*args)
        gu.check_tolerance(got, ref, f"general {pname} {M}x{N}x{K}")
    else:
        ref = orc.linear_ex_at(*args, positions[0], positions[1])
        gu.check_tolerance(got[positions[0], positions[1]], ref, f"general {pname} {M}x{N}x{K}")
    pad = wl.bits(ybuf[:, N:].cpu())
    assert (pad == SENTINEL).all(), "the kernel wrote past the N columns of a row of Y"


def _shape_for(name):
    if name == "gemv_valu_w4":
        return (3, 520, 264)
    if name.startswith("stream"):
        return (33, 264, 1032)
    if name.endswith("splitk") or name.endswith("tailsplit"):
        return (200, 264, 1032)
    return (77, 136, 520)


def _general_plan_names():
    from paper_2608_17071_amd import kernelarc
    return [n for n in kernelarc.plan_names()
            if n.startswith(("tile_", "stream_")) or n in ("gemv_valu_w4", "generic_64x64_scalar")]


@pytest.mark.parametrize("name", _general_plan_names())
def test_general_every_plan(ka, name):
    M, N, K = _shape_for(name)
    plan = ka.plan_names().index(name)
    _general_case(ka, M, N, K, 21, 0.75, -1.25, True, True, plan=plan)


@pytest.mark.parametrize("alpha,beta,with_c,with_bias", [
    (1.0, 1.0, True, False), (2.0, 0.5, True, True), (-0.5, 0.0, True, True),
    (1.0, 1.0, False, True), (0.3333333432674408, 3.0, True, False), (0.0, 1.0, True, True)])
@pytest.mark.parametrize("M,N,K", [(1, 1024, 512), (4, 96, 64), (16, 512, 1024), (64, 256, 768),
                                   (300, 520, 1032), (512, 1024, 3072)])
def test_general_scalars_and_shapes(ka, M, N, K, alpha, beta, with_c, with_bias):
    _general_case(ka, M, N, K, M + N + K, alpha, beta, with_c, with_bias)


@pytest.mark.parametrize("pads", [(0, 0, 0, 0), (8, 0, 3, 5), (3, 5, 0, 0), (0, 8, 16, 1)])
def test_general_strides(ka, pads):
    # odd X/W strides cannot take the 16-byte loads (generic kernel); odd
    # C/Y strides take the 2-byte epilogue of the MFMA kernels
    _general_case(ka, 96, 200, 136, 5, 1.5, 0.5, True, True, pads=pads)
    # the same strides on a streaming shape (16-row blocks, 16-bit R and Y)
    _general_case(ka, 24, 200, 1032, 6, 1.5, 0.5, True, True, pads=pads)


def test_general_bands(ka):
    # the banded plan with both column bands (4096 columns of 256x256 tiles,
    # 264 on the 128x128 tile) in the general form: strides, alpha, beta, bias
    plan = ka.plan_names().index("tile_256x256_k64_w4_m16a_bands")
    _general_case(ka, 4000, 4360, 200, 31, 0.75, -1.25, True, True, plan=plan)
    _general_case(ka, 4096, 4608, 136, 32, 1.0, 0.0, True, False, pads=(0, 8, 0, 16), plan=plan)


def test_general_large_k_ne_n(ka):
    # a decoder layer's down projection: K = 3.5 * hidden
    M, N, K = 4096, 4096, 14336
    pos = gu.sample_positions(M, N, rows=4, cols=3, seed=3)
    _general_case(ka, M, N, K, 9, 1.0, 1.0, True, True, pads=(0, 0, 0, 0), positions=pos)


@pytest.mark.parametrize("name", ["tile_256x256_k64_w8", "tile_64x64_k128s3_w4_splitk",
                                  "tile_256x128_k64s3_w8_lag", "gemv_valu_w4", "generic_64x64_scalar"])
def test_general_default_is_plain_bitwise(ka, name):
    plan = ka.plan_names().index(name)
    M, N, K = (2, 1024, 512) if name == "gemv_valu_w4" else (300, 520, 1032)
    g = torch.Generator().manual_seed(17)
    x = _bf16(g, (M, K), K ** -0.5).cuda()
    w = _bf16(g, (N, K), K ** -0.5).cuda()
    r = _bf16(g, (M, N), 1.0).cuda()
    gu.note(f"general-vs-plain {name} {M}x{N}x{K}")
    plain = ka.gemm_bf16_with_plan(plan, x, w, r)
    gen = ka.gemm_bf16_ex(x, w, r, None, 1.0, 1.0, plan=plan)
    plain0 = ka.gemm_bf16_with_plan(plan, x, w, None)
    gen0 = ka.gemm_bf16_ex(x, w, None, None, 1.0, 1.0, plan=plan)
    torch.cuda.synchronize()
    assert torch.equal(plain.view(torch.int16), gen.view(torch.int16))
    assert torch.equal(plain0.view(torch.int16), gen0.view(torch.int16))


def test_general_beta_zero_does_not_read_c(ka):
    M, N, K = 64, 256, 512
    g = torch.Generator().manual_seed(4)
    x = _bf16(g, (M, K), K ** -0.5).cuda()
    w = _bf16(g, (N, K), K ** -0.5).cuda()
    b = _bf16(g, (N,), 1.0).cuda()
    c = torch.full((M, N), float("nan"), dtype=torch.bfloat16, device="cuda")
    gu.note("general beta=0 NaN C")
    y = ka.gemm_bf16_ex(x, w, c, b, 1.0, 0.0)
    y0 = ka.gemm_bf16_ex(x, w, None, b, 1.0, 1.0)
    torch.cuda.synchronize()
    assert torch.isfinite(y.float()).all()
    assert torch.equal(y.view(torch.int16), y0.view(torch.int16))


@pytest.mark.parametrize("M", [200, 16])
def test_general_in_place(ka, M):
    N, K = 264, 520
    g = torch.Generator().manual_seed(6)
    X = _bf16(g, (M, K), K ** -0.5)
    W = _bf16(g, (N, K), K ** -0.5)
    C = _bf16(g, (M, N), 1.0)
    b = _bf16(g, (N,), 1.0)
    cbuf, c = _padded_dev(C, 8, NAN_BITS)
    gu.note("general in place Y == C")
    ka.gemm_bf16_ex(X.cuda(), W.cuda(), c, b.cuda(), 0.5, 2.0, out=c)
    torch.cuda.synchronize()
    ref = oracle.default().linear_ex(wl.bits(X), wl.bits(W), wl.bits(C), wl.bits(b), 0.5, 2.0)
    gu.check_tolerance(gu.to_bits(c), ref, "general in place")


def test_general_rejects(ka):
    g = torch.Generator().manual_seed(7)
    x = _bf16(g, (64, 128), 1.0).cuda()
    w = _bf16(g, (96, 128), 1.0).cuda()
    c = _bf16(g, (64, 96), 1.0).cuda()
    gemv = ka.plan_names().index("gemv_valu_w4")
    gu.note("general rejects")
    with pytest.raises(ka.KernelArcError) as e:
        ka.gemm_bf16_ex(x[:16], w, c[:16], None, 2.0, 1.0, plan=gemv)     # the GEMV takes at most 4 rows
    assert e.value.status == ka.ERR_UNSUPPORTED
    big = torch.zeros(64, 200, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(ka.KernelArcError) as e:                            # Y partially overlaps C
        ka.gemm_bf16_ex(x, w, big[:, :96], None, 1.0, 1.0, out=big[:, 8:104])
    assert e.value.status == ka.ERR_INVALID_ARG


def test_general_graph_replay(ka):
    M, N, K = 512, 1024, 3072
    g = torch.Generator().manual_seed(8)
    x = _bf16(g, (M, K), K ** -0.5).cuda()
    w = _bf16(g, (N, K), K ** -0.5).cuda()
    c = _bf16(g, (M, N), 1.0).cuda()
    b = _bf16(g, (N,), 1.0).cuda()
    gu.note("general graph replay")
    eager = ka.gemm_bf16_ex(x, w, c, b, 0.5, 1.0)
    out = torch.empty_like(eager)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        ka.gemm_bf16_ex(x, w, c, b, 0.5, 1.0, out=out)   # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(s)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=s):
        ka.gemm_bf16_ex(x, w, c, b, 0.5, 1.0, out=out)
    for _ in range(3):
        out.zero_()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int16), eager.view(torch.int16))


@pytest.mark.parametrize("name", [w.name for w in wl.GENERAL])
def test_general_bench_workloads(ka, name):
    """The benchmark's general-form shapes, launched as the benchmark launches
    them (X through its row stride, the selected plan), on sampled outputs."""
    w = wl.GENERAL_BY_NAME[name]
    t = wl.make_general_inputs(w)
    xbuf = torch.zeros((w.M, w.ldx), dtype=torch.bfloat16)
    xbuf[:, :w.K] = t["X"]
    xbuf = xbuf.cuda()
    c = t["C"].cuda() if t["C"] is not None else None
    b = t["bias"].cuda() if t["bias"] is not None else None
    plan = ka.select_plan_ex(w.M, w.N, w.K, w.has_c, w.ldx, w.K, w.N, w.N, w.alpha, w.beta, w.has_bias)
    gu.note(f"general bench {name} plan={ka.plan_name(plan)}")
    y = ka.gemm_bf16_ex(xbuf[:, :w.K], t["W"].cuda(), c, b, w.alpha, w.beta)
    torch.cuda.synchronize()
    pos = gu.sample_positions(w.M, w.N, rows=4, cols=3, seed=w.seed)
    ref = oracle.default().linear_ex_at(wl.bits(t["X"]), wl.bits(t["W"]), wl.bits(t["C"]) if t["C"] is not None else None,
                                        wl.bits(t["bias"]) if t["bias"] is not None else None, w.alpha, w.beta,
                                        pos[0], pos[1])
    gu.check_tolerance(gu.to_bits(y)[pos[0], pos[1]], ref, name)
