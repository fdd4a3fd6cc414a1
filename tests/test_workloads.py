"""Seeded input generation: determinism and the stated distributions."""
import math

import numpy as np
import torch

import oracle
from paper_2608_17071_amd import workloads as wl


def test_named_configs():
    assert (wl.TINY.M, wl.TINY.N, wl.TINY.K) == (128, 256, 256)
    assert (wl.DECODE.M, wl.DECODE.N, wl.DECODE.K) == (16, 4096, 4096)
    assert (wl.PREFILL.M, wl.PREFILL.N, wl.PREFILL.K) == (4096, 4096, 4096)
    assert (wl.SQUARE.M, wl.SQUARE.N, wl.SQUARE.K, wl.SQUARE.residual) == (8192, 8192, 8192, False)
    assert len(wl.SWEEP) == 16
    assert [w.seed for w in wl.SWEEP] == list(range(16))
    assert {(w.M, w.K) for w in wl.SWEEP} == {(m, h) for m in wl.SWEEP_M for h in wl.SWEEP_HIDDEN}
    assert all(w.N == w.K for w in wl.SWEEP)


def test_deterministic():
    a = wl.make_inputs(wl.TINY)
    b = wl.make_inputs(wl.TINY)
    assert wl.sha256(a["X"], a["W"], a["R"]) == wl.sha256(b["X"], b["W"], b["R"])
    c = wl.make_inputs(wl.custom(128, 256, 256, seed=1))
    assert wl.sha256(c["X"]) != wl.sha256(a["X"])


def test_distributions():
    w = wl.custom(256, 512, 1024)
    t = wl.make_inputs(w)
    x = t["X"].float()
    assert abs(x.std().item() * math.sqrt(1024) - 1) < 0.02
    assert abs(t["R"].float().std().item() - 1) < 0.02
    u = wl.make_inputs(wl.custom(256, 512, 1024, residual=False, dist="uniform"))
    xu = u["X"].float() * math.sqrt(1024)
    assert u["R"] is None
    assert xu.min() >= -1 and xu.max() <= 1 and abs(xu.std().item() - 1 / math.sqrt(3)) < 0.02


def test_output_rms_matches_stated_scale():
    """RMS(Yref): about sqrt(1 + 1/K) with a residual, 1/(3 sqrt K) for uniform plain."""
    orc = oracle.default()
    w = wl.TINY
    t = wl.make_inputs(w)
    Y = orc.linear(wl.bits(t["X"]), wl.bits(t["W"]), wl.bits(t["R"]))
    assert abs(np.sqrt(np.mean(Y ** 2)) - math.sqrt(1 + 1 / w.K)) < 0.03
    u = wl.make_inputs(wl.custom(64, 512, 1024, residual=False, dist="uniform"))
    Yu = orc.linear(wl.bits(u["X"]), wl.bits(u["W"]), None)
    assert abs(np.sqrt(np.mean(Yu ** 2)) * 3 * math.sqrt(1024) - 1) < 0.05


def test_rank1_inputs_are_exact():
    X, W, R, a, b, u, v = wl.rank1_integer(16, 24, 300, seed=3)
    np.testing.assert_array_equal(X.float().numpy(), np.outer(a, u))
    np.testing.assert_array_equal(W.float().numpy(), np.outer(b, v))
    assert R.float().abs().max() <= 64
    assert len(set(u.tolist())) > 1 and len(set(v.tolist())) > 1


def test_bits_roundtrip():
    t = torch.randn(5, 7).to(torch.bfloat16)
    assert torch.equal(wl.from_bits(wl.bits(t)), t)
