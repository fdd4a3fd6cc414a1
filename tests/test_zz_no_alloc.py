"""kernelarc_gemm_bf16_residual_noalloc: the entry point for callers that
cannot allocate.  Its split-K partials live in the library's static scratch;
its results must equal kernelarc_gemm_bf16_residual's (same plans, same
kernels) bit for bit, on consecutive calls that reuse the scratch (the second
smaller than the first), for the plain form (R == NULL), and on HIP-graph
replays of a captured call.
"""
import numpy as np
import pytest
import torch

from paper_2608_17071_amd import workloads as wl
from tests import gpu_util as gu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ka():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_17071_amd import kernelarc
    return kernelarc


def _inputs(M, N, K, seed):
    t = wl.make_inputs(wl.custom(M, N, K, seed=seed))
    return t["X"].cuda(), t["W"].cuda(), t["R"].cuda()


def _noalloc_raw(ka, x, w, r, y):
    """Through the C ABI with raw pointers on the current stream."""
    M, K = x.shape
    N = w.shape[0]
    st = ka.kernelarc_gemm_bf16_residual_noalloc(M, N, K, x.data_ptr(), w.data_ptr(),
                                                 r.data_ptr() if r is not None else None, y.data_ptr(),
                                                 torch.cuda.current_stream().cuda_stream)
    assert st == ka.OK, ka.kernelarc_last_error()


# (M, N, K): consecutive calls, each with a smaller output than the one
# before; the plans split K through the scratch (tail split of 256x256
# tiles, 128x128 split-K, the streaming kernel's split), run two column
# bands, or (the last shape) do not split at all.
SEQUENCE = [(6144, 2816, 4096), (4096, 5120, 5120), (512, 4096, 4096), (16, 8192, 8192), (64, 4096, 4096),
            (300, 520, 264)]


def test_matches_the_allocating_entry_point(ka):
    for i, (M, N, K) in enumerate(SEQUENCE):
        plan = ka.plan_name_for(M, N, K, True)
        x, w, r = _inputs(M, N, K, seed=60 + i)
        gu.note(f"noalloc vs residual entry {M}x{N}x{K} plan={plan}")
        want = ka.gemm_bf16_residual(x, w, r)
        want_plain = ka.gemm_bf16(x, w)
        y = torch.full((M, N), float("nan"), dtype=torch.bfloat16, device="cuda")
        _noalloc_raw(ka, x, w, r, y)
        yp = torch.full((M, N), float("nan"), dtype=torch.bfloat16, device="cuda")
        _noalloc_raw(ka, x, w, None, yp)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(gu.to_bits(y), gu.to_bits(want), err_msg=f"{M}x{N}x{K} {plan}")
        np.testing.assert_array_equal(gu.to_bits(yp), gu.to_bits(want_plain), err_msg=f"{M}x{N}x{K} plain")
    # in place (Y == R) through the binding
    M, N, K = SEQUENCE[2]
    x, w, r = _inputs(M, N, K, seed=70)
    want = gu.to_bits(ka.gemm_bf16_residual(x, w, r))
    out = ka.gemm_bf16_residual_noalloc(x, w, r, out=r)
    torch.cuda.synchronize()
    assert out.data_ptr() == r.data_ptr()
    np.testing.assert_array_equal(gu.to_bits(r), want)


def test_graph_replays(ka):
    """A captured call replays correctly, with eager no-alloc calls of another
    shape between the replays (they reuse the same scratch)."""
    M, N, K = 512, 4096, 4096
    x, w, r = _inputs(M, N, K, seed=71)
    x2, w2, r2 = _inputs(64, 4096, 4096, seed=72)
    eager = gu.to_bits(ka.gemm_bf16_residual(x, w, r))
    eager2 = gu.to_bits(ka.gemm_bf16_residual(x2, w2, r2))
    y = torch.empty(M, N, dtype=torch.bfloat16, device="cuda")
    y2 = torch.empty(64, 4096, dtype=torch.bfloat16, device="cuda")
    torch.cuda.synchronize()
    gu.note(f"noalloc graph capture {M}x{N}x{K}")
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        ka.gemm_bf16_residual_noalloc(x, w, r, out=y)
    for rep in range(3):
        y.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        np.testing.assert_array_equal(gu.to_bits(y), eager, err_msg=f"replay {rep}")
        ka.gemm_bf16_residual_noalloc(x2, w2, r2, out=y2)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(gu.to_bits(y2), eager2, err_msg=f"eager after replay {rep}")


def test_rejects_like_the_residual_entry_point(ka):
    x, w, r = _inputs(16, 64, 64, seed=73)
    y = torch.empty(16, 64, dtype=torch.bfloat16, device="cuda")
    f = ka.kernelarc_gemm_bf16_residual_noalloc
    s = torch.cuda.current_stream().cuda_stream
    assert f(-1, 64, 64, x.data_ptr(), w.data_ptr(), r.data_ptr(), y.data_ptr(), s) == ka.ERR_INVALID_ARG
    assert f(16, 64, 64, x.data_ptr(), w.data_ptr(), r.data_ptr(), None, s) == ka.ERR_INVALID_ARG
    assert f(16, 64, 64, x.data_ptr(), w.data_ptr(), r.data_ptr(), x.data_ptr(), s) == ka.ERR_INVALID_ARG
    assert f(0, 64, 64, None, None, None, None, s) == ka.OK
