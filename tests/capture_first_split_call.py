"""Run as its own process by test_gpu_capture.py (a fresh process, so the
split-K workspace does not exist yet): the first call of a split-K plan made
under stream capture must return KERNELARC_ERR_UNSUPPORTED without touching
the stream, the capture must end normally, and the same call made eagerly
afterwards must allocate the workspace and compute the right result.
Prints one line starting with CAPTURE_OK on success."""
import os
import sys

import torch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from paper_2608_17071_amd import kernelarc as ka  # noqa: E402
from paper_2608_17071_amd import workloads as wl  # noqa: E402


def main():
    M, N, K = 512, 4096, 4096
    plan = ka.select_plan(M, N, K, True)
    print(f"[capture] plan={ka.plan_name(plan)} M={M} N={N} K={K}", flush=True)
    assert ka.kernelarc_plan_uses_workspace(plan, M, N, K) == 1
    t = wl.make_inputs(wl.custom(M, N, K, seed=80))
    x, w, r = t["X"].cuda(), t["W"].cuda(), t["R"].cuda()
    # a call that needs no workspace first, so the device is probed before capture
    ka.gemm_bf16_residual(x[:1], w, r[:1])
    torch.cuda.synchronize()
    y = torch.empty(M, N, dtype=torch.bfloat16, device="cuda")
    s = torch.cuda.Stream()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        st = ka.kernelarc_gemm_bf16_residual(M, N, K, x.data_ptr(), w.data_ptr(), r.data_ptr(), y.data_ptr(),
                                             s.cuda_stream)
        err = ka.kernelarc_last_error()
    torch.cuda.synchronize()
    assert st == ka.ERR_UNSUPPORTED, (st, err)
    assert b"capture" in err, err
    print(f"[capture] under capture: status {st}: {err.decode()}", flush=True)
    y1 = ka.gemm_bf16_residual(x, w, r)          # allocates and clears the workspace
    y2 = ka.gemm_bf16_residual(x, w, r)          # reuses it
    ref = ka.gemm_bf16_with_plan(ka.plan_names().index("tile_128x128_k64_w4"), x, w, r)   # no split
    torch.cuda.synchronize()
    assert torch.equal(y1, y2)
    diff = (y1.float() - ref.float()).abs().max().item()
    bound = 1e-2 * ref.float().pow(2).mean().sqrt().item() + 2.0 ** -7 * ref.float().abs().max().item()
    assert diff <= bound, (diff, bound)
    print(f"CAPTURE_OK max |split - unsplit| {diff:.3g}", flush=True)


if __name__ == "__main__":
    main()
