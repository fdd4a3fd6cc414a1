"""Helpers shared by the GPU tests: run the HIP library, check against the oracle."""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle
from oracle import bf16_bits_to_f64
from paper_2608_17071_amd import workloads as wl

# Acceptance bound per element: |Y - Yref| <= 1e-2 * RMS(Yref) + 2^-7 * |Yref|
REL = 2.0 ** -7
ABS_RMS = 1e-2


def note(msg: str) -> None:
    """Name the case about to run on the GPU (flushed, so a fault still shows it)."""
    print(f"[gpu-case] {msg}", flush=True)
    sys.stdout.flush()


def dev(t):
    return None if t is None else t.cuda()


def to_bits(y: torch.Tensor) -> np.ndarray:
    return wl.bits(y.cpu())


def run_library(X, W, R, plan=None, residual=None, out=None):
    """Run one call on cuda:0; returns the output as bf16 bit patterns."""
    from paper_2608_17071_amd import kernelarc as ka
    if residual is None:
        residual = R is not None
    x, w = dev(X), dev(W)
    r = dev(R) if residual else None
    if plan is None:
        y = ka.gemm_bf16_residual(x, w, r, out=out) if residual else ka.gemm_bf16(x, w, out=out)
    else:
        y = ka.gemm_bf16_with_plan(plan, x, w, r, out=out)
    torch.cuda.synchronize()
    return to_bits(y)


def check_tolerance(y_bits: np.ndarray, yref: np.ndarray, what: str, rms: float | None = None) -> float:
    """Assert the acceptance bound element by element; returns max error/bound."""
    y = bf16_bits_to_f64(y_bits)
    assert np.all(np.isfinite(y)), f"{what}: non-finite output"
    if rms is None:
        rms = float(np.sqrt(np.mean(yref ** 2))) if yref.size else 0.0
    bound = ABS_RMS * rms + REL * np.abs(yref)
    err = np.abs(y - yref)
    ratio = float(np.max(err / np.maximum(bound, 1e-300))) if y.size else 0.0
    if ratio > 1.0:
        idx = np.unravel_index(int(np.argmax(err / np.maximum(bound, 1e-300))), err.shape)
        raise AssertionError(f"{what}: max err/bound {ratio:.3f} at {idx}: y={y[idx]!r} ref={yref[idx]!r}")
    return ratio


def sample_positions(M: int, N: int, rows: int = 6, cols: int = 4, seed: int = 0):
    """Whole rows and whole columns (always the first and last), as index arrays."""
    rng = np.random.default_rng(seed)
    rsel = sorted(set([0, M - 1] + list(rng.integers(0, M, size=rows))))
    csel = sorted(set([0, N - 1] + list(rng.integers(0, N, size=cols))))
    ri = np.concatenate([np.full(N, r, dtype=np.int64) for r in rsel] +
                        [np.arange(M, dtype=np.int64) for _ in csel])
    ci = np.concatenate([np.arange(N, dtype=np.int64) for _ in rsel] +
                        [np.full(M, c, dtype=np.int64) for c in csel])
    return ri, ci


def oracle_reference(X, W, R, positions=None):
    """Yref in float64 (full, or at the given (rows, cols))."""
    orc = oracle.default()
    xb, wb = wl.bits(X), wl.bits(W)
    rb = wl.bits(R) if R is not None else None
    if positions is None:
        return orc.linear(xb, wb, rb)
    return orc.linear_at(xb, wb, rb, positions[0], positions[1])
