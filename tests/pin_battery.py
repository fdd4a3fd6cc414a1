"""Checks that pin the CPU oracle to facts other than itself.

Each ``pin_*`` function takes an ``oracle.Oracle`` and raises AssertionError
when the oracle disagrees with what the definition Y = X W^T + R (Alg. 3,
alpha = beta = 1, row-major nn.Linear reading) or IEEE round-to-nearest-even
fix independently:

* exact rational arithmetic on tiny random shapes (brute force);
* a hand-worked fixture under tests/golden/;
* numpy's float64 matmul (an independent BLAS implementation);
* closed forms: W = 0 gives R, W = I gives X + R, rank-1 integer inputs give
  a_i b_j (u.v) + R_ij;
* invariants: row permutation, a common K permutation, and the transpose
  symmetry of the plain product;
* bf16 rounding: every bf16 value is a fixed point, midpoints go to the even
  neighbour, overflow goes to infinity, and float32 inputs round as torch
  rounds them.

``ALL_PINS`` is run against the real oracle (all must pass) and against
copies of the oracle with a planted mistake (at least one must fail).
"""
from __future__ import annotations

import json
import os
from fractions import Fraction

import numpy as np
import torch

from oracle import bf16_bits_to_f64
from paper_2608_17071_amd import workloads as wl

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _rand_bits(rng, shape, scale=1.0):
    t = torch.from_numpy((rng.standard_normal(shape) * scale).astype(np.float32))
    return wl.bits(t.to(torch.bfloat16)).copy()


def pin_exact_bruteforce(orc, trials=40, seed=1234):
    """Oracle within 2^-50 (sum|x w| + |r|) of the exact rational result."""
    rng = np.random.default_rng(seed)
    for _ in range(trials):
        M, N, K = (int(v) for v in rng.integers(1, 13, size=3))
        X = _rand_bits(rng, (M, K), 1.0 / np.sqrt(K))
        W = _rand_bits(rng, (N, K), 1.0 / np.sqrt(K))
        R = _rand_bits(rng, (M, N)) if rng.random() < 0.7 else None
        Y = orc.linear(X, W, R)
        xf, wf = bf16_bits_to_f64(X), bf16_bits_to_f64(W)
        rf = bf16_bits_to_f64(R) if R is not None else None
        for i in range(M):
            for j in range(N):
                exact = Fraction(0)
                mag = Fraction(0)
                for k in range(K):
                    p = Fraction(xf[i, k]) * Fraction(wf[j, k])
                    exact += p
                    mag += abs(p)
                if rf is not None:
                    exact += Fraction(rf[i, j])
                    mag += abs(Fraction(rf[i, j]))
                err = abs(Fraction(Y[i, j]) - exact)
                assert err <= mag / 2**50, (M, N, K, i, j, float(err))


def pin_golden_hand_worked(orc):
    with open(os.path.join(GOLDEN, "hand_worked_2x3x2.json")) as f:
        g = json.load(f)
    X = wl.bits(torch.tensor(g["X"], dtype=torch.float32).to(torch.bfloat16))
    W = wl.bits(torch.tensor(g["W"], dtype=torch.float32).to(torch.bfloat16))
    R = wl.bits(torch.tensor(g["R"], dtype=torch.float32).to(torch.bfloat16))
    assert (g["M"], g["K"]) == X.shape and (g["N"], g["K"]) == W.shape
    np.testing.assert_array_equal(orc.linear(X, W, R), np.array(g["Y_residual"]))
    np.testing.assert_array_equal(orc.linear(X, W, None), np.array(g["Y_plain"]))


def pin_numpy_matmul(orc, seed=7):
    """numpy float64 matmul of the same bf16 values agrees to ~1e-12."""
    rng = np.random.default_rng(seed)
    for (M, N, K) in [(33, 47, 64), (5, 128, 96), (64, 17, 256), (1, 40, 1000)]:
        X = _rand_bits(rng, (M, K), 1.0 / np.sqrt(K))
        W = _rand_bits(rng, (N, K), 1.0 / np.sqrt(K))
        R = _rand_bits(rng, (M, N))
        ref = bf16_bits_to_f64(X) @ bf16_bits_to_f64(W).T
        mag = np.abs(bf16_bits_to_f64(X)) @ np.abs(bf16_bits_to_f64(W)).T
        np.testing.assert_array_less(np.abs(orc.linear(X, W, None) - ref), 1e-13 * mag + 1e-300)
        ref_r = ref + bf16_bits_to_f64(R)
        mag_r = mag + np.abs(bf16_bits_to_f64(R))
        np.testing.assert_array_less(np.abs(orc.linear(X, W, R) - ref_r), 1e-13 * mag_r + 1e-300)


def pin_zero_weight(orc, seed=3):
    rng = np.random.default_rng(seed)
    M, N, K = 9, 31, 40
    X = _rand_bits(rng, (M, K))
    W = wl.bits(wl.zero_weight(N, K)).copy()
    R = _rand_bits(rng, (M, N))
    np.testing.assert_array_equal(orc.linear(X, W, R), bf16_bits_to_f64(R))
    assert not np.any(orc.linear(X, W, None))


def pin_identity_weight(orc, seed=4):
    rng = np.random.default_rng(seed)
    M, K = 13, 24
    X = _rand_bits(rng, (M, K))
    W = wl.bits(wl.identity_weight(K)).copy()
    R = _rand_bits(rng, (M, K))
    np.testing.assert_array_equal(orc.linear(X, W, None), bf16_bits_to_f64(X))
    np.testing.assert_array_equal(orc.linear(X, W, R),
                                  bf16_bits_to_f64(X) + bf16_bits_to_f64(R))


def pin_rank1_integer(orc):
    for (M, N, K, seed) in [(7, 11, 50, 0), (16, 3, 129, 1), (2, 64, 8, 2)]:
        X, W, R, a, b, u, v = wl.rank1_integer(M, N, K, seed)
        s = int(np.dot(u, v))
        expect = np.outer(a, b) * s
        np.testing.assert_array_equal(orc.linear(wl.bits(X), wl.bits(W), None), expect)
        np.testing.assert_array_equal(orc.linear(wl.bits(X), wl.bits(W), wl.bits(R)),
                                      expect + bf16_bits_to_f64(wl.bits(R)))


def pin_invariants(orc, seed=5):
    rng = np.random.default_rng(seed)
    M, N, K = 12, 20, 36
    X = _rand_bits(rng, (M, K))
    W = _rand_bits(rng, (N, K))
    R = _rand_bits(rng, (M, N))
    Y = orc.linear(X, W, R)
    # a row permutation of X and R permutes the rows of Y (bitwise: same k-order)
    p = rng.permutation(M)
    np.testing.assert_array_equal(orc.linear(X[p], W, R[p]), Y[p])
    # a row permutation of W and the columns of R permutes the columns of Y
    q = rng.permutation(N)
    np.testing.assert_array_equal(orc.linear(X, W[q], np.ascontiguousarray(R[:, q])), Y[:, q])
    # one permutation of K applied to X and W leaves Y unchanged (up to order)
    kp = rng.permutation(K)
    Yk = orc.linear(np.ascontiguousarray(X[:, kp]), np.ascontiguousarray(W[:, kp]), R)
    np.testing.assert_allclose(Yk, Y, rtol=0, atol=1e-12)
    # plain product: gemm(W, X) = gemm(X, W)^T
    np.testing.assert_allclose(orc.linear(W, X, None), orc.linear(X, W, None).T, rtol=0, atol=1e-12)


def pin_linear_at_matches_full(orc, seed=6):
    rng = np.random.default_rng(seed)
    M, N, K = 21, 34, 55
    X = _rand_bits(rng, (M, K))
    W = _rand_bits(rng, (N, K))
    R = _rand_bits(rng, (M, N))
    rows = rng.integers(0, M, size=50)
    cols = rng.integers(0, N, size=50)
    # the sampled entry point must evaluate the same exact expression; the
    # full entry point is pinned above, so this pins the sampled one too
    full = bf16_bits_to_f64(X) @ bf16_bits_to_f64(W).T + bf16_bits_to_f64(R)
    np.testing.assert_allclose(orc.linear_at(X, W, R, rows, cols), full[rows, cols],
                               rtol=0, atol=1e-12)


def _all_finite_bf16():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    vals = bf16_bits_to_f64(bits)
    keep = np.isfinite(vals)
    return bits[keep], vals[keep]


def pin_round_fixed_points(orc):
    bits, vals = _all_finite_bf16()
    np.testing.assert_array_equal(orc.round_bf16(vals), bits)


def pin_round_midpoints(orc):
    """Halfway between neighbours goes to the even pattern; off-centre goes nearest."""
    pos = np.arange(0x0000, 0x7F80, dtype=np.uint16)      # +0 .. largest finite
    lo, hi = pos[:-1], pos[1:]
    a, b = bf16_bits_to_f64(lo), bf16_bits_to_f64(hi)
    mid = (a + b) / 2                                       # exact in float64
    even = np.where(lo % 2 == 0, lo, hi)
    np.testing.assert_array_equal(orc.round_bf16(mid), even)
    np.testing.assert_array_equal(orc.round_bf16(-mid), even | 0x8000)
    gap = b - a
    np.testing.assert_array_equal(orc.round_bf16(mid - gap / 8), lo)
    np.testing.assert_array_equal(orc.round_bf16(mid + gap / 8), hi)


def pin_round_specials(orc):
    big = float(bf16_bits_to_f64(np.array([0x7F7F], dtype=np.uint16))[0])
    ulp = 2.0 ** (127 - 7)
    out = orc.round_bf16(np.array([big + ulp / 2, big + ulp / 2 * 0.999, -(big + ulp),
                                   np.inf, -np.inf, np.nan, 0.0, -0.0]))
    assert list(out[:5]) == [0x7F80, 0x7F7F, 0xFF80, 0x7F80, 0xFF80]
    assert (out[5] & 0x7F80) == 0x7F80 and (out[5] & 0x7F) != 0
    assert list(out[6:]) == [0x0000, 0x8000]


def pin_round_like_torch(orc, seed=8):
    """float32 inputs: torch's float32 -> bfloat16 conversion is nearest-even."""
    rng = np.random.default_rng(seed)
    f = np.concatenate([rng.standard_normal(20000) * 10.0 ** rng.uniform(-30, 30, 20000),
                        rng.standard_normal(1000) * 1e-39]).astype(np.float32)
    t = wl.bits(torch.from_numpy(f).to(torch.bfloat16))
    np.testing.assert_array_equal(orc.round_bf16(f.astype(np.float64)), t)


ALL_PINS = [
    pin_exact_bruteforce,
    pin_golden_hand_worked,
    pin_numpy_matmul,
    pin_zero_weight,
    pin_identity_weight,
    pin_rank1_integer,
    pin_invariants,
    pin_linear_at_matches_full,
    pin_round_fixed_points,
    pin_round_midpoints,
    pin_round_specials,
    pin_round_like_torch,
]
