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

The general form D = alpha X W^T + beta C + bias (leading dimensions, bias
row; ``EX_PINS``) is pinned by exact rational arithmetic with strided
operands over NaN padding, by reduction to the plain operator at
alpha = beta = 1, by the W = 0 closed form, by beta = 0 leaving C unread,
by exact scaling with power-of-two alpha, and by strided = dense.

The gated MLP input projection H = silu(X Wg^T) * (X Wu^T) (SwiGLU,
``GLU_PINS``) is pinned by exact rational k-sums with SiLU evaluated by
Python's decimal module at 60 digits (correctly rounded exp, not libm), by
closed forms at e (silu(1) = e/(1+e), silu(-1) = -1/(1+e), silu(2), silu(-2),
silu(1/2)), by numpy's matmul with scipy's logistic function, by the odd
part silu(z) - silu(-z) = z and the even part silu(z) + silu(-z) =
z tanh(z/2), by the saturated tails (z >= 40: silu(z) = z in double;
z <= -800: 0), by zero operands, and by row and column permutations.

The INT8 forms (``I8_PINS``: Y = sx[i] sw[j] sum_k qX qW (+ R) and
H = silu(sx swg Ag) (sx swu Au)) are pinned by exact Python-integer sums
(including the -128 x -128 extremes), exact rational dequantisation with
random binary32 scales, reduction to the bf16 oracles (already pinned) when
power-of-two scales make every dequantised operand an exact bf16 value, a
zero weight, and the 60-digit decimal SiLU.

The FP8 forms (``F8_PINS``: E4M3 operands with the same scales) are pinned
by the decoding of all 256 bit patterns against torch's float8_e4m3fn, the
format's landmarks (1, 448, the smallest normal and subnormal, NaN), exact
rational dequantisation with random scales, and bit-identity with the bf16
oracles when power-of-two scales make every dequantised operand an exact bf16
value.

The grouped forms over an expert-major padded layout (``GRP_PINS``: per
expert e, Y[e,i] = X[e,i] W[e]^T for the rows i below counts[e] clamped to
[0, M_pad]) are pinned by exact rational brute force with empty, partial,
full, negative and oversized counts, by reduction expert by expert to the
(pinned) plain and SwiGLU oracles, by gap rows left exactly as they were,
and by expert permutations.

``ALL_PINS`` is run against the real oracle (all must pass) and against
copies of the oracle with a planted mistake (at least one must fail).
"""
from __future__ import annotations

import json
import math
import os
from decimal import Decimal, localcontext
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


# ---- general form D = alpha X W^T + beta C + bias (strided operands) ----

_ALPHAS = (1.0, -2.0, 0.5, 0.0, 3.0517578125e-05, 1.7310791015625, -0.3333333432674408)


def _padded(rng, arr, extra):
    """arr as the leading columns of a wider buffer whose padding is NaN."""
    rows, cols = arr.shape
    buf = np.full((rows, cols + extra), 0x7FC0, np.uint16)
    buf[:, :cols] = arr
    return buf[:, :cols]


def pin_ex_exact_bruteforce(orc, trials=40, seed=4321):
    """General form within 2^-49 (|alpha| sum|x w| + |beta c| + |b|) of the
    exact rational result, with strided operands over NaN padding."""
    rng = np.random.default_rng(seed)
    for t in range(trials):
        M, N, K = (int(v) for v in rng.integers(1, 13, size=3))
        X = _padded(rng, _rand_bits(rng, (M, K), 1.0 / np.sqrt(K)), int(rng.integers(0, 5)))
        W = _padded(rng, _rand_bits(rng, (N, K), 1.0 / np.sqrt(K)), int(rng.integers(0, 5)))
        C = _padded(rng, _rand_bits(rng, (M, N)), int(rng.integers(0, 5))) if rng.random() < 0.7 else None
        b = _rand_bits(rng, (N,)) if rng.random() < 0.6 else None
        alpha = float(np.float32(_ALPHAS[t % len(_ALPHAS)]))
        beta = float(np.float32(_ALPHAS[(3 * t + 1) % len(_ALPHAS)]))
        D = orc.linear_ex(X, W, C, b, alpha, beta)
        assert np.isfinite(D).all(), (M, N, K, "non-finite output from finite operands")
        xf, wf = bf16_bits_to_f64(X), bf16_bits_to_f64(W)
        cf = bf16_bits_to_f64(C) if C is not None else None
        bf = bf16_bits_to_f64(b) if b is not None else None
        for i in range(M):
            for j in range(N):
                s = Fraction(0)
                mag = Fraction(0)
                for k in range(K):
                    p = Fraction(xf[i, k]) * Fraction(wf[j, k])
                    s += p
                    mag += abs(p)
                exact = Fraction(alpha) * s
                mag = abs(Fraction(alpha)) * mag
                if cf is not None and beta != 0.0:
                    exact += Fraction(beta) * Fraction(cf[i, j])
                    mag += abs(Fraction(beta) * Fraction(cf[i, j]))
                if bf is not None:
                    exact += Fraction(bf[j])
                    mag += abs(Fraction(bf[j]))
                err = abs(Fraction(D[i, j]) - exact)
                assert err <= mag / 2**49, (M, N, K, alpha, beta, i, j, float(err))


def pin_ex_reduces_to_base(orc, seed=11):
    """alpha = beta = 1 without bias is the plain operator, bit for bit."""
    rng = np.random.default_rng(seed)
    for M, N, K in ((5, 7, 9), (16, 3, 40), (1, 33, 17)):
        X = _rand_bits(rng, (M, K))
        W = _rand_bits(rng, (N, K))
        R = _rand_bits(rng, (M, N))
        np.testing.assert_array_equal(orc.linear_ex(X, W, R, None, 1.0, 1.0), orc.linear(X, W, R))
        np.testing.assert_array_equal(orc.linear_ex(X, W, None, None, 1.0, 1.0), orc.linear(X, W))


def pin_ex_zero_weight(orc, seed=12):
    """W = 0: D = beta C + bias (the product term vanishes for finite X)."""
    rng = np.random.default_rng(seed)
    M, N, K = 9, 11, 13
    X = _rand_bits(rng, (M, K))
    W = np.zeros((N, K), np.uint16)
    C = _rand_bits(rng, (M, N))
    b = _rand_bits(rng, (N,))
    D = orc.linear_ex(X, W, C, b, -2.0, 0.5)
    cf, bf = bf16_bits_to_f64(C), bf16_bits_to_f64(b)
    for i in range(M):
        for j in range(N):
            exact = Fraction(0.5) * Fraction(cf[i, j]) + Fraction(bf[j])
            assert abs(Fraction(D[i, j]) - exact) <= abs(exact) / 2**52, (i, j)


def pin_ex_beta_zero_skips_c(orc, seed=13):
    """beta = 0: C is not read (NaN in C does not reach D)."""
    rng = np.random.default_rng(seed)
    M, N, K = 6, 5, 8
    X = _rand_bits(rng, (M, K))
    W = _rand_bits(rng, (N, K))
    b = _rand_bits(rng, (N,))
    C = np.full((M, N), 0x7FC0, np.uint16)
    D = orc.linear_ex(X, W, C, b, 1.0, 0.0)
    assert np.isfinite(D).all()
    np.testing.assert_array_equal(D, orc.linear_ex(X, W, None, b, 1.0, 1.0))


def pin_ex_alpha_power_of_two(orc, seed=14):
    """A power-of-two alpha scales the product exactly."""
    rng = np.random.default_rng(seed)
    X = _rand_bits(rng, (7, 19))
    W = _rand_bits(rng, (9, 19))
    base = orc.linear(X, W)
    for a in (4.0, 0.125, -1.0):
        np.testing.assert_array_equal(orc.linear_ex(X, W, None, None, a, 0.0), a * base)


def pin_ex_strided_equals_dense(orc, seed=15):
    """Row-strided views (NaN padding) give the dense result, bit for bit."""
    rng = np.random.default_rng(seed)
    M, N, K = 10, 12, 21
    X = _rand_bits(rng, (M, K))
    W = _rand_bits(rng, (N, K))
    C = _rand_bits(rng, (M, N))
    b = _rand_bits(rng, (N,))
    dense = orc.linear_ex(X, W, C, b, 0.75, -1.5)
    strided = orc.linear_ex(_padded(rng, X, 5), _padded(rng, W, 3), _padded(rng, C, 7), b, 0.75, -1.5)
    np.testing.assert_array_equal(strided, dense)


def pin_ex_at_matches_full(orc, seed=16):
    rng = np.random.default_rng(seed)
    M, N, K = 8, 9, 10
    X = _padded(rng, _rand_bits(rng, (M, K)), 2)
    W = _rand_bits(rng, (N, K))
    C = _rand_bits(rng, (M, N))
    b = _rand_bits(rng, (N,))
    full = orc.linear_ex(X, W, C, b, 1.25, 2.0)
    rows = rng.integers(0, M, 40)
    cols = rng.integers(0, N, 40)
    np.testing.assert_array_equal(orc.linear_ex_at(X, W, C, b, 1.25, 2.0, rows, cols), full[rows, cols])


EX_PINS = [
    pin_ex_exact_bruteforce,
    pin_ex_reduces_to_base,
    pin_ex_zero_weight,
    pin_ex_beta_zero_skips_c,
    pin_ex_alpha_power_of_two,
    pin_ex_strided_equals_dense,
    pin_ex_at_matches_full,
]

# ----------------------------------------------------------------- SwiGLU ----
def _neg_bits(bits):
    """Exact negation of bf16 bit patterns (sign bit flipped)."""
    return (np.asarray(bits, dtype=np.uint16) ^ np.uint16(0x8000)).astype(np.uint16)


def _glu_f64(X, Wg, Wu):
    """G = X Wg^T and U = X Wu^T by numpy's float64 matmul, and the
    magnitudes |X| |Wg|^T and |X| |Wu|^T that bound their rounding."""
    xf, gf, uf = bf16_bits_to_f64(X), bf16_bits_to_f64(Wg), bf16_bits_to_f64(Wu)
    return xf @ gf.T, xf @ uf.T, np.abs(xf) @ np.abs(gf).T, np.abs(xf) @ np.abs(uf).T


def _glu_bound(G, U, magG, magU, ref, rel):
    """Error allowed for H near silu(G) U when G and U carry k-sum rounding
    up to rel * their magnitudes (|silu'| <= 1.1), plus the final rounding."""
    s = np.abs(G) / (1.0 + np.exp(-np.clip(G, -700, 700)))
    return rel * (1.1 * magG * np.abs(U) + s * magU) + 1e-15 * np.abs(ref) + 1e-300


def pin_glu_exact_bruteforce(orc, trials=30, seed=2468):
    """Oracle within 2^-46 of silu(G) U computed from the exact rational G and
    U with a 60-digit decimal exponential (over the tails too: |G| up to ~100)."""
    rng = np.random.default_rng(seed)
    for t in range(trials):
        M, N, K = (int(v) for v in rng.integers(1, 9, size=3))
        spread = (1.0, 4.0, 30.0)[t % 3]
        X = _rand_bits(rng, (M, K), spread)
        Wg = _rand_bits(rng, (N, K), 1.0 / np.sqrt(K))
        Wu = _rand_bits(rng, (N, K), 1.0 / np.sqrt(K))
        H = orc.swiglu(X, Wg, Wu)
        assert np.isfinite(H).all()
        xf, gf, uf = bf16_bits_to_f64(X), bf16_bits_to_f64(Wg), bf16_bits_to_f64(Wu)
        with localcontext() as ctx:
            ctx.prec = 60
            for i in range(M):
                for j in range(N):
                    g = sum((Fraction(xf[i, k]) * Fraction(gf[j, k]) for k in range(K)), Fraction(0))
                    u = sum((Fraction(xf[i, k]) * Fraction(uf[j, k]) for k in range(K)), Fraction(0))
                    mg = sum(abs(Fraction(xf[i, k]) * Fraction(gf[j, k])) for k in range(K))
                    mu = sum(abs(Fraction(xf[i, k]) * Fraction(uf[j, k])) for k in range(K))
                    gd = Decimal(g.numerator) / Decimal(g.denominator)
                    ud = Decimal(u.numerator) / Decimal(u.denominator)
                    sd = gd / (1 + (-gd).exp())
                    ref = sd * ud
                    bound = (Decimal(1.1) * Decimal(float(mg)) * abs(ud) + abs(sd) * Decimal(float(mu))) \
                        * Decimal(2) ** -46 + abs(ref) * Decimal(2) ** -50
                    err = abs(Decimal(float(H[i, j])) - ref)
                    assert err <= bound, (M, N, K, i, j, float(err), float(bound))


def pin_glu_closed_forms(orc):
    """K = 1 cases whose SiLU has a closed form in e."""
    e = math.e
    # X is one column of scalars, the weights are scalars: G = x*wg, U = x*wu.
    xs = [1.0, -1.0, 2.0, 0.5]
    wg = [1.0, 2.0, -1.0]
    wu = [1.0, -0.5, 3.0]
    X = wl.bits(torch.tensor(xs, dtype=torch.float32).reshape(4, 1).to(torch.bfloat16))
    Wg = wl.bits(torch.tensor(wg, dtype=torch.float32).reshape(3, 1).to(torch.bfloat16))
    Wu = wl.bits(torch.tensor(wu, dtype=torch.float32).reshape(3, 1).to(torch.bfloat16))
    silu_closed = {1.0: e / (1 + e), -1.0: -1 / (1 + e), 2.0: 2 * e * e / (1 + e * e),
                   -2.0: -2 / (1 + e * e), 0.5: 0.5 * math.sqrt(e) / (1 + math.sqrt(e)),
                   -0.5: -0.5 / (1 + math.sqrt(e)), 4.0: 4 * e ** 4 / (1 + e ** 4), -4.0: -4 / (1 + e ** 4)}
    H = orc.swiglu(X, Wg, Wu)
    for i, x in enumerate(xs):
        for j in range(3):
            ref = silu_closed[x * wg[j]] * (x * wu[j])
            assert abs(H[i, j] - ref) <= 4e-16 * abs(ref), (i, j, H[i, j], ref)


def pin_glu_scipy_expit(orc, seed=21):
    """numpy's float64 matmul with scipy's logistic function."""
    from scipy.special import expit
    rng = np.random.default_rng(seed)
    M, N, K = 23, 31, 257
    X = _rand_bits(rng, (M, K), 3.0)
    Wg = _rand_bits(rng, (N, K), 1.0 / np.sqrt(K))
    Wu = _rand_bits(rng, (N, K), 1.0 / np.sqrt(K))
    G, U, mg, mu = _glu_f64(X, Wg, Wu)
    ref = G * expit(G) * U
    H = orc.swiglu(X, Wg, Wu)
    assert (np.abs(H - ref) <= _glu_bound(G, U, mg, mu, ref, 1e-13)).all()


def pin_glu_odd_even_parts(orc, seed=22):
    """silu(z) - silu(-z) = z and silu(z) + silu(-z) = z tanh(z/2): with the
    gate weights negated, H - H' = G U and H + H' = G U tanh(G/2)."""
    rng = np.random.default_rng(seed)
    M, N, K = 17, 13, 64
    X = _rand_bits(rng, (M, K), 2.0)
    Wg = _rand_bits(rng, (N, K), 1.0 / np.sqrt(K))
    Wu = _rand_bits(rng, (N, K), 1.0 / np.sqrt(K))
    G, U, mg, mu = _glu_f64(X, Wg, Wu)
    H = orc.swiglu(X, Wg, Wu)
    Hn = orc.swiglu(X, _neg_bits(Wg), Wu)
    odd = G * U
    even = G * U * np.tanh(G / 2)
    assert (np.abs((H - Hn) - odd) <= _glu_bound(G, U, mg, mu, odd, 1e-13) * 4).all()
    assert (np.abs((H + Hn) - even) <= _glu_bound(G, U, mg, mu, even, 1e-13) * 4).all()


def pin_glu_tails(orc):
    """Integer operands: gate sums >= 40 give H = G U exactly (the sigmoid is 1
    in double), gate sums <= -800 give H = 0 (the exponential overflows)."""
    X = wl.bits(torch.tensor([[8.0, 8.0], [-16.0, 4.0]]).to(torch.bfloat16))
    Wg = wl.bits(torch.tensor([[4.0, 2.0], [-64.0, -64.0], [-4.0, 8.0]]).to(torch.bfloat16))
    Wu = wl.bits(torch.tensor([[3.0, -1.0], [1.0, 1.0], [0.5, 2.0]]).to(torch.bfloat16))
    H = orc.swiglu(X, Wg, Wu)
    xf, gf, uf = bf16_bits_to_f64(X), bf16_bits_to_f64(Wg), bf16_bits_to_f64(Wu)
    G, U = xf @ gf.T, xf @ uf.T
    for i in range(2):
        for j in range(3):
            if G[i, j] >= 40:
                assert H[i, j] == G[i, j] * U[i, j], (i, j)
            elif G[i, j] <= -800:
                assert H[i, j] == 0.0, (i, j)
    assert (G >= 40).sum() >= 2 and (G <= -800).sum() >= 1


def pin_glu_zero_operands(orc, seed=23):
    """A zero gate, a zero up projection, zero activations or K = 0 give H = 0."""
    rng = np.random.default_rng(seed)
    M, N, K = 6, 7, 33
    X = _rand_bits(rng, (M, K))
    Wg = _rand_bits(rng, (N, K))
    Wu = _rand_bits(rng, (N, K))
    z = np.zeros
    for args in ((X, z((N, K), np.uint16), Wu), (X, Wg, z((N, K), np.uint16)), (z((M, K), np.uint16), Wg, Wu)):
        assert (orc.swiglu(*args) == 0).all()
    e = np.zeros((M, 0), np.uint16)
    assert (orc.swiglu(e, np.zeros((N, 0), np.uint16), np.zeros((N, 0), np.uint16)) == 0).all()


def pin_glu_permutations(orc, seed=24):
    """Permuting X's rows permutes H's rows; permuting Wg's and Wu's rows
    together permutes H's columns (bit for bit: each element is computed on
    its own); a gate/up swap changes the result."""
    rng = np.random.default_rng(seed)
    M, N, K = 9, 11, 40
    X = _rand_bits(rng, (M, K), 2.0)
    Wg = _rand_bits(rng, (N, K), 1.0 / np.sqrt(K))
    Wu = _rand_bits(rng, (N, K), 1.0 / np.sqrt(K))
    H = orc.swiglu(X, Wg, Wu)
    pr, pc = rng.permutation(M), rng.permutation(N)
    np.testing.assert_array_equal(orc.swiglu(X[pr], Wg, Wu), H[pr])
    np.testing.assert_array_equal(orc.swiglu(X, Wg[pc], Wu[pc]), H[:, pc])
    assert not np.allclose(orc.swiglu(X, Wu, Wg), H)


def pin_glu_at_matches_full(orc, seed=25):
    rng = np.random.default_rng(seed)
    M, N, K = 8, 9, 10
    X = _rand_bits(rng, (M, K), 2.0)
    Wg = _rand_bits(rng, (N, K))
    Wu = _rand_bits(rng, (N, K))
    full = orc.swiglu(X, Wg, Wu)
    rows = rng.integers(0, M, 40)
    cols = rng.integers(0, N, 40)
    np.testing.assert_array_equal(orc.swiglu_at(X, Wg, Wu, rows, cols), full[rows, cols])


GLU_PINS = [
    pin_glu_exact_bruteforce,
    pin_glu_closed_forms,
    pin_glu_scipy_expit,
    pin_glu_odd_even_parts,
    pin_glu_tails,
    pin_glu_zero_operands,
    pin_glu_permutations,
    pin_glu_at_matches_full,
]

# ------------------------------------------------------------------- INT8 ----
def _rand_i8(rng, shape, sigma=40.0):
    """int8 values from a rounded normal, clipped to [-128, 127]."""
    return np.clip(np.rint(rng.standard_normal(shape) * sigma), -128, 127).astype(np.int8)


def _rand_scales(rng, n, lo=-12, hi=-4):
    """Positive binary32 scales with random mantissas over a range of binades."""
    return (2.0 ** rng.uniform(lo, hi, size=n)).astype(np.float32)


def _pow2_scales(rng, n, lo=-10, hi=-3):
    return (2.0 ** rng.integers(lo, hi, size=n)).astype(np.float32)


def _bf16_from_f64(values):
    """bf16 bit patterns of float64 values that are exactly representable."""
    t = torch.from_numpy(np.asarray(values, dtype=np.float64))
    out = wl.bits(t.to(torch.float32).to(torch.bfloat16)).copy()
    assert (bf16_bits_to_f64(out) == np.asarray(values)).all(), "value is not an exact bf16"
    return out


def pin_i8_exact_integer_sums(orc, trials=20, seed=31):
    """The integer sums equal Python's exact integer arithmetic, extremes included."""
    rng = np.random.default_rng(seed)
    for t in range(trials):
        M, N, K = (int(v) for v in rng.integers(1, 11, size=3))
        qX = _rand_i8(rng, (M, K), 90.0)
        qW = _rand_i8(rng, (N, K), 90.0)
        A = orc.i8_dot(qX, qW)
        for i in range(M):
            for j in range(N):
                assert A[i, j] == sum(int(qX[i, k]) * int(qW[j, k]) for k in range(K))
    K = 4099
    lo = np.full((2, K), -128, np.int8)
    assert (orc.i8_dot(lo, lo) == K * 16384).all()
    hi = np.full((1, K), 127, np.int8)
    assert (orc.i8_dot(hi, lo[:1]) == -K * 127 * 128).all()


def pin_i8_dequant_exact(orc, trials=20, seed=32):
    """Random binary32 scales: Y within 2^-52 |Y| of the exact rational
    sx sw A (+ R)."""
    rng = np.random.default_rng(seed)
    for _ in range(trials):
        M, N, K = (int(v) for v in rng.integers(1, 9, size=3))
        qX, qW = _rand_i8(rng, (M, K)), _rand_i8(rng, (N, K))
        sx, sw = _rand_scales(rng, M), _rand_scales(rng, N)
        R = _rand_bits(rng, (M, N)) if rng.random() < 0.5 else None
        Y = orc.i8_linear(qX, sx, qW, sw, R)
        rf = bf16_bits_to_f64(R) if R is not None else None
        for i in range(M):
            for j in range(N):
                a = sum(int(qX[i, k]) * int(qW[j, k]) for k in range(K))
                exact = Fraction(float(sx[i])) * Fraction(float(sw[j])) * a
                mag = abs(exact)
                if rf is not None:
                    exact += Fraction(rf[i, j])
                    mag += abs(Fraction(rf[i, j]))
                assert abs(Fraction(Y[i, j]) - exact) <= mag / 2**51 + Fraction(1, 2**1074), (i, j)


def pin_i8_matches_bf16_oracle(orc, seed=33):
    """Power-of-two scales: sx*qX and sw*qW are exact bf16 values, and the INT8
    oracle equals the (pinned) bf16 oracle on those operands, bit for bit."""
    rng = np.random.default_rng(seed)
    M, N, K = 13, 17, 96
    qX, qW = _rand_i8(rng, (M, K), 60.0), _rand_i8(rng, (N, K), 60.0)
    sx, sw = _pow2_scales(rng, M), _pow2_scales(rng, N)
    R = _rand_bits(rng, (M, N))
    Xb = _bf16_from_f64(qX.astype(np.float64) * sx[:, None])
    Wb = _bf16_from_f64(qW.astype(np.float64) * sw[:, None])
    np.testing.assert_array_equal(orc.i8_linear(qX, sx, qW, sw, R), orc.linear(Xb, Wb, R))
    np.testing.assert_array_equal(orc.i8_linear(qX, sx, qW, sw), orc.linear(Xb, Wb))
    qWu = _rand_i8(rng, (N, K), 60.0)
    swu = _pow2_scales(rng, N)
    Wub = _bf16_from_f64(qWu.astype(np.float64) * swu[:, None])
    np.testing.assert_array_equal(orc.i8_swiglu(qX, sx, qW, sw, qWu, swu), orc.swiglu(Xb, Wb, Wub))


def pin_i8_zero_weight(orc, seed=34):
    rng = np.random.default_rng(seed)
    M, N, K = 5, 6, 40
    qX = _rand_i8(rng, (M, K))
    sx, sw = _rand_scales(rng, M), _rand_scales(rng, N)
    R = _rand_bits(rng, (M, N))
    z = np.zeros((N, K), np.int8)
    np.testing.assert_array_equal(orc.i8_linear(qX, sx, z, sw, R), bf16_bits_to_f64(R))
    assert (orc.i8_swiglu(qX, sx, z, sw, _rand_i8(rng, (N, K)), sw) == 0).all()
    assert (orc.i8_swiglu(qX, sx, _rand_i8(rng, (N, K)), sw, z, sw) == 0).all()


def pin_i8_swiglu_decimal(orc, trials=12, seed=35):
    """INT8 SwiGLU within 2^-46 of silu(g) u from exact rational g and u and a
    60-digit decimal exponential (gate sums up to about +-50)."""
    rng = np.random.default_rng(seed)
    for _ in range(trials):
        M, N, K = (int(v) for v in rng.integers(1, 7, size=3))
        qX, qWg, qWu = _rand_i8(rng, (M, K)), _rand_i8(rng, (N, K)), _rand_i8(rng, (N, K))
        sx = _rand_scales(rng, M, -6, -3)
        swg, swu = _rand_scales(rng, N, -8, -4), _rand_scales(rng, N, -8, -4)
        H = orc.i8_swiglu(qX, sx, qWg, swg, qWu, swu)
        with localcontext() as ctx:
            ctx.prec = 60
            for i in range(M):
                for j in range(N):
                    ag = sum(int(qX[i, k]) * int(qWg[j, k]) for k in range(K))
                    au = sum(int(qX[i, k]) * int(qWu[j, k]) for k in range(K))
                    g = Fraction(float(sx[i])) * Fraction(float(swg[j])) * ag
                    u = Fraction(float(sx[i])) * Fraction(float(swu[j])) * au
                    gd = Decimal(g.numerator) / Decimal(g.denominator)
                    ud = Decimal(u.numerator) / Decimal(u.denominator)
                    sd = gd / (1 + (-gd).exp())
                    ref = sd * ud
                    bound = (abs(sd * ud) + Decimal(1.1) * abs(gd * ud)) * Decimal(2) ** -46 + Decimal(2) ** -1000
                    assert abs(Decimal(float(H[i, j])) - ref) <= bound, (i, j)


def pin_i8_at_matches_full(orc, seed=36):
    rng = np.random.default_rng(seed)
    M, N, K = 7, 9, 24
    qX, qW, qWu = _rand_i8(rng, (M, K)), _rand_i8(rng, (N, K)), _rand_i8(rng, (N, K))
    sx, sw, swu = _rand_scales(rng, M), _rand_scales(rng, N), _rand_scales(rng, N)
    R = _rand_bits(rng, (M, N))
    rows, cols = rng.integers(0, M, 40), rng.integers(0, N, 40)
    np.testing.assert_array_equal(orc.i8_linear_at(qX, sx, qW, sw, R, rows, cols),
                                  orc.i8_linear(qX, sx, qW, sw, R)[rows, cols])
    np.testing.assert_array_equal(orc.i8_swiglu_at(qX, sx, qW, sw, qWu, swu, rows, cols),
                                  orc.i8_swiglu(qX, sx, qW, sw, qWu, swu)[rows, cols])


I8_PINS = [
    pin_i8_exact_integer_sums,
    pin_i8_dequant_exact,
    pin_i8_matches_bf16_oracle,
    pin_i8_zero_weight,
    pin_i8_swiglu_decimal,
    pin_i8_at_matches_full,
]

# -------------------------------------------------------------------- FP8 ----
def _rand_f8(rng, shape, sigma=8.0):
    """E4M3 bit patterns of N(0,1)*sigma draws (torch rounds to the format)."""
    t = torch.from_numpy((rng.standard_normal(shape) * sigma).astype(np.float32))
    return t.to(torch.float8_e4m3fn).view(torch.uint8).numpy().copy()


def pin_f8_decode(orc):
    """All 256 E4M3 patterns decode as torch's float8_e4m3fn does; landmarks."""
    bits = np.arange(256, dtype=np.uint8)
    ours = orc.fp8_decode(bits)
    ref = torch.from_numpy(bits.copy()).view(torch.float8_e4m3fn).to(torch.float32).numpy().astype(np.float64)
    assert (np.isnan(ours) == np.isnan(ref)).all()
    ok = ~np.isnan(ref)
    np.testing.assert_array_equal(ours[ok], ref[ok])
    assert np.array_equal(np.signbit(ours[ok]), np.signbit(ref[ok]))
    land = {0x38: 1.0, 0x7E: 448.0, 0xFE: -448.0, 0x08: 2.0 ** -6, 0x01: 2.0 ** -9, 0x07: 7 * 2.0 ** -9,
            0x40: 2.0, 0x3C: 1.5}
    for b, v in land.items():
        assert ours[b] == v, (hex(b), ours[b], v)
    assert np.isnan(ours[0x7F]) and np.isnan(ours[0xFF]) and np.isfinite(ours[0x78])


def pin_f8_dequant_exact(orc, trials=15, seed=71):
    rng = np.random.default_rng(seed)
    for _ in range(trials):
        M, N, K = (int(v) for v in rng.integers(1, 8, size=3))
        qX, qW = _rand_f8(rng, (M, K)), _rand_f8(rng, (N, K))
        sx, sw = _rand_scales(rng, M), _rand_scales(rng, N)
        R = _rand_bits(rng, (M, N)) if rng.random() < 0.5 else None
        Y = orc.f8_linear(qX, sx, qW, sw, R)
        xd, wd = orc.fp8_decode(qX), orc.fp8_decode(qW)
        rf = bf16_bits_to_f64(R) if R is not None else None
        for i in range(M):
            for j in range(N):
                s_ = sum((Fraction(xd[i, k]) * Fraction(wd[j, k]) for k in range(K)), Fraction(0))
                mag = sum(abs(Fraction(xd[i, k]) * Fraction(wd[j, k])) for k in range(K))
                sc = Fraction(float(sx[i])) * Fraction(float(sw[j]))
                exact = sc * s_
                bound = sc * mag / 2**50
                if rf is not None:
                    exact += Fraction(rf[i, j])
                    bound += abs(Fraction(rf[i, j])) / 2**52
                assert abs(Fraction(Y[i, j]) - exact) <= bound + Fraction(1, 2**1074), (i, j)


def pin_f8_matches_bf16_oracle(orc, seed=72):
    """Power-of-two scales: the dequantised FP8 operands are exact bf16 values
    and the FP8 oracle equals the (pinned) bf16 oracles bit for bit."""
    rng = np.random.default_rng(seed)
    M, N, K = 11, 13, 80
    qX, qW, qWu = _rand_f8(rng, (M, K)), _rand_f8(rng, (N, K)), _rand_f8(rng, (N, K))
    sx, sw, swu = _pow2_scales(rng, M, -4, 3), _pow2_scales(rng, N, -9, -4), _pow2_scales(rng, N, -9, -4)
    R = _rand_bits(rng, (M, N))
    Xb = _bf16_from_f64(orc.fp8_decode(qX) * sx[:, None].astype(np.float64))
    Wb = _bf16_from_f64(orc.fp8_decode(qW) * sw[:, None].astype(np.float64))
    Wub = _bf16_from_f64(orc.fp8_decode(qWu) * swu[:, None].astype(np.float64))
    np.testing.assert_array_equal(orc.f8_linear(qX, sx, qW, sw, R), orc.linear(Xb, Wb, R))
    np.testing.assert_array_equal(orc.f8_swiglu(qX, sx, qW, sw, qWu, swu), orc.swiglu(Xb, Wb, Wub))


def pin_f8_at_matches_full(orc, seed=73):
    rng = np.random.default_rng(seed)
    M, N, K = 7, 9, 24
    qX, qW, qWu = _rand_f8(rng, (M, K)), _rand_f8(rng, (N, K)), _rand_f8(rng, (N, K))
    sx, sw, swu = _rand_scales(rng, M), _rand_scales(rng, N), _rand_scales(rng, N)
    R = _rand_bits(rng, (M, N))
    rows, cols = rng.integers(0, M, 40), rng.integers(0, N, 40)
    np.testing.assert_array_equal(orc.f8_linear_at(qX, sx, qW, sw, R, rows, cols),
                                  orc.f8_linear(qX, sx, qW, sw, R)[rows, cols])
    np.testing.assert_array_equal(orc.f8_swiglu_at(qX, sx, qW, sw, qWu, swu, rows, cols),
                                  orc.f8_swiglu(qX, sx, qW, sw, qWu, swu)[rows, cols])


F8_PINS = [
    pin_f8_decode,
    pin_f8_dequant_exact,
    pin_f8_matches_bf16_oracle,
    pin_f8_at_matches_full,
]


# ---------------------------------------------------------------- grouped ----
def _rows_of(counts, e, Mpad):
    return Mpad if counts is None else int(min(max(int(counts[e]), 0), Mpad))


def pin_grouped_exact_bruteforce(orc, trials=12, seed=51):
    rng = np.random.default_rng(seed)
    for t in range(trials):
        E, Mpad, N, K = (int(v) for v in rng.integers(1, 6, size=4))
        X = _rand_bits(rng, (E, Mpad, K))
        W = _rand_bits(rng, (E, N, K))
        counts = None if t % 4 == 0 else rng.integers(-2, Mpad + 3, size=E).astype(np.int32)
        Y = orc.grouped_linear(X, W, counts)
        xf, wf = bf16_bits_to_f64(X), bf16_bits_to_f64(W)
        for e in range(E):
            r = _rows_of(counts, e, Mpad)
            assert np.isnan(Y[e, r:]).all()
            for i in range(r):
                for j in range(N):
                    exact = sum((Fraction(xf[e, i, k]) * Fraction(wf[e, j, k]) for k in range(K)), Fraction(0))
                    mag = sum(abs(Fraction(xf[e, i, k]) * Fraction(wf[e, j, k])) for k in range(K))
                    assert abs(Fraction(Y[e, i, j]) - exact) <= mag / 2**50, (e, i, j)


def pin_grouped_reduces_per_expert(orc, seed=52):
    """Expert by expert, the valid rows equal the plain and SwiGLU oracles bit for bit."""
    rng = np.random.default_rng(seed)
    E, Mpad, N, K = 5, 9, 7, 33
    X = _rand_bits(rng, (E, Mpad, K), 2.0)
    W = _rand_bits(rng, (E, N, K), 1.0 / np.sqrt(K))
    Wu = _rand_bits(rng, (E, N, K), 1.0 / np.sqrt(K))
    counts = np.array([0, 3, 9, 12, -1], np.int32)
    Y = orc.grouped_linear(X, W, counts)
    H = orc.grouped_swiglu(X, W, Wu, counts)
    for e in range(E):
        r = _rows_of(counts, e, Mpad)
        if r:
            np.testing.assert_array_equal(Y[e, :r], orc.linear(X[e, :r], W[e]))
            np.testing.assert_array_equal(H[e, :r], orc.swiglu(X[e, :r], W[e], Wu[e]))
    np.testing.assert_array_equal(orc.grouped_linear(X, W)[2], orc.linear(X[2], W[2]))


def pin_grouped_gap_rows_untouched(orc, seed=53):
    rng = np.random.default_rng(seed)
    E, Mpad, N, K = 4, 6, 5, 8
    X = _rand_bits(rng, (E, Mpad, K))
    W = _rand_bits(rng, (E, N, K))
    counts = np.array([2, 0, 6, 4], np.int32)
    out = np.full((E, Mpad, N), 12345.5)
    orc.grouped_linear(X, W, counts, out=out)
    for e in range(E):
        r = int(counts[e])
        assert (out[e, r:] == 12345.5).all()
        assert not (out[e, :r] == 12345.5).any()


def pin_grouped_expert_permutation(orc, seed=54):
    rng = np.random.default_rng(seed)
    E, Mpad, N, K = 6, 5, 4, 12
    X = _rand_bits(rng, (E, Mpad, K))
    W = _rand_bits(rng, (E, N, K))
    counts = rng.integers(0, Mpad + 1, size=E).astype(np.int32)
    pe = rng.permutation(E)
    np.testing.assert_array_equal(orc.grouped_linear(X[pe], W[pe], counts[pe]),
                                  orc.grouped_linear(X, W, counts)[pe])


def pin_grouped_at_matches_full(orc, seed=55):
    rng = np.random.default_rng(seed)
    E, Mpad, N, K = 4, 7, 6, 10
    X = _rand_bits(rng, (E, Mpad, K))
    W = _rand_bits(rng, (E, N, K))
    Wu = _rand_bits(rng, (E, N, K))
    counts = np.array([7, 2, 5, 1], np.int32)
    full, fullh = orc.grouped_linear(X, W, counts), orc.grouped_swiglu(X, W, Wu, counts)
    g = rng.integers(0, E, 60)
    r = np.array([rng.integers(0, counts[e]) for e in g])
    c = rng.integers(0, N, 60)
    np.testing.assert_array_equal(orc.grouped_at(X, W, None, counts, g, r, c), full[g, r, c])
    np.testing.assert_array_equal(orc.grouped_at(X, W, Wu, counts, g, r, c), fullh[g, r, c])
    try:
        orc.grouped_at(X, W, None, counts, [1], [2], [0])      # row 2 of expert 1 is a gap row
    except ValueError:
        pass
    else:
        raise AssertionError("a gap-row position was accepted")


GRP_PINS = [
    pin_grouped_exact_bruteforce,
    pin_grouped_reduces_per_expert,
    pin_grouped_gap_rows_untouched,
    pin_grouped_expert_permutation,
    pin_grouped_at_matches_full,
]

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
] + EX_PINS + GLU_PINS + I8_PINS + F8_PINS + GRP_PINS
