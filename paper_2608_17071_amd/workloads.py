"""Seeded synthetic inputs for Y = X.W^T + R.

This module only draws and lays out input bytes; it holds none of the
operator's arithmetic.  Both the GPU library (through the tests and the
benchmark) and the CPU oracle consume exactly the bytes produced here.

Recipe (all tensors bf16, dense, row-major; X is [M,K], W is [N,K] in
nn.Linear [out, in] layout, R is [M,N]):

* ``g = torch.Generator().manual_seed(seed)``; X is drawn first, then W,
  then R, each as float32 and rounded to bf16 (nearest-even) by torch.
* ``normal``:  X, W ~ N(0,1)/sqrt(K) and R ~ N(0,1).
* ``uniform``: X, W ~ U(-1,1)/sqrt(K) (``rand*2-1``), no residual.

The named workloads are the attention-output-projection shapes the paper
motivates (Sec. "From Sequential Plateaus to Design Requirements": one
operator scored over 16 shapes with per-M configuration choices; Sec.
"Guided Sequential GEMM Boundary Study": a large square BF16 GEMM).  The
benchmark suite's own 16 shapes are not public in the paper; the sweep
below (M in {1, 64, 512, 4096} x hidden in {2048, 4096, 5120, 8192}, N = K =
hidden) stands in for them.
"""
from __future__ import annotations

import hashlib
import math
from dataclasses import dataclass

import numpy as np
import torch


@dataclass(frozen=True)
class Workload:
    name: str
    M: int
    N: int
    K: int
    residual: bool
    dist: str          # "normal" or "uniform"
    seed: int

    @property
    def flops(self) -> int:
        return 2 * self.M * self.N * self.K

    @property
    def algorithmic_bytes(self) -> int:
        """Each operand read once and Y written once, 2 bytes per element."""
        b = 2 * (self.M * self.K + self.N * self.K + self.M * self.N)
        if self.residual:
            b += 2 * self.M * self.N
        return b


SWEEP_M = (1, 64, 512, 4096)
SWEEP_HIDDEN = (2048, 4096, 5120, 8192)


def _sweep():
    out = []
    for mi, m in enumerate(SWEEP_M):
        for hi, h in enumerate(SWEEP_HIDDEN):
            s = mi * len(SWEEP_HIDDEN) + hi
            out.append(Workload(f"sweep_s{s:02d}_m{m}_h{h}", m, h, h, True, "normal", s))
    return tuple(out)


TINY = Workload("tiny_m128_n256_k256", 128, 256, 256, True, "normal", 0)
DECODE = Workload("decode_m16_h4096", 16, 4096, 4096, True, "normal", 0)
PREFILL = Workload("prefill_m4096_h4096", 4096, 4096, 4096, True, "normal", 0)
SQUARE = Workload("square_plain_8192", 8192, 8192, 8192, False, "uniform", 0)
SWEEP = _sweep()
ALL = (TINY, DECODE, PREFILL, SQUARE) + SWEEP
BY_NAME = {w.name: w for w in ALL}


# ---- the general form Y = alpha X W^T + beta C + bias ----------------------

@dataclass(frozen=True)
class GeneralWorkload:
    """A general-form call: X is the leading K columns of an [M, K + x_pad]
    buffer (row stride ldx = K + x_pad); C ([M,N], when has_c) and bias ([N],
    when has_bias) are drawn like R; alpha and beta are binary32 values."""
    name: str
    M: int
    N: int
    K: int
    alpha: float
    beta: float
    has_c: bool
    has_bias: bool
    x_pad: int
    seed: int

    @property
    def ldx(self) -> int:
        return self.K + self.x_pad

    @property
    def flops(self) -> int:
        return 2 * self.M * self.N * self.K

    @property
    def algorithmic_bytes(self) -> int:
        """X, W, C and bias read once, Y written once, 2 bytes per element."""
        b = 2 * (self.M * self.K + self.N * self.K + self.M * self.N)
        if self.has_c and self.beta != 0.0:
            b += 2 * self.M * self.N
        if self.has_bias:
            b += 2 * self.N
        return b


# The decoder layer's two residual GEMM sites at Llama-class sizes (hidden
# 4096, intermediate 14336; hidden 5120, intermediate 13824): the
# output projection with a bias, the down projection reading its input
# through a row stride (a slice of a wider activation buffer), a decode
# step with a scaled residual, and a prefill step with beta != 1 and a bias.
GENERAL = (
    GeneralWorkload("general_oproj_bias_m4096_h4096", 4096, 4096, 4096, 1.0, 1.0, True, True, 0, 101),
    GeneralWorkload("general_down_strided_m4096_n4096_k14336", 4096, 4096, 14336, 1.0, 1.0, True, False, 128, 102),
    GeneralWorkload("general_down_scaled_m16_n4096_k14336", 16, 4096, 14336, 1.0, 0.5, True, False, 0, 103),
    GeneralWorkload("general_down_bias_m512_n5120_k13824", 512, 5120, 13824, 0.5, 0.25, True, True, 0, 104),
)
GENERAL_BY_NAME = {w.name: w for w in GENERAL}


def make_general_inputs(w: GeneralWorkload) -> dict:
    """Draw X (dense [M,K]), W, C and bias as bf16 CPU tensors: X ~ N(0,1)/sqrt(K),
    W ~ N(0,1)/sqrt(K), C ~ N(0,1), bias ~ N(0,1), in that order from one seed."""
    g = torch.Generator().manual_seed(w.seed)
    scale = 1.0 / math.sqrt(w.K) if w.K > 0 else 1.0
    X = (torch.randn((w.M, w.K), generator=g) * scale).to(torch.bfloat16)
    W = (torch.randn((w.N, w.K), generator=g) * scale).to(torch.bfloat16)
    C = torch.randn((w.M, w.N), generator=g).to(torch.bfloat16)
    b = torch.randn((w.N,), generator=g).to(torch.bfloat16)
    return {"X": X, "W": W, "C": C if w.has_c else None, "bias": b if w.has_bias else None}


# ---- SwiGLU: H = silu(X Wg^T) * (X Wu^T) -----------------------------------

@dataclass(frozen=True)
class GluWorkload:
    """A SwiGLU call: X [M,K] (K = hidden size), Wg and Wu [N,K] (N =
    intermediate size), H [M,N]."""
    name: str
    M: int
    N: int
    K: int
    seed: int

    @property
    def flops(self) -> int:
        """Both projections; the SiLU-multiply adds a few operations per output."""
        return 4 * self.M * self.N * self.K

    @property
    def algorithmic_bytes(self) -> int:
        """X, Wg and Wu read once, H written once, 2 bytes per element."""
        return 2 * (self.M * self.K + 2 * self.N * self.K + self.M * self.N)


# The decoder layer's gate/up projections at Llama-class sizes (hidden 4096,
# intermediate 14336; hidden 5120, intermediate 13824): a decode step, a
# prefill chunk below the paper's INT8 threshold of M = 1000 tokens (the
# BF16 path), and a full prefill.
GLU = (
    GluWorkload("swiglu_decode_m16_h4096_i14336", 16, 14336, 4096, 201),
    GluWorkload("swiglu_m512_h5120_i13824", 512, 13824, 5120, 202),
    GluWorkload("swiglu_prefill_m4096_h4096_i14336", 4096, 14336, 4096, 203),
)
GLU_BY_NAME = {w.name: w for w in GLU}


def make_glu_inputs(w: GluWorkload) -> dict:
    """Draw X ~ N(0,1) (normalised hidden states), then Wg and Wu ~ N(0,1)/sqrt(K),
    as bf16 CPU tensors from one seed, so that the gate and up sums are about
    N(0,1) and the gate spans SiLU's curved range."""
    g = torch.Generator().manual_seed(w.seed)
    scale = 1.0 / math.sqrt(w.K) if w.K > 0 else 1.0
    X = torch.randn((w.M, w.K), generator=g).to(torch.bfloat16)
    Wg = (torch.randn((w.N, w.K), generator=g) * scale).to(torch.bfloat16)
    Wu = (torch.randn((w.N, w.K), generator=g) * scale).to(torch.bfloat16)
    return {"X": X, "Wg": Wg, "Wu": Wu}


# ---- INT8 with dequantisation scales ----------------------------------------

@dataclass(frozen=True)
class I8Workload:
    """An 8-bit call: qX [M,K], qW (or qWg, qWu) [N,K] int8 (fmt "i8") or FP8
    E4M3 (fmt "f8") with float32 scales per row of qX and per output channel;
    a bf16 residual when `residual`; SwiGLU when `swiglu`."""
    name: str
    M: int
    N: int
    K: int
    swiglu: bool
    residual: bool
    seed: int
    fmt: str = "i8"

    eight_bit = True     # 8-bit operands: the roofline uses the 8-bit MFMA peak

    @property
    def flops(self) -> int:
        """Integer multiply-adds counted as 2 operations (4MNK for SwiGLU)."""
        return (4 if self.swiglu else 2) * self.M * self.N * self.K

    @property
    def algorithmic_bytes(self) -> int:
        """int8 operands and float32 scales read once, bf16 output written once."""
        w = 2 if self.swiglu else 1
        b = self.M * self.K + w * self.N * self.K + 4 * self.M + 4 * w * self.N + 2 * self.M * self.N
        if self.residual:
            b += 2 * self.M * self.N
        return b


# The precision axis of the same layers: the o-proj / down-proj site with a
# residual (prefill and decode), the large square GEMM, and the decoder
# layer's INT8 gate/up path, which the paper takes from M = 1000 tokens up.
I8 = (
    I8Workload("i8_decode_m16_h4096", 16, 4096, 4096, False, True, 301),
    I8Workload("i8_prefill_m4096_h4096", 4096, 4096, 4096, False, True, 302),
    I8Workload("i8_square_8192", 8192, 8192, 8192, False, False, 303),
    I8Workload("swiglu_i8_m1024_h5120_i13824", 1024, 13824, 5120, True, False, 304),
    I8Workload("swiglu_i8_prefill_m4096_h4096_i14336", 4096, 14336, 4096, True, False, 305),
)
I8_BY_NAME = {w.name: w for w in I8}

# The same layers with FP8 E4M3 operands.
F8 = (
    I8Workload("f8_prefill_m4096_h4096", 4096, 4096, 4096, False, True, 311, "f8"),
    I8Workload("f8_square_8192", 8192, 8192, 8192, False, False, 312, "f8"),
    I8Workload("swiglu_f8_prefill_m4096_h4096_i14336", 4096, 14336, 4096, True, False, 313, "f8"),
)
F8_BY_NAME = {w.name: w for w in F8}


def make_i8_inputs(w: I8Workload) -> dict:
    """Draw, from one seed and in this order: qX = round(N(0,1) * 40) clipped
    to [-128, 127] (int8), or N(0,1) * 8 rounded to E4M3 (FP8); the weight(s)
    the same way; sx ~ U(0.5, 1.5)/a per row; per-channel scales
    ~ U(0.5, 1.5)/(a sqrt(K)) per weight (a = 40 for int8, 8 for FP8); R
    ~ N(0,1) in bf16 when the workload has a residual.  The dequantised sums
    are then about N(0,1) (the gate spans SiLU's curved range)."""
    g = torch.Generator().manual_seed(w.seed)
    amp = 40.0 if w.fmt == "i8" else 8.0

    def q(shape):
        if w.fmt == "f8":      # N(0,1) * 8 rounded to E4M3 by torch (|values| stay far below 448)
            return (torch.randn(shape, generator=g) * amp).to(torch.float8_e4m3fn)
        return torch.clamp(torch.round(torch.randn(shape, generator=g) * amp), -128, 127).to(torch.int8)

    qx = q((w.M, w.K))
    ws = [q((w.N, w.K)) for _ in range(2 if w.swiglu else 1)]
    sx = ((torch.rand(w.M, generator=g) + 0.5) / amp).to(torch.float32)
    kscale = amp * math.sqrt(w.K) if w.K > 0 else amp
    ss = [((torch.rand(w.N, generator=g) + 0.5) / kscale).to(torch.float32) for _ in ws]
    out = {"qX": qx, "sx": sx, "qW": ws[0], "sw": ss[0], "R": None}
    if w.swiglu:
        out["qWu"], out["swu"] = ws[1], ss[1]
    if w.residual:
        out["R"] = torch.randn((w.M, w.N), generator=g).to(torch.bfloat16)
    return out


# ---- grouped (per-expert) forms over an expert-major padded layout ---------

@dataclass(frozen=True)
class GroupedWorkload:
    """A mixture-of-experts projection: T tokens each routed to top_k of G
    experts; the token-expert rows sit expert-contiguously in a [G x M_pad]
    buffer.  swiglu: the experts' gate/up projections with the SiLU-multiply
    (N = intermediate, K = hidden); else a plain projection (e.g. the down
    projection, N = hidden, K = intermediate)."""
    name: str
    T: int
    top_k: int
    G: int
    N: int
    K: int
    swiglu: bool
    seed: int

    @property
    def counts(self) -> np.ndarray:
        return routing_counts(self.T, self.top_k, self.G, self.seed)

    @property
    def Mpad(self) -> int:
        return padded_capacity(self.counts)

    @property
    def rows(self) -> int:
        """Valid rows over all experts (= T * top_k)."""
        return int(self.counts.sum())

    @property
    def M(self) -> int:
        """Rows the projection computes: the valid rows of all experts."""
        return self.rows

    @property
    def flops(self) -> int:
        return (4 if self.swiglu else 2) * self.rows * self.N * self.K

    @property
    def algorithmic_bytes(self) -> int:
        """Valid X rows, every expert's weights and the valid output rows, once
        each (bf16), and the counts."""
        w = 2 if self.swiglu else 1
        return 2 * (self.rows * self.K + w * self.G * self.N * self.K + self.rows * self.N) + 4 * self.G


_COUNTS_CACHE: dict = {}


def routing_counts(T: int, top_k: int, G: int, seed: int) -> np.ndarray:
    """Rows per expert when each of T tokens picks its top_k of G experts by
    i.i.d. uniform router scores (torch.rand from `seed`, then topk)."""
    key = (T, top_k, G, seed)
    if key not in _COUNTS_CACHE:
        g = torch.Generator().manual_seed(seed)
        idx = torch.rand((T, G), generator=g).topk(top_k, dim=1).indices
        _COUNTS_CACHE[key] = torch.bincount(idx.flatten(), minlength=G).numpy().astype(np.int32)
    return _COUNTS_CACHE[key]


def padded_capacity(counts: np.ndarray, multiple: int = 32) -> int:
    """M_pad: the largest expert's row count rounded up to a multiple of 32."""
    m = int(counts.max()) if counts.size else 0
    return max(multiple, -(-m // multiple) * multiple)


# The mixture-of-experts layer of the paper's case study (256 experts, top-8,
# hidden 4096, intermediate 2048) at its smallest and largest token counts:
# the experts' gate/up projections with SwiGLU and their down projections.
GROUPED = (
    GroupedWorkload("moe_gate_up_t2048", 2048, 8, 256, 2048, 4096, True, 401),
    GroupedWorkload("moe_gate_up_t6144", 6144, 8, 256, 2048, 4096, True, 402),
    GroupedWorkload("moe_down_t2048", 2048, 8, 256, 4096, 2048, False, 403),
    GroupedWorkload("moe_down_t6144", 6144, 8, 256, 4096, 2048, False, 404),
)
GROUPED_BY_NAME = {w.name: w for w in GROUPED}


def make_grouped_inputs(w: GroupedWorkload, device: str = "cuda") -> dict:
    """counts from the routing draw (seed, on the host); then, from seed + 1
    on `device`'s torch generator: X rows ~ N(0,1) (the valid rows of each
    expert; gap rows zero), the weights [G, N, K] ~ N(0,1)/sqrt(K) (gate, then
    up), all bf16.  The expert weights run to billions of values, so they are
    drawn where they are used; a check copies the same bytes to the host."""
    counts = w.counts
    Mpad = w.Mpad
    g = torch.Generator(device=device).manual_seed(w.seed + 1)
    X = torch.randn((w.G, Mpad, w.K), generator=g, device=device)
    valid = torch.from_numpy(counts.astype(np.int64)).to(device)
    rows = torch.arange(Mpad, device=device)[None, :, None] < valid[:, None, None]
    X = torch.where(rows, X, torch.zeros((), device=device)).to(torch.bfloat16)
    scale = 1.0 / math.sqrt(w.K) if w.K > 0 else 1.0
    ws = []
    for _ in range(2 if w.swiglu else 1):
        t = torch.randn((w.G, w.N, w.K), generator=g, device=device)
        t.mul_(scale)
        ws.append(t.to(torch.bfloat16))
        del t
    out = {"X": X, "W": ws[0], "counts": torch.from_numpy(counts.copy()).to(device), "Mpad": Mpad}
    if w.swiglu:
        out["Wu"] = ws[1]
    return out


def custom(M: int, N: int, K: int, residual: bool = True, dist: str = "normal",
           seed: int = 0, name: str | None = None) -> Workload:
    return Workload(name or f"custom_m{M}_n{N}_k{K}", M, N, K, residual, dist, seed)


def make_inputs(w: Workload) -> dict:
    """Draw X, W (and R) on the host as bf16 CPU tensors."""
    g = torch.Generator().manual_seed(w.seed)
    scale = 1.0 / math.sqrt(w.K) if w.K > 0 else 1.0

    def draw(shape):
        if w.dist == "normal":
            return torch.randn(shape, generator=g, dtype=torch.float32)
        if w.dist == "uniform":
            return torch.rand(shape, generator=g, dtype=torch.float32) * 2.0 - 1.0
        raise ValueError(f"unknown distribution {w.dist!r}")

    X = (draw((w.M, w.K)) * scale).to(torch.bfloat16)
    W = (draw((w.N, w.K)) * scale).to(torch.bfloat16)
    out = {"X": X, "W": W, "R": None}
    if w.residual:
        out["R"] = torch.randn((w.M, w.N), generator=g, dtype=torch.float32).to(torch.bfloat16)
    return out


def bits(t: torch.Tensor) -> np.ndarray:
    """The bf16 bit patterns of a CPU tensor as a numpy uint16 array (a view)."""
    if t.dtype != torch.bfloat16:
        raise TypeError("expected a bf16 tensor")
    return t.contiguous().view(torch.int16).numpy().view(np.uint16)


def from_bits(a: np.ndarray) -> torch.Tensor:
    """bf16 CPU tensor holding the given uint16 bit patterns."""
    a = np.ascontiguousarray(a, dtype=np.uint16)
    return torch.from_numpy(a.view(np.int16).copy()).view(torch.bfloat16)


def sha256(*tensors) -> str:
    h = hashlib.sha256()
    for t in tensors:
        if t is not None:
            h.update(bits(t).tobytes())
    return h.hexdigest()


# ---- structured inputs for closed-form checks (bit patterns only) ----------

def rank1_integer(M: int, N: int, K: int, seed: int = 0, residual: bool = True):
    """X[i,k] = a_i u_k and W[j,k] = b_j v_k with small integers.

    a, b are drawn from [-8, 8]; u, v from {-1, 0, 1} and forced
    non-constant.  With R drawn from the integers in [-64, 64] every value is
    exactly representable in bf16, and every partial sum of the product is an
    integer of magnitude below 2^24.  Returns (X, W, R, a, b, u, v) with the
    tensors as bf16 and the factors as int64 numpy arrays.
    """
    rng = np.random.default_rng(seed)
    a = rng.integers(-8, 9, size=M)
    b = rng.integers(-8, 9, size=N)
    u = rng.integers(-1, 2, size=K)
    v = rng.integers(-1, 2, size=K)
    if K >= 2:
        u[0], u[-1] = 1, -1
        v[0], v[1 % K] = 1, 1
    X = torch.from_numpy(np.outer(a, u).astype(np.float32)).to(torch.bfloat16)
    W = torch.from_numpy(np.outer(b, v).astype(np.float32)).to(torch.bfloat16)
    R = None
    if residual:
        R = torch.from_numpy(rng.integers(-64, 65, size=(M, N)).astype(np.float32)).to(torch.bfloat16)
    return X, W, R, a.astype(np.int64), b.astype(np.int64), u.astype(np.int64), v.astype(np.int64)


def identity_weight(K: int) -> torch.Tensor:
    return torch.eye(K, dtype=torch.float32).to(torch.bfloat16)


def zero_weight(N: int, K: int) -> torch.Tensor:
    return torch.zeros((N, K), dtype=torch.bfloat16)
