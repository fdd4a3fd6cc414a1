"""CPU oracle for Y = X.W^T + R, its general form
D = alpha.X.W^T + beta.C + bias, the gated MLP input projection
H = silu(X.Wg^T) * (X.Wu^T), their INT8 and FP8 (E4M3) forms with per-row
and per-column dequantisation scales, and grouped (per-expert) forms over an
expert-major padded layout (TEST INFRASTRUCTURE ONLY).

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The GPU library never imports, links
or falls back to it, and the two share no code: the only thing they have in
common is the byte content of the seeded inputs.

The arithmetic lives in ``kernelarc_oracle.c`` (plain C, fp64, ascending k);
this module builds it with gcc and marshals numpy arrays through ctypes.
Inputs are bf16 bit patterns held in ``numpy.uint16`` arrays.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SOURCE = os.path.join(HERE, "kernelarc_oracle.c")
LIBRARY = os.path.join(HERE, "libkernelarc_oracle.so")

# -O2 without -ffast-math and with contraction off keeps the k-order and the
# separate multiply/add of the definition; OpenMP only splits output rows.
CFLAGS = ["-std=c11", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fopenmp",
          "-shared", "-fPIC"]


def build(source: str = SOURCE, output: str = LIBRARY) -> str:
    """Compile the oracle with gcc into a shared library; returns its path."""
    tmp = output + ".tmp"
    cmd = ["gcc", *CFLAGS, "-o", tmp, source, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, output)
    return output


_I64 = ctypes.c_int64
_P = ctypes.c_void_p


class Oracle:
    """ctypes view of one compiled oracle library."""

    def __init__(self, path: str = LIBRARY):
        if not os.path.exists(path):
            raise FileNotFoundError(
                f"oracle library {path} is not built; run __graft_entry__.build()")
        lib = ctypes.CDLL(path)
        lib.ka_oracle_linear.argtypes = [_I64, _I64, _I64, _P, _P, _P, _P]
        lib.ka_oracle_linear.restype = ctypes.c_int
        lib.ka_oracle_linear_pair.argtypes = [_I64, _I64, _I64, _P, _P, _P, _P, _P]
        lib.ka_oracle_linear_pair.restype = ctypes.c_int
        lib.ka_oracle_linear_at.argtypes = [_I64, _I64, _I64, _P, _P, _P, _I64, _P, _P, _P]
        lib.ka_oracle_linear_at.restype = ctypes.c_int
        lib.ka_oracle_linear_ex.argtypes = [_I64, _I64, _I64, ctypes.c_float, _P, _I64, _P, _I64,
                                            ctypes.c_float, _P, _I64, _P, _P]
        lib.ka_oracle_linear_ex.restype = ctypes.c_int
        lib.ka_oracle_linear_ex_at.argtypes = [_I64, _I64, _I64, ctypes.c_float, _P, _I64, _P, _I64,
                                               ctypes.c_float, _P, _I64, _P, _I64, _P, _P, _P]
        lib.ka_oracle_linear_ex_at.restype = ctypes.c_int
        lib.ka_oracle_swiglu.argtypes = [_I64, _I64, _I64, _P, _P, _P, _P]
        lib.ka_oracle_swiglu.restype = ctypes.c_int
        lib.ka_oracle_swiglu_at.argtypes = [_I64, _I64, _I64, _P, _P, _P, _I64, _P, _P, _P]
        lib.ka_oracle_swiglu_at.restype = ctypes.c_int
        lib.ka_oracle_i8_dot.argtypes = [_I64, _I64, _I64, _P, _P, _P]
        lib.ka_oracle_i8_dot.restype = ctypes.c_int
        lib.ka_oracle_i8_linear.argtypes = [_I64, _I64, _I64, _P, _P, _P, _P, _P, _P]
        lib.ka_oracle_i8_linear.restype = ctypes.c_int
        lib.ka_oracle_i8_linear_at.argtypes = [_I64, _I64, _I64, _P, _P, _P, _P, _P, _I64, _P, _P, _P]
        lib.ka_oracle_i8_linear_at.restype = ctypes.c_int
        lib.ka_oracle_i8_swiglu.argtypes = [_I64, _I64, _I64, _P, _P, _P, _P, _P, _P, _P]
        lib.ka_oracle_i8_swiglu.restype = ctypes.c_int
        lib.ka_oracle_i8_swiglu_at.argtypes = [_I64, _I64, _I64, _P, _P, _P, _P, _P, _P, _I64, _P, _P, _P]
        lib.ka_oracle_i8_swiglu_at.restype = ctypes.c_int
        lib.ka_oracle_grouped_linear.argtypes = [_I64, _I64, _I64, _I64, _P, _P, _P, _P]
        lib.ka_oracle_grouped_linear.restype = ctypes.c_int
        lib.ka_oracle_grouped_swiglu.argtypes = [_I64, _I64, _I64, _I64, _P, _P, _P, _P, _P]
        lib.ka_oracle_grouped_swiglu.restype = ctypes.c_int
        lib.ka_oracle_grouped_at.argtypes = [_I64, _I64, _I64, _I64, _P, _P, _P, _P, ctypes.c_int, _I64, _P, _P,
                                             _P, _P]
        lib.ka_oracle_grouped_at.restype = ctypes.c_int
        lib.ka_oracle_fp8_decode.argtypes = [_I64, _P, _P]
        lib.ka_oracle_fp8_decode.restype = None
        lib.ka_oracle_f8_linear.argtypes = [_I64, _I64, _I64, _P, _P, _P, _P, _P, _P]
        lib.ka_oracle_f8_linear.restype = ctypes.c_int
        lib.ka_oracle_f8_linear_at.argtypes = [_I64, _I64, _I64, _P, _P, _P, _P, _P, _I64, _P, _P, _P]
        lib.ka_oracle_f8_linear_at.restype = ctypes.c_int
        lib.ka_oracle_f8_swiglu.argtypes = [_I64, _I64, _I64, _P, _P, _P, _P, _P, _P, _P]
        lib.ka_oracle_f8_swiglu.restype = ctypes.c_int
        lib.ka_oracle_f8_swiglu_at.argtypes = [_I64, _I64, _I64, _P, _P, _P, _P, _P, _P, _I64, _P, _P, _P]
        lib.ka_oracle_f8_swiglu_at.restype = ctypes.c_int
        lib.ka_oracle_round_bf16.argtypes = [_I64, _P, _P]
        lib.ka_oracle_round_bf16.restype = None
        lib.ka_oracle_threads.argtypes = []
        lib.ka_oracle_threads.restype = ctypes.c_int
        lib.ka_oracle_set_threads.argtypes = [ctypes.c_int]
        lib.ka_oracle_set_threads.restype = None
        self.lib = lib
        self.path = path

    @staticmethod
    def _bits(a, shape):
        a = np.ascontiguousarray(a)
        if a.dtype != np.uint16:
            raise TypeError("oracle inputs are bf16 bit patterns (numpy.uint16)")
        if a.shape != shape:
            raise ValueError(f"expected shape {shape}, got {a.shape}")
        return a

    def linear(self, X, W, R=None) -> np.ndarray:
        """Y[i,j] = sum_k X[i,k] W[j,k] (+ R[i,j]) in float64."""
        M, K = X.shape
        N = W.shape[0]
        X = self._bits(X, (M, K))
        W = self._bits(W, (N, K))
        Rp = None
        if R is not None:
            R = self._bits(R, (M, N))
            Rp = R.ctypes.data
        Y = np.empty((M, N), dtype=np.float64)
        rc = self.lib.ka_oracle_linear(M, N, K, X.ctypes.data, W.ctypes.data, Rp,
                                       Y.ctypes.data)
        if rc != 0:
            raise ValueError("oracle rejected its arguments")
        return Y

    def linear_pair(self, X, W, R):
        """(X W^T, X W^T + R) in float64 from one evaluation of each k-sum:
        the values of linear(X, W) and linear(X, W, R)."""
        M, K = X.shape
        N = W.shape[0]
        X = self._bits(X, (M, K))
        W = self._bits(W, (N, K))
        R = self._bits(R, (M, N))
        Yp = np.empty((M, N), dtype=np.float64)
        Yr = np.empty((M, N), dtype=np.float64)
        rc = self.lib.ka_oracle_linear_pair(M, N, K, X.ctypes.data, W.ctypes.data, R.ctypes.data,
                                            Yp.ctypes.data, Yr.ctypes.data)
        if rc != 0:
            raise ValueError("oracle rejected its arguments")
        return Yp, Yr

    def linear_at(self, X, W, R, rows, cols) -> np.ndarray:
        """The same definition evaluated at the positions (rows[t], cols[t])."""
        M, K = X.shape
        N = W.shape[0]
        X = self._bits(X, (M, K))
        W = self._bits(W, (N, K))
        Rp = None
        if R is not None:
            R = self._bits(R, (M, N))
            Rp = R.ctypes.data
        rows = np.ascontiguousarray(rows, dtype=np.int64)
        cols = np.ascontiguousarray(cols, dtype=np.int64)
        if rows.shape != cols.shape or rows.ndim != 1:
            raise ValueError("rows and cols must be 1-D and of equal length")
        out = np.empty(rows.shape[0], dtype=np.float64)
        rc = self.lib.ka_oracle_linear_at(M, N, K, X.ctypes.data, W.ctypes.data, Rp,
                                          rows.shape[0], rows.ctypes.data,
                                          cols.ctypes.data, out.ctypes.data)
        if rc != 0:
            raise ValueError("oracle rejected its arguments")
        return out

    @staticmethod
    def _strided(a, rows, cols, what):
        """A 2-D bf16 view with unit stride along its last axis: (array, ld)."""
        if not isinstance(a, np.ndarray) or a.dtype != np.uint16:
            raise TypeError(f"{what}: oracle inputs are bf16 bit patterns (numpy.uint16)")
        if a.ndim != 2 or a.shape != (rows, cols):
            raise ValueError(f"{what}: expected shape {(rows, cols)}, got {a.shape}")
        if rows > 0 and cols > 0 and a.strides[1] != 2:
            raise ValueError(f"{what}: the last axis must be contiguous")
        ld = a.strides[0] // 2 if rows > 1 else max(cols, 1)
        if rows > 1 and (a.strides[0] % 2 or ld < cols):
            raise ValueError(f"{what}: bad row stride")
        return a, ld

    def _ex_args(self, X, W, C, bias, alpha, beta):
        M, K = X.shape
        N = W.shape[0]
        X, ldx = self._strided(X, M, K, "X")
        W, ldw = self._strided(W, N, K, "W")
        Cp, ldc = None, max(N, 1)
        if C is not None:
            C, ldc = self._strided(C, M, N, "C")
            Cp = C.ctypes.data
        bp = None
        if bias is not None:
            bias = np.ascontiguousarray(bias)
            if bias.dtype != np.uint16 or bias.shape != (N,):
                raise ValueError("bias: expected bf16 bit patterns of shape (N,)")
            bp = bias.ctypes.data
        keep = (X, W, C, bias)
        return (M, N, K, float(alpha), X.ctypes.data, ldx, W.ctypes.data, ldw,
                float(beta), Cp, ldc, bp), keep

    def linear_ex(self, X, W, C=None, bias=None, alpha=1.0, beta=1.0) -> np.ndarray:
        """D = alpha * X W^T + beta * C + bias in float64 (X, W, C may be
        row-strided views; beta = 0 leaves C unread)."""
        args, keep = self._ex_args(X, W, C, bias, alpha, beta)
        D = np.empty((args[0], args[1]), dtype=np.float64)
        rc = self.lib.ka_oracle_linear_ex(*args, D.ctypes.data)
        if rc != 0:
            raise ValueError("oracle rejected its arguments")
        del keep
        return D

    def linear_ex_at(self, X, W, C, bias, alpha, beta, rows, cols) -> np.ndarray:
        """The general form at the positions (rows[t], cols[t])."""
        args, keep = self._ex_args(X, W, C, bias, alpha, beta)
        rows = np.ascontiguousarray(rows, dtype=np.int64)
        cols = np.ascontiguousarray(cols, dtype=np.int64)
        if rows.shape != cols.shape or rows.ndim != 1:
            raise ValueError("rows and cols must be 1-D and of equal length")
        out = np.empty(rows.shape[0], dtype=np.float64)
        rc = self.lib.ka_oracle_linear_ex_at(*args, rows.shape[0], rows.ctypes.data,
                                             cols.ctypes.data, out.ctypes.data)
        if rc != 0:
            raise ValueError("oracle rejected its arguments")
        del keep
        return out

    def swiglu(self, X, Wg, Wu) -> np.ndarray:
        """H[i,j] = silu(G[i,j]) * U[i,j] in float64, with G = X Wg^T,
        U = X Wu^T and silu(z) = z / (1 + exp(-z))."""
        M, K = X.shape
        N = Wg.shape[0]
        X = self._bits(X, (M, K))
        Wg = self._bits(Wg, (N, K))
        Wu = self._bits(Wu, (N, K))
        H = np.empty((M, N), dtype=np.float64)
        rc = self.lib.ka_oracle_swiglu(M, N, K, X.ctypes.data, Wg.ctypes.data, Wu.ctypes.data,
                                       H.ctypes.data)
        if rc != 0:
            raise ValueError("oracle rejected its arguments")
        return H

    def swiglu_at(self, X, Wg, Wu, rows, cols) -> np.ndarray:
        """SwiGLU at the positions (rows[t], cols[t])."""
        M, K = X.shape
        N = Wg.shape[0]
        X = self._bits(X, (M, K))
        Wg = self._bits(Wg, (N, K))
        Wu = self._bits(Wu, (N, K))
        rows = np.ascontiguousarray(rows, dtype=np.int64)
        cols = np.ascontiguousarray(cols, dtype=np.int64)
        if rows.shape != cols.shape or rows.ndim != 1:
            raise ValueError("rows and cols must be 1-D and of equal length")
        out = np.empty(rows.shape[0], dtype=np.float64)
        rc = self.lib.ka_oracle_swiglu_at(M, N, K, X.ctypes.data, Wg.ctypes.data, Wu.ctypes.data,
                                          rows.shape[0], rows.ctypes.data, cols.ctypes.data,
                                          out.ctypes.data)
        if rc != 0:
            raise ValueError("oracle rejected its arguments")
        return out

    # ---- INT8 with dequantisation scales ------------------------------------
    @staticmethod
    def _i8(a, shape, what):
        a = np.ascontiguousarray(a)
        if a.dtype != np.int8:
            raise TypeError(f"{what}: expected int8")
        if a.shape != shape:
            raise ValueError(f"{what}: expected shape {shape}, got {a.shape}")
        return a

    @staticmethod
    def _f32(a, n, what):
        a = np.ascontiguousarray(a)
        if a.dtype != np.float32 or a.shape != (n,):
            raise ValueError(f"{what}: expected float32 of shape ({n},)")
        return a

    @staticmethod
    def _positions(rows, cols):
        rows = np.ascontiguousarray(rows, dtype=np.int64)
        cols = np.ascontiguousarray(cols, dtype=np.int64)
        if rows.shape != cols.shape or rows.ndim != 1:
            raise ValueError("rows and cols must be 1-D and of equal length")
        return rows, cols

    def i8_dot(self, qX, qW) -> np.ndarray:
        """A = qX qW^T as exact int64 sums."""
        M, K = qX.shape
        N = qW.shape[0]
        qX, qW = self._i8(qX, (M, K), "qX"), self._i8(qW, (N, K), "qW")
        A = np.empty((M, N), dtype=np.int64)
        if self.lib.ka_oracle_i8_dot(M, N, K, qX.ctypes.data, qW.ctypes.data, A.ctypes.data) != 0:
            raise ValueError("oracle rejected its arguments")
        return A

    def _i8_args(self, qX, sx, qW, sw, R):
        M, K = qX.shape
        N = qW.shape[0]
        qX, qW = self._i8(qX, (M, K), "qX"), self._i8(qW, (N, K), "qW")
        sx, sw = self._f32(sx, M, "sx"), self._f32(sw, N, "sw")
        Rp = None
        if R is not None:
            R = self._bits(R, (M, N))
            Rp = R.ctypes.data
        return (M, N, K, qX.ctypes.data, sx.ctypes.data, qW.ctypes.data, sw.ctypes.data, Rp), (qX, sx, qW, sw, R)

    def i8_linear(self, qX, sx, qW, sw, R=None) -> np.ndarray:
        """Y = sx[i] sw[j] (qX qW^T)[i,j] (+ R) in float64."""
        args, keep = self._i8_args(qX, sx, qW, sw, R)
        Y = np.empty((args[0], args[1]), dtype=np.float64)
        if self.lib.ka_oracle_i8_linear(*args, Y.ctypes.data) != 0:
            raise ValueError("oracle rejected its arguments")
        del keep
        return Y

    def i8_linear_at(self, qX, sx, qW, sw, R, rows, cols) -> np.ndarray:
        args, keep = self._i8_args(qX, sx, qW, sw, R)
        rows, cols = self._positions(rows, cols)
        out = np.empty(rows.shape[0], dtype=np.float64)
        if self.lib.ka_oracle_i8_linear_at(*args, rows.shape[0], rows.ctypes.data, cols.ctypes.data,
                                           out.ctypes.data) != 0:
            raise ValueError("oracle rejected its arguments")
        del keep
        return out

    def _i8_glu_args(self, qX, sx, qWg, swg, qWu, swu):
        M, K = qX.shape
        N = qWg.shape[0]
        qX = self._i8(qX, (M, K), "qX")
        qWg, qWu = self._i8(qWg, (N, K), "qWg"), self._i8(qWu, (N, K), "qWu")
        sx = self._f32(sx, M, "sx")
        swg, swu = self._f32(swg, N, "swg"), self._f32(swu, N, "swu")
        keep = (qX, sx, qWg, swg, qWu, swu)
        return (M, N, K) + tuple(a.ctypes.data for a in keep), keep

    def i8_swiglu(self, qX, sx, qWg, swg, qWu, swu) -> np.ndarray:
        """H = silu(sx swg (qX qWg^T)) * (sx swu (qX qWu^T)) in float64."""
        args, keep = self._i8_glu_args(qX, sx, qWg, swg, qWu, swu)
        H = np.empty((args[0], args[1]), dtype=np.float64)
        if self.lib.ka_oracle_i8_swiglu(*args, H.ctypes.data) != 0:
            raise ValueError("oracle rejected its arguments")
        del keep
        return H

    def i8_swiglu_at(self, qX, sx, qWg, swg, qWu, swu, rows, cols) -> np.ndarray:
        args, keep = self._i8_glu_args(qX, sx, qWg, swg, qWu, swu)
        rows, cols = self._positions(rows, cols)
        out = np.empty(rows.shape[0], dtype=np.float64)
        if self.lib.ka_oracle_i8_swiglu_at(*args, rows.shape[0], rows.ctypes.data, cols.ctypes.data,
                                           out.ctypes.data) != 0:
            raise ValueError("oracle rejected its arguments")
        del keep
        return out

    # ---- FP8 (E4M3 bit patterns in numpy.uint8) with dequantisation scales ----
    @staticmethod
    def _u8(a, shape, what):
        a = np.ascontiguousarray(a)
        if a.dtype != np.uint8:
            raise TypeError(f"{what}: expected E4M3 bit patterns (numpy.uint8)")
        if a.shape != shape:
            raise ValueError(f"{what}: expected shape {shape}, got {a.shape}")
        return a

    def fp8_decode(self, bits) -> np.ndarray:
        """E4M3 bit patterns to float64 (exact)."""
        b = np.ascontiguousarray(bits, dtype=np.uint8)
        out = np.empty(b.shape, dtype=np.float64)
        self.lib.ka_oracle_fp8_decode(b.size, b.ctypes.data, out.ctypes.data)
        return out

    def _f8_args(self, qX, sx, qW, sw, R):
        M, K = qX.shape
        N = qW.shape[0]
        qX, qW = self._u8(qX, (M, K), "qX"), self._u8(qW, (N, K), "qW")
        sx, sw = self._f32(sx, M, "sx"), self._f32(sw, N, "sw")
        Rp = None
        if R is not None:
            R = self._bits(R, (M, N))
            Rp = R.ctypes.data
        return (M, N, K, qX.ctypes.data, sx.ctypes.data, qW.ctypes.data, sw.ctypes.data, Rp), (qX, sx, qW, sw, R)

    def f8_linear(self, qX, sx, qW, sw, R=None) -> np.ndarray:
        """Y = sx[i] sw[j] sum_k x8(qX) x8(qW) (+ R) in float64."""
        args, keep = self._f8_args(qX, sx, qW, sw, R)
        Y = np.empty((args[0], args[1]), dtype=np.float64)
        if self.lib.ka_oracle_f8_linear(*args, Y.ctypes.data) != 0:
            raise ValueError("oracle rejected its arguments")
        del keep
        return Y

    def f8_linear_at(self, qX, sx, qW, sw, R, rows, cols) -> np.ndarray:
        args, keep = self._f8_args(qX, sx, qW, sw, R)
        rows, cols = self._positions(rows, cols)
        out = np.empty(rows.shape[0], dtype=np.float64)
        if self.lib.ka_oracle_f8_linear_at(*args, rows.shape[0], rows.ctypes.data, cols.ctypes.data,
                                           out.ctypes.data) != 0:
            raise ValueError("oracle rejected its arguments")
        del keep
        return out

    def _f8_glu_args(self, qX, sx, qWg, swg, qWu, swu):
        M, K = qX.shape
        N = qWg.shape[0]
        qX = self._u8(qX, (M, K), "qX")
        qWg, qWu = self._u8(qWg, (N, K), "qWg"), self._u8(qWu, (N, K), "qWu")
        sx = self._f32(sx, M, "sx")
        swg, swu = self._f32(swg, N, "swg"), self._f32(swu, N, "swu")
        keep = (qX, sx, qWg, swg, qWu, swu)
        return (M, N, K) + tuple(a.ctypes.data for a in keep), keep

    def f8_swiglu(self, qX, sx, qWg, swg, qWu, swu) -> np.ndarray:
        args, keep = self._f8_glu_args(qX, sx, qWg, swg, qWu, swu)
        H = np.empty((args[0], args[1]), dtype=np.float64)
        if self.lib.ka_oracle_f8_swiglu(*args, H.ctypes.data) != 0:
            raise ValueError("oracle rejected its arguments")
        del keep
        return H

    def f8_swiglu_at(self, qX, sx, qWg, swg, qWu, swu, rows, cols) -> np.ndarray:
        args, keep = self._f8_glu_args(qX, sx, qWg, swg, qWu, swu)
        rows, cols = self._positions(rows, cols)
        out = np.empty(rows.shape[0], dtype=np.float64)
        if self.lib.ka_oracle_f8_swiglu_at(*args, rows.shape[0], rows.ctypes.data, cols.ctypes.data,
                                           out.ctypes.data) != 0:
            raise ValueError("oracle rejected its arguments")
        del keep
        return out

    # ---- grouped (per-expert) forms ------------------------------------------
    def _grouped_args(self, X, W, W2, counts):
        E, Mpad, K = X.shape
        N = W.shape[1]
        X = self._bits(X, (E, Mpad, K))
        W = self._bits(W, (E, N, K))
        if W2 is not None:
            W2 = self._bits(W2, (E, N, K))
        cp = None
        if counts is not None:
            counts = np.ascontiguousarray(counts)
            if counts.dtype != np.int32 or counts.shape != (E,):
                raise ValueError("counts: expected int32 of shape (E,)")
            cp = counts.ctypes.data
        return (E, Mpad, N, K), (X, W, W2, counts), cp

    def grouped_linear(self, X, W, counts=None, out=None) -> np.ndarray:
        """Y[e,i,:] = X[e,i,:] W[e]^T for the valid rows i < counts[e] of each
        expert (float64); the other rows of `out` (default: NaN) are untouched."""
        (E, Mpad, N, K), keep, cp = self._grouped_args(X, W, None, counts)
        Y = np.full((E, Mpad, N), np.nan) if out is None else out
        if Y.dtype != np.float64 or Y.shape != (E, Mpad, N) or not Y.flags.c_contiguous:
            raise ValueError("out: expected a contiguous float64 array of shape (E, M_pad, N)")
        if self.lib.ka_oracle_grouped_linear(E, Mpad, N, K, keep[0].ctypes.data, keep[1].ctypes.data, cp,
                                             Y.ctypes.data) != 0:
            raise ValueError("oracle rejected its arguments")
        return Y

    def grouped_swiglu(self, X, Wg, Wu, counts=None, out=None) -> np.ndarray:
        """H[e,i,:] = silu(X[e,i,:] Wg[e]^T) * (X[e,i,:] Wu[e]^T) for the valid rows."""
        (E, Mpad, N, K), keep, cp = self._grouped_args(X, Wg, Wu, counts)
        H = np.full((E, Mpad, N), np.nan) if out is None else out
        if H.dtype != np.float64 or H.shape != (E, Mpad, N) or not H.flags.c_contiguous:
            raise ValueError("out: expected a contiguous float64 array of shape (E, M_pad, N)")
        if self.lib.ka_oracle_grouped_swiglu(E, Mpad, N, K, keep[0].ctypes.data, keep[1].ctypes.data,
                                             keep[2].ctypes.data, cp, H.ctypes.data) != 0:
            raise ValueError("oracle rejected its arguments")
        return H

    def grouped_at(self, X, W, W2, counts, groups, rows, cols) -> np.ndarray:
        """Either grouped form (SwiGLU when W2 is given) at (groups[t], rows[t], cols[t])."""
        (E, Mpad, N, K), keep, cp = self._grouped_args(X, W, W2, counts)
        groups = np.ascontiguousarray(groups, dtype=np.int64)
        rows, cols = self._positions(rows, cols)
        if groups.shape != rows.shape:
            raise ValueError("groups, rows and cols must have equal length")
        out = np.empty(rows.shape[0], dtype=np.float64)
        w2 = keep[2].ctypes.data if keep[2] is not None else None
        if self.lib.ka_oracle_grouped_at(E, Mpad, N, K, keep[0].ctypes.data, keep[1].ctypes.data, w2, cp,
                                         int(W2 is not None), rows.shape[0], groups.ctypes.data, rows.ctypes.data,
                                         cols.ctypes.data, out.ctypes.data) != 0:
            raise ValueError("oracle rejected its arguments")
        return out

    def threads(self) -> int:
        """OpenMP threads the oracle's loops use."""
        return int(self.lib.ka_oracle_threads())

    def set_threads(self, n: int) -> None:
        """Threads the oracle's loops use from now on (n >= 1)."""
        self.lib.ka_oracle_set_threads(int(n))

    def round_bf16(self, values) -> np.ndarray:
        """Round float64 values to bf16 bit patterns (nearest, ties to even)."""
        v = np.ascontiguousarray(values, dtype=np.float64)
        out = np.empty(v.shape, dtype=np.uint16)
        self.lib.ka_oracle_round_bf16(v.size, v.ctypes.data, out.ctypes.data)
        return out


_default: Oracle | None = None


def default() -> Oracle:
    """The oracle built in-tree (built on first use if it is missing)."""
    global _default
    if _default is None:
        if not os.path.exists(LIBRARY):
            build()
        _default = Oracle(LIBRARY)
    return _default


def bf16_bits_to_f64(bits) -> np.ndarray:
    """Exact widening of bf16 bit patterns to float64 (for the test checks)."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    with np.errstate(invalid="ignore"):          # signalling-NaN patterns
        return b.view(np.float32).astype(np.float64)
