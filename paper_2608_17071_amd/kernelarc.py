"""Python binding of the HIP library ``libkernelarc.so`` (ctypes).

Only argument marshalling happens here: shapes and dtypes are checked,
leading dimensions of X are flattened into M (the token count, Alg. 3), and
the raw device pointers plus torch's current HIP stream are handed to the
C ABI declared in ``include/kernelarc.h``.  Every arithmetic step runs in the
library's kernels; there is no other backend, and importing this module
raises if the library has not been built.

The C entry points are also exposed under their own names
(``kernelarc_gemm_bf16_residual`` and so on) for callers that manage raw
pointers themselves.
"""
from __future__ import annotations

import ctypes
import os

import torch

LIBRARY = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libkernelarc.so")

OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_LAUNCH = 0, 1, 2, 3

if not os.path.exists(LIBRARY):
    raise ImportError(
        f"{LIBRARY} is missing: build it with `python -m paper_2608_17071_amd.build` "
        "(there is no fallback implementation)")

_lib = ctypes.CDLL(LIBRARY)
_I64 = ctypes.c_int64
_P = ctypes.c_void_p

_SIGS = {
    "kernelarc_gemm_bf16_residual": (ctypes.c_int, [_I64, _I64, _I64, _P, _P, _P, _P, _P]),
    "kernelarc_gemm_bf16": (ctypes.c_int, [_I64, _I64, _I64, _P, _P, _P, _P]),
    "kernelarc_gemm_bf16_residual_noalloc": (ctypes.c_int, [_I64, _I64, _I64, _P, _P, _P, _P, _P]),
    "kernelarc_gemm_bf16_with_plan": (ctypes.c_int, [ctypes.c_int, _I64, _I64, _I64, _P, _P, _P, _P, _P]),
    "kernelarc_plan_count": (ctypes.c_int, []),
    "kernelarc_plan_name": (ctypes.c_int, [_I64, _I64, _I64, ctypes.c_int, ctypes.c_char_p, ctypes.c_size_t]),
    "kernelarc_plan_label": (ctypes.c_char_p, [ctypes.c_int]),
    "kernelarc_plan_supports": (ctypes.c_int, [ctypes.c_int, _I64, _I64, _I64, ctypes.c_int]),
    "kernelarc_select_plan": (ctypes.c_int, [_I64, _I64, _I64, ctypes.c_int]),
    "kernelarc_plan_uses_workspace": (ctypes.c_int, [ctypes.c_int, _I64, _I64, _I64]),
    "kernelarc_gemm_bf16_ex": (ctypes.c_int, [_I64, _I64, _I64, ctypes.c_float, _P, _I64, _P, _I64,
                                              ctypes.c_float, _P, _I64, _P, _P, _I64, _P]),
    "kernelarc_gemm_bf16_ex_with_plan": (ctypes.c_int, [ctypes.c_int, _I64, _I64, _I64, ctypes.c_float, _P, _I64,
                                                        _P, _I64, ctypes.c_float, _P, _I64, _P, _P, _I64, _P]),
    "kernelarc_select_plan_ex": (ctypes.c_int, [_I64, _I64, _I64, ctypes.c_int, _I64, _I64, _I64, _I64,
                                                ctypes.c_float, ctypes.c_float, ctypes.c_int]),
    "kernelarc_swiglu_bf16": (ctypes.c_int, [_I64, _I64, _I64, _P, _P, _P, _P, _P]),
    "kernelarc_swiglu_bf16_with_plan": (ctypes.c_int, [ctypes.c_int, _I64, _I64, _I64, _P, _P, _P, _P, _P]),
    "kernelarc_select_plan_swiglu": (ctypes.c_int, [_I64, _I64, _I64]),
    "kernelarc_plan_supports_swiglu": (ctypes.c_int, [ctypes.c_int, _I64, _I64, _I64]),
    "kernelarc_gemm_i8": (ctypes.c_int, [_I64, _I64, _I64, _P, _P, _P, _P, _P, _P, _P]),
    "kernelarc_gemm_i8_with_plan": (ctypes.c_int, [ctypes.c_int, _I64, _I64, _I64, _P, _P, _P, _P, _P, _P, _P]),
    "kernelarc_swiglu_i8": (ctypes.c_int, [_I64, _I64, _I64, _P, _P, _P, _P, _P, _P, _P, _P]),
    "kernelarc_swiglu_i8_with_plan": (ctypes.c_int, [ctypes.c_int, _I64, _I64, _I64, _P, _P, _P, _P, _P, _P, _P,
                                                     _P]),
    "kernelarc_select_plan_i8": (ctypes.c_int, [_I64, _I64, _I64, ctypes.c_int]),
    "kernelarc_plan_supports_i8": (ctypes.c_int, [ctypes.c_int, _I64, _I64, _I64, ctypes.c_int]),
    "kernelarc_gemm_bf16_grouped": (ctypes.c_int, [_I64, _I64, _I64, _I64, _P, _P, _P, _P, _P]),
    "kernelarc_gemm_bf16_grouped_with_plan": (ctypes.c_int, [ctypes.c_int, _I64, _I64, _I64, _I64, _P, _P, _P, _P,
                                                             _P]),
    "kernelarc_swiglu_bf16_grouped": (ctypes.c_int, [_I64, _I64, _I64, _I64, _P, _P, _P, _P, _P, _P]),
    "kernelarc_swiglu_bf16_grouped_with_plan": (ctypes.c_int, [ctypes.c_int, _I64, _I64, _I64, _I64, _P, _P, _P, _P,
                                                               _P, _P]),
    "kernelarc_select_plan_grouped": (ctypes.c_int, [_I64, _I64, _I64, _I64, ctypes.c_int]),
    "kernelarc_plan_supports_grouped": (ctypes.c_int, [ctypes.c_int, _I64, _I64, _I64, _I64, ctypes.c_int]),
    "kernelarc_gemm_f8": (ctypes.c_int, [_I64, _I64, _I64, _P, _P, _P, _P, _P, _P, _P]),
    "kernelarc_gemm_f8_with_plan": (ctypes.c_int, [ctypes.c_int, _I64, _I64, _I64, _P, _P, _P, _P, _P, _P, _P]),
    "kernelarc_swiglu_f8": (ctypes.c_int, [_I64, _I64, _I64, _P, _P, _P, _P, _P, _P, _P, _P]),
    "kernelarc_swiglu_f8_with_plan": (ctypes.c_int, [ctypes.c_int, _I64, _I64, _I64, _P, _P, _P, _P, _P, _P, _P,
                                                     _P]),
    "kernelarc_select_plan_f8": (ctypes.c_int, [_I64, _I64, _I64, ctypes.c_int]),
    "kernelarc_plan_supports_f8": (ctypes.c_int, [ctypes.c_int, _I64, _I64, _I64, ctypes.c_int]),
    "kernelarc_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "kernelarc_last_error": (ctypes.c_char_p, []),
}

for _name, (_res, _args) in _SIGS.items():
    _fn = getattr(_lib, _name)
    _fn.restype = _res
    _fn.argtypes = _args
    globals()[_name] = _fn

EXPORTED = tuple(_SIGS)


class KernelArcError(RuntimeError):
    def __init__(self, status: int, where: str):
        detail = _lib.kernelarc_last_error().decode(errors="replace")
        msg = _lib.kernelarc_status_string(status).decode()
        super().__init__(f"{where}: {msg} ({detail})" if detail else f"{where}: {msg}")
        self.status = status


def _check(status: int, where: str) -> None:
    if status != OK:
        raise KernelArcError(status, where)


def plan_count() -> int:
    return _lib.kernelarc_plan_count()


def plan_name(plan: int) -> str | None:
    """Name of plan id `plan` (None for an unknown id)."""
    n = _lib.kernelarc_plan_label(plan)
    return n.decode() if n is not None else None


def plan_name_for(M: int, N: int, K: int, residual: bool = True) -> str:
    """Name of the plan the library runs for this shape (kernelarc_plan_name)."""
    buf = ctypes.create_string_buffer(64)
    _check(_lib.kernelarc_plan_name(M, N, K, int(residual), buf, len(buf)), "kernelarc_plan_name")
    return buf.value.decode()


def plan_names() -> list[str]:
    return [plan_name(i) for i in range(plan_count())]


def select_plan(M: int, N: int, K: int, residual: bool = True) -> int:
    return _lib.kernelarc_select_plan(M, N, K, int(residual))


def plan_supports(plan: int, M: int, N: int, K: int, residual: bool = True) -> bool:
    return _lib.kernelarc_plan_supports(plan, M, N, K, int(residual)) == 1


def _stream_handle(stream=None) -> int:
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def _operands(x: torch.Tensor, w: torch.Tensor, r: torch.Tensor | None, out: torch.Tensor | None):
    if w.dim() != 2:
        raise ValueError("w must be [N, K]")
    N, K = w.shape
    if x.shape[-1] != K:
        raise ValueError(f"x's last dimension {x.shape[-1]} does not match K={K}")
    lead = tuple(x.shape[:-1])
    M = 1
    for d in lead:
        M *= d
    for name, t in (("x", x), ("w", w), ("r", r), ("out", out)):
        if t is None:
            continue
        if t.dtype != torch.bfloat16:
            raise TypeError(f"{name} must be bfloat16")
        if not t.is_cuda:
            raise ValueError(f"{name} must be a GPU tensor")
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
        if t.device != x.device:
            raise ValueError(f"{name} is on {t.device}, x on {x.device}")
    if r is not None and tuple(r.shape) != lead + (N,):
        raise ValueError(f"r must have shape {lead + (N,)}")
    if out is None:
        out = torch.empty(lead + (N,), dtype=torch.bfloat16, device=x.device)
    elif tuple(out.shape) != lead + (N,):
        raise ValueError(f"out must have shape {lead + (N,)}")
    return M, N, K, out


def gemm_bf16_residual(x, w, r, out=None, stream=None):
    """Y = X W^T + R (out may be r itself for the in-place form)."""
    M, N, K, out = _operands(x, w, r, out)
    with torch.cuda.device(x.device):
        st = _lib.kernelarc_gemm_bf16_residual(M, N, K, x.data_ptr(), w.data_ptr(), r.data_ptr(),
                                               out.data_ptr(), _stream_handle(stream))
    _check(st, "kernelarc_gemm_bf16_residual")
    return out


def gemm_bf16(x, w, out=None, stream=None):
    """Y = X W^T."""
    M, N, K, out = _operands(x, w, None, out)
    with torch.cuda.device(x.device):
        st = _lib.kernelarc_gemm_bf16(M, N, K, x.data_ptr(), w.data_ptr(), out.data_ptr(),
                                      _stream_handle(stream))
    _check(st, "kernelarc_gemm_bf16")
    return out


def gemm_bf16_residual_noalloc(x, w, r=None, out=None, stream=None):
    """Y = X W^T (+ R) with the split-K partials in the library's static
    scratch: the call allocates no device memory (``out`` must then be given
    by callers that cannot allocate)."""
    M, N, K, out = _operands(x, w, r, out)
    with torch.cuda.device(x.device):
        st = _lib.kernelarc_gemm_bf16_residual_noalloc(M, N, K, x.data_ptr(), w.data_ptr(),
                                                       r.data_ptr() if r is not None else None,
                                                       out.data_ptr(), _stream_handle(stream))
    _check(st, "kernelarc_gemm_bf16_residual_noalloc")
    return out


def gemm_bf16_with_plan(plan, x, w, r=None, out=None, stream=None):
    """Y = X W^T (+ R) with an explicit plan id."""
    M, N, K, out = _operands(x, w, r, out)
    with torch.cuda.device(x.device):
        st = _lib.kernelarc_gemm_bf16_with_plan(plan, M, N, K, x.data_ptr(), w.data_ptr(),
                                                r.data_ptr() if r is not None else None,
                                                out.data_ptr(), _stream_handle(stream))
    _check(st, f"kernelarc_gemm_bf16_with_plan({plan_name(plan)})")
    return out


def _rows(t: torch.Tensor, name: str, rows: int, cols: int) -> int:
    """Leading dimension (elements) of a 2-D bf16 GPU view with unit column stride."""
    if t.dtype != torch.bfloat16:
        raise TypeError(f"{name} must be bfloat16")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if t.dim() != 2 or tuple(t.shape) != (rows, cols):
        raise ValueError(f"{name} must have shape {(rows, cols)}, got {tuple(t.shape)}")
    if rows > 0 and cols > 1 and t.stride(1) != 1:
        raise ValueError(f"{name} must have unit stride along its last dimension")
    return t.stride(0) if rows > 1 else max(cols, 1)


def gemm_bf16_ex(x, w, c=None, bias=None, alpha=1.0, beta=1.0, out=None, stream=None, plan=None):
    """Y = alpha X W^T + beta C + bias with row-strided 2-D operands.

    x [M, K], w [N, K], c and out [M, N] may be row-strided views (unit
    stride along the last dimension); bias is [N] or None; c is not read
    when beta == 0.  ``out`` may be ``c`` itself (same view).
    """
    if x.dim() != 2 or w.dim() != 2:
        raise ValueError("x must be [M, K] and w [N, K]")
    M, K = x.shape
    N = w.shape[0]
    ldx = _rows(x, "x", M, K)
    ldw = _rows(w, "w", N, K)
    if out is None:
        out = torch.empty((M, N), dtype=torch.bfloat16, device=x.device)
    ldy = _rows(out, "out", M, N)
    ldc = _rows(c, "c", M, N) if c is not None else max(N, 1)
    if bias is not None:
        if bias.dtype != torch.bfloat16 or not bias.is_cuda or tuple(bias.shape) != (N,) or not bias.is_contiguous():
            raise ValueError(f"bias must be a contiguous bfloat16 GPU tensor of shape {(N,)}")
    for t in (w, c, bias, out):
        if t is not None and t.device != x.device:
            raise ValueError(f"operands on different devices ({t.device} vs {x.device})")
    args = (M, N, K, float(alpha), x.data_ptr(), ldx, w.data_ptr(), ldw, float(beta),
            c.data_ptr() if c is not None else None, ldc,
            bias.data_ptr() if bias is not None else None, out.data_ptr(), ldy)
    with torch.cuda.device(x.device):
        if plan is None:
            st = _lib.kernelarc_gemm_bf16_ex(*args, _stream_handle(stream))
        else:
            st = _lib.kernelarc_gemm_bf16_ex_with_plan(plan, *args, _stream_handle(stream))
    _check(st, "kernelarc_gemm_bf16_ex" if plan is None else f"kernelarc_gemm_bf16_ex_with_plan({plan_name(plan)})")
    return out


def select_plan_ex(M, N, K, has_c, ldx, ldw, ldc, ldy, alpha, beta, has_bias) -> int:
    """The plan the general form would run for these strides and scalars."""
    return _lib.kernelarc_select_plan_ex(M, N, K, int(has_c), ldx, ldw, ldc, ldy, float(alpha), float(beta),
                                         int(has_bias))


def swiglu_bf16(x, wg, wu, out=None, stream=None, plan=None):
    """H = silu(X Wg^T) * (X Wu^T) (the gated MLP input projection).

    x is [..., K] (leading dimensions flattened into M), wg and wu are
    [N, K]; the result is [..., N].  All contiguous bfloat16 GPU tensors.
    """
    if wu.dim() != 2 or tuple(wu.shape) != tuple(wg.shape):
        raise ValueError("wg and wu must both be [N, K]")
    M, N, K, out = _operands(x, wg, None, out)
    for name, t in (("wu", wu),):
        if t.dtype != torch.bfloat16 or not t.is_cuda or not t.is_contiguous() or t.device != x.device:
            raise ValueError(f"{name} must be a contiguous bfloat16 tensor on {x.device}")
    args = (M, N, K, x.data_ptr(), wg.data_ptr(), wu.data_ptr(), out.data_ptr(), _stream_handle(stream))
    with torch.cuda.device(x.device):
        if plan is None:
            st = _lib.kernelarc_swiglu_bf16(*args)
        else:
            st = _lib.kernelarc_swiglu_bf16_with_plan(plan, *args)
    _check(st, "kernelarc_swiglu_bf16" if plan is None else f"kernelarc_swiglu_bf16_with_plan({plan_name(plan)})")
    return out


def select_plan_swiglu(M: int, N: int, K: int) -> int:
    return _lib.kernelarc_select_plan_swiglu(M, N, K)


def plan_supports_swiglu(plan: int, M: int, N: int, K: int) -> bool:
    return _lib.kernelarc_plan_supports_swiglu(plan, M, N, K) == 1


def _i8_operand(t, name, shape, device, dtype=torch.int8):
    if t.dtype != dtype or not t.is_cuda or not t.is_contiguous() or tuple(t.shape) != shape:
        raise ValueError(f"{name} must be a contiguous {dtype} GPU tensor of shape {shape}")
    if t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")


def _scales(t, name, n, device):
    if t.dtype != torch.float32 or not t.is_cuda or not t.is_contiguous() or tuple(t.shape) != (n,):
        raise ValueError(f"{name} must be a contiguous float32 GPU tensor of shape ({n},)")
    if t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")


def _q8_call(fmt, swiglu, qx, sx, ws, r, out, stream, plan):
    """INT8 (fmt "i8", torch.int8 operands) or FP8 (fmt "f8", torch.float8_e4m3fn
    operands) call; ws = ((qw, sw),) or ((qwg, swg), (qwu, swu))."""
    dtype = torch.int8 if fmt == "i8" else torch.float8_e4m3fn
    if qx.dim() != 2 or any(w.dim() != 2 or w.shape[1] != qx.shape[1] for w, _ in ws):
        raise ValueError("qx must be [M, K] and the weights [N, K]")
    M, K = qx.shape
    N = ws[0][0].shape[0]
    dev = qx.device
    _i8_operand(qx, "qx", (M, K), dev, dtype)
    _scales(sx, "sx", M, dev)
    for i, (w, s) in enumerate(ws):
        _i8_operand(w, f"weight {i}", (N, K), dev, dtype)
        _scales(s, f"scale {i}", N, dev)
    for name, t in (("r", r), ("out", out)):
        if t is not None and (t.dtype != torch.bfloat16 or not t.is_cuda or not t.is_contiguous()
                              or tuple(t.shape) != (M, N) or t.device != dev):
            raise ValueError(f"{name} must be a contiguous bfloat16 GPU tensor of shape {(M, N)}")
    if out is None:
        out = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
    wargs = []
    for w, s in ws:
        wargs += [w.data_ptr(), s.data_ptr()]
    if swiglu:
        args = (M, N, K, qx.data_ptr(), sx.data_ptr(), *wargs, out.data_ptr(), _stream_handle(stream))
    else:
        args = (M, N, K, qx.data_ptr(), sx.data_ptr(), *wargs, r.data_ptr() if r is not None else None,
                out.data_ptr(), _stream_handle(stream))
    name = f"kernelarc_{'swiglu' if swiglu else 'gemm'}_{fmt}"
    with torch.cuda.device(dev):
        st = getattr(_lib, name)(*args) if plan is None else getattr(_lib, name + "_with_plan")(plan, *args)
    _check(st, name if plan is None else f"{name}_with_plan({plan_name(plan)})")
    return out


def gemm_f8(qx, sx, qw, sw, r=None, out=None, stream=None, plan=None):
    """Y = bf16(sx[i] sw[j] sum_k qX qW (+ R)) with torch.float8_e4m3fn qx [M, K],
    qw [N, K] and float32 scales sx [M], sw [N]; out may be r (in place)."""
    return _q8_call("f8", False, qx, sx, ((qw, sw),), r, out, stream, plan)


def swiglu_f8(qx, sx, qwg, swg, qwu, swu, out=None, stream=None, plan=None):
    """H = bf16(silu(sx swg (qX qWg^T)) * (sx swu (qX qWu^T))) with E4M3 operands."""
    return _q8_call("f8", True, qx, sx, ((qwg, swg), (qwu, swu)), None, out, stream, plan)


def select_plan_f8(M: int, N: int, K: int, swiglu: bool = False) -> int:
    return _lib.kernelarc_select_plan_f8(M, N, K, int(swiglu))


def plan_supports_f8(plan: int, M: int, N: int, K: int, swiglu: bool = False) -> bool:
    return _lib.kernelarc_plan_supports_f8(plan, M, N, K, int(swiglu)) == 1


def gemm_i8(qx, sx, qw, sw, r=None, out=None, stream=None, plan=None):
    """Y = bf16(sx[i] sw[j] (qX qW^T)[i,j] (+ R)): int8 qx [M, K] and qw [N, K],
    float32 per-row scales sx [M] and per-output-channel scales sw [N],
    optional bf16 residual r [M, N]; out may be r (in place)."""
    if qx.dim() != 2 or qw.dim() != 2 or qx.shape[1] != qw.shape[1]:
        raise ValueError("qx must be [M, K] and qw [N, K]")
    M, K = qx.shape
    N = qw.shape[0]
    dev = qx.device
    _i8_operand(qx, "qx", (M, K), dev)
    _i8_operand(qw, "qw", (N, K), dev)
    _scales(sx, "sx", M, dev)
    _scales(sw, "sw", N, dev)
    for name, t in (("r", r), ("out", out)):
        if t is not None and (t.dtype != torch.bfloat16 or not t.is_cuda or not t.is_contiguous()
                              or tuple(t.shape) != (M, N) or t.device != dev):
            raise ValueError(f"{name} must be a contiguous bfloat16 GPU tensor of shape {(M, N)}")
    if out is None:
        out = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
    args = (M, N, K, qx.data_ptr(), sx.data_ptr(), qw.data_ptr(), sw.data_ptr(),
            r.data_ptr() if r is not None else None, out.data_ptr(), _stream_handle(stream))
    with torch.cuda.device(dev):
        st = _lib.kernelarc_gemm_i8(*args) if plan is None else _lib.kernelarc_gemm_i8_with_plan(plan, *args)
    _check(st, "kernelarc_gemm_i8" if plan is None else f"kernelarc_gemm_i8_with_plan({plan_name(plan)})")
    return out


def swiglu_i8(qx, sx, qwg, swg, qwu, swu, out=None, stream=None, plan=None):
    """H = bf16(silu(sx swg (qX qWg^T)) * (sx swu (qX qWu^T))) with int8 operands
    and float32 scales (per row of qx, per output channel of each weight)."""
    if qx.dim() != 2 or qwg.dim() != 2 or qx.shape[1] != qwg.shape[1]:
        raise ValueError("qx must be [M, K] and qwg, qwu [N, K]")
    M, K = qx.shape
    N = qwg.shape[0]
    dev = qx.device
    _i8_operand(qx, "qx", (M, K), dev)
    _i8_operand(qwg, "qwg", (N, K), dev)
    _i8_operand(qwu, "qwu", (N, K), dev)
    _scales(sx, "sx", M, dev)
    _scales(swg, "swg", N, dev)
    _scales(swu, "swu", N, dev)
    if out is None:
        out = torch.empty((M, N), dtype=torch.bfloat16, device=dev)
    elif out.dtype != torch.bfloat16 or not out.is_contiguous() or tuple(out.shape) != (M, N) or out.device != dev:
        raise ValueError(f"out must be a contiguous bfloat16 GPU tensor of shape {(M, N)}")
    args = (M, N, K, qx.data_ptr(), sx.data_ptr(), qwg.data_ptr(), swg.data_ptr(), qwu.data_ptr(), swu.data_ptr(),
            out.data_ptr(), _stream_handle(stream))
    with torch.cuda.device(dev):
        st = _lib.kernelarc_swiglu_i8(*args) if plan is None else _lib.kernelarc_swiglu_i8_with_plan(plan, *args)
    _check(st, "kernelarc_swiglu_i8" if plan is None else f"kernelarc_swiglu_i8_with_plan({plan_name(plan)})")
    return out


def select_plan_i8(M: int, N: int, K: int, swiglu: bool = False) -> int:
    return _lib.kernelarc_select_plan_i8(M, N, K, int(swiglu))


def plan_supports_i8(plan: int, M: int, N: int, K: int, swiglu: bool = False) -> bool:
    return _lib.kernelarc_plan_supports_i8(plan, M, N, K, int(swiglu)) == 1


def _grouped_operand(t, name, shape, device):
    if t.dtype != torch.bfloat16 or not t.is_cuda or not t.is_contiguous() or tuple(t.shape) != shape:
        raise ValueError(f"{name} must be a contiguous bfloat16 GPU tensor of shape {shape}")
    if t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")


def _grouped_call(fn, fn_plan, what, x, ws, counts, out, stream, plan):
    if x.dim() != 3 or any(w.dim() != 3 for w in ws):
        raise ValueError("x must be [G, M_pad, K] and the weights [G, N, K]")
    G, Mpad, K = x.shape
    N = ws[0].shape[1]
    dev = x.device
    _grouped_operand(x, "x", (G, Mpad, K), dev)
    for i, w in enumerate(ws):
        _grouped_operand(w, f"weight {i}", (G, N, K), dev)
    if counts is not None and (counts.dtype != torch.int32 or not counts.is_cuda or not counts.is_contiguous()
                               or tuple(counts.shape) != (G,) or counts.device != dev):
        raise ValueError(f"counts must be a contiguous int32 GPU tensor of shape ({G},)")
    if out is None:
        out = torch.empty((G, Mpad, N), dtype=torch.bfloat16, device=dev)
    else:
        _grouped_operand(out, "out", (G, Mpad, N), dev)
    args = (G, Mpad, N, K, x.data_ptr(), *[w.data_ptr() for w in ws],
            counts.data_ptr() if counts is not None else None, out.data_ptr(), _stream_handle(stream))
    with torch.cuda.device(dev):
        st = fn(*args) if plan is None else fn_plan(plan, *args)
    _check(st, what if plan is None else f"{what}_with_plan({plan_name(plan)})")
    return out


def gemm_bf16_grouped(x, w, counts=None, out=None, stream=None, plan=None):
    """Y[g, i] = X[g, i] W[g]^T for the valid rows i < counts[g] of each group:
    x [G, M_pad, K], w [G, N, K], counts int32 [G] on the device (None: all
    rows); the gap rows of `out` are left untouched."""
    return _grouped_call(_lib.kernelarc_gemm_bf16_grouped, _lib.kernelarc_gemm_bf16_grouped_with_plan,
                         "kernelarc_gemm_bf16_grouped", x, (w,), counts, out, stream, plan)


def swiglu_bf16_grouped(x, wg, wu, counts=None, out=None, stream=None, plan=None):
    """H[g, i] = silu(X[g, i] Wg[g]^T) * (X[g, i] Wu[g]^T) for the valid rows."""
    return _grouped_call(_lib.kernelarc_swiglu_bf16_grouped, _lib.kernelarc_swiglu_bf16_grouped_with_plan,
                         "kernelarc_swiglu_bf16_grouped", x, (wg, wu), counts, out, stream, plan)


def select_plan_grouped(G: int, M_pad: int, N: int, K: int, swiglu: bool = False) -> int:
    return _lib.kernelarc_select_plan_grouped(G, M_pad, N, K, int(swiglu))


def plan_supports_grouped(plan: int, G: int, M_pad: int, N: int, K: int, swiglu: bool = False) -> bool:
    return _lib.kernelarc_plan_supports_grouped(plan, G, M_pad, N, K, int(swiglu)) == 1
