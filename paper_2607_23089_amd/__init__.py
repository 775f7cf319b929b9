"""MI355X (gfx950) row softmax: Python binding of the C ABI in include/rowsm.h.

Every function here only marshals arguments to the shared library
``librowsm.so`` (built by ``paper_2607_23089_amd.build``); every step of the
softmax runs in the library's HIP kernels.  There is no fallback: when the
library is missing or fails to load, the calls raise ``RowsmError``.

Raw entry points (same names and arguments as the C ABI; pointers are ints,
``stream`` a hipStream_t handle as an int, 0 = default stream):

    rowsm_forward(x, y, rows, cols, in_dtype, out_dtype, stream) -> status
    rowsm_forward_noalloc(x, y, rows, cols, in_dtype, out_dtype, stream) -> status
    rowsm_forward_variant(x, y, rows, cols, in_dtype, out_dtype, stream, variant)
    rowsm_forward_config(x, y, rows, cols, in_dtype, out_dtype, stream, cfg)
    rowsm_forward_scaled_causal(x, y, rows, cols, in_dtype, out_dtype, scale,
                                causal_period, causal_offset, stream, cfg)
    rowsm_select(rows, cols, in_dtype, out_dtype) -> variant or status
    rowsm_describe(rows, cols, in_dtype, out_dtype, variant) -> (status, text)
    rowsm_split_wait_failures() -> count (diagnostics of the exchanging forms)
    rowsm_set_split_wait_limit(polls) -> previous limit (test setting)
    rowsm_status_string(status) -> str

Tensor helper: ``softmax(x, out_dtype=None, out=None, ...)`` for torch tensors
on a GPU (marshalling only: pointers, sizes, dtype codes and the current
stream).
"""
from __future__ import annotations

import ctypes
import os

F32, BF16 = 0, 1
AUTO, SMALL, MEDIUM, LARGE = 0, 1, 2, 3
OK, EINVAL, EDTYPE, EHIP = 0, -1, -2, -3
VARIANT_NAMES = {SMALL: "small", MEDIUM: "medium", LARGE: "large"}
OP_SOFTMAX, OP_SCALED_CAUSAL, OP_LOG_SOFTMAX, OP_SOFTMAX_BACKWARD = 0, 1, 2, 3
OP_MOE_GROUP_TOP2 = 4

_PKG = os.path.dirname(os.path.abspath(__file__))
# ROWSM_LIB names another build of the library (the host-logic check build).
LIB_PATH = os.environ.get("ROWSM_LIB") or os.path.join(_PKG, "librowsm.so")

# Symbols declared in include/rowsm.h.
EXPORTS = ("rowsm_forward", "rowsm_forward_noalloc", "rowsm_select", "rowsm_forward_variant",
           "rowsm_forward_config", "rowsm_forward_scaled_causal", "rowsm_log_softmax",
           "rowsm_softmax_backward", "rowsm_moe_group_top2", "rowsm_describe",
           "rowsm_describe_op",
           "rowsm_split_wait_failures", "rowsm_set_split_wait_limit", "rowsm_stream_copy",
           "rowsm_status_string")


class RowsmError(RuntimeError):
    pass


class RowsmConfig(ctypes.Structure):
    """Mirror of ``rowsm_config`` (launch overrides; 0 / packed=-1 = default)."""
    _fields_ = [(name, ctypes.c_int32) for name in (
        "variant", "vw", "lanes_per_row", "rows_per_lane", "waves_per_row",
        "rows_per_block", "packed", "block", "tile_vectors", "blocks_per_cu",
        "split_blocks", "prefetch")]

    def __init__(self, **kw):
        super().__init__()
        self.packed = -1
        for k, v in kw.items():
            if k not in dict(self._fields_):
                raise TypeError(f"unknown rowsm_config field {k!r}")
            setattr(self, k, int(v))


_lib = None


def lib(path: str | None = None) -> ctypes.CDLL:
    """Load librowsm.so (once) and type its entry points."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise RowsmError(f"{p} is missing: build it with "
                         "`python -m paper_2607_23089_amd.build`")
    try:
        h = ctypes.CDLL(p)
    except OSError as e:
        raise RowsmError(f"cannot load {p}: {e}") from e
    vp, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int
    fwd = [vp, vp, i64, i64, i32, i32, vp]
    h.rowsm_forward.argtypes = fwd
    h.rowsm_forward.restype = i32
    h.rowsm_forward_noalloc.argtypes = fwd
    h.rowsm_forward_noalloc.restype = i32
    h.rowsm_forward_variant.argtypes = fwd + [i32]
    h.rowsm_forward_variant.restype = i32
    h.rowsm_forward_config.argtypes = fwd + [ctypes.POINTER(RowsmConfig)]
    h.rowsm_forward_config.restype = i32
    h.rowsm_forward_scaled_causal.argtypes = [vp, vp, i64, i64, i32, i32, ctypes.c_float,
                                              i64, i64, vp, ctypes.POINTER(RowsmConfig)]
    h.rowsm_forward_scaled_causal.restype = i32
    h.rowsm_log_softmax.argtypes = fwd + [ctypes.POINTER(RowsmConfig)]
    h.rowsm_log_softmax.restype = i32
    h.rowsm_softmax_backward.argtypes = [vp, vp, vp, i64, i64, i32, i32, vp,
                                         ctypes.POINTER(RowsmConfig)]
    h.rowsm_softmax_backward.restype = i32
    h.rowsm_moe_group_top2.argtypes = [vp, vp, i64, i64, i64, i32, i32, vp,
                                       ctypes.POINTER(RowsmConfig)]
    h.rowsm_moe_group_top2.restype = i32
    h.rowsm_describe_op.argtypes = [i32, i64, i64, i32, i32, ctypes.POINTER(RowsmConfig),
                                    ctypes.c_char_p, i64]
    h.rowsm_describe_op.restype = i32
    h.rowsm_select.argtypes = [i64, i64, i32, i32]
    h.rowsm_select.restype = i32
    h.rowsm_describe.argtypes = [i64, i64, i32, i32, i32, ctypes.c_char_p, i64]
    h.rowsm_describe.restype = i32
    h.rowsm_stream_copy.argtypes = [vp, vp, i64, i32, i32, vp]
    h.rowsm_stream_copy.restype = i32
    h.rowsm_split_wait_failures.argtypes = []
    h.rowsm_split_wait_failures.restype = i64
    h.rowsm_set_split_wait_limit.argtypes = [i64]
    h.rowsm_set_split_wait_limit.restype = i64
    h.rowsm_status_string.argtypes = [i32]
    h.rowsm_status_string.restype = ctypes.c_char_p
    if path is None:
        _lib = h
    return h


def rowsm_forward(x, y, rows, cols, in_dtype, out_dtype, stream=0) -> int:
    return lib().rowsm_forward(x, y, rows, cols, in_dtype, out_dtype, stream)


def rowsm_forward_noalloc(x, y, rows, cols, in_dtype, out_dtype, stream=0) -> int:
    return lib().rowsm_forward_noalloc(x, y, rows, cols, in_dtype, out_dtype, stream)


def rowsm_forward_variant(x, y, rows, cols, in_dtype, out_dtype, stream, variant) -> int:
    return lib().rowsm_forward_variant(x, y, rows, cols, in_dtype, out_dtype, stream,
                                       variant)


def rowsm_forward_config(x, y, rows, cols, in_dtype, out_dtype, stream, cfg) -> int:
    if cfg is not None and not isinstance(cfg, RowsmConfig):
        cfg = RowsmConfig(**cfg)
    ref = ctypes.byref(cfg) if cfg is not None else None
    return lib().rowsm_forward_config(x, y, rows, cols, in_dtype, out_dtype, stream, ref)


def rowsm_forward_scaled_causal(x, y, rows, cols, in_dtype, out_dtype, scale, causal_period,
                                causal_offset, stream=0, cfg=None) -> int:
    if cfg is not None and not isinstance(cfg, RowsmConfig):
        cfg = RowsmConfig(**cfg)
    ref = ctypes.byref(cfg) if cfg is not None else None
    return lib().rowsm_forward_scaled_causal(x, y, rows, cols, in_dtype, out_dtype, scale,
                                             causal_period, causal_offset, stream, ref)


def rowsm_log_softmax(x, y, rows, cols, in_dtype, out_dtype, stream=0, cfg=None) -> int:
    if cfg is not None and not isinstance(cfg, RowsmConfig):
        cfg = RowsmConfig(**cfg)
    ref = ctypes.byref(cfg) if cfg is not None else None
    return lib().rowsm_log_softmax(x, y, rows, cols, in_dtype, out_dtype, stream, ref)


def rowsm_select(rows, cols, in_dtype, out_dtype) -> int:
    return lib().rowsm_select(rows, cols, in_dtype, out_dtype)


def rowsm_describe(rows, cols, in_dtype, out_dtype, variant=AUTO):
    buf = ctypes.create_string_buffer(256)
    st = lib().rowsm_describe(rows, cols, in_dtype, out_dtype, variant, buf, len(buf))
    return st, buf.value.decode()


def rowsm_describe_op(op, rows, cols, in_dtype, out_dtype, cfg=None):
    if cfg is not None and not isinstance(cfg, RowsmConfig):
        cfg = RowsmConfig(**cfg)
    ref = ctypes.byref(cfg) if cfg is not None else None
    buf = ctypes.create_string_buffer(256)
    st = lib().rowsm_describe_op(op, rows, cols, in_dtype, out_dtype, ref, buf, len(buf))
    return st, buf.value.decode()


def rowsm_softmax_backward(y, dy, dx, rows, cols, in_dtype, out_dtype, stream=0,
                           cfg=None) -> int:
    if cfg is not None and not isinstance(cfg, RowsmConfig):
        cfg = RowsmConfig(**cfg)
    ref = ctypes.byref(cfg) if cfg is not None else None
    return lib().rowsm_softmax_backward(y, dy, dx, rows, cols, in_dtype, out_dtype, stream, ref)


def rowsm_moe_group_top2(scores, out, tokens, experts, group_size, in_dtype, out_dtype,
                         stream=0, cfg=None) -> int:
    if cfg is not None and not isinstance(cfg, RowsmConfig):
        cfg = RowsmConfig(**cfg)
    ref = ctypes.byref(cfg) if cfg is not None else None
    return lib().rowsm_moe_group_top2(scores, out, tokens, experts, group_size, in_dtype,
                                      out_dtype, stream, ref)


def rowsm_stream_copy(x, y, n, in_dtype, out_dtype, stream=0) -> int:
    return lib().rowsm_stream_copy(x, y, n, in_dtype, out_dtype, stream)


def rowsm_split_wait_failures() -> int:
    return lib().rowsm_split_wait_failures()


def rowsm_set_split_wait_limit(polls: int) -> int:
    return lib().rowsm_set_split_wait_limit(polls)


def rowsm_status_string(status) -> str:
    return lib().rowsm_status_string(status).decode()


def check(status: int) -> None:
    if status != OK:
        raise RowsmError(f"rowsm status {status}: {rowsm_status_string(status)}")


def dtype_code(dtype) -> int:
    import torch
    if dtype == torch.float32:
        return F32
    if dtype == torch.bfloat16:
        return BF16
    raise RowsmError(f"unsupported dtype {dtype}")


def _row_operands(name, x, out, out_dtype):
    """Shared marshalling of the row operations: x must be a contiguous GPU
    tensor; out (allocated when None) a contiguous tensor of x's shape on x's
    device.  Returns (out, rows, cols)."""
    import torch
    if not x.is_cuda or not x.is_contiguous():
        raise RowsmError(f"{name} needs a contiguous GPU tensor")
    if out is None:
        out = torch.empty(x.shape, dtype=out_dtype or x.dtype, device=x.device)
    elif out.shape != x.shape or not out.is_contiguous() or out.device != x.device:
        raise RowsmError("out must be a contiguous tensor of the input's shape on its device")
    cols = x.shape[-1] if x.dim() else 1
    rows = x.numel() // cols if cols else 0
    return out, rows, cols


def _stream_handle(stream, device) -> int:
    import torch
    return (stream or torch.cuda.current_stream(device)).cuda_stream


def softmax(x, out_dtype=None, out=None, variant: int = AUTO, config=None, stream=None):
    """softmax(x, dim=-1) of a contiguous fp32/bf16 GPU tensor through the
    library.  Returns ``out`` (allocated with ``out_dtype``, default x.dtype,
    when not given).  Runs on torch's current stream unless ``stream`` (a
    torch.cuda.Stream) is given."""
    out, rows, cols = _row_operands("softmax", x, out, out_dtype)
    args = (x.data_ptr(), out.data_ptr(), rows, cols, dtype_code(x.dtype),
            dtype_code(out.dtype), _stream_handle(stream, x.device))
    if config is not None:
        check(rowsm_forward_config(*args, config))
    elif variant != AUTO:
        check(rowsm_forward_variant(*args, variant))
    else:
        check(rowsm_forward(*args))
    return out


def scaled_causal_softmax(x, scale: float, causal_period: int, causal_offset: int = 0,
                          out_dtype=None, out=None, config=None, stream=None):
    """softmax(scale * x + causal mask, dim=-1) of a contiguous fp32/bf16 GPU
    tensor (see rowsm_forward_scaled_causal).  Marshalling only."""
    out, rows, cols = _row_operands("scaled_causal_softmax", x, out, out_dtype)
    check(rowsm_forward_scaled_causal(x.data_ptr(), out.data_ptr(), rows, cols,
                                      dtype_code(x.dtype), dtype_code(out.dtype), float(scale),
                                      int(causal_period), int(causal_offset),
                                      _stream_handle(stream, x.device), config))
    return out


def log_softmax(x, out_dtype=None, out=None, config=None, stream=None):
    """log(softmax(x, dim=-1)) of a contiguous fp32/bf16 GPU tensor (see
    rowsm_log_softmax).  Marshalling only."""
    out, rows, cols = _row_operands("log_softmax", x, out, out_dtype)
    check(rowsm_log_softmax(x.data_ptr(), out.data_ptr(), rows, cols, dtype_code(x.dtype),
                            dtype_code(out.dtype), _stream_handle(stream, x.device), config))
    return out


def softmax_backward(y, dy, out_dtype=None, out=None, config=None, stream=None):
    """Gradient of softmax(x, dim=-1) given its output ``y`` and the upstream
    gradient ``dy`` (contiguous GPU tensors of one shape and dtype), see
    rowsm_softmax_backward.  Returns ``out`` (dx).  Marshalling only."""
    if not dy.is_cuda or not dy.is_contiguous():
        raise RowsmError("softmax_backward needs contiguous GPU tensors")
    if dy.shape != y.shape or dy.dtype != y.dtype or dy.device != y.device:
        raise RowsmError("y and dy must share shape, dtype and device")
    out, rows, cols = _row_operands("softmax_backward", y, out, out_dtype)
    check(rowsm_softmax_backward(y.data_ptr(), dy.data_ptr(), out.data_ptr(), rows, cols,
                                 dtype_code(y.dtype), dtype_code(out.dtype),
                                 _stream_handle(stream, y.device), config))
    return out


def moe_group_top2(scores, group_size: int = 32, out_dtype=None, out=None, config=None,
                   stream=None):
    """MoE group scores of a contiguous tokens x experts fp32/bf16 GPU tensor:
    the sum of the two largest scores of every group of ``group_size``
    consecutive experts (see rowsm_moe_group_top2).  Returns ``out``
    (tokens x experts / group_size, ``out_dtype``, default fp32).
    Marshalling only."""
    import torch
    if not scores.is_cuda or not scores.is_contiguous():
        raise RowsmError("moe_group_top2 needs a contiguous GPU tensor")
    experts = scores.shape[-1] if scores.dim() else 1
    tokens = scores.numel() // experts if experts else 0
    shape = tuple(scores.shape[:-1]) + (experts // group_size if group_size else 0,)
    if out is None:
        out = torch.empty(shape, dtype=out_dtype or torch.float32, device=scores.device)
    elif tuple(out.shape) != shape or not out.is_contiguous() or out.device != scores.device:
        raise RowsmError("out must be a contiguous tokens x (experts / group_size) tensor")
    check(rowsm_moe_group_top2(scores.data_ptr(), out.data_ptr(), tokens, experts,
                               int(group_size), dtype_code(scores.dtype), dtype_code(out.dtype),
                               _stream_handle(stream, scores.device), config))
    return out


def stream_copy(x, out_dtype=None, out=None, stream=None):
    """x converted to ``out_dtype`` (default x.dtype) by the library's
    streaming copy (see rowsm_stream_copy), the measurement ceiling of the
    row kernels.  Marshalling only."""
    out, rows, cols = _row_operands("stream_copy", x, out, out_dtype)
    check(rowsm_stream_copy(x.data_ptr(), out.data_ptr(), rows * cols, dtype_code(x.dtype),
                            dtype_code(out.dtype), _stream_handle(stream, x.device)))
    return out
