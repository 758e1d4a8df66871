"""Thin ctypes binding of libsckv.so (include/sckv.h).

Argument marshalling only: every function takes torch tensors (device
memory) or numpy arrays (host memory, for span boundaries), passes raw
pointers, sizes and the current HIP stream to the C entry point of the same
name, and raises ``SckvError`` on a non-zero status.  No computation of the
method happens here, and there is no fallback: if the library is missing the
import fails.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libsckv.so")

F32, BF16 = 0, 1
STATUS_CAP, STATUS_TOKEN = 1, 2
OK, EINVAL, ESPAN, ECAP, EHIP, EUNSUP = 0, 1, 2, 3, 4, 5
_ERRNAMES = {1: "EINVAL", 2: "ESPAN", 3: "ECAP", 4: "EHIP", 5: "EUNSUP"}


class SckvError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{_ERRNAMES.get(code, code)}: {msg}")
        self.code = code


def _load():
    if not os.path.exists(_LIB_PATH):
        raise ImportError(
            f"{_LIB_PATH} is missing: build it with `python -m paper_2310_08152_amd.build` "
            "(there is no fallback implementation)")
    return ctypes.CDLL(_LIB_PATH)


lib = _load()

_p = ctypes.c_void_p
_i32 = ctypes.c_int32
_i64 = ctypes.c_int64
_f32 = ctypes.c_float
_sz = ctypes.c_size_t

_SIGS = {
    "sckv_last_error": (ctypes.c_char_p, []),
    "sckv_version": (ctypes.c_char_p, []),
    "sckv_span_meta": (ctypes.c_int, [_p, _p, _p, _i32, _i32, _i32, _p, _p, _p, _p]),
    "rope_apply": (ctypes.c_int, [_p, _p, _i32, _i32, _i32, _i64, _i64, _i32, ctypes.c_int, _p,
                                  _i32, _i32, _f32, _p]),
    "rope_apply_at": (ctypes.c_int, [_p, _p, _p, _i32, _i32, _i32, _i32, _i64, _i64, _i32,
                                     ctypes.c_int, _p, _i32, _i32, _f32, _p, _p]),
    "sckv_prefill_workspace_bytes": (_sz, [_i32, _i32]),
    "sckv_prefill_cached_workspace_bytes": (_sz, [_i32, _i32, _i32]),
    "span_masked_prefill_attn_cached": (ctypes.c_int, [_p, _p, _p, _p, _i32, _i32, _i32, _i32,
                                                       _i64, _i64, _i64, ctypes.c_int, _f32, _p,
                                                       _i32, _i32, _p, _p, _i32, _p, _sz, _p,
                                                       _p]),
    "sckv_prefill_cached_plan": (ctypes.c_int, [_p, _i32, _i32, _p, _p, _i32, _i32, _i32, _p,
                                                _sz, _p]),
    "span_masked_prefill_attn_cached_planned": (ctypes.c_int, [_p, _p, _p, _p, _i32, _i32, _i32,
                                                               _i32, _i64, _i64, _i64,
                                                               ctypes.c_int, _f32, _p, _i32, _i32,
                                                               _p, _p, _i32, _p, _sz, _p, _p]),
    "kv_extend": (ctypes.c_int, [_p, _p, _p, _p, _p, _i32, _i32, _i32, _i32, _i32, _p, _p]),
    "span_masked_prefill_attn": (ctypes.c_int, [_p, _p, _p, _p, _i32, _i32, _i32, _i32, _i64,
                                                _i64, _i64, ctypes.c_int, _f32, _p, _i32, _p, _sz,
                                                _p]),
    "sckv_prefill_plan": (ctypes.c_int, [_p, _i32, _i32, _i32, _p, _sz, _p]),
    "span_masked_prefill_attn_planned": (ctypes.c_int, [_p, _p, _p, _p, _i32, _i32, _i32, _i32,
                                                        _i64, _i64, _i64, ctypes.c_int, _f32, _p,
                                                        _i32, _p, _sz, _p]),
    "kv_compact": (ctypes.c_int, [_p, _p, _i32, _i32, _i32, _i32, _i32, ctypes.c_int, _p, _p, _p,
                                  _p, _p, _i32, _p, _p]),
    "sckv_decode_workspace_bytes": (_sz, [_i32, _i32, _i32, _i32]),
    "compacted_decode_attn": (ctypes.c_int, [_p, _p, _p, _p, _p, _p, _p, _p, _p, _i32, _p, _i32,
                                             _i32, _i32, _i32, ctypes.c_int, _f32, _f32, _p, _sz,
                                             _p, _p]),
    "kv_commit": (ctypes.c_int, [_p, _p, _p, _p, _p, _p, _i32, _i32, _i32, _p, _p]),
    "local_decode_attn": (ctypes.c_int, [_p, _p, _p, _p, _p, _i32, _p, _p, _p, _i32, _p, _i32,
                                         _i32, _i32, _i32, ctypes.c_int, _f32, _f32, _p, _sz, _p,
                                         _p]),
}
for _name, (_res, _args) in _SIGS.items():
    _f = getattr(lib, _name)
    _f.restype = _res
    _f.argtypes = _args

EXPORTS = tuple(_SIGS)


def last_error() -> str:
    return lib.sckv_last_error().decode()


def version() -> str:
    return lib.sckv_version().decode()


def _check(rc: int):
    if rc != OK:
        raise SckvError(rc, last_error())


def _ptr(t):
    """Device (torch) or host (numpy) buffer -> address; None -> NULL."""
    if t is None:
        return None
    if isinstance(t, np.ndarray):
        return t.ctypes.data
    return t.data_ptr()


def _stream(stream, *tensors):
    if stream is not None:
        return stream
    import torch
    for t in tensors:
        if t is not None and hasattr(t, "is_cuda") and t.is_cuda:
            return torch.cuda.current_stream(t.device).cuda_stream
    return None


def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    return 99  # rejected by the library


def _i32_host(a):
    a = np.ascontiguousarray(a, dtype=np.int32)
    return a


# ---------------------------------------------------------------------------
# entry points (same names as the C ABI)
# ---------------------------------------------------------------------------

def sckv_span_meta(cl, cr, n, L_meta: int, spans_dev, vu, pos=None, stream=None):
    """cl, cr: host int32 [b][s_max]; n: host int32 [b]; spans_dev, vu, pos:
    device int32 tensors ([2*b*s_max + b], [b][L_meta], [b][L_meta])."""
    cl, cr, n = _i32_host(cl), _i32_host(cr), _i32_host(n)
    b, s_max = cl.shape
    _check(lib.sckv_span_meta(_ptr(cl), _ptr(cr), _ptr(n), s_max, b, L_meta, _ptr(spans_dev),
                              _ptr(vu), _ptr(pos), _stream(stream, vu)))


def rope_apply(x, y, b: int, H: int, n: int, x_stride_bh: int, y_stride_bh: int, d_head: int,
               pos, L_meta: int, tok0: int, theta: float, stream=None):
    _check(lib.rope_apply(_ptr(x), _ptr(y), b, H, n, x_stride_bh, y_stride_bh, d_head,
                          _dtype_code(x), _ptr(pos), L_meta, tok0, theta, _stream(stream, x)))


def rope_apply_at(x, y, row0, y_rows: int, b: int, H: int, n: int, x_stride_bh: int,
                  y_stride_bh: int, d_head: int, pos, L_meta: int, tok0: int, theta: float,
                  status=None, stream=None):
    _check(lib.rope_apply_at(_ptr(x), _ptr(y), _ptr(row0), y_rows, b, H, n, x_stride_bh,
                             y_stride_bh, d_head, _dtype_code(x), _ptr(pos), L_meta, tok0, theta,
                             _ptr(status), _stream(stream, x)))


def sckv_prefill_cached_workspace_bytes(b: int, nq: int, L_cap: int) -> int:
    return int(lib.sckv_prefill_cached_workspace_bytes(b, nq, L_cap))


def span_masked_prefill_attn_cached(q, k_cache, v_cache, o, b: int, H: int, nq: int, d_head: int,
                                    q_stride_bh: int, kv_stride_bh: int, o_stride_bh: int,
                                    scale: float, vu, L_meta: int, tok0: int, row0, tok_idx,
                                    L_cap: int, ws, status=None, stream=None):
    _check(lib.span_masked_prefill_attn_cached(
        _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(o), b, H, nq, d_head, q_stride_bh,
        kv_stride_bh, o_stride_bh, _dtype_code(q), scale, _ptr(vu), L_meta, tok0, _ptr(row0),
        _ptr(tok_idx), L_cap, _ptr(ws), ws.numel() * ws.element_size(), _ptr(status),
        _stream(stream, q)))


def sckv_prefill_cached_plan(vu, L_meta: int, tok0: int, row0, tok_idx, L_cap: int, b: int,
                             nq: int, ws, stream=None):
    _check(lib.sckv_prefill_cached_plan(_ptr(vu), L_meta, tok0, _ptr(row0), _ptr(tok_idx), L_cap,
                                        b, nq, _ptr(ws), ws.numel() * ws.element_size(),
                                        _stream(stream, ws)))


def span_masked_prefill_attn_cached_planned(q, k_cache, v_cache, o, b: int, H: int, nq: int,
                                            d_head: int, q_stride_bh: int, kv_stride_bh: int,
                                            o_stride_bh: int, scale: float, vu, L_meta: int,
                                            tok0: int, row0, tok_idx, L_cap: int, ws, status=None,
                                            stream=None):
    _check(lib.span_masked_prefill_attn_cached_planned(
        _ptr(q), _ptr(k_cache), _ptr(v_cache), _ptr(o), b, H, nq, d_head, q_stride_bh,
        kv_stride_bh, o_stride_bh, _dtype_code(q), scale, _ptr(vu), L_meta, tok0, _ptr(row0),
        _ptr(tok_idx), L_cap, _ptr(ws), ws.numel() * ws.element_size(), _ptr(status),
        _stream(stream, q)))


def kv_extend(kv_len, tok_idx, pos_ids, row0_out, pos, L_meta: int, tok0: int, n: int, b: int,
              L_cap: int, status=None, stream=None):
    _check(lib.kv_extend(_ptr(kv_len), _ptr(tok_idx), _ptr(pos_ids), _ptr(row0_out), _ptr(pos),
                         L_meta, tok0, n, b, L_cap, _ptr(status), _stream(stream, kv_len)))


def sckv_prefill_workspace_bytes(b: int, L: int) -> int:
    return int(lib.sckv_prefill_workspace_bytes(b, L))


def span_masked_prefill_attn(q, k, v, o, b: int, H: int, L: int, d_head: int, q_stride_bh: int,
                             kv_stride_bh: int, o_stride_bh: int, scale: float, vu, L_meta: int,
                             ws, stream=None):
    _check(lib.span_masked_prefill_attn(_ptr(q), _ptr(k), _ptr(v), _ptr(o), b, H, L, d_head,
                                        q_stride_bh, kv_stride_bh, o_stride_bh, _dtype_code(q),
                                        scale, _ptr(vu), L_meta, _ptr(ws), ws.numel() *
                                        ws.element_size(), _stream(stream, q)))


def sckv_prefill_plan(vu, L_meta: int, b: int, L: int, ws, stream=None):
    _check(lib.sckv_prefill_plan(_ptr(vu), L_meta, b, L, _ptr(ws), ws.numel() * ws.element_size(),
                                 _stream(stream, ws)))


def span_masked_prefill_attn_planned(q, k, v, o, b: int, H: int, L: int, d_head: int,
                                     q_stride_bh: int, kv_stride_bh: int, o_stride_bh: int,
                                     scale: float, vu, L_meta: int, ws, stream=None):
    _check(lib.span_masked_prefill_attn_planned(_ptr(q), _ptr(k), _ptr(v), _ptr(o), b, H, L,
                                                d_head, q_stride_bh, kv_stride_bh, o_stride_bh,
                                                _dtype_code(q), scale, _ptr(vu), L_meta, _ptr(ws),
                                                ws.numel() * ws.element_size(),
                                                _stream(stream, q)))


def kv_compact(kv, kv_out, M: int, b: int, H: int, L_cap: int, d_head: int, kv_len, tok_idx,
               pos_ids, next_tok, vu, L_meta: int, kept_src_row, stream=None):
    _check(lib.kv_compact(_ptr(kv), _ptr(kv_out), M, b, H, L_cap, d_head, _dtype_code(kv),
                          _ptr(kv_len), _ptr(tok_idx), _ptr(pos_ids), _ptr(next_tok), _ptr(vu),
                          L_meta, _ptr(kept_src_row), _stream(stream, kv)))


def sckv_decode_workspace_bytes(b: int, H: int, L_cap: int, d_head: int) -> int:
    return int(lib.sckv_decode_workspace_bytes(b, H, L_cap, d_head))


def compacted_decode_attn(q, k_new, v_new, k_cache, v_cache, kv_len, cur_tok, vu, pos,
                          L_meta: int, o, b: int, H: int, L_cap: int, d_head: int, scale: float,
                          rope_theta: float, ws, status=None, stream=None):
    _check(lib.compacted_decode_attn(_ptr(q), _ptr(k_new), _ptr(v_new), _ptr(k_cache),
                                     _ptr(v_cache), _ptr(kv_len), _ptr(cur_tok), _ptr(vu),
                                     _ptr(pos), L_meta, _ptr(o), b, H, L_cap, d_head,
                                     _dtype_code(q), scale, rope_theta, _ptr(ws),
                                     ws.numel() * ws.element_size(), _ptr(status),
                                     _stream(stream, q)))


def kv_commit(kv_len, tok_idx, pos_ids, cur_tok, vu, pos, L_meta: int, b: int, L_cap: int,
              status=None, stream=None):
    _check(lib.kv_commit(_ptr(kv_len), _ptr(tok_idx), _ptr(pos_ids), _ptr(cur_tok), _ptr(vu),
                         _ptr(pos), L_meta, b, L_cap, _ptr(status), _stream(stream, kv_len)))


def local_decode_attn(q, k_new, v_new, k_cache, v_cache, W: int, cur_tok, vu, pos, L_meta: int,
                      o, b: int, H: int, L_cap: int, d_head: int, scale: float, rope_theta: float,
                      ws, status=None, stream=None):
    _check(lib.local_decode_attn(_ptr(q), _ptr(k_new), _ptr(v_new), _ptr(k_cache), _ptr(v_cache),
                                 W, _ptr(cur_tok), _ptr(vu), _ptr(pos), L_meta, _ptr(o), b, H,
                                 L_cap, d_head, _dtype_code(q), scale, rope_theta, _ptr(ws),
                                 ws.numel() * ws.element_size(), _ptr(status), _stream(stream, q)))
