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
    "compacted_decode_attn_noalloc": (ctypes.c_int, [_p, _p, _p, _p, _p, _p, _p, _p, _p, _i32, _p,
                                                     _i32, _i32, _i32, _i32, ctypes.c_int, _f32,
                                                     _f32, _p, _p]),
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
    """Host (numpy) buffer -> address; None -> NULL.  Device tensors go
    through _dev, which checks them first."""
    if t is None:
        return None
    if isinstance(t, np.ndarray):
        return t.ctypes.data
    return t.data_ptr()


def _fail(msg):
    raise SckvError(EINVAL, msg)


def _avail(t) -> int:
    """Elements of t's storage from its first element to the storage's end."""
    return t.untyped_storage().nbytes() // t.element_size() - t.storage_offset()


_torch = _I32 = _FLOATS = _raw_stream = None


def _tm():
    """torch, imported on first use (host-only callers never need it)."""
    global _torch, _I32, _FLOATS, _raw_stream
    if _torch is None:
        import torch
        _I32, _FLOATS = torch.int32, (torch.float32, torch.bfloat16)
        # the raw handle of the current stream of a device, without building
        # a Stream object per call
        _raw_stream = getattr(torch._C, "_cuda_getCurrentRawStream", None) or (
            lambda dev: torch.cuda.current_stream(dev).cuda_stream)
        _torch = torch
    return _torch


def _dev(t, what, kind=None, need=0, contiguous=False, nullable=False):
    """Address of a device tensor after checking what the kernels will
    assume of it: on a GPU, of the element type `kind` ("i32", "float":
    fp32 or bf16, "u8": any byte workspace), contiguous if asked, and with
    at least `need` elements from its first one to the end of its storage
    (so no kernel addresses memory outside the allocation)."""
    torch = _torch or _tm()
    if t is None:
        if nullable:
            return None
        _fail(f"{what}: missing (None)")
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        _fail(f"{what}: must be a device (cuda) tensor")
    if kind is not None:
        dt = t.dtype
        if kind == "i32" and dt != _I32:
            _fail(f"{what}: must be int32, got {dt}")
        if kind == "float" and dt not in _FLOATS:
            _fail(f"{what}: must be float32 or bfloat16, got {dt}")
    if contiguous:
        if not t.is_contiguous():
            _fail(f"{what}: must be contiguous")
        if need <= t.numel():  # a contiguous tensor holds its numel elements from the first
            return t.data_ptr()
    if need > _avail(t):
        _fail(f"{what}: {need} elements addressed, only {_avail(t)} in its storage")
    return t.data_ptr()


def _rows(t, what, b, H, n, d, stride_bh, dtype=None):
    """(b, H, n, d) slices with (b, h) stride stride_bh: rows contiguous,
    the batch stride H * stride_bh, element type as `dtype` (if given)."""
    if t is not None and t.dim() == 4:
        sh, st = t.shape, t.stride()
        four = sh[0] == b and sh[1] == H
    else:
        four = False
    if four:
        if n > 1 and st[2] != d or st[3] != 1:
            _fail(f"{what}: rows of {d} elements must be contiguous")
        if H > 1 and st[1] != stride_bh or b > 1 and st[0] != H * stride_bh:
            _fail(f"{what}: (b, h) slices must be stride_bh = {stride_bh} apart")
    elif t is not None and not t.is_contiguous():
        _fail(f"{what}: expected a (b, H, n, d) view or a contiguous tensor")
    p = _dev(t, what, "float", (b * H - 1) * stride_bh + n * d if b * H and n else 0)
    if dtype is not None and t.dtype != dtype:
        _fail(f"{what}: element type {t.dtype} differs from {dtype}")
    return p


def _stream(stream, *tensors):
    """The caller's stream, else the current stream of the first device
    tensor's GPU."""
    if stream is not None:
        return stream
    torch = _torch or _tm()
    for t in tensors:
        if isinstance(t, torch.Tensor) and t.is_cuda:
            return _raw_stream(t.get_device())
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

def _ws(ws, what="ws"):
    """A device workspace: address and size in bytes."""
    p = _dev(ws, what, contiguous=True)
    return p, ws.numel() * ws.element_size()


def sckv_span_meta(cl, cr, n, L_meta: int, spans_dev, vu, pos=None, stream=None):
    """cl, cr: host int32 [b][s_max]; n: host int32 [b]; spans_dev, vu, pos:
    device int32 tensors ([2*b*s_max + b], [b][L_meta], [b][L_meta])."""
    cl, cr, n = _i32_host(cl), _i32_host(cr), _i32_host(n)
    b, s_max = cl.shape
    if cr.shape != cl.shape or n.shape != (b,):
        _fail("sckv_span_meta: cl, cr must be [b][s_max] and n [b]")
    _check(lib.sckv_span_meta(_ptr(cl), _ptr(cr), _ptr(n), s_max, b, L_meta,
                              _dev(spans_dev, "spans_dev", "i32", 2 * b * s_max + b, True),
                              _dev(vu, "vu", "i32", b * L_meta, True),
                              _dev(pos, "pos", "i32", b * L_meta, True, nullable=True),
                              _stream(stream, vu)))


def rope_apply(x, y, b: int, H: int, n: int, x_stride_bh: int, y_stride_bh: int, d_head: int,
               pos, L_meta: int, tok0: int, theta: float, stream=None):
    px = _rows(x, "x", b, H, n, d_head, x_stride_bh)
    py = _rows(y, "y", b, H, n, d_head, y_stride_bh, x.dtype)
    pp = _dev(pos, "pos", "i32", b * L_meta, True, nullable=theta == 0)
    _check(lib.rope_apply(px, py, b, H, n, x_stride_bh, y_stride_bh, d_head, _dtype_code(x), pp,
                          L_meta, tok0, theta, _stream(stream, x)))


def rope_apply_at(x, y, row0, y_rows: int, b: int, H: int, n: int, x_stride_bh: int,
                  y_stride_bh: int, d_head: int, pos, L_meta: int, tok0: int, theta: float,
                  status=None, stream=None):
    px = _rows(x, "x", b, H, n, d_head, x_stride_bh)
    py = _rows(y, "y", b, H, y_rows, d_head, y_stride_bh, x.dtype)
    _check(lib.rope_apply_at(px, py, _dev(row0, "row0", "i32", b, True), y_rows, b, H, n,
                             x_stride_bh, y_stride_bh, d_head, _dtype_code(x),
                             _dev(pos, "pos", "i32", b * L_meta, True, nullable=theta == 0),
                             L_meta, tok0, theta,
                             _dev(status, "status", "i32", 1, nullable=True),
                             _stream(stream, x)))


def sckv_prefill_cached_workspace_bytes(b: int, nq: int, L_cap: int) -> int:
    return int(lib.sckv_prefill_cached_workspace_bytes(b, nq, L_cap))


def _cached_args(q, k_cache, v_cache, o, b, H, nq, d_head, q_stride_bh, kv_stride_bh,
                 o_stride_bh, vu, L_meta, row0, tok_idx, L_cap, ws, status):
    pq = _rows(q, "q", b, H, nq, d_head, q_stride_bh)
    pk = _rows(k_cache, "k_cache", b, H, L_cap, d_head, kv_stride_bh, q.dtype)
    pv = _rows(v_cache, "v_cache", b, H, L_cap, d_head, kv_stride_bh, q.dtype)
    po = _rows(o, "o", b, H, nq, d_head, o_stride_bh, q.dtype)
    pw, nw = _ws(ws)
    return (pq, pk, pv, po, _dev(vu, "vu", "i32", b * L_meta, True),
            _dev(row0, "row0", "i32", b, True), _dev(tok_idx, "tok_idx", "i32", b * L_cap, True),
            pw, nw, _dev(status, "status", "i32", 1, nullable=True))


def span_masked_prefill_attn_cached(q, k_cache, v_cache, o, b: int, H: int, nq: int, d_head: int,
                                    q_stride_bh: int, kv_stride_bh: int, o_stride_bh: int,
                                    scale: float, vu, L_meta: int, tok0: int, row0, tok_idx,
                                    L_cap: int, ws, status=None, stream=None):
    pq, pk, pv, po, pvu, pr0, ptok, pw, nw, pst = _cached_args(
        q, k_cache, v_cache, o, b, H, nq, d_head, q_stride_bh, kv_stride_bh, o_stride_bh, vu,
        L_meta, row0, tok_idx, L_cap, ws, status)
    _check(lib.span_masked_prefill_attn_cached(
        pq, pk, pv, po, b, H, nq, d_head, q_stride_bh, kv_stride_bh, o_stride_bh, _dtype_code(q),
        scale, pvu, L_meta, tok0, pr0, ptok, L_cap, pw, nw, pst, _stream(stream, q)))


def sckv_prefill_cached_plan(vu, L_meta: int, tok0: int, row0, tok_idx, L_cap: int, b: int,
                             nq: int, ws, stream=None):
    pw, nw = _ws(ws)
    _check(lib.sckv_prefill_cached_plan(_dev(vu, "vu", "i32", b * L_meta, True), L_meta, tok0,
                                        _dev(row0, "row0", "i32", b, True),
                                        _dev(tok_idx, "tok_idx", "i32", b * L_cap, True), L_cap,
                                        b, nq, pw, nw, _stream(stream, ws)))


def span_masked_prefill_attn_cached_planned(q, k_cache, v_cache, o, b: int, H: int, nq: int,
                                            d_head: int, q_stride_bh: int, kv_stride_bh: int,
                                            o_stride_bh: int, scale: float, vu, L_meta: int,
                                            tok0: int, row0, tok_idx, L_cap: int, ws, status=None,
                                            stream=None):
    pq, pk, pv, po, pvu, pr0, ptok, pw, nw, pst = _cached_args(
        q, k_cache, v_cache, o, b, H, nq, d_head, q_stride_bh, kv_stride_bh, o_stride_bh, vu,
        L_meta, row0, tok_idx, L_cap, ws, status)
    _check(lib.span_masked_prefill_attn_cached_planned(
        pq, pk, pv, po, b, H, nq, d_head, q_stride_bh, kv_stride_bh, o_stride_bh, _dtype_code(q),
        scale, pvu, L_meta, tok0, pr0, ptok, L_cap, pw, nw, pst, _stream(stream, q)))


def kv_extend(kv_len, tok_idx, pos_ids, row0_out, pos, L_meta: int, tok0: int, n: int, b: int,
              L_cap: int, status=None, stream=None):
    _check(lib.kv_extend(_dev(kv_len, "kv_len", "i32", b, True),
                         _dev(tok_idx, "tok_idx", "i32", b * L_cap, True),
                         _dev(pos_ids, "pos_ids", "i32", b * L_cap, True),
                         _dev(row0_out, "row0_out", "i32", b, True),
                         _dev(pos, "pos", "i32", b * L_meta, True), L_meta, tok0, n, b, L_cap,
                         _dev(status, "status", "i32", 1, nullable=True),
                         _stream(stream, kv_len)))


def sckv_prefill_workspace_bytes(b: int, L: int) -> int:
    return int(lib.sckv_prefill_workspace_bytes(b, L))


def _prefill_args(q, k, v, o, b, H, L, d_head, q_stride_bh, kv_stride_bh, o_stride_bh, vu,
                  L_meta, ws):
    pw, nw = _ws(ws)
    return (_rows(q, "q", b, H, L, d_head, q_stride_bh),
            _rows(k, "k", b, H, L, d_head, kv_stride_bh, q.dtype),
            _rows(v, "v", b, H, L, d_head, kv_stride_bh, q.dtype),
            _rows(o, "o", b, H, L, d_head, o_stride_bh, q.dtype),
            _dev(vu, "vu", "i32", b * L_meta, True), pw, nw)


def span_masked_prefill_attn(q, k, v, o, b: int, H: int, L: int, d_head: int, q_stride_bh: int,
                             kv_stride_bh: int, o_stride_bh: int, scale: float, vu, L_meta: int,
                             ws, stream=None):
    pq, pk, pv, po, pvu, pw, nw = _prefill_args(q, k, v, o, b, H, L, d_head, q_stride_bh,
                                                kv_stride_bh, o_stride_bh, vu, L_meta, ws)
    _check(lib.span_masked_prefill_attn(pq, pk, pv, po, b, H, L, d_head, q_stride_bh,
                                        kv_stride_bh, o_stride_bh, _dtype_code(q), scale, pvu,
                                        L_meta, pw, nw, _stream(stream, q)))


def sckv_prefill_plan(vu, L_meta: int, b: int, L: int, ws, stream=None):
    pw, nw = _ws(ws)
    _check(lib.sckv_prefill_plan(_dev(vu, "vu", "i32", b * L_meta, True), L_meta, b, L, pw, nw,
                                 _stream(stream, ws)))


def span_masked_prefill_attn_planned(q, k, v, o, b: int, H: int, L: int, d_head: int,
                                     q_stride_bh: int, kv_stride_bh: int, o_stride_bh: int,
                                     scale: float, vu, L_meta: int, ws, stream=None):
    pq, pk, pv, po, pvu, pw, nw = _prefill_args(q, k, v, o, b, H, L, d_head, q_stride_bh,
                                                kv_stride_bh, o_stride_bh, vu, L_meta, ws)
    _check(lib.span_masked_prefill_attn_planned(pq, pk, pv, po, b, H, L, d_head, q_stride_bh,
                                                kv_stride_bh, o_stride_bh, _dtype_code(q), scale,
                                                pvu, L_meta, pw, nw, _stream(stream, q)))


def kv_compact(kv, kv_out, M: int, b: int, H: int, L_cap: int, d_head: int, kv_len, tok_idx,
               pos_ids, next_tok, vu, L_meta: int, kept_src_row, stream=None):
    n = M * 2 * b * H * L_cap * d_head
    pkv = _dev(kv, "kv", "float", n, True)
    pout = _dev(kv_out, "kv_out", "float", n, True, nullable=True)
    if kv_out is not None and kv_out.dtype != kv.dtype:
        _fail("kv_out: element type differs from kv")
    _check(lib.kv_compact(pkv, pout, M, b, H, L_cap, d_head, _dtype_code(kv),
                          _dev(kv_len, "kv_len", "i32", b, True),
                          _dev(tok_idx, "tok_idx", "i32", b * L_cap, True),
                          _dev(pos_ids, "pos_ids", "i32", b * L_cap, True),
                          _dev(next_tok, "next_tok", "i32", b, True),
                          _dev(vu, "vu", "i32", b * L_meta, True), L_meta,
                          _dev(kept_src_row, "kept_src_row", "i32", b * L_cap, True),
                          _stream(stream, kv)))


def sckv_decode_workspace_bytes(b: int, H: int, L_cap: int, d_head: int) -> int:
    return int(lib.sckv_decode_workspace_bytes(b, H, L_cap, d_head))


def _decode_args(q, k_new, v_new, k_cache, v_cache, o, vu, pos, L_meta, b, H, L_cap, d_head,
                 theta, status):
    nh = b * H * d_head
    pq = _dev(q, "q", "float", nh, True)
    out = [pq]
    for t, nm in ((k_new, "k_new"), (v_new, "v_new")):
        out.append(_dev(t, nm, "float", nh, True))
    for t, nm in ((k_cache, "k_cache"), (v_cache, "v_cache")):
        out.append(_dev(t, nm, "float", b * H * L_cap * d_head, True))
    out.append(_dev(o, "o", "float", nh, True))
    for t, nm in ((k_new, "k_new"), (v_new, "v_new"), (k_cache, "k_cache"), (v_cache, "v_cache"),
                  (o, "o")):
        if t.dtype != q.dtype:
            _fail(f"{nm}: element type {t.dtype} differs from q's {q.dtype}")
    out.append(_dev(vu, "vu", "i32", b * L_meta, True))
    out.append(_dev(pos, "pos", "i32", b * L_meta, True, nullable=theta == 0))
    out.append(_dev(status, "status", "i32", 1, nullable=True))
    return out


def compacted_decode_attn(q, k_new, v_new, k_cache, v_cache, kv_len, cur_tok, vu, pos,
                          L_meta: int, o, b: int, H: int, L_cap: int, d_head: int, scale: float,
                          rope_theta: float, ws, status=None, stream=None):
    pq, pkn, pvn, pkc, pvc, po, pvu, ppos, pst = _decode_args(
        q, k_new, v_new, k_cache, v_cache, o, vu, pos, L_meta, b, H, L_cap, d_head, rope_theta,
        status)
    pw, nw = _ws(ws)
    _check(lib.compacted_decode_attn(pq, pkn, pvn, pkc, pvc,
                                     _dev(kv_len, "kv_len", "i32", b, True),
                                     _dev(cur_tok, "cur_tok", "i32", b, True), pvu, ppos, L_meta,
                                     po, b, H, L_cap, d_head, _dtype_code(q), scale, rope_theta,
                                     pw, nw, pst, _stream(stream, q)))


def compacted_decode_attn_noalloc(q, k_new, v_new, k_cache, v_cache, kv_len, cur_tok, vu, pos,
                                  L_meta: int, o, b: int, H: int, L_cap: int, d_head: int,
                                  scale: float, rope_theta: float, status=None, stream=None):
    """compacted_decode_attn with the library's own scratch array in place
    of a workspace (no allocation by the call)."""
    pq, pkn, pvn, pkc, pvc, po, pvu, ppos, pst = _decode_args(
        q, k_new, v_new, k_cache, v_cache, o, vu, pos, L_meta, b, H, L_cap, d_head, rope_theta,
        status)
    _check(lib.compacted_decode_attn_noalloc(pq, pkn, pvn, pkc, pvc,
                                             _dev(kv_len, "kv_len", "i32", b, True),
                                             _dev(cur_tok, "cur_tok", "i32", b, True), pvu, ppos,
                                             L_meta, po, b, H, L_cap, d_head, _dtype_code(q),
                                             scale, rope_theta, pst, _stream(stream, q)))


NOALLOC_SCRATCH_BYTES = 16 << 20  # SCKV_NOALLOC_SCRATCH_BYTES in sckv.h


def kv_commit(kv_len, tok_idx, pos_ids, cur_tok, vu, pos, L_meta: int, b: int, L_cap: int,
              status=None, stream=None):
    _check(lib.kv_commit(_dev(kv_len, "kv_len", "i32", b, True),
                         _dev(tok_idx, "tok_idx", "i32", b * L_cap, True),
                         _dev(pos_ids, "pos_ids", "i32", b * L_cap, True),
                         _dev(cur_tok, "cur_tok", "i32", b, True),
                         _dev(vu, "vu", "i32", b * L_meta, True),
                         _dev(pos, "pos", "i32", b * L_meta, True), L_meta, b, L_cap,
                         _dev(status, "status", "i32", 1, nullable=True),
                         _stream(stream, kv_len)))


def local_decode_attn(q, k_new, v_new, k_cache, v_cache, W: int, cur_tok, vu, pos, L_meta: int,
                      o, b: int, H: int, L_cap: int, d_head: int, scale: float, rope_theta: float,
                      ws, status=None, stream=None):
    pq, pkn, pvn, pkc, pvc, po, pvu, ppos, pst = _decode_args(
        q, k_new, v_new, k_cache, v_cache, o, vu, pos, L_meta, b, H, L_cap, d_head, rope_theta,
        status)
    pw, nw = _ws(ws)
    _check(lib.local_decode_attn(pq, pkn, pvn, pkc, pvc, W,
                                 _dev(cur_tok, "cur_tok", "i32", b, True), pvu, ppos, L_meta, po,
                                 b, H, L_cap, d_head, _dtype_code(q), scale, rope_theta, pw, nw,
                                 pst, _stream(stream, q)))
