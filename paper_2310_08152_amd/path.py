"""Host-side orchestration of the hot path: buffer allocation (torch, device
memory only) and the order of C-ABI calls.  No arithmetic of the method is
done here; every step runs in libsckv.so kernels.

Typical use (one batch of sequences):
    meta  = SpanMeta(spans, L_meta, device)          # span metadata, tied positions
    cache = KVCache(M, b, H, L_cap, d, dtype, device)
    prefill_plan(...)                                 # the mask's visibility plan, once
    for m in layers: prefill_layer(..., planned=True) # rotary + masked attention
    cache.compact(meta, next_tok)                     # free closed spans in place
    for step: for m: decode_layer(...); commit(...)   # generate

A prompt too long for the cache is processed block by block instead
(prefill_progressive): each block is appended to the compacted cache,
attends to it, and the spans it closes are freed before the next block.
"""
from __future__ import annotations

import math
from typing import List, Sequence, Tuple

import torch

from . import binding as B
from .workload import spans_to_arrays


class SpanMeta:
    """Device span metadata (vu) and tied position ids for a batch."""

    def __init__(self, spans: Sequence[Sequence[Tuple[int, int]]], L_meta: int, device,
                 stream=None):
        cl, cr, n = spans_to_arrays(list(spans))
        b, s_max = cl.shape
        self.b, self.L_meta, self.device = b, L_meta, torch.device(device)
        self.spans_dev = torch.empty(2 * b * s_max + b, dtype=torch.int32, device=device)
        self.vu = torch.empty(b, L_meta, dtype=torch.int32, device=device)
        self.pos = torch.empty(b, L_meta, dtype=torch.int32, device=device)
        B.sckv_span_meta(cl, cr, n, L_meta, self.spans_dev, self.vu, self.pos, stream=stream)


class KVCache:
    """(M, 2, b, H, L_cap, d) cache with per-sequence row bookkeeping."""

    def __init__(self, M: int, b: int, H: int, L_cap: int, d: int, dtype, device):
        self.M, self.b, self.H, self.L_cap, self.d = M, b, H, L_cap, d
        self.kv = torch.empty(M, 2, b, H, L_cap, d, dtype=dtype, device=device)
        self.kv_len = torch.zeros(b, dtype=torch.int32, device=device)
        self.tok_idx = torch.zeros(b, L_cap, dtype=torch.int32, device=device)
        self.pos_ids = torch.zeros(b, L_cap, dtype=torch.int32, device=device)
        self.kept_src = torch.empty(b, L_cap, dtype=torch.int32, device=device)
        self.cur_tok = torch.zeros(b, dtype=torch.int32, device=device)
        self.status = torch.zeros(1, dtype=torch.int32, device=device)
        # per-layer views, made once: indexing a tensor costs microseconds of
        # host time, and decode issues one call per layer per token
        self._k = [self.kv[m, 0] for m in range(M)]
        self._v = [self.kv[m, 1] for m in range(M)]

    def k(self, m: int):
        return self._k[m]

    def v(self, m: int):
        return self._v[m]

    def start_prompt(self, L: int, meta: SpanMeta):
        """Rows [0, L) hold prompt tokens 0..L-1; the next token is L."""
        self.tok_idx[:, :L] = torch.arange(L, dtype=torch.int32, device=self.kv.device)
        self.pos_ids[:, :L] = meta.pos[:, :L]
        self.kv_len.fill_(L)
        self.cur_tok.fill_(L)

    def compact(self, meta: SpanMeta, next_tok=None, kv_out=None, stream=None):
        nt = self.cur_tok if next_tok is None else next_tok
        B.kv_compact(self.kv, kv_out, self.M, self.b, self.H, self.L_cap, self.d, self.kv_len,
                     self.tok_idx, self.pos_ids, nt, meta.vu, meta.L_meta, self.kept_src,
                     stream=stream)

    def extend(self, meta: SpanMeta, tok0: int, n: int, row0, stream=None):
        """Rows for prompt tokens tok0 .. tok0+n-1 after the current rows;
        row0 (device int32 [b]) receives each sequence's first new row."""
        B.kv_extend(self.kv_len, self.tok_idx, self.pos_ids, row0, meta.pos, meta.L_meta, tok0, n,
                    self.b, self.L_cap, self.status, stream=stream)

    def commit(self, meta: SpanMeta, stream=None):
        B.kv_commit(self.kv_len, self.tok_idx, self.pos_ids, self.cur_tok, meta.vu, meta.pos,
                    meta.L_meta, self.b, self.L_cap, self.status, stream=stream)


class Workspace:
    """Device workspaces sized for a batch shape (block: the block size of
    block-wise prompt processing, if used)."""

    def __init__(self, b: int, H: int, L: int, L_cap: int, d: int, device, block: int = 0):
        self.prefill = torch.empty(max(1, B.sckv_prefill_workspace_bytes(b, max(L, 1))),
                                   dtype=torch.uint8, device=device)
        self.decode = torch.empty(max(1, B.sckv_decode_workspace_bytes(b, H, L_cap, d)),
                                  dtype=torch.uint8, device=device)
        self.prefill_cached = None
        if block > 0:
            self.prefill_cached = torch.empty(
                max(1, B.sckv_prefill_cached_workspace_bytes(b, block, L_cap)),
                dtype=torch.uint8, device=device)


def default_scale(d: int) -> float:
    return 1.0 / math.sqrt(d)


def rope_rows(x, y, meta: SpanMeta, n: int, tok0: int, theta: float, stream=None):
    """Rotate rows [0, n) of every (b, h) slice of x (b, H, >=n, d) into y."""
    b, H, _, d = x.shape
    B.rope_apply(x, y, b, H, n, x.stride(1), y.stride(1), d, meta.pos, meta.L_meta, tok0, theta,
                 stream=stream)


def prefill_layer(q, k, v, o, meta: SpanMeta, ws: Workspace, L: int, scale=None, stream=None,
                  planned: bool = False):
    """Masked attention of q (b,H,L,d) over key/value slices k, v (b,H,>=L,d).
    With planned=True the visibility plan already in ws (prefill_plan) is
    used instead of being rebuilt: it is the same for every layer."""
    b, H, _, d = q.shape
    f = B.span_masked_prefill_attn_planned if planned else B.span_masked_prefill_attn
    f(q, k, v, o, b, H, L, d, q.stride(1), k.stride(1), o.stride(1),
      default_scale(d) if scale is None else scale, meta.vu, meta.L_meta, ws.prefill,
      stream=stream)


def prefill_plan(meta: SpanMeta, ws: Workspace, b: int, L: int, stream=None):
    """Visibility plan of the prompt's first L tokens, shared by all layers."""
    B.sckv_prefill_plan(meta.vu, meta.L_meta, b, L, ws.prefill, stream=stream)


def decode_layer(q, k_new, v_new, cache: KVCache, m: int, meta: SpanMeta, ws: Workspace, o,
                 scale=None, theta: float = 0.0, stream=None):
    d = q.shape[-1]
    B.compacted_decode_attn(q, k_new, v_new, cache.k(m), cache.v(m), cache.kv_len, cache.cur_tok,
                            meta.vu, meta.pos, meta.L_meta, o, cache.b, cache.H, cache.L_cap, d,
                            default_scale(d) if scale is None else scale, theta, ws.decode,
                            cache.status, stream=stream)


def prefill_block(q, cache: KVCache, m: int, o, meta: SpanMeta, ws: Workspace, tok0: int, row0,
                  scale=None, stream=None, planned: bool = False):
    """Masked attention of a block's queries q (b,H,nq,d), tokens tok0.., over
    layer m of the cache, whose rows row0.. hold the block itself.  With
    planned=True the plan already in ws (prefill_block_plan) is used."""
    b, H, nq, d = q.shape
    f = B.span_masked_prefill_attn_cached_planned if planned else B.span_masked_prefill_attn_cached
    f(q, cache.k(m), cache.v(m), o, b, H, nq, d, q.stride(1), cache.k(m).stride(1), o.stride(1),
      default_scale(d) if scale is None else scale, meta.vu, meta.L_meta, tok0, row0,
      cache.tok_idx, cache.L_cap, ws.prefill_cached, status=cache.status, stream=stream)


def prefill_block_plan(cache: KVCache, meta: SpanMeta, ws: Workspace, tok0: int, nq: int, row0,
                       stream=None):
    """Plan of a block's masked attention over the cache, shared by all layers."""
    B.sckv_prefill_cached_plan(meta.vu, meta.L_meta, tok0, row0, cache.tok_idx, cache.L_cap,
                               cache.b, nq, ws.prefill_cached, stream=stream)


def prefill_progressive(q, k, v, o, cache: KVCache, meta: SpanMeta, ws: Workspace, L: int,
                        block: int, theta: float = 0.0, scale=None, stream=None,
                        on_block=None):
    """Process the prompt (tokens 0..L-1) in blocks of `block` tokens:
    for each block, append its rows to the compacted cache (keys rotated),
    run the masked attention of its queries over the cache for every layer,
    then free the spans closed within it (compaction at the block's end).

    q, k, v, o: (M, b, H, >= L, d) per-layer prompt tensors (o receives the
    outputs).  The cache starts empty; at the end it holds the rows a token
    after the prompt may see, exactly as a one-shot prefill + compaction
    leaves it.  on_block(B1), if given, is called after each block."""
    M, b, H, _, d = q.shape
    cache.kv_len.zero_()
    row0 = torch.empty(b, dtype=torch.int32, device=q.device)
    nxt = torch.empty(b, dtype=torch.int32, device=q.device)
    qr = torch.empty(b, H, block, d, dtype=q.dtype, device=q.device)
    for B0 in range(0, L, block):
        n = min(block, L - B0)
        cache.extend(meta, B0, n, row0, stream=stream)
        prefill_block_plan(cache, meta, ws, B0, n, row0, stream=stream)
        for m in range(M):
            for kv, src, th in ((0, k, theta), (1, v, 0.0)):
                x = src[m, :, :, B0:B0 + n]
                dst = cache.kv[m, kv]
                B.rope_apply_at(x, dst, row0, cache.L_cap, b, H, n, x.stride(1), dst.stride(1), d,
                                meta.pos, meta.L_meta, B0, th, status=cache.status,
                                stream=stream)
            B.rope_apply(q[m, :, :, B0:B0 + n], qr, b, H, n, q.stride(2), qr.stride(1), d,
                         meta.pos, meta.L_meta, B0, theta, stream=stream)
            prefill_block(qr[:, :, :n], cache, m, o[m, :, :, B0:B0 + n], meta, ws, B0, row0,
                          scale=scale, stream=stream, planned=True)
        nxt.fill_(B0 + n)
        cache.compact(meta, next_tok=nxt, stream=stream)
        if on_block is not None:
            on_block(B0 + n)
    cache.cur_tok.fill_(L)


# ---------------------------------------------------------------------------
# local-attention comparator: a ring of the W most recent tokens
# ---------------------------------------------------------------------------

def ring_fill(x, y, W: int, L: int, meta: SpanMeta, theta: float, L_cap: int, stream=None):
    """Rotate tokens [L-W, L) of x (b, H, >=L, d) into the ring slices y
    (b, H, L_cap, d), token t at row t mod W."""
    b, H, _, d = x.shape
    t0 = L - W
    a = t0 % W
    pieces = ((t0, t0 + (W - a), a), (t0 + (W - a), L, 0))  # (first token, end, first row)
    for ts, te, r in pieces:
        if te <= ts:
            continue
        row0 = torch.full((b,), r, dtype=torch.int32, device=x.device)
        xs = x[:, :, ts:te]
        B.rope_apply_at(xs, y, row0, L_cap, b, H, te - ts, xs.stride(1), y.stride(1), d, meta.pos,
                        meta.L_meta, ts, theta, stream=stream)


def local_decode_layer(q, k_new, v_new, cache: KVCache, m: int, W: int, meta: SpanMeta,
                       ws: Workspace, o, scale=None, theta: float = 0.0, stream=None):
    """Attention of the current token over the W most recent tokens held in
    the ring rows of layer m; the new token replaces the oldest."""
    d = q.shape[-1]
    B.local_decode_attn(q, k_new, v_new, cache.k(m), cache.v(m), W, cache.cur_tok, meta.vu,
                        meta.pos, meta.L_meta, o, cache.b, cache.H, cache.L_cap, d,
                        default_scale(d) if scale is None else scale, theta, ws.decode,
                        cache.status, stream=stream)
