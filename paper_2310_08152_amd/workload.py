"""Seeded synthetic workloads: span boundaries and input tensors.

This module produces *inputs* only.  It holds none of the method's
arithmetic: no attention mask, no token types, no position ids, no keep
rule.  Both the HIP path and the CPU oracle receive what it generates and
derive everything else on their own.

Spans are (cl, cr) pairs of indices into the transformed sequence (the
sequence that already contains the sentinel tokens): ``cl`` is where the
<CL> token sits, ``cr`` is where the <CR> token sits, ``cl < cr``.  The
"span length" ``cr - cl`` counts the <CL> token and the enclosed tokens,
i.e. the rows whose key/value memory is freed once the span is closed
(Section 3.1, paragraphs "Input Transformation" and "Manipulating
Key-Value Memory").  A span with ``cr >= L`` is still open at the end of
the sequence.

Tensor values are i.i.d. N(0, 1), drawn in fp32 from a seeded generator and
then rounded to the storage dtype (round-to-nearest-even for bf16).

The five workloads mirror the model shapes the paper evaluates (OPT-1.3B:
24 layers, 32 heads, head dim 64; a RedPajama-3B-like RoPE model: 32 layers,
32 heads, head dim 80; Section 4.1 "Models") with synthetic data standing in
for WikiText-2 / C4 text and trained weights, which are not available.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Tuple

import numpy as np

__all__ = [
    "Workload", "WORKLOADS", "get_workload",
    "spans_periodic", "spans_jittered_windows", "spans_uniform_lengths",
    "spans_streaming", "spans_to_arrays", "randn", "span_coverage",
]


@dataclass(frozen=True)
class Workload:
    name: str
    layers: int          # M
    batch: int           # b
    heads: int           # H
    d_head: int          # d
    seq_len: int         # L: transformed prompt length (sentinels included)
    dtype: str           # "f32" | "bf16"
    span_kind: str       # generator used for the prompt spans
    span_args: dict = field(default_factory=dict)
    decode_steps: int = 0
    rope_theta: float = 0.0   # 0 = no rotary embedding
    gen_tokens: int = 0       # streaming workload: generated tokens
    seed: int = 0

    @property
    def span_seed(self) -> int:
        return 1000 + self.seed

    @property
    def meta_len(self) -> int:
        """Number of original token indices the span metadata covers."""
        return self.seq_len + max(self.gen_tokens, self.decode_steps)


# Sizes follow the paper's models; the span recipes are the synthetic
# stand-ins described in the module docstring.
WORKLOADS = {
    # Tiny CPU-checkable case: <CL> at offset 8 and <CR> at offset 24 of
    # every 32-token window (span length 16, half the tokens evicted).
    "tiny-f32": Workload("tiny-f32", 1, 1, 4, 64, 256, "f32", "periodic",
                         dict(period=32, cl_off=8, cr_off=24), decode_steps=1, seed=1),
    # OPT-1.3B-shaped prefill slice: one span of length 32 per 64-token
    # window, boundaries jittered by up to 4 tokens per (sequence, window).
    "opt1.3b-prefill": Workload("opt1.3b-prefill", 1, 8, 32, 64, 2048, "bf16", "windows",
                                dict(window=64, cl_off=16, length=32, jitter=4), seed=2),
    # OPT-1.3B-shaped compaction + decode: 75% of the prompt evicted, span
    # lengths uniform in [16, 64].
    "opt1.3b-decode": Workload("opt1.3b-decode", 24, 64, 32, 64, 2048, "bf16", "uniform",
                               dict(ratio=0.75, lo=16, hi=64), decode_steps=128, seed=3),
    # 3B RoPE-shaped prefill + compaction + decode, 50% evicted.
    "3b-rope": Workload("3b-rope", 32, 16, 32, 80, 4096, "bf16", "uniform",
                        dict(ratio=0.5, lo=16, hi=64), decode_steps=128,
                        rope_theta=10000.0, seed=4),
    # Streaming: 1024-token prompt with no spans, then 1024 generated tokens
    # in which every 48-token block holds <CL> at offset 8 and <CR> at 40.
    "3b-rope-stream": Workload("3b-rope-stream", 32, 256, 32, 80, 1024, "bf16", "streaming",
                               dict(block=48, cl_off=8, cr_off=40), rope_theta=10000.0,
                               gen_tokens=1024, seed=5),
}


def get_workload(name: str) -> Workload:
    return WORKLOADS[name]


# ---------------------------------------------------------------------------
# span generators (inputs; pure index bookkeeping)
# ---------------------------------------------------------------------------

def spans_periodic(L: int, period: int, cl_off: int, cr_off: int) -> List[Tuple[int, int]]:
    out = []
    for base in range(0, L, period):
        c, r = base + cl_off, base + cr_off
        if c < L:
            out.append((c, r))
    return out


def spans_jittered_windows(L: int, window: int, cl_off: int, length: int, jitter: int,
                           rng: np.random.Generator) -> List[Tuple[int, int]]:
    out = []
    for base in range(0, L, window):
        delta = int(rng.integers(-jitter, jitter + 1))
        c = base + cl_off + delta
        out.append((c, c + length))
    return out


def spans_uniform_lengths(L: int, ratio: float, lo: int, hi: int,
                          rng: np.random.Generator) -> List[Tuple[int, int]]:
    """Span lengths ~ U[lo, hi] drawn until their sum reaches round(ratio*L).

    The last draw is trimmed so the evicted total is exact; a trimmed piece
    shorter than ``lo`` is merged into an earlier span that has room.  The
    leftover normal tokens (L - E - n, where n spans contribute n <CR> rows)
    are spread over the n+1 gaps with sorted uniform cut points.
    """
    E = int(round(ratio * L))
    lengths: List[int] = []
    total = 0
    while total < E:
        x = int(rng.integers(lo, hi + 1))
        if total + x > E:
            x = E - total
        lengths.append(x)
        total += x
    if len(lengths) > 1 and lengths[-1] < lo:
        rem = lengths.pop()
        for k in rng.permutation(len(lengths)):
            if lengths[k] + rem <= hi:
                lengths[k] += rem
                rem = 0
                break
        if rem:
            lengths.append(rem)
    n = len(lengths)
    G = L - E - n
    if G < 0:
        raise ValueError("ratio too high for the number of spans")
    cuts = np.sort(rng.integers(0, G + 1, size=n))
    gaps = np.diff(np.concatenate([[0], cuts, [G]])).astype(int)
    out = []
    pos = 0
    for k in range(n):
        pos += int(gaps[k])
        c = pos
        r = c + lengths[k]
        out.append((c, r))
        pos = r + 1
    assert pos + int(gaps[n]) == L
    return out


def spans_streaming(prompt_len: int, gen_tokens: int, block: int, cl_off: int,
                    cr_off: int) -> List[Tuple[int, int]]:
    """Spans in the generated part only; the last one may still be open."""
    out = []
    end = prompt_len + gen_tokens
    for base in range(prompt_len, end, block):
        c = base + cl_off
        if c < end:
            out.append((c, base + cr_off))
    return out


def workload_spans(w: Workload) -> List[List[Tuple[int, int]]]:
    """Per-sequence span lists for a workload, from its span seed."""
    rng = np.random.default_rng(w.span_seed)
    out = []
    for _ in range(w.batch):
        if w.span_kind == "periodic":
            s = spans_periodic(w.seq_len, **w.span_args)
        elif w.span_kind == "windows":
            s = spans_jittered_windows(w.seq_len, rng=rng, **w.span_args)
        elif w.span_kind == "uniform":
            s = spans_uniform_lengths(w.seq_len, rng=rng, **w.span_args)
        elif w.span_kind == "streaming":
            s = spans_streaming(w.seq_len, w.gen_tokens, **w.span_args)
        elif w.span_kind == "none":
            s = []
        else:
            raise ValueError(w.span_kind)
        out.append(s)
    return out


def spans_to_arrays(spans: List[List[Tuple[int, int]]], s_max: Optional[int] = None):
    """Pack per-sequence span lists into (cl[b][s_max], cr[b][s_max], n[b]) int32."""
    b = len(spans)
    if s_max is None:
        s_max = max([len(s) for s in spans] + [1])
    cl = np.zeros((b, s_max), np.int32)
    cr = np.zeros((b, s_max), np.int32)
    n = np.zeros((b,), np.int32)
    for i, s in enumerate(spans):
        n[i] = len(s)
        for k, (c, r) in enumerate(s):
            cl[i, k] = c
            cr[i, k] = r
    return cl, cr, n


def span_coverage(spans: List[Tuple[int, int]], L: int) -> int:
    """Number of rows in [0, L) that lie in some [cl, cr)."""
    return sum(max(0, min(r, L) - c) for c, r in spans if c < L)


# ---------------------------------------------------------------------------
# tensors
# ---------------------------------------------------------------------------

def randn(shape, seed: int, dtype: str = "bf16", device: str = "cpu", scale: float = 1.0):
    """i.i.d. N(0, scale^2) tensor: drawn in fp32 from a seeded torch
    generator on ``device``, then rounded to ``dtype``."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    x = torch.randn(tuple(shape), generator=g, device=device, dtype=torch.float32)
    if scale != 1.0:
        x.mul_(scale)
    return x.to(torch_dtype(dtype))


def torch_dtype(dtype: str):
    import torch
    return {"f32": torch.float32, "bf16": torch.bfloat16}[dtype]
