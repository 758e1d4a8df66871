"""CPU oracle for sentinel-token context compression (Ren, Jia and Zhu, 2023).

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or
execute this module: only the test suite, the smoke check and the CPU
baseline leg of the benchmark use it.  It shares no code with the HIP
library and imports nothing from the package.

Everything here is plain, slow and dense: float64 NumPy, one sequence at a
time, an explicit L x L boolean mask built pair by pair from the prose rules
of the paper.  Each function names the passage it follows.

Token types (Section 3.1): two sentinel tokens, <CL> and <CR>, are placed
around a contiguous span whose key/value memory will be compressed; every
other token is a "normal" token (tokens enclosed by a span are normal tokens
too).

Readings of the paper where it is silent or the figure that would settle a
point is missing (Figure 1 is not reproduced in the text):
  R1  enclosed tokens do not attend to their own <CL> (only <CR> and normal
      tokens are listed as attendable by normal tokens);
  R2  a <CR> token attends like a normal token: to earlier <CR>/normal tokens
      that are not hidden by an earlier closed span, to its own enclosed
      tokens and to itself, but not to any <CL>;
  R3  a <CL> token attends to itself only, so its output is its own value;
  R4  the rows freed from the cache are the <CL> row and the enclosed rows of
      each closed span; the <CR> row is kept;
  R5  the softmax scale is 1/sqrt(d_head) unless given;
  R6  rotary embedding is the rotate-half form over the full head dimension,
      applied at the tied (original) position of each token;
  R7  a decode step whose token is a <CL> outputs that token's value and adds
      nothing to the cache (it is never visible to a later token).

Parity status: the paper prints no numeric worked example (its Figure 1 is
an image that is not part of the text), so no stored value here comes from
the paper itself; every function is pinned by hand-derived small cases,
closed forms, library routines on special cases and brute force (see the
test suite).
"""
from __future__ import annotations

import numpy as np

NORMAL, CL, CR = 0, 1, 2

__all__ = [
    "NORMAL", "CL", "CR", "token_types", "enclosing_cr", "attention_mask", "attention_mask_rows",
    "tie_positions", "rope_rotate_half", "masked_attention", "keep_rows",
    "compact_cache", "decode_attention", "run_prompt_and_decode",
]


# ---------------------------------------------------------------------------
# Section 3.1: sentinel tokens placed around spans
# ---------------------------------------------------------------------------

def token_types(spans, L):
    """Type of every position of a transformed sequence of length L.

    ``spans`` is a list of (cl, cr): the <CL> token sits at index cl and the
    <CR> token at index cr (cr >= L means the span is not closed inside the
    sequence).  Section 3.1, first paragraph.
    """
    t = np.full(L, NORMAL, dtype=np.int64)
    for cl, cr in spans:
        if 0 <= cl < L:
            t[cl] = CL
        if 0 <= cr < L:
            t[cr] = CR
    return t


def enclosing_cr(types):
    """For each position, the index of the <CR> that closes the span the
    token is enclosed in, or -1 when the token is not enclosed.  A token of
    a span still open at the end gets len(types) (its <CR> lies beyond the
    sequence).  Section 3.1: tokens "between <CL> and <CR>"."""
    L = len(types)
    out = np.full(L, -1, dtype=np.int64)
    open_members = None
    for t in range(L):
        if types[t] == CL:
            open_members = []
        elif types[t] == CR:
            if open_members is not None:
                for j in open_members:
                    out[j] = t
            open_members = None
        elif open_members is not None:
            open_members.append(t)
    if open_members is not None:
        for j in open_members:
            out[j] = L
    return out


def attention_mask(types):
    """Modified causal mask, True = row i may attend to column j.

    Written pair by pair from the rules of Section 1 and Section 3.1:
      * causal: nothing in the future;
      * a <CL> token attends only to itself;
      * normal tokens (and <CR>, reading R2) attend to earlier <CR> and
        normal tokens, never to a <CL>;
      * tokens after a <CR> cannot attend to the tokens between that <CR>
        and its <CL>.
    """
    L = len(types)
    enc = enclosing_cr(types)
    m = np.zeros((L, L), dtype=bool)
    for i in range(L):
        for j in range(i + 1):
            if types[i] == CL:
                m[i, j] = (j == i)
                continue
            if types[j] == CL:
                continue
            if enc[j] >= 0 and i > enc[j]:
                continue
            m[i, j] = True
    return m


def attention_mask_rows(types, rows):
    """The rows ``rows`` of attention_mask(types), built pair by pair by the
    same rules, for sequences too long for the whole L x L mask."""
    L = len(types)
    enc = enclosing_cr(types)
    m = np.zeros((len(rows), L), dtype=bool)
    for r, i in enumerate(rows):
        for j in range(i + 1):
            if types[i] == CL:
                m[r, j] = (j == i)
                continue
            if types[j] == CL:
                continue
            if enc[j] >= 0 and i > enc[j]:
                continue
            m[r, j] = True
    return m


def tie_positions(types):
    """Position ids of the transformed sequence (Section 3.1, "Input
    Transformation"): sentinels take the position of the token before them,
    so normal tokens keep consecutive positions 0, 1, 2, ...  A sentinel at
    index 0 takes position 0."""
    L = len(types)
    pos = np.zeros(L, dtype=np.int64)
    nxt = 0
    for t in range(L):
        if types[t] == NORMAL:
            pos[t] = nxt
            nxt += 1
        else:
            pos[t] = pos[t - 1] if t > 0 else 0
    return pos


# ---------------------------------------------------------------------------
# Rotary position embedding (reading R6), float64
# ---------------------------------------------------------------------------

def rope_rotate_half(x, pos, theta):
    """x[..., n, d] rotated at integer positions pos[n]: the first and second
    halves of the head dimension form the (real, imaginary) pairs, pair i
    turning by angle pos * theta^(-2i/d)."""
    x = np.asarray(x, dtype=np.float64)
    d = x.shape[-1]
    half = d // 2
    inv = theta ** (-(2.0 * np.arange(half, dtype=np.float64)) / d)
    ang = np.asarray(pos, dtype=np.float64)[:, None] * inv[None, :]
    c, s = np.cos(ang), np.sin(ang)
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


# ---------------------------------------------------------------------------
# Attention under the modified mask (Section 3.1), float64
# ---------------------------------------------------------------------------

def masked_attention(q, k, v, mask, scale=None, return_probs=False):
    """softmax(scale * q k^T restricted to ``mask``) v for one sequence.

    q: [H, Lq, d]; k, v: [H, L, d]; mask: [Lq, L] bool (row attends to
    column; Lq = L for the whole sequence, fewer for sampled query rows).
    """
    q = np.asarray(q, np.float64)
    k = np.asarray(k, np.float64)
    v = np.asarray(v, np.float64)
    H, L, d = q.shape
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    s = scale * np.einsum("hid,hjd->hij", q, k)
    s = np.where(mask[None], s, -np.inf)
    mx = s.max(axis=-1, keepdims=True)
    p = np.exp(s - mx)
    p = p / p.sum(axis=-1, keepdims=True)
    o = np.einsum("hij,hjd->hid", p, v)
    return (o, p) if return_probs else o


# ---------------------------------------------------------------------------
# Freeing the key/value memory of closed spans (Section 3, "Manipulating
# Key-Value Memory for Inference-time Compression"), reading R4
# ---------------------------------------------------------------------------

def keep_rows(types, next_index):
    """keep[t] for every original index t: True when the key/value row of
    token t can still be attended by a normal token at index ``next_index``
    or later.  A <CL> row is never attendable by a later token; an enclosed
    row stops being attendable once its <CR> has been processed."""
    L = len(types)
    enc = enclosing_cr(types)
    keep = np.ones(L, dtype=bool)
    for t in range(L):
        if types[t] == CL:
            keep[t] = False
        elif enc[t] >= 0 and next_index > enc[t]:
            keep[t] = False
    return keep


def compact_cache(k, v, tok_idx, pos_ids, kv_len, types, next_index):
    """Drop freed rows from a cache, keeping the survivors in their order.

    k, v: [H, L_cap, d] (any dtype; copied as is); tok_idx, pos_ids: [L_cap];
    rows [0, kv_len) are valid and row r holds original token tok_idx[r].
    Returns (k', v', tok', pos', kv_len', kept_src) with kept_src the list of
    surviving source rows.
    """
    keep = keep_rows(types, next_index)
    kept_src = [r for r in range(kv_len) if keep[int(tok_idx[r])]]
    n = len(kept_src)
    k2, v2 = k.copy(), v.copy()
    tok2, pos2 = tok_idx.copy(), pos_ids.copy()
    for dst, src in enumerate(kept_src):
        k2[:, dst] = k[:, src]
        v2[:, dst] = v[:, src]
        tok2[dst] = tok_idx[src]
        pos2[dst] = pos_ids[src]
    return k2, v2, tok2, pos2, n, np.asarray(kept_src, dtype=np.int64)


def decode_attention(q, k_new, v_new, k_cache, v_cache, kv_len, is_cl, scale=None):
    """One generated token attending to a (compacted) cache plus itself.

    q, k_new, v_new: [H, d]; k_cache, v_cache: [H, >=kv_len, d].  Plain
    softmax attention over rows [0, kv_len) and the new row (the cache holds
    only rows that every later token may see, so no mask is needed).  A <CL>
    token attends to itself only (reading R7).
    """
    q = np.asarray(q, np.float64)
    kn = np.asarray(k_new, np.float64)
    vn = np.asarray(v_new, np.float64)
    if is_cl:
        return vn.copy()
    H, d = q.shape
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    K = np.concatenate([np.asarray(k_cache[:, :kv_len], np.float64), kn[:, None]], axis=1)
    V = np.concatenate([np.asarray(v_cache[:, :kv_len], np.float64), vn[:, None]], axis=1)
    s = scale * np.einsum("hd,hjd->hj", q, K)
    s = s - s.max(axis=-1, keepdims=True)
    p = np.exp(s)
    p = p / p.sum(axis=-1, keepdims=True)
    return np.einsum("hj,hjd->hd", p, V)


# ---------------------------------------------------------------------------
# Composition: prefix -> free in one go -> generate (Section 3, Section 4.3)
# ---------------------------------------------------------------------------

def run_prompt_and_decode(q, k, v, types_all, L, steps, scale=None, theta=0.0,
                          compact_after=None):
    """Reference for one sequence of the whole path.

    q, k, v: [H, L + steps, d] raw (unrotated) projections for every token of
    the transformed sequence; ``types_all`` covers all L + steps indices.
    The prompt [0, L) goes through masked attention; the cache is then
    compacted at next index L; each generated token t >= L attends to the
    compacted cache plus itself, is appended unless it is a <CL>, and the
    cache is compacted again after every index in ``compact_after``.

    Returns (prompt_out [H, L, d], step_outs [steps, H, d], final cache
    tuple (k, v, tok, pos, kv_len)).
    """
    H, T, d = q.shape
    pos = tie_positions(types_all)
    if theta > 0:
        q = np.stack([rope_rotate_half(q[h], pos, theta) for h in range(H)])
        k = np.stack([rope_rotate_half(k[h], pos, theta) for h in range(H)])
    else:
        q = np.asarray(q, np.float64)
        k = np.asarray(k, np.float64)
    v = np.asarray(v, np.float64)
    mask = attention_mask(types_all[:L])
    out_prompt = masked_attention(q[:, :L], k[:, :L], v[:, :L], mask, scale)
    cap = T
    kc = np.zeros((H, cap, d))
    vc = np.zeros((H, cap, d))
    kc[:, :L], vc[:, :L] = k[:, :L], v[:, :L]
    tok = np.zeros(cap, np.int64)
    tok[:L] = np.arange(L)
    pp = np.zeros(cap, np.int64)
    pp[:L] = pos[:L]
    kc, vc, tok, pp, n, _ = compact_cache(kc, vc, tok, pp, L, types_all, L)
    outs = []
    compact_after = set(compact_after or [])
    for t in range(L, L + steps):
        is_cl = types_all[t] == CL
        outs.append(decode_attention(q[:, t], k[:, t], v[:, t], kc, vc, n, is_cl, scale))
        if not is_cl:
            kc[:, n], vc[:, n] = k[:, t], v[:, t]
            tok[n], pp[n] = t, pos[t]
            n += 1
        if t in compact_after:
            kc, vc, tok, pp, n, _ = compact_cache(kc, vc, tok, pp, n, types_all, t + 1)
    return out_prompt, np.stack(outs) if outs else np.zeros((0, H, d)), (kc, vc, tok, pp, n)
