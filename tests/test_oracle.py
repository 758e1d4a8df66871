"""Pins for the CPU oracle: each check ties the oracle to something other
than itself (a hand-derived example, a library routine on a special case,
a closed form, an independent formulation, brute force on tiny inputs)."""
import itertools
import math
import os

import numpy as np
import pytest
import torch

from oracle import sckv_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "mask_two_spans_L12.txt")
INF = np.iinfo(np.int64).max


# ---------------------------------------------------------------------------
# helpers written independently of the oracle
# ---------------------------------------------------------------------------

def load_golden():
    g = {"rows": {}, "keep": {}}
    with open(GOLDEN) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, _, rest = line.partition(" ")
            if key == "spans":
                g["spans"] = [tuple(int(x) for x in s.split(":")) for s in rest.split()]
            elif key == "types":
                g["types"] = [{"N": O.NORMAL, "CL": O.CL, "CR": O.CR}[x] for x in rest.split()]
            elif key == "row":
                i, _, cols = rest.partition(":")
                g["rows"][int(i)] = [int(x) for x in cols.split()]
            elif key == "pos":
                g["pos"] = [int(x) for x in rest.split()]
            elif key == "keep":
                p, _, cols = rest.partition(":")
                g["keep"][int(p)] = [int(x) for x in cols.split()]
    return g


def vu_from_spans(spans, L):
    """Closed form, independent of the oracle: the last row that may see
    column j (j itself for a <CL>, the closing <CR> for an enclosed token,
    'forever' otherwise)."""
    vu = np.full(L, INF, dtype=np.int64)
    for c, r in spans:
        if c < L:
            vu[c] = c
        for j in range(c + 1, min(r, L)):
            vu[j] = r
    return vu


def closed_form_mask(spans, L):
    vu = vu_from_spans(spans, L)
    i = np.arange(L)[:, None]
    j = np.arange(L)[None, :]
    is_cl_row = (vu == np.arange(L))[:, None]
    return (j <= i) & (i <= vu[None, :]) & (~is_cl_row | (i == j))


def all_span_sets(L, allow_open=True):
    """Every set of non-overlapping spans (c < r, c_{k+1} > r_k) inside a
    sequence of length L; the last span may be open (r >= L)."""
    out = []

    def rec(start, acc):
        out.append(list(acc))
        for c in range(start, L):
            for r in range(c + 1, L):
                rec(r + 1, acc + [(c, r)])
            if allow_open:
                out.append(acc + [(c, L + 3)])

    rec(0, [])
    return out


def sdpa_causal(q, k, v):
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a, np.float64))
    o = torch.nn.functional.scaled_dot_product_attention(t(q)[None], t(k)[None], t(v)[None],
                                                         is_causal=True)
    return o[0].numpy()


def rnd(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


# ---------------------------------------------------------------------------
# hand-derived example (plays the role of the missing Figure 1)
# ---------------------------------------------------------------------------

def check_golden():
    g = load_golden()
    L = len(g["types"])
    types = O.token_types(g["spans"], L)
    assert list(types) == g["types"]
    m = O.attention_mask(types)
    for i in range(L):
        assert list(np.nonzero(m[i])[0]) == g["rows"][i], f"row {i}"
    assert list(O.tie_positions(types)) == g["pos"]
    for P, cols in g["keep"].items():
        keep = O.keep_rows(types, P)
        assert [t for t in range(P) if keep[t]] == cols, f"keep at {P}"


def test_golden_example():
    check_golden()


# ---------------------------------------------------------------------------
# P1 / P4: special cases that reduce to a library routine
# ---------------------------------------------------------------------------

def check_no_spans_is_causal():
    H, L, d = 3, 40, 16
    q, k, v = rnd((H, L, d), 1), rnd((H, L, d), 2), rnd((H, L, d), 3)
    m = O.attention_mask(O.token_types([], L))
    o = O.masked_attention(q, k, v, m)
    np.testing.assert_allclose(o, sdpa_causal(q, k, v), rtol=0, atol=1e-12)


def test_no_spans_is_causal_attention():
    check_no_spans_is_causal()


def test_rows_before_first_cl_are_causal():
    H, L, d = 2, 64, 8
    spans = [(20, 30), (40, 50)]
    q, k, v = rnd((H, L, d), 4), rnd((H, L, d), 5), rnd((H, L, d), 6)
    o = O.masked_attention(q, k, v, O.attention_mask(O.token_types(spans, L)))
    ref = sdpa_causal(q, k, v)
    np.testing.assert_allclose(o[:, :20], ref[:, :20], rtol=0, atol=1e-12)
    assert np.abs(o[:, 31:] - ref[:, 31:]).max() > 1e-3   # the mask does bite later


# ---------------------------------------------------------------------------
# P2: brute force over every span set on tiny sequences
# ---------------------------------------------------------------------------

def check_bruteforce_masks(Lmax=8):
    count = 0
    for L in range(1, Lmax + 1):
        for spans in all_span_sets(L):
            types = O.token_types(spans, L)
            m = O.attention_mask(types)
            assert np.array_equal(m, closed_form_mask(spans, L)), (L, spans)
            # every row sees at least itself: no empty softmax
            assert m[np.arange(L), np.arange(L)].all()
            count += 1
    return count


def test_bruteforce_mask_equals_closed_form():
    n = check_bruteforce_masks(8)
    assert n > 500


def test_mask_rows_equal_closed_form_and_sampled_attention():
    """attention_mask_rows (for sequences too long for the whole mask) gives
    the closed-form rows on every span set up to L=8, in any row order, and
    attention over sampled query rows equals those rows of the full result."""
    for L in range(1, 9):
        for spans in all_span_sets(L):
            types = O.token_types(spans, L)
            rows = list(range(L - 1, -1, -1))
            assert np.array_equal(O.attention_mask_rows(types, rows),
                                  closed_form_mask(spans, L)[rows]), (L, spans)
    H, L, d = 2, 300, 8
    spans = [(3, 40), (50, 51), (60, 200), (250, 400)]
    types = O.token_types(spans, L)
    q, k, v = rnd((H, L, d), 21), rnd((H, L, d), 22), rnd((H, L, d), 23)
    full = O.masked_attention(q, k, v, O.attention_mask(types))
    rows = [0, 3, 39, 40, 41, 60, 199, 200, 201, 250, 299]
    part = O.masked_attention(q[:, rows], k, v, O.attention_mask_rows(types, rows))
    np.testing.assert_allclose(part, full[:, rows], rtol=0, atol=1e-12)


def test_bruteforce_keep_rule_and_closed_length():
    for L in range(1, 9):
        for spans in all_span_sets(L):
            types = O.token_types(spans, L)
            for P in range(0, L + 1):
                keep = O.keep_rows(types, P)
                kept = sum(keep[:P])
                closed = P - sum(r - c for c, r in spans if r < P) \
                    - sum(1 for c, r in spans if c < P <= r)
                assert kept == closed, (L, spans, P)


def test_bruteforce_outputs_against_loop_softmax():
    rng = np.random.default_rng(7)
    H, d = 1, 3
    for L in range(1, 7):
        for spans in all_span_sets(L)[::3]:
            q, k, v = (rng.standard_normal((H, L, d)) for _ in range(3))
            types = O.token_types(spans, L)
            o = O.masked_attention(q, k, v, O.attention_mask(types))
            cf = closed_form_mask(spans, L)
            for i in range(L):
                vis = [j for j in range(L) if cf[i, j]]
                w = [math.exp(sum(q[0, i, t] * k[0, j, t] for t in range(d)) / math.sqrt(d))
                     for j in vis]
                z = sum(w)
                for t in range(d):
                    ref = sum(wj * v[0, j, t] for wj, j in zip(w, vis)) / z
                    assert abs(o[0, i, t] - ref) < 1e-12


# ---------------------------------------------------------------------------
# P3, P5, P9: exact consequences of the mask
# ---------------------------------------------------------------------------

def test_cl_rows_output_their_own_value():
    H, L, d = 2, 50, 8
    spans = [(3, 9), (15, 16), (17, 30), (44, 60)]
    q, k, v = rnd((H, L, d), 8), rnd((H, L, d), 9), rnd((H, L, d), 10)
    o = O.masked_attention(q, k, v, O.attention_mask(O.token_types(spans, L)))
    for c, _ in spans:
        assert np.array_equal(o[:, c], v[:, c])


def check_eviction_invariance():
    H, L, d = 2, 60, 8
    spans = [(5, 12), (20, 21), (22, 40)]
    q, k, v = rnd((H, L, d), 11), rnd((H, L, d), 12), rnd((H, L, d), 13)
    m = O.attention_mask(O.token_types(spans, L))
    base = O.masked_attention(q, k, v, m)
    for c, r in spans:
        k2, v2 = k.copy(), v.copy()
        k2[:, c:r] = 1e4 * np.sign(rnd((H, r - c, d), 99))
        v2[:, c:r] = -1e4
        o2 = O.masked_attention(q, k2, v2, m)
        assert np.array_equal(o2[:, r + 1:], base[:, r + 1:]), (c, r)
        assert not np.array_equal(o2[:, c:r + 1], base[:, c:r + 1])


def test_eviction_invariance():
    check_eviction_invariance()


def test_probabilities_and_convex_hull():
    H, L, d = 2, 48, 6
    spans = [(4, 10), (12, 30)]
    q, k, v = rnd((H, L, d), 14), rnd((H, L, d), 15), rnd((H, L, d), 16)
    m = O.attention_mask(O.token_types(spans, L))
    o, p = O.masked_attention(q, k, v, m, return_probs=True)
    np.testing.assert_allclose(p.sum(-1), 1.0, atol=1e-12)
    assert (p[:, ~m] == 0).all()
    for h in range(H):
        for i in range(L):
            vis = v[h, m[i]]
            assert (o[h, i] >= vis.min(0) - 1e-12).all() and (o[h, i] <= vis.max(0) + 1e-12).all()


# ---------------------------------------------------------------------------
# P6: masked full-cache attention == attention over the compacted cache
# ---------------------------------------------------------------------------

def compacted_row(q, k, v, types, i, pos=None, theta=0.0, pos_override=None):
    """Row i computed the compaction way: compact rows [0, i) at next index i,
    then decode token i against it."""
    H, L, d = k.shape
    tok = np.arange(L)
    pp = np.zeros(L, np.int64) if pos is None else pos.copy()
    k2, v2, tok2, _, n, _ = O.compact_cache(k, v, tok, pp, i, types, i)
    qi, ki = q[:, i], k[:, i]
    if theta > 0:
        kpos = pos[tok2[:n]] if pos_override is None else pos_override(n)
        kr = np.stack([O.rope_rotate_half(k2[h, :n], kpos, theta) for h in range(H)])
        qpos = np.array([pos[i] if pos_override is None else n])
        qi = np.stack([O.rope_rotate_half(q[h, i][None], qpos, theta)[0] for h in range(H)])
        ki = np.stack([O.rope_rotate_half(k[h, i][None], qpos, theta)[0] for h in range(H)])
        k2 = np.concatenate([kr, k2[:, n:]], axis=1)
    return O.decode_attention(qi, ki, v[:, i], k2, v2, n, types[i] == O.CL)


def check_masked_equals_compacted(theta=0.0):
    H, L, d = 2, 96, 8
    rng = np.random.default_rng(17)
    spans = [(2, 9), (10, 11), (12, 40), (50, 70), (80, 120)]
    types = O.token_types(spans, L)
    q, k, v = (rng.standard_normal((H, L, d)) for _ in range(3))
    pos = O.tie_positions(types)
    if theta > 0:
        qr = np.stack([O.rope_rotate_half(q[h], pos, theta) for h in range(H)])
        kr = np.stack([O.rope_rotate_half(k[h], pos, theta) for h in range(H)])
    else:
        qr, kr = q, k
    full = O.masked_attention(qr, kr, v, O.attention_mask(types))
    for i in range(L):
        row = compacted_row(q, k, v, types, i, pos, theta)
        np.testing.assert_allclose(row, full[:, i], rtol=0, atol=1e-10, err_msg=f"row {i}")


def test_masked_full_cache_equals_compacted_cache():
    check_masked_equals_compacted(0.0)


def test_masked_equals_compacted_with_rope_at_tied_positions():
    check_masked_equals_compacted(10000.0)


def test_rope_at_compacted_row_index_is_wrong():
    """Negative check: rotating keys by their compacted row index instead of
    their original position breaks the equality."""
    H, L, d = 1, 64, 8
    rng = np.random.default_rng(18)
    spans = [(4, 30)]
    types = O.token_types(spans, L)
    q, k, v = (rng.standard_normal((H, L, d)) for _ in range(3))
    pos = O.tie_positions(types)
    qr = np.stack([O.rope_rotate_half(q[h], pos, 10000.0) for h in range(H)])
    kr = np.stack([O.rope_rotate_half(k[h], pos, 10000.0) for h in range(H)])
    full = O.masked_attention(qr, kr, v, O.attention_mask(types))
    i = 50
    bad = compacted_row(q, k, v, types, i, pos, 10000.0, pos_override=lambda n: np.arange(n))
    assert np.abs(bad - full[:, i]).max() > 1e-3


# ---------------------------------------------------------------------------
# P7: compaction laws
# ---------------------------------------------------------------------------

def _cache(L, H=2, d=4, seed=19):
    rng = np.random.default_rng(seed)
    k, v = rng.standard_normal((H, L, d)), rng.standard_normal((H, L, d))
    return k, v, np.arange(L), rng.integers(0, 1000, L)


def test_compaction_idempotent_and_incremental():
    L = 120
    spans = [(3, 10), (11, 12), (20, 50), (60, 61), (70, 100), (110, 140)]
    types = O.token_types(spans, 140)
    k, v, tok, pos = _cache(L)
    one = O.compact_cache(k, v, tok, pos, L, types, L)
    assert np.all(np.diff(one[5]) > 0)
    two = O.compact_cache(*one[:4], one[4], types, L)
    assert two[4] == one[4] and np.array_equal(two[0][:, :two[4]], one[0][:, :one[4]])
    for P1 in [0, 5, 11, 13, 51, 99, 101, 120]:
        a = O.compact_cache(k, v, tok, pos, P1, types, P1)
        # the rows P1..L-1 are appended to the partially compacted cache
        n = a[4]
        k3, v3, t3, p3 = a[0].copy(), a[1].copy(), a[2].copy(), a[3].copy()
        k3[:, n:n + L - P1], v3[:, n:n + L - P1] = k[:, P1:], v[:, P1:]
        t3[n:n + L - P1], p3[n:n + L - P1] = tok[P1:], pos[P1:]
        b = O.compact_cache(k3, v3, t3, p3, n + L - P1, types, L)
        assert b[4] == one[4]
        assert np.array_equal(b[0][:, :b[4]], one[0][:, :one[4]])
        assert np.array_equal(b[2][:b[4]], one[2][:one[4]])
        assert np.array_equal(b[3][:b[4]], one[3][:one[4]])


# ---------------------------------------------------------------------------
# tie rule properties
# ---------------------------------------------------------------------------

def test_tie_positions_properties():
    rng = np.random.default_rng(20)
    for _ in range(50):
        L = int(rng.integers(1, 80))
        spans, c = [], int(rng.integers(0, 4))
        while c < L:
            r = c + int(rng.integers(1, 12))
            spans.append((c, r))
            c = r + 1 + int(rng.integers(0, 5))
        types = O.token_types(spans, L)
        pos = O.tie_positions(types)
        normal = np.nonzero(types == O.NORMAL)[0]
        assert list(pos[normal]) == list(range(len(normal)))
        for t in np.nonzero(types != O.NORMAL)[0]:
            assert pos[t] == (pos[t - 1] if t > 0 else 0)


# ---------------------------------------------------------------------------
# P8: rotary embedding
# ---------------------------------------------------------------------------

def check_rope():
    rng = np.random.default_rng(21)
    n, d, theta = 17, 10, 10000.0
    x = rng.standard_normal((n, d))
    pos = rng.integers(0, 5000, n)
    # identity at position 0
    np.testing.assert_array_equal(O.rope_rotate_half(x, np.zeros(n, int), theta), x)
    # complex-number formulation: (x1 + i x2) * exp(i * pos * w)
    half = d // 2
    w = np.array([theta ** (-2.0 * i / d) for i in range(half)])
    z = (x[:, :half] + 1j * x[:, half:]) * np.exp(1j * pos[:, None] * w[None])
    ref = np.concatenate([z.real, z.imag], axis=1)
    np.testing.assert_allclose(O.rope_rotate_half(x, pos, theta), ref, atol=1e-12)
    # d = 2 is a plain rotation by pos radians
    y = rng.standard_normal((n, 2))
    ang = pos.astype(float)
    rot = np.stack([y[:, 0] * np.cos(ang) - y[:, 1] * np.sin(ang),
                    y[:, 0] * np.sin(ang) + y[:, 1] * np.cos(ang)], axis=1)
    np.testing.assert_allclose(O.rope_rotate_half(y, pos, theta), rot, atol=1e-12)
    # relative: q(m) . k(n) depends on m - n only
    q, k = rng.standard_normal(d), rng.standard_normal(d)
    a = O.rope_rotate_half(q[None], [100], theta) @ O.rope_rotate_half(k[None], [40], theta).T
    b = O.rope_rotate_half(q[None], [1100], theta) @ O.rope_rotate_half(k[None], [1040], theta).T
    np.testing.assert_allclose(a, b, atol=1e-10)


def test_rope():
    check_rope()


# ---------------------------------------------------------------------------
# decode and the whole composition
# ---------------------------------------------------------------------------

def test_decode_cl_step_outputs_own_value():
    rng = np.random.default_rng(22)
    q, kn, vn = (rng.standard_normal((3, 8)) for _ in range(3))
    kc, vc = rng.standard_normal((3, 10, 8)), rng.standard_normal((3, 10, 8))
    assert np.array_equal(O.decode_attention(q, kn, vn, kc, vc, 10, True), vn)


def test_decode_with_empty_cache_outputs_new_value():
    rng = np.random.default_rng(23)
    q, kn, vn = (rng.standard_normal((3, 8)) for _ in range(3))
    z = np.zeros((3, 4, 8))
    np.testing.assert_allclose(O.decode_attention(q, kn, vn, z, z, 0, False), vn, atol=1e-15)


def check_streaming_equals_full_mask(theta):
    H, d = 2, 8
    L, steps = 40, 60
    T = L + steps
    spans = [(5, 15), (30, 45), (50, 52), (60, 75), (90, 120)]
    types = O.token_types(spans, T)
    rng = np.random.default_rng(24)
    q, k, v = (rng.standard_normal((H, T, d)) for _ in range(3))
    cr_steps = [r for _, r in spans if L <= r < T]
    prompt, outs, _ = O.run_prompt_and_decode(q, k, v, types, L, steps, theta=theta,
                                              compact_after=cr_steps)
    pos = O.tie_positions(types)
    if theta > 0:
        q = np.stack([O.rope_rotate_half(q[h], pos, theta) for h in range(H)])
        k = np.stack([O.rope_rotate_half(k[h], pos, theta) for h in range(H)])
    full = O.masked_attention(q, k, v, O.attention_mask(types))
    np.testing.assert_allclose(prompt, full[:, :L], atol=1e-10)
    np.testing.assert_allclose(outs.transpose(1, 0, 2), full[:, L:], atol=1e-10)


def test_streaming_equals_full_mask():
    check_streaming_equals_full_mask(0.0)
    check_streaming_equals_full_mask(10000.0)


# ---------------------------------------------------------------------------
# the pins catch plausible mistakes planted in the oracle
# ---------------------------------------------------------------------------

def _mut_mask_cl_visible(types):
    m = ORIG_MASK(types)
    for i in range(len(types)):
        if types[i] != O.CL:
            m[i, :i + 1] |= (np.asarray(types[:i + 1]) == O.CL)
    return m


def _mut_mask_cr_blind(types):
    m = ORIG_MASK(types)
    enc = O.enclosing_cr(types)
    for i in range(len(types)):
        for j in range(i + 1):
            if enc[j] >= 0 and i >= enc[j]:
                m[i, j] = False
    return m


def _mut_tie_next(types):
    pos = np.zeros(len(types), np.int64)
    nxt = 0
    for t in range(len(types)):
        pos[t] = nxt
        if types[t] == O.NORMAL:
            nxt += 1
    return pos


def _mut_keep_cl(types, P):
    keep = ORIG_KEEP(types, P)
    keep[np.asarray(types) == O.CL] = True
    return keep


def _mut_rope_sign(x, pos, theta):
    # rotating the wrong way
    return ORIG_ROPE(x, -np.asarray(pos), theta)


def _mut_no_scale(q, k, v, mask, scale=None, return_probs=False):
    return ORIG_ATTN(q, k, v, mask, 1.0, return_probs)


ORIG_MASK = O.attention_mask
ORIG_KEEP = O.keep_rows
ORIG_ROPE = O.rope_rotate_half
ORIG_ATTN = O.masked_attention


@pytest.mark.parametrize("name,attr,fn,checks", [
    ("cl-visible", "attention_mask", _mut_mask_cl_visible, [check_golden, check_bruteforce_masks]),
    ("cr-blind", "attention_mask", _mut_mask_cr_blind, [check_golden, check_bruteforce_masks]),
    ("tie-next", "tie_positions", _mut_tie_next, [check_golden]),
    ("keep-cl", "keep_rows", _mut_keep_cl, [check_golden]),
    ("rope-sign", "rope_rotate_half", _mut_rope_sign, [check_rope]),
    ("no-scale", "masked_attention", _mut_no_scale, [check_no_spans_is_causal]),
])
def test_planted_mistakes_are_caught(monkeypatch, name, attr, fn, checks):
    monkeypatch.setattr(O, attr, fn)
    for chk in checks:
        with pytest.raises(AssertionError):
            chk(4) if chk is check_bruteforce_masks else chk()
