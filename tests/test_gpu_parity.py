"""GPU parity: the HIP path (through the C ABI) against the CPU oracle on the
same seeded inputs.  Integer/index/byte results must match bit for bit;
attention outputs within max-abs 2e-2 (bf16 inputs) or 1e-5 (fp32)."""
import math

import numpy as np
import pytest
import torch

from oracle import sckv_oracle as O

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
TOL = {"bf16": 2e-2, "f32": 1e-5}
INF = 0x7fffffff


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2310_08152_amd import binding  # noqa: F401  (fails loudly without the library)


def P():
    from paper_2310_08152_amd import path
    return path


def W():
    from paper_2310_08152_amd import workload
    return workload


def f64(t):
    return t.detach().to("cpu", torch.float64).numpy()


def rnd(shape, seed, dtype):
    return W().randn(shape, seed=seed, dtype=dtype).to(DEV)


def say(msg):
    print(msg, flush=True)


def random_spans(L, rng, max_len=40, gap=8, start_at_zero=False, open_end=False):
    out, c = [], 0 if start_at_zero else int(rng.integers(0, gap + 1))
    while c < L - 1:
        r = c + int(rng.integers(1, max_len + 1))
        if r >= L:
            if open_end:
                out.append((c, L + 5))
            break
        out.append((c, r))
        c = r + 1 + int(rng.integers(0, gap + 1))
    return out


def mask_from_vu(vu):
    L = len(vu)
    i = np.arange(L)[:, None]
    j = np.arange(L)[None, :]
    cl_row = (vu == np.arange(L))[:, None]
    return (j <= i) & (i <= vu[None, :].astype(np.int64)) & (~cl_row | (i == j))


# ---------------------------------------------------------------------------
# span metadata and tied positions
# ---------------------------------------------------------------------------

SPAN_CASES = {
    "none": (lambda L, rng: [], 77),
    "start-at-zero-adjacent": (lambda L, rng: [(0, 3), (4, 9), (10, 11), (12, 30)], 64),
    "open-end": (lambda L, rng: [(5, 20), (40, 300)], 100),
    "random": (lambda L, rng: random_spans(L, rng, open_end=True), 300),
    "random-long": (lambda L, rng: random_spans(L, rng, max_len=200, gap=50), 1500),
}


@pytest.mark.parametrize("case", list(SPAN_CASES))
def test_span_meta_matches_oracle(case):
    say(f"span_meta case={case}")
    gen, L = SPAN_CASES[case]
    rng = np.random.default_rng(5)
    spans = [gen(L, rng) for _ in range(3)]
    meta = P().SpanMeta(spans, L, DEV)
    vu = meta.vu.cpu().numpy()
    pos = meta.pos.cpu().numpy()
    for s, sp in enumerate(spans):
        types = O.token_types(sp, L)
        assert np.array_equal(pos[s], O.tie_positions(types)), s
        if L <= 400:
            assert np.array_equal(mask_from_vu(vu[s]), O.attention_mask(types)), s
        for Pn in [0, 1, L // 3, L // 2, L - 1, L]:
            keep = O.keep_rows(types, Pn)
            gpu_keep = (vu[s] != np.arange(L)) & (vu[s].astype(np.int64) >= Pn)
            assert np.array_equal(gpu_keep[:Pn], keep[:Pn]), (s, Pn)


# ---------------------------------------------------------------------------
# rotary embedding
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("dtype,d", [("bf16", 64), ("bf16", 80), ("f32", 64), ("f32", 80)])
def test_rope_matches_oracle(dtype, d):
    say(f"rope dtype={dtype} d={d}")
    L = 300
    spans = [[(3, 40), (50, 51), (60, 200)], [(0, 10)]]
    meta = P().SpanMeta(spans, L, DEV)
    x = rnd((2, 3, 257, d), 11, dtype)
    y = torch.empty_like(x)
    P().rope_rows(x, y, meta, n=257, tok0=20, theta=10000.0)
    z = x.clone()
    P().rope_rows(z, z, meta, n=257, tok0=20, theta=10000.0)          # in place
    assert torch.equal(y, z)
    c = torch.empty_like(x)
    P().rope_rows(x, c, meta, n=257, tok0=20, theta=0.0)              # copy
    assert torch.equal(c, x)
    X, Y = f64(x), f64(y)
    for s in range(2):
        pos = O.tie_positions(O.token_types(spans[s], L))[20:277]
        for h in range(3):
            ref = O.rope_rotate_half(X[s, h], pos, 10000.0)
            err = np.abs(Y[s, h] - ref)
            if dtype == "bf16":
                assert (err <= 2.0 ** -8 * np.abs(ref) + 1e-3).all(), err.max()
            else:
                assert err.max() < 1e-5


# ---------------------------------------------------------------------------
# prefill
# ---------------------------------------------------------------------------

def run_prefill(q, k, v, spans, L_meta=None):
    b, H, L, d = q.shape
    meta = P().SpanMeta(spans, L_meta or L, DEV)
    ws = P().Workspace(b, H, L, L, d, DEV)
    o = torch.full_like(q, float("nan"))
    P().prefill_layer(q, k, v, o, meta, ws, L)
    torch.cuda.synchronize()
    return o


def oracle_prefill(q, k, v, spans, heads=None):
    Q, K, V = f64(q), f64(k), f64(v)
    b, H, L, d = Q.shape
    out = {}
    for s in range(b):
        m = O.attention_mask(O.token_types(spans[s], L))
        hs = range(H) if heads is None else [h for (ss, h) in heads if ss == s]
        for h in hs:
            out[(s, h)] = O.masked_attention(Q[s, h][None], K[s, h][None], V[s, h][None], m)[0]
    return out


PREFILL_CASES = [
    # name, dtype, b, H, L, d, span generator
    ("tiny-f32-config", "f32", 1, 4, 256, 64, "tiny"),
    ("f32-d80-ragged", "f32", 1, 2, 200, 80, "random"),
    ("bf16-d64-windows", "bf16", 2, 4, 2048, 64, "windows"),
    ("bf16-d80-uniform-ragged", "bf16", 2, 2, 1000, 80, "uniform"),
    ("bf16-d64-nospans", "bf16", 1, 2, 333, 64, "none"),
    ("bf16-d64-L1", "bf16", 1, 1, 1, 64, "none"),
    ("bf16-d64-L37-zero-start", "bf16", 1, 3, 37, 64, "zero"),
    ("bf16-d80-L129-open", "bf16", 2, 1, 129, 80, "open"),
    ("bf16-d64-long-spans", "bf16", 1, 2, 700, 64, "long"),
    # (sequence, head) slices are dispatched in groups of 8: a full group and a
    # partial one, with an odd head count
    ("bf16-d80-12-slices", "bf16", 3, 4, 600, 80, "uniform"),
    ("bf16-d64-20-slices", "bf16", 4, 5, 513, 64, "random"),
]


def make_spans(kind, b, L, rng):
    w = W()
    if kind == "tiny":
        return [w.spans_periodic(L, 32, 8, 24) for _ in range(b)]
    if kind == "windows":
        return [w.spans_jittered_windows(L, 64, 16, 32, 4, rng) for _ in range(b)]
    if kind == "uniform":
        return [w.spans_uniform_lengths(L, 0.5, 16, 64, rng) for _ in range(b)]
    if kind == "none":
        return [[] for _ in range(b)]
    if kind == "zero":
        return [[(0, 5), (6, 7), (8, 20), (30, 50)] for _ in range(b)]
    if kind == "open":
        return [[(10, 60), (61, 62), (100, 150)], [(128, 140)]][:b]
    if kind == "long":
        return [[(5, 400), (401, 650)] for _ in range(b)]
    return [random_spans(L, rng, open_end=True) for _ in range(b)]


@pytest.mark.parametrize("name,dtype,b,H,L,d,kind", PREFILL_CASES, ids=[c[0] for c in PREFILL_CASES])
def test_prefill_matches_oracle(name, dtype, b, H, L, d, kind):
    say(f"prefill case={name} b={b} H={H} L={L} d={d} dtype={dtype}")
    rng = np.random.default_rng(L)
    spans = make_spans(kind, b, L, rng)
    q, k, v = (rnd((b, H, L, d), 100 + i, dtype) for i in range(3))
    o = run_prefill(q, k, v, spans)
    ref = oracle_prefill(q, k, v, spans)
    Og, V = f64(o), f64(v)
    worst = 0.0
    for (s, h), r in ref.items():
        worst = max(worst, np.abs(Og[s, h] - r).max())
        for c, _ in spans[s]:
            if c < L:  # a <CL> row is its own value row, bit for bit
                assert np.array_equal(Og[s, h, c], V[s, h, c]), (s, h, c)
    assert np.isfinite(Og).all()
    assert worst <= TOL[dtype], worst


@pytest.mark.parametrize("dtype,d", [("bf16", 80), ("f32", 64)])
def test_prefill_plan_reuse_bitexact(dtype, d):
    """One plan (sckv_prefill_plan) serves several layers: each planned call
    equals span_masked_prefill_attn, which rebuilds the plan, bit for bit."""
    say(f"prefill plan reuse dtype={dtype} d={d}")
    b, H, L = 2, 3, 777
    rng = np.random.default_rng(77)
    spans = make_spans("uniform", b, L, rng)
    meta = P().SpanMeta(spans, L, DEV)
    ws = P().Workspace(b, H, L, L, d, DEV)
    layers = [tuple(rnd((b, H, L, d), 400 + 10 * m + i, dtype) for i in range(3)) for m in range(3)]
    P().prefill_plan(meta, ws, b, L)
    planned = []
    for q, k, v in layers:
        o = torch.full_like(q, float("nan"))
        P().prefill_layer(q, k, v, o, meta, ws, L, planned=True)
        planned.append(o)
    torch.cuda.synchronize()
    for (q, k, v), o in zip(layers, planned):
        ref = run_prefill(q, k, v, spans)  # plans again, in its own workspace
        assert torch.equal(o, ref)
    # the last layer against the oracle as well
    q, k, v = layers[-1]
    worst = max(np.abs(f64(planned[-1])[s_, h] - r).max()
                for (s_, h), r in oracle_prefill(q, k, v, spans).items())
    assert worst <= TOL[dtype], worst


def test_prefill_eviction_invariance_bitexact():
    say("prefill eviction invariance")
    b, H, L, d = 2, 4, 1100, 64
    rng = np.random.default_rng(9)
    spans = make_spans("uniform", b, L, rng)
    q, k, v = (rnd((b, H, L, d), 200 + i, "bf16") for i in range(3))
    o1 = run_prefill(q, k, v, spans)
    k2, v2 = k.clone(), v.clone()
    for s in range(b):
        for c, r in spans[s]:
            k2[s, :, c:r] = 1e4
            v2[s, :, c:r] = -1e4
    o2 = run_prefill(q, k2, v2, spans)
    for s in range(b):
        inside = np.zeros(L, bool)
        for c, r in spans[s]:
            inside[c:min(r, L - 1) + 1] = True
        rows = torch.from_numpy(np.nonzero(~inside)[0]).to(DEV)
        assert torch.equal(o1[s][:, rows], o2[s][:, rows])
        assert not torch.equal(o1[s], o2[s])


def test_prefill_full_size_opt13b_sampled():
    """The OPT-1.3B-shaped prefill slice at full size, 8 sampled heads."""
    w = W().get_workload("opt1.3b-prefill")
    say(f"prefill full size {w}")
    spans = W().workload_spans(w)
    shape = (w.batch, w.heads, w.seq_len, w.d_head)
    q, k, v = (W().randn(shape, seed=w.seed * 10 + i, dtype="bf16", device=DEV) for i in range(3))
    o = run_prefill(q, k, v, spans)
    rng = np.random.default_rng(0)
    picks = [(int(rng.integers(w.batch)), int(rng.integers(w.heads))) for _ in range(8)]
    for s, h in picks:
        m = O.attention_mask(O.token_types(spans[s], w.seq_len))
        r = O.masked_attention(f64(q[s, h])[None], f64(k[s, h])[None], f64(v[s, h])[None], m)[0]
        assert np.abs(f64(o[s, h]) - r).max() <= TOL["bf16"]


# ---------------------------------------------------------------------------
# compaction
# ---------------------------------------------------------------------------

def build_cache(M, b, H, L_cap, d, dtype, L, spans, seed):
    meta = P().SpanMeta(spans, L_cap, DEV)
    cache = P().KVCache(M, b, H, L_cap, d, W().torch_dtype(dtype), DEV)
    cache.kv.copy_(W().randn(cache.kv.shape, seed=seed, dtype=dtype).to(DEV))
    cache.start_prompt(L, meta)
    return meta, cache


def bits(t):
    return t.view(torch.int16 if t.element_size() == 2 else torch.int32).cpu().numpy()


@pytest.mark.parametrize("dtype,d", [("bf16", 64), ("bf16", 80), ("f32", 64), ("f32", 80)])
def test_compaction_bitexact(dtype, d):
    say(f"compaction dtype={dtype} d={d}")
    M, b, H, L_cap = 2, 4, 3, 600
    L = 520
    rng = np.random.default_rng(21)
    spans = [random_spans(L, rng, open_end=True), [(0, 100), (101, 102), (200, 519)],
             [], [(5, 550)]]
    meta, cache = build_cache(M, b, H, L_cap, d, dtype, L, spans, 31)
    next_tok = torch.tensor([L, 300, L, 520], dtype=torch.int32, device=DEV)
    before = bits(cache.kv)
    tok0, pos0 = cache.tok_idx.cpu().numpy(), cache.pos_ids.cpu().numpy()
    ref_out = torch.zeros_like(cache.kv)
    # out of place first (kv untouched), then in place
    kv_len0 = cache.kv_len.clone()
    tok_save, pos_save = cache.tok_idx.clone(), cache.pos_ids.clone()
    cache.compact(meta, next_tok, kv_out=ref_out)
    assert np.array_equal(bits(cache.kv), before)
    oop_len = cache.kv_len.clone()
    cache.kv_len.copy_(kv_len0)
    cache.tok_idx.copy_(tok_save)
    cache.pos_ids.copy_(pos_save)
    cache.compact(meta, next_tok)
    torch.cuda.synchronize()
    assert torch.equal(oop_len, cache.kv_len)
    kvl = cache.kv_len.cpu().numpy()
    after = bits(cache.kv)
    oop = bits(ref_out)
    ks = cache.kept_src.cpu().numpy()
    tok, pos = cache.tok_idx.cpu().numpy(), cache.pos_ids.cpu().numpy()
    for s in range(b):
        types = O.token_types(spans[s], L_cap)
        k_ = before[:, 0, s]
        v_ = before[:, 1, s]
        res = O.compact_cache(k_.reshape(-1, L_cap, d), v_.reshape(-1, L_cap, d), tok0[s], pos0[s],
                              L, types, int(next_tok[s]))
        n = res[4]
        assert kvl[s] == n
        assert np.array_equal(ks[s, :n], res[5]) and (ks[s, n:] == -1).all()
        assert np.array_equal(tok[s, :n], res[2][:n])
        assert np.array_equal(pos[s, :n], res[3][:n])
        got_k = after[:, 0, s].reshape(-1, L_cap, d)[:, :n]
        got_v = after[:, 1, s].reshape(-1, L_cap, d)[:, :n]
        assert np.array_equal(got_k, res[0][:, :n]) and np.array_equal(got_v, res[1][:, :n])
        assert np.array_equal(oop[:, :, s, :, :n], after[:, :, s, :, :n])
    # idempotent
    cache.compact(meta, next_tok)
    torch.cuda.synchronize()
    assert np.array_equal(cache.kv_len.cpu().numpy(), kvl)
    assert np.array_equal(bits(cache.kv), after)


def test_compaction_incremental_equals_one_shot():
    say("compaction incremental")
    M, b, H, L_cap, d = 1, 2, 2, 400, 64
    L = 400
    rng = np.random.default_rng(3)
    spans = [random_spans(L, rng), random_spans(L, rng, start_at_zero=True)]
    meta, one = build_cache(M, b, H, L_cap, d, "bf16", L, spans, 41)
    _, inc = build_cache(M, b, H, L_cap, d, "bf16", L, spans, 41)
    one.compact(meta, torch.full((b,), L, dtype=torch.int32, device=DEV))
    for Pn in [50, 120, 121, 260, 399, 400]:
        inc.compact(meta, torch.full((b,), Pn, dtype=torch.int32, device=DEV))
    torch.cuda.synchronize()
    assert torch.equal(one.kv_len, inc.kv_len)
    n = int(one.kv_len.max())
    for s in range(b):
        ns = int(one.kv_len[s])
        assert torch.equal(one.kv[:, :, s, :, :ns], inc.kv[:, :, s, :, :ns])
        assert torch.equal(one.tok_idx[s, :ns], inc.tok_idx[s, :ns])
    assert n > 0


# ---------------------------------------------------------------------------
# decode
# ---------------------------------------------------------------------------

# The launch shape follows the number of (sequence, head) slices: H=3 gives
# 24 slices, split into chunks merged by a second kernel; from H=64 (512
# slices) on, one workgroup per slice: bf16 with 4 waves at 512 slices, 2 at
# 1024, 1 (d=64) or 2 (d=80) at 2048 (H=256), and 4 again at 4096 (H=512),
# past what one round of the chip holds; fp32 512 or 256 threads.
@pytest.mark.parametrize("dtype,d,theta,H", [("bf16", 64, 0.0, 3), ("bf16", 80, 10000.0, 3),
                                             ("f32", 64, 0.0, 3), ("f32", 80, 10000.0, 3),
                                             ("bf16", 80, 10000.0, 64), ("f32", 64, 0.0, 64),
                                             ("bf16", 64, 0.0, 128), ("f32", 80, 10000.0, 128),
                                             ("bf16", 64, 10000.0, 256), ("bf16", 80, 10000.0, 256),
                                             ("bf16", 64, 0.0, 512)])
def test_decode_matches_oracle(dtype, d, theta, H):
    say(f"decode dtype={dtype} d={d} theta={theta} H={H}")
    L_cap = 700
    lens = [0, 1, 255, 256, 257, 511, 600, 699]
    b = len(lens)
    spans = [[(650, 660)] for _ in range(b)]
    meta = P().SpanMeta(spans, 1000, DEV)
    cache = P().KVCache(1, b, H, L_cap, d, W().torch_dtype(dtype), DEV)
    cache.kv.copy_(W().randn(cache.kv.shape, seed=51, dtype=dtype).to(DEV))
    cache.kv_len.copy_(torch.tensor(lens, dtype=torch.int32))
    toks = [700 + i for i in range(b)]
    toks[2] = 650  # a <CL> step
    cache.cur_tok.copy_(torch.tensor(toks, dtype=torch.int32))
    ws = P().Workspace(b, H, 1, L_cap, d, DEV)
    q, kn, vn = (rnd((b, H, d), 60 + i, dtype) for i in range(3))
    o = torch.empty_like(q)
    before = cache.kv.clone()
    P().decode_layer(q, kn, vn, cache, 0, meta, ws, o, theta=theta)
    torch.cuda.synchronize()
    assert int(cache.status) == 0
    assert torch.equal(cache.kv_len.cpu(), torch.tensor(lens, dtype=torch.int32))
    Q, KN, VN, K, V, Og = f64(q), f64(kn), f64(vn), f64(before[0, 0]), f64(before[0, 1]), f64(o)
    Kafter = f64(cache.kv[0, 0])
    for s in range(b):
        types = O.token_types(spans[s], 1000)
        t = toks[s]
        is_cl = types[t] == O.CL
        qs, ks = Q[s], KN[s]
        if theta > 0:
            p = [O.tie_positions(types)[t]]
            qs = np.stack([O.rope_rotate_half(Q[s, h][None], p, theta)[0] for h in range(H)])
            ks = np.stack([O.rope_rotate_half(KN[s, h][None], p, theta)[0] for h in range(H)])
        ref = O.decode_attention(qs, ks, VN[s], K[s], V[s], lens[s], is_cl)
        if is_cl:
            assert np.array_equal(Og[s], VN[s])
            assert torch.equal(cache.kv[:, :, s], before[:, :, s])
        else:
            assert np.abs(Og[s] - ref).max() <= TOL[dtype], (s, np.abs(Og[s] - ref).max())
            n = lens[s]
            assert np.array_equal(f64(cache.kv[0, 1, s, :, n]), VN[s])
            kerr = np.abs(Kafter[s, :, n] - ks)
            assert kerr.max() <= (2e-2 if dtype == "bf16" else 1e-5)
            assert torch.equal(cache.kv[:, :, s, :, :n], before[:, :, s, :, :n])


# A cache of at least 512 rows per wave of a slice has both first blocks of
# every wave read before the slice length is known: L_cap=2100 at 4 waves and
# L_cap=600 at one wave (H=256, d=64) read past the short slices too.
@pytest.mark.parametrize("dtype,H,d,L_cap", [("bf16", 3, 80, 600), ("bf16", 64, 80, 600),
                                             ("bf16", 128, 80, 600), ("f32", 64, 80, 600),
                                             ("bf16", 256, 64, 600), ("bf16", 64, 80, 2100)])
def test_decode_ignores_rows_past_the_slice(dtype, H, d, L_cap):
    """Rows at or past kv_len may hold anything (never written, or NaN/Inf
    bit patterns): the output over short and long slices must not change."""
    say(f"decode past-the-slice rows dtype={dtype} H={H} d={d} L_cap={L_cap}")
    lens = [0, 1, 31, 37, 100, 255, 256, L_cap - 1]
    b = len(lens)
    meta = P().SpanMeta([[] for _ in range(b)], 1000, DEV)
    cache = P().KVCache(1, b, H, L_cap, d, W().torch_dtype(dtype), DEV)
    cache.kv.copy_(W().randn(cache.kv.shape, seed=71, dtype=dtype).to(DEV))
    clean = cache.kv.clone()
    for s_, n in enumerate(lens):   # poison every row past the slice
        cache.kv[:, 0, s_, :, n:] = float("nan")
        cache.kv[:, 1, s_, :, n:] = float("inf")
    cache.kv_len.copy_(torch.tensor(lens, dtype=torch.int32))
    cache.cur_tok.copy_(torch.tensor([700 + i for i in range(b)], dtype=torch.int32))
    ws = P().Workspace(b, H, 1, L_cap, d, DEV)
    q, kn, vn = (rnd((b, H, d), 80 + i, dtype) for i in range(3))
    o = torch.empty_like(q)
    P().decode_layer(q, kn, vn, cache, 0, meta, ws, o, theta=0.0)
    torch.cuda.synchronize()
    assert int(cache.status) == 0
    assert torch.isfinite(o).all()
    Q, KN, VN, K, V, Og = f64(q), f64(kn), f64(vn), f64(clean[0, 0]), f64(clean[0, 1]), f64(o)
    for s_, n in enumerate(lens):
        ref = O.decode_attention(Q[s_], KN[s_], VN[s_], K[s_], V[s_], n, False)
        assert np.abs(Og[s_] - ref).max() <= TOL[dtype], (s_, n)


@pytest.mark.parametrize("dtype,H", [("bf16", 2), ("bf16", 256), ("bf16", 512), ("f32", 512)])
def test_decode_reports_capacity_and_token_errors(dtype, H):
    say(f"decode status dtype={dtype} H={H}")
    L_cap, d = 64, 64
    meta = P().SpanMeta([[], []], 100, DEV)
    cache = P().KVCache(1, 2, H, L_cap, d, W().torch_dtype(dtype), DEV)
    cache.kv.zero_()
    cache.kv_len.copy_(torch.tensor([L_cap, 3], dtype=torch.int32))
    cache.cur_tok.copy_(torch.tensor([10, 100], dtype=torch.int32))
    ws = P().Workspace(2, H, 1, L_cap, d, DEV)
    q = rnd((2, H, d), 1, dtype)
    o = torch.zeros_like(q)
    P().decode_layer(q, q, q, cache, 0, meta, ws, o)
    torch.cuda.synchronize()
    st = int(cache.status)
    assert st & 1 and st & 2
    assert torch.isnan(o.float()).all()
    assert int(cache.kv.abs().sum()) == 0
    cache.commit(meta)
    torch.cuda.synchronize()
    assert cache.kv_len.tolist() == [L_cap, 3]
    assert cache.cur_tok.tolist() == [11, 101]


# ---------------------------------------------------------------------------
# the whole path on a small RoPE model: masked full cache == compacted cache
# ---------------------------------------------------------------------------

E2E_CASES = {
    # prompt spans, spans crossing the prompt end, spans closing mid-generation
    "mixed-bf16-rope": ("bf16", 80, 10000.0, 300, 100,
                        [[(10, 50), (51, 52), (120, 250), (290, 330), (340, 341), (345, 380),
                          (390, 420)],
                         [(0, 299), (305, 340), (360, 361)]]),
    "mixed-f32": ("f32", 64, 0.0, 300, 100,
                  [[(10, 50), (51, 52), (120, 250), (290, 330), (340, 341), (345, 380),
                    (390, 420)],
                   [(0, 299), (305, 340), (360, 361)]]),
    # the streaming schedule: no prompt spans, <CL> at +8 and <CR> at +40 of
    # every 48 generated tokens, compaction right after each <CR>
    "streaming-bf16-rope": ("bf16", 80, 10000.0, 64, 200, "stream"),
}


@pytest.mark.parametrize("case", list(E2E_CASES))
def test_end_to_end_prompt_compact_decode(case):
    dtype, d, theta, L, steps, spans = E2E_CASES[case]
    say(f"end to end case={case}")
    M, b, H = 2, 2, 2
    T = L + steps
    if spans == "stream":
        spans = [W().spans_streaming(L, steps, 48, 8, 40) for _ in range(b)]
    types = [O.token_types(sp, T) for sp in spans]
    cr_steps = sorted({r for sp in spans for _, r in sp if L <= r < T})
    q, k, v = (rnd((M, b, H, T, d), 300 + i, dtype) for i in range(3))
    meta = P().SpanMeta(spans, T, DEV)
    cache = P().KVCache(M, b, H, T, d, W().torch_dtype(dtype), DEV)
    ws = P().Workspace(b, H, L, T, d, DEV)
    cache.start_prompt(L, meta)
    outs_prompt = []
    for m in range(M):
        qr = torch.empty(b, H, L, d, dtype=q.dtype, device=DEV)
        P().rope_rows(q[m, :, :, :L], qr, meta, L, 0, theta)
        P().rope_rows(k[m, :, :, :L], cache.k(m), meta, L, 0, theta)
        P().rope_rows(v[m, :, :, :L], cache.v(m), meta, L, 0, 0.0)
        o = torch.empty_like(qr)
        P().prefill_layer(qr, cache.k(m), cache.v(m), o, meta, ws, L)
        outs_prompt.append(o)
    cache.compact(meta)
    step_out = torch.empty(steps, M, b, H, d, dtype=q.dtype, device=DEV)
    for i, t in enumerate(range(L, T)):
        for m in range(M):
            qn = q[m, :, :, t].contiguous()
            kn = k[m, :, :, t].contiguous()
            vn = v[m, :, :, t].contiguous()
            P().decode_layer(qn, kn, vn, cache, m, meta, ws, step_out[i, m], theta=theta)
        cache.commit(meta)
        if t in cr_steps:
            cache.compact(meta)
    torch.cuda.synchronize()
    assert int(cache.status) == 0
    Q, K, V = f64(q), f64(k), f64(v)
    for m in range(M):
        for s in range(b):
            rp, rs, fin = O.run_prompt_and_decode(Q[m, s], K[m, s], V[m, s], types[s], L, steps,
                                                  theta=theta, compact_after=cr_steps)
            assert np.abs(f64(outs_prompt[m][s]) - rp).max() <= TOL[dtype]
            got = f64(step_out[:, m, s])
            assert np.abs(got - rs).max() <= TOL[dtype], np.abs(got - rs).max()
            assert int(cache.kv_len[s]) == fin[4]
            assert np.array_equal(cache.tok_idx[s, :fin[4]].cpu().numpy(), fin[2][:fin[4]])
            assert np.array_equal(cache.pos_ids[s, :fin[4]].cpu().numpy(), fin[3][:fin[4]])


def _pipeline_outputs(q, k, v, spans, L, steps, theta):
    """Prompt, compaction and decode steps (compaction after each <CR>) on
    the current stream; returns every output and the final bookkeeping."""
    M, b, H, T, d = q.shape
    meta = P().SpanMeta(spans, T, DEV)
    cache = P().KVCache(M, b, H, T, d, q.dtype, DEV)
    ws = P().Workspace(b, H, L, T, d, DEV)
    cache.start_prompt(L, meta)
    cr_steps = {r for sp in spans for _, r in sp if L <= r < T}
    outs = []
    P().prefill_plan(meta, ws, b, L)
    for m in range(M):
        qr = torch.empty(b, H, L, d, dtype=q.dtype, device=DEV)
        P().rope_rows(q[m, :, :, :L], qr, meta, L, 0, theta)
        P().rope_rows(k[m, :, :, :L], cache.k(m), meta, L, 0, theta)
        P().rope_rows(v[m, :, :, :L], cache.v(m), meta, L, 0, 0.0)
        o = torch.empty_like(qr)
        P().prefill_layer(qr, cache.k(m), cache.v(m), o, meta, ws, L, planned=True)
        outs.append(o)
    cache.compact(meta)
    for t in range(L, L + steps):
        for m in range(M):
            od = torch.empty(b, H, d, dtype=q.dtype, device=DEV)
            P().decode_layer(q[m, :, :, t].contiguous(), k[m, :, :, t].contiguous(),
                             v[m, :, :, t].contiguous(), cache, m, meta, ws, od, theta=theta)
            outs.append(od)
        cache.commit(meta)
        if t in cr_steps:
            cache.compact(meta)
    return outs, cache


def test_pipeline_on_a_side_stream_is_bitexact():
    """The whole path launched inside `torch.cuda.stream(s)` (every call on
    that stream, no explicit stream argument) gives the same bytes as on the
    default stream."""
    say("pipeline on a side stream")
    M, b, H, L, steps, d, theta = 2, 2, 4, 300, 20, 80, 10000.0
    T = L + steps
    rng = np.random.default_rng(17)
    spans = [random_spans(L, rng, max_len=30) + [(L + 3, L + 9)] for _ in range(b)]
    q, k, v = (rnd((M, b, H, T, d), 400 + i, "bf16") for i in range(3))
    torch.cuda.synchronize()
    ref, ref_cache = _pipeline_outputs(q, k, v, spans, L, steps, theta)
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        got, got_cache = _pipeline_outputs(q, k, v, spans, L, steps, theta)
    s.synchronize()
    assert int(ref_cache.status) == 0 and int(got_cache.status) == 0
    for a, c in zip(ref, got):
        assert torch.equal(a, c)
    assert torch.equal(ref_cache.kv_len, got_cache.kv_len)
    for i in range(b):  # rows past a sequence's length were never written
        n = int(ref_cache.kv_len[i])
        assert torch.equal(ref_cache.kv[:, :, i, :, :n], got_cache.kv[:, :, i, :, :n])
        assert torch.equal(ref_cache.tok_idx[i, :n], got_cache.tok_idx[i, :n])
        assert torch.equal(ref_cache.pos_ids[i, :n], got_cache.pos_ids[i, :n])


# ---------------------------------------------------------------------------
# local-attention comparator: ring of the W most recent tokens
# ---------------------------------------------------------------------------

# H=3 splits each slice into chunks (merge kernel); H=256 with b=2 gives 512
# slices, one workgroup each
@pytest.mark.parametrize("d,theta,H,W", [(80, 10000.0, 3, 50), (64, 0.0, 3, 37),
                                         (80, 10000.0, 256, 50)])
def test_local_decode_ring_matches_oracle(d, theta, H, W):
    say(f"local decode d={d} theta={theta} H={H} W={W}")
    b, L, steps = 2, 120, 70  # 70 steps wrap the ring more than once
    T = L + steps
    meta = P().SpanMeta([[] for _ in range(b)], T, DEV)
    L_cap = W + 3
    cache = P().KVCache(1, b, H, L_cap, d, torch.bfloat16, DEV)
    ws = P().Workspace(b, H, 1, L_cap, d, DEV)
    k0, v0 = (rnd((b, H, L, d), 900 + i, "bf16") for i in range(2))
    P().ring_fill(k0, cache.k(0), W, L, meta, theta, L_cap)
    P().ring_fill(v0, cache.v(0), W, L, meta, 0.0, L_cap)
    cache.cur_tok.fill_(L)
    qd, kd, vd = (rnd((steps, b, H, d), 910 + i, "bf16") for i in range(3))
    od = torch.empty(b, H, d, dtype=torch.bfloat16, device=DEV)
    got = []
    for i in range(steps):
        P().local_decode_layer(qd[i], kd[i], vd[i], cache, 0, W, meta, ws, od, theta=theta)
        got.append(f64(od))
        cache.cur_tok.add_(1)
    torch.cuda.synchronize()
    assert int(cache.status) == 0
    # oracle: keys of all tokens rotated at their positions (no sentinels:
    # position = index), attention over the last W tokens
    K = np.concatenate([f64(k0), np.transpose(f64(kd), (1, 2, 0, 3))], axis=2)
    V = np.concatenate([f64(v0), np.transpose(f64(vd), (1, 2, 0, 3))], axis=2)
    Q = f64(qd)
    worst = 0.0
    for s in range(b):
        for h in range(H):
            # unrounded fp64 rotation, as in every other test (the cache
            # itself stores the rotated keys in bf16)
            Kr = O.rope_rotate_half(K[s, h], np.arange(T), theta) if theta > 0 else K[s, h]
            for i in range(steps):
                t = L + i
                qs = Q[i, s, h][None]
                if theta > 0:
                    qs = O.rope_rotate_half(qs, [t], theta)
                lo = t - W + 1
                ref = O.decode_attention(qs, Kr[t][None], V[s, h, t][None], Kr[lo:t][None],
                                         V[s, h, lo:t][None], W - 1, False)[0]
                worst = max(worst, np.abs(got[i][s, h] - ref).max())
    assert worst <= TOL["bf16"], worst
    # the ring holds the last W tokens, token t at row t mod W
    Kc, Vc = f64(cache.k(0)), f64(cache.v(0))
    for t in range(T - W, T):
        assert np.array_equal(Vc[:, :, t % W], V[:, :, t])


# ---------------------------------------------------------------------------
# the binding refuses tensors the kernels would misread
# ---------------------------------------------------------------------------

def test_binding_rejects_bad_device_tensors():
    """Wrong element type, too small a buffer or a layout that does not
    match the strides: SckvError before the C call, nothing launched."""
    say("binding argument checks")
    B = P().B
    b, H, d, L_cap, T = 2, 2, 64, 32, 40
    q = torch.zeros((b, H, d), dtype=torch.bfloat16, device=DEV)
    kc = torch.zeros((b, H, L_cap, d), dtype=torch.bfloat16, device=DEV)
    vu = torch.zeros((b, T), dtype=torch.int32, device=DEV)
    n = torch.zeros(b, dtype=torch.int32, device=DEV)
    ws = torch.empty(B.sckv_decode_workspace_bytes(b, H, L_cap, d), dtype=torch.uint8, device=DEV)
    ok = dict(q=q, k_new=q, v_new=q, k_cache=kc, v_cache=kc, kv_len=n, cur_tok=n, vu=vu, pos=vu,
              L_meta=T, o=q.clone(), b=b, H=H, L_cap=L_cap, d_head=d, scale=0.125,
              rope_theta=0.0, ws=ws)
    bad = [dict(kv_len=n.long()),                                   # int64 lengths
           dict(k_cache=kc[:, :, :L_cap // 2]),                      # fewer rows than L_cap
           dict(q=torch.zeros((b, H, d), dtype=torch.float32, device=DEV)),  # mixed types
           dict(vu=vu[:, :T // 2]),                                  # non-contiguous view
           dict(o=torch.zeros((b, H, d - 8), dtype=torch.bfloat16, device=DEV))]  # too small
    for change in bad:
        with pytest.raises(B.SckvError) as e:
            B.compacted_decode_attn(**{**ok, **change})
        assert e.value.code == B.EINVAL, change
    # strided prefill operands must match the strides passed
    L = 16
    x = torch.zeros((b, H, L, d), dtype=torch.bfloat16, device=DEV)
    pws = torch.empty(B.sckv_prefill_workspace_bytes(b, L), dtype=torch.uint8, device=DEV)
    with pytest.raises(B.SckvError):
        B.span_masked_prefill_attn(x, x, x, x.clone(), b, H, L, d, L * d, 2 * L * d, L * d, 0.125,
                                   vu, T, pws)
    torch.cuda.synchronize()


def test_binding_launches_on_the_current_stream():
    """Without an explicit stream the calls go to torch's current stream of
    the tensors' GPU, also inside a `torch.cuda.stream` block."""
    B = P().B
    x = torch.zeros(4, device=DEV)
    assert B._stream(None, x) == torch.cuda.current_stream(x.device).cuda_stream
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        assert B._stream(None, x) == s.cuda_stream
    assert B._stream(None, x) == torch.cuda.current_stream(x.device).cuda_stream
