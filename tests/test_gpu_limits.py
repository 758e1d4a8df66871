"""Entry points at their documented size limits, against the oracle on
sampled rows: masked prefill at L = 32768 (with rotary at tied positions),
compaction of a cache of L_cap = 65536 rows, and one decode step over the
compacted 65536-row cache (a single (sequence, head) slice, so the decode
takes its split launch with the most chunks)."""
import numpy as np
import pytest
import torch

from oracle import sckv_oracle as O

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
TOL = 2e-2


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def P():
    from paper_2310_08152_amd import path
    return path


def W():
    from paper_2310_08152_amd import workload
    return workload


def f64(t):
    return t.detach().to("cpu", torch.float64).numpy()


def say(msg):
    print(msg, flush=True)


def test_prefill_at_max_length():
    L, b, H, d, theta = 32768, 1, 2, 80, 10000.0
    say(f"prefill at L={L}")
    spans = [(100, 20000)] + [(20100 + 500 * k, 20100 + 500 * k + 10 + 19 * k) for k in range(25)]
    spans += [(32700, L + 50)]  # still open at the end
    meta = P().SpanMeta([spans], L, DEV)
    q, k, v = (W().randn((b, H, L, d), seed=910 + i, device=DEV) for i in range(3))
    qr, kr = torch.empty_like(q), torch.empty_like(k)
    P().rope_rows(q, qr, meta, L, 0, theta)
    P().rope_rows(k, kr, meta, L, 0, theta)
    ws = P().Workspace(b, H, L, L, d, DEV)
    o = torch.full_like(q, float("nan"))
    P().prefill_layer(qr, kr, v, o, meta, ws, L)
    torch.cuda.synchronize()
    types = O.token_types(spans, L)
    pos = O.tie_positions(types)
    rows = [0, 99, 100, 101, 5000, 19999, 20000, 20001, 20110, 27777, 32699, 32700, 32701, 32767]
    mask = O.attention_mask_rows(types, rows)
    for h in range(H):
        Q = O.rope_rotate_half(f64(q[0, h])[rows], pos[rows], theta)
        K = O.rope_rotate_half(f64(k[0, h]), pos, theta)
        ref = O.masked_attention(Q[None], K[None], f64(v[0, h])[None], mask)[0]
        err = np.abs(f64(o[0, h])[rows] - ref).max()
        assert err <= TOL, (h, err)
    assert torch.isfinite(o).all()


def test_compaction_and_decode_at_max_capacity():
    L_cap, b, H, d, theta = 65536, 1, 1, 64, 10000.0
    say(f"compaction and decode at L_cap={L_cap}")
    rng = np.random.default_rng(65536)
    spans, c = [], int(rng.integers(0, 50))
    while c < L_cap - 2:
        r = c + int(rng.integers(2, 200))
        if r >= L_cap:
            break
        spans.append((c, r))
        c = r + 1 + int(rng.integers(0, 120))
    L_meta = L_cap + 1  # the decode step's token
    meta = P().SpanMeta([spans], L_meta, DEV)
    cache = P().KVCache(1, b, H, L_cap, d, torch.bfloat16, DEV)
    cache.kv.copy_(W().randn(cache.kv.shape, seed=920, device=DEV))
    before = cache.kv.clone()
    cache.start_prompt(L_cap, meta)
    cache.compact(meta)
    torch.cuda.synchronize()
    types = O.token_types(spans, L_meta)
    pos = O.tie_positions(types)
    keep = O.keep_rows(types, L_cap)
    kept_src = np.nonzero(keep[:L_cap])[0]
    n = len(kept_src)
    assert int(cache.kv_len[0]) == n
    assert np.array_equal(cache.tok_idx[0, :n].cpu().numpy(), kept_src)
    assert np.array_equal(cache.pos_ids[0, :n].cpu().numpy(), pos[kept_src])
    src = torch.as_tensor(kept_src, device=DEV)
    assert torch.equal(cache.kv[:, :, 0, 0, :n], before[:, :, 0, 0].index_select(2, src))

    # one decode step over the n surviving rows: token L_cap (a normal token)
    assert types[L_cap] == O.NORMAL
    q, kn, vn = (W().randn((b, H, d), seed=930 + i, device=DEV) for i in range(3))
    ws = P().Workspace(b, H, 1, L_cap, d, DEV)
    o = torch.full_like(q, float("nan"))
    P().decode_layer(q, kn, vn, cache, 0, meta, ws, o, theta=theta)
    torch.cuda.synchronize()
    assert int(cache.status) == 0
    p = [pos[L_cap]]
    qs = O.rope_rotate_half(f64(q[0]), p, theta)
    ks = O.rope_rotate_half(f64(kn[0]), p, theta)
    Kc, Vc = f64(before[0, 0, 0, :, kept_src]), f64(before[0, 1, 0, :, kept_src])
    ref = O.decode_attention(qs, ks, f64(vn[0]), Kc, Vc, n, False)
    assert np.abs(f64(o[0]) - ref).max() <= TOL
    # the new row went to row n, rotated; rows before it are untouched
    assert np.array_equal(f64(cache.kv[0, 1, 0, 0, n]), f64(vn[0, 0]))
    assert np.abs(f64(cache.kv[0, 0, 0, 0, n]) - ks[0]).max() <= TOL
