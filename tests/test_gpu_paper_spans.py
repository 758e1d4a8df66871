"""The paper's own span distribution through the whole path on the GPU.

Section 3.1 ("Input Transformation") draws span lengths from U(2, l) until
the compression ratio r is reached, and Section 4.1 sets l = 25.  Short
spans leave many partly visible key columns in every query block, the
regime in which the prefill's gathered key tiles are most fragmented (the
ratio of executed to algorithmic work is highest at r = 0.9).

At r = 0.1, 0.5 and 0.9 over a 2048-token prompt (head size 64 without
rotary positions, as in OPT; head size 80 with rotary positions, as in the
3B RoPE model), every head of every sequence goes through

  * the masked prefill on a plan built once for the prompt,
  * compaction at the end of the prompt,
  * 24 decode steps whose generated text holds two more short spans, with
    compaction right after each <CR>,

and is compared with the oracle: attention outputs within max-abs 2e-2
(bf16 inputs), <CL> rows and every compacted index, length and position bit
for bit.  The block-wise prompt path (blocks of 512, freeing after each) is
checked on the same spans at r = 0.5 and 0.9.
"""
import numpy as np
import pytest
import torch

from oracle import sckv_oracle as O

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
TOL = 2e-2
L = 2048
STEPS = 24
# spans in the generated text, lengths from the same U(2, 25) range
GEN_SPANS = [(L + 2, L + 9), (L + 12, L + 14)]


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


def say(msg):
    print(msg, flush=True)


def paper_spans(b, ratio, seed):
    rng = np.random.default_rng(seed)
    return [W().spans_uniform_lengths(L, ratio, 2, 25, rng) for _ in range(b)]


CASES = [(r, d, th) for r in (0.1, 0.5, 0.9) for d, th in ((64, 0.0), (80, 1e4))]


@pytest.mark.parametrize("ratio,d,theta", CASES,
                         ids=[f"r{r}-d{d}" + ("-rope" if th else "") for r, d, th in CASES])
def test_paper_spans_prefill_compact_decode(ratio, d, theta):
    b, H = 2, 4
    T = L + STEPS
    seed = int(ratio * 1000) + d
    prompt_spans = paper_spans(b, ratio, seed)
    spans = [sp + GEN_SPANS for sp in prompt_spans]
    say(f"paper spans r={ratio} d={d} theta={theta}: "
        f"{[len(sp) for sp in prompt_spans]} prompt spans per sequence")
    types = [O.token_types(sp, T) for sp in spans]
    cr_steps = sorted({r for _, r in GEN_SPANS})
    q, k, v = (W().randn((b, H, T, d), seed=seed * 10 + i, dtype="bf16", device=DEV)
               for i in range(3))

    meta = P().SpanMeta(spans, T, DEV)
    cache = P().KVCache(1, b, H, T, d, torch.bfloat16, DEV)
    ws = P().Workspace(b, H, L, T, d, DEV)
    cache.start_prompt(L, meta)
    qr = torch.empty(b, H, L, d, dtype=torch.bfloat16, device=DEV)
    P().rope_rows(q[:, :, :L], qr, meta, L, 0, theta)
    P().rope_rows(k[:, :, :L], cache.k(0), meta, L, 0, theta)
    P().rope_rows(v[:, :, :L], cache.v(0), meta, L, 0, 0.0)
    o = torch.full_like(qr, float("nan"))
    P().prefill_plan(meta, ws, b, L)
    P().prefill_layer(qr, cache.k(0), cache.v(0), o, meta, ws, L, planned=True)
    cache.compact(meta)
    torch.cuda.synchronize()
    after_prompt = (cache.kv_len.clone(), cache.tok_idx.clone(), cache.pos_ids.clone(),
                    cache.kept_src.clone())
    od = torch.empty(STEPS, b, H, d, dtype=torch.bfloat16, device=DEV)
    for i, t in enumerate(range(L, T)):
        P().decode_layer(q[:, :, t].contiguous(), k[:, :, t].contiguous(),
                         v[:, :, t].contiguous(), cache, 0, meta, ws, od[i], theta=theta)
        cache.commit(meta)
        if t in cr_steps:
            cache.compact(meta)
    torch.cuda.synchronize()
    assert int(cache.status) == 0

    Q, K, V, Og, Od = f64(q), f64(k), f64(v), f64(o), f64(od)
    for s in range(b):
        say(f"  oracle s={s}")
        rp, rs, fin = O.run_prompt_and_decode(Q[s], K[s], V[s], types[s], L, STEPS, theta=theta,
                                              compact_after=cr_steps)
        err_p = np.abs(Og[s] - rp).max()
        err_d = np.abs(Od[:, s] - rs).max()
        assert err_p <= TOL and err_d <= TOL, (s, err_p, err_d)
        for c, _ in prompt_spans[s]:
            # a <CL> row sees only itself: its output is its own value row
            assert np.array_equal(Og[s, :, c], V[s, :, c]), (s, c)
        # the compaction at the end of the prompt, bit for bit
        pos = O.tie_positions(types[s])
        ref = O.compact_cache(np.zeros((1, L, 1)), np.zeros((1, L, 1)), np.arange(L),
                              pos[:L].copy(), L, types[s], L)
        n = ref[4]
        assert int(after_prompt[0][s]) == n
        assert np.array_equal(after_prompt[1][s, :n].cpu().numpy(), ref[2][:n])
        assert np.array_equal(after_prompt[2][s, :n].cpu().numpy(), ref[3][:n])
        assert np.array_equal(after_prompt[3][s, :n].cpu().numpy(), ref[5])
        # the cache after the generated tokens and their spans
        n = fin[4]
        assert int(cache.kv_len[s]) == n
        assert np.array_equal(cache.tok_idx[s, :n].cpu().numpy(), fin[2][:n])
        assert np.array_equal(cache.pos_ids[s, :n].cpu().numpy(), fin[3][:n])


@pytest.mark.parametrize("ratio", [0.5, 0.9])
def test_paper_spans_blockwise_prompt(ratio):
    """Blocks of 512 prompt tokens, each appended to the compacted cache,
    attending to it and freeing what it closes; outputs against the oracle's
    masked attention over the whole prompt, the final cache against the
    one-shot path bit for bit."""
    M, b, H, d, theta, block = 1, 2, 4, 80, 1e4, 512
    seed = int(ratio * 1000) + 7
    spans = paper_spans(b, ratio, seed)
    say(f"paper spans block-wise r={ratio}: {[len(sp) for sp in spans]} spans per sequence")
    types = [O.token_types(sp, L) for sp in spans]
    pos = [O.tie_positions(t) for t in types]
    peak = 0
    for B0 in range(0, L, block):
        for s in range(b):
            kept = int(O.keep_rows(types[s], B0)[:B0].sum()) if B0 else 0
            peak = max(peak, kept + min(block, L - B0))
    q, k, v = (W().randn((M, b, H, L, d), seed=seed * 10 + i, dtype="bf16", device=DEV)
               for i in range(3))
    meta = P().SpanMeta(spans, L, DEV)
    cache = P().KVCache(M, b, H, peak, d, torch.bfloat16, DEV)
    ws = P().Workspace(b, H, block, peak, d, DEV, block=block)
    o = torch.full_like(q, float("nan"))
    P().prefill_progressive(q, k, v, o, cache, meta, ws, L, block, theta=theta)
    torch.cuda.synchronize()
    assert int(cache.status) == 0
    Og, Q, K, V = f64(o), f64(q), f64(k), f64(v)
    worst = 0.0
    for s in range(b):
        say(f"  oracle s={s}")
        mask = O.attention_mask(types[s])
        for h in range(H):
            Qs = O.rope_rotate_half(Q[0, s, h], pos[s], theta)
            Ks = O.rope_rotate_half(K[0, s, h], pos[s], theta)
            ref = O.masked_attention(Qs[None], Ks[None], V[0, s, h][None], mask)[0]
            worst = max(worst, np.abs(Og[0, s, h] - ref).max())
    assert worst <= TOL, worst
    one = P().KVCache(M, b, H, L, d, torch.bfloat16, DEV)
    P().rope_rows(k[0], one.k(0), meta, L, 0, theta)
    one.v(0).copy_(v[0])
    one.start_prompt(L, meta)
    one.compact(meta)
    torch.cuda.synchronize()
    assert torch.equal(cache.kv_len, one.kv_len)
    for s in range(b):
        n = int(one.kv_len[s])
        assert torch.equal(cache.tok_idx[s, :n], one.tok_idx[s, :n])
        assert torch.equal(cache.pos_ids[s, :n], one.pos_ids[s, :n])
        assert torch.equal(cache.kv[:, :, s, :, :n], one.kv[:, :, s, :, :n])
