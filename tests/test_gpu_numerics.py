"""Online-softmax range checks against the oracle (GPU).

The other parity tests draw q, k, v from N(0, 1), where the running maximum
of a query never moves by more than a few powers of two after the first
tile, so the kernels' rescaling paths are barely exercised.  Here the scores
span tens of powers of two (q and k scaled by 3: a standard deviation of 9
in natural-log units), and a single key row scaled by 40 makes the running
maximum jump by hundreds of powers of two in the middle of the keys (its
scores have a standard deviation of 360; Section 3.1: the mask decides which
queries see that row).  The
prefill takes the lazy rescale of its accumulators; the decode takes the
same inside a chunk and, with few (sequence, head) slices, the combine of
chunk partials whose maxima differ by that much.
"""
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


SPANS = [(10, 40), (100, 180), (300, 320), (520, 560)]  # row 500 is a normal token
OUTLIER = 500


def prefill(q, k, v, spans):
    b, H, L, d = q.shape
    meta = P().SpanMeta(spans, L, DEV)
    ws = P().Workspace(b, H, L, L, d, DEV)
    o = torch.full_like(q, float("nan"))
    P().prefill_layer(q, k, v, o, meta, ws, L)
    torch.cuda.synchronize()
    return o


@pytest.mark.parametrize("d", [64, 80])
@pytest.mark.parametrize("outlier", [False, True], ids=["wide", "wide+outlier"])
def test_prefill_wide_logit_range(d, outlier):
    b, H, L = 1, 2, 640
    say(f"prefill wide logit range d={d} outlier={outlier}")
    q = W().randn((b, H, L, d), seed=301, scale=3.0, device=DEV)
    k = W().randn((b, H, L, d), seed=302, scale=3.0, device=DEV)
    v = W().randn((b, H, L, d), seed=303, device=DEV)
    if outlier:
        k[:, :, OUTLIER] *= 40.0  # rounded to bf16; kernel and oracle read the same tensor
    spans = [SPANS]
    o = prefill(q, k, v, spans)
    types = O.token_types(SPANS, L)
    mask = O.attention_mask(types)
    Q, K, V, Og = f64(q), f64(k), f64(v), f64(o)
    for h in range(H):
        ref = O.masked_attention(Q[0, h][None], K[0, h][None], V[0, h][None], mask)[0]
        err = np.abs(Og[0, h] - ref).max()
        assert err <= TOL, (h, err)
    assert np.isfinite(Og).all()
    if outlier:
        # the row dominates some of the queries that see it: their outputs are its value row
        s = np.einsum("hid,hd->hi", Q[0], K[0, :, OUTLIER]) / np.sqrt(d)
        sees = mask[:, OUTLIER]
        dom = sees[None, :] & (s > 200.0)
        assert dom.sum() > 50
        for h in range(H):
            rows = np.nonzero(dom[h])[0]
            assert np.abs(Og[0, h, rows] - V[0, h, OUTLIER][None]).max() <= TOL


# b = 3: H = 3 gives 9 slices (1024-row chunks merged by a second kernel),
# H = 176 gives 528 slices (one four-wave workgroup each), H = 352 gives 1056
# (one two-wave workgroup each)
@pytest.mark.parametrize("H", [3, 176, 352], ids=["split-and-combine", "slice-wide", "slice-narrow"])
@pytest.mark.parametrize("d", [64, 80])
def test_decode_wide_logit_range(d, H):
    say(f"decode wide logit range d={d} H={H}")
    L_cap = 1200
    lens = [1100, 700, 2]
    b = len(lens)
    spans = [[] for _ in range(b)]
    meta = P().SpanMeta(spans, 2000, DEV)
    cache = P().KVCache(1, b, H, L_cap, d, torch.bfloat16, DEV)
    kv = W().randn(cache.kv.shape, seed=311, device=DEV)
    kv[0, 0] = W().randn(cache.kv[0, 0].shape, seed=312, scale=3.0, device=DEV)
    for s, n in enumerate(lens):
        kv[0, 0, s, :, (n * 3) // 4] *= 40.0  # one late row that some queries are drawn to
    cache.kv.copy_(kv)
    cache.kv_len.copy_(torch.tensor(lens, dtype=torch.int32))
    cache.cur_tok.copy_(torch.tensor([1500 + i for i in range(b)], dtype=torch.int32))
    ws = P().Workspace(b, H, 1, L_cap, d, DEV)
    q = W().randn((b, H, d), seed=313, scale=3.0, device=DEV)
    kn = W().randn((b, H, d), seed=314, scale=3.0, device=DEV)
    vn = W().randn((b, H, d), seed=315, device=DEV)
    o = torch.empty_like(q)
    before = cache.kv.clone()
    P().decode_layer(q, kn, vn, cache, 0, meta, ws, o, theta=0.0)
    torch.cuda.synchronize()
    assert int(cache.status) == 0
    Q, KN, VN, K, V, Og = f64(q), f64(kn), f64(vn), f64(before[0, 0]), f64(before[0, 1]), f64(o)
    assert np.isfinite(Og).all()
    for s in range(b):
        ref = O.decode_attention(Q[s], KN[s], VN[s], K[s], V[s], lens[s], False)
        err = np.abs(Og[s] - ref).max()
        assert err <= TOL, (s, err)
