"""compacted_decode_attn_noalloc, the decode step that takes its split-K
partials in the library's own scratch array instead of a caller workspace,
against compacted_decode_attn on the same inputs, through the C ABI: two
calls in a row, the second one smaller (fewer slices, fewer rows, another
head size), so the second call runs over what the first left in the array.
Outputs and the appended cache row must equal those of the workspace entry
point bit for bit (same kernels), and the oracle within max-abs 2e-2 (bf16).
A shape whose partials would not fit is rejected before anything runs."""
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
    from paper_2310_08152_amd import binding  # noqa: F401  (fails loudly without the library)


def B():
    from paper_2310_08152_amd import binding
    return binding


def W():
    from paper_2310_08152_amd import workload
    return workload


def f64(t):
    return t.detach().to("cpu", torch.float64).numpy()


def one_step(b, H, d, L_cap, kv_len, theta, seed):
    """One decode step of one layer over a cache of random rows, through
    both entry points on separate copies of the same state."""
    T = max(kv_len) + 1
    vu = torch.full((b, T), 0x7fffffff, dtype=torch.int32, device=DEV)  # no spans
    pos = torch.arange(T, dtype=torch.int32, device=DEV).repeat(b, 1)
    kv_len_t = torch.tensor(kv_len, dtype=torch.int32, device=DEV)
    cur_tok = kv_len_t.clone()  # the token after the rows held: a normal token
    cache = W().randn((2, b, H, L_cap, d), seed=seed, device=DEV)
    q, kn, vn = (W().randn((b, H, d), seed=seed + 1 + i, device=DEV) for i in range(3))
    scale = d ** -0.5
    outs = []
    caches = []
    for noalloc in (False, True):
        c = cache.clone()
        o = torch.full((b, H, d), float("nan"), dtype=torch.bfloat16, device=DEV)
        st = torch.zeros(1, dtype=torch.int32, device=DEV)
        if noalloc:
            B().compacted_decode_attn_noalloc(q, kn, vn, c[0], c[1], kv_len_t, cur_tok, vu, pos, T,
                                              o, b, H, L_cap, d, scale, theta, status=st)
        else:
            ws = torch.empty(B().sckv_decode_workspace_bytes(b, H, L_cap, d), dtype=torch.uint8,
                             device=DEV)
            B().compacted_decode_attn(q, kn, vn, c[0], c[1], kv_len_t, cur_tok, vu, pos, T, o, b,
                                      H, L_cap, d, scale, theta, ws, status=st)
        torch.cuda.synchronize()
        assert int(st) == 0
        outs.append(o)
        caches.append(c)
    assert torch.equal(outs[0], outs[1])
    assert torch.equal(caches[0], caches[1])
    # the oracle: attention over the kept rows plus the new row
    Q, KN, VN, K, V, Og = f64(q), f64(kn), f64(vn), f64(cache[0]), f64(cache[1]), f64(outs[1])
    worst = 0.0
    for s in range(b):
        n = kv_len[s]
        qs, ks = Q[s], KN[s]
        if theta > 0:
            qs = np.stack([O.rope_rotate_half(Q[s, h][None], [n], theta)[0] for h in range(H)])
            ks = np.stack([O.rope_rotate_half(KN[s, h][None], [n], theta)[0] for h in range(H)])
        ref = O.decode_attention(qs, ks, VN[s], K[s], V[s], n, False)
        worst = max(worst, np.abs(Og[s] - ref).max())
    assert worst <= TOL, worst


def test_noalloc_decode_equals_workspace_decode_twice():
    print("noalloc decode: b=2 H=8 d=80 L_cap=3000 rotary, then b=1 H=4 d=64 L_cap=700",
          flush=True)
    # 16 slices of 2000-2900 rows: three chunks each, merged from the scratch array
    one_step(2, 8, 80, 3000, [2900, 2000], 1e4, 11)
    # smaller: 4 slices of one chunk, over the partials the first call left
    one_step(1, 4, 64, 700, [650], 0.0, 21)


def test_noalloc_decode_one_workgroup_per_slice():
    """From 512 slices on the launch writes no partials at all."""
    print("noalloc decode: b=2 H=256 d=80 (512 slices)", flush=True)
    one_step(2, 256, 80, 400, [300, 399], 1e4, 31)


def test_noalloc_rejects_partials_beyond_the_scratch_array():
    b, H, d, L_cap = 1, 511, 80, 200000  # 511 slices x 196 chunks x 328 bytes > 16 MiB
    assert B().sckv_decode_workspace_bytes(b, H, L_cap, d) > B().NOALLOC_SCRATCH_BYTES
    x = torch.zeros((b, H, d), dtype=torch.bfloat16, device=DEV)
    cache = torch.zeros((b, H, 1, d), dtype=torch.bfloat16, device=DEV)
    i32 = torch.zeros(b, dtype=torch.int32, device=DEV)
    vu = torch.zeros((b, 4), dtype=torch.int32, device=DEV)
    with pytest.raises(B().SckvError) as e:
        # the size check fails before the binding's extent checks would
        # matter: call the C entry point directly
        rc = B().lib.compacted_decode_attn_noalloc(
            x.data_ptr(), x.data_ptr(), x.data_ptr(), cache.data_ptr(), cache.data_ptr(),
            i32.data_ptr(), i32.data_ptr(), vu.data_ptr(), vu.data_ptr(), 4, x.data_ptr(), b, H,
            L_cap, d, B().BF16, 0.1, 0.0, None, None)
        B()._check(rc)
    assert e.value.code == B().EUNSUP
    assert "scratch" in str(e.value)
