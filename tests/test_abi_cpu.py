"""The C ABI loads, exports every declared symbol, and rejects bad arguments
on the host before any HIP call (so these run without a GPU)."""
import ctypes
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sckv.h")


@pytest.fixture(scope="module")
def B():
    from paper_2310_08152_amd import binding
    return binding


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?[a-z_0-9]+\s*\*?\s*([a-z_][a-z_0-9]*)\s*\(", text, flags=re.M)
    return sorted(set(names))


def test_every_declared_symbol_is_exported(B):
    names = declared_functions()
    assert len(names) >= 10, names
    for n in names:
        assert hasattr(B.lib, n), n
        assert n in B.EXPORTS, n


def test_version(B):
    assert "gfx950" in B.version()


FAKE = ctypes.c_void_p(4096)  # never dereferenced: every call below fails a host check first
NULL = None


def test_span_meta_rejects_bad_spans(B):
    vu = FAKE
    def call(cl, cr, n, L=100):
        cl = np.asarray(cl, np.int32).reshape(1, -1)
        cr = np.asarray(cr, np.int32).reshape(1, -1)
        n = np.asarray([n], np.int32)
        return B.lib.sckv_span_meta(cl.ctypes.data, cr.ctypes.data, n.ctypes.data, cl.shape[1], 1,
                                    L, FAKE, vu, NULL, NULL)
    assert call([5, 10], [10, 20], 2) == B.ESPAN        # cr_0 == cl_1: overlap
    assert call([10, 5], [12, 8], 2) == B.ESPAN         # unsorted
    assert call([5], [5], 1) == B.ESPAN                 # cl == cr
    assert call([100], [120], 1) == B.ESPAN             # cl >= L_meta
    assert call([-1], [3], 1) == B.ESPAN                # negative
    assert call([1], [3], 2) == B.ESPAN                 # n > s_max
    assert "overlap" in B.last_error() or "s_max" in B.last_error()
    cl = np.zeros((1, 1), np.int32)
    assert B.lib.sckv_span_meta(cl.ctypes.data, cl.ctypes.data, cl.ctypes.data, 1, 1, 10, NULL,
                                FAKE, NULL, NULL) == B.EINVAL


def test_prefill_rejects(B):
    f = B.lib.span_masked_prefill_attn
    ws = B.lib.sckv_prefill_workspace_bytes(1, 256)
    assert ws > 0
    ok = dict(b=1, H=4, L=256, d=64, qs=256 * 64, kvs=256 * 64, os=256 * 64, dt=B.F32, scale=0.125)
    def call(**kw):
        a = dict(ok, **kw)
        return f(FAKE, FAKE, FAKE, FAKE, a["b"], a["H"], a["L"], a["d"], a["qs"], a["kvs"], a["os"],
                 a["dt"], a["scale"], FAKE, a.get("L_meta", 256), FAKE, a.get("ws", ws), NULL)
    assert call(d=96) == B.EUNSUP
    assert call(dt=7) == B.EINVAL
    assert call(L=0) == B.EINVAL
    assert call(qs=100) == B.EINVAL
    assert call(L_meta=255) == B.EINVAL
    assert call(ws=ws - 1) == B.EINVAL
    assert call(scale=0.0) == B.EINVAL
    assert call(L=40000, qs=40000 * 64, kvs=40000 * 64, os=40000 * 64, L_meta=40000) == B.EUNSUP
    assert f(NULL, FAKE, FAKE, FAKE, 1, 4, 256, 64, 256 * 64, 256 * 64, 256 * 64, B.F32, 0.1,
             FAKE, 256, FAKE, ws, NULL) == B.EINVAL
    # misaligned
    assert f(ctypes.c_void_p(4098), FAKE, FAKE, FAKE, 1, 4, 256, 64, 256 * 64, 256 * 64, 256 * 64,
             B.F32, 0.1, FAKE, 256, FAKE, ws, NULL) == B.EINVAL


def test_prefill_plan_rejects(B):
    ws = B.lib.sckv_prefill_workspace_bytes(2, 300)
    plan = B.lib.sckv_prefill_plan
    assert plan(NULL, 300, 2, 300, FAKE, ws, NULL) == B.EINVAL
    assert plan(FAKE, 300, 2, 300, NULL, ws, NULL) == B.EINVAL
    assert plan(FAKE, 300, 0, 300, FAKE, ws, NULL) == B.EINVAL
    assert plan(FAKE, 299, 2, 300, FAKE, ws, NULL) == B.EINVAL      # L_meta < L
    assert plan(FAKE, 300, 2, 300, FAKE, ws - 1, NULL) == B.EINVAL  # workspace too small
    assert plan(FAKE, 40000, 2, 40000, FAKE, ws, NULL) == B.EUNSUP  # L above 32768
    assert plan(FAKE, 300, 2, 300, ctypes.c_void_p(4104), ws, NULL) == B.EINVAL  # misaligned
    f = B.lib.span_masked_prefill_attn_planned
    def call(**kw):
        a = dict(b=2, H=4, L=300, d=80, s=300 * 80, dt=B.BF16, scale=0.1, ws=ws)
        a.update(kw)
        return f(FAKE, FAKE, FAKE, FAKE, a["b"], a["H"], a["L"], a["d"], a["s"], a["s"], a["s"],
                 a["dt"], a["scale"], FAKE, 300, FAKE, a["ws"], NULL)
    assert call(d=72) == B.EUNSUP
    assert call(H=0) == B.EINVAL
    assert call(s=100) == B.EINVAL
    assert call(ws=ws - 1) == B.EINVAL
    assert call(scale=float("inf")) == B.EINVAL
    assert "planned" in B.last_error()


def test_compact_rejects(B):
    f = B.lib.kv_compact
    args = [FAKE, NULL, 2, 1, 4, 128, 64, B.BF16, FAKE, FAKE, FAKE, FAKE, FAKE, 128, FAKE, NULL]
    bad_d = list(args); bad_d[6] = 72
    assert f(*bad_d) == B.EUNSUP
    bad_m = list(args); bad_m[2] = 0
    assert f(*bad_m) == B.EINVAL
    same = list(args); same[1] = FAKE
    assert f(*same) == B.EINVAL
    nul = list(args); nul[8] = NULL
    assert f(*nul) == B.EINVAL
    big = list(args); big[5] = 70000
    assert f(*big) == B.EUNSUP


def test_decode_rejects(B):
    f = B.lib.compacted_decode_attn
    ws = B.lib.sckv_decode_workspace_bytes(2, 4, 512, 80)
    assert ws == 2 * 4 * 1 * 82 * 4  # one 1024-row chunk per (sequence, head)
    def call(**kw):
        a = dict(d=80, dt=B.BF16, scale=0.1, theta=0.0, ws=ws, pos=FAKE, b=2, H=4, Lc=512)
        a.update(kw)
        return f(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, a["pos"], 600, FAKE, a["b"], a["H"],
                 a["Lc"], a["d"], a["dt"], a["scale"], a["theta"], FAKE, a["ws"], NULL, NULL)
    assert call(d=128) == B.EUNSUP
    assert call(ws=ws - 4) == B.EINVAL
    assert call(theta=-1.0) == B.EINVAL
    assert call(theta=1e4, pos=NULL) == B.EINVAL
    assert call(scale=float("nan")) == B.EINVAL
    assert call(b=1 << 30) == B.EUNSUP


def test_rope_and_commit_reject(B):
    assert B.lib.rope_apply(FAKE, FAKE, 1, 1, 10, 640, 640, 64, B.BF16, FAKE, 100, 95, 1e4,
                            NULL) == B.EINVAL  # rows past L_meta
    assert B.lib.rope_apply(FAKE, FAKE, 1, 1, 10, 64, 640, 64, B.BF16, FAKE, 100, 0, 1e4,
                            NULL) == B.EINVAL  # stride
    assert B.lib.rope_apply(FAKE, FAKE, 1, 1, 10, 640, 640, 48, B.BF16, FAKE, 100, 0, 1e4,
                            NULL) == B.EUNSUP
    assert B.lib.kv_commit(FAKE, FAKE, FAKE, NULL, FAKE, FAKE, 10, 1, 10, NULL, NULL) == B.EINVAL
    assert B.lib.kv_commit(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 10, 0, 10, NULL, NULL) == B.EINVAL


def test_workspace_sizes(B):
    assert B.lib.sckv_prefill_workspace_bytes(0, 10) == 0
    assert B.lib.sckv_prefill_workspace_bytes(2, 300) >= 2 * 3 * 384 * 4
    assert B.lib.sckv_decode_workspace_bytes(1, 1, 1, 64) == 66 * 4


def test_binding_raises_with_message(B):
    with pytest.raises(B.SckvError) as e:
        B.sckv_span_meta(np.array([[5, 10]]), np.array([[10, 20]]), np.array([2]), 100,
                         None, None)
    assert e.value.code == B.EINVAL or e.value.code == B.ESPAN


def test_block_entry_points_reject_bad_arguments(B):
    """Block-wise prompt processing: rope_apply_at, kv_extend and
    span_masked_prefill_attn_cached check their arguments on the host."""
    lib = B.lib
    # rope_apply_at: null row0, y slice smaller than its rows, tokens past L_meta
    assert lib.rope_apply_at(FAKE, FAKE, NULL, 64, 1, 1, 8, 8 * 64, 64 * 64, 64, B.BF16, FAKE,
                             100, 0, 1e4, NULL, NULL) == B.EINVAL
    assert lib.rope_apply_at(FAKE, FAKE, FAKE, 64, 1, 1, 8, 8 * 64, 32 * 64, 64, B.BF16, FAKE,
                             100, 0, 1e4, NULL, NULL) == B.EINVAL
    assert lib.rope_apply_at(FAKE, FAKE, FAKE, 64, 1, 1, 8, 8 * 64, 64 * 64, 64, B.BF16, FAKE,
                             100, 95, 1e4, NULL, NULL) == B.EINVAL
    assert "L_meta" in B.last_error()
    # kv_extend: null pos, tokens past L_meta, negative n
    assert lib.kv_extend(FAKE, FAKE, FAKE, FAKE, NULL, 100, 0, 8, 1, 64, NULL, NULL) == B.EINVAL
    assert lib.kv_extend(FAKE, FAKE, FAKE, FAKE, FAKE, 100, 96, 8, 1, 64, NULL, NULL) == B.EINVAL
    assert lib.kv_extend(FAKE, FAKE, FAKE, FAKE, FAKE, 100, 0, -1, 1, 64, NULL, NULL) == B.EINVAL
    # prefill over the cache
    ws = lib.sckv_prefill_cached_workspace_bytes(2, 100, 512)
    # entries + rows (one 128-query block), 16-byte summaries of 64-entry tiles, counts
    assert ws == 2 * (2 * 1 * 512 * 4) + 2 * 1 * (512 // 64) * 16 + 256
    assert lib.sckv_prefill_cached_workspace_bytes(0, 100, 512) == 0

    def call(**kw):
        a = dict(b=2, H=2, nq=100, d=64, qs=100 * 64, kvs=512 * 64, os=100 * 64, dt=B.BF16,
                 scale=0.125, L_meta=1000, tok0=0, row0=FAKE, tok=FAKE, L_cap=512, ws=ws)
        a.update(kw)
        return lib.span_masked_prefill_attn_cached(
            FAKE, FAKE, FAKE, FAKE, a["b"], a["H"], a["nq"], a["d"], a["qs"], a["kvs"], a["os"],
            a["dt"], a["scale"], FAKE, a["L_meta"], a["tok0"], a["row0"], a["tok"], a["L_cap"],
            FAKE, a["ws"], NULL, NULL)
    assert call(row0=NULL) == B.EINVAL
    assert call(tok=NULL) == B.EINVAL
    assert call(nq=600) == B.EUNSUP              # nq > L_cap
    assert call(L_meta=1 << 24) == B.EUNSUP      # tokens must fit 24 bits
    assert call(tok0=950) == B.EINVAL            # tokens [950, 1050) past L_meta
    assert call(kvs=256 * 64) == B.EINVAL        # cache slice smaller than L_cap rows
    assert call(ws=ws - 1) == B.EINVAL
    assert call(d=96) == B.EUNSUP
    assert call(scale=0.0) == B.EINVAL
    # the same checks on the planned call, and the plan's own
    def planned(**kw):
        a = dict(b=2, H=2, nq=100, d=64, qs=100 * 64, kvs=512 * 64, os=100 * 64, dt=B.BF16,
                 scale=0.125, L_meta=1000, tok0=0, row0=FAKE, tok=FAKE, L_cap=512, ws=ws)
        a.update(kw)
        return lib.span_masked_prefill_attn_cached_planned(
            FAKE, FAKE, FAKE, FAKE, a["b"], a["H"], a["nq"], a["d"], a["qs"], a["kvs"], a["os"],
            a["dt"], a["scale"], FAKE, a["L_meta"], a["tok0"], a["row0"], a["tok"], a["L_cap"],
            FAKE, a["ws"], NULL, NULL)
    assert planned(kvs=256 * 64) == B.EINVAL
    assert planned(d=96) == B.EUNSUP
    assert planned(tok0=950) == B.EINVAL
    assert "planned" in B.last_error()

    def plan(**kw):
        a = dict(L_meta=1000, tok0=0, row0=FAKE, tok=FAKE, L_cap=512, b=2, nq=100, ws=ws)
        a.update(kw)
        return lib.sckv_prefill_cached_plan(FAKE, a["L_meta"], a["tok0"], a["row0"], a["tok"],
                                            a["L_cap"], a["b"], a["nq"], FAKE, a["ws"], NULL)
    assert plan(row0=NULL) == B.EINVAL
    assert plan(nq=600) == B.EUNSUP
    assert plan(L_meta=1 << 24) == B.EUNSUP
    assert plan(tok0=950) == B.EINVAL
    assert plan(ws=ws - 1) == B.EINVAL
    assert plan(b=0) == B.EINVAL
    assert "cached_plan" in B.last_error()


def test_local_decode_rejects_bad_arguments(B):
    lib = B.lib
    ws = lib.sckv_decode_workspace_bytes(2, 4, 64, 80)

    def call(**kw):
        a = dict(W=32, L_cap=64, dt=B.BF16, d=80, ws=ws, cur=FAKE)
        a.update(kw)
        return lib.local_decode_attn(FAKE, FAKE, FAKE, FAKE, FAKE, a["W"], a["cur"], FAKE, FAKE,
                                     100, FAKE, 2, 4, a["L_cap"], a["d"], a["dt"], 0.1, 0.0, FAKE,
                                     a["ws"], NULL, NULL)
    assert call(W=64) == B.EINVAL        # W must be below L_cap
    assert call(W=0) == B.EINVAL
    assert call(dt=B.F32) == B.EUNSUP     # bf16 only
    assert call(d=72) == B.EUNSUP
    assert call(ws=ws - 4) == B.EINVAL
    assert call(cur=NULL) == B.EINVAL


def test_noalloc_decode_rejects_oversized_partials(B):
    """The allocation-free decode refuses a split launch whose partials would
    not fit in its scratch array, before any HIP call (no GPU needed)."""
    f = B.lib.compacted_decode_attn_noalloc
    b, H, d, L_cap = 1, 511, 80, 200000
    assert B.sckv_decode_workspace_bytes(b, H, L_cap, d) > B.NOALLOC_SCRATCH_BYTES
    rc = f(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 4, FAKE, b, H, L_cap, d, B.BF16,
           0.1, 0.0, NULL, NULL)
    assert rc == B.EUNSUP
    assert "scratch" in B.last_error()
    # argument checks come first, as for compacted_decode_attn
    assert f(NULL, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 4, FAKE, 1, 1, 10, 80, B.BF16,
             0.1, 0.0, NULL, NULL) == B.EINVAL
    assert f(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 4, FAKE, 1, 1, 10, 96, B.BF16,
             0.1, 0.0, NULL, NULL) == B.EUNSUP


def test_binding_rejects_host_tensors(B):
    """The binding checks every device argument before the C call: host
    tensors never reach a kernel as device pointers."""
    import torch
    x = torch.zeros((1, 1, 64), dtype=torch.bfloat16)
    i = torch.zeros(1, dtype=torch.int32)
    with pytest.raises(B.SckvError) as e:
        B.compacted_decode_attn(x, x, x, x, x, i, i, i, None, 1, x, 1, 1, 1, 64, 0.1, 0.0,
                                torch.zeros(16, dtype=torch.uint8))
    assert e.value.code == B.EINVAL and "device" in str(e.value)
