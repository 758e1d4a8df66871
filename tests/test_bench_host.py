"""Host-side accounting of bench.py, checked against the oracle (CPU).

The roofline figures divide by the algorithmic flop count of the masked
prefill (4*d per visible (row, column) pair) and report compaction by the
rows kept; both counts come from closed forms in bench.py.  Here they are
compared with the oracle's explicit mask and keep flags on random span sets
(Section 3.1: the mask; Section 3, "Manipulating Key-Value Memory": freeing)."""
import subprocess
import sys

import numpy as np
import pytest

import bench
from oracle import sckv_oracle as O
from paper_2310_08152_amd import workload as W


def random_spans(L, ratio, seed, open_tail=False):
    spans = W.spans_uniform_lengths(L, ratio, 2, 25, np.random.default_rng(seed))
    if open_tail and spans:
        c, _ = spans[-1]
        spans[-1] = (c, L + 5)  # still open at the end of the prefix
    return spans


@pytest.mark.parametrize("L,ratio,seed,open_tail", [(64, 0.3, 1, False), (200, 0.5, 2, False),
                                                    (257, 0.8, 3, True), (130, 0.0, 4, False)])
def test_algorithmic_pairs_equal_oracle_mask(L, ratio, seed, open_tail):
    spans = random_spans(L, ratio, seed, open_tail)
    H, d = 3, 16
    alg, exe = bench.prefill_work([spans], L, H, d)
    mask = O.attention_mask(O.token_types(spans, L))
    assert alg == 4 * d * H * int(mask.sum())
    assert exe >= alg


@pytest.mark.parametrize("L,ratio,seed,open_tail", [(200, 0.5, 2, False), (257, 0.8, 3, True),
                                                    (600, 0.9, 11, False), (130, 0.0, 4, False)])
def test_skipped_key_blocks_hold_no_visible_pair(L, ratio, seed, open_tail):
    """At d=64 the kernel skips a tile's second 32-key block where it lies past
    the block's list or starts after the wave's last row.  Against the
    oracle's mask: no skipped block holds a pair its wave's rows can see, and
    the executed count stays at or above the algorithmic one."""
    spans = random_spans(L, ratio, seed, open_tail)
    mask = O.attention_mask(O.token_types(spans, L))
    vu = bench.last_visible_row(spans, L)
    skipped = 0
    for I in range(0, L, bench.PF_BQ):
        cols = np.nonzero(vu[:min(I + bench.PF_BQ, L)] >= I)[0]
        for w in range(4):
            Iw = I + 32 * w
            if Iw >= L:
                continue
            rows = slice(Iw, min(Iw + 32, L))
            for t0 in range(0, len(cols), bench.PF_BK):
                if cols[t0] > Iw + 31:
                    continue  # the whole tile is skipped
                half = cols[t0 + 32:t0 + bench.PF_BK]
                if len(half) == 0 or half[0] > Iw + 31:
                    assert not mask[rows][:, half].any()
                    skipped += 1
    alg, exe = bench.prefill_work([spans], L, 1, 64)
    assert exe >= alg
    _, exe80 = bench.prefill_work([spans], L, 1, 80)
    assert exe80 // 80 - exe // 64 == 4 * 32 * 32 * skipped


@pytest.mark.parametrize("L,ratio,seed", [(64, 0.3, 5), (300, 0.6, 6), (513, 0.9, 7)])
def test_kept_rows_equal_oracle_keep_flags(L, ratio, seed):
    spans = random_spans(L, ratio, seed)
    types = O.token_types(spans, L)
    for P in sorted({1, L // 3, L // 2, L - 1, L}):
        sub = [(c, r) for c, r in spans if c < P]
        assert bench.kept_rows(sub, P) == int(O.keep_rows(types[:P], P).sum())


@pytest.mark.parametrize("L,ratio,seed", [(96, 0.4, 8), (300, 0.75, 9)])
def test_decode_bytes_follow_the_oracles_cache(L, ratio, seed):
    """The decode byte count of a step is the rows the oracle's compacted
    cache holds before that step (read as key and value) plus q, k, v in and
    o and the new row out, nothing for the step's own row twice."""
    H, d, steps = 2, 16, 5
    spans_all = [random_spans(L, ratio, seed + s) for s in range(3)]
    n_keep = [bench.kept_rows(sp, L) for sp in spans_all]
    for t in range(steps):
        rows = 0
        for sp in spans_all:
            types = O.token_types(sp, L + steps)
            cache = O.compact_cache(np.zeros((1, L + steps, 1)), np.zeros((1, L + steps, 1)),
                                    np.arange(L + steps), np.arange(L + steps), L, types, L)
            rows += cache[4] + t  # no spans after the prompt: every step appends
        want = rows * H * d * 2 * 2 + 6 * len(spans_all) * H * d * 2
        assert bench.decode_call_bytes(n_keep, t, H, d) == want


def test_multi_gpu_request_exits_with_message():
    r = subprocess.run([sys.executable, "bench.py", "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr
