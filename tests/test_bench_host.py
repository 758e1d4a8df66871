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


@pytest.mark.parametrize("L,ratio,seed", [(64, 0.3, 5), (300, 0.6, 6), (513, 0.9, 7)])
def test_kept_rows_equal_oracle_keep_flags(L, ratio, seed):
    spans = random_spans(L, ratio, seed)
    types = O.token_types(spans, L)
    for P in sorted({1, L // 3, L // 2, L - 1, L}):
        sub = [(c, r) for c, r in spans if c < P]
        assert bench.kept_rows(sub, P) == int(O.keep_rows(types[:P], P).sum())


def test_multi_gpu_request_exits_with_message():
    r = subprocess.run([sys.executable, "bench.py", "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr
