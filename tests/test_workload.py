"""Properties of the seeded input generators (harness only)."""
import numpy as np
import pytest

from paper_2310_08152_amd import workload as W


def _valid(spans, L_total):
    for (c, r), (c2, _) in zip(spans, spans[1:]):
        assert c < r < c2, (c, r, c2)
    for c, r in spans:
        assert 0 <= c < L_total and r > c


@pytest.mark.parametrize("name", list(W.WORKLOADS))
def test_workload_spans_are_valid_and_deterministic(name):
    w = W.get_workload(name)
    a = W.workload_spans(w)
    b = W.workload_spans(w)
    assert a == b
    assert len(a) == w.batch
    for s in a:
        _valid(s, w.meta_len)


def test_tiny_spans():
    s = W.workload_spans(W.get_workload("tiny-f32"))[0]
    assert s == [(32 * k + 8, 32 * k + 24) for k in range(8)]


def test_window_spans_ratio_and_jitter():
    w = W.get_workload("opt1.3b-prefill")
    for s in W.workload_spans(w):
        assert len(s) == 32
        assert W.span_coverage(s, w.seq_len) == w.seq_len // 2
        for k, (c, r) in enumerate(s):
            assert abs(c - (64 * k + 16)) <= 4 and r - c == 32


@pytest.mark.parametrize("name,ratio", [("opt1.3b-decode", 0.75), ("3b-rope", 0.5)])
def test_uniform_spans_exact_ratio(name, ratio):
    w = W.get_workload(name)
    for s in W.workload_spans(w):
        assert W.span_coverage(s, w.seq_len) == int(round(ratio * w.seq_len))
        assert all(r < w.seq_len for _, r in s)
        lengths = [r - c for c, r in s]
        assert max(lengths) <= 64


def test_streaming_schedule():
    w = W.get_workload("3b-rope-stream")
    s = W.workload_spans(w)[0]
    closed = [x for x in s if x[1] < w.meta_len]
    assert len(closed) == 21 and len(s) == 22
    assert all(r - c == 32 for c, r in s)
    assert s[0] == (1032, 1064)


def test_randn_rounds_to_bf16():
    import torch
    x = W.randn((4, 5), seed=3, dtype="bf16")
    assert x.dtype == torch.bfloat16
    y = W.randn((4, 5), seed=3, dtype="f32")
    assert torch.equal(x, y.to(torch.bfloat16))
