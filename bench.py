"""Benchmark of the sentinel-token compression hot path on one MI355X.

One step = the whole path on one batch of the 3B-RoPE-shaped workload
(32 layers, b=16, H=32, d_head=80, L=4096 transformed prompt tokens, half of
them in <CL>..<CR> spans, rotary theta 10000):
  * per layer: rotary embedding of Q and K at tied positions (K, and V, are
    written into the layer's cache slice) and span-masked prefill attention;
  * compaction of the whole (32, 2, 16, 32, 4096, 80) cache at the end of the
    prompt (frees the closed spans' rows in place);
  * 128 generated tokens: per token, 32 decode launches (one per layer: fused
    rotary + append + split-K attention over the compacted cache) and one
    commit.
Inputs (prompt Q/K/V of every layer, the generated tokens' q/k/v) are
synthetic N(0,1) bf16 tensors resident in HBM before timing starts.

value = compacted-decode attention HBM throughput (algorithmic bytes of all
decode launches / their summed HIP-event durations); the masked-prefill
TFLOP/s is reported beside it (roofline_prefill).

The same line then carries, under "configs", the other workloads the metric
names, each timed on its own after the previous one's buffers are freed:
the OPT-1.3B-shaped prefill slice (b=8, H=32, d=64, L=2048), the OPT-1.3B-
shaped compaction + 128 decode steps (24 layers, b=64), and the streaming
workload (b=256, 1024 generated tokens, compaction after every <CR>) over
its compressed cache.  cpu_baseline and cpu_baseline_prefill time the
oracle's decode and prefill on a bounded sample, one thread per host core.
Prints one JSON line.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, published
BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 MFMA, published
F32_PEAK_TFLOPS = 157.3        # MI355X dense fp32 MFMA, published
PF_BQ, PF_BK = 128, 64         # prefill query block / gathered key tile


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="3b-rope")
    ap.add_argument("--decode-steps", type=int, default=None)
    ap.add_argument("--launch-events", choices=["all", "none"], default="all")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="wall seconds of each CPU-baseline leg (decode, prefill)")
    ap.add_argument("--gen-tokens", type=int, default=None,
                    help="streaming workload: generated tokens per run (default: all)")
    ap.add_argument("--prefill-block", type=int, default=0,
                    help="process the prompt in blocks of this many tokens, freeing closed "
                         "spans after each block (0: one-shot prefill)")
    ap.add_argument("--local-attention", action="store_true",
                    help="the local-attention comparator: decode over a ring of the W most "
                         "recent tokens, W = the rows the compressed cache holds at its largest")
    ap.add_argument("--no-extra-configs", action="store_true",
                    help="the headline workload only (by default the OPT-1.3B prefill, the "
                         "OPT-1.3B compaction + decode and the streaming workload follow it)")
    ap.add_argument("--stream-tokens", type=int, default=None,
                    help="generated tokens of the streaming run among the extra configs "
                         "(default: all 1024)")
    ap.add_argument("--span-sweep", action="store_true",
                    help="span lengths U(2,25) at each of --sweep-ratios instead of the "
                         "workload's own spans")
    ap.add_argument("--sweep-ratios", type=float, nargs="+",
                    default=[0.1, 0.3, 0.5, 0.7, 0.9])
    return ap.parse_args()


# ---------------------------------------------------------------------------
# work accounting (host side, from the generated spans)
# ---------------------------------------------------------------------------

def last_visible_row(spans, L):
    """Per column j: the last row that may attend to it (the mask's column
    reach; <CL> columns reach only themselves)."""
    vu = np.full(L, np.iinfo(np.int64).max, dtype=np.int64)
    for c, r in spans:
        if c < L:
            vu[c] = c
            vu[c + 1:min(r, L)] = r
    return vu


def prefill_work(spans_all, L, H, d):
    """(algorithmic flops, executed flops) of one layer's prefill: 4*d per
    visible (row, column) pair, and 4*d per pair of every 32x64 tile a wave
    multiplies (at d=64 the kernel skips a tile's second 32-key block where
    it lies past the list's end or starts after the wave's last row, and such
    a tile counts 32x32)."""
    alg = 0
    exe = 0
    for spans in spans_all:
        vu = last_visible_row(spans, L)
        cl = vu == np.arange(L)
        # visible pairs: column j is seen by rows j..min(vu_j, L-1), CL only by itself
        reach = np.minimum(vu, L - 1) - np.arange(L) + 1
        nnz = int(reach.sum())
        # CL rows see only themselves: remove what they would otherwise see
        for i in np.nonzero(cl)[0]:
            vis = int(((np.arange(i + 1) <= i) & (vu[:i + 1] >= i)).sum())
            nnz -= vis - 1
        alg += nnz
        for I in range(0, L, PF_BQ):
            jend = min(I + PF_BQ, L)
            cols = np.nonzero(vu[:jend] >= I)[0]
            nt = (len(cols) + PF_BK - 1) // PF_BK
            for w in range(4):
                Iw = I + 32 * w
                if Iw >= L:
                    continue
                jmin = cols[::PF_BK][:nt]
                done = jmin <= Iw + 31
                exe += int(done.sum()) * PF_BK * 32
                if d == 64 and nt:
                    second = np.arange(nt) * PF_BK + 32  # list index of each tile's second block
                    has2 = second < len(cols)
                    j32 = cols[np.minimum(second, len(cols) - 1)]
                    skip2 = ~has2 | (j32 > Iw + 31)
                    exe -= int((done & skip2).sum()) * 32 * 32
    return 4 * d * alg * H, 4 * d * exe * H


def kept_rows(spans, L):
    """Rows left after freeing every span closed before index L (closed form:
    L minus the closed spans' lengths minus the <CL> of a span still open)."""
    closed = sum(r - c for c, r in spans if r < L)
    open_cl = sum(1 for c, r in spans if c < L <= r)
    return L - closed - open_cl


def decode_call_bytes(n_keep, t, H, d, elt=2):
    """Algorithmic HBM bytes of one decode call (one layer) at generated step
    t after a prompt whose compaction left n_keep[s] rows per sequence: the
    n_keep + t cache rows held before the step's own row (key and value), q,
    k_new and v_new read, o and the new key/value row written."""
    n_keep = np.asarray(n_keep, dtype=np.int64)
    b = len(n_keep)
    return int((n_keep + t).sum()) * H * d * elt * 2 + 6 * b * H * d * elt


# ---------------------------------------------------------------------------
# HBM traffic from stored rocprof counter summaries
# ---------------------------------------------------------------------------

def stored_traffic(name, workload):
    """Calibrated HBM bytes per dispatch summed over the kernels of a stored
    rocprof summary, or None if it is missing, for another workload, or
    taken from kernel sources that have changed since."""
    path = os.path.join(ROOT, "profiles", name)
    if not os.path.exists(path):
        return None
    with open(path) as f:
        d = json.load(f)
    from paper_2310_08152_amd.rocprof_summary import sources_hash
    if d.get("workload") != workload:
        return None
    if sources_hash([os.path.join(ROOT, x) for x in d["sources"]]) != d["sources_hash"]:
        return None
    return sum(k["hbm_bytes"] for k in d["kernels"].values())


def stored_mfma_busy(name, workload, kernel):
    """Share of the matrix cores' clocks a kernel kept busy, from a stored SQ
    counter summary, or None if it is missing, for another workload, or taken
    from kernel sources that have changed since."""
    path = os.path.join(ROOT, "profiles", name)
    if not os.path.exists(path):
        return None
    with open(path) as f:
        d = json.load(f)
    from paper_2310_08152_amd.rocprof_summary import sources_hash
    if d.get("workload") != workload:
        return None
    if sources_hash([os.path.join(ROOT, x) for x in d["sources"]]) != d["sources_hash"]:
        return None
    k = d["kernels"].get(kernel, {})
    return None if "mfma_busy" not in k else round(k["mfma_busy"], 4)


# ---------------------------------------------------------------------------
# CPU baseline: the oracle on a bounded sample, on the host's cores
# ---------------------------------------------------------------------------

def host_info():
    """CPU model, usable cores and host RAM of the machine the bench runs on."""
    model, ram = None, None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        with open("/proc/meminfo") as f:
            for line in f:
                if line.startswith("MemTotal"):
                    ram = round(int(line.split()[1]) / 2 ** 20, 1)
                    break
    except OSError:
        pass
    return {"cpu_model": model, "host_cores": len(os.sched_getaffinity(0)), "host_ram_gib": ram}


def run_threads(jobs, seconds):
    """Runs each job (a callable taking a deadline and returning the work it
    finished) on a thread of its own until `seconds` of wall time have
    passed; returns (total work, wall seconds).  NumPy releases the GIL in
    the oracle's array operations, so the threads run on separate cores."""
    import concurrent.futures as cf
    t0 = time.perf_counter()
    deadline = t0 + seconds
    with cf.ThreadPoolExecutor(len(jobs)) as ex:
        done = sum(ex.map(lambda j: j(deadline), jobs))
    return done, time.perf_counter() - t0


def cpu_baseline(w, spans_all, k_in, v_in, q_dec, k_dec, v_dec, seconds):
    """The oracle's decode (rotary of q and k + attention over its own
    compacted cache) on one (layer, sequence) slice per host core, all 32
    heads, step after step, for about `seconds` of wall time; bytes counted
    as for the GPU figure (cache rows read + q, k, v in, o and the new row
    out)."""
    from oracle import sckv_oracle as O
    n_thr = len(os.sched_getaffinity(0))
    L, H, d, M, b = w.seq_len, w.heads, w.d_head, w.layers, w.batch
    steps = q_dec.shape[0]
    T = L + steps
    f = lambda t: t.detach().to("cpu").double().numpy()
    jobs, done_steps = [], [0] * n_thr
    t_prep = time.perf_counter()
    for i in range(n_thr):
        m, s = i % M, (i * 7) % b
        types = O.token_types(spans_all[s], T)
        pos = O.tie_positions(types)
        K = np.stack([O.rope_rotate_half(f(k_in[m, s, h]), pos[:L], w.rope_theta)
                      for h in range(H)]) if w.rope_theta > 0 else f(k_in[m, s])
        Kc = np.zeros((H, T, d)); Vc = np.zeros((H, T, d))
        Kc[:, :L], Vc[:, :L] = K, f(v_in[m, s])
        tok = np.zeros(T, np.int64); tok[:L] = np.arange(L)
        pp = np.zeros(T, np.int64); pp[:L] = pos[:L]
        Kc, Vc, _, _, n0, _ = O.compact_cache(Kc, Vc, tok, pp, L, types, L)
        qd, kd, vd = f(q_dec[:, m, s]), f(k_dec[:, m, s]), f(v_dec[:, m, s])

        def job(deadline, i=i, Kc=Kc, Vc=Vc, n0=n0, qd=qd, kd=kd, vd=vd, pos=pos, types=types):
            work, n, st = 0, n0, 0
            while time.perf_counter() < deadline:
                t = L + st
                qr, kr = qd[st], kd[st]
                if w.rope_theta > 0:
                    qr = np.stack([O.rope_rotate_half(qd[st, h][None], [pos[t]], w.rope_theta)[0]
                                   for h in range(H)])
                    kr = np.stack([O.rope_rotate_half(kd[st, h][None], [pos[t]], w.rope_theta)[0]
                                   for h in range(H)])
                O.decode_attention(qr, kr, vd[st], Kc, Vc, n, types[t] == O.CL)
                work += n * H * d * 2 * 2 + 6 * H * d * 2
                done_steps[i] += 1
                Kc[:, n], Vc[:, n] = kr, vd[st]
                n, st = n + 1, st + 1
                if st == steps:  # start the slice's generation over
                    n, st = n0, 0
            return work
        jobs.append(job)
    t_prep = time.perf_counter() - t_prep
    done, wall = run_threads(jobs, seconds)
    return {"value": round(done / wall / 1e9, 4), "unit": "GB/s", "cores": n_thr,
            "kind": "oracle", **host_info(),
            "sample": f"fp64 NumPy oracle decode (rotary of q and k + attention over its own "
                      f"compacted cache), {n_thr} threads, each on one whole (layer, sequence) "
                      f"slice x {H} heads generating its {steps} tokens in a loop; "
                      f"{sum(done_steps)} sequence-steps in {wall:.1f} s of wall time "
                      f"(compacted caches prepared beforehand in {t_prep:.1f} s, untimed); "
                      f"bytes counted as for the GPU figure"}


def cpu_baseline_prefill(w, spans_all, q_in, k_in, v_in, seconds):
    """The oracle's masked prefill (rotary at tied positions, then dense
    fp64 attention under the explicit L x L mask) on whole (layer, sequence,
    head) slices, one thread per host core, for about `seconds` of wall
    time; algorithmic flops (4*d per visible pair) per second.  The mask of
    the sampled sequence is built once beforehand (untimed), as the GPU path
    builds its plan once per prompt."""
    from oracle import sckv_oracle as O
    n_thr = len(os.sched_getaffinity(0))
    L, H, d, M, b = w.seq_len, w.heads, w.d_head, w.layers, w.batch
    s = 1 % b
    f = lambda t: t.detach().to("cpu").double().numpy()
    t_mask = time.perf_counter()
    types = O.token_types(spans_all[s], L)
    pos = O.tie_positions(types)
    mask = O.attention_mask(types)
    nnz = int(mask.sum())
    t_mask = time.perf_counter() - t_mask
    heads = [0] * n_thr

    def job(deadline, i):
        work, k = 0, 0
        while time.perf_counter() < deadline:
            m, h = (i + k * n_thr) % M, (i * 5 + k) % H
            Q, K, V = f(q_in[m, s, h]), f(k_in[m, s, h]), f(v_in[m, s, h])
            if w.rope_theta > 0:
                Q = O.rope_rotate_half(Q, pos, w.rope_theta)
                K = O.rope_rotate_half(K, pos, w.rope_theta)
            O.masked_attention(Q[None], K[None], V[None], mask)
            work += 4 * d * nnz
            heads[i] += 1
            k += 1
        return work
    done, wall = run_threads([lambda dl, i=i: job(dl, i) for i in range(n_thr)], seconds)
    return {"value": round(done / wall / 1e12, 6), "unit": "TFLOP/s", "cores": n_thr,
            "kind": "oracle", **host_info(),
            "sample": f"fp64 NumPy oracle prefill (rotary, explicit {L}x{L} mask, dense), "
                      f"{n_thr} threads over whole (layer, sequence, head) slices of one "
                      f"sequence, {sum(heads)} slices in {wall:.1f} s of wall time (the "
                      f"sequence's mask built once beforehand in {t_mask:.1f} s, untimed); "
                      f"algorithmic flops (4*d per visible pair) as for the GPU figure"}


# ---------------------------------------------------------------------------
# streaming workload: spans open and close in the generated text
# ---------------------------------------------------------------------------

def live_rows_schedule(spans, prompt, gen):
    """Rows held after each generated token when every closed span is freed
    right after its <CR> (host bookkeeping from the span list), and the peak
    row count, reached just before a span is freed."""
    out = []
    n = prompt
    peak = prompt
    closes = {r: (r - c) for c, r in spans}
    cls = {c for c, _ in spans}
    for t in range(prompt, prompt + gen):
        if t not in cls:
            n += 1
        peak = max(peak, n)
        if t in closes:
            n -= closes[t] - 1  # the <CL> was never appended
        out.append(n)
    return out, peak


def streaming_run(w, gen, mode, warmup_tokens):
    """One streaming generation of `gen` tokens after the prompt, over the
    compressed cache (spans freed after every <CR>) or an uncompressed one
    (no spans); the cache is sized to the schedule's peak row count.
    Returns figures for the timed run, which follows an untimed warm-up of
    `warmup_tokens` tokens over the same cache."""
    import torch

    from paper_2310_08152_amd import path as P
    from paper_2310_08152_amd import workload as W

    dev = "cuda:0"
    M, b, H, d, L = w.layers, w.batch, w.heads, w.d_head, w.seq_len
    T = L + gen
    dt = W.torch_dtype(w.dtype)
    POOL = 16  # distinct synthetic token inputs, used cyclically
    qp = W.randn((POOL, M, b, H, d), seed=w.seed * 100000 + 1, dtype=w.dtype, device=dev)
    kp = W.randn((POOL, M, b, H, d), seed=w.seed * 100000 + 2, dtype=w.dtype, device=dev)
    vp = W.randn((POOL, M, b, H, d), seed=w.seed * 100000 + 3, dtype=w.dtype, device=dev)
    od = torch.empty(b, H, d, dtype=dt, device=dev)
    spans = [[(c, r) for c, r in s if c < T] for s in W.workload_spans(w)] \
        if mode == "compressed" else [[] for _ in range(b)]
    sched, peak = live_rows_schedule(spans[0], L, gen)
    L_cap = peak
    cr_steps = {r for c, r in spans[0] if L <= r < T}
    meta = P.SpanMeta(spans, T, dev)
    cache = P.KVCache(M, b, H, L_cap, d, dt, dev)
    for m in range(M):
        for kv in range(2):
            cache.kv[m, kv, :, :, :L].copy_(W.randn((b, H, L, d), seed=w.seed * 1000 + m * 2 + kv,
                                                    dtype=w.dtype, device=dev))
    ws = P.Workspace(b, H, 1, L_cap, d, dev)

    def loop(n_tok):
        cache.start_prompt(L, meta)
        for t in range(n_tok):
            i = t % POOL
            for m in range(M):
                P.decode_layer(qp[i, m], kp[i, m], vp[i, m], cache, m, meta, ws, od,
                               theta=w.rope_theta)
            cache.commit(meta)
            if L + t in cr_steps:
                cache.compact(meta)

    if warmup_tokens:
        loop(min(warmup_tokens, gen))
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    loop(gen)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1)
    if int(cache.status):
        raise RuntimeError(f"device status {int(cache.status)}")
    assert cache.kv_len.tolist() == [sched[-1]] * b, (cache.kv_len.tolist()[:4], sched[-1])
    row_b = d * 2
    # rows read by the decode launches: every step attends to the rows held
    # before its own (sched[t-1], the prompt's L at the first step)
    rows_read = sum([L] + sched[:-1])
    attn_bytes = rows_read * b * H * M * row_b * 2 + gen * M * 6 * b * H * d * 2
    gbs = attn_bytes / (ms * 1e-3) / 1e9
    return {"tokens_per_s": round(b * gen / (ms * 1e-3), 1), "ms": round(ms, 2),
            "generated": gen, "peak_rows": peak, "final_rows": sched[-1],
            "span_closes": len([r for r in cr_steps if r < L + gen]),
            "cache_bytes": int(cache.kv.numel() * cache.kv.element_size()),
            "attn_gbs": round(gbs, 1), "attn_frac_of_hbm": round(gbs / HBM_PEAK_GBS, 4),
            "attn_gbs_note": "decode bytes (cache rows read + q/k/v in, o and the new row out) "
                             "over the whole loop's time, commits and compactions included"}


def run_streaming(args, w):
    import torch

    gen = w.gen_tokens if args.gen_tokens is None else args.gen_tokens
    M, b, H, d, L = w.layers, w.batch, w.heads, w.d_head, w.seq_len
    results = {}
    for mode in ("compressed", "uncompressed"):
        results[mode] = streaming_run(w, gen, mode, gen if args.warmup else 0)
        torch.cuda.empty_cache()
    c, u = results["compressed"], results["uncompressed"]
    out = {
        "metric": "streaming attention tokens/s and peak KV bytes, compressed vs uncompressed cache",
        "value": c["tokens_per_s"], "unit": "tokens/s", "n_gpus": 1, "steps": 1,
        "warmup": args.warmup, "ms_per_step": c["ms"], "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": w.dtype, "data": "synthetic",
        "config": {"workload": f"{w.name}: decode {gen} tokens after a {L}-token prompt, "
                               f"in-place compaction after every <CR>", "layers": M, "batch": b,
                   "heads": H, "d_head": d, "prompt": L, "generated": gen,
                   "parallelism": "single-gpu"},
        "compressed": c, "uncompressed": u,
        "speedup_vs_uncompressed": round(c["tokens_per_s"] / u["tokens_per_s"], 3),
        "kv_bytes_saved": u["cache_bytes"] - c["cache_bytes"],
    }
    print(json.dumps(out), flush=True)


def extra_configs(args):
    """The other workloads the metric names, each timed on its own after the
    headline workload's buffers are freed: the OPT-1.3B-shaped prefill slice,
    the OPT-1.3B-shaped compaction + decode, and the streaming workload over
    its compressed cache."""
    import copy

    import torch

    from paper_2310_08152_amd import workload as W

    out = {}
    a = copy.copy(args)
    a.no_cpu_baseline = True
    a.decode_steps = None
    w2 = W.get_workload("opt1.3b-prefill")
    r = measure(a, w2)
    pf = r["roofline"]
    out[w2.name] = {
        "workload": f"{w2.name}: masked prefill, {w2.layers} layer, b={w2.batch}, H={w2.heads}, "
                    f"d={w2.d_head}, L={w2.seq_len}, {r['config']['evicted']:.0%} freed",
        "prefill_tflops_algorithmic": pf["achieved"], "frac_algorithmic": pf["frac"],
        "prefill_tflops_executed": pf["executed_tflops"],
        "frac_executed": round(pf["executed_tflops"] / pf["peak"], 4),
        "executed_over_algorithmic": pf["executed_over_algorithmic"],
        "floors_us": pf["floors_us"], "frac_of_roofline": pf["frac_of_roofline"],
        "avg_launch_us": pf["avg_launch_us"], "plan_us": pf["plan_us"],
        "traffic": stored_traffic("traffic_prefill_opt1.3b-prefill.json", f"{w2.name}/steps0"),
        "traffic_unit": "HBM bytes per call (rocprofv3 FETCH_SIZE + WRITE_SIZE, calibrated)",
        "mfma_busy": stored_mfma_busy("mfma_opt1.3b-prefill.json", f"{w2.name}/steps0",
                                      "prefill_attn_kernel"),
        "timed_steps": a.steps}
    torch.cuda.empty_cache()
    w3 = W.get_workload("opt1.3b-decode")
    a.steps, a.warmup = min(args.steps, 3), 1
    r = measure(a, w3)
    dec, pf = r["roofline"], r["roofline_prefill"]
    out[w3.name] = {
        "workload": f"{w3.name}: {w3.layers} layers, b={w3.batch}, H={w3.heads}, d={w3.d_head}, "
                    f"L={w3.seq_len}, {r['config']['evicted']:.0%} freed, "
                    f"{w3.decode_steps} decode steps",
        "decode_gbs": dec["achieved"], "decode_frac": dec["frac"],
        "decode_avg_launch_us": dec["avg_launch_us"], "decode_bytes_per_launch":
            dec["bytes_per_launch"],
        "compaction_gbs": r["compaction_gbs"],
        "compaction_frac": round(r["compaction_gbs"] / HBM_PEAK_GBS, 4),
        "compaction_bytes": r["compaction_bytes"], "compaction_ms": r["phases_ms"]["compaction"],
        "decode_traffic": stored_traffic("traffic_decode_opt1.3b-decode.json",
                                         f"{w3.name}/steps{w3.decode_steps}"),
        "compaction_traffic": stored_traffic("traffic_compact_opt1.3b-decode.json",
                                             f"{w3.name}/steps{w3.decode_steps}"),
        "prefill_tflops_algorithmic": pf["achieved"], "prefill_frac_algorithmic": pf["frac"],
        "prefill_tflops_executed": pf["executed_tflops"],
        "decode_tokens_per_s": r["decode_tokens_per_s"], "timed_steps": a.steps}
    torch.cuda.empty_cache()
    w5 = W.get_workload("3b-rope-stream")
    gen = w5.gen_tokens if args.stream_tokens is None else args.stream_tokens
    c = streaming_run(w5, gen, "compressed", 16)
    out[w5.name] = {"workload": f"{w5.name}: {w5.layers} layers, b={w5.batch}, H={w5.heads}, "
                                f"d={w5.d_head}, prompt {w5.seq_len}, {gen} generated tokens, "
                                f"compressed cache, compaction after every <CR>", **c}
    torch.cuda.empty_cache()
    return out


# ---------------------------------------------------------------------------
# main
# ---------------------------------------------------------------------------

def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only: the sentinel-token compression path shards "
              "over sequences/heads/layers with no exchange between GPUs, and no multi-GPU "
              "figure is produced (pass --gpus 1).", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2310_08152_amd import workload as W

    torch.cuda.set_device(0)
    w = W.get_workload(args.workload)
    if w.gen_tokens > 0:
        return run_streaming(args, w)
    if args.span_sweep:
        return run_span_sweep(args, w)
    if args.local_attention:
        return run_local_attention(args, w)
    out = measure(args, w)
    if args.workload == "3b-rope" and args.prefill_block == 0 and not args.no_extra_configs:
        torch.cuda.empty_cache()
        out["configs"] = extra_configs(args)
    print(json.dumps(out), flush=True)


def measure(args, w):
    """One bench line for a prefill (+ compaction + decode) workload."""
    import torch

    from paper_2310_08152_amd import path as P
    from paper_2310_08152_amd import workload as W

    dev = "cuda:0"
    steps = w.decode_steps if args.decode_steps is None else args.decode_steps
    M, b, H, d, L = w.layers, w.batch, w.heads, w.d_head, w.seq_len
    theta = w.rope_theta
    T = L + steps
    spans_all = W.workload_spans(w)
    pb = args.prefill_block
    L_cap_one_shot = max(L, max(kept_rows(s, L) for s in spans_all) + steps)
    if pb > 0:
        # block-wise prompt: the cache holds the survivors of earlier blocks
        # plus one block, then the decode rows
        peak = max(kept_rows(s, B0) + min(pb, L - B0) for s in spans_all for B0 in range(0, L, pb))
        L_cap = max(peak, max(kept_rows(s, L) for s in spans_all) + steps)
    else:
        L_cap = L_cap_one_shot

    # ---- inputs resident in HBM ----
    dt = W.torch_dtype(w.dtype)
    q_in = torch.empty(M, b, H, L, d, dtype=dt, device=dev)
    k_in = torch.empty_like(q_in)
    v_in = torch.empty_like(q_in)
    for m in range(M):
        for i, t in enumerate((q_in, k_in, v_in)):
            t[m].copy_(W.randn((b, H, L, d), seed=w.seed * 100000 + m * 10 + i, dtype=w.dtype,
                               device=dev))
    q_dec = W.randn((steps, M, b, H, d), seed=w.seed * 100000 + 7001, dtype=w.dtype, device=dev)
    k_dec = W.randn((steps, M, b, H, d), seed=w.seed * 100000 + 7002, dtype=w.dtype, device=dev)
    v_dec = W.randn((steps, M, b, H, d), seed=w.seed * 100000 + 7003, dtype=w.dtype, device=dev)

    meta = P.SpanMeta(spans_all, T, dev)
    cache = P.KVCache(M, b, H, L_cap, d, dt, dev)
    ws = P.Workspace(b, H, L, L_cap, d, dev, block=pb)
    qr = torch.empty(b, H, L, d, dtype=dt, device=dev)
    o = torch.empty(b, H, L, d, dtype=dt, device=dev)
    od = torch.empty(b, H, d, dtype=dt, device=dev)
    torch.cuda.synchronize()

    n_dec = steps * M
    use_ev = args.launch_events == "all"
    E = lambda: torch.cuda.Event(enable_timing=True)

    def run_step(rec):
        if rec is not None:
            rec["t0"].record()
        if pb > 0:
            # rotary, append, masked attention and freeing, block by block
            P.prefill_progressive(q_in, k_in, v_in, o.unsqueeze(0).expand(M, b, H, L, d), cache,
                                  meta, ws, L, pb, theta=theta)
            if rec is not None:
                rec["t1"].record()
                rec["t2"].record()
        else:
            cache.start_prompt(L, meta)
            # the mask's visibility plan is the same for every layer: built once
            if rec is not None and use_ev:
                rec["plan"][0].record()
            P.prefill_plan(meta, ws, b, L)
            if rec is not None and use_ev:
                rec["plan"][1].record()
            for m in range(M):
                P.rope_rows(q_in[m], qr, meta, L, 0, theta)
                P.rope_rows(k_in[m], cache.k(m), meta, L, 0, theta)
                P.rope_rows(v_in[m], cache.v(m), meta, L, 0, 0.0)
                if rec is not None and use_ev:
                    rec["pf"][m][0].record()
                P.prefill_layer(qr, cache.k(m), cache.v(m), o, meta, ws, L, planned=True)
                if rec is not None and use_ev:
                    rec["pf"][m][1].record()
            if rec is not None:
                rec["t1"].record()
            cache.compact(meta)
            if rec is not None:
                rec["t2"].record()
        for t in range(steps):
            # one event pair around the M back-to-back decode calls of a step:
            # a pair around every call would add the events' own overhead to
            # each call
            if rec is not None and use_ev:
                rec["dec"][t][0].record()
            for m in range(M):
                P.decode_layer(q_dec[t, m], k_dec[t, m], v_dec[t, m], cache, m, meta, ws, od,
                               theta=theta)
            if rec is not None and use_ev:
                rec["dec"][t][1].record()
            cache.commit(meta)
        if rec is not None:
            rec["t3"].record()

    for _ in range(args.warmup):
        run_step(None)
    torch.cuda.synchronize()
    recs = []
    for _ in range(args.steps):
        recs.append({"t0": E(), "t1": E(), "t2": E(), "t3": E(),
                     "pf": [(E(), E()) for _ in range(M)] if use_ev and pb == 0 else None,
                     "plan": (E(), E()) if use_ev and pb == 0 else None,
                     "dec": [(E(), E()) for _ in range(steps)] if use_ev else None})
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    for r in recs:
        run_step(r)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    status = int(cache.status)
    if status:
        raise RuntimeError(f"device status {status}")

    # ---- accounting ----
    n_keep = np.array([kept_rows(s, L) for s in spans_all], dtype=np.int64)
    assert np.array_equal(cache.kv_len.cpu().numpy(), n_keep + steps), "unexpected kv_len"
    dec_bytes = [decode_call_bytes(n_keep, t, H, d) for t in range(steps)]
    dec_bytes_step = M * sum(dec_bytes)
    pf_alg, pf_exe = prefill_work(spans_all, L, H, d)
    comp_bytes = 0
    for spans in spans_all:
        vu = last_visible_row(spans, L)
        keep = (vu != np.arange(L)) & (vu >= L)
        rank = np.cumsum(keep) - 1
        comp_bytes += int((keep & (rank != np.arange(L))).sum())
    comp_bytes *= 2 * M * H * d * 2 * 2      # read + write of every moved row, K and V

    step_ms = [r["t0"].elapsed_time(r["t3"]) for r in recs]
    pre_ms = [r["t0"].elapsed_time(r["t1"]) for r in recs]
    cmp_ms = [r["t1"].elapsed_time(r["t2"]) for r in recs]
    decph_ms = [r["t2"].elapsed_time(r["t3"]) for r in recs]
    if use_ev:
        dec_step_ms = np.array([[a.elapsed_time(z) for a, z in r["dec"]] for r in recs])
        pf_launch_ms = (np.array([[a.elapsed_time(z) for a, z in r["pf"]] for r in recs])
                        if pb == 0 else np.array(pre_ms) / M)
        dec_total_ms = float(dec_step_ms.sum(axis=1).mean())
        dec_avg_ms = dec_total_ms / max(n_dec, 1)
        pf_avg_ms = float(pf_launch_ms.mean())
        plan_ms = (float(np.mean([r["plan"][0].elapsed_time(r["plan"][1]) for r in recs]))
                   if pb == 0 else None)
    else:
        plan_ms = None
        dec_avg_ms = float(np.mean(decph_ms)) / max(n_dec, 1)
        pf_avg_ms = float(np.mean(pre_ms)) / M
        dec_total_ms = float(np.mean(decph_ms))
    if n_dec == 0:
        dec_total_ms = dec_avg_ms = float("nan")
    dec_gbs = dec_bytes_step / (dec_total_ms * 1e-3) / 1e9 if n_dec else float("nan")
    dec_bytes_launch = dec_bytes_step / n_dec if n_dec else 0.0
    pf_tflops_exe = pf_exe / (pf_avg_ms * 1e-3) / 1e12
    pf_tflops_alg = pf_alg / (pf_avg_ms * 1e-3) / 1e12
    mfma_peak = BF16_PEAK_TFLOPS if w.dtype == "bf16" else F32_PEAK_TFLOPS
    pf_ref_bytes = 4 * b * H * L * d * (2 if w.dtype == "bf16" else 4)  # Q, K, V in, O out
    ms_per_step = float(np.mean(step_ms))

    # the library's launch shape: one workgroup per (sequence, head) slice from
    # 512 slices on, chunks plus a merge kernel below
    if b * H >= 512:
        dec_kernel = "decode_mfma_kernel"
        dec_launch = "one compacted_decode_attn call = one kernel, one workgroup per (sequence, head)"
    else:
        dec_kernel = "decode_mfma_kernel + decode_combine_kernel"
        dec_launch = "one compacted_decode_attn call = chunk kernel + combine kernel"
    wl_key = f"{w.name}/steps{steps}"
    dec_traffic = stored_traffic("traffic_decode_3b-rope.json", wl_key)
    pf_traffic = stored_traffic("traffic_prefill_3b-rope.json", wl_key)
    cmp_traffic = stored_traffic("traffic_compact_3b-rope.json", wl_key)
    out = {
        "metric": "compacted-decode attn HBM GB/s + masked-prefill TFLOP/s vs MI355X roofline",
        "value": round(dec_gbs, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": f"{w.name}: prefill+compaction+decode", "layers": M, "batch": b,
                   "heads": H, "d_head": d, "seq_len": L,
                   "evicted": round(1.0 - float(n_keep.mean()) / L, 4),
                   "decode_steps": steps, "rope_theta": theta, "L_cap": L_cap,
                   "parallelism": "single-gpu"},
        "roofline": {"bound": "hbm", "kernel": dec_kernel + " (compacted_decode_attn)",
                     "achieved": round(dec_bytes_launch / (dec_avg_ms * 1e-3) / 1e9, 1),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(dec_bytes_launch / (dec_avg_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                     "traffic": None if dec_traffic is None else int(dec_traffic),
                     "traffic_over_algorithmic": None if dec_traffic is None
                     else round(dec_traffic / dec_bytes_launch, 4),
                     "avg_launch_us": round(dec_avg_ms * 1e3, 2),
                     "bytes_per_launch": int(dec_bytes_launch),
                     "launch": dec_launch},
        "roofline_prefill": {"bound": "mfma",
                             "kernel": "prefill_attn_kernel (span_masked_prefill_attn_planned; "
                                       "the plan kernel runs once per prompt, plan_us)",
                             "achieved": round(pf_tflops_alg, 1), "peak": mfma_peak,
                             "unit": "TFLOP/s", "frac": round(pf_tflops_alg / mfma_peak, 4),
                             "executed_tflops": round(pf_tflops_exe, 1),
                             "executed_over_algorithmic": round(pf_exe / pf_alg, 3),
                             # the two roofline floors of one call: algorithmic flops at
                             # the MFMA peak, Q, K, V read and O written once at the HBM peak
                             "floors_us": {"mfma": round(pf_alg / mfma_peak / 1e6, 1),
                                           "hbm": round(pf_ref_bytes / HBM_PEAK_GBS / 1e3, 1)},
                             "frac_of_roofline": round(max(pf_alg / mfma_peak / 1e6,
                                                           pf_ref_bytes / HBM_PEAK_GBS / 1e3)
                                                       / (pf_avg_ms * 1e3), 4),
                             "avg_launch_us": round(pf_avg_ms * 1e3, 1),
                             "plan_us": None if plan_ms is None else round(plan_ms * 1e3, 1),
                             "traffic": None if pf_traffic is None else int(pf_traffic),
                             "traffic_unit": "HBM bytes per call (Q, K, V read; O written)",
                             "mfma_busy": stored_mfma_busy("mfma_3b-rope.json", wl_key,
                                                           "prefill_attn_kernel"),
                             "mfma_busy_unit": "share of the matrix cores' clocks busy "
                                               "(SQ counters, profiles/mfma_3b-rope.json)"},
        "phases_ms": {"rope+prefill": round(float(np.mean(pre_ms)), 3),
                      "compaction": round(float(np.mean(cmp_ms)), 3),
                      "decode": round(float(np.mean(decph_ms)), 3)},
        "compaction_gbs": (round(comp_bytes / (float(np.mean(cmp_ms)) * 1e-3) / 1e9, 1)
                           if pb == 0 else None),
        "compaction_bytes": int(comp_bytes),
        "compaction_traffic": None if cmp_traffic is None else int(cmp_traffic),
        "wall_s_timed": round(wall, 3),
    }
    if steps == 0:
        # a prefill-only workload: the line reports the masked prefill
        pf = out.pop("roofline_prefill")
        for k in ("roofline", "vs_baseline"):
            out.pop(k)
        out["value"] = pf["achieved"]
        out["unit"] = "TFLOP/s"
        out["vs_baseline"] = None
        out["roofline"] = pf
        out["phases_ms"].pop("decode")
        out["config"]["workload"] = f"{w.name}: masked prefill (+ compaction)"
        out["config"].pop("decode_steps")
        if not args.no_cpu_baseline:
            out["cpu_baseline"] = cpu_baseline_prefill(w, spans_all, q_in, k_in, v_in,
                                                       args.cpu_seconds)
    elif not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w, spans_all, k_in, v_in, q_dec, k_dec, v_dec,
                                           args.cpu_seconds)
        # the oracle's prefill beside roofline_prefill
        out["cpu_baseline_prefill"] = cpu_baseline_prefill(w, spans_all, q_in, k_in, v_in,
                                                           args.cpu_seconds)
    elt = 2 if w.dtype == "bf16" else 4
    live = int(n_keep.max()) + steps  # rows held by the longest sequence at the last step
    if pb > 0:
        # the prompt phase holds rotary, appends, attention and compaction of
        # every block; prefill figures are per layer of that phase
        out["prefill_block"] = pb
        out["roofline_prefill"]["kernel"] = ("prompt phase per layer, block-wise: rope_apply_at + "
                                             "span_masked_prefill_attn_cached + kv_compact")
        # the stored counter figures are the one-shot kernel's, not this phase's
        out["roofline_prefill"]["traffic"] = out["roofline_prefill"]["mfma_busy"] = None
        out["phases_ms"]["prompt_blockwise"] = out["phases_ms"].pop("rope+prefill")
        out["phases_ms"].pop("compaction", None)
        out["compaction_gbs"] = out["compaction_bytes"] = out["compaction_traffic"] = None
        out["kv_rows_capacity"] = int(L_cap)
        out["kv_rows_capacity_one_shot"] = int(L_cap_one_shot)
    out["kv_rows_decode_max"] = live
    out["kv_bytes_decode"] = int(M * 2 * b * H * live * d * elt)
    out["kv_bytes_allocated"] = int(M * 2 * b * H * L_cap * d * elt)
    out["decode_tokens_per_s"] = (round(b * steps / (float(np.mean(decph_ms)) * 1e-3), 1)
                                  if steps else None)
    return out


def run_local_attention(args, w):
    """Decode of the workload's shape with the local-attention comparator at an
    equal KV budget: each token attends to the W most recent tokens, held in a
    ring of W rows, where W is the largest row count the compressed cache
    reaches (survivors of the prompt plus the generated tokens)."""
    import torch

    from paper_2310_08152_amd import path as P
    from paper_2310_08152_amd import workload as W_

    dev = "cuda:0"
    steps = w.decode_steps if args.decode_steps is None else args.decode_steps
    M, b, H, d, L = w.layers, w.batch, w.heads, w.d_head, w.seq_len
    theta = w.rope_theta
    spans_all = W_.workload_spans(w)
    Wr = max(kept_rows(s, L) for s in spans_all) + steps
    L_cap = Wr + 1
    dt = W_.torch_dtype(w.dtype)
    meta = P.SpanMeta([[] for _ in range(b)], L + steps, dev)
    cache = P.KVCache(M, b, H, L_cap, d, dt, dev)
    ws = P.Workspace(b, H, 1, L_cap, d, dev)
    for m in range(M):
        for i, kv in enumerate((cache.k(m), cache.v(m))):
            x = W_.randn((b, H, L, d), seed=w.seed * 100000 + m * 10 + 1 + i, dtype=w.dtype,
                         device=dev)
            P.ring_fill(x, kv, Wr, L, meta, theta if i == 0 else 0.0, L_cap)
            del x
    q_dec = W_.randn((steps, M, b, H, d), seed=w.seed * 100000 + 7001, dtype=w.dtype, device=dev)
    k_dec = W_.randn((steps, M, b, H, d), seed=w.seed * 100000 + 7002, dtype=w.dtype, device=dev)
    v_dec = W_.randn((steps, M, b, H, d), seed=w.seed * 100000 + 7003, dtype=w.dtype, device=dev)
    od = torch.empty(b, H, d, dtype=dt, device=dev)
    E = lambda: torch.cuda.Event(enable_timing=True)

    def run(rec):
        cache.cur_tok.fill_(L)
        for t in range(steps):
            if rec is not None:
                rec[t][0].record()
            for m in range(M):
                P.local_decode_layer(q_dec[t, m], k_dec[t, m], v_dec[t, m], cache, m, Wr, meta, ws,
                                     od, theta=theta)
            if rec is not None:
                rec[t][1].record()
            cache.cur_tok.add_(1)

    for _ in range(args.warmup):
        run(None)
    torch.cuda.synchronize()
    recs = [[(E(), E()) for _ in range(steps)] for _ in range(args.steps)]
    for r in recs:
        run(r)
    torch.cuda.synchronize()
    if int(cache.status):
        raise RuntimeError(f"device status {int(cache.status)}")
    dec_ms = float(np.mean([sum(a.elapsed_time(z) for a, z in r) for r in recs]))
    call_bytes = b * H * Wr * d * 2 * 2 + 6 * b * H * d * 2
    gbs = M * steps * call_bytes / (dec_ms * 1e-3) / 1e9
    out = {"metric": "local-attention comparator: decode over a ring of the W most recent tokens",
           "value": round(gbs, 1), "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
           "warmup": args.warmup, "higher_is_better": True, "vs_baseline": None,
           "dtype": w.dtype, "data": "synthetic",
           "config": {"workload": f"{w.name} shape, local attention at equal KV budget",
                      "layers": M, "batch": b, "heads": H, "d_head": d, "prompt": L,
                      "decode_steps": steps, "ring_rows": Wr, "rope_theta": theta},
           "roofline": {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS,
                        "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4),
                        "avg_launch_us": round(dec_ms * 1e3 / (M * steps), 2),
                        "bytes_per_launch": call_bytes},
           "decode_tokens_per_s": round(b * steps / (dec_ms * 1e-3), 1),
           "kv_bytes": int(M * 2 * b * H * Wr * d * (2 if w.dtype == "bf16" else 4))}
    print(json.dumps(out), flush=True)


def run_span_sweep(args, w):
    """The paper's span distribution (lengths uniform in [2, 25]) at a range
    of compression ratios on the workload's shape: prefill, compaction and
    decode throughput and the cache held during decode, per ratio."""
    import dataclasses

    import torch

    points = []
    for r in args.sweep_ratios:
        wr = dataclasses.replace(w, name=f"{w.name} U(2,25) r={r}",
                                 span_kind="uniform", span_args=dict(ratio=r, lo=2, hi=25))
        out = measure(args, wr)
        pt = {"ratio": r, "evicted": out["config"]["evicted"],
              "prefill_tflops_executed": out["roofline_prefill"]["executed_tflops"],
              "prefill_tflops_algorithmic": out["roofline_prefill"]["achieved"],
              "prefill_executed_over_algorithmic": out["roofline_prefill"]["executed_over_algorithmic"],
              "prefill_ms_per_layer": round(out["roofline_prefill"]["avg_launch_us"] / 1e3, 4),
              "compaction_gbs": out["compaction_gbs"],
              "compaction_ms": out["phases_ms"]["compaction"],
              "decode_gbs": out["value"], "decode_frac_of_hbm": out["roofline"]["frac"],
              "decode_us_per_call": out["roofline"]["avg_launch_us"],
              "decode_tokens_per_s": out["decode_tokens_per_s"],
              "kv_rows_decode_max": out["kv_rows_decode_max"],
              "kv_bytes_decode": out["kv_bytes_decode"],
              "kv_bytes_allocated": out["kv_bytes_allocated"]}
        points.append(pt)
        print(json.dumps(pt), file=sys.stderr, flush=True)
        torch.cuda.empty_cache()
    M, b, H, d, L = w.layers, w.batch, w.heads, w.d_head, w.seq_len
    steps = w.decode_steps if args.decode_steps is None else args.decode_steps
    line = {"metric": "span-length U(2,25) sweep over compression ratio: prefill TFLOP/s, "
                      "compaction GB/s, decode GB/s and tokens/s, decode-time KV bytes",
            "value": None, "unit": None, "n_gpus": 1, "steps": args.steps,
            "warmup": args.warmup, "higher_is_better": True, "vs_baseline": None,
            "dtype": w.dtype, "data": "synthetic",
            "config": {"workload": f"{w.name} shape, spans U(2,25) at each ratio",
                       "layers": M, "batch": b, "heads": H, "d_head": d, "seq_len": L,
                       "decode_steps": steps, "rope_theta": w.rope_theta},
            "sweep": points}
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
