"""Benchmark of the SparDA selection + block-sparse attention path on one MI355X.

Timed step (the headline): one decode layer at 128K context, batch 32, 32 query / 8 KV heads,
head_dim 128, 64-token blocks, k = 64 blocks (1 initial + 2 local forced):
    incremental K~ update of the block completed by the newest token
    -> Forecast scoring + top-k of every (batch, group) row
    -> block-sparse attention of all 32 query heads over the selected blocks.
value = algorithmic HBM bytes of the step / step time (GB/s); ms_per_step is the layer time.

Secondary legs on the same JSON line:
  paper_grid     -- the same decode layer with K~ on the paper's (32, 16) grid (8191 windows per
                    row, max-pooled to block scores inside the select);
  selectors      -- selection cost of the Forecast indexer against the InfLLM-V2 multi-head
                    selector it replaces (decode at 32K/128K, a prefill chunk at 128K; G = 4, 16);
  paper_config   -- decode (128K, B32) and chunked prefill (32K) at the paper's model configuration:
                    32 query / 2 KV heads, k = 96 with a 32-block local window, (32, 16) grid;
  indexer_training -- the indexer-training loss and its Forecast gradient on a 256-row chunk at
                    64K (Sec. 4.2);
  prefill_select -- the fused score + top-k kernel of a 32K chunked prefill (batch 1, every row
                    selects), reported in TFLOP/s of scored (row, candidate) pairs x 2 x 128;
  prefill_attn   -- block-sparse attention of that prefill (ms);
  pipeline       -- (with --pipeline, in a child process) the offloaded 32-layer, batch-64, 128K
                    decode step with one-layer-ahead selection and a side-stream gather from pinned
                    host pools (GB/s over PCIe, overlapped vs serial step time), and the same decode
                    run with step-to-step reuse of the staged blocks.
roofline -- the dominant kernel (decode attention): algorithmic bytes / its average duration
            measured with HIP events on the stream it runs on, against 8 TB/s.
cpu_baseline -- the CPU oracle on a sample of the decode step's rows, on this host's cores.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import paper_2606_04511_amd.sparda as sp  # noqa: E402
from paper_2606_04511_amd import inputs  # noqa: E402

HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2500.0
SCALE = 1.0 / math.sqrt(128)
METRIC = "decode select+sparse-attn us/layer & HBM GB/s at 128K; prefill select TFLOP/s"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def ws_tensor(shape, op, n_q, q_pos0, dev):
    n = sp.sparda_workspace_size(shape, op, n_q, q_pos0)
    return torch.empty(max(n, 16), dtype=torch.uint8, device=dev)


class DecodeLayer:
    """Device buffers of one decode layer at 128K and its library calls.  The timed step is the
    selection and the attention, with the compressed keys precomputed (the workload's
    definition); the one-block K~ refresh a decode step also performs is timed beside it."""

    def __init__(self, w: inputs.Workload, dev, grid=(64, 64), case=None):
        self.w = w
        T, nb = w.seq_len, w.n_blocks
        self.T, self.nb = T, nb
        self.grid = grid
        lw, sw = grid
        self.nw = (T - lw) // sw + 1  # compressed keys complete at T (one per block on the (64, 64) grid)
        self.shape = sp.SpardaShape(batch=w.batch, n_kv_heads=w.n_kv_heads, group_size=w.group_size,
                                    k_total=w.k_total, t_cap=T, nc_cap=self.nw, n_init=w.n_init, n_local=w.n_local,
                                    cmp_kernel=lw, cmp_stride=sw)
        if case is None:
            t0 = time.time()
            case = inputs.make_case(w, device=dev)
            log(f"[bench] generated {w.name} on the GPU in {time.time() - t0:.1f}s")
        self.case = c = case
        self.q, self.f, self.k, self.v = c["q"], c["f"], c["k"], c["v"]
        self.kc = torch.zeros(w.batch, w.n_kv_heads, self.nw, 128, dtype=torch.bfloat16, device=dev)
        self.sel = torch.empty(w.batch, w.n_kv_heads, 1, w.k_total, dtype=torch.int16, device=dev)
        self.cnt = torch.empty(w.batch, w.n_kv_heads, 1, dtype=torch.int16, device=dev)
        self.o = torch.empty(w.batch, w.n_q_heads, 1, 128, dtype=torch.bfloat16, device=dev)
        self.ws_sel = ws_tensor(self.shape, sp.SPARDA_OP_FORECAST_SELECT, 1, T - 1, dev)
        self.ws_att = ws_tensor(self.shape, sp.SPARDA_OP_SPARSE_ATTN, 1, T - 1, dev)
        self.ws_step = ws_tensor(self.shape, sp.SPARDA_OP_DECODE_STEP, 1, T - 1, dev)
        # K~ of every complete window is precomputed (not timed); the step refreshes the newest one.
        sp.sparda_compress_keys(self.shape, self.k, T, 0, self.nw, self.kc)
        torch.cuda.synchronize()

    def compress_new(self):
        sp.sparda_compress_keys(self.shape, self.k, self.T, self.nw - 1, self.nw, self.kc)

    def select(self):
        sp.sparda_forecast_select(self.shape, self.f, 1, self.T - 1, self.kc, self.sel, self.cnt, self.ws_sel)

    def attend(self):
        sp.sparda_sparse_attn(self.shape, self.q, 1, self.T - 1, self.k, self.v, 0, self.sel, self.cnt, SCALE, self.o,
                              self.ws_att)

    def step(self):
        """Select + attention: one fused launch where both run one workgroup per row (the 128K B32
        layer), the two calls otherwise."""
        sp.sparda_decode_step(self.shape, self.f, self.T - 1, self.kc, self.q, self.k, self.v, SCALE, self.sel,
                              self.cnt, self.o, self.ws_step)

    def step_separate(self):
        self.select()
        self.attend()

    def step_with_refresh(self):
        self.compress_new()
        self.step()

    def bytes(self):
        """Algorithmic HBM bytes of the step's parts (compress_new is the separate K~ refresh).
        The select reads every compressed key that overlaps a candidate block and is complete at
        the query: the candidate blocks themselves on the (64, 64) grid, about four windows per
        block on the (32, 16) one."""
        w = self.w
        lw, sw = self.grid
        rows = w.batch * w.n_kv_heads
        cand_lo, cand_hi = w.n_init, self.nb - 1 - w.n_local  # candidates of the decode row
        first = 0 if cand_lo * 64 - lw < 0 else (cand_lo * 64 - lw) // sw + 1
        last = min(((cand_hi + 1) * 64 - 1) // sw, (self.T - lw) // sw)
        n_keys = last - first + 1
        return {
            "compress_new": rows * (lw * 256 + 256),
            "select": rows * (256 + n_keys * 256 + w.k_total * 2 + 2),
            "attend": rows * (w.k_total * 2 * 64 * 256 + w.k_total * 2 + 2) + 2 * w.batch * w.n_q_heads * 256,
        }


def counted_traffic(kernel: str):
    """HBM bytes per launch of `kernel` from the committed rocprofv3 FETCH_SIZE / WRITE_SIZE runs
    (profiles/traffic_counters.json, calibrated on a plain 1 GiB copy), or None when the kernel's
    sources have changed since the counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "traffic_counters.json")
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        entry = json.load(fh)["kernels"].get(kernel)
    if entry is None:
        return None
    digest = hashlib.sha256(b"".join(open(os.path.join(ROOT, f), "rb").read() for f in entry["sources"])).hexdigest()
    return entry["traffic_bytes"] if digest == entry["sources_sha256"] else None


def time_events(fn, iters, stream):
    """Average ms of fn() over iters launches, HIP events on `stream` around each launch."""
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(iters)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(iters)]
    for i in range(iters):
        starts[i].record(stream)
        fn()
        ends[i].record(stream)
    torch.cuda.synchronize()
    return float(np.mean([s.elapsed_time(e) for s, e in zip(starts, ends)]))


class Flusher:
    """Reads a 1 GiB scratch buffer between timed repetitions (untimed): four times the 256 MB
    Infinity Cache and far beyond the eight 4 MB L2s, so each repetition starts from HBM.  The
    flush only reads: a flush that writes leaves the L2s full of dirty lines, and their write-back
    then lands inside the next timed call (measured: the prefill score contraction took 39.8 us
    after a 1 GiB memset, 28-29 us after a read-only pass)."""

    def __init__(self, dev):
        self.buf = torch.ones((1 << 30) // 4, dtype=torch.float32, device=dev)
        self.out = torch.empty((), dtype=torch.float32, device=dev)

    def __call__(self):
        torch.sum(self.buf, dim=0, out=self.out)


def rep_stats(fn, reps, stream, flush=None):
    """Per-launch HIP-event times of `reps` repetitions of fn() on `stream`, each after a cache
    flush when `flush` is given: median, p10, p90 and mean in ms."""
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(reps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(reps)]
    for i in range(reps):
        if flush is not None:
            flush()
        starts[i].record(stream)
        fn()
        ends[i].record(stream)
    torch.cuda.synchronize()
    t = np.array([a.elapsed_time(b) for a, b in zip(starts, ends)])
    return {"reps": reps, "median_ms": float(np.median(t)), "p10_ms": float(np.percentile(t, 10)),
            "p90_ms": float(np.percentile(t, 90)), "mean_ms": float(t.mean()), "cache_flushed": flush is not None}


def decode_small_leg(dev, reps, flush):
    """Decode at 4K (B1, k = 16) and 32K (B8, k = 64), 32 query / 8 KV heads: select + attention
    per layer, each repetition after a 1 GiB cache flush (the 32K step's 143 MB would otherwise
    stay in the Infinity Cache)."""
    stream = torch.cuda.current_stream()
    rows = []
    for name in ("decode_b1_t4k", "decode_b8_t32k"):
        w = inputs.WORKLOADS[name]
        layer = DecodeLayer(w, dev)
        for _ in range(5):
            layer.step()
        step = rep_stats(layer.step, reps, stream, flush)
        sel = rep_stats(layer.select, reps, stream, flush)
        att = rep_stats(layer.attend, reps, stream, flush)
        parts = layer.bytes()
        step_bytes = parts["select"] + parts["attend"]
        rows.append({
            "workload": f"decode layer B{w.batch} T={w.seq_len} Hq32/Hkv8 D128 block64 k{w.k_total}, select + sparse "
                        "attention on precomputed K~",
            "us_per_layer_median": step["median_ms"] * 1e3, "us_per_layer_p10": step["p10_ms"] * 1e3,
            "us_per_layer_p90": step["p90_ms"] * 1e3, "GBps_median": step_bytes / (step["median_ms"] * 1e-3) / 1e9,
            "frac_hbm_peak_median": step_bytes / (step["median_ms"] * 1e-3) / 1e9 / HBM_PEAK_GBS,
            "step_bytes": step_bytes, "select_us_median": sel["median_ms"] * 1e3,
            "attend_us_median": att["median_ms"] * 1e3, "step_stats": step})
        layer.case = None
        del layer
    return rows


def overlap_leg(layer: "DecodeLayer", dev, n_layers=32, reps=5):
    """Alg. 2's order of a decode step over n_layers layers of the 128K B32 shape (each layer
    re-using the one layer's buffers): layer l+1's selection runs on a second stream of the same
    priority while layer l attends, two (sel, cnt) sets alternating between layers and events
    ordering each attention after its selection and each selection after the attention that
    last read its set.  Reported beside the same layers run serially on one stream.  Streams
    map onto a few hardware queues, so a second stream can land on the compute stream's queue
    and serialise with it: four side streams are tried and each one's time is reported."""
    main = torch.cuda.current_stream()
    sets = [(layer.sel, layer.cnt), (torch.empty_like(layer.sel), torch.empty_like(layer.cnt))]
    ws = [layer.ws_sel, torch.empty_like(layer.ws_sel)]

    def select(i, stream):
        with torch.cuda.stream(stream):
            sp.sparda_forecast_select(layer.shape, layer.f, 1, layer.T - 1, layer.kc, sets[i][0], sets[i][1], ws[i])

    def attend(i):
        sp.sparda_sparse_attn(layer.shape, layer.q, 1, layer.T - 1, layer.k, layer.v, 0, sets[i][0], sets[i][1],
                              SCALE, layer.o, layer.ws_att)

    def serial():
        for l in range(n_layers):
            select(l % 2, main)
            attend(l % 2)

    def overlapped(side):
        ev_sel = [torch.cuda.Event(), torch.cuda.Event()]
        ev_att = [torch.cuda.Event(), torch.cuda.Event()]
        start = torch.cuda.Event()
        start.record(main)
        side.wait_event(start)
        select(0, main)
        ev_sel[0].record(main)
        for l in range(n_layers):
            cur, nxt = l % 2, 1 - l % 2
            if l + 1 < n_layers:
                if l >= 1:
                    side.wait_event(ev_att[nxt])  # attention l-1 read set nxt
                select(nxt, side)
                ev_sel[nxt].record(side)
            main.wait_event(ev_sel[cur])
            attend(cur)
            ev_att[cur].record(main)
        main.wait_event(ev_sel[(n_layers - 1) % 2])

    def wall(fn):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        fn()
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) * 1e3 / n_layers

    serial()
    ser = float(np.median([wall(serial) for _ in range(reps)]))
    per_side = []
    for _ in range(4):
        side = torch.cuda.Stream(device=dev)
        overlapped(side)
        per_side.append(float(np.median([wall(lambda: overlapped(side)) for _ in range(reps)])))
    best = min(per_side)
    return {"layers": n_layers, "us_per_layer_serial": ser * 1e3, "us_per_layer_overlapped": best * 1e3,
            "us_per_layer_overlapped_per_side_stream": [x * 1e3 for x in per_side],
            "overlap_gain": ser / best}


def prefill_leg(dev, warmup, iters, flush=None):
    w = inputs.WORKLOADS["prefill_b1_t32k"]
    T, nb = w.seq_len, w.n_blocks
    shape = sp.SpardaShape(batch=w.batch, n_kv_heads=w.n_kv_heads, group_size=w.group_size, k_total=w.k_total,
                           t_cap=T, nc_cap=nb, n_init=w.n_init, n_local=w.n_local)
    t0 = time.time()
    case = inputs.make_case(w, device=dev)
    log(f"[bench] generated {w.name} on the GPU in {time.time() - t0:.1f}s")
    kc = torch.zeros(w.batch, w.n_kv_heads, nb, 128, dtype=torch.bfloat16, device=dev)
    sp.sparda_compress_keys(shape, case["k"], T, 0, nb, kc)
    sel = torch.empty(w.batch, w.n_kv_heads, T, w.k_total, dtype=torch.int16, device=dev)
    cnt = torch.empty(w.batch, w.n_kv_heads, T, dtype=torch.int16, device=dev)
    o = torch.empty(w.batch, w.n_q_heads, T, 128, dtype=torch.bfloat16, device=dev)
    ws_s = ws_tensor(shape, sp.SPARDA_OP_FORECAST_SELECT, T, 0, dev)
    ws_a = ws_tensor(shape, sp.SPARDA_OP_SPARSE_ATTN, T, 0, dev)
    stream = torch.cuda.current_stream()

    def select():
        sp.sparda_forecast_select(shape, case["f"], T, 0, kc, sel, cnt, ws_s)

    def attend():
        sp.sparda_sparse_attn(shape, case["q"], T, 0, case["k"], case["v"], 0, sel, cnt, SCALE, o, ws_a)

    for _ in range(warmup):
        select()
    ms_sel = time_events(select, iters, stream)
    sel_stats = rep_stats(select, max(50, iters), stream, flush)
    attend()
    ms_att = time_events(attend, max(2, iters // 10), stream)

    # diagnostic: the score contraction alone (every candidate of every row scored on MFMA, each
    # row's scores reduced to their maximum on chip; no top-k, 1 float per row written)
    row_max = torch.empty(w.batch, w.n_kv_heads, T, dtype=torch.float32, device=dev)

    def score_only():
        sp.sparda_forecast_score_max(shape, case["f"], T, 0, kc, row_max)

    for _ in range(warmup):
        score_only()
    ms_score = time_events(score_only, iters, stream)
    score_stats = rep_stats(score_only, max(50, iters), stream, flush)

    # the same selection on the paper's (32, 16) key grid (row-wise path: window scores in the
    # workspace, max-pooled to block scores by the top-k kernel)
    nw = (T - 32) // 16 + 1
    shape_g = sp.SpardaShape(batch=w.batch, n_kv_heads=w.n_kv_heads, group_size=w.group_size, k_total=w.k_total,
                             t_cap=T, nc_cap=nw, n_init=w.n_init, n_local=w.n_local, cmp_kernel=32, cmp_stride=16)
    kc_g = torch.zeros(w.batch, w.n_kv_heads, nw, 128, dtype=torch.bfloat16, device=dev)
    sp.sparda_compress_keys(shape_g, case["k"], T, 0, nw, kc_g)
    ws_g = ws_tensor(shape_g, sp.SPARDA_OP_FORECAST_SELECT, T, 0, dev)

    def select_grid():
        sp.sparda_forecast_select(shape_g, case["f"], T, 0, kc_g, sel, cnt, ws_g)

    for _ in range(max(1, warmup)):
        select_grid()
    ms_sel_g = time_events(select_grid, iters, stream)
    sel_g_stats = rep_stats(select_grid, max(50, iters), stream, flush)
    del kc_g, ws_g
    # scored (row, candidate) pairs: rows whose candidates outnumber their free slots
    flops = 0
    score_flops = 0  # every causal (row, candidate) pair
    attn_flops = 0
    for r in range(T):
        blk = r // 64
        n_cand = max(0, blk - w.n_local - w.n_init + 1)
        score_flops += 2 * 128 * n_cand
        n_forced = min(w.n_init, blk + 1) + (blk - max(max(0, blk - w.n_local + 1), min(w.n_init, blk + 1)) + 1)
        if w.k_total - n_forced < n_cand:
            flops += 2 * 128 * n_cand
        n_sel_blocks = min(w.k_total, blk + 1)
        attn_flops += 4 * 128 * ((n_sel_blocks - 1) * 64 + (r % 64) + 1)
    flops *= w.batch * w.n_kv_heads
    score_flops *= w.batch * w.n_kv_heads
    attn_flops *= w.batch * w.n_q_heads
    # bytes the score-only kernel must move: F in, K~ in, one float per row out
    score_bytes = case["f"].numel() * 2 + kc.numel() * 2 + row_max.numel() * 4
    return {
        "workload": "prefill B1 T=32768 Hq32/Hkv8 D128 block64 k64, all 32768 rows",
        "select_ms": ms_sel,
        "select_tflops": flops / (ms_sel * 1e-3) / 1e12,
        "select_frac_bf16_peak": flops / (ms_sel * 1e-3) / 1e12 / BF16_PEAK_TFLOPS,
        # two flop counts: the rows that must rank their candidates (the kernel skips rows whose
        # candidates all fit the set), and every causal (row, candidate) pair
        "select_gflop": flops / 1e9,
        "select_gflop_scored_rows": flops / 1e9,
        "select_gflop_all_causal_pairs": score_flops / 1e9,
        "select_tflops_all_causal_pairs": score_flops / (ms_sel * 1e-3) / 1e12,
        "select_stats": sel_stats,
        "select_tflops_median_flushed": flops / (sel_stats["median_ms"] * 1e-3) / 1e12,
        "attn_ms": ms_att,
        "attn_tflops": attn_flops / (ms_att * 1e-3) / 1e12,
        "select_grid_32_16_ms": ms_sel_g,
        "select_grid_32_16_stats": sel_g_stats,
        "score_only_ms": ms_score,
        "score_only_gflop": score_flops / 1e9,
        "score_only_tflops": score_flops / (ms_score * 1e-3) / 1e12,
        "score_only_frac_bf16_peak": score_flops / (ms_score * 1e-3) / 1e12 / BF16_PEAK_TFLOPS,
        "score_only_GBps": score_bytes / (ms_score * 1e-3) / 1e9,
        "score_only_stats": score_stats,
        "score_only_tflops_median_flushed": score_flops / (score_stats["median_ms"] * 1e-3) / 1e12,
    }


def grid_leg(base: DecodeLayer, dev, warmup, steps, stream):
    """The same decode layer with compressed keys on the paper's (32, 16) grid (windows of 32
    tokens at stride 16, max-pooled to block scores): select + attention, same K/V/Q/F."""
    g = DecodeLayer(base.w, dev, grid=(32, 16), case=base.case)
    for _ in range(warmup):
        g.step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        g.step()
    torch.cuda.synchronize()
    ms_step = (time.perf_counter() - t0) * 1e3 / steps
    ms_sel = time_events(g.select, steps, stream)
    ms_att = time_events(g.attend, steps, stream)
    ms_cmp = time_events(g.compress_new, steps, stream)
    parts = g.bytes()
    step_bytes = parts["select"] + parts["attend"]
    res = {
        "workload": "decode layer B32 T=131072 Hq32/Hkv8 D128 block64 k64, K~ on the (32, 16) grid "
                    f"({g.nw} windows per row)",
        "us_per_layer": ms_step * 1e3,
        "GBps": step_bytes / (ms_step * 1e-3) / 1e9,
        "step_bytes": step_bytes,
        "parts_us": {"compress_new": ms_cmp * 1e3, "select": ms_sel * 1e3, "attend": ms_att * 1e3},
        "select_GBps": parts["select"] / (ms_sel * 1e-3) / 1e9,
    }
    g.kc = g.ws_sel = None
    return res


def selector_leg(dev, iters):
    """Selection cost of the Forecast indexer (one head per group, no softmax) against the InfLLM-V2
    multi-head selector it replaces (every query head, softmax, group sum), on the paper's (32, 16)
    key grid and the same compressed keys: decode rows at 32K and 128K (B32) and a 4096-row prefill
    chunk ending at 128K (B1), for G = 4 (8 KV heads) and G = 16 (2 KV heads), 32 query heads."""
    stream = torch.cuda.current_stream()
    out = {"grid": [32, 16], "decode": [], "prefill_chunk": []}

    def one(B, Hkv, G, T, n_q, k_total=64):
        nw = (T - 32) // 16 + 1
        shape = sp.SpardaShape(batch=B, n_kv_heads=Hkv, group_size=G, k_total=k_total, t_cap=T, nc_cap=nw,
                               cmp_kernel=32, cmp_stride=16)
        g = torch.Generator(device=dev).manual_seed(T + G)
        # compressed keys distributed like the mean of 32 N(0, 1) keys; F and Q rows N(0, 1)
        kc = (torch.randn((B, Hkv, nw, 128), generator=g, device=dev) * (32 ** -0.5)).to(torch.bfloat16)
        f = torch.randn((B, Hkv, n_q, 128), generator=g, device=dev).to(torch.bfloat16)
        q = torch.randn((B, Hkv * G, n_q, 128), generator=g, device=dev).to(torch.bfloat16)
        sel = torch.empty((B, Hkv, n_q, k_total), dtype=torch.int16, device=dev)
        cnt = torch.empty((B, Hkv, n_q), dtype=torch.int16, device=dev)
        q_pos0 = T - n_q
        ws_f = ws_tensor(shape, sp.SPARDA_OP_FORECAST_SELECT, n_q, q_pos0, dev)
        ws_m = ws_tensor(shape, sp.SPARDA_OP_MULTIHEAD_SELECT, n_q, q_pos0, dev)
        fc = lambda: sp.sparda_forecast_select(shape, f, n_q, q_pos0, kc, sel, cnt, ws_f)
        mh = lambda: sp.sparda_multihead_select(shape, q, n_q, q_pos0, kc, SCALE, sel, cnt, ws_m)
        fc(); mh()
        torch.cuda.synchronize()
        ms_f = time_events(fc, iters, stream)
        ms_m = time_events(mh, iters, stream)
        return {"batch": B, "kv_heads": Hkv, "G": G, "T": T, "rows_per_group": n_q, "forecast_us": ms_f * 1e3,
                "multihead_us": ms_m * 1e3, "multihead_over_forecast": ms_m / ms_f,
                "multihead_path": "fused" if ws_m.numel() <= 16 else (
                    "MFMA tiles + row-wise top-k" if n_q >= 16 else "row-wise")}

    for T in (32768, 131072):
        for Hkv, G in ((8, 4), (2, 16)):
            out["decode"].append(one(32, Hkv, G, T, 1))
    for Hkv, G in ((8, 4), (2, 16)):
        out["prefill_chunk"].append(one(1, Hkv, G, 131072, 4096))
    return out


def paper_config_leg(dev, warmup, steps):
    """The paper's model configuration (MiniCPM4.1-8B, App. C): 32 query / 2 KV heads, k = 96
    blocks including the 32-block local window and the initial block, keys on the (32, 16) grid.
    Decode at 128K (B32): select + attention per layer; chunked prefill at 32K (B1, all rows):
    the fused windowed select and the tiled attention."""
    stream = torch.cuda.current_stream()
    res = {}
    w = inputs.WORKLOADS["paper_decode_b32_t128k"]
    lay = DecodeLayer(w, dev, grid=(32, 16))
    for _ in range(warmup):
        lay.step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        lay.step()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / steps
    parts = lay.bytes()
    res["decode"] = {"workload": "decode B32 T=131072 Hq32/Hkv2 D128 block64 k96 (1 init + 32 local), (32, 16) grid",
                     "us_per_layer": ms * 1e3, "GBps": (parts["select"] + parts["attend"]) / (ms * 1e-3) / 1e9,
                     "select_us": time_events(lay.select, steps, stream) * 1e3,
                     "attend_us": time_events(lay.attend, steps, stream) * 1e3}
    del lay
    w = inputs.WORKLOADS["paper_prefill_b1_t32k"]
    T = w.seq_len
    nw = (T - 32) // 16 + 1
    shape = sp.SpardaShape(batch=w.batch, n_kv_heads=w.n_kv_heads, group_size=w.group_size, k_total=w.k_total,
                           t_cap=T, nc_cap=nw, n_init=w.n_init, n_local=w.n_local, cmp_kernel=32, cmp_stride=16)
    case = inputs.make_case(w, device=dev)
    kc = torch.zeros(w.batch, w.n_kv_heads, nw, 128, dtype=torch.bfloat16, device=dev)
    sp.sparda_compress_keys(shape, case["k"], T, 0, nw, kc)
    sel = torch.empty(w.batch, w.n_kv_heads, T, w.k_total, dtype=torch.int16, device=dev)
    cnt = torch.empty(w.batch, w.n_kv_heads, T, dtype=torch.int16, device=dev)
    o = torch.empty(w.batch, w.n_q_heads, T, 128, dtype=torch.bfloat16, device=dev)
    ws_s = ws_tensor(shape, sp.SPARDA_OP_FORECAST_SELECT, T, 0, dev)
    ws_a = ws_tensor(shape, sp.SPARDA_OP_SPARSE_ATTN, T, 0, dev)
    sel_fn = lambda: sp.sparda_forecast_select(shape, case["f"], T, 0, kc, sel, cnt, ws_s)
    att_fn = lambda: sp.sparda_sparse_attn(shape, case["q"], T, 0, case["k"], case["v"], 0, sel, cnt, SCALE, o, ws_a)
    sel_fn()
    att_fn()
    torch.cuda.synchronize()
    res["prefill"] = {"workload": "prefill B1 T=32768 Hq32/Hkv2 D128 block64 k96 (1 init + 32 local), (32, 16) grid, "
                                  "all rows", "select_ms": time_events(sel_fn, max(10, steps), stream),
                      "attn_ms": time_events(att_fn, 3, stream)}
    return res


def training_leg(dev, iters):
    """The indexer-training loss (Sec. 4.2, Eq. 6-7) with its gradient for a chunk of 256 query rows
    at the end of a 64K-token sequence (the paper's training length), 32 query / 8 KV heads, the
    (2, 1) target pooled to the (32, 16) prediction grid, k = 64; synthetic keys, queries and
    Forecast rows N(0, 1).  Useful work: the target's two passes of G scores per fine window."""
    B, H, G, T, n_q, k_top = 1, 8, 4, 65536, 256, 64
    nw = (T - 32) // 16 + 1
    shape = sp.SpardaShape(batch=B, n_kv_heads=H, group_size=G, k_total=64, t_cap=T, nc_cap=nw, cmp_kernel=32,
                           cmp_stride=16)
    g = torch.Generator(device=dev).manual_seed(77)
    k = torch.randn((B, H, T, 128), generator=g, device=dev).to(torch.bfloat16)
    q = torch.randn((B, H * G, n_q, 128), generator=g, device=dev).to(torch.bfloat16)
    f = torch.randn((B, H, n_q, 128), generator=g, device=dev).to(torch.bfloat16)
    kc = torch.empty((B, H, nw, 128), dtype=torch.bfloat16, device=dev)
    sp.sparda_compress_keys(shape, k, T, 0, nw, kc)
    loss = torch.empty((B, H, n_q), dtype=torch.float32, device=dev)
    dF = torch.empty((B, H, n_q, 128), dtype=torch.float32, device=dev)
    ws = ws_tensor(shape, sp.SPARDA_OP_INDEXER_KL, n_q, T - n_q, dev)
    fn = lambda: sp.sparda_indexer_kl(shape, q, k, f, kc, n_q, T - n_q, SCALE, k_top, loss, dF, ws)
    fn()
    torch.cuda.synchronize()
    ms = time_events(fn, iters, torch.cuda.current_stream())
    fine = sum(T - n_q + r for r in range(n_q))  # fine windows complete per row, summed
    flops = 2 * 2 * 128 * G * fine * B * H      # two passes of G dot products per fine window
    return {"workload": f"indexer KL + gradient, B{B} Hq{H * G}/Hkv{H} T={T}, {n_q}-row chunk, k={k_top}, "
                        "(2, 1) target -> (32, 16) prediction", "ms": ms, "rows_per_s": B * H * n_q / (ms * 1e-3),
            "target_tflops": flops / (ms * 1e-3) / 1e12, "target_gflop": flops / 1e9}


def cpu_baseline(layer: DecodeLayer, n_rows: int, min_seconds: float = 10.0):
    """The oracle on n_rows sampled (batch, group) rows of the decode step (select + attend on
    precomputed K~, as timed on the GPU), all host cores."""
    import oracle
    w = layer.w
    T, nb, G = layer.T, layer.nb, w.group_size
    rng = np.random.default_rng(11)
    pairs = [(int(rng.integers(w.batch)), int(rng.integers(w.n_kv_heads))) for _ in range(n_rows)]
    k = np.stack([inputs.to_u16(layer.k[b, m]) for b, m in pairs])[:, None]
    v = np.stack([inputs.to_u16(layer.v[b, m]) for b, m in pairs])[:, None]
    f = np.stack([inputs.to_u16(layer.f[b, m]) for b, m in pairs])[:, None]
    q = np.stack([inputs.to_u16(layer.q[b, m * G:(m + 1) * G]) for b, m in pairs])
    kc = np.stack([inputs.to_u16(layer.kc[b, m]) for b, m in pairs])[:, None].copy()
    oshape = oracle.Shape(batch=n_rows, n_kv_heads=1, group_size=G, k_total=w.k_total, t_cap=T, nc_cap=nb,
                          n_init=w.n_init, n_local=w.n_local)
    threads = oracle.set_threads(0)  # the OpenMP threads the oracle's loops use
    reps = 0
    t0 = time.perf_counter()
    while True:  # repeat the sample until about min_seconds of CPU work
        sel, cnt = oracle.forecast_select(oshape, f, 1, T - 1, kc)
        oracle.sparse_attn(oshape, q, 1, T - 1, k, v, 0, sel, cnt, SCALE)
        reps += 1
        if time.perf_counter() - t0 >= min_seconds:
            break
    dt = (time.perf_counter() - t0) / reps
    parts = layer.bytes()
    rows_total = w.batch * w.n_kv_heads
    sample_bytes = (parts["select"] + parts["attend"]) * n_rows / rows_total
    return {"value": sample_bytes / dt / 1e9, "unit": "GB/s", "cores": threads, "kind": "oracle",
            "sample": f"{n_rows} of {rows_total} (batch, group) rows of the 128K decode step "
                      f"(select + attend), {dt:.3f}s per pass, {reps} passes",
            "us_per_layer_equiv": dt * rows_total / n_rows * 1e6,
            "host": host_info(), "threads": threads, "small_workloads": oracle_small_workloads(threads)}


def host_info():
    """nproc and the lscpu topology of this host."""
    info = {"nproc": os.cpu_count()}
    try:
        import subprocess
        text = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        keys = {"Socket(s)": "sockets", "Core(s) per socket": "cores_per_socket", "Thread(s) per core": "threads_per_core",
                "Model name": "model"}
        for line in text.splitlines():
            k, _, v = line.partition(":")
            if k.strip() in keys:
                v = v.strip()
                info[keys[k.strip()]] = int(v) if v.isdigit() else v
    except (OSError, ValueError):
        pass
    return info


def oracle_small_workloads(threads):
    """The oracle's select + attend over every row of the 4K (B1) and 32K (B8) decode workloads,
    on one thread and on `threads`, median of 3 runs each (seconds per decode layer)."""
    import oracle
    out = {}
    for name in ("decode_b1_t4k", "decode_b8_t32k"):
        w = inputs.WORKLOADS[name]
        case = inputs.make_case(w)
        T, nb = w.seq_len, w.n_blocks
        o = oracle.Shape(batch=w.batch, n_kv_heads=w.n_kv_heads, group_size=w.group_size, k_total=w.k_total, t_cap=T,
                         nc_cap=nb, n_init=w.n_init, n_local=w.n_local)
        q, f, k, v = (inputs.to_u16(case[n]) for n in ("q", "f", "k", "v"))
        kc = oracle.compress_keys(o, k, T, 0, nb)
        res = {}
        for nt in (1, threads):
            oracle.set_threads(nt)
            times = []
            for _ in range(3):
                t0 = time.perf_counter()
                sel, cnt = oracle.forecast_select(o, f, 1, T - 1, kc)
                oracle.sparse_attn(o, q, 1, T - 1, k, v, 0, sel, cnt, SCALE)
                times.append(time.perf_counter() - t0)
            res[f"s_per_layer_{nt}_threads"] = float(np.median(times))
        out[name] = res
    oracle.set_threads(threads)
    return out


def pipeline_leg(dev, steps):
    """Offloaded 32-layer decode at 128K, batch 64 (pinned host pools, one-layer-ahead gather).

    Layer 0's KV is in HBM; layers 1..31 read their selected blocks from two pinned host pools
    (layer l uses pool (l-1) mod 2, so 2 x 34.4 GB are pinned instead of 31 x 34.4 GB).  The
    compressed keys, queries and Forecast rows are distinct per layer.  Reports the gather's
    workgroup sweep, the overlapped and serial step times, and the per-layer gather and compute
    times that bound the overlap.
    """
    from paper_2606_04511_amd import hostmem
    from paper_2606_04511_amd.pipeline import DecodePipeline
    w = inputs.WORKLOADS["pipeline_b64_t128k_l32"]
    B, H, G, T, nb, K, L = w.batch, w.n_kv_heads, w.group_size, w.seq_len, w.n_blocks, w.k_total, w.layers
    shape = sp.SpardaShape(batch=B, n_kv_heads=H, group_size=G, k_total=K, t_cap=T, nc_cap=nb)
    pool_bytes = B * H * T * 128 * 2
    t0 = time.time()
    bufs = [hostmem.PinnedBuffer(pool_bytes) for _ in range(4)]
    log(f"[bench] pinned 4 x {pool_bytes / 2**30:.1f} GiB host pools in {time.time() - t0:.1f}s")
    t0 = time.time()
    fill = torch.randn(64 * 1024 * 1024, device=dev).to(torch.bfloat16).view(torch.uint8)  # 128 MiB
    for buf in bufs:
        for off in range(0, pool_bytes, fill.numel()):
            n = min(fill.numel(), pool_bytes - off)
            buf.copy_from_device(off, fill[:n])
    torch.cuda.synchronize()
    log(f"[bench] filled the host pools in {time.time() - t0:.1f}s")
    pools = [None] + [(bufs[2 * ((l - 1) % 2)].ptr, bufs[2 * ((l - 1) % 2) + 1].ptr) for l in range(1, L)]
    gen = lambda shp, tid: inputs.normal_bf16(shp, w.seed, tid, dev)
    q = [gen((B, H * G, 1, 128), 1000 + l) for l in range(L)]
    f = [gen((B, H, 1, 128), 2000 + l) for l in range(L)]
    f0 = gen((B, H, 1, 128), 2999)
    kc = [gen((B, H, nb, 128), 3000 + l) for l in range(L)]
    k0 = gen((B, H, T, 128), 4000)
    v0 = gen((B, H, T, 128), 4001)
    moved = 2 * B * H * K * 64 * 256  # K + V bytes gathered per offloaded layer

    # gather sweep over the persistent grid size on a side stream (selection of layer 1)
    pipe = DecodePipeline(shape, T, q, f, f0, kc, k0, v0, pools, 64, dev)
    pipe.step()
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    sweep = {}
    for nwg in (8, 16, 32, 64, 128, 256):
        pipe.n_workgroups = nwg
        ms = time_events(lambda: pipe._gather(1, side), 5, side)
        sweep[str(nwg)] = {"ms": ms, "GBps": moved / (ms * 1e-3) / 1e9}
    best_nwg = int(max(sweep, key=lambda k: sweep[k]["GBps"]))
    pipe.n_workgroups = best_nwg
    dst = torch.empty(moved // 2, dtype=torch.uint8, device=dev)
    ms_cp = time_events(lambda: bufs[0].copy_to_device(0, dst), 5, torch.cuda.current_stream())

    # per-layer compute alone (select of the next layer + attention from staging) and gather alone
    comp = torch.cuda.current_stream()
    ms_compute = time_events(lambda: (pipe._select(pipe.f[1], 2), pipe._attend(1)), 10, comp)
    ms_gather = time_events(lambda: pipe._gather(1, comp), 5, comp)

    def one_step(overlap):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        pipe.step(overlap=overlap)
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) * 1e3

    # The gather's workgroup count (its CU budget, the paper's CTA count) is chosen on the
    # overlapped step, not on the gather alone: more workgroups copy no faster over the host link
    # but crowd the CUs the concurrent select and attention need.
    step_sweep = {}
    for nwg in (8, 16, 32, 64):
        pipe.n_workgroups = nwg
        one_step(True)
        step_sweep[str(nwg)] = float(np.median([one_step(True) for _ in range(2)]))
    pipe.n_workgroups = int(min(step_sweep, key=lambda k: step_sweep[k]))
    best_step_nwg = pipe.n_workgroups
    # The two modes alternate step by step so that drifts of the host link hit both alike; the
    # overlap can hide at most the compute time per layer, about 1 % of a step here.
    one_step(True)
    one_step(False)
    runs = {True: [], False: []}
    for _ in range(steps):
        for mode in (True, False):
            runs[mode].append(one_step(mode))
    ms_overlap = float(np.median(runs[True]))
    ms_serial = float(np.median(runs[False]))
    bound = (L - 1) * max(ms_gather, ms_compute) + ms_compute

    # Step-to-step reuse (the NOSI engine of App. C): a run of consecutive decode positions in
    # which every layer's Forecast rows drift (f <- rho f + sqrt(1 - rho^2) n, n ~ N(0, 1)), each
    # offloaded layer keeping its staging across steps and fetching only the new blocks.
    del pipe
    torch.cuda.empty_cache()
    n_reuse, rho = 8, 0.95
    rpipe = DecodePipeline(shape, T - n_reuse, q, f, f0, kc, k0, v0, pools, best_step_nwg, dev, reuse=True)
    g = torch.Generator(device=dev).manual_seed(w.seed + 7)
    reuse_ms, reuse_frac = [], []
    per_step = (L - 1) * B * H * K
    for i in range(n_reuse + 1):
        for x in f + [f0]:
            x.copy_((rho * x.float() + math.sqrt(1 - rho * rho) * torch.randn(x.shape, generator=g, device=dev))
                    .to(torch.bfloat16))
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        rpipe.step(overlap=True, t_ctx=T - n_reuse + i)
        torch.cuda.synchronize()
        ms = (time.perf_counter() - t0) * 1e3
        if i > 0:  # step 0 starts from empty staging
            reuse_ms.append(ms)
            reuse_frac.append(rpipe.fetched_blocks() / per_step)
    del rpipe
    for b in bufs:
        b.free()
    return {
        "workload": f"decode pipeline, {L} layers, B{B} T={T} k{K}: {moved / 1e9:.3f} GB gathered per offloaded layer",
        "gather_sweep": sweep, "step_sweep_overlap_ms": step_sweep, "n_workgroups": best_step_nwg,
        "gather_GBps": sweep[str(best_nwg)]["GBps"], "h2d_memcpy_GBps": (moved // 2) / (ms_cp * 1e-3) / 1e9,
        "gather_ms_per_layer": ms_gather, "compute_ms_per_layer": ms_compute,
        "ms_per_step_overlap": ms_overlap, "ms_per_step_serial": ms_serial,
        "ms_per_step_overlap_runs": runs[True], "ms_per_step_serial_runs": runs[False],
        "ms_per_step_bound": bound, "tokens_per_s": B / (ms_overlap * 1e-3),
        "reuse": {"steps": n_reuse, "forecast_drift_rho": rho, "ms_per_step": float(np.median(reuse_ms)),
                  "ms_per_step_runs": reuse_ms, "fetched_fraction": float(np.mean(reuse_frac)),
                  "fetched_fraction_runs": reuse_frac, "tokens_per_s": B / (float(np.median(reuse_ms)) * 1e-3),
                  "speedup_vs_full_fetch": ms_overlap / float(np.median(reuse_ms))},
    }


def peaks_leg(dev):
    """Hardware limits measured in the same run (the spec figures are 8 TB/s and 2.5 PFLOP/s):
    streaming HBM reads of 4 GiB, reads of 32768 randomly placed 16 KiB blocks (537 MB, the shape
    of a decode layer's attended KV blocks), both with the non-temporal hint and the best of three
    grid sizes, back-to-back bf16 MFMA of both gfx950 shapes (32x32x16 and 16x16x32), and a pinned
    1 GiB host to device copy."""
    import ctypes
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2606_04511_amd", "libsparda_peaks.so"))
    lib.peaks_stream_read.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
    lib.peaks_block_read.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_void_p,
                                     ctypes.c_void_p]
    lib.peaks_mfma_bf16.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
    lib.peaks_mfma32_bf16.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
    stream = torch.cuda.current_stream()
    sh = ctypes.c_void_p(stream.cuda_stream)
    nbytes = 4 << 30
    buf = torch.ones(nbytes // 2, dtype=torch.bfloat16, device=dev)
    sink = torch.zeros(4, dtype=torch.int32, device=dev)
    g = torch.Generator(device="cpu").manual_seed(4242)
    n_blocks = 32768
    idx = torch.randint(0, nbytes // 16384, (n_blocks,), generator=g, dtype=torch.int64).to(torch.int32).to(dev)

    def check(rc):
        if rc != 0:
            raise RuntimeError(f"peaks library call failed ({rc})")

    def warm_time(fn, iters):
        fn()
        torch.cuda.synchronize()
        return time_events(fn, iters, stream)

    # the best of a few grid sizes (non-temporal loads; 256 streaming workgroups, one per CU, and
    # 1024 block-reading workgroups were the fastest in a sweep of 256 to 8192)
    ms_stream = min(warm_time(lambda: check(lib.peaks_stream_read(buf.data_ptr(), nbytes, grid, sink.data_ptr(), sh)),
                              5) for grid in (256, 512, 8192))
    ms_block = min(warm_time(lambda: check(lib.peaks_block_read(buf.data_ptr(), idx.data_ptr(), n_blocks, grid,
                                                                sink.data_ptr(), sh)), 10) for grid in (512, 1024, 2048))
    grid, iters = 2048, 4000
    ms_mfma = warm_time(lambda: check(lib.peaks_mfma_bf16(grid, iters, sink.data_ptr(), sh)), 3)
    ms_mfma32 = warm_time(lambda: check(lib.peaks_mfma32_bf16(grid, iters, sink.data_ptr(), sh)), 3)
    del buf
    host = torch.empty(1 << 30, dtype=torch.uint8, pin_memory=True)
    dst = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
    ms_h2d = warm_time(lambda: dst.copy_(host, non_blocking=True), 5)
    del host, dst
    torch.cuda.synchronize()
    return {
        "hbm_stream_read_GBps": nbytes / (ms_stream * 1e-3) / 1e9,
        "hbm_block_read_GBps": n_blocks * 16384 / (ms_block * 1e-3) / 1e9,
        # the faster of the two gfx950 bf16 shapes is the hardware's measured MFMA limit
        "mfma_bf16_TFLOPs": grid * 4 * 4 * iters * 32768 / (ms_mfma32 * 1e-3) / 1e12,
        "mfma_bf16_32x32x16_TFLOPs": grid * 4 * 4 * iters * 32768 / (ms_mfma32 * 1e-3) / 1e12,
        "mfma_bf16_16x16x32_TFLOPs": grid * 4 * 8 * iters * 16384 / (ms_mfma * 1e-3) / 1e12,
        "h2d_pinned_GBps": (1 << 30) / (ms_h2d * 1e-3) / 1e9,
    }


def gather_sweep_leg(dev):
    """Gather rate against the persistent workgroup count, and the time of a decode attention
    launched while one gather runs, at B = 8 .. 64, T = 32K, 8 KV heads, k = 64 (the shape of the
    paper's CTA sweep): the data behind pipeline.gather_workgroups."""
    T, H, K = 32768, 8, 64
    rows = []
    for B in (8, 16, 32, 64):
        w = inputs.Workload("gather_sweep", batch=B, seq_len=T, n_q=1, n_kv_heads=H, group_size=4, k_total=K,
                            n_init=1, n_local=2, seed=77)
        L = DecodeLayer(w, dev)
        L.select()
        torch.cuda.synchronize()
        hk = torch.empty((B, H, T, 128), dtype=torch.bfloat16, pin_memory=True)
        hv = torch.empty((B, H, T, 128), dtype=torch.bfloat16, pin_memory=True)
        hk.copy_(L.k.cpu())
        hv.copy_(L.v.cpu())
        stg_k = torch.empty((B, H, K, 64, 128), dtype=torch.bfloat16, device=dev)
        stg_v = torch.empty_like(stg_k)
        side = torch.cuda.Stream()
        main = torch.cuda.current_stream()
        nbytes = 2 * B * H * K * 64 * 256
        for _ in range(3):
            L.attend()
        att_alone = time_events(L.attend, 20, main)
        for nwg in (4, 8, 16, 32, 64):
            g = lambda: sp.sparda_gather_blocks(L.shape, hk, hv, L.sel[:, :, 0], L.cnt[:, :, 0], stg_k, stg_v, nwg,
                                                side)
            g()
            side.synchronize()
            ms_g = time_events(g, 3, side)
            torch.cuda.synchronize()
            g()  # one gather on the side stream while the main stream runs attention launches
            n_att = max(1, int(ms_g / att_alone / 2))
            a0, a1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a0.record(main)
            for _ in range(n_att):
                L.attend()
            a1.record(main)
            torch.cuda.synchronize()
            rows.append({"batch": B, "n_workgroups": nwg, "gather_ms": ms_g, "gather_GBps": nbytes / ms_g / 1e6,
                         "attend_alone_us": att_alone * 1e3,
                         "attend_during_gather_us": a0.elapsed_time(a1) / n_att * 1e3})
            log("[bench] gather sweep " + json.dumps(rows[-1]))
        del L, hk, hv, stg_k, stg_v
        torch.cuda.empty_cache()
    return rows


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-prefill", action="store_true")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--pipeline", action="store_true",
                    help="also run the offloaded 32-layer decode pipeline (pins 4 x 17.2 GB of host memory) in a "
                         "child process; off by default while a host-side crash seen in it is unexplained")
    ap.add_argument("--no-pipeline", action="store_true", help="kept for compatibility (the default)")
    ap.add_argument("--pipeline-only", action="store_true", help=argparse.SUPPRESS)
    ap.add_argument("--gather-sweep", action="store_true",
                    help="only the gather workgroup sweep (host-link rate and interference), one JSON line")
    ap.add_argument("--no-grid", action="store_true", help="skip the decode layer on the (32, 16) key grid")
    ap.add_argument("--no-selectors", action="store_true",
                    help="skip the Forecast vs multi-head selector comparison")
    ap.add_argument("--no-training", action="store_true", help="skip the indexer-training loss leg")
    ap.add_argument("--no-paper-config", action="store_true",
                    help="skip the decode and prefill at the paper's model configuration")
    ap.add_argument("--cpu-rows", type=int, default=32)
    ap.add_argument("--reps", type=int, default=60, help="repetitions of each flushed per-call timing (>= 50)")
    ap.add_argument("--calib-copy", action="store_true", help="run a plain 1 GiB device copy (counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); the library has no multi-GPU path.",
              file=sys.stderr)
        sys.exit(2)
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    dev = torch.device("cuda:0")
    sp.load()
    if args.pipeline_only:  # the child process of --pipeline
        print(json.dumps(pipeline_leg(dev, 4)))
        return
    if args.gather_sweep:
        print(json.dumps({"gather_sweep": gather_sweep_leg(dev)}))
        return

    if args.calib_copy:
        a = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
        log("[bench] calibration copy of 1 GiB done (x3)")

    peaks = peaks_leg(dev)
    log("[bench] measured peaks: " + ", ".join(f"{k} {v:.1f}" for k, v in peaks.items()))

    w = inputs.WORKLOADS["decode_b32_t128k"]
    layer = DecodeLayer(w, dev)
    stream = torch.cuda.current_stream()
    for _ in range(args.warmup):
        layer.step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        layer.step()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = wall * 1e3 / args.steps
    parts = layer.bytes()
    step_bytes = parts["select"] + parts["attend"]
    log(f"[bench] decode step {ms_step * 1e3:.1f} us (one fused launch)")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        layer.step_with_refresh()
    torch.cuda.synchronize()
    ms_step_refresh = (time.perf_counter() - t0) * 1e3 / args.steps
    # the same step as two calls (select, then attention), timed the same way
    for _ in range(args.warmup):
        layer.step_separate()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        layer.step_separate()
    torch.cuda.synchronize()
    ms_sep = (time.perf_counter() - t0) * 1e3 / args.steps

    # per-call event timing: the step is one launch of the fused kernel, the dominant (only) kernel;
    # the select and attention calls alone for context
    ms_launch = time_events(layer.step, args.steps, stream)
    ms_sel = time_events(layer.select, args.steps, stream)
    ms_att = time_events(layer.attend, args.steps, stream)
    ms_cmp = time_events(layer.compress_new, args.steps, stream)
    # the same calls one at a time after a 1 GiB cache flush: median, p10 and p90
    flush = Flusher(dev)
    step_stats = {"step": rep_stats(layer.step, args.reps, stream, flush),
                  "select": rep_stats(layer.select, args.reps, stream, flush),
                  "attend": rep_stats(layer.attend, args.reps, stream, flush)}
    log(f"[bench] the same step as two calls: {ms_sep * 1e3:.1f} us")
    log(f"[bench] decode step after a cache flush: median {step_stats['step']['median_ms'] * 1e3:.1f} us "
        f"(p10 {step_stats['step']['p10_ms'] * 1e3:.1f}, p90 {step_stats['step']['p90_ms'] * 1e3:.1f})")
    att_bytes = parts["attend"]
    achieved = step_bytes / (ms_launch * 1e-3) / 1e9
    achieved_att = att_bytes / (ms_att * 1e-3) / 1e9
    out = {
        "metric": METRIC,
        "value": step_bytes / (ms_step * 1e-3) / 1e9,
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) bf16 with 5% planted blocks)",
        "config": {"workload": "decode layer B32 T=131072 Hq32/Hkv8 D128 block64 k64 (1 init + 2 local), "
                               "select + sparse attention on precomputed K~",
                   "batch": w.batch, "seq_len": w.seq_len, "k_blocks": w.k_total, "parallelism": "none (1 GPU)"},
        "us_per_layer": ms_step * 1e3,
        "us_per_layer_with_kcmp_refresh": ms_step_refresh * 1e3,
        "frac_hbm_peak": step_bytes / (ms_step * 1e-3) / 1e9 / HBM_PEAK_GBS,
        "step_bytes": step_bytes,
        "parts_us": {"compress_new": ms_cmp * 1e3, "select": ms_sel * 1e3, "attend": ms_att * 1e3},
        "us_per_layer_separate_calls": ms_sep * 1e3,
        "roofline": {"bound": "hbm", "kernel": "decode_step_kernel<4, 8> (select + attention of a decode row in "
                                               "one workgroup, one launch per step)",
                     "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                     "traffic": counted_traffic("decode_step_kernel<4, 8>"),
                     "algorithmic_bytes_per_launch": step_bytes, "avg_launch_ms": ms_launch,
                     "measured_peak": peaks["hbm_block_read_GBps"],
                     "frac_measured_peak": achieved / peaks["hbm_block_read_GBps"]},
        "attention_alone": {"kernel": "sparse_attn_kernel<4, 8>", "avg_launch_ms": ms_att, "achieved_GBps": achieved_att,
                            "frac": achieved_att / HBM_PEAK_GBS, "algorithmic_bytes_per_launch": att_bytes,
                            "traffic": counted_traffic("sparse_attn_kernel<4, 8>")},
        "peaks": peaks,
        "frac_measured_read_peak": step_bytes / (ms_step * 1e-3) / 1e9 / peaks["hbm_block_read_GBps"],
        "flushed_stats": step_stats,
        "us_per_layer_median_flushed": step_stats["step"]["median_ms"] * 1e3,
        "GBps_median_flushed": step_bytes / (step_stats["step"]["median_ms"] * 1e-3) / 1e9,
    }
    out["decode_overlap"] = overlap_leg(layer, dev)
    log(f"[bench] decode layers with select(l+1) beside attention(l): {out['decode_overlap']['us_per_layer_overlapped']:.1f} "
        f"us per layer (serial {out['decode_overlap']['us_per_layer_serial']:.1f})")
    out["decode_small"] = decode_small_leg(dev, args.reps, flush)
    for r in out["decode_small"]:
        log(f"[bench] {r['workload'][:32]}: {r['us_per_layer_median']:.1f} us per layer (median after a flush, "
            f"p10 {r['us_per_layer_p10']:.1f}, p90 {r['us_per_layer_p90']:.1f}), {r['GBps_median']:.0f} GB/s")
    if not args.no_grid:
        out["paper_grid"] = grid_leg(layer, dev, args.warmup, args.steps, stream)
        log(f"[bench] (32, 16) grid decode step {out['paper_grid']['us_per_layer']:.1f} us, "
            f"select {out['paper_grid']['parts_us']['select']:.1f} us")
    if not args.no_selectors:
        out["selectors"] = selector_leg(dev, max(5, args.steps // 5))
        for r in out["selectors"]["decode"] + out["selectors"]["prefill_chunk"]:
            log(f"[bench] selectors T={r['T']} n_q={r['rows_per_group']} G={r['G']}: forecast {r['forecast_us']:.1f} us, "
                f"multi-head {r['multihead_us']:.1f} us ({r['multihead_path']}), x{r['multihead_over_forecast']:.2f}")
    if not args.no_paper_config:
        out["paper_config"] = paper_config_leg(dev, args.warmup, args.steps)
        pc = out["paper_config"]
        log(f"[bench] paper configuration (Hkv2 G16 k96 local 32, (32, 16)): decode {pc['decode']['us_per_layer']:.1f} us "
            f"(select {pc['decode']['select_us']:.1f}, attend {pc['decode']['attend_us']:.1f}); prefill 32K select "
            f"{pc['prefill']['select_ms'] * 1e3:.0f} us, attention {pc['prefill']['attn_ms']:.2f} ms")
    if not args.no_training:
        out["indexer_training"] = training_leg(dev, max(3, args.steps // 10))
        log(f"[bench] indexer KL + gradient: {out['indexer_training']['ms']:.2f} ms for "
            f"{out['indexer_training']['rows_per_s'] * out['indexer_training']['ms'] * 1e-3:.0f} rows at 64K, "
            f"{out['indexer_training']['target_tflops']:.1f} TFLOP/s on the target scores")
    if not args.no_prefill:
        layer.case = None
        out["prefill"] = prefill_leg(dev, args.warmup, max(10, args.steps // 2), flush)
        out["prefill"]["select_frac_measured_mfma_peak"] = out["prefill"]["select_tflops"] / peaks["mfma_bf16_TFLOPs"]
        # against the rate of the 16x16x32 instruction the select kernel's layout needs
        out["prefill"]["select_frac_measured_16x16x32_rate"] = (out["prefill"]["select_tflops"]
                                                                / peaks["mfma_bf16_16x16x32_TFLOPs"])
        out["prefill"]["score_only_frac_measured_mfma_peak"] = (out["prefill"]["score_only_tflops"]
                                                                 / peaks["mfma_bf16_TFLOPs"])
        log(f"[bench] prefill select {out['prefill']['select_ms'] * 1e3:.1f} us, "
            f"{out['prefill']['select_tflops']:.1f} TFLOP/s; on the (32, 16) grid "
            f"{out['prefill']['select_grid_32_16_ms'] * 1e3:.1f} us; score contraction alone "
            f"{out['prefill']['score_only_ms'] * 1e3:.1f} us, {out['prefill']['score_only_tflops']:.0f} TFLOP/s "
            f"({out['prefill']['score_only_frac_bf16_peak'] * 100:.1f} % of 2.5 PF); after a cache flush: select "
            f"{out['prefill']['select_stats']['median_ms'] * 1e3:.1f} us, score contraction "
            f"{out['prefill']['score_only_stats']['median_ms'] * 1e3:.1f} us")
    if args.pipeline and not args.no_pipeline:
        # A child process, so that a failure there cannot take the rest of this line down.
        import subprocess
        layer.case = None
        res = subprocess.run([sys.executable, os.path.abspath(__file__), "--pipeline-only"], capture_output=True,
                             text=True, timeout=900)
        sys.stderr.write(res.stderr[-4000:])
        try:
            out["pipeline"] = json.loads(res.stdout.strip().splitlines()[-1])
            log(f"[bench] pipeline {out['pipeline']['ms_per_step_overlap']:.1f} ms/step overlapped, "
                f"{out['pipeline']['ms_per_step_serial']:.1f} serial; with step-to-step reuse "
                f"{out['pipeline']['reuse']['ms_per_step']:.1f} ms/step, "
                f"{100 * out['pipeline']['reuse']['fetched_fraction']:.1f} % of the blocks fetched")
        except (IndexError, ValueError, KeyError):
            out["pipeline"] = {"error": f"pipeline child exited with status {res.returncode}"}
            log(f"[bench] pipeline leg failed: status {res.returncode}")
    if not args.no_cpu:
        out["cpu_baseline"] = cpu_baseline(layer, args.cpu_rows)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
