#!/usr/bin/env python3
"""Benchmark of the ActKV compression step (score -> select -> compact) on one MI355X.

One step = one actkv_step call over one layer of a synthetic batch: every cached KV entry
of every request is scored by the attention of that request's action queries (LSE
supplied, as a paged-attention decode produces it), the top-B entries per KV head are
selected and compacted into fresh pages, and the block table is rewritten.

Prints ONE JSON line (rank 0).  Default workload: 32 requests x 35,000 cached tokens with
Qwen3-30B head shapes (32 query / 4 KV heads, head_dim 128, 16-token pages), 64 action
queries per request, 25% budget per KV head, pool window 7 -- drawn on the device from a
seeded generator.

Besides the headline step the record carries the per-stage durations, the step with the
LSE pass included, and the step with LRFU eviction (Sec. 5.1: keep scores carried over,
top-p 0.9 hit mask, decay 0.5) in the "lrfu" field.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
BF16_PEAK_TFLOPS = 2500.0      # MI355X dense bf16 MFMA, TFLOP/s
METRIC = "KV tokens scored+compacted/s per layer (1 GPU)"
SCORE_SOURCES = ["paper_2609_31395_amd/csrc/score.hip",
                 "paper_2609_31395_amd/csrc/device_common.hpp",
                 "paper_2609_31395_amd/csrc/actkv_internal.h"]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "score_kernel_batch32x35k_traffic.json")
COPY_CALIB_BYTES = 512 << 20   # the known-size copy that calibrates FETCH_SIZE / WRITE_SIZE
# fp32 VALU issue slots per second without packed fp32 (256 CUs x 4 SIMDs x 16 lanes x
# 2.4 GHz); v_exp_f32 takes 2 slots: measured on MI355X with register-only probes, a SIMD
# retires one wave64 v_exp_f32 per ~8.8 cycles against one FMA per ~4-5.6
VALU_SLOTS_PER_S = 256 * 4 * 16 * 2.4e9
EXP_SLOTS = 2
LRFU_TOP_P, LRFU_DECAY = 0.9, 0.5   # the eviction policy's settings in the paper's evaluation


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="batch32x35k")
    ap.add_argument("--cpu-sample-reqs", type=int, default=8,
                    help="requests of the workload the CPU oracle is timed on")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-plan", action="store_true",
                    help="time the CPU oracle on the whole timing plan (the tiny and single "
                         "35K-token layers at 1 thread and all threads; the 32 x 35K batch, "
                         "the ragged and adaptive batches in full; two layers of the 48-layer "
                         "model) and print that record instead of the benchmark line")
    ap.add_argument("--headline-only", action="store_true",
                    help="time only the headline step and its stages (for profiling)")
    ap.add_argument("--no-table1", action="store_true",
                    help="skip the Table 1 shapes (streaming scoring and compression ops)")
    ap.add_argument("--no-fullmodel", action="store_true",
                    help="skip the full-model leg (48 layers over one ~138 GB page pool)")
    ap.add_argument("--profile-stage",
                    choices=["score", "select", "compact", "lse", "step", "lrfu_select",
                             "lrfu_step", "inplace_compact", "streaming", "copy",
                             "fullmodel"],
                    help="only run one entry point --steps times (for counter collection); "
                         "prints a short JSON line instead of the benchmark record.  'copy' "
                         "is the calibration: a plain device-to-device copy of "
                         "COPY_CALIB_BYTES bytes; 'fullmodel' times only the full-model leg")
    ap.add_argument("--score-data-probe", action="store_true",
                    help="time the scoring kernel alone on the workload as drawn, then with "
                         "every K/V and Q element set to bf16 1.0, then to 0 (the same "
                         "instructions on data that toggles fewer bits): a power-limited "
                         "kernel runs faster on the latter; prints a JSON line")
    return ap.parse_args()


def source_digest() -> str:
    h = hashlib.sha256()
    for rel in SCORE_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def algorithmic_bytes(dp, num_kept: int) -> int:
    """HBM bytes the step cannot avoid: read K once; read Q and the LSE; write and read
    each fp32 score once; write and read each kept index once; read and write each kept
    K and V row once."""
    D, Hkv, Hq = dp.head_dim, dp.num_kv_heads, dp.num_q_heads
    sum_L = int(dp.seq_lens.astype(np.int64).sum())
    sum_n = int(dp.q_lens.astype(np.int64).sum())
    k_read = sum_L * Hkv * D * 2
    q_read = sum_n * Hq * D * 2 + sum_n * Hq * 4
    scores = 2 * 4 * sum_L * Hkv
    kept = 2 * 4 * num_kept
    rows = num_kept * D * 2 * 2 * 2
    return k_read + q_read + scores + kept + rows


def score_flops(dp) -> int:
    """Dense QK^T flops of one scoring pass: 2 * (G n_r) * L_r * D per (request, KV head)."""
    G = dp.num_q_heads // dp.num_kv_heads
    return int(sum(2 * G * int(n) * int(L) * dp.head_dim * dp.num_kv_heads
                   for L, n in zip(dp.seq_lens, dp.q_lens)))


def score_epilogue_slots(dp) -> float:
    """VALU issue slots of the scoring epilogue: per (query row, key) one FMA (scale and
    LSE), one exp2 (half rate) and one add."""
    exps = score_flops(dp) / (2 * dp.head_dim)
    return exps * (1 + EXP_SLOTS + 1)


def measure_copy_bw(dev, reps=10) -> float:
    """Device-to-device copy of COPY_CALIB_BYTES, timed with events: read plus written
    bytes per second (the practical HBM ceiling of a streaming kernel on this machine)."""
    import torch
    src = torch.empty(COPY_CALIB_BYTES, dtype=torch.uint8, device=dev).fill_(1)
    dst = torch.empty_like(src)
    dst.copy_(src)
    ev = _event_pairs(reps)
    for a, b in ev:
        a.record()
        dst.copy_(src)
        b.record()
    torch.cuda.synchronize()
    return 2 * COPY_CALIB_BYTES / (_mean_ms(ev) * 1e-3)


MALL_FLUSH_BYTES = 512 << 20   # twice the 256 MB MALL: touched between cold repetitions


def percentiles(us):
    """[p10, p90] of a list of microsecond timings."""
    return [float(np.percentile(us, 10)), float(np.percentile(us, 90))]


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def run_stage(stage, reps, bp, dp, bts, lse, scores, pooled, kept, free, freed, new_lens, ws, qy):
    """Run one entry point `reps` times on its own (inputs prepared by the full step once)."""
    import torch
    from paper_2609_31395_amd import actkv
    first = bts[0].clone()   # bts are all pristine here; the prep step gets its own copy
    actkv.step(bp, dp.q, dp.kv, first, free, lse=lse, scores=scores, pooled=pooled, kept=kept,
               freed=freed, new_lens=new_lens, ws=ws, qy=qy)
    ks = pooled.clone()   # keep scores of a previous step
    ks_kept = torch.empty(max(qy["num_kept"], 1), dtype=torch.float32, device=scores.device)
    kv0 = dp.kv.clone() if stage == "inplace_compact" else None
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(reps):
        if stage == "score":
            actkv.score(bp, dp.q, dp.kv, bts[i], lse=lse, out=scores, ws=ws)
        elif stage == "select":
            actkv.select(bp, scores, pooled=pooled, kept=kept, ws=ws)
        elif stage == "compact":
            actkv.compact(bp, dp.kv, bts[i], kept, free, freed=freed, new_lens=new_lens, ws=ws)
        elif stage == "lse":
            actkv.lse(bp, dp.q, dp.kv, bts[i], out=lse, ws=ws)
        elif stage == "lrfu_select":
            actkv.lrfu_select(bp, scores, ks, LRFU_TOP_P, LRFU_DECAY, kept=kept, ks_kept=ks_kept,
                              ws=ws)
        elif stage == "inplace_compact":
            # restores K/V and the table before each launch (a copy kernel between launches)
            dp.kv.copy_(kv0)
            bts[i].copy_(bts[-1])
            actkv.compact_inplace(bp, dp.kv, bts[i], kept, ws=ws, want_order=False)
        elif stage == "lrfu_step":
            actkv.step_lrfu(bp, dp.q, dp.kv, bts[i], free, ks, LRFU_TOP_P, LRFU_DECAY, lse=lse,
                            scores=scores, kept=kept, ks_kept=ks_kept, freed=freed,
                            new_lens=new_lens, ws=ws, qy=qy)
        else:
            actkv.step(bp, dp.q, dp.kv, bts[i], free, lse=lse, scores=scores, pooled=pooled,
                       kept=kept, freed=freed, new_lens=new_lens, ws=ws, qy=qy)
    torch.cuda.synchronize()
    print(json.dumps({"profile_stage": stage, "reps": reps,
                      "avg_us": (time.perf_counter() - t0) / reps * 1e6}))


def inplace_pairs(dp, kept) -> int:
    """Row copies the in-place compaction makes for this selection (Alg. 4): per (r, h),
    k minus the kept entries already inside [Start, Start + k)."""
    H, BS = dp.num_kv_heads, dp.page_size
    L = dp.seq_lens.astype(np.int64)
    k = np.minimum(dp.budgets.reshape(-1, H).astype(np.int64), L[:, None])
    off, pairs = 0, 0
    for r in range(L.shape[0]):
        skip = bool((dp.budgets[r * H:(r + 1) * H] >= L[r]).all())
        Y, X = -(-int(L[r]) // BS), -(-int(k[r].max()) // BS)
        start = (Y - X) * BS
        for h in range(H):
            kr = int(k[r, h])
            seg = kept[off:off + kr]
            off += kr
            if not skip:
                pairs += kr - int(((seg >= start) & (seg < start + kr)).sum())
    return pairs


def _binding(dp, dev, q_lens=None):
    from paper_2609_31395_amd import actkv
    return actkv.Problem(seq_lens=dp.seq_lens, q_lens=dp.q_lens if q_lens is None else q_lens,
                         budgets=dp.budgets, num_q_heads=dp.num_q_heads,
                         num_kv_heads=dp.num_kv_heads, head_dim=dp.head_dim,
                         num_pages=dp.num_pages, bt_stride=dp.bt_stride, sm_scale=dp.sm_scale,
                         pool_window=dp.pool_window, causal=dp.causal).to_device(dev)


def _event_pairs(n):
    import torch
    return [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(n)]


def _mean_ms(ev, skip=1):
    return float(np.mean([a.elapsed_time(b) for a, b in ev[skip:]]))


def _graph_us(body, reps_in_graph=10, replays=5):
    """GPU time per call of body(): body captured reps_in_graph times in one graph, which is
    replayed `replays` times between events."""
    import torch
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for _ in range(reps_in_graph):
            body()
    g.replay()
    torch.cuda.synchronize()
    ev = _event_pairs(replays)
    for a, b in ev:
        a.record()
        g.replay()
        b.record()
    torch.cuda.synchronize()
    return _mean_ms(ev, skip=0) * 1e3 / reps_in_graph


def run_score_data_probe(reps, bp, dp, bt0, lse, scores, ws, stream):
    """The scoring kernel alone (actkv_score with the plan flag) on three contents of the
    same K/V and Q: as drawn (bf16 N(0,1) with spikes), every element 1.0, every element 0.
    The instructions and memory accesses are the same; only the switching activity of the
    data differs.  Rounds of `reps` launches per content, interleaved, median per content."""
    import torch
    from paper_2609_31395_amd import actkv
    pp = bp.planned()
    kv0, q0 = dp.kv.clone(), dp.q.clone()
    contents = {"drawn": None, "ones": 0x3F80, "zeros": 0}
    times = {k: [] for k in contents}
    actkv.plan(bp, ws)
    for _ in range(3):
        for name, bits in contents.items():
            if bits is None:
                dp.kv.copy_(kv0)
                dp.q.copy_(q0)
            else:
                dp.kv.fill_(bits)
                dp.q.fill_(bits)
            actkv.score(pp, dp.q, dp.kv, bt0, lse=lse, out=scores, ws=ws)
            ev = _event_pairs(reps)
            for a, b in ev:
                a.record(stream)
                actkv.score(pp, dp.q, dp.kv, bt0, lse=lse, out=scores, ws=ws)
                b.record(stream)
            torch.cuda.synchronize()
            times[name] += [a.elapsed_time(b) * 1e3 for a, b in ev]
    dp.kv.copy_(kv0)
    dp.q.copy_(q0)
    return {"score_data_probe": {k: {"median_us": float(np.median(v)),
                                     "p10_p90": percentiles(v)} for k, v in times.items()},
            "workload": dp.cfg_name, "launches_per_content": 3 * reps}


def run_table1(reps, dev, stream):
    """Table 1 shapes (r requests compressed L -> B; 8 KV heads, d = 128): one streaming
    scoring step (one action query per request, LSE supplied) and one compression operation
    -- selection plus the in-place compaction of Alg. 4, and selection plus the fresh-page
    compaction -- each timed with events on the launch stream; K/V and the block table are
    restored before each compaction, outside the events.  The compression operations use
    the plan the score step leaves in the workspace (ACTKV_FLAG_PLANNED)."""
    import torch
    from paper_2609_31395_amd import actkv
    from paper_2609_31395_amd import workloads as W
    rows = []
    for name in [k for k in W.CONFIGS if k.startswith("table1_")]:
        dp = W.make_device_problem(name, device=dev)
        bp = _binding(dp, dev)
        qy = actkv.query(bp)
        ws = torch.empty(qy["workspace_bytes"], dtype=torch.uint8, device=dev)
        bt0 = torch.from_numpy(dp.block_table).to(dev)
        bt = bt0.clone()
        free = torch.from_numpy(dp.free_pages).to(dev)
        lse = actkv.lse(bp, dp.q, dp.kv, bt0, ws=ws)
        n_sc = actkv.num_scores(bp)
        acc = torch.zeros(n_sc, dtype=torch.float32, device=dev)
        pooled = torch.empty_like(acc)
        kept = torch.empty(max(qy["num_kept"], 1), dtype=torch.int32, device=dev)
        freed = torch.empty(max(qy["pages_freed"], 1), dtype=torch.int32, device=dev)
        new_lens = torch.empty(bp.num_reqs * bp.num_kv_heads, dtype=torch.int32, device=dev)
        kv0 = dp.kv.clone()
        ev_s, ev_i, ev_f = _event_pairs(reps + 1), _event_pairs(reps + 1), _event_pairs(reps + 1)
        for e in ev_s:
            e[0].record(stream)
            actkv.score_accumulate(bp, dp.q, dp.kv, bt0, acc, lse=lse, ws=ws)
            e[1].record(stream)
        # the compression operations reuse the plan the score step left in the workspace
        # (same problem): no plan kernel of their own
        pp = bp.planned()
        for e in ev_i:
            dp.kv.copy_(kv0)
            bt.copy_(bt0)
            e[0].record(stream)
            actkv.select(pp, acc, pooled=pooled, kept=kept, ws=ws)
            actkv.compact_inplace(pp, dp.kv, bt, kept, freed=freed, new_lens=new_lens, ws=ws,
                                  want_order=False)
            e[1].record(stream)
        for e in ev_f:
            bt.copy_(bt0)
            e[0].record(stream)
            actkv.select_compact(pp, acc, dp.kv, bt, free, pooled=pooled, kept=kept,
                                 freed=freed, new_lens=new_lens, ws=ws)
            e[1].record(stream)
        torch.cuda.synchronize()
        # the score step and the fresh-page compression replayed from HIP graphs: GPU time
        # without the host's launch cost (the block-table restore is captured too and its own
        # graph's time is subtracted; the in-place form would need the whole K/V restored,
        # which swamps it)
        graph = None
        try:
            def restore_bt():
                bt.copy_(bt0)

            def fresh():
                restore_bt()
                actkv.select_compact(pp, acc, dp.kv, bt, free, pooled=pooled, kept=kept,
                                     freed=freed, new_lens=new_lens, ws=ws)

            side = torch.cuda.Stream()
            side.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(side):
                fresh()
            torch.cuda.current_stream().wait_stream(side)
            torch.cuda.synchronize()
            graph = {
                "score_step_us": _graph_us(lambda: actkv.score_accumulate(
                    bp, dp.q, dp.kv, bt0, acc, lse=lse, ws=ws)),
                "compress_fresh_us": _graph_us(fresh) - _graph_us(restore_bt),
            }
        except Exception as e:   # graphs are a second view of the same work, never required
            log(f"{name}: graph replay not measured ({type(e).__name__}: {e})")
        dp.kv.copy_(kv0)
        bt.copy_(bt0)
        torch.cuda.synchronize()
        L, B = int(dp.seq_lens[0]), int(dp.budgets[0])
        score_us = _mean_ms(ev_s) * 1e3
        k_bytes = n_sc * dp.head_dim * 2
        rows.append({"config": name, "requests": bp.num_reqs, "tokens": L, "budget": B,
                     "score_step_us": score_us,
                     "score_step_hbm_frac": k_bytes / (score_us * 1e-6) / (HBM_PEAK_GBS * 1e9),
                     "compress_inplace_us": _mean_ms(ev_i) * 1e3,
                     "compress_fresh_us": _mean_ms(ev_f) * 1e3,
                     "graph": graph})
        del dp, kv0, ws
        torch.cuda.synchronize()
    return rows


def streaming_setup(dp, dev):
    """The workload as one decode step sees it: every request scores its cache with one
    action query (the first of its action queries), LSE supplied."""
    import torch
    from paper_2609_31395_amd import actkv
    ones = np.ones_like(dp.q_lens)
    bp = _binding(dp, dev, q_lens=ones)
    first = torch.from_numpy(dp.cu_q[:-1].astype(np.int64)).to(dev)
    q1 = dp.q[first].contiguous()
    qy = actkv.query(bp)
    ws = torch.empty(qy["workspace_bytes"], dtype=torch.uint8, device=dev)
    bt0 = torch.from_numpy(dp.block_table).to(dev)
    lse = actkv.lse(bp, q1, dp.kv, bt0, ws=ws)
    acc = torch.zeros(actkv.num_scores(bp), dtype=torch.float32, device=dev)
    return bp, q1, bt0, lse, acc, ws


def run_streaming_batch(dp, bp_full, reps, dev, stream):
    """One decode step of streaming scoring over the whole batch (streaming_setup)."""
    import torch
    from paper_2609_31395_amd import actkv
    bp, q1, bt0, lse, acc, ws = streaming_setup(dp, dev)
    ev = _event_pairs(reps + 1)
    for e in ev:
        e[0].record(stream)
        actkv.score_accumulate(bp, q1, dp.kv, bt0, acc, lse=lse, ws=ws)
        e[1].record(stream)
    torch.cuda.synchronize()
    us = _mean_ms(ev) * 1e3
    k_bytes = actkv.num_scores(bp) * dp.head_dim * 2
    return {"score_step_us": us, "k_bytes": k_bytes,
            "hbm_GBps": k_bytes / (us * 1e-6) / 1e9,
            "hbm_frac": k_bytes / (us * 1e-6) / (HBM_PEAK_GBS * 1e9)}


CONF_VOCAB, CONF_TOPK = 151936, 20   # Qwen3 vocabulary; the paper's k


def run_confidence(num_reqs, trace_len, reps, dev, stream):
    """The confidence monitor of one decode step (one row of fp32 logits per request over
    the Qwen3 vocabulary, top-20) and the budget update at a compression trigger (traces of
    trace_len token confidences per request; w = 64, s = 8, b = 10%, x1.75, cap 30K)."""
    import torch
    from paper_2609_31395_amd import actkv
    g = torch.Generator(device=dev).manual_seed(77)
    logits = torch.randn((num_reqs, CONF_VOCAB), generator=g, device=dev) * 3.0
    conf = torch.empty(num_reqs, dtype=torch.float32, device=dev)
    ev = _event_pairs(reps + 1)
    for e in ev:
        e[0].record(stream)
        actkv.token_confidence(logits, top_k=CONF_TOPK, out=conf)
        e[1].record(stream)
    trace = (torch.rand((num_reqs * trace_len,), generator=g, device=dev) * 2.0 + 8.0)
    offsets = np.arange(num_reqs + 1, dtype=np.int64) * trace_len
    offsets_d = torch.from_numpy(offsets).to(dev)
    budgets = torch.full((num_reqs,), 512, dtype=torch.int32, device=dev)
    out = torch.empty_like(budgets)
    eb = _event_pairs(reps + 1)
    for e in eb:
        e[0].record(stream)
        actkv.budget_update(trace, offsets, budgets, out=out, offsets_d=offsets_d)
        e[1].record(stream)
    torch.cuda.synchronize()
    us = _mean_ms(ev) * 1e3
    nbytes = num_reqs * CONF_VOCAB * 4
    return {"rows": num_reqs, "vocab": CONF_VOCAB, "top_k": CONF_TOPK,
            "token_conf_us": us, "token_conf_GBps": nbytes / (us * 1e-6) / 1e9,
            "trace_len": trace_len, "budget_update_us": _mean_ms(eb) * 1e3}


def run_copy_calibration(reps):
    """A plain copy of COPY_CALIB_BYTES bytes, `reps` times: it reads and writes exactly that
    many bytes, so it scales the HBM counters of the other kernels."""
    import torch
    src = torch.empty(COPY_CALIB_BYTES, dtype=torch.uint8, device="cuda").fill_(1)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"profile_stage": "copy", "reps": reps, "bytes": COPY_CALIB_BYTES,
                      "avg_us": (time.perf_counter() - t0) / reps * 1e6}))


def run_lrfu(c):
    """The step with LRFU eviction (Sec. 5.1: keep scores carried from step to step, top-p
    hit mask, decay), and its selection on its own, on the launch stream."""
    import torch
    from paper_2609_31395_amd import actkv
    bp, dp, qy, ws, lse, scores, pooled, kept = (c[k] for k in (
        "bp", "dp", "qy", "ws", "lse", "scores", "pooled", "kept"))
    free, freed, new_lens, bts, bt0, dev, stream, K = (c[k] for k in (
        "free", "freed", "new_lens", "bts", "bt0", "dev", "stream", "K"))
    el = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    ks = pooled.clone()   # the keep scores a previous step left
    ks_kept = torch.empty(max(qy["num_kept"], 1), dtype=torch.float32, device=dev)
    for b in bts:
        b.copy_(bt0)
    torch.cuda.synchronize()

    def lrfu_step(bt):
        actkv.step_lrfu(bp, dp.q, dp.kv, bt, free, ks, LRFU_TOP_P, LRFU_DECAY, lse=lse,
                        scores=scores, kept=kept, ks_kept=ks_kept, freed=freed,
                        new_lens=new_lens, ws=ws, qy=qy)

    lrfu_step(bts[K])   # warm-up on its own pristine copy
    torch.cuda.synchronize()
    el[0].record(stream)
    for i in range(K):
        lrfu_step(bts[i])
    el[1].record(stream)
    torch.cuda.synchronize()
    ms_lrfu = el[0].elapsed_time(el[1]) / K
    el[0].record(stream)
    for i in range(K):
        actkv.lrfu_select(bp, scores, ks, LRFU_TOP_P, LRFU_DECAY, kept=kept, ks_kept=ks_kept,
                          ws=ws)
    el[1].record(stream)
    torch.cuda.synchronize()
    ms_lrfu_select = el[0].elapsed_time(el[1]) / K
    log(f"LRFU step {ms_lrfu * 1e3:.1f} us, LRFU select {ms_lrfu_select * 1e3:.1f} us")
    for b in bts:
        b.copy_(bt0)
    return {"top_p": LRFU_TOP_P, "decay": LRFU_DECAY, "step_us": ms_lrfu * 1e3,
            "select_us": ms_lrfu_select * 1e3, "tokens_per_s": c["sum_L"] / (ms_lrfu * 1e-3)}


def run_inplace(c):
    """The step with the paper's in-place compaction (Alg. 4), and that compaction on its
    own.  K/V and the block table are restored before every launch (enqueued on the same
    stream, outside the events); the host runs ahead of the device throughout."""
    import torch
    from paper_2609_31395_amd import actkv
    bp, dp, qy, ws, lse, scores, pooled, kept = (c[k] for k in (
        "bp", "dp", "qy", "ws", "lse", "scores", "pooled", "kept"))
    new_lens, bts, bt0, dev, stream, K = (c[k] for k in (
        "new_lens", "bts", "bt0", "dev", "stream", "K"))
    kv0 = dp.kv.clone()
    nfreed_ip = actkv.query_inplace(bp)
    freed_ip = torch.empty(max(nfreed_ip, 1), dtype=torch.int32, device=dev)
    order_ip = torch.empty(max(qy["num_kept"], 1), dtype=torch.int32, device=dev)
    ev_ip = _event_pairs(2 * K + 2)
    for i in range(K + 1):
        dp.kv.copy_(kv0)
        bts[0].copy_(bt0)
        ev_ip[i][0].record(stream)
        actkv.step_inplace(bp, dp.q, dp.kv, bts[0], lse=lse, scores=scores, pooled=pooled,
                           kept=kept, freed=freed_ip, new_lens=new_lens, new_order=order_ip,
                           ws=ws, qy=qy, nfreed=nfreed_ip)
        ev_ip[i][1].record(stream)
    for i in range(K + 1):
        dp.kv.copy_(kv0)
        bts[0].copy_(bt0)
        ev_ip[K + 1 + i][0].record(stream)
        actkv.compact_inplace(bp, dp.kv, bts[0], kept, freed=freed_ip, new_lens=new_lens,
                              new_order=order_ip, ws=ws)
        ev_ip[K + 1 + i][1].record(stream)
    torch.cuda.synchronize()
    ms_ip_step = _mean_ms(ev_ip[:K + 1])
    ms_ip_compact = _mean_ms(ev_ip[K + 1:])
    ip_pairs = inplace_pairs(dp, kept[:qy["num_kept"]].cpu().numpy())
    ip_bytes = ip_pairs * 2 * 2 * dp.head_dim * 2   # K and V rows, read and written
    dp.kv.copy_(kv0)
    bts[0].copy_(bt0)
    del kv0
    torch.cuda.synchronize()
    log(f"in-place step {ms_ip_step * 1e3:.1f} us, in-place compaction {ms_ip_compact * 1e3:.1f} us"
        f" ({ip_pairs} row copies)")
    return {"step_us": ms_ip_step * 1e3, "compact_us": ms_ip_compact * 1e3,
            "row_copies": ip_pairs, "bytes_moved": ip_bytes,
            "compact_GBps": ip_bytes / (ms_ip_compact * 1e-3) / 1e9,
            "tokens_per_s": c["sum_L"] / (ms_ip_step * 1e-3)}


def run_other_configs(reps, dev, stream):
    """The step (LSE supplied) on the ragged batched workload and on its Dirichlet-budget
    variant: each block table restored before every step, outside the events."""
    import torch
    from paper_2609_31395_amd import actkv
    from paper_2609_31395_amd import workloads as W
    out = {}
    for name in ("batched", "adaptive"):
        dp = W.make_device_problem(name, device=dev)
        bp = _binding(dp, dev)
        qy = actkv.query(bp)
        ws = torch.empty(qy["workspace_bytes"], dtype=torch.uint8, device=dev)
        bt0 = torch.from_numpy(dp.block_table).to(dev)
        bt = bt0.clone()
        free = torch.from_numpy(dp.free_pages).to(dev)
        lse = actkv.lse(bp, dp.q, dp.kv, bt0, ws=ws)
        freed = torch.empty(max(qy["pages_freed"], 1), dtype=torch.int32, device=dev)
        new_lens = torch.empty(bp.num_reqs * bp.num_kv_heads, dtype=torch.int32, device=dev)
        ev = _event_pairs(reps + 1)
        for a, b in ev:
            bt.copy_(bt0)
            a.record(stream)
            actkv.step(bp, dp.q, dp.kv, bt, free, lse=lse, freed=freed, new_lens=new_lens, ws=ws,
                       qy=qy)
            b.record(stream)
        torch.cuda.synchronize()
        ms = _mean_ms(ev)
        us = [a.elapsed_time(b) * 1e3 for a, b in ev[1:]]
        tokens = int(dp.seq_lens.astype(np.int64).sum())
        t_hbm = algorithmic_bytes(dp, qy["num_kept"]) / (HBM_PEAK_GBS * 1e9)
        t_mfma = score_flops(dp) / (BF16_PEAK_TFLOPS * 1e12)
        t_valu = score_epilogue_slots(dp) / VALU_SLOTS_PER_S
        bound = max(t_hbm, t_mfma, t_valu)
        out[name] = {"requests": dp.num_reqs, "cached_tokens": tokens,
                     "action_queries": int(dp.q_lens.sum()), "kept_entries": qy["num_kept"],
                     "step_us": ms * 1e3, "step_us_p10_p90": percentiles(us),
                     "tokens_per_s": tokens / (ms * 1e-3),
                     "hbm_roofline_frac": t_hbm / (ms * 1e-3),
                     # these batches carry more query rows per cached token than the
                     # headline (32-128 queries, mean ~80): the bound is the larger of the
                     # HBM, MFMA and VALU times
                     "combined_roofline": {"t_hbm_us": t_hbm * 1e6, "t_mfma_us": t_mfma * 1e6,
                                           "t_valu_us": t_valu * 1e6, "bound_us": bound * 1e6,
                                           "frac": bound / (ms * 1e-3)}}
        del dp, ws, bt0, bt, free, lse
        torch.cuda.synchronize()
    return out


def run_small_configs(reps, dev, stream):
    """The tiny single-request layer (2,048 tokens, 8/2 heads, d = 64) and the single
    35,000-token Qwen3-30B-shaped layer: the step (LSE supplied) per repetition, timed with
    HIP events after the block table is restored and a 512 MB buffer is written, so that
    the 256 MB MALL holds none of the layer (both layers fit in it otherwise); median,
    p10 and p90.  The tiny layer is bound by kernel launches (its HBM roofline is 0.14 us)."""
    import torch
    from paper_2609_31395_amd import actkv
    from paper_2609_31395_amd import workloads as W
    out = {}
    flush = torch.empty(MALL_FLUSH_BYTES, dtype=torch.uint8, device=dev)
    for name in ("tiny", "single35k"):
        dp = W.make_device_problem(name, device=dev)
        bp = _binding(dp, dev)
        qy = actkv.query(bp)
        ws = torch.empty(qy["workspace_bytes"], dtype=torch.uint8, device=dev)
        bt0 = torch.from_numpy(dp.block_table).to(dev)
        bt = bt0.clone()
        free = torch.from_numpy(dp.free_pages).to(dev)
        lse = actkv.lse(bp, dp.q, dp.kv, bt0, ws=ws)
        freed = torch.empty(max(qy["pages_freed"], 1), dtype=torch.int32, device=dev)
        new_lens = torch.empty(bp.num_reqs * bp.num_kv_heads, dtype=torch.int32, device=dev)
        ev = _event_pairs(reps + 1)
        for i, (a, b) in enumerate(ev):
            bt.copy_(bt0)
            flush.fill_(i & 0xFF)
            a.record(stream)
            actkv.step(bp, dp.q, dp.kv, bt, free, lse=lse, freed=freed, new_lens=new_lens, ws=ws,
                       qy=qy)
            b.record(stream)
        torch.cuda.synchronize()
        us = [a.elapsed_time(b) * 1e3 for a, b in ev[1:]]
        med = float(np.median(us))
        tokens = int(dp.seq_lens.astype(np.int64).sum())
        alg = algorithmic_bytes(dp, qy["num_kept"])
        out[name] = {"requests": dp.num_reqs, "cached_tokens": tokens,
                     "kept_entries": qy["num_kept"], "step_us_median": med,
                     "step_us_p10_p90": percentiles(us), "tokens_per_s": tokens / (med * 1e-6),
                     "algorithmic_bytes": alg,
                     "hbm_roofline_frac": alg / (HBM_PEAK_GBS * 1e9) / (med * 1e-6),
                     "mall": "flushed before every repetition"}
        log(f"{name}: step {med:.1f} us (p10 {out[name]['step_us_p10_p90'][0]:.1f}, p90 "
            f"{out[name]['step_us_p10_p90'][1]:.1f}), MALL flushed")
        del dp, ws, bt0, bt, free, lse
        torch.cuda.synchronize()
    del flush
    torch.cuda.empty_cache()
    return out


def _time_oracle_step(sample, threads=None):
    """Seconds of one oracle step (all stages, fp64) on host arrays already in memory, at
    `threads` OpenMP threads (None: all the host has)."""
    import oracle
    full = oracle.num_threads()
    oracle.set_threads(threads or full)
    try:
        t1 = time.perf_counter()
        oracle.step(sample)
        return time.perf_counter() - t1, oracle.threads_in_use()
    finally:
        oracle.set_threads(full)


def run_cpu_plan(dev):
    """The CPU oracle's timing plan: the tiny and the single 35K-token layers at one thread
    and at all threads; the 32 x 35K batch, the ragged batch and its Dirichlet-budget
    variant in full at all threads; two layers of the 48-layer model, scaled by 24 to the
    whole model.  Tokens per second per layer, with the CPU model and thread counts."""
    from paper_2609_31395_amd import workloads as W
    import torch
    rows = []

    def add(name, sample, threads, scale=1.0, note=""):
        sec, used = _time_oracle_step(sample, threads)
        tokens = int(sample.seq_lens.astype(np.int64).sum())
        rows.append({"workload": name, "threads": used, "seconds": sec,
                     "cached_tokens": tokens, "tokens_per_s": tokens / sec,
                     "extrapolated_s": sec * scale if scale != 1.0 else None, "note": note})
        log(f"cpu oracle {name} ({used} threads): {sec:.2f} s, {tokens / sec:.0f} tokens/s")

    for name in ("tiny", "single35k"):
        dp = W.make_device_problem(name, device=dev)
        host = dp.host_subset(list(range(dp.num_reqs)))
        del dp
        add(name, host, 1)
        add(name, host, None)
    for name in ("batch32x35k", "batched", "adaptive"):
        dp = W.make_device_problem(name, device=dev)
        host = dp.host_subset(list(range(dp.num_reqs)))
        del dp
        torch.cuda.empty_cache()
        add(name, host, None)
        del host
    layers = W.make_device_model("model48x32", device=dev, num_layers=2)
    for li, dp in enumerate(layers):
        host = dp.host_subset(list(range(dp.num_reqs)))
        add(f"model48x32 layer {li}", host, None, scale=24.0,
            note="x24: the 48-layer step from two sampled layers")
        del host
    del layers
    torch.cuda.empty_cache()
    import oracle
    return {"cpu_model": cpu_model(), "host_threads": oracle.num_threads(), "rows": rows}


def run_fullmodel(reps, dev, stream):
    """The full-model workload: the steps of all 48 layers back to back over one shared page
    pool (LSE supplied: produced per layer by actkv_lse outside the timed region).  Every
    layer writes its compacted rows into the pool's spare pages, so the cache the layers
    read is the same in every repetition; the block tables are restored before each
    repetition, outside the events."""
    import torch
    from paper_2609_31395_amd import actkv
    from paper_2609_31395_amd import workloads as W
    torch.cuda.empty_cache()
    t0 = time.perf_counter()
    layers = W.make_device_model("model48x32", device=dev)
    torch.cuda.synchronize()
    t_gen = time.perf_counter() - t0
    spare = torch.from_numpy(layers[0].free_pages).to(dev)
    kv = layers[0].kv
    ctx, alg_bytes, flops, tokens = [], 0, 0, 0
    for dp in layers:
        bp = _binding(dp, dev)
        qy = actkv.query(bp)
        ws = torch.empty(qy["workspace_bytes"], dtype=torch.uint8, device=dev)
        bt0 = torch.from_numpy(dp.block_table).to(dev)
        lse = actkv.lse(bp, dp.q, dp.kv, bt0, ws=ws)
        freed = torch.empty(max(qy["pages_freed"], 1), dtype=torch.int32, device=dev)
        new_lens = torch.empty(bp.num_reqs * bp.num_kv_heads, dtype=torch.int32, device=dev)
        ctx.append((bp, qy, ws, bt0, bt0.clone(), lse, freed, new_lens, dp.q))
        alg_bytes += algorithmic_bytes(dp, qy["num_kept"])
        flops += score_flops(dp)
        tokens += int(dp.seq_lens.astype(np.int64).sum())
    ev = _event_pairs(reps + 1)
    for i in range(reps + 1):
        for c in ctx:
            c[4].copy_(c[3])
        ev[i][0].record(stream)
        for bp, qy, ws, _, bt, lse, freed, new_lens, q in ctx:
            actkv.step(bp, q, kv, bt, spare, lse=lse, freed=freed, new_lens=new_lens, ws=ws,
                       qy=qy)
        ev[i][1].record(stream)
    torch.cuda.synchronize()
    ms = _mean_ms(ev)
    pipe_ms = _fullmodel_pipelined(ctx, kv, spare, reps, stream)
    d0 = layers[0]
    out = {"workload": "model48x32", "layers": len(layers), "requests": d0.num_reqs,
           "seq_len_range": [int(d0.seq_lens.min()), int(d0.seq_lens.max())],
           "pool_GB": kv.numel() * kv.element_size() / 1e9, "gen_s": t_gen,
           "cached_tokens_all_layers": tokens, "step_ms": ms,
           "layer_step_us": ms * 1e3 / len(layers),
           "tokens_per_s": tokens / (ms * 1e-3),
           "hbm_roofline_frac": alg_bytes / (HBM_PEAK_GBS * 1e9) / (ms * 1e-3),
           "score_mfma_bound_ms": flops / (BF16_PEAK_TFLOPS * 1e12) * 1e3,
           "pipelined": {"step_ms": pipe_ms, "layer_step_us": pipe_ms * 1e3 / len(layers),
                         "tokens_per_s": tokens / (pipe_ms * 1e-3),
                         "hbm_roofline_frac": alg_bytes / (HBM_PEAK_GBS * 1e9) / (pipe_ms * 1e-3),
                         "schedule": "layer l's selection and compaction on a second "
                                     "stream, beside layer l+1's plan and scoring"}}
    del ctx, layers, kv, spare
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return out


def _fullmodel_pipelined(ctx, kv, spare, reps, stream):
    """The same 48 layers on two streams: layer l's plan and scoring on the first, its
    selection and compaction (gather and rewrite) on the second, after an event that marks
    its scoring done, so they overlap layer l+1's plan and scoring.  Every layer has its own
    workspace and score buffers; the compactions, which all write the pool's spare pages,
    stay in order on their stream; no layer reads the spare pages.  Returns ms per 48-layer
    step (events on the first stream, after it has waited for the second)."""
    import torch
    from paper_2609_31395_amd import actkv
    side = torch.cuda.Stream(device=kv.device)   # default priority
    bufs = []
    for bp, qy, ws, _, bt, lse, freed, new_lens, q in ctx:
        n = actkv.num_scores(bp)
        bufs.append((bp.planned(), torch.empty(n, dtype=torch.float32, device=kv.device),
                     torch.empty(n, dtype=torch.float32, device=kv.device),
                     torch.empty(max(qy["num_kept"], 1), dtype=torch.int32, device=kv.device)))
    ev = _event_pairs(reps + 1)
    for i in range(reps + 1):
        for c in ctx:
            c[4].copy_(c[3])
        side.wait_stream(stream)
        ev[i][0].record(stream)
        for (bp, qy, ws, _, bt, lse, freed, new_lens, q), (pp, sc, po, kept) in zip(ctx, bufs):
            actkv.plan(bp, ws, stream=stream)
            actkv.score(pp, q, kv, bt, lse=lse, out=sc, ws=ws, stream=stream)
            side.wait_stream(stream)
            actkv.select(pp, sc, pooled=po, kept=kept, ws=ws, stream=side)
            actkv.compact(pp, kv, bt, kept, spare, freed=freed, new_lens=new_lens, ws=ws,
                          stream=side)
        stream.wait_stream(side)
        ev[i][1].record(stream)
    torch.cuda.synchronize()
    return _mean_ms(ev)


def _leg(name, fn, *args):
    """Run one optional bench leg; a failure (say, out of device memory on a box with less
    free HBM) is logged and the leg reported as null, so the headline line still prints."""
    import torch
    try:
        return fn(*args)
    except Exception as e:   # noqa: BLE001 -- every optional leg is best effort
        log(f"{name} leg not measured: {type(e).__name__}: {e}")
        try:
            torch.cuda.synchronize()
            torch.cuda.empty_cache()
        except Exception:   # noqa: BLE001
            pass
        return None


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py: the benchmark runs on one GPU only (asked for --gpus {args.gpus}); "
              "the compression step would shard by request and KV head with no exchange "
              "between GPUs.", file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2609_31395_amd import actkv
    from paper_2609_31395_amd import workloads as W

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if args.profile_stage == "copy":
        run_copy_calibration(args.steps)
        return
    if args.cpu_plan:
        actkv.load_library()
        print(json.dumps({"cpu_plan": run_cpu_plan(torch.device("cuda:0"))}))
        return
    if args.profile_stage == "fullmodel":
        actkv.load_library()
        fm = run_fullmodel(args.steps, torch.device("cuda:0"), torch.cuda.current_stream())
        print(json.dumps({"profile_stage": "fullmodel", "reps": args.steps, **fm}))
        return
    actkv.load_library()
    dev = torch.device("cuda:0")
    t_gen = time.time()
    dp = W.make_device_problem(args.workload, device=dev)
    torch.cuda.synchronize()
    t_gen = time.time() - t_gen
    log(f"drew {args.workload} on the device in {t_gen:.1f} s")
    bp = actkv.Problem(seq_lens=dp.seq_lens, q_lens=dp.q_lens, budgets=dp.budgets,
                       num_q_heads=dp.num_q_heads, num_kv_heads=dp.num_kv_heads,
                       head_dim=dp.head_dim, num_pages=dp.num_pages, bt_stride=dp.bt_stride,
                       sm_scale=dp.sm_scale, pool_window=dp.pool_window,
                       causal=dp.causal).to_device(dev)
    qy = actkv.query(bp)
    ws = torch.empty(qy["workspace_bytes"], dtype=torch.uint8, device=dev)
    bt0 = torch.from_numpy(dp.block_table).to(dev)
    free = torch.from_numpy(dp.free_pages).to(dev)
    n_sc = actkv.num_scores(bp)
    scores = torch.empty(n_sc, dtype=torch.float32, device=dev)
    pooled = torch.empty(n_sc, dtype=torch.float32, device=dev)
    kept = torch.empty(max(qy["num_kept"], 1), dtype=torch.int32, device=dev)
    freed = torch.empty(max(qy["pages_freed"], 1), dtype=torch.int32, device=dev)
    new_lens = torch.empty(bp.num_reqs * bp.num_kv_heads, dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream()

    # The LSE the decode attention would hand over: produced once, outside the timed region.
    lse = actkv.lse(bp, dp.q, dp.kv, bt0, ws=ws)
    torch.cuda.synchronize()

    K, Wm = args.steps, args.warmup
    # every step compacts against a pristine block table: one copy per step, made up front
    # (a compacted table must never be reused with the original lengths)
    bts = [bt0.clone() for _ in range(K + max(Wm, 1))]

    if args.profile_stage == "streaming":
        bp1, q1, bt1, lse1, acc1, ws1 = streaming_setup(dp, dev)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(K + Wm):
            actkv.score_accumulate(bp1, q1, dp.kv, bt1, acc1, lse=lse1, ws=ws1)
        torch.cuda.synchronize()
        print(json.dumps({"profile_stage": "streaming", "reps": K + Wm,
                          "avg_us": (time.perf_counter() - t0) / (K + Wm) * 1e6}))
        return
    if args.score_data_probe:
        print(json.dumps(run_score_data_probe(K, bp, dp, bt0, lse, scores, ws, stream)))
        return
    if args.profile_stage:
        run_stage(args.profile_stage, K + Wm, bp, dp, bts, lse, scores, pooled, kept, free, freed,
                  new_lens, ws, qy)
        return

    def one_step(bt, with_lse=True):
        actkv.step(bp, dp.q, dp.kv, bt, free, lse=lse if with_lse else None, scores=scores,
                   pooled=pooled, kept=kept, freed=freed, new_lens=new_lens, ws=ws, qy=qy)

    for i in range(Wm):
        one_step(bts[i])
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(K + 1)]
    t0 = time.perf_counter()
    ev[0].record(stream)
    for i in range(K):
        one_step(bts[Wm + i])
        ev[i + 1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    step_ms = [ev[i].elapsed_time(ev[i + 1]) for i in range(K)]
    ms_per_step = ev[0].elapsed_time(ev[K]) / K
    log(f"timed {K} steps: {ms_per_step * 1e3:.1f} us/step")

    # ---- per-stage durations (same work: the plan once, then the three entry points with
    # the plan flag, events between them on the launch stream)
    for b in bts:
        b.copy_(bt0)
    torch.cuda.synchronize()
    pp = bp.planned()
    se = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(K)]
    for i in range(K):
        se[i][0].record(stream)
        actkv.plan(bp, ws)
        se[i][1].record(stream)
        actkv.score(pp, dp.q, dp.kv, bts[i], lse=lse, out=scores, ws=ws)
        se[i][2].record(stream)
        actkv.select(pp, scores, pooled=pooled, kept=kept, ws=ws)
        se[i][3].record(stream)
        actkv.compact(pp, dp.kv, bts[i], kept, free, freed=freed, new_lens=new_lens, ws=ws)
        se[i][4].record(stream)
    torch.cuda.synchronize()
    stage_ms = np.array([[se[i][j].elapsed_time(se[i][j + 1]) for j in range(4)]
                         for i in range(K)]).mean(axis=0)

    # ---- the scoring kernel alone: with the plan already in the workspace, actkv_score
    # launches score_kernel and nothing else (one row chunk per request here), so the events
    # around it time that kernel's launches back to back
    actkv.plan(bp, ws)
    for _ in range(2):
        actkv.score(pp, dp.q, dp.kv, bt0, lse=lse, out=scores, ws=ws)
    ek = _event_pairs(K)
    for a, b in ek:
        a.record(stream)
        actkv.score(pp, dp.q, dp.kv, bt0, lse=lse, out=scores, ws=ws)
        b.record(stream)
    torch.cuda.synchronize()
    score_kernel_us = [a.elapsed_time(b) * 1e3 for a, b in ek]
    log(f"score_kernel alone: {np.mean(score_kernel_us):.1f} us")

    # ---- the step with the LSE pass included (library computes the normaliser)
    for b in bts:
        b.copy_(bt0)
    torch.cuda.synchronize()
    el = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    one_step(bts[K], with_lse=False)   # warm-up on its own pristine copy
    torch.cuda.synchronize()
    el[0].record(stream)
    for i in range(K):
        one_step(bts[i], with_lse=False)
    el[1].record(stream)
    torch.cuda.synchronize()
    ms_with_lse = el[0].elapsed_time(el[1]) / K
    log(f"stages plan/score/select/compact (us) {np.round(stage_ms * 1e3, 1).tolist()}, step "
        f"with LSE pass {ms_with_lse * 1e3:.1f} us")

    sum_L = int(dp.seq_lens.astype(np.int64).sum())
    extra = not args.headline_only
    ctx = dict(bp=bp, dp=dp, qy=qy, ws=ws, lse=lse, scores=scores, pooled=pooled, kept=kept,
               free=free, freed=freed, new_lens=new_lens, bts=bts, bt0=bt0, dev=dev,
               stream=stream, K=K, sum_L=sum_L)
    lrfu = _leg("lrfu", run_lrfu, ctx) if extra else None
    inplace = _leg("inplace", run_inplace, ctx) if extra else None

    value = sum_L / (ms_per_step * 1e-3)
    alg_bytes = algorithmic_bytes(dp, qy["num_kept"])
    flops = score_flops(dp)
    copy_bw = measure_copy_bw(dev)
    t_hbm = alg_bytes / (HBM_PEAK_GBS * 1e9)
    t_mfma = flops / (BF16_PEAK_TFLOPS * 1e12)
    t_valu = score_epilogue_slots(dp) / VALU_SLOTS_PER_S
    score_s = float(np.mean(score_kernel_us)) * 1e-6
    achieved_tflops = flops / score_s / 1e12
    traffic = None
    if os.path.exists(TRAFFIC_FILE):
        with open(TRAFFIC_FILE) as f:
            tr = json.load(f)
        if tr.get("source_sha256") == source_digest() and tr.get("workload") == args.workload:
            traffic = int(tr["hbm_bytes_per_launch"])

    streaming = confidence = table1 = fullmodel = others = small = None
    if extra:
        streaming = _leg("streaming", run_streaming_batch, dp, bp, K, dev, stream)
        if streaming:
            log(f"streaming scoring step (1 query per request): "
                f"{streaming['score_step_us']:.1f} us, {streaming['hbm_GBps']:.0f} GB/s")
        confidence = _leg("confidence", run_confidence, dp.num_reqs, int(dp.seq_lens.max()), K,
                          dev, stream)
        if confidence:
            log(f"confidence: token confidence {confidence['token_conf_us']:.1f} us "
                f"({confidence['token_conf_GBps']:.0f} GB/s), budget update "
                f"{confidence['budget_update_us']:.1f} us")
        table1 = (_leg("table1", run_table1, max(K // 2, 5), dev, stream)
                  if not args.no_table1 else None)
        others = _leg("other_configs", run_other_configs, K, dev, stream)
        small = _leg("small_configs", run_small_configs, K, dev, stream)
        for nm, o in (others or {}).items():
            log(f"{nm}: step {o['step_us']:.1f} us, {o['tokens_per_s'] / 1e9:.3f} G tokens/s, "
                f"{o['hbm_roofline_frac']:.2f} of its HBM roofline")
        fullmodel = (_leg("fullmodel", run_fullmodel, max(K // 4, 3), dev, stream)
                     if not args.no_fullmodel else None)
        if fullmodel:
            log(f"full model (48 layers x 32 requests, 16K-64K tokens): "
                f"{fullmodel['step_ms']:.1f} ms, {fullmodel['layer_step_us']:.0f} us per layer, "
                f"{fullmodel['hbm_roofline_frac']:.2f} of the HBM roofline; selection and "
                f"compaction on a second stream: "
                f"{fullmodel['pipelined']['layer_step_us']:.0f} us per layer")
    if table1:
        for row in table1:
            gr = row["graph"] or {}
            log(f"{row['config']:16s} score step {row['score_step_us']:7.1f} us  compress "
                f"in place {row['compress_inplace_us']:7.1f} us  fresh {row['compress_fresh_us']:7.1f} us"
                + (f"  | graph: score step {gr['score_step_us']:6.1f} us, fresh "
                   f"{gr['compress_fresh_us']:6.1f} us" if gr else ""))

    def cpu_leg():
        reqs = list(range(min(args.cpu_sample_reqs, dp.num_reqs)))
        sample = dp.host_subset(reqs)
        log(f"timing the CPU oracle on {len(reqs)} requests")
        # the oracle's own full step (it derives the LSE itself), all host threads
        cpu_s, used = _time_oracle_step(sample)
        s_tokens = int(sample.seq_lens.astype(np.int64).sum())
        small = {}
        for name in ("tiny", "single35k"):
            sp = W.make_device_problem(name, device=dev)
            host = sp.host_subset(list(range(sp.num_reqs)))
            del sp
            t_one, _ = _time_oracle_step(host, 1)
            t_all, n_all = _time_oracle_step(host)
            small[name] = {"seconds_1_thread": t_one, "seconds_all_threads": t_all,
                           "threads": n_all}
            log(f"cpu oracle {name}: {t_one * 1e3:.1f} ms at 1 thread, {t_all * 1e3:.1f} ms at "
                f"{n_all}")
        return {"value": s_tokens / cpu_s, "unit": "tokens/s", "cores": used,
                "kind": "oracle", "cpu_model": cpu_model(),
                "sample": f"{len(reqs)} of {dp.num_reqs} requests of {args.workload} "
                          f"({s_tokens} cached tokens, all stages, fp64), {cpu_s:.1f} s at "
                          f"{used} threads",
                "single_layers": small}

    cpu = None
    if not args.no_cpu_baseline and args.cpu_sample_reqs > 0:
        cpu = _leg("cpu_baseline", cpu_leg)

    cfg = W.CONFIGS[args.workload]
    out = {
        "metric": METRIC,
        "value": value,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": Wm,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": args.workload,
            "description": cfg.description,
            "requests": dp.num_reqs,
            "cached_tokens": sum_L,
            "q_heads": dp.num_q_heads, "kv_heads": dp.num_kv_heads, "head_dim": dp.head_dim,
            "page_size": dp.page_size,
            "action_queries": int(dp.q_lens.sum()),
            "kept_entries": qy["num_kept"],
            "pool_window": dp.pool_window,
            "lse": "supplied (produced once by actkv_lse outside the timed region)",
            "parallelism": "single GPU",
        },
        "step_us": ms_per_step * 1e3,
        "step_us_p10_p90": [float(np.percentile(step_ms, 10) * 1e3),
                            float(np.percentile(step_ms, 90) * 1e3)],
        "hbm_roofline": {"algorithmic_bytes": alg_bytes,
                         "t_hbm_us": t_hbm * 1e6,
                         "frac": t_hbm / (ms_per_step * 1e-3),
                         "copy_GBps": copy_bw / 1e9,
                         "frac_vs_copy": (alg_bytes / copy_bw) / (ms_per_step * 1e-3)},
        "combined_roofline": {"t_hbm_us": t_hbm * 1e6, "t_mfma_us": t_mfma * 1e6,
                              "t_valu_us": t_valu * 1e6,
                              "bound_us": max(t_hbm, t_mfma, t_valu) * 1e6,
                              "frac": max(t_hbm, t_mfma, t_valu) / (ms_per_step * 1e-3)},
        "stages_us": {"plan": stage_ms[0] * 1e3, "score": stage_ms[1] * 1e3,
                      "select": stage_ms[2] * 1e3, "compact": stage_ms[3] * 1e3},
        "score_kernel_us": {"mean": float(np.mean(score_kernel_us)),
                            "p10_p90": percentiles(score_kernel_us)},
        "step_with_lse_pass_us": ms_with_lse * 1e3,
        "inplace": inplace,
        "streaming": streaming,
        "confidence": confidence,
        "table1": table1,
        "other_configs": others,
        "small_configs": small,
        "fullmodel": fullmodel,
        "lrfu": lrfu,
        "roofline": {
            "kernel": "score_kernel (actkv_score with the plan flag: that kernel alone, LSE "
                      "supplied)",
            "bound": "mfma",
            "achieved": achieved_tflops,
            "peak": BF16_PEAK_TFLOPS,
            "unit": "TFLOP/s",
            "frac": achieved_tflops / BF16_PEAK_TFLOPS,
            "traffic": traffic,
        },
        "cpu_baseline": cpu,
        "wall_s_timed": wall,
        "gen_s": t_gen,
    }
    print(json.dumps(out))


if __name__ == "__main__":
    main()
