"""Host checks of the benchmark's roofline arithmetic (no GPU): the algorithmic bytes and
flops of the 32 x 35,000 batch written out term by term, and the one-GPU contract."""
import os
import subprocess
import sys
import types

import numpy as np

import bench
from paper_2609_31395_amd import workloads as W


def _batch32x35k_shape():
    cfg = W.CONFIGS["batch32x35k"]
    R, L, n = cfg.num_reqs, cfg.seq_len[0], cfg.q_len[0]
    return types.SimpleNamespace(
        seq_lens=np.full(R, L, np.int32), q_lens=np.full(R, n, np.int32),
        num_q_heads=cfg.num_q_heads, num_kv_heads=cfg.num_kv_heads, head_dim=cfg.head_dim)


def test_algorithmic_bytes_of_the_benchmark_batch():
    dp = _batch32x35k_shape()
    R, L, n, Hq, Hkv, D = 32, 35000, 64, 32, 4, 128
    kept = R * Hkv * (L // 4)                  # 25% budget per KV head
    k_read = R * L * Hkv * D * 2               # every K row once, bf16
    q_read = R * n * Hq * D * 2                # the action queries
    lse_read = R * n * Hq * 4                  # one fp32 LSE per query row
    score_rw = 2 * 4 * R * L * Hkv             # fp32 score written, then read by the select
    kept_rw = 2 * 4 * kept                     # int32 kept index written, then read
    rows = kept * 2 * (D * 2) * 2              # kept K and V rows read and written
    want = k_read + q_read + lse_read + score_rw + kept_rw + rows
    assert want == 2_355_599_360
    assert bench.algorithmic_bytes(dp, kept) == want


def test_score_flops_and_epilogue_slots_of_the_benchmark_batch():
    dp = _batch32x35k_shape()
    G, n, L, D, Hkv, R = 8, 64, 35000, 128, 4, 32
    flops = 2 * (G * n) * L * D * Hkv * R      # one multiply-add per (row, key, channel)
    assert flops == 587_202_560_000
    assert bench.score_flops(dp) == flops
    exps = (G * n) * L * Hkv * R               # one exp2 per (query row, key)
    assert bench.score_epilogue_slots(dp) == exps * (1 + bench.EXP_SLOTS + 1)


def test_more_than_one_gpu_is_refused_with_a_message():
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    r = subprocess.run([sys.executable, os.path.join(root, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
