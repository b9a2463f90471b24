"""Layers back to back on two streams, every output equal to the one-stream sequence of
actkv_step calls, bit for bit, for two schedules: layer l's selection and compaction on the
second stream beside layer l+1's plan and scoring (the schedule the benchmark's full-model
leg times), and layer l's compaction alone there, beside layer l+1's plan, scoring and
selection.

Four layers of the full-model workload (32 requests of 16K-64K tokens, per-layer
Dirichlet budgets) over one page pool; every layer takes its fresh pages from the pool's
spare pages, as in the benchmark, so the compactions must stay in order on their stream.
Compared per layer: kept indices, pooled scores, block table, freed pages and new lengths;
after the last layer, the spare pages the compactions wrote.
"""
import numpy as np
import pytest
import torch

from paper_2609_31395_amd import actkv
from paper_2609_31395_amd import workloads as W

pytestmark = pytest.mark.gpu

LAYERS = 4


def _binding(dp, dev):
    return actkv.Problem(seq_lens=dp.seq_lens, q_lens=dp.q_lens, budgets=dp.budgets,
                         num_q_heads=dp.num_q_heads, num_kv_heads=dp.num_kv_heads,
                         head_dim=dp.head_dim, num_pages=dp.num_pages, bt_stride=dp.bt_stride,
                         sm_scale=dp.sm_scale, pool_window=dp.pool_window,
                         causal=dp.causal).to_device(dev)


@pytest.mark.parametrize("side_work", ["select_and_compact", "compact"])
def test_layer_pipeline_matches_sequential_steps(side_work):
    dev = torch.device("cuda:0")
    layers = W.make_device_model("model48x32", device=dev, num_layers=LAYERS)
    kv = layers[0].kv
    spare = torch.from_numpy(layers[0].free_pages).to(dev)
    kv0 = kv.clone()
    ctx = []
    for dp in layers:
        bp = _binding(dp, dev)
        qy = actkv.query(bp)
        bt0 = torch.from_numpy(dp.block_table).to(dev)
        ws = torch.empty(qy["workspace_bytes"], dtype=torch.uint8, device=dev)
        lse = actkv.lse(bp, dp.q, kv, bt0, ws=ws)
        n = actkv.num_scores(bp)
        ctx.append(dict(bp=bp, qy=qy, bt0=bt0, ws=ws, lse=lse, q=dp.q, n=n))

    def buffers(c):
        return dict(bt=c["bt0"].clone(),
                    sc=torch.empty(c["n"], dtype=torch.float32, device=dev),
                    po=torch.empty(c["n"], dtype=torch.float32, device=dev),
                    kept=torch.empty(max(c["qy"]["num_kept"], 1), dtype=torch.int32, device=dev),
                    freed=torch.empty(max(c["qy"]["pages_freed"], 1), dtype=torch.int32, device=dev),
                    lens=torch.empty(c["bp"].num_reqs * c["bp"].num_kv_heads, dtype=torch.int32,
                                     device=dev))

    # one stream, one actkv_step per layer
    ref = [buffers(c) for c in ctx]
    for c, b in zip(ctx, ref):
        actkv.step(c["bp"], c["q"], kv, b["bt"], spare, lse=c["lse"], scores=b["sc"],
                   pooled=b["po"], kept=b["kept"], freed=b["freed"], new_lens=b["lens"],
                   ws=c["ws"], qy=c["qy"])
    torch.cuda.synchronize()
    kv_ref = kv.clone()
    kv.copy_(kv0)

    # two streams: layer l's tail on the second stream beside layer l+1
    main = torch.cuda.current_stream()
    side = torch.cuda.Stream(device=dev)   # default priority
    got = [buffers(c) for c in ctx]
    side.wait_stream(main)
    for c, b in zip(ctx, got):
        pp = c["bp"].planned()
        actkv.plan(c["bp"], c["ws"], stream=main)
        actkv.score(pp, c["q"], kv, b["bt"], lse=c["lse"], out=b["sc"], ws=c["ws"], stream=main)
        sel_stream = side if side_work == "select_and_compact" else main
        if side_work == "select_and_compact":
            side.wait_stream(main)
        actkv.select(pp, b["sc"], pooled=b["po"], kept=b["kept"], ws=c["ws"], stream=sel_stream)
        side.wait_stream(main)
        actkv.compact(pp, kv, b["bt"], b["kept"], spare, freed=b["freed"], new_lens=b["lens"],
                      ws=c["ws"], stream=side)
    main.wait_stream(side)
    torch.cuda.synchronize()

    for l, (c, a, b) in enumerate(zip(ctx, ref, got)):
        nk = c["qy"]["num_kept"]
        nf = c["qy"]["pages_freed"]
        assert torch.equal(a["kept"][:nk], b["kept"][:nk]), f"layer {l}: kept"
        assert torch.equal(a["po"], b["po"]), f"layer {l}: pooled scores"
        assert torch.equal(a["bt"], b["bt"]), f"layer {l}: block table"
        assert torch.equal(a["freed"][:nf], b["freed"][:nf]), f"layer {l}: freed pages"
        assert torch.equal(a["lens"], b["lens"]), f"layer {l}: new lengths"
    # the spare pages hold the last layer's compacted rows; the rest of the pool is untouched
    pages = spare.long()
    assert torch.equal(kv_ref[:, pages], kv[:, pages]), "compacted rows in the spare pages"
    assert torch.equal(kv_ref, kv), "whole pool"
