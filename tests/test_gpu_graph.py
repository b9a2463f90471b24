"""The entry points only enqueue kernels (no allocation, copy, memset or synchronisation
inside), so a whole step can be captured in a HIP graph and replayed.  Each replay is checked
bit for bit against the eager step, with eager work and synchronisations between replays."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import to_dev
from paper_2609_31395_amd import actkv
from paper_2609_31395_amd import workloads as W

pytestmark = pytest.mark.gpu


def _outputs(bp, qy, dev):
    n = actkv.num_scores(bp)
    return dict(scores=torch.empty(n, dtype=torch.float32, device=dev),
                pooled=torch.empty(n, dtype=torch.float32, device=dev),
                kept=torch.empty(max(qy["num_kept"], 1), dtype=torch.int32, device=dev),
                freed=torch.empty(max(qy["pages_freed"], 1), dtype=torch.int32, device=dev),
                new_lens=torch.empty(bp.num_reqs * bp.num_kv_heads, dtype=torch.int32,
                                     device=dev))


@pytest.mark.parametrize("decode", [False, True])
def test_step_replayed_from_a_graph_matches_the_eager_step(decode):
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    actkv.load_library()
    dev = torch.device("cuda:0")
    # several queries per request (batched scoring) or one (the decode-step kernel)
    pb = W.make_custom(seq_lens=[700, 130, 2100], q_lens=[1, 1, 1] if decode else [9, 4, 33],
                       num_q_heads=8, num_kv_heads=2, head_dim=128,
                       budgets=[200, 31, 65, 130, 500, 1400], pool_window=7, spike_frac=0.02,
                       seed=21)
    bp, t = to_dev(pb)
    qy = actkv.query(bp)
    lse = torch.from_numpy(oracle.lse(pb).astype(np.float32)).to(dev)
    ws = torch.empty(qy["workspace_bytes"], dtype=torch.uint8, device=dev)
    bt0 = t["bt"].clone()

    eager = _outputs(bp, qy, dev)
    actkv.step(bp, t["q"], t["kv"], t["bt"], t["free"], lse=lse, ws=ws, qy=qy, **eager)
    torch.cuda.synchronize()
    eager_bt, eager_kv = t["bt"].clone(), t["kv"].clone()

    out = _outputs(bp, qy, dev)
    bt = t["bt"]

    def body():
        bt.copy_(bt0)   # the step compacts against the pristine block table
        actkv.step(bp, t["q"], t["kv"], bt, t["free"], lse=lse, ws=ws, qy=qy, **out)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        body()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        body()
    for rep in range(3):
        for v in out.values():
            v.fill_(-7)
        bt.fill_(-9)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for k in eager:
            assert torch.equal(out[k], eager[k]), (rep, k)
        assert torch.equal(bt, eager_bt), rep
        assert torch.equal(t["kv"], eager_kv), rep
