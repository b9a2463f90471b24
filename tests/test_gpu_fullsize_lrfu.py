"""Full-size parity of the step with LRFU eviction (actkv_step_lrfu; Sec. 5.1, Alg. 1 steps
2-6) on the 32 x 35,000-token benchmark batch (Qwen3-30B shapes), with the paper's settings
top_p = 0.9 and decay 0.5, keep scores carried in from a previous step (random, 30% of the
entries new with keep score 0), in the launch configuration bench.py times (whole batch,
LSE supplied by actkv_lse):

  * sampled requests 0, 17 and 31: scores within 2e-3 of the oracle's (fp64, own LSE);
  * every segment: pooling exactly the oracle's function of the GPU scores; the hit mask
    the oracle's top-p function of the GPU's pooled scores outside the boundary band (the
    band of tests/test_gpu_lrfu.py, from the fixed-point truncation bound); keep scores
    bit-exact as the oracle's update of the GPU's own hit mask; the selection and the kept
    keep scores exactly the oracle's TopK of those keep scores;
  * the whole batch's compaction bit for bit on the device.
"""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import assert_scores_close, segments
from paper_2609_31395_amd import actkv
from paper_2609_31395_amd import workloads as W
from test_gpu_fullsize import SAMPLE, _offsets, _shape_only, check_whole_batch_compaction
from test_gpu_lrfu import boundary_band

pytestmark = pytest.mark.gpu

TOP_P, DECAY = 0.9, 0.5


@pytest.fixture(scope="module")
def run_lrfu():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    actkv.load_library()
    dev = torch.device("cuda:0")
    dp = W.make_device_problem("batch32x35k", device=dev)
    bp = actkv.Problem(seq_lens=dp.seq_lens, q_lens=dp.q_lens, budgets=dp.budgets,
                       num_q_heads=dp.num_q_heads, num_kv_heads=dp.num_kv_heads,
                       head_dim=dp.head_dim, num_pages=dp.num_pages, bt_stride=dp.bt_stride,
                       sm_scale=dp.sm_scale, pool_window=dp.pool_window,
                       causal=dp.causal).to_device(dev)
    qy = actkv.query(bp)
    ws = torch.empty(qy["workspace_bytes"], dtype=torch.uint8, device=dev)
    bt = torch.from_numpy(dp.block_table).to(dev)
    free = torch.from_numpy(dp.free_pages).to(dev)
    n_sc = actkv.num_scores(bp)
    lse = torch.empty(int(dp.q_lens.sum()) * dp.num_q_heads, dtype=torch.float32, device=dev)
    actkv.lse(bp, dp.q, dp.kv, bt, out=lse, ws=ws)
    rng = np.random.default_rng(91)
    ks_in = (rng.random(n_sc) * 2e-3).astype(np.float32)   # the scale of pooled scores here
    ks_in[rng.random(n_sc) < 0.3] = 0.0
    ks = torch.from_numpy(ks_in).to(dev)
    scores = torch.empty(n_sc, dtype=torch.float32, device=dev)
    pooled = torch.empty_like(scores)
    hit = torch.empty(n_sc, dtype=torch.uint8, device=dev)
    kept = torch.empty(qy["num_kept"], dtype=torch.int32, device=dev)
    ks_kept = torch.empty(qy["num_kept"], dtype=torch.float32, device=dev)
    res = actkv.step_lrfu(bp, dp.q, dp.kv, bt, free, ks, TOP_P, DECAY, lse=lse, scores=scores,
                          pooled=pooled, hit=hit, kept=kept, ks_kept=ks_kept, ws=ws, qy=qy)
    torch.cuda.synchronize()
    return dict(dp=dp, ks_in=ks_in, bt_new=bt, scores=scores.cpu().numpy(),
                pooled=pooled.cpu().numpy(), hit=hit.cpu().numpy(), ks=ks.cpu().numpy(),
                kept=kept.cpu().numpy(), ks_kept=ks_kept.cpu().numpy(),
                freed=res["freed"].cpu().numpy(), new_lens=res["new_lens"].cpu().numpy())


def test_sampled_requests_score_like_the_oracle(run_lrfu):
    dp = run_lrfu["dp"]
    seg, _, _ = _offsets(dp)
    for r in SAMPLE:
        host = dp.host_subset([r])
        ref = oracle.scores(host, lse_in=None)
        assert_scores_close(run_lrfu["scores"][seg[r]:seg[r + 1]], ref,
                            what=f"request {r} scores")


def test_hit_mask_keep_scores_and_selection_on_every_segment(run_lrfu):
    dp = run_lrfu["dp"]
    pb = _shape_only(dp)
    pooled = run_lrfu["pooled"]
    np.testing.assert_array_equal(pooled, oracle.pool(pb, run_lrfu["scores"]))
    hit = run_lrfu["hit"]
    band = boundary_band(pb, pooled, TOP_P)
    bad = np.nonzero((hit != oracle.hits(pb, pooled, TOP_P)) & ~band)[0]
    assert bad.size == 0, f"hit mask differs off the boundary at {bad[:8]}"
    assert 0 < hit.sum() < hit.size
    ks2 = oracle.lrfu_update(pb, pooled, hit, DECAY, run_lrfu["ks_in"])
    np.testing.assert_array_equal(run_lrfu["ks"], ks2)
    kept = run_lrfu["kept"]
    np.testing.assert_array_equal(kept, oracle.select(pb, ks2))
    segs = segments(dp.seq_lens, dp.num_kv_heads, ks2)
    want, off = [], 0
    H = dp.num_kv_heads
    for r, L in enumerate(dp.seq_lens):
        for h in range(H):
            k = int(min(int(dp.budgets[r * H + h]), int(L)))
            want.append(segs[(r, h)][kept[off:off + k]])
            off += k
    np.testing.assert_array_equal(run_lrfu["ks_kept"], np.concatenate(want))


def test_whole_batch_compaction_is_bit_exact(run_lrfu):
    check_whole_batch_compaction(run_lrfu["dp"], run_lrfu["bt_new"], run_lrfu["kept"],
                                 run_lrfu["freed"], run_lrfu["new_lens"])
