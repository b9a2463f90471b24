"""Full-size parity in the launch configuration bench.py times (one actkv_step over the whole
batch, LSE supplied by actkv_lse), on one Qwen3-30B-shaped layer of a single 35,000-token
request (32 query / 4 KV heads, d = 128, 64 action queries, scattered pages), on the
benchmark workload -- 32 such requests -- and on the ragged batched (L ~ U[8000, 40000], 32-128 queries: two row chunks, segments
past the LDS-resident select length) and adaptive (Dirichlet budgets, some heads keep
nothing) workloads:

  * sampled requests against the oracle (which derives its own fp64 LSE): scores within
    the 2e-3 bar, the library LSE within 2e-3 in log space, selection outside near-ties;
  * on every segment, properties that hold at any size: SUM-mode segment sums equal G * n,
    pooling and selection are exactly the oracle's functions of the GPU's own scores;
  * compaction of the whole batch checked bit for bit on the device (every kept K and V row
    of every head at its fresh slot), with the block table, freed list and lengths.
"""
import types

import numpy as np
import pytest
import torch

import oracle
from gpu_util import assert_kept_matches_outside_near_ties, assert_scores_close
from paper_2609_31395_amd import actkv
from paper_2609_31395_amd import workloads as W

pytestmark = pytest.mark.gpu

WORKLOADS = ["single35k", "batch32x35k", "batched", "adaptive"]
SAMPLE = [0, 17, 31]   # requests checked against the oracle (those the workload has)


def _shape_only(dp):
    """The fields the oracle's pool / select / totals read, without the device tensors."""
    return types.SimpleNamespace(
        seq_lens=dp.seq_lens, q_lens=dp.q_lens, budgets=dp.budgets,
        num_q_heads=dp.num_q_heads, num_kv_heads=dp.num_kv_heads, head_dim=dp.head_dim,
        page_size=dp.page_size, kv=np.empty((2, dp.num_pages, 0), np.uint16),
        block_table=dp.block_table, sm_scale=dp.sm_scale, pool_window=dp.pool_window,
        causal=dp.causal)


@pytest.fixture(scope="module", params=WORKLOADS)
def run(request):
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    actkv.load_library()
    dev = torch.device("cuda:0")
    dp = W.make_device_problem(request.param, device=dev)
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
    scores = torch.empty(n_sc, dtype=torch.float32, device=dev)
    pooled = torch.empty_like(scores)
    kept = torch.empty(qy["num_kept"], dtype=torch.int32, device=dev)
    res = actkv.step(bp, dp.q, dp.kv, bt, free, lse=lse, scores=scores, pooled=pooled,
                     kept=kept, ws=ws, qy=qy)
    torch.cuda.synchronize()
    return dict(dp=dp, bp=bp, bt_new=bt, lse=lse.cpu().numpy(), scores=scores.cpu().numpy(),
                pooled=pooled.cpu().numpy(), kept=kept.cpu().numpy(),
                freed=res["freed"].cpu().numpy(), new_lens=res["new_lens"].cpu().numpy())


def _offsets(dp):
    L = dp.seq_lens.astype(np.int64)
    H = dp.num_kv_heads
    seg = np.concatenate([[0], np.cumsum(L * H)])
    k = np.minimum(dp.budgets.reshape(-1, H).astype(np.int64), L[:, None])
    kept = np.concatenate([[0], np.cumsum(k.reshape(-1))])
    return seg, kept, k


def test_sampled_requests_match_the_oracle(run):
    """Requests 0, 17 and 31 (those the workload has) against the oracle's whole step."""
    dp = run["dp"]
    seg, koff, _ = _offsets(dp)
    H, Hq = dp.num_kv_heads, dp.num_q_heads
    for r in [r for r in SAMPLE if r < dp.num_reqs]:
        host = dp.host_subset([r])
        ref = oracle.step(host)
        assert_scores_close(run["scores"][seg[r]:seg[r + 1]], ref["raw"],
                            what=f"{dp.cfg_name} request {r} scores")
        cu = dp.cu_q
        lse_gpu = run["lse"].reshape(-1, Hq)[int(cu[r]):int(cu[r + 1])]
        np.testing.assert_allclose(lse_gpu, oracle.lse(host), rtol=0, atol=2e-3,
                                   err_msg=f"{dp.cfg_name} request {r} LSE")
        assert_kept_matches_outside_near_ties(host, run["kept"][koff[r * H]:koff[(r + 1) * H]],
                                              ref["pooled"])


def test_every_segment_sums_to_g_times_n(run):
    dp = run["dp"]
    seg, _, _ = _offsets(dp)
    G = dp.num_q_heads // dp.num_kv_heads
    H = dp.num_kv_heads
    s = run["scores"].astype(np.float64)
    for r in range(dp.num_reqs):
        for h in range(H):
            a = seg[r] + h * int(dp.seq_lens[r])
            tot = s[a:a + int(dp.seq_lens[r])].sum()
            want = G * int(dp.q_lens[r])
            assert abs(tot - want) <= 1e-4 * want, (r, h, tot, want)


def test_pool_and_select_are_the_oracle_functions_of_the_gpu_scores(run):
    pb = _shape_only(run["dp"])
    pooled_ref = oracle.pool(pb, run["scores"])
    np.testing.assert_array_equal(run["pooled"], pooled_ref)
    np.testing.assert_array_equal(run["kept"], oracle.select(pb, run["pooled"]))


def check_whole_batch_compaction(dp, bt_new, kept, freed, new_lens):
    """Fresh-page compaction of a whole device batch, bit for bit on the device: every kept
    K and V row of every head at its fresh slot (the old pages are never written, so the
    pristine rows are still there), block-table rows, the freed list and the lengths."""
    dev = torch.device("cuda:0")
    H, BS = dp.num_kv_heads, dp.page_size
    _, koff, k = _offsets(dp)
    bt_old = dp.block_table
    bt_new = bt_new.cpu().numpy()
    kv = dp.kv
    kept = torch.from_numpy(np.asarray(kept).astype(np.int64)).to(dev)
    freed_ref, fresh_off = [], 0
    for r in range(dp.num_reqs):
        L = int(dp.seq_lens[r])
        Y = -(-L // BS)
        if (dp.budgets[r * H:(r + 1) * H] >= L).all():   # untouched request
            np.testing.assert_array_equal(bt_new[r], bt_old[r])
            np.testing.assert_array_equal(new_lens[r * H:(r + 1) * H], L)
            continue
        X = -(-int(k[r].max()) // BS)
        np.testing.assert_array_equal(bt_new[r, :X], dp.free_pages[fresh_off:fresh_off + X])
        assert (bt_new[r, X:Y] == -1).all()
        freed_ref.append(bt_old[r, :Y])
        fresh_off += X
        old_pages = torch.from_numpy(bt_old[r, :Y].astype(np.int64)).to(dev)
        new_pages = torch.from_numpy(bt_new[r, :X].astype(np.int64)).to(dev)
        for h in range(H):
            idx = kept[koff[r * H + h]:koff[r * H + h + 1]]
            j = torch.arange(idx.numel(), device=dev)
            src = kv[:, old_pages[idx // BS], idx % BS, h]
            dst = kv[:, new_pages[j // BS], j % BS, h]
            assert torch.equal(src, dst), f"request {r} head {h}"
        np.testing.assert_array_equal(new_lens[r * H:(r + 1) * H], k[r])
    np.testing.assert_array_equal(freed, np.concatenate(freed_ref) if freed_ref
                                  else np.zeros(0, np.int32))


def test_whole_batch_compaction_is_bit_exact(run):
    check_whole_batch_compaction(run["dp"], run["bt_new"], run["kept"], run["freed"],
                                 run["new_lens"])
