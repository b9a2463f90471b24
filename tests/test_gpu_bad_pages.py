"""Block-table and free-list entries outside [0, num_pages): the header promises that they
are never dereferenced and that the compacted slots they would feed are left unwritten,
with the block table rewritten and the old row returned as usual.  Checked on the
fresh-page gather (actkv_compact) and on the fused selection+compaction kernel
(actkv_select_compact on a small problem) against a host model of that contract: the whole
page pool bit for bit, the rewritten block table, the freed list and the new lengths.
The kept indices come from the library's own selection of random scores.
"""
import numpy as np
import pytest
import torch

from gpu_util import to_dev
from paper_2609_31395_amd import actkv
from paper_2609_31395_amd import workloads as W

pytestmark = pytest.mark.gpu
BS = 16


def _kept_counts(pb):
    H = pb.num_kv_heads
    L = pb.seq_lens.astype(np.int64)
    k = np.minimum(pb.budgets.reshape(-1, H).astype(np.int64), L[:, None])
    return k, np.concatenate([[0], np.cumsum(k.reshape(-1))])


def _expected(pb, kept, bt, free):
    """The pool, block table, freed list and lengths the contract gives."""
    H, P = pb.num_kv_heads, pb.num_pages
    kv = pb.kv.copy()
    bt_new = bt.copy()
    freed, lens = [], []
    k, koff = _kept_counts(pb)
    off = 0
    for r in range(pb.num_reqs):
        L = int(pb.seq_lens[r])
        b = pb.budgets.reshape(-1, H)[r].astype(np.int64)
        if b.min() >= L:
            lens += [L] * H
            continue
        X, Y = (int(k[r].max()) + BS - 1) // BS, (L + BS - 1) // BS
        for h in range(H):
            seg = kept[koff[r * H + h]:koff[r * H + h + 1]]
            for j, t in enumerate(seg):
                sp, dp = int(bt[r, t // BS]), int(free[off + j // BS])
                if 0 <= sp < P and 0 <= dp < P:
                    kv[:, dp, j % BS, h] = pb.kv[:, sp, t % BS, h]
            lens.append(int(k[r, h]))
        freed += list(bt[r, :Y])
        bt_new[r, :X] = free[off:off + X]
        bt_new[r, X:Y] = -1
        off += X
    return kv, bt_new, np.asarray(freed, dtype=np.int32), np.asarray(lens, dtype=np.int32)


def _plant(pb, seed):
    """Copies of the block table and free list with some entries moved outside the pool."""
    rng = np.random.default_rng(seed)
    P = pb.num_pages
    bt, free = pb.block_table.copy(), pb.free_pages.copy()
    for r in range(pb.num_reqs):
        Y = (int(pb.seq_lens[r]) + BS - 1) // BS
        for i in rng.choice(Y, size=max(1, Y // 8), replace=False):
            bt[r, i] = rng.choice([-3, P, P + 1000])
    for i in rng.choice(len(free) // 2, size=max(1, len(free) // 16), replace=False):
        free[i] = rng.choice([-1, P, P + 5])
    return bt, free


def _check(pb, kept, bt_planted, free_planted, kv_dev, bt_dev, freed, new_lens):
    kv_ref, bt_ref, freed_ref, lens_ref = _expected(pb, kept, bt_planted, free_planted)
    np.testing.assert_array_equal(bt_dev.cpu().numpy(), bt_ref)
    np.testing.assert_array_equal(freed.cpu().numpy()[:freed_ref.size], freed_ref)
    np.testing.assert_array_equal(new_lens.cpu().numpy(), lens_ref)
    got = kv_dev.cpu().numpy().view(np.uint16)
    assert np.array_equal(got, kv_ref), "page pool differs from the contract"


def _random_scores(bp, seed):
    n = actkv.num_scores(bp)
    g = torch.Generator(device="cuda").manual_seed(seed)
    return torch.rand(max(n, 1), generator=g, device="cuda")


@pytest.mark.parametrize("seed", [0, 1])
def test_gather_skips_pages_outside_the_pool(seed):
    pb = W.make_custom(seq_lens=[700, 1500, 333], q_lens=[4, 4, 4], num_q_heads=8,
                       num_kv_heads=4, head_dim=128, budgets=[300, 20, 700, 1, 600, 650, 5,
                                                              1499, 100, 333, 0, 50],
                       seed=seed)
    bp, t = to_dev(pb)
    bt_pl, free_pl = _plant(pb, seed)
    kept, _ = actkv.select(bp, _random_scores(bp, seed))
    kept_h = kept.cpu().numpy()
    bt_dev = torch.from_numpy(bt_pl).cuda()
    freed, new_lens = actkv.compact(bp, t["kv"], bt_dev, kept, torch.from_numpy(free_pl).cuda())
    torch.cuda.synchronize()
    _check(pb, kept_h, bt_pl, free_pl, t["kv"], bt_dev, freed, new_lens)


@pytest.mark.parametrize("seed", [0, 1])
def test_fused_selection_compaction_skips_pages_outside_the_pool(seed):
    # 2 requests x 4 heads, at most 512 kept per head: the single fused kernel
    pb = W.make_custom(seq_lens=[900, 400], q_lens=[2, 2], num_q_heads=8, num_kv_heads=4,
                       head_dim=128, budgets=[300, 512, 17, 200, 399, 100, 250, 1], seed=10 + seed)
    bp, t = to_dev(pb)
    bt_pl, free_pl = _plant(pb, seed)
    qy = actkv.query(bp)
    kept = torch.empty(max(qy["num_kept"], 1), dtype=torch.int32, device="cuda")
    bt_dev = torch.from_numpy(bt_pl).cuda()
    res = actkv.select_compact(bp, _random_scores(bp, 100 + seed), t["kv"], bt_dev,
                               torch.from_numpy(free_pl).cuda(), kept=kept)
    torch.cuda.synchronize()
    _check(pb, kept[:qy["num_kept"]].cpu().numpy(), bt_pl, free_pl, t["kv"], bt_dev,
           res["freed"], res["new_lens"])
