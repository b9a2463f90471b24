"""Page accounting of the fresh-page compaction, checked on the CPU (no GPU needed).

Compaction writes K/V only into the first sum_r X_r pages of the caller's free list, so
those pages must not be live: no block-table row may reference them within its first
ceil(L_r / page_size) entries.  The library takes this as the caller's guarantee; here it is
checked for every input the tests and the benchmark generate, together with what the plan
promises about the pages:

  * fresh pages used = the first fresh_pages_needed entries of the free list (the host plan,
    actkv_query), handed out in request order, each to exactly one row;
  * the freed list is the old rows of the compacted requests, in request order;
  * no page is lost or duplicated: live-after + freed + unused free = live-before + free.
"""
import numpy as np
import pytest

import oracle
from paper_2609_31395_amd import actkv
from paper_2609_31395_amd import workloads as W


def live_pages(bt, seq_lens, page_size=16):
    rows = []
    for r, L in enumerate(seq_lens):
        rows.append(bt[r, :-(-int(L) // page_size)])
    return np.concatenate(rows) if rows else np.zeros(0, np.int32)


def binding(pb):
    return actkv.Problem(seq_lens=pb.seq_lens, q_lens=pb.q_lens, budgets=pb.budgets,
                         num_q_heads=pb.num_q_heads, num_kv_heads=pb.num_kv_heads,
                         head_dim=pb.head_dim, num_pages=pb.num_pages, bt_stride=pb.bt_stride,
                         sm_scale=pb.sm_scale, pool_window=pb.pool_window, causal=pb.causal)


PROBLEMS = {
    "tiny": lambda: W.make_problem("tiny"),
    "ragged": lambda: W.make_custom(seq_lens=[100, 37, 640, 0, 16], q_lens=[7, 1, 20, 0, 16],
                                    num_q_heads=8, num_kv_heads=2, head_dim=64,
                                    budgets=[30, 50, 37, 37, 200, 1, 5, 5, 16, 16], seed=3),
    "unequal_heads": lambda: W.make_custom(seq_lens=[333, 64], q_lens=[3, 2], num_q_heads=4,
                                           num_kv_heads=4, head_dim=64,
                                           budgets=[0, 333, 17, 200, 64, 64, 64, 70], seed=5),
}


@pytest.mark.parametrize("name", sorted(PROBLEMS))
def test_fresh_pages_are_never_live_and_pages_are_conserved(name):
    pb = PROBLEMS[name]()
    live0 = live_pages(pb.block_table, pb.seq_lens)
    qy = actkv.query(binding(pb))
    fresh = pb.free_pages[:qy["fresh_pages_needed"]]
    # the caller's guarantee (ACTKV_DEBUG's check): fresh pages are not live
    assert np.intersect1d(fresh, live0).size == 0
    assert np.unique(live0).size == live0.size and np.unique(pb.free_pages).size == pb.free_pages.size
    kept = oracle.select(pb, oracle.pool(pb, oracle.scores(pb, lse_in=oracle.lse(pb).astype(np.float32))))
    _, bt2, freed, new_lens = oracle.compact(pb, kept)
    L = pb.seq_lens.astype(np.int64)
    H = pb.num_kv_heads
    k = np.minimum(pb.budgets.reshape(-1, H).astype(np.int64), L[:, None])
    compacted = [r for r in range(pb.num_reqs) if (pb.budgets[r * H:(r + 1) * H] < L[r]).any()]
    # fresh pages in request order, one row each; old rows freed in request order
    used = np.concatenate([bt2[r, :-(-int(k[r].max()) // 16)] for r in compacted]
                          + [np.zeros(0, np.int32)])
    np.testing.assert_array_equal(used, fresh)
    old_rows = np.concatenate([pb.block_table[r, :-(-int(L[r]) // 16)] for r in compacted]
                              + [np.zeros(0, np.int32)])
    np.testing.assert_array_equal(freed, old_rows)
    assert freed.size == qy["pages_freed"]
    live1 = live_pages(bt2, new_lens.reshape(-1, H).max(axis=1))
    unused = pb.free_pages[qy["fresh_pages_needed"]:]
    before = np.sort(np.concatenate([live0, pb.free_pages]))
    after = np.sort(np.concatenate([live1, freed, unused]))
    np.testing.assert_array_equal(after, before)


@pytest.mark.parametrize("name", ["batch32x35k", "batched", "adaptive", "single35k"])
def test_benchmark_workloads_hand_over_a_free_list_disjoint_from_the_live_pages(name):
    """The device-drawn workloads lay out their pages from a seeded permutation of a pool
    twice the pages in use: the unused half is the free list.  Checked on the host plan
    only (no data drawn)."""
    lay = W.device_layout(name)
    cfg, bt = lay.cfg, lay.block_table
    live = live_pages(bt, lay.seq_lens)
    qy = actkv.query(actkv.Problem(seq_lens=lay.seq_lens, q_lens=lay.q_lens,
                                   budgets=lay.budgets, num_q_heads=cfg.num_q_heads,
                                   num_kv_heads=cfg.num_kv_heads, head_dim=cfg.head_dim,
                                   num_pages=lay.num_pages, bt_stride=bt.shape[1]))
    free = lay.free_pages
    assert free.size >= qy["fresh_pages_needed"]
    assert np.intersect1d(free[:qy["fresh_pages_needed"]], live).size == 0
    assert np.unique(np.concatenate([live, free])).size == live.size + free.size
    assert live.min() >= 0 and free.max() < lay.num_pages
