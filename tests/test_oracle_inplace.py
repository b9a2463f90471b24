"""Pins of the oracle's in-place compaction (Alg. 4, slot planning of Sec. 7.2).

Pinned against what the paper and the definition fix, not against the oracle itself:
  * a hand-worked case of the closed form (Y, X, Start, End; the region running past L);
  * after compaction, new logical slot j of a head holds, bit for bit, the original row of
    the token new_order[j] -- read back through the new block table;
  * the rows that survive are exactly those of the fresh-page compaction (an independently
    pinned oracle function), only in another order;
  * kept entries already inside the target region do not move, and no row outside the
    destination slots is written;
  * the number of copies is k_h minus the kept entries inside the region;
  * the block table keeps its last X blocks, the first Y - X are freed.
"""
import numpy as np
import pytest

import oracle
from paper_2609_31395_amd import workloads as W

BS = 16


def _pb(seq_lens, budgets, H=1, seed=5):
    return W.make_custom(seq_lens=seq_lens, q_lens=[min(1, L) for L in seq_lens],
                         num_q_heads=H, num_kv_heads=H, head_dim=64, budgets=budgets,
                         pool_window=1, seed=seed)


def _row(kv, bt_row, t, h):
    page, slot = int(bt_row[t // BS]), t % BS
    return kv[:, page, slot, h]


def _segments(pb):
    """(r, h, L, k, kept offset) per segment, in kept order."""
    H, off, out = pb.num_kv_heads, 0, []
    for r, L in enumerate(pb.seq_lens):
        for h in range(H):
            k = int(min(max(int(pb.budgets[r * H + h]), 0), int(L)))
            out.append((r, h, int(L), k, off))
            off += k
    return out


def test_hand_worked_region_past_the_end():
    # L = 40, budget 10: Y = 3, X = 1, Start = 32, End = 42 > L.  Kept inside [32, 42): 33,
    # 35, 38, 39.  Destinations (not kept, ascending): 32, 34, 36, 37, 40, 41 -- the last two
    # are past L but exist in the third block.  Sources (kept outside, ascending): 2, 3, 5,
    # 20, 21, 30.  Pairs: 2->32, 3->34, 5->36, 20->37, 21->40, 30->41.
    pb = _pb([40], [10])
    kept = np.array([2, 3, 5, 20, 21, 30, 33, 35, 38, 39], np.int32)
    out = oracle.compact_inplace(pb, kept)
    assert out["pairs"] == 6
    assert out["new_order"].tolist() == [2, 33, 3, 35, 5, 20, 38, 39, 21, 30]
    bt0 = pb.block_table[0]
    assert out["freed"].tolist() == bt0[:2].tolist()
    assert out["block_table"][0, :3].tolist() == [bt0[2], -1, -1]
    assert out["new_lens"].tolist() == [10]
    # slot 40 is logical block 2, slot 8 of the old table: it now holds token 21's row
    np.testing.assert_array_equal(_row(out["kv"], bt0, 40, 0), _row(pb.kv, bt0, 21, 0))
    # read back through the new table: new slot j holds token new_order[j]
    for j, t in enumerate(out["new_order"]):
        np.testing.assert_array_equal(_row(out["kv"], out["block_table"][0], j, 0),
                                      _row(pb.kv, bt0, int(t), 0))


def test_whole_region_is_the_sequence_when_x_equals_y():
    # L = 20, budget 18: Y = X = 2, Start = 0, End = 18; only kept entries at 18, 19 move,
    # into the holes below 18; no page is freed.
    pb = _pb([20], [18])
    kept = np.array([t for t in range(20) if t not in (4, 11)], np.int32)
    out = oracle.compact_inplace(pb, kept)
    assert out["pairs"] == 2
    assert out["freed"].size == 0
    order = out["new_order"].tolist()
    assert order[4] == 18 and order[11] == 19
    assert [t for j, t in enumerate(order) if j not in (4, 11)] == [j for j in range(18)
                                                                   if j not in (4, 11)]
    np.testing.assert_array_equal(out["block_table"], pb.block_table)


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_invariants_against_the_definition_and_the_fresh_page_form(seed):
    rng = np.random.default_rng(seed)
    H = 4
    seq = [int(x) for x in rng.integers(1, 300, size=6)] + [0, 16, 33]
    bud = []
    for L in seq:
        for h in range(H):
            c = rng.random()
            bud.append(0 if c < 0.1 else (L + 5 if c < 0.2 else int(rng.integers(0, L + 1))))
    pb = _pb(seq, bud, H=H, seed=seed)
    raw = rng.random(oracle.num_scores(pb)).astype(np.float32)
    kept = oracle.select(pb, raw)
    out = oracle.compact_inplace(pb, kept)
    kv_f, bt_f, _, lens_f = oracle.compact(pb, kept)
    np.testing.assert_array_equal(out["new_lens"], lens_f)
    bt_old, kv_old = pb.block_table, pb.kv
    written = np.zeros(kv_old.shape[1:4], bool)   # (page, slot, head) destinations
    pairs, freed = 0, []
    for r, h, L, k, ko in _segments(pb):
        order = out["new_order"][ko:ko + k]
        seg_kept = kept[ko:ko + k]
        np.testing.assert_array_equal(np.sort(order), seg_kept)
        H_r = pb.budgets[r * H:(r + 1) * H]
        if (H_r >= L).all():   # untouched request
            np.testing.assert_array_equal(order, seg_kept)
            np.testing.assert_array_equal(out["block_table"][r], bt_old[r])
            continue
        Y = -(-L // BS)
        X = -(-int(np.minimum(H_r, L).max()) // BS)
        start = (Y - X) * BS
        in_region = seg_kept[(seg_kept >= start) & (seg_kept < start + k)]
        pairs += k - in_region.size
        for t in in_region:   # survivors already in place do not move
            assert order[t - start] == t
        for j, t in enumerate(order):
            np.testing.assert_array_equal(_row(out["kv"], out["block_table"][r], j, h),
                                          _row(kv_old, bt_old[r], int(t), h))
            if t != start + j:
                s = start + j
                written[bt_old[r][s // BS], s % BS, h] = True
        # the same rows as the fresh-page form, which writes them in ascending order
        for j, t in enumerate(np.sort(order)):
            np.testing.assert_array_equal(_row(kv_f, bt_f[r], j, h),
                                          _row(out["kv"], out["block_table"][r],
                                               int(np.nonzero(order == t)[0][0]), h))
        if h == 0:
            freed.extend(bt_old[r][:Y - X].tolist())
            np.testing.assert_array_equal(out["block_table"][r][:X], bt_old[r][Y - X:Y])
            assert (out["block_table"][r][X:Y] == -1).all()
    assert out["pairs"] == pairs
    assert out["freed"].tolist() == freed
    # nothing but the destination rows changed
    same = (out["kv"] == kv_old).all(axis=(0, 4))
    assert same[~written].all()


def test_same_keep_set_on_every_head_is_the_per_request_form():
    """With one keep mask for the whole request (the paper's form), every head makes the
    same pairs."""
    rng = np.random.default_rng(9)
    pb = _pb([150, 77], [40, 40, 40, 30, 30, 30], H=3)
    keep0 = np.sort(rng.choice(150, 40, replace=False)).astype(np.int32)
    keep1 = np.sort(rng.choice(77, 30, replace=False)).astype(np.int32)
    kept = np.concatenate([keep0, keep0, keep0, keep1, keep1, keep1])
    out = oracle.compact_inplace(pb, kept)
    o = out["new_order"]
    np.testing.assert_array_equal(o[0:40], o[40:80])
    np.testing.assert_array_equal(o[0:40], o[80:120])
    np.testing.assert_array_equal(o[120:150], o[150:180])
