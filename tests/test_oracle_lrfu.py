"""Pins of the oracle's LRFU eviction policy (Sec. 5.1 keep-score update, Alg. 1 steps 2-5):
the top-p hit mask against an independent brute force and hand-worked cases, the keep-score
update against the recency / frequency limits the paper states for decay 0 and 1, and the
reduction to the plain step when every entry is hit and nothing is remembered."""
import numpy as np
import pytest

import oracle
from paper_2609_31395_amd import workloads as W


def _pb(seq_lens, budgets=None, H=1, window=1):
    budgets = budgets if budgets is not None else [max(1, L // 4) for L in seq_lens
                                                   for _ in range(H)]
    return W.make_custom(seq_lens=seq_lens, q_lens=[min(1, L) for L in seq_lens], num_q_heads=H,
                         num_kv_heads=H, head_dim=64, budgets=budgets, pool_window=window,
                         seed=3)


def brute_hits(att, seq_lens, H, p):
    """Shortest prefix of the (score desc, index asc) order whose running sum reaches p x total
    (p as the float32 the entry points take)."""
    p = float(np.float32(p))
    out, off = np.zeros(att.shape[0], np.uint8), 0
    for L in seq_lens:
        for _ in range(H):
            a = att[off:off + L].astype(np.float64)
            need = p * a.sum()
            if need > 0 and p >= 1:
                out[off:off + L] = a > 0
            elif need > 0:
                order = np.lexsort((np.arange(L), -a))
                run = np.cumsum(a[order])
                m = int(np.searchsorted(run, need, side="left")) + 1   # first index reaching need
                out[off + order[:min(m, L)]] = 1
            off += L
    return out


@pytest.mark.parametrize("p", [0.0, 0.3, 0.9, 0.99, 1.0])
def test_hits_match_brute_force_with_ties_and_zeros(p):
    rng = np.random.default_rng(11)
    seq = [300, 1, 77, 0, 512]
    pb = _pb(seq, H=2)
    att = (rng.integers(0, 20, size=oracle.num_scores(pb)) / 16).astype(np.float32)
    att[rng.random(att.shape[0]) < 0.1] = 0.0
    np.testing.assert_array_equal(oracle.hits(pb, att, p), brute_hits(att, seq, 2, p))


def test_hits_hand_worked():
    pb = _pb([4])
    att = np.array([0.125, 0.5, 0.0, 0.375], np.float32)   # order: t1, t3, t0, t2; total 1
    assert oracle.hits(pb, att, 0.5).tolist() == [0, 1, 0, 0]      # 0.5 reaches 0.5
    assert oracle.hits(pb, att, 0.875).tolist() == [0, 1, 0, 1]    # 0.875 reaches 0.875
    assert oracle.hits(pb, att, 0.9).tolist() == [1, 1, 0, 1]
    assert oracle.hits(pb, att, 1.0).tolist() == [1, 1, 0, 1]      # the zero is never needed
    assert oracle.hits(pb, att, 0.0).tolist() == [0, 0, 0, 0]
    assert oracle.hits(pb, np.zeros(4, np.float32), 0.9).tolist() == [0, 0, 0, 0]


def test_top_p_is_taken_as_float32():
    """The oracle wrapper rounds top_p to float32, the type of the GPU entry point's argument.
    Two scores a0 = fl32(0.9) and a1 = 1 - a0 sum to exactly 1: with p = fl32(0.9) the first
    entry alone reaches p x total, with the double 0.9 the second is needed as well."""
    a0 = np.float32(0.9)
    a1 = np.float32(1.0 - float(a0))
    assert float(a0) + float(a1) == 1.0 and float(a0) < 0.9
    pb = _pb([2])
    att = np.array([a0, a1], np.float32)
    assert oracle.as_f32(0.9) == float(a0)
    assert oracle.hits(pb, att, 0.9).tolist() == [1, 0]
    assert oracle.hits(pb, att, float(np.nextafter(a0, np.float32(1.0)))).tolist() == [1, 1]
    ks = oracle.lrfu_update(pb, att, np.array([1, 0], np.uint8), 0.1, np.ones(2, np.float32))
    assert ks.tolist() == [float(np.float32(np.float32(0.1) * np.float32(1.0)) + a0),
                           float(np.float32(0.1))]


def test_equal_scores_are_hit_lower_index_first():
    pb = _pb([4])
    att = np.full(4, 0.25, np.float32)   # total 1
    assert oracle.hits(pb, att, 0.5).tolist() == [1, 1, 0, 0]
    assert oracle.hits(pb, att, 0.51).tolist() == [1, 1, 1, 0]


def test_hits_are_a_top_set_and_scale_free():
    rng = np.random.default_rng(5)
    pb = _pb([999])
    att = rng.lognormal(-9, 1.5, size=999).astype(np.float32)
    h = oracle.hits(pb, att, 0.9).astype(bool)
    assert att[h].min() >= att[~h].max()
    assert att[h].astype(np.float64).sum() >= 0.9 * att.astype(np.float64).sum()
    np.testing.assert_array_equal(oracle.hits(pb, att * np.float32(4), 0.9), h)


def test_decay_zero_is_recency_and_decay_one_is_frequency():
    pb = _pb([6])
    att = np.array([0.375, 0.125, 0.25, 0.0, 0.0625, 0.5], np.float32)
    hit = np.array([1, 0, 1, 0, 1, 0], np.uint8)
    ks = np.array([0.75, 0.25, 0.0, 0.875, 0.03125, 0.0], np.float32)
    # decay 0: only the current hits count
    np.testing.assert_array_equal(oracle.lrfu_update(pb, att, hit, 0.0, ks), att * hit)
    # decay 1: scores of every hit accumulate, misses keep their score
    np.testing.assert_array_equal(oracle.lrfu_update(pb, att, hit, 1.0, ks),
                                  np.array([1.125, 0.25, 0.25, 0.875, 0.09375, 0.0],
                                           np.float32))


def test_intermittent_entry_survives_with_decay():
    """Hit, miss, miss, hit: with 0 < decay < 1 the keep score decays geometrically while
    the entry is idle and is refreshed by the next hit."""
    pb = _pb([1])
    ks = np.zeros(1, np.float32)
    one = np.ones(1, np.float32)
    for h in (1, 0, 0, 1):
        ks = oracle.lrfu_update(pb, one, np.array([h], np.uint8), 0.5, ks)
    assert ks[0] == np.float32(0.125 + 1.0)


def test_all_hit_and_no_memory_reduces_to_the_plain_step():
    pb = W.make_custom(seq_lens=[400, 130], q_lens=[9, 4], num_q_heads=8, num_kv_heads=2,
                       head_dim=64, budgets=[100, 50, 30, 13], pool_window=5, spike_frac=0.02,
                       seed=9)
    plain = oracle.step(pb)
    lr = oracle.lrfu_step(pb, np.full(oracle.num_scores(pb), 7.0, np.float32), top_p=1.0,
                          decay=0.0)
    assert (plain["pooled"] > 0).all()
    assert lr["hit"].all()
    np.testing.assert_array_equal(lr["ks"], plain["pooled"])
    np.testing.assert_array_equal(lr["kept"], plain["kept"])
    np.testing.assert_array_equal(lr["kv"], plain["kv"])


def test_keep_scores_follow_the_kept_entries():
    pb = _pb([64, 40], budgets=[10, 40])
    rng = np.random.default_rng(2)
    ks = rng.random(oracle.num_scores(pb)).astype(np.float32)
    lr = oracle.lrfu_step(pb, ks, top_p=0.9, decay=0.5)
    np.testing.assert_array_equal(lr["ks_kept"][:10], lr["ks"][:64][lr["kept"][:10]])
    np.testing.assert_array_equal(lr["ks_kept"][10:], lr["ks"][64:][lr["kept"][10:]])
    assert lr["ks_kept"][:10].min() >= np.delete(lr["ks"][:64], lr["kept"][:10]).max()
