"""GPU parity: the HIP path (through the C ABI) against the CPU oracle on the same seeded
inputs.  Scores within 2e-3 relative; pooled scores, kept indices, compacted K/V, block
tables, freed lists and lengths bit-exact (selection end to end: near-ties inside the score
tolerance excluded)."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import (assert_compaction_matches, assert_kept_matches_outside_near_ties,
                      assert_scores_close, to_dev)
from paper_2609_31395_amd import actkv
from paper_2609_31395_amd import workloads as W

pytestmark = pytest.mark.gpu


def custom(**kw):
    base = dict(num_q_heads=8, num_kv_heads=2, head_dim=128, pool_window=3, spike_frac=0.02,
                seed=7)
    base.update(kw)
    return W.make_custom(**base)


# (name, problem factory) -- ragged lengths, tails, several tiles, every supported G
CASES = {
    "tiny_config": lambda: W.make_problem("tiny"),
    "ragged_g4_d128": lambda: custom(seq_lens=[100, 37, 640], q_lens=[7, 1, 20],
                                     budgets=[30, 50, 10, 37, 200, 1]),
    "two_row_chunks_g8": lambda: custom(seq_lens=[300, 129], q_lens=[70, 33], num_q_heads=16,
                                        budgets=[75, 20, 40, 129]),
    "g1": lambda: custom(seq_lens=[77], q_lens=[5], num_q_heads=2, num_kv_heads=2,
                         budgets=[19, 40]),
    "g3_sum_only": lambda: custom(seq_lens=[150, 65], q_lens=[9, 4], num_q_heads=6,
                                  budgets=[40, 11, 65, 3]),
    "g16_d64": lambda: custom(seq_lens=[200], q_lens=[4], num_q_heads=16, num_kv_heads=1,
                              head_dim=64, budgets=[50]),
    "g2_d64_pool7": lambda: custom(seq_lens=[333, 16, 64], q_lens=[16, 3, 64], num_q_heads=4,
                                   head_dim=64, pool_window=7, budgets=[80, 90, 4, 16, 0, 63]),
    "short_and_empty": lambda: custom(seq_lens=[5, 0, 12, 48], q_lens=[2, 0, 12, 0],
                                      budgets=[2, 9, 0, 0, 12, 3, 10, 20]),
    "non_causal": lambda: custom(seq_lens=[190, 70], q_lens=[12, 80], causal=False,
                                 budgets=[50, 60, 7, 70]),
}
MAXMEAN_OK = {"tiny_config", "ragged_g4_d128", "two_row_chunks_g8", "g1", "g16_d64",
              "g2_d64_pool7", "short_and_empty", "non_causal"}


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    actkv.load_library()


def _lse32(pb):
    return oracle.lse(pb).astype(np.float32)


# the two selection kernels: the default one and the small-footprint one
# (ACTKV_FLAG_SMALL_SELECT) must give the same bits
SELECT_KERNELS = ["default", "small"]


def _select(bp, raw, kernel):
    p = bp.small_select() if kernel == "small" else bp
    return actkv.select(p, torch.from_numpy(raw).cuda())


@pytest.mark.parametrize("case", sorted(CASES))
def test_lse_matches_oracle(case):
    pb = CASES[case]()
    bp, t = to_dev(pb)
    got = actkv.lse(bp, t["q"], t["kv"], t["bt"]).cpu().numpy()
    ref = oracle.lse(pb)
    np.testing.assert_allclose(got, ref, rtol=0, atol=2e-4)


# MAX_MEAN needs G in {1, 2, 4, 8, 16}: only those cases run it
AGG_CASES = [(c, a) for c in sorted(CASES) for a in ("sum", "max_mean")
             if a == "sum" or c in MAXMEAN_OK]


@pytest.mark.parametrize("case,agg", AGG_CASES)
def test_scores_with_supplied_lse(case, agg):
    pb = CASES[case]()
    lse = _lse32(pb)
    bp, t = to_dev(pb, agg=agg)
    got = actkv.score(bp, t["q"], t["kv"], t["bt"], lse=torch.from_numpy(lse).cuda())
    ref = oracle.scores(pb, lse_in=lse, agg=agg)
    assert_scores_close(got.cpu().numpy(), ref)


@pytest.mark.parametrize("case", sorted(CASES))
def test_scores_with_library_lse(case):
    pb = CASES[case]()
    bp, t = to_dev(pb)
    got = actkv.score(bp, t["q"], t["kv"], t["bt"], lse=None)
    assert_scores_close(got.cpu().numpy(), oracle.scores(pb))


@pytest.mark.parametrize("kernel", SELECT_KERNELS)
@pytest.mark.parametrize("case", sorted(CASES))
def test_select_is_bit_exact_on_the_oracle_scores(case, kernel):
    pb = CASES[case]()
    raw = oracle.scores(pb, lse_in=_lse32(pb))
    bp, t = to_dev(pb)
    kept, pooled = _select(bp, raw, kernel)
    np.testing.assert_array_equal(pooled.cpu().numpy(), oracle.pool(pb, raw))
    np.testing.assert_array_equal(kept.cpu().numpy(), oracle.select(pb, oracle.pool(pb, raw)))


@pytest.mark.parametrize("kernel", SELECT_KERNELS)
def test_select_ties_and_plateaus_are_bit_exact(kernel):
    """Many equal scores (max-pool plateaus, quantised values): ties go to the lower index."""
    pb = custom(seq_lens=[5000, 777], q_lens=[1, 1], budgets=[1234, 2500, 1, 776],
                pool_window=9)
    rng = np.random.default_rng(3)
    raw = (rng.integers(0, 40, size=oracle.num_scores(pb)) / 64).astype(np.float32)
    bp, t = to_dev(pb)
    kept, pooled = _select(bp, raw, kernel)
    np.testing.assert_array_equal(pooled.cpu().numpy(), oracle.pool(pb, raw))
    np.testing.assert_array_equal(kept.cpu().numpy(), oracle.select(pb, oracle.pool(pb, raw)))


@pytest.mark.parametrize("kernel", SELECT_KERNELS)
@pytest.mark.parametrize("window", [1, 5, 7, 9])
def test_select_long_segments_are_bit_exact(window, kernel):
    """Segments at and past the LDS-resident length (38,400 keys) take the three select
    paths: LDS (<= 38,400), registers (<= 64,512 and windows <= 7) and global memory (longer,
    or window 9).  Budgets past 38,400 kept entries write the indices in two chunks."""
    pb = custom(seq_lens=[38400, 38401, 50000, 64512, 64513], q_lens=[1] * 5, num_q_heads=1,
                num_kv_heads=1, head_dim=64, budgets=[9600, 20000, 12345, 50000, 64512],
                pool_window=window, spike_frac=0.0)
    rng = np.random.default_rng(11)
    raw = (rng.standard_exponential(oracle.num_scores(pb)) * 1e-3).astype(np.float32)
    raw[::97] = raw[5]   # a plateau of equal values across the threshold region
    bp, t = to_dev(pb)
    kept, pooled = _select(bp, raw, kernel)
    np.testing.assert_array_equal(pooled.cpu().numpy(), oracle.pool(pb, raw))
    np.testing.assert_array_equal(kept.cpu().numpy(), oracle.select(pb, oracle.pool(pb, raw)))


@pytest.mark.parametrize("kernel", SELECT_KERNELS)
@pytest.mark.parametrize("L,k", [(40000, 1), (40000, 39999), (47104, 23552), (64511, 777)])
def test_register_select_on_signed_and_tied_scores(L, k, kernel):
    """The register-resident path (38,400 < L <= 64,512) on scores of both signs (the key
    range spans all 32 bits), signed zeros and runs of equal values, at extreme budgets."""
    pb = custom(seq_lens=[L], q_lens=[1], num_q_heads=1, num_kv_heads=1, head_dim=64,
                budgets=[k], pool_window=7, spike_frac=0.0)
    rng = np.random.default_rng(L + k)
    raw = rng.standard_normal(L).astype(np.float32)
    raw[rng.random(L) < 0.2] = 0.0
    raw[rng.random(L) < 0.1] = np.float32(-0.0)
    raw[rng.random(L) < 0.2] = np.float32(0.5)
    bp, t = to_dev(pb)
    kept, pooled = _select(bp, raw, kernel)
    np.testing.assert_array_equal(pooled.cpu().numpy(), oracle.pool(pb, raw))
    np.testing.assert_array_equal(kept.cpu().numpy(), oracle.select(pb, oracle.pool(pb, raw)))


@pytest.mark.parametrize("kernel", SELECT_KERNELS)
@pytest.mark.parametrize("L,window", [(1000, 7), (40000, 7), (40000, 9), (64513, 3)])
def test_pooled_scores_write_zero_as_positive_zero(L, window, kernel):
    """Every select path (LDS, registers, global memory) writes a pooled -0 as +0 and keeps
    the oracle's selection on signed zeros."""
    pb = custom(seq_lens=[L], q_lens=[1], num_q_heads=1, num_kv_heads=1, head_dim=64,
                budgets=[L // 3], pool_window=window, spike_frac=0.0)
    rng = np.random.default_rng(L + window)
    raw = np.where(rng.random(L) < 0.5, np.float32(-0.0), np.float32(0.0)).astype(np.float32)
    raw[rng.random(L) < 0.2] = np.float32(-1.5)
    raw[rng.random(L) < 0.01] = np.float32(2.0)
    bp, t = to_dev(pb)
    kept, pooled = _select(bp, raw, kernel)
    got = pooled.cpu().numpy()
    assert not np.any((got == 0) & np.signbit(got))
    np.testing.assert_array_equal(got, oracle.pool(pb, raw))
    np.testing.assert_array_equal(kept.cpu().numpy(), oracle.select(pb, oracle.pool(pb, raw)))


@pytest.mark.parametrize("kernel", SELECT_KERNELS)
@pytest.mark.parametrize("window", [15, 63])
def test_select_wide_windows_are_bit_exact(window, kernel):
    """Pooling windows up to the largest supported (63) on segments shorter and longer than
    a tile of the small kernel (2,048 entries) and than the window itself, with k at 0, 1,
    L - 1 and L."""
    pb = custom(seq_lens=[40, 2048, 2049, 7000, 31], q_lens=[1] * 5, num_q_heads=2,
                num_kv_heads=2, head_dim=64, pool_window=window, spike_frac=0.0,
                budgets=[0, 40, 1, 2047, 2048, 2000, 6999, 3500, 31, 30])
    rng = np.random.default_rng(window)
    raw = (rng.standard_exponential(oracle.num_scores(pb)) * 1e-2).astype(np.float32)
    raw[rng.random(raw.size) < 0.3] = np.float32(0.25)
    bp, t = to_dev(pb)
    kept, pooled = _select(bp, raw, kernel)
    np.testing.assert_array_equal(pooled.cpu().numpy(), oracle.pool(pb, raw))
    np.testing.assert_array_equal(kept.cpu().numpy(), oracle.select(pb, oracle.pool(pb, raw)))


@pytest.mark.parametrize("case", sorted(CASES))
def test_compact_is_bit_exact_given_the_oracle_selection(case):
    pb = CASES[case]()
    kept = oracle.select(pb, oracle.pool(pb, oracle.scores(pb, lse_in=_lse32(pb))))
    bp, t = to_dev(pb)
    freed, new_lens = actkv.compact(bp, t["kv"], t["bt"], torch.from_numpy(kept).cuda(), t["free"])
    assert_compaction_matches(pb, kept, pb.kv, t["kv"].cpu().numpy().view(np.uint16),
                              t["bt"].cpu().numpy(), freed.cpu().numpy(), new_lens.cpu().numpy())


@pytest.mark.parametrize("lse_mode", ["supplied", "library"])
@pytest.mark.parametrize("case", sorted(CASES))
def test_step_end_to_end(case, lse_mode):
    pb = CASES[case]()
    lse = _lse32(pb) if lse_mode == "supplied" else None
    bp, t = to_dev(pb)
    n_sc = actkv.num_scores(bp)
    qy = actkv.query(bp)
    scores = torch.empty(max(n_sc, 1), dtype=torch.float32, device="cuda")
    pooled = torch.empty_like(scores)
    kept = torch.empty(max(qy["num_kept"], 1), dtype=torch.int32, device="cuda")
    res = actkv.step(bp, t["q"], t["kv"], t["bt"], t["free"],
                     lse=None if lse is None else torch.from_numpy(lse).cuda(),
                     scores=scores, pooled=pooled, kept=kept)
    torch.cuda.synchronize()
    ref = oracle.step(pb, lse_in=lse)
    assert_scores_close(scores[:n_sc].cpu().numpy(), ref["raw"])
    kept_gpu = res["kept"].cpu().numpy()
    assert_kept_matches_outside_near_ties(pb, kept_gpu, ref["pooled"])
    # pooling and selection are exact functions of the scores: check them on the GPU's own
    np.testing.assert_array_equal(pooled[:n_sc].cpu().numpy(),
                                  oracle.pool(pb, scores[:n_sc].cpu().numpy()))
    np.testing.assert_array_equal(kept_gpu, oracle.select(pb, pooled[:n_sc].cpu().numpy()))
    assert_compaction_matches(pb, kept_gpu, pb.kv, t["kv"].cpu().numpy().view(np.uint16),
                              t["bt"].cpu().numpy(), res["freed"].cpu().numpy(),
                              res["new_lens"].cpu().numpy())


def test_budget_at_least_length_leaves_everything_untouched():
    pb = custom(seq_lens=[130, 64], q_lens=[3, 3], budgets=[130, 500, 64, 64])
    bp, t = to_dev(pb)
    kv0, bt0 = t["kv"].clone(), t["bt"].clone()
    res = actkv.step(bp, t["q"], t["kv"], t["bt"], t["free"], lse=None)
    torch.cuda.synchronize()
    assert torch.equal(t["kv"], kv0) and torch.equal(t["bt"], bt0)
    assert res["freed"].numel() == 0
    assert res["new_lens"].cpu().tolist() == [130, 130, 64, 64]


def test_physical_page_order_gives_identical_logical_results():
    kw = dict(seq_lens=[410, 97], q_lens=[9, 5], budgets=[100, 40, 30, 97], pool_window=5,
              spike_frac=0.03)
    outs = []
    for ident in (True, False):
        pb = custom(identity_pages=ident, **kw)
        bp, t = to_dev(pb)
        n_sc = actkv.num_scores(bp)
        scores = torch.empty(n_sc, dtype=torch.float32, device="cuda")
        kept = torch.empty(actkv.query(bp)["num_kept"], dtype=torch.int32, device="cuda")
        res = actkv.step(bp, t["q"], t["kv"], t["bt"], t["free"], lse=None, scores=scores,
                         kept=kept)
        torch.cuda.synchronize()
        kv = t["kv"].cpu().numpy()
        bt = t["bt"].cpu().numpy()
        logical = []
        for r in range(2):
            for h in range(2):
                k = int(res["new_lens"][r * 2 + h])
                logical.append(np.stack([kv[:, bt[r, j // 16], j % 16, h] for j in range(k)]))
        outs.append((scores.cpu().numpy(), res["kept"].cpu().numpy(), logical))
    np.testing.assert_array_equal(outs[0][0], outs[1][0])
    np.testing.assert_array_equal(outs[0][1], outs[1][1])
    for a, b in zip(outs[0][2], outs[1][2]):
        np.testing.assert_array_equal(a, b)


def test_step_is_deterministic_across_runs():
    pb = custom(seq_lens=[900, 333], q_lens=[40, 8], budgets=[200, 100, 33, 300])
    res = []
    for _ in range(2):
        bp, t = to_dev(pb)
        scores = torch.empty(actkv.num_scores(bp), dtype=torch.float32, device="cuda")
        actkv.step(bp, t["q"], t["kv"], t["bt"], t["free"], lse=None, scores=scores)
        torch.cuda.synchronize()
        res.append((scores.cpu().numpy(), t["kv"].cpu().numpy(), t["bt"].cpu().numpy()))
    for a, b in zip(res[0], res[1]):
        np.testing.assert_array_equal(a, b)


def test_second_step_with_the_same_budgets_is_a_no_op():
    """After a step every compacted request holds exactly its budget (one budget for all
    heads of a request here), so a second step with the same budgets keeps everything: over
    the compacted cache it leaves the K/V cache, the block table and the free list untouched
    and frees nothing.  The third request is within budget from the start."""
    pb = custom(seq_lens=[300, 129, 40], q_lens=[7, 3, 2], budgets=[75, 75, 20, 20, 50, 50])
    bp, t = to_dev(pb)
    lse = torch.from_numpy(_lse32(pb)).cuda()
    first = actkv.step(bp, t["q"], t["kv"], t["bt"], t["free"], lse=lse)
    torch.cuda.synchronize()
    need = actkv.query(bp)["fresh_pages_needed"]
    free2 = torch.cat([t["free"][need:], first["freed"]])
    L2, q2 = [75, 20, 40], [2, 2, 2]
    bp2 = actkv.Problem(seq_lens=L2, q_lens=q2, budgets=pb.budgets, num_q_heads=pb.num_q_heads,
                        num_kv_heads=pb.num_kv_heads, head_dim=pb.head_dim,
                        num_pages=pb.num_pages, bt_stride=pb.bt_stride, sm_scale=pb.sm_scale,
                        pool_window=pb.pool_window, causal=pb.causal).to_device("cuda")
    qy2 = actkv.query(bp2)
    assert qy2["fresh_pages_needed"] == 0 and qy2["pages_freed"] == 0
    kv_before, bt_before = t["kv"].clone(), t["bt"].clone()
    free_before = free2.clone()
    second = actkv.step(bp2, t["q"][:sum(q2)].contiguous(), t["kv"], t["bt"], free2)
    torch.cuda.synchronize()
    assert torch.equal(t["kv"], kv_before)
    assert torch.equal(t["bt"], bt_before)
    assert torch.equal(free2, free_before)
    assert second["freed"].numel() == 0
    np.testing.assert_array_equal(second["new_lens"].cpu().numpy(),
                                  np.repeat(L2, pb.num_kv_heads))


def test_plan_once_then_the_stages_equal_the_step():
    """actkv_plan once, then score, select and compact with ACTKV_FLAG_PLANNED (no plan
    kernel of their own): bit-identical to actkv_step on the same inputs."""
    pb = CASES["two_row_chunks_g8"]()
    lse = torch.from_numpy(_lse32(pb)).cuda()
    bp, t = to_dev(pb)
    qy = actkv.query(bp)
    ref = actkv.step(bp, t["q"], t["kv"], t["bt"], t["free"], lse=lse,
                     scores=torch.empty(actkv.num_scores(bp), device="cuda"),
                     pooled=torch.empty(actkv.num_scores(bp), device="cuda"),
                     kept=torch.empty(qy["num_kept"], dtype=torch.int32, device="cuda"))
    torch.cuda.synchronize()
    bp2, t2 = to_dev(pb)
    ws = actkv.workspace(bp2)
    actkv.plan(bp2, ws)
    pp = bp2.planned()
    scores = actkv.score(pp, t2["q"], t2["kv"], t2["bt"], lse=lse, ws=ws)
    kept, pooled = actkv.select(pp, scores, ws=ws)
    freed, new_lens = actkv.compact(pp, t2["kv"], t2["bt"], kept, t2["free"], ws=ws)
    torch.cuda.synchronize()
    for a, b in [(scores, ref["scores"]), (pooled, ref["pooled"]), (kept, ref["kept"]),
                 (freed, ref["freed"]), (new_lens, ref["new_lens"]), (t2["kv"], t["kv"]),
                 (t2["bt"], t["bt"])]:
        assert torch.equal(a, b)


def test_a_plan_of_another_problem_makes_the_kernels_write_nothing():
    """ACTKV_FLAG_PLANNED on a workspace planned for a different problem: every kernel sees
    the signature mismatch and returns, so the outputs keep their sentinels (no fault)."""
    pa = CASES["ragged_g4_d128"]()
    pb = custom(seq_lens=[100, 37, 600], q_lens=[7, 1, 20], budgets=[30, 50, 10, 37, 200, 1])
    ba, _ = to_dev(pa)
    bb, tb = to_dev(pb)
    ws = torch.zeros(max(actkv.query(ba)["workspace_bytes"], actkv.query(bb)["workspace_bytes"]),
                     dtype=torch.uint8, device="cuda")
    actkv.plan(ba, ws)
    pp = bb.planned()
    n = actkv.num_scores(bb)
    scores = torch.full((n,), -7.0, device="cuda")
    actkv.score(pp, tb["q"], tb["kv"], tb["bt"], lse=torch.from_numpy(_lse32(pb)).cuda(),
                out=scores, ws=ws)
    kept = torch.full((actkv.query(bb)["num_kept"],), -7, dtype=torch.int32, device="cuda")
    actkv.select(pp, scores, kept=kept, ws=ws)
    bt0 = tb["bt"].clone()
    kv0 = tb["kv"].clone()
    actkv.compact(pp, tb["kv"], tb["bt"], kept, tb["free"], ws=ws)
    torch.cuda.synchronize()
    assert bool((scores == -7.0).all()) and bool((kept == -7).all())
    assert torch.equal(tb["bt"], bt0) and torch.equal(tb["kv"], kv0)
