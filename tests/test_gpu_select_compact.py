"""actkv_select_compact (selection then fresh-page compaction in one call) against
actkv_select followed by actkv_compact: every output bit-identical, both for problems that
take the fused kernel and for larger ones (separate kernels); repeated calls on one planned
workspace (the per-request counters are left at zero); and the fused path against the
oracle's compaction of its own selection.  The fused kernel runs with one workgroup per
segment (at most 32 segments keeping at most 512 entries each), or with several workgroups
per segment that each select it and copy a share of its rows (segments up to 28,672 entries,
at most 32 MiB of kept K and V rows, as many parts as keep the batch near one workgroup per
CU, at least 128 slots per part, at most 16); the block-table rewrite falls to each
request's last workgroup."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import assert_compaction_matches, to_dev
from paper_2609_31395_amd import actkv
from paper_2609_31395_amd import workloads as W

pytestmark = pytest.mark.gpu

FUSED_MAX_SEGMENTS, FUSED_MAX_K = 32, 512   # the one-part fused kernel's limits
SPLIT_MAX_KEYS, SPLIT_MAX_BYTES = 28672, 32 << 20
SPLIT_GROUPS, SPLIT_MAX, SPLIT_MIN_SLOTS = 256, 16, 128


def custom(**kw):
    base = dict(num_q_heads=8, num_kv_heads=2, head_dim=128, pool_window=3, spike_frac=0.02,
                seed=11)
    base.update(kw)
    return W.make_custom(**base)


# the fused kernel runs for the cases whose name starts with "fused_"
CASES = {
    "fused_ragged": lambda: custom(seq_lens=[900, 37, 2500, 640], q_lens=[7, 1, 20, 3],
                                   budgets=[30, 50, 10, 37, 512, 1, 200, 100]),
    "fused_untouched_and_empty": lambda: custom(seq_lens=[64, 0, 800, 5], q_lens=[3, 0, 9, 2],
                                                budgets=[64, 64, 0, 0, 100, 512, 5, 5]),
    "fused_d64_g4_wide_window": lambda: custom(seq_lens=[4100, 333], q_lens=[3, 16],
                                               num_q_heads=8, head_dim=64, pool_window=31,
                                               budgets=[500, 512, 0, 333]),
    "fused_hkv8_32_segments": lambda: custom(seq_lens=[1024] * 4, q_lens=[1] * 4,
                                             num_q_heads=32, num_kv_heads=8, budgets=512),
    "fused_hkv8_table1_like": lambda: custom(seq_lens=[2048, 2048], q_lens=[1, 1],
                                             num_q_heads=32, num_kv_heads=8, budgets=1536),
    "fused_one_part": lambda: custom(seq_lens=[900, 37, 2500, 640], q_lens=[7, 1, 20, 3],
                                     budgets=[30, 50, 10, 37, 128, 1, 120, 100]),
    "fused_split_keep_all_head": lambda: custom(seq_lens=[300, 700, 129], q_lens=[2, 5, 1],
                                                budgets=[300, 150, 700, 5, 129, 200]),
    "fused_split_max_len": lambda: custom(seq_lens=[28672, 1000], q_lens=[2, 1],
                                          budgets=[8000, 28671, 999, 1000]),
    "fused_one_part_past_the_split_length": lambda: custom(
        seq_lens=[28673, 500], q_lens=[1, 1], budgets=[500, 100, 300, 400]),
    "past_the_split_bytes": lambda: custom(seq_lens=[8192] * 4, q_lens=[1] * 4,
                                           num_q_heads=32, num_kv_heads=8, budgets=4096),
    "past_the_segment_limit": lambda: custom(seq_lens=[300] * 17, q_lens=[1] * 17,
                                             budgets=100),
    "large": lambda: custom(seq_lens=[35000] * 4, q_lens=[1] * 4, num_q_heads=8,
                            num_kv_heads=4, budgets=35000 // 2 + 7),
}


def _splits(pb):
    """Workgroups per segment of the fused kernel (1 where it does not split)."""
    k = np.minimum(pb.budgets.reshape(len(pb.seq_lens), -1), pb.seq_lens[:, None])
    if int(pb.seq_lens.max()) > SPLIT_MAX_KEYS or int(k.sum()) * 4 * pb.head_dim > SPLIT_MAX_BYTES:
        return 1
    s = min(SPLIT_GROUPS // k.size, -(-int(k.max()) // SPLIT_MIN_SLOTS), SPLIT_MAX)
    return max(s, 1)


def _fused(pb):
    k = np.minimum(pb.budgets.reshape(len(pb.seq_lens), -1), pb.seq_lens[:, None])
    return (k.size <= FUSED_MAX_SEGMENTS and int(k.max()) <= FUSED_MAX_K) or _splits(pb) > 1


def test_the_cases_cover_both_fused_forms():
    fused = [CASES[c]() for c in CASES if c.startswith("fused_")]
    assert any(_splits(pb) == 1 for pb in fused) and any(_splits(pb) >= 8 for pb in fused)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    actkv.load_library()


def _scores(pb):
    return torch.from_numpy(oracle.scores(pb, lse_in=oracle.lse(pb).astype(np.float32))).cuda()


def _outputs(t, res, pooled, kept):
    return dict(kv=t["kv"].cpu().numpy(), bt=t["bt"].cpu().numpy(),
                freed=res["freed"].cpu().numpy(), new_lens=res["new_lens"].cpu().numpy(),
                pooled=pooled.cpu().numpy(), kept=kept.cpu().numpy())


@pytest.mark.parametrize("case", sorted(CASES))
def test_select_compact_equals_select_then_compact(case):
    pb = CASES[case]()
    assert _fused(pb) == case.startswith("fused_")
    sc = _scores(pb)
    outs = []
    for fused_call in (False, True):
        bp, t = to_dev(pb)
        qy = actkv.query(bp)
        pooled = torch.full_like(sc, -1.0)
        kept = torch.full((max(qy["num_kept"], 1),), -1, dtype=torch.int32, device="cuda")
        if fused_call:
            res = actkv.select_compact(bp, sc, t["kv"], t["bt"], t["free"], pooled=pooled,
                                       kept=kept)
        else:
            actkv.select(bp, sc, pooled=pooled, kept=kept)
            freed, new_lens = actkv.compact(bp, t["kv"], t["bt"], kept[:qy["num_kept"]],
                                            t["free"])
            res = dict(freed=freed, new_lens=new_lens)
        torch.cuda.synchronize()
        outs.append(_outputs(t, res, pooled, kept))
    for name in outs[0]:
        np.testing.assert_array_equal(outs[1][name], outs[0][name], err_msg=f"{case} {name}")


@pytest.mark.parametrize("case", [c for c in sorted(CASES) if c.startswith("fused_")])
def test_fused_path_matches_the_oracle(case):
    pb = CASES[case]()
    sc = _scores(pb)
    bp, t = to_dev(pb)
    qy = actkv.query(bp)
    pooled = torch.empty_like(sc)
    kept = torch.empty(max(qy["num_kept"], 1), dtype=torch.int32, device="cuda")
    res = actkv.select_compact(bp, sc, t["kv"], t["bt"], t["free"], pooled=pooled, kept=kept)
    torch.cuda.synchronize()
    raw = sc.cpu().numpy()
    np.testing.assert_array_equal(pooled.cpu().numpy(), oracle.pool(pb, raw))
    kept_np = kept[:qy["num_kept"]].cpu().numpy()
    np.testing.assert_array_equal(kept_np, oracle.select(pb, oracle.pool(pb, raw)))
    assert_compaction_matches(pb, kept_np, pb.kv, t["kv"].cpu().numpy().view(np.uint16),
                              t["bt"].cpu().numpy(), res["freed"].cpu().numpy(),
                              res["new_lens"].cpu().numpy())


def test_repeated_calls_on_one_planned_workspace():
    """Five fused calls in a row on one workspace planned once (ACTKV_FLAG_PLANNED), each on
    a pristine block table: every call gives the first call's results (the per-request
    counters return to zero after each launch)."""
    pb = CASES["fused_ragged"]()
    sc = _scores(pb)
    bp, t = to_dev(pb)
    qy = actkv.query(bp)
    ws = actkv.workspace(bp)
    actkv.plan(bp, ws)
    pp = bp.planned()
    bt0, kv0 = t["bt"].clone(), t["kv"].clone()
    ref = None
    for _ in range(5):
        t["bt"].copy_(bt0)
        t["kv"].copy_(kv0)
        pooled = torch.empty_like(sc)
        kept = torch.empty(qy["num_kept"], dtype=torch.int32, device="cuda")
        res = actkv.select_compact(pp, sc, t["kv"], t["bt"], t["free"], pooled=pooled,
                                   kept=kept, ws=ws)
        torch.cuda.synchronize()
        got = _outputs(t, res, pooled, kept)
        if ref is None:
            ref = got
            assert not np.array_equal(got["bt"], bt0.cpu().numpy())
        for name in ref:
            np.testing.assert_array_equal(got[name], ref[name], err_msg=name)
