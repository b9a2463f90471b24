"""The pipelined step (request groups scored on the caller's stream while the previous group
is selected and compacted on a second stream; actkv_set_overlap) against the unpipelined
one: every output bit-identical, over ragged batches, several row chunks, untouched and
empty requests, every group count; and against the oracle's pooling and selection of the
GPU's own scores.  The full-size workloads run the pipelined form by default (their tests
are in test_gpu_fullsize*.py)."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import assert_compaction_matches, to_dev
from paper_2609_31395_amd import actkv
from paper_2609_31395_amd import workloads as W

pytestmark = pytest.mark.gpu


def custom(**kw):
    base = dict(num_q_heads=8, num_kv_heads=2, head_dim=128, pool_window=3, spike_frac=0.02,
                seed=5)
    base.update(kw)
    return W.make_custom(**base)


CASES = {
    "ragged": lambda: custom(seq_lens=[900, 37, 2500, 640, 1200],
                             q_lens=[7, 1, 20, 3, 64],
                             budgets=[30, 50, 10, 37, 2500, 1, 200, 100, 0, 1200]),
    "row_chunks_g8": lambda: custom(seq_lens=[300, 129, 1000, 77], q_lens=[70, 33, 90, 5],
                                    num_q_heads=16, budgets=[75, 20, 40, 129, 500, 1, 10, 77]),
    "untouched_and_empty": lambda: custom(seq_lens=[64, 0, 800, 130, 3000, 5],
                                          q_lens=[3, 0, 9, 3, 12, 2],
                                          budgets=[64, 64, 0, 0, 100, 30, 130, 500, 3000, 1,
                                                   5, 5]),
    "d64_pool7_max_mean": lambda: custom(seq_lens=[333, 4100, 64, 2049], q_lens=[16, 3, 64, 8],
                                         num_q_heads=4, head_dim=64, pool_window=7,
                                         budgets=[80, 90, 4000, 16, 0, 63, 1024, 2048]),
}
AGG = {"d64_pool7_max_mean": "max_mean"}


@pytest.fixture(autouse=True)
def _restore_overlap():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    actkv.load_library()
    yield
    actkv.set_overlap(0)


def _run(pb, groups, agg):
    actkv.set_overlap(groups)
    bp, t = to_dev(pb, agg=agg)
    n_sc = actkv.num_scores(bp)
    qy = actkv.query(bp)
    scores = torch.full((max(n_sc, 1),), -1.0, dtype=torch.float32, device="cuda")
    pooled = torch.full_like(scores, -1.0)
    kept = torch.full((max(qy["num_kept"], 1),), -1, dtype=torch.int32, device="cuda")
    res = actkv.step(bp, t["q"], t["kv"], t["bt"], t["free"], lse=None, scores=scores,
                     pooled=pooled, kept=kept)
    torch.cuda.synchronize()
    return dict(scores=scores[:n_sc].cpu().numpy(), pooled=pooled[:n_sc].cpu().numpy(),
                kept=res["kept"].cpu().numpy(), freed=res["freed"].cpu().numpy(),
                new_lens=res["new_lens"].cpu().numpy(), kv=t["kv"].cpu().numpy(),
                bt=t["bt"].cpu().numpy())


@pytest.mark.parametrize("groups", [2, 3, 8])
@pytest.mark.parametrize("case", sorted(CASES))
def test_pipelined_step_is_bit_identical_to_the_unpipelined_one(case, groups):
    pb = CASES[case]()
    agg = AGG.get(case, "sum")
    ref = _run(pb, 1, agg)
    got = _run(pb, groups, agg)
    assert actkv.get_overlap() == groups
    for name in ref:
        np.testing.assert_array_equal(got[name], ref[name], err_msg=f"{case} {name}")
    # and pooling / selection are the oracle's functions of these scores, compaction exact
    np.testing.assert_array_equal(got["pooled"], oracle.pool(pb, got["scores"]))
    np.testing.assert_array_equal(got["kept"], oracle.select(pb, got["pooled"]))
    assert_compaction_matches(pb, got["kept"], pb.kv, got["kv"].view(np.uint16), got["bt"],
                              got["freed"], got["new_lens"])


def test_small_select_flag_in_the_unpipelined_step():
    """ACTKV_FLAG_SMALL_SELECT routes the (unpipelined) step's selection through the
    small-footprint kernel: same bits as the default kernel."""
    pb = CASES["ragged"]()
    actkv.set_overlap(1)
    outs = []
    for small in (False, True):
        bp, t = to_dev(pb)
        p = bp.small_select() if small else bp
        n_sc = actkv.num_scores(bp)
        pooled = torch.empty(n_sc, dtype=torch.float32, device="cuda")
        kept = torch.empty(actkv.query(bp)["num_kept"], dtype=torch.int32, device="cuda")
        res = actkv.step(p, t["q"], t["kv"], t["bt"], t["free"], lse=None, pooled=pooled,
                         kept=kept)
        torch.cuda.synchronize()
        outs.append((pooled.cpu().numpy(), res["kept"].cpu().numpy(), t["kv"].cpu().numpy()))
    for a, b in zip(*outs):
        np.testing.assert_array_equal(a, b)
