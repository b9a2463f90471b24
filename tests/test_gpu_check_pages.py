"""actkv_check_pages: the device check of the compaction's preconditions.  A well-formed
problem reports 0; each planted fault (a fresh page that is live, one listed twice, one
outside the pool, a live block-table entry outside the pool, a device mirror that differs
from the host) reports its own bit and no other.  Every fault is planted in the check's
inputs only: no compaction ever runs on them."""
import numpy as np
import pytest
import torch

from gpu_util import to_dev
from paper_2609_31395_amd import actkv
from paper_2609_31395_amd import workloads as W

pytestmark = pytest.mark.gpu


def _problem():
    return W.make_custom(seq_lens=[300, 129, 0, 64], q_lens=[7, 3, 0, 2], num_q_heads=8,
                         num_kv_heads=2, head_dim=64, pool_window=3, seed=4,
                         budgets=[75, 20, 40, 129, 5, 5, 64, 64])


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    actkv.load_library()


def _status(bp, bt, free):
    st = actkv.check_pages(bp, bt, free)
    torch.cuda.synchronize()
    return int(st.item())


def test_a_well_formed_problem_passes():
    pb = _problem()
    bp, t = to_dev(pb)
    assert actkv.query(bp)["fresh_pages_needed"] > 0
    assert _status(bp, t["bt"], t["free"]) == 0


def test_the_benchmark_batch_passes():
    dev = torch.device("cuda:0")
    dp = W.make_device_problem("batch32x35k", device=dev)
    bp = actkv.Problem(seq_lens=dp.seq_lens, q_lens=dp.q_lens, budgets=dp.budgets,
                       num_q_heads=dp.num_q_heads, num_kv_heads=dp.num_kv_heads,
                       head_dim=dp.head_dim, num_pages=dp.num_pages, bt_stride=dp.bt_stride,
                       sm_scale=dp.sm_scale, pool_window=dp.pool_window,
                       causal=dp.causal).to_device(dev)
    bt = torch.from_numpy(dp.block_table).to(dev)
    free = torch.from_numpy(dp.free_pages).to(dev)
    assert _status(bp, bt, free) == 0
    bad = free.clone()
    bad[17_000] = bt[31, 2000]   # a live page among the 17,504 fresh ones
    assert _status(bp, bt, bad) == actkv.CHECK_FRESH_LIVE


def _planted(kind):
    pb = _problem()
    bp, t = to_dev(pb)
    need = actkv.query(bp)["fresh_pages_needed"]
    bt, free = t["bt"], t["free"]
    if kind == "fresh_live":
        free[need - 1] = bt[1, 3]
    elif kind == "fresh_dup":
        free[need - 1] = free[0]
    elif kind == "free_range_high":
        free[2] = pb.num_pages
    elif kind == "free_range_negative":
        free[0] = -1
    elif kind == "table_range":
        bt[0, 5] = pb.num_pages + 7
    elif kind == "mirror_budget":
        bp.budgets_d[3] += 1
    elif kind == "mirror_length":
        bp.seq_lens_d[1] -= 1
    elif kind == "beyond_the_fresh_pages":   # not taken by the step: not checked
        free[need] = -1
    return bp, bt, free


EXPECTED = {
    "fresh_live": actkv.CHECK_FRESH_LIVE,
    "fresh_dup": actkv.CHECK_FRESH_DUP,
    "free_range_high": actkv.CHECK_FREE_RANGE,
    "free_range_negative": actkv.CHECK_FREE_RANGE,
    "table_range": actkv.CHECK_TABLE_RANGE,
    "mirror_budget": actkv.CHECK_MIRRORS,
    "mirror_length": actkv.CHECK_MIRRORS,
    "beyond_the_fresh_pages": 0,
}


@pytest.mark.parametrize("kind", sorted(EXPECTED))
def test_each_planted_fault_reports_its_own_bit(kind):
    bp, bt, free = _planted(kind)
    assert _status(bp, bt, free) == EXPECTED[kind]


def test_status_is_reset_by_each_call():
    bp, bt, free = _planted("fresh_dup")
    status = torch.full((1,), 0x7F, dtype=torch.int32, device="cuda")
    actkv.check_pages(bp, bt, free, status=status)
    torch.cuda.synchronize()
    assert int(status.item()) == actkv.CHECK_FRESH_DUP
    pb = _problem()
    bp2, t2 = to_dev(pb)
    actkv.check_pages(bp2, t2["bt"], t2["free"], status=status)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
