"""actkv_step_noalloc (the step on the library's static scratch array, for callers that cannot
allocate) against actkv_step on the same inputs, through the C ABI: scores, pooled scores,
kept indices, the whole K/V cache, the block table, the freed pages and the lengths must be
bit-identical.  Two calls in a row, the second on a smaller problem (the array keeps the
first call's contents), and a problem larger than the array is refused before anything is
enqueued."""
import ctypes

import numpy as np
import pytest
import torch

import oracle
from gpu_util import to_dev
from paper_2609_31395_amd import actkv
from paper_2609_31395_amd import workloads as W

pytestmark = pytest.mark.gpu


def _problem_big():
    # several requests of a few thousand tokens, two row chunks in one of them, unequal
    # head budgets and an untouched request
    return W.make_custom(seq_lens=[5000, 3001, 777, 4096], q_lens=[40, 70, 3, 16],
                         num_q_heads=32, num_kv_heads=4, head_dim=128,
                         budgets=[1250, 900, 1500, 1250, 750, 750, 3001, 10,
                                  800, 800, 800, 800, 1024, 0, 4096, 2000],
                         pool_window=7, spike_frac=0.01, seed=77)


def _problem_small():
    return W.make_problem("tiny")


def _run(pb, noalloc: bool, lse):
    bp, t = to_dev(pb)
    qy = actkv.query(bp)
    n = actkv.num_scores(bp)
    scores = torch.full((max(n, 1),), -1.0, dtype=torch.float32, device="cuda")
    pooled = torch.full_like(scores, -1.0)
    kept = torch.full((max(qy["num_kept"], 1),), -1, dtype=torch.int32, device="cuda")
    freed = torch.full((max(qy["pages_freed"], 1),), -1, dtype=torch.int32, device="cuda")
    new_lens = torch.full((bp.num_reqs * bp.num_kv_heads,), -1, dtype=torch.int32, device="cuda")
    lse_d = torch.from_numpy(lse).cuda()
    if noalloc:
        actkv.step_noalloc(bp, t["q"], t["kv"], t["bt"], t["free"], freed, new_lens, lse=lse_d,
                           scores=scores, pooled=pooled, kept=kept, qy=qy)
    else:
        actkv.step(bp, t["q"], t["kv"], t["bt"], t["free"], lse=lse_d, scores=scores,
                   pooled=pooled, kept=kept, freed=freed, new_lens=new_lens, qy=qy)
    torch.cuda.synchronize()
    out = dict(scores=scores, pooled=pooled, kept=kept, freed=freed, new_lens=new_lens,
               kv=t["kv"], bt=t["bt"])
    return {k: v.cpu().numpy() for k, v in out.items()}


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    actkv.load_library()


def test_noalloc_step_matches_the_step_twice_in_a_row_second_smaller():
    for make in (_problem_big, _problem_small):
        pb = make()
        lse = oracle.lse(pb).astype(np.float32)
        want = _run(pb, False, lse)
        got = _run(pb, True, lse)
        for key in want:
            np.testing.assert_array_equal(got[key], want[key], err_msg=f"{make.__name__}: {key}")


def test_noalloc_refuses_a_problem_past_the_scratch_array():
    """32 requests of 120,000 tokens: about 230 MiB of workspace, refused by the size check
    before the library touches any pointer (all data pointers are NULL here)."""
    R, H = 32, 4
    p = actkv.Problem(seq_lens=[120_000] * R, q_lens=[64] * R, budgets=[30_000] * (R * H),
                      num_q_heads=32, num_kv_heads=H, head_dim=128, num_pages=1 << 20,
                      bt_stride=7500)
    assert actkv.query(p)["workspace_bytes"] > actkv.NOALLOC_SCRATCH_BYTES
    lib = actkv.load_library()
    c = p.cstruct()
    rc = lib.actkv_step_noalloc(ctypes.byref(c), None, None, None, None, None, 0, None, None,
                                None, None, None, None)
    assert rc == -3   # ACTKV_ERR_WORKSPACE_TOO_SMALL
