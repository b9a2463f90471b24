"""Streaming scoring (actkv_score_accumulate; Alg. 3 as the paper runs it during decode) and
the Table 1 shapes on the GPU, against the oracle.

  * n decode steps of one query each -- the cache growing by one token per step, the
    aggregate extended by a zero entry for it -- add up to one batched call with all n
    queries (and to the oracle's scores) within the score tolerance;
  * on the Table 1 shapes (8 KV heads, d = 128, one action query), the streaming scores
    match the oracle, the selection matches outside near-ties, and the in-place and
    fresh-page compactions of the GPU's selection are bit-exact.
"""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import (assert_compaction_matches, assert_kept_matches_outside_near_ties,
                      assert_scores_close, to_dev)
from paper_2609_31395_amd import actkv
from paper_2609_31395_amd import workloads as W
from test_gpu_parity import custom

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    actkv.load_library()


def _grow(acc, lens, H):
    """Re-layout of the aggregate when every sequence grows by one token: a zero entry is
    appended to each (request, KV head) segment."""
    out, off = [], 0
    for L in lens:
        for _ in range(H):
            out.append(acc[off:off + L])
            out.append(np.zeros(1, np.float32))
            off += L
    return np.concatenate(out)


@pytest.mark.parametrize("agg", ["sum", "max_mean"])
def test_streaming_steps_add_up_to_the_batched_call(agg):
    n = 6
    pb = custom(seq_lens=[300, 77, 1030], q_lens=[n, n, n], num_q_heads=8, num_kv_heads=2,
                budgets=[50] * 6, pool_window=1)
    H, Hq = pb.num_kv_heads, pb.num_q_heads
    lse = oracle.lse(pb).astype(np.float32)           # [sum n, Hq]
    bp, t = to_dev(pb, agg=agg)
    batched = actkv.score(bp, t["q"], t["kv"], t["bt"], lse=torch.from_numpy(lse).cuda())
    torch.cuda.synchronize()
    L_final = np.asarray(pb.seq_lens, np.int64)
    cu = pb.cu_q
    acc = None
    for j in range(n):
        lens = (L_final - n + j + 1).astype(np.int32)
        if acc is None:
            acc = np.zeros(int(lens.sum()) * H, np.float32)
        else:
            acc = _grow(acc, lens - 1, H)
        rows = cu[:-1] + j
        bpj = actkv.Problem(seq_lens=lens, q_lens=np.ones_like(lens), budgets=pb.budgets,
                            num_q_heads=Hq, num_kv_heads=H, head_dim=pb.head_dim,
                            num_pages=pb.num_pages, bt_stride=pb.bt_stride,
                            sm_scale=pb.sm_scale, pool_window=1, causal=True,
                            agg=agg).to_device("cuda")
        acc_d = torch.from_numpy(acc).cuda()
        qj = t["q"][torch.from_numpy(rows).cuda()].contiguous()
        lj = torch.from_numpy(np.ascontiguousarray(lse[rows])).cuda()
        actkv.score_accumulate(bpj, qj, t["kv"], t["bt"], acc_d, lse=lj)
        torch.cuda.synchronize()
        acc = acc_d.cpu().numpy()
    if agg == "max_mean":
        acc = acc / n   # each step adds the group max: the running mean is acc / steps
    assert_scores_close(acc, batched.cpu().numpy(), what="streaming vs batched")
    assert_scores_close(acc, oracle.scores(pb, lse_in=lse, agg=agg), what="streaming vs oracle")


def test_accumulator_must_be_16_byte_aligned():
    pb = custom(seq_lens=[64], q_lens=[1], budgets=[8, 8])
    bp, t = to_dev(pb)
    buf = torch.zeros(oracle.num_scores(pb) + 1, dtype=torch.float32, device="cuda")
    with pytest.raises(actkv.ActKVError):
        actkv.score_accumulate(bp, t["q"], t["kv"], t["bt"], buf[1:])


@pytest.mark.parametrize("name", ["table1_r4_1k", "table1_r4_2k", "table1_r4_6k",
                                  "table1_r64_1k", "table1_r1_6k"])
def test_table1_shapes_against_the_oracle(name):
    pb = W.make_problem(name)
    lse = oracle.lse(pb).astype(np.float32)
    bp, t = to_dev(pb)
    n = oracle.num_scores(pb)
    acc = torch.zeros(n, dtype=torch.float32, device="cuda")
    actkv.score_accumulate(bp, t["q"], t["kv"], t["bt"], acc, lse=torch.from_numpy(lse).cuda())
    kept, pooled = actkv.select(bp, acc)
    torch.cuda.synchronize()
    raw = oracle.scores(pb, lse_in=lse)
    assert_scores_close(acc.cpu().numpy(), raw)
    kept_gpu = kept.cpu().numpy()
    assert_kept_matches_outside_near_ties(pb, kept_gpu, oracle.pool(pb, raw))
    np.testing.assert_array_equal(kept_gpu, oracle.select(pb, pooled.cpu().numpy()))
    # the compression operation of Table 1: in-place compaction of this selection
    kv1, bt1 = t["kv"].clone(), t["bt"].clone()
    out = actkv.compact_inplace(bp, kv1, bt1, kept)
    torch.cuda.synchronize()
    ref = oracle.compact_inplace(pb, kept_gpu)
    np.testing.assert_array_equal(kv1.cpu().numpy().view(np.uint16), ref["kv"])
    np.testing.assert_array_equal(bt1.cpu().numpy(), ref["block_table"])
    np.testing.assert_array_equal(out["freed"].cpu().numpy(), ref["freed"])
    np.testing.assert_array_equal(out["new_order"].cpu().numpy(), ref["new_order"])
    # and the fresh-page form
    freed, new_lens = actkv.compact(bp, t["kv"], t["bt"], kept, t["free"])
    torch.cuda.synchronize()
    assert_compaction_matches(pb, kept_gpu, pb.kv, t["kv"].cpu().numpy().view(np.uint16),
                              t["bt"].cpu().numpy(), freed.cpu().numpy(),
                              new_lens.cpu().numpy())
