"""Streaming scoring (actkv_score_accumulate; Alg. 3 as the paper runs it during decode) and
the Table 1 shapes on the GPU, against the oracle.

  * n decode steps of one query each -- the cache growing by one token per step, the
    aggregate extended by a zero entry for it -- add up to one batched call with all n
    queries (and to the oracle's scores) within the score tolerance;
  * on the Table 1 shapes (8 KV heads, d = 128, one action query), the streaming scores
    match the oracle, the selection matches outside near-ties, and the in-place and
    fresh-page compactions of the GPU's selection are bit-exact;
  * decode steps (at most one query per request) run their own kernel, which adds into the
    aggregate in place: every group size and lane layout, both aggregations, both head
    sizes, requests without a query, nothing written outside the aggregate, and at full
    size (32 x 35,000 tokens) equal to the batched kernel and, on sampled requests, to the
    oracle; calls with several queries per request keep the batched path.
"""
import dataclasses

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


# Decode steps (at most one action query per request) are scored and added in one pass by
# their own kernel: every group size (lane groups 1, 2 and 4 of the 16-row tile), both
# aggregations, both head sizes, requests without a query this step, ragged page tails.
DECODE_CASES = {
    "g1": dict(num_q_heads=2, num_kv_heads=2),
    "g4": dict(num_q_heads=8, num_kv_heads=2),
    "g8": dict(num_q_heads=16, num_kv_heads=2),
    "g16_d64": dict(num_q_heads=16, num_kv_heads=1, head_dim=64),
    "g2_d64": dict(num_q_heads=4, num_kv_heads=2, head_dim=64),
    # workgroups of 6 heads in two groups, and of 8 heads in two groups
    "g1_12kv": dict(num_q_heads=12, num_kv_heads=12),
    "g2_16kv": dict(num_q_heads=32, num_kv_heads=16),
}


@pytest.mark.parametrize("agg", ["sum", "max_mean"])
@pytest.mark.parametrize("case", sorted(DECODE_CASES))
def test_decode_step_against_the_oracle(case, agg):
    kw = DECODE_CASES[case]
    lens = [300, 77, 1030, 5, 16, 129]
    H = kw["num_kv_heads"]
    pb = custom(seq_lens=lens, q_lens=[1, 1, 0, 1, 1, 1], budgets=[8] * (len(lens) * H),
                pool_window=1, **kw)
    lse = oracle.lse(pb).astype(np.float32)
    bp, t = to_dev(pb, agg=agg)
    n = oracle.num_scores(pb)
    # the aggregate inside a guarded buffer: nothing outside it may change
    buf = torch.full((n + 64,), -7.0, dtype=torch.float32, device="cuda")
    acc = buf[32:32 + n]
    acc.zero_()
    lse_d = torch.from_numpy(lse).cuda()
    actkv.score_accumulate(bp, t["q"], t["kv"], t["bt"], acc, lse=lse_d)
    torch.cuda.synchronize()
    ref = oracle.scores(pb, lse_in=lse, agg=agg)
    assert_scores_close(acc.cpu().numpy(), ref, what="decode step vs oracle")
    # a second step adds to what is there
    actkv.score_accumulate(bp, t["q"], t["kv"], t["bt"], acc, lse=lse_d)
    torch.cuda.synchronize()
    assert_scores_close(acc.cpu().numpy(), 2 * ref, what="two decode steps")
    guard = buf.cpu().numpy()
    assert (guard[:32] == -7.0).all() and (guard[32 + n:] == -7.0).all()
    # the request without a query this step is left alone
    off = int(H * sum(lens[:2]))
    assert (acc.cpu().numpy()[off:off + H * lens[2]] == 0).all()


def test_decode_step_computes_its_own_lse():
    pb = custom(seq_lens=[500, 33], q_lens=[1, 1], budgets=[8] * 4, pool_window=1,
                num_q_heads=16, num_kv_heads=2)
    bp, t = to_dev(pb)
    acc = torch.zeros(oracle.num_scores(pb), dtype=torch.float32, device="cuda")
    actkv.score_accumulate(bp, t["q"], t["kv"], t["bt"], acc)
    torch.cuda.synchronize()
    assert_scores_close(acc.cpu().numpy(), oracle.scores(pb), what="decode step, own LSE")


def test_several_queries_per_request_take_the_batched_path():
    pb = custom(seq_lens=[300, 77, 640], q_lens=[3, 1, 2], budgets=[8] * 6, pool_window=1)
    lse = oracle.lse(pb).astype(np.float32)
    bp, t = to_dev(pb)
    n = oracle.num_scores(pb)
    acc0 = np.random.default_rng(5).random(n).astype(np.float32) * 1e-3
    acc = torch.from_numpy(acc0).cuda()
    actkv.score_accumulate(bp, t["q"], t["kv"], t["bt"], acc, lse=torch.from_numpy(lse).cuda())
    torch.cuda.synchronize()
    ref = acc0.astype(np.float64) + oracle.scores(pb, lse_in=lse)
    assert_scores_close(acc.cpu().numpy(), ref, what="accumulate, several queries")


def test_decode_step_at_full_size_matches_the_batched_kernel():
    """The 32 x 35,000-token cache with one query per request (as the streaming benchmark
    runs it): the decode kernel's scores against the batched kernel's, everywhere, and
    against the oracle on two sampled requests."""
    dev = torch.device("cuda:0")
    dp = W.make_device_problem("batch32x35k", device=dev)
    ones = np.ones_like(dp.q_lens)
    bp = actkv.Problem(seq_lens=dp.seq_lens, q_lens=ones, budgets=dp.budgets,
                       num_q_heads=dp.num_q_heads, num_kv_heads=dp.num_kv_heads,
                       head_dim=dp.head_dim, num_pages=dp.num_pages, bt_stride=dp.bt_stride,
                       sm_scale=dp.sm_scale, pool_window=1, causal=dp.causal).to_device(dev)
    q1 = dp.q[torch.from_numpy(dp.cu_q[:-1].astype(np.int64)).to(dev)].contiguous()
    bt = torch.from_numpy(dp.block_table).to(dev)
    lse = actkv.lse(bp, q1, dp.kv, bt)
    acc = torch.zeros(actkv.num_scores(bp), dtype=torch.float32, device=dev)
    actkv.score_accumulate(bp, q1, dp.kv, bt, acc, lse=lse)
    batched = actkv.score(bp, q1, dp.kv, bt, lse=lse)
    torch.cuda.synchronize()
    got = acc.cpu().numpy()
    assert_scores_close(got, batched.cpu().numpy(), what="decode vs batched kernel")
    H = dp.num_kv_heads
    offs = np.concatenate([[0], np.cumsum(dp.seq_lens.astype(np.int64) * H)])
    for r in (0, dp.num_reqs - 1):
        host = dp.host_subset([r])
        # that request with its first action query only
        one = dataclasses.replace(host, q_lens=np.ones(1, np.int32), q=host.q[:1].copy(),
                                  pool_window=1)
        ref = oracle.scores(one)   # the oracle's own fp64 LSE
        assert_scores_close(got[offs[r]:offs[r + 1]], ref, what=f"request {r} vs oracle")
