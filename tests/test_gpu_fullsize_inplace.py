"""Full-size parity of the step with the in-place compaction (actkv_step_inplace, Alg. 4) in
the launch configuration bench.py times, on the benchmark, batched and adaptive workloads.
Checked on the device for the whole batch, against the definition:

  * every new slot j < k of every (request, KV head) holds, bit for bit, the K and V rows
    that token new_order[j] had before the step (read through the new block table);
  * new_order is a permutation of the kept indices, and kept entries already inside the
    target region did not move;
  * nothing but the destination rows changed anywhere in the cache;
  * block tables keep their last X blocks, the first Y - X are freed in request order;
  * selection equals the oracle's function of the GPU's own scores;
  * on sampled requests, new_order, the lengths and the freed pages equal the oracle's
    in-place compaction (Alg. 4) of the same kept entries: the ascending pairing of the kept
    entries outside the tail region with the free slots inside it.
"""
import types

import numpy as np
import pytest
import torch

import oracle
from paper_2609_31395_amd import actkv
from paper_2609_31395_amd import workloads as W
from test_gpu_fullsize import SAMPLE, WORKLOADS, _offsets, _shape_only

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", params=WORKLOADS)
def run_ip(request):
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    actkv.load_library()
    dev = torch.device("cuda:0")
    dp = W.make_device_problem(request.param, device=dev)
    bp = actkv.Problem(seq_lens=dp.seq_lens, q_lens=dp.q_lens, budgets=dp.budgets,
                       num_q_heads=dp.num_q_heads, num_kv_heads=dp.num_kv_heads,
                       head_dim=dp.head_dim, num_pages=dp.num_pages, bt_stride=dp.bt_stride,
                       sm_scale=dp.sm_scale, pool_window=dp.pool_window,
                       causal=dp.causal).to_device(dev)
    qy = actkv.query(bp)
    ws = torch.empty(qy["workspace_bytes"], dtype=torch.uint8, device=dev)
    bt = torch.from_numpy(dp.block_table).to(dev)
    lse = torch.empty(int(dp.q_lens.sum()) * dp.num_q_heads, dtype=torch.float32, device=dev)
    actkv.lse(bp, dp.q, dp.kv, bt, out=lse, ws=ws)
    kv0 = dp.kv.clone()
    n_sc = actkv.num_scores(bp)
    scores = torch.empty(n_sc, dtype=torch.float32, device=dev)
    pooled = torch.empty_like(scores)
    kept = torch.empty(qy["num_kept"], dtype=torch.int32, device=dev)
    order = torch.empty_like(kept)
    res = actkv.step_inplace(bp, dp.q, dp.kv, bt, lse=lse, scores=scores, pooled=pooled,
                             kept=kept, new_order=order, ws=ws, qy=qy)
    torch.cuda.synchronize()
    yield dict(dp=dp, kv0=kv0, bt_new=bt, scores=scores.cpu().numpy(),
               pooled=pooled.cpu().numpy(), kept=kept, order=order,
               freed=res["freed"].cpu().numpy(), new_lens=res["new_lens"].cpu().numpy())
    del kv0


def test_selection_is_the_oracle_function_of_the_gpu_scores(run_ip):
    pb = _shape_only(run_ip["dp"])
    np.testing.assert_array_equal(run_ip["pooled"], oracle.pool(pb, run_ip["scores"]))
    np.testing.assert_array_equal(run_ip["kept"].cpu().numpy(),
                                  oracle.select(pb, run_ip["pooled"]))


def test_whole_batch_inplace_compaction(run_ip):
    dp, kv0 = run_ip["dp"], run_ip["kv0"]
    kv = dp.kv
    dev = kv.device
    H, BS = dp.num_kv_heads, dp.page_size
    _, koff, k = _offsets(dp)
    bt_old = torch.from_numpy(dp.block_table).to(dev)
    bt_new = run_ip["bt_new"]
    kept, order = run_ip["kept"], run_ip["order"]
    written = torch.zeros((dp.num_pages, BS, H), dtype=torch.bool, device=dev)
    freed_ref = []
    for r in range(dp.num_reqs):
        L = int(dp.seq_lens[r])
        if (dp.budgets[r * H:(r + 1) * H] >= L).all():   # untouched request
            assert torch.equal(bt_new[r], bt_old[r])
            np.testing.assert_array_equal(run_ip["new_lens"][r * H:(r + 1) * H], L)
            continue
        Y, X = -(-L // BS), -(-int(k[r].max()) // BS)
        start = (Y - X) * BS
        assert torch.equal(bt_new[r, :X], bt_old[r, Y - X:Y])
        assert bool((bt_new[r, X:Y] == -1).all())
        freed_ref.append(dp.block_table[r, :Y - X])
        for h in range(H):
            a, b = int(koff[r * H + h]), int(koff[r * H + h + 1])
            kh = b - a
            o = order[a:b].long()
            assert torch.equal(torch.sort(o).values, kept[a:b].long()), f"request {r} head {h}"
            j = torch.arange(kh, device=dev)
            # survivors already inside the region stay put
            ks = kept[a:b].long()
            inside = ks[(ks >= start) & (ks < start + kh)]
            assert torch.equal(o[inside - start], inside)
            src = kv0[:, bt_old[r, o // BS].long(), o % BS, h]
            dst = kv[:, bt_new[r, j // BS].long(), j % BS, h]
            assert torch.equal(src, dst), f"request {r} head {h}"
            moved = o != start + j
            pos = start + j[moved]
            written[bt_old[r, pos // BS].long(), pos % BS, h] = True
        np.testing.assert_array_equal(run_ip["new_lens"][r * H:(r + 1) * H], k[r])
    np.testing.assert_array_equal(run_ip["freed"],
                                  np.concatenate(freed_ref) if freed_ref else np.zeros(0))
    changed = (kv != kv0).any(dim=-1).any(dim=0)   # [page, slot, head]
    assert not bool((changed & ~written).any()), "rows outside the destinations changed"


def test_new_order_matches_the_oracle_on_sampled_requests(run_ip):
    """The oracle's in-place compaction of request r on its own (one request, its pages
    numbered 0 .. Y-1) gives the same slot order, lengths and freed blocks (as positions in
    the request's row) as the whole-batch GPU call."""
    dp = run_ip["dp"]
    H, BS = dp.num_kv_heads, dp.page_size
    _, koff, _ = _offsets(dp)
    kept = run_ip["kept"].cpu().numpy()
    order = run_ip["order"].cpu().numpy()
    freed_off = 0
    starts = {}
    for r in range(dp.num_reqs):   # where request r's freed blocks start in the list
        starts[r] = freed_off
        L = int(dp.seq_lens[r])
        k = np.minimum(dp.budgets[r * H:(r + 1) * H].astype(np.int64), L)
        if not (dp.budgets[r * H:(r + 1) * H] >= L).all():
            freed_off += -(-L // BS) - -(-int(k.max()) // BS)
    for r in [r for r in SAMPLE if r < dp.num_reqs]:
        L = int(dp.seq_lens[r])
        Y = -(-L // BS)
        pb = types.SimpleNamespace(
            seq_lens=np.array([L], np.int32), q_lens=np.array([int(dp.q_lens[r])], np.int32),
            budgets=dp.budgets[r * H:(r + 1) * H].copy(), num_q_heads=dp.num_q_heads,
            num_kv_heads=H, head_dim=dp.head_dim, page_size=BS,
            kv=np.zeros((2, Y, BS, H, dp.head_dim), np.uint16),
            block_table=np.arange(Y, dtype=np.int32)[None, :], sm_scale=dp.sm_scale,
            pool_window=dp.pool_window, causal=dp.causal)
        a, b = int(koff[r * H]), int(koff[(r + 1) * H])
        ref = oracle.compact_inplace(pb, kept[a:b])
        np.testing.assert_array_equal(order[a:b], ref["new_order"],
                                      err_msg=f"{dp.cfg_name} request {r}")
        np.testing.assert_array_equal(run_ip["new_lens"][r * H:(r + 1) * H], ref["new_lens"])
        nf = ref["freed"].size
        got = run_ip["freed"][starts[r]:starts[r] + nf]
        np.testing.assert_array_equal(got, dp.block_table[r, ref["freed"]])
