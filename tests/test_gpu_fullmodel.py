"""Full-model compression step: the 48 layers of a Qwen3-30B-shaped model, 32 requests of
16K-64K tokens each, compressed back to back on one GPU over ONE page pool shared by all
layers (about 138 GB of bf16 K/V; byte offsets past 2^36, page ids past 4 million), with
per-layer Dirichlet(0.5) budgets.  Each layer draws its fresh pages from the pages the
previous layer freed, as a serving system returns them to the pool.

Per layer, right after its step (the next layer overwrites the pages it freed):
  * compaction bit for bit on the device: every kept K and V row of every head at its fresh
    slot, the block table, the freed list, new lengths, and fresh pages taken in order
    from the free list the layer was given;
  * kept indices ascending and in range;
  * SUM-mode segment sums equal G * n (every softmax row sums to one).
On three layers, the longest and the shortest request against the oracle (fp64 scores and
LSE; selection outside near-ties), and pooling and selection over the whole layer as the
oracle's functions of the GPU scores.
"""
import time
import types

import numpy as np
import pytest
import torch

import oracle
from gpu_util import assert_kept_matches_outside_near_ties, assert_scores_close
from paper_2609_31395_amd import actkv
from paper_2609_31395_amd import workloads as W

pytestmark = pytest.mark.gpu

SAMPLE_LAYERS = (0, 23, 47)


def _binding(dp, dev):
    return actkv.Problem(seq_lens=dp.seq_lens, q_lens=dp.q_lens, budgets=dp.budgets,
                         num_q_heads=dp.num_q_heads, num_kv_heads=dp.num_kv_heads,
                         head_dim=dp.head_dim, num_pages=dp.num_pages, bt_stride=dp.bt_stride,
                         sm_scale=dp.sm_scale, pool_window=dp.pool_window,
                         causal=dp.causal).to_device(dev)


def _kept_counts(dp):
    H = dp.num_kv_heads
    L = dp.seq_lens.astype(np.int64)
    k = np.minimum(dp.budgets.reshape(-1, H).astype(np.int64), L[:, None])
    return k, np.concatenate([[0], np.cumsum(k.reshape(-1))])


def _layer_errors(dp, bt_new, kept, freed, new_lens, free_given, scores):
    """Everything checkable about one layer's step while its old pages are intact."""
    errs = []
    dev = dp.kv.device
    R, H, BS = dp.num_reqs, dp.num_kv_heads, dp.page_size
    G = dp.num_q_heads // H
    k, koff = _kept_counts(dp)
    bt_old = dp.block_table
    if kept.size != koff[-1]:
        return [f"{kept.size} kept entries, expected {koff[-1]}"]
    # kept indices: ascending and in range in every segment
    for r in range(R):
        for h in range(H):
            idx = kept[koff[r * H + h]:koff[r * H + h + 1]]
            if idx.size and not (np.all(np.diff(idx) > 0) and idx[0] >= 0
                                 and idx[-1] < dp.seq_lens[r]):
                errs.append(f"request {r} head {h}: kept indices not ascending in range")
    # segment sums
    seg = np.concatenate([[0], np.cumsum(np.repeat(dp.seq_lens.astype(np.int64), H))])
    sums = np.add.reduceat(scores.astype(np.float64), seg[:-1])
    want = np.repeat(G * dp.q_lens.astype(np.float64), H)
    bad = np.nonzero(np.abs(sums - want) > 1e-4 * want)[0]
    if bad.size:
        errs.append(f"segment sums off G*n at segments {bad[:5]}: {sums[bad[:5]]}")
    # block table, freed list, lengths; gather lists for the row check
    freed_ref, fresh_off = [], 0
    sp, ss, dpg, ds, hh = [], [], [], [], []
    for r in range(R):
        L = int(dp.seq_lens[r])
        Y = -(-L // BS)
        if (dp.budgets[r * H:(r + 1) * H] >= L).all():
            if not np.array_equal(bt_new[r], bt_old[r]):
                errs.append(f"request {r}: untouched request's block table changed")
            if not np.array_equal(new_lens[r * H:(r + 1) * H], np.full(H, L)):
                errs.append(f"request {r}: untouched request's lengths changed")
            continue
        X = -(-int(k[r].max()) // BS)
        if not np.array_equal(bt_new[r, :X], free_given[fresh_off:fresh_off + X]):
            errs.append(f"request {r}: fresh pages not taken in order from the free list")
        if not (bt_new[r, X:Y] == -1).all():
            errs.append(f"request {r}: block table not cleared past the fresh pages")
        if not np.array_equal(new_lens[r * H:(r + 1) * H], k[r]):
            errs.append(f"request {r}: new lengths {new_lens[r * H:(r + 1) * H]} != {k[r]}")
        freed_ref.append(bt_old[r, :Y])
        fresh_off += X
        for h in range(H):
            idx = kept[koff[r * H + h]:koff[r * H + h + 1]].astype(np.int64)
            j = np.arange(idx.size)
            sp.append(bt_old[r, idx // BS])
            ss.append(idx % BS)
            dpg.append(bt_new[r, j // BS])
            ds.append(j % BS)
            hh.append(np.full(idx.size, h))
    if not np.array_equal(freed, np.concatenate(freed_ref) if freed_ref else freed[:0]):
        errs.append("freed pages differ from the old block-table rows")
    if errs:
        return errs
    ix = [torch.from_numpy(np.concatenate(a).astype(np.int64)).to(dev)
          for a in (sp, ss, dpg, ds, hh)]
    for which, name in ((0, "K"), (1, "V")):
        plane = dp.kv[which]
        a = plane[ix[0], ix[1], ix[4]]
        b = plane[ix[2], ix[3], ix[4]]
        if not torch.equal(a, b):
            n_bad = int((a != b).any(dim=1).sum())
            errs.append(f"{name} rows: {n_bad} of {a.shape[0]} differ at their fresh slots")
        del a, b
    return errs


@pytest.fixture(scope="module")
def model():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    actkv.load_library()
    torch.cuda.empty_cache()
    dev = torch.device("cuda:0")
    t0 = time.time()
    layers = W.make_device_model("model48x32", device=dev)
    torch.cuda.synchronize()
    print(f"\nmodel48x32: {len(layers)} layers, {layers[0].num_pages} pool pages drawn in "
          f"{time.time() - t0:.1f} s", flush=True)
    L = layers[0].seq_lens
    reqs = sorted({int(np.argmax(L)), int(np.argmin(L))})
    free = torch.from_numpy(layers[0].free_pages).to(dev)
    per_layer, samples = [], {}
    for l, dp in enumerate(layers):
        bp = _binding(dp, dev)
        qy = actkv.query(bp)
        ws = torch.empty(qy["workspace_bytes"], dtype=torch.uint8, device=dev)
        bt = torch.from_numpy(dp.block_table).to(dev)
        lse = torch.empty(int(dp.q_lens.sum()) * dp.num_q_heads, dtype=torch.float32,
                          device=dev)
        actkv.lse(bp, dp.q, dp.kv, bt, out=lse, ws=ws)
        scores = torch.empty(actkv.num_scores(bp), dtype=torch.float32, device=dev)
        pooled = torch.empty_like(scores)
        kept = torch.empty(qy["num_kept"], dtype=torch.int32, device=dev)
        free_given = free.cpu().numpy()
        res = actkv.step(bp, dp.q, dp.kv, bt, free, lse=lse, scores=scores, pooled=pooled,
                         kept=kept, ws=ws, qy=qy)
        torch.cuda.synchronize()
        sc = scores.cpu().numpy()
        kp = kept.cpu().numpy()
        freed = res["freed"]
        errs = _layer_errors(dp, bt.cpu().numpy(), kp, freed.cpu().numpy(),
                             res["new_lens"].cpu().numpy(), free_given, sc)
        per_layer.append(errs)
        if l in SAMPLE_LAYERS:
            samples[l] = dict(dp=dp, scores=sc, pooled=pooled.cpu().numpy(), kept=kp,
                              lse=lse.cpu().numpy(), host={r: dp.host_subset([r]) for r in reqs})
        print(f"layer {l}: {len(errs)} problems ({time.time() - t0:.1f} s)", flush=True)
        # the next layer's fresh pages are the pages this layer returned
        free = freed
        del ws, bt, lse, scores, pooled, kept
    out = dict(per_layer=per_layer, samples=samples, reqs=reqs,
               pool_bytes=dp.kv.numel() * dp.kv.element_size())
    del layers, dp, free, freed, res
    yield out
    out.clear()
    torch.cuda.empty_cache()


def test_the_pool_needs_64_bit_offsets(model):
    assert model["pool_bytes"] > 2 ** 36


def test_every_layer_compacts_bit_exact_with_chained_free_lists(model):
    bad = {l: e for l, e in enumerate(model["per_layer"]) if e}
    assert not bad, bad


@pytest.mark.parametrize("layer", SAMPLE_LAYERS)
def test_sampled_requests_match_the_oracle(model, layer):
    s = model["samples"][layer]
    dp = s["dp"]
    H, Hq = dp.num_kv_heads, dp.num_q_heads
    seg = np.concatenate([[0], np.cumsum(dp.seq_lens.astype(np.int64) * H)])
    _, koff = _kept_counts(dp)
    cu = dp.cu_q
    for r, host in s["host"].items():
        ref = oracle.step(host)
        assert_scores_close(s["scores"][seg[r]:seg[r + 1]], ref["raw"],
                            what=f"layer {layer} request {r} scores")
        lse_gpu = s["lse"].reshape(-1, Hq)[int(cu[r]):int(cu[r + 1])]
        np.testing.assert_allclose(lse_gpu, oracle.lse(host), rtol=0, atol=2e-3)
        assert_kept_matches_outside_near_ties(host, s["kept"][koff[r * H]:koff[(r + 1) * H]],
                                              ref["pooled"])


@pytest.mark.parametrize("layer", SAMPLE_LAYERS)
def test_pool_and_select_are_the_oracle_functions_of_the_gpu_scores(model, layer):
    s = model["samples"][layer]
    dp = s["dp"]
    pb = types.SimpleNamespace(
        seq_lens=dp.seq_lens, q_lens=dp.q_lens, budgets=dp.budgets,
        num_q_heads=dp.num_q_heads, num_kv_heads=dp.num_kv_heads, head_dim=dp.head_dim,
        page_size=dp.page_size, kv=np.empty((2, dp.num_pages, 0), np.uint16),
        block_table=dp.block_table, sm_scale=dp.sm_scale, pool_window=dp.pool_window,
        causal=dp.causal)
    np.testing.assert_array_equal(s["pooled"], oracle.pool(pb, s["scores"]))
    np.testing.assert_array_equal(s["kept"], oracle.select(pb, s["pooled"]))
