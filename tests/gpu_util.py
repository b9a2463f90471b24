"""Helpers for the GPU parity tests: upload a host workload to the device, run the HIP path
through the C ABI, and compare against the oracle to the stated bars."""
import numpy as np
import torch

import oracle
from paper_2609_31395_amd import actkv

# Scores: |gpu - ref| <= RTOL * |ref| + ATOL.  fp32 accumulation of <= 1024 positive terms
# per key (each exp2 within a few ulp, each logit from an fp32-accumulated bf16 product
# whose error is far below 1e-4 in the exponent) stays well inside 2e-3 relative; the
# absolute floor only absorbs flushed denormals.
RTOL, ATOL = 2e-3, 1e-30


def dev():
    return torch.device("cuda:0")


def to_dev(pb, agg="sum", lse_dtype=np.float32):
    """Device copies of a workloads.Problem plus its binding Problem."""
    d = dev()
    bp = actkv.Problem(seq_lens=pb.seq_lens, q_lens=pb.q_lens, budgets=pb.budgets,
                       num_q_heads=pb.num_q_heads, num_kv_heads=pb.num_kv_heads,
                       head_dim=pb.head_dim, num_pages=pb.num_pages, bt_stride=pb.bt_stride,
                       sm_scale=pb.sm_scale, pool_window=pb.pool_window, causal=pb.causal,
                       agg=agg).to_device(d)
    t = dict(
        q=torch.from_numpy(np.ascontiguousarray(pb.q).view(np.int16)).to(d),
        kv=torch.from_numpy(np.ascontiguousarray(pb.kv).view(np.int16)).to(d),
        bt=torch.from_numpy(np.ascontiguousarray(pb.block_table)).to(d),
        free=torch.from_numpy(np.ascontiguousarray(pb.free_pages)).to(d),
    )
    return bp, t


def assert_scores_close(got, ref, what="scores"):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    err = np.abs(got - ref)
    bound = RTOL * np.abs(ref) + ATOL
    bad = np.nonzero(~(err <= bound))[0]
    assert bad.size == 0, (
        f"{what}: {bad.size}/{got.size} outside {RTOL} rel; first {bad[:5]} "
        f"got {got[bad[:5]]} ref {ref[bad[:5]]}")


def segments(seq_lens, H, flat):
    out, off = {}, 0
    for r, L in enumerate(seq_lens):
        for h in range(H):
            out[(r, h)] = flat[off:off + int(L)]
            off += int(L)
    return out


def kept_segments(seq_lens, budgets, H, flat):
    out, off = {}, 0
    for r, L in enumerate(seq_lens):
        for h in range(H):
            k = int(min(max(int(budgets[r * H + h]), 0), int(L)))
            out[(r, h)] = flat[off:off + k]
            off += k
    assert off == len(flat)
    return out


def assert_kept_matches_outside_near_ties(pb, kept_gpu, pooled_ref):
    """Selection parity with near-ties excluded: let tau be the reference pooled score at
    rank k.  Every entry whose reference score is above tau by more than the score
    tolerance must be kept, every entry below by more must not be, and exactly k are kept
    in ascending order."""
    H = pb.num_kv_heads
    ks = kept_segments(pb.seq_lens, pb.budgets, H, np.asarray(kept_gpu))
    ps = segments(pb.seq_lens, H, np.asarray(pooled_ref))
    for (r, h), idx in ks.items():
        L = int(pb.seq_lens[r])
        k = idx.size
        assert np.all(np.diff(idx) > 0) and (k == 0 or (idx[0] >= 0 and idx[-1] < L))
        if k == 0 or k == L:
            assert k == min(int(pb.budgets[r * H + h]), L)
            if k == L:
                np.testing.assert_array_equal(idx, np.arange(L))
            continue
        v = ps[(r, h)].astype(np.float64)
        tau = np.sort(v)[::-1][k - 1]
        band = RTOL * tau
        sel = np.zeros(L, bool)
        sel[idx] = True
        must = v > tau + band
        must_not = v < tau - band
        assert sel[must].all(), f"(r={r},h={h}) missed {np.nonzero(must & ~sel)[0][:5]}"
        assert not sel[must_not].any(), f"(r={r},h={h}) took {np.nonzero(must_not & sel)[0][:5]}"


def assert_compaction_matches(pb, kept, kv_before, kv_after, bt_after, freed, new_lens):
    """The GPU compaction equals the oracle's compaction of the SAME kept indices: block
    table, freed list and lengths exactly; every defined slot of every fresh page bit for
    bit; nothing else in the pool changed."""
    kv_ref, bt_ref, freed_ref, lens_ref = oracle.compact(pb, np.asarray(kept), kv=kv_before)
    np.testing.assert_array_equal(bt_after, bt_ref)
    np.testing.assert_array_equal(freed, freed_ref)
    np.testing.assert_array_equal(new_lens, lens_ref)
    H, BS = pb.num_kv_heads, pb.page_size
    touched = np.zeros(kv_before.shape[1], bool)
    fresh_off = 0
    for r, L in enumerate(pb.seq_lens):
        b = pb.budgets[r * H:(r + 1) * H]
        if b.min() >= L:
            continue
        X = -(-int(min(b.max(), L)) // BS)
        for p in range(X):
            page = pb.free_pages[fresh_off + p]
            touched[page] = True
            for h in range(H):
                k = int(min(b[h], L))
                s_hi = min(BS, max(0, k - p * BS))
                np.testing.assert_array_equal(kv_after[:, page, :s_hi, h], kv_ref[:, page, :s_hi, h])
        fresh_off += X
    np.testing.assert_array_equal(kv_after[:, ~touched], kv_before[:, ~touched])
