"""GPU parity of the LRFU eviction (actkv_lrfu_select, actkv_step_lrfu) against the oracle.

Both sides get the same float32 top_p and decay (the oracle wrapper rounds them as the entry
point receives them).  The hit mask is compared exactly except where the prefix boundary is
within rounding of the target: the oracle sums the masses in fp64 in sorted order, the GPU
sums exact 64-bit fixed-point masses (each score truncated to a multiple of 2^-S), so an
entry whose preceding mass lies within that truncation and rounding bound of the target may
legitimately fall either way (boundary_band).  Given the GPU's hit mask, the keep-score
update is compared bit for bit, and the selection, the kept keep scores and the compaction
are compared bit for bit as the oracle's functions of the GPU's own keep scores."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import assert_compaction_matches, assert_scores_close, segments, to_dev
from paper_2609_31395_amd import actkv
from paper_2609_31395_amd import workloads as W
from test_gpu_parity import CASES

pytestmark = pytest.mark.gpu

@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    actkv.load_library()


def fixed_point_shift(vmax: float, L: int) -> int:
    """The GPU's fixed-point scale for a segment of L entries whose largest score is vmax:
    masses are floor(v * 2^S) with S = 62 - e - lg, 2^e > vmax (frexp), 2^lg >= L + 1."""
    _, e = np.frexp(np.float32(vmax))
    return 62 - int(e) - int(L + 1).bit_length()


def boundary_band(pb, att, top_p):
    """Entries whose hit decision the arithmetic does not fix.  With T the total mass and
    `before` the mass ahead of an entry in the oracle's order, both sides hit the entry when
    before < p * T (p the float32 top_p).  The GPU's fixed-point sums are short of the exact
    ones by less than one unit 2^-S per entry (at most L units, for `before` and for T), its
    product p * T rounds once in fp64, and the oracle's fp64 sums of L positive terms are
    within L * 2^-53 * T; an entry is in the band when |before - p * T| is within the sum
    of those bounds (twice over, for margin)."""
    p = oracle.as_f32(top_p)
    H = pb.num_kv_heads
    band = np.zeros(att.shape[0], bool)
    off = 0
    for L in pb.seq_lens:
        L = int(L)
        for _ in range(H):
            a = np.where(att[off:off + L] > 0, att[off:off + L], 0).astype(np.float64)
            T = a.sum()
            if T > 0 and 0 < p < 1:
                unit = 2.0 ** -fixed_point_shift(a.max(), L)
                tol = 2 * ((1 + p) * L * unit + p * T * 2.0 ** -52 + 2 * L * 2.0 ** -53 * T)
                order = np.lexsort((np.arange(L), -a))
                before = np.concatenate([[0.0], np.cumsum(a[order])[:-1]])
                near = np.abs(before - p * T) <= tol
                band[off + order[near]] = True
            off += L
    return band


def check_stage(pb, raw, ks_in, top_p, decay):
    bp, t = to_dev(pb)
    n = raw.shape[0]
    ks = torch.from_numpy(ks_in.copy()).cuda()
    pooled = torch.empty(n, dtype=torch.float32, device="cuda")
    hit = torch.empty(n, dtype=torch.uint8, device="cuda")
    out = actkv.lrfu_select(bp, torch.from_numpy(raw).cuda(), ks, top_p, decay, pooled=pooled,
                            hit=hit)
    torch.cuda.synchronize()
    pooled_ref = oracle.pool(pb, raw)
    np.testing.assert_array_equal(pooled.cpu().numpy(), pooled_ref)
    hit_gpu = hit.cpu().numpy()
    hit_ref = oracle.hits(pb, pooled_ref, top_p)
    band = boundary_band(pb, pooled_ref, top_p)
    bad = np.nonzero((hit_gpu != hit_ref) & ~band)[0]
    assert bad.size == 0, f"hit mask differs off the boundary at {bad[:8]}"
    ks_gpu = ks.cpu().numpy()
    np.testing.assert_array_equal(ks_gpu, oracle.lrfu_update(pb, pooled_ref, hit_gpu, decay,
                                                             ks_in))
    kept_gpu = out["kept"].cpu().numpy()
    np.testing.assert_array_equal(kept_gpu, oracle.select(pb, ks_gpu))
    # the keep scores that travel with the kept entries
    segs = segments(pb.seq_lens, pb.num_kv_heads, ks_gpu)
    want, off = [], 0
    for r, L in enumerate(pb.seq_lens):
        for h in range(pb.num_kv_heads):
            k = int(min(max(int(pb.budgets[r * pb.num_kv_heads + h]), 0), int(L)))
            want.append(segs[(r, h)][kept_gpu[off:off + k]])
            off += k
    np.testing.assert_array_equal(out["ks_kept"].cpu().numpy(),
                                  np.concatenate(want) if want else np.zeros(0, np.float32))
    return hit_gpu, band


@pytest.mark.parametrize("top_p,decay", [(0.9, 0.5), (0.5, 0.0), (0.97, 1.0), (1.0, 0.5),
                                         (0.0, 0.5)])
@pytest.mark.parametrize("case", sorted(CASES))
def test_lrfu_select_on_the_oracle_scores(case, top_p, decay):
    pb = CASES[case]()
    raw = oracle.scores(pb, lse_in=oracle.lse(pb).astype(np.float32))
    rng = np.random.default_rng(4)
    ks_in = (rng.random(raw.shape[0]) * raw.max(initial=1.0)).astype(np.float32)
    ks_in[rng.random(raw.shape[0]) < 0.3] = 0.0   # entries new since the last step
    check_stage(pb, raw, ks_in, top_p, decay)


def test_lrfu_select_with_ties_and_plateaus():
    pb = W.make_custom(seq_lens=[5000, 777], q_lens=[1, 1], num_q_heads=1, num_kv_heads=1,
                       head_dim=64, budgets=[1234, 300], pool_window=9)
    rng = np.random.default_rng(8)
    raw = (rng.integers(0, 40, size=oracle.num_scores(pb)) / 64).astype(np.float32)
    ks_in = (rng.integers(0, 8, size=raw.shape[0]) / 16).astype(np.float32)
    hit, band = check_stage(pb, raw, ks_in, 0.9, 0.5)
    assert hit.any() and not hit.all()


def test_lrfu_hit_boundary_at_the_float32_top_p():
    """Two scores a0 = fl32(0.9), a1 = 1 - a0 (total exactly 1, every mass exact in the GPU's
    fixed point): with the float32 top_p = a0 the first entry alone reaches the target, so
    only it is hit, on the GPU as in the oracle (the band would excuse this entry, so the
    mask is asserted directly)."""
    pb = W.make_custom(seq_lens=[2], q_lens=[1], num_q_heads=1, num_kv_heads=1, head_dim=64,
                       budgets=[1], pool_window=1)
    a0 = np.float32(0.9)
    raw = np.array([a0, np.float32(1.0 - float(a0))], np.float32)
    bp, _ = to_dev(pb)
    hit = torch.empty(2, dtype=torch.uint8, device="cuda")
    ks = torch.zeros(2, dtype=torch.float32, device="cuda")
    actkv.lrfu_select(bp, torch.from_numpy(raw).cuda(), ks, 0.9, 0.5, hit=hit)
    torch.cuda.synchronize()
    assert hit.cpu().numpy().tolist() == oracle.hits(pb, raw, 0.9).tolist() == [1, 0]
    assert ks.cpu().numpy().tolist() == [float(a0), 0.0]


def test_lrfu_select_long_segment_at_the_limit():
    pb = W.make_custom(seq_lens=[38400], q_lens=[1], num_q_heads=1, num_kv_heads=1,
                       head_dim=64, budgets=[9600], pool_window=7)
    rng = np.random.default_rng(12)
    raw = rng.lognormal(-10, 2.0, size=38400).astype(np.float32)
    ks_in = (rng.lognormal(-10, 2.0, size=38400) * (rng.random(38400) < 0.7)).astype(np.float32)
    check_stage(pb, raw, ks_in, 0.9, 0.5)


@pytest.mark.parametrize("top_p,decay", [(0.9, 0.5), (1.0, 0.25), (0.0, 0.5)])
def test_lrfu_select_segments_past_the_lds(top_p, decay):
    """Segments of 38,401-64,512 entries (register-resident keys, a kernel of their own)
    beside one that fits in LDS: budgets past 38,400 kept entries, one keeping everything,
    one keeping nothing, windows of 7."""
    L = [38401, 64512, 50000, 1000, 40000]
    pb = W.make_custom(seq_lens=L, q_lens=[1] * 5, num_q_heads=1, num_kv_heads=1, head_dim=64,
                       budgets=[9600, 50000, 0, 300, 40000], pool_window=7)
    rng = np.random.default_rng(13)
    n = sum(L)
    raw = rng.lognormal(-10, 2.0, size=n).astype(np.float32)
    raw[rng.random(n) < 0.05] = 0.0
    ks_in = (rng.lognormal(-10, 2.0, size=n) * (rng.random(n) < 0.7)).astype(np.float32)
    check_stage(pb, raw, ks_in, top_p, decay)


@pytest.mark.parametrize("case", ["tiny_config", "ragged_g4_d128", "two_row_chunks_g8",
                                  "short_and_empty"])
def test_step_lrfu_end_to_end(case):
    pb = CASES[case]()
    top_p, decay = 0.9, 0.5
    lse = oracle.lse(pb).astype(np.float32)
    rng = np.random.default_rng(6)
    n = oracle.num_scores(pb)
    ks_in = (rng.random(n) * 0.5).astype(np.float32)
    bp, t = to_dev(pb)
    qy = actkv.query(bp)
    ks = torch.from_numpy(ks_in.copy()).cuda()
    scores = torch.empty(max(n, 1), dtype=torch.float32, device="cuda")
    pooled = torch.empty_like(scores)
    hit = torch.empty(max(n, 1), dtype=torch.uint8, device="cuda")
    kept = torch.empty(max(qy["num_kept"], 1), dtype=torch.int32, device="cuda")
    res = actkv.step_lrfu(bp, t["q"], t["kv"], t["bt"], t["free"], ks, top_p, decay,
                          lse=torch.from_numpy(lse).cuda(), scores=scores, pooled=pooled,
                          hit=hit, kept=kept, qy=qy)
    torch.cuda.synchronize()
    ref = oracle.lrfu_step(pb, ks_in, top_p, decay, lse_in=lse)
    assert_scores_close(scores[:n].cpu().numpy(), ref["raw"])
    pooled_gpu = pooled[:n].cpu().numpy()
    np.testing.assert_array_equal(pooled_gpu, oracle.pool(pb, scores[:n].cpu().numpy()))
    hit_gpu = hit[:n].cpu().numpy()
    band = boundary_band(pb, pooled_gpu, top_p)
    assert not ((hit_gpu != oracle.hits(pb, pooled_gpu, top_p)) & ~band).any()
    ks_gpu = ks.cpu().numpy()
    np.testing.assert_array_equal(ks_gpu, oracle.lrfu_update(pb, pooled_gpu, hit_gpu, decay,
                                                             ks_in))
    kept_gpu = res["kept"].cpu().numpy()
    np.testing.assert_array_equal(kept_gpu, oracle.select(pb, ks_gpu))
    assert_compaction_matches(pb, kept_gpu, pb.kv, t["kv"].cpu().numpy().view(np.uint16),
                              t["bt"].cpu().numpy(), res["freed"].cpu().numpy(),
                              res["new_lens"].cpu().numpy())
