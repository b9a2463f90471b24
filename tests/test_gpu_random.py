"""Seeded random problems through the whole step, each against the oracle: request counts,
lengths (empty and single-token requests included), query counts, GQA groups, head dims,
pooling windows, budgets (zero, partial, at and past the length), causal and non-causal,
SUM and MAX_MEAN, the LSE supplied or computed by the library.  Scores within 2e-3
relative; pooling and selection exact functions of the GPU scores; compaction bit-exact.
The same problems also go through the in-place compaction (given the oracle's selection),
the LRFU selection and, with one query per request, the decode-step scoring; the confidence
monitor gets random draws of its own."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import assert_compaction_matches, assert_scores_close, to_dev
from paper_2609_31395_amd import actkv
from paper_2609_31395_amd import workloads as W

pytestmark = pytest.mark.gpu


def _random_causal(seed):
    """Whether seed's random problem is causal (its first draws, without the data)."""
    rng = np.random.default_rng(10_000 + seed)
    rng.integers(1, 5), rng.choice([1, 2, 4, 8]), rng.choice([1, 2, 3, 4, 8, 16])
    rng.choice([64, 128])
    return bool(rng.random() < 0.8)


def _random_problem(seed):
    rng = np.random.default_rng(10_000 + seed)
    R = int(rng.integers(1, 5))
    Hkv = int(rng.choice([1, 2, 4, 8]))
    G = int(rng.choice([1, 2, 3, 4, 8, 16]))
    D = int(rng.choice([64, 128]))
    causal = bool(rng.random() < 0.8)
    assert causal == _random_causal(seed)
    L = rng.integers(0, 3000, size=R)
    L[rng.random(R) < 0.15] = 0
    L[rng.random(R) < 0.1] = 1
    if causal:
        n = np.array([int(rng.integers(0, min(l, 80) + 1)) for l in L])
    else:
        n = rng.integers(0, 81, size=R)
    b = rng.integers(0, np.maximum(L, 1)[:, None] + 10, size=(R, Hkv))
    b[rng.random((R, Hkv)) < 0.1] = 0
    window = int(rng.choice([1, 3, 5, 7, 9]))
    agg = "max_mean" if (G in (1, 2, 4, 8, 16) and rng.random() < 0.3) else "sum"
    supplied = bool(rng.random() < 0.5)
    pb = W.make_custom(seq_lens=L, q_lens=n, num_q_heads=G * Hkv, num_kv_heads=Hkv,
                       head_dim=D, budgets=b.reshape(-1), pool_window=window,
                       spike_frac=0.02, seed=seed, causal=causal)
    return pb, agg, supplied


@pytest.mark.parametrize("seed", range(150))
def test_random_problem_step_matches_the_oracle(seed):
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    actkv.load_library()
    pb, agg, supplied = _random_problem(seed)
    lse = oracle.lse(pb).astype(np.float32) if supplied else None
    bp, t = to_dev(pb, agg=agg)
    n_sc = actkv.num_scores(bp)
    qy = actkv.query(bp)
    scores = torch.empty(max(n_sc, 1), dtype=torch.float32, device="cuda")
    pooled = torch.empty_like(scores)
    kept = torch.empty(max(qy["num_kept"], 1), dtype=torch.int32, device="cuda")
    res = actkv.step(bp, t["q"], t["kv"], t["bt"], t["free"],
                     lse=None if lse is None else torch.from_numpy(lse).cuda(),
                     scores=scores, pooled=pooled, kept=kept)
    torch.cuda.synchronize()
    what = (f"seed {seed}: R={pb.num_reqs} L={pb.seq_lens.tolist()} n={pb.q_lens.tolist()} "
            f"Hq/Hkv={pb.num_q_heads}/{pb.num_kv_heads} D={pb.head_dim} w={pb.pool_window} "
            f"{agg} causal={pb.causal} lse={'supplied' if supplied else 'library'}")
    raw_ref = oracle.scores(pb, lse_in=lse, agg=agg)
    got = scores[:n_sc].cpu().numpy()
    assert_scores_close(got, raw_ref, what=what)
    pooled_gpu = pooled[:n_sc].cpu().numpy()
    np.testing.assert_array_equal(pooled_gpu, oracle.pool(pb, got), err_msg=what)
    kept_gpu = res["kept"].cpu().numpy()
    np.testing.assert_array_equal(kept_gpu, oracle.select(pb, pooled_gpu), err_msg=what)
    assert_compaction_matches(pb, kept_gpu, pb.kv, t["kv"].cpu().numpy().view(np.uint16),
                              t["bt"].cpu().numpy(), res["freed"].cpu().numpy(),
                              res["new_lens"].cpu().numpy())


@pytest.mark.parametrize("seed", range(60))
def test_random_problem_inplace_compaction_matches_the_oracle(seed):
    """The in-place compaction (Alg. 4) of the oracle's selection on the same random
    problems: the whole cache, block tables, freed lists, lengths and slot order exact."""
    from test_gpu_inplace import _assert_same, _run_inplace
    pb, agg, _ = _random_problem(seed)
    kept = oracle.select(pb, oracle.pool(pb, oracle.scores(pb, agg=agg)))
    _assert_same(_run_inplace(pb, kept), oracle.compact_inplace(pb, kept))


@pytest.mark.parametrize("seed", [s for s in range(80) if _random_causal(s)][:60])
def test_random_decode_step_matches_the_oracle(seed):
    """One action query per request (the decode-step scoring kernel when G <= 16), added
    twice to an aggregate that starts at zero: twice the oracle's scores.  Decode steps are
    causal, so only the causal random problems run."""
    pb, agg, _ = _random_problem(seed)
    n1 = np.minimum(pb.q_lens, 1).astype(np.int32)
    pb1 = W.make_custom(seq_lens=pb.seq_lens, q_lens=n1, num_q_heads=pb.num_q_heads,
                        num_kv_heads=pb.num_kv_heads, head_dim=pb.head_dim,
                        budgets=pb.budgets, pool_window=pb.pool_window, spike_frac=0.0,
                        seed=seed, causal=True)
    lse = oracle.lse(pb1).astype(np.float32)
    bp, t = to_dev(pb1, agg=agg)
    n_sc = actkv.num_scores(bp)
    acc = torch.zeros(max(n_sc, 1), dtype=torch.float32, device="cuda")
    lse_d = torch.from_numpy(lse).cuda()
    for _ in range(2):
        actkv.score_accumulate(bp, t["q"], t["kv"], t["bt"], acc, lse=lse_d)
    torch.cuda.synchronize()
    ref = 2.0 * oracle.scores(pb1, lse_in=lse, agg=agg)
    assert_scores_close(acc[:n_sc].cpu().numpy(), ref, what=f"decode seed {seed}")


@pytest.mark.parametrize("seed", range(60))
def test_random_problem_lrfu_select_matches_the_oracle(seed):
    """LRFU keep scores (Sec. 5.1) on the oracle's scores of the same random problems, with
    random keep scores, top-p and decay: hit mask outside the boundary band, keep scores,
    selection and the kept keep scores exact."""
    from test_gpu_lrfu import check_stage
    pb, agg, _ = _random_problem(seed)
    rng = np.random.default_rng(20_000 + seed)
    raw = oracle.scores(pb, agg=agg).astype(np.float32)
    ks_in = (rng.random(raw.shape[0]) * rng.choice([1e-3, 0.1, 1.0])).astype(np.float32)
    ks_in[rng.random(raw.shape[0]) < 0.3] = 0.0
    top_p = float(rng.choice([0.0, 0.5, 0.9, 0.97, 1.0]))
    decay = float(rng.choice([0.0, 0.25, 0.5, 1.0]))
    check_stage(pb, raw, ks_in, top_p, decay)


@pytest.mark.parametrize("seed", range(40))
def test_random_token_confidence_matches_the_oracle(seed):
    """Token confidence (Sec. 6.1) over random vocabularies up to 262,144 logits, top-k up to
    64, rows of different scales, ties and masked logits."""
    rng = np.random.default_rng(30_000 + seed)
    rows = int(rng.integers(1, 9))
    vocab = int(rng.choice([1, 2, 63, 64, 65, 1000, 16383, 16384, 16385, 100_000, 151_936,
                            262_144]))
    k = int(rng.integers(1, 65))
    x = (rng.standard_normal((rows, vocab)) * rng.uniform(0.1, 8.0, (rows, 1))).astype(np.float32)
    if rng.random() < 0.3:
        x = np.round(x)                                   # heavy ties
    x[rng.random((rows, vocab)) < rng.choice([0.0, 0.2])] = -np.inf
    x[:, 0] = np.where(np.isinf(x[:, 0]), 0.0, x[:, 0])   # at least one finite logit per row
    got = actkv.token_confidence(torch.from_numpy(x).cuda(), top_k=k).cpu().numpy()
    np.testing.assert_allclose(got, oracle.token_confidence(x, k), rtol=1e-6, atol=1e-5,
                               err_msg=f"seed {seed}: rows={rows} vocab={vocab} k={k}")


@pytest.mark.parametrize("seed", range(40))
def test_random_budget_update_is_bit_exact(seed):
    """The budget rule (Alg. 2) on random traces and parameters: budgets, slopes, thresholds
    and retained counts bit-exact."""
    rng = np.random.default_rng(40_000 + seed)
    R = int(rng.integers(1, 7))
    w = int(rng.choice([1, 2, 8, 24, 64, 128]))
    st = int(rng.choice([1, 3, 8, 16, 64]))
    params = dict(window=w, stride=st, bottom_pct=float(rng.choice([0.0, 5.0, 10.0, 50.0, 100.0])),
                  scale_up=float(rng.choice([1.0, 1.75, 2.5])),
                  budget_upper=int(rng.choice([600, 30000])))
    seqs = []
    for _ in range(R):
        n = int(rng.integers(0, 6000))
        if n >= w:   # stay within the window count one request may have
            n = min(n, w + st * 16383)
        t = (10 + rng.choice([-1.0, 0.0, 1.0]) * np.linspace(0, 1, n)
             + 0.3 * rng.standard_normal(n))
        t[rng.random(n) < 0.1] = 9.5
        seqs.append(np.abs(t).astype(np.float32))
    budgets = rng.integers(100, 30001, size=R).astype(np.int32)
    offsets = np.concatenate([[0], np.cumsum([s.size for s in seqs])]).astype(np.int64)
    flat = torch.from_numpy(np.concatenate(seqs) if seqs else np.zeros(0, np.float32)).cuda()
    got = actkv.budget_update(flat, offsets, torch.from_numpy(budgets).cuda(), **params)
    torch.cuda.synchronize()
    ref = oracle.budget_update(seqs, budgets, **params)
    np.testing.assert_array_equal(got["budgets"].cpu().numpy(), ref["budgets"])
    np.testing.assert_array_equal(got["retained"].cpu().numpy(), ref["retained"])
    np.testing.assert_array_equal(got["slopes"].cpu().numpy().view(np.int64),
                                  ref["slopes"].view(np.int64))
    g_thr, r_thr = got["thresholds"].cpu().numpy(), ref["thresholds"]
    assert np.array_equal(np.isnan(g_thr), np.isnan(r_thr))
    np.testing.assert_array_equal(g_thr[~np.isnan(g_thr)], r_thr[~np.isnan(r_thr)])
