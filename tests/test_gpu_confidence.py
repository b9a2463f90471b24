"""GPU parity of the confidence monitor and budget rule (actkv_token_confidence,
actkv_budget_update; Sec. 6.1, Alg. 2) against the oracle.

Token confidence: |T_gpu - T_ref| <= 1e-5 + 1e-6 |T_ref|.  The GPU sums exp() in fp32 over
up to 262,144 logits (relative error of the sum within about (log2 n + 2) * 2^-24, i.e.
~1.3e-6, which is an absolute error of the log); the top-k sum is exact in fp64; the
result is rounded to fp32 (2^-24 relative).  Budget update: given the same fp32 token
confidences, budgets, slopes (fp64), thresholds and retained counts are bit-exact -- both
sides evaluate the same fp64 operations in the same order.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_31395_amd import actkv

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    actkv.load_library()


def _logits(rng, rows, vocab):
    x = rng.standard_normal((rows, vocab)).astype(np.float32)
    x *= rng.uniform(0.5, 6.0, size=(rows, 1)).astype(np.float32)
    if rows > 1:
        x[1, rng.integers(0, vocab)] += 35.0               # one near-certain token
    if rows > 2:
        x[2, rng.random(vocab) < 0.3] = -np.inf             # masked vocabulary
    if rows > 3:
        x[3] = np.round(x[3])                               # many exact ties
    return x


@pytest.mark.parametrize("vocab", [1, 100, 16384, 16385, 151936, 262144])
@pytest.mark.parametrize("k", [1, 20, 64])
def test_token_confidence_matches_the_oracle(vocab, k):
    rng = np.random.default_rng(vocab + k)
    x = _logits(rng, 5, vocab)
    got = actkv.token_confidence(torch.from_numpy(x).cuda(), top_k=k).cpu().numpy()
    ref = oracle.token_confidence(x, k)
    np.testing.assert_allclose(got, ref, rtol=1e-6, atol=1e-5)


@pytest.mark.parametrize("k", [1, 20, 64])
def test_token_confidence_on_flat_and_few_valued_rows(k):
    """Rows where thousands of logits tie at the k-th largest value (a flat row, three
    distinct values, a row masked but for a few tokens, zeros of both signs): the exact
    top-k then cannot come from a short candidate list and is found over the whole chunk."""
    V = 151936
    rng = np.random.default_rng(k)
    x = np.empty((5, V), np.float32)
    x[0] = 3.25
    x[1] = rng.integers(0, 3, V).astype(np.float32)
    x[2] = -np.inf
    x[2, rng.choice(V, 5, replace=False)] = rng.standard_normal(5).astype(np.float32)
    x[3] = np.where(rng.random(V) < 0.5, 7.0, rng.standard_normal(V)).astype(np.float32)
    x[4] = np.where(rng.random(V) < 0.5, np.float32(-0.0), np.float32(0.0))   # signed zeros
    x[4, rng.random(V) < 0.3] = -1.0
    got = actkv.token_confidence(torch.from_numpy(x).cuda(), top_k=k).cpu().numpy()
    ref = oracle.token_confidence(x, k)
    np.testing.assert_allclose(got, ref, rtol=1e-6, atol=1e-5)


def test_token_confidence_with_row_stride():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((4, 5000)).astype(np.float32)
    xt = torch.from_numpy(x).cuda()[:, :4321]
    got = actkv.token_confidence(xt, top_k=20).cpu().numpy()
    np.testing.assert_allclose(got, oracle.token_confidence(x[:, :4321], 20), rtol=1e-6,
                               atol=1e-5)


def _seqs(rng):
    out = []
    for n in (0, 10, 63, 64, 65, 200, 1000, 35000, 64 + 8 * 16383):
        trend = rng.choice([-1.0, 0.0, 1.0])
        t = 10 + trend * np.linspace(0, 1, n) + 0.3 * rng.standard_normal(n)
        if n > 500:
            t[rng.random(n) < 0.2] = 9.5   # plateaus: tied windows around the percentile
        out.append(np.abs(t).astype(np.float32))
    return out


@pytest.mark.parametrize("params", [dict(), dict(window=2, stride=1, bottom_pct=50.0),
                                    dict(window=16, stride=16, bottom_pct=0.0),
                                    dict(bottom_pct=100.0, scale_up=1.0, budget_upper=600),
                                    # blocks of gcd(w, s) tokens: 32 and 64 (lane groups
                                    # across rows of 16), 3 and 128 (not lane groups)
                                    dict(window=64, stride=32), dict(window=128, stride=64),
                                    dict(window=24, stride=9, bottom_pct=25.0),
                                    dict(window=256, stride=128, bottom_pct=30.0)])
def test_budget_update_is_bit_exact(params):
    rng = np.random.default_rng(7)
    w, st = params.get("window", 64), params.get("stride", 8)
    # traces within the 16,384-window limit of one request for these parameters
    seqs = [t for t in _seqs(rng) if t.size < w or (t.size - w) // st + 1 <= 16384]
    budgets = np.array([512, 896, 1568, 29000, 30000, 512, 700, 2744, 100], np.int32)[:len(seqs)]
    offsets = np.concatenate([[0], np.cumsum([s.size for s in seqs])]).astype(np.int64)
    flat = torch.from_numpy(np.concatenate(seqs)).cuda()
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


def test_monitor_end_to_end_over_decode_steps():
    """Per decode step one row of logits per request -> token confidence on the GPU; at the
    compression trigger the budgets and slopes from those confidences equal the oracle's."""
    rng = np.random.default_rng(3)
    R, V, steps = 4, 30000, 300
    conf = [[] for _ in range(R)]
    for i in range(steps):
        x = rng.standard_normal((R, V)).astype(np.float32)
        # request 0 grows less certain over time, request 1 more certain
        x[0, 0] += 12.0 * (1 - i / steps)
        x[1, 0] += 12.0 * (i / steps)
        t = actkv.token_confidence(torch.from_numpy(x).cuda(), top_k=20).cpu().numpy()
        np.testing.assert_allclose(t, oracle.token_confidence(x, 20), rtol=1e-6, atol=1e-5)
        for r in range(R):
            conf[r].append(t[r])
    seqs = [np.array(c, np.float32) for c in conf]
    offsets = np.concatenate([[0], np.cumsum([s.size for s in seqs])]).astype(np.int64)
    budgets = np.full(R, 512, np.int32)
    got = actkv.budget_update(torch.from_numpy(np.concatenate(seqs)).cuda(), offsets,
                              torch.from_numpy(budgets).cuda(),
                              offsets_d=torch.from_numpy(offsets).cuda())
    ref = oracle.budget_update(seqs, budgets)
    np.testing.assert_array_equal(got["budgets"].cpu().numpy(), ref["budgets"])
    np.testing.assert_array_equal(got["slopes"].cpu().numpy().view(np.int64),
                                  ref["slopes"].view(np.int64))
