"""The LSE pass (Sec. 7.1: the normaliser the scoring recovers probabilities with) against the
oracle on rows whose running maximum moves in the middle of a 2,048-key block, after the
row's first tile.  The pass sums a tile's terms 2^(alpha x - m) against the running shift m
as it stands and takes the tile's maximum only when that sum would pass 2^64, so:
  * keys whose logit towers far above everything before them (by about 100 in log2 units)
    take the rescaling branch with a finite running shift;
  * keys a few units above the running maximum are summed as terms above 1 against a shift
    below the maximum, and the partial that leaves the block carries that lower shift.
Both must give the oracle's LSE, and the scores computed with the library's LSE the
oracle's scores."""
import numpy as np
import pytest
import torch

import oracle
from gpu_util import assert_scores_close, to_dev
from paper_2609_31395_amd import actkv
from paper_2609_31395_amd import workloads as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    actkv.load_library()


def _problem(seed):
    return W.make_custom(seq_lens=[4500, 2300], q_lens=[3, 2], num_q_heads=8, num_kv_heads=2,
                         head_dim=128, budgets=[1000, 900, 500, 600], pool_window=3,
                         spike_frac=0.0, seed=seed)


def _plant(pb, r, t, h, g, j, scale):
    """K row of token t (request r, KV head h) := scale * the bf16 query row of action query
    j, query head h * G + g: its logit for that row is scale * |q|^2 * sm_scale."""
    G = pb.num_q_heads // pb.num_kv_heads
    qrow = W.bf16_to_f32(pb.q[int(pb.cu_q[r]) + j, h * G + g])
    page = int(pb.block_table[r, t // pb.page_size])
    pb.kv[0, page, t % pb.page_size, h] = W.bf16_bits(scale * qrow)
    return float(np.dot(qrow.astype(np.float64), W.bf16_to_f32(pb.kv[0, page, t % pb.page_size, h])))


# (token, scale) plants: inside block 0 after its first tile, inside block 1, and near the
# end of the request; all keys at or before the first action query's position, so every
# row sees them
TOWERING = [(700, 8.0), (2048 + 900, 9.0), (4100, 10.0)]
RISING = [(300, 0.6), (650, 0.9), (1300, 1.2), (2048 + 200, 1.5), (3000, 1.8)]


@pytest.mark.parametrize("plants", ["towering", "rising"])
def test_lse_when_the_running_max_moves_inside_a_block(plants):
    pb = _problem(31 if plants == "towering" else 32)
    alpha_log2 = float(np.float32(pb.sm_scale)) * 1.4426950408889634
    max_dot = 0.0
    for r in range(pb.num_reqs):
        L = int(pb.seq_lens[r])
        for (tok, scale) in (TOWERING if plants == "towering" else RISING):
            if tok >= L - int(pb.q_lens[r]):
                continue
            for h in range(pb.num_kv_heads):
                dot = _plant(pb, r, tok, h, g=h % 4, j=0, scale=scale)
                max_dot = max(max_dot, abs(dot))
                if plants == "towering":
                    # the planted logit stands far above 64 in log2 units: the rescaling branch
                    assert dot * alpha_log2 > 90
    bp, t = to_dev(pb)
    got = actkv.lse(bp, t["q"], t["kv"], t["bt"]).cpu().numpy()
    ref = oracle.lse(pb)
    # the planted dot products are large and of one sign (k = scale * q): their fp32
    # accumulation over D products may be off by up to D * 2^-24 * sum|q_i k_i|, which the
    # natural-log LSE carries times sm_scale; the plain tolerance covers the rest
    tol = 2e-4 + pb.head_dim * 2.0 ** -24 * max_dot * float(pb.sm_scale)
    np.testing.assert_allclose(got, ref, rtol=0, atol=tol)
    sc = actkv.score(bp, t["q"], t["kv"], t["bt"], lse=None)
    assert_scores_close(sc.cpu().numpy(), oracle.scores(pb))
