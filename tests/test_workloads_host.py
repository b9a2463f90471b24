"""Host checks of the synthetic input generators (no GPU: the device draws run on the CPU
here): the full-model workload's shared page pool and per-layer structure."""
import numpy as np
import torch

from paper_2609_31395_amd import workloads as W


def _small_model(layers=3):
    return W.make_device_model("model48x32", "cpu", num_layers=layers,
                               overrides=dict(num_reqs=5, seq_len=(40, 300), q_len=(4, 4)))


def test_model_layers_partition_one_shared_pool():
    layers = _small_model()
    kv = layers[0].kv
    assert all(l.kv.data_ptr() == kv.data_ptr() for l in layers)
    used = [np.concatenate(l.pages) for l in layers]
    spare = layers[0].free_pages
    assert all(np.array_equal(l.free_pages, spare) for l in layers)
    # every page of the pool belongs to exactly one layer's request or to the spare list,
    # and the spare list holds one layer's worth of pages
    np.testing.assert_array_equal(np.sort(np.concatenate(used + [spare])),
                                  np.arange(layers[0].num_pages))
    assert spare.size == used[0].size


def test_model_layers_share_requests_and_draw_their_own_contents():
    layers = _small_model()
    BS, H = W.PAGE_SIZE, layers[0].num_kv_heads
    for l in layers[1:]:
        np.testing.assert_array_equal(l.seq_lens, layers[0].seq_lens)
        np.testing.assert_array_equal(l.q_lens, layers[0].q_lens)
    assert not np.array_equal(layers[0].budgets, layers[1].budgets)
    assert not torch.equal(layers[0].q, layers[1].q)
    for l in layers:
        L = l.seq_lens.astype(np.int64)
        Y = -(-L // BS)
        for r in range(l.num_reqs):
            np.testing.assert_array_equal(l.block_table[r, :Y[r]], l.pages[r])
            assert (l.block_table[r, Y[r]:] == -1).all()
            # slots past L in the last page hold zeros
            last = l.kv[:, int(l.pages[r][-1])].reshape(2, BS, -1)
            assert not last[:, L[r] - (Y[r] - 1) * BS:].any()
        b = l.budgets.reshape(-1, H).astype(np.int64)
        assert (b >= 0).all() and (b <= L[:, None]).all()
        assert (b.sum(axis=1) <= np.floor(0.25 * H * L) + H).all()


def test_model_draws_are_reproducible():
    a, b = _small_model(2), _small_model(2)
    for x, y in zip(a, b):
        pages = torch.from_numpy(np.concatenate(x.pages).astype(np.int64))
        assert torch.equal(x.kv[:, pages], y.kv[:, pages])   # spare pages are left undrawn
        assert torch.equal(x.q, y.q)
        np.testing.assert_array_equal(x.budgets, y.budgets)
        np.testing.assert_array_equal(x.block_table, y.block_table)
