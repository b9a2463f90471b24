"""Host checks of the Python binding's argument validation (no GPU needed): every tensor
argument is checked for element type, contiguity and size against the problem before its
pointer reaches the C ABI, and only then for residence on the GPU.  Each case below breaks
one argument of an otherwise valid call and must raise; the valid call made of host tensors
fails only at the device check."""
import numpy as np
import pytest
import torch

from paper_2609_31395_amd import actkv

R, HQ, HKV, D, PAGES, STRIDE = 2, 4, 2, 64, 16, 3


def problem():
    p = actkv.Problem(seq_lens=[40, 17], q_lens=[4, 2], budgets=[8, 8, 8, 8], num_q_heads=HQ,
                      num_kv_heads=HKV, head_dim=D, num_pages=PAGES, bt_stride=STRIDE,
                      pool_window=3)
    # host tensors in place of the device mirrors: the device check comes last
    p.seq_lens_d = torch.from_numpy(p.seq_lens.copy())
    p.q_lens_d = torch.from_numpy(p.q_lens.copy())
    p.budgets_d = torch.from_numpy(p.budgets.copy())
    return p


def args():
    """Host tensors of the right types and sizes for every entry point."""
    p = problem()
    qy = actkv.query(p)
    n_sc = actkv.num_scores(p)
    nk = qy["num_kept"]
    return p, dict(
        q=torch.zeros((6, HQ, D), dtype=torch.bfloat16),
        kv=torch.zeros((2, PAGES, 16, HKV, D), dtype=torch.int16),
        bt=torch.zeros((R, STRIDE), dtype=torch.int32),
        lse=torch.zeros((6, HQ), dtype=torch.float32),
        free=torch.arange(8, dtype=torch.int32),
        scores=torch.zeros(n_sc, dtype=torch.float32),
        pooled=torch.zeros(n_sc, dtype=torch.float32),
        ks=torch.zeros(n_sc, dtype=torch.float32),
        hit=torch.zeros(n_sc, dtype=torch.uint8),
        kept=torch.zeros(nk, dtype=torch.int32),
        ks_kept=torch.zeros(nk, dtype=torch.float32),
        freed=torch.zeros(qy["pages_freed"], dtype=torch.int32),
        lens=torch.zeros(R * HKV, dtype=torch.int32),
        order=torch.zeros(nk, dtype=torch.int32),
        ws=torch.zeros(qy["workspace_bytes"], dtype=torch.uint8))


def call(entry, p, a):
    if entry == "lse":
        return actkv.lse(p, a["q"], a["kv"], a["bt"], out=a["lse"], ws=a["ws"])
    if entry == "score":
        return actkv.score(p, a["q"], a["kv"], a["bt"], lse=a["lse"], out=a["scores"], ws=a["ws"])
    if entry == "score_accumulate":
        return actkv.score_accumulate(p, a["q"], a["kv"], a["bt"], a["scores"], lse=a["lse"],
                                      ws=a["ws"])
    if entry == "select":
        return actkv.select(p, a["scores"], pooled=a["pooled"], kept=a["kept"], ws=a["ws"])
    if entry == "compact":
        return actkv.compact(p, a["kv"], a["bt"], a["kept"], a["free"], freed=a["freed"],
                             new_lens=a["lens"], ws=a["ws"])
    if entry == "step":
        return actkv.step(p, a["q"], a["kv"], a["bt"], a["free"], lse=a["lse"],
                          scores=a["scores"], pooled=a["pooled"], kept=a["kept"],
                          freed=a["freed"], new_lens=a["lens"], ws=a["ws"])
    if entry == "lrfu_select":
        return actkv.lrfu_select(p, a["scores"], a["ks"], 0.9, 0.5, pooled=a["pooled"],
                                 hit=a["hit"], kept=a["kept"], ks_kept=a["ks_kept"], ws=a["ws"])
    if entry == "step_lrfu":
        return actkv.step_lrfu(p, a["q"], a["kv"], a["bt"], a["free"], a["ks"], 0.9, 0.5,
                               lse=a["lse"], scores=a["scores"], pooled=a["pooled"],
                               hit=a["hit"], kept=a["kept"], ks_kept=a["ks_kept"],
                               freed=a["freed"], new_lens=a["lens"], ws=a["ws"])
    if entry == "compact_inplace":
        return actkv.compact_inplace(p, a["kv"], a["bt"], a["kept"], freed=a["freed"],
                                     new_lens=a["lens"], new_order=a["order"], ws=a["ws"])
    if entry == "step_inplace":
        return actkv.step_inplace(p, a["q"], a["kv"], a["bt"], lse=a["lse"],
                                  scores=a["scores"], pooled=a["pooled"], kept=a["kept"],
                                  freed=a["freed"], new_lens=a["lens"], new_order=a["order"],
                                  ws=a["ws"])
    raise AssertionError(entry)


# the arguments each entry point takes (by the keys of args())
USES = {
    "lse": ["q", "kv", "bt", "lse", "ws"],
    "score": ["q", "kv", "bt", "lse", "scores", "ws"],
    "score_accumulate": ["q", "kv", "bt", "lse", "scores", "ws"],
    "select": ["scores", "pooled", "kept", "ws"],
    "compact": ["kv", "bt", "kept", "free", "freed", "lens", "ws"],
    "step": ["q", "kv", "bt", "lse", "free", "scores", "pooled", "kept", "freed", "lens", "ws"],
    "lrfu_select": ["scores", "ks", "pooled", "hit", "kept", "ks_kept", "ws"],
    "step_lrfu": ["q", "kv", "bt", "lse", "free", "ks", "scores", "pooled", "hit", "kept",
                  "ks_kept", "freed", "lens", "ws"],
    "compact_inplace": ["kv", "bt", "kept", "freed", "lens", "order", "ws"],
    "step_inplace": ["q", "kv", "bt", "lse", "scores", "pooled", "kept", "freed", "lens",
                     "order", "ws"],
}


def wrong_dtype(t):
    # int64 page ids / indices are the easy mistake (torch.from_numpy of an int64 array)
    return t.to(torch.int64) if t.dtype != torch.int64 else t.to(torch.int32)


def undersized(t):
    return t.reshape(-1)[:-1]


def strided(t):
    flat = t.reshape(-1)
    return torch.stack([flat, flat], dim=1)[:, 0]   # same values, stride 2


CASES = [(e, k, how) for e, ks in USES.items() for k in ks
         for how in ("dtype", "size", "layout")
         if not (k == "ws" and how == "dtype")          # any element type carries bytes
         and not (k in ("free",) and how == "size")]    # a longer free list than needed is fine


@pytest.mark.parametrize("entry,key,how", CASES)
def test_each_bad_argument_raises_before_the_call(entry, key, how):
    p, a = args()
    if entry.endswith("inplace"):   # the in-place form frees Y - X pages per request
        a["freed"] = a["freed"][:actkv.query_inplace(p)]
    t = a[key]
    a[key] = {"dtype": wrong_dtype, "size": undersized, "layout": strided}[how](t)
    with pytest.raises((TypeError, ValueError)) as ei:
        call(entry, p, a)
    assert "must be on the GPU" not in str(ei.value), (entry, key, how, str(ei.value))


@pytest.mark.parametrize("entry", sorted(USES))
def test_valid_host_tensors_fail_only_the_device_check(entry):
    p, a = args()
    if entry.endswith("inplace"):
        a["freed"] = a["freed"][:actkv.query_inplace(p)]
    with pytest.raises(ValueError, match="must be on the GPU"):
        call(entry, p, a)


def test_a_free_list_shorter_than_the_fresh_pages_raises():
    p, a = args()
    a["free"] = a["free"][:actkv.query(p)["fresh_pages_needed"] - 1]
    with pytest.raises(ValueError, match="free_pages"):
        call("step", p, a)


def test_device_mirrors_are_checked():
    p, a = args()
    p.budgets_d = p.budgets_d.to(torch.int64)
    with pytest.raises(TypeError, match="budgets_d"):
        call("select", p, a)
    p, a = args()
    p.seq_lens_d = None
    with pytest.raises(ValueError, match="seq_lens_d"):
        call("select", p, a)


def test_token_confidence_and_budget_update_check_their_arguments():
    with pytest.raises(ValueError):
        actkv.token_confidence(torch.zeros((4, 100), dtype=torch.float64))
    with pytest.raises(ValueError):
        actkv.token_confidence(torch.zeros((4, 100), dtype=torch.float32))   # host memory
    off = np.array([0, 10, 30], np.int64)
    with pytest.raises(ValueError):
        actkv.budget_update(torch.zeros(29, dtype=torch.float32), off,
                            torch.zeros(2, dtype=torch.int32))   # one confidence short
    with pytest.raises(TypeError):
        actkv.budget_update(torch.zeros(30, dtype=torch.float32), off,
                            torch.zeros(2, dtype=torch.int64))
    with pytest.raises(ValueError, match="must be on the GPU"):
        actkv.budget_update(torch.zeros(30, dtype=torch.float32), off,
                            torch.zeros(2, dtype=torch.int32))
