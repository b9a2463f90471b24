"""Host-side checks of libactkv that need no GPU: the shared library loads and exports every
symbol the header declares, the host planning agrees with the oracle's page accounting,
and every argument error is reported before anything is enqueued."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
from paper_2609_31395_amd import actkv
from paper_2609_31395_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "actkv.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(actkv_[a-z_]+)\s*\(", text)))


def test_header_declares_the_documented_entry_points():
    names = declared_functions()
    for n in ("actkv_query", "actkv_lse", "actkv_score", "actkv_select", "actkv_compact",
              "actkv_step", "actkv_status_str"):
        assert n in names


def test_library_loads_and_exports_every_declared_symbol():
    lib = actkv.load_library()
    for name in declared_functions():
        assert hasattr(lib, name), name
    assert actkv.status_str(0) == "ok"
    assert "workspace" in actkv.status_str(-3)


def binding_problem(pb, **kw):
    return actkv.Problem(seq_lens=pb.seq_lens, q_lens=pb.q_lens, budgets=pb.budgets,
                         num_q_heads=pb.num_q_heads, num_kv_heads=pb.num_kv_heads,
                         head_dim=pb.head_dim, num_pages=pb.num_pages, bt_stride=pb.bt_stride,
                         sm_scale=pb.sm_scale, pool_window=pb.pool_window, causal=pb.causal,
                         **kw)


@pytest.mark.parametrize("seed", range(5))
def test_query_page_accounting_matches_oracle(seed):
    rng = np.random.default_rng(seed)
    R, H = int(rng.integers(1, 6)), 2
    L = rng.integers(0, 300, size=R)
    budgets = rng.integers(0, 320, size=R * H)
    if seed == 0:
        budgets[:H] = L[0] + 5   # one untouched request
    pb = W.make_custom(seq_lens=L, q_lens=np.minimum(L, 3), num_q_heads=4, num_kv_heads=H,
                       head_dim=64, budgets=budgets, seed=seed)
    q = actkv.query(binding_problem(pb))
    nk, fresh, freed = oracle.totals(pb)
    assert (q["num_kept"], q["fresh_pages_needed"], q["pages_freed"]) == (nk, fresh, freed)
    assert q["workspace_bytes"] > 0


def _tiny(**over):
    kw = dict(seq_lens=[40, 17], q_lens=[4, 2], budgets=[8, 8, 8, 8], num_q_heads=4,
              num_kv_heads=2, head_dim=128, num_pages=64, bt_stride=3, pool_window=3)
    kw.update(over)
    return actkv.Problem(**kw)


BAD = [
    (dict(pool_window=4), -1),
    (dict(pool_window=65), -1),
    (dict(pool_window=0), -1),
    (dict(q_lens=[41, 2]), -1),                      # causal query beyond the cache
    (dict(num_q_heads=3), -1),                       # Hq not a multiple of Hkv
    (dict(budgets=[8, -1, 8, 8]), -1),
    (dict(bt_stride=2), -1),                         # row too short for 40 tokens
    (dict(seq_lens=[-1, 17]), -1),
    (dict(num_pages=0), -1),
    (dict(sm_scale=-1.0), -1),
    (dict(sm_scale=float("nan")), -1),
    (dict(head_dim=96), -2),
    (dict(page_size=32), -2),
    (dict(agg="max_mean", num_q_heads=6, num_kv_heads=2), -2),   # G = 3
]


@pytest.mark.parametrize("over,code", BAD)
def test_invalid_problems_are_rejected_on_the_host(over, code):
    with pytest.raises(actkv.ActKVError) as e:
        actkv.query(_tiny(**over))
    assert e.value.code == code


def test_non_causal_queries_may_outnumber_the_cache():
    actkv.query(_tiny(q_lens=[41, 2], causal=False))


FAKE = 0x10000   # never dereferenced: every call below must fail before any launch


def _call_step(p, ws_bytes, num_free=1000, with_mirrors=True):
    lib = actkv.load_library()
    if with_mirrors:
        c = p.cstruct()
        c.seq_lens_d = c.q_lens_d = c.budgets_d = FAKE
    else:
        c = p.cstruct()
    return lib.actkv_step(ctypes.byref(c), FAKE, FAKE, FAKE, None, FAKE, num_free, None, None,
                          None, FAKE, FAKE, FAKE, ws_bytes, None)


def test_step_reports_small_workspace_before_launching():
    p = _tiny()
    need = actkv.query(p)["workspace_bytes"]
    assert _call_step(p, need - 1) == -3


def test_step_reports_short_free_list_before_launching():
    p = _tiny()
    q = actkv.query(p)
    assert q["fresh_pages_needed"] > 0
    assert _call_step(p, q["workspace_bytes"], num_free=q["fresh_pages_needed"] - 1) == -4


def test_step_requires_device_mirrors():
    p = _tiny()
    assert _call_step(p, actkv.query(p)["workspace_bytes"], with_mirrors=False) == -1


def test_compact_and_select_validate_before_launching():
    lib = actkv.load_library()
    p = _tiny()
    c = p.cstruct()
    c.seq_lens_d = c.q_lens_d = c.budgets_d = FAKE
    ws = actkv.query(p)["workspace_bytes"]
    assert lib.actkv_compact(ctypes.byref(c), FAKE, FAKE, FAKE, FAKE, 0, FAKE, FAKE, FAKE, ws,
                             None) == -4
    assert lib.actkv_select(ctypes.byref(c), FAKE, FAKE, None, FAKE, ws, None) == -1
    assert lib.actkv_score(ctypes.byref(c), FAKE, FAKE, FAKE, None, FAKE, FAKE, 16, None) == -3
    assert lib.actkv_lse(None, FAKE, FAKE, FAKE, FAKE, FAKE, ws, None) == -1


def test_select_compact_validates_before_launching():
    """actkv_select_compact refuses, before any launch: a short free list, scores given as
    pooled, a missing score array, block table or new_lens, a negative free count and a
    small workspace."""
    lib = actkv.load_library()
    p = _tiny()
    c = p.cstruct()
    c.seq_lens_d = c.q_lens_d = c.budgets_d = FAKE
    q = actkv.query(p)
    ws, need = q["workspace_bytes"], q["fresh_pages_needed"]

    def call(scores=FAKE, pooled=None, bt=FAKE, num_free=1000, new_lens=FAKE, ws_bytes=ws):
        return lib.actkv_select_compact(ctypes.byref(c), scores, pooled, None, FAKE, bt, FAKE,
                                        num_free, FAKE, new_lens, FAKE, ws_bytes, None)

    assert call(num_free=need - 1) == -4
    assert call(pooled=FAKE) == -1
    assert call(scores=None) == -1
    assert call(bt=None) == -1
    assert call(new_lens=None) == -1
    assert call(num_free=-1) == -1
    assert call(ws_bytes=ws - 1) == -3


def test_check_pages_validates_before_launching():
    """actkv_check_pages refuses, before any launch: a missing status or scratch, a short
    scratch, a short free list, a negative free count, missing device mirrors."""
    lib = actkv.load_library()
    p = _tiny()
    c = p.cstruct()
    c.seq_lens_d = c.q_lens_d = c.budgets_d = FAKE
    q = actkv.query(p)
    need = actkv.check_scratch_bytes(p.num_pages)

    def call(status=FAKE, scratch=FAKE, nbytes=need, num_free=1000, cs=c):
        return lib.actkv_check_pages(ctypes.byref(cs), FAKE, FAKE, num_free, status, scratch,
                                     nbytes, None)

    assert call(status=None) == -1
    assert call(scratch=None) == -1
    assert call(nbytes=need - 1) == -3
    assert call(num_free=q["fresh_pages_needed"] - 1) == -4
    assert call(num_free=-1) == -1
    assert call(cs=_tiny().cstruct()) == -1   # no device mirrors


def test_check_scratch_size_matches_the_header():
    for n in (1, 31, 32, 33, 4_200_000):
        assert actkv.check_scratch_bytes(n) == 8 * ((n + 31) // 32)


def test_lrfu_entry_points_validate_before_launching():
    lib = actkv.load_library()
    p = _tiny()
    c = p.cstruct()
    c.seq_lens_d = c.q_lens_d = c.budgets_d = FAKE
    ws = actkv.query(p)["workspace_bytes"]
    ok = dict(top_p=0.9, decay=0.5)

    def sel(top_p, decay, ks=FAKE + 64, ks_kept=FAKE):
        return lib.actkv_lrfu_select(ctypes.byref(c), FAKE, top_p, decay, ks, None, None, FAKE,
                                     ks_kept, FAKE, ws, None)

    assert sel(1.5, ok["decay"]) == -1
    assert sel(-0.1, ok["decay"]) == -1
    assert sel(float("nan"), ok["decay"]) == -1
    assert sel(ok["top_p"], 1.01) == -1
    assert sel(ok["top_p"], ok["decay"], ks=None) == -1
    assert sel(ok["top_p"], ok["decay"], ks_kept=None) == -1
    # a keep-score array may not alias the scores it is updated from
    assert lib.actkv_lrfu_select(ctypes.byref(c), FAKE, 0.9, 0.5, FAKE, None, None, FAKE,
                                 FAKE, FAKE, ws, None) == -1
    # the step checks its pages before anything else runs
    assert lib.actkv_step_lrfu(ctypes.byref(c), FAKE, FAKE, FAKE, None, FAKE, 0, 0.9, 0.5,
                               FAKE, FAKE, None, None, None, None, FAKE, FAKE, FAKE, ws,
                               None) == -4


@pytest.mark.parametrize("L,window,code", [(64513, 7, -2), (38401, 9, -2), (64512, 7, -1),
                                           (38400, 9, -1)])
def test_lrfu_rejects_segments_past_its_length_limit(L, window, code):
    """Up to 38,400 entries any window; up to 64,512 windows of at most 7; longer segments are
    unsupported (-2).  The call passes no keep-score buffer, which the library checks right
    after the lengths: an accepted length then reports that missing argument (-1) instead,
    and nothing is ever launched."""
    lib = actkv.load_library()
    pb = W.make_custom(seq_lens=[L], q_lens=[1], num_q_heads=1, num_kv_heads=1,
                       head_dim=64, budgets=[10], pool_window=window)
    p = binding_problem(pb)
    c = p.cstruct()
    c.seq_lens_d = c.q_lens_d = c.budgets_d = FAKE
    ws = actkv.query(p)["workspace_bytes"]
    assert lib.actkv_lrfu_select(ctypes.byref(c), FAKE, 0.9, 0.5, None, None, None, FAKE,
                                 FAKE, FAKE, ws, None) == code


def test_inplace_page_accounting_matches_oracle():
    rng = np.random.default_rng(4)
    for _ in range(5):
        seq = [int(x) for x in rng.integers(0, 200, size=5)]
        H = 3
        bud = [int(rng.integers(0, L + 20)) for L in seq for _ in range(H)]
        pb = W.make_custom(seq_lens=seq, q_lens=[min(1, L) for L in seq], num_q_heads=H,
                           num_kv_heads=H, head_dim=64, budgets=bud)
        assert actkv.query_inplace(binding_problem(pb)) == oracle.inplace_pages_freed(pb)


def test_inplace_entry_points_validate_before_launching():
    lib = actkv.load_library()
    p = _tiny()
    c = p.cstruct()
    c.seq_lens_d = c.q_lens_d = c.budgets_d = FAKE
    ws = actkv.query(p)["workspace_bytes"]
    assert actkv.query_inplace(p) > 0
    # missing block table, lengths, kept indices or freed list
    assert lib.actkv_compact_inplace(ctypes.byref(c), FAKE, None, FAKE, FAKE, FAKE, None, FAKE,
                                     ws, None) == -1
    assert lib.actkv_compact_inplace(ctypes.byref(c), FAKE, FAKE, FAKE, FAKE, None, None, FAKE,
                                     ws, None) == -1
    assert lib.actkv_compact_inplace(ctypes.byref(c), FAKE, FAKE, None, FAKE, FAKE, None, FAKE,
                                     ws, None) == -1
    assert lib.actkv_compact_inplace(ctypes.byref(c), FAKE, FAKE, FAKE, None, FAKE, None, FAKE,
                                     ws, None) == -1
    assert lib.actkv_compact_inplace(ctypes.byref(c), FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE,
                                     16, None) == -3
    assert lib.actkv_step_inplace(ctypes.byref(c), None, FAKE, FAKE, None, None, None, None,
                                  FAKE, FAKE, None, FAKE, ws, None) == -1
    assert lib.actkv_step_inplace(ctypes.byref(c), FAKE, FAKE, FAKE, None, FAKE, FAKE, None,
                                  FAKE, FAKE, None, FAKE, ws, None) == -1   # scores == pooled
    assert lib.actkv_query_inplace(None, None) == -1


def test_confidence_entry_points_validate_before_launching():
    lib = actkv.load_library()
    sz = ctypes.c_size_t()
    assert lib.actkv_token_confidence_workspace(4, 151936, 20, ctypes.byref(sz)) == 0
    assert sz.value > 0
    assert lib.actkv_token_confidence_workspace(4, 151936, 0, None) == -1
    assert lib.actkv_token_confidence_workspace(4, 151936, 65, None) == -2
    assert lib.actkv_token_confidence_workspace(4, 262145, 20, None) == -2
    assert lib.actkv_token_confidence_workspace(-1, 100, 20, None) == -1
    assert lib.actkv_token_confidence(FAKE, 4, 1000, 999, 20, FAKE, FAKE, 1 << 20, None) == -1
    assert lib.actkv_token_confidence(None, 4, 1000, 1000, 20, FAKE, FAKE, 1 << 20, None) == -1
    assert lib.actkv_token_confidence(FAKE, 4, 1000, 1000, 20, FAKE, FAKE, 16, None) == -3
    off = np.array([0, 100, 300], np.int64)

    def upd(off=off, window=64, stride=8, pct=10.0, scale=1.75, upper=30000):
        return lib.actkv_budget_update(FAKE, off.ctypes.data, FAKE, off.shape[0] - 1, window,
                                       stride, pct, scale, upper, FAKE, FAKE, None, None,
                                       None, None)
    assert upd(window=0) == -1
    assert upd(stride=0) == -1
    assert upd(pct=100.5) == -1
    assert upd(pct=float("nan")) == -1
    assert upd(scale=0.5) == -1
    assert upd(upper=-1) == -1
    assert upd(off=np.array([0, 100, 50], np.int64)) == -1
    assert upd(off=np.array([0, 64 + 8 * 16384], np.int64)) == -2   # one window too many


def test_noalloc_step_refuses_a_problem_past_its_scratch_array_on_the_host():
    """The size check of actkv_step_noalloc runs on the host before any HIP call: a problem
    needing more workspace than the static array is refused (ACTKV_ERR_WORKSPACE_TOO_SMALL)
    with every data pointer NULL."""
    import ctypes
    R, H = 32, 4
    p = actkv.Problem(seq_lens=[120_000] * R, q_lens=[64] * R, budgets=[30_000] * (R * H),
                      num_q_heads=32, num_kv_heads=H, head_dim=128, num_pages=1 << 20,
                      bt_stride=7500)
    assert actkv.query(p)["workspace_bytes"] > actkv.NOALLOC_SCRATCH_BYTES
    c = p.cstruct()
    rc = actkv.load_library().actkv_step_noalloc(ctypes.byref(c), None, None, None, None, None,
                                                 0, None, None, None, None, None, None)
    assert rc == -3
    bad = actkv.Problem(seq_lens=[10], q_lens=[11], budgets=[1], num_q_heads=1, num_kv_heads=1,
                        head_dim=64, num_pages=4, bt_stride=1)   # causal query past the cache
    c = bad.cstruct()
    assert actkv.load_library().actkv_step_noalloc(ctypes.byref(c), None, None, None, None, None,
                                                   0, None, None, None, None, None, None) == -1


def test_unknown_flags_are_rejected():
    p = _tiny()
    lib = actkv.load_library()
    import ctypes
    for flags, code in [(4, -1), (8, -1), (1 << 31, -1), (actkv.FLAG_PLANNED, 0),
                        (actkv.FLAG_SMALL_SELECT, 0),
                        (actkv.FLAG_PLANNED | actkv.FLAG_SMALL_SELECT, 0)]:
        p.flags = flags
        c = p.cstruct()
        assert lib.actkv_query(ctypes.byref(c), None, None, None, None) == code, flags


def test_overlap_setting_is_validated_and_kept():
    """actkv_set_overlap: 0 .. ACTKV_MAX_OVERLAP_GROUPS accepted and read back; anything
    else refused with the setting unchanged (host only, no device needed)."""
    lib = actkv.load_library()
    assert actkv.get_overlap() == 0
    try:
        for g in range(actkv.MAX_OVERLAP_GROUPS + 1):
            actkv.set_overlap(g)
            assert actkv.get_overlap() == g
        actkv.set_overlap(3)
        for bad in (-1, actkv.MAX_OVERLAP_GROUPS + 1, 1 << 20):
            assert lib.actkv_set_overlap(bad) == -1
            assert actkv.get_overlap() == 3
    finally:
        actkv.set_overlap(0)
