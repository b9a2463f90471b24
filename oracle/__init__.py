"""CPU oracle of the ActKV compression step -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, the package smoke check and the benchmark's CPU-baseline leg may import
this module.  It wraps ``actkv_oracle.c`` (plain C, fp64, OpenMP over independent
(request, KV head) pairs) and ``confidence_oracle.c`` (the confidence monitor and budget
rule of Alg. 2) through ctypes.  It shares no code with the HIP library; its
inputs are host numpy arrays (bf16 carried as uint16 bit patterns).

The functions take a ``problem`` object with the attributes of a synthetic workload
(``seq_lens``, ``q_lens``, ``budgets``, ``q``, ``kv``, ``block_table``, ``free_pages``,
``num_q_heads``, ``num_kv_heads``, ``head_dim``, ``page_size``, ``sm_scale``,
``pool_window``, ``causal``); any object with those attributes works.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRCS = [os.path.join(_HERE, "actkv_oracle.c"), os.path.join(_HERE, "confidence_oracle.c")]
_LIB = os.path.join(_HERE, "liboracle.so")

AGG = {"sum": 0, "max_mean": 1}


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (-O2, no fast-math, no fused multiply-add, OpenMP)."""
    if force or _stale():
        tmp = _LIB + ".tmp"
        subprocess.run(["gcc", "-O2", "-ffp-contract=off", "-fopenmp", "-fPIC", "-shared",
                        "-Wall", "-Wextra", "-o", tmp] + _SRCS + ["-lm"], check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _stale() -> bool:
    return not os.path.exists(_LIB) or any(os.path.getmtime(_LIB) < os.path.getmtime(f)
                                           for f in _SRCS)


class _Problem(ctypes.Structure):
    _fields_ = [("num_reqs", ctypes.c_int32), ("num_q_heads", ctypes.c_int32),
                ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("page_size", ctypes.c_int32), ("num_pages", ctypes.c_int64),
                ("bt_stride", ctypes.c_int32),
                ("seq_lens", ctypes.c_void_p), ("q_lens", ctypes.c_void_p),
                ("budgets", ctypes.c_void_p), ("sm_scale", ctypes.c_double),
                ("pool_window", ctypes.c_int32), ("causal", ctypes.c_int32),
                ("agg", ctypes.c_int32)]


_lib = None


def _load():
    global _lib
    if _lib is None:
        if _stale():
            build(force=True)
        lib = ctypes.CDLL(_LIB)
        P = ctypes.POINTER(_Problem)
        vp, i64 = ctypes.c_void_p, ctypes.c_int64
        lib.actkv_oracle_slot.argtypes = [vp, ctypes.c_int32, i64]
        lib.actkv_oracle_slot.restype = i64
        lib.actkv_oracle_lse.argtypes = [P, vp, vp, vp, vp]
        lib.actkv_oracle_scores.argtypes = [P, vp, vp, vp, vp, vp]
        lib.actkv_oracle_pool.argtypes = [P, vp, vp]
        lib.actkv_oracle_select.argtypes = [P, vp, vp]
        lib.actkv_oracle_totals.argtypes = [P, ctypes.POINTER(i64), ctypes.POINTER(i64),
                                            ctypes.POINTER(i64)]
        lib.actkv_oracle_compact.argtypes = [P, vp, vp, vp, vp, i64, vp, vp]
        lib.actkv_oracle_compact_inplace.argtypes = [P, vp, vp, vp, vp, vp, vp,
                                                     ctypes.POINTER(i64)]
        lib.actkv_oracle_hits.argtypes = [P, vp, ctypes.c_double, vp]
        lib.actkv_oracle_token_confidence.argtypes = [vp, i64, i64, i64, ctypes.c_int32, vp]
        lib.actkv_oracle_budget_update.argtypes = [vp, vp, ctypes.c_int32, ctypes.c_int32,
                                                   ctypes.c_int32, ctypes.c_double,
                                                   ctypes.c_double, ctypes.c_int32, vp, vp, vp,
                                                   vp, vp]
        lib.actkv_oracle_lrfu_update.argtypes = [P, vp, vp, ctypes.c_float, vp]
        lib.actkv_oracle_get_threads.restype = ctypes.c_int
        lib.actkv_oracle_set_threads.argtypes = [ctypes.c_int]
        for f in ("actkv_oracle_lse", "actkv_oracle_scores", "actkv_oracle_pool",
                  "actkv_oracle_select", "actkv_oracle_totals", "actkv_oracle_compact",
                  "actkv_oracle_hits", "actkv_oracle_lrfu_update"):
            getattr(lib, f).restype = ctypes.c_int
        _lib = lib
    return _lib


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data


class _Bound:
    """Keeps the numpy arrays referenced by the C struct alive."""

    def __init__(self, pb, agg="sum", budgets=None, pool_window=None, causal=None,
                 sm_scale=None):
        self.seq = np.ascontiguousarray(pb.seq_lens, dtype=np.int32)
        self.ql = np.ascontiguousarray(pb.q_lens, dtype=np.int32)
        self.bud = np.ascontiguousarray(pb.budgets if budgets is None else budgets,
                                        dtype=np.int32)
        bt = np.asarray(pb.block_table)
        self.st = _Problem(
            num_reqs=self.seq.shape[0], num_q_heads=pb.num_q_heads,
            num_kv_heads=pb.num_kv_heads, head_dim=pb.head_dim, page_size=pb.page_size,
            num_pages=int(np.asarray(pb.kv).shape[1]), bt_stride=int(bt.shape[1]),
            seq_lens=self.seq.ctypes.data, q_lens=self.ql.ctypes.data,
            budgets=self.bud.ctypes.data,
            sm_scale=float(pb.sm_scale if sm_scale is None else sm_scale),
            pool_window=int(pb.pool_window if pool_window is None else pool_window),
            causal=int(pb.causal if causal is None else causal), agg=AGG[agg])

    @property
    def ref(self):
        return ctypes.byref(self.st)


def _check(rc, what):
    if rc != 0:
        raise ValueError(f"oracle {what} rejected its arguments (rc={rc})")


def slot(bt_row, page_size: int, t: int) -> int:
    """Flat physical slot of logical token t (Sec. 2.5 block-table mapping)."""
    row = np.ascontiguousarray(bt_row, dtype=np.int32)
    return int(_load().actkv_oracle_slot(row.ctypes.data, page_size, t))


def num_scores(pb) -> int:
    return int(np.sum(np.asarray(pb.seq_lens, dtype=np.int64)) * pb.num_kv_heads)


def lse(pb, **kw) -> np.ndarray:
    """fp64 log-sum-exp of every action-query row, [sum n, Hq]."""
    b = _Bound(pb, **kw)
    out = np.zeros((int(b.ql.sum()), pb.num_q_heads), dtype=np.float64)
    q = np.ascontiguousarray(pb.q, dtype=np.uint16)
    kv = np.ascontiguousarray(pb.kv, dtype=np.uint16)
    bt = np.ascontiguousarray(pb.block_table, dtype=np.int32)
    _check(_load().actkv_oracle_lse(b.ref, q.ctypes.data, kv.ctypes.data, bt.ctypes.data,
                                    out.ctypes.data), "lse")
    return out


def scores(pb, lse_in: Optional[np.ndarray] = None, agg: str = "sum", **kw) -> np.ndarray:
    """Raw per-entry scores (float32, one fp64 sum rounded once), ragged [sum_r Hkv*L_r]."""
    b = _Bound(pb, agg=agg, **kw)
    out = np.zeros(num_scores(pb), dtype=np.float32)
    q = np.ascontiguousarray(pb.q, dtype=np.uint16)
    kv = np.ascontiguousarray(pb.kv, dtype=np.uint16)
    bt = np.ascontiguousarray(pb.block_table, dtype=np.int32)
    li = None if lse_in is None else np.ascontiguousarray(lse_in, dtype=np.float32)
    _check(_load().actkv_oracle_scores(b.ref, q.ctypes.data, kv.ctypes.data, bt.ctypes.data,
                                       _ptr(li), out.ctypes.data), "scores")
    return out


def pool(pb, raw: np.ndarray, **kw) -> np.ndarray:
    b = _Bound(pb, **kw)
    raw = np.ascontiguousarray(raw, dtype=np.float32)
    out = np.zeros_like(raw)
    _check(_load().actkv_oracle_pool(b.ref, raw.ctypes.data, out.ctypes.data), "pool")
    return out


def totals(pb, **kw):
    """(entries kept, fresh pages needed, pages freed) of one step."""
    b = _Bound(pb, **kw)
    a, c, d = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
    _check(_load().actkv_oracle_totals(b.ref, ctypes.byref(a), ctypes.byref(c),
                                       ctypes.byref(d)), "totals")
    return a.value, c.value, d.value


def select(pb, pooled: np.ndarray, **kw) -> np.ndarray:
    """Kept token indices, ascending per (request, KV head), concatenated in (r, h) order."""
    b = _Bound(pb, **kw)
    nk, _, _ = totals(pb, **kw)
    pooled = np.ascontiguousarray(pooled, dtype=np.float32)
    out = np.zeros(max(nk, 1), dtype=np.int32)
    _check(_load().actkv_oracle_select(b.ref, pooled.ctypes.data, out.ctypes.data), "select")
    return out[:nk]


def compact(pb, kept: np.ndarray, kv: Optional[np.ndarray] = None,
            block_table: Optional[np.ndarray] = None, free_pages: Optional[np.ndarray] = None,
            **kw):
    """Fresh-page compaction on copies of the inputs.

    Returns (kv', block_table', freed_pages, new_lens).
    """
    b = _Bound(pb, **kw)
    _, need, nfreed = totals(pb, **kw)
    kv2 = np.array(pb.kv if kv is None else kv, dtype=np.uint16, copy=True, order="C")
    bt2 = np.array(pb.block_table if block_table is None else block_table, dtype=np.int32,
                   copy=True, order="C")
    fp = np.ascontiguousarray(pb.free_pages if free_pages is None else free_pages,
                              dtype=np.int32)
    kept = np.ascontiguousarray(kept, dtype=np.int32)
    freed = np.zeros(max(nfreed, 1), dtype=np.int32)
    new_lens = np.zeros(b.bud.shape[0], dtype=np.int32)
    rc = _load().actkv_oracle_compact(b.ref, kv2.ctypes.data, bt2.ctypes.data,
                                      kept.ctypes.data if kept.size else None,
                                      fp.ctypes.data if fp.size else None, fp.shape[0],
                                      freed.ctypes.data, new_lens.ctypes.data)
    if rc == -2:
        raise ValueError("oracle compact: free list shorter than the fresh pages needed")
    _check(rc, "compact")
    return kv2, bt2, freed[:nfreed], new_lens


def step(pb, lse_in: Optional[np.ndarray] = None, agg: str = "sum", **kw) -> dict:
    """The whole compression step on copies of the inputs; returns every intermediate."""
    raw = scores(pb, lse_in=lse_in, agg=agg, **kw)
    pooled = pool(pb, raw, **kw)
    kept = select(pb, pooled, **kw)
    kv2, bt2, freed, new_lens = compact(pb, kept, **kw)
    return dict(raw=raw, pooled=pooled, kept=kept, kv=kv2, block_table=bt2, freed=freed,
                new_lens=new_lens)


def inplace_pages_freed(pb, **kw) -> int:
    """Pages the in-place compaction returns: Y - X per compacted request (Alg. 4)."""
    b = _Bound(pb, **kw)
    H, BS = pb.num_kv_heads, pb.page_size
    total = 0
    for r, L in enumerate(np.asarray(pb.seq_lens, np.int64)):
        bud = b.bud[r * H:(r + 1) * H].astype(np.int64)
        if (bud >= L).all():
            continue
        kmax = int(np.minimum(bud, L).max())
        total += -(-int(L) // BS) - (-(-kmax // BS))
    return total


def compact_inplace(pb, kept: np.ndarray, kv: Optional[np.ndarray] = None,
                    block_table: Optional[np.ndarray] = None, **kw) -> dict:
    """In-place compaction (Alg. 4) on copies of the inputs.

    Returns kv', block_table', freed pages, new_lens, new_order (the original token of
    every new slot, laid out like kept) and the number of row copies."""
    b = _Bound(pb, **kw)
    kv2 = np.array(pb.kv if kv is None else kv, dtype=np.uint16, copy=True, order="C")
    bt2 = np.array(pb.block_table if block_table is None else block_table, dtype=np.int32,
                   copy=True, order="C")
    kept = np.ascontiguousarray(kept, dtype=np.int32)
    nfreed = inplace_pages_freed(pb, **kw)
    freed = np.zeros(max(nfreed, 1), dtype=np.int32)
    new_lens = np.zeros(b.bud.shape[0], dtype=np.int32)
    new_order = np.zeros(max(kept.shape[0], 1), dtype=np.int32)
    pairs = ctypes.c_int64(0)
    rc = _load().actkv_oracle_compact_inplace(b.ref, kv2.ctypes.data, bt2.ctypes.data,
                                              kept.ctypes.data if kept.size else None,
                                              freed.ctypes.data, new_lens.ctypes.data,
                                              new_order.ctypes.data, ctypes.byref(pairs))
    _check(rc, "compact_inplace")
    return dict(kv=kv2, block_table=bt2, freed=freed[:nfreed], new_lens=new_lens,
                new_order=new_order[:kept.shape[0]], pairs=int(pairs.value))


def step_inplace(pb, lse_in: Optional[np.ndarray] = None, agg: str = "sum", **kw) -> dict:
    """The compression step with the in-place compaction of Alg. 4."""
    raw = scores(pb, lse_in=lse_in, agg=agg, **kw)
    pooled = pool(pb, raw, **kw)
    kept = select(pb, pooled, **kw)
    out = compact_inplace(pb, kept, **kw)
    out.update(raw=raw, pooled=pooled, kept=kept)
    return out


def as_f32(x: float) -> float:
    """x rounded to the nearest float32, as a Python float: the value a float32 parameter of
    the GPU entry points carries (the oracle then computes with exactly that value)."""
    return float(np.float32(x))


def hits(pb, att: np.ndarray, top_p: float, **kw) -> np.ndarray:
    """Top-p hit mask (uint8, same layout as the scores) of the scores `att` (Alg. 1 step 3).
    top_p is rounded to float32 first, the precision the GPU entry point receives it in."""
    b = _Bound(pb, **kw)
    att = np.ascontiguousarray(att, dtype=np.float32)
    out = np.zeros(att.shape[0], dtype=np.uint8)
    _check(_load().actkv_oracle_hits(b.ref, att.ctypes.data, as_f32(top_p), out.ctypes.data),
           "hits")
    return out


def lrfu_update(pb, att: np.ndarray, hit: np.ndarray, decay: float, ks: np.ndarray,
                **kw) -> np.ndarray:
    """KS' = decay * KS + hit * att in fp32 (Alg. 1 step 4), on a copy of ks."""
    b = _Bound(pb, **kw)
    att = np.ascontiguousarray(att, dtype=np.float32)
    hit = np.ascontiguousarray(hit, dtype=np.uint8)
    out = np.array(ks, dtype=np.float32, copy=True, order="C")
    _check(_load().actkv_oracle_lrfu_update(b.ref, att.ctypes.data, hit.ctypes.data,
                                            as_f32(decay), out.ctypes.data), "lrfu_update")
    return out


def lrfu_step(pb, ks: np.ndarray, top_p: float, decay: float,
              lse_in: Optional[np.ndarray] = None, agg: str = "sum", **kw) -> dict:
    """The step with LRFU keep scores (Alg. 1 steps 1-6): score, pool, hit mask, keep-score
    update, TopK on the keep scores, compaction.  `ks` holds the keep score of every cached
    entry (0 for entries new since the last step); ks_kept are those of the kept entries
    (KS'), in the order of `kept`.  top_p and decay are float32 parameters (rounded here as
    the GPU entry point receives them)."""
    raw = scores(pb, lse_in=lse_in, agg=agg, **kw)
    pooled = pool(pb, raw, **kw)
    hit = hits(pb, pooled, top_p, **kw)
    ks2 = lrfu_update(pb, pooled, hit, decay, ks, **kw)
    kept = select(pb, ks2, **kw)
    seg = np.concatenate([[0], np.cumsum(np.repeat(np.asarray(pb.seq_lens, np.int64),
                                                   pb.num_kv_heads))])
    ks_kept, off = np.zeros(kept.shape[0], np.float32), 0
    for s_i in range(seg.shape[0] - 1):
        r, h = divmod(s_i, pb.num_kv_heads)
        k = int(min(max(int(pb.budgets[r * pb.num_kv_heads + h]), 0), int(pb.seq_lens[r])))
        ks_kept[off:off + k] = ks2[seg[s_i] + kept[off:off + k]]
        off += k
    kv2, bt2, freed, new_lens = compact(pb, kept, **kw)
    return dict(raw=raw, pooled=pooled, hit=hit, ks=ks2, kept=kept, ks_kept=ks_kept, kv=kv2,
                block_table=bt2, freed=freed, new_lens=new_lens)


def token_confidence(logits: np.ndarray, k: int = 20) -> np.ndarray:
    """T per row of `logits` ([rows, vocab] float32): -(1/k) sum of the log-probabilities of
    the k most likely tokens (Sec. 6.1), fp64."""
    x = np.ascontiguousarray(logits, dtype=np.float32)
    rows, vocab = x.shape
    out = np.zeros(rows, np.float64)
    _check(_load().actkv_oracle_token_confidence(x.ctypes.data, rows, vocab, vocab, int(k),
                                                 out.ctypes.data), "token_confidence")
    return out


def budget_update(conf_seqs, budgets, window: int = 64, stride: int = 8,
                  bottom_pct: float = 10.0, scale_up: float = 1.75,
                  budget_upper: int = 30000) -> dict:
    """Alg. 2 steps 2-4 per request: trace-level confidence, trend, budget.  conf_seqs is a
    list of float32 token-confidence sequences (one per request).  Parameters are passed as
    the float32 values the GPU entry point receives."""
    seqs = [np.ascontiguousarray(c, dtype=np.float32) for c in conf_seqs]
    flat = np.concatenate(seqs) if seqs else np.zeros(0, np.float32)
    flat = np.ascontiguousarray(flat if flat.size else np.zeros(1, np.float32))
    offsets = np.concatenate([[0], np.cumsum([c.size for c in seqs])]).astype(np.int64)
    R = len(seqs)
    b_in = np.ascontiguousarray(budgets, dtype=np.int32)
    b_out = np.zeros(max(R, 1), np.int32)
    slopes = np.zeros(max(R, 1), np.float64)
    thr = np.zeros(max(R, 1), np.float64)
    kept = np.zeros(max(R, 1), np.int32)
    _check(_load().actkv_oracle_budget_update(
        flat.ctypes.data, offsets.ctypes.data, R, int(window), int(stride),
        float(np.float32(bottom_pct)), float(np.float32(scale_up)), int(budget_upper),
        b_in.ctypes.data, b_out.ctypes.data, slopes.ctypes.data, thr.ctypes.data,
        kept.ctypes.data), "budget_update")
    return dict(budgets=b_out[:R], slopes=slopes[:R], thresholds=thr[:R], retained=kept[:R])


def set_threads(n: int) -> None:
    """Threads the oracle's parallel loops use from now on (timing only)."""
    _load().actkv_oracle_set_threads(int(n))


def threads_in_use() -> int:
    """Threads the oracle's parallel loops use now (OpenMP's own count)."""
    return int(_load().actkv_oracle_get_threads())


def num_threads() -> int:
    """Threads the OpenMP oracle will use (OMP_NUM_THREADS, else the CPU count)."""
    v = os.environ.get("OMP_NUM_THREADS")
    if v and v.isdigit() and int(v) > 0:
        return int(v)
    return len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count()
