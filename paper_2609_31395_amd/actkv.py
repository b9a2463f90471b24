"""Python binding of libactkv (ctypes): argument marshalling only.

Every function here forwards to the C entry point of the same name in ``libactkv.so``
(HIP kernels for gfx950); PyTorch only supplies device memory and the current stream.
The library must be built in-tree (``python -m paper_2609_31395_amd.build``); importing
this module without it raises, and there is no fallback path.
"""
from __future__ import annotations

import ctypes
import math
import os
from dataclasses import dataclass
from typing import Optional, Sequence

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libactkv.so")

STATUS = {0: "ok", -1: "invalid argument", -2: "unsupported", -3: "workspace too small",
          -4: "out of pages", -5: "HIP error"}
AGG = {"sum": 0, "max_mean": 1}
PAGE_SIZE = 16


class ActKVError(RuntimeError):
    def __init__(self, fn: str, code: int):
        super().__init__(f"{fn} failed: {STATUS.get(code, code)} ({code})")
        self.code = code


class CProblem(ctypes.Structure):
    _fields_ = [("num_reqs", ctypes.c_int32), ("num_q_heads", ctypes.c_int32),
                ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("page_size", ctypes.c_int32), ("num_pages", ctypes.c_int64),
                ("bt_stride", ctypes.c_int32),
                ("seq_lens_h", ctypes.c_void_p), ("q_lens_h", ctypes.c_void_p),
                ("budgets_h", ctypes.c_void_p), ("seq_lens_d", ctypes.c_void_p),
                ("q_lens_d", ctypes.c_void_p), ("budgets_d", ctypes.c_void_p),
                ("sm_scale", ctypes.c_float), ("pool_window", ctypes.c_int32),
                ("causal", ctypes.c_int32), ("agg", ctypes.c_int32), ("flags", ctypes.c_uint32)]


FLAG_PLANNED = 1   # ACTKV_FLAG_PLANNED: the workspace already holds this problem's plan
FLAG_SMALL_SELECT = 2   # ACTKV_FLAG_SMALL_SELECT: selection on the small-footprint kernel
MAX_OVERLAP_GROUPS = 8   # ACTKV_MAX_OVERLAP_GROUPS
# actkv_check_pages status bits
CHECK_MIRRORS, CHECK_TABLE_RANGE, CHECK_FREE_RANGE, CHECK_FRESH_LIVE, CHECK_FRESH_DUP = (
    1, 2, 4, 8, 16)


def check_scratch_bytes(num_pages: int) -> int:
    """ACTKV_CHECK_SCRATCH_BYTES: two page bitmaps."""
    return 8 * ((int(num_pages) + 31) // 32)


_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libactkv.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: build it with `python -m paper_2609_31395_amd.build`")
    lib = ctypes.CDLL(path)
    P = ctypes.POINTER(CProblem)
    vp, i64, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_size_t
    lib.actkv_query.argtypes = [P, ctypes.POINTER(sz), ctypes.POINTER(i64), ctypes.POINTER(i64),
                                ctypes.POINTER(i64)]
    lib.actkv_plan.argtypes = [P, vp, sz, vp]
    lib.actkv_lse.argtypes = [P, vp, vp, vp, vp, vp, sz, vp]
    lib.actkv_score.argtypes = [P, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.actkv_select.argtypes = [P, vp, vp, vp, vp, sz, vp]
    lib.actkv_compact.argtypes = [P, vp, vp, vp, vp, i64, vp, vp, vp, sz, vp]
    lib.actkv_select_compact.argtypes = [P, vp, vp, vp, vp, vp, vp, i64, vp, vp, vp, sz, vp]
    lib.actkv_step.argtypes = [P, vp, vp, vp, vp, vp, i64, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.actkv_step_noalloc.argtypes = [P, vp, vp, vp, vp, vp, i64, vp, vp, vp, vp, vp, vp]
    f32 = ctypes.c_float
    lib.actkv_lrfu_select.argtypes = [P, vp, f32, f32, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.actkv_step_lrfu.argtypes = [P, vp, vp, vp, vp, vp, i64, f32, f32, vp, vp, vp, vp, vp,
                                    vp, vp, vp, vp, sz, vp]
    lib.actkv_score_accumulate.argtypes = [P, vp, vp, vp, vp, vp, vp, sz, vp]
    i32 = ctypes.c_int32
    lib.actkv_token_confidence_workspace.argtypes = [i64, i64, i32, ctypes.POINTER(sz)]
    lib.actkv_token_confidence.argtypes = [vp, i64, i64, i64, i32, vp, vp, sz, vp]
    lib.actkv_budget_update.argtypes = [vp, vp, vp, i32, i32, i32, f32, f32, i32, vp, vp, vp,
                                        vp, vp, vp]
    lib.actkv_query_inplace.argtypes = [P, ctypes.POINTER(i64)]
    lib.actkv_compact_inplace.argtypes = [P, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    lib.actkv_step_inplace.argtypes = [P, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
    for f in ("actkv_query", "actkv_plan", "actkv_lse", "actkv_score", "actkv_select", "actkv_compact",
              "actkv_select_compact",
              "actkv_step", "actkv_step_noalloc", "actkv_lrfu_select", "actkv_step_lrfu", "actkv_query_inplace",
              "actkv_compact_inplace", "actkv_step_inplace", "actkv_score_accumulate",
              "actkv_token_confidence_workspace", "actkv_token_confidence",
              "actkv_budget_update"):
        getattr(lib, f).restype = ctypes.c_int
    lib.actkv_check_pages.argtypes = [P, vp, vp, i64, vp, vp, sz, vp]
    lib.actkv_check_pages.restype = ctypes.c_int
    lib.actkv_set_overlap.argtypes = [i32]
    lib.actkv_set_overlap.restype = ctypes.c_int
    lib.actkv_get_overlap.argtypes = []
    lib.actkv_get_overlap.restype = i32
    lib.actkv_status_str.argtypes = [ctypes.c_int]
    lib.actkv_status_str.restype = ctypes.c_char_p
    _lib = lib
    return lib


@dataclass
class Problem:
    """One compression step's metadata: host arrays plus their device mirrors."""
    seq_lens: np.ndarray
    q_lens: np.ndarray
    budgets: np.ndarray
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    num_pages: int
    bt_stride: int
    sm_scale: float = 0.0
    pool_window: int = 1
    causal: bool = True
    agg: str = "sum"
    seq_lens_d: Optional[torch.Tensor] = None
    q_lens_d: Optional[torch.Tensor] = None
    budgets_d: Optional[torch.Tensor] = None
    page_size: int = PAGE_SIZE
    flags: int = 0

    def __post_init__(self):
        self.seq_lens = np.ascontiguousarray(self.seq_lens, dtype=np.int32).reshape(-1)
        self.q_lens = np.ascontiguousarray(self.q_lens, dtype=np.int32).reshape(-1)
        self.budgets = np.ascontiguousarray(self.budgets, dtype=np.int32).reshape(-1)

    def to_device(self, device="cuda") -> "Problem":
        self.seq_lens_d = torch.from_numpy(self.seq_lens).to(device)
        self.q_lens_d = torch.from_numpy(self.q_lens).to(device)
        self.budgets_d = torch.from_numpy(self.budgets).to(device)
        return self

    @property
    def num_reqs(self) -> int:
        return int(self.seq_lens.shape[0])

    def _key(self):
        """Everything the C view of the problem and its planning depend on (the host arrays'
        contents, the scalars, the device mirrors' addresses)."""
        def dptr(t):
            return None if t is None else t.data_ptr()
        return (self.seq_lens.tobytes(), self.q_lens.tobytes(), self.budgets.tobytes(),
                self.num_q_heads, self.num_kv_heads, self.head_dim, self.num_pages,
                self.bt_stride, self.sm_scale, self.pool_window, self.causal, self.agg,
                self.page_size, self.flags, dptr(self.seq_lens_d), dptr(self.q_lens_d),
                dptr(self.budgets_d))

    def _cached(self):
        """(key, C struct, query result, sizes) of the problem as it is now; rebuilt when any
        of its inputs changed since the last call."""
        key = self._key()
        c = self.__dict__.get("_cache")
        if c is None or c[0] != key:
            struct = self._make_cstruct()
            c = (key, struct, None, None)
            self.__dict__["_cache"] = c
        return c

    def cstruct(self) -> CProblem:
        return self._cached()[1]

    def _make_cstruct(self) -> CProblem:
        def dptr(t):
            return None if t is None else t.data_ptr()
        return CProblem(
            num_reqs=self.num_reqs, num_q_heads=self.num_q_heads,
            num_kv_heads=self.num_kv_heads, head_dim=self.head_dim, page_size=self.page_size,
            num_pages=self.num_pages, bt_stride=self.bt_stride,
            seq_lens_h=self.seq_lens.ctypes.data, q_lens_h=self.q_lens.ctypes.data,
            budgets_h=self.budgets.ctypes.data, seq_lens_d=dptr(self.seq_lens_d),
            q_lens_d=dptr(self.q_lens_d), budgets_d=dptr(self.budgets_d),
            sm_scale=float(self.sm_scale), pool_window=int(self.pool_window),
            causal=int(bool(self.causal)), agg=AGG[self.agg], flags=int(self.flags))

    def planned(self) -> "Problem":
        """The same problem with ACTKV_FLAG_PLANNED: calls skip the plan kernel and use the
        plan already in the workspace (from plan() or an earlier call on this problem)."""
        import dataclasses
        return dataclasses.replace(self, flags=self.flags | FLAG_PLANNED)

    def small_select(self) -> "Problem":
        """The same problem with ACTKV_FLAG_SMALL_SELECT: TopK selection runs on the
        small-footprint kernel (same results)."""
        import dataclasses
        return dataclasses.replace(self, flags=self.flags | FLAG_SMALL_SELECT)


def _check(fn: str, code: int):
    if code != 0:
        raise ActKVError(fn, code)


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


_BITS16 = (torch.bfloat16, torch.int16, torch.uint16)   # bf16 data or its bit pattern
_I32, _F32, _U8 = (torch.int32,), (torch.float32,), (torch.uint8,)


def _need(name: str, t: Optional[torch.Tensor], dtypes, numel: int, required: bool = True,
          seen: Optional[list] = None):
    """Checks one tensor argument before its pointer reaches the C ABI: element type, a
    contiguous layout, at least `numel` elements, resident on a GPU.  A missing tensor is an
    error only when `required` and the call has elements for it.  With `seen`, the device
    check is left to _on_gpu(seen) once every argument has passed the others."""
    if t is None:
        if required and numel > 0:
            raise ValueError(f"{name} is required ({numel} elements)")
        return
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor, got {type(t).__name__}")
    if dtypes is not None and t.dtype not in dtypes:
        raise TypeError(f"{name} must be {' or '.join(str(d) for d in dtypes)}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if t.numel() < numel:
        raise ValueError(f"{name} holds {t.numel()} elements, the call needs {numel}")
    if seen is None:
        _on_gpu([(name, t)])
    else:
        seen.append((name, t))


def _on_gpu(named) -> None:
    """Every tensor resident on the same GPU."""
    first = None
    for name, t in named:
        if not t.is_cuda:
            raise ValueError(f"{name} must be on the GPU, got {t.device}")
        if first is None:
            first = (name, t.get_device())
        elif t.get_device() != first[1]:
            raise ValueError(f"{name} is on cuda:{t.get_device()}, {first[0]} on cuda:{first[1]}")


class _Sizes:
    """Element counts of every array an entry point reads or writes, from the problem and
    its host-only planning query (both cached on the problem while it is unchanged; a qy
    the caller passes is not trusted for sizes)."""

    def __init__(self, p: Problem, qy: Optional[dict] = None):
        qy = query(p)
        cache = p._cached()
        st = cache[3]
        if st is None:
            R, Hkv = p.num_reqs, p.num_kv_heads
            sum_n = int(p.q_lens.astype(np.int64).sum())
            st = dict(sum_n=sum_n, q=sum_n * p.num_q_heads * p.head_dim,
                      lse=sum_n * p.num_q_heads,
                      kv=2 * int(p.num_pages) * p.page_size * Hkv * p.head_dim,
                      bt=R * int(p.bt_stride), scores=num_scores(p), kept=int(qy["num_kept"]),
                      freed=int(qy["pages_freed"]), fresh=int(qy["fresh_pages_needed"]),
                      lens=R * Hkv, ws=int(qy["workspace_bytes"]))
            p.__dict__["_cache"] = (cache[0], cache[1], cache[2], st)
        self.qy = qy
        self.__dict__.update(st)
        self.seen: list = []
        self.mirrors = []
        R, Hkv = p.num_reqs, p.num_kv_heads
        if R > 0:
            for name, t, n in (("seq_lens_d", p.seq_lens_d, R), ("q_lens_d", p.q_lens_d, R),
                               ("budgets_d", p.budgets_d, R * Hkv)):
                _need(name, t, _I32, n, seen=self.mirrors)

    def need(self, name, t, dtypes, numel, required=True):
        _need(name, t, dtypes, numel, required=required, seen=self.seen)

    def check_ws(self, ws: Optional[torch.Tensor]):
        """The caller's workspace, if any; then every argument's device (call last)."""
        if ws is not None:
            self.need("ws", ws, None, 0)
            if _ws_bytes(ws) < self.ws:
                raise ValueError(f"ws holds {_ws_bytes(ws)} bytes, the call needs {self.ws}")
        _on_gpu(self.seen + self.mirrors)

    def kv_args(self, q, kv_cache, block_table, lse=None):
        self.need("q", q, _BITS16, self.q)
        self.need("kv_cache", kv_cache, _BITS16, self.kv if self.scores or self.kept else 0)
        self.need("block_table", block_table, _I32, self.bt)
        self.need("lse", lse, _F32, self.lse, required=False)


def _numel(t: Optional[torch.Tensor]) -> int:
    return 0 if t is None else t.numel()


def _ws_bytes(ws: torch.Tensor) -> int:
    return ws.numel() * ws.element_size()


def query(p: Problem) -> dict:
    """Host-only: workspace bytes, kept entries, fresh pages needed, pages freed."""
    cache = p._cached()
    if cache[2] is not None:
        return dict(cache[2])
    lib = load_library()
    c = cache[1]
    ws, nk, fresh, freed = ctypes.c_size_t(), ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
    _check("actkv_query", lib.actkv_query(ctypes.byref(c), ctypes.byref(ws), ctypes.byref(nk),
                                          ctypes.byref(fresh), ctypes.byref(freed)))
    out = dict(workspace_bytes=ws.value, num_kept=nk.value, fresh_pages_needed=fresh.value,
               pages_freed=freed.value)
    p.__dict__["_cache"] = (cache[0], c, out, cache[3])
    return dict(out)


def query_inplace(p: Problem) -> int:
    """Host-only: pages the in-place compaction returns."""
    lib = load_library()
    c = p.cstruct()
    freed = ctypes.c_int64()
    _check("actkv_query_inplace", lib.actkv_query_inplace(ctypes.byref(c), ctypes.byref(freed)))
    return freed.value


def num_scores(p: Problem) -> int:
    return int(p.seq_lens.astype(np.int64).sum()) * p.num_kv_heads


def workspace(p: Problem, device="cuda") -> torch.Tensor:
    return torch.empty(max(query(p)["workspace_bytes"], 1), dtype=torch.uint8, device=device)


def plan(p: Problem, ws: torch.Tensor, stream=None) -> torch.Tensor:
    """Writes p's plan into ws (for later calls with p.planned())."""
    lib = load_library()
    z = _Sizes(p)
    z.need("ws", ws, None, 0)
    if _ws_bytes(ws) < z.ws:
        raise ValueError(f"ws holds {_ws_bytes(ws)} bytes, the call needs {z.ws}")
    _on_gpu(z.seen + z.mirrors)
    c = p.cstruct()
    _check("actkv_plan", lib.actkv_plan(ctypes.byref(c), _ptr(ws), _ws_bytes(ws), _stream(stream)))
    return ws


def lse(p: Problem, q: torch.Tensor, kv_cache: torch.Tensor, block_table: torch.Tensor,
        out: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None,
        stream=None) -> torch.Tensor:
    lib = load_library()
    z = _Sizes(p)
    z.kv_args(q, kv_cache, block_table)
    z.need("out", out, _F32, z.lse, required=False)
    z.check_ws(ws)
    dev = kv_cache.device
    if out is None:
        out = torch.empty((z.sum_n, p.num_q_heads), dtype=torch.float32, device=dev)
    ws = workspace(p, dev) if ws is None else ws
    c = p.cstruct()
    _check("actkv_lse", lib.actkv_lse(ctypes.byref(c), _ptr(q), _ptr(kv_cache),
                                      _ptr(block_table), _ptr(out), _ptr(ws), _ws_bytes(ws),
                                      _stream(stream)))
    return out


def score(p: Problem, q: torch.Tensor, kv_cache: torch.Tensor, block_table: torch.Tensor,
          lse: Optional[torch.Tensor] = None, out: Optional[torch.Tensor] = None,
          ws: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    lib = load_library()
    z = _Sizes(p)
    z.kv_args(q, kv_cache, block_table, lse)
    z.need("out", out, _F32, z.scores, required=False)
    z.check_ws(ws)
    dev = kv_cache.device
    if out is None:
        out = torch.empty(z.scores, dtype=torch.float32, device=dev)
    ws = workspace(p, dev) if ws is None else ws
    c = p.cstruct()
    _check("actkv_score", lib.actkv_score(ctypes.byref(c), _ptr(q), _ptr(kv_cache),
                                          _ptr(block_table), _ptr(lse), _ptr(out), _ptr(ws),
                                          _ws_bytes(ws), _stream(stream)))
    return out


def score_accumulate(p: Problem, q: torch.Tensor, kv_cache: torch.Tensor,
                     block_table: torch.Tensor, acc: torch.Tensor,
                     lse: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None,
                     stream=None) -> torch.Tensor:
    """acc += the scores of this call (streaming, one decode step)."""
    lib = load_library()
    z = _Sizes(p)
    z.kv_args(q, kv_cache, block_table, lse)
    z.need("acc", acc, _F32, z.scores)
    z.check_ws(ws)
    ws = workspace(p, kv_cache.device) if ws is None else ws
    c = p.cstruct()
    _check("actkv_score_accumulate", lib.actkv_score_accumulate(
        ctypes.byref(c), _ptr(q), _ptr(kv_cache), _ptr(block_table), _ptr(lse), _ptr(acc),
        _ptr(ws), _ws_bytes(ws), _stream(stream)))
    return acc


def select(p: Problem, scores: torch.Tensor, pooled: Optional[torch.Tensor] = None,
           kept: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None,
           stream=None, want_pooled: bool = True):
    """Returns (kept, pooled); pooled is None when not requested."""
    lib = load_library()
    z = _Sizes(p)
    z.need("scores", scores, _F32, z.scores)
    z.need("pooled", pooled, _F32, z.scores, required=False)
    z.need("kept", kept, _I32, z.kept, required=False)
    z.check_ws(ws)
    dev = scores.device
    if kept is None:
        kept = torch.empty(max(z.kept, 1), dtype=torch.int32, device=dev)
    if pooled is None and want_pooled:
        pooled = torch.empty_like(scores)
    ws = workspace(p, dev) if ws is None else ws
    c = p.cstruct()
    _check("actkv_select", lib.actkv_select(ctypes.byref(c), _ptr(scores), _ptr(pooled),
                                            _ptr(kept), _ptr(ws), _ws_bytes(ws),
                                            _stream(stream)))
    return kept[:z.kept], pooled


def _compact_outputs(z: _Sizes, kv_cache, block_table, free_pages, freed, new_lens):
    z.need("kv_cache", kv_cache, _BITS16, z.kv if z.kept else 0)
    z.need("block_table", block_table, _I32, z.bt)
    if free_pages is not None or z.fresh:
        z.need("free_pages", free_pages, _I32, z.fresh)
    z.need("freed", freed, _I32, z.freed, required=False)
    z.need("new_lens", new_lens, _I32, z.lens, required=False)


def compact(p: Problem, kv_cache: torch.Tensor, block_table: torch.Tensor, kept: torch.Tensor,
            free_pages: torch.Tensor, freed: Optional[torch.Tensor] = None,
            new_lens: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None,
            stream=None):
    """In place on kv_cache / block_table.  Returns (freed_pages, new_lens)."""
    lib = load_library()
    z = _Sizes(p)
    _compact_outputs(z, kv_cache, block_table, free_pages, freed, new_lens)
    z.need("kept", kept, _I32, z.kept)
    z.check_ws(ws)
    dev = kv_cache.device
    if freed is None:
        freed = torch.empty(max(z.freed, 1), dtype=torch.int32, device=dev)
    if new_lens is None:
        new_lens = torch.empty(z.lens, dtype=torch.int32, device=dev)
    ws = workspace(p, dev) if ws is None else ws
    c = p.cstruct()
    _check("actkv_compact", lib.actkv_compact(ctypes.byref(c), _ptr(kv_cache), _ptr(block_table),
                                              _ptr(kept), _ptr(free_pages), _numel(free_pages),
                                              _ptr(freed), _ptr(new_lens), _ptr(ws),
                                              _ws_bytes(ws), _stream(stream)))
    return freed[:z.freed], new_lens


def select_compact(p: Problem, scores: torch.Tensor, kv_cache: torch.Tensor,
                   block_table: torch.Tensor, free_pages: torch.Tensor,
                   pooled: Optional[torch.Tensor] = None, kept: Optional[torch.Tensor] = None,
                   freed: Optional[torch.Tensor] = None, new_lens: Optional[torch.Tensor] = None,
                   ws: Optional[torch.Tensor] = None, stream=None) -> dict:
    """actkv_select_compact: selection then fresh-page compaction in one call (in place on
    kv_cache / block_table).  Returns freed, new_lens and the given pooled / kept."""
    lib = load_library()
    z = _Sizes(p)
    z.need("scores", scores, _F32, z.scores)
    z.need("pooled", pooled, _F32, z.scores, required=False)
    z.need("kept", kept, _I32, z.kept, required=False)
    _compact_outputs(z, kv_cache, block_table, free_pages, freed, new_lens)
    z.check_ws(ws)
    dev = kv_cache.device
    if freed is None:
        freed = torch.empty(max(z.freed, 1), dtype=torch.int32, device=dev)
    if new_lens is None:
        new_lens = torch.empty(z.lens, dtype=torch.int32, device=dev)
    ws = workspace(p, dev) if ws is None else ws
    c = p.cstruct()
    _check("actkv_select_compact", lib.actkv_select_compact(
        ctypes.byref(c), _ptr(scores), _ptr(pooled), _ptr(kept), _ptr(kv_cache),
        _ptr(block_table), _ptr(free_pages), _numel(free_pages), _ptr(freed), _ptr(new_lens),
        _ptr(ws), _ws_bytes(ws), _stream(stream)))
    return dict(freed=freed[:z.freed], new_lens=new_lens, pooled=pooled,
                kept=None if kept is None else kept[:z.kept])


def _step_args(z: _Sizes, q, kv_cache, block_table, free_pages, lse, scores, pooled, kept,
               freed, new_lens, ws):
    z.kv_args(q, kv_cache, block_table, lse)
    _compact_outputs(z, kv_cache, block_table, free_pages, freed, new_lens)
    z.need("scores", scores, _F32, z.scores, required=False)
    z.need("pooled", pooled, _F32, z.scores, required=False)
    z.need("kept", kept, _I32, z.kept, required=False)
    z.check_ws(ws)


def step(p: Problem, q: torch.Tensor, kv_cache: torch.Tensor, block_table: torch.Tensor,
         free_pages: torch.Tensor, lse: Optional[torch.Tensor] = None,
         scores: Optional[torch.Tensor] = None, pooled: Optional[torch.Tensor] = None,
         kept: Optional[torch.Tensor] = None, freed: Optional[torch.Tensor] = None,
         new_lens: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None,
         stream=None, qy: Optional[dict] = None) -> dict:
    """The whole step, in place on kv_cache / block_table; optional intermediates."""
    lib = load_library()
    z = _Sizes(p, qy)
    _step_args(z, q, kv_cache, block_table, free_pages, lse, scores, pooled, kept, freed,
               new_lens, ws)
    dev = kv_cache.device
    if freed is None:
        freed = torch.empty(max(z.freed, 1), dtype=torch.int32, device=dev)
    if new_lens is None:
        new_lens = torch.empty(z.lens, dtype=torch.int32, device=dev)
    ws = workspace(p, dev) if ws is None else ws
    c = p.cstruct()
    _check("actkv_step", lib.actkv_step(ctypes.byref(c), _ptr(q), _ptr(kv_cache),
                                        _ptr(block_table), _ptr(lse), _ptr(free_pages),
                                        _numel(free_pages), _ptr(scores), _ptr(pooled),
                                        _ptr(kept), _ptr(freed), _ptr(new_lens), _ptr(ws),
                                        _ws_bytes(ws), _stream(stream)))
    return dict(freed=freed[:z.freed], new_lens=new_lens, scores=scores,
                pooled=pooled, kept=None if kept is None else kept[:z.kept])


NOALLOC_SCRATCH_BYTES = 64 << 20   # ACTKV_NOALLOC_SCRATCH_BYTES


def step_noalloc(p: Problem, q: torch.Tensor, kv_cache: torch.Tensor, block_table: torch.Tensor,
                 free_pages: torch.Tensor, freed: torch.Tensor, new_lens: torch.Tensor,
                 lse: Optional[torch.Tensor] = None, scores: Optional[torch.Tensor] = None,
                 pooled: Optional[torch.Tensor] = None, kept: Optional[torch.Tensor] = None,
                 stream=None, qy: Optional[dict] = None) -> dict:
    """actkv_step with the library's static scratch array as its workspace: nothing is
    allocated, here or in the library, so every output buffer comes from the caller."""
    lib = load_library()
    z = _Sizes(p, qy)
    z.need("freed", freed, _I32, z.freed)
    z.need("new_lens", new_lens, _I32, z.lens)
    _step_args(z, q, kv_cache, block_table, free_pages, lse, scores, pooled, kept, freed,
               new_lens, None)
    c = p.cstruct()
    _check("actkv_step_noalloc", lib.actkv_step_noalloc(
        ctypes.byref(c), _ptr(q), _ptr(kv_cache), _ptr(block_table), _ptr(lse),
        _ptr(free_pages), _numel(free_pages), _ptr(scores), _ptr(pooled), _ptr(kept),
        _ptr(freed), _ptr(new_lens), _stream(stream)))
    return dict(freed=freed[:z.freed], new_lens=new_lens, scores=scores, pooled=pooled,
                kept=None if kept is None else kept[:z.kept])


def compact_inplace(p: Problem, kv_cache: torch.Tensor, block_table: torch.Tensor,
                    kept: torch.Tensor, freed: Optional[torch.Tensor] = None,
                    new_lens: Optional[torch.Tensor] = None,
                    new_order: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None,
                    stream=None, want_order: bool = True) -> dict:
    """In-place compaction (Alg. 4) on kv_cache / block_table.  Returns freed, new_lens and
    new_order (None unless requested)."""
    lib = load_library()
    z = _Sizes(p)
    nfreed = query_inplace(p)
    z.need("kv_cache", kv_cache, _BITS16, z.kv if z.kept else 0)
    z.need("block_table", block_table, _I32, z.bt)
    z.need("kept", kept, _I32, z.kept)
    z.need("freed", freed, _I32, nfreed, required=False)
    z.need("new_lens", new_lens, _I32, z.lens, required=False)
    z.need("new_order", new_order, _I32, z.kept, required=False)
    z.check_ws(ws)
    dev = kv_cache.device
    if freed is None:
        freed = torch.empty(max(nfreed, 1), dtype=torch.int32, device=dev)
    if new_lens is None:
        new_lens = torch.empty(z.lens, dtype=torch.int32, device=dev)
    if new_order is None and want_order:
        new_order = torch.empty(max(z.kept, 1), dtype=torch.int32, device=dev)
    ws = workspace(p, dev) if ws is None else ws
    c = p.cstruct()
    _check("actkv_compact_inplace", lib.actkv_compact_inplace(
        ctypes.byref(c), _ptr(kv_cache), _ptr(block_table), _ptr(kept), _ptr(freed),
        _ptr(new_lens), _ptr(new_order), _ptr(ws), _ws_bytes(ws), _stream(stream)))
    return dict(freed=freed[:nfreed], new_lens=new_lens,
                new_order=None if new_order is None else new_order[:z.kept])


def step_inplace(p: Problem, q: torch.Tensor, kv_cache: torch.Tensor, block_table: torch.Tensor,
                 lse: Optional[torch.Tensor] = None, scores: Optional[torch.Tensor] = None,
                 pooled: Optional[torch.Tensor] = None, kept: Optional[torch.Tensor] = None,
                 freed: Optional[torch.Tensor] = None, new_lens: Optional[torch.Tensor] = None,
                 new_order: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None,
                 stream=None, qy: Optional[dict] = None, nfreed: Optional[int] = None) -> dict:
    """The step with the in-place compaction, in place on kv_cache / block_table."""
    lib = load_library()
    z = _Sizes(p, qy)
    nfreed = query_inplace(p) if nfreed is None else nfreed
    z.kv_args(q, kv_cache, block_table, lse)
    z.need("scores", scores, _F32, z.scores, required=False)
    z.need("pooled", pooled, _F32, z.scores, required=False)
    z.need("kept", kept, _I32, z.kept, required=False)
    z.need("freed", freed, _I32, nfreed, required=False)
    z.need("new_lens", new_lens, _I32, z.lens, required=False)
    z.need("new_order", new_order, _I32, z.kept, required=False)
    z.check_ws(ws)
    dev = kv_cache.device
    if freed is None:
        freed = torch.empty(max(nfreed, 1), dtype=torch.int32, device=dev)
    if new_lens is None:
        new_lens = torch.empty(z.lens, dtype=torch.int32, device=dev)
    ws = workspace(p, dev) if ws is None else ws
    c = p.cstruct()
    _check("actkv_step_inplace", lib.actkv_step_inplace(
        ctypes.byref(c), _ptr(q), _ptr(kv_cache), _ptr(block_table), _ptr(lse), _ptr(scores),
        _ptr(pooled), _ptr(kept), _ptr(freed), _ptr(new_lens), _ptr(new_order), _ptr(ws),
        _ws_bytes(ws), _stream(stream)))
    return dict(freed=freed[:nfreed], new_lens=new_lens, scores=scores, pooled=pooled,
                kept=None if kept is None else kept[:z.kept],
                new_order=None if new_order is None else new_order[:z.kept])


def lrfu_select(p: Problem, scores: torch.Tensor, ks: torch.Tensor, top_p: float,
                decay: float, pooled: Optional[torch.Tensor] = None,
                hit: Optional[torch.Tensor] = None, kept: Optional[torch.Tensor] = None,
                ks_kept: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None,
                stream=None) -> dict:
    """LRFU eviction; ks (fp32, same layout as scores) is updated in place.  Returns kept,
    ks_kept, and the optional pooled / hit outputs.  top_p and decay travel as float32."""
    lib = load_library()
    z = _Sizes(p)
    z.need("scores", scores, _F32, z.scores)
    z.need("ks", ks, _F32, z.scores)
    z.need("pooled", pooled, _F32, z.scores, required=False)
    z.need("hit", hit, _U8, z.scores, required=False)
    z.need("kept", kept, _I32, z.kept, required=False)
    z.need("ks_kept", ks_kept, _F32, z.kept, required=False)
    z.check_ws(ws)
    dev = scores.device
    if kept is None:
        kept = torch.empty(max(z.kept, 1), dtype=torch.int32, device=dev)
    if ks_kept is None:
        ks_kept = torch.empty(max(z.kept, 1), dtype=torch.float32, device=dev)
    ws = workspace(p, dev) if ws is None else ws
    c = p.cstruct()
    _check("actkv_lrfu_select", lib.actkv_lrfu_select(
        ctypes.byref(c), _ptr(scores), float(top_p), float(decay), _ptr(ks), _ptr(hit),
        _ptr(pooled), _ptr(kept), _ptr(ks_kept), _ptr(ws), _ws_bytes(ws), _stream(stream)))
    return dict(kept=kept[:z.kept], ks_kept=ks_kept[:z.kept], pooled=pooled, hit=hit)


def step_lrfu(p: Problem, q: torch.Tensor, kv_cache: torch.Tensor, block_table: torch.Tensor,
              free_pages: torch.Tensor, ks: torch.Tensor, top_p: float, decay: float,
              lse: Optional[torch.Tensor] = None, scores: Optional[torch.Tensor] = None,
              pooled: Optional[torch.Tensor] = None, hit: Optional[torch.Tensor] = None,
              kept: Optional[torch.Tensor] = None, ks_kept: Optional[torch.Tensor] = None,
              freed: Optional[torch.Tensor] = None, new_lens: Optional[torch.Tensor] = None,
              ws: Optional[torch.Tensor] = None, stream=None, qy: Optional[dict] = None) -> dict:
    """The whole step with LRFU eviction, in place on kv_cache / block_table / ks."""
    lib = load_library()
    z = _Sizes(p, qy)
    z.need("ks", ks, _F32, z.scores)
    z.need("hit", hit, _U8, z.scores, required=False)
    z.need("ks_kept", ks_kept, _F32, z.kept, required=False)
    _step_args(z, q, kv_cache, block_table, free_pages, lse, scores, pooled, kept, freed,
               new_lens, ws)
    dev = kv_cache.device
    if freed is None:
        freed = torch.empty(max(z.freed, 1), dtype=torch.int32, device=dev)
    if new_lens is None:
        new_lens = torch.empty(z.lens, dtype=torch.int32, device=dev)
    if ks_kept is None:
        ks_kept = torch.empty(max(z.kept, 1), dtype=torch.float32, device=dev)
    ws = workspace(p, dev) if ws is None else ws
    c = p.cstruct()
    _check("actkv_step_lrfu", lib.actkv_step_lrfu(
        ctypes.byref(c), _ptr(q), _ptr(kv_cache), _ptr(block_table), _ptr(lse),
        _ptr(free_pages), _numel(free_pages), float(top_p), float(decay), _ptr(ks),
        _ptr(ks_kept), _ptr(scores), _ptr(pooled), _ptr(hit), _ptr(kept), _ptr(freed),
        _ptr(new_lens), _ptr(ws), _ws_bytes(ws), _stream(stream)))
    return dict(freed=freed[:z.freed], new_lens=new_lens,
                ks_kept=ks_kept[:z.kept], scores=scores, pooled=pooled, hit=hit,
                kept=None if kept is None else kept[:z.kept])


def token_confidence(logits: torch.Tensor, top_k: int = 20, out: Optional[torch.Tensor] = None,
                     ws: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """Token-level confidence of every row of `logits` (fp32 [rows, >= vocab] with unit
    column stride); vocab = logits.shape[1]."""
    lib = load_library()
    if not isinstance(logits, torch.Tensor) or logits.dim() != 2:
        raise ValueError("logits must be a 2-D tensor [rows, vocab]")
    rows, vocab = int(logits.shape[0]), int(logits.shape[1])
    if logits.dtype != torch.float32 or (rows > 0 and logits.stride(1) != 1):
        raise ValueError("logits must be float32 with contiguous rows")
    if rows > 1 and logits.stride(0) < vocab:
        raise ValueError("logits rows must not overlap")
    if logits.device.type != "cuda":
        raise ValueError(f"logits must be on the GPU, got {logits.device}")
    _need("out", out, _F32, rows, required=False)
    need = ctypes.c_size_t()
    _check("actkv_token_confidence_workspace",
           lib.actkv_token_confidence_workspace(rows, vocab, int(top_k), ctypes.byref(need)))
    if ws is not None:
        _need("ws", ws, None, 0)
        if _ws_bytes(ws) < need.value:
            raise ValueError(f"ws holds {_ws_bytes(ws)} bytes, the call needs {need.value}")
    if out is None:
        out = torch.empty(max(rows, 1), dtype=torch.float32, device=logits.device)
    if ws is None:
        ws = torch.empty(max(need.value, 1), dtype=torch.uint8, device=logits.device)
    _check("actkv_token_confidence", lib.actkv_token_confidence(
        _ptr(logits), rows, vocab, int(logits.stride(0)) if rows > 0 else vocab, int(top_k),
        _ptr(out), _ptr(ws), _ws_bytes(ws), _stream(stream)))
    return out[:rows]


def budget_update(token_conf: torch.Tensor, offsets: np.ndarray, budgets: torch.Tensor,
                  window: int = 64, stride: int = 8, bottom_pct: float = 10.0,
                  scale_up: float = 1.75, budget_upper: int = 30000,
                  out: Optional[torch.Tensor] = None, stream=None,
                  offsets_d: Optional[torch.Tensor] = None) -> dict:
    """Alg. 2 steps 2-4 for every request (token confidences concatenated, int64 offsets
    [R + 1] on the host; offsets_d, when given, holds the same values on the device and
    saves the copy).  Returns the new budgets, slopes, thresholds and retained counts."""
    lib = load_library()
    off_h = np.ascontiguousarray(offsets, dtype=np.int64).reshape(-1)
    R = int(off_h.shape[0] - 1)
    if R < 0:
        raise ValueError("offsets must hold R + 1 values")
    n_conf = int(off_h[-1]) if R > 0 else 0
    seen: list = []
    _need("token_conf", token_conf, _F32, n_conf, required=n_conf > 0, seen=seen)
    _need("budgets", budgets, _I32, R, seen=seen)
    _need("out", out, _I32, R, required=False, seen=seen)
    _need("offsets_d", offsets_d, (torch.int64,), R + 1, required=False, seen=seen)
    if offsets_d is not None and offsets_d.numel() != R + 1:
        raise ValueError("offsets_d must be int64 [R + 1] on the device")
    _on_gpu(seen)
    dev = budgets.device
    off_d = torch.from_numpy(off_h).to(dev) if offsets_d is None else offsets_d
    if out is None:
        out = torch.empty(max(R, 1), dtype=torch.int32, device=dev)
    slopes = torch.empty(max(R, 1), dtype=torch.float64, device=dev)
    thr = torch.empty_like(slopes)
    kept = torch.empty(max(R, 1), dtype=torch.int32, device=dev)
    _check("actkv_budget_update", lib.actkv_budget_update(
        _ptr(token_conf), off_h.ctypes.data, _ptr(off_d), R, int(window), int(stride),
        float(bottom_pct), float(scale_up), int(budget_upper), _ptr(budgets), _ptr(out),
        _ptr(slopes), _ptr(thr), _ptr(kept), _stream(stream)))
    return dict(budgets=out[:R], slopes=slopes[:R], thresholds=thr[:R], retained=kept[:R],
                _keep=off_d)


def check_pages(p: Problem, block_table: torch.Tensor, free_pages: Optional[torch.Tensor],
                status: Optional[torch.Tensor] = None, scratch: Optional[torch.Tensor] = None,
                stream=None) -> torch.Tensor:
    """actkv_check_pages: the compaction's preconditions checked on the device.  Returns the
    one-element int32 status tensor (0: everything holds; else CHECK_* bits), valid once the
    stream gets there."""
    lib = load_library()
    z = _Sizes(p)
    z.need("block_table", block_table, _I32, z.bt)
    if free_pages is not None or z.fresh:
        z.need("free_pages", free_pages, _I32, z.fresh)
    z.need("status", status, _I32, 1, required=False)
    if scratch is not None:
        z.need("scratch", scratch, (torch.uint8,), check_scratch_bytes(p.num_pages))
    z.check_ws(None)
    dev = block_table.device
    if status is None:
        status = torch.empty(1, dtype=torch.int32, device=dev)
    if scratch is None:
        scratch = torch.empty(check_scratch_bytes(p.num_pages), dtype=torch.uint8, device=dev)
    _check("actkv_check_pages", lib.actkv_check_pages(
        ctypes.byref(p.cstruct()), _ptr(block_table), _ptr(free_pages), _numel(free_pages),
        _ptr(status), _ptr(scratch), _numel(scratch), _stream(stream)))
    return status


def set_overlap(groups: int) -> None:
    """actkv_set_overlap: 0 = automatic pipelining of large steps, 1 = never, 2 ..
    MAX_OVERLAP_GROUPS = pipeline every step that can be, in that many request groups."""
    _check("actkv_set_overlap", load_library().actkv_set_overlap(int(groups)))


def get_overlap() -> int:
    return int(load_library().actkv_get_overlap())


def status_str(code: int) -> str:
    return load_library().actkv_status_str(code).decode()


def default_sm_scale(head_dim: int) -> float:
    return float(np.float32(1.0) / np.sqrt(np.float32(head_dim)))
