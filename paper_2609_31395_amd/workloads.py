"""Seeded synthetic inputs for the ActKV compression step (score -> select -> compact).

This module only *draws* inputs: Gaussian Q/K/V rounded to bf16, planted spike keys,
a shuffled physical page pool with its block table and free list, per-(request, KV head)
budgets and the scoring flags.  None of the method's arithmetic (logits, softmax, scores,
pooling, selection, compaction) lives here, so the CPU oracle and the HIP path can both
consume these arrays without sharing any of that code.

The paper's evaluation runs agent traces from ALFWorld, HotpotQA-Web and WebShop on
Qwen3 / GPT-OSS models (Sec. 8.1).  None of those traces or weights are used: the
workloads below are synthetic stand-ins with the head shapes of Qwen3-30B
(32 query heads, 4 KV heads, head_dim 128, 16-token pages), the trace lengths the paper
reports (about 35K tokens for a 25-iteration WebShop task, Sec. 1; mean FullKV lengths
8K-33K, Sec. 8.1) and the page-pool layout of Sec. 2.5.

Recipe (all draws from numpy PCG64, one child stream per request via SeedSequence.spawn):
  * Q, K, V ~ N(0, 1) in float32, rounded to bf16 (round-to-nearest-even).
  * Spike keys: per (request, KV head) ``round(spike_frac * L)`` distinct token indices;
    their K row (before rounding) gets ``+ 3 * mean`` where ``mean`` is the average of that
    request's bf16 action queries over the G query heads that share the KV head.
  * Pages: the pool holds ``pool_factor`` times the pages in use (or a fixed count), is
    shuffled by a seeded permutation; each request takes its pages in logical order from
    the permutation, the rest form the free list.
  * Budgets: a fixed count, a fraction of L, or a Dirichlet(alpha) split of a fraction of
    ``Hkv * L`` across the KV heads of a request (floor; never above L).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Tuple

import numpy as np

PAGE_SIZE = 16


@dataclass(frozen=True)
class WorkloadConfig:
    name: str
    num_reqs: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    seq_len: Tuple[int, int]      # inclusive range; lo == hi for a fixed length
    q_len: Tuple[int, int]        # inclusive range of action queries per request
    budget: Tuple                 # ("fixed", B) | ("frac", f) | ("dirichlet", alpha, f)
    pool_window: int
    spike_frac: float
    seed: int
    pool_factor: float = 2.0
    fixed_pool_pages: Optional[int] = None
    causal: bool = True
    description: str = ""


CONFIGS: Dict[str, WorkloadConfig] = {
    "tiny": WorkloadConfig(
        "tiny", 1, 8, 2, 64, (2048, 2048), (16, 16), ("fixed", 512), 5, 0.02, 1001,
        fixed_pool_pages=256,
        description="1 request, 8q/2kv heads, d=64, 2048 tokens in 128 of 256 shuffled "
                    "pages, 16 action queries, 2% spikes, pool 5, budget 512 per KV head"),
    "single35k": WorkloadConfig(
        "single35k", 1, 32, 4, 128, (35000, 35000), (64, 64), ("frac", 0.25), 7, 0.01, 1002,
        description="1 request, Qwen3-30B heads (32q/4kv, d=128), 35,000 tokens, "
                    "64 action queries, 1% spikes, pool 7, budget 25% per KV head"),
    "batched": WorkloadConfig(
        "batched", 32, 32, 4, 128, (8000, 40000), (32, 128), ("frac", 0.25), 7, 0.01, 1003,
        description="32 requests, Qwen3-30B heads, L ~ U[8000, 40000], 32-128 action "
                    "queries, 1% spikes, pool 7, budget 25% per KV head"),
    "adaptive": WorkloadConfig(
        "adaptive", 32, 32, 4, 128, (8000, 40000), (32, 128), ("dirichlet", 0.5, 0.25), 7,
        0.01, 1004,
        description="as 'batched' with per-(request, KV head) budgets from a "
                    "Dirichlet(0.5) split of 25% of Hkv*L"),
    "batch32x35k": WorkloadConfig(
        "batch32x35k", 32, 32, 4, 128, (35000, 35000), (64, 64), ("frac", 0.25), 7, 0.01, 1006,
        description="32 requests x 35,000 tokens, Qwen3-30B heads (32q/4kv, d=128), "
                    "64 action queries each, 1% spikes, pool 7, budget 25% per KV head"),
}


# Table 1 shapes (Sec. 8, paged compression kernels): block 16, 8 KV heads, head_dim 128,
# r concurrent requests, each compressed from L to B entries.  The query-head count is not
# given; 32 (G = 4) is the Qwen3 shape with 8 KV heads.  One action query per request: the
# current decode step's query of the streaming scoring.  No pooling (the paper pools
# nothing).
TABLE1_SIZES = ((1024, 512), (2048, 1536), (6144, 4096))
TABLE1_REQS = (1, 4, 16, 64)
for _i, (_r, (_L, _B)) in enumerate([(r, lb) for r in TABLE1_REQS for lb in TABLE1_SIZES]):
    _name = f"table1_r{_r}_{_L // 1024}k"
    CONFIGS[_name] = WorkloadConfig(
        _name, _r, 32, 8, 128, (_L, _L), (1, 1), ("fixed", _B), 1, 0.01, 2000 + _i,
        description=f"Table 1 shape: {_r} request(s) compressed {_L} -> {_B} entries, 32q/8kv "
                    f"heads, d=128, one action query (decode step), no pooling")
del _i, _r, _L, _B, _name


# Full-model compression step: every layer of a 48-layer model (Qwen3-30B-A3B's depth)
# compressed back to back, over one page pool that all layers share.  The requests -- their
# lengths and action-query counts -- are the same in every layer; Q, K, V, spikes and the
# Dirichlet budgets are drawn per layer, and each layer's pages lie at random places in the
# pool.  The pool holds the pages of all layers plus one layer's worth of spare pages, so
# K/V byte offsets run past 2^36.
MODEL_CONFIGS: Dict[str, Tuple[int, WorkloadConfig]] = {
    "model48x32": (48, WorkloadConfig(
        "model48x32", 32, 32, 4, 128, (16000, 64000), (64, 64), ("dirichlet", 0.5, 0.25), 7,
        0.01, 1007,
        description="48 layers x 32 requests, L ~ U[16000, 64000], Qwen3-30B heads "
                    "(32q/4kv, d=128), 64 action queries, 1% spikes, pool 7, per-layer "
                    "Dirichlet(0.5) split of 25% of Hkv*L, one shared page pool")),
}


@dataclass
class Problem:
    """Host-side (numpy) inputs of one compression step over one layer."""
    cfg_name: str
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    page_size: int
    seq_lens: np.ndarray          # int32 [R]
    q_lens: np.ndarray            # int32 [R]
    budgets: np.ndarray           # int32 [R * Hkv]
    q: np.ndarray                 # uint16 (bf16 bits) [sum n, Hq, D]
    kv: np.ndarray                # uint16 (bf16 bits) [2, P, page_size, Hkv, D]
    block_table: np.ndarray       # int32 [R, bt_stride], -1 past each request's pages
    free_pages: np.ndarray        # int32 [num_free]
    sm_scale: float               # float32 value
    pool_window: int
    causal: bool
    k_dense: List[np.ndarray] = field(default_factory=list)   # per request uint16 [L, Hkv, D]
    v_dense: List[np.ndarray] = field(default_factory=list)
    spikes: List[List[np.ndarray]] = field(default_factory=list)  # [r][h] -> token indices

    @property
    def num_reqs(self) -> int:
        return int(self.seq_lens.shape[0])

    @property
    def num_pages(self) -> int:
        return int(self.kv.shape[1])

    @property
    def bt_stride(self) -> int:
        return int(self.block_table.shape[1])

    @property
    def cu_q(self) -> np.ndarray:
        return np.concatenate([[0], np.cumsum(self.q_lens, dtype=np.int64)])


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit pattern (uint16), round to nearest even (finite inputs)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_to_f32(b: np.ndarray) -> np.ndarray:
    """bf16 bit pattern (uint16) -> float32 (exact)."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _draw_lengths(rng, cfg: WorkloadConfig):
    lo, hi = cfg.seq_len
    L = rng.integers(lo, hi + 1, size=cfg.num_reqs).astype(np.int32)
    qlo, qhi = cfg.q_len
    n = rng.integers(qlo, qhi + 1, size=cfg.num_reqs).astype(np.int32)
    return L, n


def _draw_budgets(rng, cfg: WorkloadConfig, L: np.ndarray) -> np.ndarray:
    R, H = cfg.num_reqs, cfg.num_kv_heads
    kind = cfg.budget[0]
    if kind == "fixed":
        b = np.full((R, H), cfg.budget[1], dtype=np.int64)
    elif kind == "frac":
        b = np.repeat(np.floor(cfg.budget[1] * L.astype(np.float64))[:, None], H, axis=1)
    elif kind == "dirichlet":
        alpha, frac = cfg.budget[1], cfg.budget[2]
        w = rng.dirichlet(np.full(H, alpha), size=R)
        b = np.floor(w * H * frac * L.astype(np.float64)[:, None])
        b = np.minimum(b, L[:, None])
    else:
        raise ValueError(kind)
    return b.astype(np.int32).reshape(-1)


def make_problem(name: str, *, seed: Optional[int] = None, overrides: Optional[dict] = None,
                 keep_dense: bool = True) -> Problem:
    """Draw the inputs of workload ``name`` (see CONFIGS), optionally overriding fields."""
    cfg = CONFIGS[name]
    if overrides:
        cfg = WorkloadConfig(**{**cfg.__dict__, **overrides})
    return make_problem_from_config(cfg, seed=seed, keep_dense=keep_dense)


def make_problem_from_config(cfg: WorkloadConfig, *, seed: Optional[int] = None,
                             keep_dense: bool = True) -> Problem:
    ss = np.random.SeedSequence(cfg.seed if seed is None else seed)
    meta_ss, page_ss, budget_ss, *req_ss = ss.spawn(3 + cfg.num_reqs)
    if cfg.num_q_heads % cfg.num_kv_heads:
        raise ValueError("num_q_heads must be a multiple of num_kv_heads")
    L, n = _draw_lengths(np.random.Generator(np.random.PCG64(meta_ss)), cfg)
    budgets = _draw_budgets(np.random.Generator(np.random.PCG64(budget_ss)), cfg, L)
    used = int(((L.astype(np.int64) + PAGE_SIZE - 1) // PAGE_SIZE).sum())
    P = cfg.fixed_pool_pages if cfg.fixed_pool_pages is not None else \
        max(used + 1, int(math.ceil(cfg.pool_factor * used)))
    perm = np.random.Generator(np.random.PCG64(page_ss)).permutation(P).astype(np.int32)
    return _assemble(cfg.name, L, n, budgets, cfg.num_q_heads, cfg.num_kv_heads, cfg.head_dim,
                     cfg.spike_frac, perm, req_ss, cfg.pool_window, cfg.causal, keep_dense)


def make_custom(*, seq_lens, q_lens, num_q_heads, num_kv_heads, head_dim, budgets,
                pool_window=1, spike_frac=0.0, seed=0, pool_factor=2.0, causal=True,
                identity_pages=False, extra_pool_pages=0) -> Problem:
    """Small hand-shaped problems for tests: explicit lengths and budgets.

    ``budgets`` is an int, or an array of R*Hkv ints.  With ``identity_pages`` the pages of
    the requests are laid out contiguously in logical order (no shuffle).
    """
    seq_lens = np.asarray(seq_lens, dtype=np.int32).reshape(-1)
    q_lens = np.asarray(q_lens, dtype=np.int32).reshape(-1)
    R = seq_lens.shape[0]
    ss = np.random.SeedSequence(seed)
    page_ss, *req_ss = ss.spawn(1 + R)
    b = np.asarray(budgets, dtype=np.int64)
    b = np.full(R * num_kv_heads, int(b)) if b.ndim == 0 else b.reshape(-1)
    used = int(((seq_lens.astype(np.int64) + PAGE_SIZE - 1) // PAGE_SIZE).sum())
    P = max(used + 1, int(math.ceil(pool_factor * used))) + extra_pool_pages
    if identity_pages:
        perm = np.arange(P, dtype=np.int32)
    else:
        perm = np.random.Generator(np.random.PCG64(page_ss)).permutation(P).astype(np.int32)
    return _assemble("custom", seq_lens, q_lens, b.astype(np.int32), num_q_heads, num_kv_heads,
                     head_dim, spike_frac, perm, req_ss, pool_window, causal, True)


def _assemble(name, L, n, budgets, Hq, Hkv, D, spike_frac, perm, req_ss, pool_window, causal,
              keep_dense) -> Problem:
    """Draw Q/K/V per request, plant spikes, and scatter K/V into the shuffled page pool."""
    BS = PAGE_SIZE
    R = int(L.shape[0])
    G = Hq // Hkv
    Y = (L.astype(np.int64) + BS - 1) // BS
    used = int(Y.sum())
    P = int(perm.shape[0])
    if P < used:
        raise ValueError("page pool smaller than the pages in use")
    bt_stride = int(max(1, Y.max(initial=0)))
    block_table = np.full((R, bt_stride), -1, dtype=np.int32)
    kv = np.zeros((2, P, BS, Hkv, D), dtype=np.uint16)
    q_all = np.empty((int(n.sum()), Hq, D), dtype=np.uint16)
    k_dense, v_dense, spikes = [], [], []
    off_page, off_q = 0, 0
    for r in range(R):
        rng = np.random.Generator(np.random.PCG64(req_ss[r]))
        Lr, nr, Yr = int(L[r]), int(n[r]), int(Y[r])
        q = bf16_bits(rng.standard_normal((nr, Hq, D), dtype=np.float32))
        k = rng.standard_normal((Lr, Hkv, D), dtype=np.float32)
        v = rng.standard_normal((Lr, Hkv, D), dtype=np.float32)
        qf = bf16_to_f32(q).astype(np.float64)
        sp_r = []
        for h in range(Hkv):
            cnt = int(round(spike_frac * Lr))
            idx = np.sort(rng.choice(Lr, size=cnt, replace=False)) if cnt > 0 else \
                np.zeros(0, dtype=np.int64)
            if cnt > 0 and nr > 0:
                mean = qf[:, h * G:(h + 1) * G, :].reshape(-1, D).mean(axis=0)
                k[idx, h, :] += (3.0 * mean).astype(np.float32)
            sp_r.append(idx.astype(np.int32))
        kb, vb = bf16_bits(k), bf16_bits(v)
        pages = perm[off_page:off_page + Yr]
        block_table[r, :Yr] = pages
        pad = Yr * BS - Lr
        if Yr:
            zpad = np.zeros((pad, Hkv, D), np.uint16)
            kv[0, pages] = np.concatenate([kb, zpad]).reshape(Yr, BS, Hkv, D)
            kv[1, pages] = np.concatenate([vb, zpad]).reshape(Yr, BS, Hkv, D)
        q_all[off_q:off_q + nr] = q
        off_page += Yr
        off_q += nr
        if keep_dense:
            k_dense.append(kb)
            v_dense.append(vb)
        spikes.append(sp_r)
    free_pages = perm[used:].copy()
    sm_scale = float(np.float32(1.0) / np.sqrt(np.float32(D)))
    return Problem(name, Hq, Hkv, D, BS, L.astype(np.int32), n.astype(np.int32),
                   budgets.astype(np.int32), q_all, kv, block_table, free_pages, sm_scale,
                   int(pool_window), bool(causal), k_dense, v_dense, spikes)


# ---------------------------------------------------------------------------------------
# Device-side drawing for the full-size workloads (hundreds of millions of bf16 values).
# Same recipe as above, but the Gaussian draws come from a seeded torch generator on the
# device, so the numbers differ from the numpy path.  Lengths, query counts, budgets and
# the page permutation still come from numpy exactly as in make_problem.
# ---------------------------------------------------------------------------------------
@dataclass
class DeviceProblem:
    cfg_name: str
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    page_size: int
    seq_lens: np.ndarray
    q_lens: np.ndarray
    budgets: np.ndarray
    block_table: np.ndarray       # host copy of the pristine block table
    free_pages: np.ndarray
    sm_scale: float
    pool_window: int
    causal: bool
    q: "object"                   # torch int16 (bf16 bits) [sum n, Hq, D] on the device
    kv: "object"                  # torch int16 (bf16 bits) [2, P, BS, Hkv, D] on the device
    pages: List[np.ndarray] = field(default_factory=list)   # request r's physical pages

    @property
    def num_reqs(self) -> int:
        return int(self.seq_lens.shape[0])

    @property
    def num_pages(self) -> int:
        return int(self.kv.shape[1])

    @property
    def bt_stride(self) -> int:
        return int(self.block_table.shape[1])

    @property
    def cu_q(self) -> np.ndarray:
        return np.concatenate([[0], np.cumsum(self.q_lens, dtype=np.int64)])

    def host_subset(self, reqs: List[int]) -> Problem:
        """Copy requests `reqs` back to the host as a self-contained Problem (their own
        compact page pool, same logical content) -- used to run the oracle on a sample."""
        import torch
        BS, Hkv, D = self.page_size, self.num_kv_heads, self.head_dim
        L = self.seq_lens[reqs].astype(np.int32)
        n = self.q_lens[reqs].astype(np.int32)
        b = self.budgets.reshape(-1, Hkv)[reqs].reshape(-1).astype(np.int32)
        Y = (L.astype(np.int64) + BS - 1) // BS
        used = int(Y.sum())
        P = max(2 * used, used + 1)
        kv = np.zeros((2, P, BS, Hkv, D), np.uint16)
        bt = np.full((len(reqs), int(max(1, Y.max(initial=0)))), -1, np.int32)
        qs, kd, vd = [], [], []
        off = 0
        cu = self.cu_q
        for i, r in enumerate(reqs):
            pg = torch.from_numpy(self.pages[r].astype(np.int64)).to(self.kv.device)
            blk = self.kv.index_select(1, pg).cpu().numpy().view(np.uint16)   # [2, Y, BS, Hkv, D]
            kv[:, off:off + Y[i]] = blk
            bt[i, :Y[i]] = np.arange(off, off + Y[i], dtype=np.int32)
            flat = blk.reshape(2, -1, Hkv, D)[:, :L[i]]
            kd.append(flat[0].copy())
            vd.append(flat[1].copy())
            qs.append(self.q[int(cu[r]):int(cu[r + 1])].cpu().numpy().view(np.uint16))
            off += int(Y[i])
        free = np.arange(off, P, dtype=np.int32)
        q = np.concatenate(qs) if qs else np.zeros((0, self.num_q_heads, D), np.uint16)
        return Problem(self.cfg_name + f"[{len(reqs)} requests]", self.num_q_heads, Hkv, D, BS,
                       L, n, b, q, kv, bt, free, self.sm_scale, self.pool_window, self.causal,
                       kd, vd, [])


@dataclass
class DeviceLayout:
    """The host-side metadata of a device-drawn workload: lengths, budgets, pool size, the
    page permutation (its first `used` pages are the requests' pages in request order, the
    rest the free list) and the per-request random streams of the data."""
    cfg: WorkloadConfig
    seq_lens: np.ndarray
    q_lens: np.ndarray
    budgets: np.ndarray
    num_pages: int
    perm: np.ndarray
    used: int
    req_ss: list

    @property
    def free_pages(self) -> np.ndarray:
        return self.perm[self.used:].copy()

    @property
    def block_table(self) -> np.ndarray:
        """Request r's row: the next ceil(L_r / 16) pages of the permutation (the layout
        _fill_device writes)."""
        Y = (self.seq_lens.astype(np.int64) + PAGE_SIZE - 1) // PAGE_SIZE
        bt = np.full((self.seq_lens.shape[0], int(max(1, Y.max(initial=0)))), -1, np.int32)
        off = 0
        for r, y in enumerate(Y):
            bt[r, :y] = self.perm[off:off + y]
            off += int(y)
        return bt


def device_layout(name: str, *, seed: Optional[int] = None,
                  overrides: Optional[dict] = None) -> DeviceLayout:
    """The metadata make_device_problem draws for workload `name`, without any data."""
    cfg = CONFIGS[name]
    if overrides:
        cfg = WorkloadConfig(**{**cfg.__dict__, **overrides})
    base_seed = cfg.seed if seed is None else seed
    ss = np.random.SeedSequence(base_seed)
    meta_ss, page_ss, budget_ss, *req_ss = ss.spawn(3 + cfg.num_reqs)
    L, n = _draw_lengths(np.random.Generator(np.random.PCG64(meta_ss)), cfg)
    budgets = _draw_budgets(np.random.Generator(np.random.PCG64(budget_ss)), cfg, L)
    Y = (L.astype(np.int64) + PAGE_SIZE - 1) // PAGE_SIZE
    used = int(Y.sum())
    P = cfg.fixed_pool_pages if cfg.fixed_pool_pages is not None else \
        max(used + 1, int(math.ceil(cfg.pool_factor * used)))
    perm = np.random.Generator(np.random.PCG64(page_ss)).permutation(P).astype(np.int32)
    return DeviceLayout(cfg, L, n, budgets, P, perm, used, req_ss)


def make_device_problem(name: str, device="cuda", *, seed: Optional[int] = None,
                        overrides: Optional[dict] = None) -> DeviceProblem:
    """Draw workload `name` directly into device memory (torch, seeded)."""
    import torch
    lay = device_layout(name, seed=seed, overrides=overrides)
    cfg, L, n, budgets, P = lay.cfg, lay.seq_lens, lay.q_lens, lay.budgets, lay.num_pages
    R, Hq, Hkv, D, BS = cfg.num_reqs, cfg.num_q_heads, cfg.num_kv_heads, cfg.head_dim, PAGE_SIZE
    G = Hq // Hkv
    Y = (L.astype(np.int64) + BS - 1) // BS
    bt_stride = int(max(1, Y.max(initial=0)))
    block_table = np.full((R, bt_stride), -1, dtype=np.int32)
    kv = torch.empty((2, P, BS, Hkv, D), dtype=torch.bfloat16, device=device)
    q_all = torch.empty((int(n.sum()), Hq, D), dtype=torch.bfloat16, device=device)
    pages_list = _fill_device(kv, q_all, block_table, lay.perm[:lay.used], L, n, G,
                              cfg.spike_frac, lay.req_ss, device)
    free_pages = lay.free_pages
    sm_scale = float(np.float32(1.0) / np.sqrt(np.float32(D)))
    return DeviceProblem(cfg.name, Hq, Hkv, D, BS, L.astype(np.int32), n.astype(np.int32),
                         budgets.astype(np.int32), block_table, free_pages, sm_scale,
                         cfg.pool_window, cfg.causal, q_all.view(torch.int16),
                         kv.view(torch.int16), pages_list)


def make_device_model(name: str, device="cuda", *, num_layers: Optional[int] = None,
                      overrides: Optional[dict] = None) -> List[DeviceProblem]:
    """Draw the full-model workload `name` (see MODEL_CONFIGS) into one device page pool.

    Returns one DeviceProblem per layer.  They share the kv tensor (all layers' pages and the
    spare pages) and the request lengths; each has its own Q, budgets, block table and page
    lists.  Every layer's free_pages is the pool's spare pages, which is what a layer run on
    its own draws from; a back-to-back run of the layers can instead hand each layer the
    pages the previous layer freed.
    """
    import torch
    layers, cfg = MODEL_CONFIGS[name]
    if num_layers is not None:
        layers = int(num_layers)
    if overrides:
        cfg = WorkloadConfig(**{**cfg.__dict__, **overrides})
    ss = np.random.SeedSequence(cfg.seed)
    meta_ss, page_ss, *layer_ss = ss.spawn(2 + layers)
    R, Hq, Hkv, D, BS = cfg.num_reqs, cfg.num_q_heads, cfg.num_kv_heads, cfg.head_dim, PAGE_SIZE
    G = Hq // Hkv
    L, n = _draw_lengths(np.random.Generator(np.random.PCG64(meta_ss)), cfg)
    Y = (L.astype(np.int64) + BS - 1) // BS
    used = int(Y.sum())
    P = (layers + 1) * used
    perm = np.random.Generator(np.random.PCG64(page_ss)).permutation(P).astype(np.int32)
    spare = perm[layers * used:].copy()
    bt_stride = int(max(1, Y.max(initial=0)))
    kv = torch.empty((2, P, BS, Hkv, D), dtype=torch.bfloat16, device=device)
    sm_scale = float(np.float32(1.0) / np.sqrt(np.float32(D)))
    out = []
    for l in range(layers):
        budget_ss, *req_ss = layer_ss[l].spawn(1 + R)
        budgets = _draw_budgets(np.random.Generator(np.random.PCG64(budget_ss)), cfg, L)
        block_table = np.full((R, bt_stride), -1, dtype=np.int32)
        q_all = torch.empty((int(n.sum()), Hq, D), dtype=torch.bfloat16, device=device)
        pages_list = _fill_device(kv, q_all, block_table, perm[l * used:(l + 1) * used], L, n,
                                  G, cfg.spike_frac, req_ss, device)
        out.append(DeviceProblem(f"{cfg.name}[layer {l}]", Hq, Hkv, D, BS, L.astype(np.int32),
                                 n.astype(np.int32), budgets.astype(np.int32), block_table,
                                 spare, sm_scale, cfg.pool_window, cfg.causal,
                                 q_all.view(torch.int16), kv.view(torch.int16), pages_list))
    return out


def _fill_device(kv, q_all, block_table, pages_in_use, L, n, G, spike_frac, req_ss,
                 device) -> List[np.ndarray]:
    """Draw each request's Q, K, V on the device (one torch generator per request, seeded
    from its SeedSequence), plant the spike keys, and scatter K/V into the pages
    `pages_in_use` in request order; fills block_table and q_all, returns the page lists."""
    import torch
    BS = PAGE_SIZE
    _, _, _, Hkv, D = kv.shape
    Hq = q_all.shape[1]
    Y = (L.astype(np.int64) + BS - 1) // BS
    pages_list = []
    off_page, off_q = 0, 0
    for r in range(int(L.shape[0])):
        Lr, nr, Yr = int(L[r]), int(n[r]), int(Y[r])
        gen = torch.Generator(device=device)
        gen.manual_seed(int(req_ss[r].generate_state(1, dtype=np.uint64)[0] & 0x7FFFFFFFFFFFFFFF))
        q = torch.randn((nr, Hq, D), generator=gen, device=device).to(torch.bfloat16)
        k = torch.randn((Yr * BS, Hkv, D), generator=gen, device=device)
        v = torch.randn((Yr * BS, Hkv, D), generator=gen, device=device)
        k[Lr:] = 0
        v[Lr:] = 0
        cnt = int(round(spike_frac * Lr))
        if cnt > 0 and nr > 0:
            qf = q.float()
            for h in range(Hkv):
                mean = qf[:, h * G:(h + 1) * G, :].reshape(-1, D).double().mean(0).float()
                idx = torch.randperm(Lr, generator=gen, device=device)[:cnt]
                k[idx, h, :] += 3.0 * mean
        pages = pages_in_use[off_page:off_page + Yr]
        block_table[r, :Yr] = pages
        pg = torch.from_numpy(pages.astype(np.int64)).to(device)
        kv[0].index_copy_(0, pg, k.to(torch.bfloat16).view(Yr, BS, Hkv, D))
        kv[1].index_copy_(0, pg, v.to(torch.bfloat16).view(Yr, BS, Hkv, D))
        q_all[off_q:off_q + nr] = q
        pages_list.append(pages.copy())
        off_page += Yr
        off_q += nr
        del k, v
    return pages_list
