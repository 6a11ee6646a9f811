"""Seeded synthetic inputs for the OasisKV decode-time path.

This module draws random numbers, rounds them to bf16 and lays them out in KV
pages. It holds none of the method's arithmetic (no summaries, scores,
selection, staging or attention), so both the HIP path (through the tests and
the benchmark) and the CPU oracle can consume what it returns.

Workload recipes (the paper evaluates on models and datasets that are not
available here; these synthetic inputs stand in for them):

* ``c1`` parity: 1 request, 32 query / 8 KV heads, head_dim 128, block 16,
  context 8,192, 4 draft tokens, budget 2,048. K, V ~ N(0, 1); 8 planted
  blocks per KV head whose keys get ``+3 * sign(sum of that head's draft
  query rows)`` per coordinate.
* ``c2``: 32 requests, contexts uniform in [16K, 32K]; per (request, KV head)
  block keys scaled by ``clip((rank / max(1, 0.05 * n_cand)) ** -1.1, 0.25, 4)``
  with ``rank`` a random 1-based permutation of the candidate blocks (a
  Zipf(1.1)-like skew of block key norms).
* ``c3`` reasoning-style: 32 layers, 64 requests, context ``1024 + U[4096,
  16384]``, c2's key distribution, queries follow AR(1) over steps
  (``q_s = 0.9 q_{s-1} + 0.436 eps``), one token appended per step.
* ``c4`` long context: 8 requests x 131,072 tokens (8,192 blocks), K, V ~
  N(0, 1), 82 planted blocks (1 % of 8,191 candidates) per (request, KV head).
* ``c5`` large GQA: 16 requests x 65,536 tokens, 64 query / 8 KV heads, block
  32, 8 draft tokens, budget 4,096; keys and values are ``mu + N(0, 1)`` with a
  per-(request, KV head) mean ``mu ~ N(0, 0.5^2)`` per coordinate.

Seeds: configuration ``c`` uses base ``20260000 + 100 c``; the streams are
``base+1`` keys/values (per request, head), ``base+2`` queries (per request,
step), ``base+3`` context lengths, ``base+4`` planted ids (per request, head),
``base+5`` Zipf permutations (per request, head), ``base+6`` the physical page
permutation. Values are drawn in float32 and rounded to bf16 (round to nearest
even), so every consumer sees the same bf16 bits.
"""
from __future__ import annotations

import dataclasses
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

__all__ = [
    "Config", "CONFIGS", "config", "Workload", "make_workload",
    "f32_to_bf16_bits", "bf16_bits_to_f32",
]


# ----------------------------------------------------------------------------
# bf16 encoding (round to nearest even), done with integer bit operations
# ----------------------------------------------------------------------------

def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (nearest, ties to even); returns uint16 bits."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    if not np.all(np.isfinite(x)):
        raise ValueError("bf16 encoding of non-finite input")
    u = x.view(np.uint32)
    bias = np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Decode bf16 bits (uint16) to float32 (exact)."""
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


# ----------------------------------------------------------------------------
# Configurations
# ----------------------------------------------------------------------------

@dataclasses.dataclass(frozen=True)
class Config:
    name: str
    index: int                 # seed index c (base seed 20260000 + 100 c)
    num_reqs: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    block_size: int
    num_draft: int             # D draft (lookahead) tokens; T = 1 + D query rows
    budget: int                # KV token budget; K = budget // block_size
    ctx_kind: str              # "fixed" | "uniform" | "prompt_uniform"
    ctx_args: tuple
    key_dist: str              # "planted" | "zipf" | "mean_offset"
    n_planted: int = 0         # planted heavy-hitter blocks per (request, KV head)
    planted_frac: float = 0.0  # if > 0: n_planted = round(frac * n_cand)
    layers: int = 1
    steps: int = 1
    ar_queries: bool = False   # AR(1) queries across steps
    grow_per_step: int = 0     # tokens appended per decode step

    @property
    def T(self) -> int:
        return 1 + self.num_draft

    @property
    def G(self) -> int:
        return self.num_q_heads // self.num_kv_heads

    @property
    def K(self) -> int:
        return self.budget // self.block_size

    @property
    def base_seed(self) -> int:
        return 20260000 + 100 * self.index

    def replace(self, **kw) -> "Config":
        return dataclasses.replace(self, **kw)


CONFIGS = {
    "c1": Config("c1", 1, 1, 32, 8, 128, 16, 4, 2048, "fixed", (8192,), "planted", n_planted=8),
    "c2": Config("c2", 2, 32, 32, 8, 128, 16, 4, 2048, "uniform", (16384, 32768), "zipf"),
    "c3": Config("c3", 3, 64, 32, 8, 128, 16, 4, 2048, "prompt_uniform", (1024, 4096, 16384), "zipf",
                 layers=32, steps=64, ar_queries=True, grow_per_step=1),
    "c4": Config("c4", 4, 8, 32, 8, 128, 16, 4, 2048, "fixed", (131072,), "planted", planted_frac=0.01),
    "c5": Config("c5", 5, 16, 64, 8, 128, 32, 8, 4096, "fixed", (65536,), "mean_offset"),
}


def config(name: str, **overrides) -> Config:
    return CONFIGS[name].replace(**overrides) if overrides else CONFIGS[name]


def _rng(*key: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([int(k) for k in key])))


# ----------------------------------------------------------------------------
# Workload
# ----------------------------------------------------------------------------

def _num_threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


class Workload:
    """All inputs of one configuration: lengths, queries, paged host K/V."""

    def __init__(self, cfg: Config):
        self.cfg = cfg
        c = cfg
        if c.num_q_heads % c.num_kv_heads:
            raise ValueError("num_q_heads must be a multiple of num_kv_heads")
        rng = _rng(c.base_seed + 3)
        if c.ctx_kind == "fixed":
            lens = np.full(c.num_reqs, c.ctx_args[0], dtype=np.int64)
        elif c.ctx_kind == "uniform":
            lo, hi = c.ctx_args
            lens = rng.integers(lo, hi + 1, size=c.num_reqs)
        elif c.ctx_kind == "prompt_uniform":
            p, lo, hi = c.ctx_args
            lens = p + rng.integers(lo, hi + 1, size=c.num_reqs)
        else:
            raise ValueError(c.ctx_kind)
        # context length at step 0; tokens appended later are generated up front
        self.ctx0 = lens.astype(np.int32)
        self.max_steps = max(1, c.steps)
        self.alloc_len = (self.ctx0 + c.grow_per_step * (self.max_steps - 1)).astype(np.int64)
        B = c.block_size
        self.alloc_blocks = (self.alloc_len + B - 1) // B
        self.NBmax = int(self.alloc_blocks.max())
        self.NPhys = int(self.alloc_blocks.sum())
        perm = _rng(c.base_seed + 6).permutation(self.NPhys).astype(np.int32)
        self.block_table = np.full((c.num_reqs, self.NBmax), -1, dtype=np.int32)
        off = 0
        for r in range(c.num_reqs):
            nb = int(self.alloc_blocks[r])
            self.block_table[r, :nb] = perm[off:off + nb]
            off += nb
        self._q_cache: dict[int, np.ndarray] = {}
        self._q_state: np.ndarray | None = None
        self._q_state_step = -1

    # -- lengths ------------------------------------------------------------
    def ctx_len(self, step: int = 0) -> np.ndarray:
        return (self.ctx0 + self.cfg.grow_per_step * step).astype(np.int32)

    def local_block_pages(self, steps: int) -> tuple[np.ndarray, np.ndarray]:
        """Pages of the blocks that are a request's local block at some step in [0, steps).

        Returns the host page ids of those blocks (int64, in request and block
        order) and a [R][NBmax] int32 table that maps each of them to its index
        in that list (-1 elsewhere): the layout of a small device-resident copy
        of the active blocks, which a model would write on the GPU.
        """
        c = self.cfg
        B = c.block_size
        first = self.ctx_len(0).astype(np.int64)
        last = self.ctx_len(max(0, steps - 1)).astype(np.int64)
        table = np.full((c.num_reqs, self.NBmax), -1, dtype=np.int32)
        pages = []
        for r in range(c.num_reqs):
            if last[r] <= 0:
                continue
            b0 = max(0, int(first[r] - 1) // B)
            b1 = int(last[r] - 1) // B
            for b in range(b0, b1 + 1):
                table[r, b] = len(pages)
                pages.append(int(self.block_table[r, b]))
        return np.array(pages, dtype=np.int64), table

    def n_cand0(self, r: int) -> int:
        B = self.cfg.block_size
        return int((int(self.ctx0[r]) + B - 1) // B - 1)

    # -- queries ------------------------------------------------------------
    def _eps(self, r: int, step: int, layer: int = 0) -> np.ndarray:
        c = self.cfg
        key = (c.base_seed + 2, r, step) if layer == 0 else (c.base_seed + 2, r, step, layer)
        return _rng(*key).standard_normal((c.T, c.num_q_heads, c.head_dim), dtype=np.float32)

    def layer_queries(self, layer: int, steps: int) -> list[np.ndarray]:
        """bf16 query bits of ``steps`` consecutive decode steps of one more layer.

        Each layer has its own stream of draws; with ``ar_queries`` they follow
        the same AR(1) recipe over steps.
        """
        c = self.cfg
        state = np.stack([self._eps(r, 0, layer) for r in range(c.num_reqs)])
        out = [f32_to_bf16_bits(state)]
        for s in range(1, steps):
            eps = np.stack([self._eps(r, s, layer) for r in range(c.num_reqs)])
            state = (np.float32(0.9) * state + np.float32(0.436) * eps).astype(np.float32) if c.ar_queries else eps
            out.append(f32_to_bf16_bits(state))
        return out

    def queries_f32(self, step: int = 0) -> np.ndarray:
        """float32 query state [R][T][Hq][d] at ``step`` (before bf16 rounding)."""
        c = self.cfg
        if not c.ar_queries:
            return np.stack([self._eps(r, step) for r in range(c.num_reqs)])
        if self._q_state is None or self._q_state_step > step:
            self._q_state = np.stack([self._eps(r, 0) for r in range(c.num_reqs)])
            self._q_state_step = 0
        while self._q_state_step < step:
            s = self._q_state_step + 1
            eps = np.stack([self._eps(r, s) for r in range(c.num_reqs)])
            self._q_state = (np.float32(0.9) * self._q_state + np.float32(0.436) * eps).astype(np.float32)
            self._q_state_step = s
        return self._q_state.copy()

    def queries(self, step: int = 0) -> np.ndarray:
        """bf16 bits [R][T][Hq][d]: row 0 = verify token, rows 1..D = draft tokens."""
        if step not in self._q_cache:
            self._q_cache[step] = f32_to_bf16_bits(self.queries_f32(step))
        return self._q_cache[step]

    # -- keys / values ------------------------------------------------------
    def planted_ids(self, r: int, h: int) -> np.ndarray:
        c = self.cfg
        n_cand = self.n_cand0(r)
        n = c.n_planted if c.planted_frac <= 0 else int(round(c.planted_frac * n_cand))
        n = min(n, n_cand)
        if c.key_dist != "planted" or n <= 0:
            return np.zeros(0, dtype=np.int64)
        return np.sort(_rng(c.base_seed + 4, r, h).choice(n_cand, size=n, replace=False))

    def request_head_kv(self, r: int, h: int) -> tuple[np.ndarray, np.ndarray]:
        """bf16 bits K, V of request ``r`` / KV head ``h``: [alloc_len][d] each."""
        c = self.cfg
        L = int(self.alloc_len[r])
        d, B = c.head_dim, c.block_size
        rng = _rng(c.base_seed + 1, r, h)
        if c.key_dist == "mean_offset":
            mu_k = (0.5 * rng.standard_normal(d, dtype=np.float32)).astype(np.float32)
            mu_v = (0.5 * rng.standard_normal(d, dtype=np.float32)).astype(np.float32)
        k = rng.standard_normal((L, d), dtype=np.float32)
        v = rng.standard_normal((L, d), dtype=np.float32)
        n_cand = self.n_cand0(r)
        if c.key_dist == "planted":
            ids = self.planted_ids(r, h)
            if ids.size:
                q = bf16_bits_to_f32(self.queries(0)[r]).astype(np.float64)  # [T][Hq][d]
                rows = q[1:, h * c.G:(h + 1) * c.G, :].reshape(-1, d)
                shift = (3.0 * np.sign(rows.sum(axis=0))).astype(np.float32)
                for b in ids:
                    k[b * B:(b + 1) * B] += shift
        elif c.key_dist == "zipf":
            rank = _rng(c.base_seed + 5, r, h).permutation(n_cand).astype(np.float64) + 1.0
            scale = np.clip((rank / max(1.0, 0.05 * n_cand)) ** -1.1, 0.25, 4.0).astype(np.float32)
            k[:n_cand * B] *= np.repeat(scale, B)[:, None]
        elif c.key_dist == "mean_offset":
            k += mu_k
            v += mu_v
        else:
            raise ValueError(c.key_dist)
        return f32_to_bf16_bits(k), f32_to_bf16_bits(v)

    def request_kv(self, r: int) -> tuple[np.ndarray, np.ndarray]:
        """bf16 bits K, V of request ``r``: [Hkv][alloc_len][d] each."""
        ks, vs = zip(*(self.request_head_kv(r, h) for h in range(self.cfg.num_kv_heads)))
        return np.stack(ks), np.stack(vs)

    def fill_paged(self, host_k: np.ndarray | None = None, host_v: np.ndarray | None = None,
                   threads: int | None = None) -> tuple[np.ndarray, np.ndarray]:
        """Write every request's K/V into physical pages [NPhys][Hkv][B][d] (HTD order).

        ``host_k``/``host_v`` may be caller-provided uint16 buffers (for example
        views of pinned memory); the unused tail of a request's last page is
        zero.
        """
        c = self.cfg
        shape = (self.NPhys, c.num_kv_heads, c.block_size, c.head_dim)
        if host_k is None:
            host_k = np.empty(shape, dtype=np.uint16)
        if host_v is None:
            host_v = np.empty(shape, dtype=np.uint16)
        assert host_k.shape == shape and host_v.shape == shape
        B, d = c.block_size, c.head_dim

        def one(rh):
            r, h = rh
            k, v = self.request_head_kv(r, h)
            L = k.shape[0]
            nb = int(self.alloc_blocks[r])
            pad = nb * B - L
            if pad:
                k = np.concatenate([k, np.zeros((pad, d), np.uint16)])
                v = np.concatenate([v, np.zeros((pad, d), np.uint16)])
            pages = self.block_table[r, :nb]
            host_k[pages, h] = k.reshape(nb, B, d)
            host_v[pages, h] = v.reshape(nb, B, d)

        jobs = [(r, h) for r in range(c.num_reqs) for h in range(c.num_kv_heads)]
        n = threads or _num_threads()
        if n == 1 or len(jobs) == 1:
            for j in jobs:
                one(j)
        else:
            with ThreadPoolExecutor(n) as ex:
                list(ex.map(one, jobs))
        return host_k, host_v


def make_workload(name_or_cfg, **overrides) -> Workload:
    cfg = name_or_cfg if isinstance(name_or_cfg, Config) else config(name_or_cfg, **overrides)
    if overrides and isinstance(name_or_cfg, Config):
        cfg = cfg.replace(**overrides)
    return Workload(cfg)


def random_scores(seed: int, shape, n_distinct: int | None = None) -> np.ndarray:
    """float32 scores for selection tests; ``n_distinct`` forces many exact ties."""
    rng = _rng(seed)
    if n_distinct:
        vals = rng.standard_normal(n_distinct).astype(np.float32)
        return vals[rng.integers(0, n_distinct, size=shape)]
    return rng.standard_normal(shape).astype(np.float32) * np.float32(50.0)


def random_bf16(seed: int, shape, scale: float = 1.0, mean: float = 0.0) -> np.ndarray:
    """bf16 bits of N(mean, scale^2) values."""
    x = _rng(seed).standard_normal(shape, dtype=np.float32) * np.float32(scale) + np.float32(mean)
    return f32_to_bf16_bits(x)


def random_selection(seed: int, n_cand, k: int, prev=None, keep_frac: float = 0.6):
    """Ascending block-id selections [R][H][k] (-1 padded) and counts [R][H].

    ``n_cand`` holds the candidate count of every request. With ``prev``, about
    ``keep_frac`` of each previous selection is kept, which makes later staging
    steps deltas rather than cold fills.
    """
    rng = _rng(seed)
    n_cand = np.asarray(n_cand)
    R = n_cand.shape[0]
    H = prev[0].shape[1] if prev is not None else None
    if H is None:
        raise ValueError("pass prev=(sel, cnt) or use random_selection_h")
    return _random_selection(rng, n_cand, H, k, prev, keep_frac)


def random_selection_h(seed: int, n_cand, num_heads: int, k: int):
    return _random_selection(_rng(seed), np.asarray(n_cand), num_heads, k, None, 0.0)


def _random_selection(rng, n_cand, H, k, prev, keep_frac):
    R = n_cand.shape[0]
    sel = np.full((R, H, k), -1, np.int32)
    cnt = np.zeros((R, H), np.int32)
    for r in range(R):
        nc = int(n_cand[r])
        m = min(k, nc)
        for h in range(H):
            if prev is not None and m:
                old = prev[0][r, h, :prev[1][r, h]]
                keep = old[rng.random(old.size) < keep_frac] if old.size else old
                rest = np.setdiff1d(np.arange(nc), keep)
                extra = rng.choice(rest, size=m - min(m, keep.size), replace=False) if m > keep.size else []
                chosen = np.sort(np.concatenate([keep[:m], np.asarray(extra, dtype=keep.dtype)]).astype(np.int32))
            else:
                chosen = np.sort(rng.choice(nc, size=m, replace=False)).astype(np.int32) if m else np.zeros(0, np.int32)
            sel[r, h, :m] = chosen
            cnt[r, h] = m
    return sel, cnt
