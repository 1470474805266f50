"""Seeded synthetic decode workloads for the sparse-KV hot path.

This module only draws inputs: context lengths, queries, keys/values, planted
heavy blocks, resident hot sets, free slot lists and per-request budgets.  It
holds none of the path's arithmetic (no digest, score, selection, recall or
attention) and imports neither the GPU binding nor the oracle, so both sides
can consume the same inputs.

Shapes follow the paper's decode workloads: block size 16, head_dim 128,
bf16 KV, a 2,048-token hot budget of 16 sink + 128 local + 1,904 middle
tokens (Sec. 5 setup), long contexts of 32K-256K tokens with lognormal-like
raggedness (Sec. 5 workloads).  Five named presets are provided; see
``preset``.

Host KV store layout (one block = all KV heads, K then V):
    K part  [Hkv][bs][d]   token-major
    V part  [Hkv][d][bs]   channel-major
so one block is 2*Hkv*bs*d 16-bit elements; global block b of request r is
blk_off[r] + j.  Tokens past the end of a request's context inside its last
block are zero.

Planting.  Heavy blocks are planted in the keys of one KV head (the
retrieval head ``solo_kv_head``).  A heavy block made of the query plus
0.1 N(0,1) noise is built along the scaled direction of that head's GQA-group
mean query: every valid token of a
heavy block gets k = lam * qbar / |qbar|^2 + 0.1 * eps with lam = 2*d, so the
group-mean logit of a heavy token is lam (before noise).  ``plant_mode =
"literal"`` instead uses k = q_lead + 0.1 * eps, with q_lead the first query
head of the group.  Other KV heads keep N(0,1) keys.
"""
from __future__ import annotations

import math
import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field
from typing import Callable, Optional

import numpy as np

F16 = 0
BF16 = 1
DTYPE_CODES = {"f16": F16, "bf16": BF16}


# --------------------------------------------------------------------------- rounding


def round_to_dtype(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round float32 values to fp16 / bf16 (round-to-nearest-even); return uint16 bits."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    if dtype == "f16":
        return x.astype(np.float16).view(np.uint16)
    u = x.view(np.uint32).copy()
    t = u >> 16
    t &= 1
    t += 0x7FFF
    u += t
    u >>= 16
    return u.astype(np.uint16)


def to_float(bits: np.ndarray, dtype: str) -> np.ndarray:
    """16-bit patterns -> float32 values (exact)."""
    bits = np.asarray(bits, dtype=np.uint16)
    if dtype == "f16":
        return bits.view(np.float16).astype(np.float32)
    return (bits.astype(np.uint32) << 16).view(np.float32)


# --------------------------------------------------------------------------- specs


@dataclass
class Spec:
    """Everything that defines one synthetic layer-step workload."""

    name: str
    batch: int
    ctx_lens: list  # per-request context tokens
    num_q_heads: int = 32
    num_kv_heads: int = 8
    head_dim: int = 128
    block_size: int = 16
    dtype: str = "bf16"
    n_sink: int = 1  # forced sink blocks
    n_local: int = 8  # forced local blocks
    k_mid: list = field(default_factory=list)  # per-request middle budget (blocks)
    resident_frac: float = 0.10
    heavy: list = field(default_factory=list)  # per-request sorted heavy block indices
    planted: bool = True
    plant_mode: str = "scaled"
    free_order: str = "ascending"  # or "shuffled"
    slack_slots: int = 0  # extra free slots beyond the worst case
    n_free_override: Optional[int] = None  # force a small free list (pool exhaustion)
    resident_key: int = 0  # stream of the resident sample (layers sharing a store differ here)


@dataclass
class Workload:
    spec: Spec
    seed: int
    B: int
    Hq: int
    Hkv: int
    d: int
    bs: int
    dtype: str
    dtype_code: int
    ctx_len: np.ndarray  # int32 [B]
    n_blocks: np.ndarray  # int64 [B]
    blk_off: np.ndarray  # int64 [B+1]
    q: np.ndarray  # uint16 [B, Hq, d]
    kv: np.ndarray  # uint16 [total_blocks, 2*Hkv*bs*d]
    k_mid: np.ndarray  # int32 [B]
    n_sink: int
    n_local: int
    k_max: int
    max_blocks: int
    table0: np.ndarray  # int32 [B, max_blocks], -1 = not resident
    resident_blocks: np.ndarray  # int64 global block ids, slot i holds resident_blocks[i]
    free_slots: np.ndarray  # int32 [n_free]
    n_slots: int
    solo_kv_head: int
    heavy: list  # per-request int64 arrays of heavy block indices
    sm_scale: float

    @property
    def total_blocks(self) -> int:
        return int(self.blk_off[-1])

    @property
    def elems_per_block(self) -> int:
        return 2 * self.Hkv * self.bs * self.d

    @property
    def unit_bytes(self) -> int:
        return 2 * self.elems_per_block

    @property
    def G(self) -> int:
        return self.Hq // self.Hkv

    def shape_tuple(self):
        return (self.Hq, self.Hkv, self.d, self.bs, self.dtype_code)


# --------------------------------------------------------------------------- presets


def _forced_counts(bs: int):
    """Sink 16 tokens and local 128 tokens, as whole blocks (Sec. 5 setup)."""
    return -(-16 // bs), -(-128 // bs)


def _middle_budget(budget_tokens: int, bs: int) -> int:
    n_sink, n_local = _forced_counts(bs)
    return budget_tokens // bs - n_sink - n_local


def preset(config_id: int, *, ctx_scale: float = 1.0, batch: Optional[int] = None, layer: int = 0,
           planted: bool = True, free_order: str = "ascending", n_stores: int = 4) -> tuple:
    """(Spec, seed) of one of the five named workloads.

    1: 1 request x 4096 tokens, bs 16, 32/8 heads, fp16, middle budget 16 blocks,
       25% resident, 8 heavy blocks.
    2: 8 x 32K, bf16, 2048-token budget, 10% resident, 32 heavy blocks/request.
    3: 32 requests, contexts uniform in [64K, 128K] (ragged), 4096-token budget,
       5% resident, 32 heavy/request.
    4: one layer of a 32-layer step: 16 x 64K, per-request budgets lognormal
       (sigma 1) around 2048 tokens clipped to [256, 8192], 10% resident; layer l
       shares host store l % n_stores (keys, values, query) with other layers.
    5: 4 x 256K, bs 32, 64/8 heads, 8192-token budget, 3% resident, heavy blocks
       in 4 runs of 16 plus 64 singletons.
    ctx_scale shrinks contexts (and batch may be overridden) for oracle-sized runs.
    """
    seed = 1000 + config_id
    rng = np.random.default_rng([seed, layer, 0])
    if config_id == 1:
        B = batch or 1
        ctx = [max(1, int(4096 * ctx_scale))] * B
        spec = Spec("cfg1", B, ctx, 32, 8, 128, 16, "f16", resident_frac=0.25)
        spec.k_mid = [16] * B
        nh = [8] * B
    elif config_id == 2:
        B = batch or 8
        ctx = [max(1, int(32768 * ctx_scale))] * B
        spec = Spec("cfg2", B, ctx, 32, 8, 128, 16, "bf16", resident_frac=0.10)
        spec.k_mid = [_middle_budget(2048, 16)] * B
        nh = [32] * B
    elif config_id == 3:
        B = batch or 32
        lo, hi = int(65536 * ctx_scale), int(131072 * ctx_scale)
        ctx = [int(x) for x in rng.integers(lo, hi + 1, size=B)]
        spec = Spec("cfg3", B, ctx, 32, 8, 128, 16, "bf16", resident_frac=0.05)
        spec.k_mid = [_middle_budget(4096, 16)] * B
        nh = [32] * B
    elif config_id == 4:
        # layer l reads host store l % n_stores (keys, values, query, planted blocks);
        # its budgets and resident set are its own
        store = layer % n_stores
        rng = np.random.default_rng([seed, store, 0])
        B = batch or 16
        ctx = [max(1, int(65536 * ctx_scale))] * B
        spec = Spec(f"cfg4_l{layer}", B, ctx, 32, 8, 128, 16, "bf16", resident_frac=0.10)
        z = np.random.default_rng([seed, 1000 + layer]).standard_normal(B)
        budgets = np.clip(2048.0 * np.exp(z), 256, 8192)
        spec.k_mid = [int(b) // 16 - 9 for b in budgets]
        spec.resident_key = layer
        nh = [32] * B
    elif config_id == 5:
        B = batch or 4
        ctx = [max(1, int(262144 * ctx_scale))] * B
        spec = Spec("cfg5", B, ctx, 64, 8, 128, 32, "bf16", resident_frac=0.03)
        spec.n_sink, spec.n_local = _forced_counts(32)
        spec.k_mid = [_middle_budget(8192, 32)] * B
        nh = None
    else:
        raise ValueError(f"unknown config {config_id}")
    if config_id != 5:
        spec.n_sink, spec.n_local = _forced_counts(spec.block_size)
    spec.planted = planted
    spec.free_order = free_order
    bs = spec.block_size
    heavy = []
    for r in range(spec.batch):
        n = -(-spec.ctx_lens[r] // bs)
        lo_m, hi_m = spec.n_sink, n - spec.n_local
        if config_id == 5:
            heavy.append(_clustered_heavy(rng, lo_m, hi_m, runs=4, run_len=16, singles=64))
        else:
            m = max(0, hi_m - lo_m)
            h = min(nh[r], m)
            heavy.append(np.sort(rng.choice(m, size=h, replace=False)).astype(np.int64) + lo_m)
    spec.heavy = heavy
    return spec, seed + 7919 * (layer % n_stores if config_id == 4 else layer)


def _clustered_heavy(rng, lo: int, hi: int, runs: int, run_len: int, singles: int) -> np.ndarray:
    """Runs of contiguous heavy blocks plus singletons, all separated by >= 1 block."""
    items = [run_len] * runs + [1] * singles
    n_items = len(items)
    span = hi - lo
    need = sum(items) + (n_items - 1)
    if span < need:  # scaled-down contexts: shrink to what fits
        k = max(0, span // 3)
        return np.sort(rng.choice(span, size=min(k, span), replace=False)).astype(np.int64) + lo
    order = rng.permutation(n_items)
    slack = span - need
    cuts = np.sort(rng.integers(0, slack + 1, size=n_items))
    gaps = np.diff(np.concatenate([[0], cuts]))  # extra gap before each item
    out = []
    pos = lo
    for i, idx in enumerate(order):
        pos += int(gaps[i]) + (1 if i > 0 else 0)
        out.extend(range(pos, pos + items[idx]))
        pos += items[idx]
    return np.array(out, np.int64)


def custom(name: str, ctx_lens, *, Hq=32, Hkv=8, d=128, bs=16, dtype="bf16", k_mid=8, n_sink=1,
           n_local=2, resident_frac=0.25, heavy_per_req=4, planted=True, free_order="ascending",
           seed=7, slack_slots=0, n_free_override=None) -> tuple:
    """Spec for a hand-sized workload (edge cases, ragged tails, ties)."""
    rng = np.random.default_rng([seed, 99])
    B = len(ctx_lens)
    spec = Spec(name, B, [int(x) for x in ctx_lens], Hq, Hkv, d, bs, dtype, n_sink, n_local,
                resident_frac=resident_frac, planted=planted, free_order=free_order,
                slack_slots=slack_slots, n_free_override=n_free_override)
    spec.k_mid = list(k_mid) if isinstance(k_mid, (list, tuple, np.ndarray)) else [int(k_mid)] * B
    heavy = []
    for r in range(B):
        n = -(-spec.ctx_lens[r] // bs)
        lo_m, hi_m = n_sink, n - n_local
        m = max(0, hi_m - lo_m)
        h = min(heavy_per_req, m)
        heavy.append(np.sort(rng.choice(m, size=h, replace=False)).astype(np.int64) + lo_m if h else
                     np.zeros(0, np.int64))
    spec.heavy = heavy
    return spec, seed


# --------------------------------------------------------------------------- generation


def _fill_chunk(out: np.ndarray, seed_key, dtype: str):
    rng = np.random.default_rng(seed_key)
    tmp = rng.standard_normal(out.size, dtype=np.float32)
    out.reshape(-1)[:] = round_to_dtype(tmp, dtype)


def generate(spec: Spec, seed: int, *, kv_alloc: Optional[Callable] = None, threads: Optional[int] = None,
             store_key: int = 0, reuse_kv: Optional["Workload"] = None) -> Workload:
    """Draw a full workload.  ``kv_alloc(shape, np.uint16)`` may return a view of pinned host
    memory so the store is generated in place.  ``store_key`` selects the key/value stream.
    ``reuse_kv``: a workload drawn with the same seed, contexts and heavy blocks whose store,
    query and retrieval head are taken as they are (layers sharing one host store)."""
    B = spec.batch
    Hq, Hkv, d, bs, dtype = spec.num_q_heads, spec.num_kv_heads, spec.head_dim, spec.block_size, spec.dtype
    if Hq % Hkv:
        raise ValueError("num_q_heads must be a multiple of num_kv_heads")
    G = Hq // Hkv
    rng = np.random.default_rng([seed, 1])
    ctx_len = np.asarray(spec.ctx_lens, np.int32)
    n_blocks = (ctx_len.astype(np.int64) + bs - 1) // bs
    blk_off = np.zeros(B + 1, np.int64)
    blk_off[1:] = np.cumsum(n_blocks)
    total = int(blk_off[-1])
    E = 2 * Hkv * bs * d

    q = round_to_dtype(rng.standard_normal((B, Hq, d), dtype=np.float32), dtype).reshape(B, Hq, d)
    solo = int(rng.integers(Hkv))
    if reuse_kv is not None:
        if reuse_kv.seed != seed or not np.array_equal(reuse_kv.blk_off, blk_off):
            raise ValueError("reuse_kv must come from the same seed and contexts")
        return _finish(spec, seed, B, Hq, Hkv, d, bs, dtype, ctx_len, n_blocks, blk_off, reuse_kv.q, reuse_kv.kv,
                       reuse_kv.solo_kv_head)

    kv = kv_alloc((total, E), np.uint16) if kv_alloc else np.empty((total, E), np.uint16)
    # bulk N(0,1) keys/values, chunked by request and block range with independent streams
    CH = 256
    jobs = []
    for r in range(B):
        for c0 in range(0, int(n_blocks[r]), CH):
            c1 = min(int(n_blocks[r]), c0 + CH)
            b0, b1 = int(blk_off[r]) + c0, int(blk_off[r]) + c1
            jobs.append((b0, b1, [seed, store_key, r, c0]))
    nthreads = threads or min(16, os.cpu_count() or 1)
    if jobs:
        with ThreadPoolExecutor(max_workers=nthreads) as ex:
            list(ex.map(lambda jb: _fill_chunk(kv[jb[0]:jb[1]], jb[2], dtype), jobs))

    kv5 = kv.reshape(total, 2, Hkv, bs * d)
    # planting in the retrieval head's keys
    if spec.planted:
        qf = to_float(q, dtype).astype(np.float64)
        prng = np.random.default_rng([seed, store_key, 1 << 20])
        for r in range(B):
            hv = np.asarray(spec.heavy[r], np.int64)
            if hv.size == 0:
                continue
            grp = qf[r, solo * G:(solo + 1) * G]
            if spec.plant_mode == "scaled":
                qbar = grp.mean(axis=0)
                base = (2.0 * d) * qbar / float(qbar @ qbar)
            else:
                base = grp[0]
            for j in hv:
                noise = prng.standard_normal((bs, d))
                keys = (base[None, :] + 0.1 * noise).astype(np.float32)
                kblk = kv5[blk_off[r] + j, 0, solo].reshape(bs, d)
                kblk[:] = round_to_dtype(keys, dtype).reshape(bs, d)
    # zero the padding tokens of each request's last block
    for r in range(B):
        if n_blocks[r] == 0:
            continue
        nv = int(ctx_len[r] - (n_blocks[r] - 1) * bs)
        if nv < bs:
            last = int(blk_off[r] + n_blocks[r] - 1)
            kpart = kv5[last, 0].reshape(Hkv, bs, d)
            vpart = kv5[last, 1].reshape(Hkv, d, bs)
            kpart[:, nv:, :] = 0
            vpart[:, :, nv:] = 0

    return _finish(spec, seed, B, Hq, Hkv, d, bs, dtype, ctx_len, n_blocks, blk_off, q, kv, solo)


def _finish(spec, seed, B, Hq, Hkv, d, bs, dtype, ctx_len, n_blocks, blk_off, q, kv, solo) -> Workload:
    """Resident hot set, slot pool, free list and budgets of a drawn store."""
    # resident hot set: forced sink/local blocks plus a seeded sample of middle blocks
    k_mid = np.asarray(spec.k_mid, np.int32)
    max_blocks = int(max(1, n_blocks.max() if B else 1))
    table0 = np.full((B, max_blocks), -1, np.int32)
    resident = []
    rrng = np.random.default_rng([seed, 2, spec.resident_key])
    for r in range(B):
        n = int(n_blocks[r])
        forced = sorted(set(range(min(spec.n_sink, n))) | set(range(max(0, n - spec.n_local), n)))
        middle = np.arange(spec.n_sink, max(spec.n_sink, n - spec.n_local))
        want = int(math.floor(spec.resident_frac * n)) - len(forced)
        pick = rrng.choice(middle, size=max(0, min(want, middle.size)), replace=False) if want > 0 else []
        res = np.sort(np.concatenate([np.asarray(forced, np.int64), np.asarray(pick, np.int64)]))
        resident.append(res)
    slot = 0
    res_blocks = []
    for r in range(B):
        for j in resident[r]:
            table0[r, j] = slot
            res_blocks.append(int(blk_off[r] + j))
            slot += 1
    n_res = slot
    worst = 0
    for r in range(B):
        n = int(n_blocks[r])
        n_forced = len(set(range(min(spec.n_sink, n))) | set(range(max(0, n - spec.n_local), n)))
        worst += n_forced + max(0, min(int(k_mid[r]), n - n_forced))
    n_free = worst + spec.slack_slots if spec.n_free_override is None else spec.n_free_override
    n_slots = max(1, n_res + n_free)
    free_slots = np.arange(n_res, n_res + n_free, dtype=np.int32)
    if spec.free_order == "shuffled":
        free_slots = np.random.default_rng([seed, 3]).permutation(free_slots).astype(np.int32)
    k_max = 1
    for r in range(B):
        n = int(n_blocks[r])
        n_forced = len(set(range(min(spec.n_sink, n))) | set(range(max(0, n - spec.n_local), n)))
        k_max = max(k_max, n_forced + max(0, min(int(k_mid[r]), n - n_forced)))

    return Workload(spec=spec, seed=seed, B=B, Hq=Hq, Hkv=Hkv, d=d, bs=bs, dtype=dtype,
                    dtype_code=DTYPE_CODES[dtype], ctx_len=ctx_len, n_blocks=n_blocks, blk_off=blk_off,
                    q=q, kv=kv, k_mid=k_mid, n_sink=spec.n_sink, n_local=spec.n_local, k_max=k_max,
                    max_blocks=max_blocks, table0=table0, resident_blocks=np.asarray(res_blocks, np.int64),
                    free_slots=free_slots, n_slots=n_slots, solo_kv_head=solo, heavy=spec.heavy,
                    sm_scale=1.0 / math.sqrt(d))


def make(config_id: int, **kw) -> Workload:
    """Generate one of the five presets (see ``preset``)."""
    gen_kw = {k: kw.pop(k) for k in ("kv_alloc", "threads", "store_key") if k in kw}
    spec, seed = preset(config_id, **kw)
    return generate(spec, seed, **gen_kw)


def initial_pool(w: Workload) -> np.ndarray:
    """Host image of the slot pool at the start of a step: resident blocks in their slots,
    free slots zero.  uint16 [n_slots, elems_per_block]."""
    pool = np.zeros((w.n_slots, w.elems_per_block), np.uint16)
    if w.resident_blocks.size:
        pool[: w.resident_blocks.size] = w.kv[w.resident_blocks]
    return pool
