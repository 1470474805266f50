"""Shared helpers of the GPU parity tests: build device state from a workload and
compare every stage of the GPU path with the CPU oracle on the same inputs."""
import sys

import numpy as np

from oracle import pulse_oracle as O
from paper_2609_34555_amd import harness as H
from paper_2609_34555_amd import workloads as W

ATTN_TOL = 2e-3  # max-abs on fp32 outputs, fp32 accumulation
TIE_REL = 1e-5   # selections may differ only between scores this close to the k-th


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def build(spec, seed, coherent=True, k_max=None, store_key=0):
    holder = []
    w = W.generate(spec, seed, kv_alloc=H.pinned_allocator(holder, coherent), store_key=store_key)
    st = H.LayerState(w, holder[0].ptr, k_max=k_max)
    st.holder = holder
    return w, st


def oracle_selection(w, digests_u16, solo=None, k_max=None):
    solo = w.solo_kv_head if solo is None else solo
    s = O.score(w.q, digests_u16, w.blk_off, w.Hq, w.Hkv, w.d, w.dtype_code, solo)
    rc, idx, cnt = O.select(s, w.blk_off, w.k_mid, w.n_sink, w.n_local, k_max or w.k_max)
    return rc, idx, cnt, s


def assert_selection_ok(w, gidx, gcnt, oidx, ocnt, oscores):
    """Equal counts, ascending lists padded with -1, and any difference only among
    middle blocks whose (fp32) oracle score is within TIE_REL of the k-th score."""
    k_max = gidx.shape[1]
    n_ties = 0
    for r in range(w.B):
        assert gcnt[r] == ocnt[r], (r, gcnt[r], ocnt[r])
        g = gidx[r, : gcnt[r]]
        assert np.all(np.diff(g) > 0) and np.all(gidx[r, gcnt[r]:] == -1)
        diff = set(g.tolist()) ^ set(oidx[r, : ocnt[r]].tolist())
        if not diff:
            continue
        b0 = int(w.blk_off[r])
        n = int(w.n_blocks[r])
        lo, hi = w.n_sink, n - w.n_local
        mid = np.float32(oscores[b0 + lo: b0 + hi])
        k = min(max(int(w.k_mid[r]), 0), hi - lo)
        kth = np.sort(mid)[::-1][k - 1]
        for j in diff:
            assert lo <= j < hi, (r, j)
            assert abs(np.float32(oscores[b0 + j]) - kth) <= TIE_REL * abs(kth), (r, j, oscores[b0 + j], kth)
            n_ties += 1
    assert k_max >= 1
    return n_ties


def oracle_recall(w, idx, cnt, free_slots=None, free_head=0, table0=None):
    """The oracle's recall of selection (idx, cnt) from the workload's initial table (or table0)
    and pool; free_slots / free_head default to the workload's free list and 0."""
    table = (w.table0 if table0 is None else table0).copy()
    pool = W.initial_pool(w).view(np.uint8).reshape(w.n_slots, -1).copy()
    host = w.kv.view(np.uint8).reshape(w.total_blocks, 2 * w.elems_per_block)
    free = w.free_slots if free_slots is None else free_slots
    rc, fh, stats = O.recall(host, w.blk_off, idx, cnt, table, free, free_head, pool, w.unit_bytes)
    return rc, table, pool, fh, stats


def assert_recall_equal(st, table, pool, fh, stats):
    assert np.array_equal(st.table_np(), table)
    assert int(st.free_head.item()) == fh
    assert st.recall_stats() == tuple(stats)
    gp = st.pool.cpu().numpy().view(np.uint8).reshape(pool.shape)
    assert np.array_equal(gp, pool)


def oracle_attention(w, pool_u8, table, idx, cnt):
    pool16 = pool_u8.view(np.uint16).reshape(w.n_slots, -1)
    return O.attention(w.q, pool16, table, idx, cnt, w.blk_off, w.ctx_len, w.Hq, w.Hkv, w.bs, w.d, w.dtype_code,
                       w.sm_scale)


def assert_attention_close(st, out, lse, tol=ATTN_TOL):
    go = st.out.cpu().numpy().astype(np.float64)
    gl = st.lse.cpu().numpy().astype(np.float64)
    err = np.max(np.abs(go - out)) if out.size else 0.0
    assert err <= tol, f"max |out - oracle| = {err}"
    fin = np.isfinite(lse)
    assert np.array_equal(np.isfinite(gl), fin)
    lerr = np.max(np.abs(gl[fin] - lse[fin])) if fin.any() else 0.0
    assert lerr <= tol, f"max |lse - oracle| = {lerr}"
    return err, lerr


def full_check(w, st, chained=True, run=True):
    """Run one layer-step on the GPU (chained or stage by stage; run=False checks the
    state a previous run left) and check every stage against the oracle."""
    import torch

    if run:
        st.reset()
        if chained:
            st.decode_layer()
        else:
            st.select()
            st.recall()
            st.attention()
    torch.cuda.synchronize()
    assert st.status() == 0, f"device status {st.status()}"
    dig = st.digests.cpu().numpy().view(np.uint16)[: w.total_blocks]
    odig = O.build_digests(w.kv, w.blk_off, w.ctx_len, w.Hkv, w.bs, w.d, w.dtype_code, w.solo_kv_head)
    assert np.array_equal(dig, odig)
    gidx, gcnt = st.selection()
    rc, oidx, ocnt, osc = oracle_selection(w, odig, k_max=st.k_max)
    assert rc == 0
    ties = assert_selection_ok(w, gidx, gcnt, oidx, ocnt, osc)
    rc, table, pool, fh, stats = oracle_recall(w, gidx, gcnt)
    assert rc == 0
    assert_recall_equal(st, table, pool, fh, stats)
    out, lse = oracle_attention(w, pool, table, gidx, gcnt)
    err = assert_attention_close(st, out, lse)
    return dict(ties=ties, stats=stats, attn_err=err)


def random_case(seed):
    """A seeded small workload: batch, ragged (and empty) contexts, block size, group size,
    forced-block counts, budgets from 0 to past the middle, planted or not, free-list order."""
    rng = np.random.default_rng([seed, 3107])
    B = int(rng.integers(1, 7))
    bs = int(rng.choice([16, 32, 64]))
    Hkv = int(rng.choice([1, 2, 3, 8]))  # odd head counts: blocks of 8 KiB multiples that are not 16 KiB ones
    G = int(rng.choice([1, 2, 3, 4, 8, 16]))
    ctx = [0 if rng.random() < 0.1 else int(rng.integers(1, 24000)) for _ in range(B)]
    n_max = max(1, max(-(-c // bs) for c in ctx))
    k_mid = [int(rng.choice([0, int(rng.integers(1, 40)), int(rng.integers(1, n_max + 5))])) for _ in range(B)]
    n_sink, n_local = int(rng.integers(0, 3)), int(rng.integers(0, 9))
    spec, s = W.custom(f"rand{seed}", ctx, Hq=G * Hkv, Hkv=Hkv, bs=bs, dtype=str(rng.choice(["bf16", "f16"])),
                       k_mid=k_mid, n_sink=n_sink, n_local=n_local, resident_frac=float(rng.choice([0.0, 0.1, 0.5])),
                       heavy_per_req=int(rng.integers(0, 8)), planted=bool(rng.random() < 0.5),
                       free_order=str(rng.choice(["ascending", "shuffled"])), seed=seed)
    return spec, s


def random_case_long(seed):
    """A seeded workload with long contexts (up to 300K tokens: several 8192-block selection
    tiles at bs 16) and batches up to 24, budgets up to a few hundred blocks."""
    rng = np.random.default_rng([seed, 4219])
    B = int(rng.integers(1, 25))
    bs = int(rng.choice([16, 32]))
    Hkv = int(rng.choice([1, 2, 8]))
    G = int(rng.choice([1, 4, 8]))
    ctx = [0 if rng.random() < 0.05 else int(rng.integers(1, 300000 if r < 3 else 40000)) for r in range(B)]
    k_mid = [int(rng.integers(0, 600)) for _ in range(B)]
    spec, s = W.custom(f"long{seed}", ctx, Hq=G * Hkv, Hkv=Hkv, bs=bs, dtype=str(rng.choice(["bf16", "f16"])),
                       k_mid=k_mid, n_sink=int(rng.integers(0, 3)), n_local=int(rng.integers(0, 9)),
                       resident_frac=float(rng.choice([0.0, 0.05, 0.3])), heavy_per_req=int(rng.integers(0, 30)),
                       planted=bool(rng.random() < 0.5), free_order=str(rng.choice(["ascending", "shuffled"])),
                       seed=seed)
    return spec, s
