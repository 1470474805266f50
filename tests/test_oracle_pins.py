"""Pins of the CPU oracle against things other than itself (runs on CPU).

Each test checks the oracle against a fact fixed by the paper or by
mathematics: a hand-worked example, brute force on tiny inputs, invariants,
closed forms and special cases that reduce to a textbook computation.  A
dropped term, a wrong sign or index, or a transposed operand in the oracle
fails at least one of them.
"""
import json
import math
import os

import numpy as np
import pytest

from oracle import pulse_oracle as O
from paper_2609_34555_amd import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------- helpers

def k_view(w_kv, Hkv, bs, d):
    """keys [blocks, Hkv, bs, d] per the stated block layout"""
    nb = w_kv.shape[0]
    return w_kv.reshape(nb, 2, Hkv, bs * d)[:, 0].reshape(nb, Hkv, bs, d)


def v_view(w_kv, Hkv, bs, d):
    """values [blocks, Hkv, bs, d] (stored channel-major)"""
    nb = w_kv.shape[0]
    return w_kv.reshape(nb, 2, Hkv, bs * d)[:, 1].reshape(nb, Hkv, d, bs).transpose(0, 1, 3, 2)


def tiny(ctx, Hq=4, Hkv=2, d=8, bs=4, dtype="bf16", seed=3, k_mid=2, n_sink=1, n_local=1, planted=False,
         resident_frac=0.25, heavy=1):
    spec, s = W.custom("t", ctx, Hq=Hq, Hkv=Hkv, d=d, bs=bs, dtype=dtype, k_mid=k_mid, n_sink=n_sink,
                       n_local=n_local, resident_frac=resident_frac, heavy_per_req=heavy, planted=planted,
                       seed=seed)
    return W.generate(spec, s)


def worked():
    with open(os.path.join(GOLDEN, "worked_example.json")) as f:
        g = json.load(f)
    sh = g["shape"]
    Hq, Hkv, d, bs = sh["Hq"], sh["Hkv"], sh["d"], sh["bs"]
    L = sh["ctx_len"]
    nb = -(-L // bs)
    kv = np.zeros((nb, 2 * Hkv * bs * d), np.uint16)
    keys = np.array(g["keys"], np.float32)
    vals = np.array(g["values"], np.float32)
    for t in range(L):
        b, row = divmod(t, bs)
        for c in range(d):
            kv[b, (0 * Hkv + 0) * bs * d + row * d + c] = W.round_to_dtype(keys[t, c:c + 1], "bf16")[0]
            kv[b, Hkv * bs * d + (0 * d + c) * bs + row] = W.round_to_dtype(vals[t, c:c + 1], "bf16")[0]
    q = W.round_to_dtype(np.array(g["q"], np.float32), "bf16").reshape(1, Hq, d)
    blk_off = np.array([0, nb], np.int64)
    ctx = np.array([L], np.int32)
    return g, kv, q, blk_off, ctx, (Hq, Hkv, d, bs)


# ---------------------------------------------------------------- worked example

def test_worked_example_digest_score_select():
    g, kv, q, blk_off, ctx, (Hq, Hkv, d, bs) = worked()
    dig = O.build_digests(kv, blk_off, ctx, Hkv, bs, d, O.BF16, 0)
    assert np.array_equal(W.to_float(dig[:, 0], "bf16"), np.array(g["digest_min"], np.float32))
    assert np.array_equal(W.to_float(dig[:, 1], "bf16"), np.array(g["digest_max"], np.float32))
    s = O.score(q, dig, blk_off, Hq, Hkv, d, O.BF16, 0)
    assert np.array_equal(s, np.array(g["scores"]))
    rc, idx, cnt = O.select(s, blk_off, np.array([2], np.int32), 0, 0, 4)
    assert rc == 0 and list(idx[0, : cnt[0]]) == g["select_top2_no_forced"]
    rc, idx, cnt = O.select(s, blk_off, np.array([1], np.int32), 1, 1, 4)
    assert rc == 0 and list(idx[0, : cnt[0]]) == g["select_sink1_local1_k1"]


def test_worked_example_attention_closed_form():
    g, kv, q, blk_off, ctx, (Hq, Hkv, d, bs) = worked()
    sel = np.array([g["attention_over"] + [-1]], np.int32)
    table = np.array([[0, -1, 1]], np.int32)  # b0 in slot 0, b2 in slot 1
    pool = np.stack([kv[0], kv[2]])
    out, lse = O.attention(q, pool, table, sel, np.array([2], np.int32), blk_off, ctx, Hq, Hkv, bs, d, O.BF16, 1.0)
    e = math.exp
    Z0 = e(-1) + e(4) + 1
    Z1 = 2 * e(2) + e(6)
    want = np.array([[(e(-1) + 1) / Z0, (e(4) + 1) / Z0], [(e(2) + e(2)) / Z1, (e(6) + e(2)) / Z1]])
    assert np.allclose(out[0], want, rtol=0, atol=1e-14)
    assert np.allclose(lse[0], [math.log(Z0), math.log(Z1)], rtol=0, atol=1e-13)


def test_worked_example_mam_closed_form():
    g, kv, q, blk_off, ctx, (Hq, Hkv, d, bs) = worked()
    best, mq, mh = O.mam(q, kv, blk_off, ctx, 0, Hq, Hkv, bs, d, O.BF16, 1.0, n_sink_tok=1, n_local_tok=1)
    e = math.exp
    m0 = (e(4) + 1 + e(-6)) / (e(-1) + e(4) + 1 + e(-6) + 1)
    m1 = (e(6) + 1 + e(-4)) / (e(2) + e(6) + 1 + e(-4) + e(2))
    assert best == 0
    assert np.allclose(mq, [m0, m1], rtol=0, atol=1e-14)
    assert abs(mh[0] - (m0 + m1) / 2) < 1e-14


# ---------------------------------------------------------------- digest pins

@pytest.mark.parametrize("dtype", ["bf16", "f16"])
def test_digest_bounds_and_attained(dtype):
    w = tiny([37, 16, 5], dtype=dtype, seed=11)
    code = W.DTYPE_CODES[dtype]
    kv = w.kv.copy()
    # poke huge values into padding tokens: they must not reach the digest
    K = k_view(kv, w.Hkv, w.bs, w.d)
    for r in range(w.B):
        nv = int(w.ctx_len[r] - (w.n_blocks[r] - 1) * w.bs)
        if nv < w.bs:
            K[int(w.blk_off[r + 1] - 1), :, nv:, :] = W.round_to_dtype(np.full((1,), 100.0, np.float32), dtype)[0]
    for h in range(w.Hkv):
        dig = O.build_digests(kv, w.blk_off, w.ctx_len, w.Hkv, w.bs, w.d, code, h)
        mn = W.to_float(dig[:, 0], dtype)
        mx = W.to_float(dig[:, 1], dtype)
        Kf = W.to_float(K[:, h], dtype)  # [blocks, bs, d]
        for r in range(w.B):
            for j in range(int(w.n_blocks[r])):
                b = int(w.blk_off[r] + j)
                nv = min(w.bs, int(w.ctx_len[r]) - j * w.bs)
                toks = Kf[b, :nv]
                assert np.array_equal(mn[b], toks.min(axis=0))
                assert np.array_equal(mx[b], toks.max(axis=0))


def test_digest_block_size_one_is_identity():
    w = tiny([9, 4], bs=1, seed=5, n_local=0, n_sink=0)
    dig = O.build_digests(w.kv, w.blk_off, w.ctx_len, w.Hkv, 1, w.d, O.BF16, 1)
    K = k_view(w.kv, w.Hkv, 1, w.d)[:, 1, 0, :]
    assert np.array_equal(dig[:, 0], K) and np.array_equal(dig[:, 1], K)


def test_digest_signed_zero_order():
    # one block of 2 tokens, channel 0 holds -0 and +0: min is -0, max is +0
    Hkv, bs, d = 1, 2, 2
    kv = np.zeros((1, 2 * Hkv * bs * d), np.uint16)
    kv[0, 0 * d + 0] = 0x8000  # token 0, channel 0: -0
    kv[0, 1 * d + 0] = 0x0000  # token 1, channel 0: +0
    kv[0, 0 * d + 1] = 0x0000
    kv[0, 1 * d + 1] = 0x8000
    dig = O.build_digests(kv, np.array([0, 1], np.int64), np.array([2], np.int32), Hkv, bs, d, O.BF16, 0)
    assert list(dig[0, 0]) == [0x8000, 0x8000] and list(dig[0, 1]) == [0x0000, 0x0000]


# ---------------------------------------------------------------- score pins

@pytest.mark.parametrize("dtype", ["bf16", "f16"])
def test_score_is_upper_bound_of_group_mean_of_max_logits(dtype):
    w = tiny([64, 29], Hq=8, Hkv=2, d=16, bs=4, dtype=dtype, seed=21)
    code = W.DTYPE_CODES[dtype]
    qf = W.to_float(w.q, dtype).astype(np.float64)
    for h in range(w.Hkv):
        dig = O.build_digests(w.kv, w.blk_off, w.ctx_len, w.Hkv, w.bs, w.d, code, h)
        s = O.score(w.q, dig, w.blk_off, w.Hq, w.Hkv, w.d, code, h)
        K = W.to_float(k_view(w.kv, w.Hkv, w.bs, w.d)[:, h], dtype).astype(np.float64)
        G = w.G
        for r in range(w.B):
            for j in range(int(w.n_blocks[r])):
                b = int(w.blk_off[r] + j)
                nv = min(w.bs, int(w.ctx_len[r]) - j * w.bs)
                logits = qf[r, h * G:(h + 1) * G] @ K[b, :nv].T  # [G, nv]
                bound = logits.max(axis=1).mean()
                assert s[b] >= bound - 1e-9 * max(1.0, abs(bound))


def test_score_block_size_one_equals_group_mean_logit():
    w = tiny([50, 33], Hq=8, Hkv=2, d=16, bs=1, seed=8, n_sink=0, n_local=0)
    qf = W.to_float(w.q, "bf16").astype(np.float64)
    K = W.to_float(k_view(w.kv, w.Hkv, 1, w.d)[:, :, 0, :], "bf16").astype(np.float64)
    for h in range(w.Hkv):
        dig = O.build_digests(w.kv, w.blk_off, w.ctx_len, w.Hkv, 1, w.d, O.BF16, h)
        s = O.score(w.q, dig, w.blk_off, w.Hq, w.Hkv, w.d, O.BF16, h)
        for r in range(w.B):
            qbar = qf[r, h * w.G:(h + 1) * w.G].mean(axis=0)
            b0, b1 = int(w.blk_off[r]), int(w.blk_off[r + 1])
            exact = K[b0:b1, h] @ qbar
            assert np.allclose(s[b0:b1], exact, rtol=1e-13, atol=1e-12)


# ---------------------------------------------------------------- selection pins

def test_solohead_bs1_equals_bruteforce_exact_topk():
    """bs = 1: the digest bound is exact, so SoloHead top-k = exact top-k of the
    solo head's group-mean attention logits (brute force with lexsort)."""
    w = tiny([200, 150, 7], Hq=8, Hkv=4, d=32, bs=1, seed=31, n_sink=0, n_local=0, k_mid=12)
    qf = W.to_float(w.q, "bf16").astype(np.float64)
    K = W.to_float(k_view(w.kv, w.Hkv, 1, w.d)[:, :, 0, :], "bf16").astype(np.float64)
    h = 2
    dig = O.build_digests(w.kv, w.blk_off, w.ctx_len, w.Hkv, 1, w.d, O.BF16, h)
    s = O.score(w.q, dig, w.blk_off, w.Hq, w.Hkv, w.d, O.BF16, h)
    k_max = 16
    rc, idx, cnt = O.select(s, w.blk_off, np.full(w.B, 12, np.int32), 0, 0, k_max)
    assert rc == 0
    for r in range(w.B):
        b0, b1 = int(w.blk_off[r]), int(w.blk_off[r + 1])
        logit = K[b0:b1, h] @ qf[r, h * w.G:(h + 1) * w.G].mean(axis=0)
        order = np.lexsort((np.arange(b1 - b0), -logit))
        want = np.sort(order[: min(12, b1 - b0)])
        assert list(idx[r, : cnt[r]]) == list(want)


def test_select_matches_full_sort_with_forced_blocks():
    rng = np.random.default_rng(4)
    n = np.array([40, 3, 17, 0, 12])
    blk_off = np.concatenate([[0], np.cumsum(n)]).astype(np.int64)
    s = np.round(rng.standard_normal(int(n.sum())) * 4) / 4  # many exact ties
    k_mid = np.array([5, 2, 20, 3, 0], np.int32)
    n_sink, n_local, k_max = 2, 3, 32
    rc, idx, cnt = O.select(s, blk_off, k_mid, n_sink, n_local, k_max)
    assert rc == 0
    for r in range(len(n)):
        sc = s[blk_off[r]:blk_off[r + 1]]
        forced = [j for j in range(n[r]) if j < n_sink or j >= n[r] - n_local]
        mid = [j for j in range(n[r]) if j not in forced]
        mid_sorted = sorted(mid, key=lambda j: (-np.float32(sc[j]), j))
        want = sorted(forced + mid_sorted[: max(0, min(int(k_mid[r]), len(mid)))])
        assert list(idx[r, : cnt[r]]) == want
        assert all(x == -1 for x in idx[r, cnt[r]:])


def test_select_ties_take_lowest_index_and_edge_budgets():
    blk_off = np.array([0, 10], np.int64)
    s = np.ones(10)  # every middle block ties
    rc, idx, cnt = O.select(s, blk_off, np.array([3], np.int32), 1, 1, 10)
    assert list(idx[0, : cnt[0]]) == [0, 1, 2, 3, 9]
    rc, idx, cnt = O.select(s, blk_off, np.array([100], np.int32), 1, 1, 10)  # k >= #middle -> all
    assert list(idx[0, : cnt[0]]) == list(range(10))
    rc, idx, cnt = O.select(s, blk_off, np.array([0], np.int32), 1, 1, 10)  # k = 0 -> forced only
    assert list(idx[0, : cnt[0]]) == [0, 9]
    rc, idx, cnt = O.select(s, blk_off, np.array([-4], np.int32), 6, 6, 10)  # forced cover all blocks
    assert list(idx[0, : cnt[0]]) == list(range(10))
    rc, idx, cnt = O.select(s, blk_off, np.array([5], np.int32), 1, 1, 6)  # 7 > k_max
    assert rc == O.ERR_SELECT_OVERFLOW and cnt[0] == 0


# ---------------------------------------------------------------- recall pins

def _recall_setup(seed=12, n_free_override=None, free_order="shuffled"):
    spec, s = W.custom("r", [70, 33, 48], Hq=4, Hkv=2, d=8, bs=4, k_mid=6, n_sink=1, n_local=2,
                       resident_frac=0.3, heavy_per_req=3, seed=seed, free_order=free_order,
                       n_free_override=n_free_override)
    w = W.generate(spec, s)
    dig = O.build_digests(w.kv, w.blk_off, w.ctx_len, w.Hkv, w.bs, w.d, O.BF16, w.solo_kv_head)
    sc = O.score(w.q, dig, w.blk_off, w.Hq, w.Hkv, w.d, O.BF16, w.solo_kv_head)
    rc, idx, cnt = O.select(sc, w.blk_off, w.k_mid, w.n_sink, w.n_local, w.k_max)
    assert rc == 0
    return w, idx, cnt


def test_recall_invariants_and_bytes():
    w, idx, cnt = _recall_setup()
    table = w.table0.copy()
    pool = W.initial_pool(w).view(np.uint8).reshape(w.n_slots, -1).copy()
    pool_before = pool.copy()
    host = w.kv.view(np.uint8).reshape(w.total_blocks, -1)
    rc, fh, stats = O.recall(host, w.blk_off, idx, cnt, table, w.free_slots, 0, pool, w.unit_bytes)
    assert rc == 0
    missing = [(r, j) for r in range(w.B) for j in idx[r, : cnt[r]] if w.table0[r, j] < 0]
    assert stats[0] == len(missing) and fh == len(missing) and stats[2] == len(missing) * w.unit_bytes
    # slots: exactly the head of the free list, in (request, block) order
    assert [table[r, j] for r, j in missing] == list(w.free_slots[: len(missing)])
    # runs counted another way: breaks in consecutive missing indices per request
    runs = 0
    for r in range(w.B):
        js = np.array([j for rr, j in missing if rr == r])
        runs += int(js.size and 1 + np.count_nonzero(np.diff(js) != 1))
    assert stats[1] == runs
    # every selected block resident afterwards with the host bytes; other entries unchanged
    for r in range(w.B):
        for j in idx[r, : cnt[r]]:
            assert np.array_equal(pool[table[r, j]], host[w.blk_off[r] + j])
    changed = table != w.table0
    assert changed.sum() == len(missing)
    untouched = np.setdiff1d(np.arange(w.n_slots), w.free_slots[: len(missing)])
    assert np.array_equal(pool[untouched], pool_before[untouched])


def test_recall_pool_exhaustion_changes_nothing():
    w, idx, cnt = _recall_setup(n_free_override=2)
    table = w.table0.copy()
    pool = W.initial_pool(w).view(np.uint8).reshape(w.n_slots, -1).copy()
    before = (table.copy(), pool.copy())
    host = w.kv.view(np.uint8).reshape(w.total_blocks, -1)
    rc, fh, stats = O.recall(host, w.blk_off, idx, cnt, table, w.free_slots, 0, pool, w.unit_bytes)
    assert rc == O.ERR_POOL_EXHAUSTED and fh == 0 and stats[2] == 0 and stats[0] > 2
    assert np.array_equal(table, before[0]) and np.array_equal(pool, before[1])


def test_recall_rejects_unsorted_selection():
    w, idx, cnt = _recall_setup()
    bad = idx.copy()
    bad[0, [0, 1]] = bad[0, [1, 0]]
    table = w.table0.copy()
    pool = W.initial_pool(w).view(np.uint8).reshape(w.n_slots, -1).copy()
    host = w.kv.view(np.uint8).reshape(w.total_blocks, -1)
    rc, fh, _ = O.recall(host, w.blk_off, bad, cnt, table, w.free_slots, 0, pool, w.unit_bytes)
    assert rc == O.ERR_BAD_INDEX and fh == 0 and np.array_equal(table, w.table0)


# ---------------------------------------------------------------- attention pins

def _all_resident(w):
    """table/pool with every block resident (slot = global block id)."""
    table = np.full((w.B, w.max_blocks), -1, np.int32)
    for r in range(w.B):
        table[r, : w.n_blocks[r]] = np.arange(w.blk_off[r], w.blk_off[r + 1])
    return table, w.kv.copy()


def test_select_all_equals_dense_attention():
    w = tiny([45, 16, 3], Hq=8, Hkv=2, d=16, bs=4, seed=17)
    table, pool = _all_resident(w)
    k_max = int(w.n_blocks.max())
    idx = np.full((w.B, k_max), -1, np.int32)
    for r in range(w.B):
        idx[r, : w.n_blocks[r]] = np.arange(w.n_blocks[r])
    out, lse = O.attention(w.q, pool, table, idx, w.n_blocks.astype(np.int32), w.blk_off, w.ctx_len, w.Hq, w.Hkv,
                           w.bs, w.d, O.BF16, w.sm_scale)
    dout, dlse = O.dense_attention(w.q, w.kv, w.blk_off, w.ctx_len, w.Hq, w.Hkv, w.bs, w.d, O.BF16, w.sm_scale)
    assert np.allclose(out, dout, rtol=0, atol=1e-13) and np.allclose(lse, dlse, rtol=0, atol=1e-12)


@pytest.mark.parametrize("dtype", ["bf16", "f16"])
def test_dense_attention_matches_matrix_softmax(dtype):
    """Dense oracle vs an independent matrix formulation softmax(q K^T s) V in fp64."""
    w = tiny([23, 8], Hq=6, Hkv=3, d=16, bs=4, dtype=dtype, seed=41)
    code = W.DTYPE_CODES[dtype]
    out, lse = O.dense_attention(w.q, w.kv, w.blk_off, w.ctx_len, w.Hq, w.Hkv, w.bs, w.d, code, w.sm_scale)
    K = W.to_float(k_view(w.kv, w.Hkv, w.bs, w.d), dtype).astype(np.float64)
    V = W.to_float(v_view(w.kv, w.Hkv, w.bs, w.d), dtype).astype(np.float64)
    qf = W.to_float(w.q, dtype).astype(np.float64)
    for r in range(w.B):
        L = int(w.ctx_len[r])
        b0, b1 = int(w.blk_off[r]), int(w.blk_off[r + 1])
        for hq in range(w.Hq):
            h = hq // w.G
            Kr = K[b0:b1, h].reshape(-1, w.d)[:L]
            Vr = V[b0:b1, h].reshape(-1, w.d)[:L]
            z = (Kr @ qf[r, hq]) * w.sm_scale
            p = np.exp(z - z.max())
            assert np.allclose(out[r, hq], (p / p.sum()) @ Vr, rtol=0, atol=1e-13)
            assert abs(lse[r, hq] - (z.max() + np.log(p.sum()))) < 1e-12


def test_attention_closed_forms_uniform_and_normalisation():
    w = tiny([30, 12], Hq=4, Hkv=2, d=8, bs=4, seed=9)
    table, pool = _all_resident(w)
    k_max = int(w.n_blocks.max())
    idx = np.full((w.B, k_max), -1, np.int32)
    for r in range(w.B):
        idx[r, : w.n_blocks[r]] = np.arange(w.n_blocks[r])
    cnt = w.n_blocks.astype(np.int32)
    # q = 0 -> uniform weights: out = mean of values, lse = ln(#tokens)
    q0 = np.zeros_like(w.q)
    out, lse = O.attention(q0, pool, table, idx, cnt, w.blk_off, w.ctx_len, w.Hq, w.Hkv, w.bs, w.d, O.BF16, 1.0)
    V = W.to_float(v_view(w.kv, w.Hkv, w.bs, w.d), "bf16").astype(np.float64)
    for r in range(w.B):
        L = int(w.ctx_len[r])
        for hq in range(w.Hq):
            Vr = V[w.blk_off[r]:w.blk_off[r + 1], hq // w.G].reshape(-1, w.d)[:L]
            assert np.allclose(out[r, hq], Vr.mean(axis=0), rtol=0, atol=1e-14)
            assert abs(lse[r, hq] - math.log(L)) < 1e-13
    # all-ones values -> output exactly 1 (weights sum to one)
    ones = pool.copy()
    ones.reshape(ones.shape[0], 2, -1)[:, 1] = W.round_to_dtype(np.ones(1, np.float32), "bf16")[0]
    out, _ = O.attention(w.q, ones, table, idx, cnt, w.blk_off, w.ctx_len, w.Hq, w.Hkv, w.bs, w.d, O.BF16, w.sm_scale)
    assert np.allclose(out, 1.0, rtol=0, atol=1e-14)


def test_attention_single_token_and_slot_permutation():
    w = tiny([1, 9], Hq=4, Hkv=2, d=8, bs=4, seed=10)
    table, pool = _all_resident(w)
    k_max = int(w.n_blocks.max())
    idx = np.full((w.B, k_max), -1, np.int32)
    for r in range(w.B):
        idx[r, : w.n_blocks[r]] = np.arange(w.n_blocks[r])
    cnt = w.n_blocks.astype(np.int32)
    out, lse = O.attention(w.q, pool, table, idx, cnt, w.blk_off, w.ctx_len, w.Hq, w.Hkv, w.bs, w.d, O.BF16,
                           w.sm_scale)
    # request 0 has one token: out = its value row, lse = its logit
    V = W.to_float(v_view(w.kv, w.Hkv, w.bs, w.d), "bf16").astype(np.float64)
    K = W.to_float(k_view(w.kv, w.Hkv, w.bs, w.d), "bf16").astype(np.float64)
    qf = W.to_float(w.q, "bf16").astype(np.float64)
    for hq in range(w.Hq):
        assert np.array_equal(out[0, hq], V[0, hq // w.G, 0])
        assert abs(lse[0, hq] - w.sm_scale * float(K[0, hq // w.G, 0] @ qf[0, hq])) < 1e-13
    # moving blocks to other slots changes nothing
    perm = np.random.default_rng(0).permutation(pool.shape[0])
    pool2 = np.empty_like(pool)
    pool2[perm] = pool
    table2 = np.where(table >= 0, perm[np.maximum(table, 0)], -1).astype(np.int32)
    out2, lse2 = O.attention(w.q, pool2, table2, idx, cnt, w.blk_off, w.ctx_len, w.Hq, w.Hkv, w.bs, w.d, O.BF16,
                             w.sm_scale)
    assert np.array_equal(out, out2) and np.array_equal(lse, lse2)


def test_attention_empty_selection():
    w = tiny([0, 9], Hq=4, Hkv=2, d=8, bs=4, seed=10)
    table, pool = _all_resident(w)
    idx = np.full((w.B, 3), -1, np.int32)
    cnt = np.zeros(w.B, np.int32)
    out, lse = O.attention(w.q, pool, table, idx, cnt, w.blk_off, w.ctx_len, w.Hq, w.Hkv, w.bs, w.d, O.BF16, 1.0)
    assert np.all(out == 0) and np.all(np.isneginf(lse))


# ---------------------------------------------------------------- MAM pins

def test_mam_is_one_without_sink_and_local_and_uniform_value():
    w = tiny([40], Hq=4, Hkv=2, d=8, bs=4, seed=2)
    best, mq, mh = O.mam(w.q, w.kv, w.blk_off, w.ctx_len, 0, w.Hq, w.Hkv, w.bs, w.d, O.BF16, w.sm_scale, 0, 0)
    assert np.allclose(mq, 1.0, atol=1e-15) and best == 0
    q0 = np.zeros_like(w.q)
    best, mq, mh = O.mam(q0, w.kv, w.blk_off, w.ctx_len, 0, w.Hq, w.Hkv, w.bs, w.d, O.BF16, w.sm_scale, 3, 5)
    assert np.allclose(mq, (40 - 8) / 40, atol=1e-15)
    assert np.allclose(mh, mq.reshape(w.Hkv, w.G).mean(axis=1))


def test_mam_picks_planted_retrieval_head():
    """The generator plants heavy middle blocks in one KV head's keys; Eq. 2 ranks that
    head highest (its query heads put their mass on middle tokens)."""
    spec, s = W.preset(1)
    w = W.generate(spec, s)
    best, mq, mh = O.mam(w.q, w.kv, w.blk_off, w.ctx_len, 0, w.Hq, w.Hkv, w.bs, w.d, w.dtype_code, w.sm_scale)
    assert best == w.solo_kv_head
    assert mh[best] > 0.999 and np.sort(mh)[-2] < mh[best]


# ---------------------------------------------------------------- selection variants (Sec. 4.4.1)

def test_average_bs1_equals_bruteforce_mean_over_all_query_heads():
    """bs = 1: every head's digest bound is exact, so the averaged score is the exact
    mean over all Hq query heads of q . k (each query head against its own KV head),
    and average top-k = brute-force exact top-k of that mean."""
    w = tiny([120, 77, 9], Hq=8, Hkv=4, d=32, bs=1, seed=41, n_sink=0, n_local=0, k_mid=10)
    qf = W.to_float(w.q, "bf16").astype(np.float64)
    K = W.to_float(k_view(w.kv, w.Hkv, 1, w.d)[:, :, 0, :], "bf16").astype(np.float64)
    avg = O.average_scores(w.kv, w.q, w.blk_off, w.ctx_len, w.Hq, w.Hkv, 1, w.d, O.BF16)
    rc, idx, cnt = O.select(avg, w.blk_off, np.full(w.B, 10, np.int32), 0, 0, 12)
    assert rc == 0
    for r in range(w.B):
        b0, b1 = int(w.blk_off[r]), int(w.blk_off[r + 1])
        logit = np.zeros(b1 - b0)
        for hq in range(w.Hq):
            logit += K[b0:b1, hq // w.G] @ qf[r, hq]
        logit /= w.Hq
        assert np.allclose(avg[b0:b1], logit, rtol=1e-13, atol=1e-12)
        order = np.lexsort((np.arange(b1 - b0), -logit))
        assert list(idx[r, : cnt[r]]) == list(np.sort(order[: min(10, b1 - b0)]))


def test_average_of_identical_heads_is_the_solohead_score():
    """All KV heads holding the same keys and every GQA group the same queries: the
    average over heads equals any single head's SoloHead score."""
    w = tiny([64, 30], Hq=8, Hkv=4, d=16, bs=4, seed=9)
    kv = w.kv.reshape(w.total_blocks, 2, w.Hkv, -1).copy()
    kv[:, :, 1:] = kv[:, :, :1]
    kv = kv.reshape(w.total_blocks, -1)
    q = w.q.reshape(w.B, w.Hkv, w.G, w.d).copy()
    q[:, 1:] = q[:, :1]
    q = q.reshape(w.B, w.Hq, w.d)
    avg = O.average_scores(kv, q, w.blk_off, w.ctx_len, w.Hq, w.Hkv, w.bs, w.d, O.BF16)
    dig = O.build_digests(kv, w.blk_off, w.ctx_len, w.Hkv, w.bs, w.d, O.BF16, 2)
    solo = O.score(q, dig, w.blk_off, w.Hq, w.Hkv, w.d, O.BF16, 2)
    assert np.allclose(avg, solo, rtol=1e-14, atol=1e-12)


def test_mam_over_middle_blocks_equals_bruteforce_softmax_mass():
    """The block-level middle (all blocks but the first n_sink and last n_local) passed
    to the token-level Eq. 2 as token counts equals a direct softmax over the raw keys
    summed over those blocks' tokens (partial last block included)."""
    w = tiny([45], Hq=4, Hkv=2, d=8, bs=4, seed=17)  # 12 blocks, the last one holds 1 token
    L, bs, n = int(w.ctx_len[0]), w.bs, int(w.n_blocks[0])
    ns, nl = 2, 3
    sink_tok, local_tok = ns * bs, L - (n - nl) * bs
    best, mq, mh = O.mam(w.q, w.kv, w.blk_off, w.ctx_len, 0, w.Hq, w.Hkv, bs, w.d, O.BF16, w.sm_scale,
                         sink_tok, local_tok)
    qf = W.to_float(w.q, "bf16").astype(np.float64)[0]
    K = W.to_float(k_view(w.kv, w.Hkv, bs, w.d), "bf16").astype(np.float64)  # [blk, h, row, c]
    for hq in range(w.Hq):
        keys = K[:, hq // w.G].reshape(-1, w.d)[:L]
        lg = keys @ qf[hq] * w.sm_scale
        p = np.exp(lg - lg.max())
        p /= p.sum()
        assert abs(mq[hq] - p[ns * bs:(n - nl) * bs].sum()) < 1e-12
    assert np.allclose(mh, mq.reshape(w.Hkv, w.G).mean(axis=1))
    assert best == int(np.argmax(mh))


# ---------------------------------------------------------------- headwise baseline (Sec. 3.4)

def test_missing_counts_hand_worked():
    """Set difference and runs on a hand-worked table: selected [0, 1, 2, 5, 6, 9] with
    entries -1 at 1, 2, 5 and 9 -> 4 missing blocks in 3 runs ({1, 2}, {5}, {9});
    an empty selection and an all-resident one count nothing."""
    table = np.array([[7, -1, -1, 3, 4, -1, 8, 2, 1, -1],
                      [0, 1, 2, 3, 4, 5, 6, 7, 8, 9],
                      [-1] * 10], np.int32)
    sel = np.full((3, 8), -1, np.int32)
    sel[0, :6] = [0, 1, 2, 5, 6, 9]
    sel[1, :4] = [1, 2, 3, 4]
    cnt = np.array([6, 4, 0], np.int32)
    units, runs = O.missing_counts(sel, cnt, table)
    assert list(units) == [4, 0, 0] and list(runs) == [3, 0, 0]


def test_missing_counts_agree_with_the_recall_statistics():
    """The headwise counter and the recall (two separate implementations of Sec. 2.2's set
    difference) agree on missing blocks and runs for random selections and tables."""
    rng = np.random.default_rng(12)
    for trial in range(20):
        n = rng.integers(1, 40, size=4)
        blk_off = np.concatenate([[0], np.cumsum(n)]).astype(np.int64)
        maxb = int(n.max())
        table = np.full((4, maxb), -1, np.int32)
        k_max = maxb
        sel = np.full((4, k_max), -1, np.int32)
        cnt = np.zeros(4, np.int32)
        slot = 0
        for r in range(4):
            res = np.flatnonzero(rng.random(n[r]) < 0.4)
            table[r, res] = np.arange(slot, slot + res.size)
            slot += res.size
            c = int(rng.integers(0, n[r] + 1))
            sel[r, :c] = np.sort(rng.choice(n[r], c, replace=False))
            cnt[r] = c
        units, runs = O.missing_counts(sel, cnt, table)
        U = 16
        n_free = int(units.sum())
        free = np.arange(slot, slot + n_free, dtype=np.int32)
        pool = np.zeros((slot + n_free, U), np.uint8)
        host = np.zeros((int(blk_off[-1]), U), np.uint8)
        rc, fh, stats = O.recall(host, blk_off, sel, cnt, table.copy(), free, 0, pool, U)
        assert rc == 0
        assert stats[0] == units.sum() and stats[1] == runs.sum() and fh == n_free


def test_headwise_bs1_each_head_is_its_exact_topk_and_solo_row_is_solohead():
    """bs = 1: every KV head's headwise selection is the exact top-k of that head's
    group-mean logits (brute force), and the row of any head equals SoloHead with that head."""
    w = tiny([90, 33, 5], Hq=8, Hkv=4, d=16, bs=1, seed=41, n_sink=0, n_local=0, k_mid=9)
    k_mid = np.full(w.B, 9, np.int32)
    sel, cnt, sc = O.headwise_select(w.kv, w.q, w.blk_off, w.ctx_len, w.Hq, w.Hkv, 1, w.d, O.BF16, k_mid, 0, 0, 12)
    qf = W.to_float(w.q, "bf16").astype(np.float64)
    K = W.to_float(k_view(w.kv, w.Hkv, 1, w.d)[:, :, 0, :], "bf16").astype(np.float64)
    for h in range(w.Hkv):
        for r in range(w.B):
            b0, b1 = int(w.blk_off[r]), int(w.blk_off[r + 1])
            logit = K[b0:b1, h] @ qf[r, h * w.G:(h + 1) * w.G].mean(axis=0)
            order = np.lexsort((np.arange(b1 - b0), -logit))
            assert list(sel[h, r, : cnt[h, r]]) == list(np.sort(order[: min(9, b1 - b0)]))
        dig = O.build_digests(w.kv, w.blk_off, w.ctx_len, w.Hkv, 1, w.d, O.BF16, h)
        rc, idx, c1 = O.select(O.score(w.q, dig, w.blk_off, w.Hq, w.Hkv, w.d, O.BF16, h), w.blk_off, k_mid, 0, 0, 12)
        assert rc == 0 and np.array_equal(idx, sel[h]) and np.array_equal(c1, cnt[h])
