"""GPU parity: every stage of the gfx950 path against the CPU oracle, through the C ABI.

Sizes are ones the oracle finishes in seconds but that span several tiles of
every kernel and have ragged tails; edge cases cover empty requests, partial
last blocks, k >= #blocks, k = 0, everything resident, nothing resident, exact
duplicate blocks (ties), pool exhaustion and malformed selections."""
import numpy as np
import pytest
import torch

from oracle import pulse_oracle as O
from paper_2609_34555_amd import pulse as P
from paper_2609_34555_amd import workloads as W

from parity import (assert_attention_close, assert_recall_equal, assert_selection_ok, build, full_check,
                    oracle_attention, oracle_recall, oracle_selection, random_case, random_case_long, say)

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _name(request):
    say(f"\n[gpu] {request.node.name}")
    yield
    torch.cuda.synchronize()


# ------------------------------------------------------------------ digests

@pytest.mark.parametrize("dtype,bs,coherent", [("bf16", 16, True), ("f16", 16, False), ("bf16", 32, True),
                                               ("f16", 64, True)])
def test_digests_bitexact_every_head(dtype, bs, coherent):
    spec, s = W.custom("dg", [1000, 17, 1, 513, 64], Hq=16, Hkv=4, bs=bs, dtype=dtype, k_mid=8)
    w, st = build(spec, s, coherent=coherent)
    for h in range(w.Hkv):
        out = torch.zeros_like(st.digests)
        st.build_digests(h, out=out)
        torch.cuda.synchronize()
        got = out.cpu().numpy().view(np.uint16)[: w.total_blocks]
        want = O.build_digests(w.kv, w.blk_off, w.ctx_len, w.Hkv, w.bs, w.d, w.dtype_code, h)
        assert np.array_equal(got, want), f"head {h}"
    assert st.status() == 0


def test_digests_signed_zeros():
    spec, s = W.custom("z", [48], Hq=8, Hkv=2, bs=16, dtype="f16", k_mid=1)
    w, st = build(spec, s)
    K = w.kv.reshape(w.total_blocks, 2, w.Hkv, w.bs, w.d)
    K[0, 0, 0, :, :] = 0
    K[0, 0, 0, 3, :64] = 0x8000  # -0 in half of the channels of one token
    K[1, 0, 0, :, :] = 0x8000
    K[1, 0, 0, 5, 7] = 0
    st.build_digests(0)
    torch.cuda.synchronize()
    got = st.digests.cpu().numpy().view(np.uint16)[: w.total_blocks]
    want = O.build_digests(w.kv, w.blk_off, w.ctx_len, w.Hkv, w.bs, w.d, w.dtype_code, 0)
    assert np.array_equal(got, want)


# ------------------------------------------------------------------ selection

SELECT_CASES = [
    # name, ctx_lens, Hq, Hkv, bs, dtype, k_mid, n_sink, n_local
    ("ragged", [5000, 4096, 17, 0, 2100], 32, 8, 16, "bf16", [40, 3, 7, 5, 500], 1, 8),
    ("g1_f16", [3000, 700], 8, 8, 16, "f16", 25, 1, 2),
    ("g12", [2048, 999], 48, 4, 32, "bf16", 11, 2, 2),
    ("g16_bs64", [9000, 64], 16, 1, 64, "bf16", 30, 0, 0),
    ("k_ge_n", [400, 300], 32, 8, 16, "bf16", 1000, 1, 8),
    ("k_zero", [400, 300], 32, 8, 16, "bf16", 0, 1, 8),
    ("forced_cover", [100, 40], 32, 8, 16, "bf16", 4, 3, 5),
    ("big_n", [131072, 70000], 32, 8, 16, "bf16", [247, 100], 1, 8),
    # > 8192 middle blocks: keys re-read from L2 each radix pass, two ordered tiles
    ("uncached_two_tiles", [150000, 140000, 3000], 32, 8, 16, "bf16", [300, 5, 40], 1, 8),
    # 100 / 140 / 60 / 100 blocks: the equal-length guess of the score and select kernels
    # (100 blocks each) holds for requests 0 and 3 and fails for 1 (length) and 2 (offset)
    ("equal_length_guess", [1600, 2240, 960, 1585], 32, 8, 16, "bf16", [20, 31, 9, 50], 1, 8),
]


@pytest.mark.parametrize("case", SELECT_CASES, ids=[c[0] for c in SELECT_CASES])
def test_select_parity(case):
    name, ctx, Hq, Hkv, bs, dtype, k_mid, n_sink, n_local = case
    spec, s = W.custom(name, ctx, Hq=Hq, Hkv=Hkv, bs=bs, dtype=dtype, k_mid=k_mid, n_sink=n_sink,
                       n_local=n_local, heavy_per_req=6)
    w, st = build(spec, s)
    scores = torch.zeros(max(w.total_blocks, 1), dtype=torch.float32, device="cuda")
    st.select(scores=scores)
    torch.cuda.synchronize()
    assert st.status() == 0
    dig = st.digests.cpu().numpy().view(np.uint16)[: w.total_blocks]
    rc, oidx, ocnt, osc = oracle_selection(w, dig)
    gidx, gcnt = st.selection()
    ties = assert_selection_ok(w, gidx, gcnt, oidx, ocnt, osc)
    say(f"  boundary near-ties: {ties}")
    # scores of middle blocks agree with the exact value to fp32 rounding of a short sum
    g = scores.cpu().numpy().astype(np.float64)
    for r in range(w.B):
        b0, n = int(w.blk_off[r]), int(w.n_blocks[r])
        lo, hi = b0 + w.n_sink, b0 + n - w.n_local
        if hi > lo:
            err = np.abs(g[lo:hi] - osc[lo:hi]) / np.maximum(np.abs(osc[lo:hi]), 1.0)
            assert err.max() < 4e-6


def test_chained_layer_beyond_key_cache():
    """A chained layer-step whose requests exceed the select kernel's one tile of keys held in
    registers and its prefetched table entries (plan mode reads the rest of the table in the kernel)."""
    spec, s = W.custom("long", [150000, 9000], Hq=32, Hkv=8, bs=16, dtype="bf16", k_mid=[200, 30], n_sink=1,
                       n_local=8, resident_frac=0.1, heavy_per_req=6)
    w, st = build(spec, s)
    res = full_check(w, st, chained=True)
    say(f"  attn max err {res['attn_err']}")


def test_chained_layer_equal_length_guess():
    """A chained layer-step on requests of 100 / 140 / 60 / 100 blocks: the kernels' loads at
    equal-length offsets are used for requests 0 and 3 and reloaded for 1 and 2."""
    spec, s = W.custom("eqguess", [1600, 2240, 960, 1585], Hq=32, Hkv=8, bs=16, dtype="bf16", k_mid=[20, 31, 9, 50],
                       n_sink=1, n_local=8, resident_frac=0.1, heavy_per_req=6)
    w, st = build(spec, s)
    assert w.total_blocks == 400 and list(w.n_blocks) == [100, 140, 60, 100]
    res = full_check(w, st, chained=True)
    say(f"  stats={res['stats']} attn max err {res['attn_err']}")


def test_chained_layer_at_maximum_batch():
    """4096 requests (the largest batch the selection and recall kernels take), short ragged
    contexts: every request's plan, allocation order and attention against the oracle."""
    rng = np.random.default_rng(4096)
    ctx = [int(x) for x in rng.integers(1, 160, 4096)]
    spec, s = W.custom("maxb", ctx, Hq=8, Hkv=2, bs=16, dtype="bf16", k_mid=3, n_sink=1, n_local=1,
                       resident_frac=0.2, heavy_per_req=1)
    w, st = build(spec, s)
    res = full_check(w, st, chained=True)
    say(f"  {w.B} requests, {res['stats'][0]} recalled blocks, attn max err {res['attn_err']}")
    # the next step with the fused release (B * k_max plan entries spread over the scoring
    # grid) repeats the step exactly
    table1, fh1, stats1 = st.table.clone(), int(st.free_head.item()), st.recall_stats()
    out1 = st.out.clone()
    st.out.zero_()
    st.decode_layer(release_previous=True)
    torch.cuda.synchronize()
    assert st.status() == 0
    assert torch.equal(st.table, table1) and int(st.free_head.item()) == fh1 and st.recall_stats() == stats1
    assert torch.equal(st.out, out1)


def test_select_duplicate_blocks_take_lowest_index():
    """21 exact copies of each request's best middle block compete for 7 places: only the
    lowest-index rule decides, and both sides must pick the same blocks."""
    spec, s = W.custom("dup", [1600, 1600], Hq=32, Hkv=8, bs=16, dtype="bf16", k_mid=7, n_sink=1, n_local=8,
                       planted=False)
    w, st = build(spec, s)
    dig = O.build_digests(w.kv, w.blk_off, w.ctx_len, w.Hkv, w.bs, w.d, w.dtype_code, w.solo_kv_head)
    sc = O.score(w.q, dig, w.blk_off, w.Hq, w.Hkv, w.d, w.dtype_code, w.solo_kv_head)
    for r in range(w.B):
        b0, n = int(w.blk_off[r]), int(w.n_blocks[r])
        best = b0 + 1 + int(np.argmax(sc[b0 + 1: b0 + n - 8]))
        for j in range(30, 50):
            if b0 + j != best:
                w.kv[b0 + j] = w.kv[best]
    st.build_digests(w.solo_kv_head)
    st.select()
    torch.cuda.synchronize()
    dig = st.digests.cpu().numpy().view(np.uint16)[: w.total_blocks]
    rc, oidx, ocnt, osc = oracle_selection(w, dig)
    gidx, gcnt = st.selection()
    assert np.array_equal(gidx, oidx) and np.array_equal(gcnt, ocnt)
    for r in range(w.B):
        mid = [j for j in gidx[r, : gcnt[r]] if 1 <= j < w.n_blocks[r] - 8]
        assert len(mid) == 7 and max(mid) < 50


def test_equal_keys_across_two_tiles_chained():
    """Every block of a 9000-block request holds the same keys, so every middle score is
    equal: the first 8500 middle blocks in index order are taken, the equal keys ranked
    across the selection pass's 8192-block tile boundary.  Only the forced blocks are
    resident, so the recall plan is one run of 8500 blocks crossing that boundary;
    selection, plan, pool and attention against the oracle."""
    spec, s = W.custom("eq2t", [9000 * 16], Hq=32, Hkv=8, bs=16, dtype="bf16", k_mid=8500, n_sink=1, n_local=8,
                       resident_frac=0.0, planted=False)
    w, st = build(spec, s)
    w.kv[1:] = w.kv[0]  # one block's keys and values everywhere, resident copies included
    st.pool[: w.resident_blocks.size] = torch.from_numpy(w.kv[w.resident_blocks].view(np.int16)).cuda()
    st.build_digests(w.solo_kv_head)
    res = full_check(w, st, chained=True)
    assert res["ties"] == 0 and res["stats"][0] == 8500 and res["stats"][1] == 1, res["stats"]
    gidx, gcnt = st.selection()
    assert gcnt[0] == 8509 and np.array_equal(gidx[0, :8501], np.arange(8501))


def test_tied_keys_cut_across_two_tiles():
    """201 exact copies of a request's best middle block straddle the 8192-block tile
    boundary (blocks 8100 .. 8300) and only 150 places remain for them: the lowest-index
    rule takes the first copies in block order, with the equal-key ranks of the first tile
    carried into the second; both sides must pick the same blocks."""
    spec, s = W.custom("tie2t", [9000 * 16], Hq=32, Hkv=8, bs=16, dtype="bf16", k_mid=151, n_sink=1, n_local=8,
                       planted=False)
    w, st = build(spec, s)
    dig = O.build_digests(w.kv, w.blk_off, w.ctx_len, w.Hkv, w.bs, w.d, w.dtype_code, w.solo_kv_head)
    sc = O.score(w.q, dig, w.blk_off, w.Hq, w.Hkv, w.d, w.dtype_code, w.solo_kv_head)
    best = 1 + int(np.argmax(sc[1: 9000 - 8]))
    src = w.kv[best].copy()
    w.kv[8100:8301] = src
    st.build_digests(w.solo_kv_head)
    st.select()
    torch.cuda.synchronize()
    assert st.status() == 0
    dig = st.digests.cpu().numpy().view(np.uint16)[: w.total_blocks]
    rc, oidx, ocnt, osc = oracle_selection(w, dig)
    gidx, gcnt = st.selection()
    assert rc == 0 and np.array_equal(gidx, oidx) and np.array_equal(gcnt, ocnt)
    mid = [j for j in gidx[0, : gcnt[0]] if 1 <= j < 9000 - 8]
    copies = [j for j in mid if 8100 <= j <= 8300]
    assert len(mid) == 151 and copies[0] == 8100 and 8192 <= copies[-1] <= 8300


@pytest.mark.parametrize("seed", range(48))
def test_random_workloads_against_oracle(seed):
    """Seeded random workloads (seed 26: a batch of one empty request), each one layer-step
    (chained for even seeds, stage by stage for odd ones) checked stage by stage against the
    oracle: digests, selection (R12 near ties), table, free head, statistics, every pool byte,
    attention."""
    spec, s = random_case(seed)
    w, st = build(spec, s)
    say(f"  B={w.B} ctx={list(w.ctx_len)} bs={w.bs} G={w.Hq // w.Hkv} Hkv={w.Hkv} k_mid={list(w.k_mid)} "
        f"sink/local={w.n_sink}/{w.n_local}")
    res = full_check(w, st, chained=seed % 2 == 0)
    say(f"  stats={res['stats']} ties={res['ties']} attn max err {res['attn_err']}")


@pytest.mark.parametrize("seed", [1, 6, 7, 19, 24, 39])
def test_random_long_context_workloads_against_oracle(seed):
    """Seeded long-context workloads: batches up to 24 requests, the first three up to 300K tokens
    (up to three 8192-block selection tiles), budgets up to 600 blocks and recalls of up to
    735 MB, one layer-step (chained for even seeds, stage by stage for odd ones) checked stage
    by stage against the oracle."""
    spec, s = random_case_long(seed)
    w, st = build(spec, s)
    say(f"  B={w.B} max blocks={int(w.n_blocks.max())} bs={w.bs} G={w.Hq // w.Hkv} Hkv={w.Hkv} "
        f"sink/local={w.n_sink}/{w.n_local}")
    res = full_check(w, st, chained=seed % 2 == 0)
    say(f"  stats={res['stats']} ties={res['ties']} attn max err {res['attn_err']}")


def test_select_overflow_reports_and_empties_request():
    spec, s = W.custom("ovf", [800, 800], Hq=32, Hkv=8, bs=16, k_mid=[5, 30], n_sink=1, n_local=8)
    w, st = build(spec, s, k_max=20)
    st.select()
    torch.cuda.synchronize()
    assert st.status() == P.PULSE_ERR_SELECT_OVERFLOW
    gidx, gcnt = st.selection()
    assert gcnt[1] == 0 and np.all(gidx[1] == -1) and gcnt[0] == 14


def test_chained_layer_with_overflowing_request():
    """pulse_decode_layer when one request's selection exceeds k_max: SELECT_OVERFLOW, that
    request's selection is empty (attention out 0, lse -inf), and the other requests are
    selected, recalled and attended exactly as the oracle does on the same inputs."""
    spec, s = W.custom("ovfc", [900, 1500, 700], Hq=32, Hkv=8, bs=16, k_mid=[6, 40, 4], n_sink=1, n_local=8,
                       resident_frac=0.1, heavy_per_req=4)
    w, st = build(spec, s, k_max=24)
    st.reset()
    st.decode_layer()
    torch.cuda.synchronize()
    assert st.status() == P.PULSE_ERR_SELECT_OVERFLOW
    dig = st.digests.cpu().numpy().view(np.uint16)[: w.total_blocks]
    gidx, gcnt = st.selection()
    rc, oidx, ocnt, osc = oracle_selection(w, dig, k_max=st.k_max)
    assert rc == O.ERR_SELECT_OVERFLOW and ocnt[1] == 0 and gcnt[1] == 0 and np.all(gidx[1] == -1)
    assert_selection_ok(w, gidx, gcnt, oidx, ocnt, osc)
    rc, table, pool, fh, stats = oracle_recall(w, gidx, gcnt)
    assert rc == 0 and stats[0] > 0
    assert_recall_equal(st, table, pool, fh, stats)
    out, lse = oracle_attention(w, pool, table, gidx, gcnt)
    assert np.all(out[1] == 0) and np.all(np.isneginf(lse[1]))
    err = assert_attention_close(st, out, lse)
    say(f"  stats={stats} attn_err={err[0]:.1e}")


# ------------------------------------------------------------------ recall

RECALL_CASES = [
    ("ragged_shuffled", [5000, 4096, 17, 0, 2100], 16, "bf16", 40, 0.10, "shuffled", True),
    ("noncoherent", [3000, 2500, 2000], 16, "bf16", 60, 0.05, "ascending", False),
    ("bs32_runs", [30000, 9000], 32, "bf16", 200, 0.03, "ascending", True),
    ("all_resident", [2000, 1000], 16, "f16", 50, 1.0, "ascending", True),
    ("none_resident", [2000, 1000], 16, "bf16", 50, 0.0, "shuffled", True),
    ("hkv1_8k_unit", [4000], 16, "bf16", 30, 0.1, "ascending", True),
]


@pytest.mark.parametrize("case", RECALL_CASES, ids=[c[0] for c in RECALL_CASES])
def test_recall_parity(case):
    name, ctx, bs, dtype, k_mid, frac, order, coherent = case
    Hq, Hkv = (8, 1) if name == "hkv1_8k_unit" else (32, 8)
    spec, s = W.custom(name, ctx, Hq=Hq, Hkv=Hkv, bs=bs, dtype=dtype, k_mid=k_mid, n_sink=1, n_local=2,
                       resident_frac=frac, heavy_per_req=20, free_order=order)
    w, st = build(spec, s, coherent=coherent)
    st.select()
    st.recall()
    torch.cuda.synchronize()
    assert st.status() == 0
    gidx, gcnt = st.selection()
    rc, table, pool, fh, stats = oracle_recall(w, gidx, gcnt)
    assert rc == 0
    assert_recall_equal(st, table, pool, fh, stats)
    say(f"  missing={stats[0]} runs={stats[1]} bytes={stats[2]}")


def test_recall_pool_exhaustion_leaves_state():
    spec, s = W.custom("exh", [3000, 3000], Hq=32, Hkv=8, bs=16, k_mid=40, n_sink=1, n_local=8,
                       resident_frac=0.05, n_free_override=10)
    w, st = build(spec, s)
    st.select()
    pool0 = st.pool.clone()
    st.recall()
    torch.cuda.synchronize()
    assert st.status() == P.PULSE_ERR_POOL_EXHAUSTED
    assert torch.equal(st.table, st.table0) and int(st.free_head.item()) == 0 and torch.equal(st.pool, pool0)
    n_missing, _, nbytes = st.recall_stats()
    assert n_missing > 10 and nbytes == 0
    gidx, gcnt = st.selection()
    rc, table, pool, fh, stats = oracle_recall(w, gidx, gcnt)  # statistics as the oracle's, exactly
    assert rc == O.ERR_POOL_EXHAUSTED
    assert_recall_equal(st, table, pool, fh, stats)


def test_recall_rejects_unsorted_and_out_of_range():
    spec, s = W.custom("bad", [3000, 3000], Hq=32, Hkv=8, bs=16, k_mid=40, n_sink=1, n_local=8)
    w, st = build(spec, s)
    st.select()
    torch.cuda.synchronize()
    idx = st.sel_idx.clone()
    st.sel_idx[1, 3], st.sel_idx[1, 4] = idx[1, 4], idx[1, 3]
    st.recall()
    torch.cuda.synchronize()
    assert st.status() == P.PULSE_ERR_BAD_INDEX
    assert torch.equal(st.table, st.table0) and int(st.free_head.item()) == 0
    st.reset()
    st.sel_idx.copy_(idx)
    st.sel_idx[0, 5] = 10 ** 6  # beyond the request's blocks
    st.sel_idx[0, 6:] = -1
    st.sel_cnt[0] = 6
    st.recall()
    torch.cuda.synchronize()
    assert st.status() == P.PULSE_ERR_BAD_INDEX and torch.equal(st.table, st.table0)
    gidx, gcnt = st.selection()
    rc, table, pool, fh, stats = oracle_recall(w, gidx, gcnt)
    assert rc == O.ERR_BAD_INDEX and stats == (0, 0, 0)
    assert_recall_equal(st, table, pool, fh, stats)


BAD_FREE = ["slot_past_pool", "negative_slot", "head_past_list", "bad_slot_past_range", "table_entry_past_pool"]


@pytest.mark.parametrize("bad", BAD_FREE)
@pytest.mark.parametrize("path", ["recall_gather", "decode_layer", "engine"])
def test_recall_rejects_bad_free_slot(path, bad):
    """A free list whose entries in the range the recall takes lie outside the pool, a
    free-list head outside the list, or a selected block whose table entry lies past the pool:
    BAD_INDEX, and table, free head, statistics and every pool byte exactly as the oracle
    leaves them (nothing written, bytes 0).  A bad entry past the free-list range is never
    read.  Afterwards a clean recall on the same state matches the oracle.  Covers the
    standalone recall, the chained layer-step and the paper's engine."""
    spec, s = W.custom("badfree", [3000, 2000, 700], Hq=32, Hkv=8, bs=16, k_mid=40, n_sink=1, n_local=8,
                       resident_frac=0.05, heavy_per_req=10)
    w, st = build(spec, s)
    eng = (P.GatherScatterEngine(st.shape, n_workers=2, max_blocks_per_call=w.B * st.k_max, staging_blocks=16)
           if path == "engine" else None)
    try:
        st.select()
        torch.cuda.synchronize()
        gidx, gcnt = st.selection()
        rc0, _, _, _, clean = oracle_recall(w, gidx, gcnt)
        n_miss = clean[0]
        assert rc0 == 0 and n_miss >= 3 and n_miss < w.free_slots.size
        free, fh0, table0 = w.free_slots.copy(), 0, w.table0.copy()
        if bad == "table_entry_past_pool":
            table0[1, 0] = w.n_slots  # request 1's sink block: always selected
        elif bad == "slot_past_pool":
            free[n_miss - 1] = w.n_slots  # the last slot the recall takes
        elif bad == "negative_slot":
            free[n_miss // 2] = -3
        elif bad == "head_past_list":
            fh0 = int(w.free_slots.size) + 1
        else:
            free[n_miss] = -1  # first entry past the range: not read
        st.reset()
        st.free_slots.copy_(torch.from_numpy(free))
        st.free_head.fill_(fh0)
        st.table.copy_(torch.from_numpy(table0))
        pool0 = st.pool.clone()

        def run():
            if path == "recall_gather":
                st.recall()
            elif path == "decode_layer":
                st.decode_layer()
            else:
                seq = st.recall_gs(eng, wait=False)
                try:
                    eng.wait(seq, 20000)
                except P.PulseError as e:  # the call's device status
                    assert e.status == P.PULSE_ERR_BAD_INDEX
            torch.cuda.synchronize()

        run()
        gidx, gcnt = st.selection()
        rc, table, pool, fh, stats = oracle_recall(w, gidx, gcnt, free_slots=free, free_head=fh0, table0=table0)
        say(f"  {path}/{bad}: oracle rc={rc} stats={stats}; gpu status={st.status()} stats={st.recall_stats()}")
        if bad == "bad_slot_past_range":
            assert rc == 0 and st.status() == 0
            assert_recall_equal(st, table, pool, fh, stats)
            return
        assert rc == O.ERR_BAD_INDEX and stats[2] == 0
        assert st.status() == P.PULSE_ERR_BAD_INDEX
        assert np.array_equal(st.table_np(), table0) and torch.equal(st.pool, pool0)
        assert_recall_equal(st, table, pool, fh, stats)
        # nothing changed: a clean recall of the same selection on this state matches the oracle
        st.free_slots.copy_(torch.from_numpy(w.free_slots))
        st.free_head.fill_(0)
        st.table.copy_(st.table0)
        st.dev_status.zero_()
        run()
        assert st.status() == 0
        gidx, gcnt = st.selection()
        rc, table, pool, fh, stats = oracle_recall(w, gidx, gcnt)
        assert rc == 0 and stats == clean
        assert_recall_equal(st, table, pool, fh, stats)
    finally:
        if eng is not None:
            eng.destroy()


# ------------------------------------------------------------------ attention

ATTN_CASES = [
    # name, ctx, Hq, Hkv, bs, dtype, k_mid, planted
    ("cfg1_like_f16", [4096], 32, 8, 16, "f16", 16, True),
    ("unplanted_ragged", [5000, 4097, 17, 1, 2100], 32, 8, 16, "bf16", [40, 3, 7, 5, 100], False),
    ("planted_bs32_g8", [20000, 9000], 64, 8, 32, "bf16", 120, True),
    ("bs64_g2_f16", [7000, 100], 16, 8, 64, "f16", 33, False),
    ("g16", [3000], 16, 1, 16, "bf16", 64, False),
    ("g3", [2500, 333], 24, 8, 16, "bf16", 21, False),
    ("empty_request", [0, 900], 32, 8, 16, "bf16", 10, False),
]


@pytest.mark.parametrize("case", ATTN_CASES, ids=[c[0] for c in ATTN_CASES])
def test_attention_parity_stagewise(case):
    name, ctx, Hq, Hkv, bs, dtype, k_mid, planted = case
    spec, s = W.custom(name, ctx, Hq=Hq, Hkv=Hkv, bs=bs, dtype=dtype, k_mid=k_mid, n_sink=1, n_local=2,
                       resident_frac=0.1, heavy_per_req=5, planted=planted)
    w, st = build(spec, s)
    res = full_check(w, st, chained=False)
    say(f"  attn max err {res['attn_err']}")


def test_attention_single_token_is_value_row():
    spec, s = W.custom("one", [1, 17], Hq=8, Hkv=2, bs=16, dtype="bf16", k_mid=1, n_sink=1, n_local=1)
    w, st = build(spec, s)
    st.reset()
    st.decode_layer()
    torch.cuda.synchronize()
    V = w.kv.reshape(w.total_blocks, 2, w.Hkv, w.d, w.bs)[:, 1]
    got = st.out.cpu().numpy()
    for hq in range(w.Hq):
        want = W.to_float(V[0, hq // w.G, :, 0], "bf16")
        assert np.array_equal(got[0, hq], want)


# ------------------------------------------------------------------ chained layer-step

@pytest.mark.parametrize("cid,kw", [
    (1, {}),
    (2, dict(ctx_scale=1 / 8)),
    (3, dict(ctx_scale=1 / 16, batch=6)),
    (4, dict(ctx_scale=1 / 8, layer=5)),
    (5, dict(ctx_scale=1 / 16)),
    (2, dict(ctx_scale=1 / 8, planted=False)),
])
def test_decode_layer_presets_scaled(cid, kw):
    spec, s = W.preset(cid, **kw)
    w, st = build(spec, s)
    res = full_check(w, st, chained=True)
    say(f"  cfg{cid} {kw}: stats={res['stats']} ties={res['ties']} attn_err={res['attn_err']}")


def test_decode_layer_is_deterministic():
    spec, s = W.preset(2, ctx_scale=1 / 8)
    w, st = build(spec, s)
    outs = []
    for _ in range(2):
        st.reset()
        st.decode_layer()
        torch.cuda.synchronize()
        outs.append((st.out.clone(), st.lse.clone(), st.table.clone(), st.sel_idx.clone(), st.stats.clone()))
    for a, b in zip(outs[0], outs[1]):
        assert torch.equal(a, b)


def test_decode_layer_stage_events_all_some_none():
    """Stage events change nothing in the results, and NULL entries are skipped: the
    recorded ones still bracket their stages (recall between events 2 and 3)."""
    from paper_2609_34555_amd import pulse as P

    spec, s = W.preset(2, ctx_scale=1 / 8)
    w, st = build(spec, s)
    outs = []
    sets = [P.EventSet(6) for _ in range(3)]
    try:
        for keep in (None, (0, 1, 2, 3, 4), (2, 3)):
            a = st.layer_args()
            if keep is not None:
                a.events = sets[len(outs)].masked_ptr(keep)
            if keep == (0, 1, 2, 3, 4):  # and the one between the split-K kernel and its combine
                a.attn_split_event = sets[len(outs)].arr[5]
            st.reset()
            assert P.pulse_decode_layer(a) == 0
            torch.cuda.synchronize()
            assert st.status() == 0
            outs.append((st.out.clone(), st.lse.clone(), st.table.clone(), st.stats.clone()))
        for o in outs[1:]:
            assert all(torch.equal(x, y) for x, y in zip(outs[0], o))
        for e in sets[1:]:
            assert e.elapsed_ms(2, 3) > 0.0
        assert sets[1].elapsed_ms(0, 4) >= sets[1].elapsed_ms(2, 3)
        assert 0.0 < sets[1].elapsed_ms(3, 5) <= sets[1].elapsed_ms(3, 4)
    finally:
        for e in sets:
            e.destroy()


def test_decode_layer_config2_full_size():
    """The benchmark's workload (8 x 32K, bf16) at full size, in the same launch
    configuration the benchmark times."""
    spec, s = W.preset(2)
    w, st = build(spec, s)
    res = full_check(w, st, chained=True)
    say(f"  cfg2 full: stats={res['stats']} ties={res['ties']} attn_err={res['attn_err']}")
    heavy_hit = 0
    gidx, gcnt = st.selection()
    for r in range(w.B):
        heavy_hit += len(set(np.asarray(w.heavy[r]).tolist()) & set(gidx[r, : gcnt[r]].tolist()))
    assert heavy_hit == sum(len(h) for h in w.heavy)  # SoloHead recovers every planted block


# ------------------------------------------------------------------ headwise selection (a9)

@pytest.mark.parametrize("cid,kw", [(4, dict(ctx_scale=1 / 16, batch=4, layer=3)),
                                    (2, dict(ctx_scale=1 / 8, batch=3))])
def test_headwise_selection_and_counts(cid, kw):
    spec, s = W.preset(cid, **kw)
    w, st = build(spec, s)
    sel, cnt, miss, runs = st.headwise()
    torch.cuda.synchronize()
    assert st.status() == 0
    gsel, gcnt = sel.cpu().numpy(), cnt.cpu().numpy()
    gmiss, gruns = miss.cpu().numpy(), runs.cpu().numpy()
    osel, ocnt, osc = O.headwise_select(w.kv, w.q, w.blk_off, w.ctx_len, w.Hq, w.Hkv, w.bs, w.d, w.dtype_code,
                                        w.k_mid, w.n_sink, w.n_local, st.k_max)
    total_units = 0
    for h in range(w.Hkv):
        assert_selection_ok(w, gsel[h], gcnt[h], osel[h], ocnt[h], osc[h])
        units, nruns = O.missing_counts(gsel[h], gcnt[h], w.table0)
        assert np.array_equal(gmiss[h], units) and np.array_equal(gruns[h], nruns)
        total_units += int(units.sum())
    # SoloHead on the same step: whole blocks, one transfer stream per run
    st.reset()
    st.select()
    st.recall()
    torch.cuda.synchronize()
    n_missing, n_runs, nbytes = st.recall_stats()
    say(f"  solohead: {n_missing} blocks / {n_runs} runs / {nbytes} B;  headwise: {total_units} head-blocks / "
        f"{int(gruns.sum())} runs / {total_units * w.unit_bytes // w.Hkv} B")
    assert total_units > n_missing  # heads disagree on most non-planted blocks


@pytest.mark.parametrize("seed", range(16))
def test_random_workloads_headwise(seed):
    """Headwise selection (every KV head with its own digests) and its per-head transfer and
    run counts on the seeded random workloads, against the oracle."""
    spec, s = random_case(seed)
    w, st = build(spec, s)
    sel, cnt, miss, runs = st.headwise()
    torch.cuda.synchronize()
    assert st.status() == 0
    gsel, gcnt = sel.cpu().numpy(), cnt.cpu().numpy()
    gmiss, gruns = miss.cpu().numpy(), runs.cpu().numpy()
    osel, ocnt, osc = O.headwise_select(w.kv, w.q, w.blk_off, w.ctx_len, w.Hq, w.Hkv, w.bs, w.d, w.dtype_code,
                                        w.k_mid, w.n_sink, w.n_local, st.k_max)
    for h in range(w.Hkv):
        assert_selection_ok(w, gsel[h], gcnt[h], osel[h], ocnt[h], osc[h])
        units, nruns = O.missing_counts(gsel[h], gcnt[h], w.table0)
        assert np.array_equal(gmiss[h], units) and np.array_equal(gruns[h], nruns)


# ------------------------------------------------------------------ multi-layer step, two streams

def test_multilayer_overlapped_matches_chained_and_oracle():
    from paper_2609_34555_amd.harness import MultiLayerStep

    ml = MultiLayerStep(n_layers=6, n_stores=2, ctx_scale=1 / 32, batch=4)
    ml.reset()
    ml.run_chained()
    torch.cuda.synchronize()
    snap = [(st.out.clone(), st.lse.clone(), st.table.clone(), st.stats.clone(), st.sel_idx.clone())
            for st in ml.layers]
    ml.reset()
    ml.run_overlapped()
    torch.cuda.synchronize()
    for st, ref in zip(ml.layers, snap):
        assert st.status() == 0
        for a, b in zip((st.out, st.lse, st.table, st.stats, st.sel_idx), ref):
            assert torch.equal(a, b)
    # layers sharing a store share keys and queries but not budgets or resident sets
    assert ml.layers[0].w.kv is ml.layers[2].w.kv
    assert not np.array_equal(ml.layers[0].w.table0, ml.layers[2].w.table0)
    for i in (0, 3):
        st = ml.layers[i]
        res = full_check(st.w, st, chained=True)
        say(f"  layer {i}: stats={res['stats']} attn_err={res['attn_err']}")


# ------------------------------------------------------------------ the paper's gather-scatter engine

@pytest.mark.parametrize("cid,kw", [(2, dict(ctx_scale=1 / 8)), (5, dict(ctx_scale=1 / 16)),
                                    (3, dict(ctx_scale=1 / 16, batch=5))])
def test_gather_scatter_engine_matches_oracle(cid, kw):
    """CPU gather -> one DMA -> GPU scatter, submitted through the host-visible mailbox:
    table, free head, stats and every pool byte as the oracle; attention after completion."""
    spec, s = W.preset(cid, **kw)
    w, st = build(spec, s)
    eng = P.GatherScatterEngine(st.shape, n_workers=4, max_blocks_per_call=w.B * st.k_max, staging_blocks=64)
    try:
        for rep in range(2):  # the second call reuses the engine (sequence numbers advance)
            st.reset()
            st.select()
            seq = st.recall_gs(eng, wait=False)
            with pytest.raises(P.PulseError):  # one call in flight per engine
                st.recall_gs(eng, wait=False)
            eng.wait(seq, 20000)
            assert eng.poll(seq)
            st.attention()
            torch.cuda.synchronize()
            assert st.status() == 0
            res = full_check(w, st, run=False)
            say(f"  rep {rep}: stats={res['stats']} timing={eng.last_timing()}")
    finally:
        eng.destroy()


@pytest.mark.parametrize("seed", range(12))
def test_random_workloads_engine_and_release(seed):
    """On seeded random workloads: the recall through the gather-scatter engine as the oracle
    does it (table, free head, statistics, every pool byte, then attention); then a chained
    layer-step that first releases that recall (release_previous) reproduces the oracle's
    step from the initial state."""
    spec, s = random_case(seed)
    w, st = build(spec, s)
    eng = P.GatherScatterEngine(st.shape, n_workers=2, max_blocks_per_call=max(1, w.B * st.k_max),
                                staging_blocks=16)
    try:
        st.reset()
        st.select()
        st.recall_gs(eng)
        st.attention()
        torch.cuda.synchronize()
        assert st.status() == 0
        full_check(w, st, run=False)
        st.release(chained=False)
        torch.cuda.synchronize()
        assert st.status() == 0 and np.array_equal(st.table_np(), w.table0) and int(st.free_head.item()) == 0
        st.decode_layer()
        st.decode_layer(release_previous=True)
        torch.cuda.synchronize()
        res = full_check(w, st, run=False)
        say(f"  stats={res['stats']}")
    finally:
        eng.destroy()


@pytest.mark.parametrize("Hkv,bs", [(1, 16), (3, 16), (3, 32)])
def test_gather_scatter_engine_block_sizes(Hkv, bs):
    """The engine's scatter on blocks of 8 KiB, 24 KiB (not a multiple of its 16 KiB chunks:
    it copies them in 8 KiB chunks) and 48 KiB: every pool byte, table, free head and
    statistics as the oracle; attention after completion."""
    spec, s = W.custom(f"gs_h{Hkv}_bs{bs}", [9000, 2500], Hq=2 * Hkv, Hkv=Hkv, bs=bs, k_mid=[60, 25], n_sink=1,
                       n_local=4, resident_frac=0.1, heavy_per_req=6)
    w, st = build(spec, s)
    assert w.unit_bytes == Hkv * bs * 512
    eng = P.GatherScatterEngine(st.shape, n_workers=2, max_blocks_per_call=w.B * st.k_max, staging_blocks=16)
    try:
        st.reset()
        st.select()
        st.recall_gs(eng)
        st.attention()
        torch.cuda.synchronize()
        assert st.status() == 0
        res = full_check(w, st, run=False)
        say(f"  unit {w.unit_bytes} B: stats={res['stats']}")
    finally:
        eng.destroy()


def test_gather_scatter_engine_pool_exhaustion():
    spec, s = W.custom("gsx", [3000, 3000], Hq=32, Hkv=8, bs=16, k_mid=40, n_sink=1, n_local=8,
                       resident_frac=0.05, n_free_override=10)
    w, st = build(spec, s)
    eng = P.GatherScatterEngine(st.shape, n_workers=2, max_blocks_per_call=w.B * st.k_max, staging_blocks=16)
    try:
        st.select()
        pool0 = st.pool.clone()
        seq = st.recall_gs(eng, wait=False)
        with pytest.raises(P.PulseError) as e:
            eng.wait(seq, 20000)
        assert e.value.status == P.PULSE_ERR_POOL_EXHAUSTED
        torch.cuda.synchronize()
        assert st.status() == P.PULSE_ERR_POOL_EXHAUSTED
        assert torch.equal(st.table, st.table0) and int(st.free_head.item()) == 0 and torch.equal(st.pool, pool0)
        gidx, gcnt = st.selection()
        rc, table, pool, fh, stats = oracle_recall(w, gidx, gcnt)
        assert rc == O.ERR_POOL_EXHAUSTED
        assert_recall_equal(st, table, pool, fh, stats)
    finally:
        eng.destroy()
