"""Step-end release of a recall (the fixed-size hot set of Sec. 4.2): after a layer-step the
recalled blocks leave the table and their slots return to the free list, exactly undoing
the recall, so the next step recalls and attends identically."""
import pytest
import torch

from paper_2609_34555_amd import pulse as P
from paper_2609_34555_amd import workloads as W

from parity import build, say

pytestmark = pytest.mark.gpu


def _state(st):
    return st.table.clone(), int(st.free_head.item()), st.recall_stats()


def test_release_undoes_chained_recall_and_next_step_repeats():
    say("\n[gpu] release chained")
    spec, s = W.preset(2, ctx_scale=1 / 8)
    w, st = build(spec, s)
    st.reset()
    st.decode_layer()
    torch.cuda.synchronize()
    assert st.status() == 0
    out1, lse1 = st.out.clone(), st.lse.clone()
    table1, fh1, stats1 = _state(st)
    assert stats1[0] > 0 and fh1 == stats1[0]
    for _ in range(2):  # the second release is a no-op
        st.release(chained=True)
        torch.cuda.synchronize()
        assert st.status() == 0
        assert torch.equal(st.table, st.table0) and int(st.free_head.item()) == 0
        assert st.recall_stats() == (0, 0, 0)
    st.out.zero_()
    st.decode_layer()  # next step from the released state: same slots, same results
    torch.cuda.synchronize()
    assert st.status() == 0
    assert torch.equal(st.out, out1) and torch.equal(st.lse, lse1)
    assert torch.equal(st.table, table1) and _state(st)[1:] == (fh1, stats1)


def test_release_after_standalone_and_engine_recall():
    say("\n[gpu] release standalone / engine")
    spec, s = W.preset(2, ctx_scale=1 / 16)
    w, st = build(spec, s)
    st.reset()
    st.select()
    st.recall()
    torch.cuda.synchronize()
    assert st.status() == 0 and st.recall_stats()[0] > 0
    st.release(chained=False)
    torch.cuda.synchronize()
    assert torch.equal(st.table, st.table0) and int(st.free_head.item()) == 0
    eng = P.GatherScatterEngine(st.shape, n_workers=2, max_blocks_per_call=w.B * st.k_max, staging_blocks=32)
    try:
        st.recall_gs(eng)
        torch.cuda.synchronize()
        assert st.status() == 0 and st.recall_stats()[0] > 0
        st.release(chained=False)
        torch.cuda.synchronize()
        assert torch.equal(st.table, st.table0) and int(st.free_head.item()) == 0
    finally:
        eng.destroy()


def test_release_after_exhaustion_changes_nothing():
    say("\n[gpu] release after exhaustion")
    spec, s = W.custom("exh", [3000, 3000], Hq=32, Hkv=8, bs=16, k_mid=40, n_sink=1, n_local=8,
                       resident_frac=0.05, n_free_override=10)
    w, st = build(spec, s)
    st.reset()
    st.decode_layer()
    torch.cuda.synchronize()
    assert st.status() == P.PULSE_ERR_POOL_EXHAUSTED
    st.dev_status.zero_()
    st.release(chained=True)
    torch.cuda.synchronize()
    assert st.status() == 0
    assert torch.equal(st.table, st.table0) and int(st.free_head.item()) == 0


def _snap(st):
    return (st.out.clone(), st.lse.clone(), st.table.clone(), int(st.free_head.item()), st.recall_stats(),
            st.pool.clone())


def test_release_previous_in_scoring_kernel_equals_separate_release():
    """pulse_decode_layer with release_previous: each step first undoes the previous step's
    recall inside the scoring kernel; every step then matches decode_layer + a separate
    pulse_release_recalled bit for bit, and the first step (nothing recalled yet) and a step
    after an explicit release (statistics cleared) release nothing."""
    say("\n[gpu] release_previous vs separate release")
    spec, s = W.preset(2, ctx_scale=1 / 8)
    w, a = build(spec, s)
    _, b = build(spec, s)  # a second, identical state
    a.reset()
    b.reset()
    for step in range(3):
        a.decode_layer()
        b.decode_layer(release_previous=True)
        torch.cuda.synchronize()
        assert a.status() == 0 and b.status() == 0
        sa, sb = _snap(a), _snap(b)
        assert sa[4][0] > 0
        for x, y in zip(sa, sb):
            assert (torch.equal(x, y) if isinstance(x, torch.Tensor) else x == y), step
        a.release(chained=True)
    b.release(chained=True)  # clears the statistics: the next fused release is a no-op
    torch.cuda.synchronize()
    assert torch.equal(b.table, b.table0) and int(b.free_head.item()) == 0
    b.decode_layer(release_previous=True)
    a.decode_layer()
    torch.cuda.synchronize()
    for x, y in zip(_snap(a), _snap(b)):
        assert torch.equal(x, y) if isinstance(x, torch.Tensor) else x == y


def test_release_previous_after_exhaustion_releases_nothing():
    say("\n[gpu] release_previous after exhaustion")
    spec, s = W.custom("exh2", [3000, 3000], Hq=32, Hkv=8, bs=16, k_mid=40, n_sink=1, n_local=8,
                       resident_frac=0.05, n_free_override=10)
    w, st = build(spec, s)
    st.reset()
    st.decode_layer(release_previous=True)
    torch.cuda.synchronize()
    assert st.status() == P.PULSE_ERR_POOL_EXHAUSTED
    st.dev_status.zero_()
    st.decode_layer(release_previous=True)  # nothing was recalled: no rewind, same exhaustion
    torch.cuda.synchronize()
    assert st.status() == P.PULSE_ERR_POOL_EXHAUSTED
    assert torch.equal(st.table, st.table0) and int(st.free_head.item()) == 0


def test_release_previous_after_standalone_recall_and_reset():
    """The workspace last used by the standalone calls (another layout of the plan) and a
    reset: the fused release finds no recall in the statistics and touches nothing."""
    say("\n[gpu] release_previous after standalone use")
    spec, s = W.preset(2, ctx_scale=1 / 16)
    w, st = build(spec, s)
    st.reset()
    st.select()
    st.recall()
    st.release(chained=False)
    st.reset()
    st.decode_layer(release_previous=True)
    torch.cuda.synchronize()
    assert st.status() == 0 and st.recall_stats()[0] > 0
    first = _snap(st)
    st.decode_layer(release_previous=True)
    torch.cuda.synchronize()
    assert st.status() == 0
    for x, y in zip(first, _snap(st)):
        assert torch.equal(x, y) if isinstance(x, torch.Tensor) else x == y
