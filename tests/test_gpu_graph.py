"""A chained layer-step captured into a HIP graph (through torch's graph capture of the
stream the library launches on) and replayed: every replay, with eager steps and host
synchronisations in between, leaves the same selection, table, statistics, pool bytes and
attention output as the eager step.  The chain records no memset, so it is capturable;
each step releases the previous one's recall first (release_previous), so every replay
repeats the same work."""
import pytest
import torch

from paper_2609_34555_amd import workloads as W

from parity import build, say

pytestmark = pytest.mark.gpu


def _snapshot(st):
    torch.cuda.synchronize()
    assert st.status() == 0
    return [t.clone() for t in (st.out, st.lse, st.sel_idx, st.sel_cnt, st.table, st.free_head, st.stats, st.pool)]


def _same(a, b):
    return all(torch.equal(x, y) for x, y in zip(a, b))


@pytest.mark.parametrize("cid", [1, 2])
def test_layer_step_graph_replays_equal_eager(cid):
    spec, s = W.preset(cid, ctx_scale=1 / 8) if cid == 2 else W.preset(cid)
    w, st = build(spec, s)
    st.reset()
    st.decode_layer(release_previous=True)
    ref = _snapshot(st)
    assert int(ref[6][0].item()) > 0  # the step recalled blocks

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):  # one eager step on the capture stream first
        st.decode_layer(release_previous=True, stream=side)
    torch.cuda.current_stream().wait_stream(side)
    assert _same(_snapshot(st), ref)

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):
        st.decode_layer(release_previous=True, stream=side)
    for i in range(4):
        g.replay()
        assert _same(_snapshot(st), ref), f"replay {i}"
        st.decode_layer(release_previous=True)  # eager work between replays
        assert _same(_snapshot(st), ref), f"eager step after replay {i}"
    say(f"  preset {cid}: 4 replays and 4 eager steps equal to the first eager step")
