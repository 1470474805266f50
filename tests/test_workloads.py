"""Host-side checks of the seeded workload generator (CPU)."""
import numpy as np
import pytest

from paper_2609_34555_amd import workloads as W


def test_rounding_matches_numpy_and_is_rne():
    x = np.array([1.0, 1.00390625, 1.01171875, -2.5, 3.14159, 65504.0, 1e-8], np.float32)
    assert np.array_equal(W.round_to_dtype(x, "f16"), x.astype(np.float16).view(np.uint16))
    b = W.round_to_dtype(x, "bf16")
    # 1 + 2^-8 is a tie between 1 and 1 + 2^-7 -> even (1.0); 1 + 3*2^-8 -> 1 + 2^-6
    assert W.to_float(b[1:3], "bf16").tolist() == [1.0, 1.015625]
    assert np.all(np.abs(W.to_float(b, "bf16") - x) <= np.abs(x) * 2.0 ** -8)


def test_generation_is_deterministic_and_threads_do_not_matter():
    spec, s = W.preset(2, ctx_scale=1 / 64, batch=3)
    a = W.generate(spec, s, threads=1)
    b = W.generate(spec, s, threads=8)
    assert np.array_equal(a.kv, b.kv) and np.array_equal(a.q, b.q)
    assert np.array_equal(a.table0, b.table0) and a.solo_kv_head == b.solo_kv_head


@pytest.mark.parametrize("cid,k_mid,n_sink,n_local,bs,frac", [
    (1, 16, 1, 8, 16, 0.25), (2, 119, 1, 8, 16, 0.10), (3, 247, 1, 8, 16, 0.05), (5, 251, 1, 4, 32, 0.03)])
def test_presets_follow_the_paper_budget_split(cid, k_mid, n_sink, n_local, bs, frac):
    spec, _ = W.preset(cid)
    assert spec.block_size == bs and spec.n_sink == n_sink and spec.n_local == n_local
    assert all(k == k_mid for k in spec.k_mid) and spec.resident_frac == frac


def test_preset4_lognormal_budgets_are_clipped():
    ks = []
    for layer in range(32):
        spec, _ = W.preset(4, layer=layer)
        ks += spec.k_mid
    ks = np.array(ks)
    assert ks.min() >= 256 // 16 - 9 and ks.max() <= 8192 // 16 - 9
    assert 100 < ks.mean() < 260  # mean budget ~2.9K tokens


def test_preset5_heavy_runs_and_singletons():
    spec, _ = W.preset(5)
    for hv in spec.heavy:
        hv = np.asarray(hv)
        assert hv.size == 4 * 16 + 64 and np.all(np.diff(hv) >= 1)
        runs = np.split(hv, np.nonzero(np.diff(hv) != 1)[0] + 1)
        lens = sorted(len(r) for r in runs)
        assert lens == [1] * 64 + [16] * 4
        n = 262144 // 32
        assert hv.min() >= 1 and hv.max() < n - 4


def test_resident_set_free_list_and_kmax():
    spec, s = W.custom("x", [100, 37, 5, 64], bs=16, k_mid=3, n_sink=1, n_local=2, resident_frac=0.3,
                       heavy_per_req=2, free_order="shuffled")
    w = W.generate(spec, s)
    res_slots = set()
    for r in range(w.B):
        n = int(w.n_blocks[r])
        row = w.table0[r, :n]
        forced = set(range(min(1, n))) | set(range(max(0, n - 2), n))
        assert all(row[j] >= 0 for j in forced)  # sink and local always resident
        res_slots |= set(row[row >= 0].tolist())
        assert np.all(w.table0[r, n:] == -1)
    assert res_slots == set(range(len(res_slots)))
    assert set(w.free_slots.tolist()).isdisjoint(res_slots)
    assert len(set(w.free_slots.tolist())) == w.free_slots.size
    assert w.k_max == max(len(set(range(min(1, n))) | set(range(max(0, n - 2), n))) + min(3, max(0, n - 3))
                          for n in w.n_blocks.tolist())
    # the resident slot images are the host blocks
    pool = W.initial_pool(w)
    for i, b in enumerate(w.resident_blocks):
        assert np.array_equal(pool[i], w.kv[b])


def test_padding_tokens_are_zero():
    spec, s = W.custom("p", [21, 16, 3], Hq=4, Hkv=2, d=128, bs=16)
    w = W.generate(spec, s)
    for r in range(w.B):
        nv = int(w.ctx_len[r] - (w.n_blocks[r] - 1) * w.bs)
        last = int(w.blk_off[r + 1] - 1)
        blk = w.kv[last].reshape(2, w.Hkv, -1)
        K = blk[0].reshape(w.Hkv, w.bs, w.d)
        V = blk[1].reshape(w.Hkv, w.d, w.bs)
        assert np.all(K[:, nv:, :] == 0) and np.all(V[:, :, nv:] == 0)
        if nv == w.bs:
            assert np.any(K[:, -1, :] != 0)


def test_planted_heavy_blocks_in_middle_and_in_solo_head_only():
    spec, s = W.preset(1)
    w = W.generate(spec, s)
    hv = np.asarray(w.heavy[0])
    assert hv.size == 8 and hv.min() >= w.n_sink and hv.max() < w.n_blocks[0] - w.n_local
    K = w.kv.reshape(w.total_blocks, 2, w.Hkv, w.bs, w.d)[:, 0]
    Kf = W.to_float(K, "f16")
    norms = np.linalg.norm(Kf, axis=-1).mean(axis=-1)  # [blocks, Hkv]
    h = w.solo_kv_head
    assert norms[hv, h].min() > 2 * norms[:, h].mean() / 1.5
    others = [x for x in range(w.Hkv) if x != h]
    assert norms[hv][:, others].max() < 1.5 * np.sqrt(w.d)
