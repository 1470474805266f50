"""Host logic of the benchmark's CPU baseline: the threaded mode runs the oracle one request
at a time and must reproduce the whole-batch oracle step exactly (selection, recall
statistics, table, pool bytes, attention output)."""
from concurrent.futures import ThreadPoolExecutor

import numpy as np

import bench
from oracle import pulse_oracle as O
from paper_2609_34555_amd import workloads as W


def _step(w, ex):
    dig = O.build_digests(w.kv, w.blk_off, w.ctx_len, w.Hkv, w.bs, w.d, w.dtype_code, w.solo_kv_head)
    pool = W.initial_pool(w).view(np.uint8).reshape(w.n_slots, -1).copy()
    host = w.kv.view(np.uint8).reshape(w.total_blocks, -1)
    table = w.table0.copy()
    dt, stats, out, lse = bench._oracle_step(O, w, dig, host, pool, table, pool.view(np.uint16).reshape(w.n_slots, -1),
                                             4 if ex else 1, ex)
    return dt, stats, out, lse, table, pool


def test_threaded_oracle_step_matches_whole_batch():
    spec, seed = W.custom("ragged", [1000, 37, 4096, 517, 16], k_mid=[6, 1, 20, 9, 3], n_local=2,
                          resident_frac=0.2, heavy_per_req=3)
    w = W.generate(spec, seed)
    dt1, st1, out1, lse1, tab1, pool1 = _step(w, None)
    with ThreadPoolExecutor(4) as ex:
        dt4, st4, out4, lse4, tab4, pool4 = _step(w, ex)
    assert set(dt1) == {"score", "select", "recall", "attention"}
    assert set(dt4) == {"score+select", "recall", "attention"}
    assert st1 == st4 and st1[0] > 0
    assert np.array_equal(tab1, tab4) and np.array_equal(pool1, pool4)
    assert np.array_equal(out1, out4) and np.array_equal(lse1, lse4)


def test_host_info_fields():
    info = bench.host_info()
    assert info["nproc"] >= 1 and 1 <= info["usable_cpus"] <= info["nproc"]


def test_more_than_one_gpu_is_refused():
    """The benchmark measures one GPU; asking for more exits with a message, before any GPU work."""
    import subprocess
    import sys

    res = subprocess.run([sys.executable, bench.__file__, "--gpus", "2"], capture_output=True, text=True, timeout=120)
    assert res.returncode != 0 and "one GPU" in res.stderr and res.stdout == ""


def test_counter_traffic_only_for_unchanged_sources(tmp_path, monkeypatch):
    """Byte counters are reported for a kernel only while its sources hash as when they were
    collected; any other hash, or a kernel with no counters, gives None."""
    import hashlib
    import json

    src = tmp_path / "k.hip"
    src.write_text("kernel source\n")
    good = hashlib.sha256(src.read_bytes()).hexdigest()[:16]
    data = {"kernels": {
        "same": {"fetch_bytes": 3.0, "write_bytes": 4.0, "sources": ["k.hip"], "sources_sha256_16": good},
        "changed": {"fetch_bytes": 3.0, "write_bytes": 4.0, "sources": ["k.hip"], "sources_sha256_16": "0" * 16}}}
    (tmp_path / "profiles").mkdir()
    (tmp_path / "profiles" / "counters_cfg3.json").write_text(json.dumps(data))
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.counter_traffic("same", 3) == {"fetch": 3.0, "write": 4.0, "total": 7.0}
    assert bench.counter_traffic("same", 2) is None  # no passes taken on that preset
    assert bench.counter_traffic("changed", 3) is None
    assert bench.counter_traffic("absent", 3) is None
    src.write_text("edited\n")
    assert bench.counter_traffic("same", 3) is None


def test_default_line_is_the_largest_single_layer_preset(monkeypatch):
    """With no flags the benchmark runs preset 3 (32 requests x U[64K,128K] tokens)."""
    import sys

    monkeypatch.setattr(sys, "argv", [bench.__file__])
    args = bench.parse()
    assert args.config == 3 and args.gpus == 1 and not args.no_presets
    assert "U[65536,131072]" in bench.WORKLOADS[3]
