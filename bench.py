#!/usr/bin/env python3
"""Benchmark one decode layer-step of sparse-KV offloading on one MI355X.

A step = digest score + SoloHead selection (with the set difference) + slot
allocation and gather-scatter recall from pinned host DRAM + sparse GQA
decode attention, chained on one stream by pulse_decode_layer.

Default workload (synthetic, seeded; the largest single-layer configuration):
32 requests with contexts drawn uniformly from [64K, 128K] tokens (ragged block
tables, partial last blocks), block 16, 32 query / 8 KV heads, head_dim 128,
bf16, 4096-token hot budget (1 sink + 8 local + 247 middle blocks), 5% of
blocks resident, 32 planted heavy blocks per request.  The queries, digests,
block table and slot pool are in HBM and the full KV store (12 GiB) is in
pinned host DRAM when the timed region starts (the host tier is the method's
own data structure).

Prints one JSON line.  value = recall bytes per step / wall time per step.
With the default preset the line also carries a `presets` sub-record: the
other four workloads, each timed the same way (without CPU baseline or probes).
"""
import argparse
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "recall GB/s (host→HBM) + µs per layer-step select+recall+attend"
PCIE5_X16_GBPS = 64.0  # published MI355X host interface: PCIe 5.0 x16, per direction
HBM_GBPS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--config", type=int, default=3, choices=[1, 2, 3, 4, 5],
                    help="workload preset (3 = the default benchmark line)")
    ap.add_argument("--no-presets", action="store_true",
                    help="with the default preset: leave out the sub-record of the other four presets")
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-probes", action="store_true", help="skip link probes and memcpy baselines")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--irq", action="store_true",
                    help="report: interruptible layer-wise scheduling of a preset-4 offload batch against a "
                         "resident normal batch, every detection mode and both recall paths (not the default line)")
    ap.add_argument("--ioaa-profile", action="store_true",
                    help="report: overlap depth measured over a (B_o, B_n) grid and an IOAA admission on it")
    ap.add_argument("--recall-sweep", action="store_true",
                    help="report: recall bandwidth against the number of blocks per recall for the GPU gather "
                         "kernel, the paper's engine and one hipMemcpyAsync per block (not the default line)")
    ap.add_argument("--normal-batch", type=int, default=32)
    ap.add_argument("--summarize-counters", nargs="+", metavar="DIR",
                    help="no GPU work: turn rocprofv3 --pmc output directories of `bench.py --profile --config N` "
                         "(FETCH_SIZE, WRITE_SIZE, optionally TCC_EA0_RDREQ_sum / _32B_sum / TCC_BUBBLE_sum) into "
                         "profiles/counters_cfgN.json and print a markdown table")
    ap.add_argument("--profile", action="store_true",
                    help="profiler run: no CPU baseline, link probes or preset sub-record; adds device copies "
                         "of known size that calibrate the byte counters")
    return ap.parse_args()


def link_probes(torch, P, st, holder):
    """Host-link peak: a 1 GiB pinned->device hipMemcpyAsync and the streaming read
    kernel over the pinned KV store; plus a transfer-size sweep of per-unit copies."""
    res = {}
    nbytes = 1 << 30
    dev = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    host = torch.empty(nbytes, dtype=torch.uint8, pin_memory=True)
    host.fill_(1)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    best = 0.0
    for _ in range(3):
        e0.record()
        dev.copy_(host, non_blocking=True)
        e1.record()
        torch.cuda.synchronize()
        best = max(best, nbytes / (e0.elapsed_time(e1) * 1e-3) / 1e9)
    res["memcpy_1GiB_GBps"] = best
    store_bytes = (holder[0].nbytes // 16384) * 16384
    nb = min(store_bytes, nbytes)
    best = 0.0
    for _ in range(3):
        e0.record()
        P.pulse_probe_host_read(holder[0].ptr, dev, nb)
        e1.record()
        torch.cuda.synchronize()
        best = max(best, nb / (e0.elapsed_time(e1) * 1e-3) / 1e9)
    res["kernel_read_1GiB_GBps"] = best
    # per-unit hipMemcpyAsync sweep (the fragmented-transfer curve)
    import numpy as np

    sweep = {}
    for unit in (8 << 10, 16 << 10, 32 << 10, 64 << 10, 128 << 10, 256 << 10, 512 << 10, 1 << 20):
        n = min(512, nb // unit)
        src = np.random.default_rng(0).permutation(nb // unit)[:n].astype(np.int64)
        dst = np.arange(n, dtype=np.int64)
        times = []
        for rep in range(4):  # one warm-up, then the median of three
            e0.record()
            P.pulse_baseline_memcpy_units(holder[0].ptr, dev, src, dst, n, unit)
            e1.record()
            torch.cuda.synchronize()
            if rep:
                times.append(e0.elapsed_time(e1))
        sweep[f"{unit >> 10}KiB"] = n * unit / (statistics.median(times) * 1e-3) / 1e9
    res["memcpy_per_unit_GBps"] = sweep
    del dev, host
    return res


def memcpy_recall_baseline(torch, P, st, w):
    """The same recall done with one hipMemcpyAsync per missing block (the threaded
    per-block copy the paper's engine is compared with).  The plan is read back to
    the host first; that sync is outside the timed copies."""
    import numpy as np

    st.reset()
    st.select()
    torch.cuda.synchronize()
    idx, cnt = st.selection()
    src, dst = [], []
    g = 0
    for r in range(w.B):
        for j in idx[r, : cnt[r]]:
            if w.table0[r, j] < 0:
                src.append(int(w.blk_off[r] + j))
                dst.append(int(w.free_slots[g]))
                g += 1
    src = np.array(src, np.int64)
    dst = np.array(dst, np.int64)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    times = []
    for _ in range(5):
        e0.record()
        P.pulse_baseline_memcpy_units(st.host_ptr, st.pool, src, dst, len(src), w.unit_bytes)
        e1.record()
        torch.cuda.synchronize()
        times.append(e0.elapsed_time(e1))
    ms = statistics.median(times)
    return {"blocks": len(src), "ms": ms, "GBps": len(src) * w.unit_bytes / (ms * 1e-3) / 1e9}


def counter_traffic(kernel, cid):
    """HBM-side bytes per launch of `kernel` on preset `cid` from the committed rocprofv3
    FETCH_SIZE/WRITE_SIZE passes (scaled by the copy-kernel calibration); None if there are
    none for this preset or the kernel's sources changed since."""
    import hashlib

    path = os.path.join(ROOT, "profiles", f"counters_cfg{cid}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        k = json.load(f)["kernels"].get(kernel)
    if not k:
        return None
    h = hashlib.sha256()
    for src in k["sources"]:
        with open(os.path.join(ROOT, src), "rb") as f:
            h.update(f.read())
    if h.hexdigest()[:16] != k["sources_sha256_16"]:
        return None
    if "fetch_bytes" not in k:
        return None
    return {"fetch": k["fetch_bytes"], "write": k["write_bytes"], "total": k["fetch_bytes"] + k["write_bytes"]}


KERNEL_SOURCES = {
    "recall_copy_kernel": ["paper_2609_34555_amd/csrc/recall.hip", "paper_2609_34555_amd/csrc/pulse_internal.h"],
    "attn_splitk_kernel": ["paper_2609_34555_amd/csrc/attention.hip", "paper_2609_34555_amd/csrc/pulse_internal.h"],
    "attn_combine_kernel": ["paper_2609_34555_amd/csrc/attention.hip", "paper_2609_34555_amd/csrc/pulse_internal.h"],
    "score_kernel": ["paper_2609_34555_amd/csrc/digest.hip", "paper_2609_34555_amd/csrc/pulse_internal.h"],
    "select_kernel": ["paper_2609_34555_amd/csrc/select.hip", "paper_2609_34555_amd/csrc/pulse_internal.h"],
}


def _sources_hash(files):
    import hashlib

    h = hashlib.sha256()
    for src in files:
        with open(os.path.join(ROOT, src), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def summarize_counters(dirs, cid):
    """Per-dispatch FETCH_SIZE / WRITE_SIZE (KiB) of a profiler run of this file, scaled to bytes
    by the reading of the calibration copies (probe_copy_kernel over CALIBRATION_COPIES bytes,
    device to device, one dispatch per size in order).  With a third directory holding
    TCC_EA0_RDREQ_sum / TCC_EA0_RDREQ_32B_sum / TCC_BUBBLE_sum, the read requests are reported
    too (the calibration shows their size).  Writes profiles/counters_cfg{cid}.json."""
    import collections
    import csv

    vals = collections.defaultdict(lambda: collections.defaultdict(list))
    for d in dirs:
        with open(os.path.join(d, "bench_counter_collection.csv")) as f:
            for r in csv.DictReader(f):
                name = r["Kernel_Name"].split("(")[0].replace("void ", "").strip()
                vals[name][r["Counter_Name"]].append(float(r["Counter_Value"]))
    cal = vals["pulse::probe_copy_kernel"]
    if len(cal["FETCH_SIZE"]) != len(CALIBRATION_COPIES) or len(cal["WRITE_SIZE"]) != len(CALIBRATION_COPIES):
        raise RuntimeError("expected one calibration copy dispatch per size")
    fetch_f = [b / (k * 1024) for b, k in zip(CALIBRATION_COPIES, cal["FETCH_SIZE"])]
    write_f = [b / (k * 1024) for b, k in zip(CALIBRATION_COPIES, cal["WRITE_SIZE"])]
    fs, ws = statistics.mean(fetch_f), statistics.mean(write_f)
    calib = {"copy_bytes": list(CALIBRATION_COPIES), "fetch_KiB": cal["FETCH_SIZE"], "write_KiB": cal["WRITE_SIZE"],
             "fetch_scale_per_size": fetch_f, "write_scale_per_size": write_f, "fetch_scale": fs, "write_scale": ws}
    if "TCC_EA0_RDREQ_sum" in cal:
        calib["rdreq"] = cal["TCC_EA0_RDREQ_sum"]
        calib["rdreq_32B"] = cal.get("TCC_EA0_RDREQ_32B_sum")
        calib["bubble"] = cal.get("TCC_BUBBLE_sum")
        calib["bytes_per_read_request"] = [b / n for b, n in zip(CALIBRATION_COPIES, cal["TCC_EA0_RDREQ_sum"])]
    out = {"preset": cid, "workload": WORKLOADS[cid], "calibration": calib, "kernels": {}}
    rows = []
    for name in sorted(vals):
        if not name.startswith("pulse::") or "probe" in name:
            continue
        v = vals[name]
        fa, wa = statistics.mean(v["FETCH_SIZE"]), statistics.mean(v.get("WRITE_SIZE", [0.0]))
        rec = {"dispatches": len(v["FETCH_SIZE"]), "fetch_KiB": fa, "write_KiB": wa,
               "fetch_bytes": fa * 1024 * fs, "write_bytes": wa * 1024 * ws}
        if "TCC_EA0_RDREQ_sum" in v:
            rec["read_requests"] = statistics.mean(v["TCC_EA0_RDREQ_sum"])
            rec["read_requests_32B"] = statistics.mean(v["TCC_EA0_RDREQ_32B_sum"])
            rec["bubble"] = statistics.mean(v["TCC_BUBBLE_sum"])
        short = name.split("::")[1].split("<")[0]
        if short in KERNEL_SOURCES:
            rec["sources"] = KERNEL_SOURCES[short]
            rec["sources_sha256_16"] = _sources_hash(KERNEL_SOURCES[short])
            out["kernels"][short] = rec
        rows.append((name, rec))
    path = os.path.join(ROOT, "profiles", f"counters_cfg{cid}.json")
    with open(path, "w") as f:
        json.dump(out, f, indent=1)
    print(f"calibration: FETCH scale {fs:.4f} ({', '.join(f'{x:.4f}' for x in fetch_f)}), "
          f"WRITE scale {ws:.4f} ({', '.join(f'{x:.4f}' for x in write_f)})")
    if "bytes_per_read_request" in calib:
        print("bytes per read request of the calibration copies: "
              + ", ".join(f"{x:.2f}" for x in calib["bytes_per_read_request"]) + f"; TCC_BUBBLE {calib['bubble']}")
    print("| Kernel | Dispatches | FETCH_SIZE (KiB, avg) | WRITE_SIZE (KiB, avg) | Fetch bytes (scaled) | "
          "Write bytes (scaled) | Read requests (avg) |")
    print("|---|---|---|---|---|---|---|")
    for name, r in rows:
        rq = f"{r['read_requests']:,.0f}" if "read_requests" in r else "-"
        print(f"| `{name}` | {r['dispatches']} | {r['fetch_KiB']:.1f} | {r['write_KiB']:.1f} | {r['fetch_bytes']:,.0f} | "
              f"{r['write_bytes']:,.0f} | {rq} |")
    return out


def engine_recall_baseline(torch, P, st, w, reps=5):
    """The paper's recall engine on the same selection: GPU plan + publish into a pinned
    mailbox, CPU poller and 8 gather threads into pinned staging, one DMA per 16 MiB batch,
    GPU scatter.  Wall time from submit to the host seeing completion."""
    eng = P.GatherScatterEngine(st.shape, n_workers=8, max_blocks_per_call=w.B * st.k_max,
                                staging_blocks=max(1, (16 << 20) // w.unit_bytes))
    times, timing = [], None
    try:
        for _ in range(reps + 1):
            st.reset()
            st.select()
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            st.recall_gs(eng)
            times.append((time.perf_counter() - t0) * 1e3)
            timing = eng.last_timing()
    finally:
        eng.destroy()
    torch.cuda.synchronize()
    ms = statistics.median(times[1:])
    nbytes = st.recall_stats()[2]
    return {"ms": ms, "GBps": nbytes / (ms * 1e-3) / 1e9, "last_call": timing, "workers": 8,
            "staging_MiB": 16}


def host_info():
    """CPU model, logical CPUs usable by this process and installed memory of this host."""
    info = {"nproc": os.cpu_count(), "usable_cpus": len(os.sched_getaffinity(0))}
    try:
        with open("/proc/cpuinfo") as f:
            info["model"] = next((ln.split(":", 1)[1].strip() for ln in f if ln.startswith("model name")), None)
        with open("/proc/meminfo") as f:
            kb = next(int(ln.split()[1]) for ln in f if ln.startswith("MemTotal"))
        info["mem_GiB"] = round(kb / 2**20, 1)
    except (OSError, StopIteration, ValueError):
        pass
    return info


def _oracle_step(O, w, dig, host, pool, table, pool_u16, threads, pool_exec):
    """One layer-step through the oracle, returning its stage times (s), recall stats and
    attention output.  With a thread pool the per-request stages (score, select,
    attention) run one request per task -- the oracle's C calls release the GIL -- and
    the recall, whose slot allocation follows the global request order, runs whole."""
    import numpy as np

    t = [time.perf_counter()]
    if pool_exec is None:
        sc = O.score(w.q, dig, w.blk_off, w.Hq, w.Hkv, w.d, w.dtype_code, w.solo_kv_head)
        t.append(time.perf_counter())
        rc, idx, cnt = O.select(sc, w.blk_off, w.k_mid, w.n_sink, w.n_local, w.k_max)
    else:
        offs = w.blk_off.tolist()

        def score_select(r):
            lo, hi = offs[r], offs[r + 1]
            one = np.array([0, hi - lo], np.int64)
            s_r = O.score(w.q[r:r + 1], dig[lo:hi], one, w.Hq, w.Hkv, w.d, w.dtype_code, w.solo_kv_head)
            return O.select(s_r, one, w.k_mid[r:r + 1], w.n_sink, w.n_local, w.k_max)

        parts = list(pool_exec.map(score_select, range(w.B)))
        rc = max(p[0] for p in parts)
        idx = np.concatenate([p[1] for p in parts])
        cnt = np.concatenate([p[2] for p in parts])
    t.append(time.perf_counter())
    rc2, fh, stats = O.recall(host, w.blk_off, idx, cnt, table, w.free_slots, 0, pool, w.unit_bytes)
    t.append(time.perf_counter())
    if pool_exec is None:
        out, lse = O.attention(w.q, pool_u16, table, idx, cnt, w.blk_off, w.ctx_len, w.Hq, w.Hkv, w.bs, w.d,
                               w.dtype_code, w.sm_scale)
    else:
        def attend(r):
            one = np.array([0, offs[r + 1] - offs[r]], np.int64)
            return O.attention(w.q[r:r + 1], pool_u16, table[r:r + 1], idx[r:r + 1], cnt[r:r + 1], one,
                               w.ctx_len[r:r + 1], w.Hq, w.Hkv, w.bs, w.d, w.dtype_code, w.sm_scale)

        res = list(pool_exec.map(attend, range(w.B)))
        out = np.concatenate([o for o, _ in res])
        lse = np.concatenate([l for _, l in res])
    t.append(time.perf_counter())
    if rc or rc2:
        raise RuntimeError(f"oracle status {rc} / {rc2}")
    dt = [b - a for a, b in zip(t, t[1:])]
    names = ["score", "select", "recall", "attention"] if pool_exec is None else \
        ["score+select", "recall", "attention"]  # one task per request covers both
    return dict(zip(names, dt)), stats, out, lse


def cpu_baseline(w, seconds, sample_note="whole layer-steps of the same workload"):
    """The CPU oracle timed on this host on whole layer-steps of the same workload (digests
    are per-block state, built once outside the timing): single thread, then -- over
    requests, on up to 16 threads -- the same oracle calls one request at a time.  Both
    modes' outputs are checked to be identical."""
    from concurrent.futures import ThreadPoolExecutor

    import numpy as np

    from oracle import pulse_oracle as O
    from paper_2609_34555_amd import workloads as W

    dig = O.build_digests(w.kv, w.blk_off, w.ctx_len, w.Hkv, w.bs, w.d, w.dtype_code, w.solo_kv_head)
    pool0 = W.initial_pool(w).view(np.uint8).reshape(w.n_slots, -1)
    host = w.kv.view(np.uint8).reshape(w.total_blocks, -1)

    def run(threads, budget):
        ex = ThreadPoolExecutor(threads) if threads > 1 else None
        stage = {}
        steps, nbytes, first = 0, 0, None
        try:
            while sum(stage.values()) < budget or steps < 2:
                table = w.table0.copy()
                pool = pool0.copy()
                pool_u16 = pool.view(np.uint16).reshape(w.n_slots, -1)
                dt, stats, out, lse = _oracle_step(O, w, dig, host, pool, table, pool_u16, threads, ex)
                for k, v in dt.items():
                    stage[k] = stage.get(k, 0.0) + v
                steps += 1
                nbytes = stats[2]
                if first is None:
                    first = (out, lse)
        finally:
            if ex is not None:
                ex.shutdown()
        per_step = sum(stage.values()) / steps
        return {"value": nbytes / per_step / 1e9, "unit": "GB/s", "cores": threads, "steps": steps,
                "us_per_layer_step": per_step * 1e6,
                "stage_us": {k: v / steps * 1e6 for k, v in stage.items()}}, first

    single, ref = run(1, seconds)
    line = {"kind": "oracle", **single,
            "sample": f"{single['steps']} x {sample_note} ({w.B} requests), single thread",
            "host": host_info()}
    threads = min(16, line["host"]["usable_cpus"], w.B)
    if threads > 1:
        par, got = run(threads, seconds / 2)
        if not (np.array_equal(got[0], ref[0]) and np.array_equal(got[1], ref[1])):
            raise RuntimeError("threaded oracle run differs from the single-thread run")
        par["sample"] = (f"{par['steps']} x the same layer-steps, one request per task on {threads} threads "
                         "(score + select and attention per request; recall whole)")
        line["threaded"] = par
    return line


WORKLOADS = {
    1: "1 request x 4096 tokens, block 16, 32 q / 8 KV heads, head_dim 128, fp16, middle budget 16 blocks "
       "(+1 sink +8 local), 25% resident, 8 planted heavy blocks",
    2: "8 requests x 32768 tokens, block 16, 32 q / 8 KV heads, head_dim 128, bf16, 2048-token budget "
       "(1 sink + 8 local + 119 middle blocks), 10% resident, 32 planted heavy blocks/request",
    3: "32 requests x U[65536,131072] tokens (ragged), block 16, 32 q / 8 KV heads, head_dim 128, bf16, "
       "4096-token budget, 5% resident, 32 planted heavy blocks/request",
    4: "32 layers x (16 requests x 65536 tokens), block 16, 32 q / 8 KV heads, head_dim 128, bf16, "
       "per-(layer, request) budgets lognormal sigma 1 around 2048 tokens clipped to [256, 8192], 10% resident, "
       "layers on 4 shared host stores; recall of layer l+1 overlaps attention of layer l on two streams",
    5: "4 requests x 262144 tokens, block 32, 64 q / 8 KV heads, head_dim 128, bf16, 8192-token budget, "
       "3% resident, heavy blocks in 4 runs of 16 + 64 singletons per request",
}
DTYPES = {1: "f16", 2: "bf16", 3: "bf16", 4: "bf16", 5: "bf16"}


def base_line(cid, K, warmup):
    return {"metric": METRIC, "unit": "GB/s", "n_gpus": 1, "steps": K, "warmup": warmup,
            "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": DTYPES[cid],
            "data": "synthetic (seeded N(0,1) K/V/q, planted heavy blocks; no model weights or datasets)"}


def _event_pass(torch, P, st, K, keep, every=1, split=False):
    """K steps; every `every`-th layer-step records the stage events in `keep` (indices into
    the five of pulse_layer_args.events; the others are left out), the rest none; with
    `split`, event 5 is the split-K attention kernel's end (pulse_layer_args.attn_split_event).  Returns the EventSets of the recording steps and
    the host wall time of the K steps."""
    evs = []
    args = []
    for k in range(K):
        a = st.layer_args(release_previous=True)
        if k % every == 0:
            evs.append(P.EventSet(6))
            a.events = evs[-1].masked_ptr(keep)
            if split:
                a.attn_split_event = evs[-1].arr[5]
        args.append(a)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for a in args:
        P.pulse_decode_layer(a)
    torch.cuda.synchronize()
    return evs, time.perf_counter() - t0


def timed_steps(torch, P, st, K, warmup):
    """W untimed steps, then exactly K timed steps, bracketed by device synchronisation.  A
    step is pulse_decode_layer with release_previous set: it first undoes the previous step's
    recall (inside the scoring kernel; the hot set stays fixed-size), so every step recalls
    the same blocks.  Inside the timed region only the recall copy kernel's start and end
    events (the roofline kernel) are recorded, on every 4th step: the library attaches them to
    the kernel's launch, but recording events still costs the stream some time between launches.
    Two untimed passes of K steps follow: the scoring kernel's start and the attention's end
    only (the chain's duration), then all five plus, when a merge kernel follows the split-K
    attention kernel, that kernel's end (the per-stage split; with one workgroup per (request,
    KV head) the split-K kernel is the whole attention and carries the attention's end itself)."""
    step = st.layer_args(release_previous=True)
    st.reset()  # once, untimed: nothing recalled yet
    for _ in range(warmup):
        P.pulse_decode_layer(step)
    evs, wall = _event_pass(torch, P, st, K, (2, 3), every=4)  # the timed region
    recall = [e.elapsed_ms(2, 3) for e in evs]
    chain_evs, _ = _event_pass(torch, P, st, K, (0, 4))
    layer = [e.elapsed_ms(0, 4) for e in chain_evs]
    merge = P.pulse_attention_workgroups(st.shape, st.w.B, st.k_max) > 1
    stage_evs, _ = _event_pass(torch, P, st, K, (0, 1, 2, 3, 4), split=merge)
    P.pulse_decode_layer(step)  # untimed: leaves this step's recall statistics and tables in place
    torch.cuda.synchronize()
    stage = {"score": [], "select": [], "recall": [], "attention": [], "attention_kernel": [],
             "attention_combine": [], "layer": []}
    for e in stage_evs:
        stage["score"].append(e.elapsed_ms(0, 1))
        stage["select"].append(e.elapsed_ms(1, 2))
        stage["recall"].append(e.elapsed_ms(2, 3))
        stage["attention"].append(e.elapsed_ms(3, 4))
        if merge:
            stage["attention_kernel"].append(e.elapsed_ms(3, 5))
            stage["attention_combine"].append(e.elapsed_ms(5, 4))
        else:  # no merge kernel: the split-K kernel is the attention
            stage["attention_kernel"].append(e.elapsed_ms(3, 4))
            stage["attention_combine"].append(0.0)
        stage["layer"].append(e.elapsed_ms(0, 4))
    for e in evs + chain_evs + stage_evs:
        e.destroy()
    timed = {"recall": statistics.mean(recall), "layer": statistics.mean(layer),
             "layer_median": statistics.median(layer), "attention_merge": merge}
    return (wall, timed, {k: statistics.mean(v) for k, v in stage.items()},
            {k: statistics.median(v) for k, v in stage.items()})


def hbm_probe(torch, P, nbytes, reps=10):
    """Read bandwidth this GPU sustains over `nbytes` of device memory: the streaming read
    probe, each launch carrying its own start and stop events (as the layer-step's stage
    events are carried by its kernels), mean over `reps` launches after 3 warm-ups.  A spin
    kernel queued first keeps the GPU busy while the host enqueues the launches."""
    nbytes = max(16, (int(nbytes) // 16) * 16)
    src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    sink = torch.zeros(P.pulse_probe_hbm_sink_bytes() // 4, dtype=torch.int32, device="cuda")
    ev = P.EventSet(2 * reps)
    try:
        for _ in range(3):
            P.pulse_probe_hbm_read(src, nbytes, sink)
        torch.cuda.synchronize()
        torch.cuda._sleep(20_000_000)  # ~10 ms of GPU time ahead of the enqueues below
        for i in range(reps):
            P.pulse_probe_hbm_read(src, nbytes, sink, start_event=ev.arr[2 * i], stop_event=ev.arr[2 * i + 1])
        torch.cuda.synchronize()
        ms = statistics.mean(ev.elapsed_ms(2 * i, 2 * i + 1) for i in range(reps))
    finally:
        ev.destroy()
    del src, sink
    return nbytes / (ms * 1e-3) / 1e9


def attention_warm_cold(torch, st, attn_bytes, reps=10):
    """The attention call (split-K kernel + combine) alone, warm and cold.  In the chained
    step the recall has just written part of the selected blocks, and a working set under
    256 MB can stay in the Infinity Cache: warm launches repeat the call on the same
    selection; cold ones first read 1 GiB of other data, which evicts the working set
    without leaving dirty lines to write back.  HIP events bracket each launch on the
    current stream; mean over `reps` launches."""
    scratch = torch.ones(1 << 28, dtype=torch.float32, device="cuda")  # 1 GiB
    res = {}
    for mode in ("warm", "cold"):
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
        sink = []
        st.attention()
        torch.cuda.synchronize()
        torch.cuda._sleep(20_000_000)  # keeps the GPU busy while the launches below are enqueued
        for e0, e1 in evs:
            if mode == "cold":
                sink.append(scratch.sum())
            else:
                st.attention()
            e0.record()
            st.attention()
            e1.record()
        torch.cuda.synchronize()
        ms = statistics.mean(e0.elapsed_time(e1) for e0, e1 in evs)
        res[mode] = {"us": ms * 1e3, "GBps": attn_bytes / (ms * 1e-3) / 1e9,
                     "frac": attn_bytes / (ms * 1e-3) / 1e9 / HBM_GBPS}
    del scratch
    if st.status() != 0:
        raise RuntimeError(f"device status {st.status()} after the isolated attention runs")
    return res


def selection_variants(torch, P, st, w, reps=10):
    """Scoring + selection by the three strategies of Sec. 4.4.1 on this workload, each call
    alone: SoloHead (one KV head's digests), Average (every KV head scores, the scores are
    averaged, one selection) and headwise (every KV head selects for itself, with its transfer
    and run counts against the block table).  The digests of every head are built first
    (untimed); outputs go to buffers of their own, so the step's state is untouched.  Events
    recorded around each launch on the current stream (each interval carries a marker's cost,
    the same for all three); mean over `reps` calls after two warm-ups."""
    hd = st.all_head_digests()
    dev = st.device
    H, B, k, nt = w.Hkv, w.B, st.k_max, w.total_blocks
    sel = torch.full((H, B, k), -1, dtype=torch.int32, device=dev)
    cnt = torch.zeros((H, B), dtype=torch.int32, device=dev)
    miss, runs = torch.zeros_like(cnt), torch.zeros_like(cnt)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    nb = {"solohead": P.pulse_workspace_bytes(st.shape, B, k, nt),
          "average": P.pulse_average_workspace_bytes(st.shape, B, k, nt),
          "headwise": P.pulse_headwise_workspace_bytes(st.shape, B, k, nt)}
    ws = torch.zeros(max(max(nb.values()), 1), dtype=torch.uint8, device=dev)
    calls = {
        "solohead": lambda: P.pulse_select_solohead(st.shape, st.q, st.digests, st.blk_off, B, nt, w.solo_kv_head,
                                                    st.k_mid, w.n_sink, w.n_local, k, sel[0], cnt[0], None, status,
                                                    ws, nb["solohead"]),
        "average": lambda: P.pulse_select_average(st.shape, st.q, hd, st.blk_off, B, nt, st.k_mid, w.n_sink,
                                                  w.n_local, k, sel[0], cnt[0], None, status, ws, nb["average"]),
        "headwise": lambda: P.pulse_select_headwise(st.shape, st.q, hd, st.blk_off, B, nt, st.k_mid, w.n_sink,
                                                    w.n_local, k, st.table, w.max_blocks, w.n_slots, sel, cnt, miss,
                                                    runs, status, ws, nb["headwise"]),
    }
    out = {}
    for name, fn in calls.items():
        for _ in range(2):
            fn()
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
        torch.cuda.synchronize()
        torch.cuda._sleep(20_000_000)  # keeps the GPU busy while the launches below are enqueued
        for e0, e1 in evs:
            e0.record()
            fn()
            e1.record()
        torch.cuda.synchronize()
        out[name + "_us"] = statistics.mean(e0.elapsed_time(e1) for e0, e1 in evs) * 1e3
    if int(status.item()) != 0:
        raise RuntimeError(f"device status {int(status.item())} in the selection variants")
    per_head = int(sum(max(0, n - w.n_sink - w.n_local) for n in w.n_blocks.tolist())) * 2 * w.d * 2
    out["digest_bytes_read"] = {"solohead": per_head, "average": per_head * H, "headwise": per_head * H}
    out["digest_bytes_resident"] = {"solohead": nt * 2 * w.d * 2, "every_head": nt * 2 * w.d * 2 * H}
    del hd, ws
    st.head_digests = None
    torch.cuda.empty_cache()
    return out


def rooflines(w, st, timed, mean, rbytes, peak_measured):
    """The recall's rate from the timed region's events; attention and score from the
    all-stage pass."""
    recall_GBps = rbytes / (timed["recall"] * 1e-3) / 1e9
    sel = st.sel_cnt.cpu().numpy()
    attn_bytes = int(sel.sum()) * w.unit_bytes + w.q.nbytes + w.B * w.Hq * w.d * 4
    digest_bytes = int(sum(max(0, n - w.n_sink - w.n_local) for n in w.n_blocks.tolist())) * 2 * w.d * 2
    attn = attn_bytes / (mean["attention_kernel"] * 1e-3) / 1e9
    attn_call = attn_bytes / (mean["attention"] * 1e-3) / 1e9
    score = digest_bytes / (mean["score"] * 1e-3) / 1e9
    roof = {"bound": "host_link", "kernel": "recall_copy_kernel", "achieved": recall_GBps, "peak": PCIE5_X16_GBPS,
            "unit": "GB/s", "frac": recall_GBps / PCIE5_X16_GBPS, "peak_measured": peak_measured,
            "frac_of_measured": (recall_GBps / peak_measured) if peak_measured else None,
            "bytes_per_launch": rbytes}
    attn_roof = {"bound": "hbm", "kernel": "attn_splitk_kernel", "achieved": attn, "peak": HBM_GBPS, "unit": "GB/s",
                 "frac": attn / HBM_GBPS, "bytes_per_launch": attn_bytes,
                 "with_combine": {"achieved": attn_call, "frac": attn_call / HBM_GBPS,
                                  "us": mean["attention"] * 1e3, "combine_us": mean["attention_combine"] * 1e3,
                                  "combine_kernel": timed["attention_merge"]}}
    score_roof = {"bound": "hbm", "kernel": "score_kernel", "achieved": score, "peak": HBM_GBPS, "unit": "GB/s",
                  "frac": score / HBM_GBPS, "bytes_per_launch": digest_bytes}
    return roof, attn_roof, score_roof


CALIBRATION_COPIES = (64 << 20, 256 << 20, 1 << 30)  # device-to-device copies that scale the byte counters


def calibration_copies(torch, P):
    """Profiler runs only: device-to-device copies of known size through the library's streaming
    copy kernel (probe_copy_kernel: the recall's 16-byte load / store pattern), one dispatch per
    size in CALIBRATION_COPIES order, then one runtime copy (the hipMemcpy blit kernel) of 256 MiB.
    FETCH_SIZE / WRITE_SIZE of these dispatches give the factors that turn the counters into bytes."""
    n = max(CALIBRATION_COPIES)
    a = torch.empty(n, dtype=torch.uint8, device="cuda")
    b = torch.empty_like(a)
    a.fill_(3)
    torch.cuda.synchronize()
    for nbytes in CALIBRATION_COPIES:
        P.pulse_probe_host_read(a, b, nbytes)
        torch.cuda.synchronize()
    b[: 256 << 20].copy_(a[: 256 << 20])
    torch.cuda.synchronize()
    if not torch.equal(a[: 256 << 20], b[: 256 << 20]):
        raise RuntimeError("calibration copy mismatch")
    del a, b
    return {"probe_copy_kernel_bytes": list(CALIBRATION_COPIES), "runtime_copy_bytes": 256 << 20}


def attach_traffic(cid, roof, attn_roof, score_roof):
    """`traffic` of each roofline from the committed counter passes of this preset (null when
    there are none, or the kernel's sources changed since they were taken)."""
    rec = counter_traffic("recall_copy_kernel", cid)
    roof["traffic"] = (rec or {}).get("total")
    roof["traffic_split"] = rec
    if rec is not None:
        roof["traffic_note"] = ("fetch = the blocks read from pinned host memory over the link, write = the "
                                "same bytes stored to the HBM slot pool: each is bytes_per_launch, no re-reads")
    attn = counter_traffic("attn_splitk_kernel", cid)
    attn_roof["traffic"] = (attn or {}).get("total")
    attn_roof["traffic_split"] = attn
    score = counter_traffic("score_kernel", cid)
    score_roof["traffic"] = (score or {}).get("total")
    score_roof["traffic_split"] = score


def bench_layer(cid, args, torch, P, H, W, compact=False):
    """One workload preset: K timed layer-steps plus untimed event passes.  compact: no
    profiler calibration, link / HBM probes or CPU baseline (the presets sub-record)."""
    spec, seed = W.preset(cid)
    holder = []
    t0 = time.time()
    w = W.generate(spec, seed, kv_alloc=H.pinned_allocator(holder))
    gen_s = time.time() - t0
    st = H.LayerState(w, holder[0].ptr)
    torch.cuda.synchronize()
    K = args.steps
    wall, timed, mean, median = timed_steps(torch, P, st, K, args.warmup)
    status = st.status()
    if status != 0:
        raise RuntimeError(f"device status {P.status_string(status)}")
    n_missing, n_runs, rbytes = st.recall_stats()
    ms_per_step = wall * 1e3 / K

    extras = {}
    probes = not (args.no_probes or args.profile or compact)
    if args.profile and not compact:
        extras["calibration"] = calibration_copies(torch, P)
    if probes:
        extras["link"] = link_probes(torch, P, st, holder)
        extras["per_block_memcpy_recall"] = memcpy_recall_baseline(torch, P, st, w)
        extras["paper_engine_recall"] = engine_recall_baseline(torch, P, st, w)
    peak_measured = max([extras["link"]["memcpy_1GiB_GBps"], extras["link"]["kernel_read_1GiB_GBps"]]
                        if "link" in extras else [0.0]) or None
    roof, attn_roof, score_roof = rooflines(w, st, timed, mean, rbytes, peak_measured)
    if probes:  # measured HBM read ceilings at the kernels' own sizes, and at 1 GiB
        for r in (attn_roof, score_roof):
            r["peak_measured"] = hbm_probe(torch, P, r["bytes_per_launch"])
            r["frac_of_measured"] = r["achieved"] / r["peak_measured"]
        extras["hbm_read_1GiB_GBps"] = hbm_probe(torch, P, 1 << 30)
        attn_roof["isolated"] = attention_warm_cold(torch, st, attn_roof["bytes_per_launch"])
        extras["selection_variants"] = selection_variants(torch, P, st, w)
    attach_traffic(cid, roof, attn_roof, score_roof)
    line = base_line(cid, K, args.warmup)
    line.update({
        "value": rbytes / (ms_per_step * 1e-3) / 1e9,
        "us_per_layer_step": timed["layer"] * 1e3,
        "us_per_layer_step_median": timed["layer_median"] * 1e3,
        "ms_per_step": ms_per_step,
        "config": {"workload": WORKLOADS[cid], "preset": cid, "batch": w.B, "total_blocks": w.total_blocks,
                   "block_size": w.bs, "k_max": w.k_max, "parallelism": "single GPU"},
        "recall": {"bytes_per_step": rbytes, "blocks": n_missing, "runs": n_runs,
                   "kernel_GBps": roof["achieved"]},
        "stage_us": {k: v * 1e3 for k, v in mean.items()},
        "stage_us_median": {k: v * 1e3 for k, v in median.items()},
        "roofline": roof,
        "roofline_hbm_attention": attn_roof,
        "roofline_hbm_score": score_roof,
        "extras": extras,
        "setup_s": {"generate": gen_s},
    })
    if not (args.no_cpu_baseline or args.profile or compact):
        line["cpu_baseline"] = cpu_baseline(w, args.cpu_seconds)
    del st, w
    for store in holder:
        store.free()
    torch.cuda.empty_cache()
    return line


def presets_record(args, torch, P, H, W):
    """The other four presets, each timed as the default line (K steps after W warm-ups) but
    without probes or CPU baseline: a compact record per preset."""
    keep = ("value", "unit", "us_per_layer_step", "ms_per_step", "dtype", "config", "recall", "stage_us",
            "schedules_ms", "headwise_vs_solohead", "attention_ms_per_step")
    out = {}
    for cid in (1, 2, 4, 5):
        t = time.time()
        if cid == 4:
            line = bench_multilayer(args, torch, P, H, W, compact=True)
        else:
            line = bench_layer(cid, args, torch, P, H, W, compact=True)
        rec = {k: line[k] for k in keep if k in line}
        rec["roofline"] = {k: line["roofline"].get(k) for k in ("bound", "achieved", "peak", "frac", "traffic")}
        for name in ("roofline_hbm_attention", "roofline_hbm_score"):
            if name in line:
                r = line[name]
                rec[name] = {"achieved": r["achieved"], "peak": r["peak"], "frac": r["frac"],
                             "traffic": r.get("traffic")}
                if "with_combine" in r:
                    rec[name]["with_combine_frac"] = r["with_combine"]["frac"]
        rec["wall_s"] = time.time() - t
        out[str(cid)] = rec
        print(f"[bench] preset {cid}: {rec['value']:.2f} GB/s, {rec['us_per_layer_step']:.1f} us per layer-step",
              file=sys.stderr, flush=True)
    return out


def bench_multilayer(args, torch, P, H, W, compact=False):
    """Preset 4: a 32-layer decode step.  Timed: the two-stream schedule (recall of
    layer l+1 overlapping attention of layer l); also reported: the same step chained on
    one stream, and headwise vs SoloHead recall transfers."""
    t0 = time.time()
    ml = H.MultiLayerStep(n_layers=32, n_stores=4)
    gen_s = time.time() - t0
    torch.cuda.synchronize()
    K = args.steps

    def run(fn, ev_steps=None):
        # every step ends with (or starts by) releasing each layer's recall, so every step
        # recalls the same blocks; the tables are restored once, untimed
        ml.reset()
        for _ in range(args.warmup):
            fn(None)
        torch.cuda.synchronize()
        t = time.perf_counter()
        for k in range(K):
            fn(ev_steps[k] if ev_steps else None)
        torch.cuda.synchronize()
        return (time.perf_counter() - t) / K

    # timing events around the recall copy of every 8th layer inside the timed region (each
    # record costs a few microseconds on the I/O stream, so not every layer carries them)
    sampled = list(range(0, len(ml.layers), 8))
    rec_evs = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) if i in sampled
                else None for i in range(len(ml.layers))] for _ in range(K)]
    t_overlap = run(lambda ev: ml.run_overlapped(recall_events=ev, release=True), rec_evs)
    sampled_ms = statistics.mean(sum(step[i][0].elapsed_time(step[i][1]) for i in sampled) for step in rec_evs)
    t_chain = run(lambda ev: ml.run_chained(release_previous=True))
    for st in ml.layers:
        if st.status() != 0:
            raise RuntimeError(f"device status {P.status_string(st.status())}")
    per_layer = [st.recall_stats() for st in ml.layers]
    rbytes = sum(x[2] for x in per_layer)
    blocks = sum(x[0] for x in per_layer)
    runs = sum(x[1] for x in per_layer)
    # attention time of every layer inside one chained step (untimed)
    evs = [P.EventSet(5) for _ in ml.layers]
    ml.reset()
    for st, e in zip(ml.layers, evs):
        a = st.layer_args()
        a.events = e.masked_ptr((3, 4))
        P.pulse_decode_layer(a)
    torch.cuda.synchronize()
    attn_ms = sum(e.elapsed_ms(3, 4) for e in evs)
    for e in evs:
        e.destroy()
    # headwise vs SoloHead transfers, per layer against the same tables
    hw_units = hw_runs = 0
    for st in ml.layers:
        st.reset()
        _, _, miss, hruns = st.headwise()
        hw_units += int(miss.sum().item())
        hw_runs += int(hruns.sum().item())
        st.head_digests = None
    w0 = ml.layers[0].w
    U = w0.unit_bytes
    extras = {}
    if args.profile and not compact:
        extras["calibration"] = calibration_copies(torch, P)
    line = base_line(4, K, args.warmup)
    sampled_bytes = sum(per_layer[i][2] for i in sampled)
    recall_GBps = sampled_bytes / (sampled_ms * 1e-3) / 1e9
    line.update({
        "value": rbytes / t_overlap / 1e9,
        "us_per_layer_step": t_overlap * 1e6 / len(ml.layers),
        "ms_per_step": t_overlap * 1e3,
        "config": {"workload": WORKLOADS[4], "preset": 4, "layers": len(ml.layers), "batch": w0.B,
                   "block_size": w0.bs, "parallelism": "single GPU, two streams"},
        "recall": {"bytes_per_step": rbytes, "blocks": blocks, "runs": runs, "kernel_GBps": recall_GBps},
        "schedules_ms": {"two_stream": t_overlap * 1e3, "one_stream_chained": t_chain * 1e3},
        "headwise_vs_solohead": {
            "solohead": {"transfers": blocks, "unit_bytes": U, "runs": runs, "bytes": blocks * U},
            "headwise": {"transfers": hw_units, "unit_bytes": U // w0.Hkv, "runs": hw_runs,
                         "bytes": hw_units * U // w0.Hkv}},
        "roofline": {"bound": "host_link", "kernel": "recall_copy_kernel", "achieved": recall_GBps,
                     "peak": PCIE5_X16_GBPS, "unit": "GB/s", "frac": recall_GBps / PCIE5_X16_GBPS,
                     "bytes_per_launch": rbytes / len(ml.layers), "traffic": None,
                     "timed_layers": sampled},
        "extras": extras,
        "attention_ms_per_step": attn_ms,
        "setup_s": {"generate_and_upload": gen_s},
    })
    # every pass recalls each layer once, so the mean per-launch counter reading is the mean
    # over layers, the same average as bytes_per_launch
    rec = counter_traffic("recall_copy_kernel", 4)
    line["roofline"]["traffic"] = (rec or {}).get("total")
    line["roofline"]["traffic_split"] = rec
    if not (args.no_cpu_baseline or args.profile or compact):
        line["cpu_baseline"] = cpu_baseline(w0, args.cpu_seconds, "layer 0 of the 32-layer step")
    del ml
    torch.cuda.empty_cache()
    return line


LLAMA3_8B_FFN = 14336  # d_ff of the Llama-3-8B-shaped layers (d_model 4096 = 32 x 128)


def _irq_run(torch, ml, sched, normal, mode, engine, steps):
    ml.run_irq(sched, normal, mode=mode, engine=engine)  # warm-up
    rows = []
    for _ in range(steps):
        ml.reset()
        stats, depth = ml.run_irq(sched, normal, mode=mode, engine=engine)
        for st in ml.layers:
            if st.status() != 0:
                raise RuntimeError(f"offload device status {st.status()}")
        if normal is not None and normal.status() != 0:
            raise RuntimeError(f"normal device status {normal.status()}")
        rows.append(stats)
    return {k: statistics.mean(r[k] for r in rows) for k in rows[0]}


def bench_irq(args, torch, P, H):
    """Interruptible layer-wise scheduling (Sec. 4.2): preset 4's 32-layer offload batch
    (16 x 64K tokens) against a normal batch of args.normal_batch x 4K-token requests with
    resident KV and Llama-3-8B-shaped SwiGLU FFNs, 32 layers; every detection mode with the
    GPU gather kernel and with the gather-scatter engine as the recall path."""
    ml = H.MultiLayerStep(n_layers=32, n_stores=4)
    normal = H.NormalBatch(B=args.normal_batch, ctx=4096, n_layers=32, d_ff=LLAMA3_8B_FFN, seed=11)
    sched = P.IrqScheduler(ml.cmp_stream, ml.io_stream)
    w0 = ml.layers[0].w
    engine = P.GatherScatterEngine(ml.layers[0].shape, n_workers=8,
                                   max_blocks_per_call=max(st.w.B * st.k_max for st in ml.layers),
                                   staging_blocks=max(1, (16 << 20) // w0.unit_bytes))
    torch.cuda.synchronize()
    res = {}
    try:
        for path, eng in (("gather_kernel", None), ("gs_engine", engine)):
            for mode in ("blocking", "semi_sync", "sync", "async"):
                r = _irq_run(torch, ml, sched, normal, mode, eng, args.steps)
                wall_s = r["wall_ms"] * 1e-3
                r["offload_tokens_per_s"] = w0.B / wall_s  # one token per offload request per step
                r["normal_tokens_per_s"] = normal.B * r["normal_layers"] / normal.n_layers / wall_s
                res[f"{path}/{mode}"] = r
                print(f"[irq] {path}/{mode}: wall {r['wall_ms']:.2f} ms, normal layers {r['normal_layers']:.0f}, "
                      f"depth {r['mean_overlap_depth']:.2f}", file=sys.stderr, flush=True)
    finally:
        sched.destroy()
        engine.destroy()
    return {"report": "irq", "offload": {"workload": WORKLOADS[4], "layers": 32},
            "normal": {"batch": normal.B, "ctx": normal.ctx, "layers": normal.n_layers, "d_ff": normal.d_ff,
                       "d_model": 4096},
            "steps": args.steps, "results": res}


def bench_ioaa(args, torch, P, H):
    """Overlap depth m(B_o, B_n) measured with IRQ (semi-synchronous, gather-scatter engine)
    over a grid, then one IOAA admission (Sec. 4.3) of 30 waiting requests on that grid."""
    import numpy as np

    grid_bo, grid_bn, n_layers = [2, 4, 8, 16], [8, 16, 32], 8
    m = np.zeros((len(grid_bo), len(grid_bn)))
    detail = {}
    for i, bo in enumerate(grid_bo):
        ml = H.MultiLayerStep(n_layers=n_layers, n_stores=1, batch=bo, ctx_scale=0.5)
        sched = P.IrqScheduler(ml.cmp_stream, ml.io_stream)
        engine = P.GatherScatterEngine(ml.layers[0].shape, n_workers=8,
                                       max_blocks_per_call=max(st.w.B * st.k_max for st in ml.layers),
                                       staging_blocks=max(1, (16 << 20) // ml.layers[0].w.unit_bytes))
        try:
            for j, bn in enumerate(grid_bn):
                normal = H.NormalBatch(B=bn, ctx=4096, n_layers=n_layers, d_ff=LLAMA3_8B_FFN, seed=13)
                r = _irq_run(torch, ml, sched, normal, "semi_sync", engine, max(1, args.steps))
                m[i, j] = max(1.0, r["mean_overlap_depth"])  # one normal layer at least per offload layer
                detail[f"{bo}x{bn}"] = {"overlap_depth": r["mean_overlap_depth"], "stall_us": r["mean_stall_us"]}
                print(f"[ioaa] B_o {bo} B_n {bn}: m = {r['mean_overlap_depth']:.2f}", file=sys.stderr, flush=True)
                del normal
                torch.cuda.empty_cache()
        finally:
            sched.destroy()
            engine.destroy()
        del ml
        torch.cuda.empty_cache()
    # a waiting queue of 30 requests, lognormal lengths around 16K tokens (sigma 1)
    rng = np.random.default_rng(2026)
    lengths = np.clip(rng.lognormal(np.log(16384), 1.0, 30), 1024, 262144).astype(np.int64)
    kv_per_token = 2 * 8 * 128 * 2 * 32  # K and V, 8 KV heads x 128, bf16, 32 layers
    digest_bytes = (16384 // 16) * 2 * 128 * 2 * 32  # one head's per-block min/max, 32 layers, 16K tokens
    params = P.make_ioaa_params(40 << 30, kv_per_token, 2048, digest_bytes, 32, 8, grid_bo, grid_bn, m)
    t = time.perf_counter()
    assign, thr, nodes, leaves = P.pulse_ioaa_plan(params, lengths)
    plan_us = (time.perf_counter() - t) * 1e6
    return {"report": "ioaa", "grid_bo": grid_bo, "grid_bn": grid_bn, "overlap_depth": m.tolist(),
            "grid_detail": detail, "measured_with": "pulse_irq_step semi_sync + pulse_gs engine, 8 layers, "
                                                    "offload preset 4 shape at 32K tokens, normal 4K tokens",
            "queue": {"n": 30, "lengths": lengths.tolist(), "gpu_budget_bytes": 40 << 30,
                      "running_normal": 32, "running_offload": 8},
            "plan": {"normal": int((assign == 1).sum()), "offload": int((assign == 2).sum()),
                     "wait": int((assign == 0).sum()), "throughput_eq1": thr, "nodes_visited": nodes,
                     "assignments_evaluated": leaves,
                     "plan_us": plan_us}}


def bench_recall_sweep(args, torch, P, H, W):
    """Recall bandwidth against the number of blocks recalled in one call (the analogue of the
    paper's gather-scatter figure, Sec. 4.4.2): the preset's selection is cut down to its first
    n missing blocks (request order, block order), and the same blocks are recalled by the GPU
    gather kernel (pulse_recall_gather: plan + copy, HIP events), the paper's engine (submit to
    host-observed completion) and one hipMemcpyAsync per block (HIP events around the calls).
    Each recall starts from the initial table and free list; median of `reps` after a warm-up."""
    import numpy as np

    spec, seed = W.preset(args.config)
    holder = []
    w = W.generate(spec, seed, kv_alloc=H.pinned_allocator(holder))
    st = H.LayerState(w, holder[0].ptr)
    st.reset()
    st.select()
    torch.cuda.synchronize()
    idx, cnt = st.selection()
    missing = [(r, int(j)) for r in range(w.B) for j in idx[r, : cnt[r]] if w.table0[r, j] < 0]
    reps = 7
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    eng = P.GatherScatterEngine(st.shape, n_workers=8, max_blocks_per_call=w.B * st.k_max,
                                staging_blocks=max(1, (16 << 20) // w.unit_bytes))
    sizes = [n for n in (1, 2, 4, 8, 16, 32, 64, 128, 256, 512, 1024, 2048, 4096) if n < len(missing)]
    sizes.append(len(missing))
    rows = []
    try:
        for n in sizes:
            keep = set(missing[:n])
            sel = np.full_like(idx, -1)
            c = np.zeros_like(cnt)
            for r in range(w.B):  # the cut selection: its resident blocks and its first n missing ones
                js = [int(j) for j in idx[r, : cnt[r]] if w.table0[r, j] >= 0 or (r, int(j)) in keep]
                sel[r, : len(js)] = js
                c[r] = len(js)
            st.sel_idx.copy_(torch.from_numpy(sel))
            st.sel_cnt.copy_(torch.from_numpy(c))
            src = np.array([w.blk_off[r] + j for r, j in missing[:n]], np.int64)
            dst = np.array(w.free_slots[:n], np.int64)
            gather, engine, memcpy = [], [], []
            for rep in range(reps + 1):
                st.reset()
                torch.cuda.synchronize()
                e0.record()
                st.recall()
                e1.record()
                torch.cuda.synchronize()
                if st.recall_stats()[0] != n or st.status() != 0:
                    raise RuntimeError(f"gather recall of {n} blocks: stats {st.recall_stats()} status {st.status()}")
                gather.append(e0.elapsed_time(e1))
                st.reset()
                torch.cuda.synchronize()
                t0 = time.perf_counter()
                st.recall_gs(eng)
                engine.append((time.perf_counter() - t0) * 1e3)
                if st.recall_stats()[0] != n or st.status() != 0:
                    raise RuntimeError(f"engine recall of {n} blocks: stats {st.recall_stats()} status {st.status()}")
                e0.record()
                P.pulse_baseline_memcpy_units(st.host_ptr, st.pool, src, dst, n, w.unit_bytes)
                e1.record()
                torch.cuda.synchronize()
                memcpy.append(e0.elapsed_time(e1))
            nbytes = n * w.unit_bytes
            row = {"blocks": n, "bytes": nbytes}
            for name, t in (("gather_kernel", gather), ("engine", engine), ("per_block_memcpy", memcpy)):
                ms = statistics.median(t[1:])
                row[name] = {"us": ms * 1e3, "GBps": nbytes / (ms * 1e-3) / 1e9}
            rows.append(row)
            print(f"# {n:5d} blocks: gather {row['gather_kernel']['GBps']:6.2f}  engine {row['engine']['GBps']:6.2f}"
                  f"  per-block memcpy {row['per_block_memcpy']['GBps']:6.2f} GB/s", file=sys.stderr, flush=True)
    finally:
        eng.destroy()
    return {"report": "recall_sweep", "workload": WORKLOADS[args.config], "unit_bytes": w.unit_bytes,
            "timing": "gather: HIP events around pulse_recall_gather (plan + copy kernels); engine: host wall time "
                      "from submit to observed completion; per-block memcpy: HIP events around the n calls",
            "rows": rows}


def main():
    args = parse()
    if args.summarize_counters:
        summarize_counters(args.summarize_counters, args.config)
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the sparse-KV decode path here has no multi-GPU mode "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)
    import torch

    from paper_2609_34555_amd import harness as H
    from paper_2609_34555_amd import pulse as P
    from paper_2609_34555_amd import workloads as W

    torch.cuda.set_device(0)
    if args.recall_sweep:
        print(json.dumps(bench_recall_sweep(args, torch, P, H, W)), flush=True)
        return
    if args.irq or args.ioaa_profile:
        line = bench_irq(args, torch, P, H) if args.irq else bench_ioaa(args, torch, P, H)
        print(json.dumps(line), flush=True)
        return
    if args.config == 4:
        line = bench_multilayer(args, torch, P, H, W)
    else:
        line = bench_layer(args.config, args, torch, P, H, W)
    if args.config == 3 and not (args.no_presets or args.profile):
        line["presets"] = presets_record(args, torch, P, H, W)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
