"""ctypes binding of libpulse.so (include/pulse.h), argument marshalling only.

Every function has the name of its C entry point and forwards plain pointers:
a torch tensor argument passes ``tensor.data_ptr()``, an int passes itself,
None passes NULL.  ``stream`` defaults to torch's current HIP stream.  A
non-OK status raises PulseError.  All compute runs in the library's kernels;
there is no fallback: a missing library raises at import of the first call.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libpulse.so")

PULSE_OK = 0
PULSE_ERR_INVALID_ARG = 1
PULSE_ERR_UNSUPPORTED = 2
PULSE_ERR_WORKSPACE = 3
PULSE_ERR_POOL_EXHAUSTED = 4
PULSE_ERR_SELECT_OVERFLOW = 5
PULSE_ERR_HIP = 6
PULSE_ERR_BAD_INDEX = 7
PULSE_ERR_TIMEOUT = 8

NOALLOC_SCRATCH_BYTES = 32 << 20  # PULSE_NOALLOC_SCRATCH_BYTES: static workspace of pulse_decode_layer_noalloc
PULSE_F16 = 0
PULSE_BF16 = 1

EXPORTED = (
    "pulse_status_string", "pulse_block_bytes", "pulse_workspace_bytes", "pulse_build_digests",
    "pulse_select_solohead", "pulse_recall_gather", "pulse_sparse_decode_attn", "pulse_decode_layer",
    "pulse_decode_layer_noalloc",
    "pulse_host_alloc", "pulse_host_free", "pulse_baseline_memcpy_units", "pulse_probe_host_read",
    "pulse_events_create", "pulse_events_destroy", "pulse_event_elapsed_ms", "pulse_headwise_workspace_bytes",
    "pulse_select_headwise", "pulse_gs_engine_create", "pulse_gs_engine_destroy", "pulse_gs_recall_submit",
    "pulse_gs_recall_poll", "pulse_gs_recall_wait", "pulse_gs_last_timing", "pulse_overlap_depth",
    "pulse_ioaa_plan", "pulse_average_workspace_bytes", "pulse_select_average", "pulse_mam_workspace_bytes",
    "pulse_mam", "pulse_pick_solo_heads", "pulse_irq_create", "pulse_irq_destroy", "pulse_irq_step",
    "pulse_probe_hbm_read", "pulse_probe_hbm_sink_bytes", "pulse_release_recalled", "pulse_attention_workgroups",
)


class PulseError(RuntimeError):
    def __init__(self, status: int, where: str):
        super().__init__(f"{where}: {status_string(status)} ({status})")
        self.status = status


class pulse_shape(ctypes.Structure):
    _fields_ = [("num_q_heads", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("block_size", ctypes.c_int32), ("dtype", ctypes.c_int32)]


class pulse_recall_stats(ctypes.Structure):
    _fields_ = [("n_missing", ctypes.c_int32), ("n_runs", ctypes.c_int32), ("bytes", ctypes.c_int64)]


_P = ctypes.c_void_p


class pulse_ioaa_params(ctypes.Structure):
    _fields_ = [("gpu_budget_bytes", ctypes.c_int64), ("kv_bytes_per_token", ctypes.c_int64),
                ("offload_tokens", ctypes.c_int64), ("offload_extra_bytes", ctypes.c_int64),
                ("running_normal", ctypes.c_int32), ("running_offload", ctypes.c_int32),
                ("grid_bo", ctypes.c_void_p), ("n_bo", ctypes.c_int32), ("grid_bn", ctypes.c_void_p),
                ("n_bn", ctypes.c_int32), ("grid_m", ctypes.c_void_p)]


class pulse_layer_args(ctypes.Structure):
    _fields_ = [
        ("shape", pulse_shape), ("B", ctypes.c_int32), ("total_blocks", ctypes.c_int64), ("ctx_len", _P),
        ("blk_off", _P), ("q", _P), ("digests", _P), ("solo_kv_head", ctypes.c_int32), ("k_mid", _P),
        ("n_sink_blocks", ctypes.c_int32), ("n_local_blocks", ctypes.c_int32), ("k_max", ctypes.c_int32),
        ("sel_idx", _P), ("sel_cnt", _P), ("host_kv", _P), ("block_table", _P), ("max_blocks", ctypes.c_int32),
        ("free_slots", _P), ("free_head", _P), ("n_free", ctypes.c_int32), ("slot_pool", _P),
        ("n_slots", ctypes.c_int32), ("stats", _P), ("sm_scale", ctypes.c_float), ("out", _P), ("lse", _P),
        ("dev_status", _P), ("ws", _P), ("ws_bytes", ctypes.c_size_t), ("events", _P),
        ("release_previous", ctypes.c_int32), ("attn_split_event", _P),
    ]


class pulse_normal_layer(ctypes.Structure):
    _fields_ = [
        ("shape", pulse_shape), ("B", ctypes.c_int32), ("q", _P), ("slot_pool", _P), ("n_slots", ctypes.c_int32),
        ("block_table", _P), ("max_blocks", ctypes.c_int32), ("sel_idx", _P), ("sel_cnt", _P),
        ("k_max", ctypes.c_int32), ("ctx_len", _P), ("sm_scale", ctypes.c_float), ("out", _P), ("lse", _P),
        ("ws", _P), ("ws_bytes", ctypes.c_size_t), ("d_ff", ctypes.c_int32), ("w_gate_up", _P), ("w_down", _P),
        ("x", _P), ("gu", _P), ("h", _P), ("y", _P), ("dev_status", _P),
    ]


class pulse_irq_stats(ctypes.Structure):
    _fields_ = [("normal_layers", ctypes.c_int64), ("offload_layers", ctypes.c_int32),
                ("max_overlap_depth", ctypes.c_int32), ("mean_overlap_depth", ctypes.c_double),
                ("wall_ms", ctypes.c_double), ("mean_stall_us", ctypes.c_double),
                ("mean_resume_us", ctypes.c_double), ("mean_recall_us", ctypes.c_double)]

    def as_dict(self):
        return {k: getattr(self, k) for k, _ in self._fields_}


PULSE_IRQ_SEMI_SYNC, PULSE_IRQ_SYNC, PULSE_IRQ_ASYNC, PULSE_IRQ_BLOCKING = 0, 1, 2, 3
IRQ_MODES = {"semi_sync": PULSE_IRQ_SEMI_SYNC, "sync": PULSE_IRQ_SYNC, "async": PULSE_IRQ_ASYNC,
             "blocking": PULSE_IRQ_BLOCKING}

_lib = None


def lib():
    """The loaded libpulse.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build()")
        # torch bundles a HIP runtime with the same soname as /opt/rocm's; loading torch
        # first makes libpulse bind to that one runtime instead of mapping a second copy
        import torch  # noqa: F401

        L = ctypes.CDLL(LIB_PATH)
        bind(L, signatures())
        _lib = L
    return _lib


def bind(L, sig):
    """Set restype / argtypes of every entry of `sig` (name -> (restype, argtypes)) on library L."""
    for name, (res, args) in sig.items():
        fn = getattr(L, name)
        fn.restype = res
        fn.argtypes = args
    return L


def signatures():
    """C signatures of the exported entry points, as ctypes types."""
    I32, I64, SZ, F = ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t, ctypes.c_float
    SP = ctypes.POINTER(pulse_shape)
    sig = {
        "pulse_status_string": (ctypes.c_char_p, [ctypes.c_int]),
        "pulse_block_bytes": (SZ, [SP]),
        "pulse_workspace_bytes": (SZ, [SP, I32, I32, I64]),
        "pulse_attention_workgroups": (I32, [SP, I32, I32]),
        "pulse_build_digests": (ctypes.c_int, [SP, _P, _P, _P, I32, I64, I32, _P, _P, _P]),
        "pulse_select_solohead": (ctypes.c_int, [SP, _P, _P, _P, I32, I64, I32, _P, I32, I32, I32, _P, _P, _P,
                                                 _P, _P, SZ, _P]),
        "pulse_recall_gather": (ctypes.c_int, [SP, _P, _P, I32, _P, _P, I32, _P, I32, _P, _P, I32, _P, I32, _P,
                                               _P, _P, SZ, _P]),
        "pulse_sparse_decode_attn": (ctypes.c_int, [SP, _P, _P, I32, _P, I32, _P, _P, I32, _P, I32, F, _P, _P,
                                                    _P, _P, SZ, _P]),
        "pulse_decode_layer": (ctypes.c_int, [ctypes.POINTER(pulse_layer_args), _P]),
        "pulse_decode_layer_noalloc": (ctypes.c_int, [ctypes.POINTER(pulse_layer_args), _P]),
        "pulse_host_alloc": (ctypes.c_int, [SZ, I32, ctypes.POINTER(ctypes.c_void_p)]),
        "pulse_host_free": (ctypes.c_int, [_P]),
        "pulse_baseline_memcpy_units": (ctypes.c_int, [_P, _P, _P, _P, I32, SZ, _P]),
        "pulse_probe_host_read": (ctypes.c_int, [_P, _P, SZ, _P]),
        "pulse_probe_hbm_read": (ctypes.c_int, [_P, SZ, _P, _P, _P, _P]),
        "pulse_release_recalled": (ctypes.c_int, [SP, I32, I32, I64, _P, I32, _P, _P, _P, _P, SZ, _P]),
        "pulse_probe_hbm_sink_bytes": (SZ, []),
        "pulse_headwise_workspace_bytes": (SZ, [SP, I32, I32, I64]),
        "pulse_select_headwise": (ctypes.c_int, [SP, _P, _P, _P, I32, I64, _P, I32, I32, I32, _P, I32, I32, _P,
                                                 _P, _P, _P, _P, _P, SZ, _P]),
        "pulse_average_workspace_bytes": (SZ, [SP, I32, I32, I64]),
        "pulse_select_average": (ctypes.c_int, [SP, _P, _P, _P, I32, I64, _P, I32, I32, I32, _P, _P, _P, _P, _P,
                                                SZ, _P]),
        "pulse_mam_workspace_bytes": (SZ, [SP, I32, I32]),
        "pulse_mam": (ctypes.c_int, [SP, _P, _P, I32, _P, I32, _P, I32, I32, I32, F, _P, _P, _P, SZ, _P]),
        "pulse_pick_solo_heads": (ctypes.c_int, [_P, I32, I32, ctypes.POINTER(I32), ctypes.POINTER(I32)]),
        "pulse_irq_create": (ctypes.c_int, [_P, _P, ctypes.POINTER(ctypes.c_void_p)]),
        "pulse_irq_destroy": (ctypes.c_int, [_P]),
        "pulse_irq_step": (ctypes.c_int, [_P, ctypes.POINTER(pulse_layer_args), I32,
                                          ctypes.POINTER(pulse_normal_layer), I32, I32, I32, _P, _P,
                                          ctypes.POINTER(pulse_irq_stats)]),
        "pulse_gs_engine_create": (ctypes.c_int, [SP, I32, I64, I64, ctypes.POINTER(ctypes.c_void_p)]),
        "pulse_gs_engine_destroy": (ctypes.c_int, [_P]),
        "pulse_gs_recall_submit": (ctypes.c_int, [_P, _P, _P, I32, _P, _P, I32, _P, I32, _P, _P, I32, _P, I32, _P,
                                                  _P, _P, SZ, ctypes.POINTER(ctypes.c_int64), _P]),
        "pulse_gs_recall_poll": (ctypes.c_int, [_P, I64, ctypes.POINTER(ctypes.c_int32)]),
        "pulse_gs_recall_wait": (ctypes.c_int, [_P, I64, I32]),
        "pulse_gs_last_timing": (ctypes.c_int, [_P, ctypes.POINTER(ctypes.c_float)]),
        "pulse_overlap_depth": (ctypes.c_double, [ctypes.POINTER(pulse_ioaa_params), ctypes.c_double,
                                                  ctypes.c_double]),
        "pulse_ioaa_plan": (ctypes.c_int, [ctypes.POINTER(pulse_ioaa_params), _P, I32, _P,
                                           ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int64),
                                           ctypes.POINTER(ctypes.c_int64)]),
        "pulse_events_create": (ctypes.c_int, [I32, _P]),
        "pulse_events_destroy": (ctypes.c_int, [I32, _P]),
        "pulse_event_elapsed_ms": (ctypes.c_int, [_P, _P, ctypes.POINTER(ctypes.c_float)]),
    }
    return sig


def _ptr(x):
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if hasattr(x, "data_ptr"):
        return x.data_ptr()
    if hasattr(x, "ctypes"):  # numpy array (host buffers)
        return x.ctypes.data
    raise TypeError(f"cannot pass {type(x)} as a pointer")


def _stream(stream):
    if stream is None:
        import torch

        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _check(status: int, where: str, check: bool):
    if check and status != PULSE_OK:
        raise PulseError(status, where)
    return status


def status_string(status: int) -> str:
    return lib().pulse_status_string(int(status)).decode()


def make_shape(num_q_heads, num_kv_heads, head_dim, block_size, dtype) -> pulse_shape:
    return pulse_shape(num_q_heads, num_kv_heads, head_dim, block_size, dtype)


def pulse_block_bytes(shape: pulse_shape) -> int:
    return lib().pulse_block_bytes(ctypes.byref(shape))


def pulse_workspace_bytes(shape: pulse_shape, B: int, k_max: int, total_blocks: int) -> int:
    return lib().pulse_workspace_bytes(ctypes.byref(shape), B, k_max, total_blocks)


def pulse_attention_workgroups(shape: pulse_shape, B: int, k_max: int) -> int:
    """Split-K workgroups per (request, KV head) of the attention; above 1 a merge kernel follows."""
    return lib().pulse_attention_workgroups(ctypes.byref(shape), B, k_max)


def pulse_build_digests(shape, kv, blk_off, ctx_len, B, total_blocks, kv_head, digests, dev_status=None,
                        stream=None, check=True):
    st = lib().pulse_build_digests(ctypes.byref(shape), _ptr(kv), _ptr(blk_off), _ptr(ctx_len), B, total_blocks,
                                   kv_head, _ptr(digests), _ptr(dev_status), _stream(stream))
    return _check(st, "pulse_build_digests", check)


def pulse_select_solohead(shape, q, digests, blk_off, B, total_blocks, solo_kv_head, k_mid, n_sink_blocks,
                          n_local_blocks, k_max, sel_idx, sel_cnt, scores, dev_status, ws, ws_bytes, stream=None,
                          check=True):
    st = lib().pulse_select_solohead(ctypes.byref(shape), _ptr(q), _ptr(digests), _ptr(blk_off), B, total_blocks,
                                     solo_kv_head, _ptr(k_mid), n_sink_blocks, n_local_blocks, k_max, _ptr(sel_idx),
                                     _ptr(sel_cnt), _ptr(scores), _ptr(dev_status), _ptr(ws), ws_bytes,
                                     _stream(stream))
    return _check(st, "pulse_select_solohead", check)


def pulse_headwise_workspace_bytes(shape: pulse_shape, B: int, k_max: int, total_blocks: int) -> int:
    return lib().pulse_headwise_workspace_bytes(ctypes.byref(shape), B, k_max, total_blocks)


def pulse_select_headwise(shape, q, head_digests, blk_off, B, total_blocks, k_mid, n_sink_blocks, n_local_blocks,
                          k_max, block_table, max_blocks, n_slots, sel_idx, sel_cnt, miss_cnt, run_cnt, dev_status, ws,
                          ws_bytes, stream=None, check=True):
    st = lib().pulse_select_headwise(ctypes.byref(shape), _ptr(q), _ptr(head_digests), _ptr(blk_off), B,
                                     total_blocks, _ptr(k_mid), n_sink_blocks, n_local_blocks, k_max,
                                     _ptr(block_table), max_blocks, n_slots, _ptr(sel_idx), _ptr(sel_cnt),
                                     _ptr(miss_cnt), _ptr(run_cnt), _ptr(dev_status), _ptr(ws), ws_bytes,
                                     _stream(stream))
    return _check(st, "pulse_select_headwise", check)


def pulse_average_workspace_bytes(shape: pulse_shape, B: int, k_max: int, total_blocks: int) -> int:
    return lib().pulse_average_workspace_bytes(ctypes.byref(shape), B, k_max, total_blocks)


def pulse_select_average(shape, q, head_digests, blk_off, B, total_blocks, k_mid, n_sink_blocks, n_local_blocks,
                         k_max, sel_idx, sel_cnt, scores, dev_status, ws, ws_bytes, stream=None, check=True):
    st = lib().pulse_select_average(ctypes.byref(shape), _ptr(q), _ptr(head_digests), _ptr(blk_off), B,
                                    total_blocks, _ptr(k_mid), n_sink_blocks, n_local_blocks, k_max, _ptr(sel_idx),
                                    _ptr(sel_cnt), _ptr(scores), _ptr(dev_status), _ptr(ws), ws_bytes,
                                    _stream(stream))
    return _check(st, "pulse_select_average", check)


def pulse_mam_workspace_bytes(shape: pulse_shape, B: int, max_blocks: int) -> int:
    return lib().pulse_mam_workspace_bytes(ctypes.byref(shape), B, max_blocks)


def pulse_mam(shape, q, slot_pool, n_slots, block_table, max_blocks, ctx_len, B, n_sink_blocks, n_local_blocks,
              sm_scale, mam, dev_status, ws, ws_bytes, stream=None, check=True):
    st = lib().pulse_mam(ctypes.byref(shape), _ptr(q), _ptr(slot_pool), n_slots, _ptr(block_table), max_blocks,
                         _ptr(ctx_len), B, n_sink_blocks, n_local_blocks, float(sm_scale), _ptr(mam),
                         _ptr(dev_status), _ptr(ws), ws_bytes, _stream(stream))
    return _check(st, "pulse_mam", check)


def pulse_pick_solo_heads(mam, check=True):
    """(solo, reversed) KV heads from a host float32 array [rows, num_kv_heads]."""
    import numpy as np

    m = np.ascontiguousarray(mam, dtype=np.float32)
    if m.ndim == 1:
        m = m[None, :]
    solo, rev = ctypes.c_int32(-1), ctypes.c_int32(-1)
    st = lib().pulse_pick_solo_heads(_ptr(m), m.shape[0], m.shape[1], ctypes.byref(solo), ctypes.byref(rev))
    _check(st, "pulse_pick_solo_heads", check)
    return solo.value, rev.value


class IrqScheduler:
    """pulse_irq_* : interruptible layer-wise scheduling of an offload batch against a
    normal batch on two streams (compute, I/O)."""

    def __init__(self, compute_stream, io_stream):
        h = ctypes.c_void_p()
        _check(lib().pulse_irq_create(_stream(compute_stream), _stream(io_stream), ctypes.byref(h)),
               "pulse_irq_create", True)
        self.handle = h

    def step(self, offload_args, normal_layers, mode="semi_sync", async_ahead=4, engine=None, check=True):
        """offload_args: list of pulse_layer_args; normal_layers: list of pulse_normal_layer;
        engine: an optional GatherScatterEngine for the recalls.  Returns (stats dict,
        per-layer overlap depths)."""
        import numpy as np

        L = len(offload_args)
        off = (pulse_layer_args * L)(*offload_args)
        nn = len(normal_layers)
        nrm = (pulse_normal_layer * max(nn, 1))(*normal_layers) if nn else None
        depth = np.zeros(L, np.int32)
        st = pulse_irq_stats()
        rc = lib().pulse_irq_step(self.handle, off, L, nrm, nn, IRQ_MODES[mode] if isinstance(mode, str) else mode,
                                  async_ahead, engine.handle if engine is not None else None, depth.ctypes.data,
                                  ctypes.byref(st))
        _check(rc, "pulse_irq_step", check)
        return st.as_dict(), depth

    def destroy(self):
        if self.handle:
            lib().pulse_irq_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.destroy()
        except Exception:
            pass


def pulse_recall_gather(shape, host_kv, blk_off, B, sel_idx, sel_cnt, k_max, block_table, max_blocks, free_slots,
                        free_head, n_free, slot_pool, n_slots, stats, dev_status, ws, ws_bytes, stream=None,
                        check=True):
    st = lib().pulse_recall_gather(ctypes.byref(shape), _ptr(host_kv), _ptr(blk_off), B, _ptr(sel_idx),
                                   _ptr(sel_cnt), k_max, _ptr(block_table), max_blocks, _ptr(free_slots),
                                   _ptr(free_head), n_free, _ptr(slot_pool), n_slots, _ptr(stats), _ptr(dev_status),
                                   _ptr(ws), ws_bytes, _stream(stream))
    return _check(st, "pulse_recall_gather", check)


def pulse_release_recalled(shape, B, k_max, total_blocks, block_table, max_blocks, free_head, stats, dev_status,
                           ws, ws_bytes, stream=None, check=True):
    st = lib().pulse_release_recalled(ctypes.byref(shape), B, k_max, total_blocks, _ptr(block_table), max_blocks,
                                      _ptr(free_head), _ptr(stats), _ptr(dev_status), _ptr(ws), ws_bytes,
                                      _stream(stream))
    return _check(st, "pulse_release_recalled", check)


def pulse_sparse_decode_attn(shape, q, slot_pool, n_slots, block_table, max_blocks, sel_idx, sel_cnt, k_max,
                             ctx_len, B, sm_scale, out, lse, dev_status, ws, ws_bytes, stream=None, check=True):
    st = lib().pulse_sparse_decode_attn(ctypes.byref(shape), _ptr(q), _ptr(slot_pool), n_slots, _ptr(block_table),
                                        max_blocks, _ptr(sel_idx), _ptr(sel_cnt), k_max, _ptr(ctx_len), B,
                                        float(sm_scale), _ptr(out), _ptr(lse), _ptr(dev_status), _ptr(ws), ws_bytes,
                                        _stream(stream))
    return _check(st, "pulse_sparse_decode_attn", check)


def pulse_decode_layer(args: pulse_layer_args, stream=None, check=True):
    st = lib().pulse_decode_layer(ctypes.byref(args), _stream(stream))
    return _check(st, "pulse_decode_layer", check)


def pulse_decode_layer_noalloc(args: pulse_layer_args, stream=None, check=True):
    st = lib().pulse_decode_layer_noalloc(ctypes.byref(args), _stream(stream))
    return _check(st, "pulse_decode_layer_noalloc", check)


def pulse_host_alloc(nbytes: int, coherent: bool = True) -> int:
    p = ctypes.c_void_p()
    _check(lib().pulse_host_alloc(nbytes, 1 if coherent else 0, ctypes.byref(p)), "pulse_host_alloc", True)
    return p.value


def pulse_host_free(ptr: int):
    return _check(lib().pulse_host_free(ptr), "pulse_host_free", True)


def pulse_baseline_memcpy_units(host_kv, pool, src_units, dst_units, n, unit_bytes, stream=None, check=True):
    st = lib().pulse_baseline_memcpy_units(_ptr(host_kv), _ptr(pool), _ptr(src_units), _ptr(dst_units), n,
                                           unit_bytes, _stream(stream))
    return _check(st, "pulse_baseline_memcpy_units", check)


def pulse_probe_host_read(host_src, dev_dst, nbytes, stream=None, check=True):
    st = lib().pulse_probe_host_read(_ptr(host_src), _ptr(dev_dst), nbytes, _stream(stream))
    return _check(st, "pulse_probe_host_read", check)


def pulse_probe_hbm_read(src, nbytes, sink, stream=None, check=True, start_event=None, stop_event=None):
    st = lib().pulse_probe_hbm_read(_ptr(src), nbytes, _ptr(sink), start_event, stop_event, _stream(stream))
    return _check(st, "pulse_probe_hbm_read", check)


def pulse_probe_hbm_sink_bytes() -> int:
    return lib().pulse_probe_hbm_sink_bytes()


def make_ioaa_params(gpu_budget_bytes, kv_bytes_per_token, offload_tokens, offload_extra_bytes, running_normal,
                     running_offload, grid_bo, grid_bn, grid_m):
    """pulse_ioaa_params holding references to float64 numpy grids (kept on the struct)."""
    import numpy as np

    bo = np.ascontiguousarray(grid_bo, dtype=np.float64)
    bn = np.ascontiguousarray(grid_bn, dtype=np.float64)
    m = np.ascontiguousarray(grid_m, dtype=np.float64).reshape(bo.size, bn.size)
    p = pulse_ioaa_params(int(gpu_budget_bytes), int(kv_bytes_per_token), int(offload_tokens),
                          int(offload_extra_bytes), int(running_normal), int(running_offload), bo.ctypes.data,
                          bo.size, bn.ctypes.data, bn.size, m.ctypes.data)
    p._keep = (bo, bn, m)
    return p


def pulse_overlap_depth(params: pulse_ioaa_params, b_o: float, b_n: float) -> float:
    return lib().pulse_overlap_depth(ctypes.byref(params), float(b_o), float(b_n))


def pulse_ioaa_plan(params: pulse_ioaa_params, lengths):
    """Returns (assign int8 [n]: 0 wait / 1 normal / 2 offload, throughput, nodes_visited,
    leaves_evaluated)."""
    import numpy as np

    L = np.ascontiguousarray(lengths, dtype=np.int64)
    assign = np.zeros(L.size, np.int8)
    thr = ctypes.c_double()
    nodes = ctypes.c_int64()
    leaves = ctypes.c_int64()
    _check(lib().pulse_ioaa_plan(ctypes.byref(params), L.ctypes.data if L.size else None, L.size,
                                 assign.ctypes.data if L.size else None, ctypes.byref(thr), ctypes.byref(nodes),
                                 ctypes.byref(leaves)),
           "pulse_ioaa_plan", True)
    return assign, thr.value, nodes.value, leaves.value


class GatherScatterEngine:
    """Handle of a pulse_gs_engine (the paper's CPU-gather / one-DMA / GPU-scatter path)."""

    def __init__(self, shape: pulse_shape, n_workers: int, max_blocks_per_call: int, staging_blocks: int):
        h = ctypes.c_void_p()
        _check(lib().pulse_gs_engine_create(ctypes.byref(shape), n_workers, max_blocks_per_call, staging_blocks,
                                            ctypes.byref(h)), "pulse_gs_engine_create", True)
        self.handle = h.value

    def submit(self, host_kv, blk_off, B, sel_idx, sel_cnt, k_max, block_table, max_blocks, free_slots, free_head,
               n_free, slot_pool, n_slots, stats, dev_status, ws, ws_bytes, stream=None) -> int:
        seq = ctypes.c_int64()
        _check(lib().pulse_gs_recall_submit(self.handle, _ptr(host_kv), _ptr(blk_off), B, _ptr(sel_idx),
                                            _ptr(sel_cnt), k_max, _ptr(block_table), max_blocks, _ptr(free_slots),
                                            _ptr(free_head), n_free, _ptr(slot_pool), n_slots, _ptr(stats),
                                            _ptr(dev_status), _ptr(ws), ws_bytes, ctypes.byref(seq),
                                            _stream(stream)), "pulse_gs_recall_submit", True)
        return seq.value

    def poll(self, seq: int) -> bool:
        done = ctypes.c_int32()
        _check(lib().pulse_gs_recall_poll(self.handle, seq, ctypes.byref(done)), "pulse_gs_recall_poll", True)
        return bool(done.value)

    def wait(self, seq: int, timeout_ms: int = 10000):
        return _check(lib().pulse_gs_recall_wait(self.handle, seq, timeout_ms), "pulse_gs_recall_wait", True)

    def last_timing(self):
        ms = (ctypes.c_float * 3)()
        _check(lib().pulse_gs_last_timing(self.handle, ms), "pulse_gs_last_timing", True)
        return {"gather_ms": ms[0], "dma_scatter_tail_ms": ms[1], "total_ms": ms[2]}

    def destroy(self):
        if self.handle:
            lib().pulse_gs_engine_destroy(self.handle)
            self.handle = None


class EventSet:
    """n HIP events owned by the library's helpers (for pulse_layer_args.events)."""

    def __init__(self, n: int):
        self.n = n
        self._masked = []
        self.arr = (ctypes.c_void_p * n)()
        _check(lib().pulse_events_create(n, ctypes.cast(self.arr, ctypes.c_void_p)), "pulse_events_create", True)

    @property
    def ptr(self) -> int:
        return ctypes.addressof(self.arr)

    def masked_ptr(self, keep) -> int:
        """Address of a copy of the handle array in which the entries not in `keep` are
        NULL (pulse_decode_layer records only the non-NULL ones)."""
        masked = (ctypes.c_void_p * self.n)(*[self.arr[i] if i in keep else None for i in range(self.n)])
        self._masked.append(masked)  # kept alive as long as the set
        return ctypes.addressof(masked)

    def elapsed_ms(self, i: int, j: int) -> float:
        ms = ctypes.c_float()
        _check(lib().pulse_event_elapsed_ms(self.arr[i], self.arr[j], ctypes.byref(ms)), "pulse_event_elapsed_ms",
               True)
        return ms.value

    def destroy(self):
        if self.arr is not None:
            lib().pulse_events_destroy(self.n, ctypes.cast(self.arr, ctypes.c_void_p))
            self.arr = None
