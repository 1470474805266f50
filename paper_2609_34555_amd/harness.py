"""Device-side state of one layer-step for a generated workload.

Owns the buffers the C ABI operates on (torch device tensors and a pinned,
host-mapped KV store), the pristine copies needed to restore the block table
and free-list head between steps, and ready-made argument packs.  Used by the
tests, the smoke check and the benchmark; it does no compute of its own
beyond the caller-side setup (uploads and state restores).
"""
from __future__ import annotations

import ctypes
import math
from typing import Optional

import numpy as np
import torch

from . import pulse as P
from .workloads import BF16 as P_BF16
from .workloads import Workload


class PinnedStore:
    """Pinned, host-mapped memory from pulse_host_alloc, viewable as numpy."""

    def __init__(self, nbytes: int, coherent: bool = True):
        self.nbytes = int(nbytes)
        self.ptr = P.pulse_host_alloc(max(self.nbytes, 1), coherent)
        self.coherent = coherent

    def numpy(self, shape, dtype) -> np.ndarray:
        n = int(np.prod(shape)) * np.dtype(dtype).itemsize
        if n > self.nbytes:
            raise ValueError("view larger than the pinned allocation")
        buf = (ctypes.c_char * max(n, 1)).from_address(self.ptr)
        return np.frombuffer(buf, dtype=dtype, count=int(np.prod(shape))).reshape(shape)

    def free(self):
        if self.ptr:
            P.pulse_host_free(self.ptr)
            self.ptr = 0

    def __del__(self):
        try:
            self.free()
        except Exception:
            pass


def pinned_allocator(holder: list, coherent: bool = True):
    """kv_alloc callback for workloads.generate that places the store in pinned memory."""

    def alloc(shape, dtype):
        store = PinnedStore(int(np.prod(shape)) * np.dtype(dtype).itemsize, coherent)
        holder.append(store)
        return store.numpy(shape, dtype)

    return alloc


def _dev(a: np.ndarray, device) -> torch.Tensor:
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    return torch.from_numpy(a).to(device)


class LayerState:
    """All device buffers of one layer-step of workload ``w``.

    host_ptr: address of the pinned host-mapped store holding ``w.kv`` (the
    workload must have been generated into it)."""

    def __init__(self, w: Workload, host_ptr: int, device="cuda", k_max: Optional[int] = None,
                 build_digests: bool = True):
        self.w = w
        self.device = torch.device(device)
        self.shape = P.make_shape(w.Hq, w.Hkv, w.d, w.bs, w.dtype_code)
        self.host_ptr = int(host_ptr)
        self.k_max = int(k_max or w.k_max)
        dev = self.device
        self.ctx_len = _dev(w.ctx_len, dev)
        self.blk_off = _dev(w.blk_off, dev)
        self.q = _dev(w.q, dev)
        self.k_mid = _dev(w.k_mid, dev)
        self.table0 = _dev(w.table0, dev)
        self.table = self.table0.clone()
        self.free_slots = _dev(w.free_slots, dev) if w.free_slots.size else torch.zeros(1, dtype=torch.int32,
                                                                                        device=dev)
        self.free_head0 = torch.zeros(1, dtype=torch.int32, device=dev)
        self.free_head = self.free_head0.clone()
        E = w.elems_per_block
        self.pool = torch.zeros((w.n_slots, E), dtype=torch.int16, device=dev)
        if w.resident_blocks.size:
            self.pool[: w.resident_blocks.size] = _dev(w.kv[w.resident_blocks], dev)
        self.sel_idx = torch.full((w.B, self.k_max), -1, dtype=torch.int32, device=dev)
        self.sel_cnt = torch.zeros(w.B, dtype=torch.int32, device=dev)
        self.stats = torch.zeros(2, dtype=torch.int64, device=dev)  # pulse_recall_stats (16 bytes)
        self.dev_status = torch.zeros(1, dtype=torch.int32, device=dev)
        self.out = torch.zeros((w.B, w.Hq, w.d), dtype=torch.float32, device=dev)
        self.lse = torch.zeros((w.B, w.Hq), dtype=torch.float32, device=dev)
        self.ws_bytes = P.pulse_workspace_bytes(self.shape, w.B, self.k_max, w.total_blocks)
        self.ws = torch.zeros(max(self.ws_bytes, 1), dtype=torch.uint8, device=dev)
        self.digests = torch.zeros((max(w.total_blocks, 1), 2, w.d), dtype=torch.int16, device=dev)
        if build_digests:
            self.build_digests(w.solo_kv_head)

    # ------------------------------------------------------------------ steps
    def build_digests(self, kv_head: int, out: Optional[torch.Tensor] = None, stream=None):
        w = self.w
        dst = self.digests if out is None else out
        P.pulse_build_digests(self.shape, self.host_ptr, self.blk_off, self.ctx_len, w.B, w.total_blocks, kv_head,
                              dst, self.dev_status, stream=stream)
        return dst

    def reset(self):
        """Restore the block table and free-list head of the step's start; clear status and
        the recall statistics (no recall is left to release)."""
        self.table.copy_(self.table0)
        self.free_head.copy_(self.free_head0)
        self.dev_status.zero_()
        self.stats.zero_()

    def layer_args(self, digests: Optional[torch.Tensor] = None, release_previous: bool = False
                   ) -> P.pulse_layer_args:
        w = self.w
        a = P.pulse_layer_args()
        a.shape = self.shape
        a.B = w.B
        a.total_blocks = w.total_blocks
        a.ctx_len = self.ctx_len.data_ptr()
        a.blk_off = self.blk_off.data_ptr()
        a.q = self.q.data_ptr()
        a.digests = (self.digests if digests is None else digests).data_ptr()
        a.solo_kv_head = w.solo_kv_head
        a.k_mid = self.k_mid.data_ptr()
        a.n_sink_blocks = w.n_sink
        a.n_local_blocks = w.n_local
        a.k_max = self.k_max
        a.sel_idx = self.sel_idx.data_ptr()
        a.sel_cnt = self.sel_cnt.data_ptr()
        a.host_kv = self.host_ptr
        a.block_table = self.table.data_ptr()
        a.max_blocks = w.max_blocks
        a.free_slots = self.free_slots.data_ptr()
        a.free_head = self.free_head.data_ptr()
        a.n_free = int(w.free_slots.size)
        a.slot_pool = self.pool.data_ptr()
        a.n_slots = w.n_slots
        a.stats = self.stats.data_ptr()
        a.sm_scale = w.sm_scale
        a.out = self.out.data_ptr()
        a.lse = self.lse.data_ptr()
        a.dev_status = self.dev_status.data_ptr()
        a.ws = self.ws.data_ptr()
        a.ws_bytes = self.ws_bytes
        a.release_previous = 1 if release_previous else 0
        return a

    def decode_layer(self, stream=None, release_previous=False):
        """pulse_decode_layer; release_previous: first undo the previous layer-step's recall
        (in the scoring kernel) instead of a separate release()."""
        P.pulse_decode_layer(self.layer_args(release_previous=release_previous), stream=stream)

    def release(self, chained=True, stream=None):
        """Step-end release of the last recall (pulse_release_recalled): table and free
        head return to their state before it.  chained: the recall came from
        decode_layer (else from recall() / the engine)."""
        w = self.w
        P.pulse_release_recalled(self.shape, w.B, self.k_max, w.total_blocks if chained else 0, self.table,
                                 w.max_blocks, self.free_head, self.stats, self.dev_status, self.ws, self.ws_bytes,
                                 stream=stream)

    def select(self, scores: Optional[torch.Tensor] = None, stream=None):
        w = self.w
        P.pulse_select_solohead(self.shape, self.q, self.digests, self.blk_off, w.B, w.total_blocks, w.solo_kv_head,
                                self.k_mid, w.n_sink, w.n_local, self.k_max, self.sel_idx, self.sel_cnt, scores,
                                self.dev_status, self.ws, self.ws_bytes, stream=stream)

    def recall(self, stream=None):
        w = self.w
        P.pulse_recall_gather(self.shape, self.host_ptr, self.blk_off, w.B, self.sel_idx, self.sel_cnt, self.k_max,
                              self.table, w.max_blocks, self.free_slots, self.free_head, int(w.free_slots.size),
                              self.pool, w.n_slots, self.stats, self.dev_status, self.ws, self.ws_bytes,
                              stream=stream)

    def recall_gs(self, engine, stream=None, wait=True, timeout_ms=20000):
        """Recall through the CPU-gather / one-DMA / GPU-scatter engine (the paper's path)."""
        w = self.w
        seq = engine.submit(self.host_ptr, self.blk_off, w.B, self.sel_idx, self.sel_cnt, self.k_max, self.table,
                            w.max_blocks, self.free_slots, self.free_head, int(w.free_slots.size), self.pool,
                            w.n_slots, self.stats, self.dev_status, self.ws, self.ws_bytes, stream=stream)
        if wait:
            engine.wait(seq, timeout_ms)
        return seq

    def attention(self, stream=None):
        w = self.w
        P.pulse_sparse_decode_attn(self.shape, self.q, self.pool, w.n_slots, self.table, w.max_blocks, self.sel_idx,
                                   self.sel_cnt, self.k_max, self.ctx_len, w.B, w.sm_scale, self.out, self.lse,
                                   self.dev_status, self.ws, self.ws_bytes, stream=stream)

    def all_head_digests(self, stream=None) -> torch.Tensor:
        """Digests of every KV head, [Hkv][total_blocks][2][d] (built once)."""
        w = self.w
        if getattr(self, "head_digests", None) is None:
            self.head_digests = torch.zeros((w.Hkv, max(w.total_blocks, 1), 2, w.d), dtype=torch.int16,
                                            device=self.device)
            for h in range(w.Hkv):
                self.build_digests(h, out=self.head_digests[h], stream=stream)
        return self.head_digests

    def select_average(self, scores: Optional[torch.Tensor] = None, stream=None):
        """Average selection (all heads' scores averaged) into this step's sel_idx / sel_cnt."""
        w = self.w
        hd = self.all_head_digests(stream)
        nb = P.pulse_average_workspace_bytes(self.shape, w.B, self.k_max, w.total_blocks)
        ws = torch.zeros(max(nb, 1), dtype=torch.uint8, device=self.device)
        P.pulse_select_average(self.shape, self.q, hd, self.blk_off, w.B, w.total_blocks, self.k_mid, w.n_sink,
                               w.n_local, self.k_max, self.sel_idx, self.sel_cnt, scores, self.dev_status, ws, nb,
                               stream=stream)
        return ws

    def mam(self, stream=None) -> torch.Tensor:
        """Middle Attention Mass of every (request, KV head), [B][Hkv], over the whole context:
        every block is placed in a dense device pool for the calibration."""
        w = self.w
        dev = self.device
        pool = _dev(w.kv, dev) if w.total_blocks else torch.zeros((1, w.elems_per_block), dtype=torch.int16,
                                                                 device=dev)  # slot b = global block b
        table = np.full((w.B, w.max_blocks), -1, np.int32)
        for r in range(w.B):
            n = int(w.n_blocks[r])
            table[r, :n] = np.arange(int(w.blk_off[r]), int(w.blk_off[r]) + n, dtype=np.int32)
        table_t = _dev(table, dev)
        out = torch.zeros((w.B, w.Hkv), dtype=torch.float32, device=dev)
        nb = P.pulse_mam_workspace_bytes(self.shape, w.B, w.max_blocks)
        ws = torch.zeros(max(nb, 1), dtype=torch.uint8, device=dev)
        P.pulse_mam(self.shape, self.q, pool, max(w.total_blocks, 1), table_t, w.max_blocks, self.ctx_len, w.B,
                    w.n_sink, w.n_local, w.sm_scale, out, self.dev_status, ws, nb, stream=stream)
        torch.cuda.synchronize()  # the temporary pool, table and workspace are freed on return
        return out

    def headwise(self, stream=None):
        """Headwise selection of every KV head with its own digests against this step's
        table (nothing is recalled).  Returns (sel_idx, sel_cnt, miss_cnt, run_cnt) tensors."""
        w = self.w
        H = w.Hkv
        self.all_head_digests(stream)
        dev = self.device
        sel_idx = torch.full((H, w.B, self.k_max), -1, dtype=torch.int32, device=dev)
        sel_cnt = torch.zeros((H, w.B), dtype=torch.int32, device=dev)
        miss = torch.zeros((H, w.B), dtype=torch.int32, device=dev)
        runs = torch.zeros((H, w.B), dtype=torch.int32, device=dev)
        nb = P.pulse_headwise_workspace_bytes(self.shape, w.B, self.k_max, w.total_blocks)
        ws = torch.zeros(max(nb, 1), dtype=torch.uint8, device=dev)
        P.pulse_select_headwise(self.shape, self.q, self.head_digests, self.blk_off, w.B, w.total_blocks, self.k_mid,
                                w.n_sink, w.n_local, self.k_max, self.table, w.max_blocks, w.n_slots, sel_idx, sel_cnt,
                                miss, runs, self.dev_status, ws, nb, stream=stream)
        return sel_idx, sel_cnt, miss, runs

    # ------------------------------------------------------------------ readback
    def status(self) -> int:
        return int(self.dev_status.item())

    def recall_stats(self):
        s = self.stats.cpu().numpy()
        n_missing = int(s[0] & 0xFFFFFFFF)
        n_runs = int((s[0] >> 32) & 0xFFFFFFFF)
        return n_missing, n_runs, int(s[1])

    def selection(self):
        return self.sel_idx.cpu().numpy(), self.sel_cnt.cpu().numpy()

    def table_np(self):
        return self.table.cpu().numpy()

    def pool_np(self) -> np.ndarray:
        return self.pool.cpu().numpy().view(np.uint16)


class MultiLayerStep:
    """A decode step over many layers (preset 4): one LayerState per layer; layers
    share ``n_stores`` pinned host stores.  ``run_chained`` issues one
    pulse_decode_layer per layer on one stream.  ``run_overlapped`` keeps only the
    recalls on an I/O stream: selection of layer l+1 and attention of layer l run on a
    compute stream while layer l+1's blocks cross the host link (the queries of every
    layer are given up front)."""

    def __init__(self, n_layers: int = 32, n_stores: int = 4, device="cuda", **preset_kw):
        from . import workloads as W

        self.layers = []
        self.stores = {}
        for layer in range(n_layers):
            spec, seed = W.preset(4, layer=layer, n_stores=n_stores, **preset_kw)
            sid = layer % n_stores
            if sid not in self.stores:
                holder = []
                w = W.generate(spec, seed, kv_alloc=pinned_allocator(holder))
                self.stores[sid] = (w, holder)
            else:
                w = W.generate(spec, seed, reuse_kv=self.stores[sid][0])
            self.layers.append(LayerState(w, self.stores[sid][1][0].ptr, device=device))
        self.io_stream = torch.cuda.Stream()
        self.cmp_stream = torch.cuda.Stream()
        self.selected = [torch.cuda.Event() for _ in self.layers]
        self.recalled = [torch.cuda.Event() for _ in self.layers]

    def reset(self):
        for st in self.layers:
            st.reset()

    def run_chained(self, stream=None, release_previous=False):
        """One pulse_decode_layer per layer on one stream; release_previous: each layer first
        undoes its previous step's recall (the hot set stays fixed-size)."""
        for st in self.layers:
            st.decode_layer(stream=stream, release_previous=release_previous)

    def run_overlapped(self, recall_events=None, release=False):
        """The two-stream step.  recall_events: optional per-layer (start, end) timing events
        (or None) recorded around that layer's recall copy on the I/O stream.  release: after
        each layer's attention, release its recall on the compute stream (the step-end
        release; it overlaps the next recalls)."""
        cur = torch.cuda.current_stream()
        io, cmp_ = self.io_stream, self.cmp_stream
        io.wait_stream(cur)
        cmp_.wait_stream(cur)
        n = len(self.layers)
        self.layers[0].select(stream=cmp_)
        self.selected[0].record(cmp_)
        for i, st in enumerate(self.layers):
            io.wait_event(self.selected[i])
            ev = recall_events[i] if recall_events is not None else None
            if ev is not None:
                ev[0].record(io)
            st.recall(stream=io)
            if ev is not None:
                ev[1].record(io)
            self.recalled[i].record(io)
            if i + 1 < n:  # next layer's selection while this layer's blocks cross the link
                self.layers[i + 1].select(stream=cmp_)
                self.selected[i + 1].record(cmp_)
            cmp_.wait_event(self.recalled[i])
            st.attention(stream=cmp_)
            if release:
                st.release(chained=False, stream=cmp_)
        cur.wait_stream(io)
        cur.wait_stream(cmp_)

    def run_irq(self, sched, normal=None, mode="semi_sync", async_ahead=4, engine=None):
        """One step under the interruptible layer-wise scheduler (pulse_irq_step) with an
        optional NormalBatch and gather-scatter engine; returns (stats dict, per-layer
        overlap depths)."""
        torch.cuda.current_stream().synchronize()  # table restores done before the scheduler's streams start
        args = [st.layer_args() for st in self.layers]
        return sched.step(args, normal.layers if normal is not None else [], mode=mode, async_ahead=async_ahead,
                          engine=engine)


class NormalBatch:
    """A normal batch (Sec. 4.2): B requests whose KV cache is resident in HBM, over
    n_layers layers, each with its own KV pool and SwiGLU FFN weights (seeded random
    bf16).  ``layers`` holds the pulse_normal_layer structs of the layer scheduler."""

    def __init__(self, B: int, ctx: int, n_layers: int, Hq=32, Hkv=8, d=128, bs=16, d_ff=14336, seed=0,
                 device="cuda"):
        dev = torch.device(device)
        self.B, self.ctx, self.n_layers, self.d_ff = B, ctx, n_layers, d_ff
        self.shape = P.make_shape(Hq, Hkv, d, bs, P_BF16)
        n = -(-ctx // bs)
        self.n_blocks = n
        E = 2 * Hkv * bs * d
        D = Hq * d
        g = torch.Generator(device=dev)
        g.manual_seed(seed)
        self.table = torch.arange(B * n, dtype=torch.int32, device=dev).reshape(B, n)
        self.sel_idx = torch.arange(n, dtype=torch.int32, device=dev).repeat(B, 1).contiguous()
        self.sel_cnt = torch.full((B,), n, dtype=torch.int32, device=dev)
        self.ctx_len = torch.full((B,), ctx, dtype=torch.int32, device=dev)
        self.dev_status = torch.zeros(1, dtype=torch.int32, device=dev)
        self.ws_bytes = P.pulse_workspace_bytes(self.shape, B, n, 0)
        self.bufs = []
        self.layers = []
        for _ in range(n_layers):
            b = {
                "pool": torch.randn((B * n, E), generator=g, device=dev, dtype=torch.bfloat16).view(torch.int16),
                "q": torch.randn((B, Hq, d), generator=g, device=dev, dtype=torch.bfloat16),
                "w_gu": (torch.randn((2 * d_ff, D), generator=g, device=dev, dtype=torch.bfloat16) * 0.02),
                "w_down": (torch.randn((D, d_ff), generator=g, device=dev, dtype=torch.bfloat16) * 0.02),
                "out": torch.zeros((B, Hq, d), dtype=torch.float32, device=dev),
                "lse": torch.zeros((B, Hq), dtype=torch.float32, device=dev),
                "ws": torch.zeros(max(self.ws_bytes, 1), dtype=torch.uint8, device=dev),
                "x": torch.zeros((B, D), dtype=torch.bfloat16, device=dev),
                "gu": torch.zeros((B, 2 * d_ff), dtype=torch.bfloat16, device=dev),
                "h": torch.zeros((B, d_ff), dtype=torch.bfloat16, device=dev),
                "y": torch.zeros((B, D), dtype=torch.bfloat16, device=dev),
            }
            self.bufs.append(b)
            L = P.pulse_normal_layer()
            L.shape = self.shape
            L.B = B
            L.q = b["q"].data_ptr()
            L.slot_pool = b["pool"].data_ptr()
            L.n_slots = B * n
            L.block_table = self.table.data_ptr()
            L.max_blocks = n
            L.sel_idx = self.sel_idx.data_ptr()
            L.sel_cnt = self.sel_cnt.data_ptr()
            L.k_max = n
            L.ctx_len = self.ctx_len.data_ptr()
            L.sm_scale = 1.0 / math.sqrt(d)
            L.out = b["out"].data_ptr()
            L.lse = b["lse"].data_ptr()
            L.ws = b["ws"].data_ptr()
            L.ws_bytes = self.ws_bytes
            L.d_ff = d_ff
            L.w_gate_up = b["w_gu"].data_ptr()
            L.w_down = b["w_down"].data_ptr()
            L.x = b["x"].data_ptr()
            L.gu = b["gu"].data_ptr()
            L.h = b["h"].data_ptr()
            L.y = b["y"].data_ptr()
            L.dev_status = self.dev_status.data_ptr()
            self.layers.append(L)

    def status(self) -> int:
        return int(self.dev_status.item())
