"""ctypes wrapper of the CPU oracle (oracle/pulse_oracle.c).

TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT: only the test-suite, the smoke
check and the benchmark's CPU-baseline leg may import this module.  It never
imports the GPU package and the GPU package never imports it.

Every array is numpy; 16-bit KV/query values are passed as their uint16 bit
patterns with a dtype code (0 = fp16, 1 = bf16).  Each function names the
passage of the paper it follows; the C source states the readings taken where
the paper is silent.
"""
import ctypes
import os

import numpy as np

from . import build as _build

F16 = 0
BF16 = 1
OK = 0
ERR_INVALID_ARG = 1
ERR_POOL_EXHAUSTED = 4
ERR_SELECT_OVERFLOW = 5
ERR_BAD_INDEX = 7

_lib = None


def _load():
    global _lib
    if _lib is None:
        path = os.environ.get("PULSE_ORACLE_LIB")  # another build of pulse_oracle.c (sanitizer runs)
        if not path:
            if not os.path.exists(_build.LIB):
                _build.build_oracle()
            path = _build.LIB
        lib = ctypes.CDLL(path)
        P = ctypes.c_void_p
        I = ctypes.c_int
        lib.or_decode.restype = ctypes.c_double
        lib.or_decode.argtypes = [ctypes.c_uint16, I]
        lib.or_build_digests.argtypes = [P, P, P, I, I, I, I, I, I, P]
        lib.or_score.argtypes = [P, P, P, I, I, I, I, I, I, P]
        lib.or_select.argtypes = [P, P, I, P, I, I, I, P, P]
        lib.or_recall.argtypes = [P, P, I, P, P, I, P, I, P, P, I, P, I, ctypes.c_int64, P]
        lib.or_attention.argtypes = [P, P, I, P, I, P, P, I, P, P, I, I, I, I, I, I,
                                     ctypes.c_double, P, P]
        lib.or_dense_attention.argtypes = [P, P, P, P, I, I, I, I, I, I, ctypes.c_double, P, P]
        lib.or_mam.argtypes = [P, P, P, P, I, I, I, I, I, I, ctypes.c_double, I, I, P, P]
        for name in ("or_build_digests", "or_score", "or_select", "or_recall", "or_attention",
                     "or_dense_attention", "or_mam"):
            getattr(lib, name).restype = I
        _lib = lib
    return _lib


def _p(a):
    return a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dt):
    """Contiguous array of exactly dtype dt (no silent conversion of values)."""
    a = np.asarray(a)
    if a.dtype != np.dtype(dt):
        raise TypeError(f"expected {np.dtype(dt)}, got {a.dtype}")
    return np.ascontiguousarray(a)


def decode(bits, dtype):
    """Widen 16-bit patterns to float64 exactly (elementwise)."""
    lib = _load()
    flat = np.asarray(bits, dtype=np.uint16).ravel()
    out = np.fromiter((lib.or_decode(int(b), dtype) for b in flat), dtype=np.float64, count=flat.size)
    return out.reshape(np.shape(bits))


def build_digests(kv, blk_off, ctx_len, Hkv, bs, d, dtype, kv_head):
    """Per-block min/max key digest of one KV head (Sec. 2.1, Sec. 4.4.1).

    kv: uint16 [total_blocks, 2*Hkv*bs*d]; returns uint16 [total_blocks, 2, d]."""
    kv = _c(kv, np.uint16)
    blk_off = _c(blk_off, np.int64)
    ctx_len = _c(ctx_len, np.int32)
    B = ctx_len.shape[0]
    total = int(blk_off[-1])
    out = np.zeros((total, 2, d), np.uint16)
    rc = _load().or_build_digests(_p(kv), _p(blk_off), _p(ctx_len), B, Hkv, bs, d, dtype, kv_head, _p(out))
    if rc:
        raise ValueError(f"or_build_digests failed: {rc}")
    return out


def score(q, digests, blk_off, Hq, Hkv, d, dtype, solo_kv_head):
    """fp64 query-digest score of every block for the solo head (Sec. 4.4.1)."""
    q = _c(q, np.uint16)
    digests = _c(digests, np.uint16)
    blk_off = _c(blk_off, np.int64)
    B = blk_off.shape[0] - 1
    out = np.zeros(int(blk_off[-1]), np.float64)
    rc = _load().or_score(_p(q), _p(digests), _p(blk_off), B, Hq, Hkv, d, dtype, solo_kv_head, _p(out))
    if rc:
        raise ValueError(f"or_score failed: {rc}")
    return out


def select(scores, blk_off, k_mid, n_sink, n_local, k_max):
    """SoloHead top-k with forced sink/local blocks (Sec. 4.4.1, Sec. 5 setup).

    Returns (status, sel_idx int32 [B, k_max] padded with -1, sel_cnt int32 [B])."""
    scores = _c(scores, np.float64)
    blk_off = _c(blk_off, np.int64)
    k_mid = _c(k_mid, np.int32)
    B = blk_off.shape[0] - 1
    sel_idx = np.full((B, k_max), -1, np.int32)
    sel_cnt = np.zeros(B, np.int32)
    rc = _load().or_select(_p(scores), _p(blk_off), B, _p(k_mid), n_sink, n_local, k_max, _p(sel_idx),
                           _p(sel_cnt))
    return rc, sel_idx, sel_cnt


def recall(host_kv_bytes, blk_off, sel_idx, sel_cnt, table, free_slots, free_head, pool_bytes,
           unit_bytes):
    """Set difference, slot allocation and copy of the missing blocks (Sec. 2.2, Sec. 4.4.2).

    table (int32 [B, max_blocks]) and pool_bytes (uint8 [n_slots, unit_bytes]) are updated
    in place.  Returns (status, new_free_head, stats=(n_missing, n_runs, bytes))."""
    host_kv_bytes = _c(host_kv_bytes, np.uint8)
    blk_off = _c(blk_off, np.int64)
    sel_idx = _c(sel_idx, np.int32)
    sel_cnt = _c(sel_cnt, np.int32)
    free_slots = _c(free_slots, np.int32)
    if table.dtype != np.int32 or not table.flags.c_contiguous:
        raise TypeError("table must be C-contiguous int32")
    if pool_bytes.dtype != np.uint8 or not pool_bytes.flags.c_contiguous:
        raise TypeError("pool must be C-contiguous uint8")
    B = blk_off.shape[0] - 1
    k_max = sel_idx.shape[1]
    max_blocks = table.shape[1]
    n_slots = pool_bytes.shape[0]
    fh = np.array([free_head], np.int32)
    stats = np.zeros(3, np.int64)
    rc = _load().or_recall(_p(host_kv_bytes), _p(blk_off), B, _p(sel_idx), _p(sel_cnt), k_max, _p(table),
                           max_blocks, _p(free_slots), _p(fh), free_slots.shape[0], _p(pool_bytes), n_slots,
                           unit_bytes, _p(stats))
    return rc, int(fh[0]), tuple(int(x) for x in stats)


def attention(q, pool, table, sel_idx, sel_cnt, blk_off, ctx_len, Hq, Hkv, bs, d, dtype, sm_scale):
    """fp64 sparse GQA decode attention over the selected blocks (Sec. 2.2).

    pool: uint16 [n_slots, 2*Hkv*bs*d].  Returns (out float64 [B, Hq, d], lse float64 [B, Hq])."""
    q = _c(q, np.uint16)
    pool = _c(pool, np.uint16)
    table = _c(table, np.int32)
    sel_idx = _c(sel_idx, np.int32)
    sel_cnt = _c(sel_cnt, np.int32)
    blk_off = _c(blk_off, np.int64)
    ctx_len = _c(ctx_len, np.int32)
    B = ctx_len.shape[0]
    out = np.zeros((B, Hq, d), np.float64)
    lse = np.zeros((B, Hq), np.float64)
    rc = _load().or_attention(_p(q), _p(pool), pool.shape[0], _p(table), table.shape[1], _p(sel_idx),
                              _p(sel_cnt), sel_idx.shape[1], _p(blk_off), _p(ctx_len), B, Hq, Hkv, bs, d,
                              dtype, float(sm_scale), _p(out), _p(lse))
    if rc:
        raise ValueError(f"or_attention failed: {rc}")
    return out, lse


def dense_attention(q, host_kv, blk_off, ctx_len, Hq, Hkv, bs, d, dtype, sm_scale):
    """fp64 attention over every context token, read from the host store."""
    q = _c(q, np.uint16)
    host_kv = _c(host_kv, np.uint16)
    blk_off = _c(blk_off, np.int64)
    ctx_len = _c(ctx_len, np.int32)
    B = ctx_len.shape[0]
    out = np.zeros((B, Hq, d), np.float64)
    lse = np.zeros((B, Hq), np.float64)
    rc = _load().or_dense_attention(_p(q), _p(host_kv), _p(blk_off), _p(ctx_len), B, Hq, Hkv, bs, d, dtype,
                                    float(sm_scale), _p(out), _p(lse))
    if rc:
        raise ValueError(f"or_dense_attention failed: {rc}")
    return out, lse


def mam(q, host_kv, blk_off, ctx_len, r, Hq, Hkv, bs, d, dtype, sm_scale, n_sink_tok=16,
        n_local_tok=128):
    """Middle Attention Mass, Eq. 2, of request r; returns (best_kv_head, mam_q, mam_h).
    The middle excludes the first n_sink_tok and last n_local_tok tokens (R13: the tests
    pass the token counts of the sink and local blocks)."""
    q = _c(q, np.uint16)
    host_kv = _c(host_kv, np.uint16)
    blk_off = _c(blk_off, np.int64)
    ctx_len = _c(ctx_len, np.int32)
    mam_q = np.zeros(Hq, np.float64)
    mam_h = np.zeros(Hkv, np.float64)
    best = _load().or_mam(_p(q), _p(host_kv), _p(blk_off), _p(ctx_len), r, Hq, Hkv, bs, d, dtype,
                          float(sm_scale), n_sink_tok, n_local_tok, _p(mam_q), _p(mam_h))
    return best, mam_q, mam_h


def missing_counts(sel_idx, sel_cnt, table):
    """Set difference of a selection against the block table (Sec. 2.2): per request the
    number of selected blocks whose entry is -1, and the number of maximal runs of
    consecutive missing block indices.  Returns (units int64 [B], runs int64 [B])."""
    B = sel_cnt.shape[0]
    units = np.zeros(B, np.int64)
    runs = np.zeros(B, np.int64)
    for r in range(B):
        prev = -2
        for j in sel_idx[r, : sel_cnt[r]]:
            if table[r, j] < 0:
                units[r] += 1
                if j != prev + 1:
                    runs[r] += 1
                prev = j
    return units, runs


def average_scores(kv, q, blk_off, ctx_len, Hq, Hkv, bs, d, dtype):
    """The "average" strategy of Sec. 4.4.1: every KV head scores every block with its
    own digests (Sec. 4.4.1 with R1, R2), and (R14) the fp64 scores are averaged over the KV
    heads -- the mean over all query heads.  Returns fp64 [total_blocks]; selection on it
    is select() (R3: the decision is taken on the average rounded once to fp32)."""
    total = int(blk_off[-1])
    acc = np.zeros(total, np.float64)
    for h in range(Hkv):
        dig = build_digests(kv, blk_off, ctx_len, Hkv, bs, d, dtype, h)
        acc += score(q, dig, blk_off, Hq, Hkv, d, dtype, h)
    return acc / Hkv


def headwise_select(kv, q, blk_off, ctx_len, Hq, Hkv, bs, d, dtype, k_mid, n_sink, n_local, k_max):
    """Headwise selection baseline (Sec. 3.4; Sec. 4.4.1 'headwise'): every KV head selects
    its own blocks with its own digests.  Returns per-head (sel_idx [Hkv,B,k_max],
    sel_cnt [Hkv,B], scores [Hkv,total_blocks])."""
    B = ctx_len.shape[0]
    total = int(blk_off[-1])
    sel = np.full((Hkv, B, k_max), -1, np.int32)
    cnt = np.zeros((Hkv, B), np.int32)
    sc = np.zeros((Hkv, total), np.float64)
    for h in range(Hkv):
        dig = build_digests(kv, blk_off, ctx_len, Hkv, bs, d, dtype, h)
        sc[h] = score(q, dig, blk_off, Hq, Hkv, d, dtype, h)
        rc, sel[h], cnt[h] = select(sc[h], blk_off, k_mid, n_sink, n_local, k_max)
        if rc:
            raise ValueError(f"select failed: {rc}")
    return sel, cnt, sc
