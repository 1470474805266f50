"""Oracle of IO-Adaptive Offloading Admission (Sec. 4.3): exhaustive search.

TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT (see oracle/__init__.py).

Definitions followed:
  - Eq. 1: throughput is proportional to m/(m+1) * B_n + 1/(m+1) * B_o, with m the
    overlap depth, B_n / B_o the normal / offload batch sizes (Sec. 4.3);
  - the overlap depth is profiled offline on a grid of (B_o, B_n) and interpolated
    from the nearest profiled points (Sec. 4.3.2);
  - each waiting request is admitted to the normal batch or offloaded; branches over
    the GPU memory budget are infeasible; length monotonicity: after the longest
    normal-batch admission on a path, no shorter request goes to the offload batch
    (Sec. 4.3.1).
Readings taken where the paper is silent:
  I1  requests are decided longest first; when a request fits neither batch, it and
      every later request keep waiting (the search stops on that path);
  I2  with no offload request at all, throughput is B_n (Eq. 1 describes the
      interleaved schedule, which needs an offload batch);
  I3  interpolation is bilinear on the grid, clamped at its edges;
  I4  a normal request holds its whole KV cache on the GPU; an offloaded one holds its
      hot budget of tokens plus a fixed per-request extra (digests).
This oracle enumerates every admissible assignment; it shares nothing with the
library's pruned depth-first search.
"""
import itertools

import numpy as np


def overlap_depth(grid_bo, grid_bn, grid_m, b_o, b_n):
    """Bilinear interpolation of the profiled overlap depth, clamped at the edges (I3)."""
    bo = np.asarray(grid_bo, float)
    bn = np.asarray(grid_bn, float)
    m = np.asarray(grid_m, float).reshape(bo.size, bn.size)
    x = min(max(b_o, bo[0]), bo[-1])
    y = min(max(b_n, bn[0]), bn[-1])
    i = max(0, min(int(np.searchsorted(bo, x, side="right")) - 1, bo.size - 2)) if bo.size > 1 else 0
    j = max(0, min(int(np.searchsorted(bn, y, side="right")) - 1, bn.size - 2)) if bn.size > 1 else 0
    if bo.size == 1 and bn.size == 1:
        return float(m[0, 0])
    if bo.size == 1:
        ty = (y - bn[j]) / (bn[j + 1] - bn[j])
        return float(m[0, j] * (1 - ty) + m[0, j + 1] * ty)
    if bn.size == 1:
        tx = (x - bo[i]) / (bo[i + 1] - bo[i])
        return float(m[i, 0] * (1 - tx) + m[i + 1, 0] * tx)
    tx = (x - bo[i]) / (bo[i + 1] - bo[i])
    ty = (y - bn[j]) / (bn[j + 1] - bn[j])
    return float(m[i, j] * (1 - tx) * (1 - ty) + m[i + 1, j] * tx * (1 - ty) + m[i, j + 1] * (1 - tx) * ty
                 + m[i + 1, j + 1] * tx * ty)


def throughput(b_n, b_o, m):
    """Eq. 1 (up to its constant of proportionality); I2 when there is no offload batch."""
    if b_o == 0:
        return float(b_n)
    return m / (m + 1.0) * b_n + 1.0 / (m + 1.0) * b_o


def admissible(lengths, budget, kv_bytes_per_token, offload_tokens, offload_extra):
    """Every admissible assignment, as (order, choice): the first len(choice) requests of
    `order` (longest first) are decided (1 normal, 2 offload), the rest wait.  Admissible:
    within the memory budget, no offload after a longer normal request (Sec. 4.3.1), and
    waiting only where the next request fits neither batch (I1)."""
    n = len(lengths)
    order = sorted(range(n), key=lambda i: (-lengths[i], i))
    for k in range(n + 1):  # the first k requests (longest first) are decided, the rest wait
        for choice in itertools.product((1, 2), repeat=k):
            if any(choice[t] == 2 and 1 in choice[:t] for t in range(k)):
                continue  # monotonicity: no offload after a longer normal request
            mem, ok = 0, True
            for t in range(k):
                L = lengths[order[t]]
                mem += L * kv_bytes_per_token if choice[t] == 1 else offload_tokens * kv_bytes_per_token + offload_extra
                if mem > budget:
                    ok = False
                    break
            if not ok:
                continue
            if k < n:  # I1: waiting only when the next request fits neither batch
                L = lengths[order[k]]
                cost_n = mem + L * kv_bytes_per_token
                cost_o = mem + offload_tokens * kv_bytes_per_token + offload_extra
                can_n = cost_n <= budget
                can_o = cost_o <= budget and 1 not in choice
                if can_n or can_o:
                    continue
            yield order, choice


def count_admissible(lengths, budget, kv_bytes_per_token, offload_tokens, offload_extra):
    """Number of admissible assignments: the complete assignments at which a search over
    the pruned tree evaluates Eq. 1."""
    return sum(1 for _ in admissible(lengths, budget, kv_bytes_per_token, offload_tokens, offload_extra))


def best_assignment(lengths, budget, kv_bytes_per_token, offload_tokens, offload_extra, run_n, run_o, grid_bo,
                    grid_bn, grid_m):
    """Enumerate every admissible assignment; returns (assign [n] in {0 wait, 1 normal,
    2 offload}, throughput).  Ties keep the assignment with the most normal admissions,
    then the most offloads (any maximiser is accepted by the tests when values tie)."""
    n = len(lengths)
    best, best_thr = None, -1.0
    for order, choice in admissible(lengths, budget, kv_bytes_per_token, offload_tokens, offload_extra):
        b_n = run_n + sum(1 for c in choice if c == 1)
        b_o = run_o + sum(1 for c in choice if c == 2)
        thr = throughput(b_n, b_o, overlap_depth(grid_bo, grid_bn, grid_m, b_o, b_n))
        if thr > best_thr:
            best_thr = thr
            best = [0] * n
            for t in range(len(choice)):
                best[order[t]] = choice[t]
    return best, best_thr
