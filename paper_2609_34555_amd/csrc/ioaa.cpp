// ioaa.cpp -- IO-Adaptive Offloading Admission (Sec. 4.3), host C++.
//
// Chooses, for the waiting requests of a decode-step boundary, which join the
// normal batch (KV cache fully on the GPU) and which are offloaded (hot budget
// on the GPU, the rest recalled per layer), maximising the throughput model of
// Eq. 1:  thr = m/(m+1) * B_n + 1/(m+1) * B_o,  with the overlap depth m
// interpolated from an offline (B_o, B_n) profile (Sec. 4.3.2).
//
// Search (Sec. 4.3.1): a depth-first walk of the binary tree whose level t
// decides the t-th longest request (normal branch first, then offload).  Two
// prunes: a branch that exceeds the GPU memory budget is cut, and length
// monotonicity (no offload admission below a normal-batch one).  A request
// that fits neither batch ends the path (it and all shorter ones keep
// waiting); Eq. 1 is evaluated where a path ends.
#include <algorithm>
#include <cmath>
#include <numeric>
#include <vector>

#include "../../include/pulse.h"

namespace {

struct Search {
    const pulse_ioaa_params* p;
    std::vector<int64_t> len;  // sorted longest first
    std::vector<int8_t> cur, best;
    double best_thr = -1.0;
    int64_t nodes = 0;   // tree nodes visited
    int64_t leaves = 0;  // complete assignments at which Eq. 1 is evaluated

    double depth(double b_o, double b_n) const { return pulse_overlap_depth(p, b_o, b_n); }

    double thr(int64_t b_n, int64_t b_o) const {
        if (b_o == 0) return (double)b_n;  // no offload batch: the normal batch runs alone
        const double m = depth((double)b_o, (double)b_n);
        return m / (m + 1.0) * (double)b_n + 1.0 / (m + 1.0) * (double)b_o;
    }

    void leaf(int64_t nn, int64_t no) {
        ++leaves;
        const double t = thr(p->running_normal + nn, p->running_offload + no);
        if (t > best_thr) {
            best_thr = t;
            best = cur;
        }
    }

    void dfs(size_t i, int64_t mem, int64_t nn, int64_t no, bool any_normal) {
        ++nodes;
        if (i == len.size()) {
            leaf(nn, no);
            return;
        }
        const int64_t cost_n = len[i] * p->kv_bytes_per_token;
        const int64_t cost_o = p->offload_tokens * p->kv_bytes_per_token + p->offload_extra_bytes;
        const bool can_n = mem + cost_n <= p->gpu_budget_bytes;
        const bool can_o = !any_normal && mem + cost_o <= p->gpu_budget_bytes;
        if (!can_n && !can_o) {  // this request and all shorter ones keep waiting
            leaf(nn, no);
            return;
        }
        if (can_n) {
            cur[i] = 1;
            dfs(i + 1, mem + cost_n, nn + 1, no, true);
        }
        if (can_o) {
            cur[i] = 2;
            dfs(i + 1, mem + cost_o, nn, no + 1, any_normal);
        }
        cur[i] = 0;
    }
};

}  // namespace

extern "C" {

double pulse_overlap_depth(const pulse_ioaa_params* p, double b_o, double b_n) {
    if (!p || !p->grid_bo || !p->grid_bn || !p->grid_m || p->n_bo < 1 || p->n_bn < 1) return NAN;
    const double* bo = p->grid_bo;
    const double* bn = p->grid_bn;
    const int nbo = p->n_bo, nbn = p->n_bn;
    const double x = std::min(std::max(b_o, bo[0]), bo[nbo - 1]);
    const double y = std::min(std::max(b_n, bn[0]), bn[nbn - 1]);
    auto cell = [](const double* g, int n, double v) {
        int i = (int)(std::upper_bound(g, g + n, v) - g) - 1;
        return std::max(0, std::min(i, n - 2));
    };
    auto M = [&](int i, int j) { return p->grid_m[(size_t)i * nbn + j]; };
    if (nbo == 1 && nbn == 1) return M(0, 0);
    if (nbo == 1) {
        const int j = cell(bn, nbn, y);
        const double ty = (y - bn[j]) / (bn[j + 1] - bn[j]);
        return M(0, j) * (1 - ty) + M(0, j + 1) * ty;
    }
    if (nbn == 1) {
        const int i = cell(bo, nbo, x);
        const double tx = (x - bo[i]) / (bo[i + 1] - bo[i]);
        return M(i, 0) * (1 - tx) + M(i + 1, 0) * tx;
    }
    const int i = cell(bo, nbo, x), j = cell(bn, nbn, y);
    const double tx = (x - bo[i]) / (bo[i + 1] - bo[i]);
    const double ty = (y - bn[j]) / (bn[j + 1] - bn[j]);
    return M(i, j) * (1 - tx) * (1 - ty) + M(i + 1, j) * tx * (1 - ty) + M(i, j + 1) * (1 - tx) * ty +
           M(i + 1, j + 1) * tx * ty;
}

pulse_status pulse_ioaa_plan(const pulse_ioaa_params* p, const int64_t* lengths, int32_t n, int8_t* assign,
                             double* throughput, int64_t* nodes_visited, int64_t* leaves_evaluated) {
    if (!p || n < 0 || (n > 0 && (!lengths || !assign)) || !throughput) return PULSE_ERR_INVALID_ARG;
    if (!p->grid_bo || !p->grid_bn || !p->grid_m || p->n_bo < 1 || p->n_bn < 1) return PULSE_ERR_INVALID_ARG;
    for (int i = 1; i < p->n_bo; ++i)
        if (!(p->grid_bo[i] > p->grid_bo[i - 1])) return PULSE_ERR_INVALID_ARG;
    for (int i = 1; i < p->n_bn; ++i)
        if (!(p->grid_bn[i] > p->grid_bn[i - 1])) return PULSE_ERR_INVALID_ARG;
    if (p->kv_bytes_per_token < 0 || p->offload_tokens < 0 || p->offload_extra_bytes < 0) return PULSE_ERR_INVALID_ARG;
    for (int i = 0; i < n; ++i)
        if (lengths[i] < 0) return PULSE_ERR_INVALID_ARG;
    std::vector<int32_t> order(n);
    std::iota(order.begin(), order.end(), 0);
    std::stable_sort(order.begin(), order.end(), [&](int32_t a, int32_t b) { return lengths[a] > lengths[b]; });
    Search s;
    s.p = p;
    s.len.resize(n);
    for (int i = 0; i < n; ++i) s.len[i] = lengths[order[i]];
    s.cur.assign(n, 0);
    s.best.assign(n, 0);
    s.dfs(0, 0, 0, 0, false);
    for (int i = 0; i < n; ++i) assign[order[i]] = s.best[i];
    *throughput = s.best_thr;
    if (nodes_visited) *nodes_visited = s.nodes;
    if (leaves_evaluated) *leaves_evaluated = s.leaves;
    return PULSE_OK;
}

}  // extern "C"
