// recall.hip -- set difference, slot allocation and the gather-scatter
// recall of missing KV blocks from pinned host DRAM into the GPU slot pool.
//
// Sec. 2.2: after selection, B_recall = B_topk minus B_gpu is copied from
// DRAM to the GPU.  Sec. 4.4.2: scattered blocks should cross the host link
// as large coalesced transfers and land in the GPU KV cache.  Here the GPU
// itself gathers: wavefronts issue 16-byte non-temporal loads straight from
// the pinned, host-mapped store (the host->device crossing happens inside
// the load instructions) and store into the slots taken from the free list.
// Missing blocks are processed in (request, block) order, so every run of
// consecutive missing blocks is read as one contiguous host stream spread
// over consecutive workgroups.
//
// Plan kernel (one workgroup per request): set difference of the selection
// against the block table -> listed missing blocks, count, runs.
// Copy kernel (persistent grid): every workgroup scans the per-request
// counts (small), checks the pool capacity, then copies 4 KiB * LPT chunks;
// the chunk that starts a block also writes its block-table entry.
#include <type_traits>

#include "pulse_internal.h"

namespace pulse {

#ifndef PULSE_RECALL_GRID
#define PULSE_RECALL_GRID 128  // measured best on MI355X: more workgroups in flight slow the host link
#endif
#ifndef PULSE_RECALL_LPT
#define PULSE_RECALL_LPT 4
#endif

constexpr int kPlanThreads = 256;
constexpr int kCopyThreads = 256;
constexpr int64_t kRecallGrid = PULSE_RECALL_GRID;  // persistent copy workgroups
// Calls that can move at most kSmallRecallBytes, copying from every XCD, take
// half as many: with 64 workgroups in flight a 57 MB / 127 MB recall ran 0.6% /
// 0.35% faster than with 128, while a 490 MB one had occasional launches 5%
// slower (and none with 128).  A copy confined to fewer XCDs keeps 128 (16 per
// XCD reach the link rate from one XCD).
constexpr int64_t kRecallGridSmall = 64;
constexpr int64_t kSmallRecallBytes = (int64_t)256 << 20;
// Workgroups are dispatched to the 8 XCDs round-robin by id.  While a kernel reads
// pinned host memory, other kernels' HBM traffic through the same XCDs waits behind
// it.  With copy_xcds < 8 only the workgroups on the first copy_xcds XCDs copy: one
// XCD's 16 workgroups still reach the link rate, and the other XCDs stay free for
// concurrent kernels (which then also take a little link bandwidth); with 8, all do.
constexpr int kXcds = 8;

__device__ inline uint64_t lanemask_lt_r() {
    const int lane = threadIdx.x & 63;
    return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

__global__ __launch_bounds__(kPlanThreads) void recall_plan_kernel(
    const int64_t* __restrict__ blk_off, const int32_t* __restrict__ sel_idx, const int32_t* __restrict__ sel_cnt,
    int32_t k_max, const int32_t* __restrict__ table, int32_t max_blocks, int32_t n_slots,
    const int32_t* __restrict__ free_head, int32_t* __restrict__ miss_list, int32_t* __restrict__ miss_cnt,
    int32_t* __restrict__ run_cnt, int32_t* __restrict__ req_err, int32_t* __restrict__ misc, int32_t* status) {
    __shared__ uint32_t wc[kPlanThreads / kWave][2];
    __shared__ int32_t sh_err;
    const int r = blockIdx.x;
    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    if (r == 0 && tid == 0) misc[0] = *free_head;
    if (tid == 0) sh_err = 0;
    __syncthreads();
    const int64_t n = blk_off[r + 1] - blk_off[r];
    int32_t cnt = sel_cnt[r];
    int32_t my_err = 0;
    if (cnt < 0 || cnt > k_max) {
        my_err = PULSE_ERR_BAD_INDEX;
        cnt = 0;
    }
    const int32_t* row = sel_idx + (size_t)r * k_max;
    const int32_t* trow = table + (size_t)r * max_blocks;
    uint32_t carry = 0, runs = 0;
    for (int32_t tile = 0; tile < cnt; tile += kPlanThreads) {
        const int32_t i = tile + tid;
        const bool in = i < cnt;
        int32_t j = in ? row[i] : 0;
        const int32_t pj = (in && i > 0) ? row[i - 1] : -1;
        bool bad = in && (j < 0 || j >= n || j >= max_blocks || (i > 0 && j <= pj));
        bool miss = false, prev_miss = false;
        if (in && !bad) {
            const int32_t v = trow[j];
            if (v >= n_slots) bad = true;
            else miss = v < 0;
            // the previous listed entry continues the run iff it is block j-1 and missing
            if (i > 0 && pj == j - 1) prev_miss = trow[pj] < 0;
        }
        if (bad) my_err = PULSE_ERR_BAD_INDEX;
        const bool start = miss && !prev_miss;
        const uint64_t m_miss = __ballot(miss);
        const uint64_t m_start = __ballot(start);
        if (lane == 0) { wc[wid][0] = (uint32_t)__popcll(m_miss); wc[wid][1] = (uint32_t)__popcll(m_start); }
        __syncthreads();
        uint32_t pos = carry + (uint32_t)__popcll(m_miss & lanemask_lt_r()), tm = 0, ts = 0;
        for (int w = 0; w < kPlanThreads / kWave; ++w) {
            if (w < wid) pos += wc[w][0];
            tm += wc[w][0];
            ts += wc[w][1];
        }
        if (miss && pos < (uint32_t)k_max) miss_list[(size_t)r * k_max + pos] = j;
        carry += tm;
        runs += ts;
        __syncthreads();
    }
    if (my_err) atomicCAS(&sh_err, 0, my_err);
    __syncthreads();
    if (tid == 0) {
        miss_cnt[r] = (int32_t)carry;
        run_cnt[r] = (int32_t)runs;
        req_err[r] = sh_err;
        if (sh_err) report(status, sh_err);
    }
}

// Recalls larger than this (the 256 MB Infinity Cache) are stored non-temporally:
// such a volume cannot stay cached until the attention reads it, and storing it
// through keeps its write-back out of the attention that follows (measured: the
// attention after a 490 MB recall 13% faster; after recalls of 57-170 MB, which
// partly stay cached, normal stores are 3-8% better for it).
constexpr int64_t kNtStoreBytes = (int64_t)256 << 20;

template <int LPT, bool NT>
__device__ inline void copy_chunk(const uint8_t* __restrict__ src, uint8_t* __restrict__ dst, int tid) {
    u32x4 v[LPT];
#pragma unroll
    for (int k = 0; k < LPT; ++k)
        v[k] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(src) + tid + k * kCopyThreads);
#pragma unroll
    for (int k = 0; k < LPT; ++k) {
        if constexpr (NT)
            __builtin_nontemporal_store(v[k], reinterpret_cast<u32x4*>(dst) + tid + k * kCopyThreads);
        else
            reinterpret_cast<u32x4*>(dst)[tid + k * kCopyThreads] = v[k];
    }
}

template <int LPT>
__global__ __launch_bounds__(kCopyThreads) void recall_copy_kernel(
    const uint8_t* __restrict__ host, const int64_t* __restrict__ blk_off, int32_t B, int32_t k_max,
    int32_t* __restrict__ table, int32_t max_blocks, const int32_t* __restrict__ free_slots,
    int32_t* __restrict__ free_head, int32_t n_free, uint8_t* __restrict__ pool, int32_t n_slots, int64_t U,
    const int32_t* __restrict__ miss_list, const int32_t* __restrict__ miss_cnt,
    const int32_t* __restrict__ run_cnt, const int32_t* __restrict__ req_err, const int32_t* __restrict__ misc,
    pulse_recall_stats* __restrict__ stats, int32_t* status, int32_t copy_xcds) {
    __shared__ int32_t off[kMaxBatch + 1];
    __shared__ uint32_t wave_tot[kCopyThreads / kWave];
    __shared__ uint32_t sh_runs, sh_bad;
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
    // the free-list head snapshot is read with the counts, not after the scan: the
    // first chunk's slot lookup depends on it
    const int32_t fh0 = misc[0];
    // exclusive scan of miss_cnt: thread t owns a contiguous segment
    const int per = (B + kCopyThreads - 1) / kCopyThreads;
    const int s0 = tid * per, s1 = min(B, s0 + per);
    uint32_t acc = 0, racc = 0, bad = 0;
    for (int i = s0; i < s1; ++i) {
        acc += (uint32_t)miss_cnt[i];
        racc += (uint32_t)run_cnt[i];
        bad |= (uint32_t)(req_err[i] != 0);
    }
    uint32_t incl = acc;  // inclusive scan within the wave, then wave totals through LDS
    for (int o = 1; o < kWave; o <<= 1) {
        const uint32_t y = (uint32_t)__shfl_up((int)incl, o);
        if (lane >= o) incl += y;
    }
    if (lane == kWave - 1) wave_tot[wave] = incl;
    if (tid == 0) { sh_runs = 0; sh_bad = 0; }
    __syncthreads();
    if (racc) atomicAdd(&sh_runs, racc);
    if (bad) atomicOr(&sh_bad, 1u);
    uint32_t before = incl - acc;
    for (int w = 0; w < wave; ++w) before += wave_tot[w];
    for (int i = s0; i < s1; ++i) {
        off[i] = (int32_t)before;
        before += (uint32_t)miss_cnt[i];
    }
    if (tid == kCopyThreads - 1) off[B] = (int32_t)before;
    __syncthreads();
    const int64_t total = off[B];
    const bool ok = sh_bad == 0;
    const bool head_ok = fh0 >= 0 && fh0 <= n_free;
    const bool fits = head_ok && total <= (int64_t)n_free - fh0;
    // Every slot the recall takes must lie inside the pool.  Each workgroup checks the
    // whole range free_slots[fh0, fh0 + total) before anything is written, so either all
    // workgroups copy or none does, and on a bad slot the table, free-list head, pool and
    // byte count stay as they were.  kSlotCheckLoads independent loads per thread are in
    // flight per pass (an L2-resident list of at most B * k_max entries).
    int slot_bad = 0;
    if (ok && fits) {
        constexpr int kSlotCheckLoads = 8;
        for (int64_t g0 = tid; g0 < total; g0 += (int64_t)kSlotCheckLoads * kCopyThreads) {
            int32_t s[kSlotCheckLoads];
#pragma unroll
            for (int k = 0; k < kSlotCheckLoads; ++k) {
                const int64_t g = g0 + (int64_t)k * kCopyThreads;
                s[k] = g < total ? free_slots[fh0 + g] : 0;
            }
#pragma unroll
            for (int k = 0; k < kSlotCheckLoads; ++k) slot_bad |= (uint32_t)s[k] >= (uint32_t)n_slots;
        }
    }
    slot_bad = __syncthreads_or(slot_bad);
    const bool go = ok && fits && !slot_bad;
    if (blockIdx.x == 0 && tid == 0) {
        // a malformed selection (already reported by the plan) leaves no statistics
        stats->n_missing = ok ? (int32_t)total : 0;
        stats->n_runs = ok ? (int32_t)sh_runs : 0;
        stats->bytes = go ? total * U : 0;
        if (ok && !head_ok) report(status, PULSE_ERR_BAD_INDEX);
        else if (ok && !fits) report(status, PULSE_ERR_POOL_EXHAUSTED);
        else if (ok && slot_bad) report(status, PULSE_ERR_BAD_INDEX);
        if (go) *free_head = fh0 + (int32_t)total;
    }
    if (!go) return;
    constexpr int64_t chunk = 4096 * LPT;
    const int64_t cpb = U / chunk;
    const int64_t n_chunks = total * cpb;
    const bool nt_store = total * U > kNtStoreBytes;
    // copying workgroups: those on the first copy_xcds XCDs when the grid spans whole
    // rounds of kXcds, else all
    const bool confine = copy_xcds >= 1 && copy_xcds < kXcds && gridDim.x % kXcds == 0;
    const int xcd = (int)(blockIdx.x % kXcds);
    if (confine && xcd >= copy_xcds) return;
    const int64_t c0 = confine ? (int64_t)(blockIdx.x / kXcds) * copy_xcds + xcd : (int64_t)blockIdx.x;
    const int64_t cstride = confine ? (int64_t)(gridDim.x / kXcds) * copy_xcds : (int64_t)gridDim.x;
    // one loop per store kind, so the compiler cannot merge the two kinds of stores
    auto copy_all = [&](auto nt) {
        for (int64_t c = c0; c < n_chunks; c += cstride) {
            const int64_t g = c / cpb;
            const int64_t part = c - g * cpb;
            int lo = 0, hi = B;  // largest r with off[r] <= g
            while (hi - lo > 1) {
                const int mid = (lo + hi) >> 1;
                if (off[mid] <= g) lo = mid; else hi = mid;
            }
            const int r = lo;
            const int32_t j = miss_list[(size_t)r * k_max + (g - off[r])];
            const int32_t slot = free_slots[fh0 + g];
            if (slot < 0 || slot >= n_slots) continue;  // checked above; guards the store all the same
            const uint8_t* src = host + (blk_off[r] + j) * U + part * chunk;
            uint8_t* dst = pool + (int64_t)slot * U + part * chunk;
            copy_chunk<LPT, decltype(nt)::value>(src, dst, tid);
            if (part == 0 && tid == 0) table[(size_t)r * max_blocks + j] = slot;
        }
    };
    if (nt_store)
        copy_all(std::true_type{});
    else
        copy_all(std::false_type{});
}

// streaming host -> device copy with the load pattern of the recall kernel
__global__ __launch_bounds__(kCopyThreads) void probe_copy_kernel(const uint8_t* __restrict__ src,
                                                                 uint8_t* __restrict__ dst, int64_t n_chunks) {
    for (int64_t c = blockIdx.x; c < n_chunks; c += gridDim.x)
        copy_chunk<4, false>(src + c * 16384, dst + c * 16384, threadIdx.x);
}

// Step-end release of a recall (undo, LIFO): every block the last recall
// mapped returns to "not resident" and its slot to the free list, then the
// statistics are cleared so a second release changes nothing.  One thread
// per plan entry (request r, i-th missing block): setting its table entry to
// -1 is right whether the recall moved the block (it is undone) or not (the
// entry was still -1), so the table pass needs no statistics; thread 0 alone
// reads and clears them and moves the free-list head back.
constexpr int kReleaseThreads = 256;

__global__ __launch_bounds__(kReleaseThreads) void release_kernel(ReleaseArgs a) {
    release_entries(a, (int64_t)blockIdx.x * kReleaseThreads + threadIdx.x, (int64_t)gridDim.x * kReleaseThreads,
                    false);
}

hipError_t launch_release(const int32_t* miss_list, const int32_t* miss_cnt, int32_t B, int32_t k_max,
                          int32_t* table, int32_t max_blocks, int32_t* free_head, pulse_recall_stats* stats,
                          int32_t* status, hipStream_t st) {
    if (B == 0) return hipSuccess;
    const int64_t n = (int64_t)B * k_max;
    const ReleaseArgs a{miss_list, miss_cnt, B, k_max, table, max_blocks, free_head, stats, status};
    hipLaunchKernelGGL(release_kernel, dim3((unsigned)((n + kReleaseThreads - 1) / kReleaseThreads)),
                       dim3(kReleaseThreads), 0, st, a);
    return hipGetLastError();
}

hipError_t launch_recall_plan(const int64_t* blk_off, int32_t B, const int32_t* sel_idx, const int32_t* sel_cnt,
                              int32_t k_max, const int32_t* table, int32_t max_blocks, int32_t n_slots,
                              const int32_t* free_head, int32_t* miss_list, int32_t* miss_cnt, int32_t* run_cnt,
                              int32_t* req_err, int32_t* misc, int32_t* status, hipStream_t st) {
    if (B == 0) return hipSuccess;
    hipLaunchKernelGGL(recall_plan_kernel, dim3(B), dim3(kPlanThreads), 0, st, blk_off, sel_idx, sel_cnt, k_max,
                       table, max_blocks, n_slots, free_head, miss_list, miss_cnt, run_cnt, req_err, misc, status);
    return hipGetLastError();
}

hipError_t launch_recall_copy(const void* host_kv, const int64_t* blk_off, int32_t B, int32_t k_max, int32_t* table,
                              int32_t max_blocks, const int32_t* free_slots, int32_t* free_head, int32_t n_free,
                              void* pool, int32_t n_slots, size_t unit_bytes, const int32_t* miss_list,
                              const int32_t* miss_cnt, const int32_t* run_cnt, const int32_t* req_err,
                              const int32_t* misc, pulse_recall_stats* stats, int32_t* status, int32_t copy_xcds,
                              hipStream_t st, hipEvent_t start, hipEvent_t stop) {
    if (B == 0) return hipSuccess;
    // 16-byte loads in flight per thread: the largest of PULSE_RECALL_LPT, 4, 2 whose
    // 4 KiB * LPT chunk divides the block
    int lpt = 2;
    if (PULSE_RECALL_LPT >= 8 && unit_bytes % 32768 == 0) lpt = 8;
    else if (unit_bytes % 16384 == 0) lpt = 4;
    const int64_t chunk = 4096 * (int64_t)lpt;
    const int64_t max_chunks = (int64_t)B * k_max * (int64_t)(unit_bytes / chunk);
    const int64_t max_bytes = (int64_t)B * k_max * (int64_t)unit_bytes;
    const int64_t cap = (copy_xcds >= kXcds && max_bytes <= kSmallRecallBytes) ? kRecallGridSmall : kRecallGrid;
    const unsigned grid = (unsigned)(max_chunks < cap ? (max_chunks > 0 ? max_chunks : 1) : cap);
#define PULSE_COPY(L)                                                                                              \
    launch_timed(recall_copy_kernel<L>, dim3(grid), dim3(kCopyThreads), 0u, st, start, stop, (const uint8_t*)host_kv, \
                 blk_off, B, k_max, table, max_blocks, free_slots, free_head, n_free, (uint8_t*)pool, n_slots,        \
                 (int64_t)unit_bytes, miss_list, miss_cnt, run_cnt, req_err, misc, stats, status, copy_xcds)
    if (lpt == 8) PULSE_COPY(8);
    else if (lpt == 4) PULSE_COPY(4);
    else PULSE_COPY(2);
#undef PULSE_COPY
    return hipGetLastError();
}

hipError_t launch_probe_copy(const void* src, void* dst, size_t bytes, hipStream_t st) {
    const int64_t n_chunks = (int64_t)(bytes / 16384);
    if (n_chunks == 0) return hipSuccess;
    const unsigned grid = (unsigned)(n_chunks < 2048 ? n_chunks : 2048);
    hipLaunchKernelGGL(probe_copy_kernel, dim3(grid), dim3(kCopyThreads), 0, st, (const uint8_t*)src, (uint8_t*)dst,
                       n_chunks);
    return hipGetLastError();
}

}  // namespace pulse
