// gather_engine.hip -- the paper's own recall engine, as a second recall path
// next to the GPU-gather kernel: CPU gather into pinned staging, one large DMA,
// GPU scatter (Sec. 4.4.2), submitted without a host synchronisation through a
// host-visible mailbox polled by a CPU thread (zero-sync I/O submission,
// Sec. 4.5).
//
//   caller stream:  plan kernel (set difference)  ->  publish kernel
//                   (allocation, table / free_head / stats updates, plan and
//                   ready sequence number written to the pinned mailbox)
//   poller thread:  sees the new sequence number, splits the plan into staging
//                   batches; worker threads memcpy the blocks from the host
//                   store into pinned staging (two halves; the first batch is
//                   an eighth of a full one so the link starts early); the
//                   workers spin while a call is served, so a batch costs no
//                   thread wake-up;
//   copy stream:    one hipMemcpyAsync per batch (staging -> device staging),
//                   back to back;
//   scatter stream: per batch, after its DMA, the scatter kernel (device
//                   staging -> pool slots), so no DMA waits for a scatter;
//   completion:     the poller stores the sequence number as completed; the
//                   caller polls (semi-synchronous check) or waits with a
//                   timeout before enqueuing attention.
// No GPU stream ever waits on a host-written value, so a stalled host thread
// cannot hang the GPU.
#include <atomic>
#include <chrono>
#include <condition_variable>
#include <cstring>
#include <mutex>
#include <thread>
#include <vector>

#include "pulse_internal.h"

namespace pulse {

struct alignas(64) Mailbox {
    int64_t ready_seq;  // written last by the publish kernel (system scope)
    int64_t n_blocks;   // blocks in the plan (0 on any device error)
    int32_t status;     // device-detected error of this call (0 = ok)
    int32_t pad[11];
    // followed by int64 src_block[cap] then int32 slot[cap]
};

constexpr int kPublishThreads = 1024;

// Allocation + plan publication: one workgroup.  Mirrors the allocation of the
// GPU-gather path: the g-th missing block in (request, listed order) takes
// free_slots[free_head + g].
__global__ __launch_bounds__(kPublishThreads) void publish_plan_kernel(
    const int64_t* __restrict__ blk_off, int32_t B, int32_t k_max, int32_t* __restrict__ table, int32_t max_blocks,
    const int32_t* __restrict__ free_slots, int32_t* __restrict__ free_head, int32_t n_free, int32_t n_slots,
    int64_t U, const int32_t* __restrict__ miss_list, const int32_t* __restrict__ miss_cnt,
    const int32_t* __restrict__ run_cnt, const int32_t* __restrict__ req_err, const int32_t* __restrict__ misc,
    pulse_recall_stats* __restrict__ stats, int32_t* status, Mailbox* mb, int64_t* mb_src, int32_t* mb_slot,
    int64_t cap, int64_t seq) {
    __shared__ int32_t off[kMaxBatch + 1];
    __shared__ uint32_t sh_runs, sh_bad;
    const int tid = threadIdx.x;
    if (tid == 0) {
        uint32_t acc = 0, runs = 0, bad = 0;
        for (int i = 0; i < B; ++i) {  // B <= kMaxBatch, one thread: small
            off[i] = (int32_t)acc;
            acc += (uint32_t)miss_cnt[i];
            runs += (uint32_t)run_cnt[i];
            bad |= (uint32_t)(req_err[i] != 0);
        }
        off[B] = (int32_t)acc;
        sh_runs = runs;
        sh_bad = bad;
    }
    __syncthreads();
    const int64_t total = off[B];
    const int32_t fh0 = misc[0];
    const bool ok = sh_bad == 0;
    const bool head_ok = fh0 >= 0 && fh0 <= n_free;
    const bool fits = head_ok && total <= (int64_t)n_free - fh0;
    const bool room = total <= cap;
    // First pass: every slot the recall takes must lie inside the pool.  Nothing is
    // written (table, free-list head, statistics, mailbox plan) unless all of them do.
    int slot_bad = 0;
    if (ok && fits && room)
        for (int64_t g = tid; g < total; g += kPublishThreads)
            slot_bad |= (uint32_t)free_slots[fh0 + g] >= (uint32_t)n_slots;
    const bool any_slot_bad = __syncthreads_or(slot_bad) != 0;
    const bool go = ok && fits && room && !any_slot_bad;
    if (go) {
        for (int64_t g = tid; g < total; g += kPublishThreads) {
            int lo = 0, hi = B;
            while (hi - lo > 1) {
                const int mid = (lo + hi) >> 1;
                if (off[mid] <= g) lo = mid; else hi = mid;
            }
            const int32_t j = miss_list[(size_t)lo * k_max + (g - off[lo])];
            const int32_t slot = free_slots[fh0 + g];
            table[(size_t)lo * max_blocks + j] = slot;
            mb_src[g] = blk_off[lo] + j;
            mb_slot[g] = slot;
        }
    }
    __threadfence_system();  // every thread's plan entries reach host memory ...
    __syncthreads();         // ... before thread 0 publishes the sequence number
    if (tid == 0) {
        int32_t err = 0;
        if (!ok || !head_ok) err = PULSE_ERR_BAD_INDEX;
        else if (!fits) err = PULSE_ERR_POOL_EXHAUSTED;
        else if (!room) err = PULSE_ERR_WORKSPACE;
        else if (any_slot_bad) err = PULSE_ERR_BAD_INDEX;
        if (err) report(status, err);
        // a malformed selection (already reported by the plan) leaves no statistics
        stats->n_missing = ok ? (int32_t)total : 0;
        stats->n_runs = ok ? (int32_t)sh_runs : 0;
        stats->bytes = go ? total * U : 0;
        if (go) *free_head = fh0 + (int32_t)total;
        mb->n_blocks = go ? total : 0;
        mb->status = err;
        __threadfence_system();  // header before the sequence number
        __hip_atomic_store(&mb->ready_seq, seq, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    }
}

// device staging -> pool slots; grid-stride over (block, chunk of 4096 * V bytes): 16 KiB
// chunks (V = 4), or 8 KiB (V = 2) for blocks that are not a multiple of 16 KiB (a block is
// Hkv * bs * 512 bytes, so it is always a multiple of 8 KiB)
template <int V>
__global__ __launch_bounds__(256) void scatter_kernel(const uint8_t* __restrict__ staging,
                                                      const int32_t* __restrict__ slots, int64_t n, int64_t U,
                                                      int32_t n_slots, uint8_t* __restrict__ pool) {
    constexpr int64_t kChunk = 4096 * V;
    const int64_t cpb = U / kChunk;
    for (int64_t c = blockIdx.x; c < n * cpb; c += gridDim.x) {
        const int64_t k = c / cpb, part = c - k * cpb;
        const int32_t slot = slots[k];
        if (slot < 0 || slot >= n_slots) continue;
        const u32x4* src = reinterpret_cast<const u32x4*>(staging + k * U + part * kChunk);
        u32x4* dst = reinterpret_cast<u32x4*>(pool + (int64_t)slot * U + part * kChunk);
#pragma unroll
        for (int i = 0; i < V; ++i) dst[threadIdx.x + 256 * i] = src[threadIdx.x + 256 * i];
    }
}

}  // namespace pulse

using namespace pulse;

struct pulse_gs_engine {
    pulse_shape shape;
    size_t U = 0;
    int64_t cap = 0;            // plan entries per call
    int64_t batch_blocks = 0;   // blocks per staging half
    Mailbox* mb = nullptr;      // pinned, coherent (host view)
    int64_t* mb_src = nullptr;
    int32_t* mb_slot = nullptr;
    Mailbox* d_mb = nullptr;    // device view of the same memory
    int64_t* d_src = nullptr;
    int32_t* d_slot = nullptr;
    uint8_t* host_stage[2] = {nullptr, nullptr};
    uint8_t* dev_stage[2] = {nullptr, nullptr};
    hipEvent_t dma_done[2] = {nullptr, nullptr};   // host staging half free again
    hipEvent_t scat_done[2] = {nullptr, nullptr};  // device staging half free again
    hipStream_t copy = nullptr;                    // DMAs, back to back
    hipStream_t scat = nullptr;                    // scatter kernels, each after its DMA
    int device = 0;
    // the call being served
    std::mutex mu;
    std::condition_variable cv;
    const uint8_t* host_kv = nullptr;  // set under mu by the submitting thread
    uint8_t* pool = nullptr;
    int32_t n_slots = 0;
    const uint8_t* cur_host_kv = nullptr;  // copies read by the poller and the workers
    uint8_t* cur_pool = nullptr;
    int32_t cur_n_slots = 0;
    int64_t submitted = 0;
    std::atomic<int64_t> completed{0};
    std::atomic<int32_t> last_status{0};
    float timing_ms[3] = {0, 0, 0};  // gather, dma+scatter tail, total (poller clock)
    // threads
    std::atomic<bool> running{true};
    std::thread poller;
    int n_workers = 0;
    std::vector<std::thread> workers;
    std::mutex wmu;
    std::condition_variable wcv;
    std::atomic<int64_t> job_gen{0};   // bumped (release) once a job's fields are set
    std::atomic<int> jobs_left{0};      // workers still copying the current job
    std::atomic<bool> serving{false};   // a call is in progress: idle workers spin, not sleep
    const int64_t* job_src = nullptr;
    uint8_t* job_dst = nullptr;
    int64_t job_n = 0;

    void worker_loop(int id) {
        int64_t seen = 0;
        for (;;) {
            int64_t g = job_gen.load(std::memory_order_acquire);
            while (g == seen) {  // wait for the next job
                if (!running.load()) return;
                if (serving.load(std::memory_order_relaxed)) {
                    std::this_thread::yield();
                } else {
                    std::unique_lock<std::mutex> lk(wmu);
                    wcv.wait_for(lk, std::chrono::milliseconds(1), [&] {
                        return !running.load() || serving.load() || job_gen.load() != seen;
                    });
                }
                g = job_gen.load(std::memory_order_acquire);
            }
            seen = g;
            const int64_t n = job_n;
            const int64_t* src = job_src;
            uint8_t* dst = job_dst;
            const int64_t per = (n + n_workers - 1) / n_workers;
            const int64_t k0 = id * per, k1 = std::min<int64_t>(n, k0 + per);
            for (int64_t k = k0; k < k1; ++k)
                if (src[k] >= 0) std::memcpy(dst + k * U, cur_host_kv + src[k] * U, U);
            jobs_left.fetch_sub(1, std::memory_order_acq_rel);
        }
    }

    // All workers copy their share of the n blocks listed in src into dst; returns
    // when every share is done (spinning: the workers are spinning too).
    void gather(const int64_t* src, uint8_t* dst, int64_t n) {
        job_src = src;
        job_dst = dst;
        job_n = n;
        jobs_left.store(n_workers, std::memory_order_relaxed);
        job_gen.fetch_add(1, std::memory_order_release);
        while (jobs_left.load(std::memory_order_acquire) != 0) std::this_thread::yield();
    }

    void serve(int64_t seq) {
        using clk = std::chrono::steady_clock;
        const auto t0 = clk::now();
        {
            std::lock_guard<std::mutex> lk(wmu);  // a worker about to block sees the flag or the notify
            serving.store(true);
        }
        wcv.notify_all();
        {
            std::lock_guard<std::mutex> lk(mu);  // fields of the call, set by the submitting thread
            cur_host_kv = host_kv;
            cur_pool = pool;
            cur_n_slots = n_slots;
        }
        double gather_ms = 0;
        const int64_t n = mb->n_blocks;
        int32_t st = mb->status;
        // Batches alternate between two staging halves.  The DMAs run back to back on
        // their own stream; each scatter waits for its DMA on another stream, so a DMA
        // never waits for the previous scatter.  The first batch is an eighth of a full one
        // so the link starts early.
        int half = 0;
        for (int64_t b0 = 0, i = 0; b0 < n && st == 0; ++i) {
            const int64_t want = i == 0 ? std::max<int64_t>(1, batch_blocks / 8) : batch_blocks;
            const int64_t nb = std::min<int64_t>(want, n - b0);
            if (hipEventSynchronize(dma_done[half]) != hipSuccess) { st = PULSE_ERR_HIP; break; }
            const auto g0 = clk::now();
            gather(mb_src + b0, host_stage[half], nb);
            gather_ms += std::chrono::duration<double, std::milli>(clk::now() - g0).count();
            if (hipStreamWaitEvent(copy, scat_done[half], 0) != hipSuccess ||
                hipMemcpyAsync(dev_stage[half], host_stage[half], (size_t)nb * U, hipMemcpyHostToDevice, copy) !=
                    hipSuccess ||
                hipEventRecord(dma_done[half], copy) != hipSuccess ||
                hipStreamWaitEvent(scat, dma_done[half], 0) != hipSuccess) {
                st = PULSE_ERR_HIP;
                break;
            }
            const bool wide = U % 16384 == 0;
            const int64_t chunks = nb * (int64_t)(U / (wide ? 16384 : 8192));
            const dim3 sgrid((unsigned)std::min<int64_t>(chunks, 1024));
            if (wide)
                hipLaunchKernelGGL(scatter_kernel<4>, sgrid, dim3(256), 0, scat, dev_stage[half], d_slot + b0, nb,
                                   (int64_t)U, cur_n_slots, cur_pool);
            else
                hipLaunchKernelGGL(scatter_kernel<2>, sgrid, dim3(256), 0, scat, dev_stage[half], d_slot + b0, nb,
                                   (int64_t)U, cur_n_slots, cur_pool);
            if (hipGetLastError() != hipSuccess || hipEventRecord(scat_done[half], scat) != hipSuccess) {
                st = PULSE_ERR_HIP;
                break;
            }
            b0 += nb;
            half ^= 1;
        }
        if ((hipStreamSynchronize(copy) != hipSuccess || hipStreamSynchronize(scat) != hipSuccess) && st == 0)
            st = PULSE_ERR_HIP;
        {
            std::lock_guard<std::mutex> lk(wmu);
            serving.store(false);
        }
        const auto t1 = clk::now();
        {
            std::lock_guard<std::mutex> lk(mu);
            timing_ms[0] = (float)gather_ms;
            timing_ms[2] = (float)std::chrono::duration<double, std::milli>(t1 - t0).count();
            timing_ms[1] = timing_ms[2] - timing_ms[0];
            last_status.store(st);
            completed.store(seq);
        }
        cv.notify_all();
    }

    void poll_loop() {
        (void)hipSetDevice(device);
        int64_t handled = 0;
        while (running.load()) {
            const int64_t seq = __atomic_load_n(&mb->ready_seq, __ATOMIC_ACQUIRE);
            if (seq > handled) {
                handled = seq;
                serve(seq);
            } else {
                std::this_thread::yield();
            }
        }
    }
};

namespace pulse {
// Whether an engine was created for shape `s` (pulse_irq_step checks every offload layer).
bool gs_engine_serves(const pulse_gs_engine* e, const pulse_shape& s) {
    return e->shape.num_q_heads == s.num_q_heads && e->shape.num_kv_heads == s.num_kv_heads &&
           e->shape.head_dim == s.head_dim && e->shape.block_size == s.block_size && e->shape.dtype == s.dtype;
}
}  // namespace pulse

extern "C" {

pulse_status pulse_gs_engine_create(const pulse_shape* shape, int32_t n_workers, int64_t max_blocks_per_call,
                                    int64_t staging_blocks, pulse_gs_engine** out) {
    if (!out) return PULSE_ERR_INVALID_ARG;
    *out = nullptr;
    if (!shape) return PULSE_ERR_INVALID_ARG;
    if (!shape_supported(shape)) return PULSE_ERR_UNSUPPORTED;
    if (n_workers < 1 || n_workers > 64 || max_blocks_per_call < 1 || staging_blocks < 1)
        return PULSE_ERR_INVALID_ARG;
    auto* e = new pulse_gs_engine();
    e->shape = *shape;
    e->U = pulse_block_bytes(shape);
    e->cap = max_blocks_per_call;
    e->batch_blocks = staging_blocks;
    e->n_workers = n_workers;
    bool fail = hipGetDevice(&e->device) != hipSuccess;
    const size_t mb_bytes = sizeof(Mailbox) + (size_t)e->cap * (sizeof(int64_t) + sizeof(int32_t));
    void* p = nullptr;
    fail = fail || hipHostMalloc(&p, mb_bytes, hipHostMallocMapped | hipHostMallocCoherent) != hipSuccess;
    if (!fail) {
        std::memset(p, 0, mb_bytes);
        e->mb = static_cast<Mailbox*>(p);
        e->mb_src = reinterpret_cast<int64_t*>(e->mb + 1);
        e->mb_slot = reinterpret_cast<int32_t*>(e->mb_src + e->cap);
        void* dp = nullptr;
        fail = hipHostGetDevicePointer(&dp, p, 0) != hipSuccess;
        if (!fail) {
            e->d_mb = static_cast<Mailbox*>(dp);
            e->d_src = reinterpret_cast<int64_t*>(e->d_mb + 1);
            e->d_slot = reinterpret_cast<int32_t*>(e->d_src + e->cap);
        }
    }
    for (int h = 0; h < 2 && !fail; ++h) {
        fail = hipHostMalloc((void**)&e->host_stage[h], (size_t)staging_blocks * e->U, hipHostMallocDefault) !=
                   hipSuccess ||
               hipMalloc((void**)&e->dev_stage[h], (size_t)staging_blocks * e->U) != hipSuccess ||
               hipEventCreateWithFlags(&e->dma_done[h], hipEventDisableTiming) != hipSuccess ||
               hipEventCreateWithFlags(&e->scat_done[h], hipEventDisableTiming) != hipSuccess;
    }
    fail = fail || hipStreamCreateWithFlags(&e->copy, hipStreamNonBlocking) != hipSuccess ||
           hipStreamCreateWithFlags(&e->scat, hipStreamNonBlocking) != hipSuccess;
    for (int h = 0; h < 2 && !fail; ++h)
        fail = hipEventRecord(e->dma_done[h], e->copy) != hipSuccess ||
               hipEventRecord(e->scat_done[h], e->scat) != hipSuccess;
    if (fail) {
        pulse_gs_engine_destroy(e);
        return PULSE_ERR_HIP;
    }
    for (int i = 0; i < n_workers; ++i) e->workers.emplace_back([e, i] { e->worker_loop(i); });
    e->poller = std::thread([e] { e->poll_loop(); });
    *out = e;
    return PULSE_OK;
}

pulse_status pulse_gs_engine_destroy(pulse_gs_engine* e) {
    if (!e) return PULSE_ERR_INVALID_ARG;
    e->running.store(false);
    {
        std::lock_guard<std::mutex> lk(e->wmu);
        e->wcv.notify_all();
    }
    if (e->poller.joinable()) e->poller.join();
    for (auto& t : e->workers)
        if (t.joinable()) t.join();
    for (hipStream_t s : {e->copy, e->scat})
        if (s) {
            (void)hipStreamSynchronize(s);
            (void)hipStreamDestroy(s);
        }
    for (int h = 0; h < 2; ++h) {
        if (e->dma_done[h]) (void)hipEventDestroy(e->dma_done[h]);
        if (e->scat_done[h]) (void)hipEventDestroy(e->scat_done[h]);
        if (e->host_stage[h]) (void)hipHostFree(e->host_stage[h]);
        if (e->dev_stage[h]) (void)hipFree(e->dev_stage[h]);
    }
    if (e->mb) (void)hipHostFree(e->mb);
    delete e;
    return PULSE_OK;
}

pulse_status pulse_gs_recall_submit(pulse_gs_engine* e, const void* host_kv, const int64_t* blk_off, int32_t B,
                                    const int32_t* sel_idx, const int32_t* sel_cnt, int32_t k_max,
                                    int32_t* block_table, int32_t max_blocks, const int32_t* free_slots,
                                    int32_t* free_head, int32_t n_free, void* slot_pool, int32_t n_slots,
                                    pulse_recall_stats* stats, int32_t* dev_status, void* ws, size_t ws_bytes,
                                    int64_t* seq_out, pulse_stream_t stream) {
    if (!e || !seq_out) return PULSE_ERR_INVALID_ARG;
    *seq_out = 0;
    if (B < 0 || k_max < 1 || max_blocks < 1 || n_free < 0 || n_slots < 1) return PULSE_ERR_INVALID_ARG;
    if (B > kMaxBatch) return PULSE_ERR_UNSUPPORTED;
    if (B == 0) return PULSE_OK;
    if (!host_kv || !blk_off || !sel_idx || !sel_cnt || !block_table || !free_head || !slot_pool || !stats ||
        !dev_status || (!free_slots && n_free))
        return PULSE_ERR_INVALID_ARG;
    const WsLayout w = ws_layout(e->shape, B, k_max, 0);
    if (!ws || ws_bytes < w.total) return PULSE_ERR_WORKSPACE;
    if (e->completed.load() != e->submitted) return PULSE_ERR_INVALID_ARG;  // one call in flight at a time
    auto at32 = [&](size_t off) { return reinterpret_cast<int32_t*>(static_cast<char*>(ws) + off); };
    hipStream_t hs = (hipStream_t)stream;
    {
        std::lock_guard<std::mutex> lk(e->mu);
        e->host_kv = static_cast<const uint8_t*>(host_kv);
        e->pool = static_cast<uint8_t*>(slot_pool);
        e->n_slots = n_slots;
    }
    hipError_t err = launch_recall_plan(blk_off, B, sel_idx, sel_cnt, k_max, block_table, max_blocks, n_slots,
                                        free_head, at32(w.miss_list), at32(w.miss_cnt), at32(w.run_cnt),
                                        at32(w.req_err), at32(w.misc), dev_status, hs);
    if (err != hipSuccess) return PULSE_ERR_HIP;
    const int64_t seq = e->submitted + 1;
    hipLaunchKernelGGL(publish_plan_kernel, dim3(1), dim3(kPublishThreads), 0, hs, blk_off, B, k_max, block_table,
                       max_blocks, free_slots, free_head, n_free, n_slots, (int64_t)e->U, at32(w.miss_list),
                       at32(w.miss_cnt), at32(w.run_cnt), at32(w.req_err), at32(w.misc), stats, dev_status, e->d_mb,
                       e->d_src, e->d_slot, e->cap, seq);
    if (hipGetLastError() != hipSuccess) return PULSE_ERR_HIP;
    e->submitted = seq;
    *seq_out = seq;
    return PULSE_OK;
}

pulse_status pulse_gs_recall_poll(pulse_gs_engine* e, int64_t seq, int32_t* done) {
    if (!e || !done) return PULSE_ERR_INVALID_ARG;
    *done = e->completed.load() >= seq;
    return *done ? (pulse_status)e->last_status.load() : PULSE_OK;
}

pulse_status pulse_gs_recall_wait(pulse_gs_engine* e, int64_t seq, int32_t timeout_ms) {
    if (!e) return PULSE_ERR_INVALID_ARG;
    std::unique_lock<std::mutex> lk(e->mu);
    const bool ok = e->cv.wait_for(lk, std::chrono::milliseconds(timeout_ms < 0 ? 0 : timeout_ms),
                                   [&] { return e->completed.load() >= seq; });
    if (!ok) return PULSE_ERR_TIMEOUT;
    return (pulse_status)e->last_status.load();
}

pulse_status pulse_gs_last_timing(pulse_gs_engine* e, float* ms3) {
    if (!e || !ms3) return PULSE_ERR_INVALID_ARG;
    std::lock_guard<std::mutex> lk(e->mu);
    for (int i = 0; i < 3; ++i) ms3[i] = e->timing_ms[i];
    return PULSE_OK;
}

}  // extern "C"
