// irq.hip -- interruptible layer-wise scheduling (IRQ, Sec. 4.2) of an offload
// batch (the sparse-KV path of this library) against a normal batch whose
// KV cache is resident in HBM, with semi-synchronous completion detection
// (Sec. 4.2.2).
//
// Offload layer m: score + select + recall plan on the compute stream; the
// recall copy on the I/O stream, followed by a one-thread signal kernel that
// writes m's sequence number into pinned, host-mapped memory (the "interrupt
// line": the host reads it without any driver call).  Alternatively the recall
// goes through the gather-scatter engine (CPU gather, one DMA per batch, GPU
// scatter), whose completion is host-visible the same way.  On MI355X, kernels
// on other streams make little progress through the XCDs on which a kernel
// streams from host memory (their memory requests wait behind the host reads),
// so here the gather kernel copies from one XCD only; the engine's DMA leaves
// every XCD to the normal batch.  While that recall is in
// flight the host keeps enqueuing normal-batch layers on the compute stream
// and, at each normal layer boundary, checks the flag.  Once it is set, the
// offload batch's attention for layer m is enqueued on the compute stream
// behind a stream wait on the recall's completion event (the host read orders
// nothing on the GPU), then layer m + 1's selection, which issues the next
// recall, and so on.
//
// Detection modes (Sec. 4.2.2):
//   SEMI_SYNC  after enqueuing a normal layer (attention, then FFN) the host
//              waits for its attention only, then checks the flag while the
//              FFN still runs;
//   SYNC       the host waits for the whole normal layer before checking;
//   ASYNC      the host never waits for normal layers (up to `async_ahead`
//              queued), checking the flag between enqueues;
//   BLOCKING   no interleaving: each offload layer waits for its recall with
//              no other work, then one normal layer runs (a single-batch
//              schedule, the baseline).
//
// A normal-batch layer is decode attention over its resident KV (every
// block selected; the attention kernel of this library) followed by a SwiGLU
// FFN on the attention output: x = bf16(out), [g|u] = x W_gu^T, h = silu(g) *
// u, y = h W_down^T (bf16, fp32 accumulation; the two GEMMs are rocBLAS
// calls).  Projections and norms are left out.
#include <rocblas/rocblas.h>

#include <chrono>
#include <vector>

#include "pulse_internal.h"

namespace pulse {

__global__ void irq_signal_kernel(int64_t* flag, int64_t value) {
    if (threadIdx.x == 0 && blockIdx.x == 0)
        __hip_atomic_store(flag, value, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

__global__ __launch_bounds__(256) void to_bf16_kernel(const float* __restrict__ in, __bf16* __restrict__ out,
                                                      int64_t n) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        out[i] = (__bf16)in[i];
}

// h[b][i] = silu(gu[b][i]) * gu[b][F + i], in fp32, rounded to bf16.
__global__ __launch_bounds__(256) void swiglu_kernel(const __bf16* __restrict__ gu, __bf16* __restrict__ h, int32_t B,
                                                     int32_t F) {
    const int64_t n = (int64_t)B * F;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t b = i / F, c = i % F;
        const float g = (float)gu[b * 2 * F + c];
        const float u = (float)gu[b * 2 * F + F + c];
        h[i] = (__bf16)(g / (1.f + expf(-g)) * u);
    }
}

// The gather kernel copies from one XCD while normal-batch layers run: the link rate
// holds and the other XCDs keep serving HBM (from all XCDs, the concurrent layers
// would barely progress until the recall ends).
constexpr int32_t kIrqRecallXcds = 1;

static unsigned grid_for(int64_t n) {
    int64_t g = (n + 255) / 256;
    return (unsigned)(g < 1 ? 1 : (g > 4096 ? 4096 : g));
}

}  // namespace pulse

using namespace pulse;

struct pulse_irq {
    hipStream_t cmp = nullptr, io = nullptr;
    rocblas_handle blas = nullptr;
    int64_t* flag_host = nullptr;  // pinned, host-mapped
    int64_t* flag_dev = nullptr;
    int64_t seq = 0;
    std::vector<hipEvent_t> events;  // grown on demand, reused across steps
    size_t next_event = 0;

    hipEvent_t event() {
        if (next_event == events.size()) {
            hipEvent_t e;
            if (hipEventCreate(&e) != hipSuccess) return nullptr;
            events.push_back(e);
        }
        return events[next_event++];
    }
    bool flag_reached(int64_t v) const { return __atomic_load_n(flag_host, __ATOMIC_ACQUIRE) >= v; }
};

static pulse_status check_normal(const pulse_normal_layer* n) {
    PULSE_REQUIRE(n && shape_supported(&n->shape), PULSE_ERR_INVALID_ARG);
    PULSE_REQUIRE(n->B >= 1 && n->k_max >= 1 && n->max_blocks >= 1 && n->n_slots >= 1 && n->d_ff >= 1,
                  PULSE_ERR_INVALID_ARG);
    PULSE_REQUIRE(n->q && n->slot_pool && n->block_table && n->sel_idx && n->sel_cnt && n->ctx_len && n->out &&
                      n->w_gate_up && n->w_down && n->x && n->gu && n->h && n->y && n->dev_status,
                  PULSE_ERR_INVALID_ARG);
    PULSE_REQUIRE(n->ws && n->ws_bytes >= ws_layout(n->shape, n->B, n->k_max, 0).total, PULSE_ERR_WORKSPACE);
    return PULSE_OK;
}

// Enqueue one normal-batch layer on irq->cmp; ev_attn is recorded after its
// attention, ev_end after its FFN.
static pulse_status normal_layer(pulse_irq* irq, const pulse_normal_layer& n, hipEvent_t ev_attn, hipEvent_t ev_end) {
    const hipStream_t hs = irq->cmp;
    const WsLayout w = ws_layout(n.shape, n.B, n.k_max, 0);
    if (launch_attention(n.shape, n.q, n.slot_pool, n.n_slots, n.block_table, n.max_blocks, n.sel_idx, n.sel_cnt,
                         n.k_max, n.ctx_len, n.B, n.sm_scale, n.out, n.lse, ws_at<float>(n.ws, w.attn_o),
                         ws_at<float2>(n.ws, w.attn_ml), n.dev_status, hs) != hipSuccess)
        return PULSE_ERR_HIP;
    if (hipEventRecord(ev_attn, hs) != hipSuccess) return PULSE_ERR_HIP;
    const int32_t D = n.shape.num_q_heads * n.shape.head_dim, F = n.d_ff, B = n.B;
    const int64_t nx = (int64_t)B * D;
    hipLaunchKernelGGL(to_bf16_kernel, dim3(grid_for(nx)), dim3(256), 0, hs, n.out, (__bf16*)n.x, nx);
    if (hipGetLastError() != hipSuccess) return PULSE_ERR_HIP;
    const float one = 1.f, zero = 0.f;
    // [B][2F] = x [B][D] . W_gu^T   (column-major: (2F x B) = W_gu^T(2F x D) . x^T(D x B))
    if (rocblas_gemm_ex(irq->blas, rocblas_operation_transpose, rocblas_operation_none, 2 * F, B, D, &one,
                        n.w_gate_up, rocblas_datatype_bf16_r, D, n.x, rocblas_datatype_bf16_r, D, &zero, n.gu,
                        rocblas_datatype_bf16_r, 2 * F, n.gu, rocblas_datatype_bf16_r, 2 * F, rocblas_datatype_f32_r,
                        rocblas_gemm_algo_standard, 0, 0) != rocblas_status_success)
        return PULSE_ERR_HIP;
    hipLaunchKernelGGL(swiglu_kernel, dim3(grid_for((int64_t)B * F)), dim3(256), 0, hs, (const __bf16*)n.gu,
                       (__bf16*)n.h, B, F);
    if (hipGetLastError() != hipSuccess) return PULSE_ERR_HIP;
    // [B][D] = h [B][F] . W_down^T
    if (rocblas_gemm_ex(irq->blas, rocblas_operation_transpose, rocblas_operation_none, D, B, F, &one, n.w_down,
                        rocblas_datatype_bf16_r, F, n.h, rocblas_datatype_bf16_r, F, &zero, n.y,
                        rocblas_datatype_bf16_r, D, n.y, rocblas_datatype_bf16_r, D, rocblas_datatype_f32_r,
                        rocblas_gemm_algo_standard, 0, 0) != rocblas_status_success)
        return PULSE_ERR_HIP;
    if (hipEventRecord(ev_end, hs) != hipSuccess) return PULSE_ERR_HIP;
    return PULSE_OK;
}

extern "C" {

pulse_status pulse_irq_create(pulse_stream_t compute_stream, pulse_stream_t io_stream, pulse_irq** out) {
    PULSE_REQUIRE(out, PULSE_ERR_INVALID_ARG);
    *out = nullptr;
    pulse_irq* irq = new pulse_irq();
    irq->cmp = (hipStream_t)compute_stream;
    irq->io = (hipStream_t)io_stream;
    bool fail = hipHostMalloc((void**)&irq->flag_host, sizeof(int64_t),
                              hipHostMallocMapped | hipHostMallocCoherent) != hipSuccess;
    if (!fail) {
        *irq->flag_host = 0;
        fail = hipHostGetDevicePointer((void**)&irq->flag_dev, irq->flag_host, 0) != hipSuccess;
    }
    fail = fail || rocblas_create_handle(&irq->blas) != rocblas_status_success;
    fail = fail || rocblas_set_stream(irq->blas, irq->cmp) != rocblas_status_success;
    if (fail) {
        pulse_irq_destroy(irq);
        return PULSE_ERR_HIP;
    }
    *out = irq;
    return PULSE_OK;
}

pulse_status pulse_irq_destroy(pulse_irq* irq) {
    if (!irq) return PULSE_ERR_INVALID_ARG;
    if (irq->cmp) (void)hipStreamSynchronize(irq->cmp);
    if (irq->io) (void)hipStreamSynchronize(irq->io);
    for (hipEvent_t e : irq->events) (void)hipEventDestroy(e);
    if (irq->blas) (void)rocblas_destroy_handle(irq->blas);
    if (irq->flag_host) (void)hipHostFree(irq->flag_host);
    delete irq;
    return PULSE_OK;
}

pulse_status pulse_irq_step(pulse_irq* irq, const pulse_layer_args* offload, int32_t n_offload_layers,
                            const pulse_normal_layer* normal, int32_t n_normal_layers, int32_t mode,
                            int32_t async_ahead, pulse_gs_engine* engine, int32_t* overlap_depth,
                            pulse_irq_stats* stats) {
    PULSE_REQUIRE(irq && stats && n_offload_layers >= 1 && offload, PULSE_ERR_INVALID_ARG);
    PULSE_REQUIRE(mode >= PULSE_IRQ_SEMI_SYNC && mode <= PULSE_IRQ_BLOCKING, PULSE_ERR_INVALID_ARG);
    PULSE_REQUIRE(n_normal_layers >= 0 && (normal || n_normal_layers == 0), PULSE_ERR_INVALID_ARG);
    PULSE_REQUIRE(mode != PULSE_IRQ_ASYNC || async_ahead >= 1, PULSE_ERR_INVALID_ARG);
    for (int32_t m = 0; m < n_offload_layers; ++m) {
        pulse_status st = check_layer_args(&offload[m]);
        if (st != PULSE_OK) return st;
        PULSE_REQUIRE(offload[m].B >= 1, PULSE_ERR_INVALID_ARG);
    }
    for (int32_t l = 0; l < n_normal_layers; ++l) {
        pulse_status st = check_normal(&normal[l]);
        if (st != PULSE_OK) return st;
    }
    const auto t0 = std::chrono::steady_clock::now();
    const double wait_limit_s = 60.0;  // a recall that never signals means a broken device
    irq->next_event = 0;
    const size_t L = (size_t)n_offload_layers;
    std::vector<hipEvent_t> ev_sel(L), ev_rc0(L), ev_rc1(L), ev_att(L);
    std::vector<int32_t> depths(L, 0);
    int64_t nl = 0;  // normal layers enqueued
    std::vector<hipEvent_t> ring;  // layer-end events of queued normal layers (ASYNC throttle)
    size_t ring_head = 0;
    pulse_status result = PULSE_OK;
    int64_t engine_pending = 0;  // engine call submitted and not yet seen complete

    auto run_normal = [&](bool wait_attn, bool wait_all) -> pulse_status {
        hipEvent_t ea = irq->event(), ee = irq->event();
        if (!ea || !ee) return PULSE_ERR_HIP;
        if (mode == PULSE_IRQ_ASYNC) {
            if ((int64_t)(ring.size() - ring_head) >= async_ahead) {
                if (hipEventSynchronize(ring[ring_head]) != hipSuccess) return PULSE_ERR_HIP;
                ++ring_head;
            }
        }
        pulse_status st = normal_layer(irq, normal[nl % n_normal_layers], ea, ee);
        if (st != PULSE_OK) return st;
        ++nl;
        if (mode == PULSE_IRQ_ASYNC) ring.push_back(ee);
        if (wait_attn && hipEventSynchronize(ea) != hipSuccess) return PULSE_ERR_HIP;
        if (wait_all && hipEventSynchronize(ee) != hipSuccess) return PULSE_ERR_HIP;
        return PULSE_OK;
    };

    for (size_t m = 0; m < L && result == PULSE_OK; ++m) {
        const pulse_layer_args& a = offload[m];
        ev_sel[m] = irq->event();
        ev_rc0[m] = irq->event();
        ev_rc1[m] = irq->event();
        ev_att[m] = irq->event();
        if (!ev_sel[m] || !ev_rc0[m] || !ev_rc1[m] || !ev_att[m]) { result = PULSE_ERR_HIP; break; }
        // selection on the compute stream, then the recall: the GPU gather kernel + signal on
        // the I/O stream, or a submission to the gather-scatter engine
        if (layer_select(a, irq->cmp) != hipSuccess || hipEventRecord(ev_sel[m], irq->cmp) != hipSuccess) {
            result = PULSE_ERR_HIP;
            break;
        }
        int64_t seq = 0;
        if (engine) {
            result = pulse_gs_recall_submit(engine, a.host_kv, a.blk_off, a.B, a.sel_idx, a.sel_cnt, a.k_max,
                                            a.block_table, a.max_blocks, a.free_slots, a.free_head, a.n_free,
                                            a.slot_pool, a.n_slots, a.stats, a.dev_status, a.ws, a.ws_bytes, &seq,
                                            irq->cmp);
            if (result != PULSE_OK) break;
            engine_pending = seq;
        } else {
            seq = ++irq->seq;
            if (hipStreamWaitEvent(irq->io, ev_sel[m], 0) != hipSuccess ||
                hipEventRecord(ev_rc0[m], irq->io) != hipSuccess ||
                layer_recall(a, irq->io, kIrqRecallXcds) != hipSuccess) {
                result = PULSE_ERR_HIP;
                break;
            }
            hipLaunchKernelGGL(irq_signal_kernel, dim3(1), dim3(64), 0, irq->io, irq->flag_dev, seq);
            if (hipGetLastError() != hipSuccess || hipEventRecord(ev_rc1[m], irq->io) != hipSuccess) {
                result = PULSE_ERR_HIP;
                break;
            }
        }
        auto recall_done = [&]() -> bool {
            if (!engine) return irq->flag_reached(seq);
            int32_t done = 0;
            const pulse_status ps = pulse_gs_recall_poll(engine, seq, &done);
            if (done) engine_pending = 0;
            if (done && ps != PULSE_OK && result == PULSE_OK) result = ps;
            return done != 0;
        };
        // wait for the recall: normal layers run meanwhile, checked at layer boundaries
        int32_t depth = 0;
        const auto w0 = std::chrono::steady_clock::now();
        while (!recall_done()) {
            if (std::chrono::duration<double>(std::chrono::steady_clock::now() - w0).count() > wait_limit_s) {
                result = PULSE_ERR_TIMEOUT;
                break;
            }
            if (mode == PULSE_IRQ_BLOCKING || n_normal_layers == 0) continue;  // spin on the flag
            result = run_normal(mode == PULSE_IRQ_SEMI_SYNC, mode == PULSE_IRQ_SYNC);
            if (result != PULSE_OK) break;
            ++depth;
        }
        if (result != PULSE_OK) break;
        depths[m] = depth;
        // resume the offload batch: its attention for layer m
        // (the engine marks a call complete only after its streams have drained)
        if ((!engine && hipStreamWaitEvent(irq->cmp, ev_rc1[m], 0) != hipSuccess) ||
            hipEventRecord(ev_att[m], irq->cmp) != hipSuccess || layer_attention(a, irq->cmp) != hipSuccess) {
            result = PULSE_ERR_HIP;
            break;
        }
        if (mode == PULSE_IRQ_BLOCKING && n_normal_layers > 0) {  // single-batch schedule: one normal layer per layer
            result = run_normal(false, false);
            if (result != PULSE_OK) break;
        }
    }
    // drain both streams (the GPU work enqueued is finite in every case) and, after an
    // early exit, the engine call still in flight, so the engine can take the next one
    const bool ok_sync = hipStreamSynchronize(irq->cmp) == hipSuccess && hipStreamSynchronize(irq->io) == hipSuccess;
    if (engine && engine_pending) (void)pulse_gs_recall_wait(engine, engine_pending, (int32_t)(wait_limit_s * 1e3));
    if (result == PULSE_OK && !ok_sync) result = PULSE_ERR_HIP;
    const auto t1 = std::chrono::steady_clock::now();
    *stats = pulse_irq_stats{};
    stats->normal_layers = nl;
    stats->wall_ms = std::chrono::duration<double, std::milli>(t1 - t0).count();
    if (result != PULSE_OK) return result;
    stats->offload_layers = n_offload_layers;
    double sum_resume = 0.0, sum_recall = 0.0, sum_stall = 0.0, sum_depth = 0.0;
    int32_t max_depth = 0;
    for (size_t m = 0; m < L; ++m) {
        float r = 0.f, c = 0.f, w = 0.f;
        if (hipEventElapsedTime(&w, ev_sel[m], ev_att[m]) != hipSuccess) return PULSE_ERR_HIP;
        if (!engine && (hipEventElapsedTime(&r, ev_rc1[m], ev_att[m]) != hipSuccess ||
                        hipEventElapsedTime(&c, ev_rc0[m], ev_rc1[m]) != hipSuccess))
            return PULSE_ERR_HIP;
        sum_resume += r;
        sum_recall += c;
        sum_stall += w;
        sum_depth += depths[m];
        max_depth = depths[m] > max_depth ? depths[m] : max_depth;
        if (overlap_depth) overlap_depth[m] = depths[m];
    }
    stats->mean_stall_us = sum_stall * 1e3 / (double)L;
    stats->mean_resume_us = engine ? -1.0 : sum_resume * 1e3 / (double)L;
    stats->mean_recall_us = engine ? -1.0 : sum_recall * 1e3 / (double)L;
    stats->mean_overlap_depth = sum_depth / (double)L;
    stats->max_overlap_depth = max_depth;
    return PULSE_OK;
}

}  // extern "C"
