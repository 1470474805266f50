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
// u, y = h W_down^T (bf16, fp32 accumulation; the two GEMMs are the MFMA
// kernel below).  Projections and norms are left out.
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

// ---- the FFN's GEMMs ------------------------------------------------------
// C[M][N] = A[M][K] . Wt[N][K]^T with bf16 inputs, fp32 accumulation and a bf16
// (round-to-nearest-even) result: the shape of a decode batch's projections,
// M (requests) small and N, K model widths, so the weight rows dominate the
// traffic.  A workgroup of kGemmWaves waves owns 16 * NT output columns and
// 16 * MT rows.  Its waves split K: wave w takes kGemmUnroll consecutive
// 32-element steps at a time (every weight row is read in 256-byte runs), all
// their loads in flight before the products.  Per step a lane loads 16
// contiguous bytes of one weight row per column tile (B operand: column =
// lane % 16, k = 8 * (lane / 16) ...) and of one activation row per row tile
// (A operand), and v_mfma_f32_16x16x32_bf16 accumulates each 16 x 16 tile
// (lane holds rows 4 * (lane / 16) + v, column lane % 16).  Weights are loaded
// non-temporally: they are read once, and the activations (read by every
// workgroup) then stay in L2.  The waves' partial tiles are summed in LDS.
// K must be a multiple of 8 and rows 16-byte aligned.
constexpr int kGemmWaves = 8;

template <int MT, int NT, int U>
__global__ __launch_bounds__(kGemmWaves * kWave) void ffn_gemm_kernel(const __bf16* __restrict__ A,
                                                                      const __bf16* __restrict__ Wt,
                                                                      __bf16* __restrict__ C, int32_t M, int32_t N,
                                                                      int32_t K) {
    __shared__ float red[kGemmWaves][NT][MT][4][kWave];
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
    const int col = lane & 15, grp = lane >> 4;
    const int n0 = blockIdx.x * 16 * NT, m0 = blockIdx.y * 16 * MT;
    const __bf16* wrow[NT];
    bool n_ok[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
        const int n = n0 + 16 * nt + col;
        n_ok[nt] = n < N;
        wrow[nt] = Wt + (size_t)(n_ok[nt] ? n : 0) * K + grp * 8;
    }
    const __bf16* arow[MT];
    bool m_ok[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
        const int m = m0 + 16 * mt + col;
        m_ok[mt] = m < M;
        arow[mt] = A + (size_t)(m_ok[mt] ? m : 0) * K + grp * 8;
    }
    const u32x4 zero = {0, 0, 0, 0};
    f32x4 acc[NT][MT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) acc[nt][mt] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int steps = (K + 31) / 32;
    for (int sb = wave * U; sb < steps; sb += kGemmWaves * U) {
        u32x4 b[U][NT], a[U][MT];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int k = (sb + u) * 32;  // this lane's 8 elements start at k + 8 * grp
            const bool k_ok = k + grp * 8 < K;
#pragma unroll
            for (int nt = 0; nt < NT; ++nt)
                b[u][nt] = (k_ok && n_ok[nt])
                               ? __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(wrow[nt] + k))
                               : zero;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
                a[u][mt] = (k_ok && m_ok[mt]) ? *reinterpret_cast<const u32x4*>(arow[mt] + k) : zero;
        }
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int nt = 0; nt < NT; ++nt)
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
                    acc[nt][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a[u][mt]),
                                                                          __builtin_bit_cast(bf16x8, b[u][nt]),
                                                                          acc[nt][mt], 0, 0, 0);
    }
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int v = 0; v < 4; ++v) red[wave][nt][mt][v][lane] = acc[nt][mt][v];
    __syncthreads();
    for (int o = tid; o < 16 * MT * 16 * NT; o += kGemmWaves * kWave) {
        const int ml = o / (16 * NT), nl = o % (16 * NT);  // row of the workgroup's rows, column of its columns
        const int mt = ml / 16, i = ml % 16, nt = nl / 16;
        const int v = i % 4, src = (i / 4) * 16 + nl % 16;
        float sum = 0.f;
#pragma unroll
        for (int w = 0; w < kGemmWaves; ++w) sum += red[w][nt][mt][v][src];
        const int m = m0 + ml, n = n0 + nl;
        if (m < M && n < N) C[(size_t)m * N + n] = (__bf16)sum;
    }
}

// The same product for wide outputs (many column tiles), with the activations shared
// through LDS: a workgroup's 8 waves are CG = 8 / KG column groups of 16 * NT
// columns times KG K-groups.  K advances in chunks of KC = KG * U * 32 elements;
// each chunk of the workgroup's 16 * MT activation rows is staged once in LDS
// (double-buffered, rows padded by 16 bytes against bank conflicts) and read by
// all column groups, while every wave prefetches its weights of the next chunk.
// The K-groups' partial tiles are summed in LDS at the end.
template <int MT, int NT, int KG, int U>
__global__ __launch_bounds__(kGemmWaves * kWave) void ffn_gemm_lds_kernel(const __bf16* __restrict__ A,
                                                                          const __bf16* __restrict__ Wt,
                                                                          __bf16* __restrict__ C, int32_t M,
                                                                          int32_t N, int32_t K) {
    constexpr int CG = kGemmWaves / KG;
    constexpr int KC = KG * U * 32;    // K elements per chunk
    constexpr int ROWS = 16 * MT;
    constexpr int PITCH = KC + 8;      // elements per staged row
    constexpr int PIECES = ROWS * KC / 8;  // 16-byte pieces of a chunk
    constexpr int kThreads = kGemmWaves * kWave;
    constexpr int kStageBytes = 2 * ROWS * PITCH * 2;
    constexpr int kRedBytes = KG * CG * NT * MT * 4 * kWave * 4;
    static_assert(PIECES % kThreads == 0, "a chunk is an exact number of pieces per thread");
    __shared__ __align__(16) uint8_t smem[kStageBytes > kRedBytes ? kStageBytes : kRedBytes];
    uint16_t(*sa)[ROWS][PITCH] = reinterpret_cast<uint16_t(*)[ROWS][PITCH]>(smem);
    const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
    const int col = lane & 15, grp = lane >> 4;
    const int cg = wave % CG, kg = wave / CG;
    const int n0 = blockIdx.x * 16 * NT * CG + cg * 16 * NT, m0 = blockIdx.y * ROWS;
    const __bf16* wrow[NT];
    bool n_ok[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
        const int n = n0 + 16 * nt + col;
        n_ok[nt] = n < N;
        wrow[nt] = Wt + (size_t)(n_ok[nt] ? n : 0) * K + grp * 8;
    }
    const u32x4 zero = {0, 0, 0, 0};
    // this thread's pieces of an activation chunk: row, element offset
    auto stage_load = [&](int k0, u32x4 (&ra)[PIECES / kThreads]) {
#pragma unroll
        for (int i = 0; i < PIECES / kThreads; ++i) {
            const int pc = tid + i * kThreads;
            const int row = pc / (KC / 8), kk = (pc % (KC / 8)) * 8;
            const int m = m0 + row, k = k0 + kk;
            ra[i] = (m < M && k < K) ? *reinterpret_cast<const u32x4*>(A + (size_t)m * K + k) : zero;
        }
    };
    auto stage_store = [&](int buf, const u32x4 (&ra)[PIECES / kThreads]) {
#pragma unroll
        for (int i = 0; i < PIECES / kThreads; ++i) {
            const int pc = tid + i * kThreads;
            const int row = pc / (KC / 8), kk = (pc % (KC / 8)) * 8;
            *reinterpret_cast<u32x4*>(&sa[buf][row][kk]) = ra[i];
        }
    };
    auto load_w = [&](int k0, u32x4 (&b)[U][NT]) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int k = k0 + (kg * U + u) * 32;  // this lane's 8 elements start at k + 8 * grp
            const bool k_ok = k + grp * 8 < K;
#pragma unroll
            for (int nt = 0; nt < NT; ++nt)
                b[u][nt] = (k_ok && n_ok[nt])
                               ? __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(wrow[nt] + k))
                               : zero;
        }
    };
    f32x4 acc[NT][MT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) acc[nt][mt] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int n_chunks = (K + KC - 1) / KC;
    u32x4 ra[PIECES / kThreads], b[U][NT], bn[U][NT];
    stage_load(0, ra);
    load_w(0, b);
    stage_store(0, ra);
    __syncthreads();
    for (int it = 0; it < n_chunks; ++it) {
        const bool more = it + 1 < n_chunks;
        if (more) {  // next chunk's weights and activations in flight during this chunk's products
            load_w((it + 1) * KC, bn);
            stage_load((it + 1) * KC, ra);
        }
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                const u32x4 af = *reinterpret_cast<const u32x4*>(&sa[it & 1][16 * mt + col][(kg * U + u) * 32 + grp * 8]);
#pragma unroll
                for (int nt = 0; nt < NT; ++nt)
                    acc[nt][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, af),
                                                                          __builtin_bit_cast(bf16x8, b[u][nt]),
                                                                          acc[nt][mt], 0, 0, 0);
            }
        if (more) stage_store((it + 1) & 1, ra);
        __syncthreads();
        if (more) {
#pragma unroll
            for (int u = 0; u < U; ++u)
#pragma unroll
                for (int nt = 0; nt < NT; ++nt) b[u][nt] = bn[u][nt];
        }
    }
    // the staging buffers are free now (the loop ended with a barrier): K-group partials
    float(*red)[CG][NT][MT][4][kWave] = reinterpret_cast<float(*)[CG][NT][MT][4][kWave]>(smem);
#pragma unroll
    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int v = 0; v < 4; ++v) red[kg][cg][nt][mt][v][lane] = acc[nt][mt][v];
    __syncthreads();
    constexpr int COLS = 16 * NT * CG;
    const int nb = blockIdx.x * COLS;
    for (int o = tid; o < ROWS * COLS; o += kThreads) {
        const int ml = o / COLS, nl = o % COLS;  // row of the workgroup's rows, column of its columns
        const int g = nl / (16 * NT), nt = (nl / 16) % NT, mt = ml / 16, i = ml % 16;
        const int v = i % 4, src = (i / 4) * 16 + nl % 16;
        float sum = 0.f;
#pragma unroll
        for (int w = 0; w < KG; ++w) sum += red[w][g][nt][mt][v][src];
        const int m = m0 + ml, n = nb + nl;
        if (m < M && n < N) C[(size_t)m * N + n] = (__bf16)sum;
    }
}

// Wide outputs (N >= 16384: at least 256 workgroups of 64 columns) with at most 32 rows use
// the LDS kernel with 4 column groups of 16 columns x 2 K-groups (measured on 32 x 4096 x 28672:
// 58.9 us, against 64.0 with 128 columns per workgroup and 60.1 with 8 column groups and one
// K-group); the others the direct kernel with 16 columns per workgroup (enough workgroups for
// narrow outputs: 48 us on 32 x 14336 x 4096, 66 with 32 columns).
static hipError_t launch_ffn_gemm(const void* A, const void* Wt, void* C, int32_t M, int32_t N, int32_t K,
                                  hipStream_t st) {
    const __bf16* a = (const __bf16*)A;
    const __bf16* w = (const __bf16*)Wt;
    __bf16* c = (__bf16*)C;
    const dim3 block(kGemmWaves * kWave);
    if (N >= 16384 && M <= 32) {
        constexpr int CG = 4, NT = 1;
        const dim3 grid((unsigned)((N + 16 * NT * CG - 1) / (16 * NT * CG)), (unsigned)((M + 31) / 32));
        hipLaunchKernelGGL((ffn_gemm_lds_kernel<2, NT, kGemmWaves / CG, 4>), grid, block, 0, st, a, w, c, M, N, K);
    } else if (M <= 16) {
        hipLaunchKernelGGL((ffn_gemm_kernel<1, 1, 4>), dim3((unsigned)((N + 15) / 16), (unsigned)((M + 15) / 16)),
                           block, 0, st, a, w, c, M, N, K);
    } else if (M <= 32) {
        hipLaunchKernelGGL((ffn_gemm_kernel<2, 1, 4>), dim3((unsigned)((N + 15) / 16), (unsigned)((M + 31) / 32)),
                           block, 0, st, a, w, c, M, N, K);
    } else {
        hipLaunchKernelGGL((ffn_gemm_kernel<4, 1, 4>), dim3((unsigned)((N + 15) / 16), (unsigned)((M + 63) / 64)),
                           block, 0, st, a, w, c, M, N, K);
    }
    return hipGetLastError();
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

namespace pulse {
// gather_engine.hip: whether an engine was created for shape `s` (its block size and
// staging are that shape's)
bool gs_engine_serves(const pulse_gs_engine* e, const pulse_shape& s);
}  // namespace pulse

using namespace pulse;

struct pulse_irq {
    hipStream_t cmp = nullptr, io = nullptr;
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
    // the FFN GEMMs load 16-byte pieces of rows of length D and d_ff
    PULSE_REQUIRE(n->d_ff % 8 == 0, PULSE_ERR_UNSUPPORTED);
    for (const void* p : {n->w_gate_up, n->w_down, (const void*)n->x, (const void*)n->h})
        PULSE_REQUIRE(((uintptr_t)p & 15) == 0, PULSE_ERR_INVALID_ARG);
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
    // gu [B][2F] = x [B][D] . W_gu^T
    if (launch_ffn_gemm(n.x, n.w_gate_up, n.gu, B, 2 * F, D, hs) != hipSuccess) return PULSE_ERR_HIP;
    hipLaunchKernelGGL(swiglu_kernel, dim3(grid_for((int64_t)B * F)), dim3(256), 0, hs, (const __bf16*)n.gu,
                       (__bf16*)n.h, B, F);
    if (hipGetLastError() != hipSuccess) return PULSE_ERR_HIP;
    // y [B][D] = h [B][F] . W_down^T
    if (launch_ffn_gemm(n.h, n.w_down, n.y, B, D, F, hs) != hipSuccess) return PULSE_ERR_HIP;
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
        // the engine moves blocks of the shape it was made for
        PULSE_REQUIRE(!engine || gs_engine_serves(engine, offload[m].shape), PULSE_ERR_INVALID_ARG);
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
