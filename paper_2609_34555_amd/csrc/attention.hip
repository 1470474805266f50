// attention.hip -- split-K sparse GQA decode attention over the selected
// blocks of the slot pool, for gfx950 (the attention that follows recall,
// Sec. 2.2 and Sec. 4.2.1).
//
// One wavefront owns (request r, KV head h, split s): a contiguous range of
// the request's selected blocks.  The G query heads of h share every K/V
// byte the wave reads, so the contraction is a batched GQA tile:
//   S^T[32 tokens x 16] = K[32 x 128] . Q^T[128 x 16]   (G <= 16 query columns)
//   O[16 x 128]        += P[16 x 32]  . V[32 x 128]
// both on v_mfma_f32_16x16x32_{bf16,f16}.  Each lane's MFMA operands are 16
// contiguous bytes in HBM: K is stored token-major and V channel-major, so
// neither operand needs an LDS transpose.  The S^T tile rows are assigned
// to tokens so that its accumulator layout is exactly the P operand layout
// of the P.V product (lane = query column, 8 consecutive tokens per lane
// group), so softmax probabilities never leave registers.
//
// Precision: K, V, q are consumed as stored (products exact in fp32, fp32
// accumulation).  P is split into hi + lo 16-bit parts (two MFMAs), which
// keeps the P.V product at ~2^-16 relative error instead of the 2^-9 of a
// single bf16 rounding.  Softmax is online per 32-token step in the log2
// domain.
//
// Merging the splits: a workgroup holds W waves = W consecutive splits of one
// (r, h) (W = 8 for G <= 8, else 4); they merge through LDS.  With one
// workgroup per (r, h) it writes the result directly.  Otherwise each workgroup writes one partial (m, l, O) to
// the workspace and a combine kernel merges those few partials, one thread
// per output element, with independent loads.  (Merging in the last workgroup
// to finish instead needs a device-scope release per workgroup, an L2
// write-back on gfx950 measured at about 9 ns per workgroup, plus a merge on
// the kernel's tail and counters that start at zero in the workspace: it would
// save well under the combine launch's 3.6 us.)
#include "pulse_internal.h"

namespace pulse {

#ifndef PULSE_ATTN_TARGET_WAVES
#define PULSE_ATTN_TARGET_WAVES 2048
#endif
constexpr int kCombineThreads = kHeadDim;

// Waves per workgroup (attn_waves): 8 while the LDS merge buffer (waves x G x
// 128 floats) stays within 32 KiB, else 4.  Fewer, wider workgroups leave
// fewer partials for the combine kernel.

template <int DT>
struct Mfma;
template <>
struct Mfma<PULSE_BF16> {
    typedef bf16x8 vec;
    typedef __bf16 elem;
    __device__ static inline f32x4 mac(vec a, vec b, f32x4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
    }
    __device__ static inline void split(float p, __bf16& hi, __bf16& lo) {
        hi = (__bf16)p;
        lo = (__bf16)(p - (float)hi);
    }
};
template <>
struct Mfma<PULSE_F16> {
    typedef f16x8 vec;
    typedef _Float16 elem;
    __device__ static inline f32x4 mac(vec a, vec b, f32x4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
    }
    __device__ static inline void split(float p, _Float16& hi, _Float16& lo) {
        hi = (_Float16)p;
        lo = (_Float16)(p - (float)hi);
    }
};

template <int DT>
__device__ inline typename Mfma<DT>::vec load_vec(const uint16_t* p) {
    return __builtin_bit_cast(typename Mfma<DT>::vec, *reinterpret_cast<const u32x4*>(p));
}
template <int DT>
__device__ inline typename Mfma<DT>::vec zero_vec() {
    return __builtin_bit_cast(typename Mfma<DT>::vec, u32x4{0, 0, 0, 0});
}

// Attention of one wave over entries [e0, e0 + ne) of request r, KV head h;
// j_lane is the selected block of entry e0 + lane (loaded by the caller).
// Leaves the running max (log2 domain) and the lane-group-reduced sum for
// query column `col` in m_run / l_run, and O rows g = 4*grp + v in acc.
template <int DT, int BS>
__device__ inline void attend_split(const uint16_t* __restrict__ q, const uint16_t* __restrict__ pool,
                                    int32_t n_slots, const int32_t* __restrict__ table, int32_t max_blocks,
                                    int32_t j_lane, int ctx, int32_t Hq, int32_t Hkv, int32_t G,
                                    int r, int h, int e0, int ne, float scale_log2, int32_t* status, int lane,
                                    float& m_run, float& l_run, f32x4 (&acc)[8]) {
    using M = Mfma<DT>;
    using vec = typename M::vec;
    const int col = lane & 15;  // MFMA column: query head (QK^T), channel (PV)
    const int grp = lane >> 4;  // lane group: 8-channel / 8-token slice
#pragma unroll
    for (int t = 0; t < 8; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
    m_run = -INFINITY;
    l_run = 0.f;
    if (ne <= 0) return;
    // entry metadata, one entry per lane (ne <= 64)
    const int64_t n_r = ((int64_t)ctx + BS - 1) / BS;
    int my_slot = -1, my_nv = 0;
    if (lane < ne) {
        const int32_t j = j_lane;
        if (j >= 0 && j < n_r && j < max_blocks) {
            const int32_t sl = table[(size_t)r * max_blocks + j];
            if (sl >= 0 && sl < n_slots) {
                my_slot = sl;
                const int64_t v = (int64_t)ctx - (int64_t)j * BS;
                my_nv = v >= BS ? BS : (int)v;
            }
        }
        if (my_slot < 0) report(status, PULSE_ERR_BAD_INDEX);
    }
    // Q^T operand: lane holds q[g = col][8 channels of slice grp + 32 kc]
    vec qb[4];
    {
        const uint16_t* qr = q + ((size_t)r * Hq + (size_t)h * G + col) * kHeadDim + grp * 8;
#pragma unroll
        for (int kc = 0; kc < 4; ++kc) qb[kc] = col < G ? load_vec<DT>(qr + 32 * kc) : zero_vec<DT>();
    }
    const size_t E = (size_t)2 * Hkv * BS * kHeadDim;
    const size_t k_head = (size_t)h * BS * kHeadDim;
    const size_t v_head = (size_t)Hkv * BS * kHeadDim + (size_t)h * kHeadDim * BS;
    const int tokens = ne * BS;

    // K and V operand loads of one 32-token step starting at sequence token t0
    // K: MFMA row m = col maps to token 8*(col/4) + 4*sub + col%4;
    // V: lane group grp holds tokens 8*grp .. 8*grp+7 of channel col + 16*tile.
    auto load_k = [&](int t0, vec (&ka)[2][4]) {
        const int ka_seq = t0 + 8 * (col >> 2);
        const int ka_e = ka_seq / BS;
        const int ka_slot = __shfl(my_slot, ka_e < ne ? ka_e : 0);
        const int ka_nv = __shfl(my_nv, ka_e < ne ? ka_e : 0);
#pragma unroll
        for (int sub = 0; sub < 2; ++sub) {
            const int row = ka_seq % BS + 4 * sub + (col & 3);
            const bool ok = ka_e < ne && ka_slot >= 0 && row < ka_nv;
            const uint16_t* kp = pool + (size_t)(ok ? ka_slot : 0) * E + k_head + (size_t)row * kHeadDim + grp * 8;
#pragma unroll
            for (int kc = 0; kc < 4; ++kc) ka[sub][kc] = ok ? load_vec<DT>(kp + 32 * kc) : zero_vec<DT>();
        }
    };
    auto load_v = [&](int t0, vec (&vb)[8]) {
        const int pv_seq = t0 + 8 * grp;
        const int pv_e = pv_seq / BS;
        const int pv_slot = __shfl(my_slot, pv_e < ne ? pv_e : 0);
        const bool pv_ok = pv_e < ne && pv_slot >= 0;
        const uint16_t* vp = pool + (size_t)(pv_ok ? pv_slot : 0) * E + v_head + (size_t)col * BS + pv_seq % BS;
#pragma unroll
        for (int t = 0; t < 8; ++t) vb[t] = pv_ok ? load_vec<DT>(vp + (size_t)16 * t * BS) : zero_vec<DT>();
    };

    // One 32-token step at a time: K is loaded first, V once the S tile is issued, so
    // the V loads overlap the softmax and fewer operands are live (143 VGPRs, 3 waves
    // per SIMD).  The other resident waves hide the load latency.  Measured slower:
    // loading K and V together (154 VGPRs; 2-5%), prefetching the next step into
    // registers as well (223 VGPRs; another 1-2%), and, for splits of two steps,
    // issuing all four loads before the first product (177 VGPRs; 11% slower on
    // 8 requests x 2048 selected tokens).
#pragma unroll 1
    for (int t0 = 0; t0 < tokens; t0 += kChunkTokens) {
        vec ka[2][4], vb[8];
        load_k(t0, ka);
        const int pv_seq = t0 + 8 * grp;
        const int pv_e = pv_seq / BS;
        const int pv_slot = __shfl(my_slot, pv_e < ne ? pv_e : 0);
        const int pv_nv = __shfl(my_nv, pv_e < ne ? pv_e : 0);
        const int pv_row = pv_seq % BS;
        const bool pv_ok = pv_e < ne && pv_slot >= 0;
        // --- S^T = K . Q^T
        f32x4 s1 = {0.f, 0.f, 0.f, 0.f}, s2 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kc = 0; kc < 4; ++kc) {
            s1 = M::mac(ka[0][kc], qb[kc], s1);
            s2 = M::mac(ka[1][kc], qb[kc], s2);
        }
        load_v(t0, vb);
        // lane (col, grp) now holds query col, tokens pv_seq + 0..7
        float x[8];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            x[i] = s1[i] * scale_log2;
            x[4 + i] = s2[i] * scale_log2;
        }
        float cm = -INFINITY;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            if (!pv_ok || pv_row + i >= pv_nv) x[i] = -INFINITY;
            cm = fmaxf(cm, x[i]);
        }
        cm = fmaxf(cm, __shfl_xor(cm, 16));
        cm = fmaxf(cm, __shfl_xor(cm, 32));
        const float m_new = fmaxf(m_run, cm);
        const float m_use = m_new == -INFINITY ? 0.f : m_new;
        const float alpha = exp2f(m_run - m_use);
        float psum = 0.f;
        vec ph, pl;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const float p = exp2f(x[i] - m_use);
            psum += p;
            typename M::elem hi, lo;
            M::split(p, hi, lo);
            ph[i] = hi;
            pl[i] = lo;
        }
        l_run = l_run * alpha + psum;
        m_run = m_new;
        // rescale accumulator rows g' = 4*grp + v by alpha of query g'
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const float av = __shfl(alpha, 4 * grp + v);
#pragma unroll
            for (int t = 0; t < 8; ++t) acc[t][v] *= av;
        }
        // --- O += P . V  (hi and lo parts of P)
#pragma unroll
        for (int t = 0; t < 8; ++t) {
            acc[t] = M::mac(ph, vb[t], acc[t]);
            acc[t] = M::mac(pl, vb[t], acc[t]);
        }
    }
    l_run += __shfl_xor(l_run, 16);
    l_run += __shfl_xor(l_run, 32);
}

// grid = (workgroups per (r, h), Hkv, B); W waves per workgroup, wave w owns
// split W*blockIdx.x + w of eps entries.  Dynamic LDS: O [W][G][128] floats
// then (m, l) [W][G] float2.
template <int DT, int BS, int W>
__global__ __launch_bounds__(W * kWave) void attn_splitk_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ pool, int32_t n_slots,
    const int32_t* __restrict__ table, int32_t max_blocks, const int32_t* __restrict__ sel_idx,
    const int32_t* __restrict__ sel_cnt, int32_t k_max, const int32_t* __restrict__ ctx_len, int32_t Hq,
    int32_t Hkv, int32_t G, int32_t eps, int32_t n_wg, float scale_log2, float* __restrict__ ws_o,
    float2* __restrict__ ws_ml, float* __restrict__ out, float* __restrict__ lse, int32_t* status) {
    extern __shared__ float smem[];
    constexpr int kThreads = W * kWave;
    float* s_o = smem;                                                           // [W][G][128]
    float2* s_ml = reinterpret_cast<float2*>(smem + W * G * kHeadDim);  // [W][G]
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int col = lane & 15, grp = lane >> 4;
    const int wg = blockIdx.x, h = blockIdx.y, r = blockIdx.z;
    float* out_rh = out + ((size_t)r * Hq + (size_t)h * G) * kHeadDim;
    float* lse_rh = lse ? lse + (size_t)r * Hq + (size_t)h * G : nullptr;

    // this wave's selected blocks (one per lane) are loaded with the count they
    // depend on, not after it: one memory round trip fewer before the first K load
    const int s = wg * W + wave;
    const int e0 = s * eps;
    const int32_t j_lane = (lane < eps && e0 + lane < k_max) ? sel_idx[(size_t)r * k_max + e0 + lane] : -1;
    int32_t cnt = sel_cnt[r];
    if (cnt < 0 || cnt > k_max) {
        if (tid == 0) report(status, PULSE_ERR_BAD_INDEX);
        cnt = 0;
    }
    const int ns = (cnt + eps - 1) / eps;                // non-empty splits of (r, h)
    const int nwg = (ns + W - 1) / W;  // workgroups with work
    if (wg >= nwg) {
        if (cnt == 0 && wg == 0) {  // empty selection: out = 0, lse = -inf
            for (int i = tid; i < G * kHeadDim; i += kThreads) out_rh[i] = 0.f;
            if (lse_rh && tid < G) lse_rh[tid] = -INFINITY;
        }
        return;
    }
    const int ne = min(e0 + eps, cnt) - e0;
    float m_run, l_run;
    f32x4 acc[8];
    attend_split<DT, BS>(q, pool, n_slots, table, max_blocks, j_lane, ctx_len[r], Hq, Hkv, G, r,
                         h, e0, ne, scale_log2, status, lane, m_run, l_run, acc);
    // wave partials to LDS
    if (grp == 0 && col < G) s_ml[wave * G + col] = make_float2(m_run, l_run);
#pragma unroll
    for (int v = 0; v < 4; ++v) {
        const int g = 4 * grp + v;
        if (g < G) {
            float* o = s_o + (wave * G + g) * kHeadDim + col;
#pragma unroll
            for (int t = 0; t < 8; ++t) o[16 * t] = acc[t][v];
        }
    }
    __syncthreads();
    // merge the W waves: thread handles outputs (g, c) = (idx / 128, idx % 128)
    const size_t unit = ((size_t)r * Hkv + h) * n_wg + wg;
    for (int idx = tid; idx < G * kHeadDim; idx += kThreads) {
        const int g = idx / kHeadDim, c = idx % kHeadDim;
        float Mx = -INFINITY;
#pragma unroll
        for (int w = 0; w < W; ++w) Mx = fmaxf(Mx, s_ml[w * G + g].x);
        float L = 0.f, a = 0.f;
        if (Mx != -INFINITY) {
#pragma unroll
            for (int w = 0; w < W; ++w) {
                const float2 ml = s_ml[w * G + g];
                const float wt = ml.x == -INFINITY ? 0.f : exp2f(ml.x - Mx);
                L += ml.y * wt;
                a += s_o[(w * G + g) * kHeadDim + c] * wt;
            }
        }
        if (nwg == 1) {
            out_rh[idx] = Mx == -INFINITY ? 0.f : a / L;
            if (lse_rh && c == 0) lse_rh[g] = Mx == -INFINITY ? -INFINITY : (Mx + log2f(L)) * 0.69314718055994531f;
        } else {
            ws_o[unit * G * kHeadDim + idx] = a;
            if (c == 0) ws_ml[unit * G + g] = make_float2(Mx, L);
        }
    }
}

// Merge the workgroup partials of one (request, KV head, query head):
// grid = (G, Hkv, B), 128 threads, thread c owns output channel c.  Partials
// are read 8 at a time (16 independent loads per thread) and merged online.
// Requests whose selection fits one workgroup were finished by the attention
// kernel.
__global__ __launch_bounds__(kCombineThreads) void attn_combine_kernel(
    const float* __restrict__ ws_o, const float2* __restrict__ ws_ml, const int32_t* __restrict__ sel_cnt,
    int32_t k_max, int32_t Hq, int32_t Hkv, int32_t G, int32_t eps, int32_t n_wg, int32_t waves,
    float* __restrict__ out, float* __restrict__ lse) {
    const int c = threadIdx.x, g = blockIdx.x, h = blockIdx.y, r = blockIdx.z;
    const size_t u0 = ((size_t)r * Hkv + h) * n_wg;
    const float2* ml = ws_ml + u0 * G + g;                  // stride G
    const float* po = ws_o + (u0 * G + g) * kHeadDim + c;   // stride G * 128
    // the first 8 partials are loaded before the request's workgroup count is
    // known (n_wg bounds it); entries past that count are discarded below
    float2 mlv[8];
    float ov[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        mlv[i] = i < n_wg ? ml[(size_t)i * G] : make_float2(-INFINITY, 0.f);
        ov[i] = i < n_wg ? po[(size_t)i * G * kHeadDim] : 0.f;
    }
    int32_t cnt = sel_cnt[r];
    if (cnt < 0 || cnt > k_max) cnt = 0;
    const int ns = (cnt + eps - 1) / eps;
    const int nwg = (ns + waves - 1) / waves;
    if (nwg <= 1) return;
    float m_run = -INFINITY, L = 0.f, a = 0.f;
    for (int w0 = 0; w0 < nwg; w0 += 8) {
        if (w0 > 0) {
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const bool ok = w0 + i < nwg;
                mlv[i] = ok ? ml[(size_t)(w0 + i) * G] : make_float2(-INFINITY, 0.f);
                ov[i] = ok ? po[(size_t)(w0 + i) * G * kHeadDim] : 0.f;
            }
        } else {
#pragma unroll
            for (int i = 0; i < 8; ++i)
                if (i >= nwg) {  // not written by this call
                    mlv[i] = make_float2(-INFINITY, 0.f);
                    ov[i] = 0.f;
                }
        }
        float cm = m_run;
#pragma unroll
        for (int i = 0; i < 8; ++i) cm = fmaxf(cm, mlv[i].x);
        if (cm == -INFINITY) continue;
        const float alpha = m_run == -INFINITY ? 0.f : exp2f(m_run - cm);
        L *= alpha;
        a *= alpha;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const float wt = mlv[i].x == -INFINITY ? 0.f : exp2f(mlv[i].x - cm);
            L += mlv[i].y * wt;
            a += ov[i] * wt;
        }
        m_run = cm;
    }
    float* out_rg = out + ((size_t)r * Hq + (size_t)h * G + g) * kHeadDim;
    out_rg[c] = m_run == -INFINITY ? 0.f : a / L;
    if (lse && c == 0)
        lse[(size_t)r * Hq + (size_t)h * G + g] =
            m_run == -INFINITY ? -INFINITY : (m_run + log2f(L)) * 0.69314718055994531f;
}

AttnPlan attn_plan(int32_t B, int32_t Hkv, int32_t k_max, int32_t bs) {
    // entries per 32-token step; a split covers >= 2 steps, <= 64 entries
    const int32_t step = bs >= kChunkTokens ? 1 : kChunkTokens / bs;
    const int64_t units = (int64_t)B * Hkv;
    const int64_t target_waves = PULSE_ATTN_TARGET_WAVES;  // one round at 2 resident waves per SIMD on 256 CUs
    int64_t want = units > 0 ? (target_waves + units - 1) / units : 1;
    int64_t min_entries = (bs >= 2 * kChunkTokens) ? 1 : (2 * kChunkTokens) / bs;
    int64_t max_split = (k_max + min_entries - 1) / min_entries;
    if (want > max_split) want = max_split;
    if (want < 1) want = 1;
    int64_t eps = (k_max + want - 1) / want;
    eps = ((eps + step - 1) / step) * step;
    if (eps > 64) eps = 64;
    if (eps < 1) eps = 1;
    AttnPlan p;
    p.entries_per_split = (int32_t)eps;
    p.n_split = (int32_t)((k_max + eps - 1) / eps);
    return p;
}

// `done` (optional): the kernel's stop event, carried by the launch.
template <int DT, int BS, int W>
static void launch_attn_t(dim3 grid, size_t lds, hipStream_t st, hipEvent_t done, const void* q, const void* pool,
                          int32_t n_slots, const int32_t* table, int32_t max_blocks, const int32_t* sel_idx,
                          const int32_t* sel_cnt, int32_t k_max, const int32_t* ctx_len, int32_t Hq, int32_t Hkv,
                          int32_t G, int32_t eps, int32_t n_wg, float scale_log2, float* ws_o, float2* ws_ml,
                          float* out, float* lse, int32_t* status) {
    launch_timed(attn_splitk_kernel<DT, BS, W>, grid, dim3(W * kWave), (uint32_t)lds, st, nullptr, done,
                 (const uint16_t*)q, (const uint16_t*)pool, n_slots, table, max_blocks, sel_idx, sel_cnt, k_max,
                 ctx_len, Hq, Hkv, G, eps, n_wg, scale_log2, ws_o, ws_ml, out, lse, status);
}

hipError_t launch_attention(const pulse_shape& s, const void* q, const void* pool, int32_t n_slots,
                            const int32_t* table, int32_t max_blocks, const int32_t* sel_idx, const int32_t* sel_cnt,
                            int32_t k_max, const int32_t* ctx_len, int32_t B, float sm_scale, float* out, float* lse,
                            float* ws_o, float2* ws_ml, int32_t* status, hipStream_t st, hipEvent_t split_done,
                            hipEvent_t done) {
    if (B == 0) return hipSuccess;
    const int32_t Hkv = s.num_kv_heads, Hq = s.num_q_heads, G = Hq / Hkv;
    const AttnPlan p = attn_plan(B, Hkv, k_max, s.block_size);
    const int W = attn_waves(G);
    const int32_t n_wg = (p.n_split + W - 1) / W;
    dim3 grid((unsigned)n_wg, (unsigned)Hkv, (unsigned)B);
    const size_t lds = sizeof(float) * W * G * kHeadDim + sizeof(float2) * W * G;
    const float scale_log2 = sm_scale * 1.4426950408889634f;
    // stop event of the split-K kernel: split_done, or `done` when no combine follows it
    const hipEvent_t splitk_stop = split_done ? split_done : (n_wg <= 1 ? done : nullptr);
#define PULSE_ATTN(DT, BS, W)                                                                                        \
    launch_attn_t<DT, BS, W>(grid, lds, st, splitk_stop, q, pool, n_slots, table, max_blocks, sel_idx, sel_cnt,     \
                             k_max, ctx_len,                                                                        \
                             Hq, Hkv, G, p.entries_per_split, n_wg, scale_log2, ws_o, ws_ml, out, lse, status)
#define PULSE_ATTN_W(DT, BS) \
    if (W == 8) PULSE_ATTN(DT, BS, 8); else PULSE_ATTN(DT, BS, 4)
    if (s.dtype == PULSE_BF16) {
        if (s.block_size == 16) PULSE_ATTN_W(PULSE_BF16, 16);
        else if (s.block_size == 32) PULSE_ATTN_W(PULSE_BF16, 32);
        else PULSE_ATTN_W(PULSE_BF16, 64);
    } else {
        if (s.block_size == 16) PULSE_ATTN_W(PULSE_F16, 16);
        else if (s.block_size == 32) PULSE_ATTN_W(PULSE_F16, 32);
        else PULSE_ATTN_W(PULSE_F16, 64);
    }
#undef PULSE_ATTN_W
#undef PULSE_ATTN
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (n_wg <= 1) return (done && split_done) ? hipEventRecord(done, st) : hipSuccess;
    launch_timed(attn_combine_kernel, dim3((unsigned)G, (unsigned)Hkv, (unsigned)B), dim3(kCombineThreads), 0u, st,
                 nullptr, done, (const float*)ws_o, (const float2*)ws_ml, sel_cnt, k_max, Hq, Hkv, G,
                 p.entries_per_split, n_wg, W, out, lse);
    return hipGetLastError();
}

}  // namespace pulse
