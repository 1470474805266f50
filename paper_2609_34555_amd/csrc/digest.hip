// digest.hip -- per-block key digests of one KV head and the query-digest
// score of SoloHead selection, for gfx950.
//
// Digest (Sec. 2.1 Quest-style block digests; Sec. 4.4.1 digests kept for
// one KV head per layer): elementwise min and max of the head's keys over
// the valid tokens of each block, exact, in the KV dtype.
//
// Score (Sec. 4.4.1, query-digest score): for block b and the G query heads
// of the solo KV head,
//   s[b] = (1/G) * sum_g sum_c max(q_gc * mn_bc, q_gc * mx_bc).
// Since mn <= mx, max(q*mn, q*mx) = q * (q >= 0 ? mx : mn) exactly, so each
// channel costs one bit-select and half of a packed dot product.  Both
// kernels are HBM-bound streams over the digests (512 B per block); one
// 16-lane group owns one block, each lane 8 channels (one 16-byte load).
#include "pulse_internal.h"

namespace pulse {

// Largest r in [0, B) with blk_off[r] <= b (blk_off is non-decreasing).
__device__ inline int find_request(const int64_t* blk_off, int32_t B, int64_t b) {
    int lo = 0, hi = B;
    while (hi - lo > 1) {
        int mid = (lo + hi) >> 1;
        if (blk_off[mid] <= b) lo = mid; else hi = mid;
    }
    return lo;
}

// One wave per block: lane = (token group tg in 0..3, 8-channel slice).
__global__ __launch_bounds__(256) void build_digests_kernel(const uint16_t* __restrict__ kv,
                                                            const int64_t* __restrict__ blk_off,
                                                            const int32_t* __restrict__ ctx_len, int32_t B,
                                                            int64_t total_blocks, int32_t Hkv, int32_t bs,
                                                            int32_t kv_head, uint16_t* __restrict__ digests,
                                                            int32_t* status) {
    const int lane = threadIdx.x & 63;
    const int64_t b = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (b >= total_blocks) return;
    const int c8 = (lane & 15) * 8;
    const int tg = lane >> 4;
    u32x4* dst = reinterpret_cast<u32x4*>(digests + b * 2 * kHeadDim);
    const int r = find_request(blk_off, B, b);
    const int64_t j = b - blk_off[r];
    const int64_t nv64 = (int64_t)ctx_len[r] - j * bs;
    const int nv = nv64 >= bs ? bs : (int)nv64;
    if (j < 0 || b >= blk_off[r + 1] || nv <= 0) {
        if (lane == 0) report(status, PULSE_ERR_BAD_INDEX);
        if (tg == 0) {
            dst[c8 / 8] = u32x4{0, 0, 0, 0};
            dst[16 + c8 / 8] = u32x4{0, 0, 0, 0};
        }
        return;
    }
    const size_t E = (size_t)2 * Hkv * bs * kHeadDim;
    const uint16_t* K = kv + (size_t)b * E + (size_t)kv_head * bs * kHeadDim;
    uint32_t mn[8], mx[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) { mn[i] = 0xFFFFu; mx[i] = 0u; }
    for (int t = tg; t < nv; t += 4) {
        u32x4 v = *reinterpret_cast<const u32x4*>(K + (size_t)t * kHeadDim + c8);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            uint32_t k = key16((v[i >> 1] >> (16 * (i & 1))) & 0xFFFFu);
            mn[i] = min(mn[i], k);
            mx[i] = max(mx[i], k);
        }
    }
#pragma unroll
    for (int off = 16; off <= 32; off <<= 1)
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            mn[i] = min(mn[i], (uint32_t)__shfl_xor((int)mn[i], off));
            mx[i] = max(mx[i], (uint32_t)__shfl_xor((int)mx[i], off));
        }
    if (tg == 0) {
        u32x4 omn, omx;
#pragma unroll
        for (int p = 0; p < 4; ++p) {
            omn[p] = unkey16(mn[2 * p]) | (unkey16(mn[2 * p + 1]) << 16);
            omx[p] = unkey16(mx[2 * p]) | (unkey16(mx[2 * p + 1]) << 16);
        }
        dst[c8 / 8] = omn;
        dst[16 + c8 / 8] = omx;
    }
}

template <int DT>
__device__ inline float dot2(uint32_t a, uint32_t b, float acc) {
    if constexpr (DT == PULSE_BF16)
        return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a), __builtin_bit_cast(bf16x2, b),
                                               acc, false);
    else
        return __builtin_amdgcn_fdot2(__builtin_bit_cast(f16x2, a), __builtin_bit_cast(f16x2, b), acc, false);
}

// Two shapes of the score kernel, chosen by the number of digests read:
// small sets (up to kScoreLargeBlocks) take one 16-block iteration per
// workgroup, so more workgroups share the short stream; large ones take two
// iterations with non-temporal loads, which keep the once-read digests from
// displacing cached lines.  Both measured faster than the other's setting at
// their sizes (and than 4 or more iterations, or a grid-stride form).
constexpr int64_t kScoreLargeBlocks = 65536;

template <bool NT>
__device__ inline u32x4 score_load(const u32x4* p) {
    if constexpr (NT) return __builtin_nontemporal_load(p);
    return *p;
}

// Largest r in [0, B) with off[r] <= b, over an LDS copy of blk_off.
__device__ inline int find_request_lds(const int64_t* off, int32_t B, int64_t b) {
    int lo = 0, hi = B;
    while (hi - lo > 1) {
        int mid = (lo + hi) >> 1;
        if (off[mid] <= b) lo = mid; else hi = mid;
    }
    return lo;
}

// 256 threads = 16 groups of 16 lanes; group gi handles blocks
// base + gi + 16*it so that consecutive groups stream consecutive digests.
// blockIdx.y selects the scoring KV head when several heads score at once
// (headwise selection); with one head it is `solo`.  blk_off is staged in LDS
// so the request of a block costs no dependent global loads.
template <int DT, int G, int ITERS, bool NT>
__global__ __launch_bounds__(256) void score_kernel(const uint16_t* __restrict__ q,
                                                    const uint16_t* __restrict__ digests,
                                                    const int64_t* __restrict__ blk_off, int32_t B,
                                                    int64_t total_blocks, int32_t Hq, int32_t solo,
                                                    int32_t n_sink, int32_t n_local, float* __restrict__ scores,
                                                    ReleaseArgs rel, int32_t do_release) {
    extern __shared__ int64_t s_off[];
    const int head = gridDim.y > 1 ? (int)blockIdx.y : solo;
    digests += (size_t)blockIdx.y * total_blocks * 2 * kHeadDim;
    scores += (size_t)blockIdx.y * total_blocks;
    const int sub = threadIdx.x & 15;
    const int gi = threadIdx.x >> 4;
    const int c8 = sub * 8;
    const int64_t base = (int64_t)blockIdx.x * (16 * ITERS) + gi;
    // digest loads first: their addresses do not depend on the request
    u32x4 dmn[ITERS], dmx[ITERS];
#pragma unroll
    for (int it = 0; it < ITERS; ++it) {
        const int64_t b = base + 16 * it;
        if (b < total_blocks) {
            const u32x4* dg = reinterpret_cast<const u32x4*>(digests + (size_t)b * 2 * kHeadDim);
            dmn[it] = score_load<NT>(dg + sub);
            dmx[it] = score_load<NT>(dg + 16 + sub);
        }
    }
    // Up to G = 6, the query rows of the request that holds the first block if
    // every request had the same length (exact for equal contexts) are loaded
    // with the digests, and a wrong guess is reloaded once the offsets are
    // known.  Larger groups load them then: holding G x 4 more registers across
    // the barrier would take the kernel past 64 VGPRs (8 waves per SIMD).
    constexpr bool kEarlyQ = G <= 6;
    uint32_t qp[G][4];
    auto load_q = [&](int rq) {
        const uint16_t* qr = q + ((size_t)rq * Hq + (size_t)head * G) * kHeadDim + c8;
#pragma unroll
        for (int g = 0; g < G; ++g) {
            const u32x4 v = *reinterpret_cast<const u32x4*>(qr + (size_t)g * kHeadDim);
#pragma unroll
            for (int p = 0; p < 4; ++p) qp[g][p] = v[p];
        }
    };
    int q_r = -1;
    if constexpr (kEarlyQ) {
        q_r = base < total_blocks ? (int)(base * B / total_blocks) : 0;
        q_r = q_r < B ? q_r : B - 1;
        load_q(q_r);
    }
    // the previous step's release, on the side (independent of the scores)
    if (do_release && blockIdx.y == 0)
        release_entries(rel, (int64_t)blockIdx.x * 256 + threadIdx.x, (int64_t)gridDim.x * 256, true);
    for (int i = threadIdx.x; i <= B; i += 256) s_off[i] = blk_off[i];
    __syncthreads();
    int64_t r_lo = 0, r_hi = 0;
#pragma unroll
    for (int it = 0; it < ITERS; ++it) {
        const int64_t b = base + 16 * it;
        if (b >= total_blocks) break;
        if (b >= r_hi || b < r_lo) {
            const int cur_r = find_request_lds(s_off, B, b);
            r_lo = s_off[cur_r];
            r_hi = s_off[cur_r + 1];
            if (cur_r != q_r) {
                load_q(cur_r);
                q_r = cur_r;
            }
        }
        const int64_t j = b - r_lo;
        const int64_t n = r_hi - r_lo;
        if (j < n_sink || j >= n - n_local) continue;  // forced blocks are not scored
        float acc = 0.f;
#pragma unroll
        for (int g = 0; g < G; ++g)
#pragma unroll
            for (int p = 0; p < 4; ++p) {
                // 0xFFFF in each half whose q is non-negative (sign bit clear), formed
                // here rather than kept: G x 4 fewer live registers
                const uint32_t qm = ~(((qp[g][p] & 0x80008000u) >> 15) * 0xFFFFu);
                const uint32_t sel = (dmx[it][p] & qm) | (dmn[it][p] & ~qm);
                acc = dot2<DT>(qp[g][p], sel, acc);
            }
#pragma unroll
        for (int off = 1; off < 16; off <<= 1) acc += __shfl_xor(acc, off);
        if (sub == 0) scores[b] = acc / (float)G;
    }
}

hipError_t launch_build_digests(const pulse_shape& s, const void* kv, const int64_t* blk_off,
                                const int32_t* ctx_len, int32_t B, int64_t total_blocks, int32_t kv_head,
                                void* digests, int32_t* status, hipStream_t st) {
    if (total_blocks == 0) return hipSuccess;
    dim3 grid((unsigned)((total_blocks + 3) / 4));
    hipLaunchKernelGGL(build_digests_kernel, grid, dim3(256), 0, st, (const uint16_t*)kv, blk_off, ctx_len, B,
                       total_blocks, s.num_kv_heads, s.block_size, kv_head, (uint16_t*)digests, status);
    return hipGetLastError();
}

template <int DT, int G>
static void launch_score_t(int32_t heads, hipStream_t st, hipEvent_t ev0, hipEvent_t ev1, const void* q,
                           const void* digests, const int64_t* blk_off, int32_t B, int64_t total, int32_t Hq,
                           int32_t solo, int32_t n_sink, int32_t n_local, float* scores, const ReleaseArgs* rel) {
    const uint32_t lds = (uint32_t)(sizeof(int64_t) * ((size_t)B + 1));
    const ReleaseArgs ra = rel ? *rel : ReleaseArgs{};
    const int32_t dr = rel != nullptr;
    if (total * heads > kScoreLargeBlocks) {
        const dim3 grid((unsigned)((total + 31) / 32), (unsigned)heads);
        launch_timed(score_kernel<DT, G, 2, true>, grid, dim3(256), lds, st, ev0, ev1, (const uint16_t*)q,
                     (const uint16_t*)digests, blk_off, B, total, Hq, solo, n_sink, n_local, scores, ra, dr);
    } else {
        const dim3 grid((unsigned)((total + 15) / 16), (unsigned)heads);
        launch_timed(score_kernel<DT, G, 1, false>, grid, dim3(256), lds, st, ev0, ev1, (const uint16_t*)q,
                     (const uint16_t*)digests, blk_off, B, total, Hq, solo, n_sink, n_local, scores, ra, dr);
    }
}

template <int DT>
static void launch_score_dt(int G, int32_t heads, hipStream_t st, hipEvent_t ev0, hipEvent_t ev1, const void* q,
                            const void* digests, const int64_t* blk_off, int32_t B, int64_t total, int32_t Hq,
                            int32_t solo, int32_t n_sink, int32_t n_local, float* scores, const ReleaseArgs* rel) {
#define PULSE_SCORE_CASE(g)                                                                                    \
    case g:                                                                                                    \
        launch_score_t<DT, g>(heads, st, ev0, ev1, q, digests, blk_off, B, total, Hq, solo, n_sink, n_local,  \
                              scores, rel);                                                                    \
        break;
    switch (G) {
        PULSE_SCORE_CASE(1) PULSE_SCORE_CASE(2) PULSE_SCORE_CASE(3) PULSE_SCORE_CASE(4)
        PULSE_SCORE_CASE(5) PULSE_SCORE_CASE(6) PULSE_SCORE_CASE(7) PULSE_SCORE_CASE(8)
        PULSE_SCORE_CASE(9) PULSE_SCORE_CASE(10) PULSE_SCORE_CASE(11) PULSE_SCORE_CASE(12)
        PULSE_SCORE_CASE(13) PULSE_SCORE_CASE(14) PULSE_SCORE_CASE(15) PULSE_SCORE_CASE(16)
        default: break;
    }
#undef PULSE_SCORE_CASE
}

hipError_t launch_score(const pulse_shape& s, const void* q, const void* digests, const int64_t* blk_off,
                        int32_t B, int64_t total_blocks, int32_t solo, int32_t n_sink, int32_t n_local,
                        float* scores, int32_t heads, hipStream_t st, const ReleaseArgs* rel, hipEvent_t start,
                        hipEvent_t stop) {
    if (total_blocks == 0) {  // no blocks: no recall to release either; requested events become markers
        hipError_t e = start ? hipEventRecord(start, st) : hipSuccess;
        if (e == hipSuccess && stop) e = hipEventRecord(stop, st);
        return e;
    }
    const int G = s.num_q_heads / s.num_kv_heads;
    if (s.dtype == PULSE_BF16)
        launch_score_dt<PULSE_BF16>(G, heads, st, start, stop, q, digests, blk_off, B, total_blocks, s.num_q_heads,
                                    solo, n_sink, n_local, scores, rel);
    else
        launch_score_dt<PULSE_F16>(G, heads, st, start, stop, q, digests, blk_off, B, total_blocks, s.num_q_heads,
                                   solo, n_sink, n_local, scores, rel);
    return hipGetLastError();
}

}  // namespace pulse
