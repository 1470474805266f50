// select.hip -- SoloHead top-k block selection and the set difference
// against the GPU-resident hot set, for gfx950.
//
// Selection (Sec. 4.4.1, budget split Sec. 5 setup): per request, the first
// n_sink and last n_local blocks are forced; k' = min(max(k_mid,0), #middle)
// middle blocks of highest score are chosen, equal scores in ascending
// block order; the set is emitted ascending.  One 1024-thread workgroup per
// request:
//   1. radix select (8-bit passes over an LDS copy of the keys, starting at the
//      highest byte in which the keys differ) of the k'-th largest
//      order-preserving key of the fp32 scores -> threshold T and the number
//      need_eq of keys equal to T that are taken;
//   2. one ordered pass over the blocks in tiles of 1024 with wave ballots and
//      a cross-wave LDS scan: block j is chosen if key > T, or key == T and
//      fewer than need_eq equal keys precede it -- this is exactly the
//      lowest-index tie rule.
// With a block table the same pass also takes the set difference (Sec. 2.2:
// selected blocks whose table entry is -1 are missing) and writes the recall
// plan: missing blocks in listed order, their count and their run count.
#include "pulse_internal.h"

namespace pulse {

constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / kWave;
constexpr int kKeyCache = 8192;  // middle-block keys kept in LDS (32 KiB); larger requests read L2

__device__ inline uint64_t lanemask_lt() {
    const int lane = threadIdx.x & 63;
    return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

// grid = (B, heads): blockIdx.x = request, blockIdx.y = selecting head slot
// (always 0 for SoloHead; 0..Hkv-1 for headwise selection, whose per-head
// scores, selections and plans are stacked along the head dimension).
__global__ __launch_bounds__(kSelThreads) void select_kernel(
    const int64_t* __restrict__ blk_off, int32_t B, int64_t total_blocks, const float* __restrict__ scores,
    const int32_t* __restrict__ k_mid, int32_t n_sink, int32_t n_local, int32_t k_max, int32_t* __restrict__ sel_idx,
    int32_t* __restrict__ sel_cnt, const int32_t* __restrict__ table, int32_t max_blocks, int32_t n_slots,
    const int32_t* __restrict__ free_head, int32_t* __restrict__ miss_list, int32_t* __restrict__ miss_cnt,
    int32_t* __restrict__ run_cnt, int32_t* __restrict__ req_err, int32_t* __restrict__ misc, int32_t* status) {
    __shared__ uint32_t skey[kKeyCache];
    __shared__ uint32_t hist[256];
    __shared__ uint32_t sh_prefix, sh_kk;
    __shared__ uint32_t wc[kSelWaves][5];
    __shared__ int32_t sh_err;

    const int r = blockIdx.x;
    const int hy = blockIdx.y;
    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    const bool plan = table != nullptr;
    scores += (size_t)hy * total_blocks;
    sel_idx += (size_t)hy * B * k_max;
    sel_cnt += (size_t)hy * B;
    if (plan) {
        miss_list += (size_t)hy * B * k_max;
        miss_cnt += (size_t)hy * B;
        run_cnt += (size_t)hy * B;
        req_err += (size_t)hy * B;
    }
    const int64_t b0 = blk_off[r];
    const int64_t n = blk_off[r + 1] - b0;
    const int64_t lo = n_sink, hi = n - n_local;  // middle blocks [lo, hi)
    const int64_t nc = hi > lo ? hi - lo : 0;
    int64_t k = k_mid[r];
    k = k < 0 ? 0 : (k > nc ? nc : k);
    const int64_t cnt = (n - nc) + k;
    int32_t* out = sel_idx + (size_t)r * k_max;

    if (plan && free_head && r == 0 && hy == 0 && tid == 0) misc[0] = *free_head;
    if (tid == 0) sh_err = 0;

    if (cnt > k_max) {
        for (int i = tid; i < k_max; i += kSelThreads) out[i] = -1;
        if (tid == 0) {
            report(status, PULSE_ERR_SELECT_OVERFLOW);
            sel_cnt[r] = 0;
            if (plan) { miss_cnt[r] = 0; run_cnt[r] = 0; req_err[r] = 0; }
        }
        return;
    }

    const bool cached = nc <= kKeyCache;
    const float* msc = scores + b0 + lo;  // middle scores
    const bool all_mid = (k == nc);
    const bool none_mid = (k == 0);
    uint32_t T = 0, need_eq = 0;
    if (!all_mid && !none_mid) {
        // keys to LDS, with the block-wide min and max key
        uint32_t kmin = 0xFFFFFFFFu, kmax = 0u;
        for (int64_t i = tid; i < nc; i += kSelThreads) {
            const uint32_t key = key32(msc[i]);
            if (cached) skey[i] = key;
            kmin = min(kmin, key);
            kmax = max(kmax, key);
        }
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) {
            kmin = min(kmin, (uint32_t)__shfl_xor((int)kmin, off));
            kmax = max(kmax, (uint32_t)__shfl_xor((int)kmax, off));
        }
        if (lane == 0) { wc[wid][0] = kmin; wc[wid][1] = kmax; }
        __syncthreads();
        kmin = 0xFFFFFFFFu;
        kmax = 0u;
        for (int w = 0; w < kSelWaves; ++w) { kmin = min(kmin, wc[w][0]); kmax = max(kmax, wc[w][1]); }
        __syncthreads();  // wc is reused below
        const uint32_t diff = kmin ^ kmax;
        if (diff == 0) {
            T = kmax;  // every middle key ties: the first k in index order are taken
            need_eq = (uint32_t)k;
        } else {
            // radix passes start at the byte holding the highest bit in which keys differ
            const int top = 31 - __clz(diff);
            const int first_shift = (top / 8) * 8;
            uint32_t mask = first_shift + 8 >= 32 ? 0u : ~((1u << (first_shift + 8)) - 1u);
            uint32_t prefix = kmax & mask;
            uint32_t kk = (uint32_t)k;
            for (int shift = first_shift; shift >= 0; shift -= 8) {
                if (tid < 256) hist[tid] = 0;
                __syncthreads();
                for (int64_t i = tid; i < nc; i += kSelThreads) {
                    const uint32_t key = cached ? skey[i] : key32(msc[i]);
                    if ((key & mask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1u);
                }
                __syncthreads();
                if (wid == 0) {
                    // lane owns digits 4*lane .. 4*lane+3; find digit d with
                    // above(d) < kk <= above(d) + hist[d], above(d) = #keys with digit > d.
                    uint32_t c[4];
#pragma unroll
                    for (int i = 0; i < 4; ++i) c[i] = hist[4 * lane + i];
                    const uint32_t sum = c[0] + c[1] + c[2] + c[3];
                    uint32_t x = sum;  // inclusive suffix sum over lanes >= lane
#pragma unroll
                    for (int off = 1; off < 64; off <<= 1) {
                        const uint32_t y = (uint32_t)__shfl_down((int)x, off);
                        if (lane + off < 64) x += y;
                    }
                    uint32_t above = x - sum;
#pragma unroll
                    for (int i = 3; i >= 0; --i) {
                        if (above < kk && kk <= above + c[i]) {
                            sh_prefix = prefix | ((uint32_t)(4 * lane + i) << shift);
                            sh_kk = kk - above;
                        }
                        above += c[i];
                    }
                }
                __syncthreads();
                prefix = sh_prefix;
                kk = sh_kk;
                mask |= 255u << shift;
            }
            T = prefix;
            need_eq = kk;
        }
    }

    // ordered pass: selection positions, set difference, runs
    uint32_t eq_carry = 0, sel_carry = 0, miss_carry = 0, runs = 0, prev_bit = 0;
    int32_t my_err = 0;
    for (int64_t tile = 0; tile < n; tile += kSelThreads) {
        const int64_t j = tile + tid;
        const bool in = j < n;
        const bool forced = in && (j < lo || j >= hi);
        const bool middle = in && !forced;
        uint32_t key = 0u;
        if (middle && !all_mid && !none_mid) key = cached ? skey[j - lo] : key32(msc[j - lo]);
        const bool gt = middle && (all_mid || (!none_mid && key > T));
        const bool eq = middle && !all_mid && !none_mid && key == T;
        const uint64_t m_eq = __ballot(eq);
        if (lane == 0) wc[wid][0] = (uint32_t)__popcll(m_eq);
        __syncthreads();
        uint32_t eq_before = eq_carry + (uint32_t)__popcll(m_eq & lanemask_lt()), tile_eq = 0;
        for (int w = 0; w < kSelWaves; ++w) {
            if (w < wid) eq_before += wc[w][0];
            tile_eq += wc[w][0];
        }
        const bool sel = forced || gt || (eq && eq_before < need_eq);
        bool miss = false;
        if (plan && sel) {
            if (j >= max_blocks) {
                my_err = PULSE_ERR_BAD_INDEX;
            } else {
                const int32_t v = table[(size_t)r * max_blocks + j];
                if (v >= n_slots) my_err = PULSE_ERR_BAD_INDEX;
                else miss = v < 0;
            }
        }
        const uint64_t m_sel = __ballot(sel);
        const uint64_t m_miss = __ballot(miss);
        const uint64_t prev_in_wave = (m_miss << 1);  // bit l = miss flag of lane l-1
        if (lane == 0) {
            wc[wid][1] = (uint32_t)__popcll(m_sel);
            wc[wid][2] = (uint32_t)__popcll(m_miss);
            wc[wid][3] = (uint32_t)(m_miss >> 63);
        }
        __syncthreads();
        uint32_t sel_pos = sel_carry + (uint32_t)__popcll(m_sel & lanemask_lt());
        uint32_t miss_pos = miss_carry + (uint32_t)__popcll(m_miss & lanemask_lt());
        uint32_t tile_sel = 0, tile_miss = 0;
        for (int w = 0; w < kSelWaves; ++w) {
            if (w < wid) { sel_pos += wc[w][1]; miss_pos += wc[w][2]; }
            tile_sel += wc[w][1];
            tile_miss += wc[w][2];
        }
        const uint32_t first_prev = wid == 0 ? prev_bit : wc[wid - 1][3];
        const uint64_t prev_mask = prev_in_wave | (uint64_t)first_prev;
        const uint64_t starts = m_miss & ~prev_mask;
        if (sel && sel_pos < (uint32_t)k_max) out[sel_pos] = (int32_t)j;
        if (miss && miss_pos < (uint32_t)k_max) miss_list[(size_t)r * k_max + miss_pos] = (int32_t)j;
        if (lane == 0) wc[wid][4] = (uint32_t)__popcll(starts);
        __syncthreads();
        uint32_t tile_runs = 0;
        for (int w = 0; w < kSelWaves; ++w) tile_runs += wc[w][4];
        runs += tile_runs;
        prev_bit = wc[kSelWaves - 1][3];
        eq_carry += tile_eq;
        sel_carry += tile_sel;
        miss_carry += tile_miss;
        __syncthreads();
    }
    for (int64_t i = cnt + tid; i < k_max; i += kSelThreads) out[i] = -1;
    if (my_err) atomicCAS(&sh_err, 0, my_err);
    __syncthreads();
    if (tid == 0) {
        sel_cnt[r] = (int32_t)cnt;
        if (plan) {
            miss_cnt[r] = (int32_t)miss_carry;
            run_cnt[r] = (int32_t)runs;
            req_err[r] = sh_err;
            if (sh_err) report(status, sh_err);
        }
    }
}

hipError_t launch_select(const int64_t* blk_off, int32_t B, int64_t total_blocks, const float* scores,
                         const int32_t* k_mid, int32_t n_sink, int32_t n_local, int32_t k_max, int32_t* sel_idx,
                         int32_t* sel_cnt, const int32_t* table, int32_t max_blocks, int32_t n_slots,
                         const int32_t* free_head, int32_t* miss_list, int32_t* miss_cnt, int32_t* run_cnt,
                         int32_t* req_err, int32_t* misc, int32_t* status, int32_t heads, hipStream_t st) {
    if (B == 0) return hipSuccess;
    hipLaunchKernelGGL(select_kernel, dim3(B, heads), dim3(kSelThreads), 0, st, blk_off, B, total_blocks, scores,
                       k_mid, n_sink, n_local, k_max, sel_idx, sel_cnt, table, max_blocks, n_slots, free_head,
                       miss_list, miss_cnt, run_cnt, req_err, misc, status);
    return hipGetLastError();
}

}  // namespace pulse
