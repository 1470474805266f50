// select.hip -- SoloHead top-k block selection and the set difference
// against the GPU-resident hot set, for gfx950.
//
// Selection (Sec. 4.4.1, budget split Sec. 5 setup): per request, the first
// n_sink and last n_local blocks are forced; k' = min(max(k_mid,0), #middle)
// middle blocks of highest score are chosen, equal scores in ascending
// block order; the set is emitted ascending.  One 1024-thread workgroup per
// request:
//   1. radix select (8-bit passes over an LDS copy of the keys, on the offsets
//      key - min key, from the highest bit of the key range down) of the k'-th
//      largest order-preserving key of the fp32 scores.  It ends at the first
//      pass whose bucket holding the k'-th offset is taken whole, leaving a
//      threshold T on the decided high bits (mask M) and the number need_eq of
//      offsets with those bits equal to T that are taken;
//   2. one ordered pass over super-tiles of 8192 blocks, thread t owning 8
//      consecutive blocks as bit masks, with two workgroup scans (DPP wave
//      scans + LDS) per super-tile: block j is chosen if its masked offset is
//      above T, or equal to T and fewer than need_eq equal ones precede it --
//      exactly the lowest-index tie rule.
// With a block table the same pass also takes the set difference (Sec. 2.2:
// selected blocks whose table entry is -1 are missing) and writes the recall
// plan: missing blocks in listed order, their count and their run count.
#include "pulse_internal.h"

namespace pulse {

constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / kWave;
constexpr int kKeyCache = 8192;  // middle-block keys kept in LDS (32 KiB); larger requests read L2
constexpr int kPerThread = kKeyCache / kSelThreads;  // keys (and table entries) prefetched per thread

// Inclusive scan of x over the 64 lanes of a wave with `op`, in registers
// (DPP row shifts within 16-lane rows, then row broadcasts of lanes 15 and
// 31); lanes without a source combine with `identity`.
template <typename Op>
__device__ inline uint32_t wave_scan(uint32_t x, uint32_t identity, Op op) {
    const int id = (int)identity;
    x = op(x, (uint32_t)__builtin_amdgcn_update_dpp(id, (int)x, 0x111, 0xF, 0xF, false));  // row_shr:1
    x = op(x, (uint32_t)__builtin_amdgcn_update_dpp(id, (int)x, 0x112, 0xF, 0xF, false));  // row_shr:2
    x = op(x, (uint32_t)__builtin_amdgcn_update_dpp(id, (int)x, 0x114, 0xF, 0xF, false));  // row_shr:4
    x = op(x, (uint32_t)__builtin_amdgcn_update_dpp(id, (int)x, 0x118, 0xF, 0xF, false));  // row_shr:8
    x = op(x, (uint32_t)__builtin_amdgcn_update_dpp(id, (int)x, 0x142, 0xA, 0xF, false));  // row_bcast:15
    x = op(x, (uint32_t)__builtin_amdgcn_update_dpp(id, (int)x, 0x143, 0xC, 0xF, false));  // row_bcast:31
    return x;
}
struct OpAdd { __device__ uint32_t operator()(uint32_t a, uint32_t b) const { return a + b; } };
struct OpMin { __device__ uint32_t operator()(uint32_t a, uint32_t b) const { return a < b ? a : b; } };
struct OpMax { __device__ uint32_t operator()(uint32_t a, uint32_t b) const { return a > b ? a : b; } };

// Value of lane 63 (the wave-wide result of an inclusive scan), in every lane.
__device__ inline uint32_t last_lane(uint32_t x) { return (uint32_t)__builtin_amdgcn_readlane((int)x, 63); }

// Per-wave totals (and each wave's last bit) exchanged through LDS by the
// workgroup scans of the ordered pass.
struct ScanLds {
    uint32_t tot[kSelWaves];
    uint32_t last[kSelWaves];
};

// Exclusive prefix sum of v over the workgroup's threads in order; *total =
// the workgroup sum.  One barrier.
__device__ inline uint32_t block_scan(uint32_t v, ScanLds& sl, uint32_t& total) {
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    const uint32_t x = wave_scan(v, 0u, OpAdd());  // inclusive scan within the wave
    if (lane == 63) sl.tot[wid] = x;
    __syncthreads();
    uint32_t before = x - v, t = 0;
#pragma unroll
    for (int w = 0; w < kSelWaves; ++w) {
        const uint32_t c = sl.tot[w];
        if (w < wid) before += c;
        t += c;
    }
    total = t;
    return before;
}

// block_scan that also hands each thread the `bit` of the thread before it
// (thread 0 gets carry_bit) in *prev_bit.
__device__ inline uint32_t block_scan_last(uint32_t v, uint32_t bit, uint32_t carry_bit, ScanLds& sl,
                                           uint32_t& total, uint32_t& prev_bit) {
    const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
    uint32_t pb = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)bit, 0x138, 0xF, 0xF, false);  // wave_shr:1
    if (lane == 63) sl.last[wid] = bit;
    const uint32_t before = block_scan(v, sl, total);  // its barrier also publishes sl.last
    if (lane == 0) pb = wid == 0 ? carry_bit : sl.last[wid - 1];
    prev_bit = pb;
    return before;
}

// Workgroup sum of v (one barrier; sl must not be read concurrently).
__device__ inline uint32_t block_sum(uint32_t v, ScanLds& sl) {
    uint32_t total;
    (void)block_scan(v, sl, total);
    return total;
}

// grid = (B, heads): blockIdx.x = request, blockIdx.y = selecting head slot
// (always 0 for SoloHead; 0..Hkv-1 for headwise selection, whose per-head
// scores, selections and plans are stacked along the head dimension).
//
// Requests of at most kKeyCache blocks (the cached path) keep the key of
// block j in skey[j]; the radix passes read each thread's keys from registers
// and the ordered pass forms its masks without branches.  Longer requests
// re-read their scores from memory in every pass.
__global__ __launch_bounds__(kSelThreads) void select_kernel(
    const int64_t* __restrict__ blk_off, int32_t B, int64_t total_blocks, const float* __restrict__ scores,
    const int32_t* __restrict__ k_mid, int32_t n_sink, int32_t n_local, int32_t k_max, int32_t* __restrict__ sel_idx,
    int32_t* __restrict__ sel_cnt, const int32_t* __restrict__ table, int32_t max_blocks, int32_t n_slots,
    const int32_t* __restrict__ free_head, int32_t* __restrict__ miss_list, int32_t* __restrict__ miss_cnt,
    int32_t* __restrict__ run_cnt, int32_t* __restrict__ req_err, int32_t* __restrict__ misc, int32_t* status) {
    __shared__ __align__(16) uint32_t skey[kKeyCache];  // key of block j at [j] (cached path)
    __shared__ uint32_t hist[2][256];  // radix histograms: one counted while the other is cleared
    __shared__ uint32_t sh_prefix, sh_kk;
    __shared__ bool sh_whole;
    __shared__ uint32_t wc[kSelWaves][2];
    __shared__ ScanLds scan[2];  // double-buffered: scan[0] equal counts, scan[1] selected / missing
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
    // Loads issued before the request's extent is known, so that the common case
    // costs one memory round trip: this thread's table entries of the first
    // super-tile (blocks 8t .. 8t+7, any that exist in the row), and the scores
    // at the offsets the request has when all requests are equally long (a wrong
    // guess is reloaded once blk_off is known).
    int32_t tpre[kPerThread];
#pragma unroll
    for (int u = 0; u < kPerThread; ++u) {
        const int j = kPerThread * tid + u;
        tpre[u] = (plan && j < max_blocks) ? table[(size_t)r * max_blocks + j] : -1;
    }
    const int64_t n_eq = total_blocks / B;
    const int64_t b0_eq = (int64_t)r * n_eq;
    const bool spec = n_eq >= 1 && n_eq <= kKeyCache;
    float sv[kPerThread];
    if (spec) {
#pragma unroll
        for (int u = 0; u < kPerThread; ++u) {
            if (u * kSelThreads >= n_eq) break;  // workgroup-uniform: no key of this slot exists
            const int j = tid + u * kSelThreads;
            sv[u] = scores[b0_eq + (j < n_eq ? j : n_eq - 1)];
        }
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

    const bool cached = n <= kKeyCache;
    const int64_t t_lim = n < max_blocks ? n : max_blocks;  // table entries that exist
    const float* rsc = scores + b0;                          // this request's scores, by block
    const bool all_mid = (k == nc);
    const bool none_mid = (k == 0);
    // Threshold: a middle block is taken if its masked offset (key - key_base) & T_mask
    // is above T, or equal to T and fewer than need_eq equal ones precede it.
    // All keys equal: T_mask = 0, so every key is "equal" and the first k are taken.
    uint32_t key_base = 0, T = 0, T_mask = 0, need_eq = (uint32_t)k;
    // the radix select ended on a bucket taken whole: every key equal to T (masked) is chosen
    bool eq_all_taken = false;
    // cached path: keys of blocks tid + 1024u in registers, mid_l = those that are middle
    uint32_t kreg[kPerThread];
    uint32_t mid_l = 0;
    if (!all_mid && !none_mid) {
        uint32_t kmin = 0xFFFFFFFFu, kmax = 0u;
        if (cached) {
            const bool hit = spec && b0 == b0_eq && n == n_eq;
            float v[kPerThread];
#pragma unroll
            for (int u = 0; u < kPerThread; ++u) {  // n >= nc >= 1 here; clamped loads
                if (u * kSelThreads >= n) break;
                const int j = tid + u * kSelThreads;
                v[u] = hit ? sv[u] : rsc[j < n ? j : n - 1];
            }
#pragma unroll
            for (int u = 0; u < kPerThread; ++u) {
                if (u * kSelThreads >= n) break;
                const int j = tid + u * kSelThreads;
                const uint32_t key = key32(v[u]);
                kreg[u] = key;
                if (j < n) skey[j] = key;
                if (j >= lo && j < hi) {
                    mid_l |= 1u << u;
                    kmin = min(kmin, key);
                    kmax = max(kmax, key);
                }
            }
        } else {
            for (int64_t j = lo + tid; j < hi; j += kSelThreads) {
                const uint32_t key = key32(rsc[j]);
                kmin = min(kmin, key);
                kmax = max(kmax, key);
            }
        }
        kmin = last_lane(wave_scan(kmin, 0xFFFFFFFFu, OpMin()));
        kmax = last_lane(wave_scan(kmax, 0u, OpMax()));
        if (lane == 0) { wc[wid][0] = kmin; wc[wid][1] = kmax; }
        if (tid < 256) hist[0][tid] = 0;  // the first radix pass's histogram
        __syncthreads();
        kmin = 0xFFFFFFFFu;
        kmax = 0u;
        for (int w = 0; w < kSelWaves; ++w) { kmin = min(kmin, wc[w][0]); kmax = max(kmax, wc[w][1]); }
        key_base = kmin;
        if (kmin != kmax) {
            // Radix select on the offsets key - kmin (order-preserving, < 2^(top+1)):
            // digits of 8 bits from bit `top` down, so the first histogram spreads
            // over the keys' actual range instead of their (shared) exponent byte.
            // It stops as soon as the bucket holding the k-th offset is taken whole.
            const uint32_t span = kmax - kmin;
            const int top = 31 - __clz(span);
            uint32_t mask = top >= 31 ? 0u : ~((2u << top) - 1u);  // offset bits already decided
            uint32_t prefix = 0u;                                    // their value
            uint32_t kk = (uint32_t)k;
            for (int shift = top - 7, pass = 0;; shift -= 8, ++pass) {
                const int sh = shift > 0 ? shift : 0;
                const uint32_t dmask = shift >= 0 ? 255u : (255u >> -shift);
                uint32_t* hcur = hist[pass & 1];  // cleared before the barrier that ended the last pass
                if (cached) {
#pragma unroll
                    for (int u = 0; u < kPerThread; ++u) {
                        if (u * kSelThreads >= n) break;
                        const uint32_t off = kreg[u] - kmin;
                        if (((mid_l >> u) & 1u) && (off & mask) == prefix) atomicAdd(&hcur[(off >> sh) & dmask], 1u);
                    }
                } else {
                    for (int64_t j = lo + tid; j < hi; j += kSelThreads) {
                        const uint32_t off = key32(rsc[j]) - kmin;
                        if ((off & mask) == prefix) atomicAdd(&hcur[(off >> sh) & dmask], 1u);
                    }
                }
                __syncthreads();
                if (wid == 0) {
                    // lane owns digits 4*lane .. 4*lane+3; find digit d with
                    // above(d) < kk <= above(d) + hist[d], above(d) = #offsets with digit > d.
                    uint32_t c[4];
#pragma unroll
                    for (int i = 0; i < 4; ++i) c[i] = hcur[4 * lane + i];
                    const uint32_t sum = c[0] + c[1] + c[2] + c[3];
                    const uint32_t incl = wave_scan(sum, 0u, OpAdd());
                    uint32_t above = last_lane(incl) - incl;  // offsets in lanes above this one
#pragma unroll
                    for (int i = 3; i >= 0; --i) {
                        if (above < kk && kk <= above + c[i]) {
                            sh_prefix = prefix | ((uint32_t)(4 * lane + i) << sh);
                            sh_kk = kk - above;
                            sh_whole = kk == above + c[i];
                        }
                        above += c[i];
                    }
                } else if (tid < kWave + 256) {
                    hist[(pass + 1) & 1][tid - kWave] = 0;  // the next pass's histogram
                }
                __syncthreads();
                prefix = sh_prefix;
                kk = sh_kk;
                mask |= dmask << sh;
                if (sh == 0 || sh_whole) break;
            }
            T = prefix;
            T_mask = mask;
            need_eq = kk;
            eq_all_taken = sh_whole;
        }
    }

    // Ordered pass over super-tiles of kSelThreads * kPerThread blocks; thread t
    // owns the kPerThread consecutive blocks base + 8t .. base + 8t + 7 as bit
    // masks.  Two workgroup scans per super-tile: equal-key counts (for the
    // lowest-index tie rule), then selected / missing counts and each thread's
    // last missing bit (for run starts).
    uint32_t eq_carry = 0, sel_carry = 0, miss_carry = 0, runs = 0, prev_bit = 0;
    int32_t my_err = 0;
    const bool thr = !all_mid && !none_mid;
    const bool skip_eq = (!thr || eq_all_taken) && n <= (int64_t)kSelThreads * kPerThread;
    // bits u of [0, 8) with a <= j0 + u < b
    auto range_mask = [](int64_t a, int64_t b, int64_t j0) -> uint32_t {
        const int64_t a_rel = a - j0, b_rel = b - j0;
        const uint32_t ac = a_rel <= 0 ? 0u : (a_rel >= kPerThread ? (uint32_t)kPerThread : (uint32_t)a_rel);
        const uint32_t bc = b_rel <= 0 ? 0u : (b_rel >= kPerThread ? (uint32_t)kPerThread : (uint32_t)b_rel);
        return ((1u << bc) - 1u) & ~((1u << ac) - 1u);
    };
    for (int64_t base = 0; base < n; base += (int64_t)kSelThreads * kPerThread) {
        const int64_t j0 = base + (int64_t)kPerThread * tid;
        const uint32_t valid_m = range_mask(0, n, j0);
        const uint32_t mid_m = range_mask(lo, hi, j0);
        const uint32_t forced_m = valid_m & ~mid_m;
        uint32_t gt_m = 0, eq_m = 0;
        if (all_mid) {
            gt_m = mid_m;
        } else if (thr && mid_m) {
            uint32_t kb[kPerThread];
            if (cached) {  // j0 + 7 < kKeyCache: two 16-byte LDS reads
                const u32x4 a = *reinterpret_cast<const u32x4*>(&skey[j0]);
                const u32x4 b = *reinterpret_cast<const u32x4*>(&skey[j0 + 4]);
#pragma unroll
                for (int i = 0; i < 4; ++i) { kb[i] = a[i]; kb[4 + i] = b[i]; }
            } else {
#pragma unroll
                for (int u = 0; u < kPerThread; ++u)
                    kb[u] = ((mid_m >> u) & 1u) ? key32(rsc[j0 + u]) : 0u;
            }
#pragma unroll
            for (int u = 0; u < kPerThread; ++u) {
                const uint32_t mo = (kb[u] - key_base) & T_mask;
                gt_m |= (uint32_t)(mo > T) << u;
                eq_m |= (uint32_t)(mo == T) << u;
            }
            gt_m &= mid_m;
            eq_m &= mid_m;
        }
        // scan 1: equal keys before this thread's blocks (the lowest-index tie rule).  Not
        // needed when every equal key is taken (or none can occur) and the request is one
        // super-tile: consecutive scans of a multi-tile request need it between them, as
        // they reuse scan[1].
        uint32_t eq_tot = 0, take = kPerThread;  // equal keys still taken
        if (!skip_eq) {
            const uint32_t eq_before = eq_carry + block_scan(__popc(eq_m), scan[0], eq_tot);
            take = need_eq > eq_before ? need_eq - eq_before : 0u;
        }
        uint32_t sel_m = forced_m | gt_m;
#pragma unroll
        for (int u = 0; u < kPerThread; ++u)
            if ((eq_m >> u) & 1u) {
                if (take) { sel_m |= 1u << u; --take; }
            }
        // set difference against the block table
        uint32_t miss_m = 0;
        if (plan) {
#pragma unroll
            for (int u = 0; u < kPerThread; ++u) {
                if (!((sel_m >> u) & 1u)) continue;
                const int64_t j = j0 + u;
                if (j >= t_lim) {
                    if (j >= max_blocks) my_err = PULSE_ERR_BAD_INDEX;
                    continue;
                }
                const int32_t v = base == 0 ? tpre[u] : table[(size_t)r * max_blocks + j];
                if (v >= n_slots) my_err = PULSE_ERR_BAD_INDEX;
                else if (v < 0) miss_m |= 1u << u;
            }
        }
        // scan 2: selected (low 16 bits) and missing (high 16 bits) counts, plus
        // the previous thread's last missing bit
        uint32_t tot2;
        const uint32_t last_bit = (miss_m >> (kPerThread - 1)) & 1u;
        uint32_t prev_last;
        const uint32_t before2 =
            block_scan_last(__popc(sel_m) | ((uint32_t)__popc(miss_m) << 16), last_bit, prev_bit, scan[1], tot2,
                            prev_last);
        uint32_t sel_pos = sel_carry + (before2 & 0xFFFFu);
        uint32_t miss_pos = miss_carry + (before2 >> 16);
#pragma unroll
        for (int u = 0; u < kPerThread; ++u) {
            const int64_t j = j0 + u;
            if ((sel_m >> u) & 1u) {
                if (sel_pos < (uint32_t)k_max) out[sel_pos] = (int32_t)j;
                ++sel_pos;
            }
            if ((miss_m >> u) & 1u) {
                if (miss_pos < (uint32_t)k_max) miss_list[(size_t)r * k_max + miss_pos] = (int32_t)j;
                ++miss_pos;
            }
        }
        const uint32_t starts = miss_m & ~((miss_m << 1) | prev_last);
        runs += __popc(starts);
        prev_bit = scan[1].last[kSelWaves - 1];
        eq_carry += eq_tot;
        sel_carry += tot2 & 0xFFFFu;
        miss_carry += tot2 >> 16;
    }
    runs = block_sum(runs, scan[0]);
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
