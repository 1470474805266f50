// select.hip -- SoloHead top-k block selection, one 1024-thread workgroup
// per request (and per selecting head; Sec. 4.4.1, budget split Sec. 5
// setup), with the set difference against the GPU-resident hot set folded in
// when a block table is given (Sec. 2.2).
//
// Per request: the first n_sink and last n_local blocks are forced;
// k' = min(max(k_mid,0), #middle) middle blocks of highest score are chosen,
// equal scores in ascending block order; the set is emitted ascending.
// Thread t holds blocks j = base + u * 1024 + t of a tile of 8192 (u < 8
// rounds; requests of one tile keep their keys in registers), so each
// per-block step is one instruction for 64 consecutive blocks:
//   1. radix select (8-bit passes over the offsets key - min key of the
//      order-preserving keys of the fp32 scores, from the highest bit of the
//      key range down) of the k'-th largest offset.  It ends at the first
//      pass whose bucket holding the k'-th offset is taken whole, leaving a
//      threshold T on the decided high bits (mask M) and the number need_eq of
//      offsets with those bits equal to T that are taken;
//   2. one ordered pass per tile: block j is chosen if its masked offset is
//      above T, or equal to T and fewer than need_eq equal ones precede it
//      (exactly the lowest-index tie rule).  Positions come from per-round
//      counts packed as bytes and summed by DPP wave scans (which give each
//      lane its rank among the chosen lanes of its wave) plus a prefix over
//      the 128 (round, wave) counts of the tile, which every wave scans itself
//      from LDS after one barrier.
// With a block table the same pass writes the recall plan: missing blocks
// (table entry -1) in listed order, their count and their run count.
// The select kernel is issue-bound on its compute unit (16 waves share 4
// SIMDs), so per-block work is kept branch-free and cross-wave sums are wave
// scans of one LDS row instead of per-wave loops.
#include "pulse_internal.h"

namespace pulse {

constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / kWave;
constexpr int kRounds = 8;                          // rounds per tile
constexpr int kTile = kRounds * kSelThreads;        // blocks per tile; one-tile requests keep keys in registers
constexpr int kEntries = kRounds * kSelWaves;       // (round, wave) entries of a tile: two per lane
constexpr int kWords = kRounds / 4;                 // words of per-round byte counts

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

// Bits 0..3 of x as the bytes 0..3 of a word (0 or 1 each): the four shifted
// copies x << 7i land on distinct bit positions, so the product has no carries.
__device__ inline uint32_t spread_bytes(uint32_t x) { return ((x & 0xFu) * 0x00204081u) & 0x01010101u; }

// Exclusive prefix, in entry order e = round * kSelWaves + wave, of the
// kEntries values of an LDS row, computed by every wave: lane l holds the
// prefixes of entries 2l and 2l+1 and keeps the one of the parity of this
// wave's entries (wave w's entry of round u is u * kSelWaves + w).
struct RowScan {
    uint32_t mine, total;
    // prefix of this wave's entry of round u
    __device__ uint32_t prefix(int u, int wid) const {
        return (uint32_t)__builtin_amdgcn_readlane((int)mine, u * (kSelWaves / 2) + (wid >> 1));
    }
};
__device__ inline RowScan row_scan(const uint32_t* row, int wid) {
    const int lane = threadIdx.x & 63;
    const u32x2 a = *reinterpret_cast<const u32x2*>(row + 2 * lane);
    const uint32_t incl = wave_scan(a[0] + a[1], 0u, OpAdd());
    const uint32_t ex0 = incl - a[0] - a[1];
    RowScan t;
    t.mine = (wid & 1) ? ex0 + a[0] : ex0;
    t.total = last_lane(incl);
    return t;
}

// LDS of one selecting workgroup.
struct SelLds {
    uint32_t hist[2][256];  // radix histograms: one counted while the other is cleared
    uint32_t sh_prefix, sh_kk, sh_whole;
    uint32_t wc[kSelWaves][2];              // per-wave key min / max
    __align__(8) uint32_t eqc[kEntries];    // equal keys per (round, wave): the tie rule
    __align__(8) uint32_t cnt[kEntries];    // chosen (low 16 bits) | missing (high 16 bits) per (round, wave)
    __align__(8) uint32_t rb[kEntries];     // missing-run starts in the wave (bits 0-7), first (8) / last (9) lane missing
    int32_t sh_err;
};

// One request's selection and, with a table row, its recall plan.
//   n          the request's blocks; rsc its scores (rsc[j], j < n)
//   v          one-tile requests: the scores of blocks tid + u * 1024 that
//              exist, loaded by the caller (read only when k' is neither 0
//              nor #middle)
//   tpre       the table entries of blocks tid + u * 1024 (-1 past the row),
//              loaded by the caller
//   trow       the request's table row (plan) or nullptr (selection only)
//   out / miss the request's sel_idx / miss_list rows
__device__ inline void select_request(SelLds& L, const float* rsc, const float (&v)[kRounds],
                                      const int32_t (&tpre)[kRounds], int64_t n, int32_t k_mid_r, int32_t n_sink,
                                      int32_t n_local, int32_t k_max, int32_t* out, const int32_t* trow,
                                      int32_t max_blocks, int32_t n_slots, int32_t* miss, int32_t* sel_cnt_r,
                                      int32_t* miss_cnt_r, int32_t* run_cnt_r, int32_t* req_err_r, int32_t* status) {
    const int tid = threadIdx.x, lane = tid & 63;
    const int wid = __builtin_amdgcn_readfirstlane(tid >> 6);
    const bool plan = trow != nullptr;
    const int64_t lo = n_sink, hi = n - n_local;  // middle blocks [lo, hi)
    const int64_t nc = hi > lo ? hi - lo : 0;
    int64_t k = k_mid_r;
    k = k < 0 ? 0 : (k > nc ? nc : k);
    const int64_t cnt = (n - nc) + k;

    if (cnt > k_max) {
        for (int i = tid; i < k_max; i += kSelThreads) out[i] = -1;
        if (tid == 0) {
            report(status, PULSE_ERR_SELECT_OVERFLOW);
            *sel_cnt_r = 0;
            if (plan) { *miss_cnt_r = 0; *run_cnt_r = 0; *req_err_r = 0; }
        }
        return;
    }
    if (tid == 0) L.sh_err = 0;

    const bool cached = n <= kTile;
    const bool all_mid = (k == nc);
    const bool none_mid = (k == 0);
    // Threshold: a middle block is taken if its masked offset (key - key_base) & T_mask
    // is above T, or equal to T and fewer than need_eq equal ones precede it.
    // All keys equal: T_mask = 0, so every key is "equal" and the first k are taken.
    uint32_t key_base = 0, T = 0, T_mask = 0, need_eq = (uint32_t)k;
    // the radix select ended on a bucket taken whole: every key equal to T (masked) is chosen
    bool eq_all_taken = false;
    uint32_t kreg[kRounds];  // one-tile requests: key of block tid + 1024 u
    if (!all_mid && !none_mid) {
        uint32_t mid_l = 0;  // rounds whose block is a middle one
        uint32_t kmin = 0xFFFFFFFFu, kmax = 0u;
        if (cached) {
#pragma unroll
            for (int u = 0; u < kRounds; ++u) {
                if (u * kSelThreads >= n) break;
                const int j = tid + u * kSelThreads;
                const uint32_t key = key32(v[u]);
                kreg[u] = key;
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
        if (lane == 0) { L.wc[wid][0] = kmin; L.wc[wid][1] = kmax; }
        if (tid < 256) L.hist[0][tid] = 0;  // the first radix pass's histogram
        __syncthreads();
        // every wave folds the per-wave values, lane w taking wave w's
        const u32x2 mm = lane < kSelWaves ? *reinterpret_cast<const u32x2*>(L.wc[lane]) : u32x2{0xFFFFFFFFu, 0u};
        kmin = last_lane(wave_scan(mm[0], 0xFFFFFFFFu, OpMin()));
        kmax = last_lane(wave_scan(mm[1], 0u, OpMax()));
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
                uint32_t* hcur = L.hist[pass & 1];  // cleared before the barrier that ended the last pass
                if (cached) {
#pragma unroll
                    for (int u = 0; u < kRounds; ++u) {
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
                    const u32x4 c = *reinterpret_cast<const u32x4*>(&hcur[4 * lane]);
                    const uint32_t sum = c[0] + c[1] + c[2] + c[3];
                    const uint32_t incl = wave_scan(sum, 0u, OpAdd());
                    uint32_t above = last_lane(incl) - incl;  // offsets in lanes above this one
#pragma unroll
                    for (int i = 3; i >= 0; --i) {
                        if (above < kk && kk <= above + c[i]) {
                            L.sh_prefix = prefix | ((uint32_t)(4 * lane + i) << sh);
                            L.sh_kk = kk - above;
                            L.sh_whole = kk == above + c[i];
                        }
                        above += c[i];
                    }
                } else if (tid < kWave + 256) {
                    L.hist[(pass + 1) & 1][tid - kWave] = 0;  // the next pass's histogram
                }
                __syncthreads();
                prefix = L.sh_prefix;
                kk = L.sh_kk;
                mask |= dmask << sh;
                if (sh == 0 || L.sh_whole) break;
            }
            T = prefix;
            T_mask = mask;
            need_eq = kk;
            eq_all_taken = L.sh_whole;
        }
    }

    // Ordered pass, one tile of kTile blocks at a time; bit u of a mask is
    // round u's block j = base + u * 1024 + tid.
    const bool thr = !all_mid && !none_mid;
    const bool skip_eq = !thr || eq_all_taken;  // every equal key is taken (or none can occur)
    uint32_t sel_carry = 0, miss_carry = 0, eq_carry = 0, runs = 0, last_carry = 0;
    int32_t my_err = 0;
    for (int64_t base = 0; base < n; base += kTile) {
        const int64_t left = n - base;
        uint32_t valid_m = 0, mid_m = 0, gt_m = 0, eq_m = 0;
#pragma unroll
        for (int u = 0; u < kRounds; ++u) {
            if (u * kSelThreads >= left) break;  // workgroup-uniform
            const int64_t j = base + u * kSelThreads + tid;
            const bool valid = j < n, mid = j >= lo && j < hi;
            valid_m |= (uint32_t)valid << u;
            mid_m |= (uint32_t)mid << u;
            if (all_mid) {
                gt_m |= (uint32_t)mid << u;
            } else if (thr && mid) {
                const uint32_t key = cached ? kreg[u] : key32(rsc[j]);
                const uint32_t mo = (key - key_base) & T_mask;
                gt_m |= (uint32_t)(mo > T) << u;
                eq_m |= (uint32_t)(mo == T) << u;
            }
        }
        uint32_t take_m = eq_m;  // equal keys taken
        if (!skip_eq) {
            // the lowest-index tie rule: the rank of each equal key among the equal keys
            uint32_t xe[kWords];
#pragma unroll
            for (int h = 0; h < kWords; ++h) {
                const uint32_t be = spread_bytes(eq_m >> (4 * h));
                const uint32_t ie = wave_scan(be, 0u, OpAdd());
                xe[h] = ie - be;
                const uint32_t te = last_lane(ie);
                if (lane >= 4 * h && lane < 4 * h + 4)  // lane u writes this wave's entry of round u
                    L.eqc[lane * kSelWaves + wid] = (te >> (8 * (lane & 3))) & 0xFFu;
            }
            __syncthreads();
            const RowScan es = row_scan(L.eqc, wid);
            take_m = 0;
#pragma unroll
            for (int u = 0; u < kRounds; ++u) {
                const uint32_t rank = eq_carry + es.prefix(u, wid) + ((xe[u >> 2] >> (8 * (u & 3))) & 0xFFu);
                take_m |= (uint32_t)(((eq_m >> u) & 1u) && rank < need_eq) << u;
            }
            eq_carry += es.total;
        }
        const uint32_t sel_m = (valid_m & ~mid_m) | gt_m | take_m;
        // set difference against the block table
        uint32_t miss_m = 0;
        if (plan) {
#pragma unroll
            for (int u = 0; u < kRounds; ++u) {
                if (!((sel_m >> u) & 1u)) continue;
                const int64_t j = base + u * kSelThreads + tid;
                if (j >= max_blocks) {
                    my_err = PULSE_ERR_BAD_INDEX;
                    continue;
                }
                const int32_t tv = base == 0 ? tpre[u] : trow[j];
                if (tv >= n_slots) my_err = PULSE_ERR_BAD_INDEX;
                else miss_m |= (uint32_t)(tv < 0) << u;
            }
        }
        // Per (round, wave): chosen and missing counts and missing-run starts, as
        // bytes (round u in byte u & 3 of word u >> 2) summed over the wave by
        // DPP scans, which also give each lane its rank among the wave's chosen
        // (missing) lanes of every round.
        const uint32_t pm = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)miss_m, 0x138, 0xF, 0xF, false);  // wave_shr:1
        const uint32_t st_m = miss_m & ~pm;  // missing, the block before (in this wave's round) not
        uint32_t xs[kWords], xm[kWords];
        const uint32_t m_first = (uint32_t)__builtin_amdgcn_readlane((int)miss_m, 0);
        const uint32_t m_last = (uint32_t)__builtin_amdgcn_readlane((int)miss_m, 63);
#pragma unroll
        for (int h = 0; h < kWords; ++h) {
            const uint32_t bs = spread_bytes(sel_m >> (4 * h)), bm = spread_bytes(miss_m >> (4 * h));
            const uint32_t is = wave_scan(bs, 0u, OpAdd()), im = wave_scan(bm, 0u, OpAdd());
            xs[h] = is - bs;  // lanes below, per round
            xm[h] = im - bm;
            const uint32_t ts = last_lane(is), tm = last_lane(im);
            const uint32_t tst = last_lane(wave_scan(spread_bytes(st_m >> (4 * h)), 0u, OpAdd()));
            if (lane >= 4 * h && lane < 4 * h + 4) {  // lane u writes this wave's entry of round u
                const int sh = 8 * (lane & 3);
                const int e = lane * kSelWaves + wid;
                L.cnt[e] = ((ts >> sh) & 0xFFu) | (((tm >> sh) & 0xFFu) << 16);
                L.rb[e] = ((tst >> sh) & 0xFFu) | (((m_first >> lane) & 1u) << 8) | (((m_last >> lane) & 1u) << 9);
            }
        }
        __syncthreads();
        const RowScan cs = row_scan(L.cnt, wid);
        {
            // runs: starts counted in each entry, less those that continue the previous
            // entry's last block (the previous tile's last block for entry 0)
            const u32x2 rr = *reinterpret_cast<const u32x2*>(&L.rb[2 * lane]);
            const uint32_t l1 = (rr[1] >> 9) & 1u;
            uint32_t pl = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)l1, 0x138, 0xF, 0xF, false);  // wave_shr:1
            if (lane == 0) pl = last_carry;
            const uint32_t cont = (pl & (rr[0] >> 8) & 1u) + (((rr[0] >> 9) & 1u) & ((rr[1] >> 8) & 1u));
            runs += last_lane(wave_scan((rr[0] & 0xFFu) + (rr[1] & 0xFFu) - cont, 0u, OpAdd()));
            last_carry = last_lane(l1);
        }
#pragma unroll
        for (int u = 0; u < kRounds; ++u) {
            if (u * kSelThreads >= left) break;
            const uint32_t pf = cs.prefix(u, wid);
            const int32_t j = (int32_t)(base + u * kSelThreads + tid);
            if ((sel_m >> u) & 1u) {
                const uint32_t pos = sel_carry + (pf & 0xFFFFu) + ((xs[u >> 2] >> (8 * (u & 3))) & 0xFFu);
                if (pos < (uint32_t)k_max) out[pos] = j;
            }
            if ((miss_m >> u) & 1u) {
                const uint32_t pos = miss_carry + (pf >> 16) + ((xm[u >> 2] >> (8 * (u & 3))) & 0xFFu);
                if (pos < (uint32_t)k_max) miss[pos] = j;
            }
        }
        sel_carry += cs.total & 0xFFFFu;
        miss_carry += cs.total >> 16;
        if (base + kTile < n) __syncthreads();  // the next tile rewrites the LDS rows
    }
    for (int64_t i = cnt + tid; i < k_max; i += kSelThreads) out[i] = -1;
    if (my_err) atomicCAS(&L.sh_err, 0, my_err);
    __syncthreads();
    if (tid == 0) {
        *sel_cnt_r = (int32_t)cnt;
        if (plan) {
            *miss_cnt_r = (int32_t)miss_carry;
            *run_cnt_r = (int32_t)runs;
            *req_err_r = L.sh_err;
            if (L.sh_err) report(status, L.sh_err);
        }
    }
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
    __shared__ SelLds L;
    const int r = blockIdx.x;
    const int hy = blockIdx.y;
    const int tid = threadIdx.x;
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
    // costs one memory round trip: the scores at the offsets the request has when
    // all requests are equally long (a wrong guess is reloaded once blk_off is
    // known), then this thread's table entries of the first tile (blocks
    // tid + 1024 u that exist in the row).  The scores come first: the key phase
    // waits for them alone, and the table loads complete behind it.
    const int64_t n_eq = total_blocks / B;
    const int64_t b0_eq = (int64_t)r * n_eq;
    const bool spec = n_eq >= 1 && n_eq <= kTile;
    float sv[kRounds];
    if (spec) {
#pragma unroll
        for (int u = 0; u < kRounds; ++u) {
            if (u * kSelThreads >= n_eq) break;  // workgroup-uniform: no key of this slot exists
            const int j = tid + u * kSelThreads;
            sv[u] = scores[b0_eq + (j < n_eq ? j : n_eq - 1)];
        }
    }
    int32_t tpre[kRounds];
#pragma unroll
    for (int u = 0; u < kRounds; ++u) {
        const int j = tid + u * kSelThreads;
        tpre[u] = (plan && j < max_blocks) ? table[(size_t)r * max_blocks + j] : -1;
    }
    const int64_t b0 = blk_off[r];
    const int64_t n = blk_off[r + 1] - b0;
    const float* rsc = scores + b0;  // this request's scores, by block
    if (plan && free_head && r == 0 && hy == 0 && tid == 0) misc[0] = *free_head;
    float v[kRounds];
    if (n <= kTile) {
        const bool hit = spec && b0 == b0_eq && n == n_eq;
#pragma unroll
        for (int u = 0; u < kRounds; ++u) {  // clamped loads
            if (u * kSelThreads >= n) break;
            const int j = tid + u * kSelThreads;
            v[u] = hit ? sv[u] : rsc[j < n ? j : n - 1];
        }
    }
    select_request(L, rsc, v, tpre, n, k_mid[r], n_sink, n_local, k_max, sel_idx + (size_t)r * k_max,
                   plan ? table + (size_t)r * max_blocks : nullptr, max_blocks, n_slots,
                   plan ? miss_list + (size_t)r * k_max : nullptr, sel_cnt + r, miss_cnt + r, run_cnt + r,
                   req_err + r, status);
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
