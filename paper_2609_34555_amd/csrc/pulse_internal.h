// pulse_internal.h -- types, element helpers, workspace layout and launch
// declarations shared by the gfx950 kernels of the sparse-KV decode path.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/pulse.h"

namespace pulse {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(8))) _Float16 f16x8;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;
typedef __attribute__((ext_vector_type(2))) _Float16 f16x2;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((ext_vector_type(2))) uint32_t u32x2;

constexpr int kHeadDim = 128;
constexpr int kWave = 64;
constexpr int kMaxGroup = 16;   // G = Hq / Hkv padded to one 16-wide MFMA tile
constexpr int kChunkTokens = 32;  // attention processes 32 tokens per MFMA step
constexpr int kMaxBatch = 4096;   // requests per call: the recall and publish kernels scan their counts in LDS

// ---- timed launches ---------------------------------------------------------

// Launch with optional timing events carried by the dispatch itself
// (hipExtLaunchKernel: `start` is recorded when the kernel starts, `stop` when it
// completes), so timing a kernel adds no marker packet to the stream.
template <typename F, typename... Args>
inline void launch_timed(F kernel, dim3 grid, dim3 block, uint32_t lds, hipStream_t st, hipEvent_t start,
                         hipEvent_t stop, Args... args) {
    if (start || stop)
        hipExtLaunchKernelGGL(kernel, grid, block, lds, st, start, stop, 0u, args...);
    else
        hipLaunchKernelGGL(kernel, grid, block, lds, st, args...);
}

// ---- device status --------------------------------------------------------

__device__ inline void report(int32_t* status, int32_t code) {
    if (status) atomicCAS(status, 0, code);
}

// ---- 16-bit element helpers ------------------------------------------------

// Order-preserving map of a sign-magnitude 16-bit float pattern onto uint16:
// increasing values give increasing keys, and -0 sorts just below +0.
__device__ inline uint32_t key16(uint32_t x) { return (x & 0x8000u) ? (~x & 0xFFFFu) : (x | 0x8000u); }
__device__ inline uint32_t unkey16(uint32_t k) { return (k & 0x8000u) ? (k & 0x7FFFu) : (~k & 0xFFFFu); }

// Order-preserving map of fp32 onto uint32 (both zeros map to the key of +0).
__device__ inline uint32_t key32(float s) {
    s = s + 0.0f;  // -0 -> +0
    uint32_t u = __float_as_uint(s);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

template <int DT>
__device__ inline float elem_to_float(uint16_t x);
template <>
__device__ inline float elem_to_float<PULSE_BF16>(uint16_t x) { return __uint_as_float((uint32_t)x << 16); }
template <>
__device__ inline float elem_to_float<PULSE_F16>(uint16_t x) {
    _Float16 h;
    __builtin_memcpy(&h, &x, 2);
    return (float)h;
}

// ---- workspace layout -----------------------------------------------------

struct AttnPlan {
    int32_t entries_per_split;  // selected blocks handled by one wave
    int32_t n_split;            // splits per (request, KV head)
};

struct WsLayout {
    size_t scores;     // float [total_blocks]
    size_t miss_list;  // int32 [B][k_max]   missing block indices, listed order
    size_t miss_cnt;   // int32 [B]
    size_t run_cnt;    // int32 [B]
    size_t req_err;    // int32 [B]          per-request plan error (0 = ok)
    size_t misc;       // int32 [16]         [0] = free_head snapshot
    size_t attn_o;     // float [B][Hkv][n_wg][G][d]   (per-workgroup partials)
    size_t attn_ml;    // float2 [B][Hkv][n_wg][G]
    size_t total;
};

AttnPlan attn_plan(int32_t B, int32_t Hkv, int32_t k_max, int32_t bs);
// Waves per attention workgroup for a GQA group of G query heads.
inline int attn_waves(int G) { return G <= 8 ? 8 : 4; }
// Attention partials a call with these arguments writes: one per workgroup.
inline int64_t attn_partial_units(const pulse_shape& s, int32_t B, int32_t k_max) {
    const int G = s.num_q_heads / s.num_kv_heads;
    const AttnPlan p = attn_plan(B, s.num_kv_heads, k_max, s.block_size);
    const int W = attn_waves(G);
    return (int64_t)B * s.num_kv_heads * ((p.n_split + W - 1) / W);
}
WsLayout ws_layout(const pulse_shape& s, int32_t B, int32_t k_max, int64_t total_blocks);
bool shape_supported(const pulse_shape* s);

// ---- launchers (each returns hipSuccess or the launch error) --------------

hipError_t launch_build_digests(const pulse_shape& s, const void* kv, const int64_t* blk_off,
                                const int32_t* ctx_len, int32_t B, int64_t total_blocks, int32_t kv_head,
                                void* digests, int32_t* status, hipStream_t st);

// heads == 1: score with KV head `solo`; heads == Hkv: every head h scores with
// its own digests (digests and scores stacked along h).
// The step-end release of the previous recall (see launch_release), when the
// scoring kernel performs it on the side.
struct ReleaseArgs {
    const int32_t* miss_list;
    const int32_t* miss_cnt;
    int32_t B, k_max;
    int32_t* table;
    int32_t max_blocks;
    int32_t* free_head;
    pulse_recall_stats* stats;
    int32_t* status;
};
// Release work of thread `e0` of `stride` (grid-stride over the B * k_max plan
// entries): an entry's table slot returns to -1; thread 0 alone moves the
// free-list head back.  Standalone (fused = false): the table pass runs
// unconditionally (-1 is right whether or not the recall moved the block) and
// thread 0 clears the statistics, so a second release changes nothing.  Fused
// into the next layer-step's scoring kernel: only a recall that moved bytes is
// undone, every thread reads that from the statistics, and none clears them
// (the recall of the same step overwrites them), so no thread reads what
// another writes.
//
// The loads of a thread's first entry (its request's miss count and its list
// value), the statistics and the free-list head do not depend on one another,
// so all of them are issued before any is used: one memory round trip instead
// of a chain of three.  A list value past the request's count is read but not
// used (the list spans B * k_max entries).
__device__ inline void release_entries(const ReleaseArgs& a, int64_t e0, int64_t stride, bool fused) {
    const int64_t n_ent = (int64_t)a.B * a.k_max;
    const bool head = e0 == 0;
    int32_t n_missing = 0, fh = 0;
    int64_t bytes = 0;
    if (fused || head) {
        n_missing = a.stats->n_missing;
        bytes = a.stats->bytes;
    }
    if (head) fh = *a.free_head;
    int32_t n_first = 0, j_first = -1;
    if (e0 < n_ent) {
        n_first = a.miss_cnt[e0 / a.k_max];
        j_first = a.miss_list[e0];
    }
    if (fused && bytes <= 0) return;
    for (int64_t e = e0; e < n_ent; e += stride) {
        const int32_t r = (int32_t)(e / a.k_max), i = (int32_t)(e % a.k_max);
        const int32_t n = e == e0 ? n_first : a.miss_cnt[r];
        if (n < 0 || n > a.k_max) {
            if (i == 0) report(a.status, PULSE_ERR_BAD_INDEX);
        } else if (i < n) {
            const int32_t j = e == e0 ? j_first : a.miss_list[e];
            if (j >= 0 && j < a.max_blocks) a.table[(size_t)r * a.max_blocks + j] = -1;
            else report(a.status, PULSE_ERR_BAD_INDEX);
        }
    }
    if (head && bytes > 0) {
        if (fh < n_missing) {
            report(a.status, PULSE_ERR_BAD_INDEX);
        } else {
            *a.free_head = fh - n_missing;
            if (!fused) {
                a.stats->n_missing = 0;
                a.stats->n_runs = 0;
                a.stats->bytes = 0;
            }
        }
    }
}
// rel != nullptr: the scoring kernel also releases the recall described by rel
// (every entry's table reset, then the free-list head and statistics), which
// the kernel boundary orders before the selection that follows.
// start / stop (optional): timing events of the scoring kernel (recorded as
// markers when there is no block to score).
hipError_t launch_score(const pulse_shape& s, const void* q, const void* digests, const int64_t* blk_off,
                        int32_t B, int64_t total_blocks, int32_t solo, int32_t n_sink, int32_t n_local,
                        float* scores, int32_t heads, hipStream_t st, const ReleaseArgs* rel = nullptr,
                        hipEvent_t start = nullptr, hipEvent_t stop = nullptr);

// select (a3); when table != nullptr the set difference (a4) is folded in and
// the recall plan (miss list, counts, runs, free_head snapshot) is written.
// heads > 1 stacks scores, selections and plans along the head dimension.
hipError_t launch_select(const int64_t* blk_off, int32_t B, int64_t total_blocks, const float* scores,
                         const int32_t* k_mid, int32_t n_sink, int32_t n_local, int32_t k_max, int32_t* sel_idx,
                         int32_t* sel_cnt, const int32_t* table, int32_t max_blocks, int32_t n_slots,
                         const int32_t* free_head, int32_t* miss_list, int32_t* miss_cnt, int32_t* run_cnt,
                         int32_t* req_err, int32_t* misc, int32_t* status, int32_t heads, hipStream_t st);

hipError_t launch_recall_plan(const int64_t* blk_off, int32_t B, const int32_t* sel_idx,
                              const int32_t* sel_cnt, int32_t k_max, const int32_t* table,
                              int32_t max_blocks, int32_t n_slots, const int32_t* free_head,
                              int32_t* miss_list, int32_t* miss_cnt, int32_t* run_cnt, int32_t* req_err,
                              int32_t* misc, int32_t* status, hipStream_t st);

hipError_t launch_recall_copy(const void* host_kv, const int64_t* blk_off, int32_t B, int32_t k_max,
                              int32_t* table, int32_t max_blocks, const int32_t* free_slots,
                              int32_t* free_head, int32_t n_free, void* pool, int32_t n_slots,
                              size_t unit_bytes, const int32_t* miss_list, const int32_t* miss_cnt,
                              const int32_t* run_cnt, const int32_t* req_err, const int32_t* misc,
                              pulse_recall_stats* stats, int32_t* status, int32_t copy_xcds, hipStream_t st,
                              hipEvent_t start = nullptr, hipEvent_t stop = nullptr);

hipError_t launch_attention(const pulse_shape& s, const void* q, const void* pool, int32_t n_slots,
                            const int32_t* table, int32_t max_blocks, const int32_t* sel_idx,
                            const int32_t* sel_cnt, int32_t k_max, const int32_t* ctx_len, int32_t B,
                            float sm_scale, float* out, float* lse, float* ws_o, float2* ws_ml,
                            int32_t* status, hipStream_t st, hipEvent_t split_done = nullptr,
                            hipEvent_t done = nullptr);

hipError_t launch_average_scores(const float* sc, int64_t total_blocks, int32_t H, float* avg, hipStream_t st);
hipError_t launch_mam_selection(const int32_t* ctx_len, int32_t B, int32_t bs, int32_t max_blocks, int32_t n_sink,
                                int32_t n_local, int32_t* sel_all, int32_t* cnt_all, int32_t* sel_mid,
                                int32_t* cnt_mid, int32_t* status, hipStream_t st);
hipError_t launch_mam_finalize(const float* lse_all, const float* lse_mid, int32_t B, int32_t Hkv, int32_t G,
                               float* mam, hipStream_t st);

// Host-side argument check: return `code` from the calling entry point.
#define PULSE_REQUIRE(cond, code)   \
    do {                            \
        if (!(cond)) return (code); \
    } while (0)

// Typed pointer at a byte offset of a workspace.
template <typename T>
inline T* ws_at(void* ws, size_t off) {
    return reinterpret_cast<T*>(static_cast<char*>(ws) + off);
}

// Stages of a chained layer-step (api.hip): score + select + plan, recall,
// attention; and the full argument check of pulse_layer_args.
// Optional timing events (NULL = none): the scoring kernel's start / end, the
// recall copy kernel's start / end, the end of the attention's last kernel.
hipError_t layer_select(const pulse_layer_args& a, hipStream_t hs, hipEvent_t score_start = nullptr,
                        hipEvent_t score_stop = nullptr);
hipError_t layer_recall(const pulse_layer_args& a, hipStream_t hs, int32_t copy_xcds = 8,
                        hipEvent_t start = nullptr, hipEvent_t stop = nullptr);
hipError_t layer_attention(const pulse_layer_args& a, hipStream_t hs, hipEvent_t done = nullptr);
pulse_status check_layer_args(const pulse_layer_args* a);

hipError_t launch_release(const int32_t* miss_list, const int32_t* miss_cnt, int32_t B, int32_t k_max,
                          int32_t* table, int32_t max_blocks, int32_t* free_head, pulse_recall_stats* stats,
                          int32_t* status, hipStream_t st);
hipError_t launch_probe_hbm_read(const void* src, size_t bytes, uint32_t* sink, hipStream_t st,
                                 hipEvent_t start = nullptr, hipEvent_t stop = nullptr);
int32_t probe_hbm_sink_words();

hipError_t launch_probe_copy(const void* src, void* dst, size_t bytes, hipStream_t st);

}  // namespace pulse
