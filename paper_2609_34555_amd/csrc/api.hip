// api.hip -- the C ABI of the sparse-KV decode path (declared in
// include/pulse.h): host-side argument validation, workspace layout and
// kernel launches.  Nothing here allocates device memory or synchronises.
#include <string.h>

#include <mutex>

#include "pulse_internal.h"

namespace pulse {

bool shape_supported(const pulse_shape* s) {
    if (!s) return false;
    if (s->head_dim != kHeadDim) return false;
    if (s->block_size != 16 && s->block_size != 32 && s->block_size != 64) return false;
    if (s->num_kv_heads < 1 || s->num_q_heads < s->num_kv_heads) return false;
    if (s->num_q_heads % s->num_kv_heads) return false;
    if (s->num_q_heads / s->num_kv_heads > kMaxGroup) return false;
    if (s->dtype != PULSE_F16 && s->dtype != PULSE_BF16) return false;
    return true;
}

static size_t align_up(size_t x) { return (x + 255) & ~(size_t)255; }

WsLayout ws_layout(const pulse_shape& s, int32_t B, int32_t k_max, int64_t total_blocks) {
    WsLayout w;
    const size_t G = (size_t)(s.num_q_heads / s.num_kv_heads);
    const size_t units = (size_t)attn_partial_units(s, B, k_max);
    size_t o = 0;
    w.scores = o;    o = align_up(o + sizeof(float) * (size_t)total_blocks);
    w.miss_list = o; o = align_up(o + sizeof(int32_t) * (size_t)B * k_max);
    w.miss_cnt = o;  o = align_up(o + sizeof(int32_t) * (size_t)B);
    w.run_cnt = o;   o = align_up(o + sizeof(int32_t) * (size_t)B);
    w.req_err = o;   o = align_up(o + sizeof(int32_t) * (size_t)B);
    w.misc = o;      o = align_up(o + sizeof(int32_t) * 16);
    w.attn_o = o;    o = align_up(o + sizeof(float) * units * G * kHeadDim);
    w.attn_ml = o;   o = align_up(o + sizeof(float2) * units * G);
    w.total = o;
    return w;
}

template <typename T>
static T* at(void* ws, size_t off) {
    return reinterpret_cast<T*>(static_cast<char*>(ws) + off);
}

}  // namespace pulse

using namespace pulse;


static pulse_status hip_status(hipError_t e) { return e == hipSuccess ? PULSE_OK : PULSE_ERR_HIP; }

extern "C" {

const char* pulse_status_string(pulse_status s) {
    switch (s) {
        case PULSE_OK: return "PULSE_OK";
        case PULSE_ERR_INVALID_ARG: return "PULSE_ERR_INVALID_ARG";
        case PULSE_ERR_UNSUPPORTED: return "PULSE_ERR_UNSUPPORTED";
        case PULSE_ERR_WORKSPACE: return "PULSE_ERR_WORKSPACE";
        case PULSE_ERR_POOL_EXHAUSTED: return "PULSE_ERR_POOL_EXHAUSTED";
        case PULSE_ERR_SELECT_OVERFLOW: return "PULSE_ERR_SELECT_OVERFLOW";
        case PULSE_ERR_HIP: return "PULSE_ERR_HIP";
        case PULSE_ERR_BAD_INDEX: return "PULSE_ERR_BAD_INDEX";
        case PULSE_ERR_TIMEOUT: return "PULSE_ERR_TIMEOUT";
    }
    return "PULSE_ERR_UNKNOWN";
}

size_t pulse_block_bytes(const pulse_shape* shape) {
    if (!shape_supported(shape)) return 0;
    return (size_t)2 * shape->num_kv_heads * shape->block_size * shape->head_dim * 2;
}

size_t pulse_workspace_bytes(const pulse_shape* shape, int32_t B, int32_t k_max, int64_t total_blocks) {
    if (!shape_supported(shape) || B < 0 || k_max < 0 || total_blocks < 0) return 0;
    return ws_layout(*shape, B, k_max, total_blocks).total;
}

int32_t pulse_attention_workgroups(const pulse_shape* shape, int32_t B, int32_t k_max) {
    if (!shape_supported(shape) || B < 1 || k_max < 1) return 0;
    const AttnPlan p = attn_plan(B, shape->num_kv_heads, k_max, shape->block_size);
    const int W = attn_waves(shape->num_q_heads / shape->num_kv_heads);
    return (p.n_split + W - 1) / W;
}

pulse_status pulse_build_digests(const pulse_shape* shape, const void* kv, const int64_t* blk_off,
                                 const int32_t* ctx_len, int32_t B, int64_t total_blocks, int32_t kv_head,
                                 void* digests, int32_t* dev_status, pulse_stream_t stream) {
    PULSE_REQUIRE(shape, PULSE_ERR_INVALID_ARG);
    PULSE_REQUIRE(shape_supported(shape), PULSE_ERR_UNSUPPORTED);
    PULSE_REQUIRE(B >= 0 && total_blocks >= 0, PULSE_ERR_INVALID_ARG);
    PULSE_REQUIRE(kv_head >= 0 && kv_head < shape->num_kv_heads, PULSE_ERR_INVALID_ARG);
    if (B == 0 || total_blocks == 0) return PULSE_OK;
    PULSE_REQUIRE(kv && blk_off && ctx_len && digests, PULSE_ERR_INVALID_ARG);
    return hip_status(launch_build_digests(*shape, kv, blk_off, ctx_len, B, total_blocks, kv_head, digests,
                                           dev_status, (hipStream_t)stream));
}

static pulse_status check_select_args(const pulse_shape* shape, const void* q, const void* digests,
                                      const int64_t* blk_off, int32_t B, int64_t total_blocks, int32_t solo,
                                      const int32_t* k_mid, int32_t n_sink, int32_t n_local, int32_t k_max,
                                      int32_t* sel_idx, int32_t* sel_cnt, int32_t* dev_status) {
    PULSE_REQUIRE(shape, PULSE_ERR_INVALID_ARG);
    PULSE_REQUIRE(shape_supported(shape), PULSE_ERR_UNSUPPORTED);
    PULSE_REQUIRE(B >= 0 && total_blocks >= 0 && k_max >= 1, PULSE_ERR_INVALID_ARG);
    PULSE_REQUIRE(n_sink >= 0 && n_local >= 0, PULSE_ERR_INVALID_ARG);
    PULSE_REQUIRE(solo >= 0 && solo < shape->num_kv_heads, PULSE_ERR_INVALID_ARG);
    PULSE_REQUIRE(B <= kMaxBatch, PULSE_ERR_UNSUPPORTED);
    if (B == 0) return PULSE_OK;
    PULSE_REQUIRE(q && blk_off && k_mid && sel_idx && sel_cnt && dev_status, PULSE_ERR_INVALID_ARG);
    PULSE_REQUIRE(digests || total_blocks == 0, PULSE_ERR_INVALID_ARG);
    return PULSE_OK;
}

pulse_status pulse_select_solohead(const pulse_shape* shape, const void* q, const void* digests,
                                   const int64_t* blk_off, int32_t B, int64_t total_blocks, int32_t solo_kv_head,
                                   const int32_t* k_mid, int32_t n_sink_blocks, int32_t n_local_blocks,
                                   int32_t k_max, int32_t* sel_idx, int32_t* sel_cnt, float* scores,
                                   int32_t* dev_status, void* ws, size_t ws_bytes, pulse_stream_t stream) {
    pulse_status st = check_select_args(shape, q, digests, blk_off, B, total_blocks, solo_kv_head, k_mid,
                                        n_sink_blocks, n_local_blocks, k_max, sel_idx, sel_cnt, dev_status);
    if (st != PULSE_OK || B == 0) return st;
    const WsLayout w = ws_layout(*shape, B, k_max, total_blocks);
    PULSE_REQUIRE(ws && ws_bytes >= w.total, PULSE_ERR_WORKSPACE);
    float* sc = scores ? scores : at<float>(ws, w.scores);
    hipStream_t hs = (hipStream_t)stream;
    hipError_t e = launch_score(*shape, q, digests, blk_off, B, total_blocks, solo_kv_head, n_sink_blocks,
                                n_local_blocks, sc, 1, hs);
    if (e != hipSuccess) return PULSE_ERR_HIP;
    e = launch_select(blk_off, B, total_blocks, sc, k_mid, n_sink_blocks, n_local_blocks, k_max, sel_idx, sel_cnt,
                      nullptr, 0, 0, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, dev_status, 1, hs);
    return hip_status(e);
}

size_t pulse_headwise_workspace_bytes(const pulse_shape* shape, int32_t B, int32_t k_max, int64_t total_blocks) {
    if (!shape_supported(shape) || B < 0 || k_max < 0 || total_blocks < 0) return 0;
    const size_t H = (size_t)shape->num_kv_heads;
    size_t o = 0;
    o = align_up(o + sizeof(float) * H * (size_t)total_blocks);    // scores [Hkv][total_blocks]
    o = align_up(o + sizeof(int32_t) * H * (size_t)B * k_max);     // miss lists [Hkv][B][k_max]
    o = align_up(o + sizeof(int32_t) * H * (size_t)B);             // plan errors [Hkv][B]
    return o;
}

pulse_status pulse_select_headwise(const pulse_shape* shape, const void* q, const void* head_digests,
                                   const int64_t* blk_off, int32_t B, int64_t total_blocks, const int32_t* k_mid,
                                   int32_t n_sink_blocks, int32_t n_local_blocks, int32_t k_max,
                                   const int32_t* block_table, int32_t max_blocks, int32_t n_slots, int32_t* sel_idx,
                                   int32_t* sel_cnt, int32_t* miss_cnt, int32_t* run_cnt, int32_t* dev_status,
                                   void* ws, size_t ws_bytes, pulse_stream_t stream) {
    pulse_status st = check_select_args(shape, q, head_digests, blk_off, B, total_blocks, 0, k_mid, n_sink_blocks,
                                        n_local_blocks, k_max, sel_idx, sel_cnt, dev_status);
    if (st != PULSE_OK || B == 0) return st;
    PULSE_REQUIRE(block_table && miss_cnt && run_cnt && max_blocks >= 1 && n_slots >= 1, PULSE_ERR_INVALID_ARG);
    const size_t H = (size_t)shape->num_kv_heads;
    PULSE_REQUIRE(ws && ws_bytes >= pulse_headwise_workspace_bytes(shape, B, k_max, total_blocks),
                  PULSE_ERR_WORKSPACE);
    float* sc = at<float>(ws, 0);
    size_t o = align_up(sizeof(float) * H * (size_t)total_blocks);
    int32_t* miss_list = at<int32_t>(ws, o);
    o = align_up(o + sizeof(int32_t) * H * (size_t)B * k_max);
    int32_t* req_err = at<int32_t>(ws, o);
    hipStream_t hs = (hipStream_t)stream;
    hipError_t e = launch_score(*shape, q, head_digests, blk_off, B, total_blocks, 0, n_sink_blocks, n_local_blocks,
                                sc, (int32_t)H, hs);
    if (e != hipSuccess) return PULSE_ERR_HIP;
    e = launch_select(blk_off, B, total_blocks, sc, k_mid, n_sink_blocks, n_local_blocks, k_max, sel_idx, sel_cnt,
                      block_table, max_blocks, n_slots, nullptr, miss_list, miss_cnt, run_cnt, req_err, nullptr,
                      dev_status, (int32_t)H, hs);
    return hip_status(e);
}

size_t pulse_average_workspace_bytes(const pulse_shape* shape, int32_t B, int32_t k_max, int64_t total_blocks) {
    if (!shape_supported(shape) || B < 0 || k_max < 0 || total_blocks < 0) return 0;
    const size_t H = (size_t)shape->num_kv_heads;
    return align_up(sizeof(float) * H * (size_t)total_blocks) + align_up(sizeof(float) * (size_t)total_blocks);
}

pulse_status pulse_select_average(const pulse_shape* shape, const void* q, const void* head_digests,
                                  const int64_t* blk_off, int32_t B, int64_t total_blocks, const int32_t* k_mid,
                                  int32_t n_sink_blocks, int32_t n_local_blocks, int32_t k_max, int32_t* sel_idx,
                                  int32_t* sel_cnt, float* scores, int32_t* dev_status, void* ws, size_t ws_bytes,
                                  pulse_stream_t stream) {
    pulse_status st = check_select_args(shape, q, head_digests, blk_off, B, total_blocks, 0, k_mid, n_sink_blocks,
                                        n_local_blocks, k_max, sel_idx, sel_cnt, dev_status);
    if (st != PULSE_OK || B == 0) return st;
    PULSE_REQUIRE(ws && ws_bytes >= pulse_average_workspace_bytes(shape, B, k_max, total_blocks),
                  PULSE_ERR_WORKSPACE);
    const int32_t H = shape->num_kv_heads;
    float* sc = at<float>(ws, 0);
    float* avg = scores ? scores : at<float>(ws, align_up(sizeof(float) * (size_t)H * (size_t)total_blocks));
    hipStream_t hs = (hipStream_t)stream;
    hipError_t e = launch_score(*shape, q, head_digests, blk_off, B, total_blocks, 0, n_sink_blocks, n_local_blocks,
                                sc, H, hs);
    if (e != hipSuccess) return PULSE_ERR_HIP;
    e = launch_average_scores(sc, total_blocks, H, avg, hs);
    if (e != hipSuccess) return PULSE_ERR_HIP;
    e = launch_select(blk_off, B, total_blocks, avg, k_mid, n_sink_blocks, n_local_blocks, k_max, sel_idx, sel_cnt,
                      nullptr, 0, 0, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr, dev_status, 1, hs);
    return hip_status(e);
}

// MAM workspace: attention scratch (k_max = max_blocks), then the two
// selections, their counts, the attention output and the two lse arrays.
struct MamLayout {
    WsLayout attn;
    size_t sel_all, sel_mid, cnt_all, cnt_mid, out, lse_all, lse_mid, total;
};
static MamLayout mam_layout(const pulse_shape& s, int32_t B, int32_t max_blocks) {
    MamLayout m;
    m.attn = ws_layout(s, B, max_blocks, 0);
    const size_t sel = sizeof(int32_t) * (size_t)B * max_blocks;
    size_t o = m.attn.total;
    m.sel_all = o; o = align_up(o + sel);
    m.sel_mid = o; o = align_up(o + sel);
    m.cnt_all = o; o = align_up(o + sizeof(int32_t) * (size_t)B);
    m.cnt_mid = o; o = align_up(o + sizeof(int32_t) * (size_t)B);
    m.out = o;     o = align_up(o + sizeof(float) * (size_t)B * s.num_q_heads * kHeadDim);
    m.lse_all = o; o = align_up(o + sizeof(float) * (size_t)B * s.num_q_heads);
    m.lse_mid = o; o = align_up(o + sizeof(float) * (size_t)B * s.num_q_heads);
    m.total = o;
    return m;
}

size_t pulse_mam_workspace_bytes(const pulse_shape* shape, int32_t B, int32_t max_blocks) {
    if (!shape_supported(shape) || B < 0 || max_blocks < 0) return 0;
    return mam_layout(*shape, B, max_blocks).total;
}

pulse_status pulse_mam(const pulse_shape* shape, const void* q, const void* slot_pool, int32_t n_slots,
                       const int32_t* block_table, int32_t max_blocks, const int32_t* ctx_len, int32_t B,
                       int32_t n_sink_blocks, int32_t n_local_blocks, float sm_scale, float* mam,
                       int32_t* dev_status, void* ws, size_t ws_bytes, pulse_stream_t stream) {
    PULSE_REQUIRE(shape, PULSE_ERR_INVALID_ARG);
    PULSE_REQUIRE(shape_supported(shape), PULSE_ERR_UNSUPPORTED);
    PULSE_REQUIRE(B >= 0 && max_blocks >= 1 && n_slots >= 1 && n_sink_blocks >= 0 && n_local_blocks >= 0,
                  PULSE_ERR_INVALID_ARG);
    PULSE_REQUIRE(B <= kMaxBatch, PULSE_ERR_UNSUPPORTED);
    if (B == 0) return PULSE_OK;
    PULSE_REQUIRE(q && slot_pool && block_table && ctx_len && mam && dev_status, PULSE_ERR_INVALID_ARG);
    const MamLayout m = mam_layout(*shape, B, max_blocks);
    PULSE_REQUIRE(ws && ws_bytes >= m.total, PULSE_ERR_WORKSPACE);
    hipStream_t hs = (hipStream_t)stream;
    int32_t* sel_all = at<int32_t>(ws, m.sel_all);
    int32_t* sel_mid = at<int32_t>(ws, m.sel_mid);
    int32_t* cnt_all = at<int32_t>(ws, m.cnt_all);
    int32_t* cnt_mid = at<int32_t>(ws, m.cnt_mid);
    float* out = at<float>(ws, m.out);
    float* lse_all = at<float>(ws, m.lse_all);
    float* lse_mid = at<float>(ws, m.lse_mid);
    hipError_t e = launch_mam_selection(ctx_len, B, shape->block_size, max_blocks, n_sink_blocks, n_local_blocks,
                                        sel_all, cnt_all, sel_mid, cnt_mid, dev_status, hs);
    if (e != hipSuccess) return PULSE_ERR_HIP;
    float* ws_o = at<float>(ws, m.attn.attn_o);
    float2* ws_ml = at<float2>(ws, m.attn.attn_ml);
    e = launch_attention(*shape, q, slot_pool, n_slots, block_table, max_blocks, sel_all, cnt_all, max_blocks,
                         ctx_len, B, sm_scale, out, lse_all, ws_o, ws_ml, dev_status, hs);
    if (e != hipSuccess) return PULSE_ERR_HIP;
    e = launch_attention(*shape, q, slot_pool, n_slots, block_table, max_blocks, sel_mid, cnt_mid, max_blocks,
                         ctx_len, B, sm_scale, out, lse_mid, ws_o, ws_ml, dev_status, hs);
    if (e != hipSuccess) return PULSE_ERR_HIP;
    const int32_t G = shape->num_q_heads / shape->num_kv_heads;
    return hip_status(launch_mam_finalize(lse_all, lse_mid, B, shape->num_kv_heads, G, mam, hs));
}

pulse_status pulse_pick_solo_heads(const float* mam, int32_t rows, int32_t num_kv_heads, int32_t* solo,
                                   int32_t* reversed) {
    PULSE_REQUIRE(mam && rows >= 1 && num_kv_heads >= 1 && solo && reversed, PULSE_ERR_INVALID_ARG);
    int32_t hi = 0, lo = 0;
    double vhi = 0.0, vlo = 0.0;
    for (int32_t h = 0; h < num_kv_heads; ++h) {
        double s = 0.0;
        for (int32_t r = 0; r < rows; ++r) s += (double)mam[(size_t)r * num_kv_heads + h];
        if (h == 0 || s > vhi) { vhi = s; hi = h; }
        if (h == 0 || s < vlo) { vlo = s; lo = h; }
    }
    *solo = hi;
    *reversed = lo;
    return PULSE_OK;
}

static pulse_status check_recall_args(const pulse_shape* shape, const void* host_kv, const int64_t* blk_off,
                                      int32_t B, const int32_t* sel_idx, const int32_t* sel_cnt, int32_t k_max,
                                      int32_t* block_table, int32_t max_blocks, const int32_t* free_slots,
                                      int32_t* free_head, int32_t n_free, void* slot_pool, int32_t n_slots,
                                      pulse_recall_stats* stats, int32_t* dev_status) {
    PULSE_REQUIRE(shape, PULSE_ERR_INVALID_ARG);
    PULSE_REQUIRE(shape_supported(shape), PULSE_ERR_UNSUPPORTED);
    PULSE_REQUIRE(B >= 0 && k_max >= 1 && max_blocks >= 1 && n_free >= 0 && n_slots >= 1,
                  PULSE_ERR_INVALID_ARG);
    PULSE_REQUIRE(B <= kMaxBatch, PULSE_ERR_UNSUPPORTED);
    if (B == 0) return PULSE_OK;
    PULSE_REQUIRE(host_kv && blk_off && sel_idx && sel_cnt && block_table && free_head && slot_pool && stats &&
                      dev_status,
                  PULSE_ERR_INVALID_ARG);
    PULSE_REQUIRE(free_slots || n_free == 0, PULSE_ERR_INVALID_ARG);
    return PULSE_OK;
}

pulse_status pulse_recall_gather(const pulse_shape* shape, const void* host_kv, const int64_t* blk_off, int32_t B,
                                 const int32_t* sel_idx, const int32_t* sel_cnt, int32_t k_max,
                                 int32_t* block_table, int32_t max_blocks, const int32_t* free_slots,
                                 int32_t* free_head, int32_t n_free, void* slot_pool, int32_t n_slots,
                                 pulse_recall_stats* stats, int32_t* dev_status, void* ws, size_t ws_bytes,
                                 pulse_stream_t stream) {
    pulse_status st = check_recall_args(shape, host_kv, blk_off, B, sel_idx, sel_cnt, k_max, block_table,
                                        max_blocks, free_slots, free_head, n_free, slot_pool, n_slots, stats,
                                        dev_status);
    if (st != PULSE_OK || B == 0) return st;
    const WsLayout w = ws_layout(*shape, B, k_max, 0);
    PULSE_REQUIRE(ws && ws_bytes >= w.total, PULSE_ERR_WORKSPACE);
    hipStream_t hs = (hipStream_t)stream;
    hipError_t e = launch_recall_plan(blk_off, B, sel_idx, sel_cnt, k_max, block_table, max_blocks, n_slots,
                                      free_head, at<int32_t>(ws, w.miss_list), at<int32_t>(ws, w.miss_cnt),
                                      at<int32_t>(ws, w.run_cnt), at<int32_t>(ws, w.req_err),
                                      at<int32_t>(ws, w.misc), dev_status, hs);
    if (e != hipSuccess) return PULSE_ERR_HIP;
    e = launch_recall_copy(host_kv, blk_off, B, k_max, block_table, max_blocks, free_slots, free_head, n_free,
                           slot_pool, n_slots, pulse_block_bytes(shape), at<int32_t>(ws, w.miss_list),
                           at<int32_t>(ws, w.miss_cnt), at<int32_t>(ws, w.run_cnt), at<int32_t>(ws, w.req_err),
                           at<int32_t>(ws, w.misc), stats, dev_status, 8, hs);
    return hip_status(e);
}

pulse_status pulse_release_recalled(const pulse_shape* shape, int32_t B, int32_t k_max, int64_t total_blocks,
                                    int32_t* block_table, int32_t max_blocks, int32_t* free_head,
                                    pulse_recall_stats* stats, int32_t* dev_status, void* ws, size_t ws_bytes,
                                    pulse_stream_t stream) {
    PULSE_REQUIRE(shape, PULSE_ERR_INVALID_ARG);
    PULSE_REQUIRE(shape_supported(shape), PULSE_ERR_UNSUPPORTED);
    PULSE_REQUIRE(B >= 0 && k_max >= 1 && max_blocks >= 1 && total_blocks >= 0, PULSE_ERR_INVALID_ARG);
    PULSE_REQUIRE(B <= kMaxBatch, PULSE_ERR_UNSUPPORTED);
    if (B == 0) return PULSE_OK;
    PULSE_REQUIRE(block_table && free_head && stats && dev_status, PULSE_ERR_INVALID_ARG);
    const WsLayout w = ws_layout(*shape, B, k_max, total_blocks);
    PULSE_REQUIRE(ws && ws_bytes >= w.total, PULSE_ERR_WORKSPACE);
    return hip_status(launch_release(at<int32_t>(ws, w.miss_list), at<int32_t>(ws, w.miss_cnt), B, k_max, block_table,
                                     max_blocks, free_head, stats, dev_status, (hipStream_t)stream));
}

pulse_status pulse_sparse_decode_attn(const pulse_shape* shape, const void* q, const void* slot_pool, int32_t n_slots,
                                      const int32_t* block_table, int32_t max_blocks, const int32_t* sel_idx,
                                      const int32_t* sel_cnt, int32_t k_max, const int32_t* ctx_len, int32_t B,
                                      float sm_scale, float* out, float* lse, int32_t* dev_status, void* ws,
                                      size_t ws_bytes, pulse_stream_t stream) {
    PULSE_REQUIRE(shape, PULSE_ERR_INVALID_ARG);
    PULSE_REQUIRE(shape_supported(shape), PULSE_ERR_UNSUPPORTED);
    PULSE_REQUIRE(B >= 0 && k_max >= 1 && max_blocks >= 1 && n_slots >= 1, PULSE_ERR_INVALID_ARG);
    if (B == 0) return PULSE_OK;
    PULSE_REQUIRE(q && slot_pool && block_table && sel_idx && sel_cnt && ctx_len && out && dev_status,
                  PULSE_ERR_INVALID_ARG);
    const WsLayout w = ws_layout(*shape, B, k_max, 0);
    PULSE_REQUIRE(ws && ws_bytes >= w.total, PULSE_ERR_WORKSPACE);
    return hip_status(launch_attention(*shape, q, slot_pool, n_slots, block_table, max_blocks, sel_idx, sel_cnt,
                                       k_max, ctx_len, B, sm_scale, out, lse, at<float>(ws, w.attn_o),
                                       at<float2>(ws, w.attn_ml), dev_status, (hipStream_t)stream));
}

}  // extern "C"

namespace pulse {

// The three stages of a chained layer-step (arguments already validated).
// Score + select + recall plan; `mid` (optional) is recorded between score
// and select.
hipError_t layer_select(const pulse_layer_args& a, hipStream_t hs, hipEvent_t score_start, hipEvent_t score_stop) {
    const WsLayout w = ws_layout(a.shape, a.B, a.k_max, a.total_blocks);
    const ReleaseArgs rel{at<int32_t>(a.ws, w.miss_list), at<int32_t>(a.ws, w.miss_cnt), a.B, a.k_max,
                          a.block_table, a.max_blocks, a.free_head, a.stats, a.dev_status};
    hipError_t e = launch_score(a.shape, a.q, a.digests, a.blk_off, a.B, a.total_blocks, a.solo_kv_head,
                                a.n_sink_blocks, a.n_local_blocks, at<float>(a.ws, w.scores), 1, hs,
                                a.release_previous ? &rel : nullptr, score_start, score_stop);
    if (e != hipSuccess) return e;
    return launch_select(a.blk_off, a.B, a.total_blocks, at<float>(a.ws, w.scores), a.k_mid, a.n_sink_blocks,
                         a.n_local_blocks, a.k_max, a.sel_idx, a.sel_cnt, a.block_table, a.max_blocks, a.n_slots,
                         a.free_head, at<int32_t>(a.ws, w.miss_list), at<int32_t>(a.ws, w.miss_cnt),
                         at<int32_t>(a.ws, w.run_cnt), at<int32_t>(a.ws, w.req_err), at<int32_t>(a.ws, w.misc),
                         a.dev_status, 1, hs);
}

// Gather-scatter recall of the plan written by layer_select.
hipError_t layer_recall(const pulse_layer_args& a, hipStream_t hs, int32_t copy_xcds, hipEvent_t start,
                        hipEvent_t stop) {
    const WsLayout w = ws_layout(a.shape, a.B, a.k_max, a.total_blocks);
    return launch_recall_copy(a.host_kv, a.blk_off, a.B, a.k_max, a.block_table, a.max_blocks, a.free_slots,
                              a.free_head, a.n_free, a.slot_pool, a.n_slots, pulse_block_bytes(&a.shape),
                              at<int32_t>(a.ws, w.miss_list), at<int32_t>(a.ws, w.miss_cnt),
                              at<int32_t>(a.ws, w.run_cnt), at<int32_t>(a.ws, w.req_err), at<int32_t>(a.ws, w.misc),
                              a.stats, a.dev_status, copy_xcds, hs, start, stop);
}

// Sparse attention over the selection.
hipError_t layer_attention(const pulse_layer_args& a, hipStream_t hs, hipEvent_t done) {
    const WsLayout w = ws_layout(a.shape, a.B, a.k_max, a.total_blocks);
    return launch_attention(a.shape, a.q, a.slot_pool, a.n_slots, a.block_table, a.max_blocks, a.sel_idx, a.sel_cnt,
                            a.k_max, a.ctx_len, a.B, a.sm_scale, a.out, a.lse, at<float>(a.ws, w.attn_o),
                            at<float2>(a.ws, w.attn_ml), a.dev_status, hs, (hipEvent_t)a.attn_split_event, done);
}

// Full argument check of a chained layer-step.
pulse_status check_layer_args(const pulse_layer_args* a) {
    PULSE_REQUIRE(a, PULSE_ERR_INVALID_ARG);
    pulse_status st = check_select_args(&a->shape, a->q, a->digests, a->blk_off, a->B, a->total_blocks,
                                        a->solo_kv_head, a->k_mid, a->n_sink_blocks, a->n_local_blocks, a->k_max,
                                        a->sel_idx, a->sel_cnt, a->dev_status);
    if (st != PULSE_OK) return st;
    st = check_recall_args(&a->shape, a->host_kv, a->blk_off, a->B, a->sel_idx, a->sel_cnt, a->k_max,
                           a->block_table, a->max_blocks, a->free_slots, a->free_head, a->n_free, a->slot_pool,
                           a->n_slots, a->stats, a->dev_status);
    if (st != PULSE_OK) return st;
    if (a->B == 0) return PULSE_OK;
    PULSE_REQUIRE(a->ctx_len && a->out, PULSE_ERR_INVALID_ARG);
    PULSE_REQUIRE(a->ws && a->ws_bytes >= ws_layout(a->shape, a->B, a->k_max, a->total_blocks).total,
                  PULSE_ERR_WORKSPACE);
    return PULSE_OK;
}

}  // namespace pulse

extern "C" {

pulse_status pulse_decode_layer(const pulse_layer_args* a, pulse_stream_t stream) {
    pulse_status st = check_layer_args(a);
    if (st != PULSE_OK || a->B == 0) return st;
    hipStream_t hs = (hipStream_t)stream;
    // the timing events ride on the kernels' own launches (no marker packets); NULL entries are not recorded
    hipEvent_t* ev = (hipEvent_t*)a->events;
    auto E = [&](int i) { return ev ? ev[i] : nullptr; };
    if (layer_select(*a, hs, E(0), E(1)) != hipSuccess) return PULSE_ERR_HIP;
    if (layer_recall(*a, hs, 8, E(2), E(3)) != hipSuccess) return PULSE_ERR_HIP;
    if (layer_attention(*a, hs, E(4)) != hipSuccess) return PULSE_ERR_HIP;
    return PULSE_OK;
}

}  // extern "C"

namespace pulse {

// Workspace of pulse_decode_layer_noalloc: one array per GPU, kept for the life of
// the process.  In host code `scratch` names a host-side stand-in, not device
// memory: the device address comes from hipGetSymbolAddress, once per device.
static __device__ __align__(256) uint8_t scratch[PULSE_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
static std::mutex g_scratch_mu;
static void* g_scratch_ptr[kMaxDevices];

// Device address of the current device's scratch array; nullptr on a HIP error.
static void* scratch_for_current_device() {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return nullptr;
        g_scratch_ptr[dev] = p;
    }
    return g_scratch_ptr[dev];
}

}  // namespace pulse

extern "C" {

pulse_status pulse_decode_layer_noalloc(const pulse_layer_args* args, pulse_stream_t stream) {
    PULSE_REQUIRE(args, PULSE_ERR_INVALID_ARG);
    PULSE_REQUIRE(!args->ws && args->ws_bytes == 0, PULSE_ERR_INVALID_ARG);
    pulse_layer_args a = *args;
    // other argument errors are reported by pulse_decode_layer's own checks
    if (shape_supported(&a.shape) && a.B > 0 && a.B <= kMaxBatch && a.k_max >= 1 && a.total_blocks >= 0) {
        const size_t need = ws_layout(a.shape, a.B, a.k_max, a.total_blocks).total;
        PULSE_REQUIRE(need <= (size_t)PULSE_NOALLOC_SCRATCH_BYTES, PULSE_ERR_WORKSPACE);
        void* ws = scratch_for_current_device();
        if (!ws) return PULSE_ERR_HIP;
        a.ws = ws;
        a.ws_bytes = need;
    }
    return pulse_decode_layer(&a, stream);
}

pulse_status pulse_probe_hbm_read(const void* src, size_t bytes, void* sink, void* start_event, void* stop_event,
                                  pulse_stream_t stream) {
    PULSE_REQUIRE(bytes % 16 == 0 && (src || bytes == 0) && sink, PULSE_ERR_INVALID_ARG);
    return hip_status(launch_probe_hbm_read(src, bytes, (uint32_t*)sink, (hipStream_t)stream,
                                            (hipEvent_t)start_event, (hipEvent_t)stop_event));
}

size_t pulse_probe_hbm_sink_bytes(void) { return sizeof(uint32_t) * (size_t)probe_hbm_sink_words(); }

pulse_status pulse_events_create(int32_t n, void** events) {
    PULSE_REQUIRE(n >= 0 && (events || n == 0), PULSE_ERR_INVALID_ARG);
    for (int32_t i = 0; i < n; ++i) {
        hipEvent_t e;
        if (hipEventCreate(&e) != hipSuccess) return PULSE_ERR_HIP;
        events[i] = (void*)e;
    }
    return PULSE_OK;
}

pulse_status pulse_events_destroy(int32_t n, void* const* events) {
    PULSE_REQUIRE(n >= 0 && (events || n == 0), PULSE_ERR_INVALID_ARG);
    for (int32_t i = 0; i < n; ++i)
        if (events[i] && hipEventDestroy((hipEvent_t)events[i]) != hipSuccess) return PULSE_ERR_HIP;
    return PULSE_OK;
}

pulse_status pulse_event_elapsed_ms(void* start, void* stop, float* ms) {
    PULSE_REQUIRE(start && stop && ms, PULSE_ERR_INVALID_ARG);
    return hip_status(hipEventElapsedTime(ms, (hipEvent_t)start, (hipEvent_t)stop));
}

pulse_status pulse_host_alloc(size_t bytes, int32_t coherent, void** host_ptr) {
    PULSE_REQUIRE(host_ptr && bytes > 0, PULSE_ERR_INVALID_ARG);
    *host_ptr = nullptr;
    unsigned flags = hipHostMallocMapped | hipHostMallocPortable |
                     (coherent ? hipHostMallocCoherent : hipHostMallocNonCoherent);
    return hip_status(hipHostMalloc(host_ptr, bytes, flags));
}

pulse_status pulse_host_free(void* host_ptr) {
    PULSE_REQUIRE(host_ptr, PULSE_ERR_INVALID_ARG);
    return hip_status(hipHostFree(host_ptr));
}

pulse_status pulse_baseline_memcpy_units(const void* host_kv, void* pool, const int64_t* src_units,
                                         const int64_t* dst_units, int32_t n, size_t unit_bytes,
                                         pulse_stream_t stream) {
    PULSE_REQUIRE(n >= 0 && unit_bytes > 0, PULSE_ERR_INVALID_ARG);
    if (n == 0) return PULSE_OK;
    PULSE_REQUIRE(host_kv && pool && src_units && dst_units, PULSE_ERR_INVALID_ARG);
    for (int32_t i = 0; i < n; ++i) {
        const char* src = static_cast<const char*>(host_kv) + (size_t)src_units[i] * unit_bytes;
        char* dst = static_cast<char*>(pool) + (size_t)dst_units[i] * unit_bytes;
        if (hipMemcpyAsync(dst, src, unit_bytes, hipMemcpyHostToDevice, (hipStream_t)stream) != hipSuccess)
            return PULSE_ERR_HIP;
    }
    return PULSE_OK;
}

pulse_status pulse_probe_host_read(const void* host_src, void* dev_dst, size_t bytes, pulse_stream_t stream) {
    PULSE_REQUIRE(host_src && dev_dst && bytes > 0 && bytes % 16384 == 0, PULSE_ERR_INVALID_ARG);
    return hip_status(launch_probe_copy(host_src, dev_dst, bytes, (hipStream_t)stream));
}

}  // extern "C"
