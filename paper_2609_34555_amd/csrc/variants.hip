// variants.hip -- the selection strategies the paper compares SoloHead with,
// and the Middle Attention Mass that picks the solo head (Sec. 4.4.1, Eq. 2).
//
// Average selection: every KV head scores the blocks with its own digests
// (the score kernel over a head grid axis), the scores are averaged over the
// heads, and one top-k on the average is shared by all heads.  Averaging the
// per-KV-head scores (each already the mean over its G query heads) is the
// mean over all query heads.
//
// MAM: for query head q, the softmax mass of its full attention that falls on
// middle tokens is exp(lse_middle - lse_all), with lse the log-sum-exp of the
// scaled logits over the respective tokens; a KV head's MAM is the mean over
// its G query heads.  The two lse come from the sparse attention kernel run
// once over every block of the request and once over its middle blocks
// (those that selection ranks: neither the first n_sink nor the last n_local).
// The highest-MAM head is the SoloHead, the lowest the "reversed" choice.
#include "pulse_internal.h"

namespace pulse {

// avg[b] = (1/H) * sum_h sc[h][b], heads summed in ascending order.
__global__ __launch_bounds__(256) void average_scores_kernel(const float* __restrict__ sc, int64_t total_blocks,
                                                             int32_t H, float* __restrict__ avg) {
    const float inv = 1.f / (float)H;
    for (int64_t b = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; b < total_blocks;
         b += (int64_t)gridDim.x * blockDim.x) {
        float s = 0.f;
        for (int h = 0; h < H; ++h) s += sc[(size_t)h * total_blocks + b];
        avg[b] = s * inv;
    }
}

hipError_t launch_average_scores(const float* sc, int64_t total_blocks, int32_t H, float* avg, hipStream_t st) {
    if (total_blocks == 0) return hipSuccess;
    int64_t grid = (total_blocks + 255) / 256;
    if (grid > 2048) grid = 2048;
    hipLaunchKernelGGL(average_scores_kernel, dim3((unsigned)grid), dim3(256), 0, st, sc, total_blocks, H, avg);
    return hipGetLastError();
}

// Selections of every block (all) and of the middle blocks (mid) of each
// request, for the two attention passes of the MAM.  grid = B, 256 threads.
__global__ __launch_bounds__(256) void mam_selection_kernel(const int32_t* __restrict__ ctx_len, int32_t bs,
                                                            int32_t max_blocks, int32_t n_sink, int32_t n_local,
                                                            int32_t* __restrict__ sel_all,
                                                            int32_t* __restrict__ cnt_all,
                                                            int32_t* __restrict__ sel_mid,
                                                            int32_t* __restrict__ cnt_mid, int32_t* status) {
    const int r = blockIdx.x;
    const int64_t L = ctx_len[r];
    int64_t n = L > 0 ? (L + bs - 1) / bs : 0;
    if (n > max_blocks) {  // the table row cannot hold this request
        if (threadIdx.x == 0) report(status, PULSE_ERR_BAD_INDEX);
        n = 0;
    }
    const int64_t lo = n_sink, hi = n - n_local;
    const int64_t n_mid = hi > lo ? hi - lo : 0;
    int32_t* all = sel_all + (size_t)r * max_blocks;
    int32_t* mid = sel_mid + (size_t)r * max_blocks;
    for (int64_t j = threadIdx.x; j < max_blocks; j += blockDim.x) {
        all[j] = j < n ? (int32_t)j : -1;
        mid[j] = j < n_mid ? (int32_t)(lo + j) : -1;
    }
    if (threadIdx.x == 0) {
        cnt_all[r] = (int32_t)n;
        cnt_mid[r] = (int32_t)n_mid;
    }
}

// mam[r][h] = (1/G) sum_g exp(lse_mid[r][hG+g] - lse_all[r][hG+g]).
__global__ __launch_bounds__(256) void mam_finalize_kernel(const float* __restrict__ lse_all,
                                                           const float* __restrict__ lse_mid, int32_t B, int32_t Hkv,
                                                           int32_t G, float* __restrict__ mam) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (int64_t)B * Hkv) return;
    const int64_t r = i / Hkv, h = i % Hkv;
    float s = 0.f;
    for (int g = 0; g < G; ++g) {
        const int64_t k = r * Hkv * G + h * G + g;
        const float la = lse_all[k], lm = lse_mid[k];
        s += (lm == -INFINITY || la == -INFINITY) ? 0.f : expf(lm - la);
    }
    mam[i] = s / (float)G;
}

hipError_t launch_mam_selection(const int32_t* ctx_len, int32_t B, int32_t bs, int32_t max_blocks, int32_t n_sink,
                                int32_t n_local, int32_t* sel_all, int32_t* cnt_all, int32_t* sel_mid,
                                int32_t* cnt_mid, int32_t* status, hipStream_t st) {
    hipLaunchKernelGGL(mam_selection_kernel, dim3((unsigned)B), dim3(256), 0, st, ctx_len, bs, max_blocks, n_sink,
                       n_local, sel_all, cnt_all, sel_mid, cnt_mid, status);
    return hipGetLastError();
}

hipError_t launch_mam_finalize(const float* lse_all, const float* lse_mid, int32_t B, int32_t Hkv, int32_t G,
                               float* mam, hipStream_t st) {
    const int64_t n = (int64_t)B * Hkv;
    hipLaunchKernelGGL(mam_finalize_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, lse_all, lse_mid, B,
                       Hkv, G, mam);
    return hipGetLastError();
}

}  // namespace pulse
