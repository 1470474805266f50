/*
 * abi_parity.c -- one decode layer-step through the C ABI of libpulse.so, from
 * plain C (no Python, no torch), checked stage by stage against the CPU oracle
 * (liboracle.so, test infrastructure) on the same inputs.
 *
 * Workload: 2 ragged requests (700 and 1234 tokens, partial last blocks),
 * block 16, 8 query / 2 KV heads (G = 4), head_dim 128, bf16, seeded uniform
 * K / V / q, sink 1 + local 2 blocks forced, 10 and 20 middle blocks chosen,
 * some middle blocks already resident in the slot pool.
 *
 * Checks: digests bit-exact; selection exact up to near-ties at the k-th
 * score (1e-5 relative, the tie rule of the tests); block table, free-list
 * head, recall statistics and every pool byte exact; attention output and
 * log-sum-exp within 2e-3.  Exit status 0 on success.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "pulse.h"

/* the oracle's entry points (oracle/pulse_oracle.c) */
int or_build_digests(const uint16_t* kv, const int64_t* blk_off, const int32_t* ctx_len, int B, int Hkv, int bs,
                     int d, int dtype, int kv_head, uint16_t* digests);
int or_score(const uint16_t* q, const uint16_t* digests, const int64_t* blk_off, int B, int Hq, int Hkv, int d,
             int dtype, int solo_kv_head, double* scores);
int or_select(const double* scores, const int64_t* blk_off, int B, const int32_t* k_mid, int n_sink, int n_local,
              int k_max, int32_t* sel_idx, int32_t* sel_cnt);
int or_recall(const uint8_t* host_kv, const int64_t* blk_off, int B, const int32_t* sel_idx, const int32_t* sel_cnt,
              int k_max, int32_t* table, int max_blocks, const int32_t* free_slots, int32_t* free_head, int n_free,
              uint8_t* pool, int n_slots, int64_t unit_bytes, int64_t* stats);
int or_attention(const uint16_t* q, const uint16_t* pool, int n_slots, const int32_t* table, int max_blocks,
                 const int32_t* sel_idx, const int32_t* sel_cnt, int k_max, const int64_t* blk_off,
                 const int32_t* ctx_len, int B, int Hq, int Hkv, int bs, int d, int dtype, double sm_scale,
                 double* out, double* lse);

enum { B = 2, HQ = 8, HKV = 2, D = 128, BS = 16, K_MAX = 32, N_SINK = 1, N_LOCAL = 2, SOLO = 1 };

#define CHECK_HIP(x)                                                            \
    do {                                                                        \
        hipError_t e_ = (x);                                                    \
        if (e_ != hipSuccess) {                                                 \
            fprintf(stderr, "%s:%d %s: %s\n", __FILE__, __LINE__, #x,          \
                    hipGetErrorString(e_));                                     \
            return 2;                                                           \
        }                                                                       \
    } while (0)
#define CHECK_PULSE(x)                                                          \
    do {                                                                        \
        pulse_status s_ = (x);                                                  \
        if (s_ != PULSE_OK) {                                                   \
            fprintf(stderr, "%s:%d %s: %s\n", __FILE__, __LINE__, #x,          \
                    pulse_status_string(s_));                                   \
            return 2;                                                           \
        }                                                                       \
    } while (0)
#define EXPECT(cond, ...)                                                       \
    do {                                                                        \
        if (!(cond)) {                                                          \
            fprintf(stderr, "mismatch: " __VA_ARGS__);                          \
            fputc('\n', stderr);                                                \
            return 1;                                                           \
        }                                                                       \
    } while (0)

static uint64_t rng_state = 0x9E3779B97F4A7C15ull;
static double uniform(void) { /* xorshift64*: uniform in [0, 1) */
    rng_state ^= rng_state >> 12;
    rng_state ^= rng_state << 25;
    rng_state ^= rng_state >> 27;
    return (double)((rng_state * 0x2545F4914F6CDD1Dull) >> 11) * 0x1.0p-53;
}
static int desc(const void* a, const void* b) {
    const float x = *(const float*)a, y = *(const float*)b;
    return (x < y) - (x > y);
}
static uint16_t to_bf16(float f) { /* round to nearest even */
    uint32_t u;
    memcpy(&u, &f, 4);
    return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

int main(void) {
    const int32_t ctx[B] = {700, 1234};
    int64_t blk_off[B + 1] = {0};
    int32_t n_blk[B];
    for (int r = 0; r < B; ++r) {
        n_blk[r] = (ctx[r] + BS - 1) / BS;
        blk_off[r + 1] = blk_off[r] + n_blk[r];
    }
    const int64_t total = blk_off[B];
    const int max_blocks = n_blk[1] > n_blk[0] ? n_blk[1] : n_blk[0];
    const int64_t E = 2LL * HKV * BS * D; /* elements per block */
    const int64_t U = E * 2;              /* bytes per block */
    const pulse_shape shape = {HQ, HKV, D, BS, PULSE_BF16};
    if ((int64_t)pulse_block_bytes(&shape) != U) return 2;

    /* host store (pinned, host-mapped): K token-major then V channel-major per block; padding tokens zero */
    uint16_t* host = NULL;
    CHECK_PULSE(pulse_host_alloc((size_t)(total * U), 1, (void**)&host));
    for (int r = 0; r < B; ++r)
        for (int j = 0; j < n_blk[r]; ++j) {
            uint16_t* blk = host + (blk_off[r] + j) * E;
            for (int64_t e = 0; e < E; ++e) {
                const int64_t kv_split = (int64_t)HKV * BS * D;
                const int t = e < kv_split ? (int)((e / D) % BS) : (int)((e - kv_split) % BS);
                const int valid = j * BS + t < ctx[r];
                blk[e] = valid ? to_bf16((float)(4.0 * uniform() - 2.0)) : 0;
            }
        }
    uint16_t q[B * HQ * D];
    for (int i = 0; i < B * HQ * D; ++i) q[i] = to_bf16((float)(2.0 * uniform() - 1.0));

    /* resident set: sink, local and every 7th middle block; slots 0.. in (request, block) order */
    int32_t* table0 = malloc(sizeof(int32_t) * B * max_blocks);
    for (int i = 0; i < B * max_blocks; ++i) table0[i] = -1;
    int n_res = 0;
    for (int r = 0; r < B; ++r)
        for (int j = 0; j < n_blk[r]; ++j)
            if (j < N_SINK || j >= n_blk[r] - N_LOCAL || j % 7 == 3) table0[r * max_blocks + j] = n_res++;
    const int n_slots = n_res + B * K_MAX, n_free = B * K_MAX;
    int32_t* free_slots = malloc(sizeof(int32_t) * n_free);
    for (int i = 0; i < n_free; ++i) free_slots[i] = n_res + i;
    uint8_t* pool0 = calloc((size_t)n_slots, (size_t)U);
    for (int r = 0; r < B; ++r)
        for (int j = 0; j < n_blk[r]; ++j) {
            const int32_t s = table0[r * max_blocks + j];
            if (s >= 0) memcpy(pool0 + (int64_t)s * U, (uint8_t*)host + (blk_off[r] + j) * U, (size_t)U);
        }
    const int32_t k_mid[B] = {10, 20};

    /* device buffers */
    int64_t* d_blk_off;
    int32_t *d_ctx, *d_kmid, *d_sel, *d_cnt, *d_table, *d_free, *d_fh, *d_status;
    uint16_t *d_q, *d_dig;
    uint8_t* d_pool;
    pulse_recall_stats* d_stats;
    float *d_out, *d_lse;
    void* d_ws;
    const size_t ws_bytes = pulse_workspace_bytes(&shape, B, K_MAX, total);
    CHECK_HIP(hipMalloc((void**)&d_blk_off, sizeof(blk_off)));
    CHECK_HIP(hipMalloc((void**)&d_ctx, sizeof(ctx)));
    CHECK_HIP(hipMalloc((void**)&d_kmid, sizeof(k_mid)));
    CHECK_HIP(hipMalloc((void**)&d_sel, sizeof(int32_t) * B * K_MAX));
    CHECK_HIP(hipMalloc((void**)&d_cnt, sizeof(int32_t) * B));
    CHECK_HIP(hipMalloc((void**)&d_table, sizeof(int32_t) * B * max_blocks));
    CHECK_HIP(hipMalloc((void**)&d_free, sizeof(int32_t) * n_free));
    CHECK_HIP(hipMalloc((void**)&d_fh, sizeof(int32_t)));
    CHECK_HIP(hipMalloc((void**)&d_status, sizeof(int32_t)));
    CHECK_HIP(hipMalloc((void**)&d_q, sizeof(q)));
    CHECK_HIP(hipMalloc((void**)&d_dig, sizeof(uint16_t) * total * 2 * D));
    CHECK_HIP(hipMalloc((void**)&d_pool, (size_t)n_slots * U));
    CHECK_HIP(hipMalloc((void**)&d_stats, sizeof(pulse_recall_stats)));
    CHECK_HIP(hipMalloc((void**)&d_out, sizeof(float) * B * HQ * D));
    CHECK_HIP(hipMalloc((void**)&d_lse, sizeof(float) * B * HQ));
    CHECK_HIP(hipMalloc(&d_ws, ws_bytes));
    CHECK_HIP(hipMemcpy(d_blk_off, blk_off, sizeof(blk_off), hipMemcpyHostToDevice));
    CHECK_HIP(hipMemcpy(d_ctx, ctx, sizeof(ctx), hipMemcpyHostToDevice));
    CHECK_HIP(hipMemcpy(d_kmid, k_mid, sizeof(k_mid), hipMemcpyHostToDevice));
    CHECK_HIP(hipMemcpy(d_table, table0, sizeof(int32_t) * B * max_blocks, hipMemcpyHostToDevice));
    CHECK_HIP(hipMemcpy(d_free, free_slots, sizeof(int32_t) * n_free, hipMemcpyHostToDevice));
    CHECK_HIP(hipMemcpy(d_q, q, sizeof(q), hipMemcpyHostToDevice));
    CHECK_HIP(hipMemcpy(d_pool, pool0, (size_t)n_slots * U, hipMemcpyHostToDevice));
    CHECK_HIP(hipMemset(d_fh, 0, sizeof(int32_t)));
    CHECK_HIP(hipMemset(d_status, 0, sizeof(int32_t)));
    CHECK_HIP(hipMemset(d_stats, 0, sizeof(pulse_recall_stats)));

    /* a1 digests of the solo head, then one chained layer-step */
    CHECK_PULSE(pulse_build_digests(&shape, host, d_blk_off, d_ctx, B, total, SOLO, d_dig, d_status, NULL));
    pulse_layer_args a;
    memset(&a, 0, sizeof(a));
    a.shape = shape;
    a.B = B;
    a.total_blocks = total;
    a.ctx_len = d_ctx;
    a.blk_off = d_blk_off;
    a.q = d_q;
    a.digests = d_dig;
    a.solo_kv_head = SOLO;
    a.k_mid = d_kmid;
    a.n_sink_blocks = N_SINK;
    a.n_local_blocks = N_LOCAL;
    a.k_max = K_MAX;
    a.sel_idx = d_sel;
    a.sel_cnt = d_cnt;
    a.host_kv = host;
    a.block_table = d_table;
    a.max_blocks = max_blocks;
    a.free_slots = d_free;
    a.free_head = d_fh;
    a.n_free = n_free;
    a.slot_pool = d_pool;
    a.n_slots = n_slots;
    a.stats = d_stats;
    a.sm_scale = (float)(1.0 / sqrt((double)D));
    a.out = d_out;
    a.lse = d_lse;
    a.dev_status = d_status;
    a.ws = d_ws;
    a.ws_bytes = ws_bytes;
    CHECK_PULSE(pulse_decode_layer(&a, NULL));
    CHECK_HIP(hipDeviceSynchronize());

    int32_t status = -1, fh = -1, gcnt[B], gsel[B * K_MAX];
    pulse_recall_stats gstats;
    uint16_t* gdig = malloc(sizeof(uint16_t) * total * 2 * D);
    int32_t* gtable = malloc(sizeof(int32_t) * B * max_blocks);
    uint8_t* gpool = malloc((size_t)n_slots * U);
    float gout[B * HQ * D], glse[B * HQ];
    CHECK_HIP(hipMemcpy(&status, d_status, sizeof(int32_t), hipMemcpyDeviceToHost));
    CHECK_HIP(hipMemcpy(&fh, d_fh, sizeof(int32_t), hipMemcpyDeviceToHost));
    CHECK_HIP(hipMemcpy(gcnt, d_cnt, sizeof(gcnt), hipMemcpyDeviceToHost));
    CHECK_HIP(hipMemcpy(gsel, d_sel, sizeof(gsel), hipMemcpyDeviceToHost));
    CHECK_HIP(hipMemcpy(&gstats, d_stats, sizeof(gstats), hipMemcpyDeviceToHost));
    CHECK_HIP(hipMemcpy(gdig, d_dig, sizeof(uint16_t) * total * 2 * D, hipMemcpyDeviceToHost));
    CHECK_HIP(hipMemcpy(gtable, d_table, sizeof(int32_t) * B * max_blocks, hipMemcpyDeviceToHost));
    CHECK_HIP(hipMemcpy(gpool, d_pool, (size_t)n_slots * U, hipMemcpyDeviceToHost));
    CHECK_HIP(hipMemcpy(gout, d_out, sizeof(gout), hipMemcpyDeviceToHost));
    CHECK_HIP(hipMemcpy(glse, d_lse, sizeof(glse), hipMemcpyDeviceToHost));
    EXPECT(status == 0, "device status %s", pulse_status_string((pulse_status)status));

    /* digests: bit-exact */
    uint16_t* odig = malloc(sizeof(uint16_t) * total * 2 * D);
    EXPECT(or_build_digests(host, blk_off, ctx, B, HKV, BS, D, PULSE_BF16, SOLO, odig) == 0, "oracle digests");
    EXPECT(memcmp(odig, gdig, sizeof(uint16_t) * total * 2 * D) == 0, "digests differ");

    /* selection: equal counts; a differing block only at a near-tie with the k-th middle score */
    double* osc = malloc(sizeof(double) * total);
    int32_t osel[B * K_MAX], ocnt[B];
    EXPECT(or_score(q, odig, blk_off, B, HQ, HKV, D, PULSE_BF16, SOLO, osc) == 0, "oracle score");
    EXPECT(or_select(osc, blk_off, B, k_mid, N_SINK, N_LOCAL, K_MAX, osel, ocnt) == 0, "oracle select");
    int ties = 0;
    for (int r = 0; r < B; ++r) {
        EXPECT(gcnt[r] == ocnt[r], "request %d: %d selected, oracle %d", r, gcnt[r], ocnt[r]);
        for (int i = 1; i < gcnt[r]; ++i) EXPECT(gsel[r * K_MAX + i] > gsel[r * K_MAX + i - 1], "not ascending");
        /* the k-th largest fp32 middle score (k = k_mid <= #middle here) */
        const int lo = N_SINK, hi = n_blk[r] - N_LOCAL;
        float mid[128];
        EXPECT(hi - lo <= 128 && k_mid[r] <= hi - lo, "request %d: middle blocks exceed the test's buffer", r);
        for (int j = lo; j < hi; ++j) mid[j - lo] = (float)osc[blk_off[r] + j];
        qsort(mid, (size_t)(hi - lo), sizeof(float), desc);
        const float kth = mid[k_mid[r] - 1];
        for (int pass = 0; pass < 2; ++pass) { /* blocks in one selection and not in the other */
            const int32_t* x = pass ? osel : gsel;
            const int32_t* y = pass ? gsel : osel;
            for (int i = 0; i < gcnt[r]; ++i) {
                int found = 0;
                for (int i2 = 0; i2 < gcnt[r]; ++i2) found |= y[r * K_MAX + i2] == x[r * K_MAX + i];
                if (found) continue;
                const int32_t j = x[r * K_MAX + i];
                EXPECT(j >= lo && j < hi, "request %d: forced block %d differs", r, j);
                const float v = (float)osc[blk_off[r] + j];
                EXPECT(fabsf(v - kth) <= 1e-5f * fabsf(kth), "request %d: block %d score %g, k-th %g", r, j, v, kth);
                ++ties;
            }
        }
    }

    /* recall of the GPU's selection: table, free head, statistics, every pool byte */
    int32_t* otable = malloc(sizeof(int32_t) * B * max_blocks);
    memcpy(otable, table0, sizeof(int32_t) * B * max_blocks);
    uint8_t* opool = malloc((size_t)n_slots * U);
    memcpy(opool, pool0, (size_t)n_slots * U);
    int32_t ofh = 0;
    int64_t ostats[3];
    EXPECT(or_recall((const uint8_t*)host, blk_off, B, gsel, gcnt, K_MAX, otable, max_blocks, free_slots, &ofh, n_free,
                     opool, n_slots, U, ostats) == 0,
           "oracle recall");
    EXPECT(memcmp(otable, gtable, sizeof(int32_t) * B * max_blocks) == 0, "block table differs");
    EXPECT(ofh == fh, "free head %d, oracle %d", fh, ofh);
    EXPECT(gstats.n_missing == ostats[0] && gstats.n_runs == ostats[1] && gstats.bytes == ostats[2],
           "stats (%d, %d, %lld), oracle (%lld, %lld, %lld)", gstats.n_missing, gstats.n_runs,
           (long long)gstats.bytes, (long long)ostats[0], (long long)ostats[1], (long long)ostats[2]);
    EXPECT(ostats[0] > 0, "nothing recalled");
    EXPECT(memcmp(opool, gpool, (size_t)n_slots * U) == 0, "pool bytes differ");

    /* attention over the GPU's selection */
    double oout[B * HQ * D], olse[B * HQ];
    EXPECT(or_attention(q, (const uint16_t*)opool, n_slots, otable, max_blocks, gsel, gcnt, K_MAX, blk_off, ctx, B, HQ,
                        HKV, BS, D, PULSE_BF16, (double)a.sm_scale, oout, olse) == 0,
           "oracle attention");
    double err = 0.0;
    for (int i = 0; i < B * HQ * D; ++i) err = fmax(err, fabs((double)gout[i] - oout[i]));
    for (int i = 0; i < B * HQ; ++i) err = fmax(err, fabs((double)glse[i] - olse[i]));
    EXPECT(err <= 2e-3, "attention max |gpu - oracle| = %g", err);

    printf("c abi parity ok: missing=%lld runs=%lld bytes=%lld ties=%d attn_max_err=%.2e\n", (long long)ostats[0],
           (long long)ostats[1], (long long)ostats[2], ties, err);
    CHECK_PULSE(pulse_host_free(host));
    hipFree(d_blk_off); hipFree(d_ctx); hipFree(d_kmid); hipFree(d_sel); hipFree(d_cnt); hipFree(d_table);
    hipFree(d_free); hipFree(d_fh); hipFree(d_status); hipFree(d_q); hipFree(d_dig); hipFree(d_pool);
    hipFree(d_stats); hipFree(d_out); hipFree(d_lse); hipFree(d_ws);
    free(table0); free(free_slots); free(pool0); free(gdig); free(gtable); free(gpool); free(odig); free(osc);
    free(otable); free(opool);
    return 0;
}
