/*
 * pulse_oracle.c -- CPU oracle for the per-layer decode hot path of
 * I/O-centric sparse KV-cache offloading (PulseInfer, arXiv 2609.34555).
 *
 * TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT.  Only the test-suite, the
 * smoke check and the benchmark's CPU-baseline leg load this library.  It
 * shares no code, header, table or helper with the GPU library; the block
 * layout below is restated here from its specification.
 *
 * Plain scalar C99, fp64 arithmetic, no blocking, fusion or reordering.
 * Passages followed:
 *   - sparse-offload workflow: select the top-k blocks, take the set
 *     difference against the GPU-resident hot set, copy the missing blocks
 *     from DRAM to the GPU (Sec. 2.2 and its figure of the offloading flow);
 *   - Quest-style per-block key digests and query-digest scores (Sec. 2.1,
 *     Sec. 4.4.1, where the averaged strategy speaks of query-digest scores);
 *   - SoloHead: one KV head keeps digests and selects a top-k block set that
 *     every KV head of the layer shares (Sec. 4.4.1);
 *   - hot set = sink + local + selected middle tokens; sink and local stay
 *     resident and only middle tokens are recalled (Sec. 4.2, Sec. 5 setup);
 *   - Middle Attention Mass, Eq. 2, averaged over the GQA query heads of a
 *     KV head (Sec. 4.4.1);
 *   - gather the scattered blocks, one large copy, scatter into the GPU KV
 *     cache (Sec. 4.4.2).
 *
 * Readings taken where the paper is silent (numbered as in the repository's
 * list of readings; R10-R12 concern inputs and tests, not this arithmetic):
 *   R1  digest = per-block, per-channel min and max of the keys over the
 *       block's valid tokens, kept in the KV dtype; -0 orders below +0.
 *   R2  score = (1/G) * sum_g sum_c max(q_gc*mn_c, q_gc*mx_c) over the G
 *       query heads of the solo KV head (mean of per-query-head bounds);
 *       no 1/sqrt(d) factor (it does not change the ranking).
 *   R3  the selection decision is taken on the exact score rounded once to
 *       fp32.
 *   R4  equal fp32 keys are ordered by ascending block index; the selection
 *       is emitted in ascending block order.
 *   R5  forced blocks: the first n_sink and the last n_local blocks of a
 *       request; k' = min(max(k_mid,0), #middle) middle blocks are chosen.
 *   R6  missing blocks are taken in (request asc, listed order) order; the
 *       i-th gets free_slots[free_head + i].
 *   R7  a run is a maximal stretch of listed missing blocks of one request
 *       whose indices increase by exactly one.
 *   R8  digests and attention use the valid tokens of a partial last block
 *       only.
 *   R9  attention: softmax over the valid tokens of the selected blocks of
 *       sm_scale * q.k, output sum_t p_t v_t, lse = log sum_t exp(logit_t);
 *       an empty selection gives out = 0, lse = -inf; the KV head of query
 *       head hq is hq / G (consecutive GQA groups).
 *   R13 MAM's middle tokens are those outside the sink and local token
 *       counts the caller passes (block-aligned counts give the blocks that
 *       selection ranks).
 *   R14 (pulse_oracle.py) the Average strategy averages the per-KV-head
 *       scores of R2 over the KV heads: the mean over all query heads.
 *
 * Block layout, in 16-bit elements, of one KV block of Hkv heads (host store
 * and slot pool alike):
 *   K(h, t, c) at ((0 * Hkv + h) * bs + t) * d + c        token-major keys
 *   V(h, t, c) at Hkv*bs*d + (h * d + c) * bs + t         channel-major values
 * Global block b of request r is blk_off[r] + j; its first element is at
 * b * 2 * Hkv * bs * d.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define OR_F16 0
#define OR_BF16 1

/* status codes restated from the boundary's specification */
#define OR_OK 0
#define OR_ERR_INVALID_ARG 1
#define OR_ERR_POOL_EXHAUSTED 4
#define OR_ERR_SELECT_OVERFLOW 5
#define OR_ERR_BAD_INDEX 7

/* ---- element decoding (exact widening to double) ---------------------- */

double or_decode(uint16_t bits, int dtype) {
    if (dtype == OR_BF16) {
        uint32_t u = ((uint32_t)bits) << 16;
        float f;
        memcpy(&f, &u, sizeof f);
        return (double)f;
    }
    /* IEEE binary16 */
    int sign = bits >> 15;
    int ex = (bits >> 10) & 0x1f;
    int man = bits & 0x3ff;
    double v;
    if (ex == 0)
        v = ldexp((double)man, -24);
    else if (ex == 31)
        v = man ? NAN : INFINITY;
    else
        v = ldexp((double)(man + 1024), ex - 25);
    return sign ? -v : v;
}

static int64_t kv_elems_per_block(int Hkv, int bs, int d) { return (int64_t)2 * Hkv * bs * d; }

static int64_t k_at(int Hkv, int bs, int d, int h, int t, int c) {
    (void)Hkv;
    return ((int64_t)h * bs + t) * d + c;
}

static int64_t v_at(int Hkv, int bs, int d, int h, int t, int c) {
    return (int64_t)Hkv * bs * d + ((int64_t)h * d + c) * bs + t;
}

static int valid_tokens(int64_t ctx, int64_t j, int bs) {
    int64_t v = ctx - j * bs;
    if (v >= bs) return bs;
    return v > 0 ? (int)v : 0;
}

/* blk_off must describe ceil(ctx_len / bs) blocks per request */
static int check_layout(const int64_t* blk_off, const int32_t* ctx_len, int B, int bs) {
    if (blk_off[0] != 0) return OR_ERR_INVALID_ARG;
    for (int r = 0; r < B; ++r) {
        int64_t n = blk_off[r + 1] - blk_off[r];
        if (ctx_len[r] < 0 || n != ((int64_t)ctx_len[r] + bs - 1) / bs) return OR_ERR_INVALID_ARG;
    }
    return OR_OK;
}

/* -0 orders below +0 (R1); inputs are finite */
static int value_less(uint16_t a, uint16_t b, int dtype) {
    double x = or_decode(a, dtype), y = or_decode(b, dtype);
    if (x < y) return 1;
    if (x > y) return 0;
    return (a >> 15) && !(b >> 15);
}

/* ---- a1: per-block key digest of one KV head (Sec. 2.1, Sec. 4.4.1; R1) -- */

int or_build_digests(const uint16_t* kv, const int64_t* blk_off, const int32_t* ctx_len, int B,
                     int Hkv, int bs, int d, int dtype, int kv_head, uint16_t* digests) {
    if (check_layout(blk_off, ctx_len, B, bs)) return OR_ERR_INVALID_ARG;
    if (kv_head < 0 || kv_head >= Hkv) return OR_ERR_INVALID_ARG;
    const int64_t E = kv_elems_per_block(Hkv, bs, d);
    for (int r = 0; r < B; ++r) {
        int64_t n = blk_off[r + 1] - blk_off[r];
        for (int64_t j = 0; j < n; ++j) {
            int64_t b = blk_off[r] + j;
            const uint16_t* blk = kv + b * E;
            int nv = valid_tokens(ctx_len[r], j, bs);
            for (int c = 0; c < d; ++c) {
                uint16_t mn = blk[k_at(Hkv, bs, d, kv_head, 0, c)];
                uint16_t mx = mn;
                for (int t = 1; t < nv; ++t) {
                    uint16_t x = blk[k_at(Hkv, bs, d, kv_head, t, c)];
                    if (value_less(x, mn, dtype)) mn = x;
                    if (value_less(mx, x, dtype)) mx = x;
                }
                digests[(b * 2 + 0) * d + c] = mn;
                digests[(b * 2 + 1) * d + c] = mx;
            }
        }
    }
    return OR_OK;
}

/* ---- a2: query-digest score of the solo head (Sec. 4.4.1; R2) ---------- */

int or_score(const uint16_t* q, const uint16_t* digests, const int64_t* blk_off, int B, int Hq,
             int Hkv, int d, int dtype, int solo_kv_head, double* scores) {
    if (Hkv <= 0 || Hq % Hkv) return OR_ERR_INVALID_ARG;
    if (solo_kv_head < 0 || solo_kv_head >= Hkv) return OR_ERR_INVALID_ARG;
    const int G = Hq / Hkv;
    for (int r = 0; r < B; ++r) {
        for (int64_t b = blk_off[r]; b < blk_off[r + 1]; ++b) {
            double s = 0.0;
            for (int g = 0; g < G; ++g) {
                const uint16_t* qr = q + ((int64_t)r * Hq + (int64_t)solo_kv_head * G + g) * d;
                for (int c = 0; c < d; ++c) {
                    double qc = or_decode(qr[c], dtype);
                    double lo = qc * or_decode(digests[(b * 2 + 0) * d + c], dtype);
                    double hi = qc * or_decode(digests[(b * 2 + 1) * d + c], dtype);
                    s += lo > hi ? lo : hi;
                }
            }
            scores[b] = s / G;
        }
    }
    return OR_OK;
}

/* ---- a3: SoloHead top-k block selection (Sec. 4.4.1, Sec. 5 setup; R3-R5) */

typedef struct {
    float key;
    int32_t j;
} cand_t;

static int cand_cmp(const void* pa, const void* pb) {
    const cand_t* a = (const cand_t*)pa;
    const cand_t* b = (const cand_t*)pb;
    if (a->key > b->key) return -1;
    if (a->key < b->key) return 1;
    return (a->j > b->j) - (a->j < b->j);
}

int or_select(const double* scores, const int64_t* blk_off, int B, const int32_t* k_mid,
              int n_sink, int n_local, int k_max, int32_t* sel_idx, int32_t* sel_cnt) {
    if (n_sink < 0 || n_local < 0 || k_max < 1) return OR_ERR_INVALID_ARG;
    int status = OR_OK;
    for (int r = 0; r < B; ++r) {
        int64_t n = blk_off[r + 1] - blk_off[r];
        int32_t* out = sel_idx + (int64_t)r * k_max;
        for (int i = 0; i < k_max; ++i) out[i] = -1;
        char* chosen = (char*)calloc(n > 0 ? (size_t)n : 1, 1);
        cand_t* cand = (cand_t*)malloc((n > 0 ? (size_t)n : 1) * sizeof(cand_t));
        int64_t nc = 0;
        for (int64_t j = 0; j < n; ++j) {
            int forced = j < n_sink || j >= n - n_local;
            if (forced) {
                chosen[j] = 1;
            } else {
                cand[nc].key = (float)scores[blk_off[r] + j];
                cand[nc].j = (int32_t)j;
                ++nc;
            }
        }
        int64_t k = k_mid[r] < 0 ? 0 : k_mid[r];
        if (k > nc) k = nc;
        qsort(cand, (size_t)nc, sizeof(cand_t), cand_cmp);
        for (int64_t i = 0; i < k; ++i) chosen[cand[i].j] = 1;
        int64_t cnt = 0;
        for (int64_t j = 0; j < n; ++j) cnt += chosen[j];
        if (cnt > k_max) {
            status = OR_ERR_SELECT_OVERFLOW;
            sel_cnt[r] = 0;
        } else {
            int64_t p = 0;
            for (int64_t j = 0; j < n; ++j)
                if (chosen[j]) out[p++] = (int32_t)j;
            sel_cnt[r] = (int32_t)cnt;
        }
        free(chosen);
        free(cand);
    }
    return status;
}

/* ---- a4-a6: set difference, slot allocation, gather-scatter recall
 *      (Sec. 2.2, Sec. 4.4.2; R6, R7) -------------------------------------- */

int or_recall(const uint8_t* host_kv, const int64_t* blk_off, int B, const int32_t* sel_idx,
              const int32_t* sel_cnt, int k_max, int32_t* table, int max_blocks,
              const int32_t* free_slots, int32_t* free_head, int n_free, uint8_t* pool, int n_slots,
              int64_t unit_bytes, int64_t* stats /* n_missing, n_runs, bytes */) {
    /* validate every index before any state changes */
    int64_t total = 0, runs = 0;
    for (int r = 0; r < B; ++r) {
        int64_t n = blk_off[r + 1] - blk_off[r];
        if (sel_cnt[r] < 0 || sel_cnt[r] > k_max) return OR_ERR_BAD_INDEX;
        int32_t prev_missing = -2;
        for (int i = 0; i < sel_cnt[r]; ++i) {
            int32_t j = sel_idx[(int64_t)r * k_max + i];
            if (j < 0 || j >= n || j >= max_blocks) return OR_ERR_BAD_INDEX;
            if (i > 0 && j <= sel_idx[(int64_t)r * k_max + i - 1]) return OR_ERR_BAD_INDEX;
            int32_t slot = table[(int64_t)r * max_blocks + j];
            if (slot >= n_slots) return OR_ERR_BAD_INDEX;
            if (slot < 0) {
                if (j != prev_missing + 1) ++runs;
                prev_missing = j;
                ++total;
            }
        }
    }
    stats[0] = total;
    stats[1] = runs;
    stats[2] = 0;
    if (*free_head < 0 || *free_head > n_free) return OR_ERR_BAD_INDEX;
    if (total > (int64_t)n_free - *free_head) return OR_ERR_POOL_EXHAUSTED;
    for (int64_t g = 0; g < total; ++g) {
        int32_t slot = free_slots[*free_head + g];
        if (slot < 0 || slot >= n_slots) return OR_ERR_BAD_INDEX;
    }
    /* allocate and copy, in (request asc, listed order) order */
    int64_t g = 0;
    for (int r = 0; r < B; ++r) {
        for (int i = 0; i < sel_cnt[r]; ++i) {
            int32_t j = sel_idx[(int64_t)r * k_max + i];
            int32_t* entry = table + (int64_t)r * max_blocks + j;
            if (*entry >= 0) continue;
            int32_t slot = free_slots[*free_head + g];
            *entry = slot;
            memcpy(pool + (int64_t)slot * unit_bytes, host_kv + (blk_off[r] + j) * unit_bytes,
                   (size_t)unit_bytes);
            ++g;
        }
    }
    *free_head += (int32_t)total;
    stats[2] = total * unit_bytes;
    return OR_OK;
}

/* ---- a7: sparse GQA decode attention over the selected blocks
 *      (Sec. 2.2 attention after recall, Sec. 4.2.1; R8, R9) --------------- */

static void attend_one(const uint16_t* qrow, const uint16_t* const* blocks, const int* nvalid,
                       int nb, int Hkv, int bs, int d, int dtype, int h, double sm_scale,
                       double* out, double* lse) {
    int64_t ntok = 0;
    for (int i = 0; i < nb; ++i) ntok += nvalid[i];
    for (int c = 0; c < d; ++c) out[c] = 0.0;
    if (ntok == 0) {
        *lse = -INFINITY;
        return;
    }
    double* logit = (double*)malloc((size_t)ntok * sizeof(double));
    int64_t p = 0;
    double m = -INFINITY;
    for (int i = 0; i < nb; ++i)
        for (int t = 0; t < nvalid[i]; ++t) {
            double s = 0.0;
            for (int c = 0; c < d; ++c)
                s += or_decode(qrow[c], dtype) * or_decode(blocks[i][k_at(Hkv, bs, d, h, t, c)], dtype);
            s *= sm_scale;
            logit[p++] = s;
            if (s > m) m = s;
        }
    double denom = 0.0;
    for (int64_t u = 0; u < ntok; ++u) denom += exp(logit[u] - m);
    p = 0;
    for (int i = 0; i < nb; ++i)
        for (int t = 0; t < nvalid[i]; ++t) {
            double w = exp(logit[p++] - m) / denom;
            for (int c = 0; c < d; ++c) out[c] += w * or_decode(blocks[i][v_at(Hkv, bs, d, h, t, c)], dtype);
        }
    *lse = m + log(denom);
    free(logit);
}

int or_attention(const uint16_t* q, const uint16_t* pool, int n_slots, const int32_t* table,
                 int max_blocks, const int32_t* sel_idx, const int32_t* sel_cnt, int k_max,
                 const int64_t* blk_off, const int32_t* ctx_len, int B, int Hq, int Hkv, int bs, int d,
                 int dtype, double sm_scale, double* out, double* lse) {
    if (Hkv <= 0 || Hq % Hkv) return OR_ERR_INVALID_ARG;
    if (check_layout(blk_off, ctx_len, B, bs)) return OR_ERR_INVALID_ARG;
    const int G = Hq / Hkv;
    const int64_t E = kv_elems_per_block(Hkv, bs, d);
    const uint16_t** blocks = (const uint16_t**)malloc((size_t)(k_max > 0 ? k_max : 1) * sizeof(void*));
    int* nvalid = (int*)malloc((size_t)(k_max > 0 ? k_max : 1) * sizeof(int));
    int status = OR_OK;
    for (int r = 0; r < B && status == OR_OK; ++r) {
        int64_t n = blk_off[r + 1] - blk_off[r];
        int nb = sel_cnt[r];
        if (nb < 0 || nb > k_max) {
            status = OR_ERR_BAD_INDEX;
            break;
        }
        for (int i = 0; i < nb; ++i) {
            int32_t j = sel_idx[(int64_t)r * k_max + i];
            if (j < 0 || j >= n || j >= max_blocks) {
                status = OR_ERR_BAD_INDEX;
                break;
            }
            int32_t slot = table[(int64_t)r * max_blocks + j];
            if (slot < 0 || slot >= n_slots) {
                status = OR_ERR_BAD_INDEX;
                break;
            }
            blocks[i] = pool + (int64_t)slot * E;
            nvalid[i] = valid_tokens(ctx_len[r], j, bs);
        }
        if (status != OR_OK) break;
        for (int hq = 0; hq < Hq; ++hq)
            attend_one(q + ((int64_t)r * Hq + hq) * d, blocks, nvalid, nb, Hkv, bs, d, dtype, hq / G,
                       sm_scale, out + ((int64_t)r * Hq + hq) * d, lse + (int64_t)r * Hq + hq);
    }
    free(blocks);
    free(nvalid);
    return status;
}

/* dense reference: every block of the request, read from the host store */
int or_dense_attention(const uint16_t* q, const uint16_t* host_kv, const int64_t* blk_off,
                       const int32_t* ctx_len, int B, int Hq, int Hkv, int bs, int d, int dtype,
                       double sm_scale, double* out, double* lse) {
    if (Hkv <= 0 || Hq % Hkv) return OR_ERR_INVALID_ARG;
    if (check_layout(blk_off, ctx_len, B, bs)) return OR_ERR_INVALID_ARG;
    const int G = Hq / Hkv;
    const int64_t E = kv_elems_per_block(Hkv, bs, d);
    for (int r = 0; r < B; ++r) {
        int64_t n = blk_off[r + 1] - blk_off[r];
        const uint16_t** blocks = (const uint16_t**)malloc((size_t)(n > 0 ? n : 1) * sizeof(void*));
        int* nvalid = (int*)malloc((size_t)(n > 0 ? n : 1) * sizeof(int));
        for (int64_t j = 0; j < n; ++j) {
            blocks[j] = host_kv + (blk_off[r] + j) * E;
            nvalid[j] = valid_tokens(ctx_len[r], j, bs);
        }
        for (int hq = 0; hq < Hq; ++hq)
            attend_one(q + ((int64_t)r * Hq + hq) * d, blocks, nvalid, (int)n, Hkv, bs, d, dtype, hq / G,
                       sm_scale, out + ((int64_t)r * Hq + hq) * d, lse + (int64_t)r * Hq + hq);
        free(blocks);
        free(nvalid);
    }
    return OR_OK;
}

/* ---- Middle Attention Mass, Eq. 2, for one request (Sec. 4.4.1) --------
 * MAM_q = sum over middle tokens of the softmax attention weight of query
 * head q over all context tokens; middle excludes the first n_sink_tok and
 * the last n_local_tok tokens.  KV-head MAM = mean over its GQA query heads.
 * Returns the KV head of highest MAM (lowest index on ties) or -1. */
int or_mam(const uint16_t* q, const uint16_t* host_kv, const int64_t* blk_off, const int32_t* ctx_len,
           int r, int Hq, int Hkv, int bs, int d, int dtype, double sm_scale, int n_sink_tok,
           int n_local_tok, double* mam_q, double* mam_h) {
    if (Hkv <= 0 || Hq % Hkv) return -1;
    const int G = Hq / Hkv;
    const int64_t E = kv_elems_per_block(Hkv, bs, d);
    const int64_t L = ctx_len[r];
    if (L <= 0) return -1;
    double* logit = (double*)malloc((size_t)L * sizeof(double));
    for (int hq = 0; hq < Hq; ++hq) {
        const uint16_t* qrow = q + ((int64_t)r * Hq + hq) * d;
        int h = hq / G;
        double m = -INFINITY;
        for (int64_t t = 0; t < L; ++t) {
            const uint16_t* blk = host_kv + (blk_off[r] + t / bs) * E;
            double s = 0.0;
            for (int c = 0; c < d; ++c)
                s += or_decode(qrow[c], dtype) * or_decode(blk[k_at(Hkv, bs, d, h, (int)(t % bs), c)], dtype);
            logit[t] = s * sm_scale;
            if (logit[t] > m) m = logit[t];
        }
        double denom = 0.0, middle = 0.0;
        for (int64_t t = 0; t < L; ++t) {
            double e = exp(logit[t] - m);
            denom += e;
            if (t >= n_sink_tok && t < L - n_local_tok) middle += e;
        }
        mam_q[hq] = middle / denom;
    }
    int best = 0;
    for (int h = 0; h < Hkv; ++h) {
        double s = 0.0;
        for (int g = 0; g < G; ++g) s += mam_q[h * G + g];
        mam_h[h] = s / G;
        if (mam_h[h] > mam_h[best]) best = h;
    }
    free(logit);
    return best;
}
