/*
 * SparCML reference oracle -- TEST INFRASTRUCTURE ONLY (see oracle.h).
 *
 * Each function restates, in the plainest sequential form, a definition from
 * Renggli et al., "SparCML", arXiv 1802.08021.  Nothing here is blocked,
 * fused or reordered beyond what the definition states; the only library
 * primitives used are qsort (top-k by full sort) and sqrt.  Values are fp32
 * (the value type of the sparse streams, §5.1 "Vector Representations");
 * the QSGD norm, which the paper leaves unspecified, is accumulated in fp64.
 *
 * Build: gcc -O2 -std=c11 -ffp-contract=off -fno-fast-math -pthread -shared -fPIC.
 */
#include "oracle.h"

#include <math.h>
#include <pthread.h>
#include <stdatomic.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------------ */
/* Work items that are independent by definition (the nodes of one level of
 * the reduction tree, the ranks of top-k and quantization) may be spread
 * over threads; each item reads only its own inputs and writes only its own
 * outputs, so the results are the same bits for any thread count.  The
 * default is one thread (a plain loop). */

static int g_threads = 1;

void orc_set_threads(int n) { g_threads = n < 1 ? 1 : (n > 256 ? 256 : n); }
int orc_get_threads(void) { return g_threads; }

typedef void (*orc_item_fn)(void* ctx, int i);

typedef struct {
    orc_item_fn fn;
    void* ctx;
    int n;
    atomic_int next;
} orc_pool;

static void* pool_worker(void* arg)
{
    orc_pool* p = (orc_pool*)arg;
    for (;;) {
        int i = atomic_fetch_add(&p->next, 1);
        if (i >= p->n) break;
        p->fn(p->ctx, i);
    }
    return NULL;
}

/* fn(ctx, i) for i in [0, n): in order on the calling thread, or claimed one
 * at a time by min(threads, n) threads (the caller is one of them). */
static void for_each_item(int n, orc_item_fn fn, void* ctx)
{
    int t = g_threads < n ? g_threads : n;
    if (t <= 1) {
        for (int i = 0; i < n; ++i) fn(ctx, i);
        return;
    }
    orc_pool p;
    p.fn = fn;
    p.ctx = ctx;
    p.n = n;
    atomic_init(&p.next, 0);
    pthread_t th[256];
    int started = 0;
    for (int k = 1; k < t; ++k, ++started)
        if (pthread_create(&th[started], NULL, pool_worker, &p) != 0) break;
    pool_worker(&p); /* also finishes whatever a thread that failed to start would have taken */
    for (int k = 0; k < started; ++k) pthread_join(th[k], NULL);
}

/* ------------------------------------------------------------------------ */
/* Philox4x32-10 (Salmon et al., SC'11).  State: four 32-bit words; key: two.
 * One round multiplies words 0 and 2 by the two Philox constants, splits
 * each 64-bit product into high/low halves and mixes the high halves with
 * words 1 and 3 and the round key; the key is bumped by the two Weyl
 * constants between rounds. */
void orc_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4])
{
    const uint32_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u;
    const uint32_t W0 = 0x9E3779B9u, W1 = 0xBB67AE85u;
    uint32_t x0 = ctr[0], x1 = ctr[1], x2 = ctr[2], x3 = ctr[3];
    uint32_t k0 = key[0], k1 = key[1];
    for (int round = 0; round < 10; ++round) {
        if (round > 0) {
            k0 += W0;
            k1 += W1;
        }
        uint64_t p0 = (uint64_t)M0 * (uint64_t)x0;
        uint64_t p1 = (uint64_t)M1 * (uint64_t)x2;
        uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
        uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
        uint32_t y0 = hi1 ^ x1 ^ k0;
        uint32_t y1 = lo1;
        uint32_t y2 = hi0 ^ x3 ^ k1;
        uint32_t y3 = lo0;
        x0 = y0; x1 = y1; x2 = y2; x3 = y3;
    }
    out[0] = x0; out[1] = x1; out[2] = x2; out[3] = x3;
}

/* ------------------------------------------------------------------------ */
/* Sparse streams and their pairwise sum (§5.1).                            */

typedef struct {
    int dense;      /* representation flag (§5.1 "Switching to a Dense Format") */
    uint64_t nnz;   /* sparse: number of pairs; dense: N */
    uint32_t* idx;  /* sparse only */
    float* val;     /* sparse: nnz values; dense: N values */
    int owned;      /* buffers belong to the oracle (freed after use) */
} onode;

static int is_pow2(int p) { return p >= 1 && (p & (p - 1)) == 0; }

static void node_free(onode* n)
{
    if (n->owned) {
        free(n->idx);
        free(n->val);
    }
    n->idx = NULL;
    n->val = NULL;
}

/* Both sparse, result sparse: ordered merge of the two index lists; an index
 * present in both gets the fp32 sum of the two values. */
static int sum_sparse_sparse(const onode* a, const onode* b, onode* o)
{
    uint64_t cap = a->nnz + b->nnz;
    o->dense = 0;
    o->owned = 1;
    o->idx = (uint32_t*)malloc((cap ? cap : 1) * sizeof(uint32_t));
    o->val = (float*)malloc((cap ? cap : 1) * sizeof(float));
    if (!o->idx || !o->val) return -4;
    uint64_t i = 0, j = 0, n = 0;
    while (i < a->nnz || j < b->nnz) {
        if (j >= b->nnz || (i < a->nnz && a->idx[i] < b->idx[j])) {
            o->idx[n] = a->idx[i];
            o->val[n] = a->val[i];
            ++i;
        } else if (i >= a->nnz || b->idx[j] < a->idx[i]) {
            o->idx[n] = b->idx[j];
            o->val[n] = b->val[j];
            ++j;
        } else {
            o->idx[n] = a->idx[i];
            o->val[n] = a->val[i] + b->val[j];
            ++i;
            ++j;
        }
        ++n;
    }
    o->nnz = n;
    return 0;
}

/* Add every pair of a sparse stream into a dense vector. */
static void scatter_add(float* D, const onode* s)
{
    for (uint64_t i = 0; i < s->nnz; ++i) D[s->idx[i]] += s->val[i];
}

/* One node of the reduction tree: the four cases of §5.1 "Efficient
 * Summation" for overlapping index sets, with the switch rule: two sparse
 * inputs whose nnz upper bound |H1|+|H2| exceeds the threshold give a dense
 * result. */
static int sum_pair(const onode* L, const onode* R, uint64_t N, uint64_t thr, onode* o)
{
    if (!L->dense && !R->dense) {
        if (L->nnz + R->nnz <= thr) return sum_sparse_sparse(L, R, o);
        o->dense = 1;
        o->owned = 1;
        o->nnz = N;
        o->idx = NULL;
        o->val = (float*)calloc(N, sizeof(float)); /* all +0.0 */
        if (!o->val) return -4;
        scatter_add(o->val, L);
        scatter_add(o->val, R);
        return 0;
    }
    if (L->dense && R->dense) {
        /* dense + dense: elementwise sum (into a fresh vector) */
        o->dense = 1;
        o->owned = 1;
        o->nnz = N;
        o->idx = NULL;
        o->val = (float*)malloc(N * sizeof(float));
        if (!o->val) return -4;
        for (uint64_t j = 0; j < N; ++j) o->val[j] = L->val[j] + R->val[j];
        return 0;
    }
    /* one dense, one sparse: copy the dense one, add the sparse pairs */
    const onode* D = L->dense ? L : R;
    const onode* S = L->dense ? R : L;
    o->dense = 1;
    o->owned = 1;
    o->nnz = N;
    o->idx = NULL;
    o->val = (float*)malloc(N * sizeof(float));
    if (!o->val) return -4;
    memcpy(o->val, D->val, N * sizeof(float));
    scatter_add(o->val, S);
    return 0;
}

/* One level of the tree as independent items: item g sums node a = g and
 * b = g + off (App. A's step in front, off = P2) or a = 2g, b = 2g + 1
 * (recursive doubling, off = 0) into out[g]; its inputs are released once
 * it succeeds. */
typedef struct {
    onode* in;
    onode* out;
    int* rc;
    uint64_t N, thr;
    int off;
} pair_level;

static void pair_item(void* ctx, int g)
{
    pair_level* lv = (pair_level*)ctx;
    onode* a = lv->off ? &lv->in[g] : &lv->in[2 * g];
    onode* b = lv->off ? &lv->in[g + lv->off] : &lv->in[2 * g + 1];
    lv->rc[g] = sum_pair(a, b, lv->N, lv->thr, &lv->out[g]);
    if (lv->rc[g] == 0) {
        node_free(a);
        node_free(b);
    }
}

int orc_sparse_reduce(int P, const uint32_t* const* idx, const float* const* val,
                      const uint64_t* nnz, uint64_t N, double delta,
                      uint32_t* out_idx, uint64_t out_cap, float* out_val,
                      uint64_t* out_nnz, int* out_dense,
                      uint64_t* node_nnz, uint8_t* node_dense)
{
    if (P < 1 || N == 0 || N > 0xFFFFFFFFull || !(delta > 0.0)) return -1;
    if (!idx || !val || !nnz || !out_val || !out_nnz || !out_dense) return -1;
    /* threshold on the number of sparse items (§5.1), as a fraction of N */
    double t = floor(delta * (double)N);
    uint64_t thr = t >= 18446744073709551615.0 ? UINT64_MAX : (uint64_t)t;

    for (int r = 0; r < P; ++r) {
        if (nnz[r] > N) return -2;
        if (nnz[r] && (!idx[r] || !val[r])) return -1;
        for (uint64_t i = 0; i < nnz[r]; ++i) {
            if (idx[r][i] >= N) return -2;
            if (i > 0 && idx[r][i] <= idx[r][i - 1]) return -2;
        }
    }

    onode* cur = (onode*)calloc((size_t)P, sizeof(onode));
    if (!cur) return -4;
    for (int r = 0; r < P; ++r) {
        cur[r].dense = 0;
        cur[r].nnz = nnz[r];
        cur[r].idx = (uint32_t*)idx[r];
        cur[r].val = (float*)val[r];
        cur[r].owned = 0;
    }

    int rc = 0;
    if (P == 1 && nnz[0] > thr) {
        /* a single stream with more than thr items cannot stay sparse */
        onode d = {1, N, NULL, (float*)calloc(N, sizeof(float)), 1};
        if (!d.val) { free(cur); return -4; }
        scatter_add(d.val, &cur[0]);
        cur[0] = d;
    }

    /* P not a power of two (App. A): a step in front reduces the
     * participants to the largest power of two P2 <= P -- rank P2 + i sends
     * its stream to rank i, which sums the two (a tree node under the same
     * switch rule), for i < P - P2; the other ranks take part unchanged. */
    int width = P;
    uint64_t node_base = 0;
    if (!is_pow2(P)) {
        int P2 = 1;
        while (2 * P2 <= P) P2 *= 2;
        const int rem = P - P2;
        onode* fold = (onode*)calloc((size_t)rem, sizeof(onode));
        int* frc = (int*)calloc((size_t)rem, sizeof(int));
        if (!fold || !frc) rc = -4;
        if (rc == 0) {
            pair_level lv = {cur, fold, frc, N, thr, P2};
            for_each_item(rem, pair_item, &lv);
            for (int i = 0; i < rem; ++i)
                if (frc[i] && rc == 0) rc = frc[i];
        }
        if (rc) {
            for (int i = 0; fold && i < rem; ++i) node_free(&fold[i]);
            for (int r = 0; r < P; ++r) node_free(&cur[r]);
            free(fold);
            free(frc);
            free(cur);
            return rc;
        }
        for (int i = 0; i < rem; ++i) {
            if (node_nnz) node_nnz[i] = fold[i].nnz;
            if (node_dense) node_dense[i] = (uint8_t)fold[i].dense;
            cur[i] = fold[i];
        }
        free(fold);
        free(frc);
        width = P2;
        node_base = (uint64_t)rem;
    }

    /* Recursive doubling (§5.3.1): in round t the partners at distance
     * 2^(t-1) hold the sums of adjacent blocks of 2^(t-1) ranks; their sum is
     * node g of level t, made of nodes 2g and 2g+1 of level t-1. */
    while (width > 1) {
        int half = width / 2;
        onode* next = (onode*)calloc((size_t)half, sizeof(onode));
        int* grc = (int*)calloc((size_t)half, sizeof(int));
        if (!next || !grc) {
            free(next);
            free(grc);
            rc = -4;
            break;
        }
        /* the nodes of one level are independent of each other */
        pair_level lv = {cur, next, grc, N, thr, 0};
        for_each_item(half, pair_item, &lv);
        for (int g = 0; g < half; ++g) {
            if (grc[g] && rc == 0) rc = grc[g];
            if (node_nnz) node_nnz[node_base + g] = next[g].nnz;
            if (node_dense) node_dense[node_base + g] = (uint8_t)next[g].dense;
        }
        free(grc);
        if (rc) {
            for (int g = 0; g < half; ++g) node_free(&next[g]);
            free(next);
            break;
        }
        free(cur);
        cur = next;
        node_base += (uint64_t)half;
        width = half;
    }
    if (rc) {
        for (int r = 0; r < width; ++r) node_free(&cur[r]);
        free(cur);
        return rc;
    }

    onode* root = &cur[0];
    if (root->dense) {
        memcpy(out_val, root->val, N * sizeof(float));
        *out_nnz = N;
        *out_dense = 1;
    } else {
        if (root->nnz > out_cap) {
            node_free(root);
            free(cur);
            return -3;
        }
        if (root->nnz) {
            memcpy(out_idx, root->idx, root->nnz * sizeof(uint32_t));
            memcpy(out_val, root->val, root->nnz * sizeof(float));
        }
        *out_nnz = root->nnz;
        *out_dense = 0;
    }
    node_free(root);
    free(cur);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Top-k by magnitude (§2.2, Alg. 1).                                        */

typedef struct {
    uint32_t key;
    uint32_t idx;
} okv;

static uint32_t mag_key(float v)
{
    uint32_t b;
    memcpy(&b, &v, sizeof b);
    return b & 0x7FFFFFFFu; /* |v| as an ordered integer */
}

static int cmp_key_desc_idx_asc(const void* pa, const void* pb)
{
    const okv* a = (const okv*)pa;
    const okv* b = (const okv*)pb;
    if (a->key != b->key) return a->key > b->key ? -1 : 1;
    if (a->idx != b->idx) return a->idx < b->idx ? -1 : 1;
    return 0;
}

static int cmp_u32(const void* pa, const void* pb)
{
    uint32_t a = *(const uint32_t*)pa, b = *(const uint32_t*)pb;
    return a < b ? -1 : (a > b ? 1 : 0);
}

typedef struct {
    const float* x;
    uint64_t N, k;
    uint32_t* out_idx;
    float* out_val;
    float* residual;
    int* rc;
} topk_rows;

/* Rank r's row: full sort by key, the first k taken, reported in index order. */
static void topk_row(void* ctx, int r)
{
    topk_rows* t = (topk_rows*)ctx;
    const uint64_t N = t->N, k = t->k;
    okv* all = (okv*)malloc(N * sizeof(okv));
    if (!all) {
        t->rc[r] = -4;
        return;
    }
    const float* row = t->x + (uint64_t)r * N;
    for (uint64_t j = 0; j < N; ++j) {
        all[j].key = mag_key(row[j]);
        all[j].idx = (uint32_t)j;
    }
    qsort(all, N, sizeof(okv), cmp_key_desc_idx_asc);
    uint32_t* sel = t->out_idx + (uint64_t)r * k;
    for (uint64_t i = 0; i < k; ++i) sel[i] = all[i].idx;
    qsort(sel, k, sizeof(uint32_t), cmp_u32);
    float* v = t->out_val + (uint64_t)r * k;
    for (uint64_t i = 0; i < k; ++i) v[i] = row[sel[i]];
    if (t->residual) {
        float* res = t->residual + (uint64_t)r * N;
        if (res != row) memcpy(res, row, N * sizeof(float));
        for (uint64_t i = 0; i < k; ++i) res[sel[i]] = 0.0f;
    }
    free(all);
    t->rc[r] = 0;
}

int orc_topk(int P, const float* x, uint64_t N, uint64_t k,
             uint32_t* out_idx, float* out_val, float* residual)
{
    if (P < 1 || N == 0 || N > 0xFFFFFFFFull || k > N || !x) return -1;
    if (k && (!out_idx || !out_val)) return -1;
    int* rc = (int*)calloc((size_t)P, sizeof(int));
    if (!rc) return -4;
    topk_rows t = {x, N, k, out_idx, out_val, residual, rc};
    for_each_item(P, topk_row, &t); /* rows are independent */
    int e = 0;
    for (int r = 0; r < P; ++r)
        if (rc[r] && e == 0) e = rc[r];
    free(rc);
    return e;
}

typedef struct {
    const float* grad;
    float* eps;
    uint64_t N, bucket, kb, K;
    float alpha;
    uint32_t* out_idx;
    float* out_val;
    int* rc;
} topkb_rows;

/* Rank r's row, bucket by bucket in order. */
static void topk_bucketed_row(void* ctx, int r)
{
    topkb_rows* t = (topkb_rows*)ctx;
    const uint64_t N = t->N, bucket = t->bucket, kb = t->kb;
    const uint64_t nb = (N + bucket - 1) / bucket;
    okv* b = (okv*)malloc(bucket * sizeof(okv));
    float* acc = (float*)malloc(bucket * sizeof(float));
    if (!b || !acc) {
        free(b);
        free(acc);
        t->rc[r] = -4;
        return;
    }
    float* e = t->eps + (uint64_t)r * N;
    const float* g = t->grad ? t->grad + (uint64_t)r * N : NULL;
    uint64_t o = (uint64_t)r * t->K;
    for (uint64_t q = 0; q < nb; ++q) {
        const uint64_t j0 = q * bucket;
        const uint64_t len = N - j0 < bucket ? N - j0 : bucket;
        /* Alg. 1: acc = eps + alpha * grad (fp32, two roundings) */
        for (uint64_t j = 0; j < len; ++j) {
            acc[j] = g ? e[j0 + j] + t->alpha * g[j0 + j] : e[j0 + j];
            b[j].key = mag_key(acc[j]);
            b[j].idx = (uint32_t)(j0 + j);
        }
        /* the bucket's kb largest magnitudes, lowest index on ties */
        qsort(b, len, sizeof(okv), cmp_key_desc_idx_asc);
        const uint64_t take = len < kb ? len : kb;
        uint32_t sel[64];
        for (uint64_t i = 0; i < take; ++i) sel[i] = b[i].idx;
        qsort(sel, take, sizeof(uint32_t), cmp_u32);
        /* eps = acc - TopK(acc): the selected entries leave, the rest stay */
        for (uint64_t j = 0; j < len; ++j) e[j0 + j] = acc[j];
        for (uint64_t i = 0; i < take; ++i) {
            t->out_idx[o + i] = sel[i];
            t->out_val[o + i] = acc[sel[i] - j0];
            e[sel[i]] = 0.0f;
        }
        o += take;
    }
    free(b);
    free(acc);
    t->rc[r] = 0;
}

int orc_topk_bucketed(int P, const float* grad, float* eps, uint64_t N, float alpha,
                      uint64_t bucket, uint64_t kb, uint32_t* out_idx, float* out_val)
{
    if (P < 1 || N == 0 || N > 0xFFFFFFFFull || !eps || bucket == 0 || kb == 0 || kb > 64) return -1;
    if (!out_idx || !out_val) return -1;
    const uint64_t nb = (N + bucket - 1) / bucket;
    const uint64_t last = N - (nb - 1) * bucket;
    const uint64_t K = (nb - 1) * kb + (last < kb ? last : kb); /* entries per rank */
    int* rc = (int*)calloc((size_t)P, sizeof(int));
    if (!rc) return -4;
    topkb_rows t = {grad, eps, N, bucket, kb, K, alpha, out_idx, out_val, rc};
    for_each_item(P, topk_bucketed_row, &t); /* rows are independent */
    int e = 0;
    for (int r = 0; r < P; ++r)
        if (rc[r] && e == 0) e = rc[r];
    free(rc);
    return e;
}

/* ------------------------------------------------------------------------ */
/* QSGD stochastic quantization (§2.2, §6).                                  */

static int valid_bits(int bits) { return bits == 2 || bits == 4 || bits == 8; }

/* L2 norm of v[0..n): squares summed by an adjacent-pair binary tree in
 * fp64, zero-padded to a power of two, rounded once to fp32. */
static int l2_scale(const float* v, uint64_t n, float* scale)
{
    uint64_t m = 1;
    while (m < n) m <<= 1;
    double* t = (double*)calloc(m, sizeof(double));
    if (!t) return -4;
    for (uint64_t j = 0; j < n; ++j) t[j] = (double)v[j] * (double)v[j];
    for (uint64_t w = m; w > 1; w >>= 1)
        for (uint64_t i = 0; i < w / 2; ++i) t[i] = t[2 * i] + t[2 * i + 1];
    double norm2 = n ? t[0] : 0.0;
    free(t);
    *scale = (float)sqrt(norm2);
    return 0;
}

/* Quantize elements j0 .. j0+n-1 of stream r (v points at element j0) with
 * one scale: codes OR-ed into q (zeroed by the caller), deq may be NULL. */
static void quantize_span(const float* v, uint64_t j0, uint64_t n, int r, int bits,
                          const uint32_t key[2], float scale, uint8_t* q, float* deq)
{
    const uint32_t s = (1u << (bits - 1)) - 1u; /* magnitude levels 0..s */
    const int per_byte = 8 / bits;
    if (scale == 0.0f) {
        if (deq)
            for (uint64_t i = 0; i < n; ++i) deq[j0 + i] = 0.0f;
        return; /* every code is 0 */
    }
    const float inv = (float)s / scale;  /* levels per unit of norm */
    const float unit = scale / (float)s; /* value of one level */
    for (uint64_t i = 0; i < n; ++i) {
        const uint64_t j = j0 + i;
        float a = fabsf(v[i]) * inv;
        uint32_t l = (uint32_t)a; /* floor, a >= 0 */
        float f = a - (float)l;   /* exact */
        uint32_t ctr[4] = {(uint32_t)(j >> 2), (uint32_t)r, 0u, 0u};
        uint32_t word[4];
        orc_philox4x32_10(ctr, key, word);
        float u = (float)(word[j & 3] >> 8) * 0x1p-24f; /* uniform [0,1) */
        if (u < f) l += 1u; /* round up with probability f */
        if (l > s) l = s;
        uint32_t sign = (v[i] < 0.0f && l > 0u) ? 1u : 0u;
        uint32_t code = (sign << (bits - 1)) | l;
        q[j / per_byte] |= (uint8_t)(code << ((j % per_byte) * bits));
        if (deq) {
            float mag = (float)l * unit;
            deq[j] = l == 0u ? 0.0f : (sign ? -mag : mag);
        }
    }
}

typedef struct {
    const float* const* val;
    const uint64_t* nnz;
    int bits;
    uint64_t bucket;
    uint32_t key[2];
    uint8_t* const* out_q;
    float* out_scale;
    float* const* out_deq;
    const uint64_t* first_scale; /* per stream: index of its first scale */
    int* rc;
} quant_streams;

/* Stream r: its buckets in order, each with its own L2 scale. */
static void quantize_stream(void* ctx, int r)
{
    quant_streams* t = (quant_streams*)ctx;
    const int bits = t->bits;
    const int per_byte = 8 / bits;
    const uint64_t n = t->nnz[r];
    const float* v = t->val[r];
    uint8_t* q = t->out_q[r];
    const uint64_t nbytes = (n + per_byte - 1) / per_byte;
    if (nbytes) memset(q, 0, nbytes);
    float* deq = t->out_deq ? t->out_deq[r] : NULL;
    const uint64_t B = t->bucket ? t->bucket : (n ? n : 1);
    const uint64_t nb = t->bucket ? (n + B - 1) / B : 1;
    for (uint64_t b = 0; b < nb; ++b) {
        const uint64_t j0 = b * B;
        const uint64_t len = n - j0 < B ? n - j0 : B;
        float scale;
        if (l2_scale(v + j0, len, &scale)) {
            t->rc[r] = -4;
            return;
        }
        t->out_scale[t->first_scale[r] + b] = scale;
        quantize_span(v + j0, j0, len, r, bits, t->key, scale, q, deq);
    }
    t->rc[r] = 0;
}

int orc_quantize_bucketed(int P, const float* const* val, const uint64_t* nnz, int bits,
                          uint64_t bucket, uint64_t seed, uint8_t* const* out_q,
                          float* out_scale, float* const* out_deq)
{
    if (P < 1 || !valid_bits(bits) || !val || !nnz || !out_q || !out_scale) return -1;
    for (int r = 0; r < P; ++r)
        if (nnz[r] && (!val[r] || !out_q[r])) return -1;
    uint64_t* first = (uint64_t*)malloc((size_t)P * sizeof(uint64_t));
    int* rc = (int*)calloc((size_t)P, sizeof(int));
    if (!first || !rc) {
        free(first);
        free(rc);
        return -4;
    }
    uint64_t so = 0; /* stream r's scales follow those of streams 0..r-1 */
    for (int r = 0; r < P; ++r) {
        first[r] = so;
        so += bucket ? (nnz[r] + bucket - 1) / bucket : 1;
    }
    quant_streams t = {val, nnz, bits, bucket,
                       {(uint32_t)(seed & 0xFFFFFFFFu), (uint32_t)(seed >> 32)},
                       out_q, out_scale, out_deq, first, rc};
    for_each_item(P, quantize_stream, &t); /* streams are independent */
    int e = 0;
    for (int r = 0; r < P; ++r)
        if (rc[r] && e == 0) e = rc[r];
    free(first);
    free(rc);
    return e;
}

int orc_quantize(int P, const float* const* val, const uint64_t* nnz, int bits,
                 uint64_t seed, uint8_t* const* out_q, float* out_scale,
                 float* const* out_deq)
{
    return orc_quantize_bucketed(P, val, nnz, bits, 0, seed, out_q, out_scale, out_deq);
}

int orc_dequantize_bucketed(const uint8_t* q, const float* scales, int bits, uint64_t bucket,
                            uint64_t n, float* out)
{
    if (!valid_bits(bits) || (n && (!q || !out || !scales))) return -1;
    const uint32_t s = (1u << (bits - 1)) - 1u;
    const int per_byte = 8 / bits;
    const uint32_t lmask = s, smask = 1u << (bits - 1);
    for (uint64_t j = 0; j < n; ++j) {
        const float unit = scales[bucket ? j / bucket : 0] / (float)s;
        uint32_t code = (q[j / per_byte] >> ((j % per_byte) * bits)) & ((1u << bits) - 1u);
        uint32_t l = code & lmask;
        float mag = (float)l * unit;
        out[j] = l == 0u ? 0.0f : ((code & smask) ? -mag : mag);
    }
    return 0;
}

int orc_dequantize(const uint8_t* q, float scale, int bits, uint64_t n, float* out)
{
    return orc_dequantize_bucketed(q, &scale, bits, 0, n, out);
}

/* ------------------------------------------------------------------------ */

int orc_densify(const uint32_t* idx, const float* val, uint64_t nnz, uint64_t N,
                float* dense)
{
    if (N == 0 || !dense || (nnz && (!idx || !val))) return -1;
    for (uint64_t j = 0; j < N; ++j) dense[j] = 0.0f;
    for (uint64_t i = 0; i < nnz; ++i) {
        if (idx[i] >= N) return -2;
        dense[idx[i]] = val[i];
    }
    return 0;
}
