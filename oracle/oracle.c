/*
 * Oracle for the sparse-embedding hot path -- TEST INFRASTRUCTURE ONLY.
 * Plain single-threaded C; see oracle.h for the contract of each function and
 * the passage of the paper it follows.  Only the tests, the smoke check and the
 * benchmark's CPU-baseline leg may load this code.
 */
#include "oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

/* Forward lookup, Sec. 4.1.1. */
int64_t orc_gather(const float *W, int64_t V, int64_t D,
                   const int32_t *ids, int64_t T, float *out) {
    int64_t bad = 0;
    for (int64_t t = 0; t < T; ++t) {
        int64_t id = ids[t];
        for (int64_t j = 0; j < D; ++j)
            out[t * D + j] = (id >= 0 && id < V) ? W[id * D + j] : 0.0f;
        if (id < 0 || id >= V) ++bad;
    }
    return bad;
}

/* A COO coordinate: (row index, token position). */
typedef struct {
    int64_t id;
    int64_t t;
} orc_coord;

static int orc_coord_cmp(const void *a, const void *b) {
    const orc_coord *x = (const orc_coord *)a, *y = (const orc_coord *)b;
    if (x->id != y->id) return x->id < y->id ? -1 : 1;
    if (x->t != y->t) return x->t < y->t ? -1 : 1;
    return 0;
}

/* Exact widening of one gradient element to fp64. */
static double orc_grad_elem(const void *grad, int32_t is_bf16, int64_t idx) {
    if (is_bf16) {
        uint32_t bits = (uint32_t)((const uint16_t *)grad)[idx] << 16;
        float f;
        memcpy(&f, &bits, sizeof f);
        return (double)f;
    }
    return (double)((const float *)grad)[idx];
}

/* COALESCE and UNIQUE of Algorithm 1, Sec. 4.2.2: sort the coordinates by
 * (index, position), then sum each run of equal index. */
int64_t orc_coalesce(const int32_t *ids, int64_t T, const void *grad,
                     int32_t grad_is_bf16, int64_t D, int64_t V,
                     int32_t *uniq_ids, int32_t *seg_offsets, float *uniq_grad,
                     double *sum_f64, double *absum, int64_t *n_invalid) {
    orc_coord *c = (orc_coord *)malloc(sizeof(orc_coord) * (size_t)(T > 0 ? T : 1));
    double *acc = (double *)malloc(sizeof(double) * (size_t)(D > 0 ? D : 1));
    double *aab = (double *)malloc(sizeof(double) * (size_t)(D > 0 ? D : 1));
    int64_t n = 0, bad = 0;
    for (int64_t t = 0; t < T; ++t) {
        if (ids[t] < 0 || ids[t] >= V) { ++bad; continue; }
        c[n].id = ids[t];
        c[n].t = t;
        ++n;
    }
    qsort(c, (size_t)n, sizeof(orc_coord), orc_coord_cmp);

    int64_t U = 0;
    for (int64_t s = 0; s < n;) {
        int64_t e = s;
        while (e < n && c[e].id == c[s].id) ++e;
        for (int64_t j = 0; j < D; ++j) { acc[j] = 0.0; aab[j] = 0.0; }
        for (int64_t i = s; i < e; ++i) {
            for (int64_t j = 0; j < D; ++j) {
                double g = orc_grad_elem(grad, grad_is_bf16, c[i].t * D + j);
                acc[j] += g;
                aab[j] += fabs(g);
            }
        }
        uniq_ids[U] = (int32_t)c[s].id;
        seg_offsets[U] = (int32_t)s;
        for (int64_t j = 0; j < D; ++j) {
            uniq_grad[U * D + j] = (float)acc[j];
            if (sum_f64) sum_f64[U * D + j] = acc[j];
            if (absum) absum[U * D + j] = aab[j];
        }
        ++U;
        s = e;
    }
    seg_offsets[U] = (int32_t)n;
    if (n_invalid) *n_invalid = bad;
    free(c);
    free(acc);
    free(aab);
    return U;
}

/* Pack by owner for the gradient AlltoAll, Sec. 4.1.1 / 4.1.2. */
int64_t orc_pack_by_owner(const int32_t *uniq_ids, const float *uniq_grad,
                          int64_t U, int64_t D, const int32_t *row_owner,
                          int64_t V, int32_t P, int32_t *send_ids,
                          float *send_rows, int32_t *send_counts,
                          int32_t *send_offsets) {
    int64_t bad = 0;
    int32_t *own = (int32_t *)malloc(sizeof(int32_t) * (size_t)(U > 0 ? U : 1));
    int32_t *run = (int32_t *)calloc((size_t)(P > 0 ? P : 1), sizeof(int32_t));
    for (int32_t p = 0; p < P; ++p) send_counts[p] = 0;
    for (int64_t k = 0; k < U; ++k) {
        int64_t id = uniq_ids[k];
        own[k] = -1;
        if (id < 0 || id >= V || row_owner[id] < 0 || row_owner[id] >= P) { ++bad; continue; }
        own[k] = row_owner[id];
        send_counts[own[k]] += 1;
    }
    send_offsets[0] = 0;
    for (int32_t p = 0; p < P; ++p) send_offsets[p + 1] = send_offsets[p] + send_counts[p];
    for (int64_t k = 0; k < U; ++k) {
        if (own[k] < 0) continue;
        int64_t pos = (int64_t)send_offsets[own[k]] + run[own[k]]++;
        send_ids[pos] = uniq_ids[k];
        for (int64_t j = 0; j < D; ++j) send_rows[pos * D + j] = uniq_grad[k * D + j];
    }
    free(own);
    free(run);
    return bad;
}

static int orc_int32_cmp(const void *a, const void *b) {
    const int32_t x = *(const int32_t *)a, y = *(const int32_t *)b;
    return (x > y) - (x < y);
}

/* Set split of Algorithm 1 (Vertical Sparse Scheduling, Sec. 4.2.2): a
 * coalesced row is prior when its index is also in the next batch's data.
 * Membership by binary search in a sorted copy of the next batch's ids. */
int64_t orc_vertical_split(const int32_t *uniq_ids, int64_t U,
                           const int32_t *next_ids, int64_t T_next,
                           int32_t *is_prior) {
    int32_t *nx = (int32_t *)malloc(sizeof(int32_t) * (size_t)(T_next > 0 ? T_next : 1));
    for (int64_t t = 0; t < T_next; ++t) nx[t] = next_ids[t];
    qsort(nx, (size_t)T_next, sizeof(int32_t), orc_int32_cmp);
    int64_t n_prior = 0;
    for (int64_t k = 0; k < U; ++k) {
        const int32_t key = uniq_ids[k];
        is_prior[k] = bsearch(&key, nx, (size_t)T_next, sizeof(int32_t), orc_int32_cmp) != NULL;
        n_prior += is_prior[k];
    }
    free(nx);
    return n_prior;
}

/* Row-wise Adam, Sec. 4.1.1 and Sec. 5.7; Kingma & Ba, Algorithm 1. */
int64_t orc_sparse_adam(float *W, float *m, float *v, int64_t V, int64_t D,
                        const int32_t *row_ids, const float *rows,
                        const int32_t *offsets, int32_t shard_begin,
                        int32_t shard_end, double lr, double beta1,
                        double beta2, double eps, int64_t step) {
    const double bc1 = 1.0 - pow(beta1, (double)step);
    const double bc2 = 1.0 - pow(beta2, (double)step);
    int64_t bad = 0;
    for (int64_t i = offsets[shard_begin]; i < offsets[shard_end]; ++i) {
        int64_t r = row_ids[i];
        if (r < 0 || r >= V) { ++bad; continue; }
        for (int64_t j = 0; j < D; ++j) {
            double g = rows[i * D + j];
            double mm = beta1 * (double)m[r * D + j] + (1.0 - beta1) * g;
            double vv = beta2 * (double)v[r * D + j] + (1.0 - beta2) * g * g;
            double mhat = mm / bc1;
            double vhat = vv / bc2;
            double w = (double)W[r * D + j] - lr * mhat / (sqrt(vhat) + eps);
            m[r * D + j] = (float)mm;
            v[r * D + j] = (float)vv;
            W[r * D + j] = (float)w;
        }
    }
    return bad;
}

/* Lookup requests of the row-wise partition, Sec. 4.1.1. */
int64_t orc_lookup_request(const int32_t *ids, int64_t T, int64_t V,
                           const int32_t *row_owner, int32_t P,
                           int32_t *req_ids, int32_t *req_counts,
                           int32_t *req_offsets, int32_t *inverse) {
    /* the distinct ids that take part, ascending */
    int32_t *u = (int32_t *)malloc(sizeof(int32_t) * (size_t)(T > 0 ? T : 1));
    int64_t n = 0;
    for (int64_t t = 0; t < T; ++t) {
        const int32_t id = ids[t];
        if (id >= 0 && id < V && row_owner[id] >= 0 && row_owner[id] < P) u[n++] = id;
    }
    qsort(u, (size_t)n, sizeof(int32_t), orc_int32_cmp);
    int64_t U = 0;
    for (int64_t k = 0; k < n; ++k)
        if (k == 0 || u[k] != u[k - 1]) u[U++] = u[k];
    /* grouped by owner, ascending inside an owner */
    for (int32_t p = 0; p < P; ++p) req_counts[p] = 0;
    for (int64_t k = 0; k < U; ++k) req_counts[row_owner[u[k]]] += 1;
    req_offsets[0] = 0;
    for (int32_t p = 0; p < P; ++p) req_offsets[p + 1] = req_offsets[p] + req_counts[p];
    int32_t *run = (int32_t *)calloc((size_t)(P > 0 ? P : 1), sizeof(int32_t));
    for (int64_t k = 0; k < U; ++k) {
        const int32_t p = row_owner[u[k]];
        req_ids[req_offsets[p] + run[p]++] = u[k];
    }
    /* each token's place in the request */
    for (int64_t t = 0; t < T; ++t) {
        const int32_t id = ids[t];
        inverse[t] = -1;
        if (id < 0 || id >= V || row_owner[id] < 0 || row_owner[id] >= P) continue;
        const int32_t p = row_owner[id];
        const int32_t *blk = req_ids + req_offsets[p];
        const int32_t *hit = (const int32_t *)bsearch(&id, blk, (size_t)(req_offsets[p + 1] - req_offsets[p]),
                                                      sizeof(int32_t), orc_int32_cmp);
        inverse[t] = hit != NULL ? (int32_t)(hit - req_ids) : -1;
    }
    free(run);
    free(u);
    return U;
}

/* Column-wise partition, Sec. 4.1.1.  First column of owner p. */
static int64_t orc_col_begin(int64_t p, int64_t D, int32_t P) { return p * D / P; }

void orc_pack_by_column(const float *rows, int64_t R, int64_t C, int64_t D,
                        int32_t P, float *blocks) {
    for (int32_t p = 0; p < P; ++p) {
        const int64_t a = orc_col_begin(p, D, P);
        const int64_t w = orc_col_begin(p + 1, D, P) - a;
        for (int64_t r = 0; r < R; ++r)
            for (int64_t j = 0; j < w; ++j)
                blocks[C * a + r * w + j] = rows[r * D + a + j];
    }
}

int64_t orc_gather_by_column(const float *shards, int64_t V, int64_t D,
                             int32_t P, const int32_t *ids, int64_t T,
                             float *blocks) {
    int64_t bad = 0;
    for (int64_t t = 0; t < T; ++t) bad += ids[t] < 0 || ids[t] >= V;
    for (int32_t p = 0; p < P; ++p) {
        const int64_t a = orc_col_begin(p, D, P);
        const int64_t w = orc_col_begin(p + 1, D, P) - a;
        const float *shard = shards + V * a;
        for (int64_t t = 0; t < T; ++t) {
            const int64_t id = ids[t];
            const int ok = id >= 0 && id < V;
            for (int64_t j = 0; j < w; ++j)
                blocks[T * a + t * w + j] = ok ? shard[id * w + j] : 0.0f;
        }
    }
    return bad;
}

void orc_assemble_by_column(const float *blocks, int64_t C, int64_t row0,
                            int64_t R, int64_t D, int32_t P, float *rows) {
    for (int32_t p = 0; p < P; ++p) {
        const int64_t a = orc_col_begin(p, D, P);
        const int64_t w = orc_col_begin(p + 1, D, P) - a;
        for (int64_t r = 0; r < R; ++r)
            for (int64_t j = 0; j < w; ++j)
                rows[r * D + a + j] = blocks[C * a + (row0 + r) * w + j];
    }
}

/* Table 2 of Sec. 4.1.2. */
double orc_comm_cost(int32_t scheme, int64_t N, int64_t S, double M,
                     double alpha, double B, double beta) {
    const double n = (double)N;
    switch (scheme) {
    case 0: return 2.0 * (n - 1.0) * (alpha * M / (n * B) + beta);
    case 1: return 2.0 * (n - 1.0) * (M / (n * B) + beta);
    case 2: return 2.0 * n * (alpha * M / ((double)S * B) + beta);
    case 3: return (n - 1.0) * (alpha * M / B + beta);
    default: return -1.0;
    }
}
