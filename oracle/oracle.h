/*
 * Oracle for the sparse-embedding hot path -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, single-threaded CPU definition of what the hot path computes,
 * used by the tests, the smoke check and the CPU-baseline leg of the benchmark
 * to judge the GPU library.  Nothing in the product path may call it.  It
 * shares no code, header, table or helper with the GPU library.
 *
 * Paper: EmbRace, "Accelerating Sparse Communication for Distributed Training
 * of Deep Neural Networks" (ICPP '22).
 *
 * Floating point: sums and the optimizer arithmetic are carried in fp64 and
 * rounded once to fp32 when stored (the paper fixes no precision).
 * Integers (ids, counts, offsets) are exact.
 */
#ifndef EMB_ORACLE_H
#define EMB_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Forward embedding lookup (Sec. 4.1.1: every process looks up its training
 * data in the embedding table).  out[t][j] = W[ids[t]][j] for ids in [0, V);
 * an id outside [0, V) yields a zero row.  Returns the number of such ids. */
int64_t orc_gather(const float *W, int64_t V, int64_t D,
                   const int32_t *ids, int64_t T, float *out);

/* COALESCE + UNIQUE of Algorithm 1 (Sec. 4.2.2, "Coalescing Gradients"):
 * the sparse COO gradient (Sec. 2.1) has one row per token; rows with the same
 * index are summed into one.  Tokens with an id outside [0, V) are dropped.
 *   uniq_ids[U]      the distinct ids, ascending
 *   seg_offsets[U+1] exclusive scan of per-id multiplicities (seg_offsets[U]
 *                    = number of valid tokens)
 *   uniq_grad[U][D]  fp64 sum (tokens in increasing t) rounded once to fp32
 *   sum_f64[U][D]    the same sums before rounding        (may be NULL)
 *   absum[U][D]      sums of |G| (the error-bound scale)  (may be NULL)
 * grad is fp32 [T][D] (grad_is_bf16 == 0) or bf16 bit patterns (uint16).
 * Returns U; *n_invalid receives the number of dropped tokens (may be NULL). */
int64_t orc_coalesce(const int32_t *ids, int64_t T, const void *grad,
                     int32_t grad_is_bf16, int64_t D, int64_t V,
                     int32_t *uniq_ids, int32_t *seg_offsets, float *uniq_grad,
                     double *sum_f64, double *absum, int64_t *n_invalid);

/* Pack the coalesced rows by owner shard (Sec. 4.1.1 / 4.1.2: the gradients
 * are exchanged with an AlltoAll, each peer receiving the rows it owns).
 *   owner(k)          = row_owner[uniq_ids[k]]
 *   send_counts[p]    = #{k : owner(k) = p}
 *   send_offsets[P+1] = exclusive scan of send_counts
 *   rows are placed in owner-major order, ascending k inside an owner.
 * Rows whose id is outside [0, V) or whose owner is outside [0, P) are not
 * sent.  Returns the number of such rows. */
int64_t orc_pack_by_owner(const int32_t *uniq_ids, const float *uniq_grad,
                          int64_t U, int64_t D, const int32_t *row_owner,
                          int64_t V, int32_t P, int32_t *send_ids,
                          float *send_rows, int32_t *send_counts,
                          int32_t *send_offsets);

/* The set split of Vertical Sparse Scheduling (Algorithm 1; Sec. 4.2.2,
 * "Minimum Dependency of Embedding"): with the next iteration's data known in
 * advance, the coalesced rows whose index also occurs in the next batch are
 * the prior rows (i_prior = D_u intersect D_next), the others the delayed rows
 * (i_delayed = D_u minus i_prior).
 *   is_prior[k] = 1 if uniq_ids[k] occurs among next_ids[0 .. T_next), else 0.
 * Returns the number of prior rows.  INDEX_SELECT of the prior and delayed
 * rows is then a plain selection by is_prior. */
int64_t orc_vertical_split(const int32_t *uniq_ids, int64_t U,
                           const int32_t *next_ids, int64_t T_next,
                           int32_t *is_prior);

/* Row-wise (lazy) Adam on the received rows (Sec. 4.1.1: each process updates
 * its embedding parameters with the new gradients; Sec. 5.7: Adam, with the
 * global step counter passed in by the caller).  Kingma & Ba, Algorithm 1:
 *   m <- b1 m + (1-b1) g ;  v <- b2 v + (1-b2) g^2
 *   w <- w - lr * (m / (1-b1^t)) / (sqrt(v / (1-b2^t)) + eps)
 * applied to rows row_ids[i], i in [offsets[shard_begin], offsets[shard_end]).
 * Rows not listed keep W, m, v unchanged.  Row ids outside [0, V) are skipped;
 * returns their number. */
int64_t orc_sparse_adam(float *W, float *m, float *v, int64_t V, int64_t D,
                        const int32_t *row_ids, const float *rows,
                        const int32_t *offsets, int32_t shard_begin,
                        int32_t shard_end, double lr, double beta1,
                        double beta2, double eps, int64_t step);

/* Lookup requests of the row-wise partition (Sec. 4.1.1: every process looks
 * up its training data in the embedding table; with rows partitioned by
 * owner, a process asks each owner for the rows it needs).  A token takes
 * part when its id is in [0, V) and row_owner[id] in [0, P).
 *   req_ids[U]        the distinct ids of the tokens that take part, grouped by
 *                     owner (owner 0 first), ascending inside an owner
 *   req_counts[P], req_offsets[P+1]: the owner groups
 *   inverse[T]        k with req_ids[k] = ids[t] for a token that takes part,
 *                     -1 for one that does not
 * Returns U. */
int64_t orc_lookup_request(const int32_t *ids, int64_t T, int64_t V,
                           const int32_t *row_owner, int32_t P,
                           int32_t *req_ids, int32_t *req_counts,
                           int32_t *req_offsets, int32_t *inverse);

/* Column-wise partition (Sec. 4.1.1: the table is split along the embedding
 * dimension, every part keeping the whole vocabulary).  The paper does not say
 * how D columns split when P does not divide D; here owner p holds columns
 * [floor(p D / P), floor((p + 1) D / P)), so widths differ by at most one.
 * Block p of a column-block layout of capacity C is the [C][w(p)] row-major
 * slice of owner p's columns at float offset C * floor(p D / P).
 *   orc_pack_by_column:     rows[R][D]       -> blocks (rows r < R of each block)
 *   orc_gather_by_column:   shards (C = V)   -> blocks of capacity T, row t of
 *                           block p = owner p's columns of table row ids[t]
 *                           (zeros for an id outside [0, V); returns their count)
 *   orc_assemble_by_column: blocks (C), rows [row0, row0 + R) -> rows[R][D] */
void orc_pack_by_column(const float *rows, int64_t R, int64_t C, int64_t D,
                        int32_t P, float *blocks);
int64_t orc_gather_by_column(const float *shards, int64_t V, int64_t D,
                             int32_t P, const int32_t *ids, int64_t T,
                             float *blocks);
void orc_assemble_by_column(const float *blocks, int64_t C, int64_t row0,
                            int64_t R, int64_t D, int32_t P, float *rows);

/* Communication cost of a sparse tensor by approach (Sec. 4.1.2, Table 2):
 * N workers, S parameter servers (PS only; the table's entry is S = n nodes),
 * table of M bytes, gradient density alpha, bandwidth B, start latency beta.
 *   scheme 0 AlltoAll  2(N-1)(alpha M / (N B) + beta)
 *          1 AllReduce 2(N-1)(M / (N B) + beta)
 *          2 PS        2N(alpha M / (S B) + beta)
 *          3 AllGather (N-1)(alpha M / B + beta)
 * Returns -1 for an unknown scheme. */
double orc_comm_cost(int32_t scheme, int64_t N, int64_t S, double M,
                     double alpha, double B, double beta);

#ifdef __cplusplus
}
#endif
#endif
