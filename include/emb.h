/*
 * emb.h -- C ABI of the sparse-embedding hot path on one MI355X (gfx950).
 *
 * The path is one GPU's share of sparse embedding-table training in EmbRace
 * (Li et al., "EmbRace: Accelerating Sparse Communication for Distributed
 * Training of Deep Neural Networks", ICPP '22):
 *
 *   emb_gather             forward lookup of the batch's rows       (Sec. 4.1.1)
 *   emb_grad_coalesce      COALESCE + UNIQUE of the sparse gradient (Sec. 4.2.2,
 *                          Algorithm 1)
 *   emb_pack_by_owner      per-owner send buffers, counts, offsets  (Sec. 4.1.1,
 *                          Sec. 4.1.2: the payload of the gradient AlltoAll)
 *   emb_sparse_adam_apply  row-wise Adam on the rows a shard owns   (Sec. 4.1.1,
 *                          Sec. 5.7)
 *
 * with, around them: the owner-major coalesce that writes the send layout
 * directly, and its prior/delayed split (Algorithm 1); the receiver side of
 * the exchange (a simulated AlltoAll and the merge); the column-wise partition
 * of Sec. 4.1.1 (gradient pack, every owner's lookup, the join of the lookup
 * results); the Table 2 cost model; and a step executor.
 *
 * Conventions for every call:
 *  - Array arguments are DEVICE pointers (memory of the current HIP device);
 *    scalars are passed by value.  The caller allocates and owns every buffer;
 *    the calls of the path never allocate, free or keep a pointer after
 *    returning.  The one allocation of the library is the signal memory of
 *    emb_step_signals_create (a few words per handle, kept in a pool for reuse
 *    and never returned to the runtime).
 *  - Tables and gradient rows are dense row-major [rows][D] arrays.  Ids are
 *    int32 row indices in [0, V).
 *  - `stream` is a hipStream_t (NULL: the null stream).  Calls only enqueue
 *    work on it and return without synchronising; outputs are valid once the
 *    stream has reached that point.  Data-dependent sizes (the unique count,
 *    per-owner counts) stay in device memory: later calls read them there, and
 *    grids are sized by the caller's capacity arguments.
 *  - The return value is a host status (EMB_OK or an EMB_ERR_* code).  Argument
 *    errors are found on the host before anything is enqueued.  Errors that
 *    depend on device data (an id or owner out of range) are OR-ed as
 *    EMB_DEV_* flags into *dev_status (an optional int32 in device memory,
 *    NULL to ignore); the caller clears it and reads it after synchronising.
 *  - Calls are reentrant; concurrent calls need distinct outputs and
 *    workspaces.
 */
#ifndef EMB_H
#define EMB_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define EMB_ABI_VERSION 3

/* host status codes */
#define EMB_OK 0
#define EMB_ERR_INVALID_ARG 1 /* null pointer, size or range out of bounds */
#define EMB_ERR_WORKSPACE 2   /* workspace smaller than the size query */
#define EMB_ERR_LAUNCH 3      /* the HIP runtime refused a launch */
#define EMB_ERR_UNSUPPORTED 4 /* valid but not supported by this library */

/* gradient element types */
#define EMB_F32 0  /* IEEE binary32 */
#define EMB_BF16 1 /* bfloat16 (upper half of a binary32), widened exactly */

/* device status flags */
#define EMB_DEV_ID_OUT_OF_RANGE 1    /* a token or row id was outside [0, V) */
#define EMB_DEV_OWNER_OUT_OF_RANGE 2 /* row_owner[id] was outside [0, P) */
#define EMB_DEV_STALLED 4            /* internal: a workgroup gave up waiting for the result \
                                        of an earlier one; the outputs are invalid */

int emb_abi_version(void);
const char *emb_status_string(int status);

/*
 * Forward lookup (Sec. 4.1.1: each process looks up its batch in the
 * embedding table).  out[t][j] = table[ids[t]][j] for t < T, j < D: a bit copy.
 *   table [V][D] fp32, ids [T] int32, out [T][D] fp32.
 * An id outside [0, V) yields a zero row and sets EMB_DEV_ID_OUT_OF_RANGE.
 * T == 0 is a no-op.  Requires 1 <= V < 2^31, D >= 1, T >= 0.
 */
int emb_gather(const float *table, int64_t V, int32_t D, const int32_t *ids,
               int32_t T, float *out, int32_t *dev_status, void *stream);

/*
 * COALESCE and UNIQUE of Algorithm 1 (Sec. 4.2.2, "Coalescing Gradients"):
 * the embedding gradient is a sparse COO tensor (Sec. 2.1) with one row per
 * token; rows with the same index are summed into one.
 *   ids [T] int32, grad [T][D] fp32 (EMB_F32) or bf16 (EMB_BF16).
 * Outputs, sized by the capacity T (the unique count U <= T):
 *   uniq_ids    [T]     the U distinct valid ids, ascending
 *   seg_offsets [T + 1] seg_offsets[k] = number of valid tokens whose id is
 *                       below uniq_ids[k]; seg_offsets[U] = valid tokens
 *   uniq_grad   [T][D]  fp32 per-id sums of the gradient rows
 *   num_unique  [1]     U
 * Entries past U are left unspecified.  Tokens with an id outside [0, V) are
 * left out and set EMB_DEV_ID_OUT_OF_RANGE.
 * Sums are accumulated in fp32 in a fixed order that depends only on the ids
 * (sorted position order, in chunks of 32 tokens, then an ordered combine of
 * the chunk partials; a batch of at most 2048 tokens is summed by one
 * workgroup in plain sorted position order): results are bitwise
 * reproducible run to run.
 * Workgroups of one launch hand prefix sums to each other (decoupled
 * look-back); every wait is bounded and a timeout sets EMB_DEV_STALLED.
 * workspace: device memory of at least
 * emb_grad_coalesce_workspace_bytes(T, V, D, grad_dtype) bytes, 256-byte
 * aligned; its contents on entry do not matter.
 * Requires 1 <= V < 2^31, D >= 1, 0 <= T < 2^30.  grad must be 4-byte (fp32)
 * or 2-byte (bf16) aligned.
 */
size_t emb_grad_coalesce_workspace_bytes(int32_t T, int64_t V, int32_t D,
                                         int32_t grad_dtype);
int emb_grad_coalesce(const int32_t *ids, int32_t T, const void *grad,
                      int32_t grad_dtype, int32_t D, int64_t V,
                      int32_t *uniq_ids, int32_t *seg_offsets,
                      float *uniq_grad, int32_t *num_unique, void *workspace,
                      size_t workspace_bytes, int32_t *dev_status,
                      void *stream);

/*
 * Pack the coalesced rows into per-owner send buffers (Sec. 4.1.1 / 4.1.2: the
 * sparse gradients are exchanged with an AlltoAll; each of the P shards
 * receives the rows it owns).  The P shards are partitions of one table on
 * this device.
 *   uniq_ids [cap_rows], uniq_grad [cap_rows][D], num_unique [1]: the rows
 *   k < *num_unique (read on the device; must be <= cap_rows).
 *   row_owner [V] int32: owner shard of each table row, in [0, P).
 * Outputs:
 *   send_counts  [P]     rows per owner
 *   send_offsets [P + 1] exclusive scan of send_counts
 *   send_ids     [cap_rows], send_rows [cap_rows][D]: owner p's rows at
 *   [send_offsets[p], send_offsets[p + 1]), in the order of the input (so
 *   ascending id when the input is emb_grad_coalesce output); rows are bit
 *   copies.
 * A row whose id is outside [0, V) or whose owner is outside [0, P) is not
 * sent and sets EMB_DEV_ID_OUT_OF_RANGE / EMB_DEV_OWNER_OUT_OF_RANGE.
 * workspace: at least emb_pack_by_owner_workspace_bytes(cap_rows, P) bytes.
 * Requires 1 <= P <= 1024, cap_rows >= 0, D >= 1, 1 <= V < 2^31.
 */
size_t emb_pack_by_owner_workspace_bytes(int32_t cap_rows, int32_t P);
int emb_pack_by_owner(const int32_t *uniq_ids, const float *uniq_grad,
                      const int32_t *num_unique, int32_t cap_rows, int32_t D,
                      const int32_t *row_owner, int64_t V, int32_t P,
                      int32_t *send_ids, float *send_rows,
                      int32_t *send_counts, int32_t *send_offsets,
                      void *workspace, size_t workspace_bytes,
                      int32_t *dev_status, void *stream);

/*
 * emb_grad_coalesce and emb_pack_by_owner in one call (Algorithm 1's COALESCE
 * and UNIQUE, Sec. 4.2.2, with the per-owner send layout of Sec. 4.1.2): the
 * tokens are sorted by (row_owner[id], id), so the distinct ids come out
 * already grouped by owner, ascending inside each owner, and the summed rows
 * are written straight into the send buffers.  The outputs equal those of
 * emb_pack_by_owner applied to the output of emb_grad_coalesce:
 *   send_ids  [T], send_rows [T][D]: owner p's rows at
 *             [send_offsets[p], send_offsets[p + 1])
 *   send_counts [P], send_offsets [P + 1]
 *   num_unique [1]: rows sent (= send_offsets[P])
 *   seg_offsets [T + 1]: seg_offsets[k + 1] - seg_offsets[k] tokens were summed
 *             into send row k (offsets in the owner-major token order)
 * except that the order of the fp32 additions inside a row may differ (same
 * rule: position order in chunks of 32 sorted tokens, then an ordered combine,
 * or plain position order for at most 2048 tokens; bitwise reproducible run to
 * run).  A token whose id is outside [0, V) or
 * whose owner is outside [0, P) is left out and sets EMB_DEV_ID_OUT_OF_RANGE /
 * EMB_DEV_OWNER_OUT_OF_RANGE.
 * workspace: emb_grad_coalesce_workspace_bytes(T, V, D, grad_dtype) bytes,
 * 256-byte aligned.  Requires what emb_grad_coalesce requires, 1 <= P <= 1024,
 * and bits(V) + bits(P) <= 32, where bits(n) is the number of bits of n - 1
 * (EMB_ERR_UNSUPPORTED otherwise; use the two calls).
 */
int emb_grad_coalesce_by_owner(const int32_t *ids, int32_t T,
                               const void *grad, int32_t grad_dtype,
                               int32_t D, int64_t V,
                               const int32_t *row_owner, int32_t P,
                               int32_t *send_ids, int32_t *seg_offsets,
                               float *send_rows, int32_t *send_counts,
                               int32_t *send_offsets, int32_t *num_unique,
                               void *workspace, size_t workspace_bytes,
                               int32_t *dev_status, void *stream);

/*
 * emb_grad_coalesce_by_owner for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation): the same arguments, outputs and rules, without the workspace.
 * The call allocates nothing and calls no allocating routine; its workspace is
 * a static device array of EMB_NOALLOC_SCRATCH_BYTES (16 MiB) that each device
 * the library runs on holds until the process ends (its address is looked up
 * once per device, at the first call on it).
 * Returns EMB_ERR_WORKSPACE, before anything touches the device, when
 * emb_grad_coalesce_workspace_bytes(T, V, D, grad_dtype) exceeds
 * EMB_NOALLOC_SCRATCH_BYTES (e.g. more than about 380k tokens of 256 floats, or
 * 182k of 1024).  Every call on one device shares the array, which keeps the
 * last call's contents (the call clears what must start at zero itself): calls
 * in order on one stream are safe; calls that can overlap on one device
 * (different streams, nothing ordering them) race on it.
 */
#define EMB_NOALLOC_SCRATCH_BYTES ((size_t)16 << 20)
int emb_grad_coalesce_by_owner_noalloc(const int32_t *ids, int32_t T,
                                       const void *grad, int32_t grad_dtype,
                                       int32_t D, int64_t V,
                                       const int32_t *row_owner, int32_t P,
                                       int32_t *send_ids, int32_t *seg_offsets,
                                       float *send_rows, int32_t *send_counts,
                                       int32_t *send_offsets,
                                       int32_t *num_unique,
                                       int32_t *dev_status, void *stream);

/*
 * emb_grad_coalesce_by_owner with the set split of Vertical Sparse Scheduling
 * (Algorithm 1; Sec. 4.2.2, "Minimum Dependency of Embedding").  With the next
 * batch's ids known in advance (next_ids [T_next]), a coalesced row is prior
 * when its id occurs in the next batch (i_prior = D_u intersect D_next) and
 * delayed otherwise.  The send layout holds 2P groups: the prior rows of
 * owners 0 .. P-1, then the delayed rows of owners 0 .. P-1, each group in
 * ascending id:
 *   send_counts [2P], send_offsets [2P + 1]: group g is
 *   [send_offsets[g], send_offsets[g + 1]); prior rows are
 *   [send_offsets[0], send_offsets[P]), delayed [send_offsets[P], send_offsets[2P]).
 * The other outputs and rules are those of emb_grad_coalesce_by_owner.  Ids
 * of next_ids outside [0, V) match no row.  Adam is then applied to each part
 * (emb_sparse_adam_apply with offsets send_offsets and send_offsets + P), both
 * with the same step (Sec. 5.7).
 * workspace: emb_grad_coalesce_split_workspace_bytes(T, T_next, V, D,
 * grad_dtype) bytes, 256-byte aligned.  Requires 0 <= T_next < 2^30 and
 * bits(V) + bits(P) + 1 <= 32 (EMB_ERR_UNSUPPORTED otherwise).
 */
size_t emb_grad_coalesce_split_workspace_bytes(int32_t T, int32_t T_next,
                                               int64_t V, int32_t D,
                                               int32_t grad_dtype);
int emb_grad_coalesce_split(const int32_t *ids, int32_t T,
                            const int32_t *next_ids, int32_t T_next,
                            const void *grad, int32_t grad_dtype, int32_t D,
                            int64_t V, const int32_t *row_owner, int32_t P,
                            int32_t *send_ids, int32_t *seg_offsets,
                            float *send_rows, int32_t *send_counts,
                            int32_t *send_offsets, int32_t *num_unique,
                            void *workspace, size_t workspace_bytes,
                            int32_t *dev_status, void *stream);

/*
 * The receiver side of the sparse-gradient AlltoAll (Sec. 4.1.1 / 4.1.2: every
 * worker sends each owner the coalesced rows it owns; an owner then sums the
 * rows it received for the same index), simulated on this device for P
 * workers whose send layouts sit side by side:
 *   send_ids [P][cap_rows], send_rows [P][cap_rows][D], send_offsets [P][P + 1]:
 *   worker w's rows for owner p at [send_offsets[w][p], send_offsets[w][p + 1])
 *   of its own block (the layout of emb_grad_coalesce_by_owner / emb_pack_by_owner).
 * emb_exchange_simulated moves every block to its receiver (a P x P block
 * transpose; rows are bit copies):
 *   recv_offsets [P][P + 1]: owner p receives worker w's rows at
 *   [recv_offsets[p][w], recv_offsets[p][w + 1]), and all its rows end at
 *   recv_offsets[p][P]; receivers follow each other (owner-major).
 *   recv_ids [P * cap_rows], recv_rows [P * cap_rows][D]; recv_total [1] = rows received.
 * Offsets are clamped into [0, cap_rows]; rows outside a worker's blocks are
 * not sent.  D == 0 moves the ids alone (send_rows and recv_rows may be NULL):
 * the lookup requests of emb_lookup_request.  Requires 1 <= P <= 1024,
 * P * cap_rows < 2^30, D >= 0.
 *
 * emb_receive_merge then coalesces the received rows of every owner (their
 * ids can repeat across senders): emb_grad_coalesce_by_owner over the first
 * *recv_total of the cap received rows (fp32), with the same outputs, rules
 * and workspace (emb_grad_coalesce_workspace_bytes(cap, V, D, EMB_F32)).  Rows
 * of one index are summed in sender order.  The result equals the owner-major
 * coalesce of all workers' tokens together (to the fp32 summation bound).
 */
int emb_exchange_simulated(const int32_t *send_ids, const float *send_rows,
                           const int32_t *send_offsets, int32_t P,
                           int32_t cap_rows, int32_t D, int32_t *recv_ids,
                           float *recv_rows, int32_t *recv_offsets,
                           int32_t *recv_total, void *stream);
int emb_receive_merge(const int32_t *recv_ids, const float *recv_rows,
                      const int32_t *recv_total, int32_t cap, int32_t D,
                      int64_t V, const int32_t *row_owner, int32_t P,
                      int32_t *merged_ids, int32_t *seg_offsets,
                      float *merged_rows, int32_t *merged_counts,
                      int32_t *merged_offsets, int32_t *num_unique,
                      void *workspace, size_t workspace_bytes,
                      int32_t *dev_status, void *stream);

/*
 * Lookup requests of the row-wise partition (Sec. 4.1.1: every process looks
 * up the embeddings of its own training data; with the rows partitioned, the
 * rows a worker needs live with their owners, so the forward pass asks each
 * owner for them and gets them back, the exchange that the column-wise
 * partition replaces by the lookup-result AlltoAll).  Each distinct row is
 * asked for once per worker, however many of its tokens use it.
 *   ids [T] int32; row_owner [V] int32.  A token takes part when its id is in
 *   [0, V) (else EMB_DEV_ID_OUT_OF_RANGE) and its owner in [0, P) (else
 *   EMB_DEV_OWNER_OUT_OF_RANGE).
 * Outputs (device):
 *   req_ids     [T]     the U distinct ids of the tokens that take part,
 *                       grouped by owner (owner 0 first), ascending inside a
 *                       group: the send layout of emb_exchange_simulated (D = 0)
 *   req_counts  [P], req_offsets [P + 1]: owner p's requests at
 *                       [req_offsets[p], req_offsets[p + 1])
 *   num_unique  [1]     U
 *   inverse     [T]     k with req_ids[k] = ids[t] for a token that takes
 *                       part, -1 for one that does not
 * The owners answer with emb_gather of the ids they receive; the rows that
 * come back in request order, [U][D], expand to the batch's lookup with
 * emb_gather(rows, U, D, inverse, T, out) (tokens that take no part get zero
 * rows).  Entries of req_ids past U are left unspecified.
 * workspace: device memory of at least emb_lookup_request_workspace_bytes(T, V)
 * bytes, 256-byte aligned; contents on entry do not matter.  T == 0 writes the
 * empty result.  Requires 1 <= V < 2^31, 1 <= P <= 1024, 0 <= T < 2^30;
 * EMB_ERR_UNSUPPORTED when bits(V) + bits(P) > 32 (the composite sort key of
 * emb_grad_coalesce_by_owner).
 */
size_t emb_lookup_request_workspace_bytes(int32_t T, int64_t V);
int emb_lookup_request(const int32_t *ids, int32_t T, int64_t V,
                       const int32_t *row_owner, int32_t P, int32_t *req_ids,
                       int32_t *req_counts, int32_t *req_offsets,
                       int32_t *num_unique, int32_t *inverse, void *workspace,
                       size_t workspace_bytes, int32_t *dev_status,
                       void *stream);

/*
 * Column-wise partition (Sec. 4.1.1: the table is split by columns before
 * training, so every process keeps the whole vocabulary for its slice of the
 * embedding dimension and all owners receive the same number of rows; the
 * lookup results are redistributed with one AlltoAll, the sparse gradients
 * with another).  This is the paper's own partition; the owner-major calls
 * above are the row-wise one.
 *
 * Owner p of P holds the float columns [off(p), off(p + 1)) of every row, with
 * off(p) = floor(p * D / P) and width w(p) = off(p + 1) - off(p).
 * The COLUMN-BLOCK LAYOUT of capacity C is C * D floats holding P blocks:
 * block p is the [C][w(p)] row-major slice of owner p's columns, at float
 * offset C * off(p); row r of block p is at C * off(p) + r * w(p).  With
 * C = V it is the partitioned table (shard p = block p, all V rows); the
 * shards of exp_avg and exp_avg_sq use the same layout.
 * All three calls are bit copies.  Every call requires 1 <= P <= min(D, 1024)
 * (each owner holds at least one column) and D * P < 2^31.
 *
 * emb_pack_by_column: the gradient payload of the column-wise AlltoAll.
 *   rows [cap_rows][D] (the uniq_grad of emb_grad_coalesce); the first R rows
 *   are packed, R = *num_rows (device int32, clamped into [0, cap_rows]) or
 *   R = cap_rows when num_rows is NULL (this partitions a table: rows = the
 *   [V][D] table, cap_rows = V).
 *   blocks: column-block layout of capacity cap_rows; rows >= R not written.
 *   send_counts [P] (device, may be NULL): R for every owner.  Each owner gets
 *   the same R ids (the uniq_ids of the coalesce, not copied) with its w(p)
 *   columns of each row.
 *   Owner p then applies emb_sparse_adam_apply to its shard (table, exp_avg,
 *   exp_avg_sq at float offset V * off(p), D = w(p)) with the rows of block p.
 *
 * emb_gather_by_column: the lookup of every owner (Sec. 4.1.1: each process
 *   looks up the training data of all processes in its part of the table).
 *   shards: the table in column-block layout of capacity V; ids [T].
 *   blocks: column-block layout of capacity T; block p row t =
 *   columns off(p) .. off(p + 1) - 1 of table row ids[t].  Worker q's tokens
 *   at rows [t0, t1) of every block are what owner p sends q.  An id outside
 *   [0, V) gives zeros and sets EMB_DEV_ID_OUT_OF_RANGE.  Requires
 *   1 <= V < 2^31, T >= 0.
 *
 * emb_assemble_by_column: the receiving side of the lookup-result AlltoAll.
 *   blocks: column-block layout of capacity C; rows [row0, row0 + R) of every
 *   block are joined into rows [R][D].  With the blocks of
 *   emb_gather_by_column and worker q's token range this yields exactly the
 *   rows emb_gather would return for q's ids from the unpartitioned table.
 *   Requires C >= 0, row0 >= 0, R >= 0, row0 + R <= C.
 */
int emb_pack_by_column(const float *rows, const int32_t *num_rows,
                       int32_t cap_rows, int32_t D, int32_t P, float *blocks,
                       int32_t *send_counts, void *stream);
int emb_gather_by_column(const float *shards, int64_t V, int32_t D, int32_t P,
                         const int32_t *ids, int32_t T, float *blocks,
                         int32_t *dev_status, void *stream);
int emb_assemble_by_column(const float *blocks, int64_t C, int64_t row0,
                           int32_t R, int32_t D, int32_t P, float *rows,
                           void *stream);

/*
 * Communication cost model of a sparse gradient (Sec. 4.1.2, Table 2): the
 * time of one training step's exchange of an embedding table of M bytes whose
 * gradient has density alpha (the fraction of rows with a nonzero gradient,
 * U / V for one batch), for N workers, with bandwidth B between any two
 * workers and start-up latency beta per message:
 *   EMB_COMM_ALLTOALL   2 (N - 1) (alpha M / (N B) + beta)
 *                       (lookup results and gradients, each alpha M / N per peer)
 *   EMB_COMM_ALLREDUCE  2 (N - 1) (M / (N B) + beta)    (dense ring)
 *   EMB_COMM_PS         2 N (alpha M / (S B) + beta)    (S servers; Table 2
 *                       states the lower bound, S = n nodes)
 *   EMB_COMM_ALLGATHER  (N - 1) (alpha M / B + beta)
 * Host-only arithmetic in double.  *seconds receives the cost in the units of
 * M / B and beta (host pointer).  S is read for EMB_COMM_PS only.
 * Requires N >= 1, S >= 1, M >= 0, 0 <= alpha <= 1, B > 0, beta >= 0.
 */
#define EMB_COMM_ALLTOALL 0
#define EMB_COMM_ALLREDUCE 1
#define EMB_COMM_PS 2
#define EMB_COMM_ALLGATHER 3
int emb_comm_cost(int32_t scheme, int64_t N, int64_t S, double M,
                  double alpha, double B, double beta, double *seconds);

/*
 * Row-wise (lazy) Adam on received rows (Sec. 4.1.1: each process updates its
 * embedding rows with the exchanged gradients; Sec. 5.7: Adam with a global
 * step counter that the caller owns and advances once per iteration).
 * Kingma & Ba, Algorithm 1, for each listed row r and column j:
 *   m <- b1 m + (1 - b1) g ;  v <- b2 v + (1 - b2) g^2
 *   w <- w - lr * (m / (1 - b1^step)) / (sqrt(v / (1 - b2^step)) + eps)
 * computed in fp32 (bias corrections formed in fp64 on the host).
 *   table, exp_avg, exp_avg_sq [V][D] fp32, updated in place.
 *   row_ids [cap_rows], rows [cap_rows][D]: the rows i in
 *   [offsets[shard_begin], offsets[shard_end]) are applied, with offsets
 *   [P + 1] in device memory (the send_offsets of emb_pack_by_owner);
 *   that range must lie within [0, cap_rows).
 * Rows not listed keep table, exp_avg and exp_avg_sq bit-unchanged.  Listed
 * row ids must be distinct (true of pack output); an id outside [0, V) is
 * skipped and sets EMB_DEV_ID_OUT_OF_RANGE.
 * Requires 1 <= P <= 1024, 0 <= shard_begin <= shard_end <= P, step >= 1,
 * 0 <= beta1, beta2 < 1, eps >= 0.
 */
int emb_sparse_adam_apply(float *table, float *exp_avg, float *exp_avg_sq,
                          int64_t V, int32_t D, const int32_t *row_ids,
                          const float *rows, const int32_t *offsets, int32_t P,
                          int32_t shard_begin, int32_t shard_end,
                          int32_t cap_rows, double lr, double beta1,
                          double beta2, double eps, int64_t step,
                          int32_t *dev_status, void *stream);

/*
 * The update's coefficients for one step (Kingma & Ba, Algorithm 1, as
 * emb_sparse_adam_apply forms them: bias corrections in fp64, each
 * coefficient rounded once to fp32), written to out[EMB_ADAM_COEFFS_WORDS]
 * (host memory): beta1, 1 - beta1, beta2, 1 - beta2, lr / (1 - beta1^step),
 * 1 / (1 - beta2^step), eps, 0.  Copied to device memory and named by
 * emb_step_args.adam_coeffs, they let steps captured in a graph advance the
 * step count on every replay (Sec. 5.7: the step counter grows once per
 * iteration).  Host arithmetic only; EMB_ERR_INVALID_ARG as for
 * emb_sparse_adam_apply's hyper-parameters.
 */
#define EMB_ADAM_COEFFS_WORDS 8
int emb_adam_coeffs(double lr, double beta1, double beta2, double eps,
                    int64_t step, float *out);

/*
 * ---------------------------------------------------------------------------
 * Step executor.  Not a step of the path itself: it enqueues the four calls
 * above for one training step of one table, in data order, on up to four streams,
 * so that the latency-bound coalesce/pack work of a step overlaps the
 * bandwidth-bound lookup and update of neighbouring steps (the sparse
 * gradient work runs in GPU idle time, as in Vertical Sparse Scheduling,
 * Sec. 4.2.2, here on one GPU).  One host call per step keeps the host ahead
 * of the GPU.
 *
 * The caller rotates buffer sets (coalesce and pack workspaces, uniq_* and
 * send_* outputs; two unless `sets` says more) between consecutive steps and
 * gives each set its own events; `reuse` is nonzero when the set was used
 * before.  Below, "s-2" is the set's previous step, s - sets.  The streams may
 * differ between sets, and a set's streams may change from one use to the
 * next (with the `coalesce` stream alternating between two streams, the sorts
 * of consecutive steps run side by side): the waits on a set's previous use
 * are issued whatever the streams, and cost nothing when the stage waited for
 * ran on the waiting stream.  `lookup_update` must be the same stream for
 * every step of a table (the lookup of a step follows the previous update in
 * stream order), and a table's steps change between split and not split only
 * once the work enqueued so far has completed.
 *
 * by_owner == 0: emb_grad_coalesce on the `coalesce` stream, emb_pack_by_owner
 * on the `pack` stream, lookup and update on `lookup_update`, with the waits
 *   coalesce(s) after pack(s-2)                (same unique-row buffers)
 *   pack(s)     after coalesce(s), update(s-2) (reads unique rows; same send buffers)
 *   update(s)   after pack(s)                  (reads the packed rows)
 *   lookup(s+1) after update(s)                (same stream; reads the table)
 * (events coalesced, packed, updated).
 *
 * by_owner != 0: emb_grad_coalesce_by_owner in its two halves.  The sort of
 * the (owner, id) keys, which does not read the gradients, runs on the
 * `coalesce` stream; the reduction, which writes the send buffers directly,
 * on the `pack` stream; the lookup and the update on `lookup_update`;
 * uniq_ids, uniq_grad and ws_pack are not used.  Waits:
 *   sort(s)     after reduce(s-2)              (same coalesce workspace)
 *   reduce(s)   after sort(s), update(s-2)     (reads the sorted keys; same send buffers)
 * (with sets >= 4 and no split: sort(s) after update(s-sets), which followed
 * reduce(s-sets), and reduce(s) after sort(s) only: one wait fewer per step)
 *   update(s)   after reduce(s)                (reads the send rows)
 *   lookup(s+1) after update(s)                (same stream; reads the table)
 * (events sorted, coalesced, updated).  The sorts thus run up to a step
 * ahead, and a step's reduction runs beside the previous update and its own
 * lookup.
 *
 * split != 0 (with by_owner): Vertical Sparse Scheduling (Sec. 4.2.2,
 * Algorithm 1).  The coalesce is emb_grad_coalesce_split with the next
 * batch's ids (args.next_ids, which must be the ids of the next call), and the
 * update runs in two parts: the prior rows (needed by the next lookup) on
 * `lookup_update` right after the lookup, the delayed rows on the `delayed`
 * stream, beside the next lookup, which reads none of them.  Both parts use
 * the same Adam step.  Waits, in addition to the above:
 *   lookup(s)   after delayed update of the step two back (its rows may be in
 *               this batch; this one is two steps whatever `sets` is)
 *   prior(s)    after reduce(s)
 *   delayed(s)  after reduce(s), lookup(s)     (reads the send rows; lookup(s) reads its rows)
 *   reduce(s)   after delayed update(s-2)      (same send buffers)
 * (events gathered: the end of the lookup, delayed_done: the end of the
 * delayed update).  The pair timing[4..5] times the prior update and
 * timing[6..7] the delayed one.
 *
 * With all streams equal the calls simply run one after another, and the
 * results are bitwise the same either way.
 *
 * Graph capture.  While `lookup_update` is being captured into a HIP graph
 * (stream capture, events only: step signals and timing events are refused
 * with EMB_ERR_UNSUPPORTED), the executor records every stage end as an event
 * node instead of attaching events to dispatches.  The captured steps must not
 * wait for steps enqueued before the capture began: each buffer set's first use
 * in a capture has reuse == 0 (a replayed graph runs after the work before it
 * on its stream, whole).  With args.adam_coeffs the update reads its
 * coefficients from device memory when it runs, so a replay can apply other
 * step numbers than the ones the capture saw.
 * ---------------------------------------------------------------------------
 */
typedef struct {
  void *lookup_update;          /* stream of emb_gather and emb_sparse_adam_apply */
  void *coalesce;               /* stream of emb_grad_coalesce (by_owner: of its sort) */
  void *pack;                   /* stream of emb_pack_by_owner */
  void *delayed;                /* split: stream of the delayed update */
  void *sorted, *coalesced, *packed, *updated; /* events of this step's buffer set
                                   (sorted: by_owner only; packed: by_owner == 0 only) */
  void *gathered, *delayed_done; /* split only: events of this step's buffer set */
  int32_t reuse;                /* the buffer set was used two steps ago */
  int32_t by_owner;             /* use emb_grad_coalesce_by_owner instead of coalesce + pack */
  int32_t split;                /* by_owner with the prior / delayed split */
  void *timing[8];              /* optional timing events (NULL to skip): begin/end of
                                   gather, coalesce, pack, adam, each recorded on the
                                   stream the (first / last) kernel runs on; the adam
                                   pair takes the update kernel's own start and end
                                   from its dispatch; by_owner records no pack pair */
  void *signals;                /* optional step signals of the table
                                   (emb_step_signals_create): when set, the waits above
                                   go through them and the events sorted .. delayed_done
                                   and `reuse` are not used (they may be NULL) */
  int32_t sets;                 /* buffer sets the caller rotates (0: 2; at most 64): the
                                   waits for a set's earlier use ("s-2" above) reach back
                                   this many steps; `reuse` means the set was used `sets`
                                   steps ago.  With events the split needs 2 */
} emb_step_schedule;

typedef struct {
  float *table, *exp_avg, *exp_avg_sq; /* [V][D] fp32, updated in place */
  int64_t V;
  int32_t D;
  const int32_t *row_owner; /* [V] */
  int32_t P;
  const int32_t *ids;       /* [T] */
  int32_t T;
  const int32_t *next_ids;  /* split: [T_next] ids of the next call's batch */
  int32_t T_next;
  const void *grad;         /* [T][D], grad_dtype */
  int32_t grad_dtype;
  int32_t cap_rows;         /* capacity of the uniq_*, seg_offsets and send_* buffers (>= T, T_next) */
  float *lookup;            /* [T][D] gather output */
  int32_t *uniq_ids, *seg_offsets, *num_unique;
  float *uniq_grad;
  int32_t *send_ids, *send_counts, *send_offsets; /* counts [P] and offsets [P + 1]; split: [2P], [2P + 1] */
  float *send_rows;
  void *ws_coalesce;
  size_t ws_coalesce_bytes;
  void *ws_pack;
  size_t ws_pack_bytes;
  double lr, beta1, beta2, eps;
  int64_t step;             /* Adam step (>= 1), one per iteration (Sec. 5.7) */
  int32_t *dev_status;      /* optional */
  const void *adam_coeffs;  /* optional, 16-byte aligned device memory: this step's
                               EMB_ADAM_COEFFS_WORDS update coefficients (emb_adam_coeffs),
                               read by the update kernel when it runs instead of those of
                               `step` (for steps replayed from a graph) */
} emb_step_args;

/* Events for the schedule (hipEventCreateWithFlags; timing: nonzero for
 * timing events).  A host-side runtime object, not device memory. */
int emb_event_create(void **event, int32_t timing);
int emb_event_destroy(void *event);
/* Milliseconds between two completed timing events. */
int emb_event_elapsed_ms(void *start, void *end, float *ms);

/* Step signals: the cross-stream order of emb_train_step kept through stream
 * memory operations instead of events.  A handle holds two words of HIP
 * signal memory per stage (sorted, coalesced, packed, updated, gathered,
 * delayed_done), for steps of even and of odd number, and a step counter.
 * Each emb_train_step call that names the handle takes the next step number n;
 * the end of a stage writes n into its word of n's parity
 * (hipStreamWriteValue32) and a stream that must follow the stage of step
 * n - k waits until the word of (n - k)'s parity reaches n - k
 * (hipStreamWaitValue32, >=).  (With the two parities on two streams, as when
 * the odd and even steps' coalesce runs on two streams, each word has a single
 * writer.)
 * The order is the one listed above for the events.  A wait never targets
 * more than the value of the last write already enqueued for its word (a
 * stage that did not run in the step waited for is waited for at its last
 * run, or not at all), so every wait refers to an earlier enqueued write and
 * the waits cannot deadlock, whatever modes the calls of a handle mix.
 * On this runtime a wait on
 * a pending event costs the host about four times as much as this write and
 * wait, and with the host running ahead of the GPU nearly every wait is on a
 * pending event; the GPU-side order is the same.
 * Use one handle per table (both of its buffer sets), from one host thread.
 * If a call fails part-way, every stage of its step is marked done so that no
 * later wait blocks.  destroy: only once the work of every step enqueued with
 * the handle has completed; the signal memory is kept for a later handle (it
 * is never returned to the runtime).  create returns EMB_ERR_UNSUPPORTED if
 * the device cannot wait on stream values. */
int emb_step_signals_create(void **signals);
int emb_step_signals_destroy(void *signals);

/* Enqueue one training step of one table (see above).  Returns the first
 * failing call's status; nothing after it is enqueued. */
int emb_train_step(const emb_step_args *args, const emb_step_schedule *sched);

/* Two-thread enqueue.  Not a step of the method: a host-side way to enqueue
 * the same steps for callers whose host time per step bounds them (small
 * batches: the executor issues a dozen HIP calls per step, and a wait on an
 * event still pending on another stream alone costs the host about 10 us).
 * emb_train_step_queued enqueues the sort and the reduction of the step (on
 * `coalesce` and `pack`) from the calling thread and hands the rest (the
 * lookup, the wait for the reduction and the update, on `lookup_update`) to
 * the queue's worker thread, which enqueues the handed steps in call order on
 * the device that was current at the call.  The stream order is exactly the
 * one emb_train_step gives.  Before the calling thread waits on a buffer
 * set's earlier use, it waits (on the host, at most 30 s, else
 * EMB_ERR_LAUNCH) until the worker has enqueued that use's update.
 * Restrictions: events (no step signals), by_owner without the split, not
 * under graph capture, `coalesce` and `pack` other streams than
 * `lookup_update` (each stream is fed by one thread; EMB_ERR_UNSUPPORTED
 * otherwise); one queue per table,
 * used from one thread; timing events in `sched` are recorded as usual, those
 * of the lookup and the update by the worker.
 * Until emb_step_queue_flush has returned, the handed parts of the steps may
 * not be enqueued yet: call it before enqueuing anything on `lookup_update`
 * that must follow them, and before reading what they write.  flush and
 * destroy return the first error of a handed part (a failed part stops its
 * own step only, as in emb_train_step); destroy enqueues what was handed
 * before it stops the worker.  The queue is host memory and a thread; the
 * library allocates nothing on the device for it. */
int emb_step_queue_create(void **queue);
int emb_step_queue_flush(void *queue);
int emb_step_queue_destroy(void *queue);
int emb_train_step_queued(void *queue, const emb_step_args *args, const emb_step_schedule *sched);

#ifdef __cplusplus
}
#endif
#endif /* EMB_H */
