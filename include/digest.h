/*
 * digest.h -- C ABI of the MI355X (gfx950) hot path of DIGEST:
 * one graph partition's GCN layer with stale halo representations, plus the
 * periodic push/pull of representations through a representation store.
 *
 * Paper: "Distributed Graph Neural Network Training with Periodic Stale
 * Representation Synchronization" (DIGEST), arXiv 2206.00057.
 *
 * Model of one partition m (Sec. 2 Eq. 2, Sec. 3.1 Eq. 4-5):
 *   H^{l} = sigma( P_in H_in^{l-1} W^l + P_out H~_out^{l-1} W^l ),
 * where P_in / P_out are the columns of the GCN propagation matrix P_m
 * (rows = the partition's own nodes) that point inside / outside the
 * partition, H_in are fresh own rows and H~_out are stale rows of the
 * out-of-partition neighbours ("halo") pulled from the store (Sec. 3.2).
 *
 * Conventions for every call below
 *   - Status: 0 (DIGEST_OK) or a negative digest_status.  On error nothing
 *     has been enqueued, outputs are untouched and the handle stays valid;
 *     digest_last_error() returns a message (thread-local).
 *   - Device pointers are caller-owned (e.g. PyTorch tensors), fp32,
 *     row-major, contiguous, 4-byte aligned (16-byte aligned rows run
 *     faster); node ids are int64 at the ABI.
 *   - hip_stream is a hipStream_t (NULL = the default stream); every device
 *     call only enqueues work on it and never synchronises the host, except
 *     digest_profile_read.
 *   - A handle is not thread-safe; distinct handles are independent.
 *   - Terminology: "level" l is the representation H^{l} (width d_l);
 *     layer l (1..L) maps level l-1 to level l.  Level 0 is the feature
 *     matrix X.  The store of level l is an [n_global, d_l] array.
 */
#ifndef DIGEST_H
#define DIGEST_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct digest_partition digest_partition;

typedef enum {
    DIGEST_OK = 0,
    DIGEST_EINVAL = -1,  /* malformed argument (ids, CSR, widths, layer/level, NULL) */
    DIGEST_ENOMEM = -2,  /* host allocation failed, or workspace too small */
    DIGEST_EHIP = -3,    /* HIP runtime error (message in digest_last_error) */
    DIGEST_ESTATE = -4   /* call out of order (see each call) */
} digest_status;

enum { DIGEST_ACT_RELU = 0, DIGEST_ACT_IDENTITY = 1 };
enum { DIGEST_PUSH_BOUNDARY = 0, DIGEST_PUSH_ALL_OWNED = 1 };
enum { DIGEST_PULL_ROWS = 0, DIGEST_PULL_AGGREGATE = 1 };

/* Message describing the last non-OK status returned on this thread. */
const char *digest_last_error(void);

/*
 * Build one partition (host only: no HIP call is made here).
 *
 * Eq. 2 splits a node's neighbours into in-subgraph and out-of-subgraph
 * sets; Sec. 3.2 defines the out-of-subgraph set of a partition as every
 * neighbour of an owned node that is not owned ("halo").
 *
 *   n_global       number of nodes of the whole graph, 1 <= n_global < 2^31.
 *   indptr         [n_owned+1] CSR row pointers of P_m: row i belongs to
 *                  owned[i]; indptr[0] == 0, non-decreasing, nnz < 2^31.
 *   indices        [nnz] GLOBAL column ids; each must be owned or halo.
 *                  Repeated (row, column) entries are allowed and summed.
 *   values         [nnz] entries of P (the GCN-normalised adjacency with
 *                  self loops, computed by the caller; not renormalised).
 *   owned          [n_owned] distinct ids in [0, n_global) (n_owned >= 0).
 *   halo           [n_halo] distinct ids in [0, n_global), disjoint from
 *                  owned; unreferenced halo ids are allowed.  Halo slot j
 *                  gets local column n_owned + j.
 *   n_layers, widths  L >= 1 and d_0..d_L (each in [1, 65536]).
 *   out            receives the handle.
 * All host arrays are copied; the caller may free them on return.
 * Derived here: the local CSR, the boundary rows (owned rows with at least
 * one halo column, ascending: the rows the push writes), and the CSR of
 * P_in^T (row c lists the owned rows i with an entry in column c, i
 * ascending).
 * Errors: DIGEST_EINVAL for any violation above, DIGEST_ENOMEM.
 */
digest_status digest_partition_create(int64_t n_global, const int64_t *indptr,
                                      const int64_t *indices, const float *values,
                                      const int64_t *owned, int64_t n_owned,
                                      const int64_t *halo, int64_t n_halo,
                                      int32_t n_layers, const int32_t *widths,
                                      digest_partition **out);

/* Release a handle (NULL is ignored).  The bound workspace is the caller's. */
void digest_partition_destroy(digest_partition *p);

/* Sizes: boundary rows (owned rows with at least one halo column, in
 * ascending row order: bnd[0..n_boundary)), nnz of P_m, nnz of the owned
 * block P_in, and the device workspace bytes the handle needs.  Any output
 * pointer may be NULL. */
digest_status digest_partition_query(const digest_partition *p, int64_t *n_boundary,
                                     int64_t *nnz, int64_t *nnz_in,
                                     size_t *workspace_bytes);

/*
 * Bind caller-allocated device memory (>= workspace_bytes, 256-byte
 * aligned) and upload the partition's index structures into it on
 * hip_stream.  The library owns the layout of this memory (local CSR,
 * P_in^T, id lists, one halo buffer and one halo aggregate per level, the
 * aggregated input AH of each layer kept for the backward, reduction
 * scratch) until the next bind
 * or destroy.  Re-binding resets the pull/forward state: every level must
 * be pulled again, and every backward (GCN or GAT) needs a forward after
 * the bind.
 * Errors: DIGEST_EINVAL (NULL, misaligned), DIGEST_ENOMEM (too small),
 * DIGEST_EHIP.
 */
digest_status digest_partition_bind_workspace(digest_partition *p, void *dev_ptr,
                                              size_t bytes, void *hip_stream);

/* Test hook (host arrays, host-side copy of the maps; any may be NULL):
 * col_local[nnz] local column numbers, boundary_gid / boundary_local
 * [n_boundary] global ids and owned-row numbers of the pushed rows. */
digest_status digest_partition_export_maps(const digest_partition *p, int32_t *col_local,
                                           int64_t *boundary_gid,
                                           int32_t *boundary_local);

/* Test hook: CSR of P_in^T (t_indptr[n_owned+1], t_src[nnz_in], t_vals[nnz_in]);
 * row c lists the owned rows with an entry in owned column c, ascending. */
digest_status digest_partition_export_transpose(const digest_partition *p,
                                                int64_t *t_indptr, int32_t *t_src,
                                                float *t_vals);

/* Test hook: copy the halo buffer of `level` ([n_halo, d_level], filled by
 * digest_pull) into the caller's device array `out` on hip_stream.
 * Errors: DIGEST_EINVAL, DIGEST_ESTATE (no workspace; pull mode
 * DIGEST_PULL_AGGREGATE, which keeps no halo rows), DIGEST_EHIP. */
digest_status digest_partition_read_halo(const digest_partition *p, int32_t level, float *out,
                                         void *hip_stream);

/*
 * What a pull of this handle keeps (host-side state, no device work):
 *   DIGEST_PULL_ROWS (the default): the halo rows in the halo buffer, and
 *     the halo aggregate formed from them (digest_pull).
 *   DIGEST_PULL_AGGREGATE: the halo aggregate alone, gathered straight from
 *     the store; the halo buffer is left alone, so a pull moves the halo
 *     rows once instead of twice.  For callers that use the GCN layer only:
 *     the calls that read halo rows (the GAT layer and the halo read-back)
 *     return DIGEST_ESTATE.
 * A change of mode marks every level as not pulled.  Callers that capture
 * graphs set the mode before the capture.
 * Errors: DIGEST_EINVAL (NULL, unknown mode).
 */
digest_status digest_partition_set_pull_mode(digest_partition *p, int32_t mode);

/*
 * Pull (Sec. 3.2; Algorithm 1 pulls when r mod N == 0): gather the stale
 * rows of the halo nodes of level `level` out of the store into the
 * handle's halo buffer of that level:  halo_buf[j, :] = store[halo[j], :].
 * The same call forms the halo aggregate of the level, the halo rows'
 * share of Eq. 5's aggregation for the boundary rows,
 *   S[b, :] = sum_j P_out[bnd[b], j] halo_buf[j, :]   (n_boundary rows),
 * which stays constant until the next pull of the level; the GCN forward of
 * layer level+1 reads it instead of the halo rows (a handle with a GAT
 * workspace bound skips it here and forms it in each GCN forward).  In pull
 * mode DIGEST_PULL_AGGREGATE the call forms S from the store's rows directly
 * and leaves the halo buffer as it was.
 *   level  0..L-1 (level 0 = the static features X, pulled once).
 *   store  device [n_global, d_level].
 * Errors: DIGEST_EINVAL, DIGEST_ESTATE (no workspace bound), DIGEST_EHIP.
 */
digest_status digest_pull(digest_partition *p, int32_t level, const float *store,
                          void *hip_stream);

/*
 * Push (Sec. 3.2; Algorithm 1 pushes when (r-1) mod N == 0): write freshly
 * computed own rows of level `level` into the store:
 *   store[owned[b], :] = h_own[b, :]  for b in the boundary rows
 *   (mode DIGEST_PUSH_BOUNDARY), or for every owned row (mode
 *   DIGEST_PUSH_ALL_OWNED, the paper's wording).
 * The boundary rows are the owned rows with a halo column.  They are the
 * only rows other partitions read when P is structurally symmetric (an
 * edge u -> v implies v -> u, as for the GCN normalisation of an
 * undirected graph): a node in another partition's halo then has that
 * partition's node among its own columns.  For a directed P use
 * DIGEST_PUSH_ALL_OWNED, or rows some other partition reads may never be
 * written.
 * Other store rows are untouched.
 *   level  1..L-1 (the stale levels; level 0 is static, level L is never
 *          stored).   h_own  device [n_owned, d_level].
 *   store  device [n_global, d_level].
 * Errors: DIGEST_EINVAL, DIGEST_ESTATE (no workspace), DIGEST_EHIP.
 */
digest_status digest_push(digest_partition *p, int32_t level, const float *h_own,
                          float *store, int32_t mode, void *hip_stream);

/*
 * Layer forward (Eq. 5):  h_out = act(P_in h_in W + P_out halo_buf[layer-1] W)
 *   layer  1..L.   h_in  device [n_owned, d_{layer-1}] (fresh own rows).
 *   w      device [d_{layer-1}, d_layer].   h_out device [n_owned, d_layer].
 *   act    DIGEST_ACT_RELU or DIGEST_ACT_IDENTITY (the paper uses ReLU on
 *          hidden layers and raw logits at the last layer).
 * The halo term enters through the level's halo aggregate S (digest_pull):
 * P_out halo_buf = E S, with E placing S's rows at the boundary rows, so
 * that h_out = act(P_s [h_in; S] W) with P_s = [P_in | E] (the same result
 * up to float rounding).
 * Order of the two products (the same result up to float rounding): a
 * layer is computed transform-first, T = [h_in; S] W over the
 * n_owned + n_boundary rows, then h_out = act(P_s T), when a cost model of
 * the layer's forward and backward says that is cheaper: it weighs the
 * gathered bytes of the sparse aggregations (P_s and P_in^T at width d_out,
 * against P_s at width d_in plus, above layer 1, the input gradient's
 * aggregation), the GEMM flops (over n_owned + n_boundary rows against
 * n_owned rows) and the row copies at measured MI355X rates.  Otherwise the
 * layer aggregates first, AH = P_s [h_in; S], then h_out = act(AH W),
 * keeping AH in the workspace for the backward.
 * Errors: DIGEST_EINVAL, DIGEST_ESTATE (no workspace, or level layer-1 never
 * pulled while the partition has halo nodes), DIGEST_EHIP.
 */
digest_status digest_layer_forward(digest_partition *p, int32_t layer, const float *h_in,
                                   const float *w, float *h_out, int32_t act,
                                   void *hip_stream);

/*
 * Layer backward (Eq. 6 with the upstream gradient; GCN backward of
 * Appendix A.3) of the last forward of `layer`:
 *   D     = dh_out * 1[h_out > 0]  (ReLU) or dh_out (identity)
 *   dw    = (P_m [h_in; halo])^T D                      (overwritten)
 *   dh_in = P_in^T D W^T           if dh_in != NULL    (overwritten)
 * The stale halo rows are constants of the layer: they get no gradient.
 * A transform-first layer forms dw as [h_in; S]^T (P_s^T D): the owned
 * rows' P_in^T D and, for the boundary rows, D's own rows.
 *   h_in   the same device array the forward of this layer read (it must
 *          be unchanged); h_out, dh_out device [n_owned, d_layer];
 *   w device [d_{layer-1}, d_layer];  dw device [d_{layer-1}, d_layer];
 *   dh_in device [n_owned, d_{layer-1}].
 * Errors: DIGEST_EINVAL, DIGEST_ESTATE (no forward of this layer since the
 * workspace was bound, or level layer-1 pulled again since that forward:
 * the halo rows the forward used are gone), DIGEST_EHIP.
 */
digest_status digest_layer_backward(digest_partition *p, int32_t layer, const float *h_in,
                                    const float *h_out, const float *dh_out,
                                    const float *w, float *dw, float *dh_in,
                                    void *hip_stream);

/*
 * Halo gradient (the stale-gradient term of the appendix's DIGEST backward,
 * P_out^T D W^T): the gradient of this subgraph's loss with respect to the
 * rows of its halo nodes at level layer-1, from the last forward of
 * `layer` (2..L):
 *   D       = dh_out * 1[h_out > 0] (ReLU) or dh_out (identity)
 *   dh_halo = P_out^T D W^T          [n_halo, d_{layer-1}], halo slot order
 * (row j belongs to halo node halo[j]).  digest_layer_backward drops this
 * term (halo rows are constants of the iteration); exchanging it through
 * digest_push_add / digest_pull_add gives the owners of the halo nodes the
 * gradient of the other subgraphs' losses.
 *   h_out, dh_out device [n_owned, d_layer]; w device [d_{layer-1}, d_layer].
 * Errors: DIGEST_EINVAL (layer < 2, NULL), DIGEST_ESTATE (no forward of the
 * layer, no workspace), DIGEST_EHIP.
 */
digest_status digest_halo_gradient(digest_partition *p, int32_t layer, const float *h_out,
                                   const float *dh_out, const float *w, float *dh_halo,
                                   void *hip_stream);

/*
 * Layer backward with the halo gradient (the appendix's DIGEST backward
 * with its stale-gradient term): the outputs of digest_layer_backward
 * (dw, dh_in) and the dh_halo of digest_halo_gradient, from shared
 * products.  Aggregating first, the transposed aggregation runs over all of
 * P_m^T, so D W^T is formed once for the owned and the halo rows;
 * transform-first, P_in^T D and P_out^T D share D (and its ReLU mask).
 *   layer 2..L;  dh_in device [n_owned, d_{layer-1}] (required when
 *   n_owned > 0);  dh_halo device [n_halo, d_{layer-1}] (required when
 *   n_halo > 0); other arguments as for digest_layer_backward.
 * Results equal those of the two separate calls up to float32 rounding
 * order.
 * Errors: those of digest_layer_backward; DIGEST_EINVAL for layer 1 or a
 * NULL dh_in / dh_halo.
 */
digest_status digest_layer_backward_halo(digest_partition *p, int32_t layer, const float *h_in,
                                         const float *h_out, const float *dh_out,
                                         const float *w, float *dw, float *dh_in,
                                         float *dh_halo, void *hip_stream);

/*
 * Gradient push: add this subgraph's halo gradient of level `level` into a
 * gradient store indexed by node id, gstore[halo[j], :] += dh_halo[j, :]
 * (float32 adds; the halo ids are distinct, so one call never adds twice to
 * a row; calls for different subgraphs on one stream add in call order).
 *   level 1..L-1;  dh_halo device [n_halo, d_level];  gstore device
 *   [n_global, d_level].
 * Errors: DIGEST_EINVAL, DIGEST_ESTATE (no workspace), DIGEST_EHIP.
 */
digest_status digest_push_add(digest_partition *p, int32_t level, const float *dh_halo,
                              float *gstore, void *hip_stream);

/*
 * Gradient pull: add what the other subgraphs pushed for this subgraph's
 * own nodes to its gradient and clear those store rows for the next use:
 *   dh_own[i, :] += gstore[owned[i], :];  gstore[owned[i], :] = 0.
 *   level 1..L-1;  gstore device [n_global, d_level];  dh_own device
 *   [n_owned, d_level] (e.g. the dh_in of the next layer's backward).
 * Errors: DIGEST_EINVAL, DIGEST_ESTATE (no workspace), DIGEST_EHIP.
 */
digest_status digest_pull_add(digest_partition *p, int32_t level, float *gstore, float *dh_own,
                              void *hip_stream);

/*
 * GAT layer over stale halo rows: the stale-representation layer of Eq. 4
 * with the attention aggregation of the GAT model the paper's experiments
 * train (single head; the paper cites the model and gives no formulas):
 *   z_v     = x_v W          for every local row v: owned rows from h_in,
 *                            halo rows from the stale halo buffer of level
 *                            layer-1 (digest_pull)
 *   s_v     = z_v . att[:,0] (source score),  t_i = z_i . att[:,1] (target)
 *   e_ik    = LeakyReLU(t_i + s_{col k}, negative_slope)
 *             over the entries k of owned row i (the CSR given at create;
 *             its values are not used, only its structure)
 *   alpha   = softmax of e over each row's entries
 *   h_out_i = act(sum_k alpha_ik z_{col k})   (an empty row gives act(0))
 * The GAT calls need a second workspace, bound once after
 * digest_partition_bind_workspace; it keeps z, the scores and alpha of
 * every layer from the forward for the backward.  The GCN calls are
 * unaffected by it.
 */

/* Bytes of the GAT workspace (256-byte aligned device memory). */
digest_status digest_gat_query(const digest_partition *p, size_t *workspace_bytes);

/* Bind the GAT workspace (caller-owned device memory, at least the queried
 * size, 256-byte aligned); uploads the transposed-entry permutation and
 * waits for the upload.  Errors: DIGEST_EINVAL, DIGEST_ENOMEM (too small),
 * DIGEST_EHIP. */
digest_status digest_gat_bind_workspace(digest_partition *p, void *dev_ptr, size_t bytes,
                                        void *hip_stream);

/*
 * GAT forward of `layer` (1..L):
 *   h_in  device [n_owned, d_{layer-1}];  w device [d_{layer-1}, d_layer];
 *   att   device [d_layer, 2] row-major (column 0 source, column 1 target);
 *   negative_slope in [0, 1] (the GAT model uses 0.2);
 *   h_out device [n_owned, d_layer];  act DIGEST_ACT_RELU or _IDENTITY.
 *   d_layer <= 512.
 * Errors: DIGEST_EINVAL (range, NULL, width), DIGEST_ESTATE (no workspace
 * or GAT workspace, level layer-1 never pulled, pull mode
 * DIGEST_PULL_AGGREGATE with halo nodes), DIGEST_EHIP.
 */
digest_status digest_gat_forward(digest_partition *p, int32_t layer, const float *h_in,
                                 const float *w, const float *att, float negative_slope,
                                 float *h_out, int32_t act, void *hip_stream);

/*
 * GAT backward of `layer`, by the chain rule through the forward; halo rows
 * are constants (no gradient), but their z rows depend on W, so they
 * contribute to dw and datt:
 *   D_i      = dh_out_i * act'(h_out_i)
 *   dpre_ik  = alpha_ik (D_i . z_{col k} - D_i . o_i) LeakyReLU'(t_i + s_{col k})
 *   dz_{col k} += alpha_ik D_i + dpre_ik att[:,0];  dz_i += dpre_ik att[:,1]
 *   datt     = [sum dpre_ik z_{col k}, sum dpre_ik z_i]      [d_layer, 2]
 *   dw       = sum over local rows v of x_v^T dz_v           [d_{layer-1}, d_layer]
 *   dh_in_i  = dz_i W^T (owned rows; NULL skips it)
 *   h_in, h_out, dh_out, w, att: as in and out of the forward of the layer.
 * LeakyReLU'(x) is 1 for x > 0 and negative_slope otherwise (at 0 too), and
 * act' is the ReLU mask h_out > 0.  Sums run in a fixed order (no float
 * atomics).
 * Errors: DIGEST_EINVAL, DIGEST_ESTATE (no GAT forward of the layer since
 * the GAT bind, or level layer-1 pulled again since it, pull mode
 * DIGEST_PULL_AGGREGATE with halo nodes), DIGEST_EHIP.
 */
digest_status digest_gat_backward(digest_partition *p, int32_t layer, const float *h_in,
                                  const float *h_out, const float *dh_out, const float *w,
                                  const float *att, float *dw, float *datt, float *dh_in,
                                  void *hip_stream);

/*
 * Local loss head (Eq. 3 with cross entropy), over all n_owned rows:
 *   loss    = -(1/n) sum_i log softmax(logits_i)[labels_i]   (device, 1 float)
 *   dlogits = (softmax(logits) - onehot(labels)) / n          [n_owned, d_L]
 *   labels  device int32 [n_owned]; a label outside [0, d_L) makes that
 *           row's dlogits zero and the loss NaN (checked on the device).
 * Errors: DIGEST_EINVAL, DIGEST_ESTATE (no workspace), DIGEST_EHIP.
 */
digest_status digest_softmax_xent(digest_partition *p, const float *logits,
                                  const int32_t *labels, float *dlogits, float *loss,
                                  void *hip_stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the loss
 * head of digest_softmax_xent without a partition handle or workspace.  It
 * allocates nothing.  Its per-block partial sums go to a fixed device array
 * of the library (DIGEST_STATIC_SCRATCH_FLOATS floats; each GPU the library
 * runs on holds its own copy until the process ends); every block writes
 * its sum before the final mean reads it, so nothing must start at zero.
 * Every call on one GPU shares that array and leaves its contents there:
 * calls that overlap on one GPU (on different streams, or from different
 * host threads) race and must be ordered by the caller.
 *   n_rows      0 <= n_rows <= DIGEST_STATIC_SCRATCH_FLOATS * r(n_classes),
 *               with r(C) = 32 rows for C <= 8, 16 for C <= 64, 8 for
 *               C <= 128 and 4 beyond (the rows one partial sum covers).
 *   n_classes   1 .. 65536.
 *   logits, dlogits  device [n_rows, n_classes];  labels device int32
 *               [n_rows];  loss device, 1 float.  Results as for
 *               digest_softmax_xent (a label outside [0, n_classes) gives
 *               that row zero dlogits and the loss NaN).
 *   hip_stream  a stream of the current device (NULL: its default stream).
 * Errors: DIGEST_EINVAL (sizes, NULL, n_rows above the limit, a stream of
 * another device), DIGEST_EHIP.
 */
#define DIGEST_STATIC_SCRATCH_FLOATS 262144
digest_status digest_softmax_xent_static(int64_t n_rows, int32_t n_classes,
                                         const float *logits, const int32_t *labels,
                                         float *dlogits, float *loss, void *hip_stream);

/*
 * Global parameter update of Algorithm 1 (AGG): each of the M subgraphs
 * took one local SGD step from the same global parameters, W_m = W -
 * lr * grad_m, and the new global parameters are their average (the
 * convergence analysis of Appendix A.3 averages the local gradients):
 *   w[e] <- w[e] - lr * (1/M) * sum_{m < M} grads[m][e]   for e < count,
 * the sum taken in m order (deterministic).
 *   w      device, count floats (updated in place).
 *   grads  HOST array of M device pointers, each to count floats (e.g. the
 *          dw of one subgraph's digest_layer_backward); not modified.
 *   n_grads M, 1 <= M <= 64.   count >= 0.
 * Not tied to a partition handle; enqueued on hip_stream.
 * Errors: DIGEST_EINVAL (M out of range, negative count, NULL), DIGEST_EHIP.
 */
digest_status digest_sgd_average(float *w, const float *const *grads, int32_t n_grads,
                                 int64_t count, float lr, void *hip_stream);

/*
 * Synchronisation schedule of Algorithm 1 (pure, host only): in round
 * iter (1-based) with interval K >= 1, *do_pull = (iter mod K == 0) and
 * *do_push = ((iter-1) mod K == 0); both apply to levels 1..L-1.
 * Errors: DIGEST_EINVAL (K < 1, iter < 1, NULL).
 */
digest_status digest_sync_period(int32_t K, int64_t iter, int32_t *do_pull,
                                 int32_t *do_push);

/*
 * Instrumentation: while enabled, every kernel the handle launches is
 * bracketed by HIP events on its own stream.  digest_profile_read
 * synchronises on those events and returns the summed duration (ms) and
 * launch count of each (kernel kind, layer) since the last read, then
 * clears them.  Both arrays hold digest_profile_kernel_count() * (L + 1)
 * entries; entry kind * (L + 1) + slot, where slot is the layer (1..L) for
 * the layer kernels, the level (0..L-1) for pull and push, and L for the
 * loss head.  Kernel kinds are numbered 0..digest_profile_kernel_count()-1.
 */
digest_status digest_profile_enable(digest_partition *p, int32_t on);
digest_status digest_profile_read(digest_partition *p, double *total_ms, int64_t *launches);
int32_t digest_profile_kernel_count(void);
const char *digest_profile_kernel_name(int32_t kind);

/*
 * Launch plan of one layer as the library runs it (host only; a pure
 * function of the partition's sizes and widths), for tests and measurement.
 * The two products of Eq. 5 associate either way; the plan records which
 * order and which kernels the layer calls use.
 *   transform_first     1: an identity layer runs as P_m ([h_in; halo] W)
 *                       (forward) with G = P_m^T D over every local row
 *                       (backward); 0: (P_m [h_in; halo]) W with AH kept.
 *   forward_narrow      1: the product with W runs on the narrow-output
 *                       kernel (W held in LDS); 0: the MFMA GEMM, or the
 *                       fused pass when forward_fused is 1.
 *   dw_slices           split-K slices of the weight gradient, summed in
 *                       slice order (1: no split).
 *   dgrad_narrow_first  aggregate-first layers: 1 if the input gradient is
 *                       (P_in^T D) W^T (aggregated at width d_layer), 0 if
 *                       P_in^T (D W^T).
 *   dgrad_fused         transform-first layers: 1 if dh_in = G_own W^T is
 *                       formed in the epilogue of the transposed
 *                       aggregation (when the caller asks for dh_in).
 *   tiers_fwd, tiers_bwd  sliced passes of the forward aggregation (P_m)
 *                       and of the transposed one (P_in^T) of this layer,
 *                       which run before one pass over the remaining
 *                       entries (0: a single pass).  The source rows are
 *                       ranked by how many entries read them; tier t takes
 *                       the entries that read the rows ranked
 *                       [t R, (t+1) R), R = tier_rows_fwd / _bwd, and its
 *                       pass gathers 32-float column slices of them, each
 *                       slice on one XCD, so that one XCD's slices of the R
 *                       rows stay in its L2.  Each pass adds into the
 *                       output in tier order (a fixed summation order).
 *                       Planned at create, and only when the environment
 *                       variable DIGEST_SPMM_TIER_BYTES gives a per-XCD L2
 *                       budget (unset or 0, the default: no tiers, which
 *                       measured fastest on the workloads at hand); then a
 *                       cost model picks the tier count, or
 *                       DIGEST_SPMM_TIERS forces one.
 *   tier_entries_fwd, tier_entries_bwd  entries the sliced passes take.
 *   forward_fused       aggregate-first layers with at least 16,384 owned
 *                       rows, 65 <= d_layer-1 <= 256 and the MFMA GEMM as
 *                       their product: 1 if the forward runs as one pass
 *                       (kernel
 *                       kind "spmm_gemm_fwd") in which each tile of 32 rows
 *                       is aggregated into LDS and multiplied by W there,
 *                       the tiles of other workgroups gathering meanwhile;
 *                       rows of more than 64 entries are aggregated first
 *                       by a long-row pass ("spmm_fwd").  AH is still
 *                       stored for the backward.  The environment variable
 *                       DIGEST_FUSE=0 turns this off, =2 fuses at any row
 *                       count; the forward also falls back to two passes
 *                       when h_in (d_layer-1 a multiple of 4) is not
 *                       16-byte aligned.
 *   backward_fused      ReLU aggregate-first layers 2..L-1 with at least
 *                       16,384 owned rows and 65 <= d_layer <= 256, when
 *                       dh_in is asked for (and no halo gradient): 1 if the
 *                       input gradient runs as (P_in^T D) W^T in one pass
 *                       ("spmm_gemm_bwd"), D = dh_out masked by h_out > 0
 *                       formed once ("relu_mask", also the weight
 *                       gradient's operand), W^T formed once
 *                       ("transpose_w"), rows of P_in^T with more than 64
 *                       entries aggregated first ("spmm_bwd_transposed").
 *                       The same DIGEST_FUSE switch.
 * Errors: DIGEST_EINVAL (NULL, layer outside 1..L).
 */
typedef struct {
    int32_t transform_first;
    int32_t forward_narrow;
    int32_t dw_slices;
    int32_t dgrad_narrow_first;
    int32_t dgrad_fused;
    int32_t tiers_fwd;
    int32_t tiers_bwd;
    int32_t tier_rows_fwd;
    int32_t tier_rows_bwd;
    int64_t tier_entries_fwd;
    int64_t tier_entries_bwd;
    int32_t forward_fused;
    int32_t backward_fused;
} digest_layer_plan;

digest_status digest_partition_plan(const digest_partition *p, int32_t layer,
                                    digest_layer_plan *out);

/*
 * Algorithmic cost of one launch of each instrumented (kernel kind, slot),
 * indexed like digest_profile_read, for the launches that one round of the
 * GCN layers (model DIGEST_MODEL_GCN: every forward with act ReLU below
 * layer L and identity at L, the loss head, every backward with dh_in for
 * layers >= 2, the pulls of levels 0..L-1 and pushes of levels 1..L-1) or
 * of the GAT layers (DIGEST_MODEL_GAT) makes under the plan above:
 *   bytes    the bytes that must move if every operand is read once and
 *            every output written once (the compulsory traffic: a source
 *            row of an aggregation counts once however many entries read it);
 *   flops    floating-point operations of the dense products (0 otherwise);
 *   entries  entries of the sparse operand of an aggregation (0 otherwise).
 * Each array holds digest_profile_kernel_count() * (L + 1) entries; kinds
 * the round does not launch are 0.
 * Errors: DIGEST_EINVAL (NULL, unknown model).
 */
enum { DIGEST_MODEL_GCN = 0, DIGEST_MODEL_GAT = 1 };
digest_status digest_profile_model(const digest_partition *p, int32_t model, double *bytes,
                                   double *flops, int64_t *entries);

#ifdef __cplusplus
}
#endif

#endif /* DIGEST_H */
