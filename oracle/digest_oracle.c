/*
 * DIGEST per-partition GCN layer: CPU ORACLE.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may call, link or
 * load this file; only the tests, the package smoke check and the CPU leg of
 * the benchmark do.  It shares no code, header or constant with the HIP
 * library: index maps, aggregation, transform, loss and backward are all
 * written out again here, plainly, in double precision.
 *
 * What it computes (paper: "Distributed Graph Neural Network Training with
 * Periodic Stale Representation Synchronization", arXiv 2206.00057):
 *
 *   - partition maps: the split of a node's neighbours into in-subgraph and
 *     out-of-subgraph sets (Sec. 2, Eq. 2), the halo set of a subgraph
 *     (Sec. 3.2, definition of the pulled set) and the owned rows that other
 *     subgraphs read (the push of Sec. 3.2);
 *   - pull / push of stale representations (Sec. 3.2);
 *   - the DIGEST GCN layer H' = sigma(P_in H_in W + P_out H~_out W)
 *     (Sec. 3.1, Eq. 5 and Eq. 4), aggregation first, then the dense
 *     transform;
 *   - the mean softmax cross-entropy local loss of Eq. 3;
 *   - the layer backward by the chain rule (Sec. 3.1 Eq. 6 and the GCN
 *     backward of Appendix A.3), with the stale halo rows held constant;
 *   - the synchronisation schedule of Algorithm 1 (pull when r mod N == 0,
 *     push when (r-1) mod N == 0, for layers other than the last);
 *   - the halo gradient P_out^T D W^T, the stale-gradient term of the DIGEST
 *     backward in Appendix A.3 (what a subgraph's rows contribute to the
 *     gradient of its halo nodes' representations);
 *   - the global parameter update of Algorithm 1 (AGG of the M locally
 *     updated models; each took one SGD step from the same global W, so
 *     the average is W minus the learning rate times the mean gradient,
 *     as the convergence proof of Appendix A.3 averages local gradients).
 *
 * Precision: every sum is accumulated in double; a value is rounded to float
 * only where a tensor is written out (AH, H_out, dW, dH_in, dlogits).
 * OpenMP splits independent output rows (or independent feature columns)
 * across threads; it never changes the order of any single sum.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* Activation codes understood by the oracle. */
#define ORACLE_RELU 0
#define ORACLE_IDENTITY 1

int oracle_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Thread count of the OpenMP loops from here on (n >= 1); returns the new
   count.  Host plumbing for timing the oracle single-threaded. */
int oracle_set_num_threads(int n)
{
#ifdef _OPENMP
    if (n >= 1)
        omp_set_num_threads(n);
    return omp_get_max_threads();
#else
    (void)n;
    return 1;
#endif
}

/* ------------------------------------------------------------------------ */
/* Partition maps (Eq. 2; halo set and push set of Sec. 3.2)                */
/* ------------------------------------------------------------------------ */

/*
 * Local numbering: owned node owned[i] -> i; halo node halo[j] -> n_own + j.
 * col_local[k] is the local number of the k-th CSR column (CSR order kept).
 * boundary_local lists, ascending, the owned rows that have at least one
 * out-of-partition (halo) column: the rows another subgraph pulls.
 *
 * Returns 0, or -1 when an id is out of range, an id repeats, owned and halo
 * overlap, a column is neither owned nor halo, or indptr is malformed.
 */
int oracle_partition_maps(int64_t n_global, const int64_t *indptr,
                          const int64_t *indices, int64_t n_own,
                          const int64_t *owned, int64_t n_halo,
                          const int64_t *halo, int32_t *col_local,
                          int32_t *boundary_local, int64_t *n_boundary)
{
    int64_t *where = (int64_t *)malloc(sizeof(int64_t) * (size_t)(n_global > 0 ? n_global : 1));
    if (!where)
        return -1;
    for (int64_t v = 0; v < n_global; ++v)
        where[v] = -1;
    int bad = 0;
    for (int64_t i = 0; i < n_own && !bad; ++i) {
        int64_t g = owned[i];
        if (g < 0 || g >= n_global || where[g] != -1)
            bad = 1;
        else
            where[g] = i;
    }
    for (int64_t j = 0; j < n_halo && !bad; ++j) {
        int64_t g = halo[j];
        if (g < 0 || g >= n_global || where[g] != -1)
            bad = 1;
        else
            where[g] = n_own + j;
    }
    if (!bad && indptr[0] != 0)
        bad = 1;
    for (int64_t i = 0; i < n_own && !bad; ++i)
        if (indptr[i + 1] < indptr[i])
            bad = 1;
    int64_t nb = 0;
    for (int64_t i = 0; i < n_own && !bad; ++i) {
        int reads_halo = 0;
        for (int64_t k = indptr[i]; k < indptr[i + 1]; ++k) {
            int64_t g = indices[k];
            if (g < 0 || g >= n_global || where[g] < 0) {
                bad = 1;
                break;
            }
            col_local[k] = (int32_t)where[g];
            if (where[g] >= n_own)
                reads_halo = 1;
        }
        if (reads_halo)
            boundary_local[nb++] = (int32_t)i;
    }
    free(where);
    if (bad)
        return -1;
    *n_boundary = nb;
    return 0;
}

/*
 * Transpose of the owned-by-owned block P_in (the part of the local CSR
 * whose columns are owned).  Row c of the result lists the pairs (i, a_ic)
 * with a_ic an entry of row i in column c, ordered by i ascending and, for
 * repeated (i, c), in the input CSR order.  Returns nnz of the block.
 */
int64_t oracle_owned_transpose(int64_t n_own, const int64_t *indptr,
                               const int32_t *col_local, const float *values,
                               int64_t *t_indptr, int32_t *t_src,
                               float *t_vals)
{
    for (int64_t c = 0; c <= n_own; ++c)
        t_indptr[c] = 0;
    for (int64_t i = 0; i < n_own; ++i)
        for (int64_t k = indptr[i]; k < indptr[i + 1]; ++k)
            if (col_local[k] < n_own)
                t_indptr[col_local[k] + 1] += 1;
    for (int64_t c = 0; c < n_own; ++c)
        t_indptr[c + 1] += t_indptr[c];
    int64_t *fill = (int64_t *)malloc(sizeof(int64_t) * (size_t)(n_own > 0 ? n_own : 1));
    for (int64_t c = 0; c < n_own; ++c)
        fill[c] = t_indptr[c];
    for (int64_t i = 0; i < n_own; ++i)
        for (int64_t k = indptr[i]; k < indptr[i + 1]; ++k) {
            int32_t c = col_local[k];
            if (c < n_own) {
                t_src[fill[c]] = (int32_t)i;
                t_vals[fill[c]] = values[k];
                fill[c] += 1;
            }
        }
    free(fill);
    return t_indptr[n_own];
}

/* ------------------------------------------------------------------------ */
/* Pull and push (Sec. 3.2)                                                 */
/* ------------------------------------------------------------------------ */

/* Pull: the halo buffer row j becomes the stored (stale) row of halo[j]. */
void oracle_pull(const float *store, int64_t d, int64_t n_halo,
                 const int64_t *halo, float *halo_buf)
{
    for (int64_t j = 0; j < n_halo; ++j)
        memcpy(halo_buf + j * d, store + halo[j] * d, sizeof(float) * (size_t)d);
}

/* Push: for each listed owned row, the store row of its node is overwritten
 * by the freshly computed representation.  Other store rows are untouched. */
void oracle_push(const float *h_own, int64_t d, const int64_t *owned,
                 int64_t n_rows, const int32_t *rows, float *store)
{
    for (int64_t b = 0; b < n_rows; ++b)
        memcpy(store + owned[rows[b]] * d, h_own + (int64_t)rows[b] * d,
               sizeof(float) * (size_t)d);
}

/* ------------------------------------------------------------------------ */
/* Forward (Eq. 5)                                                          */
/* ------------------------------------------------------------------------ */

/*
 * Aggregation: AH = P_in H_in + P_out H~_out, i.e. for owned row i the sum
 * over its CSR entries (a, c) of a * src(c), where src(c) is the fresh owned
 * row c (c < n_own) or the pulled stale halo row c - n_own.
 */
void oracle_aggregate(int64_t n_own, const int64_t *indptr,
                      const int32_t *col_local, const float *values,
                      const float *h_own, const float *halo_buf, int64_t d,
                      float *ah)
{
#pragma omp parallel
    {
        double *acc = (double *)malloc(sizeof(double) * (size_t)(d > 0 ? d : 1));
#pragma omp for schedule(dynamic, 64)
        for (int64_t i = 0; i < n_own; ++i) {
            for (int64_t f = 0; f < d; ++f)
                acc[f] = 0.0;
            for (int64_t k = indptr[i]; k < indptr[i + 1]; ++k) {
                int64_t c = col_local[k];
                const float *src = c < n_own ? h_own + c * d
                                             : halo_buf + (c - n_own) * d;
                double a = (double)values[k];
                for (int64_t f = 0; f < d; ++f)
                    acc[f] += a * (double)src[f];
            }
            for (int64_t f = 0; f < d; ++f)
                ah[i * d + f] = (float)acc[f];
        }
        free(acc);
    }
}

/* Transform and activation: H_out = sigma(AH W); sigma is ReLU or identity. */
void oracle_transform(int64_t n, int64_t d_in, int64_t d_out, const float *ah,
                      const float *w, int act, float *h_out)
{
#pragma omp parallel
    {
        double *z = (double *)malloc(sizeof(double) * (size_t)(d_out > 0 ? d_out : 1));
#pragma omp for schedule(static)
        for (int64_t i = 0; i < n; ++i) {
            for (int64_t o = 0; o < d_out; ++o)
                z[o] = 0.0;
            for (int64_t f = 0; f < d_in; ++f) {
                double a = (double)ah[i * d_in + f];
                const float *wrow = w + f * d_out;
                for (int64_t o = 0; o < d_out; ++o)
                    z[o] += a * (double)wrow[o];
            }
            for (int64_t o = 0; o < d_out; ++o) {
                double v = z[o];
                if (act == ORACLE_RELU && !(v > 0.0))
                    v = 0.0;
                h_out[i * d_out + o] = (float)v;
            }
        }
        free(z);
    }
}

/* ------------------------------------------------------------------------ */
/* Local loss (Eq. 3): mean softmax cross-entropy over the owned rows       */
/* ------------------------------------------------------------------------ */

/*
 * loss = -(1/n) sum_i log softmax(z_i)[y_i];  dlogits = (softmax(z) - onehot(y)) / n.
 * Returns 0, or -1 if a label is outside [0, C).
 */
int oracle_softmax_xent(int64_t n, int64_t C, const float *logits,
                        const int32_t *labels, float *dlogits, double *loss)
{
    for (int64_t i = 0; i < n; ++i)
        if (labels[i] < 0 || labels[i] >= C)
            return -1;
    double total = 0.0;
    for (int64_t i = 0; i < n; ++i) {
        const float *z = logits + i * C;
        double zmax = (double)z[0];
        for (int64_t c = 1; c < C; ++c)
            if ((double)z[c] > zmax)
                zmax = (double)z[c];
        double s = 0.0;
        for (int64_t c = 0; c < C; ++c)
            s += exp((double)z[c] - zmax);
        double log_s = log(s);
        total += -((double)z[labels[i]] - zmax - log_s);
        for (int64_t c = 0; c < C; ++c) {
            double p = exp((double)z[c] - zmax - log_s);
            double g = p - (c == labels[i] ? 1.0 : 0.0);
            dlogits[i * C + c] = (float)(g / (double)n);
        }
    }
    *loss = n > 0 ? total / (double)n : 0.0;
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Backward (Eq. 6 and the GCN backward of Appendix A.3)                    */
/* ------------------------------------------------------------------------ */

/*
 * Given the upstream gradient dH_out of this layer's output:
 *   D     = dH_out * sigma'(Z)          (sigma'(z) = 1[z > 0] for ReLU, read off
 *                                        H_out > 0; identity: D = dH_out)
 *   dW    = (AH)^T D                    with AH = P_in H_in + P_out H~_out
 *   dH_in = P_in^T (D W^T)              stale halo rows are constants: they
 *                                        receive no gradient
 * AH is recomputed here from (h_own, halo_buf) exactly as the forward did.
 * dh_in may be NULL (first layer: the features need no gradient).
 */
void oracle_layer_backward(int64_t n_own, const int64_t *indptr,
                           const int32_t *col_local, const float *values,
                           const float *h_own, const float *halo_buf,
                           int64_t d_in, int64_t d_out, const float *w,
                           const float *h_out, const float *dh_out, int act,
                           float *dw, float *dh_in)
{
    float *ah = (float *)malloc(sizeof(float) * (size_t)(n_own * d_in > 0 ? n_own * d_in : 1));
    oracle_aggregate(n_own, indptr, col_local, values, h_own, halo_buf, d_in, ah);

    double *dz = (double *)malloc(sizeof(double) * (size_t)(n_own * d_out > 0 ? n_own * d_out : 1));
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n_own; ++i)
        for (int64_t o = 0; o < d_out; ++o) {
            int64_t e = i * d_out + o;
            double g = (double)dh_out[e];
            if (act == ORACLE_RELU && !(h_out[e] > 0.0f))
                g = 0.0;
            dz[e] = g;
        }

    /* dW[f][o] = sum over owned rows i of AH[i][f] * D[i][o]. */
#pragma omp parallel
    {
        double *acc = (double *)malloc(sizeof(double) * (size_t)(d_out > 0 ? d_out : 1));
#pragma omp for schedule(static)
        for (int64_t f = 0; f < d_in; ++f) {
            for (int64_t o = 0; o < d_out; ++o)
                acc[o] = 0.0;
            for (int64_t i = 0; i < n_own; ++i) {
                double a = (double)ah[i * d_in + f];
                const double *drow = dz + i * d_out;
                for (int64_t o = 0; o < d_out; ++o)
                    acc[o] += a * drow[o];
            }
            for (int64_t o = 0; o < d_out; ++o)
                dw[f * d_out + o] = (float)acc[o];
        }
        free(acc);
    }

    if (dh_in) {
        /* G = D W^T, kept in double. */
        double *g = (double *)malloc(sizeof(double) * (size_t)(n_own * d_in > 0 ? n_own * d_in : 1));
#pragma omp parallel for schedule(static)
        for (int64_t i = 0; i < n_own; ++i)
            for (int64_t f = 0; f < d_in; ++f) {
                double s = 0.0;
                for (int64_t o = 0; o < d_out; ++o)
                    s += dz[i * d_out + o] * (double)w[f * d_out + o];
                g[i * d_in + f] = s;
            }
        /* dH_in[c] = sum over entries (i, c) of P_in of a_ic * G[i]:
         * a scatter along the rows of P_in; threads own disjoint feature
         * columns, so each sum still runs over i in ascending order. */
        double *acc = (double *)calloc((size_t)(n_own * d_in > 0 ? n_own * d_in : 1), sizeof(double));
#pragma omp parallel
        {
#ifdef _OPENMP
            int nt = omp_get_num_threads(), t = omp_get_thread_num();
#else
            int nt = 1, t = 0;
#endif
            int64_t f0 = d_in * t / nt, f1 = d_in * (t + 1) / nt;
            for (int64_t i = 0; i < n_own; ++i)
                for (int64_t k = indptr[i]; k < indptr[i + 1]; ++k) {
                    int64_t c = col_local[k];
                    if (c >= n_own)
                        continue; /* halo column: constant, no gradient */
                    double a = (double)values[k];
                    for (int64_t f = f0; f < f1; ++f)
                        acc[c * d_in + f] += a * g[i * d_in + f];
                }
        }
        for (int64_t e = 0; e < n_own * d_in; ++e)
            dh_in[e] = (float)acc[e];
        free(acc);
        free(g);
    }
    free(dz);
    free(ah);
}

/* ------------------------------------------------------------------------ */
/* GAT layer with stale halo rows: the stale-representation layer of Eq. 4  */
/* with an attention aggregation (the GAT model of the experiments,         */
/* single head; formulas from the GAT model the paper cites)                */
/* ------------------------------------------------------------------------ */

/* z_v = x_v W for every local row v (owned rows from h_own, halo rows from
   the stale halo buffer), in double: [(n_own + n_halo) x d_out]. */
static double *gat_transform(int64_t n_own, int64_t n_halo, const float *h_own,
                             const float *halo_buf, int64_t d_in, int64_t d_out,
                             const float *w)
{
    int64_t R = n_own + n_halo;
    double *z = (double *)malloc(sizeof(double) * (size_t)(R * d_out > 0 ? R * d_out : 1));
#pragma omp parallel for schedule(static)
    for (int64_t v = 0; v < R; ++v) {
        const float *x = v < n_own ? h_own + v * d_in : halo_buf + (v - n_own) * d_in;
        double *zv = z + v * d_out;
        for (int64_t o = 0; o < d_out; ++o)
            zv[o] = 0.0;
        /* every z_v[o] sums over f in ascending order */
        for (int64_t f = 0; f < d_in; ++f) {
            double xf = (double)x[f];
            const float *wf = w + f * d_out;
            for (int64_t o = 0; o < d_out; ++o)
                zv[o] += xf * (double)wf[o];
        }
    }
    return z;
}

/* Source scores s_v = z_v . att[:,0] (every local row) and target scores
   t_i = z_i . att[:,1] (owned rows); att is [d_out][2] row-major. */
static void gat_scores(int64_t n_own, int64_t R, int64_t d_out, const double *z,
                       const float *att, double *s, double *t)
{
    for (int64_t v = 0; v < R; ++v) {
        double a = 0.0, b = 0.0;
        for (int64_t o = 0; o < d_out; ++o) {
            a += z[v * d_out + o] * (double)att[2 * o];
            b += z[v * d_out + o] * (double)att[2 * o + 1];
        }
        s[v] = a;
        if (v < n_own)
            t[v] = b;
    }
}

static double leaky(double x, double slope) { return x > 0.0 ? x : slope * x; }

/* Attention weights of row i: alpha_k = softmax over the row's entries of
   LeakyReLU(t_i + s_{col_k}); written to a[k - indptr[i]]. */
static void gat_row_alpha(int64_t i, const int64_t *indptr, const int32_t *col_local,
                          const double *s, const double *t, double slope, double *a)
{
    int64_t kb = indptr[i], ke = indptr[i + 1];
    double m = -INFINITY;
    for (int64_t k = kb; k < ke; ++k) {
        double e = leaky(t[i] + s[col_local[k]], slope);
        a[k - kb] = e;
        if (e > m)
            m = e;
    }
    double sum = 0.0;
    for (int64_t k = kb; k < ke; ++k) {
        a[k - kb] = exp(a[k - kb] - m);
        sum += a[k - kb];
    }
    for (int64_t k = kb; k < ke; ++k)
        a[k - kb] /= sum;
}

/*
 * GAT forward on one partition:
 *   z_v      = x_v W                              every local row
 *   e_ik     = LeakyReLU(t_i + s_{col_k})         entries k of owned row i
 *   alpha_ik = softmax over row i of e_ik
 *   h_out_i  = act(sum_k alpha_ik z_{col_k})      (an empty row gives act(0))
 * Optional alpha output: the weights in CSR entry order [nnz].
 */
void oracle_gat_forward(int64_t n_own, int64_t n_halo, const int64_t *indptr,
                        const int32_t *col_local, const float *h_own, const float *halo_buf,
                        int64_t d_in, int64_t d_out, const float *w, const float *att,
                        double slope, int act, float *h_out, float *alpha)
{
    int64_t R = n_own + n_halo;
    double *z = gat_transform(n_own, n_halo, h_own, halo_buf, d_in, d_out, w);
    double *s = (double *)malloc(sizeof(double) * (size_t)(R > 0 ? R : 1));
    double *t = (double *)malloc(sizeof(double) * (size_t)(n_own > 0 ? n_own : 1));
    gat_scores(n_own, R, d_out, z, att, s, t);
#pragma omp parallel
    {
        int64_t maxrow = 1;
        for (int64_t i = 0; i < n_own; ++i)
            if (indptr[i + 1] - indptr[i] > maxrow)
                maxrow = indptr[i + 1] - indptr[i];
        double *a = (double *)malloc(sizeof(double) * (size_t)maxrow);
        double *o = (double *)malloc(sizeof(double) * (size_t)(d_out > 0 ? d_out : 1));
#pragma omp for schedule(static)
        for (int64_t i = 0; i < n_own; ++i) {
            gat_row_alpha(i, indptr, col_local, s, t, slope, a);
            for (int64_t q = 0; q < d_out; ++q)
                o[q] = 0.0;
            for (int64_t k = indptr[i]; k < indptr[i + 1]; ++k) {
                const double *zc = z + (int64_t)col_local[k] * d_out;
                for (int64_t q = 0; q < d_out; ++q)
                    o[q] += a[k - indptr[i]] * zc[q];
                if (alpha)
                    alpha[k] = (float)a[k - indptr[i]];
            }
            for (int64_t q = 0; q < d_out; ++q) {
                double v = o[q];
                if (act == ORACLE_RELU && v < 0.0)
                    v = 0.0;
                h_out[i * d_out + q] = (float)v;
            }
        }
        free(o);
        free(a);
    }
    free(t);
    free(s);
    free(z);
}

/*
 * GAT backward on one partition, by the chain rule through the forward
 * above (halo rows are constants: they get no gradient, but their z rows
 * depend on W, so they contribute to dW and to the attention gradient):
 *   D_i     = dh_out_i * act'(h_out_i)        (mask h_out > 0 for ReLU)
 *   c_i     = D_i . o_i,  o_i = sum_k alpha_ik z_{col_k}
 *   dpre_ik = alpha_ik (D_i . z_{col_k} - c_i) * LeakyReLU'(t_i + s_{col_k})
 *   dz_v    = sum over entries (i,k) with col_k = v of
 *               (alpha_ik D_i + dpre_ik att[:,0])
 *             + (v owned) (sum_k dpre_vk) att[:,1]
 *   datt[:,0] = sum_v (sum over entries reading v of dpre) z_v
 *   datt[:,1] = sum_i (sum_k dpre_ik) z_i
 *   dW = sum over local rows v of x_v^T dz_v;  dh_in_i = dz_i W^T (owned i)
 * att and datt are [d_out][2]; dh_in may be NULL.
 *
 * Every sum has one fixed order, whatever the thread count: the entries
 * that feed a column in ascending (row, entry) order, rows and columns in
 * ascending order.  Threads split independent rows (first pass), columns
 * (the scatter: each thread scans every entry and applies those whose
 * column it owns) and feature blocks of dW.
 */
void oracle_gat_backward(int64_t n_own, int64_t n_halo, const int64_t *indptr,
                         const int32_t *col_local, const float *h_own, const float *halo_buf,
                         int64_t d_in, int64_t d_out, const float *w, const float *att,
                         double slope, int act, const float *h_out, const float *dh_out,
                         float *dw, float *datt, float *dh_in)
{
    int64_t R = n_own + n_halo;
    int64_t nnz = n_own > 0 ? indptr[n_own] - indptr[0] : 0;
    int64_t e0 = n_own > 0 ? indptr[0] : 0;
    size_t one = 1;
    double *z = gat_transform(n_own, n_halo, h_own, halo_buf, d_in, d_out, w);
    double *s = (double *)malloc(sizeof(double) * (size_t)(R > 0 ? R : 1));
    double *t = (double *)malloc(sizeof(double) * (size_t)(n_own > 0 ? n_own : 1));
    gat_scores(n_own, R, d_out, z, att, s, t);
    double *D = (double *)malloc(sizeof(double) * (size_t)(n_own * d_out > 0 ? n_own * d_out : 1));
    double *alpha = (double *)malloc(sizeof(double) * (nnz > 0 ? (size_t)nnz : one));
    double *dpre = (double *)malloc(sizeof(double) * (nnz > 0 ? (size_t)nnz : one));
    double *rsum = (double *)malloc(sizeof(double) * (size_t)(n_own > 0 ? n_own : 1));

    /* First pass, owned rows independently: D_i, the row's weights, o_i,
       c_i and every dpre_ik, and their sum over the row. */
#pragma omp parallel
    {
        double *o = (double *)malloc(sizeof(double) * (size_t)(d_out > 0 ? d_out : 1));
#pragma omp for schedule(static)
        for (int64_t i = 0; i < n_own; ++i) {
            int64_t kb = indptr[i], ke = indptr[i + 1];
            double *a = alpha + (kb - e0);
            double *Di = D + i * d_out;
            gat_row_alpha(i, indptr, col_local, s, t, slope, a);
            for (int64_t q = 0; q < d_out; ++q) {
                double g = (double)dh_out[i * d_out + q];
                if (act == ORACLE_RELU && !(h_out[i * d_out + q] > 0.0f))
                    g = 0.0;
                Di[q] = g;
                o[q] = 0.0;
            }
            for (int64_t k = kb; k < ke; ++k) {
                const double *zc = z + (int64_t)col_local[k] * d_out;
                for (int64_t q = 0; q < d_out; ++q)
                    o[q] += a[k - kb] * zc[q];
            }
            double c = 0.0;
            for (int64_t q = 0; q < d_out; ++q)
                c += Di[q] * o[q];
            double rs = 0.0;
            for (int64_t k = kb; k < ke; ++k) {
                int64_t col = col_local[k];
                const double *zc = z + col * d_out;
                double dalpha = 0.0;
                for (int64_t q = 0; q < d_out; ++q)
                    dalpha += Di[q] * zc[q];
                double pre = t[i] + s[col];
                double dp = a[k - kb] * (dalpha - c) * (pre > 0.0 ? 1.0 : slope);
                dpre[k - e0] = dp;
                rs += dp;
            }
            rsum[i] = rs;
        }
        free(o);
    }

    /* Scatter into the columns: the thread that owns a column (blocks of
       64 columns dealt round robin) applies its entries in (row, entry)
       order. */
    double *dz = (double *)calloc((size_t)(R * d_out > 0 ? R * d_out : 1), sizeof(double));
    double *csum = (double *)calloc((size_t)(R > 0 ? R : 1), sizeof(double));
#pragma omp parallel
    {
        int64_t nt = 1, me = 0;
#ifdef _OPENMP
        nt = omp_get_num_threads();
        me = omp_get_thread_num();
#endif
        for (int64_t i = 0; i < n_own; ++i) {
            const double *Di = D + i * d_out;
            for (int64_t k = indptr[i]; k < indptr[i + 1]; ++k) {
                int64_t col = col_local[k];
                if ((col / 64) % nt != me)
                    continue;
                double a = alpha[k - e0], dp = dpre[k - e0];
                double *dzc = dz + col * d_out;
                for (int64_t q = 0; q < d_out; ++q)
                    dzc[q] += a * Di[q] + dp * (double)att[2 * q];
                csum[col] += dp;
            }
        }
    }
    for (int64_t i = 0; i < n_own; ++i)
        for (int64_t q = 0; q < d_out; ++q)
            dz[i * d_out + q] += rsum[i] * (double)att[2 * q + 1];

    double *da = (double *)calloc((size_t)(2 * d_out > 0 ? 2 * d_out : 1), sizeof(double));
    for (int64_t v = 0; v < R; ++v)
        for (int64_t q = 0; q < d_out; ++q) {
            da[2 * q] += csum[v] * z[v * d_out + q];
            if (v < n_own)
                da[2 * q + 1] += rsum[v] * z[v * d_out + q];
        }
    for (int64_t e = 0; e < 2 * d_out; ++e)
        datt[e] = (float)da[e];

    /* dW[f][q] = sum over local rows v (ascending) of x_v[f] dz_v[q], a block
       of features per task so that dz streams once per block. */
    {
        int64_t nt = 1;
#ifdef _OPENMP
        nt = omp_get_max_threads();
#endif
        int64_t fb = d_in / (2 * nt);
        fb = fb < 1 ? 1 : (fb > 16 ? 16 : fb);
        int64_t nblk = (d_in + fb - 1) / fb;
#pragma omp parallel
        {
            double *acc = (double *)malloc(sizeof(double) * (size_t)(fb * d_out > 0 ? fb * d_out : 1));
#pragma omp for schedule(dynamic, 1)
            for (int64_t b = 0; b < nblk; ++b) {
                int64_t f0 = b * fb, fn = d_in - f0 < fb ? d_in - f0 : fb;
                for (int64_t e = 0; e < fn * d_out; ++e)
                    acc[e] = 0.0;
                for (int64_t v = 0; v < R; ++v) {
                    const float *x = v < n_own ? h_own + v * d_in : halo_buf + (v - n_own) * d_in;
                    const double *dzv = dz + v * d_out;
                    for (int64_t j = 0; j < fn; ++j) {
                        double xf = (double)x[f0 + j];
                        double *aj = acc + j * d_out;
                        for (int64_t q = 0; q < d_out; ++q)
                            aj[q] += xf * dzv[q];
                    }
                }
                for (int64_t j = 0; j < fn; ++j)
                    for (int64_t q = 0; q < d_out; ++q)
                        dw[(f0 + j) * d_out + q] = (float)acc[j * d_out + q];
            }
            free(acc);
        }
    }
    if (dh_in) {
#pragma omp parallel for schedule(static)
        for (int64_t i = 0; i < n_own; ++i)
            for (int64_t f = 0; f < d_in; ++f) {
                double acc = 0.0;
                for (int64_t q = 0; q < d_out; ++q)
                    acc += dz[i * d_out + q] * (double)w[f * d_out + q];
                dh_in[i * d_in + f] = (float)acc;
            }
    }
    free(da);
    free(csum);
    free(dz);
    free(rsum);
    free(dpre);
    free(alpha);
    free(D);
    free(t);
    free(s);
    free(z);
}

/* ------------------------------------------------------------------------ */
/* Synchronisation schedule (Algorithm 1)                                   */
/* ------------------------------------------------------------------------ */

/* Round r (1-based), interval K: pull when r mod K == 0, push when
 * (r - 1) mod K == 0.  Returns -1 for K < 1 or r < 1. */
int oracle_sync_period(int32_t K, int64_t r, int32_t *do_pull, int32_t *do_push)
{
    if (K < 1 || r < 1)
        return -1;
    *do_pull = (r % K) == 0;
    *do_push = ((r - 1) % K) == 0;
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Global parameter update (Algorithm 1, AGG)                               */
/* ------------------------------------------------------------------------ */

/* w[e] <- w[e] - lr * (1/M) * sum_m grads[m][e] for e < count: the average of
 * the M local models W - lr * grad_m.  The sum runs over m in order, in
 * double.  Returns -1 for M < 1. */
int oracle_sgd_average(float *w, const float *const *grads, int32_t M, int64_t count, float lr)
{
    if (M < 1)
        return -1;
    for (int64_t e = 0; e < count; ++e) {
        double g = 0.0;
        for (int32_t m = 0; m < M; ++m)
            g += (double)grads[m][e];
        w[e] = (float)((double)w[e] - (double)lr * (g / (double)M));
    }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Halo gradient (Appendix A.3, the P_out^T term)                           */
/* ------------------------------------------------------------------------ */

/* dh_halo[j] = sum over entries (i, n_own + j) of P of a_ij * (D W^T)[i],
 * D = dh_out masked by h_out > 0 for ReLU; entries in CSR order, double. */
void oracle_halo_gradient(int64_t n_own, int64_t n_halo, const int64_t *indptr,
                          const int32_t *col_local, const float *values, int64_t d_in,
                          int64_t d_out, const float *w, const float *h_out,
                          const float *dh_out, int act, float *dh_halo)
{
    double *acc = (double *)calloc((size_t)(n_halo * d_in > 0 ? n_halo * d_in : 1), sizeof(double));
    double *G = (double *)malloc(sizeof(double) * (size_t)(n_own * d_in > 0 ? n_own * d_in : 1));
    /* G[i] = D[i] W^T, rows independent */
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n_own; ++i)
        for (int64_t f = 0; f < d_in; ++f) {
            double s = 0.0;
            for (int64_t o = 0; o < d_out; ++o) {
                double dz = (double)dh_out[i * d_out + o];
                if (act == ORACLE_RELU && !(h_out[i * d_out + o] > 0.0f))
                    dz = 0.0;
                s += dz * (double)w[f * d_out + o];
            }
            G[i * d_in + f] = s;
        }
    /* scatter into the halo rows, owned rows in ascending order */
    for (int64_t i = 0; i < n_own; ++i) {
        const double *g = G + i * d_in;
        for (int64_t k = indptr[i]; k < indptr[i + 1]; ++k) {
            int64_t c = col_local[k];
            if (c < n_own)
                continue; /* in-subgraph column: the ordinary backward */
            double a = (double)values[k];
            for (int64_t f = 0; f < d_in; ++f)
                acc[(c - n_own) * d_in + f] += a * g[f];
        }
    }
    for (int64_t e = 0; e < n_halo * d_in; ++e)
        dh_halo[e] = (float)acc[e];
    free(G);
    free(acc);
}

