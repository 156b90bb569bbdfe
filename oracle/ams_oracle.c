/*
 * ams_oracle.c -- float64 CPU oracle of one AMS image-embedding training step.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this library.  It shares no code,
 * header, table or helper with the HIP library it checks.
 *
 * It computes the plain definitions, slowly and in float64:
 *
 *   dedup      one sorted set of the batch's image IDs (behaviors and ads),
 *              with inverse index and stable occurrence order.  Requests for the
 *              same image are served once and their gradients are merged at the
 *              image's owner (section 4.2; Algorithm 1, SERVEREMBED and
 *              SERVERUPDATE).  Dedup is exact: embedding the unique set equals
 *              embedding every occurrence.
 *   mlp fwd    the trainable embedding model, a fully connected net with ReLU
 *              between layers (4096-256-64-12 in section 5.1; ReLU per the
 *              measured workloads, PReLU in section 7.2 is not used), applied to
 *              each unique image's feature row (the fixed VGG16 part is a
 *              precomputed input, sections 5.1 and 7.3).
 *   pool fwd   the behavior-image aggregators of section 5.2: sum, max, and
 *              attentive pooling with the ad image embedding as query,
 *              w = softmax_j(e_j . a), u = sum_j w_j e_j.
 *   pool bwd   the per-occurrence embedding gradients, then their sum per
 *              unique image in ascending occurrence order (Algorithm 1: the
 *              embedding gradients of one image are collected by its server).
 *   mlp bwd    delta_E = grad of E(I) times delta_e (Algorithm 1, SERVERUPDATE):
 *              weight and bias gradients summed over unique images in ascending
 *              order.  No gradient flows into the fixed feature table.
 *
 * For the joint step (the worker of Algorithm 1 next to the image path):
 *
 *   bag fwd    per sample and ID table, the sum of the table rows of its
 *              behaviors' IDs and of its ad's ID (the sparse ID features of
 *              section 3.2, embedded from key-value tables as in section 4.1,
 *              sum-pooled like the behavior images).
 *   ctr        the CTR MLP on [pooled user image vector, ad image embedding,
 *              one bag per table], ReLU between layers, softmax over the
 *              classes and cross-entropy with the click label (section 3.1),
 *              averaged over the batch; its backward gives the worker
 *              gradients and the gradients of every input field, among them
 *              delta_e for the image path (Algorithm 1, WORKERITERATION).
 *   adagrad    the sparse Adagrad step of the touched ID rows: accum += g^2,
 *              row -= lr g / (sqrt(accum) + eps), elementwise.
 * The merged gradient of an ID row is the SUM aggregator's backward with the
 * bag gradient as upstream (orc_pool_bwd, mode SUM).
 *
 *   adam       the dense update of the server's embedding model and the
 *              worker's CTR model (Algorithm 1: update E, update W; section
 *              7.2 trains with Adam): m = b1 m + (1-b1) g, v = b2 v + (1-b2) g^2,
 *              p -= lr (m / (1-b1^t)) / (sqrt(v / (1-b2^t)) + eps).
 *   query pool one channel of the multiple-query attentive pooling of section
 *              5.2: attention over the behavior image embeddings with a query
 *              given per sample (the ad's ID embedding for the ID channel),
 *              w = softmax_j(e_j . q_i), u_i = sum_j w_j e_j; its backward
 *              gives the behaviors' embedding gradients (merged per unique
 *              image) and the query gradient.
 *
 *   concat     the concatenate aggregator of section 5.2: a sample's behavior
 *              embeddings side by side, padded with zeros or truncated to a
 *              fixed count; its backward hands each kept position its slice
 *              of the upstream gradient, merged per unique image.
 *   dense      a fully connected net with PReLU (a learnable slope per
 *              channel, the activation of section 7.2) or ReLU between
 *              layers, forward and backward from the last layer's gradient,
 *              with the slopes' gradients.  With it the oracle's Python side
 *              composes the CTR model with PReLU and the pre-rank model of
 *              section 6: a user tower and an ad tower, the score their inner
 *              product, the logistic loss with the click label.
 *
 * Readings where the paper is silent (documented with the library): no
 * activation after the last layer unless final_relu is set; ReLU'(0) = 0;
 * the max-pool argmax is the first (lowest) position attaining the maximum;
 * an empty behavior segment pools to zero and gets no gradient; the ad
 * embedding receives the upstream gradient g_a plus the attention term.
 *
 * Inputs in bf16 are converted exactly to float64; no intermediate rounding of
 * the GPU path is emulated.  Every loop runs in a fixed order, so results do
 * not depend on the OpenMP thread count.
 *
 * Return codes: 0 ok, 1 bad argument, 2 image ID out of range.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_F32 0
#define ORC_BF16 1

#define POOL_SUM 0
#define POOL_MAX 1
#define POOL_ATT 2

static double load_elem(const void *p, int dtype, size_t i)
{
    if (dtype == ORC_F32)
        return (double)((const float *)p)[i];
    /* bf16: the upper 16 bits of an IEEE single */
    uint32_t bits = ((uint32_t)((const uint16_t *)p)[i]) << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
}

int orc_num_threads(void);
#ifdef _OPENMP
#include <omp.h>
int orc_num_threads(void) { return omp_get_max_threads(); }
void orc_set_threads(int n) { if (n > 0) omp_set_num_threads(n); }
#else
int orc_num_threads(void) { return 1; }
void orc_set_threads(int n) { (void)n; }
#endif

/* ------------------------------------------------------------------ dedup */

typedef struct { int32_t id; int32_t k; } occ_pair;

static int cmp_pair(const void *a, const void *b)
{
    const occ_pair *x = (const occ_pair *)a, *y = (const occ_pair *)b;
    if (x->id != y->id) return x->id < y->id ? -1 : 1;
    if (x->k != y->k) return x->k < y->k ? -1 : 1;
    return 0;
}

/* first index i in sorted uniq[0..n) with uniq[i] >= key */
static int32_t lower_bound_i32(const int32_t *uniq, int32_t n, int32_t key)
{
    int32_t lo = 0, hi = n;
    while (lo < hi) {
        int32_t mid = lo + (hi - lo) / 2;
        if (uniq[mid] < key) lo = mid + 1; else hi = mid;
    }
    return lo;
}

/*
 * ids[n_occ]: behavior IDs then ad IDs.  Outputs (caller-allocated):
 *   uniq[n_u]        distinct IDs, ascending
 *   inv[n_occ]       uniq[inv[k]] == ids[k]
 *   occ_perm[n_occ]  occurrence indices ordered by (ID, k): a stable sort
 *   uniq_off[n_u+1]  occ_perm[uniq_off[u] .. uniq_off[u+1]) are the occurrences of uniq[u]
 *   *n_uniq          n_u
 */
int orc_dedup(const int32_t *ids, int64_t n_occ, int32_t n_ids,
              int32_t *uniq, int32_t *inv, int32_t *occ_perm,
              int32_t *uniq_off, int32_t *n_uniq)
{
    if (n_occ < 0 || n_occ > INT32_MAX || n_ids < 0) return 1;
    for (int64_t k = 0; k < n_occ; ++k)
        if (ids[k] < 0 || ids[k] >= n_ids) return 2;
    occ_pair *p = (occ_pair *)malloc((size_t)(n_occ > 0 ? n_occ : 1) * sizeof *p);
    if (!p) return 1;
    for (int64_t k = 0; k < n_occ; ++k) { p[k].id = ids[k]; p[k].k = (int32_t)k; }
    qsort(p, (size_t)n_occ, sizeof *p, cmp_pair);
    int32_t nu = 0;
    for (int64_t i = 0; i < n_occ; ++i) {
        occ_perm[i] = p[i].k;
        if (i == 0 || p[i].id != p[i - 1].id) {
            uniq[nu] = p[i].id;
            uniq_off[nu] = (int32_t)i;
            ++nu;
        }
    }
    uniq_off[nu] = (int32_t)n_occ;
    for (int64_t k = 0; k < n_occ; ++k)
        inv[k] = lower_bound_i32(uniq, nu, ids[k]);
    *n_uniq = nu;
    free(p);
    return 0;
}

/* ---------------------------------------------------------------- MLP fwd */

/*
 * n_layers >= 1, dims[0..n_layers]: widths, input first.
 * T: feature table rows of width dims[0] (float32 or bf16), rows[u] selects
 * the row of unique image u (0 <= rows[u] < n_rows).
 * W[l]: [dims[l+1] x dims[l]] row-major (storage dtype), b[l]: float32[dims[l+1]].
 * Z (out): pre-activations of every layer, concatenated layer by layer, each
 *          [n x dims[l+1]].  E (out): [n x dims[n_layers]] final output.
 */
int orc_mlp_fwd(int n_layers, const int32_t *dims, int dtype,
                const void *T, int64_t n_rows, const int32_t *rows, int32_t n,
                const void *const *W, const float *const *b, int final_relu,
                double *Z, double *E)
{
    if (n_layers < 1 || n < 0) return 1;
    for (int32_t u = 0; u < n; ++u)
        if (rows[u] < 0 || rows[u] >= n_rows) return 2;
    size_t zoff[16];
    if (n_layers > 15) return 1;
    zoff[0] = 0;
    for (int l = 0; l < n_layers; ++l) zoff[l + 1] = zoff[l] + (size_t)n * dims[l + 1];
    const int F = dims[0];

#pragma omp parallel
    {
        int wmax = 0;
        for (int l = 0; l <= n_layers; ++l) if (dims[l] > wmax) wmax = dims[l];
        double *h = (double *)malloc(sizeof(double) * (size_t)wmax);
        double *hn = (double *)malloc(sizeof(double) * (size_t)wmax);
#pragma omp for schedule(static)
        for (int32_t u = 0; u < n; ++u) {
            for (int i = 0; i < F; ++i)
                h[i] = load_elem(T, dtype, (size_t)rows[u] * F + i);
            for (int l = 0; l < n_layers; ++l) {
                const int in = dims[l], out = dims[l + 1];
                double *z = Z + zoff[l] + (size_t)u * out;
                for (int o = 0; o < out; ++o) {
                    double acc = (double)b[l][o];
                    for (int i = 0; i < in; ++i)
                        acc += load_elem(W[l], dtype, (size_t)o * in + i) * h[i];
                    z[o] = acc;
                }
                const int last = (l == n_layers - 1);
                for (int o = 0; o < out; ++o)
                    hn[o] = (!last || final_relu) ? (z[o] > 0.0 ? z[o] : 0.0) : z[o];
                memcpy(h, hn, sizeof(double) * (size_t)out);
            }
            memcpy(E + (size_t)u * dims[n_layers], h, sizeof(double) * (size_t)dims[n_layers]);
        }
        free(h);
        free(hn);
    }
    return 0;
}

/* ---------------------------------------------------------------- MLP bwd */

/*
 * Given the forward's pre-activations Z and dE[n x D] (gradient of the loss
 * w.r.t. E), writes dW[l] ([dims[l+1] x dims[l]], float64, concatenated) and
 * db[l] ([dims[l+1]], concatenated).  Every entry is a sum over unique images
 * u = 0, 1, ..., n-1 in that order.  dZ_scratch may be NULL (allocated here);
 * if given it receives the pre-activation gradients, laid out like Z.
 */
int orc_mlp_bwd(int n_layers, const int32_t *dims, int dtype,
                const void *T, int64_t n_rows, const int32_t *rows, int32_t n,
                const void *const *W, int final_relu,
                const double *Z, const double *dE, double *dW, double *db,
                double *dZ_out)
{
    if (n_layers < 1 || n_layers > 15 || n < 0) return 1;
    for (int32_t u = 0; u < n; ++u)
        if (rows[u] < 0 || rows[u] >= n_rows) return 2;
    size_t zoff[16], woff[16], boff[16];
    zoff[0] = woff[0] = boff[0] = 0;
    for (int l = 0; l < n_layers; ++l) {
        zoff[l + 1] = zoff[l] + (size_t)n * dims[l + 1];
        woff[l + 1] = woff[l] + (size_t)dims[l + 1] * dims[l];
        boff[l + 1] = boff[l] + (size_t)dims[l + 1];
    }
    double *dZ = dZ_out ? dZ_out : (double *)malloc(sizeof(double) * (zoff[n_layers] > 0 ? zoff[n_layers] : 1));
    if (!dZ) return 1;

    /* 1. pre-activation gradients, one unique image at a time */
    const int L = n_layers;
#pragma omp parallel for schedule(static)
    for (int32_t u = 0; u < n; ++u) {
        const int D = dims[L];
        double *dz = dZ + zoff[L - 1] + (size_t)u * D;
        const double *z = Z + zoff[L - 1] + (size_t)u * D;
        for (int o = 0; o < D; ++o) {
            double g = dE[(size_t)u * D + o];
            dz[o] = final_relu ? (z[o] > 0.0 ? g : 0.0) : g;
        }
        for (int l = L - 1; l >= 1; --l) {
            const int in = dims[l], out = dims[l + 1];
            const double *dzo = dZ + zoff[l] + (size_t)u * out;
            double *dzi = dZ + zoff[l - 1] + (size_t)u * in;
            const double *zi = Z + zoff[l - 1] + (size_t)u * in;
            for (int i = 0; i < in; ++i) {
                double acc = 0.0;
                for (int o = 0; o < out; ++o)
                    acc += load_elem(W[l], dtype, (size_t)o * in + i) * dzo[o];
                dzi[i] = zi[i] > 0.0 ? acc : 0.0;
            }
        }
    }

    /* 2. weight gradients dW_l[o][i] = sum_u dz_l[u][o] * h_{l-1}[u][i] */
    for (int l = 0; l < L; ++l) {
        const int in = dims[l], out = dims[l + 1];
        double *dWl = dW + woff[l];
        memset(dWl, 0, sizeof(double) * (size_t)out * in);
        const double *dz = dZ + zoff[l];
        const int CB = 64;
        const int nblk = (in + CB - 1) / CB;
#pragma omp parallel for schedule(static)
        for (int blk = 0; blk < nblk; ++blk) {
            const int c0 = blk * CB, c1 = c0 + CB < in ? c0 + CB : in;
            double hrow[64];
            for (int32_t u = 0; u < n; ++u) {
                for (int c = c0; c < c1; ++c) {
                    if (l == 0) {
                        hrow[c - c0] = load_elem(T, dtype, (size_t)rows[u] * in + c);
                    } else {
                        double zz = Z[zoff[l - 1] + (size_t)u * in + c];
                        hrow[c - c0] = zz > 0.0 ? zz : 0.0;
                    }
                }
                for (int o = 0; o < out; ++o) {
                    const double g = dz[(size_t)u * out + o];
                    double *row = dWl + (size_t)o * in;
                    for (int c = c0; c < c1; ++c)
                        row[c] += g * hrow[c - c0];
                }
            }
        }
        double *dbl = db + boff[l];
        for (int o = 0; o < out; ++o) {
            double acc = 0.0;
            for (int32_t u = 0; u < n; ++u) acc += dz[(size_t)u * out + o];
            dbl[o] = acc;
        }
    }
    if (!dZ_out) free(dZ);
    return 0;
}

/* --------------------------------------------------------------- pool fwd */

/*
 * Samples i = 0..B-1; behaviors of sample i are occurrences
 * j in [seg_off[i], seg_off[i+1]) with embedding E[inv[j]]; the ad of sample
 * i is occurrence n_beh + i with embedding A[i] = E[inv[n_beh + i]].
 * U[B x D] pooled user vector.  argmax[B x D] (MAX, may be NULL otherwise):
 * first j attaining the max, -1 for an empty segment.  w[n_beh] (ATT):
 * attention weights.
 */
int orc_pool_fwd(int mode, int32_t B, int32_t D, const int32_t *seg_off,
                 int64_t n_beh, const int32_t *inv, const double *E,
                 double *U, double *A, int32_t *argmax, double *w)
{
    if (B < 0 || D <= 0 || mode < 0 || mode > 2) return 1;
    if (B > 0 && (seg_off[0] != 0 || seg_off[B] != n_beh)) return 1;
#pragma omp parallel for schedule(static)
    for (int32_t i = 0; i < B; ++i) {
        const int64_t j0 = seg_off[i], j1 = seg_off[i + 1];
        const double *a = E + (size_t)inv[n_beh + i] * D;
        double *u = U + (size_t)i * D;
        for (int d = 0; d < D; ++d) A[(size_t)i * D + d] = a[d];
        for (int d = 0; d < D; ++d) u[d] = 0.0;
        if (mode == POOL_SUM) {
            for (int64_t j = j0; j < j1; ++j) {
                const double *e = E + (size_t)inv[j] * D;
                for (int d = 0; d < D; ++d) u[d] += e[d];
            }
        } else if (mode == POOL_MAX) {
            for (int d = 0; d < D; ++d) {
                int32_t best = -1;
                double m = 0.0;
                for (int64_t j = j0; j < j1; ++j) {
                    const double v = E[(size_t)inv[j] * D + d];
                    if (best < 0 || v > m) { m = v; best = (int32_t)j; }
                }
                u[d] = best < 0 ? 0.0 : m;
                if (argmax) argmax[(size_t)i * D + d] = best;
            }
        } else {
            if (j1 == j0) continue;
            double smax = -INFINITY;
            for (int64_t j = j0; j < j1; ++j) {
                const double *e = E + (size_t)inv[j] * D;
                double s = 0.0;
                for (int d = 0; d < D; ++d) s += e[d] * a[d];
                w[j] = s;                       /* logit, normalised below */
                if (s > smax) smax = s;
            }
            double den = 0.0;
            for (int64_t j = j0; j < j1; ++j) den += exp(w[j] - smax);
            for (int64_t j = j0; j < j1; ++j) w[j] = exp(w[j] - smax) / den;
            for (int64_t j = j0; j < j1; ++j) {
                const double *e = E + (size_t)inv[j] * D;
                for (int d = 0; d < D; ++d) u[d] += w[j] * e[d];
            }
        }
    }
    return 0;
}

/* --------------------------------------------------------------- pool bwd */

/*
 * Loss L = sum(gU * U) + sum(gA * A) (gA may be NULL: zero).
 * ge (out, optional, [n_occ x D]): gradient w.r.t. each occurrence's
 * embedding.  dE (out, [n_u x D]): ge summed per unique image in ascending
 * occurrence order.  dA_att (out, optional, [B x D]): the attention term
 * that flows into the ad embedding.
 */
int orc_pool_bwd(int mode, int32_t B, int32_t D, const int32_t *seg_off,
                 int64_t n_beh, const int32_t *inv, int32_t n_u,
                 const double *E, const double *U, const double *A,
                 const int32_t *argmax, const double *w,
                 const double *gU, const double *gA,
                 double *dE, double *ge_out, double *dA_att)
{
    if (B < 0 || D <= 0 || D > 64 || mode < 0 || mode > 2 || n_u < 0) return 1;
    const int64_t n_occ = n_beh + B;
    double *ge = ge_out ? ge_out : (double *)malloc(sizeof(double) * (size_t)(n_occ > 0 ? n_occ : 1) * D);
    if (!ge) return 1;
#pragma omp parallel for schedule(static)
    for (int32_t i = 0; i < B; ++i) {
        const int64_t j0 = seg_off[i], j1 = seg_off[i + 1];
        const double *g = gU + (size_t)i * D;
        const double *a = A + (size_t)i * D;
        double da[64];
        for (int d = 0; d < D; ++d) da[d] = 0.0;
        if (mode == POOL_SUM) {
            for (int64_t j = j0; j < j1; ++j)
                for (int d = 0; d < D; ++d) ge[(size_t)j * D + d] = g[d];
        } else if (mode == POOL_MAX) {
            for (int64_t j = j0; j < j1; ++j)
                for (int d = 0; d < D; ++d)
                    ge[(size_t)j * D + d] = (argmax[(size_t)i * D + d] == j) ? g[d] : 0.0;
        } else {
            const double *u = U + (size_t)i * D;
            double c = 0.0;
            for (int d = 0; d < D; ++d) c += g[d] * u[d];
            for (int64_t j = j0; j < j1; ++j) {
                const double *e = E + (size_t)inv[j] * D;
                double dw = 0.0;
                for (int d = 0; d < D; ++d) dw += g[d] * e[d];
                const double ds = w[j] * (dw - c);
                for (int d = 0; d < D; ++d) {
                    ge[(size_t)j * D + d] = w[j] * g[d] + ds * a[d];
                    da[d] += ds * e[d];
                }
            }
        }
        for (int d = 0; d < D; ++d) {
            ge[(size_t)(n_beh + i) * D + d] = (gA ? gA[(size_t)i * D + d] : 0.0) + da[d];
            if (dA_att) dA_att[(size_t)i * D + d] = da[d];
        }
    }
    memset(dE, 0, sizeof(double) * (size_t)n_u * D);
    for (int64_t k = 0; k < n_occ; ++k)
        for (int d = 0; d < D; ++d)
            dE[(size_t)inv[k] * D + d] += ge[(size_t)k * D + d];
    if (!ge_out) free(ge);
    return 0;
}

/* ---------------------------------------------------------------- bag fwd */

/*
 * bag[i][d] = sum_{j in [seg_off[i], seg_off[i+1])} table[idx[j]][d]
 *             + table[idx[n_beh + i]][d]
 * summed in ascending j, the ad row last.  table is float32 [n_rows x D];
 * idx holds row numbers of `table` (raw IDs of a whole table, or positions
 * in a table of just the touched rows).
 */
int orc_bag_fwd(int32_t B, int32_t D, const int32_t *seg_off, int64_t n_beh,
                const int32_t *idx, int64_t n_rows, const float *table, double *bag)
{
    if (B < 0 || D < 1) return 1;
    for (int64_t k = 0; k < n_beh + B; ++k)
        if (idx[k] < 0 || idx[k] >= n_rows) return 2;
#pragma omp parallel for schedule(static)
    for (int32_t i = 0; i < B; ++i) {
        double *o = bag + (size_t)i * D;
        for (int d = 0; d < D; ++d) o[d] = 0.0;
        for (int64_t j = seg_off[i]; j < seg_off[i + 1]; ++j)
            for (int d = 0; d < D; ++d) o[d] += (double)table[(size_t)idx[j] * D + d];
        for (int d = 0; d < D; ++d) o[d] += (double)table[(size_t)idx[n_beh + i] * D + d];
    }
    return 0;
}

/* --------------------------------------------------------------- CTR MLP */

/*
 * X [B x dims[0]] float64 input rows; W[l] float32 [dims[l+1] x dims[l]],
 * b[l] float32 [dims[l+1]]; labels int32 [B] in [0, C), C = dims[n_layers].
 * Forward: Z_l = H_{l-1} W_l^T + b_l, H_l = ReLU(Z_l) below the last layer,
 * logits Z_L; p = softmax(Z_L) (max subtracted); loss = mean_i (lse_i - Z_L[i][y_i]).
 * Backward of the mean loss: dZ_L = (p - onehot(y)) / B; dW_l = sum_i dZ_l[i]^T
 * H_{l-1}[i] and db_l = sum_i dZ_l[i] (ascending i); dH_{l-1} = dZ_l W_l,
 * dZ_{l-1} = dH_{l-1} * [Z_{l-1} > 0]; dX = dZ_1 W_1.
 * Outputs: *loss, prob [B x C], Z (concatenated per layer, [B x dims[l+1]]),
 * dW, db (concatenated per layer), dX [B x dims[0]].
 */
int orc_ctr_fwd_bwd(int32_t B, int n_layers, const int32_t *dims, const float *const *W,
                    const float *const *b, const double *X, const int32_t *labels,
                    double *loss, double *prob, double *Z, double *dW, double *db, double *dX)
{
    if (B < 1 || n_layers < 1 || n_layers > 15) return 1;
    const int C = dims[n_layers];
    for (int32_t i = 0; i < B; ++i)
        if (labels[i] < 0 || labels[i] >= C) return 1;
    size_t zoff[16], woff[16], boff[16];
    zoff[0] = woff[0] = boff[0] = 0;
    int wmax = 0;
    for (int l = 0; l < n_layers; ++l) {
        zoff[l + 1] = zoff[l] + (size_t)B * dims[l + 1];
        woff[l + 1] = woff[l] + (size_t)dims[l] * dims[l + 1];
        boff[l + 1] = boff[l] + (size_t)dims[l + 1];
    }
    for (int l = 0; l <= n_layers; ++l) if (dims[l] > wmax) wmax = dims[l];
    /* forward, sample by sample */
    double *lossv = (double *)malloc(sizeof(double) * (size_t)B);
#pragma omp parallel
    {
        double *h = (double *)malloc(sizeof(double) * (size_t)wmax);
#pragma omp for schedule(static)
        for (int32_t i = 0; i < B; ++i) {
            for (int k = 0; k < dims[0]; ++k) h[k] = X[(size_t)i * dims[0] + k];
            for (int l = 0; l < n_layers; ++l) {
                const int in = dims[l], out = dims[l + 1];
                double *z = Z + zoff[l] + (size_t)i * out;
                for (int o = 0; o < out; ++o) {
                    double acc = (double)b[l][o];
                    for (int k = 0; k < in; ++k) acc += (double)W[l][(size_t)o * in + k] * h[k];
                    z[o] = acc;
                }
                for (int o = 0; o < out; ++o) h[o] = (l < n_layers - 1) ? (z[o] > 0.0 ? z[o] : 0.0) : z[o];
            }
            const double *zl = Z + zoff[n_layers - 1] + (size_t)i * C;
            double m = zl[0];
            for (int c = 1; c < C; ++c) if (zl[c] > m) m = zl[c];
            double se = 0.0;
            for (int c = 0; c < C; ++c) se += exp(zl[c] - m);
            const double lse = m + log(se);
            for (int c = 0; c < C; ++c) prob[(size_t)i * C + c] = exp(zl[c] - lse);
            lossv[i] = lse - zl[labels[i]];
        }
        free(h);
    }
    double tot = 0.0;
    for (int32_t i = 0; i < B; ++i) tot += lossv[i];
    *loss = tot / B;
    free(lossv);
    /* backward: dZ of every layer, then the weight gradients */
    double *dZ = (double *)malloc(sizeof(double) * zoff[n_layers]);
    for (int32_t i = 0; i < B; ++i)
        for (int c = 0; c < C; ++c)
            dZ[zoff[n_layers - 1] + (size_t)i * C + c] =
                (prob[(size_t)i * C + c] - (c == labels[i] ? 1.0 : 0.0)) / B;
    for (int l = n_layers - 1; l >= 0; --l) {
        const int in = dims[l], out = dims[l + 1];
        const double *dz = dZ + zoff[l];
#pragma omp parallel for schedule(static)
        for (int32_t i = 0; i < B; ++i) {
            for (int k = 0; k < in; ++k) {
                double acc = 0.0;
                for (int o = 0; o < out; ++o) acc += dz[(size_t)i * out + o] * (double)W[l][(size_t)o * in + k];
                if (l > 0) {
                    const double zp = Z[zoff[l - 1] + (size_t)i * in + k];
                    dZ[zoff[l - 1] + (size_t)i * in + k] = zp > 0.0 ? acc : 0.0;
                } else {
                    dX[(size_t)i * in + k] = acc;
                }
            }
        }
        /* dW_l[o][k] = sum_i dz[i][o] h_{l-1}[i][k], h_{-1} = X */
#pragma omp parallel for schedule(static)
        for (int o = 0; o < out; ++o) {
            double *row = dW + woff[l] + (size_t)o * in;
            for (int k = 0; k < in; ++k) row[k] = 0.0;
            double bsum = 0.0;
            for (int32_t i = 0; i < B; ++i) {
                const double g = dz[(size_t)i * out + o];
                bsum += g;
                for (int k = 0; k < in; ++k) {
                    double hk;
                    if (l == 0) hk = X[(size_t)i * in + k];
                    else {
                        const double zp = Z[zoff[l - 1] + (size_t)i * in + k];
                        hk = zp > 0.0 ? zp : 0.0;
                    }
                    row[k] += g * hk;
                }
            }
            db[boff[l] + o] = bsum;
        }
    }
    free(dZ);
    return 0;
}

/* ---------------------------------------------------------------- adagrad */

/*
 * Sparse Adagrad on n touched rows (row-compact arrays [n x D]):
 * accum += g^2; rows -= lr * g / (sqrt(accum) + eps), elementwise.
 */
int orc_adagrad_rows(int32_t n, int32_t D, const double *grad, double lr, double eps,
                     double *rows, double *accum)
{
    if (n < 0 || D < 1) return 1;
    for (size_t e = 0; e < (size_t)n * D; ++e) {
        accum[e] += grad[e] * grad[e];
        rows[e] -= lr * grad[e] / (sqrt(accum[e]) + eps);
    }
    return 0;
}

/* ------------------------------------------------------ query attention */

/*
 * Q [B x D]: the query of each sample.  For sample i with behaviors
 * j in [seg_off[i], seg_off[i+1]): s_j = e_j . q_i, w = softmax(s) (max
 * subtracted), u_i = sum_j w_j e_j; an empty segment pools to 0.  U [B x D],
 * w [n_beh] out.
 */
int orc_pool_query_fwd(int32_t B, int32_t D, const int32_t *seg_off, int64_t n_beh,
                       const int32_t *inv, const double *E, const double *Q, double *U, double *w)
{
    if (B < 0 || D <= 0) return 1;
    if (B > 0 && (seg_off[0] != 0 || seg_off[B] != n_beh)) return 1;
#pragma omp parallel for schedule(static)
    for (int32_t i = 0; i < B; ++i) {
        const int64_t j0 = seg_off[i], j1 = seg_off[i + 1];
        const double *q = Q + (size_t)i * D;
        double *u = U + (size_t)i * D;
        for (int d = 0; d < D; ++d) u[d] = 0.0;
        if (j1 == j0) continue;
        double smax = -INFINITY;
        for (int64_t j = j0; j < j1; ++j) {
            const double *e = E + (size_t)inv[j] * D;
            double sv = 0.0;
            for (int d = 0; d < D; ++d) sv += e[d] * q[d];
            w[j] = sv;
            if (sv > smax) smax = sv;
        }
        double den = 0.0;
        for (int64_t j = j0; j < j1; ++j) den += exp(w[j] - smax);
        for (int64_t j = j0; j < j1; ++j) w[j] = exp(w[j] - smax) / den;
        for (int64_t j = j0; j < j1; ++j) {
            const double *e = E + (size_t)inv[j] * D;
            for (int d = 0; d < D; ++d) u[d] += w[j] * e[d];
        }
    }
    return 0;
}

/*
 * Backward of orc_pool_query_fwd for the loss sum(gU * U): with
 * c_i = gU_i . u_i and ds_j = w_j (gU_i . e_j - c_i), the gradient of
 * occurrence j is ge_j = w_j gU_i + ds_j q_i (the ads' occurrences get none
 * from this channel); dE[u] = sum of ge_j over the behaviors j of image u in
 * ascending j (dE [n_u x D], overwritten); dQ_i = sum_j ds_j e_j.
 */
int orc_pool_query_bwd(int32_t B, int32_t D, const int32_t *seg_off, int64_t n_beh,
                       const int32_t *inv, int32_t n_u, const double *E, const double *Q,
                       const double *U, const double *w, const double *gU, double *dE, double *dQ)
{
    if (B < 0 || D <= 0 || n_u < 0) return 1;
    double *ge = (double *)malloc(sizeof(double) * (size_t)(n_beh > 0 ? n_beh : 1) * D);
#pragma omp parallel for schedule(static)
    for (int32_t i = 0; i < B; ++i) {
        const int64_t j0 = seg_off[i], j1 = seg_off[i + 1];
        const double *g = gU + (size_t)i * D, *u = U + (size_t)i * D, *q = Q + (size_t)i * D;
        double c = 0.0;
        for (int d = 0; d < D; ++d) c += g[d] * u[d];
        double *dq = dQ + (size_t)i * D;
        for (int d = 0; d < D; ++d) dq[d] = 0.0;
        for (int64_t j = j0; j < j1; ++j) {
            const double *e = E + (size_t)inv[j] * D;
            double dw = 0.0;
            for (int d = 0; d < D; ++d) dw += g[d] * e[d];
            const double ds = w[j] * (dw - c);
            for (int d = 0; d < D; ++d) {
                ge[(size_t)j * D + d] = w[j] * g[d] + ds * q[d];
                dq[d] += ds * e[d];
            }
        }
    }
    memset(dE, 0, sizeof(double) * (size_t)n_u * D);
    for (int64_t j = 0; j < n_beh; ++j)
        for (int d = 0; d < D; ++d) dE[(size_t)inv[j] * D + d] += ge[(size_t)j * D + d];
    free(ge);
    return 0;
}

/* ------------------------------------------------------------------- Adam */

/* One Adam step t >= 1 on n parameters, in place (all float64). */
int orc_adam(int64_t n, double *param, const double *grad, double *m, double *v, double lr, double b1,
             double b2, double eps, int64_t t)
{
    if (n < 0 || t < 1) return 1;
    const double c1 = 1.0 - pow(b1, (double)t), c2 = 1.0 - pow(b2, (double)t);
    for (int64_t i = 0; i < n; ++i) {
        m[i] = b1 * m[i] + (1.0 - b1) * grad[i];
        v[i] = b2 * v[i] + (1.0 - b2) * grad[i] * grad[i];
        param[i] -= lr * (m[i] / c1) / (sqrt(v[i] / c2) + eps);
    }
    return 0;
}

/* --------------------------------------------------- concatenate aggregator */

/*
 * U [B x Lc*D]: sample i's first Lc behavior embeddings in list order, one
 * after the other (U[i][p*D + d] = E[inv[seg_off[i] + p]][d]); positions past
 * the sample's length are zero (pad), behaviors past Lc are dropped
 * (truncate).  A [B x D]: the ad's embedding E[inv[n_beh + i]].
 */
int orc_pool_concat_fwd(int32_t B, int32_t D, int32_t Lc, const int32_t *seg_off, int64_t n_beh,
                        const int32_t *inv, const double *E, double *U, double *A)
{
    if (B < 0 || D <= 0 || Lc < 1) return 1;
    if (B > 0 && (seg_off[0] != 0 || seg_off[B] != n_beh)) return 1;
    for (int32_t i = 0; i < B; ++i) {
        const int64_t j0 = seg_off[i], n = seg_off[i + 1] - j0;
        for (int32_t p = 0; p < Lc; ++p)
            for (int d = 0; d < D; ++d)
                U[((size_t)i * Lc + p) * D + d] = p < n ? E[(size_t)inv[j0 + p] * D + d] : 0.0;
        for (int d = 0; d < D; ++d) A[(size_t)i * D + d] = E[(size_t)inv[n_beh + i] * D + d];
    }
    return 0;
}

/*
 * Backward of orc_pool_concat_fwd for the loss sum(gU * U) + sum(gA * A)
 * (gA may be NULL: zero).  Behavior j at position p of its sample i gets
 * gU[i][p] if p < Lc and zero otherwise; the ad of sample i gets gA[i].
 * dE [n_u x D] (overwritten): those summed per unique image in ascending
 * occurrence order.
 */
int orc_pool_concat_bwd(int32_t B, int32_t D, int32_t Lc, const int32_t *seg_off, int64_t n_beh,
                        const int32_t *inv, int32_t n_u, const double *gU, const double *gA, double *dE)
{
    if (B < 0 || D <= 0 || Lc < 1 || n_u < 0) return 1;
    memset(dE, 0, sizeof(double) * (size_t)n_u * D);
    int32_t i = 0;
    for (int64_t k = 0; k < n_beh + B; ++k) {
        double *o = dE + (size_t)inv[k] * D;
        if (k < n_beh) {
            while (seg_off[i + 1] <= k) ++i;
            const int64_t p = k - seg_off[i];
            if (p < Lc)
                for (int d = 0; d < D; ++d) o[d] += gU[((size_t)i * Lc + p) * D + d];
        } else if (gA) {
            for (int d = 0; d < D; ++d) o[d] += gA[(size_t)(k - n_beh) * D + d];
        }
    }
    return 0;
}

/* ------------------------------------------------- dense net with PReLU */

/*
 * A fully connected net dims[0] -> ... -> dims[L] on B rows X [B x dims[0]],
 * float32 weights W[l] [dims[l+1] x dims[l]] and biases b[l], float64
 * arithmetic: Z_l = H_{l-1} W_l^T + b_l with H_{-1} = X, and below the last
 * layer H_l = act(Z_l) with act(z) = z for z > 0 and a z otherwise, a the
 * layer's per-channel slope slope[l][o] (PReLU, the activation of section
 * 7.2); slope == NULL or slope[l] == NULL means a = 0 (ReLU).  The last
 * layer is linear.  Z (out): every layer's Z_l, concatenated.
 */
static double act_slope(const float *const *slope, int l, int o)
{
    return (slope && slope[l]) ? (double)slope[l][o] : 0.0;
}

int orc_dense_fwd(int32_t B, int L, const int32_t *dims, const float *const *W, const float *const *b,
                  const float *const *slope, const double *X, double *Z)
{
    if (B < 0 || L < 1 || L > 15) return 1;
    size_t zoff = 0;
    for (int l = 0; l < L; ++l) {
        const int in = dims[l], out = dims[l + 1];
        const double *Zp = Z + zoff - (l > 0 ? (size_t)B * in : 0);
#pragma omp parallel for schedule(static)
        for (int32_t i = 0; i < B; ++i)
            for (int o = 0; o < out; ++o) {
                double acc = (double)b[l][o];
                for (int k = 0; k < in; ++k) {
                    double h;
                    if (l == 0) h = X[(size_t)i * in + k];
                    else {
                        const double z = Zp[(size_t)i * in + k];
                        h = z > 0.0 ? z : act_slope(slope, l - 1, k) * z;
                    }
                    acc += (double)W[l][(size_t)o * in + k] * h;
                }
                Z[zoff + (size_t)i * out + o] = acc;
            }
        zoff += (size_t)B * out;
    }
    return 0;
}

/*
 * Backward of orc_dense_fwd from dZL [B x dims[L]], the gradient of the last
 * layer's output: dW_l = sum_i dZ_l[i]^T H_{l-1}[i] and db_l = sum_i dZ_l[i]
 * (ascending i); dH_{l-1} = dZ_l W_l; dZ_{l-1} = dH_{l-1} act'(Z_{l-1}) with
 * act'(z) = 1 for z > 0 and a otherwise (ReLU'(0) = 0); the slope gradient
 * dslope_{l-1}[k] = sum_i dH_{l-1}[i][k] min(Z_{l-1}[i][k], 0); dX = dZ_0 W_0.
 * dW, db, dslope (the hidden layers' widths) are concatenated per layer.
 */
int orc_dense_bwd(int32_t B, int L, const int32_t *dims, const float *const *W, const float *const *slope,
                  const double *X, const double *Z, const double *dZL, double *dW, double *db,
                  double *dslope, double *dX)
{
    if (B < 0 || L < 1 || L > 15) return 1;
    size_t zoff[16], woff[16], boff[16], soff[16];
    zoff[0] = woff[0] = boff[0] = soff[0] = 0;
    for (int l = 0; l < L; ++l) {
        zoff[l + 1] = zoff[l] + (size_t)B * dims[l + 1];
        woff[l + 1] = woff[l] + (size_t)dims[l] * dims[l + 1];
        boff[l + 1] = boff[l] + (size_t)dims[l + 1];
        soff[l + 1] = soff[l] + (l < L - 1 ? (size_t)dims[l + 1] : 0);
    }
    double *dZ = (double *)malloc(sizeof(double) * (zoff[L] > 0 ? zoff[L] : 1));
    memcpy(dZ + zoff[L - 1], dZL, sizeof(double) * (size_t)B * dims[L]);
    for (int l = L - 1; l >= 0; --l) {
        const int in = dims[l], out = dims[l + 1];
        const double *dz = dZ + zoff[l];
#pragma omp parallel for schedule(static)
        for (int o = 0; o < out; ++o) {
            double bs = 0.0;
            for (int k = 0; k < in; ++k) dW[woff[l] + (size_t)o * in + k] = 0.0;
            for (int32_t i = 0; i < B; ++i) {
                const double g = dz[(size_t)i * out + o];
                bs += g;
                for (int k = 0; k < in; ++k) {
                    double h;
                    if (l == 0) h = X[(size_t)i * in + k];
                    else {
                        const double z = Z[zoff[l - 1] + (size_t)i * in + k];
                        h = z > 0.0 ? z : act_slope(slope, l - 1, k) * z;
                    }
                    dW[woff[l] + (size_t)o * in + k] += g * h;
                }
            }
            db[boff[l] + o] = bs;
        }
        /* one thread per input unit k: rows i ascending, as in a serial loop */
#pragma omp parallel for schedule(static)
        for (int k = 0; k < in; ++k) {
            double ds = 0.0;
            for (int32_t i = 0; i < B; ++i) {
                double dh = 0.0;
                for (int o = 0; o < out; ++o) dh += dz[(size_t)i * out + o] * (double)W[l][(size_t)o * in + k];
                if (l == 0) {
                    dX[(size_t)i * in + k] = dh;
                } else {
                    const double z = Z[zoff[l - 1] + (size_t)i * in + k];
                    dZ[zoff[l - 1] + (size_t)i * in + k] = z > 0.0 ? dh : act_slope(slope, l - 1, k) * dh;
                    if (!(z > 0.0)) ds += dh * z;
                }
            }
            if (l > 0) dslope[soff[l - 1] + k] = ds;
        }
    }
    free(dZ);
    return 0;
}
