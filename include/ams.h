/*
 * ams.h -- C ABI of libams, the MI355X (gfx950) hot path of one Advanced Model
 * Server training step for the shared image-embedding model.
 *
 * One step (section 4.2; Algorithm 1, SERVEREMBED and SERVERUPDATE) is:
 *   ams_dedup      the batch's image IDs (behavior images, then ad images) are
 *                  reduced to one sorted set, so each image is fetched and
 *                  embedded once and its gradients are merged at one place;
 *   ams_embed_fwd  each unique image's feature row is gathered from the table
 *                  and run through the trainable embedding model, a fully
 *                  connected net 4096-256-64-12 (section 5.1), ReLU between
 *                  layers;
 *   ams_pool_fwd   each sample's behavior embeddings are aggregated into one
 *                  user vector by sum, max, or attentive pooling with the ad
 *                  image embedding as query (section 5.2);
 *   ams_pool_bwd   the upstream gradients are taken back through the pooling
 *                  and summed per unique image (Algorithm 1: gradients for the
 *                  same image are collected by the same server);
 *   ams_embed_bwd  the merged embedding gradients are back-propagated through
 *                  the embedding model into its weight and bias gradients
 *                  (Algorithm 1, SERVERUPDATE).  The feature table is fixed
 *                  (the frozen VGG16 part, section 5.1): no gradient flows to it.
 *
 * Conventions shared by every call
 * --------------------------------
 * Pointers:   every array argument is a DEVICE pointer unless marked "host".
 *             The caller allocates and frees all memory, including workspaces;
 *             the library allocates no device memory and keeps no mutable
 *             global state, so calls on different streams with different
 *             workspaces may run concurrently.
 * Streams:    `stream` is a hipStream_t passed as void* (NULL = the null
 *             stream).  Calls only enqueue work and never synchronize.
 * Counts:     the number of unique images n_u is produced on the device by
 *             ams_dedup (*n_uniq) and read there by later calls; they take a
 *             host upper bound `n_uniq_cap` (n_u <= n_uniq_cap <= n_occ) that
 *             sizes grids and buffers.  Work past n_u is skipped and outputs
 *             past n_u are left unspecified.  A bound below the real n_u
 *             leaves the rows past it uncomputed and the occurrences that
 *             refer to them dropped (read as zero rows): results are then
 *             unspecified, but no call reads or writes outside the
 *             buffers the bound sizes.
 * Layouts:    row-major.  Feature table T is [n_rows x dims[0]].  Weights
 *             W_l are [dims[l+1] x dims[l]] (out x in), biases float32
 *             [dims[l+1]].  E, U, A, dE, dU, dA have row stride D = dims[last]
 *             floats.  IDs are int32.
 * Precision:  AMS_F32: T and W float32, float32 MFMA with float32 accumulation.
 *             AMS_F32_X3: T and W float32 as AMS_F32.  The 4096-wide layer's
 *             forward product (dims[1] a multiple of 256) runs on bf16 MFMA:
 *             every float32 operand is split exactly into three bf16 parts
 *             h + m + l (round to nearest at each step; exact for
 *             |x| >= 2^-100, where all parts are normal) and six of the nine
 *             part products (hh, hm, mh, hl, lh, mm) are accumulated in
 *             float32; the three left out stay below 2^-22 |x y| per
 *             product, about one float32 rounding.  Everything else as
 *             AMS_F32.
 *             AMS_BF16: T and W bfloat16; bf16 MFMA with float32 accumulation
 *             for the 4096-wide layer and its weight gradient (whose
 *             activation-gradient operand is rounded to bf16).  The smaller
 *             layers also run on bf16 MFMA, but each float32 activation or
 *             gradient operand enters as a pair of bf16 values (high part
 *             plus the rounded remainder, together within 2^-18 of the
 *             float32 value) against the exact bf16 weights, so they keep
 *             float32-level accuracy.  E, U, A, the attention weights and
 *             every gradient are float32.  H1_save is bf16 in this mode
 *             (the rounding of the float32 H1), float32 otherwise.
 * Determinism: every output is bitwise reproducible for identical inputs on
 *             the same device (fixed reduction orders, no float atomics).
 * Errors:     calls return an ams_status.  Problems visible on the host are
 *             reported before anything is enqueued.  An image ID outside its
 *             range can only be seen on the device: ams_dedup then writes
 *             AMS_ERR_ID_RANGE into *dev_status (read it after a sync) and
 *             its outputs are unspecified; later calls never read outside T.
 *             Nothing is printed and no call aborts.
 */
#ifndef AMS_H
#define AMS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    AMS_OK = 0,
    AMS_ERR_NULL = 1,       /* a required pointer is NULL */
    AMS_ERR_SIZE = 2,       /* a size is negative, too large, or inconsistent */
    AMS_ERR_DTYPE = 3,      /* unknown storage dtype */
    AMS_ERR_DIMS = 4,       /* layer widths this build does not support */
    AMS_ERR_WORKSPACE = 5,  /* ws_bytes below the matching *_workspace() size */
    AMS_ERR_HIP = 6,        /* a HIP launch or runtime call failed */
    AMS_ERR_ID_RANGE = 7,   /* (device) an image ID is outside [0, n_ids) */
    AMS_ERR_MODE = 8,       /* unknown pooling mode */
    AMS_ERR_CAPACITY = 9    /* beyond the fixed scratch of ams_dedup_noalloc */
} ams_status;

typedef enum { AMS_F32 = 0, AMS_BF16 = 1, AMS_F32_X3 = 2 } ams_dtype;

/* Aggregators of section 5.2.  ATT: w_j = softmax_j(e_j . a_i) over the
 * sample's behaviors, u_i = sum_j w_j e_j, with a_i the ad image embedding. */
typedef enum { AMS_POOL_SUM = 0, AMS_POOL_MAX = 1, AMS_POOL_ATT = 2 } ams_pool;

/* Shape of the trainable embedding model (section 5.1: 4096-256-64-12).
 * Supported: n_layers 2 or 3; dims[0] a multiple of 64 in [64, 65536];
 * dims[1] a multiple of 64 in [64, 256]; hidden dims[2] (3 layers) in [1, 64];
 * output D = dims[n_layers] in [1, 32].  final_relu = 1 puts a ReLU after the
 * last layer as well (default 0: the embedding is the last layer's affine
 * output). */
typedef struct {
    int32_t n_layers;
    int32_t dims[4];
    int32_t dtype;       /* ams_dtype of T and the weights */
    int32_t final_relu;
} ams_mlp;

/* Text of a status code (host, static storage, never NULL). */
const char *ams_status_str(ams_status s);

/* Library version and the GPU architecture it was built for (host). */
const char *ams_build_info(void);

/* ------------------------------------------------------------ timing ----
 * Per-kernel timing, for benchmarks and diagnostics.  While enabled, every
 * kernel that a call enqueues is bracketed by two HIP events recorded on the
 * call's stream; ams_timing_read waits for the recorded events, sums the
 * elapsed times per kernel name and clears the record.  The switch and the
 * record are process-wide: use it from one host thread at a time.  Off by
 * default; when off it costs one relaxed load per launch.
 *
 * ams_timing_read: out[cap] receives up to cap entries in order of first
 * launch; *n_out is the number of distinct kernels recorded (may exceed cap).
 * Returns AMS_ERR_NULL for a NULL n_out (or NULL out with cap > 0), and
 * AMS_ERR_HIP if an event could not be created, recorded or read (those
 * launches are left out of the sums; the record is cleared all the same). */
typedef struct {
    char name[32];       /* kernel name, NUL-terminated */
    int64_t launches;    /* timed launches since the last read */
    double total_ms;     /* summed event-to-event time of those launches */
} ams_kernel_time;

ams_status ams_timing_enable(int on);
ams_status ams_timing_read(ams_kernel_time *out, int cap, int *n_out);

/* ------------------------------------------------------------- dedup ----
 * Requests for the same image are processed once (section 4.2).
 *
 * ids[n_occ]        the batch's image IDs: all behavior IDs (sample by sample)
 *                   followed by the B ad IDs.  0 <= ids[k] < n_ids.
 * uniq[n_occ]       out: the n_u distinct IDs in ascending order.
 * inv[n_occ]        out: uniq[inv[k]] == ids[k].
 * occ_perm[n_occ]   out: occurrence indices sorted by (ID, k): a stable sort.
 * uniq_off[n_occ+1] out: occurrences of uniq[u] are
 *                   occ_perm[uniq_off[u] .. uniq_off[u+1]); uniq_off[n_u] = n_occ.
 * n_uniq[1]         out: n_u.
 * dev_status[1]     out: AMS_OK, or AMS_ERR_ID_RANGE if some ID is out of range.
 * ws, ws_bytes      workspace of at least ams_dedup_workspace(n_occ, n_ids) bytes;
 *                   that size also serves every smaller n_occ and n_ids (one
 *                   workspace for several ID tables).
 * n_occ == 0 is valid (n_u = 0).  Host errors: NULL, SIZE (n_occ < 0,
 * n_occ > 2^30 - 1, n_ids < 1), WORKSPACE.  Outputs are bit-exact: they are
 * the unique canonical answer.  *dev_status = AMS_ERR_HIP reports an internal
 * wait that did not complete (outputs then unspecified). */
size_t ams_dedup_workspace(int64_t n_occ, int32_t n_ids);
ams_status ams_dedup(const int32_t *ids, int64_t n_occ, int32_t n_ids,
                     int32_t *uniq, int32_t *inv, int32_t *occ_perm,
                     int32_t *uniq_off, int32_t *n_uniq, int32_t *dev_status,
                     void *ws, size_t ws_bytes, void *stream);

/* ------------------------------------------- dedup without allocation ----
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): ams_dedup
 * with the workspace replaced by a fixed scratch array that the library's
 * code object holds on every GPU it runs on (about 19 MB each, kept until
 * the process ends).  Arguments, outputs, determinism and device status as
 * ams_dedup; the outputs are bit-identical to ams_dedup's.  The call itself
 * allocates nothing (no hipMalloc, no allocating library routine); its first
 * call on a device looks up that device's scratch address once.
 *   n_occ <= AMS_DEDUP_NOALLOC_MAX_OCC (2^20), else AMS_ERR_CAPACITY before
 *   anything is enqueued; any n_ids >= 1 (IDs of up to 31 bits).
 * Every call on one GPU shares that GPU's scratch: calls that overlap on one
 * GPU (different streams without ordering, or several host threads) race
 * and give unspecified results.  Calls ordered on one stream are safe; each
 * call clears the parts of the scratch that must start at zero itself.
 * Host errors: SIZE, CAPACITY, NULL; AMS_ERR_HIP if the scratch address
 * cannot be found or a launch fails. */
#define AMS_DEDUP_NOALLOC_MAX_OCC (1 << 20)
ams_status ams_dedup_noalloc(const int32_t *ids, int64_t n_occ, int32_t n_ids,
                             int32_t *uniq, int32_t *inv, int32_t *occ_perm,
                             int32_t *uniq_off, int32_t *n_uniq, int32_t *dev_status,
                             void *stream);

/* --------------------------------------------------------- embed fwd ----
 * SERVEREMBED (Algorithm 1): e = E(I) for every unique image.
 *
 * mlp (host)        model shape and dtype (see ams_mlp).
 * T                 feature table [n_rows x dims[0]], dtype mlp->dtype.
 * uniq, n_uniq      from ams_dedup; rows uniq[0..n_u) of T are embedded.
 *                   A row index outside [0, n_rows) reads as a zero row.
 * W1,b1,W2,b2,W3,b3 weights (dtype) and float32 biases; W3/b3 ignored when
 *                   n_layers == 2.
 * slope             NULL: ReLU between layers.  Otherwise a host array with
 *                   one device array per hidden layer (slope[0] [dims[1]],
 *                   and for 3 layers slope[1] [dims[2]], float32, none NULL):
 *                   PReLU, z for z > 0 and slope[c] z otherwise, a learnable
 *                   slope per channel (the activation of section 7.2).
 *                   AMS_F32 and AMS_F32_X3; AMS_BF16 with dims[1] = 256 and,
 *                   for 3 layers, dims[2] a multiple of 4 with dims[2]*D <=
 *                   1024 (the bf16 tails): other bf16 shapes return DTYPE.
 * H1_save           out, optional: first hidden layer [cap x dims[1]] (bf16 in
 *                   AMS_BF16 mode, float32 otherwise): post-ReLU, or with
 *                   PReLU the pre-activation Z1 (bias included).  Needed by
 *                   ams_embed_bwd; pass NULL for inference only.
 * H2_save           out, optional (3 layers): second hidden layer [cap x
 *                   dims[2]] float32, post-ReLU, or with PReLU Z2.
 * E                 out: embeddings [cap x D] float32 (row u for uniq[u]).
 * ws                at least ams_embed_workspace(mlp, cap) bytes. */
size_t ams_embed_workspace(const ams_mlp *mlp, int32_t n_uniq_cap);
ams_status ams_embed_fwd(const ams_mlp *mlp, const void *T, int64_t n_rows,
                         const int32_t *uniq, const int32_t *n_uniq,
                         int32_t n_uniq_cap,
                         const void *W1, const float *b1,
                         const void *W2, const float *b2,
                         const void *W3, const float *b3,
                         const float *const *slope,
                         void *H1_save, float *H2_save, float *E,
                         void *ws, size_t ws_bytes, void *stream);

/* --------------------------------------------------------- embed bwd ----
 * SERVERUPDATE (Algorithm 1): delta_E = grad E(I) . delta_e.
 *
 * Inputs as in ams_embed_fwd plus the forward's H1_save/H2_save, its E
 * (read only when final_relu = 1, for the last layer's ReLU mask; may be NULL
 * otherwise) and dE [cap x D] float32 (from ams_pool_bwd).  Outputs, all float32 and fully
 * overwritten (not accumulated): dW1 [dims[1] x dims[0]], db1, dW2, db2,
 * dW3, db3 (dW3/db3 ignored when n_layers == 2).  Every gradient is a sum over
 * the n_u unique images in a fixed order.  ReLU'(0) = 0.  slope as in
 * ams_embed_fwd (the same arrays, and H1_save / H2_save from that call);
 * with PReLU, act'(z) = 1 for z > 0 and slope otherwise, and dslope (host
 * array of device arrays, or NULL: not stored) receives each hidden layer's
 * slope gradient, sum over unique images of dH * min(Z, 0), overwritten. */
ams_status ams_embed_bwd(const ams_mlp *mlp, const void *T, int64_t n_rows,
                         const int32_t *uniq, const int32_t *n_uniq,
                         int32_t n_uniq_cap,
                         const void *W1, const void *W2, const void *W3,
                         const float *const *slope,
                         const void *H1_save, const float *H2_save,
                         const float *E_fwd, const float *dE,
                         float *dW1, float *db1, float *dW2, float *db2,
                         float *dW3, float *db3, float *const *dslope,
                         void *ws, size_t ws_bytes, void *stream);

/* ---------------------------------------------------------- pool fwd ----
 * User behavior image aggregator (section 5.2).
 *
 * mode              ams_pool.
 * B, D              samples and embedding width (1 <= D <= 32).
 * seg_off[B+1]      CSR offsets of the behavior lists: sample i owns
 *                   occurrences j in [seg_off[i], seg_off[i+1]);
 *                   seg_off[0] = 0, seg_off[B] = n_beh, non-decreasing.
 * inv[n_beh+B]      from ams_dedup (behaviors then ads).
 * n_uniq_cap        rows of E (host).  An occurrence whose unique index is
 *                   n_uniq_cap or more (only possible when the caller's
 *                   capacity is below the real unique count) reads a zero
 *                   row: results are then unspecified, but nothing outside
 *                   E is read.
 * E [n_uniq_cap x D] embeddings from ams_embed_fwd.
 * U [B x D]         out: pooled user vectors (empty segment -> 0).
 * A [B x D]         out: the ad image embedding of each sample, E[inv[n_beh+i]].
 * saved             out: MAX: int32 [B x D] index j of the first maximum
 *                   (-1 for an empty segment); ATT: float32 [n_beh] attention
 *                   weights; SUM: unused (may be NULL). */
ams_status ams_pool_fwd(int32_t mode, int32_t B, int32_t D,
                        const int32_t *seg_off, int64_t n_beh,
                        const int32_t *inv, int32_t n_uniq_cap, const float *E,
                        float *U, float *A, void *saved, void *stream);

/* ---------------------------------------------------------- pool bwd ----
 * Loss gradient through the aggregator, merged per unique image.
 *
 * dU [B x D]        upstream gradient of U; dA [B x D] of A (NULL = zero).
 * occ_perm, uniq_off, n_uniq from ams_dedup; E, U, A, saved from the forward.
 * dE [cap x D]      out: for each unique image, the sum over its occurrences
 *                   (in ascending occurrence order) of the gradient w.r.t.
 *                   that occurrence's embedding; fully overwritten for u < n_u.
 *                   E and dE have n_uniq_cap rows: occurrences whose unique
 *                   index is n_uniq_cap or more (a capacity below the real
 *                   unique count) are dropped and read E as a zero row, so
 *                   no access leaves the caller's buffers.
 * ws                at least ams_pool_workspace(mode, B, n_beh, D, cap) bytes. */
size_t ams_pool_workspace(int32_t mode, int32_t B, int64_t n_beh, int32_t D,
                          int32_t n_uniq_cap);
ams_status ams_pool_bwd(int32_t mode, int32_t B, int32_t D,
                        const int32_t *seg_off, int64_t n_beh,
                        const int32_t *inv, const int32_t *occ_perm,
                        const int32_t *uniq_off, const int32_t *n_uniq,
                        int32_t n_uniq_cap,
                        const float *E, const float *U, const float *A,
                        const void *saved, const float *dU, const float *dA,
                        float *dE, void *ws, size_t ws_bytes, void *stream);

/* --------------------------------------------------- query pooling ----
 * One channel of multiple-query attentive pooling (section 5.2): attention
 * over a sample's behavior image embeddings with a query given per sample
 * (for the ID channel, the ad's ID embedding; the image channel is
 * ams_pool_fwd's AMS_POOL_ATT, whose query is the ad image embedding).  The
 * channels' pooled vectors are concatenated by the caller.
 *
 * fwd:  Q [B x D] queries (device); U [B x D] out: u_i = sum_j w_j e_j with
 *       w = softmax_j(e_j . q_i) (max subtracted; an empty segment pools to
 *       0); w [n_beh] out: the attention weights.  Other arguments (E with
 *       n_uniq_cap rows) as in ams_pool_fwd.
 * bwd:  with dU [B x D] the loss gradient of U, the gradient of behavior j is
 *       w_j dU_i + ds_j q_i, ds_j = w_j (dU_i . e_j - dU_i . u_i); dE[u]
 *       receives the sum over the behaviors of image u in ascending order
 *       (the ads' occurrences get nothing from this channel): overwritten
 *       when accumulate = 0, added to the existing dE when accumulate = 1
 *       (so the two channels of one step merge into one dE; every row u < n_u
 *       is written by one thread, no atomics); dQ [B x D] out: sum_j ds_j e_j.
 *       ws: at least ams_pool_workspace(AMS_POOL_ATT, B, n_beh, D, cap) bytes.
 * Host errors as ams_pool_fwd / ams_pool_bwd. */
ams_status ams_pool_query_fwd(int32_t B, int32_t D, const int32_t *seg_off, int64_t n_beh,
                              const int32_t *inv, int32_t n_uniq_cap, const float *E,
                              const float *Q, float *U, float *w, void *stream);
ams_status ams_pool_query_bwd(int32_t B, int32_t D, const int32_t *seg_off, int64_t n_beh,
                              const int32_t *inv, const int32_t *occ_perm,
                              const int32_t *uniq_off, const int32_t *n_uniq,
                              int32_t n_uniq_cap, const float *E, const float *Q,
                              const float *U, const float *w, const float *dU,
                              float *dQ, float *dE, int32_t accumulate,
                              void *ws, size_t ws_bytes, void *stream);

/* -------------------------------------------------- concat pooling ----
 * The concatenate aggregator (section 5.2): a sample's behavior embeddings
 * side by side, padded or truncated to Lc of them.
 *
 * fwd:  U [B x Lc*D] out: U[i][p*D + d] = E[inv[seg_off[i] + p]][d] for the
 *       first Lc behaviors of sample i in list order, zero for positions
 *       past its length; later behaviors are dropped.  A [B x D] out: the
 *       ad's embedding E[inv[n_beh + i]].  Lc >= 1, Lc * D <= INT32_MAX.
 * bwd:  dU [B x Lc*D], dA [B x D] (NULL = zero) the loss gradients of U and
 *       A.  The behavior at position p of sample i gets dU[i][p*D .. p*D+D)
 *       when p < Lc and nothing otherwise; the ad of sample i gets dA[i].
 *       dE [cap x D] (overwritten for u < n_u): their sums per unique image
 *       in ascending occurrence order, as ams_pool_bwd merges them.
 *       ws: at least ams_pool_workspace(AMS_POOL_SUM, B, n_beh, D, cap).
 * Other arguments and host errors as ams_pool_fwd / ams_pool_bwd. */
ams_status ams_pool_concat_fwd(int32_t B, int32_t D, int32_t Lc, const int32_t *seg_off,
                               int64_t n_beh, const int32_t *inv, int32_t n_uniq_cap,
                               const float *E, float *U, float *A, void *stream);
ams_status ams_pool_concat_bwd(int32_t B, int32_t D, int32_t Lc, const int32_t *seg_off,
                               int64_t n_beh, const int32_t *inv, const int32_t *occ_perm,
                               const int32_t *uniq_off, const int32_t *n_uniq,
                               int32_t n_uniq_cap, const float *dU, const float *dA,
                               float *dE, void *ws, size_t ws_bytes, void *stream);

/* =================================================== joint step (worker) ====
 * The worker side of a joint training step (Algorithm 1, WORKERITERATION):
 * sparse ID features embedded from key-value tables (section 4.1) next to the
 * image embeddings, the CTR model on top of them trained with cross-entropy
 * (section 3.1), whose input gradients are the delta_e pushed to the image
 * path (ams_pool_bwd / ams_embed_bwd), and a sparse Adagrad step on the ID
 * rows the batch touched.  ID tables are float32 [n_rows x D] row-major;
 * their IDs per table are laid out like the image IDs: one per behavior
 * (sample by sample) then one per ad. */

/* ---------------------------------------------------------- bag fwd ----
 * bag[i][d] = sum over j in [seg_off[i], seg_off[i+1]) of table[ids[j]][d]
 *             + table[ids[n_beh + i]][d]
 * B samples, 1 <= D <= 32, ids[n_beh + B] (device), table [n_rows x D]
 * (device), bag [B x D] out (device).  An ID outside [0, n_rows) reads as a
 * zero row (ams_dedup over the same IDs reports it).  The sum over a
 * sample's behaviors has a fixed association; the ad row is added last.
 * Host errors: SIZE, DIMS (D), NULL. */
ams_status ams_bag_fwd(int32_t B, int32_t D, const int32_t *seg_off, int64_t n_beh,
                       const int32_t *ids, const float *table, int64_t n_rows,
                       float *bag, void *stream);

/* ---------------------------------------------------------- bag bwd ----
 * Merged gradient of the touched rows of one ID table.  With inv, occ_perm,
 * uniq_off, n_uniq from ams_dedup over that table's IDs and dbag [B x D] the
 * loss gradient of the bags: grad[u] = sum over the occurrences k of uniq[u]
 * (ascending k) of dbag[sample of k], for u < n_u; grad is [n_uniq_cap x D]
 * and fully written for u < n_u.  This is the SUM aggregator's backward with
 * dbag as the upstream gradient of behaviors and ads (ams_pool_bwd, SUM):
 * deterministic, no atomics, hot IDs split at fixed boundaries.
 * dad: NULL, or [B x D] a second gradient of each sample's ad row (device),
 * for a table whose ad row also serves elsewhere, as the query of the ID
 * channel of MultiQueryAttentivePooling (section 5.2: dQ from
 * ams_pool_query_bwd): the ad occurrence of sample i then contributes
 * dbag[i] + dad[i].
 * ws: at least ams_bag_workspace(B, n_beh, D, n_uniq_cap) bytes. */
size_t ams_bag_workspace(int32_t B, int64_t n_beh, int32_t D, int32_t n_uniq_cap);
ams_status ams_bag_bwd(int32_t B, int32_t D, const int32_t *seg_off, int64_t n_beh,
                       const int32_t *inv, const int32_t *occ_perm, const int32_t *uniq_off,
                       const int32_t *n_uniq, int32_t n_uniq_cap, const float *dbag,
                       const float *dad, float *grad, void *ws, size_t ws_bytes, void *stream);

/* ------------------------------------------------------------- CTR -----
 * The CTR MLP (the basic net's MLP, section 3.2): dims[0] inputs (the
 * concatenated fields), ReLU or PReLU between layers (section 7.2: PReLU,
 * z for z > 0 and a z otherwise with a learnable slope a per channel),
 * dims[n_layers] = C classes, softmax and cross-entropy with the labels,
 * averaged over the B samples.  Supported: n_layers 2 or 3; dims[0] <= 128;
 * hidden widths <= 256; 2 <= C <= 8; 1..8 input fields; widths whose
 * activations fit the block's LDS (DIMS otherwise).  float32 throughout. */
typedef struct {
    int32_t n_layers;
    int32_t dims[4];
} ams_ctr;

/* fields, field_dims, W, b, dW, db, dfields are HOST arrays of DEVICE
 * pointers (field_dims: host widths):
 *   fields[f]   [B x field_dims[f]]: sample i's input row is fields[0][i] ++
 *               fields[1][i] ++ ...; the widths sum to dims[0];
 *   labels      [B] int32 in [0, C) (device); a sample whose label is outside
 *               that range adds nothing to the loss or to any gradient;
 *   W[l], b[l]  [dims[l+1] x dims[l]] and [dims[l+1]] float32 (device);
 *   slope       NULL (ReLU everywhere) or, for each layer l < n_layers-1,
 *               the PReLU slopes [dims[l+1]] of its activation (device;
 *               an entry NULL: ReLU there); ReLU'(0) = 0, PReLU'(0) = a;
 *   loss        [1] out: mean cross-entropy over the B samples (device);
 *   prob        [B x C] out, softmax probabilities (device, may be NULL);
 *   dW[l], db[l] out: gradients of the mean loss, overwritten (device);
 *   dslope      NULL or per hidden layer the slope gradient [dims[l+1]]
 *               (device, out; written where that layer has slopes):
 *               sum over samples of dH * min(Z, 0), Z the pre-activation;
 *   dfields     gradients of the mean loss w.r.t. each field, [B x
 *               field_dims[f]] (device); dfields itself or any entry may be
 *               NULL (not written).
 * Every gradient is a sum over samples in a fixed order.
 * ws: at least ams_ctr_workspace(net, B) bytes.  Host errors: NULL, DIMS,
 * SIZE (B < 1), WORKSPACE. */
size_t ams_ctr_workspace(const ams_ctr *net, int32_t B);
ams_status ams_ctr_fwd_bwd(const ams_ctr *net, int32_t B, int32_t n_fields,
                           const float *const *fields, const int32_t *field_dims,
                           const int32_t *labels, const float *const *W,
                           const float *const *b, const float *const *slope,
                           float *loss, float *prob, float *const *dW, float *const *db,
                           float *const *dslope, float *const *dfields,
                           void *ws, size_t ws_bytes, void *stream);

/* --------------------------------------------------------- pre-rank ----
 * The pre-rank model of section 6: a user tower and an ad tower, each a
 * net of the CTR kind (ams_ctr: 1 to 3 layers, ReLU or PReLU between them,
 * the last layer linear) on its own fields, with outputs of equal width R
 * (1..64), the user and ad representations; the score of a sample is
 * their inner product s = <u, a>, its click probability sigmoid(s).  The
 * loss is softplus(s) - y s (the logistic loss) for labels y in {0, 1},
 * summed over the samples and divided by B; a sample with another label
 * adds nothing to the loss or any gradient.  The behavior images enter the
 * user tower sum-pooled (ams_pool_fwd, AMS_POOL_SUM) and the ad image the
 * ad tower; the input-field gradients carry delta_e back to them.
 * Per tower, arguments as ams_ctr_fwd_bwd's (u: user, a: ad): fields and
 * field_dims, W, b, slope, and the outputs dW, db, dslope, dfields.
 * prob [B] out (may be NULL): sigmoid(s) of every sample, labels aside.
 * ws: at least ams_dssm_workspace(user_net, ad_net, B) bytes.
 * Host errors: NULL, DIMS (widths, or R unequal), SIZE (B < 1), WORKSPACE. */
size_t ams_dssm_workspace(const ams_ctr *user_net, const ams_ctr *ad_net, int32_t B);
ams_status ams_dssm_fwd_bwd(const ams_ctr *user_net, const ams_ctr *ad_net, int32_t B,
                            int32_t n_user_fields, const float *const *user_fields,
                            const int32_t *user_field_dims, int32_t n_ad_fields,
                            const float *const *ad_fields, const int32_t *ad_field_dims,
                            const int32_t *labels,
                            const float *const *Wu, const float *const *bu,
                            const float *const *slope_u,
                            const float *const *Wa, const float *const *ba,
                            const float *const *slope_a,
                            float *loss, float *prob,
                            float *const *dWu, float *const *dbu, float *const *dslope_u,
                            float *const *dWa, float *const *dba, float *const *dslope_a,
                            float *const *duser_fields, float *const *dad_fields,
                            void *ws, size_t ws_bytes, void *stream);

/* ---------------------------------------------------------- Adagrad ----
 * Sparse Adagrad on the touched rows of an ID table, in place: for u < n_u
 * (uniq, n_uniq from ams_dedup over the table's IDs) and d < D, with
 * g = grad[u][d] and r = uniq[u]:
 *   accum[r][d] += g * g;  table[r][d] -= lr * g / (sqrt(accum[r][d]) + eps).
 * Rows are distinct, so the update has no races; untouched rows are left as
 * they are.  A row index outside [0, n_rows) is skipped.  table and accum are
 * [n_rows x D] float32 (device).  Host errors: SIZE, NULL. */
ams_status ams_adagrad_rows(int32_t D, const int32_t *uniq, const int32_t *n_uniq,
                            int32_t n_uniq_cap, const float *grad, float *table,
                            int64_t n_rows, float *accum, float lr, float eps,
                            void *stream);

/* ------------------------------------------------------------- Adam -----
 * The dense update (Algorithm 1: update E on the servers and W on the
 * workers; section 7.2 trains with Adam).  For i < n, with g = grad[i]:
 *   m[i] = b1 m[i] + (1 - b1) g;   v[i] = b2 v[i] + (1 - b2) g^2;
 *   param[i] -= lr (m[i] / (1 - b1^t)) / (sqrt(v[i] / (1 - b2^t)) + eps)
 * in float32, in place (device arrays of n floats); t >= 1 is the step
 * number (host), lr the step's learning rate (section 7.2: 1e-3, times 0.9
 * after every 24,000 batches; the schedule is the caller's).  param is the
 * float32 master copy; param_bf16 (device, may be NULL) receives its
 * round-to-nearest-even bf16 copy, the weights the bf16 kernels read.
 * Host errors: SIZE (n < 0 or t < 1), NULL. */
ams_status ams_adam_update(int64_t n, float *param, const float *grad, float *m, float *v,
                           float lr, float b1, float b2, float eps, int64_t t,
                           uint16_t *param_bf16, void *stream);

/* ============================================================= probes ====
 * Achievable-peak probes of the device (they compute nothing of the method):
 * the rates the part delivers for plain HBM streams, for gathering table
 * rows in the order the first-layer kernels visit them, and for MFMA on
 * operands read from memory, to stand beside the kernels' rates and the
 * vendor peaks.  Every pointer is a device pointer; `blocks` workgroups of
 * 256 threads.  Host errors: SIZE, NULL (DTYPE for ams_peak_mfma).
 *
 * ams_peak_copy    dst = src, `bytes` (a multiple of 16), grid-stride.
 * ams_peak_read    reads `bytes` of src; out[blocks * 256] receives one xor
 *                  per thread.
 * ams_peak_gather  reads rows[0..n) of the table T [n_table x 8192 bytes]
 *                  (row_bytes must be 8192, else SIZE) the way the bf16
 *                  first layer visits them: 512-thread blocks, each a
 *                  contiguous range of the list in tiles of 256 rows, a tile
 *                  in 64 stages of 128 bytes per row, 3 stages ahead.
 *                  pattern 0: register loads, each lane 16-byte pieces of
 *                  its own row (every load touches 32 rows: the MFMA operand
 *                  layout); 1: register loads of whole 128-byte lines (8 rows
 *                  per load); 2: as 1, non-temporal; 3: whole-line
 *                  non-temporal DMA into a 3-slot LDS ring, 2 stages ahead,
 *                  one barrier per stage; 4: as 3 plus a 32 KB slice of W
 *                  (2 MB: 256 rows of 8192 bytes, needed only here) per stage
 *                  into a 2-slot ring.  Other patterns: MODE.  A row index
 *                  outside [0, n_table) reads row 0; out[blocks * 512]
 *                  receives one xor per thread.
 * ams_peak_mfma    dtype AMS_BF16 (v_mfma_f32_32x32x16_bf16, 32768 flops) or
 *                  AMS_F32 (v_mfma_f32_32x32x2_f32, 4096 flops): every wave
 *                  runs iters x 16 independent products on operands read from
 *                  ops (524288 bytes); out[blocks * 256] one float per
 *                  thread. */
ams_status ams_peak_copy(const void *src, void *dst, int64_t bytes, int32_t blocks, void *stream);
ams_status ams_peak_read(const void *src, int64_t bytes, int32_t blocks, uint32_t *out, void *stream);
ams_status ams_peak_gather(const void *T, int64_t n_table, int32_t row_bytes, const int32_t *rows,
                           int32_t n, int32_t pattern, const void *W, int32_t blocks, uint32_t *out,
                           void *stream);
ams_status ams_peak_mfma(int32_t dtype, const void *ops, int32_t iters, int32_t blocks, float *out,
                         void *stream);

#ifdef __cplusplus
}
#endif

#endif /* AMS_H */
