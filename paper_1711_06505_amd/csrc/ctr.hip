// ctr.hip -- the worker side of one joint training step (Algorithm 1,
// WORKERITERATION) next to the image path:
//   ams_bag_fwd      per sample and ID table, the sum of the table rows of its
//                    behaviors' IDs and of its ad's ID (sparse ID features
//                    embedded from key-value tables, section 4.1);
//   ams_bag_bwd      the gradient of every touched row: the bag gradient of
//                    each occurrence's sample, summed per unique ID in
//                    ascending occurrence order (the segmented reduction of
//                    the SUM aggregator's backward);
//   ams_ctr_fwd_bwd  the CTR MLP on the concatenated input fields, softmax over
//                    the classes and mean cross-entropy with the click labels
//                    (section 3.1), and its backward: the worker's weight
//                    gradients and the gradient of every input field (among
//                    them delta_e of the image path);
//   ams_adagrad_rows sparse Adagrad on the touched rows of an ID table.
// No float atomics: every sum runs in a fixed order.
#include "ams_device.h"

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / AMS_WAVE;
constexpr int kCtrBS = 16;                  // samples per block of the CTR kernel
constexpr int kCtrThreads = 512;            // threads per block of the CTR and tower kernels (2 waves per SIMD)
constexpr int kCtrMaxIn = 128, kCtrMaxHidden = 256, kCtrMaxC = 8, kTowerMaxOut = 64;
constexpr int kCtrMaxLayers = 3, kCtrMaxFields = 8;

// ------------------------------------------------------------ bag forward

// One wave per sample: lane l adds the rows of behaviors l, l + 64, ... in
// that order; the lanes' partial rows are summed by a fixed butterfly, then
// the ad row.  Behaviors go in rounds of U per lane (8 for rows up to 16
// floats, else 4) with every ID load, then every row load, of a round in
// flight together.  An ID outside [0, n_rows) reads as a zero row (dedup
// reports it).
template <int DM>
__global__ __launch_bounds__(kThreads) void bag_fwd_k(int B, int D, const int32_t *__restrict__ seg_off,
                                                      int64_t n_beh, const int32_t *__restrict__ ids,
                                                      const float *__restrict__ table, int64_t n_rows,
                                                      float *__restrict__ bag)
{
    const int lane = ams_lane();
    const int i = blockIdx.x * kWaves + threadIdx.x / AMS_WAVE;
    if (i >= B) return;
    const int j0 = seg_off[i], j1 = seg_off[i + 1];
    float acc[DM];
#pragma unroll
    for (int d = 0; d < DM; ++d) acc[d] = 0.f;
    const bool vec4 = (D & 3) == 0 && ((uintptr_t)table & 15) == 0;
    constexpr int kBagU = DM <= 16 ? 8 : 4;
    // every load of a round unconditional (a position past the sample reads
    // its last ID, an ID outside the table reads row 0), masked once all are
    // in flight; no table rows at all: nothing to read
    if (n_rows > 0) {
        for (int jr = j0; jr < j1; jr += kBagU * AMS_WAVE) {
            int id[kBagU];
#pragma unroll
            for (int u = 0; u < kBagU; ++u) {
                const int j = jr + u * AMS_WAVE + lane;
                id[u] = ids[j < j1 ? j : j1 - 1];
            }
            bool ok[kBagU];
#pragma unroll
            for (int u = 0; u < kBagU; ++u) {
                const int j = jr + u * AMS_WAVE + lane;
                ok[u] = j < j1 && id[u] >= 0 && (int64_t)id[u] < n_rows;
            }
            if (vec4) {
                float4 v[kBagU][DM / 4];
#pragma unroll
                for (int u = 0; u < kBagU; ++u) {
                    const float *r = table + (size_t)(ok[u] ? id[u] : 0) * D;
#pragma unroll
                    for (int d4 = 0; d4 < DM / 4; ++d4) v[u][d4] = *(const float4 *)(r + (4 * d4 < D ? 4 * d4 : 0));
                }
#pragma unroll
                for (int u = 0; u < kBagU; ++u)
#pragma unroll
                    for (int d4 = 0; d4 < DM / 4; ++d4) {
                        const bool take = ok[u] && 4 * d4 < D;
                        acc[4 * d4] += take ? v[u][d4].x : 0.f;
                        acc[4 * d4 + 1] += take ? v[u][d4].y : 0.f;
                        acc[4 * d4 + 2] += take ? v[u][d4].z : 0.f;
                        acc[4 * d4 + 3] += take ? v[u][d4].w : 0.f;
                    }
            } else {
                float v[kBagU][DM];
#pragma unroll
                for (int u = 0; u < kBagU; ++u) {
                    const float *r = table + (size_t)(ok[u] ? id[u] : 0) * D;
#pragma unroll
                    for (int d = 0; d < DM; ++d) v[u][d] = r[d < D ? d : 0];
                }
#pragma unroll
                for (int u = 0; u < kBagU; ++u)
#pragma unroll
                    for (int d = 0; d < DM; ++d) acc[d] += (ok[u] && d < D) ? v[u][d] : 0.f;
            }
        }
    }
    float mine = 0.f;
#pragma unroll
    for (int d = 0; d < DM; ++d) {
        const float s = ams_wave_sum(acc[d]);
        if (lane == d) mine = s;
    }
    if (lane < D) {
        const int id = ids[n_beh + i];
        const float a = (id >= 0 && (int64_t)id < n_rows) ? table[(size_t)id * D + lane] : 0.f;
        bag[(size_t)i * D + lane] = mine + a;
    }
}

// ---------------------------------------------------------------- CTR MLP

struct CtrArgs {
    int L;                                   // layers (1 to 3)
    int dims[kCtrMaxLayers + 1];
    int n_fields;
    int fdim[kCtrMaxFields];
    const float *field[kCtrMaxFields];
    float *dfield[kCtrMaxFields];
    const float *W[kCtrMaxLayers];
    const float *b[kCtrMaxLayers];
    const float *slope[kCtrMaxLayers];       // PReLU slopes after layer l < L-1; NULL: ReLU
};

// A block's partial row holds, per layer, dW [O x K], db [O] and, below the
// last layer, the slope gradient [O], each layer's part starting on a
// 16-byte boundary (padded to 4 floats); after the net(s) come 4 floats
// whose first is the loss sum, so rows are 16-byte multiples.
__host__ __device__ inline int net_layer_size(const CtrArgs &a, int l)
{
    return (a.dims[l + 1] * a.dims[l] + a.dims[l + 1] * (l < a.L - 1 ? 2 : 1) + 3) & ~3;
}

__host__ __device__ inline int net_part_size(const CtrArgs &a)
{
    int n = 0;
    for (int l = 0; l < a.L; ++l) n += net_layer_size(a, l);
    return n;
}

// Parts of a layer split over threads: forward P * kCtrBS * O, backward-data
// P * kCtrBS * K (P is chosen as in ctr_dense_fwd / ctr_dense_bwd_data).
__host__ __device__ inline int ctr_fwd_parts(int K, int O)
{
    int P = kCtrThreads / O;
    if (P < 1) P = 1;
    if (P > (K + 15) / 16) P = (K + 15) / 16;
    return P;
}

__host__ __device__ inline int ctr_bwd_parts(int K, int O)
{
    int P = kCtrThreads / K;
    if (P < 1) P = 1;
    if (P > (O + 7) / 8) P = (O + 7) / 8;
    return P;
}

// Activation of a hidden unit: ReLU, or PReLU with slope a (z for z > 0,
// a z otherwise), whose pre-activation is kept in z_out for the backward.
__device__ __forceinline__ float ctr_act(float v, const float *slope, int o, float *z_out)
{
    if (!slope) return fmaxf(v, 0.f);
    *z_out = v;
    return v > 0.f ? v : slope[o] * v;
}

// out[s][o] = bias[o] + sum_k in[s][k] W[o][k] for the block's kCtrBS
// samples, activated below the last layer (`hidden`).  Work item (o, part p
// of P): the K range of part p (a multiple of 4 wide), its W row streamed as
// float4 (the next one loaded while the current one is used), all samples
// accumulated together, k ascending (in[s][k..k+3] is one 16-byte LDS read,
// the same address for the whole wave: a broadcast).  With P > 1 (narrow layers) the
// parts go to `scr` [P][kCtrBS][O] and are added in part order.  With PReLU
// the pre-activations go to zout [kCtrBS][O].
__device__ __forceinline__ void ctr_dense_fwd(const float *in, int K, float *out, int O, const float *__restrict__ W,
                                              const float *__restrict__ bias, bool hidden,
                                              const float *__restrict__ slope, float *zout, float *scr, int t)
{
    const int P = ctr_fwd_parts(K, O);
    const int KC = (((K + P - 1) / P) + 3) & ~3;
    for (int it = t; it < O * P; it += kCtrThreads) {
        const int o = it % O, pp = it / O;
        const int k0 = pp * KC, k1 = min(K, k0 + KC);
        float acc[kCtrBS];
#pragma unroll
        for (int s = 0; s < kCtrBS; ++s) acc[s] = 0.f;
        const float *wr = W + (size_t)o * K;
        if ((K & 3) == 0) {
            // k0 and k1 are multiples of 4: 16 k per step in four groups of
            // four, each sample's inputs of a group one 16-byte LDS read; the
            // next step's 16 weights are loaded while this step computes
            float4 wn[4];
#pragma unroll
            for (int q = 0; q < 4; ++q)
                wn[q] = k0 + 4 * q < k1 ? *(const float4 *)(wr + k0 + 4 * q) : make_float4(0.f, 0.f, 0.f, 0.f);
            for (int kb = k0; kb < k1; kb += 16) {
                float4 wv[4];
#pragma unroll
                for (int q = 0; q < 4; ++q) wv[q] = wn[q];
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    if (kb + 16 + 4 * q < k1) wn[q] = *(const float4 *)(wr + kb + 16 + 4 * q);
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    if (kb + 4 * q < k1) {
                        float4 x[kCtrBS];
#pragma unroll
                        for (int s = 0; s < kCtrBS; ++s) x[s] = *(const float4 *)(in + s * K + kb + 4 * q);
#pragma unroll
                        for (int s = 0; s < kCtrBS; ++s) {
                            acc[s] = fmaf(x[s].x, wv[q].x, acc[s]);
                            acc[s] = fmaf(x[s].y, wv[q].y, acc[s]);
                            acc[s] = fmaf(x[s].z, wv[q].z, acc[s]);
                            acc[s] = fmaf(x[s].w, wv[q].w, acc[s]);
                        }
                    }
                }
            }
        } else {
            for (int k = k0; k < k1; ++k) {
                const float wk = wr[k];
#pragma unroll
                for (int s = 0; s < kCtrBS; ++s) acc[s] = fmaf(in[s * K + k], wk, acc[s]);
            }
        }
        if (P == 1) {
            const float bo = bias[o];
#pragma unroll
            for (int s = 0; s < kCtrBS; ++s) {
                const float v = acc[s] + bo;
                out[s * O + o] = hidden ? ctr_act(v, slope, o, zout + s * O + o) : v;
            }
        } else {
#pragma unroll
            for (int s = 0; s < kCtrBS; ++s) scr[(pp * kCtrBS + s) * O + o] = acc[s];
        }
    }
    if (P > 1) {
        __syncthreads();
        for (int e = t; e < kCtrBS * O; e += kCtrThreads) {
            const int o = e % O;
            float v = bias[o];
            for (int pp = 0; pp < P; ++pp) v += scr[pp * kCtrBS * O + e];
            out[e] = hidden ? ctr_act(v, slope, o, zout + e) : v;
        }
    }
}

// Gradient into a layer's input: d[s][k] = sum_o gout[s][o] W[o][k], then
// through the activation that produced the input when `act` (below the
// first layer): ReLU takes d where in > 0; PReLU reads its pre-activation z
// from gin (left there by the forward) and takes d for z > 0, slope[k] d
// otherwise, and adds d min(z, 0) over the block's samples (ascending) into
// the slope gradient dsl[k].  Work item (k, part p of P over O, o ascending);
// the lanes of a wave take consecutive k, so each W row read is contiguous
// across the wave.  Parts are added in order through `scr` as in the
// forward.
__device__ __forceinline__ void ctr_act_bwd(float *gin, const float *in, int K, int k, const float (&d)[kCtrBS],
                                            bool act, const float *__restrict__ slope, float *dsl)
{
    if (!act) {
#pragma unroll
        for (int s = 0; s < kCtrBS; ++s) gin[s * K + k] = d[s];
    } else if (!slope) {
#pragma unroll
        for (int s = 0; s < kCtrBS; ++s) gin[s * K + k] = in[s * K + k] > 0.f ? d[s] : 0.f;
        if (dsl) dsl[k] = 0.f;
    } else {
        const float a = slope[k];
        float ds = 0.f;
#pragma unroll
        for (int s = 0; s < kCtrBS; ++s) {
            const float z = gin[s * K + k];
            const bool pos = z > 0.f;
            gin[s * K + k] = pos ? d[s] : a * d[s];
            ds = fmaf(pos ? 0.f : z, d[s], ds);
        }
        dsl[k] = ds;
    }
}

__device__ __forceinline__ void ctr_dense_bwd_data(const float *gout, int O, float *gin, const float *in, int K,
                                                   const float *__restrict__ W, bool act,
                                                   const float *__restrict__ slope, float *dsl, float *scr, int t)
{
    const int P = ctr_bwd_parts(K, O);
    const int OC = (((O + P - 1) / P) + 3) & ~3;
    for (int it = t; it < K * P; it += kCtrThreads) {
        const int k = it % K, pp = it / K;
        const int o0 = pp * OC, o1 = min(O, o0 + OC);
        float acc[kCtrBS];
#pragma unroll
        for (int s = 0; s < kCtrBS; ++s) acc[s] = 0.f;
        if ((O & 3) == 0) {
            // 16 o per step in groups of four: the samples' gradients of a
            // group as 16-byte LDS reads; the next step's 16 W values are
            // loaded while this step computes
            float wn[16];
#pragma unroll
            for (int q = 0; q < 16; ++q) wn[q] = o0 + q < o1 ? W[(size_t)(o0 + q) * K + k] : 0.f;
            for (int ob = o0; ob < o1; ob += 16) {
                float w[16];
#pragma unroll
                for (int q = 0; q < 16; ++q) w[q] = wn[q];
#pragma unroll
                for (int q = 0; q < 16; ++q)
                    if (ob + 16 + q < o1) wn[q] = W[(size_t)(ob + 16 + q) * K + k];
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    if (ob + 4 * q < o1) {
                        float4 g[kCtrBS];
#pragma unroll
                        for (int s = 0; s < kCtrBS; ++s) g[s] = *(const float4 *)(gout + s * O + ob + 4 * q);
#pragma unroll
                        for (int s = 0; s < kCtrBS; ++s) {
                            acc[s] = fmaf(g[s].x, w[4 * q], acc[s]);
                            acc[s] = fmaf(g[s].y, w[4 * q + 1], acc[s]);
                            acc[s] = fmaf(g[s].z, w[4 * q + 2], acc[s]);
                            acc[s] = fmaf(g[s].w, w[4 * q + 3], acc[s]);
                        }
                    }
                }
            }
        } else {
            for (int o = o0; o < o1; ++o) {
                const float wo = W[(size_t)o * K + k];
#pragma unroll
                for (int s = 0; s < kCtrBS; ++s) acc[s] = fmaf(gout[s * O + o], wo, acc[s]);
            }
        }
        if (P == 1) {
            ctr_act_bwd(gin, in, K, k, acc, act, slope, dsl);
        } else {
#pragma unroll
            for (int s = 0; s < kCtrBS; ++s) scr[(pp * kCtrBS + s) * K + k] = acc[s];
        }
    }
    if (P > 1) {
        __syncthreads();
        for (int k = t; k < K; k += kCtrThreads) {
            float d[kCtrBS];
#pragma unroll
            for (int s = 0; s < kCtrBS; ++s) {
                float v = 0.f;
                for (int pp = 0; pp < P; ++pp) v += scr[(pp * kCtrBS + s) * K + k];
                d[s] = v;
            }
            ctr_act_bwd(gin, in, K, k, d, act, slope, dsl);
        }
    }
}

// Partial dW[o][k] = sum_s gout[s][o] in[s][k] over the block's samples and
// db[o] = sum_s gout[s][o], in 4 x 4 register tiles (8 LDS words per sample
// feed 16 FMAs); written to the block's partial row at p (dW, then db).
__device__ __forceinline__ void ctr_dense_bwd_weight(const float *gout, int O, const float *in, int K,
                                                     float *__restrict__ p, int t)
{
    const int to = (O + 3) / 4, tk = (K + 3) / 4;
    const bool v4 = ((O | K) & 3) == 0;
    for (int it = t; it < to * tk; it += kCtrThreads) {
        const int o0 = 4 * (it / tk), k0 = 4 * (it % tk);
        float acc[4][4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) acc[i][j] = 0.f;
        if (v4) {
            // two 16-byte LDS reads per sample feed 16 FMAs
#pragma unroll 4
            for (int s = 0; s < kCtrBS; ++s) {
                const float4 g = *(const float4 *)(gout + s * O + o0);
                const float4 x = *(const float4 *)(in + s * K + k0);
                const float gv[4] = {g.x, g.y, g.z, g.w}, xv[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(gv[i], xv[j], acc[i][j]);
            }
        } else {
#pragma unroll 4
            for (int s = 0; s < kCtrBS; ++s) {
                float g[4], x[4];
#pragma unroll
                for (int i = 0; i < 4; ++i) g[i] = o0 + i < O ? gout[s * O + o0 + i] : 0.f;
#pragma unroll
                for (int j = 0; j < 4; ++j) x[j] = k0 + j < K ? in[s * K + k0 + j] : 0.f;
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(g[i], x[j], acc[i][j]);
            }
        }
        if (v4) {
            // a row of the tile is 16 contiguous bytes; across the lanes of a
            // wave (consecutive k0) the stores are contiguous
#pragma unroll
            for (int i = 0; i < 4; ++i)
                *(float4 *)(p + (o0 + i) * K + k0) = make_float4(acc[i][0], acc[i][1], acc[i][2], acc[i][3]);
        } else {
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    if (o0 + i < O && k0 + j < K) p[(o0 + i) * K + k0 + j] = acc[i][j];
        }
    }
    for (int o = t; o < O; o += kCtrThreads) {
        float acc = 0.f;
#pragma unroll
        for (int s = 0; s < kCtrBS; ++s) acc += gout[s * O + o];
        p[O * K + o] = acc;
    }
}

// LDS of one net for a block of kCtrBS samples: act (every layer's
// activations, [kCtrBS][dims[l]] each, the input fields first) and grd (the
// loss gradient of each act[l]; with PReLU a hidden layer's slot holds its
// pre-activations between the forward and the backward).
__host__ __device__ inline int ctr_act_floats(const CtrArgs &a)
{
    int n = 0;
    for (int l = 0; l <= a.L; ++l) n += kCtrBS * a.dims[l];
    return n;
}

// scr: the parts of narrow layers, forward and backward.
__host__ __device__ inline int ctr_scr_floats(const CtrArgs &a)
{
    int n = 0;
    for (int l = 0; l < a.L; ++l) {
        const int K = a.dims[l], O = a.dims[l + 1];
        const int pf = ctr_fwd_parts(K, O), pb = ctr_bwd_parts(K, O);
        if (pf > 1 && pf * kCtrBS * O > n) n = pf * kCtrBS * O;
        if (pb > 1 && pb * kCtrBS * K > n) n = pb * kCtrBS * K;
    }
    return n;
}

struct NetLds {
    float *act, *grd;
    int off[kCtrMaxLayers + 1];
};

__device__ __forceinline__ NetLds net_lds(const CtrArgs &a, float *base)
{
    NetLds n;
    n.act = base;
    n.grd = base + ctr_act_floats(a);
    n.off[0] = 0;
    for (int l = 0; l < a.L; ++l) n.off[l + 1] = n.off[l] + kCtrBS * a.dims[l];
    return n;
}

// input fields, concatenated; rows past B read 0
__device__ __forceinline__ void net_load(const CtrArgs &a, const NetLds &n, int b0, int B, int t)
{
    const int K0 = a.dims[0];
    int c0 = 0;
    for (int f = 0; f < a.n_fields; ++f) {
        const int w = a.fdim[f];
        for (int e = t; e < kCtrBS * w; e += kCtrThreads) {
            const int s = e / w, k = e % w;
            n.act[s * K0 + c0 + k] = (b0 + s < B) ? a.field[f][(size_t)(b0 + s) * w + k] : 0.f;
        }
        c0 += w;
    }
}

// Every layer in turn (the caller synchronises before: act[0] loaded).
__device__ __forceinline__ void net_forward(const CtrArgs &a, const NetLds &n, float *scr, int t)
{
    for (int l = 0; l < a.L; ++l) {
        const bool hidden = l < a.L - 1;
        ctr_dense_fwd(n.act + n.off[l], a.dims[l], n.act + n.off[l + 1], a.dims[l + 1], a.W[l], a.b[l], hidden,
                      hidden ? a.slope[l] : nullptr, n.grd + n.off[l + 1], scr, t);
        __syncthreads();
    }
}

// From the loss gradient of the last layer's output (in grd, synchronised):
// each layer's weight, bias and slope gradients over the block's samples into
// the partial row p, and the gradient of the input fields into grd[0].
__device__ __forceinline__ void net_backward(const CtrArgs &a, const NetLds &n, float *scr, float *p, int t)
{
    int wo[kCtrMaxLayers];
    int woff = 0;
    for (int l = 0; l < a.L; ++l) {
        wo[l] = woff;
        woff += net_layer_size(a, l);
    }
    for (int l = a.L - 1; l >= 0; --l) {
        const int K = a.dims[l], O = a.dims[l + 1];
        const float *gout = n.grd + n.off[l + 1], *in = n.act + n.off[l];
        ctr_dense_bwd_weight(gout, O, in, K, p + wo[l], t);
        // the activation below layer l belongs to layer l - 1: its slot
        // follows that layer's dW and db
        float *dsl = l > 0 ? p + wo[l - 1] + K * a.dims[l - 1] + K : nullptr;
        ctr_dense_bwd_data(gout, O, n.grd + n.off[l], in, K, a.W[l], l > 0, l > 0 ? a.slope[l - 1] : nullptr, dsl,
                           scr, t);
        __syncthreads();
    }
}

__device__ __forceinline__ void net_store_dfields(const CtrArgs &a, const NetLds &n, int b0, int B, int t)
{
    const int K0 = a.dims[0];
    int c0 = 0;
    for (int f = 0; f < a.n_fields; ++f) {
        const int w = a.fdim[f];
        if (a.dfield[f])
            for (int e = t; e < kCtrBS * w; e += kCtrThreads) {
                const int s = e / w, k = e % w;
                if (b0 + s < B) a.dfield[f][(size_t)(b0 + s) * w + k] = n.grd[s * K0 + c0 + k];
            }
        c0 += w;
    }
}

inline size_t ctr_lds_bytes(const CtrArgs &a)
{
    return (size_t)(2 * ctr_act_floats(a) + ctr_scr_floats(a) + kCtrBS) * 4;
}

// One block = kCtrBS samples: forward through every layer in LDS, softmax
// and cross-entropy, then the backward; the block's gradient and loss sums
// (over its samples, ascending) go to its partial row.
__global__ __launch_bounds__(kCtrThreads) void ctr_fb_k(CtrArgs a, int B, const int32_t *__restrict__ labels,
                                                     float *__restrict__ prob, float *__restrict__ part, int PS)
{
    extern __shared__ float lds[];
    const NetLds n = net_lds(a, lds);
    float *scr = lds + 2 * ctr_act_floats(a);
    float *lossv = scr + ctr_scr_floats(a);
    const int t = threadIdx.x;
    const int b0 = blockIdx.x * kCtrBS;
    const int L = a.L, C = a.dims[L];
    net_load(a, n, b0, B, t);
    __syncthreads();
    net_forward(a, n, scr, t);
    // softmax, cross-entropy, dlogits = (p - onehot(y)) / B
    if (t < kCtrBS) {
        const int s = t, i = b0 + s;
        const float *z = n.act + n.off[L] + s * C;
        float *gz = n.grd + n.off[L] + s * C;
        float ls = 0.f;
        const int y = i < B ? labels[i] : -1;
        if (i < B && y >= 0 && y < C) {
            float m = z[0];
            for (int c = 1; c < C; ++c) m = fmaxf(m, z[c]);
            float se = 0.f;
            for (int c = 0; c < C; ++c) se += expf(z[c] - m);
            const float lse = m + logf(se);
            for (int c = 0; c < C; ++c) {
                const float pc = expf(z[c] - lse);
                if (prob) prob[(size_t)i * C + c] = pc;
                gz[c] = (pc - (c == y ? 1.f : 0.f)) / (float)B;
            }
            ls = lse - z[y];
        } else {
            for (int c = 0; c < C; ++c) gz[c] = 0.f;
            if (i < B && prob)
                for (int c = 0; c < C; ++c) prob[(size_t)i * C + c] = 0.f;
        }
        lossv[s] = ls;
    }
    __syncthreads();
    float *p = part + (size_t)blockIdx.x * PS;
    net_backward(a, n, scr, p, t);
    net_store_dfields(a, n, b0, B, t);
    if (t == 0) {
        float ls = 0.f;
        for (int s = 0; s < kCtrBS; ++s) ls += lossv[s];
        p[PS - 4] = ls;
    }
}

// Pre-rank model (section 6): a user tower and an ad tower on their own
// fields, score s = <u, a> of their outputs, click probability sigmoid(s),
// logistic loss softplus(s) - y s for y in {0, 1} (other labels add
// nothing), divided by B.  Same block layout as the CTR kernel with both
// towers in LDS; the partial row holds the user tower's gradients, then the
// ad tower's, then the loss sum.
__global__ __launch_bounds__(kCtrThreads) void dssm_fb_k(CtrArgs u, CtrArgs v, int B, const int32_t *__restrict__ labels,
                                                      float *__restrict__ prob, float *__restrict__ part, int PS)
{
    extern __shared__ float lds[];
    const NetLds nu = net_lds(u, lds);
    const NetLds nv = net_lds(v, lds + 2 * ctr_act_floats(u));
    float *scr = lds + 2 * ctr_act_floats(u) + 2 * ctr_act_floats(v);
    float *lossv = scr + max(ctr_scr_floats(u), ctr_scr_floats(v));
    const int t = threadIdx.x;
    const int b0 = blockIdx.x * kCtrBS;
    const int R = u.dims[u.L];
    net_load(u, nu, b0, B, t);
    net_load(v, nv, b0, B, t);
    __syncthreads();
    net_forward(u, nu, scr, t);
    net_forward(v, nv, scr, t);
    if (t < kCtrBS) {
        const int s = t, i = b0 + s;
        const float *zu = nu.act + nu.off[u.L] + s * R, *zv = nv.act + nv.off[v.L] + s * R;
        float sc = 0.f;
        for (int r = 0; r < R; ++r) sc = fmaf(zu[r], zv[r], sc);
        const float pr = 1.f / (1.f + expf(-sc));
        const int y = i < B ? labels[i] : -1;
        float ls = 0.f, g = 0.f;
        if (i < B) {
            if (prob) prob[i] = pr;
            if (y == 0 || y == 1) {
                ls = fmaxf(sc, 0.f) + log1pf(expf(-fabsf(sc))) - (float)y * sc;
                g = (pr - (float)y) / (float)B;
            }
        }
        float *gu = nu.grd + nu.off[u.L] + s * R, *gv = nv.grd + nv.off[v.L] + s * R;
        for (int r = 0; r < R; ++r) {
            gu[r] = g * zv[r];
            gv[r] = g * zu[r];
        }
        lossv[s] = ls;
    }
    __syncthreads();
    float *p = part + (size_t)blockIdx.x * PS;
    net_backward(u, nu, scr, p, t);
    net_backward(v, nv, scr, p + net_part_size(u), t);
    net_store_dfields(u, nu, b0, B, t);
    net_store_dfields(v, nv, b0, B, t);
    if (t == 0) {
        float ls = 0.f;
        for (int s = 0; s < kCtrBS; ++s) ls += lossv[s];
        p[PS - 4] = ls;
    }
}

// Where the reduced partial rows go: per layer (of one net, or of the two
// towers one after the other) dW, db and, below a net's last layer, the
// slope gradient (NULL: not stored), at the offsets of the partial row; the loss sum sits at PS - 4.
struct RedLayer {
    int off, K, O, hidden;
    float *dW, *db, *ds;
};

struct CtrOut {
    int nl;
    RedLayer ly[2 * kCtrMaxLayers];
    float *loss;
    int B;
};

// Fixed-order sum of the blocks' partial rows, scattered into the gradients
// and the mean loss.  A block takes 64 elements; wave q of its 4 sums the
// q-th quarter of the G rows (eight running chains over g = 8 i + r, added
// r = 0..7), and the quarters are added in order.
constexpr int kRedCols = kThreads / 4;

__global__ __launch_bounds__(kThreads) void ctr_reduce_k(const float *__restrict__ part, int G, int PS, CtrOut o)
{
    __shared__ float q4[4][kRedCols];
    const int c = threadIdx.x % kRedCols, qt = threadIdx.x / kRedCols;
    const int e = blockIdx.x * kRedCols + c;
    const int g0 = (int)((int64_t)qt * G / 4), g1 = (int)((int64_t)(qt + 1) * G / 4);
    float s[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    if (e < PS) {
        int g = g0;
        for (; g + 8 <= g1; g += 8)
#pragma unroll
            for (int r = 0; r < 8; ++r) s[r] += part[(size_t)(g + r) * PS + e];
        for (int r = 0; g + r < g1; ++r) s[r] += part[(size_t)(g + r) * PS + e];
    }
    float sub = 0.f;
#pragma unroll
    for (int r = 0; r < 8; ++r) sub += s[r];
    q4[qt][c] = sub;
    __syncthreads();
    if (qt != 0 || e >= PS) return;
    const float tot = ((q4[0][c] + q4[1][c]) + q4[2][c]) + q4[3][c];
    if (e == PS - 4) {
        *o.loss = tot / (float)o.B;
        return;
    }
    for (int l = 0; l < o.nl; ++l) {
        const RedLayer &y = o.ly[l];
        int x = e - y.off;
        if (x < 0) return;                     // padding before this layer
        const int nw = y.O * y.K;
        if (x < nw) {
            y.dW[x] = tot;
            return;
        }
        x -= nw;
        if (x < y.O) {
            y.db[x] = tot;
            return;
        }
        x -= y.O;
        if (y.hidden && x < y.O) {
            if (y.ds) y.ds[x] = tot;
            return;
        }
    }
}

// ---------------------------------------------------------------- Adagrad

// One thread per 4 elements of a touched row when D % 4 == 0 and the arrays
// are 16-byte aligned (vec4), else per element; a grid-stride loop over the
// n_u rows the device counted (the grid is sized for at most kAdaBlocks, not
// for the host cap, whose blocks past n_u would each still be dispatched).
constexpr int kAdaBlocks = 2048;
__device__ __forceinline__ float ada_one(float p, float g, float &a, float lr, float eps)
{
    a = a + g * g;
    return p - lr * g / (sqrtf(a) + eps);
}

__global__ __launch_bounds__(kThreads) void adagrad_k(int D, const int32_t *__restrict__ uniq,
                                                      const int32_t *__restrict__ n_uniq_p, int cap,
                                                      const float *__restrict__ grad, float *__restrict__ table,
                                                      int64_t n_rows, float *__restrict__ accum, float lr, float eps,
                                                      int vec4)
{
    const int n_u = min(*n_uniq_p, cap);
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    if (vec4) {
        const int D4 = D / 4;
        const int64_t n4 = (int64_t)n_u * D4;
        for (int64_t e = (int64_t)blockIdx.x * kThreads + threadIdx.x; e < n4; e += stride) {
            const int u = (int)(e / D4), d = (int)(e % D4) * 4;
            const int r = uniq[u];
            if (r < 0 || (int64_t)r >= n_rows) continue;
            const float4 g = *(const float4 *)(grad + (size_t)u * D + d);
            const size_t x = (size_t)r * D + d;
            float4 a = *(const float4 *)(accum + x), t = *(const float4 *)(table + x);
            t.x = ada_one(t.x, g.x, a.x, lr, eps);
            t.y = ada_one(t.y, g.y, a.y, lr, eps);
            t.z = ada_one(t.z, g.z, a.z, lr, eps);
            t.w = ada_one(t.w, g.w, a.w, lr, eps);
            *(float4 *)(accum + x) = a;
            *(float4 *)(table + x) = t;
        }
    } else {
        const int64_t n = (int64_t)n_u * D;
        for (int64_t e = (int64_t)blockIdx.x * kThreads + threadIdx.x; e < n; e += stride) {
            const int u = (int)(e / D), d = (int)(e % D);
            const int r = uniq[u];
            if (r < 0 || (int64_t)r >= n_rows) continue;
            const size_t x = (size_t)r * D + d;
            float a = accum[x];
            table[x] = ada_one(table[x], grad[e], a, lr, eps);
            accum[x] = a;
        }
    }
}

// ------------------------------------------------------------------- Adam

struct AdamK {
    float lr, b1, b2, eps, c1, c2;
};

__device__ __forceinline__ float adam_one(float p, float g, float &m, float &v, const AdamK &k)
{
    m = k.b1 * m + (1.f - k.b1) * g;
    v = k.b2 * v + (1.f - k.b2) * g * g;
    return p - k.lr * (m / k.c1) / (sqrtf(v / k.c2) + k.eps);
}

// Scalar form: any alignment.
__global__ __launch_bounds__(kThreads) void adam_k(int64_t n, float *__restrict__ param,
                                                   const float *__restrict__ grad, float *__restrict__ m,
                                                   float *__restrict__ v, AdamK k, uint16_t *__restrict__ pb)
{
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n; i += (int64_t)gridDim.x * kThreads) {
        float mi = m[i], vi = v[i];
        const float p = adam_one(param[i], grad[i], mi, vi, k);
        m[i] = mi;
        v[i] = vi;
        param[i] = p;
        if (pb) pb[i] = ams_f32_to_bf16(p);
    }
}

// 16-byte form (param, grad, m, v 16-byte aligned, the bf16 copy 8-byte
// aligned): quad q = elements 4q..4q+3; the n % 4 last elements go to the
// first threads of the grid.  Same arithmetic per element as adam_k.
__global__ __launch_bounds__(kThreads) void adam4_k(int64_t n, float *__restrict__ param,
                                                    const float *__restrict__ grad, float *__restrict__ m,
                                                    float *__restrict__ v, AdamK k, uint16_t *__restrict__ pb)
{
    const int64_t nq = n / 4, t0 = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    for (int64_t q = t0; q < nq; q += (int64_t)gridDim.x * kThreads) {
        const float4 g = ((const float4 *)grad)[q];
        float4 p = ((float4 *)param)[q], mm = ((float4 *)m)[q], vv = ((float4 *)v)[q];
        p.x = adam_one(p.x, g.x, mm.x, vv.x, k);
        p.y = adam_one(p.y, g.y, mm.y, vv.y, k);
        p.z = adam_one(p.z, g.z, mm.z, vv.z, k);
        p.w = adam_one(p.w, g.w, mm.w, vv.w, k);
        ((float4 *)param)[q] = p;
        ((float4 *)m)[q] = mm;
        ((float4 *)v)[q] = vv;
        if (pb)
            ((uint2 *)pb)[q] = make_uint2((uint32_t)ams_f32_to_bf16(p.x) | ((uint32_t)ams_f32_to_bf16(p.y) << 16),
                                          (uint32_t)ams_f32_to_bf16(p.z) | ((uint32_t)ams_f32_to_bf16(p.w) << 16));
    }
    const int64_t i = 4 * nq + t0;
    if (i < n) {
        float mi = m[i], vi = v[i];
        const float p = adam_one(param[i], grad[i], mi, vi, k);
        m[i] = mi;
        v[i] = vi;
        param[i] = p;
        if (pb) pb[i] = ams_f32_to_bf16(p);
    }
}

size_t al256(size_t x) { return (x + 255) & ~(size_t)255; }

// Widths a net of the CTR kind accepts: 1..kCtrMaxLayers layers, inputs up
// to kCtrMaxIn, hidden widths up to kCtrMaxHidden; the output width is
// checked by the caller (classes, or a tower's representation).
bool net_dims_ok(const ams_ctr *net, int min_layers)
{
    if (!net || net->n_layers < min_layers || net->n_layers > kCtrMaxLayers) return false;
    if (net->dims[0] < 1 || net->dims[0] > kCtrMaxIn) return false;
    for (int l = 1; l < net->n_layers; ++l)
        if (net->dims[l] < 1 || net->dims[l] > kCtrMaxHidden) return false;
    return true;
}

bool ctr_ok(const ams_ctr *net)
{
    if (!net_dims_ok(net, 2)) return false;
    const int C = net->dims[net->n_layers];
    return C >= 2 && C <= kCtrMaxC;
}

bool tower_ok(const ams_ctr *net)
{
    if (!net_dims_ok(net, 1)) return false;
    const int R = net->dims[net->n_layers];
    return R >= 1 && R <= kTowerMaxOut;
}

// LDS a block may have on the current device (gfx950's 160 KiB if it cannot
// be asked).
size_t lds_limit()
{
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&n, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess || n <= 0)
        n = 160 * 1024;
    return (size_t)n;
}

// Fill a net's arguments; NULL pointers where the ABI requires them give NULL.
ams_status net_args(const ams_ctr *net, int32_t n_fields, const float *const *fields, const int32_t *field_dims,
                    const float *const *W, const float *const *b, const float *const *slope,
                    float *const *dfields, CtrArgs &a)
{
    if (!fields || !field_dims || !W || !b) return AMS_ERR_NULL;
    if (n_fields < 1 || n_fields > kCtrMaxFields) return AMS_ERR_DIMS;
    a = CtrArgs{};
    a.L = net->n_layers;
    for (int l = 0; l <= a.L; ++l) a.dims[l] = net->dims[l];
    a.n_fields = n_fields;
    int width = 0;
    for (int f = 0; f < n_fields; ++f) {
        if (field_dims[f] < 1) return AMS_ERR_DIMS;
        if (!fields[f]) return AMS_ERR_NULL;
        a.fdim[f] = field_dims[f];
        a.field[f] = fields[f];
        a.dfield[f] = dfields ? dfields[f] : nullptr;
        width += field_dims[f];
    }
    if (width != a.dims[0]) return AMS_ERR_DIMS;
    for (int l = 0; l < a.L; ++l) {
        if (!W[l] || !b[l]) return AMS_ERR_NULL;
        a.W[l] = W[l];
        a.b[l] = b[l];
        a.slope[l] = (slope && l < a.L - 1) ? slope[l] : nullptr;
    }
    return AMS_OK;
}

// Reduction targets of one net's layers, appended to o.
// base: where this net's part of the partial row starts.
ams_status net_out(const CtrArgs &a, float *const *dW, float *const *db, float *const *dslope, int base, CtrOut &o)
{
    if (!dW || !db) return AMS_ERR_NULL;
    for (int l = 0; l < a.L; ++l) {
        if (!dW[l] || !db[l]) return AMS_ERR_NULL;
        RedLayer &y = o.ly[o.nl++];
        y.off = base;
        base += net_layer_size(a, l);
        y.K = a.dims[l];
        y.O = a.dims[l + 1];
        y.hidden = l < a.L - 1;
        y.dW = dW[l];
        y.db = db[l];
        y.ds = (y.hidden && dslope && a.slope[l]) ? dslope[l] : nullptr;
    }
    return AMS_OK;
}

}  // namespace

extern "C" ams_status ams_bag_fwd(int32_t B, int32_t D, const int32_t *seg_off, int64_t n_beh,
                                  const int32_t *ids, const float *table, int64_t n_rows, float *bag, void *stream)
{
    if (B < 0 || n_beh < 0 || n_beh > INT32_MAX || n_rows < 0) return AMS_ERR_SIZE;
    if (D < 1 || D > 32) return AMS_ERR_DIMS;
    if (B == 0) return AMS_OK;
    if (!seg_off || !ids || !table || !bag) return AMS_ERR_NULL;
    hipStream_t st = (hipStream_t)stream;
    const int grid = (B + kWaves - 1) / kWaves;
    if (D <= 16)
        AMS_LAUNCH("bag_fwd", st, bag_fwd_k<16><<<grid, kThreads, 0, st>>>(B, D, seg_off, n_beh, ids, table, n_rows, bag));
    else
        AMS_LAUNCH("bag_fwd", st, bag_fwd_k<32><<<grid, kThreads, 0, st>>>(B, D, seg_off, n_beh, ids, table, n_rows, bag));
    return ams_launch_status();
}

extern "C" size_t ams_bag_workspace(int32_t B, int64_t n_beh, int32_t D, int32_t n_uniq_cap)
{
    return ams_pool_workspace(AMS_POOL_SUM, B, n_beh, D, n_uniq_cap);
}

extern "C" ams_status ams_bag_bwd(int32_t B, int32_t D, const int32_t *seg_off, int64_t n_beh, const int32_t *inv,
                                  const int32_t *occ_perm, const int32_t *uniq_off, const int32_t *n_uniq,
                                  int32_t n_uniq_cap, const float *dbag, const float *dad, float *grad, void *ws,
                                  size_t ws_bytes, void *stream)
{
    (void)n_uniq;
    if (B > 0 && !dbag) return AMS_ERR_NULL;
    // the SUM aggregator's backward with the bag gradient as the upstream
    // gradient of behaviors and ads alike, the ads also taking dad
    return pool_bwd_sum_ads(B, D, seg_off, n_beh, inv, occ_perm, uniq_off, n_uniq_cap, dbag, dbag, dad, grad, ws,
                            ws_bytes, stream);
}

extern "C" size_t ams_ctr_workspace(const ams_ctr *net, int32_t B)
{
    if (!ctr_ok(net) || B < 0) return 0;
    CtrArgs a{};
    a.L = net->n_layers;
    for (int l = 0; l <= a.L; ++l) a.dims[l] = net->dims[l];
    const int G = (B + kCtrBS - 1) / kCtrBS;
    return al256((size_t)(G > 0 ? G : 1) * (net_part_size(a) + 4) * 4);
}

extern "C" ams_status ams_ctr_fwd_bwd(const ams_ctr *net, int32_t B, int32_t n_fields, const float *const *fields,
                                      const int32_t *field_dims, const int32_t *labels, const float *const *W,
                                      const float *const *b, const float *const *slope, float *loss, float *prob,
                                      float *const *dW, float *const *db, float *const *dslope,
                                      float *const *dfields, void *ws, size_t ws_bytes, void *stream)
{
    if (!net) return AMS_ERR_NULL;
    if (!ctr_ok(net)) return AMS_ERR_DIMS;
    if (B < 1) return AMS_ERR_SIZE;
    CtrArgs a;
    ams_status s = net_args(net, n_fields, fields, field_dims, W, b, slope, dfields, a);
    if (s != AMS_OK) return s;
    CtrOut o{};
    s = net_out(a, dW, db, dslope, 0, o);
    if (s != AMS_OK) return s;
    if (!labels || !loss) return AMS_ERR_NULL;
    const size_t lds = ctr_lds_bytes(a);
    if (lds > lds_limit()) return AMS_ERR_DIMS;
    const int G = (B + kCtrBS - 1) / kCtrBS;
    const int PS = net_part_size(a) + 4;
    if (!ws || ws_bytes < (size_t)G * PS * 4) return AMS_ERR_WORKSPACE;
    hipStream_t st = (hipStream_t)stream;
    float *part = (float *)ws;
    AMS_LAUNCH("ctr_fwd_bwd", st, ctr_fb_k<<<G, kCtrThreads, lds, st>>>(a, B, labels, prob, part, PS));
    o.loss = loss;
    o.B = B;
    AMS_LAUNCH("ctr_reduce", st, ctr_reduce_k<<<(PS + kRedCols - 1) / kRedCols, kThreads, 0, st>>>(part, G, PS, o));
    return ams_launch_status();
}

extern "C" size_t ams_dssm_workspace(const ams_ctr *user_net, const ams_ctr *ad_net, int32_t B)
{
    if (!tower_ok(user_net) || !tower_ok(ad_net) || B < 0) return 0;
    CtrArgs u{}, v{};
    u.L = user_net->n_layers;
    v.L = ad_net->n_layers;
    for (int l = 0; l <= u.L; ++l) u.dims[l] = user_net->dims[l];
    for (int l = 0; l <= v.L; ++l) v.dims[l] = ad_net->dims[l];
    const int G = (B + kCtrBS - 1) / kCtrBS;
    return al256((size_t)(G > 0 ? G : 1) * (net_part_size(u) + net_part_size(v) + 4) * 4);
}

extern "C" ams_status ams_dssm_fwd_bwd(const ams_ctr *user_net, const ams_ctr *ad_net, int32_t B,
                                       int32_t n_user_fields, const float *const *user_fields,
                                       const int32_t *user_field_dims, int32_t n_ad_fields,
                                       const float *const *ad_fields, const int32_t *ad_field_dims,
                                       const int32_t *labels, const float *const *Wu, const float *const *bu,
                                       const float *const *slope_u, const float *const *Wa,
                                       const float *const *ba, const float *const *slope_a, float *loss,
                                       float *prob, float *const *dWu, float *const *dbu,
                                       float *const *dslope_u, float *const *dWa, float *const *dba,
                                       float *const *dslope_a, float *const *duser_fields,
                                       float *const *dad_fields, void *ws, size_t ws_bytes, void *stream)
{
    if (!user_net || !ad_net) return AMS_ERR_NULL;
    if (!tower_ok(user_net) || !tower_ok(ad_net)) return AMS_ERR_DIMS;
    if (user_net->dims[user_net->n_layers] != ad_net->dims[ad_net->n_layers]) return AMS_ERR_DIMS;
    if (B < 1) return AMS_ERR_SIZE;
    CtrArgs u, v;
    ams_status s = net_args(user_net, n_user_fields, user_fields, user_field_dims, Wu, bu, slope_u, duser_fields, u);
    if (s != AMS_OK) return s;
    s = net_args(ad_net, n_ad_fields, ad_fields, ad_field_dims, Wa, ba, slope_a, dad_fields, v);
    if (s != AMS_OK) return s;
    CtrOut o{};
    s = net_out(u, dWu, dbu, dslope_u, 0, o);
    if (s != AMS_OK) return s;
    s = net_out(v, dWa, dba, dslope_a, net_part_size(u), o);
    if (s != AMS_OK) return s;
    if (!labels || !loss) return AMS_ERR_NULL;
    const size_t lds = (size_t)(2 * ctr_act_floats(u) + 2 * ctr_act_floats(v) +
                                max(ctr_scr_floats(u), ctr_scr_floats(v)) + kCtrBS) * 4;
    if (lds > lds_limit()) return AMS_ERR_DIMS;
    const int G = (B + kCtrBS - 1) / kCtrBS;
    const int PS = net_part_size(u) + net_part_size(v) + 4;
    if (!ws || ws_bytes < (size_t)G * PS * 4) return AMS_ERR_WORKSPACE;
    hipStream_t st = (hipStream_t)stream;
    float *part = (float *)ws;
    AMS_LAUNCH("dssm_fwd_bwd", st, dssm_fb_k<<<G, kCtrThreads, lds, st>>>(u, v, B, labels, prob, part, PS));
    o.loss = loss;
    o.B = B;
    AMS_LAUNCH("ctr_reduce", st, ctr_reduce_k<<<(PS + kRedCols - 1) / kRedCols, kThreads, 0, st>>>(part, G, PS, o));
    return ams_launch_status();
}

extern "C" ams_status ams_adagrad_rows(int32_t D, const int32_t *uniq, const int32_t *n_uniq, int32_t n_uniq_cap,
                                       const float *grad, float *table, int64_t n_rows, float *accum, float lr,
                                       float eps, void *stream)
{
    if (D < 1 || n_uniq_cap < 0 || n_rows < 0) return AMS_ERR_SIZE;
    if (n_uniq_cap == 0) return AMS_OK;
    if (!uniq || !n_uniq || !grad || !table || !accum) return AMS_ERR_NULL;
    hipStream_t st = (hipStream_t)stream;
    const int vec4 = (D % 4 == 0) && ((((uintptr_t)grad) | ((uintptr_t)table) | ((uintptr_t)accum)) & 15) == 0;
    const int64_t n = (int64_t)n_uniq_cap * (vec4 ? D / 4 : D);
    const int64_t g = (n + kThreads - 1) / kThreads;
    AMS_LAUNCH("adagrad_rows", st, adagrad_k<<<(unsigned)(g < kAdaBlocks ? g : kAdaBlocks), kThreads, 0, st>>>(
                                       D, uniq, n_uniq, n_uniq_cap, grad, table, n_rows, accum, lr, eps, vec4));
    return ams_launch_status();
}

extern "C" ams_status ams_adam_update(int64_t n, float *param, const float *grad, float *m, float *v, float lr,
                                      float b1, float b2, float eps, int64_t t, uint16_t *param_bf16, void *stream)
{
    if (n < 0 || t < 1) return AMS_ERR_SIZE;
    if (n == 0) return AMS_OK;
    if (!param || !grad || !m || !v) return AMS_ERR_NULL;
    // bias corrections of step t, formed in double on the host
    AdamK k{lr, b1, b2, eps, (float)(1.0 - pow((double)b1, (double)t)), (float)(1.0 - pow((double)b2, (double)t))};
    hipStream_t st = (hipStream_t)stream;
    const bool v4 = ((((uintptr_t)param | (uintptr_t)grad | (uintptr_t)m | (uintptr_t)v) & 15) == 0) &&
                    (((uintptr_t)param_bf16 & 7) == 0);
    const int64_t work = v4 ? (n + 3) / 4 : n;
    int64_t g = (work + kThreads - 1) / kThreads;
    if (g > 4096) g = 4096;
    if (v4)
        AMS_LAUNCH("adam_update", st, adam4_k<<<(unsigned)g, kThreads, 0, st>>>(n, param, grad, m, v, k, param_bf16));
    else
        AMS_LAUNCH("adam_update", st, adam_k<<<(unsigned)g, kThreads, 0, st>>>(n, param, grad, m, v, k, param_bf16));
    return ams_launch_status();
}
