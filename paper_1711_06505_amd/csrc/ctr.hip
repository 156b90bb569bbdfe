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
constexpr int kCtrMaxIn = 128, kCtrMaxHidden = 256, kCtrMaxC = 8;
constexpr int kCtrMaxLayers = 3, kCtrMaxFields = 8;

// ------------------------------------------------------------ bag forward

// One wave per sample: lane l adds the rows of behaviors l, l + 64, ...;
// the lanes' partial rows are summed by a fixed butterfly, then the ad row.
// An ID outside [0, n_rows) reads as a zero row (dedup reports it).
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
    const bool vec4 = (D & 3) == 0;
    for (int j = j0 + lane; j < j1; j += AMS_WAVE) {
        const int id = ids[j];
        if (id < 0 || (int64_t)id >= n_rows) continue;
        const float *r = table + (size_t)id * D;
        if (vec4) {
#pragma unroll
            for (int d4 = 0; d4 < DM / 4; ++d4)
                if (4 * d4 < D) {
                    const float4 v = *(const float4 *)(r + 4 * d4);
                    acc[4 * d4] += v.x;
                    acc[4 * d4 + 1] += v.y;
                    acc[4 * d4 + 2] += v.z;
                    acc[4 * d4 + 3] += v.w;
                }
        } else {
#pragma unroll
            for (int d = 0; d < DM; ++d)
                if (d < D) acc[d] += r[d];
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
    int L;                                   // layers (2 or 3)
    int dims[kCtrMaxLayers + 1];
    int n_fields;
    int fdim[kCtrMaxFields];
    const float *field[kCtrMaxFields];
    float *dfield[kCtrMaxFields];
    const float *W[kCtrMaxLayers];
    const float *b[kCtrMaxLayers];
};

__host__ __device__ inline int ctr_part_size(const CtrArgs &a)
{
    int n = 1;                               // + the block's loss sum
    for (int l = 0; l < a.L; ++l) n += a.dims[l + 1] * a.dims[l] + a.dims[l + 1];
    return n;
}

// Parts of a layer split over threads: forward P * kCtrBS * O, backward-data
// P * kCtrBS * K (P is chosen as in ctr_dense_fwd / ctr_dense_bwd_data).
__host__ __device__ inline int ctr_fwd_parts(int K, int O)
{
    int P = kThreads / O;
    if (P < 1) P = 1;
    if (P > (K + 15) / 16) P = (K + 15) / 16;
    return P;
}

__host__ __device__ inline int ctr_bwd_parts(int K, int O)
{
    int P = kThreads / K;
    if (P < 1) P = 1;
    if (P > (O + 7) / 8) P = (O + 7) / 8;
    return P;
}

// out[s][o] = bias[o] + sum_k in[s][k] W[o][k] (ReLU'd unless last) for the
// block's kCtrBS samples.  Work item (o, part p of P): the K range of part p
// (a multiple of 4 wide), its W row streamed in float4 runs of 16, all
// samples accumulated together (in[s][k] is the same LDS word for the whole
// wave: a broadcast).  With P > 1 (narrow layers) the parts go to `scr`
// [P][kCtrBS][O] and are added in part order.
__device__ __forceinline__ void ctr_dense_fwd(const float *in, int K, float *out, int O, const float *__restrict__ W,
                                              const float *__restrict__ bias, bool relu, float *scr, int t)
{
    const int P = ctr_fwd_parts(K, O);
    const int KC = (((K + P - 1) / P) + 3) & ~3;
    for (int it = t; it < O * P; it += kThreads) {
        const int o = it % O, pp = it / O;
        const int k0 = pp * KC, k1 = min(K, k0 + KC);
        float acc[kCtrBS];
#pragma unroll
        for (int s = 0; s < kCtrBS; ++s) acc[s] = 0.f;
        const float *wr = W + (size_t)o * K;
        const bool v4 = (K & 3) == 0;
        for (int kb = k0; kb < k1; kb += 16) {
            float w[16];
            if (v4 && kb + 16 <= k1) {
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const float4 x = *(const float4 *)(wr + kb + 4 * q);
                    w[4 * q] = x.x;
                    w[4 * q + 1] = x.y;
                    w[4 * q + 2] = x.z;
                    w[4 * q + 3] = x.w;
                }
            } else {
#pragma unroll
                for (int q = 0; q < 16; ++q) w[q] = kb + q < k1 ? wr[kb + q] : 0.f;
            }
#pragma unroll
            for (int q = 0; q < 16; ++q) {
                if (kb + q >= k1) break;
#pragma unroll
                for (int s = 0; s < kCtrBS; ++s) acc[s] = fmaf(in[s * K + kb + q], w[q], acc[s]);
            }
        }
        if (P == 1) {
            const float bo = bias[o];
#pragma unroll
            for (int s = 0; s < kCtrBS; ++s) {
                const float v = acc[s] + bo;
                out[s * O + o] = relu ? fmaxf(v, 0.f) : v;
            }
        } else {
#pragma unroll
            for (int s = 0; s < kCtrBS; ++s) scr[(pp * kCtrBS + s) * O + o] = acc[s];
        }
    }
    if (P > 1) {
        __syncthreads();
        for (int e = t; e < kCtrBS * O; e += kThreads) {
            const int o = e % O;
            float v = bias[o];
            for (int pp = 0; pp < P; ++pp) v += scr[pp * kCtrBS * O + e];
            out[e] = relu ? fmaxf(v, 0.f) : v;
        }
    }
}

// gin[s][k] = sum_o gout[s][o] W[o][k] (masked by [in > 0] when `mask`).
// Work item (k, part p of P over O); the lanes of a wave take consecutive k,
// so each W row read is contiguous across the wave; 8 rows in flight.  Parts
// are added in order through `scr` as in the forward.
__device__ __forceinline__ void ctr_dense_bwd_data(const float *gout, int O, float *gin, const float *in, int K,
                                                   const float *__restrict__ W, bool mask, float *scr, int t)
{
    const int P = ctr_bwd_parts(K, O);
    const int OC = (O + P - 1) / P;
    for (int it = t; it < K * P; it += kThreads) {
        const int k = it % K, pp = it / K;
        const int o0 = pp * OC, o1 = min(O, o0 + OC);
        float acc[kCtrBS];
#pragma unroll
        for (int s = 0; s < kCtrBS; ++s) acc[s] = 0.f;
        for (int ob = o0; ob < o1; ob += 8) {
            float w[8];
#pragma unroll
            for (int q = 0; q < 8; ++q) w[q] = ob + q < o1 ? W[(size_t)(ob + q) * K + k] : 0.f;
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                if (ob + q >= o1) break;
#pragma unroll
                for (int s = 0; s < kCtrBS; ++s) acc[s] = fmaf(gout[s * O + ob + q], w[q], acc[s]);
            }
        }
        if (P == 1) {
#pragma unroll
            for (int s = 0; s < kCtrBS; ++s) gin[s * K + k] = (!mask || in[s * K + k] > 0.f) ? acc[s] : 0.f;
        } else {
#pragma unroll
            for (int s = 0; s < kCtrBS; ++s) scr[(pp * kCtrBS + s) * K + k] = acc[s];
        }
    }
    if (P > 1) {
        __syncthreads();
        for (int e = t; e < kCtrBS * K; e += kThreads) {
            float v = 0.f;
            for (int pp = 0; pp < P; ++pp) v += scr[pp * kCtrBS * K + e];
            gin[e] = (!mask || in[e] > 0.f) ? v : 0.f;
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
    for (int it = t; it < to * tk; it += kThreads) {
        const int o0 = 4 * (it / tk), k0 = 4 * (it % tk);
        float acc[4][4];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) acc[i][j] = 0.f;
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
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if (o0 + i < O && k0 + j < K) p[(o0 + i) * K + k0 + j] = acc[i][j];
    }
    for (int o = t; o < O; o += kThreads) {
        float acc = 0.f;
#pragma unroll
        for (int s = 0; s < kCtrBS; ++s) acc += gout[s * O + o];
        p[O * K + o] = acc;
    }
}

// One block = kCtrBS samples: forward through every layer in LDS, softmax
// and cross-entropy, then the backward; the block's weight-gradient and loss
// sums (over its samples, ascending) go to its partial row.
// Dynamic LDS, sized by ctr_lds_floats for the actual widths: act (every
// layer's activations, [kCtrBS][dims[l]] each), grd (their loss gradients),
// scr (parts of narrow layers in the backward), the samples' losses.
__host__ __device__ inline int ctr_act_floats(const CtrArgs &a)
{
    int n = 0;
    for (int l = 0; l <= a.L; ++l) n += kCtrBS * a.dims[l];
    return n;
}

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

inline size_t ctr_lds_bytes(const CtrArgs &a)
{
    return (size_t)(2 * ctr_act_floats(a) + ctr_scr_floats(a) + kCtrBS) * 4;
}

__global__ __launch_bounds__(kThreads) void ctr_fb_k(CtrArgs a, int B, const int32_t *__restrict__ labels,
                                                     float *__restrict__ prob, float *__restrict__ part, int PS)
{
    extern __shared__ float lds[];
    const int na = ctr_act_floats(a);
    float *act = lds;                        // act[l]: [kCtrBS][dims[l]] per layer
    float *grd = lds + na;                   // the loss gradient of each act[l]
    float *scr = lds + 2 * na;               // parts of narrow layers in the backward
    float *lossv = scr + ctr_scr_floats(a);
    const int t = threadIdx.x;
    const int b0 = blockIdx.x * kCtrBS;
    const int L = a.L;
    int off[kCtrMaxLayers + 1];
    off[0] = 0;
    for (int l = 0; l < L; ++l) off[l + 1] = off[l] + kCtrBS * a.dims[l];
    const int K0 = a.dims[0], C = a.dims[L];
    // input fields, concatenated; rows past B read 0
    {
        int c0 = 0;
        for (int f = 0; f < a.n_fields; ++f) {
            const int w = a.fdim[f];
            for (int e = t; e < kCtrBS * w; e += kThreads) {
                const int s = e / w, k = e % w;
                act[s * K0 + c0 + k] = (b0 + s < B) ? a.field[f][(size_t)(b0 + s) * w + k] : 0.f;
            }
            c0 += w;
        }
    }
    __syncthreads();
    for (int l = 0; l < L; ++l) {
        ctr_dense_fwd(act + off[l], a.dims[l], act + off[l + 1], a.dims[l + 1], a.W[l], a.b[l], l < L - 1, scr, t);
        __syncthreads();
    }
    // softmax, cross-entropy, dlogits = (p - onehot(y)) / B
    if (t < kCtrBS) {
        const int s = t, n = b0 + s;
        const float *z = act + off[L] + s * C;
        float *gz = grd + off[L] + s * C;
        float ls = 0.f;
        const int y = n < B ? labels[n] : -1;
        if (n < B && y >= 0 && y < C) {
            float m = z[0];
            for (int c = 1; c < C; ++c) m = fmaxf(m, z[c]);
            float se = 0.f;
            for (int c = 0; c < C; ++c) se += expf(z[c] - m);
            const float lse = m + logf(se);
            for (int c = 0; c < C; ++c) {
                const float p = expf(z[c] - lse);
                if (prob) prob[(size_t)n * C + c] = p;
                gz[c] = (p - (c == y ? 1.f : 0.f)) / (float)B;
            }
            ls = lse - z[y];
        } else {
            for (int c = 0; c < C; ++c) gz[c] = 0.f;
            if (n < B && prob)
                for (int c = 0; c < C; ++c) prob[(size_t)n * C + c] = 0.f;
        }
        lossv[s] = ls;
    }
    __syncthreads();
    float *p = part + (size_t)blockIdx.x * PS;
    int woff = 0;
    int wo[kCtrMaxLayers];
    for (int l = 0; l < L; ++l) {
        wo[l] = woff;
        woff += a.dims[l + 1] * a.dims[l] + a.dims[l + 1];
    }
    for (int l = L - 1; l >= 0; --l) {
        const int K = a.dims[l], O = a.dims[l + 1];
        const float *gout = grd + off[l + 1], *in = act + off[l];
        // weight and bias gradients of layer l over this block's samples
        ctr_dense_bwd_weight(gout, O, in, K, p + wo[l], t);
        ctr_dense_bwd_data(gout, O, grd + off[l], in, K, a.W[l], l > 0, scr, t);
        __syncthreads();
    }
    // input-field gradients
    {
        int c0 = 0;
        for (int f = 0; f < a.n_fields; ++f) {
            const int w = a.fdim[f];
            if (a.dfield[f])
                for (int e = t; e < kCtrBS * w; e += kThreads) {
                    const int s = e / w, k = e % w;
                    if (b0 + s < B) a.dfield[f][(size_t)(b0 + s) * w + k] = grd[s * K0 + c0 + k];
                }
            c0 += w;
        }
    }
    if (t == 0) {
        float ls = 0.f;
        for (int s = 0; s < kCtrBS; ++s) ls += lossv[s];
        p[PS - 1] = ls;
    }
}

struct CtrOut {
    int L;
    int dims[kCtrMaxLayers + 1];
    float *dW[kCtrMaxLayers];
    float *db[kCtrMaxLayers];
    float *loss;
    int B;
};

// Fixed-order sum of the blocks' partial rows (eight running chains over
// g = 8 i + r, added r = 0..7), scattered into dW, db and the mean loss.
__global__ __launch_bounds__(kThreads) void ctr_reduce_k(const float *__restrict__ part, int G, int PS, CtrOut o)
{
    const int e = blockIdx.x * kThreads + threadIdx.x;
    if (e >= PS) return;
    float s[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    int g = 0;
    for (; g + 8 <= G; g += 8)
#pragma unroll
        for (int r = 0; r < 8; ++r) s[r] += part[(size_t)(g + r) * PS + e];
    for (int r = 0; g + r < G; ++r) s[r] += part[(size_t)(g + r) * PS + e];
    float tot = 0.f;
#pragma unroll
    for (int r = 0; r < 8; ++r) tot += s[r];
    if (e == PS - 1) {
        *o.loss = tot / (float)o.B;
        return;
    }
    int x = e;
    for (int l = 0; l < o.L; ++l) {
        const int nw = o.dims[l + 1] * o.dims[l];
        if (x < nw) {
            o.dW[l][x] = tot;
            return;
        }
        x -= nw;
        if (x < o.dims[l + 1]) {
            o.db[l][x] = tot;
            return;
        }
        x -= o.dims[l + 1];
    }
}

// ---------------------------------------------------------------- Adagrad

__global__ __launch_bounds__(kThreads) void adagrad_k(int D, const int32_t *__restrict__ uniq,
                                                      const int32_t *__restrict__ n_uniq_p, int cap,
                                                      const float *__restrict__ grad, float *__restrict__ table,
                                                      int64_t n_rows, float *__restrict__ accum, float lr, float eps)
{
    const int n_u = min(*n_uniq_p, cap);
    const int64_t e = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (e >= (int64_t)n_u * D) return;
    const int u = (int)(e / D), d = (int)(e % D);
    const int r = uniq[u];
    if (r < 0 || (int64_t)r >= n_rows) return;
    const float g = grad[e];
    const size_t x = (size_t)r * D + d;
    const float acc = accum[x] + g * g;
    accum[x] = acc;
    table[x] -= lr * g / (sqrtf(acc) + eps);
}

// ------------------------------------------------------------------- Adam

__global__ __launch_bounds__(kThreads) void adam_k(int64_t n, float *__restrict__ param,
                                                   const float *__restrict__ grad, float *__restrict__ m,
                                                   float *__restrict__ v, float lr, float b1, float b2, float eps,
                                                   float c1, float c2, uint16_t *__restrict__ pb)
{
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n; i += (int64_t)gridDim.x * kThreads) {
        const float g = grad[i];
        const float mi = b1 * m[i] + (1.f - b1) * g;
        const float vi = b2 * v[i] + (1.f - b2) * g * g;
        m[i] = mi;
        v[i] = vi;
        const float p = param[i] - lr * (mi / c1) / (sqrtf(vi / c2) + eps);
        param[i] = p;
        if (pb) pb[i] = ams_f32_to_bf16(p);
    }
}

size_t al256(size_t x) { return (x + 255) & ~(size_t)255; }

bool ctr_ok(const ams_ctr *net)
{
    if (!net || net->n_layers < 2 || net->n_layers > kCtrMaxLayers) return false;
    if (net->dims[0] < 1 || net->dims[0] > kCtrMaxIn) return false;
    for (int l = 1; l < net->n_layers; ++l)
        if (net->dims[l] < 1 || net->dims[l] > kCtrMaxHidden) return false;
    const int C = net->dims[net->n_layers];
    return C >= 2 && C <= kCtrMaxC;
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
                                  int32_t n_uniq_cap, const float *dbag, float *grad, void *ws, size_t ws_bytes,
                                  void *stream)
{
    if (B > 0 && !dbag) return AMS_ERR_NULL;
    // the SUM aggregator's backward with the bag gradient as the upstream
    // gradient of behaviors and ads alike (it reads neither E, U nor A)
    return ams_pool_bwd(AMS_POOL_SUM, B, D, seg_off, n_beh, inv, occ_perm, uniq_off, n_uniq, n_uniq_cap,
                        grad, dbag, dbag, nullptr, dbag, dbag, grad, ws, ws_bytes, stream);
}

extern "C" size_t ams_ctr_workspace(const ams_ctr *net, int32_t B)
{
    if (!ctr_ok(net) || B < 0) return 0;
    CtrArgs a{};
    a.L = net->n_layers;
    for (int l = 0; l <= a.L; ++l) a.dims[l] = net->dims[l];
    const int G = (B + kCtrBS - 1) / kCtrBS;
    return al256((size_t)(G > 0 ? G : 1) * ctr_part_size(a) * 4);
}

extern "C" ams_status ams_ctr_fwd_bwd(const ams_ctr *net, int32_t B, int32_t n_fields, const float *const *fields,
                                      const int32_t *field_dims, const int32_t *labels, const float *const *W,
                                      const float *const *b, float *loss, float *prob, float *const *dW,
                                      float *const *db, float *const *dfields, void *ws, size_t ws_bytes,
                                      void *stream)
{
    if (!net || !fields || !field_dims || !W || !b || !dW || !db) return AMS_ERR_NULL;
    if (!ctr_ok(net)) return AMS_ERR_DIMS;
    if (B < 1) return AMS_ERR_SIZE;
    if (n_fields < 1 || n_fields > kCtrMaxFields) return AMS_ERR_DIMS;
    CtrArgs a{};
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
        if (!W[l] || !b[l] || !dW[l] || !db[l]) return AMS_ERR_NULL;
        a.W[l] = W[l];
        a.b[l] = b[l];
    }
    if (!labels || !loss) return AMS_ERR_NULL;
    const int G = (B + kCtrBS - 1) / kCtrBS;
    const int PS = ctr_part_size(a);
    if (!ws || ws_bytes < (size_t)G * PS * 4) return AMS_ERR_WORKSPACE;
    hipStream_t st = (hipStream_t)stream;
    float *part = (float *)ws;
    AMS_LAUNCH("ctr_fwd_bwd", st, ctr_fb_k<<<G, kThreads, ctr_lds_bytes(a), st>>>(a, B, labels, prob, part, PS));
    CtrOut o{};
    o.L = a.L;
    for (int l = 0; l <= a.L; ++l) o.dims[l] = a.dims[l];
    for (int l = 0; l < a.L; ++l) {
        o.dW[l] = dW[l];
        o.db[l] = db[l];
    }
    o.loss = loss;
    o.B = B;
    AMS_LAUNCH("ctr_reduce", st, ctr_reduce_k<<<(PS + kThreads - 1) / kThreads, kThreads, 0, st>>>(part, G, PS, o));
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
    const int64_t n = (int64_t)n_uniq_cap * D;
    AMS_LAUNCH("adagrad_rows", st, adagrad_k<<<(unsigned)((n + kThreads - 1) / kThreads), kThreads, 0, st>>>(
                                       D, uniq, n_uniq, n_uniq_cap, grad, table, n_rows, accum, lr, eps));
    return ams_launch_status();
}

extern "C" ams_status ams_adam_update(int64_t n, float *param, const float *grad, float *m, float *v, float lr,
                                      float b1, float b2, float eps, int64_t t, uint16_t *param_bf16, void *stream)
{
    if (n < 0 || t < 1) return AMS_ERR_SIZE;
    if (n == 0) return AMS_OK;
    if (!param || !grad || !m || !v) return AMS_ERR_NULL;
    // bias corrections of step t, formed in double on the host
    const float c1 = (float)(1.0 - pow((double)b1, (double)t));
    const float c2 = (float)(1.0 - pow((double)b2, (double)t));
    hipStream_t st = (hipStream_t)stream;
    int64_t g = (n + kThreads - 1) / kThreads;
    if (g > 4096) g = 4096;
    AMS_LAUNCH("adam_update", st, adam_k<<<(unsigned)g, kThreads, 0, st>>>(n, param, grad, m, v, lr, b1, b2, eps, c1,
                                                                          c2, param_bf16));
    return ams_launch_status();
}
