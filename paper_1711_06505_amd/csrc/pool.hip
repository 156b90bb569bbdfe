// pool.hip -- ams_pool_fwd / ams_pool_bwd: the user behavior image aggregator
// of section 5.2 (sum, max, attentive pooling with the ad image embedding as
// query) and its backward, merged per unique image as Algorithm 1 merges the
// embedding gradients of one image at its server.
//
// Forward: one wave per sample; lanes stride over the sample's behaviors,
// fetch E[inv[j]] (12 floats, L2 resident) and reduce across the wave in a
// fixed butterfly order.  Attentive pooling reads its segment's embeddings
// once (logits with a running softmax per lane, two rows in flight), then
// normalises the stored logits into weights.
//
// Backward: (1) one wave per sample computes the per-sample terms of the
// attention gradient and tags every behavior occurrence with its sample;
// (2) one wave per chunk of 64 positions of the stable occurrence order
// evaluates each occurrence's embedding gradient and sums runs of equal
// unique image with a segmented lane scan on DPP moves -- runs wholly inside the chunk go
// straight to dE, runs that cross a chunk edge leave a partial; (3) one wave
// per chunk in which a crossing run starts adds that run's partials in chunk
// order.  Fixed orders throughout: no float atomics, bitwise reproducible.
#include "ams_device.h"

#include <climits>
#include <type_traits>

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / AMS_WAVE;
// Internal mode: attentive pooling with a query given per sample (one channel
// of multiple-query attentive pooling, section 5.2).  It runs the attentive
// kernels with the query read from Q[i] instead of the ad's embedding; the
// ads' occurrences get no gradient from it and the attention term
// sum_j ds_j e_j is the query's gradient.
constexpr int kPoolQuery = 3;
// Internal mode: the concatenate aggregator's backward (section 5.2).  The
// behavior at position p of sample i takes row p of the sample's upstream
// block dU[i] ([Lc x D]) when p < Lc and nothing otherwise; an ad takes dA.
constexpr int kPoolConcat = 4;

// Row `row` of a [. x D] float array into DM registers (zero past D): 16-byte
// loads when D is a multiple of 4 and the array starts on a 16-byte
// boundary (then every row does), else one load per element.
template <int DM>
__device__ __forceinline__ void load_row(const float *__restrict__ E, int row, int D, float (&e)[DM])
{
    const float *p = E + (size_t)row * D;
    if (((D & 3) | ((uintptr_t)E & 15)) == 0) {
#pragma unroll
        for (int d4 = 0; d4 < DM / 4; ++d4) {
            const float4 v = 4 * d4 < D ? *(const float4 *)(p + 4 * d4) : make_float4(0.f, 0.f, 0.f, 0.f);
            e[4 * d4] = v.x;
            e[4 * d4 + 1] = v.y;
            e[4 * d4 + 2] = v.z;
            e[4 * d4 + 3] = v.w;
        }
    } else {
#pragma unroll
        for (int d = 0; d < DM; ++d) e[d] = d < D ? p[d] : 0.f;
    }
}

// Row `row` of E when it is below the row count `cap`, else a zero row: a
// caller whose capacity is below the real unique count gets unspecified
// values, never an access past its buffers.
template <int DM>
__device__ __forceinline__ void load_row_cap(const float *__restrict__ E, int row, int cap, int D, float (&e)[DM])
{
    if ((unsigned)row < (unsigned)cap) load_row<DM>(E, row, D, e);
    else {
#pragma unroll
        for (int d = 0; d < DM; ++d) e[d] = 0.f;
    }
}

// Calls f with the register width DM (12, 16 or 32) that covers D.
template <class F>
void with_dm(int D, F f)
{
    if (D <= 12) f(std::integral_constant<int, 12>{});
    else if (D <= 16) f(std::integral_constant<int, 16>{});
    else f(std::integral_constant<int, 32>{});
}

template <int MODE, int DM>
__global__ __launch_bounds__(kThreads) void pool_fwd_k(int B, int D, const int32_t *__restrict__ seg_off,
                                                       int64_t n_beh, const int32_t *__restrict__ inv, int cap,
                                                       const float *__restrict__ E, float *__restrict__ U,
                                                       float *__restrict__ A, void *__restrict__ saved,
                                                       const float *__restrict__ Q)
{
    const int lane = ams_lane();
    const int i = blockIdx.x * kWaves + threadIdx.x / AMS_WAVE;
    if (i >= B) return;
    const int j0 = seg_off[i], j1 = seg_off[i + 1];
    const int ad_row = inv[n_beh + i];
    if (MODE != kPoolQuery && lane < D)
        A[(size_t)i * D + lane] = (unsigned)ad_row < (unsigned)cap ? E[(size_t)ad_row * D + lane] : 0.f;
    float out[DM];
    // sum and max: lane l takes behaviors l, l + 64, ... in that order, in
    // rounds of PU per lane with the round's index loads, then its row
    // loads, in flight together
    constexpr int PU = DM <= 16 ? 4 : 2;
    auto load_round = [&](int jr, float (&e)[PU][DM]) {
        int r[PU];
#pragma unroll
        for (int q = 0; q < PU; ++q) {
            const int j = jr + q * AMS_WAVE + lane;
            r[q] = j < j1 ? inv[j] : -1;
            if (r[q] >= cap) r[q] = -1;
        }
#pragma unroll
        for (int q = 0; q < PU; ++q) {
            if (r[q] >= 0) load_row<DM>(E, r[q], D, e[q]);
            else {
#pragma unroll
                for (int d = 0; d < DM; ++d) e[q][d] = 0.f;
            }
        }
    };
    if (MODE == AMS_POOL_SUM) {
        float acc[DM];
#pragma unroll
        for (int d = 0; d < DM; ++d) acc[d] = 0.f;
        for (int jr = j0; jr < j1; jr += PU * AMS_WAVE) {
            float e[PU][DM];
            load_round(jr, e);
#pragma unroll
            for (int q = 0; q < PU; ++q)
                if (jr + q * AMS_WAVE + lane < j1) {
#pragma unroll
                    for (int d = 0; d < DM; ++d) acc[d] += e[q][d];
                }
        }
#pragma unroll
        for (int d = 0; d < DM; ++d) out[d] = ams_wave_sum(acc[d]);
    } else if (MODE == AMS_POOL_MAX) {
        float best[DM];
        int bidx[DM];
#pragma unroll
        for (int d = 0; d < DM; ++d) {
            best[d] = 0.f;
            bidx[d] = -1;
        }
        for (int jr = j0; jr < j1; jr += PU * AMS_WAVE) {
            float e[PU][DM];
            load_round(jr, e);
#pragma unroll
            for (int q = 0; q < PU; ++q) {
                const int j = jr + q * AMS_WAVE + lane;
                if (j >= j1) continue;
#pragma unroll
                for (int d = 0; d < DM; ++d)
                    if (bidx[d] < 0 || e[q][d] > best[d]) {
                        best[d] = e[q][d];
                        bidx[d] = j;
                    }
            }
        }
        // first maximum over the segment: larger value wins, ties -> lower j
#pragma unroll
        for (int d = 0; d < DM; ++d) {
            float v = best[d];
            int x = bidx[d];
#pragma unroll
            for (int o = AMS_WAVE / 2; o > 0; o >>= 1) {
                const float ov = __shfl_xor(v, o, AMS_WAVE);
                const int ox = __shfl_xor(x, o, AMS_WAVE);
                const bool take = ox >= 0 && (x < 0 || ov > v || (ov == v && ox < x));
                if (take) {
                    v = ov;
                    x = ox;
                }
            }
            out[d] = x < 0 ? 0.f : v;
            if (lane == d && d < D) ((int32_t *)saved)[(size_t)i * D + d] = x;
        }
    } else {
        // one pass over the embeddings with a running (online) softmax per
        // lane: max m, denominator den and weighted sum acc, rescaled when
        // the max grows; the lanes are then brought to the wave's max M.
        // The logits are kept in w and normalised in a second, cheap pass.
        float a[DM];
        if (MODE == kPoolQuery) load_row<DM>(Q, i, D, a);
        else load_row_cap<DM>(E, ad_row, cap, D, a);
        float *w = (float *)saved;
        float m = -INFINITY, den = 0.f, acc[DM];
#pragma unroll
        for (int d = 0; d < DM; ++d) acc[d] = 0.f;
        auto take = [&](int j, const float (&e)[DM]) {
            float sc = 0.f;
#pragma unroll
            for (int d = 0; d < DM; ++d) sc += e[d] * a[d];
            w[j] = sc;
            const float mn = fmaxf(m, sc);
            const float r = expf(m - mn), p = expf(sc - mn);    // m = -inf: r = 0
            den = den * r + p;
#pragma unroll
            for (int d = 0; d < DM; ++d) acc[d] = acc[d] * r + p * e[d];
            m = mn;
        };
        int j = j0 + lane;
        for (; j + AMS_WAVE < j1; j += 2 * AMS_WAVE) {   // two rows in flight
            const int r0 = inv[j], r1 = inv[j + AMS_WAVE];
            float e0[DM], e1[DM];
            load_row_cap<DM>(E, r0, cap, D, e0);
            load_row_cap<DM>(E, r1, cap, D, e1);
            take(j, e0);
            take(j + AMS_WAVE, e1);
        }
        if (j < j1) {
            float e0[DM];
            load_row_cap<DM>(E, inv[j], cap, D, e0);
            take(j, e0);
        }
        const float M = ams_wave_max(m);
        const float f = m == -INFINITY ? 0.f : expf(m - M);      // lanes without behaviors add nothing
        den = ams_wave_sum(den * f);
        const float inv_den = j1 > j0 ? 1.f / den : 0.f;
#pragma unroll
        for (int d = 0; d < DM; ++d) out[d] = ams_wave_sum(acc[d] * f) * inv_den;
        for (int jj = j0 + lane; jj < j1; jj += AMS_WAVE) w[jj] = expf(w[jj] - M) * inv_den;
    }
    float mine = 0.f;
#pragma unroll
    for (int d = 0; d < DM; ++d)
        if (lane == d) mine = out[d];
    if (lane < D) U[(size_t)i * D + lane] = mine;
}

// Concatenate aggregator: U[i] = the embeddings of sample i's first Lc
// behaviors side by side (zero rows past its length), A[i] = its ad's.  One
// thread per output element, grid-stride: the writes are contiguous, the
// embedding rows come from L2.
__global__ __launch_bounds__(kThreads) void pool_concat_fwd_k(int B, int D, int Lc,
                                                              const int32_t *__restrict__ seg_off, int64_t n_beh,
                                                              const int32_t *__restrict__ inv, int cap,
                                                              const float *__restrict__ E, float *__restrict__ U,
                                                              float *__restrict__ A)
{
    const int64_t row = (int64_t)Lc * D, nU = (int64_t)B * row, n = nU + (int64_t)B * D;
    for (int64_t e = (int64_t)blockIdx.x * kThreads + threadIdx.x; e < n; e += (int64_t)gridDim.x * kThreads) {
        if (e < nU) {
            const int i = (int)(e / row);
            const int r = (int)(e - (int64_t)i * row);
            const int p = r / D, d = r - p * D;
            const int j0 = seg_off[i], len = seg_off[i + 1] - j0;
            const int row_u = p < len ? inv[j0 + p] : -1;
            U[e] = (unsigned)row_u < (unsigned)cap ? E[(size_t)row_u * D + d] : 0.f;
        } else {
            const int64_t x = e - nU;
            const int i = (int)(x / D), d = (int)(x - (int64_t)i * D);
            const int r = inv[n_beh + i];
            A[x] = (unsigned)r < (unsigned)cap ? E[(size_t)r * D + d] : 0.f;
        }
    }
}

// The record of occurrence k, written in occurrence order for the stable-order
// pass to read with one access: its unique index, and its sample i for a
// behavior or -1 - i for the ad of sample i; with attention also the
// behavior's weight w_j and its score gradient ds_j (float bits).
template <int MODE>
constexpr bool wide_rec() { return MODE == AMS_POOL_ATT || MODE == kPoolQuery; }

// (1) per sample: the records of its occurrences; attention terms
// c_i = g_i . u_i and da_i = sum_j ds_j e_j, ds_j = w_j (g_i . e_j - c_i).
// Sum mode with a second upstream gradient of the ads (dA2): da_i = dA_i +
// dA2_i, the ad rows' gradient the stable-order pass then reads.
template <int MODE, int DM>
__global__ __launch_bounds__(kThreads) void pool_bwd_sample(int B, int D, const int32_t *__restrict__ seg_off,
                                                            int64_t n_beh, const int32_t *__restrict__ inv, int cap,
                                                            const float *__restrict__ E,
                                                            const float *__restrict__ U,
                                                            const float *__restrict__ wsaved,
                                                            const float *__restrict__ dU,
                                                            void *__restrict__ rec,
                                                            float *__restrict__ cvec,
                                                            float *__restrict__ da,
                                                            const float *__restrict__ dA,
                                                            const float *__restrict__ dA2)
{
    const int lane = ams_lane();
    const int i = blockIdx.x * kWaves + threadIdx.x / AMS_WAVE;
    if (i >= B) return;
    if (MODE == AMS_POOL_SUM && dA2 && lane < D)
        da[(size_t)i * D + lane] = (dA ? dA[(size_t)i * D + lane] : 0.f) + dA2[(size_t)i * D + lane];
    const int j0 = seg_off[i], j1 = seg_off[i + 1];
    if (lane == 0) {
        const int k = (int)(n_beh + i);
        if (wide_rec<MODE>()) ((int4 *)rec)[k] = make_int4(inv[k], -1 - i, 0, 0);
        else ((int2 *)rec)[k] = make_int2(inv[k], -1 - i);
    }
    if (!wide_rec<MODE>()) {
        int2 *r2 = (int2 *)rec;
        int j = j0 + lane;
        for (; j + AMS_WAVE < j1; j += 2 * AMS_WAVE) {
            const int u0 = inv[j], u1 = inv[j + AMS_WAVE];
            r2[j] = make_int2(u0, i);
            r2[j + AMS_WAVE] = make_int2(u1, i);
        }
        if (j < j1) r2[j] = make_int2(inv[j], i);
    }
    if (MODE != AMS_POOL_ATT && MODE != kPoolQuery) return;
    float g[DM], u[DM];
    load_row<DM>(dU, i, D, g);
    load_row<DM>(U, i, D, u);
    float c = 0.f;
#pragma unroll
    for (int d = 0; d < DM; ++d) c += g[d] * u[d];
    float acc[DM];
#pragma unroll
    for (int d = 0; d < DM; ++d) acc[d] = 0.f;
    int4 *r4 = (int4 *)rec;
    auto take = [&](int j, int r, const float (&e)[DM]) {
        float dw = 0.f;
#pragma unroll
        for (int d = 0; d < DM; ++d) dw += g[d] * e[d];
        const float wj = wsaved[j];
        const float ds = wj * (dw - c);
        r4[j] = make_int4(r, i, __float_as_int(wj), __float_as_int(ds));
#pragma unroll
        for (int d = 0; d < DM; ++d) acc[d] += ds * e[d];
    };
    int j = j0 + lane;
    for (; j + AMS_WAVE < j1; j += 2 * AMS_WAVE) {       // two rows in flight
        const int r0 = inv[j], r1 = inv[j + AMS_WAVE];
        float e0[DM], e1[DM];
        load_row_cap<DM>(E, r0, cap, D, e0);
        load_row_cap<DM>(E, r1, cap, D, e1);
        take(j, r0, e0);
        take(j + AMS_WAVE, r1, e1);
    }
    if (j < j1) {
        const int r0 = inv[j];
        float e0[DM];
        load_row_cap<DM>(E, r0, cap, D, e0);
        take(j, r0, e0);
    }
    float mine = 0.f;
#pragma unroll
    for (int d = 0; d < DM; ++d) {
        const float v = ams_wave_sum(acc[d]);
        if (lane == d) mine = v;
    }
    if (lane < D) da[(size_t)i * D + lane] = mine;
    if (lane == 0) cvec[i] = c;
}

// One step of the segmented scan: every lane reads (key, values) of the lane
// that the DPP control CTRL names (row_mask RM: rows not in it read nothing)
// and adds the values when the keys are equal.  Lanes with no source keep the
// `old` operand: a key no lane holds, values 0.
template <int CTRL, int RM, int DM>
__device__ __forceinline__ void seg_step(int u, float (&v)[DM])
{
    const int ou = __builtin_amdgcn_update_dpp(INT_MIN, u, CTRL, RM, 0xF, false);
    const bool join = ou == u;
#pragma unroll
    for (int d = 0; d < DM; ++d) {
        const float ov = __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v[d]), CTRL, RM, 0xF, false));
        if (join) v[d] += ov;
    }
}

// Inclusive segmented scan over the 64 lanes (runs of equal u contiguous;
// u is never INT_MIN) on DPP moves, no LDS: within each row of 16 lanes
// Hillis-Steele steps from 1, 2, 4 and 8 lanes back (row_shr); then lane 15
// of rows 0 and 2 into rows 1 and 3 (row_bcast:15), then lane 31 into rows 2
// and 3 (row_bcast:31).  A lane joins a source only when the keys match, so
// its run then covers every lane in between; after the last step a lane
// holds the sum from its run's first lane in the wave.  Fixed order, so
// deterministic.
template <int DM>
__device__ __forceinline__ void seg_scan(int u, float (&v)[DM])
{
    seg_step<0x111, 0xF, DM>(u, v);
    seg_step<0x112, 0xF, DM>(u, v);
    seg_step<0x114, 0xF, DM>(u, v);
    seg_step<0x118, 0xF, DM>(u, v);
    seg_step<0x142, 0xA, DM>(u, v);
    seg_step<0x143, 0xC, DM>(u, v);
}

// (2) segmented sums over chunks of 64 positions of the stable occurrence
// order.  A wave takes CPW consecutive chunks and issues each level of their
// dependent loads for all of them before using any (the stable order; then
// each position's unique index and sample; then the rows), so CPW chains of
// random reads are in flight per lane instead of one; each chunk is then
// scanned and written as one.
template <int MODE, int DM>
constexpr int seg_cpw() { return DM > 16 || MODE == AMS_POOL_MAX ? 2 : 4; }

template <int MODE, int DM, int CPW>
__global__ __launch_bounds__(kThreads) void pool_bwd_seg(int D, int n_occ, int cap,
                                                         const int32_t *__restrict__ occ_perm,
                                                         const int32_t *__restrict__ uniq_off,
                                                         const float *__restrict__ A,
                                                         const void *__restrict__ saved,
                                                         const float *__restrict__ dU,
                                                         const float *__restrict__ dA,
                                                         const void *__restrict__ rec,
                                                         const float *__restrict__ da, int nch,
                                                         float *__restrict__ dE,
                                                         float *__restrict__ head_part,
                                                         float *__restrict__ tail_part,
                                                         int32_t *__restrict__ cross, int accumulate,
                                                         const int32_t *__restrict__ seg_off, int Lc)
{
    constexpr bool ATT = MODE == AMS_POOL_ATT || MODE == kPoolQuery;
    const int lane = ams_lane();
    const int ch0 = (blockIdx.x * kWaves + threadIdx.x / AMS_WAVE) * CPW;
    if (ch0 >= nch) return;
    // level 1: the stable order
    int k[CPW];
#pragma unroll
    for (int c = 0; c < CPW; ++c) {
        const int p = (ch0 + c) * AMS_WAVE + lane;
        k[c] = p < n_occ ? occ_perm[p] : 0;
    }
    // level 2: the record of each position's occurrence (unique index, sample,
    // attention weight).  An occurrence whose unique index is at or past the
    // caller's capacity (possible only when the capacity is below the real
    // unique count) is dropped: its row of dE does not exist.  si: the sample
    // of a behavior, -1 - i for the ad of sample i, or INT_MIN (nothing)
    int uk[CPW], si[CPW];
    float wk[CPW], dsk[CPW];
#pragma unroll
    for (int c = 0; c < CPW; ++c) {
        const int p = (ch0 + c) * AMS_WAVE + lane;
        uk[c] = -1;
        si[c] = INT_MIN;
        wk[c] = 0.f;
        dsk[c] = 0.f;
        if (p < n_occ) {
            if constexpr (ATT) {
                const int4 r = ((const int4 *)rec)[k[c]];
                uk[c] = r.x;
                si[c] = r.y;
                wk[c] = __int_as_float(r.z);
                dsk[c] = __int_as_float(r.w);
            } else {
                const int2 r = ((const int2 *)rec)[k[c]];
                uk[c] = r.x;
                si[c] = r.y;
            }
        }
    }
    // level 3: the rows each position's gradient is made of
    float r[CPW][DM];            // dU of the behavior's sample (concat: its slice), or the ad's dA
    float a[ATT ? CPW : 1][DM];  // attentive: the sample's query row, or the ad's attention term da
    int am[MODE == AMS_POOL_MAX ? CPW : 1][DM];
#pragma unroll
    for (int c = 0; c < CPW; ++c) {
        const bool valid = si[c] != INT_MIN && uk[c] < cap;
        const bool beh = valid && si[c] >= 0;
        const bool ad = valid && si[c] < 0 && MODE != kPoolQuery;
        const int i = beh ? si[c] : (ad ? -1 - si[c] : 0);
#pragma unroll
        for (int d = 0; d < DM; ++d) r[c][d] = 0.f;
        if (beh && MODE != kPoolConcat) load_row<DM>(dU, i, D, r[c]);
        if (beh && MODE == kPoolConcat) {
            const int pos = k[c] - seg_off[i];
            if (pos < Lc) load_row<DM>(dU + (size_t)i * Lc * D, pos, D, r[c]);
        }
        if (ad && dA) load_row<DM>(dA, i, D, r[c]);
        if constexpr (MODE == AMS_POOL_MAX) {
            const int32_t *amr = (const int32_t *)saved + (size_t)i * D;
#pragma unroll
            for (int d = 0; d < DM; ++d) am[c][d] = (beh && d < D) ? amr[d] : -1;
        }
        if constexpr (ATT) {
#pragma unroll
            for (int d = 0; d < DM; ++d) a[c][d] = 0.f;
            if (beh) load_row<DM>(A, i, D, a[c]);
            if (ad && MODE == AMS_POOL_ATT) load_row<DM>(da, i, D, a[c]);
        }
    }
    // each chunk: its positions' gradients, summed per run of one image
#pragma unroll
    for (int c = 0; c < CPW; ++c) {
        const int ch = ch0 + c;
        if (ch >= nch) break;
        const int c0 = ch * AMS_WAVE, c1 = c0 + AMS_WAVE;
        const bool valid = si[c] != INT_MIN && uk[c] < cap;
        const bool beh = valid && si[c] >= 0;
        int u = valid ? uk[c] : -1 - lane;       // distinct per invalid lane: never joins a run
        float v[DM];
#pragma unroll
        for (int d = 0; d < DM; ++d) v[d] = 0.f;
        if (beh) {
            if (MODE == AMS_POOL_SUM || MODE == kPoolConcat) {
#pragma unroll
                for (int d = 0; d < DM; ++d) v[d] = r[c][d];
            } else if (MODE == AMS_POOL_MAX) {
#pragma unroll
                for (int d = 0; d < DM; ++d) v[d] = am[MODE == AMS_POOL_MAX ? c : 0][d] == k[c] ? r[c][d] : 0.f;
            } else {   // attentive: w_j g_i + ds_j a_i; A holds the query rows in the query mode
#pragma unroll
                for (int d = 0; d < DM; ++d) v[d] = wk[c] * r[c][d] + dsk[c] * a[ATT ? c : 0][d];
            }
        } else if (valid && MODE != kPoolQuery) {   // an ad: dA (+ the attention term)
#pragma unroll
            for (int d = 0; d < DM; ++d) v[d] = r[c][d];
            if (MODE == AMS_POOL_ATT) {
#pragma unroll
                for (int d = 0; d < DM; ++d) v[d] += a[ATT ? c : 0][d];
            }
        }
        seg_scan<DM>(u, v);
        const int nu_next = __shfl_down(u, 1, AMS_WAVE);
        const bool run_end = valid && (lane == AMS_WAVE - 1 || nu_next != u);
        int cross_u = -1;
        if (run_end) {
            const int s0 = uniq_off[u], e0 = uniq_off[u + 1];
            float *dst;
            if (s0 < c0) {
                dst = head_part + (size_t)ch * D;          // run began in an earlier chunk
            } else if (e0 > c1) {
                dst = tail_part + (size_t)ch * D;          // run starts here, continues later
                cross_u = u;
            } else {
                dst = dE + (size_t)u * D;                   // whole run inside this chunk
                if (accumulate) {
#pragma unroll
                    for (int d = 0; d < DM; ++d)
                        if (d < D) v[d] += dst[d];
                }
            }
#pragma unroll
            for (int d = 0; d < DM; ++d)
                if (d < D) dst[d] = v[d];
        }
        // only lane 63 can end a run that continues past the chunk
        const int cu = __shfl(cross_u, AMS_WAVE - 1, AMS_WAVE);
        if (lane == 0) cross[ch] = cu;
    }
}

// A row of D floats read as DM/4 16-byte loads with no condition: D == DM
// and 16-byte aligned rows (the fast path of the fix-up below).
template <int DM>
__device__ __forceinline__ void load_row_full(const float *__restrict__ p, float (&e)[DM])
{
#pragma unroll
    for (int d4 = 0; d4 < DM / 4; ++d4) {
        const float4 v = *(const float4 *)(p + 4 * d4);
        e[4 * d4] = v.x;
        e[4 * d4 + 1] = v.y;
        e[4 * d4 + 2] = v.z;
        e[4 * d4 + 3] = v.w;
    }
}

// Chunks per block of the head-part block sums.
constexpr int kFixBlock = 512;

// Sum of a wave's items: lane l adds items l, l + 64, ... in ascending order,
// U rows in flight (the last group clamps its index and drops the extra
// rows); then a butterfly over the lanes.  Lane d < D returns coordinate d.
template <int DM, class Row>
__device__ __forceinline__ float sum_items(int n_items, int D, bool full, Row row)
{
    constexpr int U = DM > 16 ? 4 : 8;
    const int lane = ams_lane();
    float acc[DM];
#pragma unroll
    for (int d = 0; d < DM; ++d) acc[d] = 0.f;
    if (n_items <= AMS_WAVE) {                  // one item per lane at most: one load each
        const float *rp = row(min(lane, n_items - 1));
        if (full) load_row_full<DM>(rp, acc);
        else load_row<DM>(rp, 0, D, acc);
        if (lane >= n_items) {
#pragma unroll
            for (int d = 0; d < DM; ++d) acc[d] = 0.f;
        }
        n_items = 0;                            // (the loop below does nothing)
    }
    for (int t0 = lane; t0 < n_items; t0 += U * AMS_WAVE) {
        float h[U][DM];
#pragma unroll
        for (int q = 0; q < U; ++q) {
            const float *rp = row(min(t0 + q * AMS_WAVE, n_items - 1));
            if (full) load_row_full<DM>(rp, h[q]);
            else load_row<DM>(rp, 0, D, h[q]);
        }
#pragma unroll
        for (int q = 0; q < U; ++q) {
            const bool take = t0 + q * AMS_WAVE < n_items;
#pragma unroll
            for (int d = 0; d < DM; ++d) acc[d] += take ? h[q][d] : 0.f;
        }
    }
    float mine = 0.f;
#pragma unroll
    for (int d = 0; d < DM; ++d) {
        const float s = ams_wave_sum(acc[d]);
        if (lane == d) mine = s;
    }
    return mine;
}

// (3a) block sums of the head parts: bsum[b] = sum of the head parts of
// chunks b*kFixBlock .. (b+1)*kFixBlock - 1.  Only blocks that lie inside
// one run's head chunks are ever used, where every one of those head parts
// was written.
template <int DM>
__global__ __launch_bounds__(kThreads) void pool_bwd_bsum(int D, int nch, bool full,
                                                          const float *__restrict__ head_part,
                                                          float *__restrict__ bsum)
{
    const int b = blockIdx.x * kWaves + threadIdx.x / AMS_WAVE;
    if (b >= nch / kFixBlock) return;                     // whole blocks only
    const float *base = head_part + (size_t)b * kFixBlock * D;
    const float s = sum_items<DM>(kFixBlock, D, full, [&](int t) { return base + (size_t)t * D; });
    if (ams_lane() < D) bsum[(size_t)b * D + ams_lane()] = s;
}

// Head chunks a lane adds by itself in the fix-up.
template <int DM>
constexpr int fix_short() { return DM > 16 ? 2 : 4; }

// Below this many 64-position chunks the backward runs one chunk per wave
// (stable-order pass and fix-up): the grid is then small enough that more
// waves, not longer ones, keep the part busy.
constexpr int kSmallChunks = 16384;

// (3b) the fix-up of a run that starts in chunk ch and crosses chunk edges:
// tail part of ch plus the sum of the head parts of chunks ch + 1 .. last
// (the run's last chunk).  A wave sums items lane-strided, then by the
// butterfly of ams_wave_sum: the head parts before the first whole block of
// kFixBlock chunks inside the range, the block sums, the head parts after
// the last one (a hot image's run of thousands of chunks costs at most
// 2 kFixBlock head parts and one block sum per block).  In the large-grid
// kernel a run of at most fix_short head chunks is summed by one lane in the
// butterfly's association, (h0 + h2) + (h1 + h3), so which kernel or path
// takes a run changes nothing in its sum.
template <int DM>
__device__ __forceinline__ void fix_one_lane(int D, bool full, int ch, int u, int last,
                                             const float *__restrict__ head_part,
                                             const float *__restrict__ tail_part, float *__restrict__ dE,
                                             int accumulate)
{
    constexpr int NS = fix_short<DM>();
    auto row = [&](const float *base, int r, float (&e)[DM]) {
        if (full) load_row_full<DM>(base + (size_t)r * D, e);
        else load_row<DM>(base, r, D, e);
    };
    static_assert(NS == 2 || NS == 4, "the butterfly's association below");
    const int n = last - ch;
    float t[DM], h[NS][DM];
    row(tail_part, ch, t);
#pragma unroll
    for (int q = 0; q < NS; ++q) row(head_part, min(ch + 1 + q, last), h[q]);
#pragma unroll
    for (int q = 0; q < NS; ++q)
#pragma unroll
        for (int d = 0; d < DM; ++d) h[q][d] = q < n ? h[q][d] : 0.f;
#pragma unroll
    for (int d = 0; d < DM; ++d) {
        const float sh = NS == 4 ? (h[0][d] + h[NS / 2][d]) + (h[1][d] + h[NS - 1][d]) : h[0][d] + h[1][d];
        t[d] = t[d] + sh;
    }
    float *dst = dE + (size_t)u * D;
    if (accumulate) {
        float o[DM];
        load_row<DM>(dE, u, D, o);              // dE: the caller's buffer, any alignment
#pragma unroll
        for (int d = 0; d < DM; ++d) t[d] = o[d] + t[d];
    }
#pragma unroll
    for (int d = 0; d < DM; ++d)
        if (d < D) dst[d] = t[d];
}

template <int DM>
__device__ __forceinline__ void fix_one_wave(int D, bool full, int cb, int ub, int lb,
                                             const float *__restrict__ head_part,
                                             const float *__restrict__ tail_part,
                                             const float *__restrict__ bsum, float *__restrict__ dE,
                                             int accumulate)
{
    const int first = cb + 1;
    const int jb = (first + kFixBlock - 1) / kFixBlock, je = (lb + 1) / kFixBlock;
    int n1 = lb - cb, n2 = 0, n3 = 0;
    if (jb < je) {
        n1 = jb * kFixBlock - first;
        n2 = je - jb;
        n3 = lb + 1 - je * kFixBlock;
    }
    const float s = sum_items<DM>(n1 + n2 + n3, D, full, [&](int t) {
        if (t < n1) return head_part + (size_t)(first + t) * D;
        if (t < n1 + n2) return bsum + (size_t)(jb + t - n1) * D;
        return head_part + ((size_t)je * kFixBlock + (t - n1 - n2)) * D;
    });
    const int lane = ams_lane();
    if (lane < D) {
        const float r = tail_part[(size_t)cb * D + lane] + s;
        dE[(size_t)ub * D + lane] = accumulate ? dE[(size_t)ub * D + lane] + r : r;
    }
}

// One wave per chunk (small grids).
template <int DM>
__global__ __launch_bounds__(kThreads) void pool_bwd_fix(int D, int nch, bool full,
                                                         const int32_t *__restrict__ uniq_off,
                                                         const int32_t *__restrict__ cross,
                                                         const float *__restrict__ head_part,
                                                         const float *__restrict__ tail_part,
                                                         const float *__restrict__ bsum,
                                                         float *__restrict__ dE, int accumulate)
{
    const int ch = blockIdx.x * kWaves + threadIdx.x / AMS_WAVE;
    if (ch >= nch) return;
    const int u = cross[ch];
    if (u < 0) return;
    const int last = (uniq_off[u + 1] - 1) / AMS_WAVE;
    fix_one_wave<DM>(D, full, ch, u, last, head_part, tail_part, bsum, dE, accumulate);
}

// 64 chunks per wave, one per lane (large grids): short runs by their lanes;
// the block's long runs gathered in LDS and shared out over its waves.
template <int DM>
__global__ __launch_bounds__(kThreads) void pool_bwd_fix64(int D, int nch, bool full,
                                                           const int32_t *__restrict__ uniq_off,
                                                           const int32_t *__restrict__ cross,
                                                           const float *__restrict__ head_part,
                                                           const float *__restrict__ tail_part,
                                                           const float *__restrict__ bsum,
                                                           float *__restrict__ dE, int accumulate)
{
    __shared__ int lr_ch[kWaves * AMS_WAVE], lr_u[kWaves * AMS_WAVE], lr_last[kWaves * AMS_WAVE];
    __shared__ int lr_cnt[kWaves];
    const int lane = ams_lane(), wave = threadIdx.x / AMS_WAVE;
    const int ch = (blockIdx.x * kWaves + wave) * AMS_WAVE + lane;
    const int u = ch < nch ? cross[ch] : -1;
    const int last = u >= 0 ? (uniq_off[u + 1] - 1) / AMS_WAVE : ch;
    const bool is_long = u >= 0 && last - ch > fix_short<DM>();
    if (u >= 0 && !is_long) fix_one_lane<DM>(D, full, ch, u, last, head_part, tail_part, dE, accumulate);
    const uint64_t todo = __ballot(is_long);
    if (lane == 0) lr_cnt[wave] = __popcll(todo);
    __syncthreads();
    int off = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
        off += w < wave ? lr_cnt[w] : 0;
        tot += lr_cnt[w];
    }
    if (is_long) {
        const int i = off + __popcll(todo & ((1ull << lane) - 1));
        lr_ch[i] = ch;
        lr_u[i] = u;
        lr_last[i] = last;
    }
    __syncthreads();
    for (int i = wave; i < tot; i += kWaves)
        fix_one_wave<DM>(D, full, lr_ch[i], lr_u[i], lr_last[i], head_part, tail_part, bsum, dE, accumulate);
}

size_t al256(size_t x) { return (x + 255) & ~(size_t)255; }

struct PoolPlan {
    size_t off_rec, off_c, off_da, off_head, off_tail, off_cross, off_bsum, total;
    int nch;
};

// Workspace of the backward; the records are 16 bytes with attention
// (ams_pool_workspace's AMS_POOL_ATT also covers the query mode), 8 without.
PoolPlan plan_pool(bool wide, int32_t B, int64_t n_beh, int32_t D)
{
    PoolPlan p{};
    const int64_t n_occ = n_beh + B;
    p.nch = (int)((n_occ + AMS_WAVE - 1) / AMS_WAVE);
    size_t o = 0;
    p.off_rec = o; o += al256((size_t)n_occ * (wide ? 16 : 8));
    p.off_c = o; o += al256((size_t)B * 4);
    p.off_da = o; o += al256((size_t)B * D * 4);
    p.off_head = o; o += al256((size_t)p.nch * D * 4);
    p.off_tail = o; o += al256((size_t)p.nch * D * 4);
    p.off_cross = o; o += al256((size_t)p.nch * 4);
    p.off_bsum = o; o += al256((size_t)(p.nch / kFixBlock) * D * 4);
    p.total = o;
    return p;
}

template <int MODE, int DM>
void launch_fwd(int B, int D, const int32_t *seg_off, int64_t n_beh, const int32_t *inv, int cap, const float *E,
                float *U, float *A, void *saved, hipStream_t st, const float *Q = nullptr)
{
    AMS_LAUNCH("pool_fwd_k", st, pool_fwd_k<MODE, DM><<<(B + kWaves - 1) / kWaves, kThreads, 0, st>>>(B, D, seg_off, n_beh, inv, cap,
                                                                         E, U, A, saved, Q));
}

template <int MODE, int DM>
void launch_bwd(int B, int D, const int32_t *seg_off, int64_t n_beh, const int32_t *inv, int cap,
                const int32_t *occ_perm, const int32_t *uniq_off, const float *E, const float *U,
                const float *A, const void *saved, const float *dU, const float *dA, float *dE,
                char *ws, const PoolPlan &p, hipStream_t st, float *dQ = nullptr, int accumulate = 0,
                int Lc = 0, const float *dA2 = nullptr)
{
    void *rec = ws + p.off_rec;
    float *cvec = (float *)(ws + p.off_c);
    // the attention term of each sample: the query's gradient in the query mode
    float *da = MODE == kPoolQuery ? dQ : (float *)(ws + p.off_da);
    float *head = (float *)(ws + p.off_head);
    float *tail = (float *)(ws + p.off_tail);
    int32_t *cross = (int32_t *)(ws + p.off_cross);
    float *bsum = (float *)(ws + p.off_bsum);
    const int n_occ = (int)(n_beh + B);
    // head and tail rows start at 256-byte boundaries, so rows of D == DM
    // floats (D a multiple of 4) are 16-byte aligned
    const bool full = D == DM;
    if (B > 0)
        AMS_LAUNCH("pool_bwd_sample", st, pool_bwd_sample<MODE, DM><<<(B + kWaves - 1) / kWaves, kThreads, 0, st>>>(
            B, D, seg_off, n_beh, inv, cap, E, U, (const float *)saved, dU, rec, cvec, da, dA, dA2));
    // sum mode with a second ad gradient: the ads read the folded rows
    if (MODE == AMS_POOL_SUM && dA2) dA = da;
    const bool small = p.nch < kSmallChunks;
#define SEG_LAUNCH(CPWV)                                                                                     \
    AMS_LAUNCH("pool_bwd_seg", st, (pool_bwd_seg<MODE, DM, CPWV><<<(p.nch + kWaves * CPWV - 1) / (kWaves * CPWV), \
                                                                  kThreads, 0, st>>>(                        \
                                       D, n_occ, cap, occ_perm, uniq_off, A, saved, dU, dA, rec, da, p.nch, dE, \
                                       head, tail, cross, accumulate, seg_off, Lc)))
    if (small) SEG_LAUNCH(1);
    else SEG_LAUNCH((seg_cpw<MODE, DM>()));
#undef SEG_LAUNCH
    // a whole block of chunks inside one run's head chunks starts at block 1
    // or later (the run starts in an earlier chunk), so it needs 2 blocks
    const int nblk = p.nch / kFixBlock;
    if (p.nch >= 2 * kFixBlock)
        AMS_LAUNCH("pool_bwd_bsum", st, pool_bwd_bsum<DM><<<(nblk + kWaves - 1) / kWaves, kThreads, 0, st>>>(
            D, p.nch, full, head, bsum));
    if (small)
        AMS_LAUNCH("pool_bwd_fix", st, pool_bwd_fix<DM><<<(p.nch + kWaves - 1) / kWaves, kThreads, 0, st>>>(
            D, p.nch, full, uniq_off, cross, head, tail, bsum, dE, accumulate));
    else
        AMS_LAUNCH("pool_bwd_fix", st, pool_bwd_fix64<DM><<<(p.nch + kWaves * AMS_WAVE - 1) / (kWaves * AMS_WAVE),
                                                           kThreads, 0, st>>>(D, p.nch, full, uniq_off, cross, head,
                                                                              tail, bsum, dE, accumulate));
}

ams_status check_common(int32_t mode, int32_t B, int32_t D, int64_t n_beh)
{
    if (mode < AMS_POOL_SUM || mode > AMS_POOL_ATT) return AMS_ERR_MODE;
    if (B < 0 || n_beh < 0 || D < 1 || D > 32) return AMS_ERR_SIZE;
    if (n_beh + (int64_t)B > (int64_t)INT32_MAX - 1) return AMS_ERR_SIZE;
    return AMS_OK;
}

}  // namespace

extern "C" ams_status ams_pool_fwd(int32_t mode, int32_t B, int32_t D, const int32_t *seg_off, int64_t n_beh,
                                   const int32_t *inv, int32_t n_uniq_cap, const float *E, float *U, float *A,
                                   void *saved, void *stream)
{
    ams_status s = check_common(mode, B, D, n_beh);
    if (s != AMS_OK) return s;
    if (n_uniq_cap < 0) return AMS_ERR_SIZE;
    if (B == 0) return AMS_OK;
    if (!seg_off || !inv || !E || !U || !A) return AMS_ERR_NULL;
    if (mode != AMS_POOL_SUM && !saved) return AMS_ERR_NULL;
    hipStream_t st = (hipStream_t)stream;
    with_dm(D, [&](auto dm) {
        constexpr int DM = decltype(dm)::value;
        switch (mode) {
        case AMS_POOL_SUM: launch_fwd<AMS_POOL_SUM, DM>(B, D, seg_off, n_beh, inv, n_uniq_cap, E, U, A, saved, st); break;
        case AMS_POOL_MAX: launch_fwd<AMS_POOL_MAX, DM>(B, D, seg_off, n_beh, inv, n_uniq_cap, E, U, A, saved, st); break;
        default: launch_fwd<AMS_POOL_ATT, DM>(B, D, seg_off, n_beh, inv, n_uniq_cap, E, U, A, saved, st);
        }
    });
    return ams_launch_status();
}

extern "C" size_t ams_pool_workspace(int32_t mode, int32_t B, int64_t n_beh, int32_t D, int32_t n_uniq_cap)
{
    (void)n_uniq_cap;
    if (check_common(mode, B, D, n_beh) != AMS_OK) return 0;
    return plan_pool(mode == AMS_POOL_ATT, B, n_beh, D).total;
}

ams_status pool_bwd_sum_ads(int32_t B, int32_t D, const int32_t *seg_off, int64_t n_beh, const int32_t *inv,
                            const int32_t *occ_perm, const int32_t *uniq_off, int32_t n_uniq_cap, const float *dU,
                            const float *dA, const float *dA2, float *dE, void *ws, size_t ws_bytes, void *stream)
{
    ams_status s = check_common(AMS_POOL_SUM, B, D, n_beh);
    if (s != AMS_OK) return s;
    if (n_uniq_cap < 0) return AMS_ERR_SIZE;
    if (n_beh + B == 0) return AMS_OK;
    if (!seg_off || !inv || !occ_perm || !uniq_off || !dE) return AMS_ERR_NULL;
    if (B > 0 && !dU) return AMS_ERR_NULL;
    const PoolPlan p = plan_pool(false, B, n_beh, D);
    if (!ws || ws_bytes < p.total) return AMS_ERR_WORKSPACE;
    hipStream_t st = (hipStream_t)stream;
    with_dm(D, [&](auto dm) {
        launch_bwd<AMS_POOL_SUM, decltype(dm)::value>(B, D, seg_off, n_beh, inv, n_uniq_cap, occ_perm, uniq_off,
                                                      nullptr, nullptr, nullptr, nullptr, dU, dA, dE, (char *)ws, p,
                                                      st, nullptr, 0, 0, dA2);
    });
    return ams_launch_status();
}

extern "C" ams_status ams_pool_bwd(int32_t mode, int32_t B, int32_t D, const int32_t *seg_off, int64_t n_beh,
                                   const int32_t *inv, const int32_t *occ_perm, const int32_t *uniq_off,
                                   const int32_t *n_uniq, int32_t n_uniq_cap, const float *E, const float *U,
                                   const float *A, const void *saved, const float *dU, const float *dA,
                                   float *dE, void *ws, size_t ws_bytes, void *stream)
{
    ams_status s = check_common(mode, B, D, n_beh);
    if (s != AMS_OK) return s;
    (void)n_uniq;
    if (n_uniq_cap < 0) return AMS_ERR_SIZE;
    const int64_t n_occ = n_beh + B;
    if (n_occ == 0) return AMS_OK;
    if (!seg_off || !inv || !occ_perm || !uniq_off || !E || !dE) return AMS_ERR_NULL;
    if (B > 0 && (!U || !A || !dU)) return AMS_ERR_NULL;
    if (mode != AMS_POOL_SUM && B > 0 && !saved) return AMS_ERR_NULL;
    const PoolPlan p = plan_pool(mode == AMS_POOL_ATT, B, n_beh, D);
    if (!ws || ws_bytes < p.total) return AMS_ERR_WORKSPACE;
    hipStream_t st = (hipStream_t)stream;
    char *w = (char *)ws;
    with_dm(D, [&](auto dm) {
        constexpr int DM = decltype(dm)::value;
        switch (mode) {
        case AMS_POOL_SUM:
            launch_bwd<AMS_POOL_SUM, DM>(B, D, seg_off, n_beh, inv, n_uniq_cap, occ_perm, uniq_off, E, U, A, saved, dU, dA, dE,
                                         w, p, st);
            break;
        case AMS_POOL_MAX:
            launch_bwd<AMS_POOL_MAX, DM>(B, D, seg_off, n_beh, inv, n_uniq_cap, occ_perm, uniq_off, E, U, A, saved, dU, dA, dE,
                                         w, p, st);
            break;
        default:
            launch_bwd<AMS_POOL_ATT, DM>(B, D, seg_off, n_beh, inv, n_uniq_cap, occ_perm, uniq_off, E, U, A, saved, dU, dA, dE,
                                         w, p, st);
        }
    });
    return ams_launch_status();
}

extern "C" ams_status ams_pool_query_fwd(int32_t B, int32_t D, const int32_t *seg_off, int64_t n_beh,
                                         const int32_t *inv, int32_t n_uniq_cap, const float *E, const float *Q,
                                         float *U, float *w, void *stream)
{
    ams_status s = check_common(AMS_POOL_ATT, B, D, n_beh);
    if (s != AMS_OK) return s;
    if (n_uniq_cap < 0) return AMS_ERR_SIZE;
    if (B == 0) return AMS_OK;
    if (!seg_off || !inv || !E || !Q || !U || !w) return AMS_ERR_NULL;
    hipStream_t st = (hipStream_t)stream;
    with_dm(D, [&](auto dm) {
        launch_fwd<kPoolQuery, decltype(dm)::value>(B, D, seg_off, n_beh, inv, n_uniq_cap, E, U, nullptr, w, st, Q);
    });
    return ams_launch_status();
}

extern "C" ams_status ams_pool_query_bwd(int32_t B, int32_t D, const int32_t *seg_off, int64_t n_beh,
                                         const int32_t *inv, const int32_t *occ_perm, const int32_t *uniq_off,
                                         const int32_t *n_uniq, int32_t n_uniq_cap, const float *E, const float *Q,
                                         const float *U, const float *w, const float *dU, float *dQ, float *dE,
                                         int32_t accumulate, void *ws, size_t ws_bytes, void *stream)
{
    ams_status s = check_common(AMS_POOL_ATT, B, D, n_beh);
    if (s != AMS_OK) return s;
    (void)n_uniq;
    if (n_uniq_cap < 0) return AMS_ERR_SIZE;
    const int64_t n_occ = n_beh + B;
    if (n_occ == 0) return AMS_OK;
    if (!seg_off || !inv || !occ_perm || !uniq_off || !E || !dE) return AMS_ERR_NULL;
    if (B > 0 && (!Q || !U || !w || !dU || !dQ)) return AMS_ERR_NULL;
    const PoolPlan p = plan_pool(true, B, n_beh, D);
    if (!ws || ws_bytes < p.total) return AMS_ERR_WORKSPACE;
    hipStream_t st = (hipStream_t)stream;
    char *wsc = (char *)ws;
    with_dm(D, [&](auto dm) {
        launch_bwd<kPoolQuery, decltype(dm)::value>(B, D, seg_off, n_beh, inv, n_uniq_cap, occ_perm, uniq_off, E, U, Q, w, dU,
                                                    nullptr, dE, wsc, p, st, dQ, accumulate != 0);
    });
    return ams_launch_status();
}

extern "C" ams_status ams_pool_concat_fwd(int32_t B, int32_t D, int32_t Lc, const int32_t *seg_off, int64_t n_beh,
                                          const int32_t *inv, int32_t n_uniq_cap, const float *E, float *U, float *A,
                                          void *stream)
{
    ams_status s = check_common(AMS_POOL_SUM, B, D, n_beh);
    if (s != AMS_OK) return s;
    if (n_uniq_cap < 0 || Lc < 1 || (int64_t)Lc * D > INT32_MAX) return AMS_ERR_SIZE;
    if (B == 0) return AMS_OK;
    if (!seg_off || !inv || !E || !U || !A) return AMS_ERR_NULL;
    hipStream_t st = (hipStream_t)stream;
    const int64_t n = (int64_t)B * ((int64_t)Lc * D + D);
    int64_t g = (n + kThreads - 1) / kThreads;
    if (g > 8192) g = 8192;
    AMS_LAUNCH("pool_concat_fwd", st, pool_concat_fwd_k<<<(unsigned)g, kThreads, 0, st>>>(B, D, Lc, seg_off, n_beh, inv,
                                                                                          n_uniq_cap, E, U, A));
    return ams_launch_status();
}

extern "C" ams_status ams_pool_concat_bwd(int32_t B, int32_t D, int32_t Lc, const int32_t *seg_off, int64_t n_beh,
                                          const int32_t *inv, const int32_t *occ_perm, const int32_t *uniq_off,
                                          const int32_t *n_uniq, int32_t n_uniq_cap, const float *dU,
                                          const float *dA, float *dE, void *ws, size_t ws_bytes, void *stream)
{
    ams_status s = check_common(AMS_POOL_SUM, B, D, n_beh);
    if (s != AMS_OK) return s;
    (void)n_uniq;
    if (n_uniq_cap < 0 || Lc < 1 || (int64_t)Lc * D > INT32_MAX) return AMS_ERR_SIZE;
    const int64_t n_occ = n_beh + B;
    if (n_occ == 0) return AMS_OK;
    if (!seg_off || !inv || !occ_perm || !uniq_off || !dE) return AMS_ERR_NULL;
    if (B > 0 && !dU) return AMS_ERR_NULL;
    const PoolPlan p = plan_pool(false, B, n_beh, D);
    if (!ws || ws_bytes < p.total) return AMS_ERR_WORKSPACE;
    hipStream_t st = (hipStream_t)stream;
    char *w = (char *)ws;
    with_dm(D, [&](auto dm) {
        launch_bwd<kPoolConcat, decltype(dm)::value>(B, D, seg_off, n_beh, inv, n_uniq_cap, occ_perm, uniq_off, nullptr, nullptr,
                                                     nullptr, nullptr, dU, dA, dE, w, p, st, nullptr, 0, Lc);
    });
    return ams_launch_status();
}
