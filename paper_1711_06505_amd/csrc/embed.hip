// embed.hip -- ams_embed_fwd / ams_embed_bwd: the trainable image embedding
// model of section 5.1 (fully connected, e.g. 4096-256-64-12, ReLU between
// layers) run once per unique image (SERVEREMBED in Algorithm 1), and its
// weight gradients from the merged embedding gradients (SERVERUPDATE).
//
// Forward
//   l1_fwd_*   Z1 = X_u W1^T + b1, H1 = ReLU(Z1), where X_u = T[uniq] is never
//              materialised: every workgroup gathers its 64 feature rows
//              straight from the table into LDS (the row gather is the
//              dominant HBM stream).  MFMA 32x32 tiles: fp32 operands
//              (v_mfma_f32_32x32x2_f32) or bf16 (v_mfma_f32_32x32x16_bf16), fp32
//              accumulation.
//   tail_fwd   the remaining small layers (256 -> 64 -> 12) in fp32, one wave
//              per unique image, weights transposed in LDS.
// Backward
//   tail_bwd   per unique image: dZ_last = dE (masked by the last ReLU if any),
//              dH/dZ of the small layers, dZ1 = (W2^T dZ2) * [H1 > 0]; partial
//              dW2, dW3, db* per fixed block of rows.
//   dw1_*      dW1 = dZ1^T X_u, split over fixed chunks of unique images
//              (deterministic split-K), gathering X_u rows again from T.
//   *_reduce   fixed-order sums of the partials.
// No float atomics anywhere: results are bitwise reproducible.
#include "ams_device.h"

typedef float v16f __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

namespace {

constexpr int kThreads = 256;
constexpr int kTailBlocks = 256;      // fixed row partition of the tail backward
constexpr int kMaxH1 = 256;
constexpr int kMaxH2 = 64;
constexpr int kMaxD = 32;

// Map a linear block index onto (outer, inner) tiles so that the `inner`
// tiles sharing one outer tile run on the same XCD (blocks are dealt to the 8
// XCDs round-robin) and are dispatched back to back, sharing that XCD's L2.
// The grid must have ceil(outer/8) * 8 * inner blocks; returns false for
// padding blocks.
__device__ __forceinline__ bool xcd_tile(int b, int n_outer, int n_inner, int &outer, int &inner)
{
    const int g = b / (8 * n_inner), r = b % (8 * n_inner);
    outer = g * 8 + (r & 7);
    inner = r >> 3;
    return outer < n_outer;
}

__device__ __forceinline__ v16f mfma_f32(float a, float b, v16f c)
{
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ v16f mfma_bf16(uint4 a, uint4 b, v16f c)
{
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// Row index of element j of a 32x32 MFMA accumulator held by `lane`
// (column = lane % 32).
__device__ __forceinline__ int acc_row(int j, int lane) { return 8 * (j >> 2) + 4 * (lane >> 5) + (j & 3); }

// ----------------------------------------------------------- layer 1 fwd

// fp32: block tile 64 rows x NT columns, K step 32, double-buffered LDS.
// Waves are 2 x 2; wave (wm, wn) owns 32 rows x NT/2 columns.  Within a K
// step, lane l supplies k = 16*(l/32) + i to MFMA i (the sum over k does not
// care which k goes to which MFMA as long as A and B agree), so each lane reads
// 16 contiguous floats per operand with four 16-byte LDS loads.
template <int NT>
__global__ __launch_bounds__(kThreads) void l1_fwd_f32(const float *__restrict__ T, int64_t n_rows,
                                                        int F, const int32_t *__restrict__ uniq,
                                                        const int32_t *__restrict__ n_uniq_p,
                                                        int cap, int n_mt, const float *__restrict__ W1,
                                                        const float *__restrict__ b1, int H,
                                                        float *__restrict__ H1)
{
    constexpr int BM = 64, BK = 32, LD = BK + 4;
    constexpr int NB = NT / 64;              // 32-column MFMA blocks per wave
    constexpr int BQ = NT / 32;              // float4 loads of B per thread
    __shared__ float As[2][BM * LD];
    __shared__ float Bs[2][NT * LD];
    __shared__ int rid[BM];

    const int n_u = min(*n_uniq_p, cap);   // never past the caller's buffers
    int mt, nt;
    if (!xcd_tile(blockIdx.x, n_mt, H / NT, mt, nt)) return;
    const int m0 = mt * BM;
    if (m0 >= n_u) return;
    const int n0 = nt * NT;
    const int t = threadIdx.x;
    if (t < BM) {
        int id = -1;
        if (m0 + t < n_u) {
            id = uniq[m0 + t];
            if (id < 0 || (int64_t)id >= n_rows) id = -1;   // reads as a zero row
        }
        rid[t] = id;
    }
    __syncthreads();

    const float *ap[2];
    int aoff[2];
#pragma unroll
    for (int q = 0; q < 2; ++q) {
        const int idx = t + kThreads * q;
        const int r = idx >> 3, c = (idx & 7) * 4;
        ap[q] = rid[r] >= 0 ? T + (size_t)rid[r] * F + c : nullptr;
        aoff[q] = r * LD + c;
    }
    const float *bp[BQ];
    int boff[BQ];
#pragma unroll
    for (int q = 0; q < BQ; ++q) {
        const int idx = t + kThreads * q;
        const int r = idx >> 3, c = (idx & 7) * 4;
        bp[q] = W1 + (size_t)(n0 + r) * F + c;
        boff[q] = r * LD + c;
    }
    float4 ra[2], rb[BQ];
    auto gload = [&](int k0) {
#pragma unroll
        for (int q = 0; q < 2; ++q)
            ra[q] = ap[q] ? *(const float4 *)(ap[q] + k0) : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int q = 0; q < BQ; ++q) rb[q] = *(const float4 *)(bp[q] + k0);
    };
    auto sstore = [&](int buf) {
#pragma unroll
        for (int q = 0; q < 2; ++q) *(float4 *)&As[buf][aoff[q]] = ra[q];
#pragma unroll
        for (int q = 0; q < BQ; ++q) *(float4 *)&Bs[buf][boff[q]] = rb[q];
    };

    const int lane = ams_lane(), wave = t / AMS_WAVE;
    const int wm = wave >> 1, wn = wave & 1, h = lane >> 5, r32 = lane & 31;
    v16f acc[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[nb] = (v16f){};

    gload(0);
    sstore(0);
    __syncthreads();
    const int S = F / BK;
    for (int s = 0; s < S; ++s) {
        const int buf = s & 1;
        if (s + 1 < S) gload((s + 1) * BK);
        float a[16], b[NB][16];
        const float *pa = &As[buf][(wm * 32 + r32) * LD + h * 16];
#pragma unroll
        for (int q = 0; q < 4; ++q) *(float4 *)&a[4 * q] = *(const float4 *)(pa + 4 * q);
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
            const float *pb = &Bs[buf][(wn * (NT / 2) + nb * 32 + r32) * LD + h * 16];
#pragma unroll
            for (int q = 0; q < 4; ++q) *(float4 *)&b[nb][4 * q] = *(const float4 *)(pb + 4 * q);
        }
#pragma unroll
        for (int i = 0; i < 16; ++i)
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) acc[nb] = mfma_f32(a[i], b[nb][i], acc[nb]);
        if (s + 1 < S) sstore(buf ^ 1);
        __syncthreads();
    }

#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
        const int col = n0 + wn * (NT / 2) + nb * 32 + r32;
        const float bias = b1[col];
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            const int row = m0 + wm * 32 + acc_row(j, lane);
            if (row < n_u) H1[(size_t)row * H + col] = fmaxf(acc[nb][j] + bias, 0.f);
        }
    }
}

// bf16: same tiling with K step 64; lane l supplies k = 32*(l/32) + 8*i + e to
// element e of MFMA i.  Writes fp32 H1 (for the tail layers) and, if asked,
// the bf16 copy kept for the backward.
template <int NT>
__global__ __launch_bounds__(kThreads) void l1_fwd_bf16(const uint16_t *__restrict__ T,
                                                         int64_t n_rows, int F,
                                                         const int32_t *__restrict__ uniq,
                                                         const int32_t *__restrict__ n_uniq_p,
                                                         int cap, int n_mt, const uint16_t *__restrict__ W1,
                                                         const float *__restrict__ b1, int H,
                                                         float *__restrict__ H1f,
                                                         uint16_t *__restrict__ H1b)
{
    constexpr int BM = 64, BK = 64, LD = BK + 8;   // bf16 elements
    constexpr int NB = NT / 64;
    constexpr int BQ = NT / 32;
    __shared__ uint16_t As[2][BM * LD];
    __shared__ uint16_t Bs[2][NT * LD];
    __shared__ int rid[BM];

    const int n_u = min(*n_uniq_p, cap);   // never past the caller's buffers
    int mt, nt;
    if (!xcd_tile(blockIdx.x, n_mt, H / NT, mt, nt)) return;
    const int m0 = mt * BM;
    if (m0 >= n_u) return;
    const int n0 = nt * NT;
    const int t = threadIdx.x;
    if (t < BM) {
        int id = -1;
        if (m0 + t < n_u) {
            id = uniq[m0 + t];
            if (id < 0 || (int64_t)id >= n_rows) id = -1;
        }
        rid[t] = id;
    }
    __syncthreads();

    const uint16_t *ap[2];
    int aoff[2];
#pragma unroll
    for (int q = 0; q < 2; ++q) {
        const int idx = t + kThreads * q;
        const int r = idx >> 3, c = (idx & 7) * 8;
        ap[q] = rid[r] >= 0 ? T + (size_t)rid[r] * F + c : nullptr;
        aoff[q] = r * LD + c;
    }
    const uint16_t *bp[BQ];
    int boff[BQ];
#pragma unroll
    for (int q = 0; q < BQ; ++q) {
        const int idx = t + kThreads * q;
        const int r = idx >> 3, c = (idx & 7) * 8;
        bp[q] = W1 + (size_t)(n0 + r) * F + c;
        boff[q] = r * LD + c;
    }
    uint4 ra[2], rb[BQ];
    auto gload = [&](int k0) {
#pragma unroll
        for (int q = 0; q < 2; ++q) ra[q] = ap[q] ? *(const uint4 *)(ap[q] + k0) : make_uint4(0, 0, 0, 0);
#pragma unroll
        for (int q = 0; q < BQ; ++q) rb[q] = *(const uint4 *)(bp[q] + k0);
    };
    auto sstore = [&](int buf) {
#pragma unroll
        for (int q = 0; q < 2; ++q) *(uint4 *)&As[buf][aoff[q]] = ra[q];
#pragma unroll
        for (int q = 0; q < BQ; ++q) *(uint4 *)&Bs[buf][boff[q]] = rb[q];
    };

    const int lane = ams_lane(), wave = t / AMS_WAVE;
    const int wm = wave >> 1, wn = wave & 1, h = lane >> 5, r32 = lane & 31;
    v16f acc[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[nb] = (v16f){};

    gload(0);
    sstore(0);
    __syncthreads();
    const int S = F / BK;
    for (int s = 0; s < S; ++s) {
        const int buf = s & 1;
        if (s + 1 < S) gload((s + 1) * BK);
        uint4 a[4], b[NB][4];
        const uint16_t *pa = &As[buf][(wm * 32 + r32) * LD + h * 32];
#pragma unroll
        for (int q = 0; q < 4; ++q) a[q] = *(const uint4 *)(pa + 8 * q);
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
            const uint16_t *pb = &Bs[buf][(wn * (NT / 2) + nb * 32 + r32) * LD + h * 32];
#pragma unroll
            for (int q = 0; q < 4; ++q) b[nb][q] = *(const uint4 *)(pb + 8 * q);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) acc[nb] = mfma_bf16(a[i], b[nb][i], acc[nb]);
        if (s + 1 < S) sstore(buf ^ 1);
        __syncthreads();
    }

#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
        const int col = n0 + wn * (NT / 2) + nb * 32 + r32;
        const float bias = b1[col];
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            const int row = m0 + wm * 32 + acc_row(j, lane);
            if (row < n_u) {
                const float v = fmaxf(acc[nb][j] + bias, 0.f);
                H1f[(size_t)row * H + col] = v;
                if (H1b) H1b[(size_t)row * H + col] = ams_f32_to_bf16(v);
            }
        }
    }
}

// ------------------------------------------------------- tail layers fwd

__device__ __forceinline__ float ld_w(const void *W, int bf16, size_t i)
{
    return bf16 ? ams_bf16_to_f32(((const uint16_t *)W)[i]) : ((const float *)W)[i];
}

// One wave per unique image.  Layer a: H (<= 256) -> M (<= 64); for a
// 3-layer model layer b: M -> D (<= 32).  Weights transposed into LDS so that
// lanes (outputs) read consecutive addresses and the input vector broadcasts.
template <int L>
__global__ __launch_bounds__(kThreads) void tail_fwd(const float *__restrict__ H1, int H, int M,
                                                      int D, const void *__restrict__ W2,
                                                      const float *__restrict__ b2,
                                                      const void *__restrict__ W3,
                                                      const float *__restrict__ b3, int wbf16,
                                                      int final_relu,
                                                      const int32_t *__restrict__ n_uniq_p, int cap,
                                                      float *__restrict__ H2_save,
                                                      float *__restrict__ E)
{
    __shared__ float W2t[kMaxH1 * kMaxH2];
    __shared__ float W3t[kMaxH2 * kMaxD];
    __shared__ float hrow[kThreads / AMS_WAVE][kMaxH1];
    __shared__ float h2row[kThreads / AMS_WAVE][kMaxH2];
    const int t = threadIdx.x, lane = ams_lane(), wave = t / AMS_WAVE;
    for (int e = t; e < M * H; e += kThreads) W2t[(e % H) * M + e / H] = ld_w(W2, wbf16, e);
    if (L == 3)
        for (int e = t; e < D * M; e += kThreads) W3t[(e % M) * D + e / M] = ld_w(W3, wbf16, e);
    __syncthreads();
    const int n_u = min(*n_uniq_p, cap);   // never past the caller's buffers
    const bool relu_a = (L == 3) || final_relu;
    for (int u = blockIdx.x * (kThreads / AMS_WAVE) + wave; u < n_u; u += gridDim.x * (kThreads / AMS_WAVE)) {
        for (int i = lane; i < H; i += AMS_WAVE) hrow[wave][i] = H1[(size_t)u * H + i];
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
        __builtin_amdgcn_wave_barrier();
        float z = 0.f;
        if (lane < M) {
            z = b2[lane];
            for (int i = 0; i < H; ++i) z += W2t[i * M + lane] * hrow[wave][i];
            if (relu_a) z = fmaxf(z, 0.f);
        }
        if (L == 3) {
            if (lane < M) {
                h2row[wave][lane] = z;
                if (H2_save) H2_save[(size_t)u * M + lane] = z;
            }
            __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
            __builtin_amdgcn_wave_barrier();
            if (lane < D) {
                float e = b3[lane];
                for (int o = 0; o < M; ++o) e += W3t[o * D + lane] * h2row[wave][o];
                if (final_relu) e = fmaxf(e, 0.f);
                E[(size_t)u * D + lane] = e;
            }
        } else {
            if (lane < M) E[(size_t)u * M + lane] = z;
        }
        __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
        __builtin_amdgcn_wave_barrier();
    }
}

// ------------------------------------------------------- tail layers bwd

// Block g owns unique images [g n_u / G, (g+1) n_u / G) in ascending order.
// Thread t owns hidden unit i = t of layer 1 (column i of dW2, dZ1[:, i],
// db1[i]) and a slice of dW3.  Partial layout per block:
//   [dW2: Mo x H][db2: Mo][dW3: D x M][db3: D][db1: H]
// where Mo = M for 3 layers (Mo = D for 2 layers, and dW3/db3 are empty).
template <int L>
__global__ __launch_bounds__(kThreads) void tail_bwd(const void *__restrict__ H1s, int h1_bf16,
                                                      const float *__restrict__ H2s,
                                                      const float *__restrict__ Efwd,
                                                      const float *__restrict__ dE,
                                                      const void *__restrict__ W2,
                                                      const void *__restrict__ W3, int wbf16,
                                                      int H, int M, int D, int final_relu,
                                                      const int32_t *__restrict__ n_uniq_p, int cap,
                                                      void *__restrict__ dZ1, int dz1_bf16,
                                                      float *__restrict__ part, int PS)
{
    __shared__ float W2s[kMaxH2 * kMaxH1];
    __shared__ float W3s[kMaxD * kMaxH2];
    __shared__ float dzl[kMaxD];
    __shared__ float h2s[kMaxH2];
    __shared__ float dz2s[kMaxH2];
    const int t = threadIdx.x;
    const int Mo = (L == 3) ? M : D;                  // width of the layer feeding dW2's rows
    for (int e = t; e < Mo * H; e += kThreads) W2s[e] = ld_w(W2, wbf16, e);
    if (L == 3)
        for (int e = t; e < D * M; e += kThreads) W3s[e] = ld_w(W3, wbf16, e);
    const int n_u = min(*n_uniq_p, cap);   // never past the caller's buffers
    const int r0 = (int)((int64_t)blockIdx.x * n_u / gridDim.x);
    const int r1 = (int)((int64_t)(blockIdx.x + 1) * n_u / gridDim.x);

    float dW2a[kMaxH2];
#pragma unroll
    for (int o = 0; o < kMaxH2; ++o) dW2a[o] = 0.f;
    float dW3a[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) dW3a[q] = 0.f;
    float db1a = 0.f, db2a = 0.f, db3a = 0.f;
    __syncthreads();

    for (int u = r0; u < r1; ++u) {
        if (t < D) {
            float g = dE[(size_t)u * D + t];
            if (final_relu && !(Efwd[(size_t)u * D + t] > 0.f)) g = 0.f;
            dzl[t] = g;
        }
        if (L == 3 && t < M) h2s[t] = H2s[(size_t)u * M + t];
        __syncthreads();
        if (L == 3) {
            if (t < M) {
                float dh = 0.f;
                for (int d = 0; d < D; ++d) dh += W3s[d * M + t] * dzl[d];
                const float dz = h2s[t] > 0.f ? dh : 0.f;
                dz2s[t] = dz;
                db2a += dz;
            }
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                const int e = t + kThreads * q;
                if (e < D * M) dW3a[q] += dzl[e / M] * h2s[e % M];
            }
            if (t < D) db3a += dzl[t];
        } else {
            if (t < D) {
                dz2s[t] = dzl[t];
                db2a += dzl[t];
            }
        }
        __syncthreads();
        if (t < H) {
            const float h1 = h1_bf16 ? ams_bf16_to_f32(((const uint16_t *)H1s)[(size_t)u * H + t])
                                     : ((const float *)H1s)[(size_t)u * H + t];
            float dh = 0.f;
#pragma unroll
            for (int o = 0; o < kMaxH2; ++o)
                if (o < Mo) dh += W2s[o * H + t] * dz2s[o];
            const float dz = h1 > 0.f ? dh : 0.f;
            if (dz1_bf16)
                ((uint16_t *)dZ1)[(size_t)u * H + t] = ams_f32_to_bf16(dz);
            else
                ((float *)dZ1)[(size_t)u * H + t] = dz;
            db1a += dz;
#pragma unroll
            for (int o = 0; o < kMaxH2; ++o)
                if (o < Mo) dW2a[o] += dz2s[o] * h1;
        }
        __syncthreads();
    }

    float *p = part + (size_t)blockIdx.x * PS;
    if (t < H)
#pragma unroll
        for (int o = 0; o < kMaxH2; ++o)
            if (o < Mo) p[o * H + t] = dW2a[o];
    p += Mo * H;
    if (t < Mo) p[t] = db2a;
    p += Mo;
    if (L == 3) {
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            const int e = t + kThreads * q;
            if (e < D * M) p[e] = dW3a[q];
        }
        p += D * M;
        if (t < D) p[t] = db3a;
        p += D;
    }
    if (t < H) p[t] = db1a;
}

// out[e] = sum over g = 0..G-1 (in order) of part[g * PS + e].
__global__ __launch_bounds__(kThreads) void partial_reduce(const float *__restrict__ part, int G,
                                                           size_t PS, float *__restrict__ out)
{
    const size_t e = (size_t)blockIdx.x * kThreads + threadIdx.x;
    if (e >= PS) return;
    float s = 0.f;
    for (int g = 0; g < G; ++g) s += part[(size_t)g * PS + e];
    out[e] = s;
}

// Scatter the reduced tail partials into the caller's gradient arrays.
__global__ __launch_bounds__(kThreads) void tail_unpack(const float *__restrict__ r, int L, int H,
                                                         int M, int D, float *__restrict__ dW2,
                                                         float *__restrict__ db2,
                                                         float *__restrict__ dW3,
                                                         float *__restrict__ db3,
                                                         float *__restrict__ db1)
{
    const int Mo = (L == 3) ? M : D;
    const int n2 = Mo * H, n3 = (L == 3) ? D * M : 0, nb3 = (L == 3) ? D : 0;
    const int total = n2 + Mo + n3 + nb3 + H;
    for (int e = blockIdx.x * kThreads + threadIdx.x; e < total; e += gridDim.x * kThreads) {
        int x = e;
        if (x < n2) { dW2[x] = r[e]; continue; }
        x -= n2;
        if (x < Mo) { db2[x] = r[e]; continue; }
        x -= Mo;
        if (x < n3) { dW3[x] = r[e]; continue; }
        x -= n3;
        if (x < nb3) { db3[x] = r[e]; continue; }
        x -= nb3;
        db1[x] = r[e];
    }
}

// ------------------------------------------------------------- dW1 split-K

// Partial dW1 of chunk c: sum over unique images u in [c n_u / KC,
// (c+1) n_u / KC) of dZ1[u][m] X_u[n].  Block tile BM (m) x 64 (n), K step 32
// images.  The contraction index u is the row index of both operands; the
// fp32 32x32x2 MFMA takes one k per lane, so tiles are staged [k][m] / [k][n]
// as loaded (no transpose) and lanes 0-31 / 32-63 read rows k and k+1.
// TT is the storage type of T and dZ1 (float, or uint16_t for bf16 whose
// products are exact in fp32).
template <int BM, typename TT>
__global__ __launch_bounds__(kThreads) void dw1_part(const TT *__restrict__ T, int64_t n_rows,
                                                      int F, const int32_t *__restrict__ uniq,
                                                      const int32_t *__restrict__ n_uniq_p, int cap,
                                                      const TT *__restrict__ dZ1, int H, int KC,
                                                      float *__restrict__ part)
{
    constexpr int BN = 64, BK = 32;
    constexpr int LDA = BM + 32, LDB = BN + 32;       // row strides = 32 mod 64 banks
    constexpr int AQ = BM / 32;                        // 4-element loads of A per thread
    constexpr int MB = BM / 64;                        // 32-row MFMA blocks per wave
    __shared__ float As[2][BK * LDA];
    __shared__ float Bs[2][BK * LDB];

    const int nmt = H / BM, nnt = F / BN;
    int outer, mt;
    if (!xcd_tile(blockIdx.x, nnt * KC, nmt, outer, mt)) return;
    const int nt = outer % nnt, c = outer / nnt;
    const int n_u = min(*n_uniq_p, cap);   // never past the caller's buffers
    const int u0 = (int)((int64_t)c * n_u / KC), u1 = (int)((int64_t)(c + 1) * n_u / KC);
    const int m0 = mt * BM, n0 = nt * BN;
    const int t = threadIdx.x;

    int ar[AQ], ac[AQ], br[2], bc[2];
#pragma unroll
    for (int q = 0; q < AQ; ++q) {
        const int idx = t + kThreads * q;
        ar[q] = idx / (BM / 4);
        ac[q] = (idx % (BM / 4)) * 4;
    }
#pragma unroll
    for (int q = 0; q < 2; ++q) {
        const int idx = t + kThreads * q;
        br[q] = idx >> 4;
        bc[q] = (idx & 15) * 4;
    }
    float4 ra[AQ], rb[2];
    auto ld4 = [](const TT *p) -> float4 {
        if constexpr (sizeof(TT) == 4) {
            return *(const float4 *)p;
        } else {
            const uint2 v = *(const uint2 *)p;
            return make_float4(__uint_as_float(v.x << 16), __uint_as_float(v.x & 0xffff0000u),
                               __uint_as_float(v.y << 16), __uint_as_float(v.y & 0xffff0000u));
        }
    };
    auto gload = [&](int k0) {
#pragma unroll
        for (int q = 0; q < AQ; ++q) {
            const int u = k0 + ar[q];
            ra[q] = u < u1 ? ld4(dZ1 + (size_t)u * H + m0 + ac[q]) : make_float4(0.f, 0.f, 0.f, 0.f);
        }
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            const int u = k0 + br[q];
            int id = u < u1 ? uniq[u] : -1;
            if (id < 0 || (int64_t)id >= n_rows) id = -1;
            rb[q] = id >= 0 ? ld4(T + (size_t)id * F + n0 + bc[q]) : make_float4(0.f, 0.f, 0.f, 0.f);
        }
    };
    auto sstore = [&](int buf) {
#pragma unroll
        for (int q = 0; q < AQ; ++q) *(float4 *)&As[buf][ar[q] * LDA + ac[q]] = ra[q];
#pragma unroll
        for (int q = 0; q < 2; ++q) *(float4 *)&Bs[buf][br[q] * LDB + bc[q]] = rb[q];
    };

    const int lane = ams_lane(), wave = t / AMS_WAVE;
    const int wm = wave >> 1, wn = wave & 1, h = lane >> 5, r32 = lane & 31;
    v16f acc[MB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) acc[mb] = (v16f){};

    if (u0 < u1) {
        gload(u0);
        sstore(0);
    }
    __syncthreads();
    const int S = (u1 - u0 + BK - 1) / BK;
    for (int s = 0; s < S; ++s) {
        const int buf = s & 1;
        if (s + 1 < S) gload(u0 + (s + 1) * BK);
        const float *pa = &As[buf][h * LDA + wm * (BM / 2) + r32];
        const float *pb = &Bs[buf][h * LDB + wn * 32 + r32];
#pragma unroll
        for (int kk = 0; kk < BK / 2; ++kk) {
            const float bv = pb[2 * kk * LDB];
#pragma unroll
            for (int mb = 0; mb < MB; ++mb) acc[mb] = mfma_f32(pa[2 * kk * LDA + mb * 32], bv, acc[mb]);
        }
        if (s + 1 < S) sstore(buf ^ 1);
        __syncthreads();
    }

    float *out = part + (size_t)c * H * F;
    const int col = n0 + wn * 32 + r32;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            const int row = m0 + wm * (BM / 2) + mb * 32 + acc_row(j, lane);
            out[(size_t)row * F + col] = acc[mb][j];
        }
}

// ----------------------------------------------------------------- host

bool mlp_ok(const ams_mlp *m)
{
    if (!m || (m->n_layers != 2 && m->n_layers != 3)) return false;
    const int F = m->dims[0], H = m->dims[1];
    if (F < 64 || F > 65536 || F % 64) return false;
    if (H < 64 || H > kMaxH1 || H % 64) return false;
    if (m->n_layers == 3 && (m->dims[2] < 1 || m->dims[2] > kMaxH2)) return false;
    const int D = m->dims[m->n_layers];
    if (D < 1 || D > kMaxD) return false;
    if (m->n_layers == 3 && D * m->dims[2] > 8 * kThreads) return false;
    return true;
}

size_t al256(size_t x) { return (x + 255) & ~(size_t)255; }

int dw1_chunks(int H, int F)
{
    const int bm = (H % 128 == 0) ? 128 : 64;
    const int tiles = (H / bm) * (F / 64);
    int kc = 2048 / tiles;
    return kc < 1 ? 1 : (kc > 32 ? 32 : kc);
}

int tail_part_size(const ams_mlp *m)
{
    const int L = m->n_layers, H = m->dims[1], D = m->dims[L];
    const int M = (L == 3) ? m->dims[2] : D;
    return M * H + M + ((L == 3) ? D * M + D : 0) + H;
}

struct BwdPlan {
    size_t off_dz1, off_tail, off_tailsum, off_dw1, total;
    int kc;
};

BwdPlan plan_bwd(const ams_mlp *m, int32_t cap)
{
    BwdPlan p{};
    const int H = m->dims[1], F = m->dims[0];
    const size_t es = (m->dtype == AMS_BF16) ? 2 : 4;
    p.kc = dw1_chunks(H, F);
    size_t o = 0;
    p.off_dz1 = o; o += al256((size_t)cap * H * es);
    p.off_tail = o; o += al256((size_t)kTailBlocks * tail_part_size(m) * 4);
    p.off_tailsum = o; o += al256((size_t)tail_part_size(m) * 4);
    p.off_dw1 = o; o += al256((size_t)p.kc * H * F * 4);
    p.total = o;
    return p;
}

}  // namespace

extern "C" size_t ams_embed_workspace(const ams_mlp *mlp, int32_t n_uniq_cap)
{
    if (!mlp_ok(mlp) || n_uniq_cap < 0) return 0;
    const size_t fwd = al256((size_t)n_uniq_cap * mlp->dims[1] * 4);
    const size_t bwd = plan_bwd(mlp, n_uniq_cap).total;
    return fwd > bwd ? fwd : bwd;
}

extern "C" ams_status ams_embed_fwd(const ams_mlp *mlp, const void *T, int64_t n_rows,
                                    const int32_t *uniq, const int32_t *n_uniq, int32_t cap,
                                    const void *W1, const float *b1, const void *W2,
                                    const float *b2, const void *W3, const float *b3,
                                    void *H1_save, float *H2_save, float *E, void *ws,
                                    size_t ws_bytes, void *stream)
{
    if (!mlp) return AMS_ERR_NULL;
    if (mlp->dtype != AMS_F32 && mlp->dtype != AMS_BF16) return AMS_ERR_DTYPE;
    if (!mlp_ok(mlp)) return AMS_ERR_DIMS;
    if (cap < 0 || n_rows < 0) return AMS_ERR_SIZE;
    const int L = mlp->n_layers;
    if (!T || !uniq || !n_uniq || !W1 || !b1 || !W2 || !b2 || !E) return AMS_ERR_NULL;
    if (L == 3 && (!W3 || !b3)) return AMS_ERR_NULL;
    if (cap == 0) return AMS_OK;
    const int F = mlp->dims[0], H = mlp->dims[1], D = mlp->dims[L];
    const int M = (L == 3) ? mlp->dims[2] : D;
    const bool bf = mlp->dtype == AMS_BF16;
    const bool h1_in_ws = bf || !H1_save;
    if (h1_in_ws && (!ws || ws_bytes < al256((size_t)cap * H * 4))) return AMS_ERR_WORKSPACE;
    hipStream_t st = (hipStream_t)stream;
    float *H1f = h1_in_ws ? (float *)ws : (float *)H1_save;

    const int n_mt = (cap + 63) / 64;
    const int NT = (H % 128 == 0) ? 128 : 64;
    const int grid = ((n_mt + 7) / 8) * 8 * (H / NT);
    if (!bf) {
        if (NT == 128)
            l1_fwd_f32<128><<<grid, kThreads, 0, st>>>((const float *)T, n_rows, F, uniq, n_uniq, cap, n_mt,
                                                       (const float *)W1, b1, H, H1f);
        else
            l1_fwd_f32<64><<<grid, kThreads, 0, st>>>((const float *)T, n_rows, F, uniq, n_uniq, cap, n_mt,
                                                      (const float *)W1, b1, H, H1f);
    } else {
        if (NT == 128)
            l1_fwd_bf16<128><<<grid, kThreads, 0, st>>>((const uint16_t *)T, n_rows, F, uniq, n_uniq,
                                                        cap, n_mt, (const uint16_t *)W1, b1, H, H1f,
                                                        (uint16_t *)H1_save);
        else
            l1_fwd_bf16<64><<<grid, kThreads, 0, st>>>((const uint16_t *)T, n_rows, F, uniq, n_uniq,
                                                       cap, n_mt, (const uint16_t *)W1, b1, H, H1f,
                                                       (uint16_t *)H1_save);
    }
    int tg = (cap + 3) / 4;
    if (tg > 256) tg = 256;
    if (L == 3)
        tail_fwd<3><<<tg, kThreads, 0, st>>>(H1f, H, M, D, W2, b2, W3, b3, bf, mlp->final_relu, n_uniq,
                                             cap, H2_save, E);
    else
        tail_fwd<2><<<tg, kThreads, 0, st>>>(H1f, H, M, D, W2, b2, W3, b3, bf, mlp->final_relu, n_uniq,
                                             cap, H2_save, E);
    return ams_launch_status();
}

extern "C" ams_status ams_embed_bwd(const ams_mlp *mlp, const void *T, int64_t n_rows,
                                    const int32_t *uniq, const int32_t *n_uniq, int32_t cap,
                                    const void *W1, const void *W2, const void *W3,
                                    const void *H1_save, const float *H2_save,
                                    const float *E_fwd, const float *dE, float *dW1, float *db1,
                                    float *dW2, float *db2, float *dW3, float *db3, void *ws,
                                    size_t ws_bytes, void *stream)
{
    (void)W1;
    if (!mlp) return AMS_ERR_NULL;
    if (mlp->dtype != AMS_F32 && mlp->dtype != AMS_BF16) return AMS_ERR_DTYPE;
    if (!mlp_ok(mlp)) return AMS_ERR_DIMS;
    if (cap < 0 || n_rows < 0) return AMS_ERR_SIZE;
    const int L = mlp->n_layers;
    if (!T || !uniq || !n_uniq || !W2 || !H1_save || !dE || !dW1 || !db1 || !dW2 || !db2)
        return AMS_ERR_NULL;
    if (L == 3 && (!W3 || !H2_save || !dW3 || !db3)) return AMS_ERR_NULL;
    if (mlp->final_relu && !E_fwd) return AMS_ERR_NULL;
    const BwdPlan p = plan_bwd(mlp, cap);
    if (!ws || ws_bytes < p.total) return AMS_ERR_WORKSPACE;
    const int F = mlp->dims[0], H = mlp->dims[1], D = mlp->dims[L];
    const int M = (L == 3) ? mlp->dims[2] : D;
    const bool bf = mlp->dtype == AMS_BF16;
    hipStream_t st = (hipStream_t)stream;
    char *w = (char *)ws;
    void *dz1 = w + p.off_dz1;
    float *tail = (float *)(w + p.off_tail);
    float *tailsum = (float *)(w + p.off_tailsum);
    float *dw1p = (float *)(w + p.off_dw1);
    const int PS = tail_part_size(mlp);

    if (L == 3)
        tail_bwd<3><<<kTailBlocks, kThreads, 0, st>>>(H1_save, bf, H2_save, E_fwd, dE, W2, W3, bf, H, M, D,
                                                      mlp->final_relu, n_uniq, cap, dz1, bf, tail, PS);
    else
        tail_bwd<2><<<kTailBlocks, kThreads, 0, st>>>(H1_save, bf, H2_save, E_fwd, dE, W2, W3, bf, H, M, D,
                                                      mlp->final_relu, n_uniq, cap, dz1, bf, tail, PS);
    partial_reduce<<<(PS + kThreads - 1) / kThreads, kThreads, 0, st>>>(tail, kTailBlocks, (size_t)PS,
                                                                         tailsum);
    tail_unpack<<<(PS + kThreads - 1) / kThreads, kThreads, 0, st>>>(tailsum, L, H, M, D, dW2, db2,
                                                                      dW3, db3, db1);

    const int bm = (H % 128 == 0) ? 128 : 64;
    const int nmt = H / bm, outer = (F / 64) * p.kc;
    const int grid = ((outer + 7) / 8) * 8 * nmt;
    if (!bf) {
        if (bm == 128)
            dw1_part<128, float><<<grid, kThreads, 0, st>>>((const float *)T, n_rows, F, uniq, n_uniq, cap,
                                                             (const float *)dz1, H, p.kc, dw1p);
        else
            dw1_part<64, float><<<grid, kThreads, 0, st>>>((const float *)T, n_rows, F, uniq, n_uniq, cap,
                                                            (const float *)dz1, H, p.kc, dw1p);
    } else {
        if (bm == 128)
            dw1_part<128, uint16_t><<<grid, kThreads, 0, st>>>((const uint16_t *)T, n_rows, F, uniq,
                                                                n_uniq, cap, (const uint16_t *)dz1, H, p.kc,
                                                                dw1p);
        else
            dw1_part<64, uint16_t><<<grid, kThreads, 0, st>>>((const uint16_t *)T, n_rows, F, uniq,
                                                               n_uniq, cap, (const uint16_t *)dz1, H, p.kc,
                                                               dw1p);
    }
    const size_t nw = (size_t)H * F;
    partial_reduce<<<(unsigned)((nw + kThreads - 1) / kThreads), kThreads, 0, st>>>(dw1p, p.kc, nw, dW1);
    return ams_launch_status();
}
