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
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

namespace {

constexpr int kThreads = 256;
constexpr int kTailBlocks = 256;      // fixed row partition of the tail backward

// The tail backward's blocks: with n_u unique images, blocks [0, tail_active)
// each take an equal share of at least kTailMinRows rows and write a partial
// slot; the rest of the grid leaves at once, and the reduction of the slots
// reads only the active ones (a small batch then moves far fewer partials).
constexpr int kTailMinRows = 64;
__host__ __device__ constexpr int tail_active(int n_u, int G)
{
    const int g = (n_u + kTailMinRows - 1) / kTailMinRows;
    return g < 1 ? 1 : (g > G ? G : g);
}
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

// fp32 forward of the 4096-wide layer.  Block tile 64 rows x NT columns, K
// step 32 floats, 4 waves in 2 x 2 (wave (wm, wn) owns 32 rows x NT/2 cols).
//
// Operands stream straight from HBM into a 3-slot LDS ring with
// global_load_lds_dwordx4 (no staging registers): stage s+2 is in flight
// while stage s feeds the MFMAs.  Each slot is its own __shared__ array and
// the loop is unrolled by 3 so that the compiler can tell the slot being
// filled from the slot being read, and each wave waits only for its own
// oldest stage (s_waitcnt vmcnt) and its own LDS reads (lgkmcnt) before a
// bare s_barrier; after the barrier the slot read in the previous stage is
// refilled.  A scheduling barrier keeps each stage's MFMAs ahead of the next
// stage's wait, so the wait finds the LDS reads long completed.
//
// One DMA instruction moves 1 KB = 8 tile rows of 128 B; lane l writes 16 B
// to slot (l % 8) of row l / 8.  Rows are XOR-swizzled by ring_swz(row) so
// that the MFMA operand reads (16 B per lane, 32 consecutive rows) hit
// distinct banks.  Within a K step lane l supplies k = 16*(l/32) + i to MFMA
// i (A and B agree, so the sum over k is unchanged).
//
// Rows past n_u and rows whose ID is outside the table stream a row of W1
// instead (always a valid address); rows past n_u are never stored and rows
// with an out-of-range ID get the exact result of a zero feature row,
// ReLU(b1), in the epilogue.
__device__ __forceinline__ int ring_swz(int row) { return (row & 7) ^ ((row >> 1) & 4); }

typedef __attribute__((address_space(3))) void lds_void_t;

__device__ __forceinline__ void dma16(const void *src, void *lds_dst)
{
    __builtin_amdgcn_global_load_lds(src, (lds_void_t *)lds_dst, 16, 0, 0);
}

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding).
#define AMS_WAIT_VM(n) \
    __builtin_amdgcn_s_waitcnt(((n) & 0xF) | (((n) >> 4) << 14) | (0x7 << 4) | (0xF << 8))
// ... and every LDS access of this wave completed as well (before a barrier
// after which another wave's DMA may overwrite what this wave read).
#define AMS_WAIT_VM_LDS(n) \
    __builtin_amdgcn_s_waitcnt(((n) & 0xF) | (((n) >> 4) << 14) | (0x7 << 4))

template <int NT>
struct L1Ring {
    static constexpr int BM = 64, BK = 32;
    static constexpr int ROWS = BM + NT;                 // A rows then B rows
    static constexpr int SLOT = ROWS * BK;               // floats per ring slot
    static constexpr int PER_WAVE = ROWS / 8 / 4;        // DMA instructions per wave per stage
};

template <int NT>
__device__ __forceinline__ void l1_issue(float *slot, const float *const *src, int k0, int wave)
{
#pragma unroll
    for (int q = 0; q < L1Ring<NT>::PER_WAVE; ++q)
        dma16(src[q] + k0, slot + (wave * L1Ring<NT>::PER_WAVE + q) * 256);
}

// Operands of one K step: for k-group g (4 consecutive k per lane) the A
// row's 16 bytes and the 16 bytes of each B row; the reads of group g+1 are
// issued while the MFMAs of group g run (sched_group_barrier fixes the
// interleave: 1 + NB LDS reads, then 4 NB MFMAs).
template <int NT>
__device__ __forceinline__ void l1_compute(const float *slot, v16f *acc, int lane, int wave)
{
    constexpr int NB = NT / 64;
    const int h = lane >> 5, r32 = lane & 31, wm = wave >> 1, wn = wave & 1;
    const int ra = wm * 32 + r32;
    float4 a[4], b[4][NB];
#pragma unroll
    for (int g = 0; g < 4; ++g) {
        const int q = h * 4 + g;
        a[g] = *(const float4 *)&slot[ra * 32 + ((q ^ ring_swz(ra)) << 2)];
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
            const int rb = 64 + wn * (NT / 2) + nb * 32 + r32;
            b[g][nb] = *(const float4 *)&slot[rb * 32 + ((q ^ ring_swz(rb)) << 2)];
        }
    }
#pragma unroll
    for (int g = 0; g < 4; ++g) {
        const float av[4] = {a[g].x, a[g].y, a[g].z, a[g].w};
#pragma unroll
        for (int e = 0; e < 4; ++e)
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) {
                const float bv[4] = {b[g][nb].x, b[g][nb].y, b[g][nb].z, b[g][nb].w};
                acc[nb] = mfma_f32(av[e], bv[e], acc[nb]);
            }
    }
    // group 0's reads first, then (reads of g+1, MFMAs of g)
    __builtin_amdgcn_sched_group_barrier(0x100, 1 + NB, 0);
#pragma unroll
    for (int g = 0; g < 4; ++g) {
        if (g < 3) __builtin_amdgcn_sched_group_barrier(0x100, 1 + NB, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 4 * NB, 0);
    }
}

template <int NT>
__global__ __launch_bounds__(kThreads) void l1_fwd_f32(const float *__restrict__ T, int64_t n_rows,
                                                        int F, const int32_t *__restrict__ uniq,
                                                        const int32_t *__restrict__ n_uniq_p,
                                                        int cap, int n_mt, const float *__restrict__ W1,
                                                        const float *__restrict__ b1, int H,
                                                        float *__restrict__ H1, int keep_z)
{
    using R = L1Ring<NT>;
    constexpr int NB = NT / 64;
    constexpr int PW = R::PER_WAVE;
    __shared__ __attribute__((aligned(16))) float ring0[R::SLOT];
    __shared__ __attribute__((aligned(16))) float ring1[R::SLOT];
    __shared__ __attribute__((aligned(16))) float ring2[R::SLOT];
    __shared__ int rid[R::BM];

    const int n_u = min(*n_uniq_p, cap);   // never past the caller's buffers
    int mt, nt;
    if (!xcd_tile(blockIdx.x, n_mt, H / NT, mt, nt)) return;
    const int m0 = mt * R::BM;
    if (m0 >= n_u) return;
    const int n0 = nt * NT;
    const int t = threadIdx.x, lane = ams_lane(), wave = t / AMS_WAVE;
    if (t < R::BM) {
        int id = -1;
        if (m0 + t < n_u) {
            id = uniq[m0 + t];
            if (id < 0 || (int64_t)id >= n_rows) id = -1;   // reads as a zero row
        }
        rid[t] = id;
    }
    __syncthreads();

    // per-lane source of each of this wave's DMA instructions
    const float *src[PW];
#pragma unroll
    for (int q = 0; q < PW; ++q) {
        const int row = (wave * PW + q) * 8 + (lane >> 3);
        const int chunk = (lane & 7) ^ ring_swz(row);
        if (row < R::BM) {
            const int id = rid[row];
            src[q] = (id >= 0 ? T + (size_t)id * F : W1) + chunk * 4;
        } else {
            src[q] = W1 + (size_t)(n0 + row - R::BM) * F + chunk * 4;
        }
    }

    v16f acc[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[nb] = (v16f){};

    const int S = F / R::BK;
    // stage s lives in ring slot s % 3; stage s + 2 is issued while s computes.
    // Past the end the last stage is reloaded into a slot nobody reads again,
    // which keeps every wave's count of outstanding DMA uniform.
#define L1_STAGE(cur, nxt, s)                                                    \
    do {                                                                         \
        __builtin_amdgcn_sched_barrier(0);                                         \
        AMS_WAIT_VM_LDS(PW);                                                     \
        __builtin_amdgcn_s_barrier();                                            \
        __builtin_amdgcn_sched_barrier(0);                                       \
        l1_issue<NT>(nxt, src, min((s) + 2, S - 1) * R::BK, wave);               \
        __builtin_amdgcn_sched_barrier(0);                                       \
        l1_compute<NT>(cur, acc, lane, wave);                                    \
    } while (0)

    l1_issue<NT>(ring0, src, 0, wave);
    l1_issue<NT>(ring1, src, min(1, S - 1) * R::BK, wave);
    int s = 0;
    for (; s + 3 <= S; s += 3) {
        L1_STAGE(ring0, ring2, s);
        L1_STAGE(ring1, ring0, s + 1);
        L1_STAGE(ring2, ring1, s + 2);
    }
    if (s < S) L1_STAGE(ring0, ring2, s);
    if (s + 1 < S) L1_STAGE(ring1, ring0, s + 1);
#undef L1_STAGE
    AMS_WAIT_VM(0);

#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
        const int col = n0 + (wave & 1) * (NT / 2) + nb * 32 + (lane & 31);
        const float bias = b1[col];
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            const int r = (wave >> 1) * 32 + acc_row(j, lane);
            const int row = m0 + r;
            const float z = rid[r] >= 0 ? acc[nb][j] + bias : bias;
            if (row < n_u) H1[(size_t)row * H + col] = keep_z ? z : fmaxf(z, 0.f);
        }
    }
}

// Stream-K forward of the 4096-wide layer (used when H is a multiple of
// 256).  Work = (BM-row x 256-column tile, K stage) iterations in tile-major
// order; a K stage is 128 bytes of every operand row (32 fp32 or 64 bf16).
// Each of G persistent workers (one 8-wave block per CU) takes an equal
// contiguous share, so every CU gets the same MFMA work for any number of
// unique images.  A tile fully inside one worker's share is finished in place
// (bias, ReLU); a tile cut by a share boundary leaves one partial accumulator
// tile per worker, and the tail forward (which reads H1 anyway) adds the
// pieces in K order.  Waves are 4 (M) x 2 (N), each BM/4 rows x 128 columns;
// rows stream HBM->LDS by DMA with the row swizzle of l1_fwd_f32, through a
// ring of R slots of BM + 256 rows (BM = 128, R = 3: 48 KB per slot, two
// stages in flight while one is consumed).  A 256-row tile with a 2-slot ring
// (64 KB slots) halves the W1 bytes per gathered byte but measured slower in
// bf16 at every workload here: one stage in flight, and too few tiles to fill
// the chip at ~13k unique images.
// With the whole hidden width in one tile a feature row is read from HBM once.
//
// fp32: within a stage lane l supplies k = 16*(l/32) + 4*g + e to element e
// of k-group g (one 32x32x2 MFMA per element).  bf16: the same 16-byte chunk
// holds 8 values, k = 32*(l/32) + 8*g + e, one 32x32x16 MFMA per group.  A
// and B agree, so the sum over the stage's k is unchanged.
constexpr int kSkThreads = 512;
constexpr int kSkBN = 256;
constexpr int kSkNB = kSkBN / 64;                         // 32-column MFMA blocks per wave: 4
constexpr int kSkMinIters = 32;                           // smallest share worth a worker

template <int BM_, int R_, int RB_>
struct SkShape {
    static constexpr int BM = BM_;                           // image rows per tile
    static constexpr int R = R_;                             // ring slots
    static constexpr int RB = RB_;                           // bytes of an operand row per stage
    static constexpr int MB = BM / 128;                      // 32-row MFMA blocks per wave
    static constexpr int ROWS = BM + kSkBN;                  // A rows then B rows
    static constexpr int SLOT = ROWS * RB / 4;               // floats per ring slot
    static constexpr int CPR = RB / 16;                      // 16-byte chunks per stage row
    static constexpr int RPI = 64 / CPR;                     // rows per DMA instruction
    static constexpr int PW = ROWS / RPI / (kSkThreads / 64); // DMA instructions per wave
    static constexpr int G = CPR / 2;                        // k groups per stage (chunk h G + g)
    static constexpr int TILE = BM * kSkBN;                  // floats per partial tile
};

// 128-row tiles, 128-byte stage rows, 3 slots (48 KB each) for both types.
// (256-row bf16 tiles with 64-byte stages and a 4-slot ring cut the W1
// stream per row in half and the layer-1 time by 7% on 163k unique rows, but
// doubled the partial-tile bytes the tail kernel adds up, which cost as much
// again.)
template <typename TT>
struct Sk : SkShape<128, 3, 128> {};

template <typename TT>
constexpr int sk_bk() { return Sk<TT>::RB / (int)sizeof(TT); }   // K per stage

// Chunk swizzle of a 128-byte stage row: chunk ^ (row / 2 % 8).  The LDS
// serves a 16-byte read for 16 lanes per cycle over 64 banks; rows r and
// r + 1 fall in different bank halves, so the even (odd) rows of 16
// consecutive ones need 8 distinct chunk positions (the one-tile-per-block
// ring's swizzle, bits 0-2 of the row, gives 4: counters showed 2-way
// conflicts).  A lane's rows differ by multiples of 32, which leave it
// unchanged.
template <class K>
__device__ __forceinline__ int sk_swz(int row)
{
    static_assert(K::CPR == 8, "stage rows of 8 chunks");
    return (row >> 1) & 7;
}

struct SkPlan {
    int n_u, n_cb, S, g;            // g = workers in use
    int64_t total;
    __device__ int64_t it0(int w) const { return total * w / g; }
    __device__ int owner(int64_t it) const { return (int)(((it + 1) * g - 1) / total); }
};

__device__ __forceinline__ SkPlan sk_plan(int n_u, int H, int F, int G, int bk, int bm)
{
    SkPlan p;
    p.n_u = n_u;
    p.n_cb = H / kSkBN;
    p.S = F / bk;
    const int64_t tiles = (int64_t)((n_u + bm - 1) / bm) * p.n_cb;
    p.total = tiles * p.S;
    const int64_t want = (p.total + kSkMinIters - 1) / kSkMinIters;
    p.g = (int)(want < G ? want : G);
    if (p.g < 1) p.g = 1;
    return p;
}

// src[q] are byte pointers; k0b is the stage's byte offset within a row
template <typename TT>
__device__ __forceinline__ void sk_issue(float *slot, const char *const *src, int64_t k0b, int wave)
{
#pragma unroll
    for (int q = 0; q < Sk<TT>::PW; ++q) dma16(src[q] + k0b, slot + (wave * Sk<TT>::PW + q) * 256);
}

template <typename TT>
__device__ __forceinline__ void sk_compute(const float *slot, v16f (*acc)[kSkNB], int lane, int wave)
{
    using K = Sk<TT>;
    constexpr int G = K::G, RF = K::RB / 4;                    // k groups, floats per stage row
    const int h = lane >> 5, r32 = lane & 31, wm = wave >> 1, wn = wave & 1;
    uint4 a[G][K::MB], b[G][kSkNB];
    // every row this lane reads is r32 plus a multiple of 32, which leaves the
    // swizzle unchanged: one lane offset per k group, the blocks at constant
    // distances from it
    const int sw = sk_swz<K>(r32);
    const float *pa = slot + (wm * 32 * K::MB + r32) * RF;
    const float *pb = slot + (K::BM + wn * (kSkBN / 2) + r32) * RF;
#pragma unroll
    for (int g = 0; g < G; ++g) {
        const int off = ((h * G + g) ^ sw) << 2;
#pragma unroll
        for (int mb = 0; mb < K::MB; ++mb) a[g][mb] = *(const uint4 *)(pa + mb * 32 * RF + off);
#pragma unroll
        for (int nb = 0; nb < kSkNB; ++nb) b[g][nb] = *(const uint4 *)(pb + nb * 32 * RF + off);
    }
    constexpr int PER_G = sizeof(TT) == 4 ? 4 : 1;           // MFMAs per (group, block)
#pragma unroll
    for (int g = 0; g < G; ++g) {
        if constexpr (sizeof(TT) == 4) {
#pragma unroll
            for (int mb = 0; mb < K::MB; ++mb) {
                const float av[4] = {__uint_as_float(a[g][mb].x), __uint_as_float(a[g][mb].y),
                                     __uint_as_float(a[g][mb].z), __uint_as_float(a[g][mb].w)};
#pragma unroll
                for (int e = 0; e < 4; ++e)
#pragma unroll
                    for (int nb = 0; nb < kSkNB; ++nb) {
                        const float bv[4] = {__uint_as_float(b[g][nb].x), __uint_as_float(b[g][nb].y),
                                             __uint_as_float(b[g][nb].z), __uint_as_float(b[g][nb].w)};
                        acc[mb][nb] = mfma_f32(av[e], bv[e], acc[mb][nb]);
                    }
            }
        } else {
#pragma unroll
            for (int mb = 0; mb < K::MB; ++mb)
#pragma unroll
                for (int nb = 0; nb < kSkNB; ++nb) acc[mb][nb] = mfma_bf16(a[g][mb], b[g][nb], acc[mb][nb]);
        }
    }
    // group 0's reads first, then (reads of g+1, MFMAs of g)
    __builtin_amdgcn_sched_group_barrier(0x100, K::MB + kSkNB, 0);
#pragma unroll
    for (int g = 0; g < G; ++g) {
        if (g < G - 1) __builtin_amdgcn_sched_group_barrier(0x100, K::MB + kSkNB, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, PER_G * K::MB * kSkNB, 0);
    }
}

// Epilogue of a stream-K segment.  whole: the segment covered the tile's full
// K, so H1 = act(acc + b1) is written (b1 alone for a row whose ID is out of
// range; keep_z keeps the pre-activation); otherwise acc goes to this
// worker's partial tile `piece` (row-major, kSkBN floats per row).
template <int MB>
__device__ __forceinline__ void sk_store(const v16f (&acc)[MB][kSkNB], bool whole, const int *rid, int m0, int n0,
                                         int n_u, int H, const float *__restrict__ b1, int keep_z,
                                         float *__restrict__ H1, uint16_t *__restrict__ H1b,
                                         uint16_t *__restrict__ H1lo, float *__restrict__ piece, int lane, int wave)
{
    const int wm = wave >> 1, wn = wave & 1, r32 = lane & 31;
    // this lane's rows are rl0 + 32 mb + 8 (j / 4) + j % 4, its columns
    // c0 + 32 nb (MFMA accumulator layout)
    const int rl0 = wm * 32 * MB + 4 * (lane >> 5);
    const int c0 = wn * (kSkBN / 2) + r32;
    if (whole) {
        float bias[kSkNB];
#pragma unroll
        for (int nb = 0; nb < kSkNB; ++nb) bias[nb] = b1[n0 + c0 + nb * 32];
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
            for (int j = 0; j < 16; ++j) {
                const int r = rl0 + mb * 32 + 8 * (j >> 2) + (j & 3);
                if (m0 + r >= n_u) continue;
                const bool ok = rid[r] >= 0;
                const size_t o = (size_t)(m0 + r) * H + n0 + c0;
#pragma unroll
                for (int nb = 0; nb < kSkNB; ++nb) {
                    const float z0 = ok ? acc[mb][nb][j] + bias[nb] : bias[nb];
                    const float z = keep_z ? z0 : fmaxf(z0, 0.f);
                    if (H1) H1[o + nb * 32] = z;
                    if (H1b) {
                        const uint16_t hi = ams_f32_to_bf16(z);
                        H1b[o + nb * 32] = hi;
                        if (H1lo) H1lo[o + nb * 32] = ams_f32_to_bf16(z - ams_bf16_to_f32(hi));
                    }
                }
            }
    } else {
        float *pp = piece + rl0 * kSkBN + c0;
#pragma unroll
        for (int mb = 0; mb < MB; ++mb)
#pragma unroll
            for (int j = 0; j < 16; ++j)
#pragma unroll
                for (int nb = 0; nb < kSkNB; ++nb)
                    pp[(mb * 32 + 8 * (j >> 2) + (j & 3)) * kSkBN + nb * 32] = acc[mb][nb][j];
    }
}

// H1b (bf16 mode): the bf16 copy of H1 kept for the backward, written with H1
// for tiles finished in place; H1lo, if given, the bf16 rounding of what H1b
// leaves out (H1 = H1b + H1lo to 2^-18 relative), the fp32-level operand of
// the bf16 layer-2 product.
template <typename TT>
__global__ __launch_bounds__(kSkThreads) void l1sk(const TT *__restrict__ T, int64_t n_rows, int F,
                                                   const int32_t *__restrict__ uniq,
                                                   const int32_t *__restrict__ n_uniq_p, int cap,
                                                   const TT *__restrict__ W1, const float *__restrict__ b1,
                                                   int H, int G, float *__restrict__ H1,
                                                   uint16_t *__restrict__ H1b, uint16_t *__restrict__ H1lo,
                                                   float *__restrict__ pbuf, int keep_z)
{
    using K = Sk<TT>;
    constexpr int BK = sk_bk<TT>();
    __shared__ __attribute__((aligned(16))) float ring0[K::SLOT];
    __shared__ __attribute__((aligned(16))) float ring1[K::SLOT];
    __shared__ __attribute__((aligned(16))) float ring2[K::SLOT];
    __shared__ int rid[K::BM];

    const int n_u = min(*n_uniq_p, cap);
    if (n_u <= 0) return;
    const SkPlan P = sk_plan(n_u, H, F, G, BK, K::BM);
    // workers with consecutive shares sit on one XCD (blocks go round-robin)
    const int w = (blockIdx.x & 7) * (G >> 3) + (blockIdx.x >> 3);
    if (w >= P.g) return;
    const int64_t it1 = P.it0(w + 1);
    const int t = threadIdx.x, lane = ams_lane(), wave = t / AMS_WAVE;
    const int S = P.S;
    const size_t row_bytes = (size_t)F * sizeof(TT);
    bool first = true;
    for (int64_t it = P.it0(w); it < it1;) {
        const int tile = (int)(it / S);
        const int ks = (int)(it % S);
        const int ke = (int)min<int64_t>(S, ks + (it1 - it));
        const int m0 = (tile / P.n_cb) * K::BM, n0 = (tile % P.n_cb) * kSkBN;
        __syncthreads();                        // previous segment done with rid and the ring
        if (t < K::BM) {
            int id = -1;
            if (m0 + t < n_u) {
                id = uniq[m0 + t];
                if (id < 0 || (int64_t)id >= n_rows) id = -1;
            }
            rid[t] = id;
        }
        __syncthreads();
        const char *src[K::PW];
#pragma unroll
        for (int q = 0; q < K::PW; ++q) {
            const int row = (wave * K::PW + q) * K::RPI + lane / K::CPR;
            const int chunk = (lane % K::CPR) ^ sk_swz<K>(row);
            if (row < K::BM) {
                const int id = rid[row];
                src[q] = (id >= 0 ? (const char *)T + (size_t)id * row_bytes : (const char *)W1) + chunk * 16;
            } else {
                src[q] = (const char *)W1 + (size_t)(n0 + row - K::BM) * row_bytes + chunk * 16;
            }
        }
        v16f acc[K::MB][kSkNB];
#pragma unroll
        for (int mb = 0; mb < K::MB; ++mb)
#pragma unroll
            for (int nb = 0; nb < kSkNB; ++nb) acc[mb][nb] = (v16f){};
        const int n = ke - ks;
        // 3 slots: at the top of stage s, stages s and s+1 may be in flight;
        // the wait leaves only s+1, the barrier (everyone done with the slot
        // of s-1) lets stage s+2 be issued into that slot, and stage s is
        // computed meanwhile.  Past the end the last stage is loaded again
        // (same data, into a slot nobody reads).
        static_assert(K::R == 3, "three ring slots");
        {
#define SK_STAGE(cur, nxt, s)                                                      \
    do {                                                                           \
        __builtin_amdgcn_sched_barrier(0);                                         \
        AMS_WAIT_VM_LDS(K::PW);                                                    \
        __builtin_amdgcn_s_barrier();                                              \
        __builtin_amdgcn_sched_barrier(0);                                         \
        sk_issue<TT>(nxt, src, (int64_t)(ks + min((s) + 2, n - 1)) * K::RB, wave); \
        __builtin_amdgcn_sched_barrier(0);                                         \
        sk_compute<TT>(cur, acc, lane, wave);                                      \
    } while (0)
            sk_issue<TT>(ring0, src, (int64_t)ks * K::RB, wave);
            sk_issue<TT>(ring1, src, (int64_t)(ks + min(1, n - 1)) * K::RB, wave);
            int s = 0;
            for (; s + 3 <= n; s += 3) {
                SK_STAGE(ring0, ring2, s);
                SK_STAGE(ring1, ring0, s + 1);
                SK_STAGE(ring2, ring1, s + 2);
            }
            if (s < n) SK_STAGE(ring0, ring2, s);
            if (s + 1 < n) SK_STAGE(ring1, ring0, s + 1);
#undef SK_STAGE
        }
        AMS_WAIT_VM(0);

        sk_store<K::MB>(acc, ks == 0 && ke == S, rid, m0, n0, n_u, H, b1, keep_z, H1, H1b, H1lo,
                        pbuf + ((size_t)w * 2 + (first ? 0 : 1)) * K::TILE, lane, wave);
        first = false;
        it += n;
    }
}

// ------------------------------------------------ bf16 layer 1, row split
// Z1 = T[uniq] W1^T for bf16 storage (H = 256, F = 4096) on large batches:
// each of G persistent blocks (one per CU) takes a contiguous range of the
// unique rows with the whole K, so no tile is cut (no partial tiles for the
// tail to add), and all blocks sweep K in step, so each XCD's L2 serves a W1
// slice to its 32 CUs at about the same time.  A block is 8 waves (two per
// SIMD) working in tiles of 256 rows; wave (wm, wn) computes rows
// 128 wm .. + 127 against units 64 wn .. + 63 (eight 32x32 accumulator
// blocks, 128 registers).
//
// The gathered feature rows are the dominant HBM stream.  They move by
// direct DMA (global_load_lds_dwordx4) into a 3-slot LDS ring, 2 stages
// ahead, one 64-k stage being 128 contiguous bytes of each of the tile's 256
// rows: every DMA instruction reads 8 whole 128-byte lines (8 rows), the
// access pattern that reads a scattered row set fastest (a lane-per-row
// pattern, 16 bytes of 32 rows per instruction, reached about 80 % of it),
// and carries the non-temporal hint so the streamed rows do not push W1 out
// of L2.  The stage's W1 slice (256 rows x 128 bytes) moves into a 2-slot
// ring the same way, 1 stage ahead.  Both operands are then 16-byte LDS
// reads (slot rows swizzled by 16-byte chunk, chunk ^ ((row >> 1) & 7), so a
// quarter-wave's reads of 16 rows hit distinct banks; the DMA lanes read the
// permuted chunks from global memory, within the same line).
//
// One stage sequence runs across all tiles of the block: the rows of the
// next tile's first two stages are in flight while the last stages of a
// tile and its epilogue run, and the next tile's IDs are loaded at the
// tile's first stage.  Every vector memory instruction of the stages (4 W1
// DMAs and 4 row DMAs per wave and stage, the 4 ID loads at a tile's first
// stage) comes from inline assembly, so the compiler adds no waits of its
// own: stage g waits with s_waitcnt vmcnt(4) (vmcnt(8) right after the ID
// loads), which completes everything up to its own W1 DMA (issued one stage
// earlier, after its rows).  Stages past the block's last tile issue the
// same DMAs from a zero row, so every stage issues the same count.
//
// DMA geometry: instruction q (0..3) of wave w fills the 8 slot rows
// 32 w + 8 q .. + 7, lane i row 32 w + 8 q + i / 8, 16-byte chunk i % 8;
// for feature rows, slot row 32 w + 8 q + a holds the tile's row
// 32 w + 4 a + q, so a lane's four rows are consecutive entries of uniq.
namespace rs {
constexpr int kThreads = 512;
constexpr int kWaves = kThreads / AMS_WAVE;
constexpr int kWavesPerSimd = kWaves / 4;
constexpr int BM = 256;                      // rows per tile
constexpr int BN = 256;                      // hidden units (the whole width)
constexpr int KS = 64;                       // k per stage: 128 bytes of a row
constexpr int kF = 4096;                     // feature width (the stages are unrolled for it)
constexpr int S = kF / KS;                   // stages per tile
constexpr int NX = 3;                        // feature-row slots (rows issued 2 stages ahead)
constexpr int NW = 2;                        // W1 slots (1 stage ahead)
constexpr int SLOT = BM * KS * 2;            // bytes per slot (32 KB, also BN * KS * 2)
constexpr int DMA = 4;                       // DMA instructions per wave and slot (8 slot rows each)
constexpr int WAIT = 4;                      // ops a stage may leave in flight (the next stage's rows)
constexpr int WAIT_AFTER_IDS = 8;            // ... and the 4 ID loads issued one stage earlier
static_assert(BM == BN && (NX + NW) * SLOT <= 160 * 1024, "the rings fit the LDS");
static_assert(DMA * 1024 * kWaves == SLOT && kWaves == 8, "four slot-row groups of 8 per wave; 2 x 4 waves");
static_assert(WAIT == DMA && WAIT_AFTER_IDS == DMA + 4, "wait counts follow the issue order");
static_assert(S > 3, "the next tile's first two stages are issued from the last two");
}  // namespace rs

// A zero feature row: rows past the block's range, rows whose ID is outside
// the table and the stages past the last tile read it (their products are
// then exactly 0, and Z1 = b1 for a bad ID).
__device__ __attribute__((aligned(256))) uint16_t rs_zero_row[rs::kF];

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// DMA of 64 lanes x 16 bytes from per-lane addresses, non-temporal, into
// LDS at lds_addr + 16 lane.
__device__ __forceinline__ void rs_dma_row(const char *src, uint32_t lds_addr)
{
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off nt"
                 :
                 : "s"(lds_addr), "v"(src)
                 : "memory", "m0");
}

// DMA of 64 lanes x 16 bytes from base + voff into LDS at lds_addr + 16 lane.
__device__ __forceinline__ void rs_dma16(const void *base, uint32_t voff, uint32_t lds_addr)
{
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2"
                 :
                 : "s"(lds_addr), "v"(voff), "s"(base)
                 : "memory", "m0");
}

// 4-byte load whose completion the stages count themselves.
__device__ __forceinline__ void rs_ld_id(int &v, const int32_t *p)
{
    asm volatile("global_load_dword %0, %1, off" : "=v"(v) : "v"(p) : "memory");
}

// 16-byte chunk swizzle of the 128-byte slot rows.  The LDS serves a
// 16-byte read for 16 lanes per cycle over 64 banks, so rows r and r + 1 sit
// in different bank halves and the even (odd) rows of 16 consecutive ones
// must use 8 distinct chunk positions: chunk ^ (row / 2 % 8).
__device__ __forceinline__ int rs_swz(int row) { return (row >> 1) & 7; }

// One stage's products from X slot xs and W1 slot ws: 4 k steps of 16, each
// 4 (row blocks) x 2 (unit blocks) MFMAs; the k step's 6 operand reads are
// issued while the previous step's products run.
__device__ __forceinline__ void rs_compute(const char *xs, const char *ws, const int (&ao)[4], const int (&bo)[4],
                                           v16f (&acc)[8])
{
    u32x4 a[4][4], b[4][2];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
#pragma unroll
        for (int rb = 0; rb < 4; ++rb) a[j][rb] = *(const u32x4 *)(xs + ao[j] + rb * 4096);
#pragma unroll
        for (int cb = 0; cb < 2; ++cb) b[j][cb] = *(const u32x4 *)(ws + bo[j] + cb * 4096);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int rb = 0; rb < 4; ++rb)
#pragma unroll
            for (int cb = 0; cb < 2; ++cb)
                acc[rb * 2 + cb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                    __builtin_bit_cast(bf16x8, a[j][rb]), __builtin_bit_cast(bf16x8, b[j][cb]), acc[rb * 2 + cb], 0, 0,
                    0);
    __builtin_amdgcn_sched_group_barrier(0x100, 6, 0);
#pragma unroll
    for (int j = 0; j < 3; ++j) {
        __builtin_amdgcn_sched_group_barrier(0x100, 6, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);
}

// H1b / H1lo: the bf16 rounding of H1 = ReLU(Z1 + b1) (keep_z: of Z1 + b1,
// the pre-activation PReLU keeps) and the bf16 rounding of what it leaves
// out (the tail's fp32-level layer-2 operand).
__global__ __launch_bounds__(rs::kThreads) __attribute__((amdgpu_waves_per_eu(rs::kWavesPerSimd, rs::kWavesPerSimd))) void l1rs_bf16(
    const uint16_t *__restrict__ T, int64_t n_rows, const int32_t *__restrict__ uniq,
    const int32_t *__restrict__ n_uniq_p, int cap, const uint16_t *__restrict__ W1, const float *__restrict__ b1,
    int G, uint16_t *__restrict__ H1b, uint16_t *__restrict__ H1lo, int keep_z)
{
    using namespace rs;
    __shared__ __attribute__((aligned(1024))) char ring[(NX + NW) * SLOT];
    const int n_u = min(*n_uniq_p, cap);
    if (n_u <= 0) return;
    const int r0 = (int)((int64_t)n_u * blockIdx.x / G), r1 = (int)((int64_t)n_u * (blockIdx.x + 1) / G);
    if (r0 >= r1) return;
    const int n_tiles = (r1 - r0 + BM - 1) / BM;
    const int lane = ams_lane(), h = lane >> 5, r32 = lane & 31;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / AMS_WAVE);
    const int wm = wave >> 2, wn = wave & 3;
    constexpr size_t row_bytes = (size_t)kF * 2;
    const uint32_t lds0 = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)ring);
    const uint32_t lds_x = lds0 + 4 * wave * 1024, lds_w = lds0 + NX * SLOT + 4 * wave * 1024;

    // this lane's DMA rows: slot row 32 wave + 8 q + lane / 8, chunk lane % 8
    // holding source chunk (lane % 8) ^ rs_swz(slot row)
    int co[DMA];
    uint32_t wdq[DMA];
#pragma unroll
    for (int q = 0; q < DMA; ++q) {
        const int srow = 32 * wave + 8 * q + (lane >> 3);
        co[q] = ((lane & 7) ^ rs_swz(srow)) << 4;
        wdq[q] = (uint32_t)(srow * row_bytes) + co[q];
    }
    // the tile rows of this lane's DMAs: 32 wave + 4 (lane / 8) + q
    const int lrow = 32 * wave + 4 * (lane >> 3);
    auto row_src = [&](int id, int r, int q) -> const char * {
        const bool ok = r < r1 && id >= 0 && (int64_t)id < n_rows;
        return (ok ? (const char *)T + (size_t)id * row_bytes : (const char *)rs_zero_row) + co[q];
    };
    // operand read offsets: A slot row 128 wm + 32 rb + r32, B slot row
    // 64 wn + 32 cb + r32, k step j taking chunk 2 j + h (k = 16 j + 8 h ..)
    int ao[4], bo[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int c = ((2 * j + h) ^ rs_swz(r32)) << 4;
        ao[j] = (128 * wm + r32) * 128 + c;
        bo[j] = (64 * wn + r32) * 128 + c;
    }
    // prologue: the biases and tile 0's IDs (waited for here, before any
    // DMA is in flight), then X(0), W(0), X(1)
    float bias[2];
#pragma unroll
    for (int cb = 0; cb < 2; ++cb) bias[cb] = b1[64 * wn + 32 * cb + r32];
    const char *xp[DMA];
#pragma unroll
    for (int q = 0; q < DMA; ++q) {
        const int r = r0 + lrow + q;
        xp[q] = row_src(uniq[min(r, r1 - 1)], r, q);
    }
    asm volatile("" ::"v"(bias[0]), "v"(bias[1]), "v"(xp[0]), "v"(xp[1]), "v"(xp[2]), "v"(xp[3]));
    const char *wb = (const char *)W1;
    uint32_t xs_d = 0;                       // X slot the next row DMA fills (bytes from the ring)
#pragma unroll
    for (int q = 0; q < DMA; ++q) {
        rs_dma_row(xp[q], lds_x + q * 1024);
        xp[q] += 128;
        asm volatile("" : "+v"(xp[q]));
    }
#pragma unroll
    for (int q = 0; q < DMA; ++q) rs_dma16(wb, wdq[q], lds_w + q * 1024);
    wb += 128;
#pragma unroll
    for (int q = 0; q < DMA; ++q) {
        rs_dma_row(xp[q], lds_x + SLOT + q * 1024);
        xp[q] += 128;
        asm volatile("" : "+v"(xp[q]));
    }
    xs_d = 2 * SLOT;
    uint32_t xs_c = 0;                       // X slot the next stage computes from
    int idn[DMA];

    for (int m = 0; m < n_tiles; ++m) {
        const int m0 = r0 + m * BM;
        const bool live = m0 + 128 * wm < r1;     // (uniform per wave)
        v16f acc[8];
#pragma unroll
        for (int x = 0; x < 8; ++x) acc[x] = (v16f){};
#pragma unroll
        for (int k = 0; k < S; ++k) {
            // this stage's rows and W1 slice have landed (all waves: the
            // barrier), and every wave is done with the slots refilled below
            if (k == 1)
                asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)" ::"n"(WAIT_AFTER_IDS) : "memory");
            else
                asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)" ::"n"(WAIT) : "memory");
            __builtin_amdgcn_sched_barrier(0);
            if (k == 2) {
                // the ID loads of stage 0 have landed: until here their
                // registers stay reserved whatever uses the values later
#pragma unroll
                for (int q = 0; q < DMA; ++q) asm volatile("" : "+v"(idn[q]));
            }
            __builtin_amdgcn_s_barrier();
            __builtin_amdgcn_sched_barrier(0);
            // W1 of the next stage (k + 1, the next tile's 0 after 63)
#pragma unroll
            for (int q = 0; q < DMA; ++q) rs_dma16(wb, wdq[q], lds_w + ((k + 1) & 1) * SLOT + q * 1024);
            wb = (k == S - 2) ? (const char *)W1 : wb + 128;
            asm volatile("" : "+s"(wb));
            // rows of stage k + 2 (the next tile's first two from k = S - 2)
            if (k == S - 2) {
#pragma unroll
                for (int q = 0; q < DMA; ++q) xp[q] = row_src(idn[q], m0 + BM + lrow + q, q);
            }
#pragma unroll
            for (int q = 0; q < DMA; ++q) {
                rs_dma_row(xp[q], lds_x + xs_d + q * 1024);
                xp[q] += 128;
                asm volatile("" : "+v"(xp[q]));
            }
            xs_d = xs_d == (NX - 1) * SLOT ? 0 : xs_d + SLOT;
            if (k == 0) {
                // the next tile's IDs (rows past the range are clamped, then zero rows)
#pragma unroll
                for (int q = 0; q < DMA; ++q) rs_ld_id(idn[q], uniq + min(m0 + BM + lrow + q, r1 - 1));
            }
            __builtin_amdgcn_sched_barrier(0);
            if (live) rs_compute(ring + xs_c, ring + NX * SLOT + (k & 1) * SLOT, ao, bo, acc);
            xs_c = xs_c == (NX - 1) * SLOT ? 0 : xs_c + SLOT;
            __builtin_amdgcn_sched_barrier(0);        // the products stay ahead of the next wait
        }
        if (!live) continue;
        // accumulator element j of block (rb, cb): slot row 128 wm + 32 rb +
        // 8 (j / 4) + 4 h + j % 4, i.e. tile row 32 (4 wm + rb) + 16 h + 4 (j % 4) + j / 4;
        // unit 64 wn + 32 cb + r32
        const int rbase = m0 + 128 * wm + 16 * h;
        typedef __attribute__((address_space(1))) uint16_t gu16;
        gu16 *hb = (gu16 *)(H1b + (size_t)rbase * BN + 64 * wn + r32);
        gu16 *hl = (gu16 *)(H1lo + (size_t)rbase * BN + 64 * wn + r32);
        asm volatile("" : "+v"(hb), "+v"(hl));
#pragma unroll
        for (int rb = 0; rb < 4; ++rb)
#pragma unroll
            for (int j = 0; j < 16; ++j) {
                const int dr = 32 * rb + 4 * (j & 3) + (j >> 2);
                if (rbase + dr >= r1) continue;
#pragma unroll
                for (int cb = 0; cb < 2; ++cb) {
                    const float z0 = acc[rb * 2 + cb][j] + bias[cb];
                    const float z = keep_z ? z0 : fmaxf(z0, 0.f);
                    const uint16_t hi = ams_f32_to_bf16(z);
                    hb[dr * BN + 32 * cb] = hi;
                    hl[dr * BN + 32 * cb] = ams_f32_to_bf16(z - ams_bf16_to_f32(hi));
                }
            }
    }
    // the DMAs issued past the last stage land before the block leaves
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

// ------------------------------------------- float32 layer 1 on bf16 MFMA
// (AMS_F32_X3.)  A float32 x is the exact sum of three bf16 values h =
// bf16(x), m = bf16(x - h), l = bf16(x - h - m), each rounded to nearest:
// both residuals are exact in float32 (x and h are within a factor 2 of each
// other), and at most 8 significant bits are left for l (exact while l is a
// normal number, |x| >= 2^-100).  Of the nine part
// products of x y the six kept (hh, hm, mh, hl, lh, mm) leave out
// |ml + lm + ll| < 2^-22 |x y| (|m| <= 2^-8 |x|, |l| <= 2^-16 |x|), and each
// part product is exact in the float32 accumulator.  A 16-deep k step is six
// bf16 MFMAs (6 x 32 cycles) in place of eight float32 ones (8 x 64).

__device__ __forceinline__ uint32_t cvt_pk_bf16(float a, float b)
{
    const bf16x2 v = {(__bf16)a, (__bf16)b};      // round to nearest even
    return __builtin_bit_cast(uint32_t, v);
}

// x[0..7] -> the three bf16x8 parts (element e in bits 16 e .. 16 e + 15)
__device__ __forceinline__ void split3x8(const float (&x)[8], uint4 &h, uint4 &m, uint4 &l)
{
    uint32_t hp[4], mp[4], lp[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const float x0 = x[2 * e], x1 = x[2 * e + 1];
        hp[e] = cvt_pk_bf16(x0, x1);
        const float r0 = x0 - __uint_as_float(hp[e] << 16), r1 = x1 - __uint_as_float(hp[e] & 0xffff0000u);
        mp[e] = cvt_pk_bf16(r0, r1);
        const float q0 = r0 - __uint_as_float(mp[e] << 16), q1 = r1 - __uint_as_float(mp[e] & 0xffff0000u);
        lp[e] = cvt_pk_bf16(q0, q1);
    }
    h = make_uint4(hp[0], hp[1], hp[2], hp[3]);
    m = make_uint4(mp[0], mp[1], mp[2], mp[3]);
    l = make_uint4(lp[0], lp[1], lp[2], lp[3]);
}

// W[n] float32 -> bf16 planes P[0, n) = h, P[n, 2n) = m, P[2n, 3n) = l; n % 8 == 0
__global__ __launch_bounds__(kThreads) void split3_k(const float *__restrict__ W, int64_t n, uint16_t *__restrict__ P)
{
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n / 8; i += (int64_t)gridDim.x * kThreads) {
        const float4 a = *(const float4 *)(W + 8 * i), b = *(const float4 *)(W + 8 * i + 4);
        const float x[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
        uint4 h, m, l;
        split3x8(x, h, m, l);
        *(uint4 *)(P + 8 * i) = h;
        *(uint4 *)(P + n + 8 * i) = m;
        *(uint4 *)(P + 2 * n + 8 * i) = l;
    }
}

// Stream-K layer 1 with the split: the tiles, shares and partial tiles of
// l1sk<float> (128 x 256 tiles, 32 k per stage).  A stage slot holds the
// 128 feature rows (float32, 128 bytes each, chunk c at c ^ (row / 2 % 8),
// as in l1sk)
// and the three bf16 planes of the tile's 256 W1 rows (64 bytes each,
// chunk c at c ^ ((row >> 2) & 3)); 64 KB per slot, two slots.  Every wave
// issues 2 DMA instructions of feature rows and 6 of planes per stage (the
// gathers spread over all waves).  Each wave splits its feature operand after
// the LDS read; W1 comes split (split3_k).  (Deeper rings with 16-k stages,
// and four waves with double-buffered operands, measured no faster: the
// stream of W1 parts, 6 MB per tile, sets the pace.)
struct X3 {
    static constexpr int BM = 128;
    static constexpr int BK = 32;                          // k per stage
    static constexpr int A_FL = BM * 32;                   // floats of feature rows per slot
    static constexpr int PL_FL = kSkBN * 16;               // floats per W1 plane per slot
    static constexpr int SLOT = A_FL + 3 * PL_FL;          // 16384 floats
    static constexpr int PW = SLOT / 256 / (kSkThreads / AMS_WAVE);   // DMA instructions per wave
    static constexpr int TILE = BM * kSkBN;
};
static_assert(X3::TILE == Sk<float>::TILE && X3::BM == Sk<float>::BM && X3::BK == sk_bk<float>(),
              "the split kernel leaves its partial tiles in the float32 layout");
static_assert(X3::PW == 8 && X3::A_FL / 256 == 2 * (kSkThreads / AMS_WAVE), "2 feature-row instructions per wave");

__device__ __forceinline__ void x3_compute(const float *slot, v16f (&acc)[1][kSkNB], int lane, int wave)
{
    const int h = lane >> 5, r32 = lane & 31, wm = wave >> 1, wn = wave & 1;
    // rows read are r32 plus multiples of 32: one swizzle per lane
    const float *pa = slot + (wm * 32 + r32) * 32;
    const int swa = (r32 >> 1) & 7;
    const float *pb = slot + X3::A_FL + (wn * (kSkBN / 2) + r32) * 16;
    const int swb = (r32 >> 2) & 3;
#pragma unroll
    for (int g = 0; g < 2; ++g) {
        const int ca = 4 * g + 2 * h;                      // k = 16 g + 8 h .. + 7
        const float4 x0 = *(const float4 *)(pa + ((ca ^ swa) << 2));
        const float4 x1 = *(const float4 *)(pa + (((ca + 1) ^ swa) << 2));
        const int cb = ((2 * g + h) ^ swb) << 2;
        uint4 bh[kSkNB], bm[kSkNB], bl[kSkNB];
#pragma unroll
        for (int nb = 0; nb < kSkNB; ++nb) {
            bh[nb] = *(const uint4 *)(pb + nb * 32 * 16 + cb);
            bm[nb] = *(const uint4 *)(pb + X3::PL_FL + nb * 32 * 16 + cb);
            bl[nb] = *(const uint4 *)(pb + 2 * X3::PL_FL + nb * 32 * 16 + cb);
        }
        const float x[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
        uint4 ah, am, al;
        split3x8(x, ah, am, al);
#pragma unroll
        for (int nb = 0; nb < kSkNB; ++nb) {
            v16f c = acc[0][nb];
            c = mfma_bf16(ah, bh[nb], c);
            c = mfma_bf16(ah, bm[nb], c);
            c = mfma_bf16(am, bh[nb], c);
            c = mfma_bf16(ah, bl[nb], c);
            c = mfma_bf16(al, bh[nb], c);
            c = mfma_bf16(am, bm[nb], c);
            acc[0][nb] = c;
        }
    }
}

__global__ __launch_bounds__(kSkThreads) void l1sk_x3(const float *__restrict__ T, int64_t n_rows, int F,
                                                      const int32_t *__restrict__ uniq,
                                                      const int32_t *__restrict__ n_uniq_p, int cap,
                                                      const float *__restrict__ W1,
                                                      const uint16_t *__restrict__ W1p,
                                                      const float *__restrict__ b1, int H, int G,
                                                      float *__restrict__ H1, float *__restrict__ pbuf,
                                                      int keep_z)
{
    __shared__ __attribute__((aligned(16))) float ring0[X3::SLOT];
    __shared__ __attribute__((aligned(16))) float ring1[X3::SLOT];
    __shared__ int rid[X3::BM];

    const int n_u = min(*n_uniq_p, cap);
    if (n_u <= 0) return;
    const SkPlan P = sk_plan(n_u, H, F, G, X3::BK, X3::BM);
    const int w = (blockIdx.x & 7) * (G >> 3) + (blockIdx.x >> 3);
    if (w >= P.g) return;
    const int64_t it1 = P.it0(w + 1);
    const int t = threadIdx.x, lane = ams_lane(), wave = t / AMS_WAVE;
    const int S = P.S;
    const size_t plane = (size_t)H * F;
    bool first = true;
    for (int64_t it = P.it0(w); it < it1;) {
        const int tile = (int)(it / S);
        const int ks = (int)(it % S);
        const int ke = (int)min<int64_t>(S, ks + (it1 - it));
        const int m0 = (tile / P.n_cb) * X3::BM, n0 = (tile % P.n_cb) * kSkBN;
        __syncthreads();                        // previous segment done with rid and the ring
        if (t < X3::BM) {
            int id = -1;
            if (m0 + t < n_u) {
                id = uniq[m0 + t];
                if (id < 0 || (int64_t)id >= n_rows) id = -1;
            }
            rid[t] = id;
        }
        __syncthreads();
        const char *src[X3::PW];
#pragma unroll
        for (int q = 0; q < X3::PW; ++q) {
            if (q < 2) {                        // feature rows 8 ja .. 8 ja + 7
                const int ja = 2 * wave + q;
                const int row = 8 * ja + (lane >> 3);
                const int chunk = (lane & 7) ^ ((row >> 1) & 7);
                const int id = rid[row];
                src[q] = (id >= 0 ? (const char *)(T + (size_t)id * F) : (const char *)W1) + chunk * 16;
            } else {                            // plane jb / 16, W1 rows 16 (jb % 16) .. + 15
                const int jb = 6 * wave + q - 2, pl = jb >> 4;
                const int rb = 16 * (jb & 15) + (lane >> 2);
                const int chunk = (lane & 3) ^ ((rb >> 2) & 3);
                src[q] = (const char *)(W1p + pl * plane + (size_t)(n0 + rb) * F) + chunk * 16;
            }
        }
        v16f acc[1][kSkNB];
#pragma unroll
        for (int nb = 0; nb < kSkNB; ++nb) acc[0][nb] = (v16f){};
        const int n = ke - ks;
        auto issue = [&](float *slot, int st) {
#pragma unroll
            for (int q = 0; q < 2; ++q) dma16(src[q] + (int64_t)st * 128, slot + (2 * wave + q) * 256);
#pragma unroll
            for (int q = 2; q < X3::PW; ++q)
                dma16(src[q] + (int64_t)st * 64, slot + X3::A_FL + (6 * wave + q - 2) * 256);
        };
        // 2 slots: at the top of stage s only stage s is in flight; after the
        // barrier (everyone is done with the other slot) stage s+1 is issued
        // into it and stage s is computed meanwhile.
#define X3_STAGE(cur, nxt, s)                                                      \
    do {                                                                           \
        __builtin_amdgcn_sched_barrier(0);                                         \
        AMS_WAIT_VM_LDS(0);                                                        \
        __builtin_amdgcn_s_barrier();                                              \
        __builtin_amdgcn_sched_barrier(0);                                         \
        if ((s) + 1 < n) issue(nxt, ks + (s) + 1);                                 \
        __builtin_amdgcn_sched_barrier(0);                                         \
        x3_compute(cur, acc, lane, wave);                                          \
    } while (0)
        issue(ring0, ks);
        int s = 0;
        for (; s + 2 <= n; s += 2) {
            X3_STAGE(ring0, ring1, s);
            X3_STAGE(ring1, ring0, s + 1);
        }
        if (s < n) X3_STAGE(ring0, ring1, s);
#undef X3_STAGE
        AMS_WAIT_VM(0);
        sk_store<1>(acc, ks == 0 && ke == S, rid, m0, n0, n_u, H, b1, keep_z, H1, nullptr, nullptr,
                    pbuf + ((size_t)w * 2 + (first ? 0 : 1)) * X3::TILE, lane, wave);
        first = false;
        it += n;
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

// ------------------------------------------------------- tail layers

__device__ __forceinline__ float ld_w(const void *W, int bf16, size_t i)
{
    return bf16 ? ams_bf16_to_f32(((const uint16_t *)W)[i]) : ((const float *)W)[i];
}

// Four consecutive elements (index i, a multiple of 4) of a float32 or bf16 array.
__device__ __forceinline__ float4 ld4_any(const void *p, int bf16, size_t i)
{
    if (bf16) {
        const uint2 v = *(const uint2 *)((const uint16_t *)p + i);
        return make_float4(__uint_as_float(v.x << 16), __uint_as_float(v.x & 0xffff0000u),
                           __uint_as_float(v.y << 16), __uint_as_float(v.y & 0xffff0000u));
    }
    return *(const float4 *)((const float *)p + i);
}

// Both tail kernels walk their unique images in chunks of 32 rows and run
// the small contractions on fp32 MFMA (32x32x2) with operands in LDS.  Layer
// widths: H = dims[1] (64..256, a multiple of 64), Mo = width of the second
// layer's output (dims[2] for 3 layers, D for 2), padded to 64 with zeros.
constexpr int kTailRows = 32;

// Forward: Z2 = H1 W2^T + b2 for a chunk of 32 rows.  Wave w computes output
// columns 32 (w & 1) .. +32 over the K half w >> 1; the two halves are added
// in a fixed order.  Each lane keeps its W2 operands for the whole kernel in
// registers (row o of W2, 16 consecutive k per 32-k block) and reads its H1
// row straight from global memory, so only the small combine tiles use LDS.
// Then H2 = ReLU(Z2) and, for 3 layers, E = H2 W3^T + b3.
//
// After the stream-K forward (sk_bk != 0: its K per stage) the K half of wave w lies in one
// column tile of layer 1 (the row block's only tile when H = 256).  If a
// worker finished that tile in place its H1 is read as is; otherwise the wave
// adds the workers' partial tiles in K order, applies b1 and ReLU (ReLU(b1)
// for a row whose ID is out of range) and writes the finished H1 for the
// backward.
template <int L, bool PR>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2))) void tail_fwd(float *__restrict__ H1, int H, int M,
                                                      int D, const void *__restrict__ W2,
                                                      const float *__restrict__ b2,
                                                      const void *__restrict__ W3,
                                                      const float *__restrict__ b3, int wbf16,
                                                      int final_relu,
                                                      const int32_t *__restrict__ n_uniq_p, int cap,
                                                      float *__restrict__ H2_save,
                                                      float *__restrict__ E, int sk_bk, int F, int G,
                                                      const float *__restrict__ pbuf,
                                                      uint16_t *__restrict__ H1b,
                                                      const float *__restrict__ b1,
                                                      const int32_t *__restrict__ uniq, int64_t n_rows,
                                                      const float *__restrict__ s1, const float *__restrict__ s2)
{
    constexpr int KB = kMaxH1 / 2 / 32;       // 32-k blocks in a K half (at most 4)
    constexpr int KH = KB / 2;                // ... added up by each wave of a K half's pair
    // (rows 72 floats apart: the two lane halves' rows, 4 apart, then fall
    // in opposite bank halves when a wave stores its accumulator)
    __shared__ float Zp[2][kTailRows][kMaxH2 + 8];
    __shared__ float W3s[kMaxD * (kMaxH2 + 1)];
    __shared__ float h2s[kTailRows][kMaxH2 + 1];
    __shared__ __attribute__((aligned(16))) float H1s[kTailRows][kMaxH1 + 4];   // finished rows of a cut tile
    __shared__ __attribute__((aligned(16))) float b1s[kMaxH1];
    __shared__ float b2s[kMaxH2], b3s[kMaxD];
    const int t = threadIdx.x, lane = ams_lane(), wave = t / AMS_WAVE;
    const int h = lane >> 5, r32 = lane & 31;
    const int kh = wave >> 1, nb = wave & 1, khalf = H / 2, nkb = khalf / 32;
    const int o = nb * 32 + r32;              // this lane's B row (output column)
    const int n_u = min(*n_uniq_p, cap);
    if (blockIdx.x * kTailRows >= n_u) return;    // the grid is sized by cap: no chunk for this block
    // this lane's W2 operands and W3 (D * M <= 8 kThreads): every load
    // unconditional (an index outside the weights reads element 0 and is
    // dropped) and inside one branch on the storage type, so they are all in
    // flight together instead of one wait each
    float4 breg[KB][4];
    float w3v[8];
    auto w2_at = [&](int kb, int q) { return (size_t)o * H + kh * khalf + kb * 32 + 16 * h + 4 * q; };
    if (wbf16) {
        uint2 r2[KB][4];
        uint16_t r3[8];
#pragma unroll
        for (int kb = 0; kb < KB; ++kb)
#pragma unroll
            for (int q = 0; q < 4; ++q)
                r2[kb][q] = *(const uint2 *)((const uint16_t *)W2 + ((kb < nkb && o < M) ? w2_at(kb, q) : 0));
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int e = t + i * kThreads;
            r3[i] = L == 3 ? ((const uint16_t *)W3)[e < D * M ? e : 0] : (uint16_t)0;
        }
#pragma unroll
        for (int kb = 0; kb < KB; ++kb)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const uint2 v = r2[kb][q];
                breg[kb][q] = (kb < nkb && o < M)
                                  ? make_float4(__uint_as_float(v.x << 16), __uint_as_float(v.x & 0xffff0000u),
                                                __uint_as_float(v.y << 16), __uint_as_float(v.y & 0xffff0000u))
                                  : make_float4(0.f, 0.f, 0.f, 0.f);
            }
#pragma unroll
        for (int i = 0; i < 8; ++i) w3v[i] = ams_bf16_to_f32(r3[i]);
    } else {
#pragma unroll
        for (int kb = 0; kb < KB; ++kb)
#pragma unroll
            for (int q = 0; q < 4; ++q)
                breg[kb][q] = *(const float4 *)((const float *)W2 + ((kb < nkb && o < M) ? w2_at(kb, q) : 0));
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int e = t + i * kThreads;
            w3v[i] = L == 3 ? ((const float *)W3)[e < D * M ? e : 0] : 0.f;
        }
#pragma unroll
        for (int kb = 0; kb < KB; ++kb)
#pragma unroll
            for (int q = 0; q < 4; ++q)
                if (!(kb < nkb && o < M)) breg[kb][q] = make_float4(0.f, 0.f, 0.f, 0.f);
    }
    // W3 and the biases into LDS (the bias loads unconditional, in flight together)
    const float b3v = L == 3 ? b3[t < D ? t : 0] : 0.f;
    const float b2v = b2[t < M ? t : 0];
    const float b1v = sk_bk ? b1[t < H ? t : 0] : 0.f;
    if (L == 3) {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int e = t + i * kThreads;
            if (e < D * M) W3s[(e / M) * (kMaxH2 + 1) + e % M] = w3v[i];
        }
        if (t < D) b3s[t] = b3v;
    }
    if (t < M) b2s[t] = b2v;
    if (sk_bk && t < H) b1s[t] = b1v;
    const bool relu_a = (L == 3) || final_relu;
    for (int c0 = blockIdx.x * kTailRows; c0 < n_u; c0 += gridDim.x * kTailRows) {
        const int row = c0 + r32;
        const int rowc = min(row, n_u - 1);
        float *hrow = H1 + (size_t)rowc * H + kh * khalf + 16 * h;
        float4 areg[KB][4];
        // this wave's K half lies in one column tile of the stream-K grid
        const int cbase = kh * khalf;                    // first column of the half
        const int cb = cbase / kSkBN;
        int wa = 0, wb = -1, slot_a = 0;
        if (sk_bk) {
            // the chunk's 32 rows lie in one row tile (BM is a multiple of
            // 32): the plan is the same for the whole wave, worked out on the
            // scalar unit
            const SkPlan P = sk_plan(n_u, H, F, G, sk_bk, Sk<float>::BM);
            const int tile = __builtin_amdgcn_readfirstlane((c0 / Sk<float>::BM) * P.n_cb + cb);
            wa = __builtin_amdgcn_readfirstlane(P.owner((int64_t)tile * P.S));
            wb = __builtin_amdgcn_readfirstlane(P.owner((int64_t)(tile + 1) * P.S - 1));
            // only the first contributor can hold this tile as its second piece
            slot_a = (tile == (int)(P.it0(wa) / P.S)) ? 0 : 1;
        }
        const bool split = wb > wa;             // the same for the whole block (one column tile)
        if (split) {
            // tile cut by share boundaries: the two waves of this K half each
            // add up half of its 32-k blocks, the pieces in K order with the
            // loads of up to three shares in flight together (a tile spans at
            // most three shares; more are looped), apply b1 and the
            // activation, store H1 and pass the rows on through LDS
            const int id = uniq[rowc];
            const int rl = rowc % Sk<float>::BM;
            const float *pr = pbuf + (size_t)rl * kSkBN + (cbase - cb * kSkBN) + 16 * h;
            float4 v[3][KH][4];
            // (a 32-k block past the half reloads block 0: every load of a
            // share is issued unconditionally; such blocks are never used)
            auto load_share = [&](int w, int sl, float4 (&x)[KH][4]) {
                const float *pw = pr + ((size_t)w * 2 + sl) * Sk<float>::TILE;
#pragma unroll
                for (int i = 0; i < KH; ++i)
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const int kb = nb * KH + i;
                        x[i][q] = *(const float4 *)(pw + (kb < nkb ? kb * 32 : 0) + 4 * q);
                    }
            };
            auto add = [&](float4 (&acc4)[KH][4], const float4 (&x)[KH][4]) {
#pragma unroll
                for (int i = 0; i < KH; ++i)
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        acc4[i][q].x += x[i][q].x;
                        acc4[i][q].y += x[i][q].y;
                        acc4[i][q].z += x[i][q].z;
                        acc4[i][q].w += x[i][q].w;
                    }
            };
            load_share(wa, slot_a, v[0]);
            if (wa + 1 <= wb) load_share(wa + 1, 0, v[1]);
            if (wa + 2 <= wb) load_share(wa + 2, 0, v[2]);
            float4 sum[KH][4];
#pragma unroll
            for (int i = 0; i < KH; ++i)
#pragma unroll
                for (int q = 0; q < 4; ++q) sum[i][q] = make_float4(0.f, 0.f, 0.f, 0.f);
            add(sum, v[0]);
            if (wa + 1 <= wb) add(sum, v[1]);
            if (wa + 2 <= wb) add(sum, v[2]);
            for (int w = wa + 3; w <= wb; ++w) {
                load_share(w, 0, v[0]);
                add(sum, v[0]);
            }
            const bool ok = id >= 0 && (int64_t)id < n_rows;
#pragma unroll
            for (int i = 0; i < KH; ++i)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int kb = nb * KH + i;
                    if (kb >= nkb) continue;
                    const int col = cbase + kb * 32 + 16 * h + 4 * q;
                    float4 a = sum[i][q];
                    const float4 c = *(const float4 *)&b1s[col];
                    a.x = ok ? a.x + c.x : c.x;
                    a.y = ok ? a.y + c.y : c.y;
                    a.z = ok ? a.z + c.z : c.z;
                    a.w = ok ? a.w + c.w : c.w;
                    // PReLU keeps Z1 in H1 (activated below); ReLU stores H1
                    if (!PR) a = make_float4(fmaxf(a.x, 0.f), fmaxf(a.y, 0.f), fmaxf(a.z, 0.f), fmaxf(a.w, 0.f));
                    if (row < n_u) {
                        *(float4 *)(H1 + (size_t)rowc * H + col) = a;
                        if (H1b) {
                            uint16_t *hb = H1b + (size_t)rowc * H + col;
                            const uint32_t lo = ams_f32_to_bf16(a.x) | ((uint32_t)ams_f32_to_bf16(a.y) << 16);
                            const uint32_t hi = ams_f32_to_bf16(a.z) | ((uint32_t)ams_f32_to_bf16(a.w) << 16);
                            *(uint2 *)hb = make_uint2(lo, hi);
                        }
                    }
                    *(float4 *)&H1s[r32][col] = a;
                }
        }
        __syncthreads();                        // the pair's rows are in H1s
        if (split) {
#pragma unroll
            for (int kb = 0; kb < KB; ++kb)
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    areg[kb][q] = kb >= nkb ? make_float4(0.f, 0.f, 0.f, 0.f)
                                            : *(const float4 *)&H1s[r32][cbase + kb * 32 + 16 * h + 4 * q];
        } else {
            // every row load issued before any is used (a block past the
            // half reloads block 0 and is zeroed)
#pragma unroll
            for (int kb = 0; kb < KB; ++kb)
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    areg[kb][q] = *(const float4 *)(hrow + (kb < nkb ? kb * 32 : 0) + 4 * q);
#pragma unroll
            for (int kb = 0; kb < KB; ++kb)
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    if (kb >= nkb) areg[kb][q] = make_float4(0.f, 0.f, 0.f, 0.f);
        }
        if (PR) {
            // layer 1's PReLU on this lane's operands (Z1 -> H1), slope per column
#pragma unroll
            for (int kb = 0; kb < KB; ++kb)
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    if (kb < nkb) {
                        const float4 a = *(const float4 *)&s1[kh * khalf + kb * 32 + 16 * h + 4 * q];
                        float4 &z = areg[kb][q];
                        z.x = z.x > 0.f ? z.x : a.x * z.x;
                        z.y = z.y > 0.f ? z.y : a.y * z.y;
                        z.z = z.z > 0.f ? z.z : a.z * z.z;
                        z.w = z.w > 0.f ? z.w : a.w * z.w;
                    }
        }
        v16f acc = (v16f){};
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) {
            if (kb >= nkb) break;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                acc = mfma_f32(areg[kb][q].x, breg[kb][q].x, acc);
                acc = mfma_f32(areg[kb][q].y, breg[kb][q].y, acc);
                acc = mfma_f32(areg[kb][q].z, breg[kb][q].z, acc);
                acc = mfma_f32(areg[kb][q].w, breg[kb][q].w, acc);
            }
        }
        __syncthreads();                       // previous chunk's readers of Zp / h2s are done
#pragma unroll
        for (int j = 0; j < 16; ++j) Zp[kh][acc_row(j, lane)][o] = acc[j];
        __syncthreads();
        for (int e = t; e < kTailRows * M; e += kThreads) {
            const int r = e / M, oo = e % M;
            float z = Zp[0][r][oo] + Zp[1][r][oo] + b2s[oo];
            const float zpre = z;                // saved for layer 2's PReLU backward
            if (PR && L == 3) z = z > 0.f ? z : s2[oo] * z;
            else if (relu_a) z = fmaxf(z, 0.f);
            h2s[r][oo] = z;
            if (c0 + r < n_u) {
                if (L == 3) {
                    if (H2_save) H2_save[(size_t)(c0 + r) * M + oo] = PR ? zpre : z;
                } else {
                    E[(size_t)(c0 + r) * M + oo] = z;
                }
            }
        }
        if (L == 3) {
            __syncthreads();
            for (int e = t; e < kTailRows * D; e += kThreads) {
                const int r = e / D, d = e % D;
                if (c0 + r >= n_u) continue;
                float v = b3s[d];
                for (int oo = 0; oo < M; ++oo) v += W3s[d * (kMaxH2 + 1) + oo] * h2s[r][oo];
                if (final_relu) v = fmaxf(v, 0.f);
                E[(size_t)(c0 + r) * D + d] = v;
            }
        }
    }
}

// ---- bf16 forward tail (H = 256) ----
//
// tail_fwd_bf16: the small layers after the bf16 row-split first layer
// (whole rows stored as an H1b / H1lo pair), for 32-row chunks (one chunk per
// wave at a time, no block-level sync in the loop); tail_fwd_bf16_q below
// serves the stream-K layer.  Every product runs on v_mfma_f32_32x32x16_bf16 with its fp32
// activation split into a high and a low bf16 part (x = hi + lo to 2^-18
// relative); the weights are exact in bf16 and each part's products are exact
// in fp32, so the results carry fp32 accumulation of fp32-level operands.
//
// Layer 2: Z2^T = W2 H1^T.  First operand a W2 row (16 bytes of 8
// consecutive k, LDS), second the chunk's H1 row, the (H1b, H1lo) pair the
// first layer stored.  K step s covers k = 16 s .. +15, lane half h supplying
// k = 16 s + 8 h + e.  The accumulator holds Z2[row = lane % 32][o = 32 ob +
// acc_row(j, lane)]: each lane owns one image row and 32 of its outputs.
// H2 = ReLU(Z2 + b2) is stored as float4 runs of 4 outputs.
// Layer 3 (3 layers): Z3^T = W3 H2^T; k step (ob, p) takes the outputs this
// lane already holds, o = 32 ob + 16 p + 4 h + {0..3} and the same + 8, so
// H2 goes into the MFMA straight from the registers; W3 rows sit in LDS padded
// to 68 bf16 (conflict-free 8-byte reads).  E = Z3 + b3 (ReLU if final).
// W2 sits in LDS [64 o][256 k] bf16, rows past the layer width zero, 16-byte
// chunks stored at chunk ^ (o & 15): the rows are 512 bytes (all starting at
// bank 0), so 16 lanes' rows need 16 distinct chunk positions.
constexpr int kW3S = kMaxH2 + 4;               // bf16 per W3 row in LDS

__device__ __forceinline__ uint32_t pack_bf16(float a, float b)
{
    return (uint32_t)ams_f32_to_bf16(a) | ((uint32_t)ams_f32_to_bf16(b) << 16);
}

// The eight fp32 values hi + lo of a pair of bf16x8 operands.
__device__ __forceinline__ void join8(uint4 hi, uint4 lo, float (&x)[8])
{
    const uint32_t h[4] = {hi.x, hi.y, hi.z, hi.w}, l[4] = {lo.x, lo.y, lo.z, lo.w};
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const uint32_t hw = h[e >> 1], lw = l[e >> 1];
        const float a = __uint_as_float((e & 1) ? (hw & 0xffff0000u) : (hw << 16));
        const float b = __uint_as_float((e & 1) ? (lw & 0xffff0000u) : (lw << 16));
        x[e] = a + b;
    }
}

// hi/lo split of 8 fp32 values into two bf16x8 operands
__device__ __forceinline__ void split8(const float (&x)[8], uint4 &hi, uint4 &lo)
{
    uint16_t hb[8];
    float r[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        hb[e] = ams_f32_to_bf16(x[e]);
        r[e] = x[e] - ams_bf16_to_f32(hb[e]);
    }
    hi = make_uint4(hb[0] | ((uint32_t)hb[1] << 16), hb[2] | ((uint32_t)hb[3] << 16),
                    hb[4] | ((uint32_t)hb[5] << 16), hb[6] | ((uint32_t)hb[7] << 16));
    lo = make_uint4(pack_bf16(r[0], r[1]), pack_bf16(r[2], r[3]), pack_bf16(r[4], r[5]), pack_bf16(r[6], r[7]));
}

// PR: PReLU between the layers with per-channel slopes s1 [H] and s2 [M]
// (3 layers).  H1b / H1lo then hold Z1 (split tiles: stored here) and the
// layer-2 operand is the fp32 activation re-split into hi / lo; H2_save holds
// Z2 and the layer-3 operand is its activation.
template <int L, bool PR>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2))) void tail_fwd_bf16(const uint16_t *__restrict__ H1b,
                                                          const uint16_t *__restrict__ H1lo,
                                                          int M, int D, const uint16_t *__restrict__ W2,
                                                          const float *__restrict__ b2,
                                                          const uint16_t *__restrict__ W3,
                                                          const float *__restrict__ b3, int final_relu,
                                                          const int32_t *__restrict__ n_uniq_p, int cap,
                                                          float *__restrict__ H2_save, float *__restrict__ E,
                                                          const float *__restrict__ s1, const float *__restrict__ s2)
{
    constexpr int H = kMaxH1;
    constexpr int KS = H / 16;                 // k steps
    __shared__ __attribute__((aligned(16))) uint16_t W2s[kMaxH2 * kMaxH1];
    __shared__ __attribute__((aligned(16))) uint16_t W3s[32 * kW3S];
    __shared__ __attribute__((aligned(16))) float S1s[PR ? H : 4];      // layer 1's slopes
    __shared__ float S2s[PR ? kMaxH2 : 1];                               // layer 2's slopes (3 layers)
    const int t = threadIdx.x, lane = ams_lane(), wave = t / AMS_WAVE;
    const int h = lane >> 5, r32 = lane & 31;
    const int Mo = (L == 3) ? M : D;           // width of the second layer's output
    // the grid is sized by the capacity: a block with no 32-row chunk below
    // n_u leaves before staging the weights
    const int n_u = min(*n_uniq_p, cap);
    if ((int64_t)blockIdx.x * (kThreads / AMS_WAVE) * 32 >= n_u) return;
    constexpr int cpr = H / 8;                 // 16-byte chunks per W2 row
    // W2 and W3 into LDS with every load of the block in flight together
    static_assert(kMaxH2 * cpr % kThreads == 0, "W2 chunks per thread");
    {
        uint4 v[kMaxH2 * cpr / kThreads];
#pragma unroll
        for (int i = 0; i < kMaxH2 * cpr / kThreads; ++i) {
            const int idx = t + i * kThreads, o = idx / cpr, c = idx % cpr;
            v[i] = o < Mo ? *(const uint4 *)&W2[(size_t)o * H + c * 8] : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int i = 0; i < kMaxH2 * cpr / kThreads; ++i) {
            const int idx = t + i * kThreads, o = idx / cpr, c = idx % cpr;
            *(uint4 *)&W2s[o * H + ((c ^ (o & 15)) << 3)] = v[i];
        }
    }
    if (L == 3) {
        // every load unconditional (an index past W3 reads element 0 and is
        // dropped), so they are all in flight together
        constexpr int n3 = (32 * kW3S + kThreads - 1) / kThreads;
        uint16_t v[n3];
#pragma unroll
        for (int i = 0; i < n3; ++i) {
            const int e = t + i * kThreads, d = e / kW3S, o = e % kW3S;
            const bool ok = e < 32 * kW3S && d < D && o < M;
            const uint16_t x = W3[ok ? d * M + o : 0];
            v[i] = ok ? x : (uint16_t)0;
        }
#pragma unroll
        for (int i = 0; i < n3; ++i) {
            const int e = t + i * kThreads;
            if (e < 32 * kW3S) W3s[e] = v[i];
        }
    }
    if (PR) {
        for (int i = t; i < H; i += kThreads) S1s[i] = s1[i];
        if (L == 3)
            for (int i = t; i < kMaxH2; i += kThreads) S2s[i] = i < M ? s2[i] : 0.f;
    }
    // this lane's outputs o = 32 ob + 8 q + 4 h + r and their biases
    float bias[2][16];
#pragma unroll
    for (int ob = 0; ob < 2; ++ob)
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            const int o = 32 * ob + acc_row(j, lane);
            const float bv = b2[o < Mo ? o : 0];           // unconditional loads, all in flight
            bias[ob][j] = o < Mo ? bv : 0.f;
        }
    __syncthreads();

    const bool relu2 = (L == 3 && !PR) || (L == 2 && final_relu);
    for (int c0 = (blockIdx.x * (kThreads / AMS_WAVE) + wave) * 32; c0 < n_u;
         c0 += gridDim.x * (kThreads / AMS_WAVE) * 32) {
        const int row = c0 + r32;
        const bool live = row < n_u;
        const int rowc = min(row, n_u - 1);
        const size_t roff = (size_t)rowc * H + 8 * h;
        // quarters of 64 k, double-buffered: quarter qt + 1's loads are
        // issued before quarter qt's products (the scheduling barriers keep
        // later quarters' loads from being hoisted, which runs out of
        // registers)
        v16f acc[2] = {(v16f){}, (v16f){}};
        uint4 bh[2][KS / 4], bl[2][KS / 4];
        auto load_q = [&](int qt, uint4 (&hb)[KS / 4], uint4 (&lb)[KS / 4]) {
#pragma unroll
            for (int s4 = 0; s4 < KS / 4; ++s4) {
                hb[s4] = *(const uint4 *)(H1b + roff + 16 * (qt * (KS / 4) + s4));
                lb[s4] = *(const uint4 *)(H1lo + roff + 16 * (qt * (KS / 4) + s4));
            }
        };
        load_q(0, bh[0], bl[0]);
#pragma unroll
        for (int qt = 0; qt < 4; ++qt) {
            __builtin_amdgcn_sched_barrier(0);
            if (qt < 3) load_q(qt + 1, bh[(qt + 1) & 1], bl[(qt + 1) & 1]);
            __builtin_amdgcn_sched_barrier(0);
            uint4 (&ch)[KS / 4] = bh[qt & 1];
            uint4 (&cl)[KS / 4] = bl[qt & 1];
            if (PR) {   // the operand: PReLU(Z1) in fp32, split again
#pragma unroll
                for (int s4 = 0; s4 < KS / 4; ++s4) {
                    const int k0 = 16 * (qt * (KS / 4) + s4) + 8 * h;
                    float x[8];
                    join8(ch[s4], cl[s4], x);
                    const float4 a0 = *(const float4 *)&S1s[k0], a1 = *(const float4 *)&S1s[k0 + 4];
                    const float a[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};
#pragma unroll
                    for (int e = 0; e < 8; ++e) x[e] = x[e] > 0.f ? x[e] : a[e] * x[e];
                    split8(x, ch[s4], cl[s4]);
                }
            }
#pragma unroll
            for (int s4 = 0; s4 < KS / 4; ++s4) {
                const int ss = qt * (KS / 4) + s4;
#pragma unroll
                for (int ob = 0; ob < 2; ++ob) {
                    const int o = 32 * ob + r32;
                    const uint4 av = *(const uint4 *)&W2s[o * H + (((2 * ss + h) ^ (o & 15)) << 3)];
                    acc[ob] = mfma_bf16(av, ch[s4], acc[ob]);
                    acc[ob] = mfma_bf16(av, cl[s4], acc[ob]);
                }
            }
        }
        float z[2][16];
#pragma unroll
        for (int ob = 0; ob < 2; ++ob)
#pragma unroll
            for (int j = 0; j < 16; ++j) {
                const float v = acc[ob][j] + bias[ob][j];
                z[ob][j] = relu2 ? fmaxf(v, 0.f) : v;
            }
        float *out2 = (L == 3) ? H2_save : E;  // where the second layer's output goes
        const int w2 = (L == 3) ? M : D;
        if (live && out2) {
#pragma unroll
            for (int ob = 0; ob < 2; ++ob)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int o = 32 * ob + 8 * q + 4 * h;
                    float *dst = out2 + (size_t)row * w2 + o;
                    if ((w2 & 3) == 0 && o + 3 < w2) {
                        *(float4 *)dst = make_float4(z[ob][4 * q], z[ob][4 * q + 1], z[ob][4 * q + 2], z[ob][4 * q + 3]);
                    } else {
#pragma unroll
                        for (int r = 0; r < 4; ++r)
                            if (o + r < w2) dst[r] = z[ob][4 * q + r];
                    }
                }
        }
        if constexpr (L == 3) {
            v16f a3 = (v16f){};
#pragma unroll
            for (int ob = 0; ob < 2; ++ob)
#pragma unroll
                for (int p = 0; p < 2; ++p) {
                    float x[8];
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        x[e] = z[ob][8 * p + e];           // o = 32 ob + 16 p + 4 h + e
                        x[4 + e] = z[ob][8 * p + 4 + e];   // o = 32 ob + 16 p + 8 + 4 h + e
                    }
                    if (PR) {                              // Z2 -> H2
                        const int ob0 = 32 * ob + 16 * p + 4 * h;
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            x[e] = x[e] > 0.f ? x[e] : S2s[ob0 + e] * x[e];
                            x[4 + e] = x[4 + e] > 0.f ? x[4 + e] : S2s[ob0 + 8 + e] * x[4 + e];
                        }
                    }
                    uint4 hi, lo;
                    split8(x, hi, lo);
                    const uint16_t *wr = &W3s[r32 * kW3S + 32 * ob + 16 * p + 4 * h];
                    const uint2 w0 = *(const uint2 *)wr, w1 = *(const uint2 *)(wr + 8);
                    const uint4 wv = make_uint4(w0.x, w0.y, w1.x, w1.y);
                    a3 = mfma_bf16(wv, hi, a3);
                    a3 = mfma_bf16(wv, lo, a3);
                }
            if (live) {
#pragma unroll
                for (int j = 0; j < 16; ++j) {
                    const int d = acc_row(j, lane);
                    if (d < D) {
                        float v = a3[j] + b3[d];
                        if (final_relu) v = fmaxf(v, 0.f);
                        E[(size_t)row * D + d] = v;
                    }
                }
            }
        }
    }
}

// The rest of a chunk after layer 2's products (acc[ob][j]: row lane % 32,
// output 32 ob + acc_row(j, lane)): Z2 + b2 and its activation, stored to
// H2_save (3 layers; Z2 itself with PReLU) or E (2 layers), then for 3
// layers E = H2 W3^T + b3 on MFMA with W3 rows in LDS (kW3S bf16 apart) and
// H2 split into hi and lo parts straight from the registers.
template <int L, bool PR>
__device__ __forceinline__ void tfb_finish(const v16f (&acc)[2], const float (&bias)[2][16], bool relu2,
                                           const uint16_t *W3s, const float *S2s, const float *__restrict__ b3,
                                           int final_relu, int M, int D, int row, bool live,
                                           float *__restrict__ H2_save, float *__restrict__ E, int lane)
{
    const int h = lane >> 5, r32 = lane & 31;
    float z[2][16];
#pragma unroll
    for (int ob = 0; ob < 2; ++ob)
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            const float v = acc[ob][j] + bias[ob][j];
            z[ob][j] = relu2 ? fmaxf(v, 0.f) : v;
        }
    float *out2 = (L == 3) ? H2_save : E;  // where the second layer's output goes
    const int w2 = (L == 3) ? M : D;
    if (live && out2) {
#pragma unroll
        for (int ob = 0; ob < 2; ++ob)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int o = 32 * ob + 8 * q + 4 * h;
                float *dst = out2 + (size_t)row * w2 + o;
                if ((w2 & 3) == 0 && o + 3 < w2) {
                    *(float4 *)dst = make_float4(z[ob][4 * q], z[ob][4 * q + 1], z[ob][4 * q + 2], z[ob][4 * q + 3]);
                } else {
#pragma unroll
                    for (int r = 0; r < 4; ++r)
                        if (o + r < w2) dst[r] = z[ob][4 * q + r];
                }
            }
    }
    if constexpr (L == 3) {
        v16f a3 = (v16f){};
#pragma unroll
        for (int ob = 0; ob < 2; ++ob)
#pragma unroll
            for (int p = 0; p < 2; ++p) {
                float x[8];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    x[e] = z[ob][8 * p + e];           // o = 32 ob + 16 p + 4 h + e
                    x[4 + e] = z[ob][8 * p + 4 + e];   // o = 32 ob + 16 p + 8 + 4 h + e
                }
                if (PR) {                              // Z2 -> H2
                    const int ob0 = 32 * ob + 16 * p + 4 * h;
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        x[e] = x[e] > 0.f ? x[e] : S2s[ob0 + e] * x[e];
                        x[4 + e] = x[4 + e] > 0.f ? x[4 + e] : S2s[ob0 + 8 + e] * x[4 + e];
                    }
                }
                uint4 hi, lo;
                split8(x, hi, lo);
                const uint16_t *wr = &W3s[r32 * kW3S + 32 * ob + 16 * p + 4 * h];
                const uint2 w0 = *(const uint2 *)wr, w1 = *(const uint2 *)(wr + 8);
                const uint4 wv = make_uint4(w0.x, w0.y, w1.x, w1.y);
                a3 = mfma_bf16(wv, hi, a3);
                a3 = mfma_bf16(wv, lo, a3);
            }
        if (live) {
#pragma unroll
            for (int j = 0; j < 16; ++j) {
                const int d = acc_row(j, lane);
                if (d < D) {
                    float v = a3[j] + b3[d];
                    if (final_relu) v = fmaxf(v, 0.f);
                    E[(size_t)row * D + d] = v;
                }
            }
        }
    }
}

// tail_fwd_bf16_q: the same small layers after the stream-K first layer, for
// the stream-K path's batches (below the row-split size): one block per
// 32-row chunk (blocks loop over chunks), wave q taking layer 2's
// contraction over k = 64 q .. + 63.  A wave's W2 operands come straight
// from global memory (rows o = 32 ob + lane % 32), the chunk's H1 quarter
// from the stream-K pieces (added in K order, b1 and the activation applied,
// H1b stored, as in tail_fwd_bf16) or from the finished rows; every load of
// a wave is issued before the first is used, so a chunk costs one memory
// round trip where one wave walking all four quarters costs four.  The four
// quarters' products (the same MFMA sequence per quarter as tail_fwd_bf16)
// are added in q order through LDS, and wave 0 finishes the chunk.
template <int L, bool PR>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2))) void tail_fwd_bf16_q(
    uint16_t *__restrict__ H1b, const uint16_t *__restrict__ H1lo, const float *__restrict__ pbuf, int F, int G,
    const float *__restrict__ b1, const int32_t *__restrict__ uniq, int64_t n_rows, int M, int D,
    const uint16_t *__restrict__ W2, const float *__restrict__ b2, const uint16_t *__restrict__ W3,
    const float *__restrict__ b3, int final_relu, const int32_t *__restrict__ n_uniq_p, int cap,
    float *__restrict__ H2_save, float *__restrict__ E, const float *__restrict__ s1, const float *__restrict__ s2)
{
    constexpr int H = kMaxH1;
    static_assert(kThreads == 4 * AMS_WAVE, "one wave per K quarter");
    __shared__ __attribute__((aligned(16))) float Zq[4][2][16][AMS_WAVE];   // quarter partials, lane-major
    __shared__ __attribute__((aligned(16))) uint16_t W3s[32 * kW3S];
    __shared__ __attribute__((aligned(16))) float B1s[kMaxH1];
    __shared__ __attribute__((aligned(16))) float S1s[PR ? kMaxH1 : 4];
    __shared__ float S2s[PR ? kMaxH2 : 1];
    const int t = threadIdx.x, lane = ams_lane(), q = t / AMS_WAVE;
    const int h = lane >> 5, r32 = lane & 31;
    const int Mo = (L == 3) ? M : D;
    const int n_u = min(*n_uniq_p, cap);
    if (blockIdx.x * 32 >= n_u) return;
    // this wave's W2 operands (rows past Mo read row 0 and are zeroed), all
    // in flight together, then W3, b1 and the slopes into LDS
    uint4 aw[4][2];
#pragma unroll
    for (int s4 = 0; s4 < 4; ++s4)
#pragma unroll
        for (int ob = 0; ob < 2; ++ob) {
            const int o = 32 * ob + r32;
            aw[s4][ob] = *(const uint4 *)&W2[(size_t)(o < Mo ? o : 0) * H + 64 * q + 16 * s4 + 8 * h];
        }
#pragma unroll
    for (int s4 = 0; s4 < 4; ++s4)
#pragma unroll
        for (int ob = 0; ob < 2; ++ob)
            if (32 * ob + r32 >= Mo) aw[s4][ob] = make_uint4(0, 0, 0, 0);
    if (L == 3)
        for (int e = t; e < 32 * kW3S; e += kThreads) {
            const int d = e / kW3S, o = e % kW3S;
            W3s[e] = (d < D && o < M) ? W3[d * M + o] : (uint16_t)0;
        }
    for (int i = t; i < H; i += kThreads) B1s[i] = b1[i];
    if (PR) {
        for (int i = t; i < H; i += kThreads) S1s[i] = s1[i];
        if (L == 3)
            for (int i = t; i < kMaxH2; i += kThreads) S2s[i] = i < M ? s2[i] : 0.f;
    }
    // wave 0's layer-2 biases (output 32 ob + acc_row(j, lane))
    float bias[2][16];
#pragma unroll
    for (int ob = 0; ob < 2; ++ob)
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            const int o = 32 * ob + acc_row(j, lane);
            const float bv = b2[o < Mo ? o : 0];
            bias[ob][j] = o < Mo ? bv : 0.f;
        }
    __syncthreads();

    const bool relu2 = (L == 3 && !PR) || (L == 2 && final_relu);
    using K = Sk<uint16_t>;
    const SkPlan P = sk_plan(n_u, H, F, G, sk_bk<uint16_t>(), K::BM);
    for (int c0 = blockIdx.x * 32; c0 < n_u; c0 += gridDim.x * 32) {
        const int row = c0 + r32;
        const bool live = row < n_u;
        const int rowc = min(row, n_u - 1);
        const int tile = c0 / K::BM;
        const int wa = P.owner((int64_t)tile * P.S), wb = P.owner((int64_t)(tile + 1) * P.S - 1);
        const bool split = wb > wa;
        const int slot_a = (tile == (int)(P.it0(wa) / P.S)) ? 0 : 1;   // first contributor's piece
        uint4 bh[4], bl[4];
        if (split) {
            const int id = uniq[rowc];
            const bool id_ok = id >= 0 && (int64_t)id < n_rows;
            const int rl = rowc % K::BM;
            const bool has1 = wa + 1 <= wb, has2 = wa + 2 <= wb;
            const float *pw0 = pbuf + ((size_t)wa * 2 + slot_a) * K::TILE + rl * kSkBN;
            const float *pw1 = has1 ? pbuf + ((size_t)(wa + 1) * 2) * K::TILE + rl * kSkBN : pw0;
            const float *pw2 = has2 ? pbuf + ((size_t)(wa + 2) * 2) * K::TILE + rl * kSkBN : pw0;
            float4 pv[3][4][2];
#pragma unroll
            for (int s4 = 0; s4 < 4; ++s4) {
                const int k0 = 64 * q + 16 * s4 + 8 * h;
                pv[0][s4][0] = *(const float4 *)(pw0 + k0);
                pv[0][s4][1] = *(const float4 *)(pw0 + k0 + 4);
                pv[1][s4][0] = *(const float4 *)(pw1 + k0);
                pv[1][s4][1] = *(const float4 *)(pw1 + k0 + 4);
                pv[2][s4][0] = *(const float4 *)(pw2 + k0);
                pv[2][s4][1] = *(const float4 *)(pw2 + k0 + 4);
            }
#pragma unroll
            for (int s4 = 0; s4 < 4; ++s4) {
                const int k0 = 64 * q + 16 * s4 + 8 * h;
                float x[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int pi = 0; pi < 3; ++pi) {
                    if (pi == 0 || (pi == 1 ? has1 : has2)) {
                        const float4 v0 = pv[pi][s4][0], v1 = pv[pi][s4][1];
                        x[0] += v0.x; x[1] += v0.y; x[2] += v0.z; x[3] += v0.w;
                        x[4] += v1.x; x[5] += v1.y; x[6] += v1.z; x[7] += v1.w;
                    }
                }
                for (int w = wa + 3; w <= wb; ++w) {     // (a tile spans at most 3 shares)
                    const float *pc = pbuf + ((size_t)w * 2) * K::TILE + rl * kSkBN + k0;
                    const float4 v0 = *(const float4 *)pc, v1 = *(const float4 *)(pc + 4);
                    x[0] += v0.x; x[1] += v0.y; x[2] += v0.z; x[3] += v0.w;
                    x[4] += v1.x; x[5] += v1.y; x[6] += v1.z; x[7] += v1.w;
                }
                const float4 c0v = *(const float4 *)&B1s[k0], c1v = *(const float4 *)&B1s[k0 + 4];
                const float bb[8] = {c0v.x, c0v.y, c0v.z, c0v.w, c1v.x, c1v.y, c1v.z, c1v.w};
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    x[e] = id_ok ? x[e] + bb[e] : bb[e];
                    if (!PR) x[e] = fmaxf(x[e], 0.f);
                }
                split8(x, bh[s4], bl[s4]);
                if (live) *(uint4 *)(H1b + (size_t)row * H + k0) = bh[s4];
            }
        } else {
            const size_t roff = (size_t)rowc * H + 64 * q + 8 * h;
#pragma unroll
            for (int s4 = 0; s4 < 4; ++s4) {
                bh[s4] = *(const uint4 *)(H1b + roff + 16 * s4);
                bl[s4] = *(const uint4 *)(H1lo + roff + 16 * s4);
            }
        }
        if (PR) {   // the operand: PReLU(Z1) in fp32, split again
#pragma unroll
            for (int s4 = 0; s4 < 4; ++s4) {
                const int k0 = 64 * q + 16 * s4 + 8 * h;
                float x[8];
                join8(bh[s4], bl[s4], x);
                const float4 a0 = *(const float4 *)&S1s[k0], a1 = *(const float4 *)&S1s[k0 + 4];
                const float a[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};
#pragma unroll
                for (int e = 0; e < 8; ++e) x[e] = x[e] > 0.f ? x[e] : a[e] * x[e];
                split8(x, bh[s4], bl[s4]);
            }
        }
        v16f acc[2] = {(v16f){}, (v16f){}};
#pragma unroll
        for (int s4 = 0; s4 < 4; ++s4)
#pragma unroll
            for (int ob = 0; ob < 2; ++ob) {
                acc[ob] = mfma_bf16(aw[s4][ob], bh[s4], acc[ob]);
                acc[ob] = mfma_bf16(aw[s4][ob], bl[s4], acc[ob]);
            }
#pragma unroll
        for (int ob = 0; ob < 2; ++ob)
#pragma unroll
            for (int j = 0; j < 16; ++j) Zq[q][ob][j][lane] = acc[ob][j];
        __syncthreads();
        if (q == 0) {
            v16f z[2];
#pragma unroll
            for (int ob = 0; ob < 2; ++ob)
#pragma unroll
                for (int j = 0; j < 16; ++j)
                    z[ob][j] = ((Zq[0][ob][j][lane] + Zq[1][ob][j][lane]) + Zq[2][ob][j][lane]) + Zq[3][ob][j][lane];
            tfb_finish<L, PR>(z, bias, relu2, W3s, S2s, b3, final_relu, M, D, row, live, H2_save, E, lane);
        }
        __syncthreads();                        // Zq is free for the next chunk
    }
}

// Backward of the small layers, entirely in registers.  Block g owns unique
// images [g n_u / G, (g+1) n_u / G), walked in chunks of 32 rows; wave w of
// the 4 owns H1 columns [64 w, 64 w + 64).  Per chunk, with dzl = dE (masked
// by the last ReLU if any):
//   dZ2 = (dzl W3) * [H2 > 0] on MFMA (for 2 layers dZ2 = dzl), computed in
//       two layouts by swapping the MFMA operands: lanes <-> rows (operand of
//       dH1) and lanes <-> outputs o (operand of dW2);
//   dH1 = dZ2 W2 on MFMA, dZ1 = dH1 * [H1 > 0], written out for dW1;
//   dW2 += dZ2^T H1, dW3 += dzl^T H2 (waves 0, 1) on MFMA; db* by lane sums.
// The 32 k of each MFMA sum are assigned to (lane half, step) so that the k
// of step j in half h is the accumulator row acc_row(j, lane): an
// accumulator then serves as an operand of the next product unchanged, and
// the H1 values that mask dZ1 are the same registers that feed dW2.
// Partials per block: [dW2: Mo x H][db2: Mo][dW3: D x M][db3: D][db1: H].
// One wave per SIMD (4 waves x 64 columns), so that a whole chunk's loads fit
// in registers and are in flight together.
constexpr int kTbThreads = 256;
constexpr int kTbCols = kMaxH1 / (kTbThreads / AMS_WAVE);   // 64 columns per wave

template <typename T>
__device__ __forceinline__ float ldf(const T *p, size_t i)
{
    if constexpr (sizeof(T) == 2) return ams_bf16_to_f32(p[i]);
    else return p[i];
}

template <typename T>
__device__ __forceinline__ void stf(T *p, size_t i, float v)
{
    if constexpr (sizeof(T) == 2) p[i] = ams_f32_to_bf16(v);
    else p[i] = v;
}

// Buffer loads: a resource descriptor carries the byte size of the valid
// range, and the hardware returns 0 for an offset past it, so the loads of a
// chunk need no row bounds checks or branches (gfx9 descriptor word 3).
typedef __amdgpu_buffer_rsrc_t brsrc_t;

__device__ __forceinline__ brsrc_t make_buf(const void *p, uint32_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), 0, bytes, 0x00020000);
}

template <typename T>
__device__ __forceinline__ float buf_ld(brsrc_t r, uint32_t elem)
{
    if constexpr (sizeof(T) == 2)
        return ams_bf16_to_f32(__builtin_amdgcn_raw_buffer_load_b16(r, elem * 2, 0, 0));
    else
        return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, elem * 4, 0, 0));
}

typedef unsigned int v2u32 __attribute__((ext_vector_type(2)));
typedef unsigned int v4u32 __attribute__((ext_vector_type(4)));

// Four consecutive elements from elem (a multiple of 4): one 16-byte (fp32)
// or 8-byte (bf16) buffer load, 0 past the descriptor's size.
template <typename T>
__device__ __forceinline__ float4 buf_ld4(brsrc_t r, uint32_t elem)
{
    if constexpr (sizeof(T) == 2) {
        const v2u32 v = __builtin_amdgcn_raw_buffer_load_b64(r, elem * 2, 0, 0);
        return make_float4(__uint_as_float(v[0] << 16), __uint_as_float(v[0] & 0xffff0000u),
                           __uint_as_float(v[1] << 16), __uint_as_float(v[1] & 0xffff0000u));
    } else {
        const v4u32 v = __builtin_amdgcn_raw_buffer_load_b128(r, elem * 4, 0, 0);
        return make_float4(__uint_as_float(v[0]), __uint_as_float(v[1]), __uint_as_float(v[2]),
                           __uint_as_float(v[3]));
    }
}

// Buffer store: dropped by the hardware past the descriptor's size.
template <typename T>
__device__ __forceinline__ void buf_st(brsrc_t r, uint32_t elem, float v)
{
    if constexpr (sizeof(T) == 2)
        __builtin_amdgcn_raw_buffer_store_b16(ams_f32_to_bf16(v), r, elem * 2, 0, 0);
    else
        __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), r, elem * 4, 0, 0);
}

// Upstream gradient of the last layer at (chunk row rr, d), masked by its
// ReLU; 0 for d >= D and (by the descriptor) for rows past the chunk.
// (rE has size 0 when there is no final ReLU: its loads read 0 and are not
// used.)
__device__ __forceinline__ float tb_dzl(brsrc_t rdE, brsrc_t rE, int final_relu, int rr, int d, int D)
{
    const uint32_t x = (uint32_t)(rr * D + d);   // d >= D reads a neighbour (or 0) and is masked
    const float g = buf_ld<float>(rdE, x), e = buf_ld<float>(rE, x);
    return (d < D && (!final_relu || e > 0.f)) ? g : 0.f;
}

template <int L, int SD, typename TW, typename TH, bool PR>
__global__ __launch_bounds__(kTbThreads) void tail_bwd(const TH *__restrict__ H1s,
                                                        const float *__restrict__ H2s,
                                                        const float *__restrict__ Efwd,
                                                        const float *__restrict__ dE,
                                                        const TW *__restrict__ W2,
                                                        const TW *__restrict__ W3, int H, int M, int D,
                                                        int final_relu, const int32_t *__restrict__ n_uniq_p,
                                                        int cap, TH *__restrict__ dZ1, float *__restrict__ part,
                                                        int PS, float *__restrict__ zero_row, int zero_n,
                                                        const float *__restrict__ s1, const float *__restrict__ s2)
{
    const int n_u = min(*n_uniq_p, cap);
    const int n_act = tail_active(n_u, (int)gridDim.x);
    if ((int)blockIdx.x >= n_act) return;          // (block 0 is always active)
    // the zero row that dW1's padding rows stream (read by the next launch)
    if (blockIdx.x == 0)
        for (int i = threadIdx.x; i < zero_n; i += kTbThreads) zero_row[i] = 0.f;
    const int lane = ams_lane(), wave = threadIdx.x / AMS_WAVE;
    const int h = lane >> 5, r32 = lane & 31;
    const int Mo = (L == 3) ? M : D;
    const int i0 = kTbCols * wave;            // this wave's H1 columns: icol(ib) = i0 + 32 ib + r32

    // W2 (fp32, zero-padded to 64 x 256) and W3 (2 SD x 64) in LDS: operands of
    // dH1 and dZ2, re-read per chunk (registers hold the chunk's data)
    __shared__ __attribute__((aligned(16))) float W2s[kMaxH2 * kMaxH1];
    __shared__ float W3s[2 * SD * kMaxH2];
    __shared__ float S2s[PR ? kMaxH2 : 1];     // layer 2's PReLU slopes (3 layers)
    if (PR && L == 3)
        for (int o = threadIdx.x; o < kMaxH2; o += kTbThreads) S2s[o] = o < M ? s2[o] : 0.f;
    {
        // four consecutive i per load (H is a multiple of 64), all 16 loads
        // of a thread in flight together
        const brsrc_t rW2 = make_buf(W2, (uint32_t)(Mo * H * sizeof(TW)));   // rows o >= Mo read 0
        constexpr int N4 = kMaxH2 * kMaxH1 / 4 / kTbThreads;
        float4 v[N4];
#pragma unroll
        for (int k = 0; k < N4; ++k) {
            const int e = 4 * ((int)threadIdx.x + k * kTbThreads), o = e / kMaxH1, i = e % kMaxH1;
            v[k] = buf_ld4<TW>(rW2, (uint32_t)(o * H + min(i, H - 4)));
        }
#pragma unroll
        for (int k = 0; k < N4; ++k) {
            const int e = 4 * ((int)threadIdx.x + k * kTbThreads), i = e % kMaxH1;
            *(float4 *)&W2s[e] = i < H ? v[k] : make_float4(0.f, 0.f, 0.f, 0.f);
        }
        const brsrc_t rW3 = make_buf(L == 3 ? W3 : W2, L == 3 ? (uint32_t)(D * M * sizeof(TW)) : 0u);
        static_assert(2 * SD * kMaxH2 % kTbThreads == 0, "W3 entries per thread");
#pragma unroll
        for (int i = 0; i < 2 * SD * kMaxH2 / kTbThreads; ++i) {
            const int e = threadIdx.x + i * kTbThreads, d = e / kMaxH2, o = e % kMaxH2;
            const float x = buf_ld<TW>(rW3, (uint32_t)(d * M + min(o, M - 1)));
            W3s[e] = o < M ? x : 0.f;
        }
    }
    __syncthreads();

    const int r0 = (int)((int64_t)blockIdx.x * n_u / n_act);
    const int r1 = (int)((int64_t)(blockIdx.x + 1) * n_u / n_act);

    v16f dw2[2][2] = {{(v16f){}, (v16f){}}, {(v16f){}, (v16f){}}};   // [o block][i block]
    v16f dw3 = (v16f){};                     // wave ob < 2: lanes <-> o, rows d
    float db1a[2] = {0.f, 0.f}, db2a[2] = {0.f, 0.f}, db3a = 0.f;
    // PReLU: slope gradients (sum of dH * min(Z, 0)) like db1 / db2, and this
    // lane's two layer-1 slopes (columns i0 + 32 ib + r32)
    float ds1a[2] = {0.f, 0.f}, ds2a[2] = {0.f, 0.f};
    float sl1[2] = {0.f, 0.f};
    if (PR)
#pragma unroll
        for (int ib = 0; ib < 2; ++ib) sl1[ib] = (i0 + 32 * ib + r32 < H) ? s1[i0 + 32 * ib + r32] : 0.f;
    const bool w3_wave = (L == 3) && wave < 2 && 32 * wave < M;

    for (int c0 = r0; c0 < r1; c0 += 32) {
        // descriptors over the chunk's rows [c0, min(c0 + 32, r1))
        const uint32_t nr = (uint32_t)min(32, r1 - c0);
        const brsrc_t rdE = make_buf(dE + (size_t)c0 * D, nr * D * 4);
        const brsrc_t rE = make_buf(final_relu ? Efwd + (size_t)c0 * D : dE, final_relu ? nr * D * 4 : 0);
        const brsrc_t rH2 = make_buf(L == 3 ? H2s + (size_t)c0 * M : dE, L == 3 ? nr * M * 4 : 0);
        const brsrc_t rH1 = make_buf(H1s + (size_t)c0 * H, nr * H * (uint32_t)sizeof(TH));
        const brsrc_t rZ1 = make_buf(dZ1 + (size_t)c0 * H, nr * H * (uint32_t)sizeof(TH));
        // phase 2's operands loaded with phase 1's (one memory round trip per
        // chunk; one wave per SIMD leaves the registers for it)
        float dA3[16];                          // dzl[row][d = r32] (dW3's operand, db3)
#pragma unroll
        for (int jj = 0; jj < 16; ++jj) dA3[jj] = tb_dzl(rdE, rE, final_relu, acc_row(jj, lane), r32, D);
        float h2Av[2][16];                      // H2 (or dzl) [row][o = r32 + 32 ob]
#pragma unroll
        for (int ob = 0; ob < 2; ++ob)
#pragma unroll
            for (int jj = 0; jj < 16; ++jj) {
                const int rr = acc_row(jj, lane), o = r32 + 32 * ob;
                if (L == 3) {
                    const float x = buf_ld<float>(rH2, (uint32_t)(rr * M + o));
                    h2Av[ob][jj] = o < M ? x : 0.f;
                } else {
                    h2Av[ob][jj] = tb_dzl(rdE, rE, final_relu, rr, o, D);
                }
            }
        // ==== phase 1: dZ2 with lanes <-> rows, dH1, dZ1 (one o block at a time)
        float dzB[SD];                         // dzl[r32][2 s + h]
#pragma unroll
        for (int st = 0; st < SD; ++st) dzB[st] = tb_dzl(rdE, rE, final_relu, r32, 2 * st + h, D);
        float h1v[2][16];                       // (columns past H read other data; never stored)
#pragma unroll
        for (int ib = 0; ib < 2; ++ib)
#pragma unroll
            for (int jj = 0; jj < 16; ++jj)
                h1v[ib][jj] = buf_ld<TH>(rH1, (uint32_t)(acc_row(jj, lane) * H + i0 + 32 * ib + r32));
        v16f a1[2] = {(v16f){}, (v16f){}};
#pragma unroll
        for (int ob = 0; ob < 2; ++ob) {
            float dz2B[16];
            if constexpr (L == 3) {
                float h2B[16];
#pragma unroll
                for (int jj = 0; jj < 16; ++jj) {
                    const int o = acc_row(jj, lane) + 32 * ob;
                    const float x = buf_ld<float>(rH2, (uint32_t)(r32 * M + o));
                    h2B[jj] = o < M ? x : 0.f;
                }
                v16f aB = (v16f){};
#pragma unroll
                for (int st = 0; st < SD; ++st)   // [o][row]: lanes <-> rows (zeros past D)
                    aB = mfma_f32(W3s[(2 * st + h) * kMaxH2 + r32 + 32 * ob], dzB[st], aB);
#pragma unroll
                for (int jj = 0; jj < 16; ++jj) {
                    if (PR) dz2B[jj] = h2B[jj] > 0.f ? aB[jj] : S2s[acc_row(jj, lane) + 32 * ob] * aB[jj];
                    else dz2B[jj] = h2B[jj] > 0.f ? aB[jj] : 0.f;
                }
            } else {   // 2 layers: dZ2 = dzl itself
#pragma unroll
                for (int jj = 0; jj < 16; ++jj)
                    dz2B[jj] = tb_dzl(rdE, rE, final_relu, r32, acc_row(jj, lane) + 32 * ob, D);
            }
#pragma unroll
            for (int ib = 0; ib < 2; ++ib) {
                float w2v[16];
#pragma unroll
                for (int jj = 0; jj < 16; ++jj)
                    w2v[jj] = W2s[(acc_row(jj, lane) + 32 * ob) * kMaxH1 + ((i0 + 32 * ib + r32) & (kMaxH1 - 1))];
#pragma unroll
                for (int jj = 0; jj < 16; ++jj) a1[ib] = mfma_f32(dz2B[jj], w2v[jj], a1[ib]);
            }
        }
#pragma unroll
        for (int ib = 0; ib < 2; ++ib) {
            // dZ1 = dH1 * [H1 > 0], written out (stores past the chunk are
            // dropped by the descriptor; columns past H are not stored); db1
            const int icol = i0 + 32 * ib + r32;
            float cs = 0.f, css = 0.f;
#pragma unroll
            for (int jj = 0; jj < 16; ++jj) {
                const bool pos = h1v[ib][jj] > 0.f;
                const float dz = pos ? a1[ib][jj] : (PR ? sl1[ib] * a1[ib][jj] : 0.f);
                cs += dz;
                if (PR) css += pos ? 0.f : a1[ib][jj] * h1v[ib][jj];
                if (icol < H) buf_st<TH>(rZ1, (uint32_t)(acc_row(jj, lane) * H + icol), dz);
            }
            db1a[ib] += cs + __shfl_xor(cs, 32, AMS_WAVE);
            if (PR) {
                ds1a[ib] += css + __shfl_xor(css, 32, AMS_WAVE);
                // from here on the H1 operand of dW2 is the activation
#pragma unroll
                for (int jj = 0; jj < 16; ++jj)
                    if (!(h1v[ib][jj] > 0.f)) h1v[ib][jj] *= sl1[ib];
            }
        }
        __builtin_amdgcn_sched_barrier(0);

        // ==== phase 2: dZ2 with lanes <-> o; dW2, db2, dW3, db3 (one o block at a time)
        {
            float c3 = 0.f;
#pragma unroll
            for (int jj = 0; jj < 16; ++jj) c3 += dA3[jj];
            db3a += c3 + __shfl_xor(c3, 32, AMS_WAVE);
        }
#pragma unroll
        for (int ob = 0; ob < 2; ++ob) {
            float h2A[16], dz2A[16];
#pragma unroll
            for (int jj = 0; jj < 16; ++jj) h2A[jj] = h2Av[ob][jj];
            if constexpr (L == 3) {
                v16f aA = (v16f){};
#pragma unroll
                for (int st = 0; st < SD; ++st)   // [row][o]: lanes <-> o (zeros past D)
                    aA = mfma_f32(dzB[st], W3s[(2 * st + h) * kMaxH2 + r32 + 32 * ob], aA);
                if (PR) {
                    const float a2 = S2s[r32 + 32 * ob];
                    float css = 0.f;
#pragma unroll
                    for (int jj = 0; jj < 16; ++jj) {
                        const bool pos = h2A[jj] > 0.f;
                        dz2A[jj] = pos ? aA[jj] : a2 * aA[jj];
                        css += pos ? 0.f : aA[jj] * h2A[jj];
                        if (!pos) h2A[jj] *= a2;        // H2 = PReLU(Z2): dW3's operand
                    }
                    ds2a[ob] += css + __shfl_xor(css, 32, AMS_WAVE);
                } else {
#pragma unroll
                    for (int jj = 0; jj < 16; ++jj) dz2A[jj] = h2A[jj] > 0.f ? aA[jj] : 0.f;
                }
            } else {
#pragma unroll
                for (int jj = 0; jj < 16; ++jj) dz2A[jj] = h2A[jj];
            }
#pragma unroll
            for (int ib = 0; ib < 2; ++ib)   // dW2 += dZ2^T H1
#pragma unroll
                for (int jj = 0; jj < 16; ++jj) dw2[ob][ib] = mfma_f32(dz2A[jj], h1v[ib][jj], dw2[ob][ib]);
            float cs = 0.f;
#pragma unroll
            for (int jj = 0; jj < 16; ++jj) cs += dz2A[jj];
            db2a[ob] += cs + __shfl_xor(cs, 32, AMS_WAVE);
            if (w3_wave && wave == ob) {   // dW3 += dzl^T H2 over this o block
#pragma unroll
                for (int jj = 0; jj < 16; ++jj) dw3 = mfma_f32(dA3[jj], h2A[jj], dw3);
            }
        }
    }

    float *p = part + (size_t)blockIdx.x * PS;
#pragma unroll
    for (int ob = 0; ob < 2; ++ob)
#pragma unroll
        for (int ib = 0; ib < 2; ++ib) {
            const int icol = i0 + 32 * ib + r32;
#pragma unroll
            for (int jj = 0; jj < 16; ++jj) {
                const int o = acc_row(jj, lane) + 32 * ob;
                if (o < Mo && icol < H) p[(size_t)o * H + icol] = dw2[ob][ib][jj];
            }
        }
    p += Mo * H;
    if (wave == 0 && h == 0) {
        if (r32 < Mo) p[r32] = db2a[0];
        if (32 + r32 < Mo) p[32 + r32] = db2a[1];
    }
    p += Mo;
    if (L == 3) {
        if (w3_wave) {
            const int o = 32 * wave + r32;
#pragma unroll
            for (int jj = 0; jj < 16; ++jj) {
                const int d = acc_row(jj, lane);
                if (d < D && o < M) p[d * M + o] = dw3[jj];
            }
        }
        p += D * M;
        if (wave == 0 && h == 0 && r32 < D) p[r32] = db3a;
        p += D;
    }
    if (h == 0) {
        if (i0 + r32 < H) p[i0 + r32] = db1a[0];
        if (i0 + 32 + r32 < H) p[i0 + 32 + r32] = db1a[1];
    }
    if (PR) {
        p += H;
        if (h == 0) {
            if (i0 + r32 < H) p[i0 + r32] = ds1a[0];
            if (i0 + 32 + r32 < H) p[i0 + 32 + r32] = ds1a[1];
        }
        p += H;
        if (L == 3 && wave == 0 && h == 0) {
            if (r32 < M) p[r32] = ds2a[0];
            if (32 + r32 < M) p[32 + r32] = ds2a[1];
        }
    }
}

// Sum of the tail backward's block partials, written straight into dW2, db2,
// dW3, db3, db1 and (PReLU) the slope gradients.  Thread (e, q) of a block
// (64 elements x kRedQ groups) sums partials g = q, q + kRedQ, ... in eight
// running chains (independent loads in flight); the chains, then the groups,
// are added in a fixed order, so the result is deterministic.
constexpr int kRedQ = 16;
constexpr int kRedThreads = 64 * kRedQ;
__device__ __forceinline__ void tail_reduce_block(int blk, const float *__restrict__ part, int G_grid, int PS, int L,
                                                  int H, int M, int D, float *__restrict__ dW2,
                                                  float *__restrict__ db2, float *__restrict__ dW3,
                                                  float *__restrict__ db3, float *__restrict__ db1,
                                                  float *__restrict__ ds1, float *__restrict__ ds2,
                                                  const int32_t *__restrict__ n_uniq_p, int cap)
{
    // the slots the tail backward's active blocks wrote
    const int G = tail_active(min(*n_uniq_p, cap), G_grid);
    __shared__ float sq[kRedQ][64];
    const int t = threadIdx.x, q = t >> 6;
    const int e = blk * 64 + (t & 63);
    float c[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    if (e < PS) {
        int k = 0;
        for (; q + kRedQ * (k + 7) < G; k += 8)
#pragma unroll
            for (int r = 0; r < 8; ++r) c[r] += part[(size_t)(q + kRedQ * (k + r)) * PS + e];
        for (int r = 0; r < 8 && q + kRedQ * (k + r) < G; ++r) c[r] += part[(size_t)(q + kRedQ * (k + r)) * PS + e];
    }
    float tot = 0.f;
#pragma unroll
    for (int r = 0; r < 8; ++r) tot += c[r];
    sq[q][t & 63] = tot;
    __syncthreads();
    if (q != 0 || e >= PS) return;
    float v = sq[0][t];
#pragma unroll
    for (int j = 1; j < kRedQ; ++j) v += sq[j][t];
    const int Mo = (L == 3) ? M : D;
    const int n2 = Mo * H, n3 = (L == 3) ? D * M : 0, nb3 = (L == 3) ? D : 0;
    int x = e;
    if (x < n2) { dW2[x] = v; return; }
    x -= n2;
    if (x < Mo) { db2[x] = v; return; }
    x -= Mo;
    if (x < n3) { dW3[x] = v; return; }
    x -= n3;
    if (x < nb3) { db3[x] = v; return; }
    x -= nb3;
    if (x < H) { db1[x] = v; return; }
    x -= H;                                     // PReLU slope gradients (slots unused with ReLU)
    if (x < H) { if (ds1) ds1[x] = v; return; }
    x -= H;
    if (L == 3 && x < M && ds2) ds2[x] = v;
}

// out[e] = sum of part[g * PS + e] over g = 0..G-1, in a fixed association:
// eight running sums over g = 8i + r, added r = 0..7 at the end (the eight
// independent load chains keep the reads in flight).
__device__ __forceinline__ void partial_reduce_elem(size_t e, const float *__restrict__ part, int G, size_t PS,
                                                    float *__restrict__ out)
{
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
    out[e] = tot;
}

// The backward's two fixed-order sums in one launch (they read what the tail
// backward and the dW1 product wrote, both earlier on the stream): blocks
// [0, n_dw) add the dW1 partials, kRedThreads elements each; the blocks after
// them add the tail's block partials into dW2, db2, dW3, db3, db1 and the
// slope gradients, 64 elements each.  Every sum keeps its association.
__global__ __launch_bounds__(kRedThreads) void bwd_reduce(const float *__restrict__ dw1p, int kc, size_t nw,
                                                         float *__restrict__ dW1, int n_dw,
                                                         const float *__restrict__ tail, int G_grid, int PS, int L,
                                                         int H, int M, int D, float *__restrict__ dW2,
                                                         float *__restrict__ db2, float *__restrict__ dW3,
                                                         float *__restrict__ db3, float *__restrict__ db1,
                                                         float *__restrict__ ds1, float *__restrict__ ds2,
                                                         const int32_t *__restrict__ n_uniq_p, int cap)
{
    if ((int)blockIdx.x < n_dw)
        partial_reduce_elem((size_t)blockIdx.x * kRedThreads + threadIdx.x, dw1p, kc, nw, dW1);
    else
        tail_reduce_block((int)blockIdx.x - n_dw, tail, G_grid, PS, L, H, M, D, dW2, db2, dW3, db3, db1, ds1, ds2,
                          n_uniq_p, cap);
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

// fp32 dW1 partial of chunk c with the same 3-slot DMA ring as the forward.
// Block tile 128 (m, dZ1 columns) x 128 (n, feature columns), K step 32
// unique images, 8 waves in 2 (m) x 4 (n), each 64 x 32.  Per stage the A
// tile is 32 rows x 512 B of dZ1 and the B tile 32 rows x 512 B of gathered
// feature rows, 16 DMA instructions of 2 rows each; every wave issues 2 A and
// 2 B instructions.  The 16-byte chunk index of odd rows is XOR-ed with 8 (a
// 128-byte shift) so that lanes 0-31 (row k) and 32-63 (row k+1) of one
// 4-byte operand read fall in different banks.  Rows past the chunk and rows
// with an out-of-range ID read the zero row.  One block per CU: the host
// picks the chunk count so that tiles x chunks = CUs.
//
// The image IDs that address the B rows are loaded two stages ahead, before
// the DMA of the stage that is issued with them, so at the top of stage s
// "wait until at most 6 vector-memory ops are outstanding" leaves exactly the
// IDs of stage s+3 and the DMA of stage s+1 in flight.
struct DwRing {
    static constexpr int BM = 256, BN = 128, BK = 32, WAVES = 8;   // BM = H: a block owns all of dW1's rows
    static constexpr int A_FLOATS = BK * BM, B_FLOATS = BK * BN;
    static constexpr int SLOT = A_FLOATS + B_FLOATS;              // 48 KB
    static constexpr int PA = 4, PB = 2;                 // A / B DMA instructions per wave
    static constexpr int OUTSTANDING = PA + PB + PB;     // vm ops allowed in flight at a stage top
};
constexpr int kDwThreads = DwRing::WAVES * AMS_WAVE;

__device__ __forceinline__ int dw_chunk_swz(int row) { return (row & 1) << 3; }

// IDs of this lane's two B rows of the stage starting at image u_base.
__device__ __forceinline__ void dw1_load_ids(const int32_t *__restrict__ uniq, int u_base, int u1, int wave,
                                             int lane, int (&id)[2])
{
#pragma unroll
    for (int q = 0; q < DwRing::PB; ++q) {
        const int row = 2 * (DwRing::PB * wave + q) + (lane >> 5);
        const int u = u_base + row;
        const int v = uniq[min(u, u1 - 1)];          // always issued: uniform op count
        id[q] = u < u1 ? v : -1;
    }
}

__device__ __forceinline__ void dw1_issue(float *slot, const float *__restrict__ T, int64_t n_rows, int F,
                                          const float *__restrict__ dZ1, int H, int m0, int n0, int u_base,
                                          int u1, const float *__restrict__ zero_row, const int (&id)[2],
                                          int wave, int lane)
{
    const int c = lane & 31;
    // A: one 1-KB dZ1 row per instruction, lane = 16-byte chunk
#pragma unroll
    for (int q = 0; q < DwRing::PA; ++q) {
        const int row = DwRing::PA * wave + q;
        const int u = u_base + row;
        dma16((u < u1 ? dZ1 + (size_t)u * H + m0 : zero_row) + 4 * (lane ^ dw_chunk_swz(row)), slot + row * 256);
    }
#pragma unroll
    for (int q = 0; q < DwRing::PB; ++q) {
        const int j = DwRing::PB * wave + q;
        const int row = 2 * j + (lane >> 5);
        const bool ok = id[q] >= 0 && (int64_t)id[q] < n_rows;
        dma16((ok ? T + (size_t)id[q] * F + n0 : zero_row) + 4 * (c ^ dw_chunk_swz(row)),
              slot + DwRing::A_FLOATS + j * 256);
    }
}

// 16 MFMA steps of 2 k per stage; step kk needs two B and two A values per
// lane (waves are 4 (h) x 2 (f), 64 x 64 each).  Reads run two steps ahead of the MFMAs (sched_group_barrier fixes
// the interleave), so the 4-byte LDS reads are never waited on.
__device__ __forceinline__ void dw1_compute(const float *slot, v16f *acc, int lane, int wave)
{
    const int h = lane >> 5, r32 = lane & 31, wm = wave >> 1, wn = wave & 1;
    const float *A = slot, *B = slot + DwRing::A_FLOATS;
    float av[DwRing::BK / 2][2], bv[DwRing::BK / 2][2];
#pragma unroll
    for (int kk = 0; kk < DwRing::BK / 2; ++kk) {
        const int k = 2 * kk + h;
        const int sw = dw_chunk_swz(k) << 2;
#pragma unroll
        for (int nb = 0; nb < 2; ++nb) bv[kk][nb] = B[k * DwRing::BN + ((wn * 64 + nb * 32 + r32) ^ sw)];
#pragma unroll
        for (int mb = 0; mb < 2; ++mb) av[kk][mb] = A[k * DwRing::BM + ((wm * 64 + mb * 32 + r32) ^ sw)];
    }
#pragma unroll
    for (int kk = 0; kk < DwRing::BK / 2; ++kk)
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
            for (int nb = 0; nb < 2; ++nb) acc[mb * 2 + nb] = mfma_f32(av[kk][mb], bv[kk][nb], acc[mb * 2 + nb]);
    __builtin_amdgcn_sched_group_barrier(0x100, 8, 0);
#pragma unroll
    for (int kk = 0; kk < DwRing::BK / 2; ++kk) {
        if (kk + 2 < DwRing::BK / 2) __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 4, 0);
    }
}

__global__ __launch_bounds__(kDwThreads) void dw1_part_f32(const float *__restrict__ T, int64_t n_rows,
                                                            int F, const int32_t *__restrict__ uniq,
                                                            const int32_t *__restrict__ n_uniq_p, int cap,
                                                            const float *__restrict__ dZ1, int H, int KC,
                                                            const float *__restrict__ zero_row,
                                                            float *__restrict__ part)
{
    using R = DwRing;
    __shared__ __attribute__((aligned(16))) float ring0[R::SLOT];
    __shared__ __attribute__((aligned(16))) float ring1[R::SLOT];
    __shared__ __attribute__((aligned(16))) float ring2[R::SLOT];

    const int nnt = F / R::BN;
    // the column tiles of one chunk go to one XCD: they share its dZ1 rows
    int c, nt;
    if (!xcd_tile(blockIdx.x, KC, nnt, c, nt)) return;
    const int n_u = min(*n_uniq_p, cap);
    const int u0 = (int)((int64_t)c * n_u / KC), u1 = (int)((int64_t)(c + 1) * n_u / KC);
    const int m0 = 0, n0 = nt * R::BN;
    const int lane = ams_lane(), wave = threadIdx.x / AMS_WAVE;

    v16f acc[4] = {(v16f){}, (v16f){}, (v16f){}, (v16f){}};
    const int S = (u1 - u0 + R::BK - 1) / R::BK;
    if (S > 0) {
        int id0[2], id1[2], id2[2];
#define DW_BASE(s) (u0 + min((s), S - 1) * R::BK)
        // prologue: IDs of stages 0..2 resident, IDs of stage 3 in flight, DMA 0 and 1 issued
        dw1_load_ids(uniq, DW_BASE(0), u1, wave, lane, id0);
        dw1_load_ids(uniq, DW_BASE(1), u1, wave, lane, id1);
        dw1_load_ids(uniq, DW_BASE(2), u1, wave, lane, id2);
        AMS_WAIT_VM(0);
        int idn[2];
        dw1_load_ids(uniq, DW_BASE(3), u1, wave, lane, idn);
        dw1_issue(ring0, T, n_rows, F, dZ1, H, m0, n0, DW_BASE(0), u1, zero_row, id0, wave, lane);
        dw1_issue(ring1, T, n_rows, F, dZ1, H, m0, n0, DW_BASE(1), u1, zero_row, id1, wave, lane);
#define DW_STAGE(cur, nxt, ids_next_dma, ids_load, s)                                          \
    do {                                                                                        \
        __builtin_amdgcn_sched_barrier(0);                                         \
        AMS_WAIT_VM_LDS(R::OUTSTANDING);                                                        \
        __builtin_amdgcn_s_barrier();                                                           \
        __builtin_amdgcn_sched_barrier(0);                                                      \
        dw1_load_ids(uniq, DW_BASE((s) + 4), u1, wave, lane, ids_load);                         \
        dw1_issue(nxt, T, n_rows, F, dZ1, H, m0, n0, DW_BASE((s) + 2), u1, zero_row, ids_next_dma, \
                  wave, lane);                                                                  \
        __builtin_amdgcn_sched_barrier(0);                                                      \
        dw1_compute(cur, acc, lane, wave);                                                      \
    } while (0)
        // register roles rotate with the 3-stage unroll: at stage s the IDs of
        // stage s+2 feed the DMA and those of stage s+4 are loaded
        id0[0] = idn[0];
        id0[1] = idn[1];
        // now: id2 = stage 2, id0 = stage 3 (in flight), id1 free
        int s = 0;
        for (; s + 3 <= S; s += 3) {
            DW_STAGE(ring0, ring2, id2, id1, s);       // DMA stage s+2, load stage s+4
            DW_STAGE(ring1, ring0, id0, id2, s + 1);   // DMA stage s+3, load stage s+5
            DW_STAGE(ring2, ring1, id1, id0, s + 2);   // DMA stage s+4, load stage s+6
        }
        if (s < S) DW_STAGE(ring0, ring2, id2, id1, s);
        if (s + 1 < S) DW_STAGE(ring1, ring0, id0, id2, s + 1);
#undef DW_STAGE
#undef DW_BASE
        AMS_WAIT_VM(0);
    }

    float *out = part + (size_t)c * H * F;
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int nb = 0; nb < 2; ++nb) {
            const int col = n0 + (wave & 1) * 64 + nb * 32 + (lane & 31);
#pragma unroll
            for (int j = 0; j < 16; ++j) {
                const int row = m0 + (wave >> 1) * 64 + mb * 32 + acc_row(j, lane);
                out[(size_t)row * F + col] = acc[mb * 2 + nb][j];
            }
        }
}

// bf16 partial dW1 = dZ1^T T[uniq] over one fixed chunk of unique images,
// for H = 256: a block owns all 256 rows of dW1 and 128 of its columns, so a
// feature row is read once per chunk.  The contraction runs over unique
// images, the row index of both operands, while the bf16 MFMA wants 8
// consecutive k per lane: both tiles sit in LDS row-major ([image][column])
// and are read with ds_read_b64_tr_b16, which hands lane j of a 16-lane group
// column (base + j) of four consecutive rows when lane i of the group points
// at row (i / 4), columns 4 (i % 4) .. +3.  Two such reads give the 8 values
// of one operand.
//
// Stage = 64 images (4 MFMA k-steps of 16): A = dZ1 rows (64 x 256 bf16,
// 32 KB), B = feature rows (64 x 128 bf16, 16 KB), DMA'd through a 3-slot
// ring like the fp32 kernel.  16-byte chunks are stored at chunk ^ 4 (row & 3):
// the 4 rows x 64 bytes that a half-wave's transpose reads touch then fall
// in distinct banks.  Waves are 4 (h) x 2 (f), 64 x 64 each.
// BN = 128 (64 unique images per stage, 48 KB slots) serves the smaller
// unique counts; from kDwTrWideCap slots on, 256-column tiles run as
// dw1_rs_bf16 (below), which keeps the same operand layout.
template <int BN_>
struct DwTrT {
    static constexpr int BM = 256, BN = BN_, BK = BN_ == 256 ? 32 : 64, WAVES = 8;
    static constexpr int NB = BN / 64;                            // 32-column blocks per wave
    static constexpr int KK = BK / 16;                            // MFMA k steps per stage
    static constexpr int A_BYTES = BK * BM * 2, B_BYTES = BK * BN * 2;
    static constexpr int SLOT = (A_BYTES + B_BYTES) / 4;           // floats per slot
    static constexpr int PA = A_BYTES / 1024 / WAVES;             // DMA instructions per wave
    static constexpr int PB = B_BYTES / 1024 / WAVES;
    static constexpr int CPR = BN * 2 / 16, RPI = 64 / CPR;       // B: 16-byte chunks per row, rows per DMA
    static constexpr int OUTSTANDING = PA + PB + PB;              // DMA of s+1, IDs of s+3
};
using DwTr = DwTrT<128>;
// dW1 tile width for `cap` unique-image slots: the wide tile pays off once
// each of its blocks has enough rows to amortise its 256 KB partial tile.
constexpr int kDwTrWideCap = 131072;
inline int dwtr_bn(int F, int32_t cap) { return (cap >= kDwTrWideCap && F % 256 == 0) ? 256 : 128; }

__device__ __forceinline__ int dwtr_swz(int row) { return (row & 3) << 2; }

typedef short v4s __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4s lds_v4s_t;

__device__ __forceinline__ uint2 ds_read_tr16(const void *p)
{
    const v4s v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s_t *)p);
    return __builtin_bit_cast(uint2, v);
}

// IDs of this lane's B rows (one per B DMA instruction) of the stage at u_base
template <class R>
__device__ __forceinline__ void dwtr_load_ids(const int32_t *__restrict__ uniq, int u_base, int u1, int wave,
                                              int lane, int (&id)[R::PB])
{
#pragma unroll
    for (int q = 0; q < R::PB; ++q) {
        const int row = R::RPI * (R::PB * wave + q) + lane / R::CPR;
        const int u = u_base + row;
        const int v = uniq[min(u, u1 - 1)];           // always issued: uniform op count
        id[q] = u < u1 ? v : -1;
    }
}

template <class R>
__device__ __forceinline__ void dwtr_issue(float *slot, const uint16_t *__restrict__ T, int64_t n_rows, int F,
                                           const uint16_t *__restrict__ dZ1, int n0, int u_base, int u1,
                                           const void *__restrict__ zero_row, const int (&id)[R::PB], int wave,
                                           int lane)
{
    // A: 512-byte rows, 2 per instruction
#pragma unroll
    for (int q = 0; q < R::PA; ++q) {
        const int j = R::PA * wave + q;
        const int row = 2 * j + (lane >> 5), pc = lane & 31;
        const int u = u_base + row;
        const int lc = pc ^ dwtr_swz(row);
        const char *src = u < u1 ? (const char *)(dZ1 + (size_t)u * R::BM) + lc * 16
                                 : (const char *)zero_row + lc * 16;
        dma16(src, slot + j * 256);
    }
    // B: BN columns from n0 per row, RPI rows per instruction
#pragma unroll
    for (int q = 0; q < R::PB; ++q) {
        const int j = R::PB * wave + q;
        const int row = R::RPI * j + lane / R::CPR, pc = lane % R::CPR;
        const int lc = pc ^ dwtr_swz(row);
        const bool ok = id[q] >= 0 && (int64_t)id[q] < n_rows;
        const char *src = ok ? (const char *)(T + (size_t)id[q] * F + n0) + lc * 16
                             : (const char *)zero_row + lc * 16;
        dma16(src, slot + R::A_BYTES / 4 + j * 256);
    }
}

// Byte offset of (row, col) in a swizzled bf16 tile with `rb`-byte rows.
__device__ __forceinline__ int dwtr_off(int row, int col, int rb)
{
    return row * rb + (((col >> 3) ^ dwtr_swz(row)) << 4) + ((col & 7) << 1);
}

template <class R>
__device__ __forceinline__ void dwtr_compute(const float *slot, v16f *acc, int lane, int wave)
{
    const char *A = (const char *)slot, *B = (const char *)slot + R::A_BYTES;
    const int g = lane >> 4, i = lane & 15;
    const int wm = wave >> 1, wn = wave & 1;
    // this lane's transpose-read address: row (i / 4) of its group's 4-row
    // block, columns 4 (i % 4) .. +3 of its group's 16-column half
    const int r_in = 8 * (g >> 1) + (i >> 2);
    const int c_in = 16 * (g & 1) + 4 * (i & 3);
    constexpr int NB = R::NB, KK = R::KK;
    uint4 a[KK][2], b[KK][NB];
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
        const int r0 = 16 * kk + r_in;
#pragma unroll
        for (int mb = 0; mb < 2; ++mb) {
            const int col = wm * 64 + mb * 32 + c_in;
            const uint2 lo = ds_read_tr16(A + dwtr_off(r0, col, R::BM * 2));
            const uint2 hi = ds_read_tr16(A + dwtr_off(r0 + 4, col, R::BM * 2));
            a[kk][mb] = make_uint4(lo.x, lo.y, hi.x, hi.y);
        }
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
            const int col = wn * (R::BN / 2) + nb * 32 + c_in;
            const uint2 lo = ds_read_tr16(B + dwtr_off(r0, col, R::BN * 2));
            const uint2 hi = ds_read_tr16(B + dwtr_off(r0 + 4, col, R::BN * 2));
            b[kk][nb] = make_uint4(lo.x, lo.y, hi.x, hi.y);
        }
    }
#pragma unroll
    for (int kk = 0; kk < KK; ++kk)
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) acc[mb * NB + nb] = mfma_bf16(a[kk][mb], b[kk][nb], acc[mb * NB + nb]);
    // k-step 0's reads first, then (reads of kk+1, MFMAs of kk)
    __builtin_amdgcn_sched_group_barrier(0x100, 4 + 2 * NB, 0);
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
        if (kk < KK - 1) __builtin_amdgcn_sched_group_barrier(0x100, 4 + 2 * NB, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 2 * NB, 0);
    }
}

template <int BN>
__global__ __launch_bounds__(DwTrT<BN>::WAVES * AMS_WAVE) void dw1_part_bf16(
    const uint16_t *__restrict__ T, int64_t n_rows, int F, const int32_t *__restrict__ uniq,
    const int32_t *__restrict__ n_uniq_p, int cap, const uint16_t *__restrict__ dZ1, int KC,
    const void *__restrict__ zero_row, float *__restrict__ part)
{
    using R = DwTrT<BN>;
    __shared__ __attribute__((aligned(16))) float ring0[R::SLOT];
    __shared__ __attribute__((aligned(16))) float ring1[R::SLOT];
    __shared__ __attribute__((aligned(16))) float ring2[R::SLOT];

    const int nnt = F / R::BN;
    // the column tiles of one chunk go to one XCD: they share its dZ1 rows
    int c, nt;
    if (!xcd_tile(blockIdx.x, KC, nnt, c, nt)) return;
    const int n_u = min(*n_uniq_p, cap);
    const int u0 = (int)((int64_t)c * n_u / KC), u1 = (int)((int64_t)(c + 1) * n_u / KC);
    const int n0 = nt * R::BN;
    const int lane = ams_lane(), wave = threadIdx.x / AMS_WAVE;

    v16f acc[2 * R::NB];
#pragma unroll
    for (int x = 0; x < 2 * R::NB; ++x) acc[x] = (v16f){};
    const int S = (u1 - u0 + R::BK - 1) / R::BK;
    if (S > 0) {
        int id0[2], id1[2], id2[2];
#define DT_BASE(s) (u0 + min((s), S - 1) * R::BK)
        dwtr_load_ids<R>(uniq, DT_BASE(0), u1, wave, lane, id0);
        dwtr_load_ids<R>(uniq, DT_BASE(1), u1, wave, lane, id1);
        dwtr_load_ids<R>(uniq, DT_BASE(2), u1, wave, lane, id2);
        AMS_WAIT_VM(0);
        int idn[2];
        dwtr_load_ids<R>(uniq, DT_BASE(3), u1, wave, lane, idn);
        dwtr_issue<R>(ring0, T, n_rows, F, dZ1, n0, DT_BASE(0), u1, zero_row, id0, wave, lane);
        dwtr_issue<R>(ring1, T, n_rows, F, dZ1, n0, DT_BASE(1), u1, zero_row, id1, wave, lane);
#define DT_STAGE(cur, nxt, ids_next_dma, ids_load, s)                                           \
    do {                                                                                         \
        __builtin_amdgcn_sched_barrier(0);                                                       \
        AMS_WAIT_VM_LDS(R::OUTSTANDING);                                                         \
        __builtin_amdgcn_s_barrier();                                                            \
        __builtin_amdgcn_sched_barrier(0);                                                       \
        dwtr_load_ids<R>(uniq, DT_BASE((s) + 4), u1, wave, lane, ids_load);                         \
        dwtr_issue<R>(nxt, T, n_rows, F, dZ1, n0, DT_BASE((s) + 2), u1, zero_row, ids_next_dma, wave, \
                   lane);                                                                        \
        __builtin_amdgcn_sched_barrier(0);                                                       \
        dwtr_compute<R>(cur, acc, lane, wave);                                                      \
    } while (0)
        id0[0] = idn[0];
        id0[1] = idn[1];
        // id2 = stage 2, id0 = stage 3 (in flight), id1 free
        int s = 0;
        for (; s + 3 <= S; s += 3) {
            DT_STAGE(ring0, ring2, id2, id1, s);
            DT_STAGE(ring1, ring0, id0, id2, s + 1);
            DT_STAGE(ring2, ring1, id1, id0, s + 2);
        }
        if (s < S) DT_STAGE(ring0, ring2, id2, id1, s);
        if (s + 1 < S) DT_STAGE(ring1, ring0, id0, id2, s + 1);
#undef DT_STAGE
#undef DT_BASE
        AMS_WAIT_VM(0);
    }

    float *out = part + (size_t)c * R::BM * F;
    const int wm = wave >> 1, wn = wave & 1;
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int nb = 0; nb < R::NB; ++nb) {
            const int col = n0 + wn * (R::BN / 2) + nb * 32 + (lane & 31);
#pragma unroll
            for (int j = 0; j < 16; ++j) {
                const int row = wm * 64 + mb * 32 + acc_row(j, lane);
                out[(size_t)row * F + col] = acc[mb * R::NB + nb][j];
            }
        }
}

// ---- bf16 dW1 for large unique counts ----
// Partial dW1 of chunk c (of KC) over feature columns n0 .. n0 + 255, the
// same contraction and operand layout as dw1_part_bf16, with 256-column tiles (a block owns all 256
// hidden rows x 256 feature columns of one chunk of the unique images; 8
// waves in 4 (m) x 2 (n), each 64 x 128) with the first layer's row-split
// pipeline: a stage is 64 unique images (2048 MFMA cycles per SIMD, so the
// fixed cost of a stage is paid half as often), the dZ1 rows of a stage
// (64 x 512 bytes, an L2 hit for all but the first of the chunk's 16 column
// blocks, which run on one XCD) move by DMA into a 2-slot LDS ring one stage
// ahead, and the stage's pieces of the gathered feature rows (64 x 512
// bytes, the HBM stream) by non-temporal DMA into a 3-slot ring two stages
// ahead; every DMA instruction reads two whole 512-byte row pieces.  The
// IDs of a stage's rows are uniform per wave (its 8 rows) and come by
// scalar loads one stage before their DMA is issued, so the vector memory
// queue holds only DMAs and each stage waits with s_waitcnt vmcnt(4): the
// next stage's feature rows may stay in flight.  Slot rows are 512 bytes,
// swizzled by 16-byte chunk as dwtr_swz (for the transposed operand reads);
// stages past the chunk DMA the zero row.
namespace dwr {
constexpr int kThreads = 512;
constexpr int kWaves = kThreads / AMS_WAVE;
constexpr int BM = 256, BN = 256, BK = 64;    // hidden rows, feature columns, images per stage
constexpr int KK = BK / 16;                   // MFMA k steps per stage
constexpr int NB = BN / 64;                   // 32-column blocks per wave (a wave spans BN / 2 columns)
constexpr int NA = 2, NX = 3;                 // dZ1 slots (1 stage ahead), feature-row slots (2 ahead)
constexpr int SLOT = BK * 512;                // 32 KB: 64 rows of 512 bytes (both operands)
constexpr int DMA = 4;                        // DMA instructions per wave and slot (2 rows each)
constexpr int WAIT = 4;                       // ops a stage may leave in flight (the next stage's rows)
static_assert(BM * 2 == 512 && BN * 2 == 512, "both operands have 512-byte slot rows");
static_assert((NA + NX) * SLOT <= 160 * 1024, "the rings fit the LDS");
static_assert(DMA * 1024 * kWaves == SLOT && kWaves == 8, "8 slot rows per wave, 2 per DMA instruction");
static_assert(WAIT == DMA, "wait count follows the issue order");
}  // namespace dwr

__device__ __forceinline__ void dwr_dma(const char *src, uint32_t lds_addr)
{
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off"
                 :
                 : "s"(lds_addr), "v"(src)
                 : "memory", "m0");
}

// One stage's products: A = dZ1 slot [image][hidden], B = feature slot
// [image][column]; both operands by transposed 8-byte reads (dwtr_compute's
// lane mapping), the next k step's reads issued while this one's products run.
__device__ __forceinline__ void dwr_compute(const char *A, const char *B, v16f (&acc)[2 * dwr::NB], int lane,
                                            int wave)
{
    using namespace dwr;
    const int g = lane >> 4, i = lane & 15;
    const int wm = wave >> 1, wn = wave & 1;
    const int r_in = 8 * (g >> 1) + (i >> 2);
    const int c_in = 16 * (g & 1) + 4 * (i & 3);
    uint4 a[KK][2], b[KK][NB];
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
        const int r0 = 16 * kk + r_in;
#pragma unroll
        for (int mb = 0; mb < 2; ++mb) {
            const int col = wm * 64 + mb * 32 + c_in;
            const uint2 lo = ds_read_tr16(A + dwtr_off(r0, col, 512));
            const uint2 hi = ds_read_tr16(A + dwtr_off(r0 + 4, col, 512));
            a[kk][mb] = make_uint4(lo.x, lo.y, hi.x, hi.y);
        }
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
            const int col = wn * (BN / 2) + nb * 32 + c_in;
            const uint2 lo = ds_read_tr16(B + dwtr_off(r0, col, 512));
            const uint2 hi = ds_read_tr16(B + dwtr_off(r0 + 4, col, 512));
            b[kk][nb] = make_uint4(lo.x, lo.y, hi.x, hi.y);
        }
    }
#pragma unroll
    for (int kk = 0; kk < KK; ++kk)
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) acc[mb * NB + nb] = mfma_bf16(a[kk][mb], b[kk][nb], acc[mb * NB + nb]);
    __builtin_amdgcn_sched_group_barrier(0x100, 4 + 2 * NB, 0);
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
        if (kk < KK - 1) __builtin_amdgcn_sched_group_barrier(0x100, 4 + 2 * NB, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 2 * NB, 0);
    }
}

__global__ __launch_bounds__(dwr::kThreads) __attribute__((amdgpu_waves_per_eu(2, 2))) void dw1_rs_bf16(
    const uint16_t *__restrict__ T, int64_t n_rows, int F, const int32_t *__restrict__ uniq,
    const int32_t *__restrict__ n_uniq_p, int cap, const uint16_t *__restrict__ dZ1, int KC,
    float *__restrict__ part)
{
    using namespace dwr;
    __shared__ __attribute__((aligned(1024))) char ring[(NA + NX) * SLOT];
    const int nnt = F / BN;
    // the column tiles of one chunk go to one XCD: they share its dZ1 rows
    int c, nt;
    if (!xcd_tile(blockIdx.x, KC, nnt, c, nt)) return;
    const int n_u = min(*n_uniq_p, cap);
    const int u0 = (int)((int64_t)c * n_u / KC), u1 = (int)((int64_t)(c + 1) * n_u / KC);
    const int n0 = nt * BN;
    const int lane = ams_lane();
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / AMS_WAVE);

    v16f acc[2 * NB];
#pragma unroll
    for (int x = 0; x < 2 * NB; ++x) acc[x] = (v16f){};
    const int S = (u1 - u0 + BK - 1) / BK;
    if (S > 0) {
        const uint32_t lds0 = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)ring);
        const uint32_t lds_a = lds0 + 4 * wave * 1024, lds_x = lds0 + NA * SLOT + 4 * wave * 1024;
        // DMA instruction q of this wave: slot rows 8 wave + 2 q + lane / 32,
        // chunk lane % 32 holding source chunk (lane % 32) ^ dwtr_swz(row)
        const int half = lane >> 5;
        int co[DMA];
#pragma unroll
        for (int q = 0; q < DMA; ++q) co[q] = ((lane & 31) ^ dwtr_swz(8 * wave + 2 * q + half)) << 4;
        const char *zero = (const char *)rs_zero_row;
        asm volatile("" : "+s"(zero));             // once, not per DMA
        auto a_src = [&](int s, int q) -> const char * {
            const int u = u0 + s * BK + 8 * wave + 2 * q + half;
            return (u < u1 ? (const char *)(dZ1 + (size_t)u * BM) : zero) + co[q];
        };
        // the IDs of stage s's rows 8 wave .. + 7 (uniform per wave)
        auto load_ids = [&](int s, int (&id)[8]) {
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int u = u0 + s * BK + 8 * wave + e;
                const int v = uniq[min(u, u1 - 1)];
                id[e] = u < u1 ? v : -1;
            }
        };
        auto x_src = [&](const int (&id)[8], int q) -> const char * {
            // lane half 0 takes row 2 q, half 1 row 2 q + 1 (a select, not an
            // indexed read, which would put the IDs in scratch memory)
            const int v = id[2 * q] + ((id[2 * q + 1] - id[2 * q]) & -half);
            const bool ok = v >= 0 && (int64_t)v < n_rows;
            const char *row = (const char *)(T + (size_t)(ok ? v : 0) * F + n0);
            return (ok ? row : zero) + co[q];
        };
        // prologue: X(0), dZ1(0), X(1), in the order a stage issues them
        int id[8];
        load_ids(0, id);
#pragma unroll
        for (int q = 0; q < DMA; ++q) rs_dma_row(x_src(id, q), lds_x + q * 1024);
#pragma unroll
        for (int q = 0; q < DMA; ++q) dwr_dma(a_src(0, q), lds_a + q * 1024);
        load_ids(1, id);
#pragma unroll
        for (int q = 0; q < DMA; ++q) rs_dma_row(x_src(id, q), lds_x + SLOT + q * 1024);
        load_ids(2, id);
        uint32_t xs_d = 2 * SLOT, xs_c = 0;       // feature slot to fill next, to compute from next
        for (int s = 0; s < S; ++s) {
            // stage s's dZ1 and feature rows have landed (all waves: the
            // barrier), and every wave is done with the slots refilled below
            asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)" ::"n"(WAIT) : "memory");
            __builtin_amdgcn_sched_barrier(0);
            __builtin_amdgcn_s_barrier();
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int q = 0; q < DMA; ++q) dwr_dma(a_src(s + 1, q), lds_a + ((s + 1) & 1) * SLOT + q * 1024);
#pragma unroll
            for (int q = 0; q < DMA; ++q) rs_dma_row(x_src(id, q), lds_x + xs_d + q * 1024);
            xs_d = xs_d == (NX - 1) * SLOT ? 0 : xs_d + SLOT;
            __builtin_amdgcn_sched_barrier(0);
            dwr_compute(ring + (s & 1) * SLOT, ring + NA * SLOT + xs_c, acc, lane, wave);
            xs_c = xs_c == (NX - 1) * SLOT ? 0 : xs_c + SLOT;
            __builtin_amdgcn_sched_barrier(0);
            load_ids(s + 3, id);                   // for the feature rows the next stage issues
        }
        // the DMAs issued past the last stage land before the block leaves
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    }

    float *out = part + (size_t)c * BM * F;
    const int wm = wave >> 1, wn = wave & 1;
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
            const int col = n0 + wn * (BN / 2) + nb * 32 + (lane & 31);
#pragma unroll
            for (int j = 0; j < 16; ++j) {
                const int row = wm * 64 + mb * 32 + acc_row(j, lane);
                out[(size_t)row * F + col] = acc[mb * NB + nb][j];
            }
        }
}

// ---- bf16 backward tail (H = 256) ----
//
// Per 32-row chunk of the block's unique images, all in LDS + registers:
//   phase A (all 256 threads, fp32): thread (o = t % 64, row group g = t / 64)
//     takes rows g + 4 k; with dzl = dE (masked by a final ReLU) and its W3
//     column in registers it forms dZ2 = (dzl W3) * [H2 > 0] (3 layers; dZ2 =
//     dzl for 2), splits it into a high and a low bf16 part (dZ2 = hi + lo to
//     2^-18 relative) in two tiles, and keeps running sums of db2 and (3
//     layers) dW3 = dzl^T H2 over its rows; the four row groups are added in
//     a fixed order at the end; threads d < D sum db3 over the chunk's rows;
//   phase B (wave w owns H1 columns i in [64 w, 64 w + 64)):
//     dH1 = dZ2 W2 on v_mfma_f32_32x32x16_bf16, one product per part (first
//     operand a dZ2 row, second a row of W2^T, both 16-byte LDS reads; W2 and
//     the saved H1 are exact in bf16, so both products are fp32-accurate), so
//     a lane holds dH1[rows 8 q + 4 h + r][i]; the H1 values of exactly those
//     (row, i) come from transposed LDS reads (ds_read_b64_tr_b16) of the H1
//     tile, give the ReLU mask dZ1 = dH1 * [H1 > 0] (summed into db1 in fp32,
//     rounded to bf16 into the wave's own columns of the H1 tile, from where
//     the block stores whole rows), and are at once the second operand of
//     dW2 += dZ2^T H1 (k = the chunk's rows, lane half h supplying rows
//     8 q + 4 h + r, q = 2 s, 2 s + 1), whose first operand is read
//     transposed from the dZ2 tiles.
// The next chunk's H1, H2 and dE are loaded into registers while the current
// one is computed.  Block partials have the layout of tail_bwd's
// ([dW2][db2][dW3][db3][db1]) and go through the same fixed-order reduction.
// Tile rows are padded so that a half-wave's reads spread over the banks:
// the dZ2 and W2^T tiles by 16 bytes (16-byte reads of 16 rows), the H1 tile
// by 32 (a transposed read takes 32 bytes of 4 consecutive rows, which then
// start 8 banks apart).
constexpr int kTbfBlocks = 512;
constexpr int kH1S = kMaxH1 * 2 + 32;       // bytes per H1 tile row
constexpr int kZ2S = kMaxH2 * 2 + 16;       // bytes per dZ2 tile row
constexpr int kW2S = kMaxH2 * 2 + 16;       // bytes per W2^T tile row

// Transposed read of a bf16 tile (stride bytes per row) for the 16-lane
// group of `lane`: rows R0..R0+3, columns C0..C0+15; the lane receives column
// C0 + (lane % 16) of the four rows.
__device__ __forceinline__ uint2 tr4(const char *tile, int stride, int R0, int C0, int lane)
{
    const int i16 = lane & 15;
    return ds_read_tr16(tile + (R0 + (i16 >> 2)) * stride + (C0 + 4 * (i16 & 3)) * 2);
}

__device__ __forceinline__ float bf16_elem(uint2 v, int r)
{
    const uint32_t w = r < 2 ? v.x : v.y;
    return __uint_as_float((r & 1) ? (w & 0xffff0000u) : (w << 16));
}

// DM: upper bound of D (16 or 32), the length of the per-thread dzl rows.
// PR: PReLU with slopes s1 [H], s2 [M] (3 layers): H1b holds Z1 and H2s Z2;
// the masks become 1 / slope, the dW2 and dW3 operands are the activations
// (dW2's re-rounded to bf16 from Z1's bf16), and the slope gradients
// sum dH * min(Z, 0) go to the two partial slots after db1.
template <int L, int DM, bool PR>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2)))
void tail_bwd_bf16(const uint16_t *__restrict__ H1b, const float *__restrict__ H2s,
                   const float *__restrict__ Efwd, const float *__restrict__ dE,
                   const uint16_t *__restrict__ W2, const uint16_t *__restrict__ W3, int M, int D,
                   int final_relu, const int32_t *__restrict__ n_uniq_p, int cap,
                   uint16_t *__restrict__ dZ1, float *__restrict__ part, int PS,
                   float *__restrict__ zero_row, int zero_n,
                   const float *__restrict__ s1, const float *__restrict__ s2)
{
    const int n_u = min(*n_uniq_p, cap);
    const int n_act = tail_active(n_u, (int)gridDim.x);
    if ((int)blockIdx.x >= n_act) return;          // (block 0 is always active)
    constexpr int H = kMaxH1;
    __shared__ __attribute__((aligned(16))) char H1t[32 * kH1S];      // H1, then dZ1, of the chunk
    __shared__ __attribute__((aligned(16))) char Z2t[32 * kZ2S];      // dZ2, high bf16 part
    __shared__ __attribute__((aligned(16))) char Z2l[32 * kZ2S];      // dZ2, low bf16 part
    __shared__ __attribute__((aligned(16))) char W2T[H * kW2S];
    __shared__ __attribute__((aligned(16))) float H2t[32 * kMaxH2];
    __shared__ __attribute__((aligned(16))) float Lt[32 * DM];

    const int t = threadIdx.x, lane = ams_lane(), wave = t / AMS_WAVE;
    const int h = lane >> 5, r32 = lane & 31;
    // the zero row that dW1's padding rows stream (read by the next launch)
    if (blockIdx.x == 0)
        for (int i = t; i < zero_n; i += kThreads) zero_row[i] = 0.f;
    const int Mo = (L == 3) ? M : D;
    // W2 transposed into LDS: thread t takes the 8 x 8 tile of rows
    // o0 = 8 (t % 8) .. + 7 and columns i0 = 8 (t / 8) .. + 7 (eight 16-byte
    // loads, all in flight together), transposes it in registers and writes
    // 8 rows of W2^T, 16 bytes each: the 8 threads of a column block fill
    // 128 contiguous bytes of a W2^T row, the next 8 the row 8 further on
    // (kW2S apart: the other bank half), so 16 lanes' writes meet no bank
    // twice
    static_assert(kMaxH2 * H == 64 * kThreads && kMaxH2 == 64, "one 8 x 8 tile per thread");
    {
        const int o0 = 8 * (t % 8), i0 = 8 * (t / 8);
        uint4 v[8];
#pragma unroll
        for (int a = 0; a < 8; ++a)
            v[a] = o0 + a < Mo ? *(const uint4 *)&W2[(size_t)(o0 + a) * H + i0] : make_uint4(0, 0, 0, 0);
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            uint32_t w[4];
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const uint4 r0 = v[2 * k], r1 = v[2 * k + 1];
                const uint32_t a0 = (j >> 1) == 0 ? r0.x : (j >> 1) == 1 ? r0.y : (j >> 1) == 2 ? r0.z : r0.w;
                const uint32_t a1 = (j >> 1) == 0 ? r1.x : (j >> 1) == 1 ? r1.y : (j >> 1) == 2 ? r1.z : r1.w;
                const uint32_t lo = (j & 1) ? (a0 >> 16) : (a0 & 0xffffu);
                const uint32_t hi = (j & 1) ? (a1 & 0xffff0000u) : (a1 << 16);
                w[k] = lo | hi;
            }
            *(uint4 *)(W2T + (i0 + j) * kW2S + o0 * 2) = make_uint4(w[0], w[1], w[2], w[3]);
        }
    }
    const int po = t & 63, pg = t >> 6;        // phase-A role: output o, row group
    const float sl2 = (PR && L == 3 && po < M) ? s2[po] : 0.f;
    float sl1[2];                              // slopes of phase B's columns 64 wave + 32 ib + r32
#pragma unroll
    for (int ib = 0; ib < 2; ++ib) sl1[ib] = PR ? s1[64 * wave + 32 * ib + r32] : 0.f;
    float w3c[DM];                             // W3[:, po] (3 layers)
    if (L == 3) {
        uint16_t wv[DM];                       // unconditional loads (index 0 past W3), all in flight
#pragma unroll
        for (int d = 0; d < DM; ++d) wv[d] = W3[(d < D && po < M) ? d * M + po : 0];
#pragma unroll
        for (int d = 0; d < DM; ++d) w3c[d] = (d < D && po < M) ? ams_bf16_to_f32(wv[d]) : 0.f;
    } else {
#pragma unroll
        for (int d = 0; d < DM; ++d) w3c[d] = 0.f;
    }

    const int r0 = (int)((int64_t)blockIdx.x * n_u / n_act);
    const int r1 = (int)((int64_t)(blockIdx.x + 1) * n_u / n_act);

    v16f dw2[2][2] = {{(v16f){}, (v16f){}}, {(v16f){}, (v16f){}}};   // [o block][i block]
    float db1a[2] = {0.f, 0.f}, ds1a[2] = {0.f, 0.f};
    float db2p = 0.f, db3p = 0.f, ds2p = 0.f;
    float dw3a[DM];
#pragma unroll
    for (int d = 0; d < DM; ++d) dw3a[d] = 0.f;
    uint4 pH1[4];
    float4 pH2[2];
    float pdz[4];
    auto fetch = [&](int c0) {
        const int nr = min(32, r1 - c0);
#pragma unroll
        for (int m = 0; m < 4; ++m) {
            const int idx = t + kThreads * m, row = idx >> 5, ch = idx & 31;
            pH1[m] = row < nr ? *(const uint4 *)(H1b + (size_t)(c0 + row) * H + ch * 8) : make_uint4(0, 0, 0, 0);
        }
        if (L == 3) {
#pragma unroll
            for (int m = 0; m < 2; ++m) {
                const int idx = t + kThreads * m, row = idx >> 4, c4 = idx & 15;
                pH2[m] = (row < nr && 4 * c4 < M) ? *(const float4 *)(H2s + (size_t)(c0 + row) * M + 4 * c4)
                                                  : make_float4(0.f, 0.f, 0.f, 0.f);
            }
        }
        // dE (and the forward's E for a final ReLU): unconditional loads,
        // index 0 of the chunk past its rows, all in flight
        float ev[4];
#pragma unroll
        for (int m = 0; m < 4; ++m) {
            const int idx = t + kThreads * m;
            const size_t at = (size_t)c0 * D + (idx < nr * D ? idx : 0);
            pdz[m] = dE[at];
            ev[m] = final_relu ? Efwd[at] : 1.f;
        }
#pragma unroll
        for (int m = 0; m < 4; ++m) {
            const int idx = t + kThreads * m;
            pdz[m] = (idx < nr * D && ev[m] > 0.f) ? pdz[m] : 0.f;
        }
    };

    if (r0 < r1) fetch(r0);
    for (int c0 = r0; c0 < r1; c0 += 32) {
        const int nr = min(32, r1 - c0);
        __syncthreads();                       // the previous chunk's tiles are consumed
#pragma unroll
        for (int m = 0; m < 4; ++m) {
            const int idx = t + kThreads * m, row = idx >> 5, ch = idx & 31;
            *(uint4 *)(H1t + row * kH1S + ch * 16) = pH1[m];
        }
        if (L == 3) {
#pragma unroll
            for (int m = 0; m < 2; ++m) {
                const int idx = t + kThreads * m, row = idx >> 4, c4 = idx & 15;
                *(float4 *)&H2t[row * kMaxH2 + 4 * c4] = pH2[m];
            }
        }
#pragma unroll
        for (int m = 0; m < 4; ++m) {
            const int idx = t + kThreads * m;
            if (idx < 32 * DM) Lt[idx] = 0.f;
        }
        __syncthreads();
#pragma unroll
        for (int m = 0; m < 4; ++m) {
            const int idx = t + kThreads * m;
            if (idx < 32 * D) Lt[(idx / D) * DM + idx % D] = pdz[m];
        }
        __syncthreads();
        if (c0 + 32 < r1) fetch(c0 + 32);

        // ---- phase A: dZ2 (fp32, split into two bf16 tiles), db2, dW3, db3
        if (L == 3 && t < D) {
            float a = 0.f;
            for (int rr = 0; rr < 32; ++rr) a += Lt[rr * DM + t];
            db3p += a;
        }
#pragma unroll 2
        for (int k = 0; k < 8; ++k) {
            const int rr = pg + 4 * k;
            float zl[DM];
#pragma unroll
            for (int d4 = 0; d4 < DM / 4; ++d4) {
                const float4 v = *(const float4 *)&Lt[rr * DM + 4 * d4];
                zl[4 * d4] = v.x;
                zl[4 * d4 + 1] = v.y;
                zl[4 * d4 + 2] = v.z;
                zl[4 * d4 + 3] = v.w;
            }
            float dz2;
            if constexpr (L == 3) {
                float a = 0.f;
#pragma unroll
                for (int d = 0; d < DM; ++d) a = fmaf(zl[d], w3c[d], a);
                const float h2 = H2t[rr * kMaxH2 + po];      // PReLU: Z2
                float act = h2;
                if (PR) {
                    dz2 = h2 > 0.f ? a : sl2 * a;
                    ds2p += h2 > 0.f ? 0.f : a * h2;
                    act = h2 > 0.f ? h2 : sl2 * h2;
                } else {
                    dz2 = h2 > 0.f ? a : 0.f;
                }
#pragma unroll
                for (int d = 0; d < DM; ++d) dw3a[d] = fmaf(zl[d], act, dw3a[d]);
            } else {
                dz2 = 0.f;
#pragma unroll
                for (int d = 0; d < DM; ++d)
                    if (d == po) dz2 = zl[d];
            }
            db2p += dz2;
            const uint16_t zh = ams_f32_to_bf16(dz2);
            *(uint16_t *)(Z2t + rr * kZ2S + po * 2) = zh;
            *(uint16_t *)(Z2l + rr * kZ2S + po * 2) = ams_f32_to_bf16(dz2 - ams_bf16_to_f32(zh));
        }
        __syncthreads();                       // dZ2 tiles complete

        // ---- phase B: dH1, dZ1, db1, dW2 for this wave's 64 columns
        {
            const int i0 = 64 * wave;
            v16f acc[2] = {(v16f){}, (v16f){}};
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                const uint4 ah = *(const uint4 *)(Z2t + r32 * kZ2S + (16 * s + 8 * h) * 2);
                const uint4 al = *(const uint4 *)(Z2l + r32 * kZ2S + (16 * s + 8 * h) * 2);
#pragma unroll
                for (int ib = 0; ib < 2; ++ib) {
                    const uint4 b = *(const uint4 *)(W2T + (i0 + 32 * ib + r32) * kW2S + (16 * s + 8 * h) * 2);
                    acc[ib] = mfma_bf16(ah, b, acc[ib]);
                    acc[ib] = mfma_bf16(al, b, acc[ib]);
                }
            }
            const int cg = 16 * ((lane >> 4) & 1);
            uint2 hv[2][4];
#pragma unroll
            for (int ib = 0; ib < 2; ++ib)
#pragma unroll
                for (int q = 0; q < 4; ++q) hv[ib][q] = tr4(H1t, kH1S, 8 * q + 4 * h, i0 + 32 * ib + cg, lane);
#pragma unroll
            for (int ib = 0; ib < 2; ++ib) {
                const int icol = i0 + 32 * ib + r32;
                float cs = 0.f, css = 0.f;
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    float av[4];               // PReLU: the activation, dW2's operand
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const float z1 = bf16_elem(hv[ib][q], r), g = acc[ib][4 * q + r];
                        float dz;
                        if (PR) {
                            dz = z1 > 0.f ? g : sl1[ib] * g;
                            css += z1 > 0.f ? 0.f : g * z1;
                            av[r] = z1 > 0.f ? z1 : sl1[ib] * z1;
                        } else {
                            dz = z1 > 0.f ? g : 0.f;
                        }
                        cs += dz;
                        // this wave's own columns of the H1 tile now hold dZ1
                        *(uint16_t *)(H1t + (8 * q + 4 * h + r) * kH1S + icol * 2) = ams_f32_to_bf16(dz);
                    }
                    if (PR) hv[ib][q] = make_uint2(pack_bf16(av[0], av[1]), pack_bf16(av[2], av[3]));
                }
                db1a[ib] += cs + __shfl_xor(cs, 32, AMS_WAVE);
                if (PR) ds1a[ib] += css + __shfl_xor(css, 32, AMS_WAVE);
            }
#pragma unroll
            for (int s = 0; s < 2; ++s) {
                uint4 a[2][2];                 // [part][o block]
#pragma unroll
                for (int ob = 0; ob < 2; ++ob)
#pragma unroll
                    for (int pt = 0; pt < 2; ++pt) {
                        const char *zt = pt ? Z2l : Z2t;
                        const uint2 r0v = tr4(zt, kZ2S, 16 * s + 4 * h, 32 * ob + cg, lane);
                        const uint2 r1v = tr4(zt, kZ2S, 16 * s + 8 + 4 * h, 32 * ob + cg, lane);
                        a[pt][ob] = make_uint4(r0v.x, r0v.y, r1v.x, r1v.y);
                    }
#pragma unroll
                for (int ib = 0; ib < 2; ++ib) {
                    const uint4 b = make_uint4(hv[ib][2 * s].x, hv[ib][2 * s].y, hv[ib][2 * s + 1].x,
                                               hv[ib][2 * s + 1].y);
#pragma unroll
                    for (int ob = 0; ob < 2; ++ob) {
                        dw2[ob][ib] = mfma_bf16(a[0][ob], b, dw2[ob][ib]);
                        dw2[ob][ib] = mfma_bf16(a[1][ob], b, dw2[ob][ib]);
                    }
                }
            }
        }
        __syncthreads();                       // dZ1 tile complete: whole rows out
#pragma unroll
        for (int m = 0; m < 4; ++m) {
            const int idx = t + kThreads * m, row = idx >> 5, ch = idx & 31;
            if (row < nr) *(uint4 *)(dZ1 + (size_t)(c0 + row) * H + ch * 8) = *(const uint4 *)(H1t + row * kH1S + ch * 16);
        }
    }

    float *p = part + (size_t)blockIdx.x * PS;
    const int i0 = 64 * wave;
#pragma unroll
    for (int ob = 0; ob < 2; ++ob)
#pragma unroll
        for (int ib = 0; ib < 2; ++ib)
#pragma unroll
            for (int j = 0; j < 16; ++j) {
                const int o = acc_row(j, lane) + 32 * ob;
                if (o < Mo) p[(size_t)o * H + i0 + 32 * ib + r32] = dw2[ob][ib][j];
            }
    p += Mo * H;
    // the four row groups of db2, dW3 and db3, added in a fixed order
    float *red = (float *)H1t;                 // 4 x DM x 64 floats (16 KB at DM = 16)
    __syncthreads();
    H2t[t] = db2p;
    __syncthreads();
    if (t < Mo) p[t] = ((H2t[t] + H2t[64 + t]) + H2t[128 + t]) + H2t[192 + t];
    p += Mo;
    if (L == 3) {
        for (int d0 = 0; d0 < DM; d0 += 16) {  // in slices of 16 d (the tile holds 4 x 16 x 64)
            __syncthreads();
#pragma unroll
            for (int d = 0; d < 16; ++d) red[(pg * 16 + d) * 64 + po] = dw3a[d0 + d];
            __syncthreads();
            for (int e = t; e < 16 * 64; e += kThreads) {
                const int d = d0 + e / 64, o = e % 64;
                if (d < D && o < M)
                    p[d * M + o] = ((red[(0 * 16 + e / 64) * 64 + o] + red[(1 * 16 + e / 64) * 64 + o]) +
                                    red[(2 * 16 + e / 64) * 64 + o]) + red[(3 * 16 + e / 64) * 64 + o];
            }
        }
        p += D * M;
        if (t < D) p[t] = db3p;
        p += D;
    }
    if (h == 0) {
        p[i0 + r32] = db1a[0];
        p[i0 + 32 + r32] = db1a[1];
    }
    if (PR) {   // slope gradients: [H], then [M] from the four row groups in a fixed order
        p += H;
        if (h == 0) {
            p[i0 + r32] = ds1a[0];
            p[i0 + 32 + r32] = ds1a[1];
        }
        p += H;
        if (L == 3) {
            __syncthreads();
            H2t[t] = ds2p;
            __syncthreads();
            if (t < M) p[t] = ((H2t[t] + H2t[64 + t]) + H2t[128 + t]) + H2t[192 + t];
        }
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

int sk_workers();

bool use_dw_ring(const ams_mlp *m) { return m->dtype != AMS_BF16 && m->dims[1] == DwRing::BM && m->dims[0] % DwRing::BN == 0; }
bool use_dw_tr(const ams_mlp *m) { return m->dtype == AMS_BF16 && m->dims[1] == DwTr::BM && m->dims[0] % DwTr::BN == 0; }

// Split-K chunk count of dW1: the DMA-ring kernel takes one block per CU
// (tiles x chunks = CUs); the fallback kernel aims at ~1024 blocks.
int dw1_chunks(const ams_mlp *m, int32_t cap)
{
    const int H = m->dims[1], F = m->dims[0];
    int kc;
    if (use_dw_ring(m)) {
        kc = sk_workers() / (F / DwRing::BN);
    } else if (use_dw_tr(m)) {
        kc = sk_workers() / (F / dwtr_bn(F, cap));
    } else {
        const int bm = (H % 128 == 0) ? 128 : 64;
        kc = 1024 / ((H / bm) * (F / 64));
    }
    return kc < 1 ? 1 : (kc > 32 ? 32 : kc);
}

// [dW2][db2][dW3][db3][db1], then the PReLU slope gradients [H][M] (their
// slots are always there and written only in PReLU mode).
int tail_part_size(const ams_mlp *m)
{
    const int L = m->n_layers, H = m->dims[1], D = m->dims[L];
    const int M = (L == 3) ? m->dims[2] : D;
    return M * H + M + ((L == 3) ? D * M + D : 0) + H + H + ((L == 3) ? M : 0);
}

// The bf16 backward tail (bf16 MFMA) serves H = 256 with a second-layer
// width that is a multiple of 4; other shapes use the fp32-MFMA tail.
bool use_tail_bf16(const ams_mlp *m)
{
    return m->dtype == AMS_BF16 && m->dims[1] == kMaxH1 &&
           (m->n_layers == 2 || (m->dims[2] % 4 == 0 && m->dims[2] * m->dims[3] <= 4 * kThreads));
}

int tail_blocks(const ams_mlp *m) { return use_tail_bf16(m) ? kTbfBlocks : kTailBlocks; }

struct BwdPlan {
    size_t off_zero, off_dz1, off_tail, off_dw1, total;
    int kc;
};

BwdPlan plan_bwd(const ams_mlp *m, int32_t cap)
{
    BwdPlan p{};
    const int H = m->dims[1], F = m->dims[0];
    const size_t es = (m->dtype == AMS_BF16) ? 2 : 4;
    p.kc = dw1_chunks(m, cap);
    size_t o = 0;
    p.off_zero = o; o += al256((size_t)(F > H ? F : H) * 4);
    p.off_dz1 = o; o += al256((size_t)cap * H * es);
    p.off_tail = o; o += al256((size_t)tail_blocks(m) * tail_part_size(m) * 4);
    p.off_dw1 = o; o += al256((size_t)p.kc * H * F * 4);
    p.total = o;
    return p;
}

// Stream-K workers: one per compute unit of the current device (a multiple
// of 8, the XCD count), 256 on MI355X.
int sk_workers()
{
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n < 8)
        n = 256;
    return (n / 8) * 8;
}

bool use_stream_k(const ams_mlp *m) { return m->dims[1] % kSkBN == 0; }

// The row-split bf16 first layer (H = 256, F = 4096) once the capacity
// holds at least two of its 256-row tiles per CU: it then gives every CU
// whole tiles and its output needs no partial-tile pass.  Below that (the
// 1024-sample batches, ~50 unique rows per CU) each CU would stream all of W1
// for a few rows, and the stream-K kernel, which splits K instead, is faster.
bool use_row_split(const ams_mlp *m, int32_t cap)
{
    return m->dtype == AMS_BF16 && m->dims[1] == rs::BN && m->dims[0] == rs::kF &&
           (int64_t)cap >= 2 * (int64_t)rs::BM * sk_workers();
}

}  // namespace

extern "C" size_t ams_embed_workspace(const ams_mlp *mlp, int32_t n_uniq_cap)
{
    if (!mlp_ok(mlp) || n_uniq_cap < 0) return 0;
    // forward: fp32 H1 (bf16 mode, or when the caller keeps no fp32 H1_save),
    // then the stream-K partial tiles (two per worker)
    size_t fwd = al256((size_t)n_uniq_cap * mlp->dims[1] * 4);
    if (use_stream_k(mlp)) {
        fwd += al256((size_t)sk_workers() * 2 * (mlp->dtype == AMS_BF16 ? Sk<uint16_t>::TILE : Sk<float>::TILE) * 4);
        if (mlp->dtype == AMS_F32_X3) fwd += al256((size_t)3 * mlp->dims[0] * mlp->dims[1] * 2);   // W1 parts
    }
    const size_t bwd = plan_bwd(mlp, n_uniq_cap).total;
    return fwd > bwd ? fwd : bwd;
}

// PReLU slopes of the hidden layers: NULL (ReLU), or one array per hidden
// layer.  float32 paths, and bf16 where the bf16 tails run both directions
// (first layer 256 wide: stream-K or row-split).
ams_status prelu_slopes(const ams_mlp *mlp, const float *const *slope, const float **s1, const float **s2)
{
    *s1 = *s2 = nullptr;
    if (!slope) return AMS_OK;
    if (mlp->dtype == AMS_BF16 && !(use_stream_k(mlp) && use_tail_bf16(mlp))) return AMS_ERR_DTYPE;
    for (int l = 0; l < mlp->n_layers - 1; ++l)
        if (!slope[l]) return AMS_ERR_NULL;
    *s1 = slope[0];
    if (mlp->n_layers == 3) *s2 = slope[1];
    return AMS_OK;
}

extern "C" ams_status ams_embed_fwd(const ams_mlp *mlp, const void *T, int64_t n_rows,
                                    const int32_t *uniq, const int32_t *n_uniq, int32_t cap,
                                    const void *W1, const float *b1, const void *W2,
                                    const float *b2, const void *W3, const float *b3,
                                    const float *const *slope, void *H1_save, float *H2_save, float *E,
                                    void *ws, size_t ws_bytes, void *stream)
{
    if (!mlp) return AMS_ERR_NULL;
    if (mlp->dtype != AMS_F32 && mlp->dtype != AMS_BF16 && mlp->dtype != AMS_F32_X3) return AMS_ERR_DTYPE;
    if (!mlp_ok(mlp)) return AMS_ERR_DIMS;
    if (cap < 0 || n_rows < 0) return AMS_ERR_SIZE;
    const int L = mlp->n_layers;
    if (!T || !uniq || !n_uniq || !W1 || !b1 || !W2 || !b2 || !E) return AMS_ERR_NULL;
    if (L == 3 && (!W3 || !b3)) return AMS_ERR_NULL;
    const float *s1, *s2;
    {
        const ams_status ps = prelu_slopes(mlp, slope, &s1, &s2);
        if (ps != AMS_OK) return ps;
    }
    const bool pr = s1 != nullptr;
    if (cap == 0) return AMS_OK;
    const int F = mlp->dims[0], H = mlp->dims[1], D = mlp->dims[L];
    const int M = (L == 3) ? mlp->dims[2] : D;
    const bool bf = mlp->dtype == AMS_BF16;
    const bool h1_in_ws = bf || !H1_save;
    const bool sk = use_stream_k(mlp);
    const int G = sk ? sk_workers() : 0;
    const size_t h1_bytes = al256((size_t)cap * H * 4);
    const bool x3 = sk && mlp->dtype == AMS_F32_X3;
    const size_t pbuf_bytes = sk ? al256((size_t)G * 2 * (bf ? Sk<uint16_t>::TILE : Sk<float>::TILE) * 4) : 0;
    const size_t need = h1_bytes + pbuf_bytes + (x3 ? al256((size_t)3 * F * H * 2) : 0);
    if ((h1_in_ws || sk) && (!ws || ws_bytes < need)) return AMS_ERR_WORKSPACE;
    hipStream_t st = (hipStream_t)stream;
    float *H1f = h1_in_ws ? (float *)ws : (float *)H1_save;
    // bf16 stream-K path: H1 as a pair of bf16 arrays in the workspace's H1
    // region, the low part first, then the high part unless the caller keeps
    // it (H1_save, read by the backward)
    uint16_t *h1lo = (uint16_t *)ws;
    uint16_t *h1b = H1_save ? (uint16_t *)H1_save : (uint16_t *)ws + (size_t)cap * H;
    float *pbuf = (float *)((char *)ws + h1_bytes);

    const int n_mt = (cap + 63) / 64;
    const int NT = (H % 128 == 0) ? 128 : 64;
    const int grid = ((n_mt + 7) / 8) * 8 * (H / NT);
    if (x3) {
        // W1's three bf16 parts, then the split stream-K product
        uint16_t *w1p = (uint16_t *)((char *)ws + h1_bytes + pbuf_bytes);
        const int64_t nw = (int64_t)H * F;
        const int sg = (int)std::min<int64_t>((nw / 8 + kThreads - 1) / kThreads, 2048);
        AMS_LAUNCH("split3_w1", st, split3_k<<<sg, kThreads, 0, st>>>((const float *)W1, nw, w1p));
        AMS_LAUNCH("l1sk_x3", st, l1sk_x3<<<G, kSkThreads, 0, st>>>((const float *)T, n_rows, F, uniq, n_uniq, cap,
                                                                   (const float *)W1, w1p, b1, H, G, H1f, pbuf,
                                                                   (int)pr));
    } else if (sk && !bf) {
        AMS_LAUNCH("l1sk_f32", st, l1sk<float><<<G, kSkThreads, 0, st>>>((const float *)T, n_rows, F, uniq, n_uniq, cap,
                                                                      (const float *)W1, b1, H, G, H1f, nullptr, nullptr, pbuf,
                                                                      (int)pr));
    } else if (sk && use_row_split(mlp, cap)) {
        AMS_LAUNCH("l1rs_bf16", st, l1rs_bf16<<<G, rs::kThreads, 0, st>>>((const uint16_t *)T, n_rows, uniq, n_uniq,
                                                                        cap, (const uint16_t *)W1, b1, G, h1b, h1lo,
                                                                        (int)pr));
        pbuf = nullptr;
    } else if (sk) {
        AMS_LAUNCH("l1sk_bf16", st, l1sk<uint16_t><<<G, kSkThreads, 0, st>>>((const uint16_t *)T, n_rows, F, uniq, n_uniq,
                                                                           cap, (const uint16_t *)W1, b1, H, G, nullptr,
                                                                           h1b, h1lo, pbuf, (int)pr));
    } else if (!bf) {
        if (NT == 128)
            AMS_LAUNCH("l1_fwd_f32", st, l1_fwd_f32<128><<<grid, kThreads, 0, st>>>((const float *)T, n_rows, F, uniq, n_uniq, cap, n_mt,
                                                       (const float *)W1, b1, H, H1f, (int)pr));
        else
            AMS_LAUNCH("l1_fwd_f32", st, l1_fwd_f32<64><<<grid, kThreads, 0, st>>>((const float *)T, n_rows, F, uniq, n_uniq, cap, n_mt,
                                                      (const float *)W1, b1, H, H1f, (int)pr));
    } else {
        if (NT == 128)
            AMS_LAUNCH("l1_fwd_bf16", st, l1_fwd_bf16<128><<<grid, kThreads, 0, st>>>((const uint16_t *)T, n_rows, F, uniq, n_uniq,
                                                        cap, n_mt, (const uint16_t *)W1, b1, H, H1f,
                                                        (uint16_t *)H1_save));
        else
            AMS_LAUNCH("l1_fwd_bf16", st, l1_fwd_bf16<64><<<grid, kThreads, 0, st>>>((const uint16_t *)T, n_rows, F, uniq, n_uniq,
                                                       cap, n_mt, (const uint16_t *)W1, b1, H, H1f,
                                                       (uint16_t *)H1_save));
    }
    if (sk && bf && pbuf) {
        // after the stream-K layer: a block per 32-row chunk, a wave per K
        // quarter (split tiles finished on the way), two blocks per CU
        int tg = (cap + 31) / 32;
        if (tg > 2 * G) tg = 2 * G;
#define TFQ_LAUNCH(LL, PRV)                                                                                \
    AMS_LAUNCH("tail_fwd_bf16", st, (tail_fwd_bf16_q<LL, PRV><<<tg, kThreads, 0, st>>>(                      \
                                        h1b, h1lo, pbuf, F, G, b1, uniq, n_rows, M, D, (const uint16_t *)W2, \
                                        b2, LL == 3 ? (const uint16_t *)W3 : nullptr, LL == 3 ? b3 : nullptr, \
                                        mlp->final_relu, n_uniq, cap, H2_save, E, s1, s2)))
        if (L == 3 && pr) TFQ_LAUNCH(3, true);
        else if (L == 3) TFQ_LAUNCH(3, false);
        else if (pr) TFQ_LAUNCH(2, true);
        else TFQ_LAUNCH(2, false);
#undef TFQ_LAUNCH
        return ams_launch_status();
    }
    if (sk && bf) {
        // after the row-split layer (whole tiles): two resident blocks per CU
        // stage W2 once and loop over chunks, a wave per chunk
        int tg = (cap + 4 * 32 - 1) / (4 * 32);
        if (tg > 2 * G) tg = 2 * G;
#define TFB_LAUNCH(LL, PRV)                                                                                \
    AMS_LAUNCH("tail_fwd_bf16", st, (tail_fwd_bf16<LL, PRV><<<tg, kThreads, 0, st>>>(                        \
                                        h1b, h1lo, M, D, (const uint16_t *)W2,                               \
                                        b2, LL == 3 ? (const uint16_t *)W3 : nullptr, LL == 3 ? b3 : nullptr, \
                                        mlp->final_relu, n_uniq, cap, H2_save, E, s1, s2)))
        if (L == 3 && pr) TFB_LAUNCH(3, true);
        else if (L == 3) TFB_LAUNCH(3, false);
        else if (pr) TFB_LAUNCH(2, true);
        else TFB_LAUNCH(2, false);
#undef TFB_LAUNCH
        return ams_launch_status();
    }
    // K per stream-K stage, which fixes the plan the tail reads the partial
    // tiles by (the bf16 stream-K path returned above)
    const int skk = !sk ? 0 : x3 ? X3::BK : sk_bk<float>();
    // at most the two blocks per CU that fit at once (LDS); the kernel loops
    // over chunks, and blocks sized for cap but past n_u would each still
    // cost a dispatch (with 1024 blocks for ~400 chunks the launch took
    // 34 us while each wave lived 6 us)
    int tg = (cap + kTailRows - 1) / kTailRows;
    if (tg > 2 * sk_workers()) tg = 2 * sk_workers();
#define TF_LAUNCH(LL, PRV)                                                                                 \
    AMS_LAUNCH("tail_fwd", st, (tail_fwd<LL, PRV><<<tg, kThreads, 0, st>>>(                                   \
                                   H1f, H, M, D, W2, b2, W3, b3, bf, mlp->final_relu, n_uniq, cap, H2_save, E, \
                                   skk, F, G, pbuf, bf ? (uint16_t *)H1_save : nullptr, b1, uniq, n_rows, s1, s2)))
    if (L == 3 && pr) TF_LAUNCH(3, true);
    else if (L == 3) TF_LAUNCH(3, false);
    else if (pr) TF_LAUNCH(2, true);
    else TF_LAUNCH(2, false);
#undef TF_LAUNCH
    return ams_launch_status();
}

extern "C" ams_status ams_embed_bwd(const ams_mlp *mlp, const void *T, int64_t n_rows,
                                    const int32_t *uniq, const int32_t *n_uniq, int32_t cap,
                                    const void *W1, const void *W2, const void *W3,
                                    const float *const *slope, const void *H1_save, const float *H2_save,
                                    const float *E_fwd, const float *dE, float *dW1, float *db1,
                                    float *dW2, float *db2, float *dW3, float *db3, float *const *dslope,
                                    void *ws, size_t ws_bytes, void *stream)
{
    (void)W1;
    if (!mlp) return AMS_ERR_NULL;
    if (mlp->dtype != AMS_F32 && mlp->dtype != AMS_BF16 && mlp->dtype != AMS_F32_X3) return AMS_ERR_DTYPE;
    if (!mlp_ok(mlp)) return AMS_ERR_DIMS;
    if (cap < 0 || n_rows < 0) return AMS_ERR_SIZE;
    const int L = mlp->n_layers;
    if (!T || !uniq || !n_uniq || !W2 || !H1_save || !dE || !dW1 || !db1 || !dW2 || !db2)
        return AMS_ERR_NULL;
    if (L == 3 && (!W3 || !H2_save || !dW3 || !db3)) return AMS_ERR_NULL;
    if (mlp->final_relu && !E_fwd) return AMS_ERR_NULL;
    const float *s1, *s2;
    {
        const ams_status ps = prelu_slopes(mlp, slope, &s1, &s2);
        if (ps != AMS_OK) return ps;
    }
    const bool pr = s1 != nullptr;
    float *ds1 = (pr && dslope) ? dslope[0] : nullptr;
    float *ds2 = (pr && dslope && L == 3) ? dslope[1] : nullptr;
    const BwdPlan p = plan_bwd(mlp, cap);
    if (!ws || ws_bytes < p.total) return AMS_ERR_WORKSPACE;
    const int F = mlp->dims[0], H = mlp->dims[1], D = mlp->dims[L];
    const int M = (L == 3) ? mlp->dims[2] : D;
    const bool bf = mlp->dtype == AMS_BF16;
    hipStream_t st = (hipStream_t)stream;
    char *w = (char *)ws;
    float *zero = (float *)(w + p.off_zero);
    void *dz1 = w + p.off_dz1;
    float *tail = (float *)(w + p.off_tail);
    float *dw1p = (float *)(w + p.off_dw1);
    const int PS = tail_part_size(mlp);

#define TB_LAUNCH(LL, TW, TH, PRV)                                                                     \
    if (D <= 16)                                                                                        \
        AMS_LAUNCH("tail_bwd", st, (tail_bwd<LL, 8, TW, TH, PRV><<<kTailBlocks, kTbThreads, 0, st>>>(    \
                                       (const TH *)H1_save, H2_save, E_fwd, dE, (const TW *)W2, (const TW *)W3, \
                                       H, M, D, mlp->final_relu, n_uniq, cap, (TH *)dz1, tail, PS, zero, \
                                       F > H ? F : H, s1, s2)));                                         \
    else                                                                                                \
    AMS_LAUNCH("tail_bwd", st, (tail_bwd<LL, 16, TW, TH, PRV><<<kTailBlocks, kTbThreads, 0, st>>>(           \
                                   (const TH *)H1_save, H2_save, E_fwd, dE, (const TW *)W2, (const TW *)W3, \
                                   H, M, D, mlp->final_relu, n_uniq, cap, (TH *)dz1, tail, PS, zero,     \
                                   F > H ? F : H, s1, s2)))
    const int TG = tail_blocks(mlp);
    if (use_tail_bf16(mlp)) {
#define TBF_LAUNCH(LL, DM, PRV)                                                                         \
    AMS_LAUNCH("tail_bwd_bf16", st, (tail_bwd_bf16<LL, DM, PRV><<<TG, kThreads, 0, st>>>(                \
                                        (const uint16_t *)H1_save, H2_save, E_fwd, dE, (const uint16_t *)W2, \
                                        (const uint16_t *)W3, M, D, mlp->final_relu, n_uniq, cap,          \
                                        (uint16_t *)dz1, tail, PS, zero, F > H ? F : H, s1, s2)))
        if (pr) {
            if (L == 3 && D <= 16) TBF_LAUNCH(3, 16, true);
            else if (L == 3) TBF_LAUNCH(3, 32, true);
            else if (D <= 16) TBF_LAUNCH(2, 16, true);
            else TBF_LAUNCH(2, 32, true);
        } else {
            if (L == 3 && D <= 16) TBF_LAUNCH(3, 16, false);
            else if (L == 3) TBF_LAUNCH(3, 32, false);
            else if (D <= 16) TBF_LAUNCH(2, 16, false);
            else TBF_LAUNCH(2, 32, false);
        }
#undef TBF_LAUNCH
    } else if (L == 3 && bf) {
        TB_LAUNCH(3, uint16_t, uint16_t, false);
    } else if (L == 3 && pr) {
        TB_LAUNCH(3, float, float, true);
    } else if (L == 3) {
        TB_LAUNCH(3, float, float, false);
    } else if (bf) {
        TB_LAUNCH(2, uint16_t, uint16_t, false);
    } else if (pr) {
        TB_LAUNCH(2, float, float, true);
    } else {
        TB_LAUNCH(2, float, float, false);
    }
#undef TB_LAUNCH

    const int bm = (H % 128 == 0) ? 128 : 64;
    const int nmt = H / bm, outer = (F / 64) * p.kc;
    const int grid = ((outer + 7) / 8) * 8 * nmt;
    if (use_dw_ring(mlp)) {
        const int grid8 = ((p.kc + 7) / 8) * 8 * (F / DwRing::BN);
        AMS_LAUNCH("dw1_part_f32", st, dw1_part_f32<<<grid8, kDwThreads, 0, st>>>((const float *)T, n_rows, F, uniq, n_uniq, cap,
                                                   (const float *)dz1, H, p.kc, zero, dw1p));
    } else if (use_dw_tr(mlp)) {
        const int bn = dwtr_bn(F, cap);
        const int gtr = ((p.kc + 7) / 8) * 8 * (F / bn);
        if (bn == 256)          // (use_dw_tr: H = 256)
            AMS_LAUNCH("dw1_rs_bf16", st, dw1_rs_bf16<<<gtr, dwr::kThreads, 0, st>>>(
                                              (const uint16_t *)T, n_rows, F, uniq, n_uniq, cap, (const uint16_t *)dz1,
                                              p.kc, dw1p));
        else
            AMS_LAUNCH("dw1_part_bf16", st, dw1_part_bf16<128><<<gtr, DwTr::WAVES * AMS_WAVE, 0, st>>>(
                                                (const uint16_t *)T, n_rows, F, uniq, n_uniq, cap, (const uint16_t *)dz1,
                                                p.kc, zero, dw1p));
    } else if (!bf) {
        if (bm == 128)
            AMS_LAUNCH("dw1_part", st, dw1_part<128, float><<<grid, kThreads, 0, st>>>((const float *)T, n_rows, F, uniq, n_uniq, cap,
                                                             (const float *)dz1, H, p.kc, dw1p));
        else
            AMS_LAUNCH("dw1_part", st, dw1_part<64, float><<<grid, kThreads, 0, st>>>((const float *)T, n_rows, F, uniq, n_uniq, cap,
                                                            (const float *)dz1, H, p.kc, dw1p));
    } else {
        if (bm == 128)
            AMS_LAUNCH("dw1_part", st, dw1_part<128, uint16_t><<<grid, kThreads, 0, st>>>((const uint16_t *)T, n_rows, F, uniq,
                                                                n_uniq, cap, (const uint16_t *)dz1, H, p.kc,
                                                                dw1p));
        else
            AMS_LAUNCH("dw1_part", st, dw1_part<64, uint16_t><<<grid, kThreads, 0, st>>>((const uint16_t *)T, n_rows, F, uniq,
                                                               n_uniq, cap, (const uint16_t *)dz1, H, p.kc,
                                                               dw1p));
    }
    // the dW1 partials and the tail's partials summed by one launch (four
    // dW1 elements per thread as float4 measured twice as slow: 21 vs 10 us)
    const size_t nw = (size_t)H * F;
    const int n_dw = (int)((nw + kRedThreads - 1) / kRedThreads);
    AMS_LAUNCH("bwd_reduce", st, bwd_reduce<<<n_dw + (PS + 63) / 64, kRedThreads, 0, st>>>(
                                     dw1p, p.kc, nw, dW1, n_dw, tail, TG, PS, L, H, M, D, dW2, db2, dW3, db3, db1, ds1,
                                     ds2, n_uniq, cap));
    return ams_launch_status();
}
