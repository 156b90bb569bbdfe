// peaks.hip -- achievable-peak probes of the GPU the library runs on: HBM
// copy and read bandwidth, the bandwidth of gathering table rows in the
// order the first-layer kernels visit them, and the MFMA rate on operands
// read from memory.  They compute nothing of the method; bench.py --peaks
// times them to put the kernels' rates beside what the part delivers (the
// vendor peaks stay the reference the roofline fractions use).
#include "ams_device.h"

namespace {

constexpr int kThreads = 256;

typedef float v16f __attribute__((ext_vector_type(16)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

// dst = src, 16 bytes per thread and step, grid-stride.
__global__ __launch_bounds__(kThreads) void peak_copy_k(const uint4 *__restrict__ src, uint4 *__restrict__ dst,
                                                        int64_t n)
{
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n; i += (int64_t)gridDim.x * kThreads)
        dst[i] = src[i];
}

// Reads src (16 bytes per thread and step, four in flight) and writes one
// xor per thread, so no load can be dropped.
__global__ __launch_bounds__(kThreads) void peak_read_k(const uint4 *__restrict__ src, int64_t n,
                                                        uint32_t *__restrict__ out)
{
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    uint32_t x = 0;
    int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    for (; i + 3 * stride < n; i += 4 * stride) {
        const uint4 a = src[i], b = src[i + stride], c = src[i + 2 * stride], d = src[i + 3 * stride];
        x ^= a.x ^ a.y ^ a.z ^ a.w ^ b.x ^ b.y ^ b.z ^ b.w ^ c.x ^ c.y ^ c.z ^ c.w ^ d.x ^ d.y ^ d.z ^ d.w;
    }
    for (; i < n; i += stride) {
        const uint4 a = src[i];
        x ^= a.x ^ a.y ^ a.z ^ a.w;
    }
    out[(int64_t)blockIdx.x * kThreads + threadIdx.x] = x;
}

// Gathers of 8192-byte table rows rows[0..n) the way the bf16 first layer
// meets them: 512-thread blocks, each a contiguous range of the list in
// tiles of 256 rows, a tile in 64 stages of 128 bytes per row (32 KB per
// stage), loads 3 stages ahead, one xor per thread kept so no load is
// dropped.  A row index outside [0, n_table) reads row 0.
namespace pg {
constexpr int kBlk = 512, kRowBytes = 8192, kStage = 128, kStages = kRowBytes / kStage, kTileRows = 256;
constexpr int kAhead = 3;
}

// Register loads (compiler-visible, so its own waits are exact), 4 per lane
// and stage.  ORD 0: lane (r, h) of a wave takes 16-byte pieces 4 h .. 4 h + 3
// of its row r (the MFMA operand layout: every load touches 32 rows);
// ORD 1: load i of a wave covers 8 whole 128-byte lines (8 rows).  NT: the
// non-temporal hint.  The empty asm per stage takes the stage's values after
// the loads of the stages ahead are issued.
template <int ORD, int NT>
__global__ __launch_bounds__(pg::kBlk) void peak_gather_reg_k(const char *__restrict__ T, int64_t n_table,
                                                                  const int32_t *__restrict__ rows, int n,
                                                                  uint32_t *__restrict__ out)
{
    using namespace pg;
    const int lane = ams_lane(), wave = threadIdx.x / AMS_WAVE;
    const int r0 = (int)((int64_t)n * blockIdx.x / gridDim.x), r1 = (int)((int64_t)n * (blockIdx.x + 1) / gridDim.x);
    uint4 x = make_uint4(0, 0, 0, 0);
    for (int m0 = r0; m0 < r1; m0 += kTileRows) {
        const char *p[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int row = ORD == 0 ? (lane & 31) : 8 * i + (lane >> 3);
            const int off = ORD == 0 ? 16 * (4 * (lane >> 5) + i) : 16 * (lane & 7);
            const int r = m0 + 32 * wave + row;
            int id = rows[r < r1 ? r : r0];
            if (id < 0 || (int64_t)id >= n_table) id = 0;
            p[i] = T + (size_t)id * kRowBytes + off;
        }
        typedef unsigned int u4 __attribute__((ext_vector_type(4)));
        u4 v[kAhead + 1][4];
        auto ld = [&](int st, u4 (&d)[4]) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const u4 *q = (const u4 *)(p[i] + st * kStage);
                d[i] = NT ? __builtin_nontemporal_load(q) : *q;
            }
        };
#pragma unroll
        for (int st = 0; st < kAhead; ++st) ld(st, v[st]);
#pragma unroll
        for (int st = 0; st < kStages; ++st) {
            if (st + kAhead < kStages) ld(st + kAhead, v[(st + kAhead) % (kAhead + 1)]);
            u4 (&c)[4] = v[st % (kAhead + 1)];
            asm volatile("" : "+v"(c[0]), "+v"(c[1]), "+v"(c[2]), "+v"(c[3]));
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                x.x ^= c[i].x;
                x.y ^= c[i].y;
                x.z ^= c[i].z;
                x.w ^= c[i].w;
            }
        }
    }
    out[(size_t)blockIdx.x * kBlk + threadIdx.x] = x.x ^ x.y ^ x.z ^ x.w;
}

// 16-byte DMA of every lane into LDS at lds + 16 lane (no register is written).
template <int NT>
__device__ __forceinline__ void pg_dma(const char *src, uint32_t lds)
{
    if (NT)
        asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off nt" ::"s"(lds), "v"(src)
                     : "memory", "m0");
    else
        asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off" ::"s"(lds), "v"(src)
                     : "memory", "m0");
}

// Whole-line DMA into a 3-slot LDS ring (non-temporal, 2 stages ahead), one
// barrier per stage.  WSTREAM: each stage also DMAs a 32 KB slice of W (256
// rows of 8192 bytes, an L2-resident 2 MB array) into a 2-slot ring, one
// stage ahead, as the first layer moves its weight slices.
template <int WSTREAM>
__global__ __launch_bounds__(pg::kBlk) void peak_gather_dma_k(const char *__restrict__ T, int64_t n_table,
                                                                  const int32_t *__restrict__ rows, int n,
                                                                  const char *__restrict__ W,
                                                                  uint32_t *__restrict__ out)
{
    using namespace pg;
    constexpr int SLOT = kTileRows * kStage;                   // 32 KB
    __shared__ __attribute__((aligned(1024))) char ring[(3 + 2 * WSTREAM) * SLOT];
    const int lane = ams_lane(), wave = __builtin_amdgcn_readfirstlane(threadIdx.x / AMS_WAVE);
    const int r0 = (int)((int64_t)n * blockIdx.x / gridDim.x), r1 = (int)((int64_t)n * (blockIdx.x + 1) / gridDim.x);
    const uint32_t xb = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)ring) + 4 * wave * 1024;
    const uint32_t wb = xb + 3 * SLOT;
    uint32_t x = 0;
    for (int m0 = r0; m0 < r1; m0 += kTileRows) {
        // DMA q of this wave: 8 rows (32 wave + 8 q ..), whole lines
        const char *p[4], *w[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int r = m0 + 32 * wave + 8 * q + (lane >> 3);
            int id = rows[r < r1 ? r : r0];
            if (id < 0 || (int64_t)id >= n_table) id = 0;
            p[q] = T + (size_t)id * kRowBytes + 16 * (lane & 7);
            w[q] = WSTREAM ? W + (size_t)(32 * wave + 8 * q + (lane >> 3)) * kRowBytes + 16 * (lane & 7) : nullptr;
        }
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        // prologue: rows of stages 0, 1; W of stage 0 between them (the order
        // a stage issues: W of the next stage, then rows two ahead).  The
        // pointers advance by one stage per issue (opaque to the compiler, so
        // it does not precompute every stage's addresses)
        auto adv = [](const char *&q, int by) {
            q += by;
            asm volatile("" : "+v"(q));
        };
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            pg_dma<1>(p[q], xb + q * 1024);
            adv(p[q], kStage);
        }
        if (WSTREAM) {
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                pg_dma<0>(w[q], wb + q * 1024);
                adv(w[q], kStage);
            }
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            pg_dma<1>(p[q], xb + SLOT + q * 1024);
            adv(p[q], kStage);
        }
#pragma unroll
        for (int st = 0; st < kStages; ++st) {
            // this stage's rows (and W) landed: only the next stage's rows may be in flight
            asm volatile("s_waitcnt vmcnt(4) lgkmcnt(0)" ::: "memory");
            __builtin_amdgcn_s_barrier();
            if (WSTREAM) {                          // W of stage st + 1 (the last one again past the end)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    pg_dma<0>(w[q], wb + ((st + 1) & 1) * SLOT + q * 1024);
                    if (st + 2 < kStages) adv(w[q], kStage);
                }
            }
#pragma unroll
            for (int q = 0; q < 4; ++q) {           // rows of stage st + 2 (the last one again past the end)
                pg_dma<1>(p[q], xb + ((st + 2) % 3) * SLOT + q * 1024);
                if (st + 3 < kStages) adv(p[q], kStage);
            }
            x ^= *(const uint32_t *)(ring + (st % 3) * SLOT + threadIdx.x * 16);
        }
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __builtin_amdgcn_s_barrier();
    }
    out[(size_t)blockIdx.x * kBlk + threadIdx.x] = x;
}

// MFMA rate on operands read from memory: each wave reads its own 16-byte
// operands (a[lane], b[lane], 4 each), then runs `iters` rounds of 16
// independent products, 8 accumulator blocks x 2 k steps; one float per
// thread is written.  bf16: v_mfma_f32_32x32x16_bf16 (32768 flops each);
// f32: v_mfma_f32_32x32x2_f32 (4096 flops each).
template <bool BF16>
__global__ __launch_bounds__(kThreads) void peak_mfma_k(const uint4 *__restrict__ ops, int iters,
                                                        float *__restrict__ out)
{
    const int lane = ams_lane();
    const uint4 *o = ops + ((int64_t)(blockIdx.x * (kThreads / AMS_WAVE) + threadIdx.x / AMS_WAVE) % 64) * 512;
    uint4 a[2], b[2];
#pragma unroll
    for (int k = 0; k < 2; ++k) {
        a[k] = o[k * 128 + lane];
        b[k] = o[k * 128 + 64 + lane];
    }
    v16f acc[8];
#pragma unroll
    for (int nb = 0; nb < 8; ++nb) acc[nb] = (v16f){};
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int k = 0; k < 2; ++k)
#pragma unroll
            for (int nb = 0; nb < 8; ++nb) {
                if constexpr (BF16) {
                    acc[nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a[k]),
                                                                       __builtin_bit_cast(bf16x8, b[k]), acc[nb], 0,
                                                                       0, 0);
                } else {
                    acc[nb] = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a[k].x ^ nb),
                                                                    __uint_as_float(b[k].y), acc[nb], 0, 0, 0);
                }
            }
    }
    float s = 0.f;
#pragma unroll
    for (int nb = 0; nb < 8; ++nb)
#pragma unroll
        for (int j = 0; j < 16; ++j) s += acc[nb][j];
    out[(int64_t)blockIdx.x * kThreads + threadIdx.x] = s;
}

}  // namespace

extern "C" ams_status ams_peak_copy(const void *src, void *dst, int64_t bytes, int32_t blocks, void *stream)
{
    if (bytes < 0 || bytes % 16 || blocks < 1) return AMS_ERR_SIZE;
    if (bytes == 0) return AMS_OK;
    if (!src || !dst) return AMS_ERR_NULL;
    hipStream_t st = (hipStream_t)stream;
    AMS_LAUNCH("peak_copy", st, peak_copy_k<<<blocks, kThreads, 0, st>>>((const uint4 *)src, (uint4 *)dst, bytes / 16));
    return ams_launch_status();
}

extern "C" ams_status ams_peak_read(const void *src, int64_t bytes, int32_t blocks, uint32_t *out, void *stream)
{
    if (bytes < 0 || bytes % 16 || blocks < 1) return AMS_ERR_SIZE;
    if (!src || !out) return AMS_ERR_NULL;
    hipStream_t st = (hipStream_t)stream;
    AMS_LAUNCH("peak_read", st, peak_read_k<<<blocks, kThreads, 0, st>>>((const uint4 *)src, bytes / 16, out));
    return ams_launch_status();
}

extern "C" ams_status ams_peak_gather(const void *T, int64_t n_table, int32_t row_bytes, const int32_t *rows,
                                      int32_t n, int32_t pattern, const void *W, int32_t blocks, uint32_t *out,
                                      void *stream)
{
    if (n_table < 1 || n < 0 || blocks < 1 || row_bytes != pg::kRowBytes) return AMS_ERR_SIZE;
    if (pattern < 0 || pattern > 4) return AMS_ERR_MODE;
    if (n == 0) return AMS_OK;
    if (!T || !rows || !out || (pattern == 4 && !W)) return AMS_ERR_NULL;
    hipStream_t st = (hipStream_t)stream;
    const char *t = (const char *)T;
    switch (pattern) {
    case 0: AMS_LAUNCH("peak_gather", st, peak_gather_reg_k<0, 0><<<blocks, pg::kBlk, 0, st>>>(t, n_table, rows, n, out)); break;
    case 1: AMS_LAUNCH("peak_gather", st, peak_gather_reg_k<1, 0><<<blocks, pg::kBlk, 0, st>>>(t, n_table, rows, n, out)); break;
    case 2: AMS_LAUNCH("peak_gather", st, peak_gather_reg_k<1, 1><<<blocks, pg::kBlk, 0, st>>>(t, n_table, rows, n, out)); break;
    case 3: AMS_LAUNCH("peak_gather", st, peak_gather_dma_k<0><<<blocks, pg::kBlk, 0, st>>>(t, n_table, rows, n, nullptr, out)); break;
    default: AMS_LAUNCH("peak_gather", st, peak_gather_dma_k<1><<<blocks, pg::kBlk, 0, st>>>(t, n_table, rows, n, (const char *)W, out)); break;
    }
    return ams_launch_status();
}

extern "C" ams_status ams_peak_mfma(int32_t dtype, const void *ops, int32_t iters, int32_t blocks, float *out,
                                    void *stream)
{
    if (iters < 1 || blocks < 1) return AMS_ERR_SIZE;
    if (dtype != AMS_F32 && dtype != AMS_BF16) return AMS_ERR_DTYPE;
    if (!ops || !out) return AMS_ERR_NULL;
    hipStream_t st = (hipStream_t)stream;
    if (dtype == AMS_BF16)
        AMS_LAUNCH("peak_mfma_bf16", st, peak_mfma_k<true><<<blocks, kThreads, 0, st>>>((const uint4 *)ops, iters, out));
    else
        AMS_LAUNCH("peak_mfma_f32", st, peak_mfma_k<false><<<blocks, kThreads, 0, st>>>((const uint4 *)ops, iters, out));
    return ams_launch_status();
}
