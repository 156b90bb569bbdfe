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

// Gather of table rows rows[0..n) (row_bytes each) in the first layer's
// order: each block takes a contiguous range of the list in tiles of `tile`
// rows and visits a tile in stages of `chunk` bytes per row (stage s reads
// bytes s*chunk .. of every row of the tile), `chunk` contiguous bytes per
// row and stage, 16 bytes per thread and load, eight loads per thread in
// flight.  chunk == row_bytes visits each row whole.  A row index outside
// [0, n_table) is read as row 0.
__global__ __launch_bounds__(kThreads) void peak_gather_k(const uint4 *__restrict__ T, int64_t n_table,
                                                          int row_bytes, const int32_t *__restrict__ rows, int n,
                                                          int tile, int chunk, uint32_t *__restrict__ out)
{
    const int r0 = (int)((int64_t)n * blockIdx.x / gridDim.x), r1 = (int)((int64_t)n * (blockIdx.x + 1) / gridDim.x);
    const int per_row = chunk / 16;                 // 16-byte pieces of a row per stage
    const int stages = row_bytes / chunk;
    const int64_t row_u4 = row_bytes / 16;
    uint32_t x = 0;
    for (int m0 = r0; m0 < r1; m0 += tile) {
        const int nr = min(tile, r1 - m0);
        const int pieces = nr * per_row;            // 16-byte loads of one stage
        for (int s = 0; s < stages; ++s) {
            for (int p0 = threadIdx.x; p0 < pieces; p0 += 8 * kThreads) {
                uint4 v[8];
#pragma unroll
                for (int u = 0; u < 8; ++u) {
                    const int p = p0 + u * kThreads;
                    if (p < pieces) {
                        int r = rows[m0 + p / per_row];
                        if (r < 0 || r >= n_table) r = 0;
                        v[u] = T[(int64_t)r * row_u4 + (int64_t)s * per_row + p % per_row];
                    } else {
                        v[u] = make_uint4(0, 0, 0, 0);
                    }
                }
#pragma unroll
                for (int u = 0; u < 8; ++u) x ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
            }
        }
    }
    out[(int64_t)blockIdx.x * kThreads + threadIdx.x] = x;
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
                                      int32_t n, int32_t tile, int32_t chunk, int32_t blocks, uint32_t *out,
                                      void *stream)
{
    if (n_table < 1 || n < 0 || tile < 1 || blocks < 1 || chunk < 16 || chunk % 16 || row_bytes % chunk)
        return AMS_ERR_SIZE;
    if (n == 0) return AMS_OK;
    if (!T || !rows || !out) return AMS_ERR_NULL;
    hipStream_t st = (hipStream_t)stream;
    AMS_LAUNCH("peak_gather", st, peak_gather_k<<<blocks, kThreads, 0, st>>>((const uint4 *)T, n_table, row_bytes,
                                                                               rows, n, tile, chunk, out));
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
