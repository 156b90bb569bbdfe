// ams_device.h -- device-side helpers shared by the libams kernels (gfx950,
// wave64).  Internal to the library; the public contract is include/ams.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/ams.h"

#define AMS_WAVE 64

#define AMS_HIP_TRY(expr)                                   \
    do {                                                    \
        if ((expr) != hipSuccess) return AMS_ERR_HIP;       \
    } while (0)

// Per-kernel timing (ams_timing_enable): when on, every launch is bracketed by
// a pair of HIP events on the launching stream, read back by ams_timing_read.
extern int ams_timing_flag;
void ams_timing_begin(const char *name, hipStream_t st);
void ams_timing_end(hipStream_t st);

#define AMS_LAUNCH(name, st, ...)                                    \
    do {                                                             \
        const bool ams_timed_ = __atomic_load_n(&ams_timing_flag, __ATOMIC_RELAXED) != 0; \
        if (ams_timed_) ams_timing_begin(name, st);                  \
        __VA_ARGS__;                                                 \
        if (ams_timed_) ams_timing_end(st);                          \
    } while (0)

// Launch check: a failed enqueue is reported as AMS_ERR_HIP.
static inline ams_status ams_launch_status()
{
    return hipGetLastError() == hipSuccess ? AMS_OK : AMS_ERR_HIP;
}

__device__ __forceinline__ int ams_lane() { return (int)(threadIdx.x & (AMS_WAVE - 1)); }

__device__ __forceinline__ uint64_t ams_ballot(bool p) { return (uint64_t)__ballot(p); }

__device__ __forceinline__ uint64_t ams_lanemask_lt()
{
    const int l = ams_lane();
    return l == 0 ? 0ull : (~0ull >> (64 - l));
}

// Inclusive scan of an int over the 64 lanes of a wave (fixed order).
__device__ __forceinline__ int ams_wave_incl_scan(int v)
{
    const int l = ams_lane();
#pragma unroll
    for (int o = 1; o < AMS_WAVE; o <<= 1) {
        int t = __shfl_up(v, o, AMS_WAVE);
        if (l >= o) v += t;
    }
    return v;
}

// Butterfly sum over the wave: every lane ends with the same value, and the
// association order depends only on the lane layout (deterministic).
__device__ __forceinline__ float ams_wave_sum(float v)
{
#pragma unroll
    for (int o = AMS_WAVE / 2; o > 0; o >>= 1) v += __shfl_xor(v, o, AMS_WAVE);
    return v;
}

__device__ __forceinline__ float ams_wave_max(float v)
{
#pragma unroll
    for (int o = AMS_WAVE / 2; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, AMS_WAVE));
    return v;
}

// bf16 <-> fp32 (round to nearest even; NaN kept quiet).
__device__ __forceinline__ float ams_bf16_to_f32(uint16_t b)
{
    return __uint_as_float(((uint32_t)b) << 16);
}

__device__ __forceinline__ uint16_t ams_f32_to_bf16(float f)
{
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40);
    u += 0x7fffu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

// The SUM aggregator's backward (ams_pool_bwd, AMS_POOL_SUM) with a second
// upstream gradient of the ads: the ad of sample i contributes dA[i] + dA2[i]
// (dA or dA2 NULL: nothing from it).  Shared by the ID-bag backward.
ams_status pool_bwd_sum_ads(int32_t B, int32_t D, const int32_t *seg_off, int64_t n_beh, const int32_t *inv,
                            const int32_t *occ_perm, const int32_t *uniq_off, int32_t n_uniq_cap, const float *dU,
                            const float *dA, const float *dA2, float *dE, void *ws, size_t ws_bytes, void *stream);
