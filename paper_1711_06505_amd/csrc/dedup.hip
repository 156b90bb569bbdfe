// dedup.hip -- ams_dedup: the batch's image IDs reduced to one sorted set with
// inverse index and stable occurrence order (section 4.2: requests for the
// same image are processed once; Algorithm 1: an image's gradients are
// collected in one place).
//
// Method: a stable LSD radix sort of (ID, occurrence index) over the
// ceil(log2 n_ids) significant bits, at most 8 bits per pass, then head flags
// and an exclusive scan give the unique set, its CSR offsets and the inverse.
//
// Per radix pass three kernels run: a per-tile digit histogram, one exclusive
// scan over the digit-major [digit][tile] counts, and a scatter in which every
// wave ranks its keys with 64-lane ballots (lanes holding the same digit find
// each other bit by bit) and running per-wave digit counters in LDS.  Tiles,
// waves, rows and lanes are visited in index order, so the sort is stable and
// the result bit-exact.
#include "ams_device.h"

namespace {

constexpr int kThreads = 256;                 // 4 waves
constexpr int kRows = 8;                      // rows of 64 keys per wave
constexpr int kTile = kThreads * kRows;       // 2048 keys per tile
constexpr int kMaxBits = 8;
constexpr int kUniqItems = 8;                 // positions per thread, unique pass
constexpr int kUniqTile = kThreads * kUniqItems;
constexpr int kScanThreads = 1024;

__global__ void dd_init(int32_t *n_uniq, int32_t *dev_status, int32_t *uniq_off, int n_occ)
{
    if (threadIdx.x == 0 && blockIdx.x == 0) {
        *dev_status = AMS_OK;
        *n_uniq = 0;
        if (n_occ == 0) uniq_off[0] = 0;
    }
}

// Per-tile histogram of one digit; the first pass also range-checks the IDs.
__global__ __launch_bounds__(kThreads) void dd_hist(const uint32_t *__restrict__ keys, int n,
                                                    int shift, int bits, int32_t *__restrict__ hist,
                                                    int ntiles, uint32_t n_ids,
                                                    int32_t *__restrict__ dev_status, int check)
{
    __shared__ int h[1 << kMaxBits];
    const int t = threadIdx.x;
    const uint32_t mask = (1u << bits) - 1u;
    h[t] = 0;
    __syncthreads();
    const int base = blockIdx.x * kTile;
    bool bad = false;
    for (int i = t; i < kTile; i += kThreads) {
        const int idx = base + i;
        if (idx < n) {
            const uint32_t k = keys[idx];
            bad |= (k >= n_ids);
            atomicAdd(&h[(k >> shift) & mask], 1);
        }
    }
    if (check && bad) *dev_status = AMS_ERR_ID_RANGE;
    __syncthreads();
    if (t < (1 << bits)) hist[t * ntiles + blockIdx.x] = h[t];
}

// Exclusive scan of len ints in place by one workgroup; *total (optional)
// receives the sum.  Each thread owns one contiguous run.
__global__ __launch_bounds__(kScanThreads) void dd_scan(int32_t *__restrict__ a, int len,
                                                        int32_t *__restrict__ total)
{
    __shared__ int wsum[kScanThreads / AMS_WAVE];
    const int t = threadIdx.x;
    const int per = (len + kScanThreads - 1) / kScanThreads;
    const int lo = min(len, t * per), hi = min(len, lo + per);
    int s = 0;
    for (int i = lo; i < hi; ++i) s += a[i];
    const int incl = ams_wave_incl_scan(s);
    const int w = t / AMS_WAVE;
    if (ams_lane() == AMS_WAVE - 1) wsum[w] = incl;
    __syncthreads();
    if (t < AMS_WAVE) {
        int v = t < kScanThreads / AMS_WAVE ? wsum[t] : 0;
        int vi = ams_wave_incl_scan(v);
        if (t < kScanThreads / AMS_WAVE) wsum[t] = vi - v;   // exclusive per wave
        if (t == kScanThreads / AMS_WAVE - 1 && total) *total = vi;
    }
    __syncthreads();
    int run = wsum[w] + incl - s;
    for (int i = lo; i < hi; ++i) {
        const int v = a[i];
        a[i] = run;
        run += v;
    }
}

// Stable scatter of one radix pass.  vals_in == nullptr means the identity
// (occurrence index) for the first pass.
__global__ __launch_bounds__(kThreads) void dd_scatter(const uint32_t *__restrict__ kin,
                                                       const int32_t *__restrict__ vin,
                                                       uint32_t *__restrict__ kout,
                                                       int32_t *__restrict__ vout, int n, int shift,
                                                       int bits, const int32_t *__restrict__ offs,
                                                       int ntiles)
{
    __shared__ int cnt[kThreads / AMS_WAVE][1 << kMaxBits];
    __shared__ int woff[kThreads / AMS_WAVE][1 << kMaxBits];
    const int t = threadIdx.x, lane = ams_lane(), wave = t / AMS_WAVE;
    const uint32_t mask = (1u << bits) - 1u;
    for (int d = lane; d < (1 << kMaxBits); d += AMS_WAVE) cnt[wave][d] = 0;
    __syncthreads();

    const int base = blockIdx.x * kTile + wave * (kRows * AMS_WAVE);
    const uint64_t lt = ams_lanemask_lt();
    uint32_t key[kRows];
    int32_t val[kRows];
    int rank[kRows];
#pragma unroll
    for (int r = 0; r < kRows; ++r) {
        const int idx = base + r * AMS_WAVE + lane;
        const bool valid = idx < n;
        key[r] = valid ? kin[idx] : 0u;
        val[r] = valid ? (vin ? vin[idx] : idx) : 0;
        const uint32_t d = (key[r] >> shift) & mask;
        uint64_t peers = ams_ballot(valid);
        for (int b = 0; b < bits; ++b) {
            const bool bit = (d >> b) & 1u;
            const uint64_t bb = ams_ballot(bit);
            peers &= bit ? bb : ~bb;
        }
        const int below = __popcll(peers & lt);
        const int c = valid ? cnt[wave][d] : 0;
        rank[r] = c + below;
        // every lane of the wave has read its counter before the leader of
        // each digit group advances it (one wave, LDS ops in program order)
        __builtin_amdgcn_wave_barrier();
        if (valid && below == 0) cnt[wave][d] = c + __popcll(peers);
        __builtin_amdgcn_wave_barrier();
    }
    __syncthreads();
    if (t < (1 << bits)) {
        int run = offs[t * ntiles + blockIdx.x];
#pragma unroll
        for (int w = 0; w < kThreads / AMS_WAVE; ++w) {
            woff[w][t] = run;
            run += cnt[w][t];
        }
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kRows; ++r) {
        const int idx = base + r * AMS_WAVE + lane;
        if (idx < n) {
            const uint32_t d = (key[r] >> shift) & mask;
            const int pos = woff[wave][d] + rank[r];
            kout[pos] = key[r];
            vout[pos] = val[r];
        }
    }
}

// Head flags of the sorted keys, counted per tile.
__global__ __launch_bounds__(kThreads) void dd_head_count(const uint32_t *__restrict__ k, int n,
                                                          int32_t *__restrict__ bsum)
{
    __shared__ int ws[kThreads / AMS_WAVE];
    const int t = threadIdx.x;
    const int i0 = blockIdx.x * kUniqTile + t * kUniqItems;
    int c = 0;
#pragma unroll
    for (int q = 0; q < kUniqItems; ++q) {
        const int i = i0 + q;
        if (i < n) c += (i == 0 || k[i] != k[i - 1]) ? 1 : 0;
    }
    const int incl = ams_wave_incl_scan(c);
    if (ams_lane() == AMS_WAVE - 1) ws[t / AMS_WAVE] = incl;
    __syncthreads();
    if (t == 0) {
        int s = 0;
        for (int w = 0; w < kThreads / AMS_WAVE; ++w) s += ws[w];
        bsum[blockIdx.x] = s;
    }
}

// Unique set, CSR offsets, stable occurrence order and inverse index.
__global__ __launch_bounds__(kThreads) void dd_finalize(const uint32_t *__restrict__ k,
                                                        const int32_t *__restrict__ v, int n,
                                                        const int32_t *__restrict__ boff,
                                                        int32_t *__restrict__ uniq,
                                                        int32_t *__restrict__ inv,
                                                        int32_t *__restrict__ occ_perm,
                                                        int32_t *__restrict__ uniq_off)
{
    __shared__ int ws[kThreads / AMS_WAVE];
    const int t = threadIdx.x, w = t / AMS_WAVE;
    const int i0 = blockIdx.x * kUniqTile + t * kUniqItems;
    int flag[kUniqItems];
    int c = 0;
#pragma unroll
    for (int q = 0; q < kUniqItems; ++q) {
        const int i = i0 + q;
        flag[q] = (i < n && (i == 0 || k[i] != k[i - 1])) ? 1 : 0;
        c += flag[q];
    }
    const int incl = ams_wave_incl_scan(c);
    if (ams_lane() == AMS_WAVE - 1) ws[w] = incl;
    __syncthreads();
    int before = boff[blockIdx.x];
    for (int x = 0; x < w; ++x) before += ws[x];
    int run = before + incl - c;   // heads strictly before position i0
#pragma unroll
    for (int q = 0; q < kUniqItems; ++q) {
        const int i = i0 + q;
        if (i >= n) break;
        run += flag[q];
        const int rank = run - 1;
        const int32_t occ = v[i];
        occ_perm[i] = occ;
        inv[occ] = rank;
        if (flag[q]) {
            uniq[rank] = (int32_t)k[i];
            uniq_off[rank] = i;
        }
        if (i == n - 1) uniq_off[rank + 1] = n;
    }
}

int id_bits(int32_t n_ids)
{
    int b = 1;
    while (b < 31 && (1ll << b) < (long long)n_ids) ++b;
    return b;
}

struct DedupPlan {
    int bits, passes, width, ntiles, nutiles;
    size_t off_kb, off_va, off_vb, off_hist, off_bsum, total;
};

DedupPlan plan_dedup(int64_t n_occ, int32_t n_ids)
{
    DedupPlan p{};
    p.bits = id_bits(n_ids);
    p.passes = (p.bits + kMaxBits - 1) / kMaxBits;
    p.width = (p.bits + p.passes - 1) / p.passes;
    p.ntiles = (int)((n_occ + kTile - 1) / kTile);
    p.nutiles = (int)((n_occ + kUniqTile - 1) / kUniqTile);
    auto al = [](size_t x) { return (x + 255) & ~(size_t)255; };
    const size_t nb = al((size_t)n_occ * 4);
    size_t o = 0;
    // keys_a aliases nothing: the caller's ids are read directly in pass 0
    const size_t off_ka = o; o += nb;
    p.off_kb = o; o += nb;
    p.off_va = o; o += nb;
    p.off_vb = o; o += nb;
    p.off_hist = o; o += al((size_t)(1 << p.width) * (size_t)(p.ntiles > 0 ? p.ntiles : 1) * 4);
    p.off_bsum = o; o += al((size_t)(p.nutiles > 0 ? p.nutiles : 1) * 4);
    p.total = o;
    (void)off_ka;
    return p;
}

}  // namespace

extern "C" size_t ams_dedup_workspace(int64_t n_occ, int32_t n_ids)
{
    if (n_occ < 0 || n_ids < 1) return 0;
    return plan_dedup(n_occ, n_ids).total;
}

extern "C" ams_status ams_dedup(const int32_t *ids, int64_t n_occ, int32_t n_ids, int32_t *uniq,
                                int32_t *inv, int32_t *occ_perm, int32_t *uniq_off,
                                int32_t *n_uniq, int32_t *dev_status, void *ws, size_t ws_bytes,
                                void *stream)
{
    if (n_occ < 0 || n_occ > (int64_t)INT32_MAX - 1 || n_ids < 1) return AMS_ERR_SIZE;
    if (!uniq_off || !n_uniq || !dev_status) return AMS_ERR_NULL;
    if (n_occ > 0 && (!ids || !uniq || !inv || !occ_perm || !ws)) return AMS_ERR_NULL;
    const DedupPlan p = plan_dedup(n_occ, n_ids);
    if (n_occ > 0 && ws_bytes < p.total) return AMS_ERR_WORKSPACE;
    hipStream_t st = (hipStream_t)stream;
    const int n = (int)n_occ;

    dd_init<<<1, 64, 0, st>>>(n_uniq, dev_status, uniq_off, n);
    if (n == 0) return ams_launch_status();

    char *w = (char *)ws;
    uint32_t *ka = (uint32_t *)w;
    uint32_t *kb = (uint32_t *)(w + p.off_kb);
    int32_t *va = (int32_t *)(w + p.off_va);
    int32_t *vb = (int32_t *)(w + p.off_vb);
    int32_t *hist = (int32_t *)(w + p.off_hist);
    int32_t *bsum = (int32_t *)(w + p.off_bsum);

    const uint32_t *kin = (const uint32_t *)ids;
    const int32_t *vin = nullptr;
    uint32_t *bufk[2] = {ka, kb};
    int32_t *bufv[2] = {va, vb};
    for (int pass = 0; pass < p.passes; ++pass) {
        const int shift = pass * p.width;
        const int bits = (p.bits - shift) < p.width ? (p.bits - shift) : p.width;
        uint32_t *kout = bufk[pass & 1];
        int32_t *vout = bufv[pass & 1];
        dd_hist<<<p.ntiles, kThreads, 0, st>>>(kin, n, shift, bits, hist, p.ntiles,
                                               (uint32_t)n_ids, dev_status, pass == 0);
        dd_scan<<<1, kScanThreads, 0, st>>>(hist, (1 << bits) * p.ntiles, nullptr);
        dd_scatter<<<p.ntiles, kThreads, 0, st>>>(kin, vin, kout, vout, n, shift, bits, hist,
                                                  p.ntiles);
        kin = kout;
        vin = vout;
    }
    dd_head_count<<<p.nutiles, kThreads, 0, st>>>(kin, n, bsum);
    dd_scan<<<1, kScanThreads, 0, st>>>(bsum, p.nutiles, n_uniq);
    dd_finalize<<<p.nutiles, kThreads, 0, st>>>(kin, vin, n, bsum, uniq, inv, occ_perm, uniq_off);
    return ams_launch_status();
}
