// dedup.hip -- ams_dedup: the batch's image IDs reduced to one sorted set with
// inverse index and stable occurrence order (section 4.2: requests for the
// same image are processed once; Algorithm 1: an image's gradients are
// collected in one place).
//
// Method: a stable LSD radix sort of (ID, occurrence index) over the
// ceil(log2 n_ids) significant bits, at most 8 bits per pass, then head flags
// and a scan give the unique set, its CSR offsets and the inverse index.
//
// Kernels (P = number of radix passes):
//   dd_prep        global digit histograms of every pass in one read of the
//                  IDs (per-block partials, no atomics across blocks), the ID
//                  range check, and zeroing of the look-back words;
//   dd_pass  x P   per 2048-key tile: local ranks from 64-lane ballots (lanes
//                  holding the same digit find each other bit by bit) and
//                  per-wave running counters in LDS; the tile's position among
//                  earlier tiles comes from decoupled look-back over the
//                  per-tile digit counts they publish; then a stable scatter;
//   dd_unique      head flags of the sorted keys, rank by the same look-back,
//                  and the outputs; the tile that completes a count of
//                  finished tiles writes the device status (the passes' error
//                  flag, the unique pass's own look-back bound hits carried in
//                  the count, and the range check).
// Tiles, waves, rows and lanes are visited in index order, so the sort is
// stable and every output bit-exact.  A tile only waits for earlier tiles to
// publish, and blocks are dispatched in index order, so every wait ends.
#include "ams_device.h"

#include <climits>
#include <mutex>

namespace {

constexpr int kThreads = 256;                 // 4 waves
constexpr int kWaves = kThreads / AMS_WAVE;
constexpr int kRows = 8;                      // rows of 64 keys per wave
constexpr int kTile = kThreads * kRows;       // 2048 keys per tile
constexpr int kMaxBits = 8;
constexpr int kRadix = 1 << kMaxBits;
constexpr int kMaxPasses = 4;
constexpr int kPrepBlocks = 32;                // partial histograms a pass sums

// look-back words: 2-bit state in the top bits, count below
constexpr uint32_t kAgg = 1u << 30;           // this tile's own count is published
constexpr uint32_t kPrefix = 2u << 30;        // the inclusive prefix up to this tile
constexpr uint32_t kValMask = (1u << 30) - 1;
constexpr int64_t kMaxOcc = (1 << 30) - 1;    // prefix counts stay below the state bits

__device__ __forceinline__ uint32_t ld_relaxed(const uint32_t *p)
{
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// The look-back words carry everything they communicate (no other data is
// published through them), so relaxed device-scope atomics suffice; they go
// around the per-XCD caches without the cache write-back/invalidate that
// release/acquire ordering would add.
__device__ __forceinline__ void st_relaxed(uint32_t *p, uint32_t v)
{
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Exclusive prefix of this tile's count over all earlier tiles (decoupled
// look-back).  words[t * stride] is this tile's word, earlier tiles' words at
// words[(t - 1) * stride], ...; with stride = the radix, the threads of a
// block (one digit each) read consecutive words.  Publishes the aggregate
// first, then the inclusive prefix.  Every tile publishes before it waits, so
// each wait ends; the wait is nevertheless bounded (kSpinLimit re-reads), and
// a bound that is hit is recorded in *err instead of spinning on.
constexpr int kSpinLimit = 1 << 22;

__device__ uint32_t lookback(uint32_t *words, int stride, int t, uint32_t count, int32_t *err)
{
    if (t == 0) {
        st_relaxed(&words[0], kPrefix | count);
        return 0;
    }
    st_relaxed(&words[(size_t)t * stride], kAgg | count);
    // walk back in batches of independent reads (one round trip each); the
    // nearest inclusive prefix is usually a few tiles back, so a batch of 16
    // (measured against 8, 32, 64 and 128: 20.3 against 21.5, 22.6, 32.7 and
    // 42.9 us per pass on 750k keys) keeps the reads that are not needed few
    constexpr int kBatch = 16;
    uint32_t excl = 0;
    int spins = 0;
    for (int hi = t - 1; hi >= 0;) {
        const int nb = hi + 1 < kBatch ? hi + 1 : kBatch;
        uint32_t w[kBatch];
        bool ready = true;
#pragma unroll
        for (int i = 0; i < kBatch; ++i) {
            w[i] = i < nb ? ld_relaxed(&words[(size_t)(hi - i) * stride]) : kPrefix;
            ready &= (w[i] & ~kValMask) != 0;
        }
        if (!ready) {                             // some tile of the batch has not published
            if (++spins < kSpinLimit) continue;
            __hip_atomic_store(err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            break;
        }
        spins = 0;
        bool done = false;
#pragma unroll
        for (int i = 0; i < kBatch; ++i) {
            if (done || i >= nb) continue;
            excl += w[i] & kValMask;
            done = (w[i] & ~kValMask) == kPrefix;
        }
        if (done) break;
        hi -= nb;
    }
    st_relaxed(&words[(size_t)t * stride], kPrefix | (excl + count));
    return excl;
}

// The same look-back walked by one whole wave: lane i reads the word of tile
// (hi - i), so 64 earlier tiles cost one round trip.  The lowest lane holding
// an inclusive prefix is the nearest one; the sum runs up to it.
__device__ uint32_t lookback_wave(uint32_t *words, int t, uint32_t count, bool &hit)
{
    const int lane = ams_lane();
    if (t == 0) {
        if (lane == 0) st_relaxed(&words[0], kPrefix | count);
        return 0;
    }
    if (lane == 0) st_relaxed(&words[t], kAgg | count);
    uint32_t excl = 0;
    int spins = 0;
    for (int hi = t - 1; hi >= 0;) {
        const int j = hi - lane;
        const uint32_t w = j >= 0 ? ld_relaxed(&words[j]) : kPrefix;   // before tile 0: prefix 0
        if (ams_ballot((w & ~kValMask) == 0) != 0) {                   // not all published yet
            if (++spins < kSpinLimit) continue;
            hit = true;
            break;
        }
        spins = 0;
        const uint64_t pre = ams_ballot((w & ~kValMask) == kPrefix);
        const int stop = pre ? __ffsll((unsigned long long)pre) - 1 : AMS_WAVE - 1;
        const int v = lane <= stop ? (int)(w & kValMask) : 0;
        excl += (uint32_t)__shfl(ams_wave_incl_scan(v), AMS_WAVE - 1, AMS_WAVE);
        if (pre) break;
        hi -= AMS_WAVE;
    }
    if (lane == 0) st_relaxed(&words[t], kPrefix | (excl + count));
    return excl;
}

struct Plan {
    int bits, passes, width, ntiles;
};

__device__ __forceinline__ int pass_bits(const Plan &P, int pass)
{
    const int shift = pass * P.width;
    return (P.bits - shift) < P.width ? (P.bits - shift) : P.width;
}

// Global digit histograms (partials per prep block), range check, zeroing.
// 1024 threads per block: one LDS histogram per wave (a hot ID's digit then
// contends within one wave only), 16 waves adding at once.
constexpr int kPrepThreads = 1024;
constexpr int kPrepWaves = kPrepThreads / AMS_WAVE;
__global__ __launch_bounds__(kPrepThreads) void dd_prep(const uint32_t *__restrict__ keys, int n, Plan P,
                                                        uint32_t n_ids, int32_t *__restrict__ hpart,
                                                        int32_t *__restrict__ bad,
                                                        uint32_t *__restrict__ words, int n_words)
{
    // eight keys per thread are loaded before their counts are added
    constexpr int U = 8;
    __shared__ int h[kPrepWaves][kMaxPasses][kRadix];
    const int t = threadIdx.x, wave = t / AMS_WAVE;
    for (int i = t; i < kPrepWaves * kMaxPasses * kRadix; i += kPrepThreads) (&h[0][0][0])[i] = 0;
    for (int i = blockIdx.x * kPrepThreads + t; i < n_words; i += gridDim.x * kPrepThreads) words[i] = 0;
    __syncthreads();
    bool out = false;
    const int stride = gridDim.x * kPrepThreads;
    for (int i0 = blockIdx.x * kPrepThreads + t; i0 < n; i0 += U * stride) {
        uint32_t k[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int i = i0 + u * stride;
            k[u] = i < n ? keys[i] : 0xffffffffu;
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (k[u] == 0xffffffffu && i0 + u * stride >= n) continue;
            out |= (k[u] >= n_ids);
            for (int p = 0; p < P.passes; ++p) {
                const uint32_t mask = (1u << pass_bits(P, p)) - 1u;
                atomicAdd(&h[wave][p][(k[u] >> (p * P.width)) & mask], 1);
            }
        }
    }
    const int any_out = __syncthreads_or(out);
    if (t < kRadix)
        for (int p = 0; p < P.passes; ++p) {
            int c = 0;
            for (int w = 0; w < kPrepWaves; ++w) c += h[w][p][t];
            hpart[((size_t)blockIdx.x * kMaxPasses + p) * kRadix + t] = c;
        }
    if (t == 0) bad[blockIdx.x] = any_out;
}

// One stable radix pass.  vin == nullptr means the identity (first pass).
__global__ __launch_bounds__(kThreads) void dd_pass(const uint32_t *__restrict__ kin,
                                                    const int32_t *__restrict__ vin,
                                                    uint32_t *__restrict__ kout, int32_t *__restrict__ vout,
                                                    int n, Plan P, int pass,
                                                    const int32_t *__restrict__ hpart, int n_prep,
                                                    uint32_t *__restrict__ words, int32_t *__restrict__ err)
{
    __shared__ int cnt[kWaves][kRadix];
    __shared__ int scan_tmp[kWaves];
    const int t = threadIdx.x, lane = ams_lane(), wave = t / AMS_WAVE;
    const int shift = pass * P.width, bits = pass_bits(P, pass);
    const uint32_t mask = (1u << bits) - 1u;
    const int tbase = blockIdx.x * kTile + wave * (kRows * AMS_WAVE);
    const uint64_t lt = ams_lanemask_lt();
    uint32_t key[kRows];
    int32_t val[kRows];
    int rank[kRows];
    // every load of the block first, all independent (one memory round trip):
    // the tile's keys and values (clamped, branch-free), then this pass's
    // per-block digit partials
#pragma unroll
    for (int r = 0; r < kRows; ++r) {
        const int idx = min(tbase + r * AMS_WAVE + lane, n - 1);
        key[r] = kin[idx];
        val[r] = vin ? vin[idx] : idx;
    }
    int part[kPrepBlocks];
#pragma unroll
    for (int b = 0; b < kPrepBlocks; ++b)
        part[b] = hpart[((size_t)min(b, n_prep - 1) * kMaxPasses + pass) * kRadix + t];
    for (int d = lane; d < kRadix; d += AMS_WAVE) cnt[wave][d] = 0;

    // global exclusive digit offsets of this pass (the same in every tile)
    int tot = 0;
#pragma unroll
    for (int b = 0; b < kPrepBlocks; ++b) tot += b < n_prep ? part[b] : 0;
    const int incl = ams_wave_incl_scan(tot);
    if (lane == AMS_WAVE - 1) scan_tmp[wave] = incl;
    __syncthreads();
    int gbase = incl - tot;
    for (int w = 0; w < wave; ++w) gbase += scan_tmp[w];

#pragma unroll
    for (int r = 0; r < kRows; ++r) {
        const int idx = tbase + r * AMS_WAVE + lane;
        const bool valid = idx < n;
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
    // this tile's count of digit t, and its position among earlier tiles
    // (2^width look-back words per tile; digits past this pass's bits are
    // empty everywhere)
    const int R = 1 << P.width;
    int tile_cnt = 0;
    for (int w = 0; w < kWaves; ++w) tile_cnt += cnt[w][t];
    uint32_t before = 0;
    if (t < (1 << bits))
        before = lookback(words + ((size_t)pass * P.ntiles) * R + t, R, blockIdx.x, (uint32_t)tile_cnt, err);
    // wave offsets inside the tile
    int run = gbase + (int)before;
    for (int w = 0; w < kWaves; ++w) {
        const int c = cnt[w][t];
        cnt[w][t] = run;
        run += c;
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kRows; ++r) {
        const int idx = tbase + r * AMS_WAVE + lane;
        if (idx < n) {
            const uint32_t d = (key[r] >> shift) & mask;
            const int pos = cnt[wave][d] + rank[r];
            kout[pos] = key[r];
            vout[pos] = val[r];
        }
    }
}

// Unique set, CSR offsets, stable occurrence order, inverse index, count,
// and the device status: each tile adds 1 + (hit << 32) to *done (one
// relaxed 64-bit add: tiles finished in the low word, look-back bound hits of
// this pass in the high word); the tile whose add completes the count reads
// the passes' error flag and the range check (earlier launches, ordered by
// the kernel boundaries) and writes the status.  Only the count itself is
// communicated between tiles, so no ordering beyond the add's atomicity is
// needed.
__global__ __launch_bounds__(kThreads) void dd_unique(const uint32_t *__restrict__ k,
                                                      const int32_t *__restrict__ v, int n,
                                                      uint32_t *__restrict__ words, const int32_t *__restrict__ err,
                                                      unsigned long long *__restrict__ done,
                                                      const int32_t *__restrict__ bad, int n_prep,
                                                      int32_t *__restrict__ uniq, int32_t *__restrict__ inv,
                                                      int32_t *__restrict__ occ_perm,
                                                      int32_t *__restrict__ uniq_off,
                                                      int32_t *__restrict__ n_uniq, int32_t *__restrict__ dev_status)
{
    constexpr int kItems = kTile / kThreads;  // 8 consecutive positions per thread
    __shared__ int ws[kWaves];
    __shared__ uint32_t tile_base;
    const int t = threadIdx.x, w = t / AMS_WAVE;
    const int i0 = blockIdx.x * kTile + t * kItems;
    static_assert(kItems == 8, "two 16-byte loads per thread");
    // a thread's 8 keys and values: two 16-byte loads each when all 8 are in
    // range (i0 is a multiple of 8), else one by one
    const bool full = i0 + kItems <= n;
    uint32_t kk[kItems];
    int32_t vv[kItems];
    if (full) {
        const uint4 a = *(const uint4 *)(k + i0), b = *(const uint4 *)(k + i0 + 4);
        const int4 x = *(const int4 *)(v + i0), y = *(const int4 *)(v + i0 + 4);
        kk[0] = a.x; kk[1] = a.y; kk[2] = a.z; kk[3] = a.w; kk[4] = b.x; kk[5] = b.y; kk[6] = b.z; kk[7] = b.w;
        vv[0] = x.x; vv[1] = x.y; vv[2] = x.z; vv[3] = x.w; vv[4] = y.x; vv[5] = y.y; vv[6] = y.z; vv[7] = y.w;
    } else {
#pragma unroll
        for (int q = 0; q < kItems; ++q) {
            kk[q] = i0 + q < n ? k[i0 + q] : 0u;
            vv[q] = i0 + q < n ? v[i0 + q] : 0;
        }
    }
    const uint32_t kprev = (i0 > 0 && i0 < n) ? k[i0 - 1] : 0u;
    int flag[kItems];
    int c = 0;
#pragma unroll
    for (int q = 0; q < kItems; ++q) {
        const int i = i0 + q;
        const uint32_t before = q == 0 ? kprev : kk[q - 1];
        flag[q] = (i < n && (i == 0 || kk[q] != before)) ? 1 : 0;
        c += flag[q];
    }
    const int incl = ams_wave_incl_scan(c);
    if (ams_lane() == AMS_WAVE - 1) ws[w] = incl;
    __syncthreads();
    bool hit = false;                          // (wave 0: this tile's look-back bound)
    if (w == 0) {
        int tot = 0;
        for (int x = 0; x < kWaves; ++x) tot += ws[x];
        const uint32_t b = lookback_wave(words, blockIdx.x, (uint32_t)tot, hit);
        if (t == 0) tile_base = b;
    }
    __syncthreads();
    int run = (int)tile_base + incl - c;      // heads strictly before position i0
    for (int x = 0; x < w; ++x) run += ws[x];
    // (the caller's occ_perm may start anywhere: 16-byte stores only when aligned)
    const bool vec_out = full && (((uintptr_t)occ_perm & 15) == 0);
    if (vec_out) {
        *(int4 *)(occ_perm + i0) = make_int4(vv[0], vv[1], vv[2], vv[3]);
        *(int4 *)(occ_perm + i0 + 4) = make_int4(vv[4], vv[5], vv[6], vv[7]);
    }
#pragma unroll
    for (int q = 0; q < kItems; ++q) {
        const int i = i0 + q;
        if (i >= n) break;
        run += flag[q];
        const int rank = run - 1;
        const int32_t occ = vv[q];
        if (!vec_out) occ_perm[i] = occ;
        inv[occ] = rank;
        if (flag[q]) {
            uniq[rank] = (int32_t)kk[q];
            uniq_off[rank] = i;
        }
        if (i == n - 1) {
            uniq_off[rank + 1] = n;
            *n_uniq = rank + 1;
        }
    }
    if (t == 0) {
        const unsigned long long old = __hip_atomic_fetch_add(done, 1ull + ((unsigned long long)hit << 32),
                                                              __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if ((uint32_t)old == gridDim.x - 1) {
            const bool lb = (old >> 32) != 0 || hit ||
                            __hip_atomic_load(err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0;
            int any_bad = 0;
            for (int b = 0; b < n_prep; ++b) any_bad |= bad[b];
            *dev_status = lb ? AMS_ERR_HIP : (any_bad ? AMS_ERR_ID_RANGE : AMS_OK);
        }
    }
}

__global__ void dd_empty(int32_t *n_uniq, int32_t *dev_status, int32_t *uniq_off)
{
    if (threadIdx.x == 0 && blockIdx.x == 0) {
        *dev_status = AMS_OK;
        *n_uniq = 0;
        uniq_off[0] = 0;
    }
}

constexpr int id_bits(int32_t n_ids)
{
    int b = 1;
    while (b < 31 && (1ll << b) < (long long)n_ids) ++b;
    return b;
}

struct Layout {
    Plan P;
    int n_prep, n_words, i_err, i_done;
    size_t off_kb, off_va, off_vb, off_hpart, off_bad, off_words, total;
};

constexpr Layout layout(int64_t n_occ, int32_t n_ids)
{
    Layout L{};
    L.P.bits = id_bits(n_ids);
    L.P.passes = (L.P.bits + kMaxBits - 1) / kMaxBits;
    L.P.width = (L.P.bits + L.P.passes - 1) / L.P.passes;
    L.P.ntiles = (int)((n_occ + kTile - 1) / kTile);
    L.n_prep = L.P.ntiles < kPrepBlocks ? (L.P.ntiles > 0 ? L.P.ntiles : 1) : kPrepBlocks;
    // look-back words (1 << width per tile and pass, then one per tile for
    // the unique pass), the passes' error flag, and the unique pass's 64-bit
    // completion count at an even word (the region is 256-byte aligned)
    const int n_lb = L.P.passes * L.P.ntiles * (1 << L.P.width) + L.P.ntiles;
    L.i_err = n_lb;
    L.i_done = (n_lb + 2) & ~1;
    L.n_words = L.i_done + 2;
    auto al = [](size_t x) constexpr { return (x + 255) & ~(size_t)255; };
    const size_t nb = al((size_t)n_occ * 4);
    size_t o = nb;                           // keys ping (pong is the caller's ids on pass 0)
    L.off_kb = o; o += nb;
    L.off_va = o; o += nb;
    L.off_vb = o; o += nb;
    L.off_hpart = o; o += al((size_t)L.n_prep * kMaxPasses * kRadix * 4);
    L.off_bad = o; o += al((size_t)L.n_prep * 4);
    L.off_words = o; o += al((size_t)L.n_words * 4);
    L.total = o;
    return L;
}

// Workspace that serves every ID range up to n_ids (and, the layout growing
// with n_occ, every smaller batch): the look-back words grow with the digit
// width, which is not monotonic in n_ids (100 IDs: one 7-bit pass; 1000: two
// of 5), so the largest layout over the bit counts up to n_ids's.
constexpr size_t workspace_bound(int64_t n_occ, int32_t n_ids)
{
    size_t t = 0;
    const int B = id_bits(n_ids);
    for (int b = 1; b <= B; ++b) {
        const size_t x = layout(n_occ, b == B ? n_ids : (int32_t)(1u << b)).total;
        t = x > t ? x : t;
    }
    return t;
}

// Enqueues the whole dedup with its workspace at `w` (layout L).
ams_status dedup_enqueue(const int32_t *ids, int n, int32_t n_ids, int32_t *uniq, int32_t *inv,
                         int32_t *occ_perm, int32_t *uniq_off, int32_t *n_uniq, int32_t *dev_status,
                         char *w, const Layout &L, hipStream_t st)
{
    if (n == 0) {
        AMS_LAUNCH("dd_empty", st, dd_empty<<<1, 64, 0, st>>>(n_uniq, dev_status, uniq_off));
        return ams_launch_status();
    }
    uint32_t *ka = (uint32_t *)w;
    uint32_t *kb = (uint32_t *)(w + L.off_kb);
    int32_t *va = (int32_t *)(w + L.off_va);
    int32_t *vb = (int32_t *)(w + L.off_vb);
    int32_t *hpart = (int32_t *)(w + L.off_hpart);
    int32_t *bad = (int32_t *)(w + L.off_bad);
    uint32_t *words = (uint32_t *)(w + L.off_words);
    int32_t *err = (int32_t *)(words + L.i_err);
    unsigned long long *done = (unsigned long long *)(words + L.i_done);

    // dd_prep also zeroes every look-back word, the error flag and the count
    AMS_LAUNCH("dd_prep", st, dd_prep<<<L.n_prep, kPrepThreads, 0, st>>>((const uint32_t *)ids, n, L.P, (uint32_t)n_ids, hpart, bad, words,
                                          L.n_words));
    const uint32_t *kin = (const uint32_t *)ids;
    const int32_t *vin = nullptr;
    uint32_t *bufk[2] = {ka, kb};
    int32_t *bufv[2] = {va, vb};
    for (int pass = 0; pass < L.P.passes; ++pass) {
        uint32_t *kout = bufk[pass & 1];
        int32_t *vout = bufv[pass & 1];
        AMS_LAUNCH("dd_pass", st, dd_pass<<<L.P.ntiles, kThreads, 0, st>>>(kin, vin, kout, vout, n, L.P, pass, hpart, L.n_prep, words,
                                                 err));
        kin = kout;
        vin = vout;
    }
    AMS_LAUNCH("dd_unique", st, dd_unique<<<L.P.ntiles, kThreads, 0, st>>>(
                                    kin, vin, n, words + (size_t)L.P.passes * L.P.ntiles * (1 << L.P.width), err, done,
                                    bad, L.n_prep, uniq, inv, occ_perm, uniq_off, n_uniq, dev_status));
    return ams_launch_status();
}

// ------------------------------------------------ no-allocation variant ----
// Scratch of ams_dedup_noalloc: the workspace of the largest batch it takes
// (kNoAllocMaxOcc occurrences, IDs of up to 31 bits: four radix passes),
// 19.0 MB in every GPU's copy of the library's code object.  Host code never
// passes `scratch` itself to a kernel (on the host it names a stand-in, not
// device memory): the device address comes from hipGetSymbolAddress, looked
// up once per device with that device current.
constexpr int64_t kNoAllocMaxOcc = AMS_DEDUP_NOALLOC_MAX_OCC;
constexpr size_t kScratchBytes = workspace_bound(kNoAllocMaxOcc, INT32_MAX);
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices];

// Device address of this device's scratch (nullptr on failure).
void *scratch_on_current_device()
{
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return nullptr;
        g_scratch_ptr[dev] = ptr;
    }
    return g_scratch_ptr[dev];
}

}  // namespace

extern "C" size_t ams_dedup_workspace(int64_t n_occ, int32_t n_ids)
{
    if (n_occ < 0 || n_ids < 1) return 0;
    return workspace_bound(n_occ, n_ids);
}

extern "C" ams_status ams_dedup(const int32_t *ids, int64_t n_occ, int32_t n_ids, int32_t *uniq,
                                int32_t *inv, int32_t *occ_perm, int32_t *uniq_off,
                                int32_t *n_uniq, int32_t *dev_status, void *ws, size_t ws_bytes,
                                void *stream)
{
    if (n_occ < 0 || n_occ > kMaxOcc || n_ids < 1) return AMS_ERR_SIZE;
    if (!uniq_off || !n_uniq || !dev_status) return AMS_ERR_NULL;
    if (n_occ > 0 && (!ids || !uniq || !inv || !occ_perm || !ws)) return AMS_ERR_NULL;
    const Layout L = layout(n_occ, n_ids);
    if (n_occ > 0 && ws_bytes < L.total) return AMS_ERR_WORKSPACE;
    return dedup_enqueue(ids, (int)n_occ, n_ids, uniq, inv, occ_perm, uniq_off, n_uniq, dev_status, (char *)ws, L,
                         (hipStream_t)stream);
}

extern "C" ams_status ams_dedup_noalloc(const int32_t *ids, int64_t n_occ, int32_t n_ids, int32_t *uniq,
                                        int32_t *inv, int32_t *occ_perm, int32_t *uniq_off,
                                        int32_t *n_uniq, int32_t *dev_status, void *stream)
{
    if (n_occ < 0 || n_ids < 1) return AMS_ERR_SIZE;
    if (n_occ > kNoAllocMaxOcc) return AMS_ERR_CAPACITY;
    if (!uniq_off || !n_uniq || !dev_status) return AMS_ERR_NULL;
    if (n_occ > 0 && (!ids || !uniq || !inv || !occ_perm)) return AMS_ERR_NULL;
    const Layout L = layout(n_occ, n_ids);
    if (L.total > kScratchBytes) return AMS_ERR_CAPACITY;
    char *w = (char *)scratch_on_current_device();
    if (!w) return AMS_ERR_HIP;
    return dedup_enqueue(ids, (int)n_occ, n_ids, uniq, inv, occ_perm, uniq_off, n_uniq, dev_status, w, L,
                         (hipStream_t)stream);
}
