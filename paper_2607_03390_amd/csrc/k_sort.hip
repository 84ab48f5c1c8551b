// LSD radix sort of (uint32 key, uint32 value) pairs, 8-bit digits, for the
// two sorts of a frame (Sec. III-A, per-tile depth order):
//  1. the visible Gaussians by depth (float bits of a positive depth are
//     ordered like the depths), input in Gaussian index order;
//  2. the Gaussian-tile keys by tile id, input in depth order.
// Both sorts are stable, so each tile's list ends up ordered by
// (depth bits, Gaussian index): deterministic and identical to a direct sort
// of the 64-bit (tile, depth) keys, at a third of the HBM traffic (the depth
// passes run over the Gaussians, not over their tile copies).
//
// Structure for gfx950, per 8-bit pass: an upsweep kernel counts each
// partition's digits (1024 keys per partition up to 2M keys, 3840 above), a column scan turns those counts into
// per-(digit, partition) offsets and digit totals, and a downsweep kernel
// ranks each partition in LDS and scatters it (the digit bases are a block
// scan of the 256 totals).  No block ever waits on another and no
// device-wide atomic is contended (same-address atomics serialise across the
// eight XCDs), so the sort is deterministic and needs no forward-progress
// assumption.  Ranking is stable (a wave's 64-lane match over the digit bits
// plus per-wave digit counters in input order).  Keys are staged in LDS in
// digit order before the scatter so that writes of one digit run are
// contiguous.  The key count may live on the device (grids sized for an upper
// bound; partitions past the count do no work and are not scanned), so no
// host round trip is needed.
#include "tgs_internal.h"

namespace tgs {

namespace {

constexpr int kSortThreads = 256;
constexpr int kRadix = 256;
// Keys per thread: partitions of 256 * IPT keys.  Large partitions for large
// sorts (fewer counts to scan), small ones for small sorts (enough blocks to
// fill the chip).
constexpr int kIptLarge = 15;   // 3840-key partitions
constexpr int kIptSmall = 4;    // 1024-key partitions

__device__ inline uint32_t key_count(const uint32_t *n_dev, uint32_t n_host) {
    return n_dev ? *n_dev : n_host;
}

__device__ inline uint32_t block_exclusive_scan256(uint32_t v, uint32_t *s_wave) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    uint32_t inc = v;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const uint32_t o = __shfl_up(inc, d);
        if (lane >= d) inc += o;
    }
    if (lane == 63) s_wave[wave] = inc;
    __syncthreads();
    uint32_t off = 0;
#pragma unroll
    for (int w = 0; w < 4; ++w)
        if (w < wave) off += s_wave[w];
    __syncthreads();
    return off + inc - v;
}

// Digit counts of one partition: counts[d * np + part].
template <int IPT>
__global__ __launch_bounds__(kSortThreads) void sort_upsweep_kernel(const uint32_t *__restrict__ kin,
                                                                    const uint32_t *n_dev,
                                                                    uint32_t n_host, int shift,
                                                                    uint32_t np, uint32_t *counts) {
    constexpr uint32_t kTile = kSortThreads * IPT;
    __shared__ uint32_t s_h[4][kRadix];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const uint32_t K = key_count(n_dev, n_host);
    const uint32_t part = blockIdx.x;
    if (part * kTile >= K) return;   // block-uniform: beyond the keys
    for (int k = tid; k < 4 * kRadix; k += kSortThreads) (&s_h[0][0])[k] = 0u;
    __syncthreads();
    const uint32_t wbase = part * kTile + (uint32_t)wave * (64u * IPT);
#pragma unroll
    for (int j = 0; j < IPT; ++j) {
        const uint32_t idx = wbase + (uint32_t)(j * 64 + lane);
        if (idx < K) atomicAdd(&s_h[wave][(kin[idx] >> shift) & 255u], 1u);
    }
    __syncthreads();
    counts[(size_t)tid * np + part] = s_h[0][tid] + s_h[1][tid] + s_h[2][tid] + s_h[3][tid];
}

// One block per digit: exclusive scan of the digit's counts over the
// partitions that hold keys (in place) and the digit's total.  Each thread
// scans 8 consecutive partitions, so one round covers 2048 partitions.
__global__ __launch_bounds__(256) void sort_colscan_kernel(const uint32_t *n_dev, uint32_t n_host,
                                                           uint32_t tile, uint32_t np,
                                                           uint32_t *counts, uint32_t *totals) {
    __shared__ uint32_t s_scan[4];
    __shared__ uint32_t s_run;
    const int d = blockIdx.x;
    const uint32_t K = key_count(n_dev, n_host);
    const uint32_t npa = (K + tile - 1) / tile;   // <= np
    uint32_t run = 0;
    uint32_t *col = counts + (size_t)d * np;
    for (uint32_t c = 0; c < npa; c += 2048) {
        const uint32_t p0 = c + 8u * threadIdx.x;
        uint32_t v[8], sum = 0;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            v[j] = p0 + j < npa ? col[p0 + j] : 0u;
            sum += v[j];
        }
        const uint32_t ex = block_exclusive_scan256(sum, s_scan);
        uint32_t o = run + ex;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            if (p0 + j < npa) col[p0 + j] = o;
            o += v[j];
        }
        if (threadIdx.x == 255) s_run = o;
        __syncthreads();
        run = s_run;
        __syncthreads();
    }
    if (threadIdx.x == 0) totals[d] = run;
}

template <int IPT>
__global__ __launch_bounds__(kSortThreads) void sort_downsweep_kernel(
    const uint32_t *__restrict__ kin, const uint32_t *__restrict__ vin, uint32_t *__restrict__ kout,
    uint32_t *__restrict__ vout, const uint32_t *n_dev, uint32_t n_host, int shift, uint32_t np,
    const uint32_t *__restrict__ offsets, const uint32_t *__restrict__ totals) {
    constexpr uint32_t kTile = kSortThreads * IPT;
    __shared__ uint32_t s_keys[kTile];
    __shared__ uint32_t s_vals[kTile];
    __shared__ uint32_t s_wh[4 * kRadix];     // per-wave digit counters, then wave prefixes
    __shared__ uint32_t s_dstart[kRadix];     // block-local start of each digit
    __shared__ uint32_t s_gbase[kRadix];      // global start of this block's digit run
    __shared__ uint32_t s_scan[4];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const uint32_t K = key_count(n_dev, n_host);
    const uint32_t part = blockIdx.x;
    const uint32_t base = part * kTile;
    if (base >= K) return;   // block-uniform
    for (int k = tid; k < 4 * kRadix; k += kSortThreads) s_wh[k] = 0u;
    // global start of digit tid: digits below it, then partitions before this one
    s_gbase[tid] = block_exclusive_scan256(totals[tid], s_scan) + offsets[(size_t)tid * np + part];
    __syncthreads();
    const uint32_t wbase = base + (uint32_t)wave * (64u * IPT);
    const uint64_t lt_mask = (1ull << lane) - 1ull;

    uint32_t key[IPT], val[IPT], rank[IPT];
#pragma unroll
    for (int j = 0; j < IPT; ++j) {
        const uint32_t idx = wbase + (uint32_t)(j * 64 + lane);
        const bool valid = idx < K;
        key[j] = valid ? kin[idx] : 0xffffffffu;
        val[j] = valid ? vin[idx] : 0u;
    }
#pragma unroll
    for (int j = 0; j < IPT; ++j) {
        const uint32_t idx = wbase + (uint32_t)(j * 64 + lane);
        const bool valid = idx < K;
        const uint32_t d = (key[j] >> shift) & 255u;
        uint64_t peers = __ballot(valid);
#pragma unroll
        for (int b = 0; b < 8; ++b) {
            const bool bit = (d >> b) & 1u;
            const uint64_t m = __ballot(bit);
            peers &= bit ? m : ~m;
        }
        const uint32_t below = (uint32_t)__popcll(peers & lt_mask);
        uint32_t before = 0;
        if (valid) before = s_wh[wave * kRadix + d];
        __builtin_amdgcn_wave_barrier();
        if (valid && below == 0) s_wh[wave * kRadix + d] = before + (uint32_t)__popcll(peers);
        __builtin_amdgcn_wave_barrier();
        rank[j] = before + below;
    }
    __syncthreads();

    const int d = tid;
    const uint32_t c0 = s_wh[d], c1 = s_wh[kRadix + d], c2 = s_wh[2 * kRadix + d],
                   c3 = s_wh[3 * kRadix + d];
    const uint32_t total = c0 + c1 + c2 + c3;
    __syncthreads();
    s_wh[d] = 0u;
    s_wh[kRadix + d] = c0;
    s_wh[2 * kRadix + d] = c0 + c1;
    s_wh[3 * kRadix + d] = c0 + c1 + c2;
    s_dstart[d] = block_exclusive_scan256(total, s_scan);
    __syncthreads();

#pragma unroll
    for (int j = 0; j < IPT; ++j) {
        const uint32_t idx = wbase + (uint32_t)(j * 64 + lane);
        if (idx < K) {
            const uint32_t dj = (key[j] >> shift) & 255u;
            const uint32_t pos = s_dstart[dj] + s_wh[wave * kRadix + dj] + rank[j];
            s_keys[pos] = key[j];
            s_vals[pos] = val[j];
        }
    }
    __syncthreads();

    const uint32_t n_valid = K - base < kTile ? K - base : kTile;
    for (uint32_t i = tid; i < n_valid; i += kSortThreads) {
        const uint32_t kk = s_keys[i];
        const uint32_t dj = (kk >> shift) & 255u;
        const uint32_t out = s_gbase[dj] + (i - s_dstart[dj]);
        kout[out] = kk;
        vout[out] = s_vals[i];
    }
}

inline int ipt_for(uint32_t n_max) { return n_max <= (2u << 20) ? kIptSmall : kIptLarge; }
inline uint32_t n_partitions(uint32_t K, int ipt) {
    const uint32_t tile = (uint32_t)(kSortThreads * ipt);
    return (K + tile - 1) / tile;
}

template <int IPT>
void sort_passes(const uint32_t *n_dev, uint32_t n_max, int begin_bit, int passes, uint32_t *ki,
                 uint32_t *vi, uint32_t *ko, uint32_t *vo, uint32_t *scratch, hipStream_t st) {
    const uint32_t np = n_partitions(n_max, IPT);
    uint32_t *totals = scratch;
    uint32_t *table = scratch + kRadix;
    for (int p = 0; p < passes; ++p) {
        const int shift = begin_bit + 8 * p;
        sort_upsweep_kernel<IPT><<<np, kSortThreads, 0, st>>>(ki, n_dev, n_max, shift, np, table);
        sort_colscan_kernel<<<kRadix, 256, 0, st>>>(n_dev, n_max, kSortThreads * IPT, np, table,
                                                    totals);
        sort_downsweep_kernel<IPT><<<np, kSortThreads, 0, st>>>(ki, vi, ko, vo, n_dev, n_max, shift,
                                                                np, table, totals);
        uint32_t *t = ki; ki = ko; ko = t;
        t = vi; vi = vo; vo = t;
    }
}

}  // namespace

int sort_passes_for_bits(int bits) { return (bits + 7) / 8; }

size_t sort_scratch_words(uint32_t max_keys, int passes) {
    // digit totals + one (digit x partition) offset table, reused by every pass
    (void)passes;
    return (size_t)kRadix + (size_t)kRadix * (n_partitions(max_keys, ipt_for(max_keys)) + 1);
}

int launch_sort_u32(const uint32_t *n_dev, uint32_t n_max, int begin_bit, int passes,
                    uint32_t *keys, uint32_t *vals, uint32_t *keys_alt, uint32_t *vals_alt,
                    uint32_t *scratch, hipStream_t st) {
    if (n_max <= 1 || passes <= 0) return 0;
    if (ipt_for(n_max) == kIptSmall)
        sort_passes<kIptSmall>(n_dev, n_max, begin_bit, passes, keys, vals, keys_alt, vals_alt,
                               scratch, st);
    else
        sort_passes<kIptLarge>(n_dev, n_max, begin_bit, passes, keys, vals, keys_alt, vals_alt,
                               scratch, st);
    return passes & 1;
}

}  // namespace tgs
