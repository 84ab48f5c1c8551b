// Blend order of the tiles to rasterise, run by the standalone order kernel
// or, in frames with a per-tile sort, by the first block of that launch.
#pragma once

#include "match.h"
#include "tgs_internal.h"

namespace tgs {

// Blend order of the tiles to rasterise: longest lists first, bucketed by
// floor(log2(length)).  Tile lists are bimodal (a few thousand long tiles
// next to many short ones); launched in raster order, long tiles dispatched
// last would set the blend's tail.  Tiles are independent, so the order
// within a bucket changes only scheduling, never a result; the split set is
// a union of whole buckets.
// Bucket of a list length: floor(log2(len)) + 1, 0 for an empty list.
__device__ inline uint32_t length_bucket(const uint2 *ranges, int t) {
    const uint2 r = ranges[t];
    const uint32_t len = r.y - r.x;
    return len ? 32u - (uint32_t)__clz(len) : 0u;
}

constexpr int kOrderBuckets = 33;
// LDS words of order_tiles_block<NT, ...>: bucket counters per wave (at
// most).
constexpr int order_lds_words(int nt) { return (nt / 64) * kOrderBuckets; }

// Ranks N items per lane against running bucket counters wc[33] (in
// order: item k before item k + 1, lanes in order): lanes with equal
// buckets are matched over the six bucket bits and the lowest lane of each
// group advances the counter by the group's size with one LDS atomic, whose
// old value the group shares.  The N atomics are all issued before the
// first result is used.
template <int N>
__device__ inline void wave_bucket_rank(uint32_t *wc, const uint32_t (&b)[N], const bool (&active)[N],
                                        uint32_t (&rank)[N]) {
    const int lane = threadIdx.x & 63;
    const uint64_t lt = (1ull << lane) - 1ull;
    uint64_t pm[N];
#pragma unroll
    for (int k = 0; k < N; ++k) pm[k] = __ballot(active[k]);
    match_digits<N>(b, 6, pm);
    int leader[N];
    uint32_t base[N];
#pragma unroll
    for (int k = 0; k < N; ++k) {
        leader[k] = pm[k] ? __ffsll((long long)pm[k]) - 1 : lane;
        base[k] = 0u;
        if (active[k] && lane == leader[k]) base[k] = atomicAdd(&wc[b[k]], (uint32_t)__popcll(pm[k]));
    }
#pragma unroll
    for (int k = 0; k < N; ++k) rank[k] = __shfl(base[k], leader[k]) + (uint32_t)__popcll(pm[k] & lt);
}

// Bucket totals of the per-wave counts wc[w][b] (kWaves rows), then each
// wave's start in every bucket (buckets longest first, waves in order), in
// place; the split count and the longest bucket for the host.  Run by the
// first 64 threads between two barriers.
template <int kWaves>
__device__ inline void order_bucket_starts(const OrderK &o, uint32_t *s_cnt) {
    const int tid = threadIdx.x;
    // lane l holds bucket 32 - l
    const int b = 32 - tid;
    uint32_t c = 0;
    if (b >= 0) {
#pragma unroll
        for (int w = 0; w < kWaves; ++w) c += s_cnt[w * kOrderBuckets + b];
    }
    uint32_t inc = c;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const uint32_t x = __shfl_up(inc, d);
        if (tid >= d) inc += x;
    }
    if (b >= 0) {
        uint32_t run = inc - c;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) {
            const uint32_t x = s_cnt[w * kOrderBuckets + b];
            s_cnt[w * kOrderBuckets + b] = run;
            run += x;
        }
    }
    // the tiles the blend splits, a prefix of the order: those of the
    // buckets from the lowest one >= split_bucket that leaves at most
    // max_split tiles in it and above (whole buckets)
    const int sb = o.split_bucket;
    const uint64_t fit = __ballot(sb >= 1 && b >= sb && inc <= (uint32_t)o.max_split);
    const uint32_t ns = __shfl(inc, fit ? 63 - __clzll((long long)fit) : 0);
    if (o.n_split && tid == 0) *o.n_split = fit ? ns : 0u;
    const uint64_t nz = __ballot(c != 0u);
    // the host reads this value some frames later: no fence needed
    if (o.max_bucket && tid == 0)
        __hip_atomic_store(o.max_bucket, nz ? (uint32_t)(32 - (__ffsll((long long)nz) - 1)) : 0u,
                           __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

// One block of NT threads orders the tiles (s_cnt: order_lds_words(NT)
// words of LDS).  The tiles are counted per bucket; the counters then
// become the starts in every bucket, and every tile goes to its start plus
// its rank.  PER_WAVE: each wave counts on counters of its own (within a
// bucket the tiles keep the input's order: wave, item, lane); else all
// waves share one set (fewer registers; within a bucket the order depends
// on the timing of the waves).
template <int NT, bool PER_WAVE>
__device__ void order_tiles_block(const OrderK &o, uint32_t *s_cnt) {
    constexpr int kPer = 8;   // tiles per thread and round: all loads of a round in flight
    constexpr int kWaves = PER_WAVE ? NT / 64 : 1;
    const int tid = threadIdx.x, wave = tid >> 6;
    const int n = o.n_dev ? (int)*o.n_dev : o.n_host;
    uint32_t *wc = s_cnt + (PER_WAVE ? wave : 0) * kOrderBuckets;
    for (int k = tid; k < kWaves * kOrderBuckets; k += NT) s_cnt[k] = 0u;
    __syncthreads();
    int t[kPer];
    uint32_t bk[kPer], rank[kPer];
    bool act[kPer];
    // every lane runs every round (bounds are block-uniform) so that the
    // wave-level matching sees the whole wave
    auto load_rank = [&](int c0) {
#pragma unroll
        for (int k = 0; k < kPer; ++k) {
            const int i = c0 + k * NT + tid;
            act[k] = i < n;
            t[k] = act[k] ? (o.tile_in ? o.tile_in[i] : i) : 0;
        }
#pragma unroll
        for (int k = 0; k < kPer; ++k) bk[k] = act[k] ? length_bucket(o.ranges, t[k]) : 0u;
        wave_bucket_rank<kPer>(wc, bk, act, rank);
    };
    if (n <= kPer * NT) {
        // one round: the tiles and their ranks stay in registers
        load_rank(0);
        __syncthreads();
        if (tid < 64) order_bucket_starts<kWaves>(o, s_cnt);
        __syncthreads();
#pragma unroll
        for (int k = 0; k < kPer; ++k)
            if (act[k]) o.tile_out[wc[bk[k]] + rank[k]] = t[k];
    } else {
        // several rounds: counted, then loaded and ranked again from the
        // wave's starts
        for (int c0 = 0; c0 < n; c0 += kPer * NT) load_rank(c0);
        __syncthreads();
        if (tid < 64) order_bucket_starts<kWaves>(o, s_cnt);
        __syncthreads();
        for (int c0 = 0; c0 < n; c0 += kPer * NT) {
            load_rank(c0);
#pragma unroll
            for (int k = 0; k < kPer; ++k)
                if (act[k]) o.tile_out[rank[k]] = t[k];
        }
    }
}

}  // namespace tgs
