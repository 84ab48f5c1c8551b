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
// (which, within a bucket, depends on LDS atomics) changes only scheduling,
// never a result.
// Bucket of a list length: floor(log2(len)) + 1, 0 for an empty list.
__device__ inline uint32_t length_bucket(const uint2 *ranges, int t) {
    const uint2 r = ranges[t];
    const uint32_t len = r.y - r.x;
    return len ? 32u - (uint32_t)__clz(len) : 0u;
}

// Wave-aggregated LDS atomics without a loop, for N items per lane: lanes
// with equal buckets are matched over the six bucket bits; the lowest lane
// of each group adds the group's size (one LDS atomic instruction per item
// for all groups) and the others take consecutive slots after its old
// value.  Items are counted in order (item k before item k + 1), and every
// match and atomic of the N items is issued before the first result is used.
template <int N>
__device__ inline void wave_bucket_add(uint32_t *s_cnt, const uint32_t (&b)[N], const bool (&active)[N],
                                       uint32_t (&slot)[N]) {
    const int lane = threadIdx.x & 63;
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
        if (active[k] && lane == leader[k]) base[k] = atomicAdd(&s_cnt[b[k]], (uint32_t)__popcll(pm[k]));
    }
#pragma unroll
    for (int k = 0; k < N; ++k)
        slot[k] = __shfl(base[k], leader[k]) + (uint32_t)__popcll(pm[k] & ((1ull << lane) - 1ull));
}

// One block of NT threads orders the tiles (s_cnt: 33 words of LDS).
template <int NT>
__device__ void order_tiles_block(const OrderK &o, uint32_t *s_cnt) {
    constexpr int kPer = 8;   // tiles per thread and round: all loads of a round in flight
    const int tid = threadIdx.x;
    const int n = o.n_dev ? (int)*o.n_dev : o.n_host;
    const int *tile_in = o.tile_in;
    const uint2 *ranges = o.ranges;
    int *tile_out = o.tile_out;
    uint32_t *max_bucket = o.max_bucket;
    if (tid < 33) s_cnt[tid] = 0u;
    __syncthreads();
    // up to kPer * NT tiles (one round) the tiles and buckets stay in
    // registers between the counting and the placing pass; more take a
    // second load
    const bool one_round = n <= kPer * NT;
    int t[kPer];
    uint32_t bk[kPer];
    bool act[kPer];
    // every lane runs every round (bounds are block-uniform) so that the
    // wave-level aggregation sees the whole wave
    for (int pass = 0; pass < 2; ++pass) {
        for (int c0 = 0; c0 < n; c0 += kPer * NT) {
            if (pass == 0 || !one_round) {
#pragma unroll
                for (int k = 0; k < kPer; ++k) {
                    const int i = c0 + k * NT + tid;
                    act[k] = i < n;
                    t[k] = act[k] ? (tile_in ? tile_in[i] : i) : 0;
                }
#pragma unroll
                for (int k = 0; k < kPer; ++k) bk[k] = act[k] ? length_bucket(ranges, t[k]) : 0u;
            }
            // one LDS atomic per bucket present in the wave and item (lists
            // fall into a dozen buckets: per-lane atomics contend)
            uint32_t slot[kPer];
            wave_bucket_add<kPer>(s_cnt, bk, act, slot);
            if (pass == 1) {
#pragma unroll
                for (int k = 0; k < kPer; ++k)
                    if (act[k]) tile_out[slot[k]] = t[k];
            }
        }
        __syncthreads();
        if (pass == 0 && tid < 64) {
            // bucket starts, longest lists first: lane l holds bucket 32 - l
            const int b = 32 - tid;
            const uint32_t c = b >= 0 ? s_cnt[b] : 0u;
            uint32_t inc = c;
#pragma unroll
            for (int d = 1; d < 64; d <<= 1) {
                const uint32_t o = __shfl_up(inc, d);
                if (tid >= d) inc += o;
            }
            if (b >= 0) s_cnt[b] = inc - c;
            // the tiles the blend splits, a prefix of the order: those of
            // the buckets from the lowest one >= split_bucket that leaves at
            // most max_split tiles in it and above (whole buckets, so the set
            // does not depend on the order within a bucket)
            const int sb = o.split_bucket;
            const uint64_t fit = __ballot(sb >= 1 && b >= sb && inc <= (uint32_t)o.max_split);
            const uint32_t ns = __shfl(inc, fit ? 63 - __clzll((long long)fit) : 0);
            if (o.n_split && tid == 0) *o.n_split = fit ? ns : 0u;
            const uint64_t nz = __ballot(c != 0u);
            // the host reads this value some frames later: no fence needed
            if (max_bucket && tid == 0)
                __hip_atomic_store(max_bucket, nz ? (uint32_t)(32 - (__ffsll((long long)nz) - 1)) : 0u,
                                   __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
        }
        __syncthreads();
    }
}


}  // namespace tgs
