// LSD radix sort of (uint32 key, uint32 value) pairs, digits of up to 8
// bits, for the two sorts of a frame (Sec. III-A, per-tile depth order):
//  1. the Gaussians that have keys, by depth (float bits of a positive depth
//     are ordered like the depths), input in Gaussian index order;
//  2. the Gaussian-tile keys by tile id, input in depth order.
// Both sorts are stable, so each tile's list ends up ordered by
// (depth bits, Gaussian index): deterministic and identical to a direct sort
// of the 64-bit (tile, depth) keys, at a third of the HBM traffic (the depth
// passes run over the Gaussians, not over their tile copies).
//
// Structure for gfx950, per pass: an upsweep kernel counts each partition's
// digits (1024 keys per partition for an expected count up to 2M keys, 3840
// above, 5120 for 16-bit keys) into
// a partition-major table, a column scan turns those counts into offsets
// within 16 chunks of partitions plus per-chunk digit sums, and a downsweep
// kernel ranks each partition in LDS and scatters it (the digit bases are a
// block scan of the 256 totals, plus the sums of earlier chunks).  No block
// ever waits on another and no device-wide atomic is contended (same-address
// atomics serialise across the eight XCDs), so the sort is deterministic and
// needs no forward-progress assumption.  Ranking is stable (a wave's 64-lane
// match over the digit bits plus per-wave digit counters in input order).
// A pass sorts only the bits its keys can have: the tile sort spreads the
// tile id's bits evenly over its passes, and the top depth digit has 7 bits
// (depths are positive).
// Keys are staged in LDS in digit order before the scatter so that writes of
// one digit run are contiguous.  Key counts live on the device (grids sized
// for an upper bound; partitions past the count do no work and are not
// scanned), so no host round trip is needed.
//
// The depth sort folds two neighbouring steps into its first and last pass:
//  - the first pass reads every Gaussian and keeps those with a key count
//    above zero (the compaction), writing the number kept; in a
//    selective-rendering frame its upsweep first recounts each Gaussian's
//    keys over the selected tiles of its rectangle;
//  - the last pass also carries each Gaussian's key count as a weight and
//    writes, at each sorted position, the exclusive prefix of the weights:
//    where the Gaussian's tile keys start, and the owner of every 1024-key
//    block of the emission.  It publishes the frame's counters to the host.
#include "match.h"
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
// keys below 2^16 (tile ids of grids up to 65536 tiles) are staged in LDS as
// 16-bit values, which leaves room for 5120-key partitions at four blocks
// per CU
constexpr int kIptLarge16 = 20;

enum { kPlain = 0, kFirst = 1, kLast = 2 };

__device__ inline uint32_t key_count(const uint32_t *n_dev, uint32_t n_host) {
    return n_dev ? *n_dev : n_host;
}

__device__ inline uint32_t sat32(uint64_t v) { return v > 0xffffffffull ? 0xffffffffu : (uint32_t)v; }

template <typename T>
__device__ inline T block_exclusive_scan256(T v, T *s_wave, T *total = nullptr) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    T inc = v;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const T o = __shfl_up(inc, d);
        if (lane >= d) inc += o;
    }
    if (lane == 63) s_wave[wave] = inc;
    __syncthreads();
    T off = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
        const T x = s_wave[w];
        if (w < wave) off += x;
        tot += x;
    }
    __syncthreads();
    if (total) *total = tot;
    return off + inc - v;
}

// Operands of the first and last depth-sort passes.
struct DepthIo {
    uint32_t *count;            // key count per Gaussian
    const ushort4 *rect;        // first pass of a selective frame: recount from
    const uint32_t *rowpre;     // the rectangles and the tile mask's row prefix
    int TX;                     // sums (rowpre NULL: count is final)
    uint32_t *offs;             // last pass: start of each sorted Gaussian's keys
    uint32_t *kfirst;           // last pass: owner of each key block (key_blocks(cap))
    Counters *cnt;
    HostCounters *host;         // last pass: the frame's counters, tag last
    uint32_t tag, cap;
    const uint32_t *pre_partial;   // preprocess per-block survivor / newly-visible counts
    int n_pre;
    // 1 (fewer than 2^24 Gaussians): the value the passes carry is
    // index << 8 | min(count, 255), so the last pass reads the key counts
    // below 255 from it instead of gathering them by index
    int pack;
};

// Key count of the Gaussian a carried value stands for, and its index.
__device__ inline uint32_t carried_count(const DepthIo &io, uint32_t v) {
    if (!io.pack) return io.count[v];
    const uint32_t c = v & 255u;
    return c < 255u ? c : io.count[v >> 8];
}
__device__ inline uint32_t carried_index(const DepthIo &io, uint32_t v) {
    return io.pack ? v >> 8 : v;
}

// Digit counts of one partition: counts[part * 256 + d] (one coalesced 1 KB
// row per block); in the last depth pass also the digit weight sums:
// weights[part * 256 + d].  The LDS counters are per wave and, in the last
// depth pass, per lane & 3 as well: its digits (the top bits of depths)
// take a handful of values, and lanes adding to one address serialise.
template <int IPT, int MODE>
__global__ __launch_bounds__(kSortThreads) void sort_upsweep_kernel(
    const uint32_t *__restrict__ kin, const uint32_t *__restrict__ vin, const uint32_t *n_dev,
    uint32_t n_host, int shift, int nbits, uint32_t np, DepthIo io, uint32_t *counts,
    uint32_t *weights) {
    constexpr uint32_t kTile = kSortThreads * IPT;
    constexpr int kCopies = MODE == kLast ? 4 : 1;
    constexpr int kRows = 4 * kCopies;
    __shared__ uint32_t s_h[kRows][kRadix];
    __shared__ uint32_t s_w[MODE == kLast ? kRows : 1][kRadix];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const uint32_t K = MODE == kFirst ? n_host : key_count(n_dev, n_host);
    const uint32_t part = blockIdx.x;
    if (part * kTile >= K) return;   // block-uniform: beyond the keys
    for (int k = tid; k < kRows * kRadix; k += kSortThreads) {
        (&s_h[0][0])[k] = 0u;
        if (MODE == kLast) (&s_w[0][0])[k] = 0u;
    }
    __syncthreads();
    const int row = wave * kCopies + (lane & (kCopies - 1));
    const uint32_t wbase = part * kTile + (uint32_t)wave * (64u * IPT);
    // every load first (clamped index, no branch), then the counting
    uint32_t dg[IPT], wv[MODE == kLast ? IPT : 1];
    bool keep[IPT];
#pragma unroll
    for (int j = 0; j < IPT; ++j) {
        const uint32_t idx = wbase + (uint32_t)(j * 64 + lane);
        keep[j] = idx < K;
        const uint32_t ic = keep[j] ? idx : K - 1u;
        dg[j] = (kin[ic] >> shift) & ((1u << nbits) - 1u);
        if (MODE == kFirst) {
            uint32_t c;
            if (io.rowpre) {
                c = masked_count(io.rect[ic], io.rowpre, io.TX);
                if (keep[j]) io.count[idx] = c;
            } else {
                c = io.count[ic];
            }
            keep[j] = keep[j] && c > 0u;
        }
        if (MODE == kLast) wv[j] = vin[ic];
    }
#pragma unroll
    for (int j = 0; j < IPT; ++j) {
        if (keep[j]) {
            atomicAdd(&s_h[row][dg[j]], 1u);
            if (MODE == kLast) atomicAdd(&s_w[row][dg[j]], carried_count(io, wv[j]));
        }
    }
    __syncthreads();
    uint32_t hc = 0;
#pragma unroll
    for (int r = 0; r < kRows; ++r) hc += s_h[r][tid];
    counts[(size_t)part * kRadix + tid] = hc;
    if (MODE == kLast) {
        uint32_t wc = 0;
#pragma unroll
        for (int r = 0; r < kRows; ++r) wc += s_w[r][tid];
        weights[(size_t)part * kRadix + tid] = wc;
    }
}

// The partitions holding keys are cut into kChunks chunks of L consecutive
// partitions.  One block per (table, chunk, group of 16 digits): exclusive
// scan, within the chunk, of each digit's counts (table 0) or weights
// (table 1), in place, and the chunk's digit sums in chunk_sums[c * 256 + d]
// (saturated to 32 bits).  A row of 16 digits is one 64-byte line, so every
// load uses whole lines.  The downsweep adds the sums of earlier chunks.
constexpr int kChunks = 16;

__device__ inline uint32_t chunk_len(uint32_t npa) {
    const uint32_t L = (npa + kChunks - 1) / kChunks;
    return L ? L : 1u;
}

__global__ __launch_bounds__(256) void sort_colscan_kernel(const uint32_t *n_dev, uint32_t n_host,
                                                           uint32_t tile, uint32_t np,
                                                           uint32_t *counts, uint32_t *chunk_sums) {
    __shared__ uint64_t s_sum[16][16];
    const int tid = threadIdx.x;
    const int g = blockIdx.x & 15, c = (blockIdx.x >> 4) % kChunks, table = blockIdx.x / (16 * kChunks);
    const int dl = tid & 15, lane = tid >> 4, d = 16 * g + dl;
    const uint32_t K = key_count(n_dev, n_host);
    const uint32_t npa = (K + tile - 1) / tile;   // <= np
    const uint32_t L = chunk_len(npa);
    const uint32_t S = (L + 15) / 16;             // partitions per thread
    uint32_t *tab = counts + (size_t)table * np * kRadix;
    uint32_t p0 = (uint32_t)c * L + (uint32_t)lane * S;
    uint32_t p1 = p0 + S;
    const uint32_t cend = (uint32_t)(c + 1) * L < npa ? (uint32_t)(c + 1) * L : npa;
    if (p1 > cend) p1 = cend;
    // sub-chunks of up to kKeep partitions stay in registers between the sum
    // and the write-back (one read of the table); longer ones are read twice
    constexpr uint32_t kKeep = 16;
    uint32_t keep[kKeep];
    uint64_t sum = 0;
    if (S <= kKeep) {
#pragma unroll
        for (uint32_t k = 0; k < kKeep; ++k) {
            keep[k] = p0 + k < p1 ? tab[(size_t)(p0 + k) * kRadix + d] : 0u;
            sum += keep[k];
        }
    } else {
        // long runs (huge sorts): eight loads in flight per step
        uint32_t p = p0;
        for (; p + 8 <= p1; p += 8) {
            uint32_t v[8];
#pragma unroll
            for (int k = 0; k < 8; ++k) v[k] = tab[(size_t)(p + k) * kRadix + d];
#pragma unroll
            for (int k = 0; k < 8; ++k) sum += v[k];
        }
        for (; p < p1; ++p) sum += tab[(size_t)p * kRadix + d];
    }
    s_sum[lane][dl] = sum;
    __syncthreads();
    if (tid < 16) {
        uint64_t run = 0;
        for (int l = 0; l < 16; ++l) {
            const uint64_t v = s_sum[l][tid];
            s_sum[l][tid] = run;
            run += v;
        }
        chunk_sums[(size_t)table * kChunks * kRadix + (size_t)c * kRadix + 16 * g + tid] = sat32(run);
    }
    __syncthreads();
    uint64_t o = s_sum[lane][dl];
    if (S <= kKeep) {
#pragma unroll
        for (uint32_t k = 0; k < kKeep; ++k) {
            if (p0 + k < p1) tab[(size_t)(p0 + k) * kRadix + d] = sat32(o);
            o += keep[k];
        }
    } else {
        uint32_t p = p0;
        for (; p + 8 <= p1; p += 8) {
            uint32_t v[8];
#pragma unroll
            for (int k = 0; k < 8; ++k) v[k] = tab[(size_t)(p + k) * kRadix + d];
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                tab[(size_t)(p + k) * kRadix + d] = sat32(o);
                o += v[k];
            }
        }
        for (; p < p1; ++p) {
            const uint32_t v = tab[(size_t)p * kRadix + d];
            tab[(size_t)p * kRadix + d] = sat32(o);
            o += v;
        }
    }
}

// Last depth pass, block 0: the frame's totals to the device counters and,
// tag last, to the host.
__device__ void publish_counters(const DepthIo &io, uint64_t n_keys, uint32_t *s_red) {
    const int tid = threadIdx.x;
    // eight pairs per thread and step, loaded before they are summed
    uint32_t a = 0, b = 0;
    const uint2 *pp = reinterpret_cast<const uint2 *>(io.pre_partial);
    for (int k0 = 0; k0 < io.n_pre; k0 += 8 * kSortThreads) {
        uint2 v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int k = k0 + u * kSortThreads + tid;
            v[u] = k < io.n_pre ? pp[k] : make_uint2(0u, 0u);
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            a += v[u].x;
            b += v[u].y;
        }
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        a += __shfl_xor(a, o);
        b += __shfl_xor(b, o);
    }
    if ((tid & 63) == 0) {
        s_red[2 * (tid >> 6)] = a;
        s_red[2 * (tid >> 6) + 1] = b;
    }
    __syncthreads();
    if (tid == 0) {
        const uint32_t surv = s_red[0] + s_red[2] + s_red[4] + s_red[6];
        const uint32_t newly = s_red[1] + s_red[3] + s_red[5] + s_red[7];
        const uint32_t k32 = sat32(n_keys);
        const uint32_t sorted = k32 <= io.cap ? k32 : 0u;
        io.cnt->n_keys = k32;
        io.cnt->n_sorted = sorted;
        io.cnt->n_survivors = surv;
        io.cnt->n_newly = newly;
        // n_visible and n_selected were written by earlier kernels
        publish_host(io.host, k32, surv, newly, io.cnt->n_selected, io.cnt->n_visible, sorted,
                     io.tag);
    }
    __syncthreads();
}

// KT: the type the keys are staged in (uint16_t: every key below 2^16).
// nbits: the pass's digit width (1..8): the digit is key bits [shift,
// shift + nbits).
template <int IPT, int MODE, typename KT>
__global__ __launch_bounds__(kSortThreads) void sort_downsweep_kernel(
    const uint32_t *__restrict__ kin, const uint32_t *__restrict__ vin, uint32_t *__restrict__ kout,
    uint32_t *__restrict__ vout, const uint32_t *n_dev, uint32_t n_host, int shift, int nbits,
    uint32_t np, const uint32_t *__restrict__ offsets, const uint32_t *__restrict__ chunk_sums,
    DepthIo io) {
    constexpr uint32_t kTile = kSortThreads * IPT;
    __shared__ KT s_keys[kTile];
    __shared__ uint32_t s_vals[kTile];
    __shared__ uint32_t s_wt[MODE == kLast ? kTile : 1];   // weights, then their exclusive scan
    __shared__ uint32_t s_wh[4 * kRadix];     // per-wave digit counters, then wave prefixes
    __shared__ uint32_t s_dstart[kRadix];     // block-local start of each digit
    __shared__ uint32_t s_gbase[kRadix];      // global start of this block's digit run,
                                              // then that minus the block-local start
    __shared__ uint32_t s_wbase[MODE == kLast ? kRadix : 1];   // global weight prefix of the run
    __shared__ uint32_t s_scan[4];
    __shared__ uint64_t s_scan64[4];
    __shared__ uint32_t s_nvalid;
    __shared__ uint32_t s_wtot;   // last pass: the block's weight total

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const uint32_t K = MODE == kFirst ? n_host : key_count(n_dev, n_host);
    const uint32_t part = blockIdx.x;
    const uint32_t base = part * kTile;
    const uint32_t c_mine = part / chunk_len((K + kTile - 1) / kTile);
    // digit tid: its total over all chunks and its sum over the chunks before this one
    uint64_t tot = 0, pre = 0, wtot = 0, wpre = 0;
#pragma unroll
    for (int c = 0; c < kChunks; ++c) {
        const uint32_t v = chunk_sums[c * kRadix + tid];
        tot += v;
        if ((uint32_t)c < c_mine) pre += v;
        if (MODE == kLast) {
            const uint32_t w = chunk_sums[kChunks * kRadix + c * kRadix + tid];
            wtot += w;
            if ((uint32_t)c < c_mine) wpre += w;
        }
    }
    // block 0 publishes the pass's totals (also when there is nothing to sort)
    if (MODE == kFirst && part == 0) {
        uint32_t n_kept;
        (void)block_exclusive_scan256<uint32_t>(sat32(tot), s_scan, &n_kept);
        if (tid == 0) io.cnt->n_visible = n_kept;
    }
    if (MODE == kLast && part == 0) {
        uint64_t n_keys;
        (void)block_exclusive_scan256<uint64_t>(wtot, s_scan64, &n_keys);
        publish_counters(io, n_keys, s_wh);
    }
    if (base >= K) return;   // block-uniform
    // issue every global load of the block before the first barrier
    const uint32_t wbase = base + (uint32_t)wave * (64u * IPT);
    const uint64_t lt_mask = (1ull << lane) - 1ull;
    const uint32_t dmask = (1u << nbits) - 1u;
    // 16-bit keys: each item's rank is kept in the upper half of its key
    constexpr bool kPack = sizeof(KT) == 2;
    uint32_t key[IPT], val[IPT], rank[kPack ? 1 : IPT], wt[MODE == kLast ? IPT : 1];
    bool ok[IPT];
#pragma unroll
    for (int j = 0; j < IPT; ++j) {
        const uint32_t idx = wbase + (uint32_t)(j * 64 + lane);
        ok[j] = idx < K;
        // clamped index: every load is issued, none behind a branch (the
        // values of lanes past the end are never used)
        const uint32_t ic = ok[j] ? idx : K - 1u;
        key[j] = kin[ic];
        if (MODE == kFirst) {
            const uint32_t c = io.count[ic];
            val[j] = io.pack ? idx << 8 | (c < 255u ? c : 255u) : idx;
            ok[j] = ok[j] && c > 0u;
        } else {
            val[j] = vin[ic];
        }
    }
    const uint32_t off_mine = offsets[(size_t)part * kRadix + tid];
    const uint32_t woff_mine = MODE == kLast ? offsets[(size_t)np * kRadix + (size_t)part * kRadix + tid] : 0u;
    if (MODE == kLast) {
#pragma unroll
        for (int j = 0; j < IPT; ++j) wt[j] = ok[j] ? carried_count(io, val[j]) : 0u;
    }
    for (int k = tid; k < 4 * kRadix; k += kSortThreads) s_wh[k] = 0u;
    // global start of digit tid: digits below it, then partitions before this one
    s_gbase[tid] = block_exclusive_scan256<uint32_t>(sat32(tot), s_scan) + sat32(pre) + off_mine;
    if (MODE == kLast) {
        const uint64_t wb = block_exclusive_scan256<uint64_t>(wtot, s_scan64);
        s_wbase[tid] = sat32(wb + wpre + woff_mine);
    }
    __syncthreads();
    // Rank: the lanes holding the same digit (matched over a group of items
    // at once), then the per-wave digit counters in input order.
    constexpr int kG = IPT % 5 == 0 ? 5 : 4;
    static_assert(IPT % kG == 0, "items per thread must be a multiple of the group");
#pragma unroll
    for (int j0 = 0; j0 < IPT; j0 += kG) {
        uint32_t dg[kG];
        uint64_t pm[kG];
#pragma unroll
        for (int g = 0; g < kG; ++g) {
            dg[g] = (key[j0 + g] >> shift) & dmask;
            pm[g] = __ballot(ok[j0 + g]);
        }
        match_digits<kG>(dg, nbits, pm);
#pragma unroll
        for (int g = 0; g < kG; ++g) {
            const int j = j0 + g;
            const bool valid = ok[j];
            const uint32_t d = dg[g];
            const uint64_t peers = pm[g];
            const uint32_t below = (uint32_t)__popcll(peers & lt_mask);
            uint32_t before = 0;
            if (valid) before = s_wh[wave * kRadix + d];
            __builtin_amdgcn_wave_barrier();
            if (valid && below == 0) s_wh[wave * kRadix + d] = before + (uint32_t)__popcll(peers);
            __builtin_amdgcn_wave_barrier();
            if constexpr (kPack) key[j] = (key[j] & 0xffffu) | ((before + below) << 16);
            else rank[j] = before + below;
        }
    }
    __syncthreads();

    const int d = tid;
    const uint32_t c0 = s_wh[d], c1 = s_wh[kRadix + d], c2 = s_wh[2 * kRadix + d],
                   c3 = s_wh[3 * kRadix + d];
    const uint32_t total = c0 + c1 + c2 + c3;
    uint32_t n_valid;
    // the scan's barriers also order the counter reads above before the
    // writes below
    const uint32_t dstart = block_exclusive_scan256<uint32_t>(total, s_scan, &n_valid);
    // per wave: where its items of digit d start in the block's staging
    s_wh[d] = dstart;
    s_wh[kRadix + d] = dstart + c0;
    s_wh[2 * kRadix + d] = dstart + c0 + c1;
    s_wh[3 * kRadix + d] = dstart + c0 + c1 + c2;
    s_dstart[d] = dstart;
    s_gbase[d] -= dstart;
    if (tid == 0) s_nvalid = n_valid;
    __syncthreads();

    // staging reads first (a digit of any item is in range), then the writes
    // of the kept items
#pragma unroll
    for (int j = 0; j < IPT; ++j) {
        uint32_t kj, rk;
        if constexpr (kPack) {
            kj = key[j] & 0xffffu;
            rk = key[j] >> 16;
        } else {
            kj = key[j];
            rk = rank[j];
        }
        const uint32_t dj = (kj >> shift) & dmask;
        const uint32_t pos = s_wh[wave * kRadix + dj] + rk;
        if (ok[j]) {
            s_keys[pos] = (KT)kj;
            s_vals[pos] = val[j];
            if (MODE == kLast) s_wt[pos] = wt[j];
        }
    }
    __syncthreads();
    const uint32_t nv = s_nvalid;

    if (MODE == kLast) {
        // exclusive scan of the weights in staged (digit, then input) order
        uint32_t w[IPT], sum = 0;
#pragma unroll
        for (int j = 0; j < IPT; ++j) {
            const uint32_t p = (uint32_t)tid * IPT + j;
            w[j] = p < nv ? s_wt[p] : 0u;
            sum += w[j];
        }
        uint32_t wtot;
        uint32_t o = block_exclusive_scan256<uint32_t>(sum, s_scan, &wtot);
#pragma unroll
        for (int j = 0; j < IPT; ++j) {
            const uint32_t p = (uint32_t)tid * IPT + j;
            if (p < nv) s_wt[p] = o;
            o += w[j];
        }
        if (tid == 0) s_wtot = wtot;
        __syncthreads();
    }

    if (MODE != kLast) {
        // every staged slot is read (in bounds; slots past nv are unused),
        // then the kept items are stored: all LDS reads of the thread in
        // flight at once
        uint32_t sk[IPT], sv[IPT], od[IPT];
#pragma unroll
        for (int j = 0; j < IPT; ++j) {
            const uint32_t i = (uint32_t)(j * kSortThreads + tid);
            sk[j] = (uint32_t)s_keys[i];
            sv[j] = s_vals[i];
        }
#pragma unroll
        for (int j = 0; j < IPT; ++j) od[j] = s_gbase[(sk[j] >> shift) & dmask];
#pragma unroll
        for (int j = 0; j < IPT; ++j) {
            const uint32_t i = (uint32_t)(j * kSortThreads + tid);
            if (i < nv) {
                kout[od[j] + i] = sk[j];
                vout[od[j] + i] = sv[j];
            }
        }
        return;
    }
    for (uint32_t i = tid; i < nv; i += kSortThreads) {
        const uint32_t kk = (uint32_t)s_keys[i];
        const uint32_t dj = (kk >> shift) & dmask;
        const uint32_t out = s_gbase[dj] + i;
        if (MODE == kLast) {
            const uint32_t o = s_wbase[dj] + (s_wt[i] - s_wt[s_dstart[dj]]);
            io.offs[out] = o;
            // the Gaussian's key count is its weight: the next prefix minus this one
            const uint32_t c = (i + 1 < nv ? s_wt[i + 1] : s_wtot) - s_wt[i];
            mark_key_blocks(io.kfirst, (uint32_t)key_blocks(io.cap), out, o, c);
        } else {
            kout[out] = kk;
        }
        vout[out] = MODE == kLast ? carried_index(io, s_vals[i]) : s_vals[i];
    }
}

inline int ipt_for(uint32_t n_max) { return n_max <= (2u << 20) ? kIptSmall : kIptLarge; }
inline uint32_t n_partitions(uint32_t K, int ipt) {
    const uint32_t tile = (uint32_t)(kSortThreads * ipt);
    const uint32_t np = (K + tile - 1) / tile;
    return np ? np : 1u;
}

// counted: the count table already holds the pass's digit counts (one row
// per partition, written by the key emission), so it has no counting launch.
template <int IPT, int MODE, typename KT = uint32_t>
void one_pass(const uint32_t *n_dev, uint32_t n_max, int shift, int nbits, const uint32_t *ki,
              const uint32_t *vi, uint32_t *ko, uint32_t *vo, uint32_t *scratch, const DepthIo &io,
              bool counted, hipStream_t st) {
    // at least one block: the last depth pass always publishes the counters
    const uint32_t np = n_partitions(n_max, IPT);
    uint32_t *chunk_sums = scratch;                 // [2][kChunks][256]
    uint32_t *table = sort_count_rows(scratch);     // [2][np][256]
    const uint32_t *nd = MODE == kFirst ? nullptr : n_dev;
    const int tables = MODE == kLast ? 2 : 1;
    if (!counted)
        sort_upsweep_kernel<IPT, MODE><<<np, kSortThreads, 0, st>>>(
            ki, vi, nd, n_max, shift, nbits, np, io, table, table + (size_t)np * kRadix);
    sort_colscan_kernel<<<tables * 16 * kChunks, 256, 0, st>>>(nd, n_max, kSortThreads * IPT, np,
                                                                table, chunk_sums);
    sort_downsweep_kernel<IPT, MODE, KT><<<np, kSortThreads, 0, st>>>(ki, vi, ko, vo, nd, n_max, shift,
                                                                  nbits, np, table, chunk_sums, io);
}

template <int IPT>
void depth_passes(uint32_t n, const uint32_t *dkey, uint32_t *k_a, uint32_t *v_a, uint32_t *k_b,
                  uint32_t *v_b, uint32_t *scratch, const DepthIo &io, hipStream_t st) {
    const uint32_t *n_vis = &io.cnt->n_visible;
    one_pass<IPT, kFirst>(nullptr, n, 0, 8, dkey, nullptr, k_a, v_a, scratch, io, false, st);
    one_pass<IPT, kPlain>(n_vis, n, 8, 8, k_a, v_a, k_b, v_b, scratch, io, false, st);
    one_pass<IPT, kPlain>(n_vis, n, 16, 8, k_b, v_b, k_a, v_a, scratch, io, false, st);
    // kept depths are positive (above the near plane): the sign bit is zero
    one_pass<IPT, kLast>(n_vis, n, 24, 7, k_a, v_a, nullptr, v_b, scratch, io, false, st);
}

template <int IPT, typename KT = uint32_t>
void plain_passes(const uint32_t *n_dev, uint32_t n_max, int begin_bit, int bits, uint32_t *ki,
                  uint32_t *vi, uint32_t *ko, uint32_t *vo, uint32_t *scratch, bool counted,
                  hipStream_t st) {
    const DepthIo none{};
    // digits of (nearly) equal width: fewer runs per partition in the widest
    // pass, so its scattered writes come in longer pieces
    const int passes = sort_passes_for_bits(bits);
    int shift = begin_bit;
    for (int p = 0; p < passes; ++p) {
        const int nb = bits / passes + (p < bits % passes ? 1 : 0);
        one_pass<IPT, kPlain, KT>(n_dev, n_max, shift, nb, ki, vi, ko, vo, scratch, none,
                                  counted && p == 0, st);
        shift += nb;
        uint32_t *t = ki; ki = ko; ko = t;
        t = vi; vi = vo; vo = t;
    }
}

}  // namespace

int sort_passes_for_bits(int bits) { return (bits + 7) / 8; }

size_t sort_scratch_words(uint32_t max_keys) {
    // chunk sums of counts and weights, then a (partition x digit) count table
    // and weight table, reused by every pass
    // (sized for the small partitions: a sort may take them for any count)
    const uint32_t np = n_partitions(max_keys, kIptSmall);
    return (size_t)2 * kChunks * kRadix + (size_t)2 * kRadix * np;
}

uint32_t *sort_count_rows(uint32_t *scratch) { return scratch + 2 * kChunks * kRadix; }

int sort_first_digit_bits(int bits) {
    const int passes = sort_passes_for_bits(bits);
    return passes > 0 ? bits / passes + (bits % passes ? 1 : 0) : 0;
}

// Items per thread of a plain sort: by the expected count (the grid covers
// n_max either way), 16-bit staging where every key is below 2^16.
static int plain_ipt(uint32_t n_max, uint32_t n_hint, int begin_bit, int bits) {
    if (ipt_for(n_hint < n_max ? n_hint : n_max) == kIptSmall) return kIptSmall;
    return begin_bit + bits <= 16 ? kIptLarge16 : kIptLarge;
}

// Counted rows are taken where a partition is one block of the emission
// (1024 keys).  Larger partitions could sum several rows, but their column
// scan over five times the rows cost more than the counting launch it
// replaces (room full frame: 4.8 -> 8.5 us against 5.3 us).
bool sort_takes_rows(uint32_t n_max, uint32_t n_hint, int begin_bit, int bits) {
    static_assert(kKeyBlock == kSortThreads * kIptSmall, "a counted row is a small partition");
    if (n_max <= 1 || sort_passes_for_bits(bits) <= 0) return false;
    return plain_ipt(n_max, n_hint, begin_bit, bits) == kIptSmall;
}

int launch_sort_u32(const uint32_t *n_dev, uint32_t n_max, uint32_t n_hint, int begin_bit,
                    int bits, uint32_t *keys, uint32_t *vals, uint32_t *keys_alt,
                    uint32_t *vals_alt, uint32_t *scratch, bool counted, hipStream_t st) {
    const int passes = sort_passes_for_bits(bits);
    if (n_max <= 1 || passes <= 0) return 0;
    counted = counted && sort_takes_rows(n_max, n_hint, begin_bit, bits);
    switch (plain_ipt(n_max, n_hint, begin_bit, bits)) {
        case kIptSmall:
            plain_passes<kIptSmall>(n_dev, n_max, begin_bit, bits, keys, vals, keys_alt, vals_alt,
                                    scratch, counted, st);
            break;
        case kIptLarge16:
            plain_passes<kIptLarge16, uint16_t>(n_dev, n_max, begin_bit, bits, keys, vals, keys_alt,
                                                vals_alt, scratch, counted, st);
            break;
        default:
            plain_passes<kIptLarge>(n_dev, n_max, begin_bit, bits, keys, vals, keys_alt, vals_alt,
                                    scratch, counted, st);
            break;
    }
    return passes & 1;
}

void launch_depth_sort(int n, uint32_t *count, const ushort4 *rect, const uint32_t *rowpre, int TX,
                       const uint32_t *dkey, uint32_t *k_a, uint32_t *v_a, uint32_t *k_b,
                       uint32_t *v_b, uint32_t *offs, uint32_t *kfirst, uint32_t *scratch,
                       Counters *cnt, uint32_t cap, const uint32_t *pre_partial, int n_pre,
                       HostCounters *host, uint32_t tag, hipStream_t st) {
    DepthIo io;
    io.count = count;
    io.rect = rect;
    io.rowpre = rowpre;
    io.TX = TX;
    io.offs = offs;
    io.kfirst = kfirst;
    io.cnt = cnt;
    io.host = host;
    io.tag = tag;
    io.cap = cap;
    io.pre_partial = pre_partial;
    io.n_pre = n_pre;
    io.pack = n < (1 << 24) ? 1 : 0;
    const uint32_t nn = (uint32_t)(n > 0 ? n : 0);
    if (ipt_for(nn) == kIptSmall)
        depth_passes<kIptSmall>(nn, dkey, k_a, v_a, k_b, v_b, scratch, io, st);
    else
        depth_passes<kIptLarge>(nn, dkey, k_a, v_a, k_b, v_b, scratch, io, st);
}

}  // namespace tgs
