// Per-tile depth order without a global depth sort (Sec. III-A): an
// alternative to sorting every visible Gaussian by depth before emitting
// its keys, for frames whose tile lists are short.
//
//  1. Key counts are scanned in Gaussian index order (two kernels: block
//     partials, then the emission of the compacted (index, key offset)
//     pairs, each block summing the partials before it; block 0 publishes
//     the frame's counters).
//  2. Keys are emitted in index order and stably sorted by tile (the same
//     duplication and tile-sort kernels as the depth-ordered path), so each
//     tile's list comes out in index order.
//  3. One block per tile sorts its list by (depth bits, Gaussian index): a
//     stable LSD radix sort on the depth bits (passes of 8, 8, 8 and 7 bits,
//     depths being positive; the list in index order stays in index order
//     among equal depths) with the (depth key, index) pairs in LDS and 1-8
//     entries per thread, for lists
//     of up to 4096 entries; the same sort over global memory for longer
//     ones (correct for any length, meant for the rare list that outgrows
//     the bound).
// The per-tile lists are identical to those of the depth-ordered path.  One
// more block of the short-list launch computes the blend order of the tiles
// (order.h).
#include "match.h"
#include "order.h"
#include "tgs_internal.h"

namespace tgs {

namespace {

constexpr int kScanThreads = 256;
constexpr int kScanPer = 4;                               // Gaussians per thread
constexpr int kScanBlock = kScanThreads * kScanPer;       // 1024 Gaussians per block
// per-tile sort: lists of up to 2048 entries on 256-thread blocks (1-8
// entries per thread), longer ones on 512-thread blocks (8 per thread, or
// the global-memory path above 4096)
constexpr int kShortThreads = 256;
constexpr int kShortCap = 2048;
constexpr int kLongThreads = 512;
constexpr int kSegCap = 4096;

__device__ inline uint32_t sat32u(uint64_t v) { return v > 0xffffffffull ? 0xffffffffu : (uint32_t)v; }

// Inclusive scan across the block of one value per thread (256 threads);
// s_wave holds 4 entries.  Returns the exclusive prefix; *total the sum.
template <typename T>
__device__ inline T block_exscan(T v, T *s_wave, T *total) {
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
    for (int w = 0; w < (int)(blockDim.x >> 6); ++w) {
        const T x = s_wave[w];
        if (w < wave) off += x;
        tot += x;
    }
    __syncthreads();
    *total = tot;
    return off + inc - v;
}

// Per 1024-Gaussian block: keys and Gaussians with keys.  In a
// selective-rendering frame each count is first replaced by the selected
// tiles of the Gaussian's rectangle.  Thread t holds Gaussians
// base + 4t .. base + 4t + 3 (consecutive, so the emission's in-block scan
// follows index order).
__global__ __launch_bounds__(kScanThreads) void count_partials_kernel(int n, uint32_t *count,
                                                                      const ushort4 *rect,
                                                                      const uint32_t *rowpre, int TX,
                                                                      uint32_t *part) {
    __shared__ uint32_t s_w[4];
    const int base = blockIdx.x * kScanBlock + threadIdx.x * kScanPer;
    uint32_t keys = 0, nz = 0;
    if (rowpre) {
        // the four rectangles are loaded before the first count
        ushort4 r[kScanPer];
#pragma unroll
        for (int k = 0; k < kScanPer; ++k)
            r[k] = base + k < n ? rect[base + k] : make_ushort4(1, 0, 0, 0);
#pragma unroll
        for (int k = 0; k < kScanPer; ++k) {
            const uint32_t c = masked_count(r[k], rowpre, TX);
            if (base + k < n) count[base + k] = c;
            keys += c;
            nz += c ? 1u : 0u;
        }
    } else {
#pragma unroll
        for (int k = 0; k < kScanPer; ++k) {
            const uint32_t c = base + k < n ? count[base + k] : 0u;
            keys += c;
            nz += c ? 1u : 0u;
        }
    }
    uint32_t tk, tn;
    (void)block_exscan<uint32_t>(keys, s_w, &tk);
    (void)block_exscan<uint32_t>(nz, s_w, &tn);
    if (threadIdx.x == 0) {
        part[2 * blockIdx.x] = tk;
        part[2 * blockIdx.x + 1] = tn;
    }
}

// Sum over a 256-thread block of 64-bit and 32-bit values; every thread gets
// the totals.  s64 / s32 hold 4 entries each.
__device__ inline void block_sum2(unsigned long long &x, uint32_t &y, unsigned long long *s64,
                                  uint32_t *s32) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        x += __shfl_xor(x, o);
        y += __shfl_xor(y, o);
    }
    if ((threadIdx.x & 63) == 0) {
        s64[threadIdx.x >> 6] = x;
        s32[threadIdx.x >> 6] = y;
    }
    __syncthreads();
    x = s64[0] + s64[1] + s64[2] + s64[3];
    y = s32[0] + s32[1] + s32[2] + s32[3];
    __syncthreads();
}

// Sum of the pairs v[0, m) over a 256-thread block: eight pairs per thread
// and step, all loaded before they are summed; every thread gets the totals
// (x 64-bit, y 32-bit).
__device__ inline void block_sum_pairs(const uint2 *v, int m, unsigned long long &x, uint32_t &y,
                                       unsigned long long *s64, uint32_t *s32) {
    x = 0ull;
    y = 0u;
    for (int k0 = 0; k0 < m; k0 += 8 * kScanThreads) {
        uint2 t[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int k = k0 + u * kScanThreads + (int)threadIdx.x;
            t[u] = k < m ? v[k] : make_uint2(0u, 0u);
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            x += t[u].x;
            y += t[u].y;
        }
    }
    block_sum2(x, y, s64, s32);
}

// Per 1024-Gaussian block: the Gaussians with keys, in index order, at
// compacted positions: vidx[p] = index, voffs[p] = start of its keys.  The
// block's bases (keys and kept Gaussians of the blocks before it) are summed
// from their partials by the block itself: a few KB read from cache, instead
// of a one-block scan kernel between the two launches.  Block 0 (at least one
// is launched), first to start, also sums every partial and writes the
// frame's totals to the device counters and, tag last, to the host.
__global__ __launch_bounds__(kScanThreads) void count_emit_kernel(
    int n, int nb, const uint32_t *count, const uint32_t *part, uint32_t *vidx, uint32_t *voffs,
    uint32_t *kfirst, const uint32_t *pre_partial, int n_pre, Counters *cnt, HostCounters *host,
    uint32_t tag, uint32_t cap) {
    __shared__ uint32_t s_w[4];
    __shared__ unsigned long long s_k[4];
    const int tid = threadIdx.x;
    const int blk = blockIdx.x;
    // this block's counts first: their loads overlap the partial sums
    const int base = blk * kScanBlock + tid * kScanPer;
    uint32_t c[kScanPer], keys = 0, nz = 0;
#pragma unroll
    for (int k = 0; k < kScanPer; ++k) {
        c[k] = blk < nb && base + k < n ? count[base + k] : 0u;
        keys += c[k];
        nz += c[k] ? 1u : 0u;
    }
    const uint2 *pp = reinterpret_cast<const uint2 *>(part);
    unsigned long long bk;
    uint32_t bn;
    block_sum_pairs(pp, blk < nb ? blk : nb, bk, bn, s_k, s_w);   // blocks before this one
    if (blk < nb) {
        uint32_t tk, tn;
        uint32_t ok = block_exscan<uint32_t>(keys, s_w, &tk) + sat32u(bk);
        uint32_t on = block_exscan<uint32_t>(nz, s_w, &tn) + bn;
#pragma unroll
        for (int k = 0; k < kScanPer; ++k) {
            if (c[k]) {
                vidx[on] = (uint32_t)(base + k);
                voffs[on] = ok;
                mark_key_blocks(kfirst, (uint32_t)key_blocks(cap), on, ok, c[k]);
                ++on;
                ok += c[k];
            }
        }
    }
    if (blk != 0) return;   // block-uniform
    unsigned long long tot_k, sv;
    uint32_t tot_n, nw;
    block_sum_pairs(pp, nb, tot_k, tot_n, s_k, s_w);
    // survivors and newly visible Gaussians from the preprocess partials
    block_sum_pairs(reinterpret_cast<const uint2 *>(pre_partial), n_pre, sv, nw, s_k, s_w);
    if (tid == 0) {
        const uint32_t n_surv = (uint32_t)sv, n_newly = nw;
        const uint32_t k32 = sat32u(tot_k);
        const uint32_t sorted = k32 <= cap ? k32 : 0u;
        cnt->n_visible = tot_n;
        cnt->n_keys = k32;
        cnt->n_sorted = sorted;
        cnt->n_survivors = n_surv;
        cnt->n_newly = n_newly;
        // n_selected was written by the tile selection
        publish_host(host, k32, n_surv, n_newly, cnt->n_selected, tot_n, sorted, tag);
    }
}

// ---------------------------------------------------------------------------
// per-tile sort
// ---------------------------------------------------------------------------

// Stable in-block LSD radix sort of vals[0, L) by dkey[vals[i]] (four 8-bit
// passes, ping-pong with tmp; the depth keys are gathered again each pass).
template <int NT>
__device__ void segment_lsd(uint32_t *vals, uint32_t *tmp, uint32_t L, const uint32_t *dkey,
                            uint32_t *s_hist, uint32_t *s_wcnt, uint32_t *s_run) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    constexpr int kWaves = NT / 64;
    constexpr int kSegThreads = NT;
    const uint64_t lt = (1ull << lane) - 1ull;
    uint32_t *src = vals, *dst = tmp;
    for (int pass = 0; pass < 4; ++pass) {
        const int shift = 8 * pass;
        for (int d = tid; d < 256; d += kSegThreads) s_hist[d] = 0u;
        __syncthreads();
        for (uint32_t i = tid; i < L; i += kSegThreads)
            atomicAdd(&s_hist[(dkey[src[i]] >> shift) & 255u], 1u);
        __syncthreads();
        if (tid < 64) {
            // exclusive scan of the 256 digit counts by one wave (4 per lane)
            uint32_t v[4], sum = 0;
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                v[k] = s_hist[4 * tid + k];
                sum += v[k];
            }
            uint32_t inc = sum;
#pragma unroll
            for (int d = 1; d < 64; d <<= 1) {
                const uint32_t o = __shfl_up(inc, d);
                if (lane >= d) inc += o;
            }
            uint32_t run = inc - sum;
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                s_run[4 * tid + k] = run;
                run += v[k];
            }
        }
        __syncthreads();
        // stable scatter, one chunk of kSegThreads entries at a time
        for (uint32_t c0 = 0; c0 < L; c0 += kSegThreads) {
            const uint32_t i = c0 + tid;
            const bool ok = i < L;
            const uint32_t v = ok ? src[i] : 0u;
            const uint32_t d = ok ? (dkey[v] >> shift) & 255u : 0u;
            const uint32_t dg[1] = {d};
            uint64_t pm[1] = {__ballot(ok)};
            match_digits<1>(dg, 8, pm);
            const uint64_t peers = pm[0];
            for (int k = tid; k < kWaves * 256; k += kSegThreads) s_wcnt[k] = 0u;
            __syncthreads();
            if (ok && (peers & lt) == 0) s_wcnt[wave * 256 + d] = (uint32_t)__popcll(peers);
            __syncthreads();
            if (ok) {
                uint32_t before = 0;
                for (int w = 0; w < wave; ++w) before += s_wcnt[w * 256 + d];
                dst[s_run[d] + before + (uint32_t)__popcll(peers & lt)] = v;
            }
            __syncthreads();
            for (int dd = tid; dd < 256; dd += kSegThreads) {
                uint32_t t = 0;
                for (int w = 0; w < kWaves; ++w) t += s_wcnt[w * 256 + dd];
                s_run[dd] += t;
            }
            __syncthreads();
        }
        uint32_t *t = src;
        src = dst;
        dst = t;
    }
    // four passes: the result is back in vals
}

// Stable LSD radix sort of the list vals[0, L) (L <= 256 IPT) by its depth
// keys, in LDS.  Entry e of the current order sits at wave e / (64 IPT),
// item (e mod 64 IPT) / 64, lane e mod 64, so ranking items in order within
// a wave and waves in order keeps the sort stable.  Each pass ranks the
// digits (64-lane match over the 8 digit bits plus per-wave counters),
// scatters the (key, index) pairs into LDS in digit order and reloads them.
template <int IPT, int NT>
__device__ void seg_sort_lds(uint32_t *vals, uint32_t L, const uint32_t *dkey, uint2 *s_kv,
                             uint32_t *s_wh, uint32_t *s_dstart, uint32_t *s_scan) {
    constexpr int kWaves = NT / 64;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const uint64_t lt = (1ull << lane) - 1ull;
    const uint32_t wbase = (uint32_t)wave * 64u * IPT;
    uint32_t key[IPT], val[IPT];
    bool ok[IPT];
#pragma unroll
    for (int j = 0; j < IPT; ++j) {
        const uint32_t idx = wbase + (uint32_t)(j * 64 + lane);
        ok[j] = idx < L;
        val[j] = ok[j] ? vals[idx] : 0u;
    }
#pragma unroll
    for (int j = 0; j < IPT; ++j) key[j] = ok[j] ? dkey[val[j]] : 0u;
    for (int pass = 0; pass < 4; ++pass) {
        const int shift = 8 * pass;
        for (int k = tid; k < kWaves * 256; k += NT) s_wh[k] = 0u;
        __syncthreads();
        uint32_t rank[IPT];
        // depths are positive: the top digit has 7 bits
        const int nbits = pass == 3 ? 7 : 8;
        constexpr int kG = IPT < 4 ? IPT : 4;
#pragma unroll
        for (int j0 = 0; j0 < IPT; j0 += kG) {
            uint32_t dg[kG];
            uint64_t pm[kG];
#pragma unroll
            for (int g = 0; g < kG; ++g) {
                dg[g] = (key[j0 + g] >> shift) & 255u;
                pm[g] = __ballot(ok[j0 + g]);
            }
            match_digits<kG>(dg, nbits, pm);
#pragma unroll
            for (int g = 0; g < kG; ++g) {
                const int j = j0 + g;
                const bool valid = ok[j];
                const uint32_t d = dg[g];
                const uint64_t peers = pm[g];
                const uint32_t below = (uint32_t)__popcll(peers & lt);
                uint32_t before = 0;
                if (valid) before = s_wh[wave * 256 + d];
                __builtin_amdgcn_wave_barrier();
                if (valid && below == 0) s_wh[wave * 256 + d] = before + (uint32_t)__popcll(peers);
                __builtin_amdgcn_wave_barrier();
                rank[j] = before + below;
            }
        }
        __syncthreads();
        {
            // thread = digit: per-wave starts within the digit, digit starts
            const int d = tid;
            uint32_t total = 0;
            if (d < 256) {
#pragma unroll
                for (int w = 0; w < kWaves; ++w) {
                    const uint32_t c = s_wh[w * 256 + d];
                    s_wh[w * 256 + d] = total;
                    total += c;
                }
            }
            uint32_t tot;
            const uint32_t start = block_exscan<uint32_t>(total, s_scan, &tot);
            if (d < 256) s_dstart[d] = start;
        }
        __syncthreads();
#pragma unroll
        for (int j = 0; j < IPT; ++j) {
            if (ok[j]) {
                const uint32_t d = (key[j] >> shift) & 255u;
                s_kv[s_dstart[d] + s_wh[wave * 256 + d] + rank[j]] = make_uint2(key[j], val[j]);
            }
        }
        __syncthreads();
#pragma unroll
        for (int j = 0; j < IPT; ++j) {
            if (ok[j]) {
                const uint2 kv = s_kv[wbase + (uint32_t)(j * 64 + lane)];
                key[j] = kv.x;
                val[j] = kv.y;
            }
        }
        __syncthreads();   // every reload is done before the next scatter
    }
#pragma unroll
    for (int j = 0; j < IPT; ++j)
        if (ok[j]) vals[wbase + (uint32_t)(j * 64 + lane)] = val[j];
}

// One block per tile: its list [ranges.x, ranges.y) of vals, in index order,
// sorted by (depth bits, index) in place.  Short lists (up to 2048 entries):
// up to 256 by counting, longer ones by the LDS radix sort.
// Lists above 2048 entries: left to the long-list kernel (long_lists != 0),
// else sorted here over global memory (tmp), for frames where they are rare
// enough that a launch of their own costs more than it saves.
// With with_order, block 0 computes the blend order of the tiles (it needs
// only the list lengths, which the sort leaves unchanged) while the other
// blocks sort tile blockIdx.x - 1: the order costs no launch of its own.
__global__ __launch_bounds__(kShortThreads) void segment_sort_short_kernel(const uint2 *ranges,
                                                                         uint32_t *vals,
                                                                         uint32_t *tmp,
                                                                         const uint32_t *dkey,
                                                                         int long_lists,
                                                                         OrderK order,
                                                                         int with_order) {
    __shared__ uint2 s_kv[kShortCap];
    __shared__ uint32_t s_wh[(kShortThreads / 64) * 256];
    __shared__ uint32_t s_dstart[256];
    __shared__ uint32_t s_scan[kShortThreads / 64];
    __shared__ uint32_t s_ocnt[order_lds_words(kShortThreads)];
    int tile = (int)blockIdx.x;
    if (with_order) {
        if (tile == 0) {   // block-uniform
            order_tiles_block<kShortThreads, false>(order, s_ocnt);
            return;
        }
        tile -= 1;
    }
    const uint2 r = ranges[tile];
    const uint32_t L = r.y - r.x;
    if (L <= 1) return;   // block-uniform
    if (L > (uint32_t)kShortCap) {
        if (long_lists) return;
        uint32_t *s_hist = reinterpret_cast<uint32_t *>(s_kv);   // 256
        uint32_t *s_run = s_hist + 256;                          // 256
        segment_lsd<kShortThreads>(vals + r.x, tmp + r.x, L, dkey, s_hist, s_wh, s_run);
        return;
    }
    uint32_t *v = vals + r.x;
    if (L <= (uint32_t)kShortThreads) {
        // one entry per thread, ranked by counting: entry i goes to
        // #{j : d_j < d_i} + #{j < i : d_j = d_i} (the list is in index order,
        // so position breaks depth ties by index); one barrier in all
        uint32_t *s_d = reinterpret_cast<uint32_t *>(s_kv);
        const uint32_t i = threadIdx.x;
        uint32_t val = 0, d = 0;
        if (i < L) {
            val = v[i];
            d = dkey[val];
            s_d[i] = d;
        }
        __syncthreads();
        if (i < L) {
            uint32_t rank = 0;
            for (uint32_t j = 0; j < L; ++j) {
                const uint32_t dj = s_d[j];
                rank += (dj < d || (dj == d && j < i)) ? 1u : 0u;
            }
            v[rank] = val;
        }
    } else if (L <= 512) seg_sort_lds<2, kShortThreads>(v, L, dkey, s_kv, s_wh, s_dstart, s_scan);
    else if (L <= 1024) seg_sort_lds<4, kShortThreads>(v, L, dkey, s_kv, s_wh, s_dstart, s_scan);
    else seg_sort_lds<8, kShortThreads>(v, L, dkey, s_kv, s_wh, s_dstart, s_scan);
}

// The same for lists above 2048 entries: in LDS up to 4096, over global
// memory (tmp: scratch of the same layout as vals) beyond.
__global__ __launch_bounds__(kLongThreads) void segment_sort_long_kernel(const uint2 *ranges,
                                                                       uint32_t *vals, uint32_t *tmp,
                                                                       const uint32_t *dkey) {
    __shared__ uint2 s_kv[kSegCap];
    __shared__ uint32_t s_wh[(kLongThreads / 64) * 256];
    __shared__ uint32_t s_dstart[256];
    __shared__ uint32_t s_scan[kLongThreads / 64];
    const uint2 r = ranges[blockIdx.x];
    const uint32_t L = r.y - r.x;
    if (L <= (uint32_t)kShortCap) return;   // block-uniform
    if (L > (uint32_t)kSegCap) {
        uint32_t *s_hist = reinterpret_cast<uint32_t *>(s_kv);   // 256
        uint32_t *s_run = s_hist + 256;                          // 256
        segment_lsd<kLongThreads>(vals + r.x, tmp + r.x, L, dkey, s_hist, s_wh, s_run);
        return;
    }
    uint32_t *v = vals + r.x;
    seg_sort_lds<8, kLongThreads>(v, L, dkey, s_kv, s_wh, s_dstart, s_scan);
}

}  // namespace

int count_scan_blocks(int n) { return (n + kScanBlock - 1) / kScanBlock; }

void launch_count_scan(int n, uint32_t *count, const ushort4 *rect, const uint32_t *rowpre, int TX,
                       uint32_t *part, uint32_t *vidx, uint32_t *voffs, uint32_t *kfirst,
                       Counters *cnt, uint32_t cap, const uint32_t *pre_partial, int n_pre,
                       HostCounters *host, uint32_t tag, hipStream_t st) {
    const int nb = count_scan_blocks(n > 0 ? n : 0);
    if (nb > 0)
        count_partials_kernel<<<nb, kScanThreads, 0, st>>>(n, count, rect, rowpre, TX, part);
    // at least one block: the last one publishes the counters
    count_emit_kernel<<<nb > 0 ? nb : 1, kScanThreads, 0, st>>>(n, nb, count, part, vidx, voffs,
                                                                kfirst, pre_partial, n_pre, cnt,
                                                                host, tag, cap);
}

void launch_segment_sort(int n_tiles, const uint2 *ranges, uint32_t *vals, uint32_t *tmp,
                         const uint32_t *dkey, bool long_lists, const OrderK *order,
                         hipStream_t st) {
    if (n_tiles <= 0) return;
    if (long_lists)
        segment_sort_long_kernel<<<n_tiles, kLongThreads, 0, st>>>(ranges, vals, tmp, dkey);
    const bool with_order = order && order->n_host > 0;
    segment_sort_short_kernel<<<n_tiles + (with_order ? 1 : 0), kShortThreads, 0, st>>>(
        ranges, vals, tmp, dkey, long_lists ? 1 : 0, with_order ? *order : OrderK{},
        with_order ? 1 : 0);
}

}  // namespace tgs
