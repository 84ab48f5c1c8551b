// Gaussian-tile duplication (Sec. III-A) around the two sorts of a frame:
//  - masked key counts: in a selective-rendering frame a Gaussian's count is
//    the number of selected tiles of its rectangle, from per-row prefix sums
//    of the tile mask (one subtraction per row);
//  - compaction of the Gaussians with at least one key, in index order, into
//    (depth bits, index) pairs for the depth sort;
//  - exclusive scan of the key counts in depth order;
//  - key emission in depth order, one output key per lane so every store is
//    coalesced (the owning Gaussian is found by a binary search over the
//    wave's 64 offsets held in LDS);
//  - per-tile [start, end) ranges of the tile-sorted keys.
// The scans are reduce-then-scan over 4096-element blocks (no block waits on
// another, no contended atomics); their totals stay on the device, so the
// depth sort needs no host round trip.
#include "tgs_internal.h"

namespace tgs {

namespace {

constexpr int kScanThreads = 256;
constexpr int kScanItems = 16;
constexpr int kScanTile = kScanThreads * kScanItems;   // 4096

__device__ inline uint32_t masked_count(ushort4 r, const uint32_t *rowpre, int TX) {
    if (r.x > r.z || r.y > r.w) return 0u;
    uint32_t c = 0;
    for (int y = r.y; y <= r.w; ++y) {
        const uint32_t *row = rowpre + (size_t)y * (TX + 1);
        c += row[r.z + 1] - row[r.x];
    }
    return c;
}

__global__ __launch_bounds__(256) void count_masked_kernel(int n, const ushort4 *rect,
                                                           const uint32_t *rowpre, int TX,
                                                           uint32_t *count) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) count[i] = masked_count(rect[i], rowpre, TX);
}

// Exclusive block scan of 64-bit values over 256 threads.
__device__ inline uint64_t block_exclusive_scan64(uint64_t v, uint64_t *s_wave, uint64_t *total) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    uint64_t inc = v;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const uint64_t o = __shfl_up(inc, d);
        if (lane >= d) inc += o;
    }
    if (lane == 63) s_wave[wave] = inc;
    __syncthreads();
    uint64_t off = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
        const uint64_t x = s_wave[w];
        if (w < wave) off += x;
        tot += x;
    }
    __syncthreads();
    *total = tot;
    return off + inc - v;
}

// The two scans of a frame are reduce-then-scan: per-block sums, one block
// scanning the sums, then a downsweep that recomputes the local values.
// Thread t of block b owns the 16 consecutive elements b*4096 + 16t + j, read
// with 16-byte loads; one block scan per block.

// MODE 0: flags (count[i] > 0) over Gaussians i < n (n on the host).
// MODE 1: key counts count[didx[s]] over sorted positions s < cnt->n_visible.
template <int MODE>
__device__ inline void load16(uint32_t first, int n, const uint32_t *count, const uint32_t *didx,
                              const Counters *cnt, uint32_t v[kScanItems]) {
    const uint32_t lim = MODE == 0 ? (uint32_t)n : cnt->n_visible;
    const uint32_t *src = MODE == 0 ? count : didx;
    if (first + kScanItems <= lim) {
#pragma unroll
        for (int j = 0; j < kScanItems; j += 4) {
            const uint4 q = *reinterpret_cast<const uint4 *>(src + first + j);
            v[j] = q.x; v[j + 1] = q.y; v[j + 2] = q.z; v[j + 3] = q.w;
        }
    } else {
#pragma unroll
        for (int j = 0; j < kScanItems; ++j) v[j] = first + j < lim ? src[first + j] : 0xffffffffu;
    }
#pragma unroll
    for (int j = 0; j < kScanItems; ++j) {
        if (first + j >= lim) v[j] = 0u;
        else if (MODE == 0) v[j] = v[j] > 0u ? 1u : 0u;
        else v[j] = count[v[j]];
    }
}

template <int MODE>
__global__ __launch_bounds__(kScanThreads) void scan_reduce_kernel(int n, const uint32_t *count,
                                                                   const uint32_t *didx,
                                                                   const Counters *cnt,
                                                                   uint64_t *block_sums) {
    uint32_t v[kScanItems];
    load16<MODE>(blockIdx.x * (uint32_t)kScanTile + threadIdx.x * kScanItems, n, count, didx, cnt, v);
    uint64_t sum = 0;
#pragma unroll
    for (int j = 0; j < kScanItems; ++j) sum += v[j];
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) sum += __shfl_xor(sum, o);
    __shared__ uint64_t s_sum[4];
    if ((threadIdx.x & 63) == 0) s_sum[threadIdx.x >> 6] = sum;
    __syncthreads();
    if (threadIdx.x == 0) block_sums[blockIdx.x] = s_sum[0] + s_sum[1] + s_sum[2] + s_sum[3];
}

// One block: exclusive scan of the block sums in place; the total goes to
// cnt->n_visible (MODE 0) or cnt->n_keys (MODE 1, saturated; cnt->n_sorted is
// the same count when it fits the key capacity, else 0).
template <int MODE>
__global__ __launch_bounds__(1024) void scan_top_kernel(int nb, uint64_t *block_sums,
                                                        const uint32_t *pre_partial, int n_pre,
                                                        uint32_t cap, Counters *cnt,
                                                        HostCounters *host, uint32_t tag) {
    __shared__ uint64_t s_wave[16];
    __shared__ uint64_t s_carry;
    __shared__ uint32_t s_pre[16][2];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    if (MODE == 0) {
        // survivor and newly-visible counts of the preprocess blocks
        uint32_t a = 0, b = 0;
        for (int k = threadIdx.x; k < n_pre; k += 1024) {
            a += pre_partial[2 * k];
            b += pre_partial[2 * k + 1];
        }
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) {
            a += __shfl_xor(a, o);
            b += __shfl_xor(b, o);
        }
        if (lane == 0) {
            s_pre[wave][0] = a;
            s_pre[wave][1] = b;
        }
    }
    if (threadIdx.x == 0) s_carry = 0;
    __syncthreads();
    if (MODE == 0 && threadIdx.x == 0) {
        uint32_t a = 0, b = 0;
        for (int w = 0; w < 16; ++w) {
            a += s_pre[w][0];
            b += s_pre[w][1];
        }
        cnt->n_survivors = a;
        cnt->n_newly = b;
    }
    for (int c = 0; c < nb; c += 1024) {
        const int i = c + threadIdx.x;
        const uint64_t v = i < nb ? block_sums[i] : 0;
        uint64_t inc = v;
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
            const uint64_t o = __shfl_up(inc, d);
            if (lane >= d) inc += o;
        }
        if (lane == 63) s_wave[wave] = inc;
        __syncthreads();
        uint64_t off = 0, tot = 0;
        for (int w = 0; w < 16; ++w) {
            const uint64_t x = s_wave[w];
            if (w < wave) off += x;
            tot += x;
        }
        const uint64_t carry = s_carry;
        if (i < nb) block_sums[i] = carry + off + inc - v;
        __syncthreads();
        if (threadIdx.x == 0) s_carry = carry + tot;
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        const uint64_t total = s_carry;
        const uint32_t t32 = total > 0xffffffffull ? 0xffffffffu : (uint32_t)total;
        if (MODE == 0) {
            cnt->n_visible = t32;
        } else {
            const uint32_t sorted = t32 <= cap ? t32 : 0u;
            cnt->n_keys = t32;
            cnt->n_sorted = sorted;
            // every other counter was written by an earlier kernel
            volatile HostCounters *h = host;
            h->n_keys = t32;
            h->n_survivors = cnt->n_survivors;
            h->n_newly = cnt->n_newly;
            h->n_selected = cnt->n_selected;
            h->n_visible = cnt->n_visible;
            h->n_sorted = sorted;
            __threadfence_system();
            h->tag = tag;
        }
    }
}

// MODE 0: compaction of the Gaussians with keys into (depth bits, index).
// MODE 1: offs[s] = exclusive prefix of the key counts in depth order.
template <int MODE>
__global__ __launch_bounds__(kScanThreads) void scan_down_kernel(int n, const uint32_t *count,
                                                                 const uint32_t *didx,
                                                                 const Counters *cnt,
                                                                 const uint64_t *block_sums,
                                                                 const float4 *g1, uint32_t *out_a,
                                                                 uint32_t *out_b) {
    __shared__ uint64_t s_wave[4];
    const uint32_t first = blockIdx.x * (uint32_t)kScanTile + threadIdx.x * kScanItems;
    uint32_t v[kScanItems];
    load16<MODE>(first, n, count, didx, cnt, v);
    uint64_t local = 0;
#pragma unroll
    for (int j = 0; j < kScanItems; ++j) local += v[j];
    uint64_t tot;
    uint64_t run = block_sums[blockIdx.x] + block_exclusive_scan64(local, s_wave, &tot);
    if (MODE == 0) {
#pragma unroll
        for (int j = 0; j < kScanItems; ++j) {
            if (v[j]) {
                out_a[run] = __float_as_uint(g1[first + j].z);
                out_b[run] = first + j;
                ++run;
            }
        }
    } else {
        const uint32_t lim = cnt->n_visible;
        uint32_t o[kScanItems];
#pragma unroll
        for (int j = 0; j < kScanItems; ++j) {
            o[j] = (uint32_t)run;
            run += v[j];
        }
        if (first + kScanItems <= lim) {
#pragma unroll
            for (int j = 0; j < kScanItems; j += 4)
                *reinterpret_cast<uint4 *>(out_a + first + j) = make_uint4(o[j], o[j + 1], o[j + 2], o[j + 3]);
        } else {
#pragma unroll
            for (int j = 0; j < kScanItems; ++j)
                if (first + j < lim) out_a[first + j] = o[j];
        }
    }
}

// One output key per lane.  Wave w owns sorted positions [64w, 64w+64).
// Past the key capacity (cnt->n_sorted == 0 with keys) nothing is emitted:
// the host grows the buffers and renders the frame again.
__global__ __launch_bounds__(256) void duplicate_kernel(const Counters *cnt,
                                                        const uint32_t *__restrict__ didx,
                                                        const uint32_t *__restrict__ offs,
                                                        const ushort4 *__restrict__ rect,
                                                        const uint32_t *rowpre, const int *sel_cols,
                                                        int TX, int n_tiles, uint32_t *tkey,
                                                        uint32_t *tval, uint2 *ranges) {
    __shared__ uint32_t s_off[4][64];
    __shared__ uint32_t s_g[4][64];
    __shared__ ushort4 s_rect[4][64];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    for (int t = blockIdx.x * blockDim.x + threadIdx.x; t < n_tiles; t += gridDim.x * blockDim.x)
        ranges[t] = make_uint2(0u, 0u);
    const uint32_t V = cnt->n_visible, K = cnt->n_sorted;
    const uint32_t w0 = (blockIdx.x * 4u + (uint32_t)wave) * 64u;
    if (K == 0u || w0 >= V) return;
    const uint32_t s = w0 + lane;
    const uint32_t m = V - w0 < 64u ? V - w0 : 64u;
    if (s < V) {
        const uint32_t g = didx[s];
        s_off[wave][lane] = offs[s];
        s_g[wave][lane] = g;
        s_rect[wave][lane] = rect[g];
    }
    // the LDS arrays are private to the wave: a wave-level barrier suffices
    __builtin_amdgcn_wave_barrier();
    const uint32_t start = s_off[wave][0];
    const uint32_t end = w0 + 64u < V ? offs[w0 + 64u] : K;
    for (uint32_t p = start + lane; p < end; p += 64u) {
        // owner: the last j with s_off[j] <= p (offsets strictly increase)
        uint32_t lo = 0, hi = m - 1;
        while (lo < hi) {
            const uint32_t mid = (lo + hi + 1) >> 1;
            if (s_off[wave][mid] <= p) lo = mid;
            else hi = mid - 1;
        }
        uint32_t r = p - s_off[wave][lo];
        const ushort4 rc = s_rect[wave][lo];
        int tx, ty;
        if (!rowpre) {
            const uint32_t w = (uint32_t)(rc.z - rc.x + 1);
            ty = rc.y + (int)(r / w);
            tx = rc.x + (int)(r % w);
        } else {
            // r-th selected tile of the rectangle, rows first: O(1) per row
            ty = rc.y;
            const uint32_t *row = rowpre + (size_t)ty * (TX + 1);
            for (;; ++ty, row += TX + 1) {
                const uint32_t c = row[rc.z + 1] - row[rc.x];
                if (r < c) break;
                r -= c;
            }
            tx = sel_cols[(size_t)ty * TX + row[rc.x] + r];
        }
        tkey[p] = (uint32_t)(ty * TX + tx);
        tval[p] = s_g[wave][lo];
    }
}

__global__ __launch_bounds__(256) void ranges_zero_kernel(int n_tiles, uint2 *ranges) {
    const int t = blockIdx.x * blockDim.x + threadIdx.x;
    if (t < n_tiles) ranges[t] = make_uint2(0u, 0u);
}

__global__ __launch_bounds__(256) void ranges_kernel(const Counters *cnt, const uint32_t *keys,
                                                     uint2 *ranges) {
    const uint32_t K = cnt->n_sorted;
    for (uint32_t k = blockIdx.x * blockDim.x + threadIdx.x; k < K; k += gridDim.x * blockDim.x) {
        const uint32_t t = keys[k];
        if (k == 0 || keys[k - 1] != t) ranges[t].x = k;
        if (k == K - 1 || keys[k + 1] != t) ranges[t].y = k + 1;
    }
}

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

// Wave-aggregated LDS atomic: each distinct bucket of the wave takes one
// atomicAdd; returns this lane's slot (old value + rank among its peers).
__device__ inline uint32_t wave_bucket_add(uint32_t *s_cnt, uint32_t b, bool active) {
    const int lane = threadIdx.x & 63;
    const uint64_t lt_mask = (1ull << lane) - 1ull;
    uint64_t todo = __ballot(active);
    uint32_t slot = 0;
    while (todo) {
        const int leader = __ffsll((long long)todo) - 1;
        const uint32_t lb = __shfl(b, leader);
        const uint64_t peers = __ballot(active && b == lb);
        uint32_t base = 0;
        if (lane == leader) base = atomicAdd(&s_cnt[lb], (uint32_t)__popcll(peers));
        base = __shfl(base, leader);
        if (active && b == lb) slot = base + (uint32_t)__popcll(peers & lt_mask);
        todo &= ~peers;
    }
    return slot;
}

__global__ __launch_bounds__(1024) void order_tiles_kernel(int n_host, const uint32_t *n_dev,
                                                           const int *tile_in,
                                                           const uint2 *ranges, int *tile_out) {
    __shared__ uint32_t s_cnt[33];
    const int tid = threadIdx.x;
    const int n = n_dev ? (int)*n_dev : n_host;
    if (tid < 33) s_cnt[tid] = 0u;
    __syncthreads();
    // loop bounds are uniform over the block so that every lane takes part
    // in the wave-level aggregation
    for (int c = 0; c < n; c += 1024) {
        const int i = c + tid;
        const bool active = i < n;
        const uint32_t b = active ? length_bucket(ranges, tile_in ? tile_in[i] : i) : 0u;
        (void)wave_bucket_add(s_cnt, b, active);
    }
    __syncthreads();
    if (tid == 0) {
        uint32_t run = 0;
        for (int b = 32; b >= 0; --b) {
            const uint32_t c = s_cnt[b];
            s_cnt[b] = run;
            run += c;
        }
    }
    __syncthreads();
    for (int c = 0; c < n; c += 1024) {
        const int i = c + tid;
        const bool active = i < n;
        const int t = active ? (tile_in ? tile_in[i] : i) : 0;
        const uint32_t b = active ? length_bucket(ranges, t) : 0u;
        const uint32_t slot = wave_bucket_add(s_cnt, b, active);
        if (active) tile_out[slot] = t;
    }
}

inline uint32_t scan_parts(uint32_t n) { return (n + kScanTile - 1) / kScanTile; }

}  // namespace

size_t scan_scratch_bytes(int n) {
    return (size_t)(scan_parts((uint32_t)(n > 0 ? n : 1)) + 1) * sizeof(uint64_t);
}

void launch_count_masked(int n, const ushort4 *rect, const uint32_t *rowpre, int TX,
                         uint32_t *count, hipStream_t st) {
    if (n <= 0) return;
    count_masked_kernel<<<(n + 255) / 256, 256, 0, st>>>(n, rect, rowpre, TX, count);
}

void launch_visible_scans(int n, const uint32_t *count, const float4 *g1, uint32_t *dkey,
                          uint32_t *didx, void *scratch, const uint32_t *pre_partial,
                          Counters *cnt, hipStream_t st) {
    const uint32_t nb = scan_parts((uint32_t)(n > 0 ? n : 1));
    uint64_t *sums = static_cast<uint64_t *>(scratch);
    scan_reduce_kernel<0><<<nb, kScanThreads, 0, st>>>(n, count, nullptr, cnt, sums);
    scan_top_kernel<0><<<1, 1024, 0, st>>>((int)nb, sums, pre_partial,
                                           n > 0 ? preprocess_blocks(n) : 0, 0u, cnt, nullptr, 0u);
    scan_down_kernel<0><<<nb, kScanThreads, 0, st>>>(n, count, nullptr, cnt, sums, g1, dkey, didx);
}

void launch_sorted_count_scan(int n, const uint32_t *didx, const uint32_t *count, uint32_t *offs,
                              void *scratch, Counters *cnt, uint32_t cap, HostCounters *host,
                              uint32_t tag, hipStream_t st) {
    const uint32_t nb = scan_parts((uint32_t)(n > 0 ? n : 1));
    uint64_t *sums = static_cast<uint64_t *>(scratch);
    scan_reduce_kernel<1><<<nb, kScanThreads, 0, st>>>(n, count, didx, cnt, sums);
    scan_top_kernel<1><<<1, 1024, 0, st>>>((int)nb, sums, nullptr, 0, cap, cnt, host, tag);
    scan_down_kernel<1><<<nb, kScanThreads, 0, st>>>(n, count, didx, cnt, sums, nullptr, offs,
                                                     nullptr);
}

void launch_duplicate(int n, const Counters *cnt, const uint32_t *didx, const uint32_t *offs,
                      const ushort4 *rect, const uint32_t *rowpre, const int *sel_cols, int TX,
                      int n_tiles, uint32_t *tkey, uint32_t *tval, uint2 *ranges, hipStream_t st) {
    if (n <= 0) {
        ranges_zero_kernel<<<(n_tiles + 255) / 256, 256, 0, st>>>(n_tiles, ranges);
        return;
    }
    const uint32_t waves = ((uint32_t)n + 63) / 64;
    duplicate_kernel<<<(waves + 3) / 4, 256, 0, st>>>(cnt, didx, offs, rect, rowpre, sel_cols, TX,
                                                      n_tiles, tkey, tval, ranges);
}

void launch_ranges(uint32_t cap, const Counters *cnt, const uint32_t *keys, uint2 *ranges,
                   hipStream_t st) {
    // grid-stride over at most 2048 blocks: the key count is on the device
    const uint32_t blocks = (cap + 255) / 256 < 2048u ? (cap + 255) / 256 : 2048u;
    if (cap > 0) ranges_kernel<<<blocks, 256, 0, st>>>(cnt, keys, ranges);
}

void launch_order_tiles(int n, const uint32_t *n_dev, const int *tile_in, const uint2 *ranges,
                        int *tile_out, hipStream_t st) {
    if (n > 0) order_tiles_kernel<<<1, 1024, 0, st>>>(n, n_dev, tile_in, ranges, tile_out);
}

}  // namespace tgs
