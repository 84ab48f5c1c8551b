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
// The scans are single-pass chained scans (decoupled look-back over
// 4096-element partitions numbered by an atomic ticket); their totals stay on
// the device, so the sorts need no host round trip.
#include "tgs_internal.h"

namespace tgs {

namespace {

constexpr int kScanThreads = 256;
constexpr int kScanItems = 16;
constexpr int kScanTile = kScanThreads * kScanItems;   // 4096
constexpr uint64_t kSFlagAgg = 1ull << 62;
constexpr uint64_t kSFlagInc = 2ull << 62;
constexpr uint64_t kSValMask = (1ull << 62) - 1;

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

__device__ inline uint64_t ld_agent64(const uint64_t *p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline void st_agent64(uint64_t *p, uint64_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
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

// Partition prefix by decoupled look-back (one lane per block does the walk).
__device__ inline uint64_t chained_prefix(uint64_t *status, uint32_t part, uint64_t block_total,
                                          uint64_t *s_prefix) {
    if (threadIdx.x == 0) {
        uint64_t excl = 0;
        if (part == 0) {
            st_agent64(status, kSFlagInc | block_total);
        } else {
            st_agent64(status + part, kSFlagAgg | block_total);
            int p = (int)part - 1;
            while (true) {
                const uint64_t w = ld_agent64(status + p);
                const uint64_t flag = w & ~kSValMask;
                if (flag == 0) {
                    __builtin_amdgcn_s_sleep(1);
                    continue;
                }
                excl += w & kSValMask;
                if (flag == kSFlagInc) break;
                --p;
            }
            st_agent64(status + part, kSFlagInc | (excl + block_total));
        }
        *s_prefix = excl;
    }
    __syncthreads();
    return *s_prefix;
}

// Compacts the Gaussians with count > 0, in index order, into
// (depth bits, index) pairs; the number of such Gaussians goes to
// cnt->n_visible.
__global__ __launch_bounds__(kScanThreads) void compact_visible_kernel(
    int n, const uint32_t *__restrict__ count, const float4 *__restrict__ g1, uint32_t *dkey,
    uint32_t *didx, uint64_t *status, uint32_t *ticket, Counters *cnt) {
    __shared__ uint64_t s_wave[4];
    __shared__ uint64_t s_prefix;
    __shared__ uint32_t s_part;
    if (threadIdx.x == 0) s_part = atomicAdd(ticket, 1u);
    __syncthreads();
    const uint32_t part = s_part;
    const uint32_t base = part * (uint32_t)kScanTile;
    if (base >= (uint32_t)n) {
        if (part == 0 && threadIdx.x == 0) cnt->n_visible = 0u;
        return;
    }
    const uint32_t first = base + threadIdx.x * kScanItems;
    uint32_t flags = 0, local = 0;
#pragma unroll
    for (int j = 0; j < kScanItems; j += 4) {
        const uint32_t i = first + j;
        uint4 c = make_uint4(0u, 0u, 0u, 0u);
        if (i + 3 < (uint32_t)n) {
            c = *reinterpret_cast<const uint4 *>(count + i);
        } else {
            if (i < (uint32_t)n) c.x = count[i];
            if (i + 1 < (uint32_t)n) c.y = count[i + 1];
            if (i + 2 < (uint32_t)n) c.z = count[i + 2];
        }
        const uint32_t f = (c.x > 0u ? 1u : 0u) | (c.y > 0u ? 2u : 0u) | (c.z > 0u ? 4u : 0u) |
                           (c.w > 0u ? 8u : 0u);
        flags |= f << j;
    }
    local = (uint32_t)__popc(flags);
    uint64_t block_total;
    const uint64_t texcl = block_exclusive_scan64(local, s_wave, &block_total);
    const uint64_t prefix = chained_prefix(status, part, block_total, &s_prefix);
    uint32_t pos = (uint32_t)(prefix + texcl);
#pragma unroll
    for (int j = 0; j < kScanItems; ++j) {
        if (flags & (1u << j)) {
            const uint32_t i = first + j;
            dkey[pos] = __float_as_uint(g1[i].z);
            didx[pos] = i;
            ++pos;
        }
    }
    if (base + kScanTile >= (uint32_t)n && threadIdx.x == 0)
        cnt->n_visible = (uint32_t)(prefix + block_total);
}

// Exclusive scan of the key counts in depth order: offs[s] for the sorted
// position s of Gaussian didx[s]; total -> cnt->n_keys (saturated).
__global__ __launch_bounds__(kScanThreads) void scan_sorted_counts_kernel(
    const uint32_t *__restrict__ didx, const uint32_t *__restrict__ count, uint32_t *offs,
    uint64_t *status, uint32_t *ticket, Counters *cnt) {
    __shared__ uint64_t s_wave[4];
    __shared__ uint64_t s_prefix;
    __shared__ uint32_t s_part;
    if (threadIdx.x == 0) s_part = atomicAdd(ticket, 1u);
    __syncthreads();
    const uint32_t n = cnt->n_visible;
    const uint32_t part = s_part;
    const uint32_t base = part * (uint32_t)kScanTile;
    if (base >= n) {
        if (part == 0 && threadIdx.x == 0) cnt->n_keys = 0u;
        return;
    }
    const uint32_t first = base + threadIdx.x * kScanItems;
    uint32_t c[kScanItems];
    uint64_t local = 0;
#pragma unroll
    for (int j = 0; j < kScanItems; ++j) {
        const uint32_t s = first + j;
        c[j] = s < n ? count[didx[s]] : 0u;
        local += c[j];
    }
    uint64_t block_total;
    const uint64_t texcl = block_exclusive_scan64(local, s_wave, &block_total);
    const uint64_t prefix = chained_prefix(status, part, block_total, &s_prefix);
    uint64_t run = prefix + texcl;
#pragma unroll
    for (int j = 0; j < kScanItems; ++j) {
        const uint32_t s = first + j;
        if (s < n) offs[s] = (uint32_t)run;
        run += c[j];
    }
    if (base + kScanTile >= n && threadIdx.x == 0) {
        const uint64_t K = prefix + block_total;
        cnt->n_keys = K > 0xffffffffull ? 0xffffffffu : (uint32_t)K;
    }
}

// One output key per lane.  Wave w owns sorted positions [64w, 64w+64).
__global__ __launch_bounds__(256) void duplicate_kernel(uint32_t V, uint32_t K,
                                                        const uint32_t *__restrict__ didx,
                                                        const uint32_t *__restrict__ offs,
                                                        const ushort4 *__restrict__ rect,
                                                        const uint32_t *rowpre, int TX,
                                                        uint32_t *tkey, uint32_t *tval) {
    __shared__ uint32_t s_off[4][64];
    __shared__ uint32_t s_g[4][64];
    __shared__ ushort4 s_rect[4][64];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const uint32_t w0 = (blockIdx.x * 4u + (uint32_t)wave) * 64u;
    if (w0 >= V) return;
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
            ty = rc.y;
            for (;; ++ty) {
                const uint32_t *row = rowpre + (size_t)ty * (TX + 1);
                const uint32_t c = row[rc.z + 1] - row[rc.x];
                if (r < c) break;
                r -= c;
            }
            const uint32_t *row = rowpre + (size_t)ty * (TX + 1);
            const uint32_t b = row[rc.x];
            int xl = rc.x, xh = rc.z;   // smallest x with row[x+1] - b > r
            while (xl < xh) {
                const int mid = (xl + xh) >> 1;
                if (row[mid + 1] - b > r) xh = mid;
                else xl = mid + 1;
            }
            tx = xl;
        }
        tkey[p] = (uint32_t)(ty * TX + tx);
        tval[p] = s_g[wave][lo];
    }
}

__global__ __launch_bounds__(256) void ranges_zero_kernel(int n_tiles, uint2 *ranges) {
    const int t = blockIdx.x * blockDim.x + threadIdx.x;
    if (t < n_tiles) ranges[t] = make_uint2(0u, 0u);
}

__global__ __launch_bounds__(256) void ranges_kernel(uint32_t K, const uint32_t *keys,
                                                     uint2 *ranges) {
    const uint32_t k = blockIdx.x * blockDim.x + threadIdx.x;
    if (k >= K) return;
    const uint32_t t = keys[k];
    if (k == 0 || keys[k - 1] != t) ranges[t].x = k;
    if (k == K - 1 || keys[k + 1] != t) ranges[t].y = k + 1;
}

__global__ __launch_bounds__(256) void clear64_kernel(uint64_t *p, size_t n) {
    for (size_t k = blockIdx.x * (size_t)blockDim.x + threadIdx.x; k < n;
         k += (size_t)gridDim.x * blockDim.x)
        p[k] = 0ull;
}

inline uint32_t scan_parts(uint32_t n) { return (n + kScanTile - 1) / kScanTile; }

}  // namespace

size_t scan_scratch_bytes(int n) {
    // two chained scans: status words + tickets for each
    const size_t parts = scan_parts((uint32_t)(n > 0 ? n : 1)) + 1;
    return 2 * (parts + 1) * sizeof(uint64_t);
}

void launch_count_masked(int n, const ushort4 *rect, const uint32_t *rowpre, int TX,
                         uint32_t *count, hipStream_t st) {
    if (n <= 0) return;
    count_masked_kernel<<<(n + 255) / 256, 256, 0, st>>>(n, rect, rowpre, TX, count);
}

void launch_visible_scans(int n, const uint32_t *count, const float4 *g1, uint32_t *dkey,
                          uint32_t *didx, void *scratch, Counters *cnt, hipStream_t st) {
    const uint32_t parts = scan_parts((uint32_t)(n > 0 ? n : 1));
    uint64_t *status = static_cast<uint64_t *>(scratch);
    const size_t words = 2 * ((size_t)parts + 2);
    clear64_kernel<<<(unsigned)((words + 255) / 256), 256, 0, st>>>(status, words);
    uint32_t *ticket = reinterpret_cast<uint32_t *>(status + parts + 1);
    compact_visible_kernel<<<parts, kScanThreads, 0, st>>>(n, count, g1, dkey, didx, status,
                                                           ticket, cnt);
}

void launch_sorted_count_scan(int n, const uint32_t *didx, const uint32_t *count, uint32_t *offs,
                              void *scratch, Counters *cnt, hipStream_t st) {
    const uint32_t parts = scan_parts((uint32_t)(n > 0 ? n : 1));
    uint64_t *status = static_cast<uint64_t *>(scratch) + parts + 2;
    uint32_t *ticket = reinterpret_cast<uint32_t *>(status + parts + 1);
    scan_sorted_counts_kernel<<<parts, kScanThreads, 0, st>>>(didx, count, offs, status, ticket, cnt);
}

void launch_duplicate(uint32_t V, uint32_t K, const uint32_t *didx, const uint32_t *offs,
                      const ushort4 *rect, const uint32_t *rowpre, int TX, uint32_t *tkey,
                      uint32_t *tval, hipStream_t st) {
    if (V == 0 || K == 0) return;
    const uint32_t waves = (V + 63) / 64;
    duplicate_kernel<<<(waves + 3) / 4, 256, 0, st>>>(V, K, didx, offs, rect, rowpre, TX, tkey, tval);
}

void launch_ranges(uint32_t K, int n_tiles, const uint32_t *keys, uint2 *ranges, hipStream_t st) {
    ranges_zero_kernel<<<(n_tiles + 255) / 256, 256, 0, st>>>(n_tiles, ranges);
    if (K > 0) ranges_kernel<<<(K + 255) / 256, 256, 0, st>>>(K, keys, ranges);
}

}  // namespace tgs
