// Gaussian-tile duplication (Sec. III-A): per-Gaussian key counts, their
// exclusive scan, key emission and per-tile ranges of the sorted keys.
//
// A Gaussian's count is the number of tiles of its rectangle, or, in a
// selective-rendering frame, the number of selected tiles of its rectangle,
// taken from per-row prefix sums of the tile mask (one subtraction per row).
// The scan is a deterministic reduce-then-scan over 4096-Gaussian blocks;
// keys are emitted in Gaussian index order, so a stable radix sort breaks
// depth ties by index.
#include "tgs_internal.h"

namespace tgs {

namespace {

constexpr int kScanThreads = 256;
constexpr int kScanItems = 16;
constexpr int kScanBlock = kScanThreads * kScanItems;

__device__ inline uint32_t tile_count(ushort4 r, const uint32_t *rowpre, int TX) {
    if (r.x > r.z || r.y > r.w) return 0u;
    if (!rowpre) return (uint32_t)(r.z - r.x + 1) * (uint32_t)(r.w - r.y + 1);
    uint32_t c = 0;
    for (int y = r.y; y <= r.w; ++y) {
        const uint32_t *row = rowpre + (size_t)y * (TX + 1);
        c += row[r.z + 1] - row[r.x];
    }
    return c;
}

// inclusive scan over the 64 lanes of a wave
__device__ inline uint32_t wave_inclusive_scan(uint32_t v) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const uint32_t o = __shfl_up(v, d);
        if (lane >= d) v += o;
    }
    return v;
}

// exclusive scan over a 256-thread block; returns the block total in *total
__device__ inline uint32_t block_exclusive_scan(uint32_t v, uint32_t *s_wave, uint32_t *total) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const uint32_t inc = wave_inclusive_scan(v);
    if (lane == 63) s_wave[wave] = inc;
    __syncthreads();
    uint32_t off = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
        const uint32_t x = s_wave[w];
        if (w < wave) off += x;
        tot += x;
    }
    __syncthreads();
    *total = tot;
    return off + inc - v;
}

__global__ __launch_bounds__(kScanThreads) void scan_reduce_kernel(int n, const ushort4 *rect,
                                                                   const uint32_t *rowpre, int TX,
                                                                   uint64_t *block_sums) {
    __shared__ uint32_t s_wave[4];
    const int base = blockIdx.x * kScanBlock;
    uint64_t sum = 0;
    for (int j = 0; j < kScanItems; ++j) {
        const int i = base + j * kScanThreads + threadIdx.x;
        if (i < n) sum += tile_count(rect[i], rowpre, TX);
    }
    // 64-bit block reduction
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int d = 32; d >= 1; d >>= 1) sum += __shfl_down(sum, d);
    __shared__ uint64_t s_sum[4];
    if (lane == 0) s_sum[wave] = sum;
    __syncthreads();
    if (threadIdx.x == 0) block_sums[blockIdx.x] = s_sum[0] + s_sum[1] + s_sum[2] + s_sum[3];
    (void)s_wave;
}

// single block: exclusive scan of the block sums in place, total -> counters
__global__ __launch_bounds__(1024) void scan_top_kernel(int nb, uint64_t *block_sums,
                                                        Counters *cnt) {
    __shared__ uint64_t s_wave[16];
    __shared__ uint64_t s_carry;
    if (threadIdx.x == 0) s_carry = 0;
    __syncthreads();
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
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
        const uint64_t K = s_carry;
        cnt->n_keys = K > 0xffffffffull ? 0xffffffffu : (uint32_t)K;
    }
}

__global__ __launch_bounds__(kScanThreads) void scan_down_kernel(int n, const ushort4 *rect,
                                                                 const uint32_t *rowpre, int TX,
                                                                 const uint64_t *block_sums,
                                                                 uint32_t *offsets) {
    __shared__ uint32_t s_wave[4];
    const int base = blockIdx.x * kScanBlock;
    uint64_t run = block_sums[blockIdx.x];
    for (int j = 0; j < kScanItems; ++j) {
        const int i = base + j * kScanThreads + threadIdx.x;
        const uint32_t c = i < n ? tile_count(rect[i], rowpre, TX) : 0u;
        uint32_t tot;
        const uint32_t ex = block_exclusive_scan(c, s_wave, &tot);
        if (i < n) offsets[i] = (uint32_t)(run + ex);
        run += tot;
    }
}

__global__ __launch_bounds__(256) void duplicate_kernel(int n, const ushort4 *rect, const float4 *g1,
                                                        const uint32_t *offsets, const uint8_t *sel,
                                                        int TX, uint64_t *keys, uint32_t *vals) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const ushort4 r = rect[i];
    if (r.x > r.z || r.y > r.w) return;
    const uint64_t dbits = (uint64_t)__float_as_uint(g1[i].z);
    uint32_t o = offsets[i];
    for (int y = r.y; y <= r.w; ++y)
        for (int x = r.x; x <= r.z; ++x) {
            const uint32_t t = (uint32_t)(y * TX + x);
            if (sel && !sel[t]) continue;
            keys[o] = ((uint64_t)t << 32) | dbits;
            vals[o] = (uint32_t)i;
            ++o;
        }
}

__global__ __launch_bounds__(256) void ranges_zero_kernel(int n_tiles, uint2 *ranges) {
    const int t = blockIdx.x * blockDim.x + threadIdx.x;
    if (t < n_tiles) ranges[t] = make_uint2(0u, 0u);
}

__global__ __launch_bounds__(256) void ranges_kernel(uint32_t K, const uint64_t *keys,
                                                     uint2 *ranges) {
    const uint32_t k = blockIdx.x * blockDim.x + threadIdx.x;
    if (k >= K) return;
    const uint32_t t = (uint32_t)(keys[k] >> 32);
    if (k == 0 || (uint32_t)(keys[k - 1] >> 32) != t) ranges[t].x = k;
    if (k == K - 1 || (uint32_t)(keys[k + 1] >> 32) != t) ranges[t].y = k + 1;
}

}  // namespace

size_t scan_scratch_words(int n) {
    // block sums are 64-bit
    return 2 * (size_t)((n + kScanBlock - 1) / kScanBlock + 1);
}

void launch_scan(int n, const ushort4 *rect, const uint32_t *rowpre, int TX, uint32_t *offsets,
                 uint32_t *scratch, Counters *cnt, hipStream_t st) {
    uint64_t *block_sums = reinterpret_cast<uint64_t *>(scratch);
    const int nb = (n + kScanBlock - 1) / kScanBlock;
    if (nb > 0)
        scan_reduce_kernel<<<nb, kScanThreads, 0, st>>>(n, rect, rowpre, TX, block_sums);
    scan_top_kernel<<<1, 1024, 0, st>>>(nb, block_sums, cnt);
    if (nb > 0)
        scan_down_kernel<<<nb, kScanThreads, 0, st>>>(n, rect, rowpre, TX, block_sums, offsets);
}

void launch_duplicate(int n, const ushort4 *rect, const float4 *g1, const uint32_t *offsets,
                      const uint8_t *sel, int TX, uint64_t *keys, uint32_t *vals, hipStream_t st) {
    if (n <= 0) return;
    duplicate_kernel<<<(n + 255) / 256, 256, 0, st>>>(n, rect, g1, offsets, sel, TX, keys, vals);
}

void launch_ranges(uint32_t K, int n_tiles, const uint64_t *keys, uint2 *ranges, hipStream_t st) {
    ranges_zero_kernel<<<(n_tiles + 255) / 256, 256, 0, st>>>(n_tiles, ranges);
    if (K > 0) ranges_kernel<<<(K + 255) / 256, 256, 0, st>>>(K, keys, ranges);
}

}  // namespace tgs
