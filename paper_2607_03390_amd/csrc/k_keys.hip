// Gaussian-tile duplication (Sec. III-A) around the two sorts of a frame:
//  - key emission in depth order, a fixed slice of output keys per block with
//    coalesced stores (owners from a search over the sorted offsets and an
//    LDS max-scan);
//  - per-tile [start, end) ranges of the tile-sorted keys and the blend
//    order of the tiles.
// Counts stay on the device, so nothing here needs a host round trip.
#include "order.h"
#include "tgs_internal.h"

namespace tgs {

namespace {


// Tile of the r-th key of a Gaussian with tile rectangle rc: row-major over
// the rectangle, or (rowpre != NULL) over its selected tiles, rows first,
// O(1) per row from the per-row prefix sums of the tile mask.
__device__ inline uint32_t key_tile(uint32_t r, ushort4 rc, const uint32_t *rowpre,
                                    const int *sel_cols, int TX) {
    int tx, ty;
    if (!rowpre) {
        const uint32_t w = (uint32_t)(rc.z - rc.x + 1);
        ty = rc.y + (int)(r / w);
        tx = rc.x + (int)(r % w);
    } else {
        // four rows per step (eight independent loads), then the row
        // holding the r-th selected tile among them
        ty = rc.y;
        const size_t s = (size_t)(TX + 1);
        const uint32_t *row = rowpre + (size_t)ty * s;
        for (;;) {
            if (ty > (int)rc.w) {   // r past the Gaussian's count: cannot happen
                tx = rc.x;
                ty = rc.w;
                break;
            }
            uint32_t c[4], b[4];
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const bool in = ty + k <= (int)rc.w;
                b[k] = in ? row[k * s + rc.x] : 0u;
                c[k] = in ? row[k * s + rc.z + 1] - b[k] : 0u;
            }
            int k = 0;
            while (k < 3 && r >= c[k]) {
                r -= c[k];
                ++k;
            }
            if (r < c[k]) {
                ty += k;
                tx = sel_cols[(size_t)ty * TX + b[k] + r];
                break;
            }
            r -= c[k];
            ty += 4;
            row += 4 * s;
        }
    }
    return (uint32_t)(ty * TX + tx);
}

// Block b emits output keys [1024 b, 1024 b + 1024), four per thread at
// consecutive positions across the block (coalesced stores), whatever the
// Gaussians' key counts: a Gaussian spanning thousands of tiles is spread
// over many blocks instead of holding one wave.  The owner of the block's
// first key comes from the key-block table written with the offsets; the
// Gaussians starting inside the block mark their first position in LDS and
// an inclusive max-scan gives every position its owner.  Past the key
// capacity (cnt->n_sorted == 0 with keys) nothing is emitted: the host grows
// the buffers and renders the frame again.
constexpr int kDupKeys = kKeyBlock;
static_assert(kDupKeys % 256 == 0, "whole keys per thread");

__global__ __launch_bounds__(256) void duplicate_kernel(const Counters *cnt,
                                                        const uint32_t *__restrict__ didx,
                                                        const uint32_t *__restrict__ offs,
                                                        const uint32_t *__restrict__ kfirst,
                                                        const ushort4 *__restrict__ rect,
                                                        const uint32_t *rowpre, const int *sel_cols,
                                                        int TX, int n_tiles, uint32_t *tkey,
                                                        uint32_t *tval, uint2 *ranges) {
    __shared__ int s_owner[kDupKeys];           // window index of each position's owner
    __shared__ uint32_t s_off[kDupKeys + 1];    // offsets of window Gaussians j0 + k
    __shared__ uint32_t s_g[kDupKeys + 1];      // their Gaussian indices
    __shared__ int s_wmax[4];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    for (int t = blockIdx.x * blockDim.x + tid; t < n_tiles; t += gridDim.x * blockDim.x)
        ranges[t] = make_uint2(0u, 0u);
    const uint32_t V = cnt->n_visible, K = cnt->n_sorted;
    const uint32_t P0 = blockIdx.x * (uint32_t)kDupKeys;
    if (K == 0u || P0 >= K) return;   // block-uniform
    const uint32_t P1 = K - P0 < (uint32_t)kDupKeys ? K : P0 + kDupKeys;
    for (int k = tid; k < kDupKeys; k += 256) s_owner[k] = -1;
    const uint32_t j0 = kfirst[blockIdx.x];   // owner of key P0 (offs[j0] <= P0)
    __syncthreads();
    // at most kDupKeys Gaussians after j0 start inside the block's keys
    for (int k = tid; k <= kDupKeys; k += 256) {
        const uint32_t j = j0 + (uint32_t)k;
        if (j < V) {
            const uint32_t o = offs[j];
            s_off[k] = o;
            s_g[k] = didx[j];
            if (k == 0) s_owner[0] = 0;
            else if (o < P1) s_owner[o - P0] = k;
        }
    }
    __syncthreads();
    // inclusive max-scan of the marks: kPer consecutive entries per thread
    constexpr int kPer = kDupKeys / 256;
    int v[kPer], m = -1;
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
        m = max(m, s_owner[kPer * tid + i]);
        v[i] = m;
    }
    int inc = m;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const int o = __shfl_up(inc, d);
        if (lane >= d) inc = max(inc, o);
    }
    int ex = __shfl_up(inc, 1);
    if (lane == 0) ex = -1;
    if (lane == 63) s_wmax[wave] = inc;
    __syncthreads();
    for (int w = 0; w < wave; ++w) ex = max(ex, s_wmax[w]);
#pragma unroll
    for (int i = 0; i < kPer; ++i) s_owner[kPer * tid + i] = max(v[i], ex);
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
        const uint32_t i = (uint32_t)(tid + 256 * k);
        const uint32_t p = P0 + i;
        if (p < P1) {
            const int w = s_owner[i];
            const uint32_t g = s_g[w];
            tkey[p] = key_tile(p - s_off[w], rect[g], rowpre, sel_cols, TX);
            tval[p] = g;
        }
    }
}

__global__ __launch_bounds__(256) void ranges_zero_kernel(int n_tiles, uint2 *ranges) {
    const int t = blockIdx.x * blockDim.x + threadIdx.x;
    if (t < n_tiles) ranges[t] = make_uint2(0u, 0u);
}

// Four consecutive sorted keys per thread (one 16-byte load) and the key on
// either side: the thread writes the start / end of every tile run that
// begins / ends among its four.
__global__ __launch_bounds__(256) void ranges_kernel(const Counters *cnt, const uint32_t *keys,
                                                     uint2 *ranges) {
    const uint64_t K = cnt->n_sorted;
    const uint64_t G = (K + 3) / 4;
    for (uint64_t g = blockIdx.x * (uint64_t)blockDim.x + threadIdx.x; g < G;
         g += (uint64_t)gridDim.x * blockDim.x) {
        const uint64_t k0 = 4 * g;
        uint32_t t[4];
        if (k0 + 4 <= K) {
            const uint4 v = *reinterpret_cast<const uint4 *>(keys + k0);
            t[0] = v.x;
            t[1] = v.y;
            t[2] = v.z;
            t[3] = v.w;
        } else {
#pragma unroll
            for (int j = 0; j < 4; ++j) t[j] = k0 + j < K ? keys[k0 + j] : 0xffffffffu;
        }
        const uint32_t prev = k0 > 0 ? keys[k0 - 1] : 0xffffffffu;
        const uint32_t next = k0 + 4 < K ? keys[k0 + 4] : 0xffffffffu;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const uint64_t k = k0 + j;
            if (k >= K) break;
            const uint32_t tp = j == 0 ? prev : t[j - 1];
            const uint32_t tn = j == 3 ? next : t[j + 1];
            if (k == 0 || tp != t[j]) ranges[t[j]].x = (uint32_t)k;
            if (k == K - 1 || tn != t[j]) ranges[t[j]].y = (uint32_t)(k + 1);
        }
    }
}

__global__ __launch_bounds__(1024) void order_tiles_kernel(OrderK o) {
    __shared__ uint32_t s_cnt[33];
    order_tiles_block<1024>(o, s_cnt);
}

}  // namespace

void launch_duplicate(int n, uint32_t cap, const Counters *cnt, const uint32_t *didx,
                      const uint32_t *offs, const uint32_t *kfirst, const ushort4 *rect,
                      const uint32_t *rowpre, const int *sel_cols, int TX, int n_tiles,
                      uint32_t *tkey, uint32_t *tval, uint2 *ranges, hipStream_t st) {
    if (n <= 0 || cap == 0) {
        ranges_zero_kernel<<<(n_tiles + 255) / 256, 256, 0, st>>>(n_tiles, ranges);
        return;
    }
    const uint32_t blocks = (cap + kDupKeys - 1) / kDupKeys;
    duplicate_kernel<<<blocks, 256, 0, st>>>(cnt, didx, offs, kfirst, rect, rowpre, sel_cols, TX,
                                             n_tiles, tkey, tval, ranges);
}

void launch_ranges(uint32_t cap, const Counters *cnt, const uint32_t *keys, uint2 *ranges,
                   hipStream_t st) {
    // sized for the key capacity (the key count is on the device), at most
    // 65535 blocks, grid-stride beyond
    const uint64_t groups = ((uint64_t)cap + 3) / 4;
    const uint32_t blocks = (uint32_t)((groups + 255) / 256 < 65535u ? (groups + 255) / 256 : 65535u);
    if (cap > 0) ranges_kernel<<<blocks, 256, 0, st>>>(cnt, keys, ranges);
}

void launch_order_tiles(const OrderK &o, hipStream_t st) {
    if (o.n_host > 0) order_tiles_kernel<<<1, 1024, 0, st>>>(o);
}

}  // namespace tgs
