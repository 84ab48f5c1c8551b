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

// Tile (tx, ty) of the r-th key of a Gaussian with tile rectangle rc:
// row-major over the rectangle, or (rowpre != NULL) over its selected tiles,
// rows first, O(1) per row from the per-row prefix sums of the tile mask.
__device__ inline void key_tile_xy(uint32_t r, ushort4 rc, const uint32_t *rowpre,
                                   const int *sel_cols, int TX, int &tx, int &ty) {
    if (!rowpre) {
        const uint32_t w = (uint32_t)(rc.z - rc.x + 1);
        ty = rc.y + (int)(r / w);
        tx = rc.x + (int)(r % w);
        return;
    }
    // four rows per step (eight independent loads), then the row holding the
    // r-th selected tile among them
    ty = rc.y;
    const size_t s = (size_t)(TX + 1);
    const uint32_t *row = rowpre + (size_t)ty * s;
    for (;;) {
        if (ty > (int)rc.w) {   // r past the Gaussian's count: cannot happen
            tx = rc.x;
            ty = rc.w;
            return;
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
            return;
        }
        r -= c[k];
        ty += 4;
        row += 4 * s;
    }
}

// Inputs of key generation: the cnt->n_visible Gaussians in emission order
// (didx), the start of each one's keys (offs, strictly increasing: every
// emitted Gaussian has keys), the owner of every kKeyBlock-th key (kfirst),
// and the tile rectangles / selection.
struct DupIo {
    const Counters *cnt;
    const uint32_t *didx;
    const uint32_t *offs;
    const uint32_t *kfirst;
    const ushort4 *rect;
    const uint32_t *rowpre;
    const int *sel_cols;
    int TX;
    int n_tiles;
    uint2 *ranges;   // cleared by the first kernel of the emission
    uint32_t *rows;  // optional: digit counts of each block's keys for the tile sort
    int row_bits;    // width of that digit (key bits [0, row_bits))
};

// Window of the Gaussians owning output positions [P0, P1) (P0 a multiple
// of kKeyBlock, P1 - P0 <= KD): from j0, the owner of P0, to the owner of
// P1 (the next block's first key) or, for the block holding the last key K,
// to the last Gaussian.  Entry k >= 1 starts at or after P0 + k (strictly
// increasing offsets), so at most KD entries can start before P1.
template <int KD>
__device__ inline void dup_window(const DupIo &io, uint32_t P0, uint32_t P1, uint32_t K,
                                  uint32_t V, uint32_t &j0, uint32_t &nw) {
    j0 = io.kfirst[P0 / kKeyBlock];
    const uint32_t jn = P1 < K ? io.kfirst[P1 / kKeyBlock] + 1u : V;
    nw = jn - j0 < (uint32_t)KD ? jn - j0 : (uint32_t)KD;
}

// Owners of the output positions [P0, P1) by a block of NT threads: s_off[k]
// / s_g[k] = start and Gaussian index of window entry k (those starting
// before P1), s_owner[i] = the window entry owning position P0 + i.  The
// window is read in one step (every load in flight at once).  Ends with a
// barrier.
template <int KD, int NT>
__device__ inline void dup_owners(const DupIo &io, uint32_t P0, uint32_t P1, uint32_t K,
                                  uint32_t V, int *s_owner, uint32_t *s_off, uint32_t *s_g,
                                  int *s_wmax) {
    static_assert(KD % NT == 0 && KD % kKeyBlock == 0, "whole steps and key blocks");
    constexpr int kPer = KD / NT;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    uint32_t j0, nw;
    dup_window<KD>(io, P0, P1, K, V, j0, nw);
    // clamped indices, no branches: every load is issued before the first wait
    uint32_t o[kPer], g[kPer];
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
        const uint32_t k = (uint32_t)(tid + NT * i), kc = k < nw ? k : nw - 1u;
        o[i] = io.offs[j0 + kc];
        g[i] = io.didx[j0 + kc];
    }
    for (int k = tid; k < KD; k += NT) s_owner[k] = -1;
    __syncthreads();
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
        const int k = tid + NT * i;
        if ((uint32_t)k < nw && (k == 0 || o[i] < P1)) {
            s_off[k] = o[i];
            s_g[k] = g[i];
            s_owner[k == 0 ? 0 : (int)(o[i] - P0)] = k;
        }
    }
    __syncthreads();
    // inclusive max-scan of the marks: kPer consecutive entries per thread
    int v[kPer], m = -1;
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
        m = max(m, s_owner[kPer * tid + i]);
        v[i] = m;
    }
    int inc = m;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const int t = __shfl_up(inc, d);
        if (lane >= d) inc = max(inc, t);
    }
    int ex = __shfl_up(inc, 1);
    if (lane == 0) ex = -1;
    if (lane == 63) s_wmax[wave] = inc;
    __syncthreads();
    for (int w = 0; w < wave; ++w) ex = max(ex, s_wmax[w]);
#pragma unroll
    for (int i = 0; i < kPer; ++i) s_owner[kPer * tid + i] = max(v[i], ex);
    __syncthreads();
}

// Block b emits output keys [1024 b, 1024 b + 1024), four per thread at
// consecutive positions across the block (coalesced stores), whatever the
// Gaussians' key counts: a Gaussian spanning thousands of tiles is spread
// over many blocks instead of holding one wave.  Owners of the positions
// come from the key-block table and the window of Gaussians starting inside
// the block (dup_owners).  Past the key capacity (cnt->n_sorted == 0 with
// keys) nothing is emitted: the host grows the buffers and renders the
// frame again.  With io.rows, the block also counts its keys' first
// tile-sort digit into row blockIdx.x (LDS counters per wave), so that the
// sort's first pass needs no counting launch of its own.
constexpr int kDupKeys = kKeyBlock;

__global__ __launch_bounds__(256) void duplicate_kernel(DupIo io, uint32_t *tkey, uint32_t *tval) {
    __shared__ int s_owner[kDupKeys];
    __shared__ uint32_t s_off[kDupKeys];
    __shared__ uint32_t s_g[kDupKeys];
    __shared__ int s_wmax[4];
    __shared__ uint32_t s_hist[4][256];
    const int tid = threadIdx.x;
    for (int t = blockIdx.x * blockDim.x + tid; t < io.n_tiles; t += gridDim.x * blockDim.x)
        io.ranges[t] = make_uint2(0u, 0u);
    const uint32_t V = io.cnt->n_visible, K = io.cnt->n_sorted;
    const uint32_t P0 = blockIdx.x * (uint32_t)kDupKeys;
    if (K == 0u || P0 >= K) return;   // block-uniform
    if (io.rows) {
#pragma unroll
        for (int w = 0; w < 4; ++w) s_hist[w][tid] = 0u;   // ordered by dup_owners' barriers
    }
    const uint32_t P1 = K - P0 < (uint32_t)kDupKeys ? K : P0 + kDupKeys;
    dup_owners<kDupKeys, 256>(io, P0, P1, K, V, s_owner, s_off, s_g, s_wmax);
    // positions past the keys take the last key's owner (no branch before
    // the stores, so every rectangle load is in flight together)
    constexpr int kPer = kDupKeys / 256;
    uint32_t g[kPer], r[kPer];
    ushort4 rc[kPer];
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
        const uint32_t p = P0 + (uint32_t)(tid + 256 * k), pc = p < P1 ? p : P1 - 1u;
        const int w = s_owner[pc - P0];
        g[k] = s_g[w];
        r[k] = pc - s_off[w];
        rc[k] = io.rect[g[k]];
    }
#pragma unroll
    for (int k = 0; k < kPer; ++k) {
        const uint32_t p = P0 + (uint32_t)(tid + 256 * k);
        int tx, ty;
        key_tile_xy(r[k], rc[k], io.rowpre, io.sel_cols, io.TX, tx, ty);
        if (p < P1) {
            const uint32_t key = (uint32_t)(ty * io.TX + tx);
            tkey[p] = key;
            tval[p] = g[k];
            if (io.rows) atomicAdd(&s_hist[tid >> 6][key & ((1u << io.row_bits) - 1u)], 1u);
        }
    }
    if (io.rows) {
        __syncthreads();
        io.rows[(size_t)blockIdx.x * 256 + tid] = s_hist[0][tid] + s_hist[1][tid] + s_hist[2][tid] +
                                                  s_hist[3][tid];
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
    __shared__ uint32_t s_cnt[order_lds_words(1024)];
    order_tiles_block<1024, true>(o, s_cnt);
}

}  // namespace

void launch_duplicate(int n, uint32_t cap, const Counters *cnt, const uint32_t *didx,
                      const uint32_t *offs, const uint32_t *kfirst, const ushort4 *rect,
                      const uint32_t *rowpre, const int *sel_cols, int TX, int n_tiles,
                      uint32_t *tkey, uint32_t *tval, uint2 *ranges, uint32_t *rows, int row_bits,
                      hipStream_t st) {
    if (n <= 0 || cap == 0) {
        ranges_zero_kernel<<<(n_tiles + 255) / 256, 256, 0, st>>>(n_tiles, ranges);
        return;
    }
    const uint32_t blocks = (cap + kDupKeys - 1) / kDupKeys;
    const DupIo io{cnt, didx, offs, kfirst, rect, rowpre, sel_cols, TX, n_tiles, ranges,
                   row_bits > 0 ? rows : nullptr, row_bits};
    duplicate_kernel<<<blocks, 256, 0, st>>>(io, tkey, tval);
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
