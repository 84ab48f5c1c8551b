// Temporal kernels of a TemporalGS frame (Sec. III-C..E):
//  - forward warp of the temporal geometry buffer into the current view
//    (Eq. 3): nearest destination pixel, minimum depth and maximum standard
//    deviation by integer atomics on the float bits (both are non-negative,
//    so unsigned order is float order and the result is order-independent);
//  - depth fill, backward correspondence query and unmatched tiles, one
//    block per tile with a block-wide OR (fill_query.h; with the
//    full-resolution geometry buffer the preprocess launch runs it);
//  - occluded tiles of the newly visible Gaussians, one wave per
//    (Gaussian, tile) pair with a wave ballot over the tile's 256 pixels,
//    the pairs of 1024 Gaussians dealt out over the four waves of a block;
//  - tile selection and compaction in one launch, one block per tile row,
//    including the per-row prefix sums of the mask used by the key counts.
// (The stitching of the tiles that are not re-rendered, Eq. 4, runs in the
// blend launch: stitch.h.)
// All of these are HBM- or latency-bound; none is a dense contraction.
#include "fill_query.h"
#include "tgs_internal.h"

namespace tgs {

namespace {

__global__ __launch_bounds__(256) void temporal_init_kernel(int n_px, float *dmin, float *smax) {
    const int k = blockIdx.x * blockDim.x + threadIdx.x;
    if (k < n_px) {
        dmin[k] = kNoHit;
        smax[k] = 0.0f;
    }
}

__global__ __launch_bounds__(256) void forward_warp_kernel(WarpK w, const float *__restrict__ D,
                                                           const float *__restrict__ S, float *dmin,
                                                           float *smax) {
    const int q = blockIdx.x * blockDim.x + threadIdx.x;
    if (q >= w.W * w.H) return;
    const float d = D[q];
    if (d == kNoHit) return;
    const int x = q % w.W, y = q / w.W;
    const float rx = ((float)x - w.kref[2]) / w.kref[0];
    const float ry = ((float)y - w.kref[3]) / w.kref[1];
    const float Px = d * rx, Py = d * ry, Pz = d;
    const float *M = w.M;
    const float X = ((M[0] * Px + M[1] * Py) + M[2] * Pz) + M[3];
    const float Y = ((M[4] * Px + M[5] * Py) + M[6] * Pz) + M[7];
    const float Z = ((M[8] * Px + M[9] * Py) + M[10] * Pz) + M[11];
    if (!(Z > w.z_near)) return;
    const float u = w.kcur[0] * (X / Z) + w.kcur[2];
    const float v = w.kcur[1] * (Y / Z) + w.kcur[3];
    const float xf = floorf(u + 0.5f), yf = floorf(v + 0.5f);
    if (!(xf >= 0.0f && xf <= (float)(w.W - 1) && yf >= 0.0f && yf <= (float)(w.H - 1))) return;
    const int p = (int)yf * w.W + (int)xf;
    atomicMin(reinterpret_cast<unsigned int *>(dmin + p), __float_as_uint(Z));
    atomicMax(reinterpret_cast<unsigned int *>(smax + p), __float_as_uint(S[q]) & 0x7fffffffu);
}

__global__ __launch_bounds__(256) void fill_query_kernel(FillK f) { fill_query_tile(f, blockIdx.x); }

__device__ inline uint32_t block_exclusive_scan256(uint32_t v, uint32_t *s_wave, uint32_t *total) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    uint32_t inc = v;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const uint32_t o = __shfl_up(inc, d);
        if (lane >= d) inc += o;
    }
    if (lane == 63) s_wave[wave] = inc;
    __syncthreads();
    uint32_t off = 0, tot = 0;
#pragma unroll
    for (int x = 0; x < 4; ++x) {
        const uint32_t c = s_wave[x];
        if (x < wave) off += c;
        tot += c;
    }
    __syncthreads();
    *total = tot;
    return off + inc - v;
}

// value of x in lane j (j uniform across the wave)
__device__ inline float lane_f(float x, int j) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), j));
}

// Tiles that Gaussian i can reach with alpha >= 1/255: its rectangle cut to
// the tiles meeting the box of the alpha >= 1/255 ellipse (enlarged by 0.2%
// + 0.05 px, from the record; negative half extents: alpha < 1/255
// everywhere).  No pixel outside that box can reach the threshold.  Returns
// the number of tiles (0: none) and the first column and row and the column
// count in *box.
__device__ inline uint32_t occ_box(int i, const float4 *g, const ushort4 *rect, int3 *box) {
    const ushort4 r = rect[i];
    const float4 a = g[4 * (size_t)i];
    const float hx = g[4 * (size_t)i + 2].w, hy = g[4 * (size_t)i + 1].w;
    if (r.x > r.z || r.y > r.w || !(hx >= 0.0f)) return 0u;
    const int ex0 = max((int)r.x, (int)ceilf((a.x - hx - 15.0f) * 0.0625f));
    const int ex1 = min((int)r.z, (int)floorf((a.x + hx) * 0.0625f));
    const int ey0 = max((int)r.y, (int)ceilf((a.y - hy - 15.0f) * 0.0625f));
    const int ey1 = min((int)r.w, (int)floorf((a.y + hy) * 0.0625f));
    if (ex0 > ex1 || ey0 > ey1) return 0u;
    *box = make_int3(ex0, ey0, ex1 - ex0 + 1);
    return (uint32_t)((ex1 - ex0 + 1) * (ey1 - ey0 + 1));
}

constexpr int kOccThreads = 256;
constexpr int kOccPer = 4;                                 // consecutive Gaussians per thread
constexpr int kOccBlock = kOccThreads * kOccPer;           // 1024 Gaussians per block
constexpr int kOccWaves = kOccThreads / 64;

// Exclusive scan across a block of kOccThreads threads, one value each;
// *total = the block's sum.
__device__ inline uint32_t occ_block_scan(uint32_t v, uint32_t *s_wave, uint32_t *total) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    uint32_t inc = v;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const uint32_t o = __shfl_up(inc, d);
        if (lane >= d) inc += o;
    }
    if (lane == 63) s_wave[wave] = inc;
    __syncthreads();
    uint32_t off = 0, tot = 0;
#pragma unroll
    for (int x = 0; x < kOccWaves; ++x) {
        const uint32_t c = s_wave[x];
        if (x < wave) off += c;
        tot += c;
    }
    __syncthreads();
    *total = tot;
    return off + inc - v;
}

// One block per 1024 Gaussians, four consecutive ones per thread (a launch
// of few waves: most blocks find no newly visible Gaussian).  The newly
// visible ones that can reach a tile are compacted in LDS with the start of
// their (Gaussian, tile) pairs (two block scans, index order).  Wave w takes
// the pairs p = w (mod 4), 64 at a time: lane
// l finds the owner and tile of its pair (the searches run side by side),
// then the wave tests the pairs one after another with their data broadcast
// from the lanes: each lane tests four pixel centres and a ballot marks the
// tile.  Dealing the pairs out one by one spreads a block's pairs, however
// few Gaussians hold them, evenly over its four waves.  Marks are plain
// byte stores of 1, so concurrent writers agree.
__global__ __launch_bounds__(kOccThreads) void occluded_kernel(WarpK w, int n,
                                                               const uint8_t *__restrict__ status,
                                                               const float4 *__restrict__ g,
                                                               const ushort4 *__restrict__ rect,
                                                               uint8_t *oc) {
    __shared__ uint32_t s_idx[kOccBlock];   // compacted Gaussians
    __shared__ uint32_t s_off[kOccBlock];   // start of their pairs
    __shared__ uint32_t s_wave[kOccWaves];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int i0 = blockIdx.x * kOccBlock + tid * kOccPer;
    uint32_t c[kOccPer], na = 0u, np = 0u;
#pragma unroll
    for (int k = 0; k < kOccPer; ++k) {
        c[k] = 0u;
        if (i0 + k < n && (status[i0 + k] & 2u)) {
            int3 box;
            c[k] = occ_box(i0 + k, g, rect, &box);
        }
        na += c[k] ? 1u : 0u;
        np += c[k];
    }
    uint32_t total, n_act;
    uint32_t oa = occ_block_scan(na, s_wave, &n_act);
    uint32_t op = occ_block_scan(np, s_wave, &total);
#pragma unroll
    for (int k = 0; k < kOccPer; ++k) {
        if (c[k]) {
            s_idx[oa] = (uint32_t)(i0 + k);
            s_off[oa] = op;
            ++oa;
            op += c[k];
        }
    }
    __syncthreads();
    const uint32_t mine = total > (uint32_t)wave ? (total - (uint32_t)wave + kOccWaves - 1) / kOccWaves : 0u;
    for (uint32_t r0 = 0; r0 < mine; r0 += 64u) {
        const uint32_t r = r0 + (uint32_t)lane;
        int tx = 0, ty = 0;
        float4 a = make_float4(0.0f, 0.0f, 0.0f, 0.0f), b = a;
        if (r < mine) {
            const uint32_t p = (uint32_t)wave + kOccWaves * r;
            // owner of pair p: the last entry whose start is <= p (starts
            // increase strictly: every entry has a pair)
            uint32_t lo = 0, hi = n_act;
            while (hi - lo > 1u) {
                const uint32_t mid = (lo + hi) >> 1;
                if (s_off[mid] <= p) lo = mid;
                else hi = mid;
            }
            const int gi = (int)s_idx[lo];
            int3 box;
            (void)occ_box(gi, g, rect, &box);
            const int k = (int)(p - s_off[lo]);
            tx = box.x + k % box.z;
            ty = box.y + k / box.z;
            a = g[4 * (size_t)gi];
            b = g[4 * (size_t)gi + 1];
        }
        const int m = (int)min(64u, mine - r0);
        for (int j = 0; j < m; ++j) {
            const int jx = __builtin_amdgcn_readlane(tx, j), jy = __builtin_amdgcn_readlane(ty, j);
            const float ax = lane_f(a.x, j), ay = lane_f(a.y, j), az = lane_f(a.z, j),
                        aw = lane_f(a.w, j), bx = lane_f(b.x, j), by = lane_f(b.y, j);
            float amax = 0.0f;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int px = lane + 64 * q;
                const int x = jx * kTile + (px & 15), y = jy * kTile + (px >> 4);
                if (x < w.W && y < w.H) {
                    const float dx = ax - (float)x, dy = ay - (float)y;
                    const float power = -0.5f * (az * dx * dx + bx * dy * dy) - aw * dx * dy;
                    if (!(power > 0.0f)) amax = fmaxf(amax, fminf(kAlphaMax, by * __expf(power)));
                }
            }
            const uint64_t hit = __ballot(!(amax < kAlphaMin));
            if (hit != 0ull && lane == 0) oc[jy * w.TX + jx] = 1;
        }
    }
}

// One block per tile row: selected = occluded | unmatched (or every tile),
// the row's exclusive prefix sums rowpre[ty][0..TX] (rowpre[ty][TX] is the
// row's count) and its entries of the ascending list of selected tiles (the
// tiles not selected fill the list from the end, descending).  The
// list offset of the row, the selected tiles of the rows above, is counted
// by the block itself from the occluded and unmatched flags (a few KB read
// from cache), so no second launch waits for the other rows.  The last row
// also stores the total.
__global__ __launch_bounds__(256) void select_kernel(int TX, int TY, int mode, const uint8_t *oc,
                                                     const uint8_t *um, uint8_t *sel,
                                                     uint32_t *rowpre, int *sel_list, int *sel_cols,
                                                     uint8_t *mask_out, Counters *cnt) {
    __shared__ uint32_t s_wave[4];
    const int ty = blockIdx.x;
    // selected tiles above the row: four flags per 32-bit word, then a byte tail
    const uint32_t above = (uint32_t)ty * (uint32_t)TX;
    uint32_t part = 0;
    if (mode) {
        part = threadIdx.x == 0 ? above : 0u;
    } else {
        const uint32_t nw = above / 4u;
        const uint32_t *ow = reinterpret_cast<const uint32_t *>(oc);
        const uint32_t *uw = reinterpret_cast<const uint32_t *>(um);
        for (uint32_t k = threadIdx.x; k < nw; k += 256) {
            const uint32_t f = (ow[k] | uw[k]) & 0x01010101u;   // flags are 0 or 1
            part += (f * 0x01010101u) >> 24;
        }
        for (uint32_t t = 4u * nw + threadIdx.x; t < above; t += 256) part += (uint32_t)(oc[t] | um[t]);
    }
    uint32_t off;
    (void)block_exclusive_scan256(part, s_wave, &off);
    uint32_t *row = rowpre + (size_t)ty * (TX + 1);
    uint32_t run = 0;
    for (int c = 0; c < TX; c += 256) {
        const int x = c + threadIdx.x;
        const int t = ty * TX + x;
        uint32_t f = 0;
        if (x < TX) {
            f = mode ? 1u : (uint32_t)(oc[t] | um[t]);
            sel[t] = (uint8_t)f;
            if (mask_out) mask_out[t] = (uint8_t)f;
        }
        uint32_t tot;
        const uint32_t ex = block_exclusive_scan256(f, s_wave, &tot);
        if (x < TX) {
            row[x] = run + ex;
            if (f) {
                sel_list[off + run + ex] = t;
                sel_cols[(size_t)ty * TX + run + ex] = x;
            } else {
                // the others from the end: tiles not selected above the row,
                // then those of the row before this one
                sel_list[TX * TY - 1 - ((above - off) + ((uint32_t)x - run - ex))] = t;
            }
        }
        run += tot;
    }
    if (threadIdx.x == 0) {
        row[TX] = run;
        if (ty == TY - 1) cnt->n_selected = off + run;
    }
}

template <typename T>
__global__ __launch_bounds__(256) void fill_kernel(T *p, size_t n, T v) {
    for (size_t k = blockIdx.x * (size_t)blockDim.x + threadIdx.x; k < n;
         k += (size_t)gridDim.x * blockDim.x)
        p[k] = v;
}

template <typename T>
void fill(T *p, size_t n, T v, hipStream_t st) {
    if (n == 0) return;
    size_t blocks = (n + 255) / 256;
    if (blocks > 4096) blocks = 4096;
    fill_kernel<T><<<(unsigned)blocks, 256, 0, st>>>(p, n, v);
}

}  // namespace

void launch_temporal_init(int n_px, float *dmin, float *smax, hipStream_t st) {
    if (n_px > 0) temporal_init_kernel<<<(n_px + 255) / 256, 256, 0, st>>>(n_px, dmin, smax);
}

void launch_forward_warp(const WarpK &w, const float *D, const float *S, float *dmin, float *smax,
                         hipStream_t st) {
    const int n = w.W * w.H;
    forward_warp_kernel<<<(n + 255) / 256, 256, 0, st>>>(w, D, S, dmin, smax);
}

void launch_fill_query(const FillK &f, hipStream_t st) {
    fill_query_kernel<<<f.w.TX * f.w.TY, f.w.tp * f.w.tp, 0, st>>>(f);
}

void launch_occluded(const WarpK &w, int n, const uint8_t *status, const float4 *g,
                     const ushort4 *rect, uint8_t *oc, hipStream_t st) {
    if (n <= 0) return;
    occluded_kernel<<<(n + kOccBlock - 1) / kOccBlock, kOccThreads, 0, st>>>(w, n, status, g, rect,
                                                                            oc);
}

void launch_select(int TX, int TY, int mode, const uint8_t *oc, const uint8_t *um, uint8_t *sel,
                   int *sel_list, uint32_t *rowpre, int *sel_cols, uint8_t *mask_out,
                   Counters *cnt, hipStream_t st) {
    select_kernel<<<TY, 256, 0, st>>>(TX, TY, mode, oc, um, sel, rowpre, sel_list, sel_cols,
                                      mask_out, cnt);
}

void launch_fill_u8(uint8_t *p, size_t n, uint8_t v, hipStream_t st) { fill<uint8_t>(p, n, v, st); }
void launch_fill_f32(float *p, size_t n, float v, hipStream_t st) { fill<float>(p, n, v, st); }
void launch_fill_i32(int *p, size_t n, int v, hipStream_t st) { fill<int>(p, n, v, st); }

}  // namespace tgs
