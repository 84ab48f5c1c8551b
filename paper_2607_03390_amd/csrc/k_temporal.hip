// Temporal kernels of a TemporalGS frame (Sec. III-C..E):
//  - forward warp of the temporal geometry buffer into the current view
//    (Eq. 3): nearest destination pixel, minimum depth and maximum standard
//    deviation by integer atomics on the float bits (both are non-negative,
//    so unsigned order is float order and the result is order-independent);
//  - depth fill, backward correspondence query and unmatched tiles, one
//    block per tile with a block-wide OR;
//  - occluded tiles of the newly visible Gaussians, one wave per
//    (Gaussian, tile) pair with a wave ballot over the tile's 256 pixels;
//  - tile selection and compaction, one block per tile row, including the
//    per-row prefix sums of the mask used by the key counts;
//  - stitching of the warped reference image into the tiles that are not
//    re-rendered (Eq. 4, bilinear).
// All of these are HBM- or latency-bound; none is a dense contraction.
#include "tgs_internal.h"

namespace tgs {

namespace {

__global__ __launch_bounds__(256) void temporal_init_kernel(int n_px, int n_tiles, float *dmin,
                                                            float *smax, uint8_t *oc) {
    const int k = blockIdx.x * blockDim.x + threadIdx.x;
    if (k < n_px) {
        dmin[k] = kNoHit;
        smax[k] = 0.0f;
    }
    if (k < n_tiles) oc[k] = 0;
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

// One block of tp x tp threads per tile (tp = 16 on the image, 8 on the
// half-resolution geometry-buffer grid, where a tile is 8 x 8 cells).
__global__ __launch_bounds__(256) void fill_query_kernel(WarpK w, const float *__restrict__ dmin,
                                                         float *dfill, float2 *uv, uint8_t *um) {
    const int tile = blockIdx.x;
    const int tx = tile % w.TX, ty = tile / w.TX;
    const int px = tx * w.tp + (int)(threadIdx.x % (unsigned)w.tp);
    const int py = ty * w.tp + (int)(threadIdx.x / (unsigned)w.tp);
    int bad = 0;
    if (px < w.W && py < w.H) {
        const int q = py * w.W + px;
        float d = dmin[q];
        if (d == kNoHit && px >= 1 && py >= 1 && px <= w.W - 2 && py <= w.H - 2) {
            const float *r0 = dmin + (size_t)(py - 1) * w.W + px;
            const float *r1 = r0 + w.W, *r2 = r1 + w.W;
            const float n0 = r0[-1], n1 = r0[0], n2 = r0[1], n3 = r1[-1], n4 = r1[1], n5 = r2[-1],
                        n6 = r2[0], n7 = r2[1];
            if (n0 != kNoHit && n1 != kNoHit && n2 != kNoHit && n3 != kNoHit && n4 != kNoHit &&
                n5 != kNoHit && n6 != kNoHit && n7 != kNoHit) {
                float s = n0;
                s = s + n1;
                s = s + n2;
                s = s + n3;
                s = s + n4;
                s = s + n5;
                s = s + n6;
                s = s + n7;
                d = s / 8.0f;
            }
        }
        dfill[q] = d;
        bool ok = false;
        float u = -1.0f, v = -1.0f;
        if (d != kNoHit) {
            const float rx = ((float)px - w.kcur[2]) / w.kcur[0];
            const float ry = ((float)py - w.kcur[3]) / w.kcur[1];
            const float Px = d * rx, Py = d * ry, Pz = d;
            const float *M = w.Minv;
            const float X = ((M[0] * Px + M[1] * Py) + M[2] * Pz) + M[3];
            const float Y = ((M[4] * Px + M[5] * Py) + M[6] * Pz) + M[7];
            const float Z = ((M[8] * Px + M[9] * Py) + M[10] * Pz) + M[11];
            if (Z > w.z_near) {
                u = w.kref[0] * (X / Z) + w.kref[2];
                v = w.kref[1] * (Y / Z) + w.kref[3];
                ok = u >= 0.0f && u <= (float)(w.W - 1) && v >= 0.0f && v <= (float)(w.H - 1);
            }
        }
        uv[q] = ok ? make_float2(u, v) : make_float2(-1.0f, -1.0f);
        bad = ok ? 0 : 1;
    }
    const int any = __syncthreads_or(bad);
    if (threadIdx.x == 0) um[tile] = (uint8_t)(any ? 1 : 0);
}

// Each wave scans 64 status bytes at a time; for every newly visible
// Gaussian among them the whole wave tests its rectangle's tiles, four pixel
// centres per lane, with a ballot per tile.
__global__ __launch_bounds__(256) void occluded_kernel(WarpK w, int n,
                                                       const uint8_t *__restrict__ status,
                                                       const float4 *g, const ushort4 *rect,
                                                       uint8_t *oc) {
    const int lane = threadIdx.x & 63;
    const int wave = (int)((blockIdx.x * blockDim.x + threadIdx.x) >> 6);
    const int n_waves = (int)((gridDim.x * blockDim.x) >> 6);
    for (int base = wave * 64; base < n; base += n_waves * 64) {
        const int me = base + lane;
        const bool nv = me < n && (status[me] & 2u);
        uint64_t todo = __ballot(nv);
        while (todo) {
            const int l = __ffsll((unsigned long long)todo) - 1;
            todo &= todo - 1ull;
            const int i = base + l;
            const ushort4 r = rect[i];
            if (r.x > r.z || r.y > r.w) continue;
            const float4 a = g[4 * (size_t)i];
            const float4 b = g[4 * (size_t)i + 1];
            if (!(b.y >= 0.999f * kAlphaMin)) continue;   // alpha < 1/255 everywhere
            // tiles meeting the box of the alpha >= 1/255 ellipse (enlarged
            // by 0.2% + 0.05 px): no pixel outside it can reach the threshold
            const float kq = 2.0f * __logf(fmaxf(255.0f * b.y, 1.0f)) + 1e-3f;
            const float det = a.z * b.x - a.w * a.w;
            const float hx = sqrtf(kq * b.x / det) * 1.002f + 0.05f;
            const float hy = sqrtf(kq * a.z / det) * 1.002f + 0.05f;
            const int ex0 = max((int)r.x, (int)ceilf((a.x - hx - 15.0f) * 0.0625f));
            const int ex1 = min((int)r.z, (int)floorf((a.x + hx) * 0.0625f));
            const int ey0 = max((int)r.y, (int)ceilf((a.y - hy - 15.0f) * 0.0625f));
            const int ey1 = min((int)r.w, (int)floorf((a.y + hy) * 0.0625f));
            for (int ty = ey0; ty <= ey1; ++ty)
                for (int tx = ex0; tx <= ex1; ++tx) {
                    float amax = 0.0f;
#pragma unroll
                    for (int k = 0; k < 4; ++k) {
                        const int p = lane + 64 * k;
                        const int x = tx * kTile + (p & 15), y = ty * kTile + (p >> 4);
                        if (x < w.W && y < w.H) {
                            const float dx = a.x - (float)x, dy = a.y - (float)y;
                            const float power = -0.5f * (a.z * dx * dx + b.x * dy * dy) - a.w * dx * dy;
                            if (!(power > 0.0f))
                                amax = fmaxf(amax, fminf(kAlphaMax, b.y * __expf(power)));
                        }
                    }
                    const uint64_t hit = __ballot(!(amax < kAlphaMin));
                    if (hit != 0ull && lane == 0) oc[ty * w.TX + tx] = 1;
                }
        }
    }
}

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

// One block per tile row: selected = occluded | unmatched (or every tile),
// and the row's exclusive prefix sums rowpre[ty][0..TX] (rowpre[ty][TX] is the
// row's count).
__global__ __launch_bounds__(256) void select_rows_kernel(int TX, int mode, const uint8_t *oc,
                                                          const uint8_t *um, uint8_t *sel,
                                                          uint32_t *rowpre, uint8_t *mask_out) {
    __shared__ uint32_t s_wave[4];
    const int ty = blockIdx.x;
    uint32_t *row = rowpre + (size_t)ty * (TX + 1);
    uint32_t run = 0;
    for (int c = 0; c < TX; c += 256) {
        const int x = c + threadIdx.x;
        const int t = ty * TX + x;
        uint32_t s = 0;
        if (x < TX) {
            s = mode ? 1u : (uint32_t)(oc[t] | um[t]);
            sel[t] = (uint8_t)s;
            if (mask_out) mask_out[t] = (uint8_t)s;
        }
        uint32_t tot;
        const uint32_t ex = block_exclusive_scan256(s, s_wave, &tot);
        if (x < TX) row[x] = run + ex;
        run += tot;
    }
    if (threadIdx.x == 0) row[TX] = run;
}

// One block per tile row: the ascending list of selected tiles; the last row
// also stores the total.
__global__ __launch_bounds__(256) void select_list_kernel(int TX, int TY, const uint8_t *sel,
                                                          const uint32_t *rowpre, int *sel_list,
                                                          int *sel_cols, Counters *cnt) {
    __shared__ uint32_t s_sum[4];
    const int ty = blockIdx.x;
    uint32_t part = 0;
    for (int r = threadIdx.x; r < ty; r += 256) part += rowpre[(size_t)r * (TX + 1) + TX];
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) part += __shfl_xor(part, o);
    if ((threadIdx.x & 63) == 0) s_sum[threadIdx.x >> 6] = part;
    __syncthreads();
    const uint32_t off = s_sum[0] + s_sum[1] + s_sum[2] + s_sum[3];
    const uint32_t *row = rowpre + (size_t)ty * (TX + 1);
    for (int x = threadIdx.x; x < TX; x += 256) {
        const int t = ty * TX + x;
        if (sel[t]) {
            sel_list[off + row[x]] = t;
            sel_cols[(size_t)ty * TX + row[x]] = x;
        }
    }
    if (ty == TY - 1 && threadIdx.x == 0) cnt->n_selected = off + row[TX];
}

__global__ __launch_bounds__(256) void stitch_kernel(WarpK w, const uint8_t *sel,
                                                     const float *__restrict__ tab,
                                                     const float2 *__restrict__ uv, float *rgb) {
    const int tile = blockIdx.x;
    if (sel[tile]) return;
    const int tx = tile % w.TX, ty = tile / w.TX;
    const int px = tx * kTile + (threadIdx.x & 15), py = ty * kTile + (threadIdx.x >> 4);
    if (px >= w.W || py >= w.H) return;
    const size_t HW = (size_t)w.W * w.H;
    const size_t q = (size_t)py * w.W + px;
    const float2 c = uv[q];
    if (!(c.x >= 0.0f && c.y >= 0.0f)) {   // unmatched pixels only occur in selected tiles
        rgb[q] = rgb[HW + q] = rgb[2 * HW + q] = 0.0f;
        return;
    }
    const int x0 = (int)floorf(c.x), y0 = (int)floorf(c.y);
    const int x1 = min(x0 + 1, w.W - 1), y1 = min(y0 + 1, w.H - 1);
    const float ax = c.x - (float)x0, ay = c.y - (float)y0;
    const size_t i00 = (size_t)y0 * w.W + x0, i10 = (size_t)y0 * w.W + x1;
    const size_t i01 = (size_t)y1 * w.W + x0, i11 = (size_t)y1 * w.W + x1;
#pragma unroll
    for (int ch = 0; ch < 3; ++ch) {
        const float *I = tab + ch * HW;
        const float top = (1.0f - ax) * I[i00] + ax * I[i10];
        const float bot = (1.0f - ax) * I[i01] + ax * I[i11];
        rgb[ch * HW + q] = (1.0f - ay) * top + ay * bot;
    }
}

// Eq. 4 from a half-resolution repaired depth: pixel (x, y) takes the depth
// of its block (x >> 1, y >> 1), is unprojected and moved to the reference
// view at full resolution, and samples the reference image bilinearly at
// the projection clamped to the image (the block matched; the pixel itself
// may land up to about a pixel outside).
__global__ __launch_bounds__(256) void stitch_depth_kernel(WarpK w, int Wg, const uint8_t *sel,
                                                           const float *__restrict__ tab,
                                                           const float *__restrict__ dfill,
                                                           float *rgb) {
    const int tile = blockIdx.x;
    if (sel[tile]) return;
    const int tx = tile % w.TX, ty = tile / w.TX;
    const int px = tx * kTile + (threadIdx.x & 15), py = ty * kTile + (threadIdx.x >> 4);
    if (px >= w.W || py >= w.H) return;
    const size_t HW = (size_t)w.W * w.H;
    const size_t q = (size_t)py * w.W + px;
    const float d = dfill[(size_t)(py >> 1) * Wg + (px >> 1)];
    bool ok = false;
    float u = 0.0f, v = 0.0f;
    if (d != kNoHit) {
        const float rx = ((float)px - w.kcur[2]) / w.kcur[0];
        const float ry = ((float)py - w.kcur[3]) / w.kcur[1];
        const float Px = d * rx, Py = d * ry, Pz = d;
        const float *M = w.Minv;
        const float X = ((M[0] * Px + M[1] * Py) + M[2] * Pz) + M[3];
        const float Y = ((M[4] * Px + M[5] * Py) + M[6] * Pz) + M[7];
        const float Z = ((M[8] * Px + M[9] * Py) + M[10] * Pz) + M[11];
        if (Z > w.z_near) {
            u = fminf(fmaxf(w.kref[0] * (X / Z) + w.kref[2], 0.0f), (float)(w.W - 1));
            v = fminf(fmaxf(w.kref[1] * (Y / Z) + w.kref[3], 0.0f), (float)(w.H - 1));
            ok = true;
        }
    }
    if (!ok) {   // cannot occur outside selected tiles
        rgb[q] = rgb[HW + q] = rgb[2 * HW + q] = 0.0f;
        return;
    }
    const int x0 = (int)floorf(u), y0 = (int)floorf(v);
    const int x1 = min(x0 + 1, w.W - 1), y1 = min(y0 + 1, w.H - 1);
    const float ax = u - (float)x0, ay = v - (float)y0;
    const size_t i00 = (size_t)y0 * w.W + x0, i10 = (size_t)y0 * w.W + x1;
    const size_t i01 = (size_t)y1 * w.W + x0, i11 = (size_t)y1 * w.W + x1;
#pragma unroll
    for (int ch = 0; ch < 3; ++ch) {
        const float *I = tab + ch * HW;
        const float top = (1.0f - ax) * I[i00] + ax * I[i10];
        const float bot = (1.0f - ax) * I[i01] + ax * I[i11];
        rgb[ch * HW + q] = (1.0f - ay) * top + ay * bot;
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

void launch_temporal_init(int n_px, int n_tiles, float *dmin, float *smax, uint8_t *oc,
                          Counters *cnt, hipStream_t st) {
    const int n = n_px > n_tiles ? n_px : n_tiles;
    temporal_init_kernel<<<(n + 255) / 256, 256, 0, st>>>(n_px, n_tiles, dmin, smax, oc);
    (void)cnt;
}

void launch_forward_warp(const WarpK &w, const float *D, const float *S, float *dmin, float *smax,
                         hipStream_t st) {
    const int n = w.W * w.H;
    forward_warp_kernel<<<(n + 255) / 256, 256, 0, st>>>(w, D, S, dmin, smax);
}

void launch_fill_query(const WarpK &w, const float *dmin, float *dfill, float2 *uv, uint8_t *um,
                       hipStream_t st) {
    fill_query_kernel<<<w.TX * w.TY, w.tp * w.tp, 0, st>>>(w, dmin, dfill, uv, um);
}

void launch_stitch_depth(const WarpK &w, int Wg, const uint8_t *sel, const float *tab,
                         const float *dfill, float *rgb, hipStream_t st) {
    stitch_depth_kernel<<<w.TX * w.TY, 256, 0, st>>>(w, Wg, sel, tab, dfill, rgb);
}

void launch_occluded(const WarpK &w, int n, const uint8_t *status, const float4 *g,
                     const ushort4 *rect, uint8_t *oc, hipStream_t st) {
    if (n <= 0) return;
    int blocks = (n + 255) / 256;
    if (blocks > 1024) blocks = 1024;
    occluded_kernel<<<blocks, 256, 0, st>>>(w, n, status, g, rect, oc);
}

void launch_select(int TX, int TY, int mode, const uint8_t *oc, const uint8_t *um, uint8_t *sel,
                   int *sel_list, uint32_t *rowpre, int *sel_cols, uint8_t *mask_out,
                   Counters *cnt, hipStream_t st) {
    select_rows_kernel<<<TY, 256, 0, st>>>(TX, mode, oc, um, sel, rowpre, mask_out);
    select_list_kernel<<<TY, 256, 0, st>>>(TX, TY, sel, rowpre, sel_list, sel_cols, cnt);
}

void launch_stitch(const WarpK &w, const uint8_t *sel, const float *tab, const float2 *uv,
                   float *rgb, hipStream_t st) {
    stitch_kernel<<<w.TX * w.TY, 256, 0, st>>>(w, sel, tab, uv, rgb);
}

void launch_fill_u8(uint8_t *p, size_t n, uint8_t v, hipStream_t st) { fill<uint8_t>(p, n, v, st); }
void launch_fill_f32(float *p, size_t n, float v, hipStream_t st) { fill<float>(p, n, v, st); }
void launch_fill_i32(int *p, size_t n, int v, hipStream_t st) { fill<int>(p, n, v, st); }

}  // namespace tgs
