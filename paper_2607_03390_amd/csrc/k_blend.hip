// Per-tile front-to-back alpha blending (Sec. III-A) and, on reference
// frames, the temporal priors it produces: the per-pixel depth and depth
// standard deviation of Eq. 1/2 (temporal geometry buffer), a copy of the
// image (temporal appearance buffer) and the set of Gaussians with a
// positive blending weight somewhere (temporal Gaussian buffer, Sec. III-C).
//
// One 256-thread block (four wave64s, one per 8x8 quadrant) per 16x16 tile,
// one pixel per thread.
// The tile's sorted Gaussians are staged through LDS in batches of 256
// records (48 bytes each, one coalesced gather per thread); every wave then
// reads each record as an LDS broadcast.  A pixel stops at the Gaussian that
// would take its transmittance below 1e-4; the block leaves as soon as all
// 256 pixels have stopped.  The work is VALU-bound (one exp and ~25 lane-ops
// per pixel-Gaussian pair).
//
// Eq. 1/2 are accumulated in one pass around a pivot (the first composited
// depth): D = d0 + S1/W, sigma^2 = S2/W - (S1/W)^2, which avoids the
// cancellation of the unshifted form at large depths.  Gaussians that a wave
// composites are flagged through a wave ballot, so the temporal Gaussian
// buffer costs one scalar test per record and wave.
#include <hip/hip_ext.h>

#include "tgs_internal.h"

namespace tgs {

namespace {

// Wave votes on the execution mask itself (no 0/1 vector temporaries).
__device__ inline bool wave_any(bool p) { return __builtin_amdgcn_ballot_w64(p) != 0ull; }
__device__ inline bool wave_all(bool p) { return __builtin_amdgcn_ballot_w64(!p) == 0ull; }

template <bool CAPTURE, bool CONTRIB, bool COUNT>
__global__ __launch_bounds__(256) void blend_kernel(BlendArgs a) {
    // Staged per Gaussian: (u, v, qa, qb) and (qc, opacity, depth, -) where
    // q* = conic coefficients pre-scaled by -log2(e) (and 1/2 on the squares)
    // so that log2 of the Gaussian falloff is a three-FMA quadratic form and
    // the opacity is one v_exp_f32.
    __shared__ float4 s_g0[256];
    __shared__ float4 s_g1[256];
    __shared__ float4 s_col[256];
    __shared__ int s_idx[256];
    __shared__ uint32_t s_flag[256];
    // Wave w (the 8x8 quadrant w of the tile: column half w & 1, row half
    // w >> 1) visits only the staged Gaussians whose alpha >= 1/255 ellipse,
    // conservatively enlarged, meets its quadrant, in staging (= depth)
    // order.  A square region touches fewer footprints than a 16x4 strip of
    // the same area.
    __shared__ uint16_t s_list[4][256];   // byte offsets (16 * staging slot)
    __shared__ uint32_t s_cnt[4][4];

    if (a.n_tiles_dev && blockIdx.x >= *a.n_tiles_dev) return;   // block-uniform
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int tile = a.tile_list ? a.tile_list[blockIdx.x] : (int)blockIdx.x;
    const int tx = tile % a.TX, ty = tile / a.TX;
    const int qx = wave & 1, qy = wave >> 1;
    const int px = tx * kTile + 8 * qx + (lane & 7), py = ty * kTile + 8 * qy + (lane >> 3);
    const bool inside = px < a.W && py < a.H;
    const float fpx = (float)px, fpy = (float)py;
    const float tile_x0 = (float)(tx * kTile), tile_y0 = (float)(ty * kTile);
    const uint2 range = a.ranges[tile];
    constexpr float kLog2e = 1.4426950408889634f;
    const uint64_t lt_mask = (1ull << lane) - 1ull;

    float T = 1.0f, cr = 0.0f, cg = 0.0f, cb = 0.0f;
    float sw = 0.0f, s1 = 0.0f, s2 = 0.0f, d0 = 0.0f;
    bool pivot = false;
    bool done = !inside;
    uint32_t stop_pos = range.y;   // list position of the stopping Gaussian (+1 below)
    uint32_t n_hit = 0;            // pairs with alpha >= 1/255 before the pixel stopped

    for (uint32_t b = range.x; b < range.y; b += 256) {
        if (__syncthreads_count(done) == 256) break;
        const uint32_t k = b + tid;
        uint32_t strips = 0;
        if (k < range.y) {
            const int idx = (int)a.vals[k];
            const float4 g0 = a.g0[idx];
            const float4 g1 = a.g1[idx];
            s_idx[tid] = idx;
            s_g0[tid] = make_float4(g0.x, g0.y, -0.5f * kLog2e * g0.z, -kLog2e * g0.w);
            s_g1[tid] = make_float4(-0.5f * kLog2e * g1.x, g1.y, g1.z, 0.0f);
            s_col[tid] = a.col[idx];
            // alpha >= 1/255  <=>  d^T conic d <= 2 ln(255 o): an ellipse with
            // half extents sqrt(k Sigma'_xx), sqrt(k Sigma'_yy); enlarged by
            // 0.2% + 0.05 px so that every pixel left out has alpha well below
            // the threshold.
            if (g1.y >= 0.999f * kAlphaMin) {
                const float kq = 2.0f * __logf(fmaxf(255.0f * g1.y, 1.0f)) + 1e-3f;
                const float det = g0.z * g1.x - g0.w * g0.w;
                const float hx = sqrtf(kq * g1.x / det) * 1.002f + 0.05f;
                const float hy = sqrtf(kq * g0.z / det) * 1.002f + 0.05f;
#pragma unroll
                for (int w = 0; w < 4; ++w) {
                    const float xlo = tile_x0 + 8.0f * (w & 1), ylo = tile_y0 + 8.0f * (w >> 1);
                    if (g0.x + hx >= xlo && g0.x - hx <= xlo + 7.0f && g0.y + hy >= ylo &&
                        g0.y - hy <= ylo + 7.0f)
                        strips |= 1u << w;
                }
            }
        }
        if (CAPTURE) s_flag[tid] = 0u;
        // order-preserving compaction of each strip's Gaussians
        uint64_t bal[4];
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            bal[w] = __ballot((strips >> w) & 1u);
            if (lane == 0) s_cnt[wave][w] = (uint32_t)__popcll(bal[w]);
        }
        __syncthreads();
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            if ((strips >> w) & 1u) {
                uint32_t pos = (uint32_t)__popcll(bal[w] & lt_mask);
                for (int sw2 = 0; sw2 < wave; ++sw2) pos += s_cnt[sw2][w];
                s_list[w][pos] = (uint16_t)(16 * tid);
            }
        }
        // the same for every lane of the wave: keep the loop on scalar registers
        const uint32_t n_mine = __builtin_amdgcn_readfirstlane(
            s_cnt[0][wave] + s_cnt[1][wave] + s_cnt[2][wave] + s_cnt[3][wave]);
        __syncthreads();
        // a wave whose pixels have all stopped skips the batch
        const uint32_t n_run = wave_all(done) ? 0u : n_mine;
        for (uint32_t e = 0; e < n_run; ++e) {
            const uint32_t jo = s_list[wave][e];
            const int j = (int)(jo >> 4);
            // staged records by byte offset: one LDS address for all three arrays
            const float4 g0 = *reinterpret_cast<const float4 *>(reinterpret_cast<const char *>(s_g0) + jo);
            const float4 g1 = *reinterpret_cast<const float4 *>(reinterpret_cast<const char *>(s_g1) + jo);
            const float dx = g0.x - fpx, dy = g0.y - fpy;
            // log2 of exp(power) with power = -(A dx^2 + 2B dx dy + C dy^2)/2
            const float p2 = __builtin_fmaf(dx, __builtin_fmaf(g0.z, dx, g0.w * dy), g1.x * dy * dy);
            const float alpha = fminf(kAlphaMax, g1.y * __builtin_amdgcn_exp2f(p2));
            // skipped: finished pixels, power > 0, alpha < 1/255; each vote
            // below is a single compare, so it is the compare's lane mask
            float alpha_eff = (done || p2 > 0.0f) ? 0.0f : alpha;
            // keep the select materialised (an empty constraint, no code):
            // otherwise the compiler turns it back into three combined masks
            // and rebuilds a vector 0/1 for the vote
            __asm__ volatile("" : "+v"(alpha_eff));
            const bool hit = alpha_eff >= kAlphaMin;
            if (!wave_any(hit)) continue;
            if (COUNT) n_hit += hit ? 1u : 0u;
            const float Tn = T * (1.0f - alpha);
            const bool inc = hit && Tn >= kTMin;
            const float w = inc ? alpha * T : 0.0f;
            const float4 c = *reinterpret_cast<const float4 *>(reinterpret_cast<const char *>(s_col) + jo);
            cr = __builtin_fmaf(w, c.x, cr);
            cg = __builtin_fmaf(w, c.y, cg);
            cb = __builtin_fmaf(w, c.z, cb);
            T = inc ? Tn : T;
            bool all_done = false;
            if (wave_any(Tn < kTMin)) {   // rare: a pixel may stop at this Gaussian
                const bool stop = hit && Tn < kTMin;
                if (COUNT && stop) stop_pos = b + (uint32_t)j;
                done = done || stop;
                all_done = wave_all(done);
            }
            if (CAPTURE) {
                const float dep = g1.z;
                d0 = (inc && !pivot) ? dep : d0;
                pivot = pivot || inc;
                const float dd = dep - d0;
                sw += w;
                s1 = __builtin_fmaf(w, dd, s1);
                s2 = __builtin_fmaf(w * dd, dd, s2);
                // w > 0 exactly where the pixel composites (alpha, T > 0)
                const bool any_inc = wave_any(w > 0.0f);
                if (any_inc && lane == 0) s_flag[j] = 1u;
                if (CONTRIB && any_inc) {
                    float mw = w;
#pragma unroll
                    for (int o = 32; o >= 1; o >>= 1) mw = fmaxf(mw, __shfl_xor(mw, o));
                    if (lane == 0)
                        atomicMax(reinterpret_cast<unsigned int *>(a.contrib + s_idx[j]),
                                  __float_as_uint(mw));
                }
            }
            if (all_done) break;
        }
        __syncthreads();
        if (CAPTURE && a.g_flag && k < range.y && s_flag[tid]) a.g_flag[s_idx[tid]] = 1u;
    }

    if (COUNT) {
        // evaluated list entries: up to and including the stopping one
        unsigned long long e = inside ? (unsigned long long)(stop_pos < range.y ? stop_pos + 1 : range.y) - range.x : 0ull;
        unsigned long long h = n_hit;
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) {
            e += __shfl_xor(e, o);
            h += __shfl_xor(h, o);
        }
        if (lane == 0 && e) atomicAdd(a.pairs, e);
        if (lane == 0 && h) atomicAdd(a.hits, h);
    }
    if (!inside) return;
    const size_t HW = (size_t)a.W * a.H;
    const size_t q = (size_t)py * a.W + px;
    a.rgb[q] = cr;
    a.rgb[HW + q] = cg;
    a.rgb[2 * HW + q] = cb;
    if (a.tab) {
        a.tab[q] = cr;
        a.tab[HW + q] = cg;
        a.tab[2 * HW + q] = cb;
    }
    if (CAPTURE) {
        float D = a.empty_depth, S = 0.0f;
        if (sw > 0.0f) {
            const float m1 = s1 / sw;
            D = d0 + m1;
            S = sqrtf(fmaxf(0.0f, s2 / sw - m1 * m1));
        }
        if (a.depth) a.depth[q] = D;
        if (a.sigma) a.sigma[q] = S;
        if (a.alpha) a.alpha[q] = 1.0f - T;
        if (a.tgb_depth) a.tgb_depth[q] = D;
        if (a.tgb_sigma) a.tgb_sigma[q] = S;
    }
}

// Adaptive frustum (Sec. III-D): min / max NDC of the projected means of the
// temporal Gaussian buffer.  Two levels: a fixed grid of blocks reduces
// grid-strided slices into partials, one block reduces the partials (no
// contended atomics; min / max are exact, so the result is deterministic).
constexpr int kAfcBlocks = kAfcPartials;

__global__ __launch_bounds__(256) void afc_partial_kernel(int n, const uint8_t *g_flag,
                                                          const float4 *g0, int W, int H,
                                                          int *partial) {
    __shared__ int s_red[4][4];
    int v[4] = {float_to_ordered(__builtin_inff()), float_to_ordered(__builtin_inff()),
                float_to_ordered(-__builtin_inff()), float_to_ordered(-__builtin_inff())};
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) {
        if (!g_flag[i]) continue;
        const float4 r = g0[i];
        const int nx = float_to_ordered((2.0f * r.x + 1.0f) / (float)W - 1.0f);
        const int ny = float_to_ordered((2.0f * r.y + 1.0f) / (float)H - 1.0f);
        v[0] = min(v[0], nx);
        v[1] = min(v[1], ny);
        v[2] = max(v[2], nx);
        v[3] = max(v[3], ny);
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        v[0] = min(v[0], __shfl_xor(v[0], o));
        v[1] = min(v[1], __shfl_xor(v[1], o));
        v[2] = max(v[2], __shfl_xor(v[2], o));
        v[3] = max(v[3], __shfl_xor(v[3], o));
    }
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    if (lane == 0)
        for (int k = 0; k < 4; ++k) s_red[wave][k] = v[k];
    __syncthreads();
    if (threadIdx.x < 4) {
        const int k = threadIdx.x;
        int r = s_red[0][k];
        for (int w = 1; w < 4; ++w) r = k < 2 ? min(r, s_red[w][k]) : max(r, s_red[w][k]);
        partial[blockIdx.x * 4 + k] = r;
    }
}

__global__ __launch_bounds__(64) void afc_final_kernel(const int *partial, int n_partial,
                                                       int *fbox) {
    int v[4] = {float_to_ordered(__builtin_inff()), float_to_ordered(__builtin_inff()),
                float_to_ordered(-__builtin_inff()), float_to_ordered(-__builtin_inff())};
    for (int b = threadIdx.x; b < n_partial; b += 64) {
        v[0] = min(v[0], partial[b * 4 + 0]);
        v[1] = min(v[1], partial[b * 4 + 1]);
        v[2] = max(v[2], partial[b * 4 + 2]);
        v[3] = max(v[3], partial[b * 4 + 3]);
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        v[0] = min(v[0], __shfl_xor(v[0], o));
        v[1] = min(v[1], __shfl_xor(v[1], o));
        v[2] = max(v[2], __shfl_xor(v[2], o));
        v[3] = max(v[3], __shfl_xor(v[3], o));
    }
    if (threadIdx.x == 0)
        for (int k = 0; k < 4; ++k) fbox[k] = v[k];
}

}  // namespace

template <bool CAPTURE, bool CONTRIB>
void launch_blend_v(const BlendArgs &a, int n_blocks, hipStream_t st, hipEvent_t e0, hipEvent_t e1) {
    if (a.pairs)
        hipExtLaunchKernelGGL(blend_kernel<CAPTURE, CONTRIB, true>, dim3(n_blocks), dim3(256), 0, st,
                              e0, e1, 0, a);
    else
        hipExtLaunchKernelGGL(blend_kernel<CAPTURE, CONTRIB, false>, dim3(n_blocks), dim3(256), 0, st,
                              e0, e1, 0, a);
}

void launch_blend(const BlendArgs &a, int n_blocks, hipStream_t st, hipEvent_t start,
                  hipEvent_t stop) {
    if (n_blocks <= 0) return;
    const bool capture = a.depth || a.sigma || a.alpha || a.tgb_depth || a.tgb_sigma || a.g_flag ||
                         a.contrib;
    if (a.contrib)
        launch_blend_v<true, true>(a, n_blocks, st, start, stop);
    else if (capture)
        launch_blend_v<true, false>(a, n_blocks, st, start, stop);
    else
        launch_blend_v<false, false>(a, n_blocks, st, start, stop);
}

void launch_afc_bounds(int n, const uint8_t *g_flag, const float4 *g0, int W, int H, int *fbox,
                       hipStream_t st) {
    // fbox[0..3] is the result; fbox[4..] holds kAfcBlocks x 4 partials
    int *partial = fbox + 4;
    afc_partial_kernel<<<kAfcBlocks, 256, 0, st>>>(n, g_flag, g0, W, H, partial);
    afc_final_kernel<<<1, 64, 0, st>>>(partial, kAfcBlocks, fbox);
}

}  // namespace tgs
