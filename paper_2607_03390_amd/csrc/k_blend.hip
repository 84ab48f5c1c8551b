// Per-tile front-to-back alpha blending (Sec. III-A) and, on reference
// frames, the temporal priors it produces: the per-pixel depth and depth
// standard deviation of Eq. 1/2 (temporal geometry buffer), a copy of the
// image (temporal appearance buffer) and the set of Gaussians with a
// positive blending weight somewhere (temporal Gaussian buffer, Sec. III-C).
//
// One 256-thread block (four wave64s) per 16x16 tile, one pixel per thread.
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
#include "tgs_internal.h"

namespace tgs {

namespace {

template <bool CAPTURE, bool CONTRIB, bool COUNT>
__global__ __launch_bounds__(256) void blend_kernel(BlendArgs a) {
    __shared__ float4 s_g0[256];
    __shared__ float4 s_g1[256];
    __shared__ float4 s_col[256];
    __shared__ int s_idx[256];
    __shared__ uint32_t s_flag[256];

    const int tid = threadIdx.x, lane = tid & 63;
    const int tile = a.tile_list ? a.tile_list[blockIdx.x] : (int)blockIdx.x;
    const int tx = tile % a.TX, ty = tile / a.TX;
    const int px = tx * kTile + (tid & 15), py = ty * kTile + (tid >> 4);
    const bool inside = px < a.W && py < a.H;
    const float fpx = (float)px, fpy = (float)py;
    const uint2 range = a.ranges[tile];

    float T = 1.0f, cr = 0.0f, cg = 0.0f, cb = 0.0f;
    float sw = 0.0f, s1 = 0.0f, s2 = 0.0f, d0 = 0.0f;
    bool pivot = false;
    bool done = !inside;
    uint32_t evaluated = 0;

    for (uint32_t b = range.x; b < range.y; b += 256) {
        if (__syncthreads_count(done) == 256) break;
        const uint32_t k = b + tid;
        if (k < range.y) {
            const int idx = (int)a.vals[k];
            s_idx[tid] = idx;
            s_g0[tid] = a.g0[idx];
            s_g1[tid] = a.g1[idx];
            s_col[tid] = a.col[idx];
        }
        if (CAPTURE) s_flag[tid] = 0u;
        __syncthreads();
        const int cnt = (int)min(256u, range.y - b);
        for (int j = 0; j < cnt; ++j) {
            bool inc = false;
            float w = 0.0f;
            if (!done) {
                if (COUNT) ++evaluated;
                const float4 g0 = s_g0[j];
                const float4 g1 = s_g1[j];
                const float dx = g0.x - fpx, dy = g0.y - fpy;
                const float power = -0.5f * (g0.z * dx * dx + g1.x * dy * dy) - g0.w * dx * dy;
                if (!(power > 0.0f)) {
                    const float alpha = fminf(kAlphaMax, g1.y * __expf(power));
                    if (!(alpha < kAlphaMin)) {
                        const float Tn = T * (1.0f - alpha);
                        if (Tn < kTMin) {
                            done = true;
                        } else {
                            w = alpha * T;
                            const float4 c = s_col[j];
                            cr = __builtin_fmaf(w, c.x, cr);
                            cg = __builtin_fmaf(w, c.y, cg);
                            cb = __builtin_fmaf(w, c.z, cb);
                            if (CAPTURE) {
                                if (!pivot) { d0 = g1.z; pivot = true; }
                                const float dd = g1.z - d0;
                                sw += w;
                                s1 = __builtin_fmaf(w, dd, s1);
                                s2 = __builtin_fmaf(w * dd, dd, s2);
                            }
                            T = Tn;
                            inc = true;
                        }
                    }
                }
            }
            if (CAPTURE) {
                const uint64_t m = __ballot(inc);
                if (m != 0ull && lane == 0) s_flag[j] = 1u;
                if (CONTRIB && m != 0ull) {
                    float mw = w;
#pragma unroll
                    for (int o = 32; o >= 1; o >>= 1) mw = fmaxf(mw, __shfl_xor(mw, o));
                    if (lane == 0)
                        atomicMax(reinterpret_cast<unsigned int *>(a.contrib + s_idx[j]),
                                  __float_as_uint(mw));
                }
            }
        }
        __syncthreads();
        if (CAPTURE && a.g_flag && k < range.y && s_flag[tid]) a.g_flag[s_idx[tid]] = 1u;
    }

    if (COUNT) {
        unsigned long long e = evaluated;
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) e += __shfl_xor(e, o);
        if (lane == 0 && e) atomicAdd(a.pairs, e);
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
        float D = kNoHit, S = 0.0f;
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

__global__ __launch_bounds__(64) void afc_init_kernel(int *fbox) {
    if (threadIdx.x < 4) {
        const float v = threadIdx.x < 2 ? __builtin_inff() : -__builtin_inff();
        fbox[threadIdx.x] = float_to_ordered(v);
    }
}

__global__ __launch_bounds__(256) void afc_bounds_kernel(int n, const uint8_t *g_flag,
                                                         const float4 *g0, int W, int H,
                                                         int *fbox) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    int mnx = float_to_ordered(__builtin_inff()), mny = mnx;
    int mxx = float_to_ordered(-__builtin_inff()), mxy = mxx;
    if (i < n && g_flag[i]) {
        const float4 r = g0[i];
        const float nx = (2.0f * r.x + 1.0f) / (float)W - 1.0f;
        const float ny = (2.0f * r.y + 1.0f) / (float)H - 1.0f;
        mnx = mxx = float_to_ordered(nx);
        mny = mxy = float_to_ordered(ny);
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        mnx = min(mnx, __shfl_xor(mnx, o));
        mny = min(mny, __shfl_xor(mny, o));
        mxx = max(mxx, __shfl_xor(mxx, o));
        mxy = max(mxy, __shfl_xor(mxy, o));
    }
    if ((threadIdx.x & 63) == 0) {
        atomicMin(&fbox[0], mnx);
        atomicMin(&fbox[1], mny);
        atomicMax(&fbox[2], mxx);
        atomicMax(&fbox[3], mxy);
    }
}

}  // namespace

template <bool CAPTURE, bool CONTRIB>
void launch_blend_v(const BlendArgs &a, int n_blocks, hipStream_t st) {
    if (a.pairs)
        blend_kernel<CAPTURE, CONTRIB, true><<<n_blocks, 256, 0, st>>>(a);
    else
        blend_kernel<CAPTURE, CONTRIB, false><<<n_blocks, 256, 0, st>>>(a);
}

void launch_blend(const BlendArgs &a, int n_blocks, hipStream_t st) {
    if (n_blocks <= 0) return;
    const bool capture = a.depth || a.sigma || a.alpha || a.tgb_depth || a.tgb_sigma || a.g_flag ||
                         a.contrib;
    if (a.contrib)
        launch_blend_v<true, true>(a, n_blocks, st);
    else if (capture)
        launch_blend_v<true, false>(a, n_blocks, st);
    else
        launch_blend_v<false, false>(a, n_blocks, st);
}

void launch_afc_bounds(int n, const uint8_t *g_flag, const float4 *g0, int W, int H, int *fbox,
                       hipStream_t st) {
    afc_init_kernel<<<1, 64, 0, st>>>(fbox);
    if (n > 0) afc_bounds_kernel<<<(n + 255) / 256, 256, 0, st>>>(n, g_flag, g0, W, H, fbox);
}

}  // namespace tgs
