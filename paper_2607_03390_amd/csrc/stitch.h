// Stitching of a tile that is not re-rendered (Eq. 4): each pixel takes the
// reference image (temporal appearance buffer) sampled bilinearly where its
// surface point lands in the reference view.  One 256-thread block per tile,
// one pixel per thread.  The blend launch of a TemporalGS frame runs these
// on the blocks past the selected tiles, so the stitching fills the
// blend's tail instead of a launch of its own.
#pragma once

#include "tgs_internal.h"

namespace tgs {

// Bilinear sample of the three planes of tab at (u, v) in [0, W-1] x [0, H-1]
// into pixel q of rgb.
__device__ inline void stitch_sample(const WarpK &w, const float *__restrict__ tab, float u,
                                     float v, size_t q, float *rgb) {
    const size_t HW = (size_t)w.W * w.H;
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

// Full-resolution geometry buffer: the per-pixel correspondences of the
// backward query (negative: unmatched, which occurs in selected tiles only).
__device__ inline void stitch_tile_uv(const WarpK &w, int tile, const float *__restrict__ tab,
                                      const float2 *__restrict__ uv, float *rgb) {
    const int tx = tile % w.TX, ty = tile / w.TX;
    const int px = tx * kTile + (threadIdx.x & 15), py = ty * kTile + (threadIdx.x >> 4);
    if (px >= w.W || py >= w.H) return;
    const size_t HW = (size_t)w.W * w.H;
    const size_t q = (size_t)py * w.W + px;
    const float2 c = uv[q];
    if (!(c.x >= 0.0f && c.y >= 0.0f)) {
        rgb[q] = rgb[HW + q] = rgb[2 * HW + q] = 0.0f;
        return;
    }
    stitch_sample(w, tab, c.x, c.y, q, rgb);
}

// Half-resolution geometry buffer (grid width Wg): pixel (x, y) takes the
// repaired depth of its block (x >> 1, y >> 1), is unprojected and moved to
// the reference view at full resolution, and samples the reference image at
// the projection clamped to the image (the block matched; the pixel itself
// may land up to about a pixel outside).
__device__ inline void stitch_tile_depth(const WarpK &w, int Wg, int tile,
                                         const float *__restrict__ tab,
                                         const float *__restrict__ dfill, float *rgb) {
    const int tx = tile % w.TX, ty = tile / w.TX;
    const int px = tx * kTile + (threadIdx.x & 15), py = ty * kTile + (threadIdx.x >> 4);
    if (px >= w.W || py >= w.H) return;
    const size_t HW = (size_t)w.W * w.H;
    const size_t q = (size_t)py * w.W + px;
    const float d = dfill[(size_t)(py >> 1) * Wg + (px >> 1)];
    if (d != kNoHit) {
        const float rx = ((float)px - w.kcur[2]) / w.kcur[0];
        const float ry = ((float)py - w.kcur[3]) / w.kcur[1];
        const float Px = d * rx, Py = d * ry, Pz = d;
        const float *M = w.Minv;
        const float X = ((M[0] * Px + M[1] * Py) + M[2] * Pz) + M[3];
        const float Y = ((M[4] * Px + M[5] * Py) + M[6] * Pz) + M[7];
        const float Z = ((M[8] * Px + M[9] * Py) + M[10] * Pz) + M[11];
        if (Z > w.z_near) {
            const float u = fminf(fmaxf(w.kref[0] * (X / Z) + w.kref[2], 0.0f), (float)(w.W - 1));
            const float v = fminf(fmaxf(w.kref[1] * (Y / Z) + w.kref[3], 0.0f), (float)(w.H - 1));
            stitch_sample(w, tab, u, v, q, rgb);
            return;
        }
    }
    rgb[q] = rgb[HW + q] = rgb[2 * HW + q] = 0.0f;   // cannot occur outside selected tiles
}

}  // namespace tgs
