// Depth fill and backward correspondence query of one tile of a TemporalGS
// frame (Sec. III-E), run by its own kernel or by the blocks of the
// preprocess launch past the Gaussians.
#pragma once

#include "tgs_internal.h"

namespace tgs {

// One block of tp x tp threads per tile (tp = 16 on the image, 8 on the
// half-resolution geometry-buffer grid, where a tile is 8 x 8 cells).
// The block also clears its tile's occluded flag for this frame and resets
// its cells of the other warp pair (dmin_next, smax_next) for the next one.
__device__ inline void fill_query_tile(const FillK &f, int tile) {
    const WarpK &w = f.w;
    const float *__restrict__ dmin = f.dmin;
    float *dfill = f.dfill;
    float2 *uv = f.uv;
    uint8_t *um = f.um, *oc = f.oc;
    float *dmin_next = f.dmin_next, *smax_next = f.smax_next;
    const int tx = tile % w.TX, ty = tile / w.TX;
    const int px = tx * w.tp + (int)(threadIdx.x % (unsigned)w.tp);
    const int py = ty * w.tp + (int)(threadIdx.x / (unsigned)w.tp);
    int bad = 0;
    if (threadIdx.x == 0) oc[tile] = 0;
    if (px < w.W && py < w.H) {
        const int q = py * w.W + px;
        dmin_next[q] = kNoHit;
        smax_next[q] = 0.0f;
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

}  // namespace tgs
