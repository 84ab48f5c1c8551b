// Per-Gaussian stage of a frame (3DGS preprocess, Sec. III-A) with the
// temporal dynamic culling of Sec. III-D and the newly-visible test of the
// occluded-tile detection (Sec. III-E) folded in.
//
// One thread per Gaussian.  Only the mean (16 bytes, one coalesced 1 KB
// request per wave) is read for a culled Gaussian; the geometry (32 bytes)
// for the survivors and the SH coefficients (192 of the 240 bytes per
// Gaussian at degree 3) for survivors that touch a tile, each Gaussian's
// bytes contiguous so that sparse survivors fetch only their own lines.  The
// kernel is HBM-bound.  In TemporalGS frames the launch also carries the
// depth fill / correspondence query (fill_query.h) on its blocks past the
// Gaussians', and in reference frames it clears the temporal Gaussian buffer.
// Quantities that decide a discrete outcome (near cull, frustum
// and occlusion tests, tile rectangle, sort depth) are computed in fp32 in a
// fixed order with contraction disabled for the whole library, so they are
// reproducible by any implementation that follows the same order.
#include "fill_query.h"
#include <hip/hip_ext.h>

#include "tgs_internal.h"

namespace tgs {

namespace {

template <int DEG>
__device__ inline void sh_colour(const SceneDev &s, int i, float dx, float dy, float dz,
                                 float &r, float &g, float &b) {
    constexpr int K = (DEG + 1) * (DEG + 1);
    constexpr int SLOTS = (3 * K + 3) / 4;
    float basis[K];
    basis[0] = 0.28209479177387814f;
    if constexpr (DEG >= 1) {
        const float C1 = 0.4886025119029199f;
        float inv = 1.0f / sqrtf(dx * dx + dy * dy + dz * dz);
        float x = dx * inv, y = dy * inv, z = dz * inv;
        basis[1] = -C1 * y;
        basis[2] = C1 * z;
        basis[3] = -C1 * x;
        if constexpr (DEG >= 2) {
            float xx = x * x, yy = y * y, zz = z * z, xy = x * y, yz = y * z, xz = x * z;
            basis[4] = 1.0925484305920792f * xy;
            basis[5] = -1.0925484305920792f * yz;
            basis[6] = 0.31539156525252005f * (2.0f * zz - xx - yy);
            basis[7] = -1.0925484305920792f * xz;
            basis[8] = 0.5462742152960396f * (xx - yy);
            if constexpr (DEG >= 3) {
                basis[9] = -0.5900435899266435f * y * (3.0f * xx - yy);
                basis[10] = 2.890611442640554f * xy * z;
                basis[11] = -0.4570457994644658f * y * (4.0f * zz - xx - yy);
                basis[12] = 0.3731763325901154f * z * (2.0f * zz - 3.0f * xx - 3.0f * yy);
                basis[13] = -0.4570457994644658f * x * (4.0f * zz - xx - yy);
                basis[14] = 1.445305721320277f * z * (xx - yy);
                basis[15] = -0.5900435899266435f * x * (xx - 3.0f * yy);
            }
        }
    }
    float f[4 * SLOTS];
    const float4 *p = s.sh + (size_t)i * SLOTS;
#pragma unroll
    for (int j = 0; j < SLOTS; ++j) {
        const float4 v = p[j];
        f[4 * j + 0] = v.x;
        f[4 * j + 1] = v.y;
        f[4 * j + 2] = v.z;
        f[4 * j + 3] = v.w;
    }
    float acc0 = 0.0f, acc1 = 0.0f, acc2 = 0.0f;
#pragma unroll
    for (int k = 0; k < K; ++k) {
        acc0 = __builtin_fmaf(basis[k], f[3 * k + 0], acc0);
        acc1 = __builtin_fmaf(basis[k], f[3 * k + 1], acc1);
        acc2 = __builtin_fmaf(basis[k], f[3 * k + 2], acc2);
    }
    r = fmaxf(acc0 + 0.5f, 0.0f);
    g = fmaxf(acc1 + 0.5f, 0.0f);
    b = fmaxf(acc2 + 0.5f, 0.0f);
}

// Blocks at or past n_pre (a TemporalGS frame with the full-resolution
// geometry buffer) run the depth fill / correspondence query of tile
// blockIdx.x - n_pre instead: independent of the preprocess, so it fills in
// beside it rather than taking a launch of its own.
template <int DEG>
__global__ __launch_bounds__(256) void preprocess_kernel(SceneDev s, CamK cam, CullK cull,
                                                         Records rec, Counters *cnt, FillK fill,
                                                         int n_pre) {
    if ((int)blockIdx.x >= n_pre) {   // block-uniform
        fill_query_tile(fill, (int)blockIdx.x - n_pre);
        return;
    }
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    bool survivor = false, newly = false;
    ushort4 rect = make_ushort4(1, 1, 0, 0);
    uint32_t keys = 0;

    if (i < s.n) {
        const float4 mo = s.mean_op[i];
        const float mx = mo.x, my = mo.y, mz = mo.z;
        const float *V = cam.V;
        const float tx = ((V[0] * mx + V[1] * my) + V[2] * mz) + V[3];
        const float ty = ((V[4] * mx + V[5] * my) + V[6] * mz) + V[7];
        const float tz = ((V[8] * mx + V[9] * my) + V[10] * mz) + V[11];
        bool alive = tz > cull.z_near;                      // near-plane culling
        float u = 0.0f, v = 0.0f;
        if (alive) {
            u = cam.fx * (tx / tz) + cam.cx;
            v = cam.fy * (ty / tz) + cam.cy;
            if (cull.afc) {                                 // adaptive frustum culling
                const float nx = (2.0f * u + 1.0f) / (float)cam.W - 1.0f;
                const float ny = (2.0f * v + 1.0f) / (float)cam.H - 1.0f;
                alive = ordered_to_float(cull.fbox[0]) <= nx && nx <= ordered_to_float(cull.fbox[2]) &&
                        ordered_to_float(cull.fbox[1]) <= ny && ny <= ordered_to_float(cull.fbox[3]);
            }
        }
        if (alive && cull.toc) {                            // occlusion culling, newly visible
            const float pxf = floorf(u + 0.5f), pyf = floorf(v + 0.5f);
            if (pxf >= 0.0f && pxf <= (float)(cam.W - 1) && pyf >= 0.0f &&
                pyf <= (float)(cam.H - 1) && !cull.g_rendered[i]) {
                // the geometry-buffer cell holding that pixel (its 2x2 block
                // when the buffer is downscaled)
                const int p = ((int)pyf >> cull.tgb_shift) * cull.tgb_w + ((int)pxf >> cull.tgb_shift);
                const float dm = cull.dmin[p];
                // with lambda2 = 0 the cull needs only the depth (dm + 0 * sm
                // is dm: sm is finite), so sm is read for the survivors only
                if (cull.lambda2 == 0.0f && tz > dm) {
                    alive = false;
                } else {
                    const float sm = cull.smax[p];
                    if (tz > dm + cull.lambda2 * sm) alive = false;
                    else if (tz <= dm - cull.lambda1 * sm) newly = true;
                }
            }
        }
        survivor = alive;
        if (alive) {
            // 3D covariance R S S^T R^T from the normalised quaternion
            const float4 sq = s.geo[2 * (size_t)i];
            const float4 qv = s.geo[2 * (size_t)i + 1];
            const float q0 = sq.w, q1 = qv.x, q2 = qv.y, q3 = qv.z;
            const float qn = sqrtf(((q0 * q0 + q1 * q1) + q2 * q2) + q3 * q3);
            const float r = q0 / qn, x = q1 / qn, y = q2 / qn, z = q3 / qn;
            float R[9];
            R[0] = 1.0f - 2.0f * (y * y + z * z);
            R[1] = 2.0f * (x * y - r * z);
            R[2] = 2.0f * (x * z + r * y);
            R[3] = 2.0f * (x * y + r * z);
            R[4] = 1.0f - 2.0f * (x * x + z * z);
            R[5] = 2.0f * (y * z - r * x);
            R[6] = 2.0f * (x * z - r * y);
            R[7] = 2.0f * (y * z + r * x);
            R[8] = 1.0f - 2.0f * (x * x + y * y);
            const float sc[3] = {sq.x, sq.y, sq.z};
            float M[9];
#pragma unroll
            for (int a = 0; a < 3; ++a)
#pragma unroll
                for (int c = 0; c < 3; ++c) M[a * 3 + c] = R[a * 3 + c] * sc[c];
            float S[9];
#pragma unroll
            for (int a = 0; a < 3; ++a)
#pragma unroll
                for (int c = 0; c < 3; ++c)
                    S[a * 3 + c] = (M[a * 3 + 0] * M[c * 3 + 0] + M[a * 3 + 1] * M[c * 3 + 1]) +
                                   M[a * 3 + 2] * M[c * 3 + 2];
            // EWA projection: J W Sigma W^T J^T + 0.3 I
            const float txc = fminf(cam.limx, fmaxf(-cam.limx, tx / tz)) * tz;
            const float tyc = fminf(cam.limy, fmaxf(-cam.limy, ty / tz)) * tz;
            const float j00 = cam.fx / tz, j02 = -(cam.fx * txc) / (tz * tz);
            const float j11 = cam.fy / tz, j12 = -(cam.fy * tyc) / (tz * tz);
            float A[6];
#pragma unroll
            for (int c = 0; c < 3; ++c) {
                A[c] = j00 * V[c] + j02 * V[8 + c];
                A[3 + c] = j11 * V[4 + c] + j12 * V[8 + c];
            }
            float B[6];
#pragma unroll
            for (int a = 0; a < 2; ++a)
#pragma unroll
                for (int c = 0; c < 3; ++c)
                    B[a * 3 + c] = (A[a * 3 + 0] * S[c] + A[a * 3 + 1] * S[3 + c]) + A[a * 3 + 2] * S[6 + c];
            const float ca = ((B[0] * A[0] + B[1] * A[1]) + B[2] * A[2]) + 0.3f;
            const float cb = (B[0] * A[3] + B[1] * A[4]) + B[2] * A[5];
            const float cc = ((B[3] * A[3] + B[4] * A[4]) + B[5] * A[5]) + 0.3f;
            const float det = ca * cc - cb * cb;
            if (det > 0.0f && (!cull.footprint || mo.w >= kAlphaMin)) {
                const float dinv = 1.0f / det;
                // Tile rectangle: tiles whose pixel-centre span meets the box
                // [u-hx, u+hx] x [v-hy, v+hy].
                float hx, hy;
                if (cull.footprint) {
                    // Bounding box of the ellipse where the Gaussian can reach
                    // alpha >= 1/255: d^T Sigma'^-1 d <= 2 ln(255 o).  kq bounds
                    // that from above without a transcendental (exact exponent
                    // plus the tangent of log2 at sqrt 2 for the mantissa, which
                    // lies above log2 on [1, 2)), so the rectangle is exactly
                    // reproducible; half extents sqrt(kq Sigma'_xx),
                    // sqrt(kq Sigma'_yy), enlarged by 0.1% + 0.01 px.
                    const uint32_t xb = __float_as_uint(fmaxf(255.0f * mo.w, 1.0f));
                    const int e = (int)((xb >> 23) & 255u) - 127;
                    const float m = __uint_as_float((xb & 0x007fffffu) | 0x3f800000u);
                    float t = m - 1.4142135f;
                    t = 1.0201394f * t;
                    t = 0.5f + t;
                    float L = (float)e + t;
                    L = L + 1e-4f;
                    const float kq = 1.3862944f * L;
                    hx = sqrtf(kq * ca) * 1.001f + 0.01f;
                    hy = sqrtf(kq * cc) * 1.001f + 0.01f;
                } else {
                    // 3DGS: 3 sigma of the larger eigenvalue of Sigma', rounded up
                    const float mid = 0.5f * (ca + cc);
                    const float lam = mid + sqrtf(fmaxf(0.0f, mid * mid - det));
                    hx = hy = ceilf(3.0f * sqrtf(lam));
                }
                const float x0 = fmaxf(0.0f, ceilf(((u - hx) - 15.0f) / 16.0f));
                const float x1 = fminf((float)(cam.TX - 1), floorf((u + hx) / 16.0f));
                const float y0 = fmaxf(0.0f, ceilf(((v - hy) - 15.0f) / 16.0f));
                const float y1 = fminf((float)(cam.TY - 1), floorf((v + hy) / 16.0f));
                if (x0 <= x1 && y0 <= y1) {
                    rect = make_ushort4((unsigned short)x0, (unsigned short)y0,
                                        (unsigned short)x1, (unsigned short)y1);
                    keys = (uint32_t)(rect.z - rect.x + 1) * (uint32_t)(rect.w - rect.y + 1);
                    float cr, cg, cbl;
                    sh_colour<DEG>(s, i, mx - cam.campos[0], my - cam.campos[1],
                                   mz - cam.campos[2], cr, cg, cbl);
                    const float con_a = cc * dinv, con_b = -cb * dinv, con_c = ca * dinv;
                    // blend culling box: alpha >= 1/255 <=> d^T Sigma'^-1 d <=
                    // 2 ln(255 o), an ellipse with half extents sqrt(k Sigma'_xx),
                    // sqrt(k Sigma'_yy); enlarged so that every pixel left out
                    // has alpha well below the threshold
                    float bx = -1.0f, by = -1.0f, kq = 0.0f;
                    if (mo.w >= 0.999f * kAlphaMin) {
                        kq = 2.0f * __logf(fmaxf(255.0f * mo.w, 1.0f)) + 1e-3f;
                        bx = sqrtf(kq * ca) * 1.002f + 0.05f;
                        by = sqrtf(kq * cc) * 1.002f + 0.05f;
                    }
                    constexpr float kLog2e = 1.4426950408889634f;
                    float4 *r = rec.g + 4 * (size_t)i;
                    r[0] = make_float4(u, v, con_a, con_b);
                    r[1] = make_float4(con_c, mo.w, tz, by);
                    r[2] = make_float4(cr, cg, cbl, bx);
                    r[3] = make_float4(-0.5f * kLog2e * con_a, -kLog2e * con_b, -0.5f * kLog2e * con_c, kq);
                }
            }
        }
        rec.rect[i] = rect;
        rec.count[i] = keys;
        rec.dkey[i] = __float_as_uint(tz);
        rec.status[i] = (uint8_t)((survivor ? 1 : 0) | (newly ? 2 : 0));
        if (cull.clear_flag) cull.clear_flag[i] = 0u;
    }

    // per-block counts (no contended device-wide atomics)
    __shared__ uint32_t s_cnt[4][2];
    const uint64_t surv_mask = __ballot(survivor);
    const uint64_t newly_mask = __ballot(newly);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    if (lane == 0) {
        s_cnt[wave][0] = (uint32_t)__popcll(surv_mask);
        s_cnt[wave][1] = (uint32_t)__popcll(newly_mask);
    }
    __syncthreads();
    if (threadIdx.x < 2)
        rec.partial[2 * blockIdx.x + threadIdx.x] = s_cnt[0][threadIdx.x] + s_cnt[1][threadIdx.x] +
                                                    s_cnt[2][threadIdx.x] + s_cnt[3][threadIdx.x];
    (void)cnt;
}

}  // namespace

void launch_preprocess(const SceneDev &s, const CamK &cam, const CullK &cull, Records rec,
                       Counters *cnt, const FillK *fill, hipStream_t st, hipEvent_t start,
                       hipEvent_t stop) {
    const int n_pre = s.n > 0 ? preprocess_blocks(s.n) : 0;
    // the fill blocks need 256 threads per tile: full-resolution grid only
    const bool with_fill = fill && fill->w.tp * fill->w.tp == 256;
    if (fill && !with_fill) launch_fill_query(*fill, st);
    const int n_fill = with_fill ? fill->w.TX * fill->w.TY : 0;
    if (n_pre + n_fill <= 0) return;
    const FillK f = with_fill ? *fill : FillK{};
    const dim3 grid(n_pre + n_fill), block(256);
    // start / stop (may be NULL) are attached to the dispatch itself
    switch (s.deg) {
        case 0:
            hipExtLaunchKernelGGL(preprocess_kernel<0>, grid, block, 0, st, start, stop, 0, s, cam, cull,
                                  rec, cnt, f, n_pre);
            break;
        case 1:
            hipExtLaunchKernelGGL(preprocess_kernel<1>, grid, block, 0, st, start, stop, 0, s, cam, cull,
                                  rec, cnt, f, n_pre);
            break;
        case 2:
            hipExtLaunchKernelGGL(preprocess_kernel<2>, grid, block, 0, st, start, stop, 0, s, cam, cull,
                                  rec, cnt, f, n_pre);
            break;
        default:
            hipExtLaunchKernelGGL(preprocess_kernel<3>, grid, block, 0, st, start, stop, 0, s, cam, cull,
                                  rec, cnt, f, n_pre);
            break;
    }
}

}  // namespace tgs
