/*
 * TemporalGS CPU oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, single-threaded reference of the TemporalGS frame path:
 * the 3DGS tile rasteriser the method plugs into (Sec. III-A), the temporal
 * priors (Sec. III-C, Eq. 1-3), temporal dynamic culling (Sec. III-D) and
 * selective rendering (Sec. III-E, Eq. 4).  Only the test-suite, the package
 * smoke check and the benchmark's CPU-baseline leg load this file; the
 * product path never does.  It shares no code with the HIP library.
 *
 * Precision.  Every quantity that feeds a discrete decision (near cull, tile
 * rectangle, sort key, frustum/occlusion tests, warp destinations, fill,
 * correspondence, alpha thresholds) is evaluated in IEEE fp32 in the order
 * written below, compiled without contraction (-ffp-contract=off), because
 * such decisions must be taken in the precision of the kernel that takes
 * them.  Continuous outputs (SH colour, blended colour, Eq. 1/2 depth
 * moments, bilinear stitching) are accumulated in fp64.
 *
 * The only non-reproducible fp32 step is exp() in the blending opacity; the
 * oracle records, per pixel and per (Gaussian, tile) pair, where a decision
 * lies within a stated margin of its threshold so that tests can exclude it.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define OR_NOHIT 1001.0f          /* z_far (1000) + epsilon (1), Sec. III-C */
#define OR_ALPHA_MIN (1.0f / 255.0f)
#define OR_ALPHA_MAX 0.99f
#define OR_T_MIN 1e-4f
/* margins: decisions this close to their threshold are reported as uncertain */
#define OR_MARGIN_ALPHA (1e-5 / 255.0)
#define OR_MARGIN_T (1e-4 * 1e-4)
#define OR_MARGIN_POWER 1e-6
/* Relative difference between two evaluations of one alpha from the same
 * fp32 exponent (exp2 implementations and the opacity product), in units of
 * roundoff u = 2^-24: bounds the difference of each composited weight, and
 * through it of Eq. 1/2, reported per pixel. */
#define OR_U32 5.9604644775390625e-8
#define OR_ALPHA_ULPS 4.0
/* log2(e) as a float: the blend takes alpha = o 2^p2 with the exponent in
 * base 2 */
#define OR_LOG2E 1.4426950408889634f

enum { OR_TILES_3SIGMA = 0, OR_TILES_FOOTPRINT = 1 };
enum { OR_NEAR_CULLED = 0, OR_AFC_CULLED = 1, OR_TOC_CULLED = 2, OR_DEGENERATE = 3,
       OR_NO_TILES = 4, OR_VISIBLE = 5 };

typedef struct {
    float w2c[16];
    float fx, fy, cx, cy;
    int32_t width, height;
} or_camera;

/* ------------------------------------------------------------------------ */
/* small helpers                                                            */
/* ------------------------------------------------------------------------ */

static uint32_t f2u(float f) { uint32_t u; memcpy(&u, &f, 4); return u; }

/* Camera centre c = -R^T t of a rigid world->camera matrix, in double. */
void or_camera_centre(const float *w2c, float *c)
{
    for (int i = 0; i < 3; ++i) {
        double s = (double)w2c[0 * 4 + i] * (double)w2c[3]
                 + (double)w2c[1 * 4 + i] * (double)w2c[7]
                 + (double)w2c[2 * 4 + i] * (double)w2c[11];
        c[i] = (float)(-s);
    }
}

/* Relative pose of Eq. 3: M = W_cur * W_ref^-1 (reference camera -> current
 * camera) and its inverse, both as 3x4 row-major fp32, formed in double with
 * the rigid inverse [R^T | -R^T t]. */
static void rigid_inverse(const double *a, double *inv)
{
    for (int i = 0; i < 3; ++i) {
        for (int j = 0; j < 3; ++j) inv[i * 4 + j] = a[j * 4 + i];
        inv[i * 4 + 3] = -(a[0 * 4 + i] * a[3] + a[1 * 4 + i] * a[7] + a[2 * 4 + i] * a[11]);
    }
    inv[12] = inv[13] = inv[14] = 0.0; inv[15] = 1.0;
}

static void mat4_mul(const double *a, const double *b, double *c)
{
    for (int i = 0; i < 4; ++i)
        for (int j = 0; j < 4; ++j) {
            double s = 0.0;
            for (int k = 0; k < 4; ++k) s += a[i * 4 + k] * b[k * 4 + j];
            c[i * 4 + j] = s;
        }
}

void or_relative_pose(const float *w2c_ref, const float *w2c_cur, float *m, float *minv)
{
    double r[16], c[16], rinv[16], cinv[16], t[16];
    for (int i = 0; i < 16; ++i) { r[i] = w2c_ref[i]; c[i] = w2c_cur[i]; }
    r[12] = r[13] = r[14] = 0.0; r[15] = 1.0;
    c[12] = c[13] = c[14] = 0.0; c[15] = 1.0;
    rigid_inverse(r, rinv);
    rigid_inverse(c, cinv);
    mat4_mul(c, rinv, t);
    for (int i = 0; i < 12; ++i) m[i] = (float)t[i];
    mat4_mul(r, cinv, t);
    for (int i = 0; i < 12; ++i) minv[i] = (float)t[i];
}

/* Rotation from a quaternion (w,x,y,z), normalised first (Sec. III-A; the
 * covariance parameterisation of the cited 3DGS work). */
void or_quat_to_rot(const float *q, float *R)
{
    float n = sqrtf(((q[0] * q[0] + q[1] * q[1]) + q[2] * q[2]) + q[3] * q[3]);
    float r = q[0] / n, x = q[1] / n, y = q[2] / n, z = q[3] / n;
    R[0] = 1.0f - 2.0f * (y * y + z * z);
    R[1] = 2.0f * (x * y - r * z);
    R[2] = 2.0f * (x * z + r * y);
    R[3] = 2.0f * (x * y + r * z);
    R[4] = 1.0f - 2.0f * (x * x + z * z);
    R[5] = 2.0f * (y * z - r * x);
    R[6] = 2.0f * (x * z - r * y);
    R[7] = 2.0f * (y * z + r * x);
    R[8] = 1.0f - 2.0f * (x * x + y * y);
}

/* 3D covariance Sigma = R S S^T R^T, returned as the full 3x3 matrix. */
void or_cov3d(const float *scale, const float *q, float *S)
{
    float R[9], M[9];
    or_quat_to_rot(q, R);
    for (int i = 0; i < 3; ++i)
        for (int j = 0; j < 3; ++j) M[i * 3 + j] = R[i * 3 + j] * scale[j];
    for (int i = 0; i < 3; ++i)
        for (int j = 0; j < 3; ++j)
            S[i * 3 + j] = (M[i * 3 + 0] * M[j * 3 + 0] + M[i * 3 + 1] * M[j * 3 + 1]) + M[i * 3 + 2] * M[j * 3 + 2];
}

/* Real spherical harmonics up to degree 3 (3DGS colour model), in double.
 * basis[k] for k < (deg+1)^2 at unit direction (x,y,z). */
void or_sh_basis(int deg, double x, double y, double z, double *basis)
{
    const double C0 = 0.28209479177387814;
    const double C1 = 0.4886025119029199;
    const double C2[5] = {1.0925484305920792, -1.0925484305920792, 0.31539156525252005,
                          -1.0925484305920792, 0.5462742152960396};
    const double C3[7] = {-0.5900435899266435, 2.890611442640554, -0.4570457994644658,
                          0.3731763325901154, -0.4570457994644658, 1.445305721320277,
                          -0.5900435899266435};
    basis[0] = C0;
    if (deg < 1) return;
    basis[1] = -C1 * y;
    basis[2] = C1 * z;
    basis[3] = -C1 * x;
    if (deg < 2) return;
    double xx = x * x, yy = y * y, zz = z * z, xy = x * y, yz = y * z, xz = x * z;
    basis[4] = C2[0] * xy;
    basis[5] = C2[1] * yz;
    basis[6] = C2[2] * (2.0 * zz - xx - yy);
    basis[7] = C2[3] * xz;
    basis[8] = C2[4] * (xx - yy);
    if (deg < 3) return;
    basis[9] = C3[0] * y * (3.0 * xx - yy);
    basis[10] = C3[1] * xy * z;
    basis[11] = C3[2] * y * (4.0 * zz - xx - yy);
    basis[12] = C3[3] * z * (2.0 * zz - 3.0 * xx - 3.0 * yy);
    basis[13] = C3[4] * x * (4.0 * zz - xx - yy);
    basis[14] = C3[5] * z * (xx - yy);
    basis[15] = C3[6] * x * (xx - 3.0 * yy);
}

/* ------------------------------------------------------------------------ */
/* Per-Gaussian stage: near-plane cull, projection, adaptive frustum culling */
/* (Sec. III-D), temporal occlusion culling and the newly-visible test       */
/* (Sec. III-D/III-E), then 2D covariance, extent, tile rectangle, colour    */
/* for the survivors (Sec. III-A).                                           */
/* ------------------------------------------------------------------------ */

typedef struct {
    int32_t afc;             /* apply adaptive frustum culling            */
    float fbox[4];           /* F_min.x, F_min.y, F_max.x, F_max.y (NDC)  */
    int32_t toc;             /* apply occlusion culling + newly-visible   */
    const float *dmin;       /* warped min depth on the TGB grid          */
    const float *smax;       /* warped max std on the TGB grid            */
    const uint8_t *g_rendered; /* temporal Gaussian buffer [N]            */
    float lambda1, lambda2;
    int32_t tgb_shift;       /* TGB grid = image >> tgb_shift (0 or 1)    */
    int32_t tgb_w;           /* width of the TGB grid                     */
} or_cull;

int32_t or_gaussians(int32_t n, int32_t sh_degree, const float *means, const float *scales,
                     const float *rots, const float *opac, const float *sh, const or_camera *cam,
                     float z_near, const or_cull *cull, int32_t tile_bound,
                     int32_t *status, uint8_t *newly_visible, float *mean2d, float *ndc,
                     float *depth, float *conic, float *extent, int32_t *rect, double *rgb)
{
    const float *V = cam->w2c;
    const int W = cam->width, H = cam->height;
    const int TX = (W + 15) / 16, TY = (H + 15) / 16;
    const float tanfx = (0.5f * (float)W) / cam->fx;
    const float tanfy = (0.5f * (float)H) / cam->fy;
    const float limx = 1.3f * tanfx, limy = 1.3f * tanfy;
    float campos[3];
    or_camera_centre(V, campos);
    const int ncoef = (sh_degree + 1) * (sh_degree + 1);
    int32_t survivors = 0;

    for (int i = 0; i < n; ++i) {
        const float mx = means[3 * i], my = means[3 * i + 1], mz = means[3 * i + 2];
        newly_visible[i] = 0;
        rect[4 * i + 0] = 1; rect[4 * i + 1] = 1; rect[4 * i + 2] = 0; rect[4 * i + 3] = 0;
        mean2d[2 * i] = mean2d[2 * i + 1] = 0.0f;
        ndc[2 * i] = ndc[2 * i + 1] = 0.0f;
        depth[i] = 0.0f;
        conic[3 * i] = conic[3 * i + 1] = conic[3 * i + 2] = 0.0f;
        extent[2 * i] = extent[2 * i + 1] = 0.0f;
        float x0 = 1.0f, x1 = 0.0f, y0 = 1.0f, y1 = 0.0f;
        rgb[3 * i] = rgb[3 * i + 1] = rgb[3 * i + 2] = 0.0;

        /* view-space position */
        float tx = ((V[0] * mx + V[1] * my) + V[2] * mz) + V[3];
        float ty = ((V[4] * mx + V[5] * my) + V[6] * mz) + V[7];
        float tz = ((V[8] * mx + V[9] * my) + V[10] * mz) + V[11];
        if (!(tz > z_near)) { status[i] = OR_NEAR_CULLED; continue; }
        depth[i] = tz;

        /* projected mean and its NDC (Pix2NDC, Sec. III-D) */
        float u = cam->fx * (tx / tz) + cam->cx;
        float v = cam->fy * (ty / tz) + cam->cy;
        mean2d[2 * i] = u; mean2d[2 * i + 1] = v;
        float nx = (2.0f * u + 1.0f) / (float)W - 1.0f;
        float ny = (2.0f * v + 1.0f) / (float)H - 1.0f;
        ndc[2 * i] = nx; ndc[2 * i + 1] = ny;

        if (cull && cull->afc) {
            if (!(cull->fbox[0] <= nx && nx <= cull->fbox[2] &&
                  cull->fbox[1] <= ny && ny <= cull->fbox[3])) { status[i] = OR_AFC_CULLED; continue; }
        }
        if (cull && cull->toc) {
            /* nearest pixel of the projected mean; only on-screen means are tested */
            float pxf = floorf(u + 0.5f), pyf = floorf(v + 0.5f);
            if (pxf >= 0.0f && pxf <= (float)(W - 1) && pyf >= 0.0f && pyf <= (float)(H - 1) &&
                !cull->g_rendered[i]) {
                /* the TGB cell holding that pixel (a 2x2 block when downscaled) */
                int p = ((int)pyf >> cull->tgb_shift) * cull->tgb_w + ((int)pxf >> cull->tgb_shift);
                float dm = cull->dmin[p], sm = cull->smax[p];
                if (tz > dm + cull->lambda2 * sm) { status[i] = OR_TOC_CULLED; continue; }
                if (tz <= dm - cull->lambda1 * sm) newly_visible[i] = 1;
            }
        }
        ++survivors;

        /* 2D covariance: J W Sigma W^T J^T plus the 0.3 px low-pass */
        float txtz = tx / tz, tytz = ty / tz;
        float txc = fminf(limx, fmaxf(-limx, txtz)) * tz;
        float tyc = fminf(limy, fmaxf(-limy, tytz)) * tz;
        float j00 = cam->fx / tz, j02 = -(cam->fx * txc) / (tz * tz);
        float j11 = cam->fy / tz, j12 = -(cam->fy * tyc) / (tz * tz);
        float A[6];
        for (int j = 0; j < 3; ++j) {
            A[j] = j00 * V[0 * 4 + j] + j02 * V[2 * 4 + j];
            A[3 + j] = j11 * V[1 * 4 + j] + j12 * V[2 * 4 + j];
        }
        float S[9];
        or_cov3d(&scales[3 * i], &rots[4 * i], S);
        float B[6];
        for (int r = 0; r < 2; ++r)
            for (int j = 0; j < 3; ++j)
                B[r * 3 + j] = (A[r * 3 + 0] * S[0 * 3 + j] + A[r * 3 + 1] * S[1 * 3 + j]) + A[r * 3 + 2] * S[2 * 3 + j];
        float ca = ((B[0] * A[0] + B[1] * A[1]) + B[2] * A[2]) + 0.3f;
        float cb = (B[0] * A[3] + B[1] * A[4]) + B[2] * A[5];
        float cc = ((B[3] * A[3] + B[4] * A[4]) + B[5] * A[5]) + 0.3f;
        float det = ca * cc - cb * cb;
        if (!(det > 0.0f)) { status[i] = OR_DEGENERATE; continue; }
        float dinv = 1.0f / det;
        conic[3 * i] = cc * dinv;
        conic[3 * i + 1] = -cb * dinv;
        conic[3 * i + 2] = ca * dinv;

        /* Tile rectangle: the tiles whose pixel-centre span [16k, 16k+15]
         * meets the box [u-hx, u+hx] x [v-hy, v+hy] (Sec. III-A duplicates a
         * Gaussian into every tile it intersects).
         * OR_TILES_3SIGMA (3DGS): hx = hy = ceil(3 sqrt(lambda_max(Sigma'))).
         * OR_TILES_FOOTPRINT: the bounding box of the ellipse where the
         * Gaussian can reach alpha >= 1/255.  A pixel at offset d does so
         * only if o exp(-q/2) >= 1/255 with q = d^T Sigma'^-1 d, i.e.
         * q <= 2 ln(255 o); the box has half extents sqrt(kq Sigma'_xx),
         * sqrt(kq Sigma'_yy).  kq bounds 2 ln(255 o) from above without a
         * transcendental: log2 x = e + log2 m (x = m 2^e, m in [1,2)), and
         * log2 m lies below its tangent at sqrt(2).  The box is enlarged by
         * 0.1% + 0.01 px, so every pixel left out has alpha well below
         * 1/255; opacity below 1/255 reaches no pixel. */
        {
            float hx, hy;
            if (tile_bound == OR_TILES_FOOTPRINT) {
                if (!(opac[i] >= OR_ALPHA_MIN)) { status[i] = OR_NO_TILES; goto colour; }
                float x = fmaxf(255.0f * opac[i], 1.0f);
                uint32_t xb = f2u(x);
                int e = (int)((xb >> 23) & 255u) - 127;
                uint32_t mb = (xb & 0x007fffffu) | 0x3f800000u;
                float m;
                memcpy(&m, &mb, 4);
                float t = m - 1.4142135f;
                t = 1.0201394f * t;
                t = 0.5f + t;
                float L = (float)e + t;
                L = L + 1e-4f;
                float kq = 1.3862944f * L;
                hx = sqrtf(kq * ca) * 1.001f + 0.01f;
                hy = sqrtf(kq * cc) * 1.001f + 0.01f;
            } else {
                float mid = 0.5f * (ca + cc);
                float lam = mid + sqrtf(fmaxf(0.0f, mid * mid - det));
                hx = hy = ceilf(3.0f * sqrtf(lam));
            }
            extent[2 * i] = hx;
            extent[2 * i + 1] = hy;
            x0 = fmaxf(0.0f, ceilf(((u - hx) - 15.0f) / 16.0f));
            x1 = fminf((float)(TX - 1), floorf((u + hx) / 16.0f));
            y0 = fmaxf(0.0f, ceilf(((v - hy) - 15.0f) / 16.0f));
            y1 = fminf((float)(TY - 1), floorf((v + hy) / 16.0f));
            status[i] = (x0 <= x1 && y0 <= y1) ? OR_VISIBLE : OR_NO_TILES;
        }
    colour:
        /* colour from SH along the viewing direction, +0.5, clamped at 0 */
        {
            double dx = (double)mx - campos[0], dy = (double)my - campos[1], dz = (double)mz - campos[2];
            double dn = sqrt(dx * dx + dy * dy + dz * dz);
            double basis[16];
            or_sh_basis(sh_degree, dx / dn, dy / dn, dz / dn, basis);
            for (int ch = 0; ch < 3; ++ch) {
                double sacc = 0.0;
                for (int k = 0; k < ncoef; ++k) sacc += basis[k] * (double)sh[((size_t)i * ncoef + k) * 3 + ch];
                sacc += 0.5;
                rgb[3 * i + ch] = sacc > 0.0 ? sacc : 0.0;
            }
        }
        if (status[i] == OR_VISIBLE) {
            rect[4 * i + 0] = (int)x0; rect[4 * i + 1] = (int)y0;
            rect[4 * i + 2] = (int)x1; rect[4 * i + 3] = (int)y1;
        }
    }
    return survivors;
}

/* ------------------------------------------------------------------------ */
/* Duplication + per-tile depth sort (Sec. III-A): each tile's list holds    */
/* the visible Gaussians whose rectangle contains it, front to back by       */
/* (depth bits, Gaussian index).  tile_sel == NULL selects every tile.       */
/* ------------------------------------------------------------------------ */

typedef struct { uint32_t dbits; int32_t idx; } or_item;

static int item_cmp(const void *a, const void *b)
{
    const or_item *x = (const or_item *)a, *y = (const or_item *)b;
    if (x->dbits != y->dbits) return x->dbits < y->dbits ? -1 : 1;
    return (x->idx > y->idx) - (x->idx < y->idx);
}

/* Pass 1: per-tile counts; returns total K.  tile_start has TX*TY+1 entries. */
int64_t or_tile_counts(int32_t n, const int32_t *status, const int32_t *rect, int32_t TX, int32_t TY,
                       const uint8_t *tile_sel, int64_t *tile_start)
{
    const int nt = TX * TY;
    for (int t = 0; t <= nt; ++t) tile_start[t] = 0;
    for (int i = 0; i < n; ++i) {
        if (status[i] != OR_VISIBLE) continue;
        for (int y = rect[4 * i + 1]; y <= rect[4 * i + 3]; ++y)
            for (int x = rect[4 * i + 0]; x <= rect[4 * i + 2]; ++x)
                if (!tile_sel || tile_sel[y * TX + x]) tile_start[y * TX + x + 1]++;
    }
    for (int t = 0; t < nt; ++t) tile_start[t + 1] += tile_start[t];
    return tile_start[nt];
}

/* Pass 2: fill and sort. items has K entries. */
void or_tile_lists(int32_t n, const int32_t *status, const int32_t *rect, const float *depth,
                   int32_t TX, int32_t TY, const uint8_t *tile_sel, const int64_t *tile_start,
                   int32_t *items)
{
    const int nt = TX * TY;
    int64_t *fill = (int64_t *)malloc(sizeof(int64_t) * (size_t)nt);
    for (int t = 0; t < nt; ++t) fill[t] = tile_start[t];
    int64_t K = tile_start[nt];
    or_item *buf = (or_item *)malloc(sizeof(or_item) * (size_t)(K > 0 ? K : 1));
    for (int i = 0; i < n; ++i) {
        if (status[i] != OR_VISIBLE) continue;
        for (int y = rect[4 * i + 1]; y <= rect[4 * i + 3]; ++y)
            for (int x = rect[4 * i + 0]; x <= rect[4 * i + 2]; ++x) {
                int t = y * TX + x;
                if (tile_sel && !tile_sel[t]) continue;
                buf[fill[t]].dbits = f2u(depth[i]);
                buf[fill[t]].idx = i;
                fill[t]++;
            }
    }
    for (int t = 0; t < nt; ++t) {
        int64_t s = tile_start[t], e = tile_start[t + 1];
        if (e - s > 1) qsort(buf + s, (size_t)(e - s), sizeof(or_item), item_cmp);
    }
    for (int64_t k = 0; k < K; ++k) items[k] = buf[k].idx;
    free(buf);
    free(fill);
}

/* ------------------------------------------------------------------------ */
/* Front-to-back alpha blending of one pixel over an ordered candidate set   */
/* (Sec. III-A), with the weights w_i = alpha_i T_i that define Eq. 1, Eq. 2  */
/* and the temporal Gaussian buffer.                                         */
/* ------------------------------------------------------------------------ */

typedef struct {
    const float *mean2d, *conic, *opac, *depth;
    const double *rgb;
    const float *bg;         /* background colour [3] */
    float *maxw;             /* [N] or NULL */
    uint8_t *g_certain;      /* [N] or NULL: included before any margin event */
    uint8_t *g_uncertain;    /* [N] or NULL: at/after a margin event          */
    double *wbuf, *dbuf;     /* scratch of list length                         */
} or_blend_ctx;

typedef struct {
    double rgb[3], D, sigma, alpha;
    int32_t margin_pos;
    int64_t evaluated, hits;
    int32_t ninc;            /* Gaussians composited                          */
    float spread;            /* largest |d - d0| among them (d0: the first)   */
    float wrel;              /* bound on the relative error of any of their   */
                             /* weights alpha T in fp32: the alpha's own      */
                             /* evaluation and the transmittance product      */
                             /* before it                                     */
} or_pixel;

static void blend_pixel(const or_blend_ctx *c, const int32_t *list, int64_t len, float px, float py,
                        or_pixel *out)
{
    float T = 1.0f;
    double C[3] = {0.0, 0.0, 0.0};
    double chain = 0.0, wrel = 0.0;   /* relative error of T, and the largest of a weight */
    int64_t ninc = 0, hits = 0;
    int32_t mpos = -1;
    int64_t j;
    for (j = 0; j < len; ++j) {
        int i = list[j];
        float dx = c->mean2d[2 * i] - px, dy = c->mean2d[2 * i + 1] - py;
        float A = c->conic[3 * i], B = c->conic[3 * i + 1], Cc = c->conic[3 * i + 2];
        /* the exponent -(A dx^2 + C dy^2)/2 - B dx dy in base 2, evaluated as
         * the blend kernel evaluates it: a conic pre-scaled by -log2(e) (1/2
         * on the squares) and fused multiply-adds.  For an elongated
         * footprint the terms are thousands of times the result, so any
         * other order of evaluation would differ by far more than a unit of
         * roundoff; taken in the kernel's order the alpha decisions and
         * weights differ only by the exp2 implementations. */
        const float qa = (-0.5f * OR_LOG2E) * A, qb = -OR_LOG2E * B, qc = (-0.5f * OR_LOG2E) * Cc;
        float power = fmaf(dx, fmaf(qa, dx, qb * dy), qc * dy * dy);
        int margin = fabs((double)power) <= OR_MARGIN_POWER;
        int include = 0, stop = 0;
        if (!(power > 0.0f)) {
            float alpha = fminf(OR_ALPHA_MAX, c->opac[i] * exp2f(power));
            if (fabs((double)alpha - (double)OR_ALPHA_MIN) <= OR_MARGIN_ALPHA) margin = 1;
            if (!(alpha < OR_ALPHA_MIN)) {
                ++hits;   /* composited, or the pair that stops the pixel */
                float Tn = T * (1.0f - alpha);
                if (fabs((double)Tn - (double)OR_T_MIN) <= OR_MARGIN_T) margin = 1;
                if (Tn < OR_T_MIN) {
                    stop = 1;
                } else {
                    float w = alpha * T;
                    /* alpha's relative error: its exponent's (zero where the
                     * 0.99 cap decides); 1 - alpha carries alpha / (1 - alpha)
                     * of it into every later transmittance */
                    const double ra = alpha == OR_ALPHA_MAX ? 0.0 : OR_ALPHA_ULPS * OR_U32;
                    const double rw = ra + chain + 2.0 * OR_U32;
                    if (rw > wrel) wrel = rw;
                    chain += (double)alpha / (1.0 - (double)alpha) * ra + 2.0 * OR_U32;
                    for (int ch = 0; ch < 3; ++ch) C[ch] += (double)w * c->rgb[3 * i + ch];
                    c->wbuf[ninc] = (double)w;
                    c->dbuf[ninc] = (double)c->depth[i];
                    ++ninc;
                    if (c->maxw && w > c->maxw[i]) c->maxw[i] = w;
                    include = 1;
                    T = Tn;
                }
            }
        }
        if (margin && mpos < 0) mpos = (int32_t)j;
        if (include) {
            if (mpos < 0) { if (c->g_certain) c->g_certain[i] = 1; }
            else if (c->g_uncertain) c->g_uncertain[i] = 1;
        }
        if (stop) break;
    }
    out->evaluated = j < len ? j + 1 : len;
    out->hits = hits;
    if (mpos >= 0 && c->g_uncertain)
        for (int64_t k = mpos; k < len; ++k) c->g_uncertain[list[k]] = 1;
    /* the background seen through the transmittance left: rgb = C + T bg */
    for (int ch = 0; ch < 3; ++ch) out->rgb[ch] = C[ch] + (double)T * (double)c->bg[ch];
    out->alpha = 1.0 - (double)T;
    /* the arithmetic size of Eq. 1/2 at this pixel: terms and depth spread */
    out->ninc = (int32_t)ninc;
    out->wrel = (float)wrel;
    out->spread = 0.0f;
    for (int64_t k = 1; k < ninc; ++k) {
        double e = fabs(c->dbuf[k] - c->dbuf[0]);
        if (e > out->spread) out->spread = (float)e;
    }
    /* Eq. 1 and Eq. 2 (two-pass) over the included weights */
    double sw = 0.0, swd = 0.0;
    for (int64_t k = 0; k < ninc; ++k) { sw += c->wbuf[k]; swd += c->wbuf[k] * c->dbuf[k]; }
    if (sw > 0.0) {
        double D = swd / sw, s2 = 0.0;
        for (int64_t k = 0; k < ninc; ++k) s2 += c->wbuf[k] * (c->dbuf[k] - D) * (c->dbuf[k] - D);
        out->D = D;
        out->sigma = sqrt(s2 / sw);
    } else {
        out->D = (double)OR_NOHIT;
        out->sigma = 0.0;
    }
    out->margin_pos = mpos;
}

/* Tiled blend over the listed tiles (all tiles if render_tiles == NULL).
 * Outputs are planar [3][H][W] / [H][W]; only pixels of rendered tiles are
 * written.  Returns the number of (pixel, Gaussian) pairs evaluated (list
 * entries up to and including the stopping one); *out_hits (if not NULL)
 * receives the number of those pairs whose alpha reaches 1/255. */
int64_t or_blend(int32_t W, int32_t H, const int64_t *tile_start, const int32_t *items,
                 const int32_t *render_tiles, int32_t n_render,
                 const float *mean2d, const float *conic, const float *opac, const float *depth,
                 const double *rgb, const float *bg, double *out_rgb, double *out_D, double *out_sigma,
                 double *out_alpha, int32_t *out_margin_pos, float *maxw, uint8_t *g_certain,
                 uint8_t *g_uncertain, int64_t *out_hits, int32_t *out_ninc, float *out_spread,
                 float *out_wrel)
{
    const int TX = (W + 15) / 16, TY = (H + 15) / 16;
    int64_t maxlen = 1;
    for (int t = 0; t < TX * TY; ++t)
        if (tile_start[t + 1] - tile_start[t] > maxlen) maxlen = tile_start[t + 1] - tile_start[t];
    or_blend_ctx c = {mean2d, conic, opac, depth, rgb, bg, maxw, g_certain, g_uncertain,
                      (double *)malloc(sizeof(double) * (size_t)maxlen),
                      (double *)malloc(sizeof(double) * (size_t)maxlen)};
    int64_t evaluated = 0, hits = 0;
    const int nr = render_tiles ? n_render : TX * TY;
    for (int r = 0; r < nr; ++r) {
        int t = render_tiles ? render_tiles[r] : r;
        int tx = t % TX, ty = t / TX;
        const int32_t *list = items + tile_start[t];
        int64_t len = tile_start[t + 1] - tile_start[t];
        for (int y = ty * 16; y < ty * 16 + 16 && y < H; ++y)
            for (int x = tx * 16; x < tx * 16 + 16 && x < W; ++x) {
                or_pixel p;
                blend_pixel(&c, list, len, (float)x, (float)y, &p);
                size_t q = (size_t)y * W + x;
                for (int ch = 0; ch < 3; ++ch) out_rgb[(size_t)ch * W * H + q] = p.rgb[ch];
                if (out_D) out_D[q] = p.D;
                if (out_sigma) out_sigma[q] = p.sigma;
                if (out_alpha) out_alpha[q] = p.alpha;
                if (out_margin_pos) out_margin_pos[q] = p.margin_pos;
                if (out_ninc) out_ninc[q] = p.ninc;
                if (out_spread) out_spread[q] = p.spread;
                if (out_wrel) out_wrel[q] = p.wrel;
                evaluated += p.evaluated;
                hits += p.hits;
            }
    }
    free(c.wbuf);
    free(c.dbuf);
    if (out_hits) *out_hits = hits;
    return evaluated;
}

/* Brute force: every pixel blends ALL visible Gaussians in global
 * (depth bits, index) order whose rectangle contains the pixel's tile -- no
 * per-tile lists, no keys.  Must reproduce or_blend bit for bit. */
void or_blend_bruteforce(int32_t W, int32_t H, int32_t n, const int32_t *status, const int32_t *rect,
                         const float *mean2d, const float *conic, const float *opac,
                         const float *depth, const double *rgb, const float *bg,
                         int32_t every_gaussian, double *out_rgb, double *out_D, double *out_sigma,
                         double *out_alpha)
{
    /* every_gaussian != 0: each pixel blends every Gaussian that has a 2D
     * footprint (tile rectangle or not), so the tile rectangles themselves
     * are under test; otherwise each pixel takes the Gaussians whose
     * rectangle contains its tile, in depth order. */
    or_item *order = (or_item *)malloc(sizeof(or_item) * (size_t)(n > 0 ? n : 1));
    int m = 0;
    for (int i = 0; i < n; ++i)
        if (status[i] == OR_VISIBLE || (every_gaussian && status[i] == OR_NO_TILES)) {
            order[m].dbits = f2u(depth[i]); order[m].idx = i; ++m;
        }
    qsort(order, (size_t)m, sizeof(or_item), item_cmp);
    int32_t *list = (int32_t *)malloc(sizeof(int32_t) * (size_t)(m > 0 ? m : 1));
    or_blend_ctx c = {mean2d, conic, opac, depth, rgb, bg, NULL, NULL, NULL,
                      (double *)malloc(sizeof(double) * (size_t)(m > 0 ? m : 1)),
                      (double *)malloc(sizeof(double) * (size_t)(m > 0 ? m : 1))};
    for (int y = 0; y < H; ++y)
        for (int x = 0; x < W; ++x) {
            int tx = x / 16, ty = y / 16, len = 0;
            for (int k = 0; k < m; ++k) {
                const int32_t *r = &rect[4 * order[k].idx];
                if (every_gaussian || (tx >= r[0] && tx <= r[2] && ty >= r[1] && ty <= r[3]))
                    list[len++] = order[k].idx;
            }
            or_pixel p;
            blend_pixel(&c, list, len, (float)x, (float)y, &p);
            size_t q = (size_t)y * W + x;
            for (int ch = 0; ch < 3; ++ch) out_rgb[(size_t)ch * W * H + q] = p.rgb[ch];
            out_D[q] = p.D;
            out_sigma[q] = p.sigma;
            out_alpha[q] = p.alpha;
        }
    free(c.wbuf); free(c.dbuf); free(list); free(order);
}

/* Adaptive frustum (Sec. III-D): component-wise min / max of the NDC of the
 * projected means of the temporal Gaussian buffer.  Returns its size. */
int32_t or_afc_bounds(int32_t n, const uint8_t *g_rendered, const float *ndc, float *fbox)
{
    int32_t cnt = 0;
    fbox[0] = fbox[1] = INFINITY;
    fbox[2] = fbox[3] = -INFINITY;
    for (int i = 0; i < n; ++i) {
        if (!g_rendered[i]) continue;
        ++cnt;
        fbox[0] = fminf(fbox[0], ndc[2 * i]);
        fbox[1] = fminf(fbox[1], ndc[2 * i + 1]);
        fbox[2] = fmaxf(fbox[2], ndc[2 * i]);
        fbox[3] = fmaxf(fbox[3], ndc[2 * i + 1]);
    }
    return cnt;
}

/* ------------------------------------------------------------------------ */
/* Temporal geometry buffer warping (Eq. 3), depth fill and correspondence   */
/* query (Sec. III-E), stitching (Eq. 4).                                    */
/* ------------------------------------------------------------------------ */

/* Forward warp of the reference TGB into the current view: nearest pixel,
 * minimum depth and maximum std at each destination; defaults NOHIT / 0. */
void or_forward_warp(int32_t W, int32_t H, const float *D, const float *S,
                     const float *kref /*fx,fy,cx,cy*/, const float *kcur, const float *M,
                     float z_near, float *dmin, float *smax)
{
    for (size_t q = 0; q < (size_t)W * H; ++q) { dmin[q] = OR_NOHIT; smax[q] = 0.0f; }
    for (int y = 0; y < H; ++y)
        for (int x = 0; x < W; ++x) {
            size_t q = (size_t)y * W + x;
            float d = D[q];
            if (d == OR_NOHIT) continue;
            float rx = ((float)x - kref[2]) / kref[0];
            float ry = ((float)y - kref[3]) / kref[1];
            float Px = d * rx, Py = d * ry, Pz = d;
            float X = ((M[0] * Px + M[1] * Py) + M[2] * Pz) + M[3];
            float Y = ((M[4] * Px + M[5] * Py) + M[6] * Pz) + M[7];
            float Z = ((M[8] * Px + M[9] * Py) + M[10] * Pz) + M[11];
            if (!(Z > z_near)) continue;
            float u = kcur[0] * (X / Z) + kcur[2];
            float v = kcur[1] * (Y / Z) + kcur[3];
            float xf = floorf(u + 0.5f), yf = floorf(v + 0.5f);
            if (!(xf >= 0.0f && xf <= (float)(W - 1) && yf >= 0.0f && yf <= (float)(H - 1))) continue;
            size_t p = (size_t)yf * W + (size_t)xf;
            if (Z < dmin[p]) dmin[p] = Z;
            if (S[q] > smax[p]) smax[p] = S[q];
        }
}

/* Depth fill: a no-hit pixel whose eight neighbours are all valid takes
 * their average; border pixels are never filled.  One pass over dmin. */
void or_depth_fill(int32_t W, int32_t H, const float *dmin, float *dfill)
{
    for (int y = 0; y < H; ++y)
        for (int x = 0; x < W; ++x) {
            size_t q = (size_t)y * W + x;
            float d = dmin[q];
            if (d != OR_NOHIT) { dfill[q] = d; continue; }
            dfill[q] = OR_NOHIT;
            if (x < 1 || y < 1 || x > W - 2 || y > H - 2) continue;
            float nb[8];
            int k = 0, ok = 1;
            for (int dy = -1; dy <= 1; ++dy)
                for (int dx = -1; dx <= 1; ++dx) {
                    if (!dx && !dy) continue;
                    nb[k] = dmin[(size_t)(y + dy) * W + (x + dx)];
                    if (nb[k] == OR_NOHIT) ok = 0;
                    ++k;
                }
            if (!ok) continue;
            float s = nb[0];
            for (k = 1; k < 8; ++k) s = s + nb[k];
            dfill[q] = s / 8.0f;
        }
}

/* Backward correspondence query: unproject the repaired depth in the current
 * view, move it to the reference view, project; a pixel is matched when the
 * point is in front of the near plane and lands inside [0,W-1]x[0,H-1].
 * A tile (tile_px x tile_px pixels of this grid: 16 at full resolution, 8 on
 * the half-resolution TGB grid) is unmatched when any of its in-grid pixels
 * is unmatched. */
void or_backward_query(int32_t W, int32_t H, int32_t tile_px, const float *dfill, const float *kcur,
                       const float *kref, const float *Minv, float z_near, float *uv,
                       uint8_t *matched, uint8_t *tile_um)
{
    const int TX = (W + tile_px - 1) / tile_px, TY = (H + tile_px - 1) / tile_px;
    memset(tile_um, 0, (size_t)TX * TY);
    for (int y = 0; y < H; ++y)
        for (int x = 0; x < W; ++x) {
            size_t q = (size_t)y * W + x;
            int ok = 0;
            float u = -1.0f, v = -1.0f;
            float d = dfill[q];
            if (d != OR_NOHIT) {
                float rx = ((float)x - kcur[2]) / kcur[0];
                float ry = ((float)y - kcur[3]) / kcur[1];
                float Px = d * rx, Py = d * ry, Pz = d;
                float X = ((Minv[0] * Px + Minv[1] * Py) + Minv[2] * Pz) + Minv[3];
                float Y = ((Minv[4] * Px + Minv[5] * Py) + Minv[6] * Pz) + Minv[7];
                float Z = ((Minv[8] * Px + Minv[9] * Py) + Minv[10] * Pz) + Minv[11];
                if (Z > z_near) {
                    u = kref[0] * (X / Z) + kref[2];
                    v = kref[1] * (Y / Z) + kref[3];
                    ok = u >= 0.0f && u <= (float)(W - 1) && v >= 0.0f && v <= (float)(H - 1);
                }
            }
            matched[q] = (uint8_t)ok;
            uv[2 * q] = ok ? u : -1.0f;
            uv[2 * q + 1] = ok ? v : -1.0f;
            if (!ok) tile_um[(y / tile_px) * TX + (x / tile_px)] = 1;
        }
}

/* Occluded tiles: for every newly visible Gaussian, each tile of its
 * rectangle whose largest opacity over the tile's pixel centres reaches
 * 1/255.  oc_margin marks tiles where that maximum lies within the margin. */
void or_occluded_tiles(int32_t W, int32_t H, int32_t n, const uint8_t *newly_visible,
                       const int32_t *status, const int32_t *rect, const float *mean2d,
                       const float *conic, const float *opac, uint8_t *oc, uint8_t *oc_margin)
{
    const int TX = (W + 15) / 16, TY = (H + 15) / 16;
    memset(oc, 0, (size_t)TX * TY);
    memset(oc_margin, 0, (size_t)TX * TY);
    for (int i = 0; i < n; ++i) {
        if (!newly_visible[i] || status[i] != OR_VISIBLE) continue;
        float A = conic[3 * i], B = conic[3 * i + 1], Cc = conic[3 * i + 2];
        for (int ty = rect[4 * i + 1]; ty <= rect[4 * i + 3]; ++ty)
            for (int tx = rect[4 * i + 0]; tx <= rect[4 * i + 2]; ++tx) {
                float amax = 0.0f;
                int pmargin = 0;
                for (int y = ty * 16; y < ty * 16 + 16 && y < H; ++y)
                    for (int x = tx * 16; x < tx * 16 + 16 && x < W; ++x) {
                        float dx = mean2d[2 * i] - (float)x, dy = mean2d[2 * i + 1] - (float)y;
                        float power = -0.5f * (A * dx * dx + Cc * dy * dy) - B * dx * dy;
                        if (fabs((double)power) <= OR_MARGIN_POWER) pmargin = 1;
                        if (power > 0.0f) continue;
                        float alpha = fminf(OR_ALPHA_MAX, opac[i] * expf(power));
                        if (alpha > amax) amax = alpha;
                    }
                int t = ty * TX + tx;
                if (!(amax < OR_ALPHA_MIN)) oc[t] = 1;
                if (pmargin || fabs((double)amax - (double)OR_ALPHA_MIN) <= OR_MARGIN_ALPHA) oc_margin[t] = 1;
            }
    }
}

/* Eq. 4 for the tiles that are not re-rendered: bilinear sample of the
 * reference image (TAB, planar [3][H][W]) at the correspondence (u,v). */
void or_stitch(int32_t W, int32_t H, const float *tab, const float *uv, const uint8_t *tile_sel,
               double *out_rgb)
{
    const int TX = (W + 15) / 16;
    for (int y = 0; y < H; ++y)
        for (int x = 0; x < W; ++x) {
            if (tile_sel[(y / 16) * TX + (x / 16)]) continue;
            size_t q = (size_t)y * W + x;
            float u = uv[2 * q], v = uv[2 * q + 1];
            if (!(u >= 0.0f && v >= 0.0f)) {   /* unmatched: cannot occur outside selected tiles */
                for (int ch = 0; ch < 3; ++ch) out_rgb[(size_t)ch * W * H + q] = 0.0;
                continue;
            }
            int x0 = (int)floorf(u), y0 = (int)floorf(v);
            int x1 = x0 + 1 < W ? x0 + 1 : W - 1;
            int y1 = y0 + 1 < H ? y0 + 1 : H - 1;
            double ax = (double)(u - (float)x0), ay = (double)(v - (float)y0);
            for (int ch = 0; ch < 3; ++ch) {
                const float *I = tab + (size_t)ch * W * H;
                double i00 = I[(size_t)y0 * W + x0], i10 = I[(size_t)y0 * W + x1];
                double i01 = I[(size_t)y1 * W + x0], i11 = I[(size_t)y1 * W + x1];
                out_rgb[(size_t)ch * W * H + q] =
                    (1.0 - ay) * ((1.0 - ax) * i00 + ax * i10) + ay * ((1.0 - ax) * i01 + ax * i11);
            }
        }
}

/* ------------------------------------------------------------------------ */
/* Temporal geometry buffer downscaled by 2 (Sec. IV-B, large scenes).       */
/* ------------------------------------------------------------------------ */

/* Eq. 1 and Eq. 2 over each 2x2 block of pixels taken as one pixel: the
 * block's composited weights are the union of its pixels', so with
 * A_p = sum of w over pixel p (= its alpha), D_p and sigma_p its Eq. 1/2,
 *   D_h = sum_p A_p D_p / sum_p A_p,
 *   sigma_h^2 = sum_p A_p (sigma_p^2 + (D_p - D_h)^2) / sum_p A_p
 * (pooled mean and variance).  A block with no composited weight gets
 * (empty_depth, 0).  Grid: ceil(W/2) x ceil(H/2); pixels outside the image
 * count as empty. */
void or_tgb_pool(int32_t W, int32_t H, const double *D, const double *S, const double *A,
                 float empty_depth, float *Dh, float *Sh)
{
    const int Wh = (W + 1) / 2, Hh = (H + 1) / 2;
    for (int j = 0; j < Hh; ++j)
        for (int i = 0; i < Wh; ++i) {
            double sa = 0.0, sad = 0.0;
            for (int dy = 0; dy < 2; ++dy)
                for (int dx = 0; dx < 2; ++dx) {
                    int x = 2 * i + dx, y = 2 * j + dy;
                    if (x >= W || y >= H) continue;
                    size_t q = (size_t)y * W + x;
                    if (A[q] > 0.0) { sa += A[q]; sad += A[q] * D[q]; }
                }
            size_t h = (size_t)j * Wh + i;
            if (!(sa > 0.0)) { Dh[h] = empty_depth; Sh[h] = 0.0f; continue; }
            double d = sad / sa, sv = 0.0;
            for (int dy = 0; dy < 2; ++dy)
                for (int dx = 0; dx < 2; ++dx) {
                    int x = 2 * i + dx, y = 2 * j + dy;
                    if (x >= W || y >= H) continue;
                    size_t q = (size_t)y * W + x;
                    if (A[q] > 0.0) sv += A[q] * (S[q] * S[q] + (D[q] - d) * (D[q] - d));
                }
            Dh[h] = (float)d;
            Sh[h] = (float)sqrt(sv / sa);
        }
}

/* Eq. 4 with a half-resolution TGB: each full-resolution pixel of a tile
 * that is not re-rendered is unprojected with the repaired depth of its 2x2
 * block (grid Wh x Hh), moved to the reference view and projected with the
 * full-resolution intrinsics; the reference image is sampled bilinearly at
 * that point, clamped to [0,W-1]x[0,H-1] (the block matched, the pixel may
 * land up to about a pixel outside). */
void or_stitch_depth(int32_t W, int32_t H, const float *tab, int32_t Wh, const float *dfill_h,
                     const float *kcur, const float *kref, const float *Minv, float z_near,
                     const uint8_t *tile_sel, double *out_rgb)
{
    const int TX = (W + 15) / 16;
    for (int y = 0; y < H; ++y)
        for (int x = 0; x < W; ++x) {
            if (tile_sel[(y / 16) * TX + (x / 16)]) continue;
            size_t q = (size_t)y * W + x;
            float d = dfill_h[(size_t)(y >> 1) * Wh + (x >> 1)];
            float u = -1.0f, v = -1.0f;
            int ok = 0;
            if (d != OR_NOHIT) {
                float rx = ((float)x - kcur[2]) / kcur[0];
                float ry = ((float)y - kcur[3]) / kcur[1];
                float Px = d * rx, Py = d * ry, Pz = d;
                float X = ((Minv[0] * Px + Minv[1] * Py) + Minv[2] * Pz) + Minv[3];
                float Y = ((Minv[4] * Px + Minv[5] * Py) + Minv[6] * Pz) + Minv[7];
                float Z = ((Minv[8] * Px + Minv[9] * Py) + Minv[10] * Pz) + Minv[11];
                if (Z > z_near) {
                    u = kref[0] * (X / Z) + kref[2];
                    v = kref[1] * (Y / Z) + kref[3];
                    u = fminf(fmaxf(u, 0.0f), (float)(W - 1));
                    v = fminf(fmaxf(v, 0.0f), (float)(H - 1));
                    ok = 1;
                }
            }
            if (!ok) {   /* cannot occur outside selected tiles */
                for (int ch = 0; ch < 3; ++ch) out_rgb[(size_t)ch * W * H + q] = 0.0;
                continue;
            }
            int x0 = (int)floorf(u), y0 = (int)floorf(v);
            int x1 = x0 + 1 < W ? x0 + 1 : W - 1;
            int y1 = y0 + 1 < H ? y0 + 1 : H - 1;
            double ax = (double)(u - (float)x0), ay = (double)(v - (float)y0);
            for (int ch = 0; ch < 3; ++ch) {
                const float *I = tab + (size_t)ch * W * H;
                double i00 = I[(size_t)y0 * W + x0], i10 = I[(size_t)y0 * W + x1];
                double i01 = I[(size_t)y1 * W + x0], i11 = I[(size_t)y1 * W + x1];
                out_rgb[(size_t)ch * W * H + q] =
                    (1.0 - ay) * ((1.0 - ax) * i00 + ax * i10) + ay * ((1.0 - ax) * i01 + ax * i11);
            }
        }
}
