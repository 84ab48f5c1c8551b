// Per-tile front-to-back alpha blending (Sec. III-A) and, on reference
// frames, the temporal priors it produces: the per-pixel depth and depth
// standard deviation of Eq. 1/2 (temporal geometry buffer), a copy of the
// image (temporal appearance buffer) and the set of Gaussians with a
// positive blending weight somewhere (temporal Gaussian buffer, Sec. III-C).
//
// One 256-thread block (four wave64s, one per 8x8 quadrant, each as four
// 16-lane groups on 4x4 sub-blocks) per 16x16 tile, one pixel per thread.
// The tile's sorted Gaussians are staged through LDS in batches of 255
// records (48 bytes each, one coalesced gather per thread; the 256th slot is
// a sentinel that pads the lists); every wave then reads each record as an
// LDS broadcast.  A pixel stops at the Gaussian that
// would take its transmittance below 1e-4; the block leaves as soon as all
// 256 pixels have stopped.  The work is VALU-bound (one exp and ~25 lane-ops
// per pixel-Gaussian pair).
//
// Eq. 1/2 are accumulated in one pass around a pivot (the first composited
// depth): D = d0 + S1/W, sigma^2 = S2/W - (S1/W)^2, which avoids the
// cancellation of the unshifted form at large depths.  Gaussians that a wave
// composites are flagged through a wave ballot, so the temporal Gaussian
// buffer costs one scalar test per record and wave.
//
// The tiles with the longest lists (the first of the blend order, counted
// by the order kernel) are blended by four blocks each, one per 8x8
// quadrant, four lanes per pixel on four consecutive list entries: on large
// scenes a few tiles with tens of batches would otherwise set the launch's
// tail.  In a TemporalGS frame the blocks past the selected tiles stitch the
// other tiles from the reference image (stitch.h) while the long tiles
// finish.
#include <hip/hip_ext.h>

#include "stitch.h"
#include "tgs_internal.h"

namespace tgs {

namespace {

constexpr int kBatch = 255;   // Gaussians staged per batch (slot 255: the sentinel)

// Wave votes on the execution mask itself (no 0/1 vector temporaries).
__device__ inline bool wave_any(bool p) { return __builtin_amdgcn_ballot_w64(p) != 0ull; }
__device__ inline bool wave_all(bool p) { return __builtin_amdgcn_ballot_w64(!p) == 0ull; }

// Broadcast of lane K of each group of four lanes (DPP quad_perm).
template <int K>
__device__ inline float quad_bcast(float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v),
                                                              K | (K << 2) | (K << 4) | (K << 6),
                                                              0xf, 0xf, false));
}
template <int K>
__device__ inline uint32_t quad_bcast_u(uint32_t v) {
    return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, K | (K << 2) | (K << 4) | (K << 6), 0xf,
                                              0xf, false);
}
// Inclusive prefix sum over the wave's lanes, in lane order, of four byte
// fields at once (no field's total may exceed 255): within rows of 16 lanes
// by shifts of 1, 2, 4 and 8, then the rows' totals by the row broadcasts of
// lanes 15 and 31.
__device__ inline uint32_t wave_incl_sum_bytes(uint32_t x) {
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x111, 0xf, 0xf, false);   // row_shr:1
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x112, 0xf, 0xf, false);   // row_shr:2
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x114, 0xf, 0xf, false);   // row_shr:4
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x118, 0xf, 0xf, false);   // row_shr:8
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x142, 0xa, 0xf, false);   // row_bcast:15
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x143, 0xc, 0xf, false);   // row_bcast:31
    return x;
}

// Sum over each group of four lanes (quad_perm [1,0,3,2], then [2,3,0,1]).
__device__ inline float quad_sum(float v) {
    v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0xb1,
                                                            0xf, 0xf, false));
    v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x4e,
                                                            0xf, 0xf, false));
    return v;
}

// LDS of one blend block.  Staged per Gaussian: (u, v, qa, qb) and (qc,
// opacity, depth, f), f set once a pixel composites the Gaussian (the
// temporal Gaussian buffer, written at the slot's own address), where q* = conic coefficients pre-scaled by -log2(e)
// (and 1/2 on the squares, by the preprocess) so that log2 of the Gaussian
// falloff is a three-FMA quadratic form and the opacity is one v_exp_f32.
// The tile is cut into sixteen 4x4 sub-blocks; sub-block list L (quadrant
// L >> 2, sub-block L & 3 within it: column 2 (L >> 2 & 1) + (L & 1), row
// 2 (L >> 3) + (L >> 1 & 1)) holds the staging slots of the Gaussians whose
// alpha >= 1/255 ellipse, conservatively enlarged, meets the sub-block, in
// staging (= depth) order: a footprint a few pixels wide meets a 4x4 block
// about 60 % as often as the 8x8 quadrant.
struct BlendLds {
    float4 g0[256];
    float4 g1[256];
    float4 col[256];
    int idx[256];
    __align__(16) uint8_t list[16][256];
    __align__(16) uint16_t mask[256];   // sub-blocks each staged Gaussian meets
};

// One 16x16 tile, or (QUAD) one 8x8 quadrant q of it.
//  - tile: each wave covers an 8x8 quadrant as four 16-lane groups, one per
//    sub-block, and every iteration advances the four lists at once (the
//    wave's trip count is its longest list);
//  - quadrant (the longest lists of the frame, whose tiles would set the
//    launch's tail): each wave covers one sub-block, four lanes per pixel
//    taking four consecutive entries of its list per iteration, composited
//    in list order through the quad's transmittance products.  The four
//    blocks of a tile each stage the whole list.
template <bool CAPTURE, bool CONTRIB, bool COUNT, bool QUAD>
__device__ __attribute__((always_inline)) inline void blend_block(const BlendArgs &a, BlendLds &s,
                                                                  int tile, int q) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int tx = tile % a.TX, ty = tile / a.TX;
    if (tid == 0 && (!QUAD || q == 0)) {
        if (a.mark_sel) a.mark_sel[tile] = 1u;
        if (a.mark_mask) a.mark_mask[tile] = 1u;
    }
    // lane -> pixel.  Tile: wave = 8x8 quadrant, lane >> 4 = 4x4 sub-block
    // within it.  Quadrant: wave = sub-block, lane >> 2 = pixel of it,
    // lane & 3 = entry of the group of four.
    const int k = lane & 3;
    int px, py, my_list;
    if (QUAD) {
        const int pix = lane >> 2;
        px = tx * kTile + 8 * (q & 1) + 4 * (wave & 1) + (pix & 3);
        py = ty * kTile + 8 * (q >> 1) + 4 * (wave >> 1) + (pix >> 2);
        my_list = 4 * q + wave;
    } else {
        const int grp = lane >> 4;
        px = tx * kTile + 8 * (wave & 1) + 4 * (grp & 1) + (lane & 3);
        py = ty * kTile + 8 * (wave >> 1) + 4 * (grp >> 1) + ((lane >> 2) & 3);
        my_list = 4 * wave + grp;
    }
    const bool inside = px < a.W && py < a.H;
    float fpx = (float)px, fpy = (float)py;
    // kept in registers through the loops (cheaper than converting them
    // again in every iteration, which the register allocator would prefer)
    __asm__ volatile("" : "+v"(fpx), "+v"(fpy));
    const float tile_x0 = (float)(tx * kTile), tile_y0 = (float)(ty * kTile);
    const uint2 range = a.ranges[tile];

    float T = 1.0f, cr = 0.0f, cg = 0.0f, cb = 0.0f;
    float sw = 0.0f, s1 = 0.0f, s2 = 0.0f, d0 = 0.0f;
    bool pivot = false;
    // stopped lanes as a wave mask on scalar registers (lanes outside the
    // image start stopped): tested and updated without vector instructions
    uint64_t done = __builtin_amdgcn_ballot_w64(!inside);
    uint32_t stop_pos = range.y;   // list position of the stopping Gaussian (+1 below)
    uint32_t n_hit = 0;            // pairs with alpha >= 1/255 before the pixel stopped

    // Batches of 255 Gaussians in slots 0..254; slot 255 holds a sentinel
    // (opacity 0, conic 0: alpha 0 at every pixel) that pads every list, so
    // entries past a list's end need no test of their own.
    // this thread's entry index of the next batch, loaded while the current
    // batch is blended: a batch then waits for one dependent global load
    // (its records) instead of two, which sets the pace of the tiles with
    // thousands of batches
    int nidx = (tid < kBatch && range.x + tid < range.y) ? (int)a.vals[range.x + tid] : 0;
    for (uint32_t b = range.x; b < range.y; b += kBatch) {
        if (__syncthreads_and(done == ~0ull)) break;
        reinterpret_cast<uint4 *>(&s.list[0][0])[tid] =
            make_uint4(0xffffffffu, 0xffffffffu, 0xffffffffu, 0xffffffffu);
        const uint32_t kb = b + tid;
        uint32_t lists = 0;   // bit L: the staged Gaussian meets sub-block L
        if (tid == kBatch) {
            s.g0[tid] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
            s.g1[tid] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
            s.col[tid] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
            s.idx[tid] = 0;
        } else if (kb < range.y) {
            const int idx = nidx;
            const float4 *r = a.g + 4 * (size_t)idx;
            const float4 r0 = r[0], r1 = r[1], r2 = r[2], r3 = r[3];
            s.idx[tid] = idx;
            s.g0[tid] = make_float4(r0.x, r0.y, r3.x, r3.y);
            s.g1[tid] = make_float4(r3.z, r1.y, r1.z, 0.0f);
            s.col[tid] = r2;
            const float hx = r2.w, hy = r1.w;
            if (hx >= 0.0f) {
                // sub-blocks the culling box meets: list L covers column
                // cx = 2 (w & 1) + (g & 1), row cy = 2 (w >> 1) + (g >> 1)
                // (w = L >> 2, g = L & 3); kColL[c] / kRowL[c] are the lists
                // of column / row c
                constexpr uint32_t kColL[4] = {0x0505u, 0x0a0au, 0x5050u, 0xa0a0u};
                constexpr uint32_t kRowL[4] = {0x0033u, 0x00ccu, 0x3300u, 0xcc00u};
                uint32_t box = 0u, rows = 0u;
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    const float x0 = tile_x0 + 4.0f * c, y0 = tile_y0 + 4.0f * c;
                    box |= (r0.x + hx >= x0 && r0.x - hx <= x0 + 3.0f) ? kColL[c] : 0u;
                    rows |= (r0.y + hy >= y0 && r0.y - hy <= y0 + 3.0f) ? kRowL[c] : 0u;
                }
                box &= rows;
                // and whose centre lies within sqrt(k) + m of the mean in the
                // metric of the conic (q(d) = a dx^2 + 2 b dx dy + c dy^2;
                // k = 2 ln(255 o), from the record; m = the largest q-length
                // from a sub-block's centre to its corner pixel centres, at
                // offset (1.5, +-1.5)): by the triangle inequality of that
                // norm no pixel centre of a sub-block farther out has
                // q <= k, i.e. alpha >= 1/255.  Enlarged by 0.2 % + 0.01,
                // which also covers the hardware square root (1 ulp) and the
                // rounding of q.  The terms of q are taken per column and per
                // row, then one FMA and one add per sub-block, without branches.
                const float ca = r0.z, cbq = r0.w, cc = r1.x;
                const float m = __builtin_amdgcn_sqrtf(2.25f * (ca + cc + 2.0f * fabsf(cbq)));
                const float rr = (__builtin_amdgcn_sqrtf(r3.w) + m) * 1.002f + 0.01f;
                const float R = rr * rr;
                float ax[4], bx[4], dyr[4], cy2[4];
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    const float dx = tile_x0 + (4.0f * c + 1.5f) - r0.x;
                    const float dy = tile_y0 + (4.0f * c + 1.5f) - r0.y;
                    ax[c] = ca * dx * dx;
                    bx[c] = 2.0f * cbq * dx;
                    dyr[c] = dy;
                    cy2[c] = cc * dy * dy;
                }
#pragma unroll
                for (int L = 0; L < 16; ++L) {
                    const int w = L >> 2, g = L & 3;
                    const int cx = 2 * (w & 1) + (g & 1), cy = 2 * (w >> 1) + (g >> 1);
                    const float qf = __builtin_fmaf(bx[cx], dyr[cy], ax[cx] + cy2[cy]);
                    lists |= !(qf > R) ? (1u << L) : 0u;
                }
                lists &= box;
                // a quadrant block lists its own four sub-blocks only
                if (QUAD) lists &= 0xfu << (4 * q);
            }
        }
        // Order-preserving compaction: every staged Gaussian's sub-block
        // bits go to LDS, then each wave builds the lists it walks (tile:
        // its four sub-blocks; quadrant: its one) from all the staged
        // Gaussians.  Lane l takes slots 4l .. 4l + 3; its entries' offsets
        // are one wave-wide prefix sum of its per-list counts, four lists
        // packed one byte each (a list holds at most 255 entries).
        s.mask[tid] = (uint16_t)lists;
        __syncthreads();
        constexpr int kNL = QUAD ? 1 : 4;
        const int L0 = QUAD ? my_list : 4 * wave;
        const uint2 m4 = reinterpret_cast<const uint2 *>(s.mask)[lane];
        uint32_t own[kNL], packed = 0;
#pragma unroll
        for (int gl = 0; gl < kNL; ++gl) {
            const uint32_t L = (uint32_t)(L0 + gl);
            // bit k: slot 4 lane + k meets sub-block L
            own[gl] = __builtin_amdgcn_ubfe(m4.x, L, 1) | __builtin_amdgcn_ubfe(m4.x, 16 + L, 1) << 1 |
                      __builtin_amdgcn_ubfe(m4.y, L, 1) << 2 | __builtin_amdgcn_ubfe(m4.y, 16 + L, 1) << 3;
            packed |= (uint32_t)__popc(own[gl]) << (8 * gl);
        }
        const uint32_t incl = wave_incl_sum_bytes(packed);
        const uint32_t excl = incl - packed;
        const uint32_t tot = __builtin_amdgcn_readlane(incl, 63);
        uint32_t n_long = 0;
#pragma unroll
        for (int gl = 0; gl < kNL; ++gl) {
            uint8_t *dst = &s.list[L0 + gl][0];
            uint32_t o = (excl >> (8 * gl)) & 255u;
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                if ((own[gl] >> k) & 1u) dst[o] = (uint8_t)(4 * lane + k);
                o += (own[gl] >> k) & 1u;
            }
            n_long = max(n_long, (tot >> (8 * gl)) & 255u);
        }
        // the wave's trip count, the same for every lane (on scalar
        // registers): its longest list (tile; shorter lists are padded), or
        // its list's length rounded up to whole groups of four (quadrant).
        // The wave reads only the lists it wrote: no barrier before the walk.
        if (QUAD) n_long = (n_long + 3u) & ~3u;
        {
            const uint32_t kn = b + kBatch + tid;
            nidx = (tid < kBatch && kn < range.y) ? (int)a.vals[kn] : 0;
        }
        // a wave whose pixels have all stopped skips the batch
        const uint32_t n_run = done == ~0ull ? 0u : n_long;
        if (QUAD) {
            for (uint32_t e = 0; e < n_run; e += 4) {
                // the group's four slots in one aligned 32-bit LDS load
                const uint32_t j = (*reinterpret_cast<const uint32_t *>(&s.list[my_list][e]) >> (8 * k)) & 255u;
                const uint32_t jo = j << 4;   // byte offset into the staged arrays
                const float4 g0 = *reinterpret_cast<const float4 *>(reinterpret_cast<const char *>(s.g0) + jo);
                const float4 g1 = *reinterpret_cast<const float4 *>(reinterpret_cast<const char *>(s.g1) + jo);
                const float dx = g0.x - fpx, dy = g0.y - fpy;
                const float p2 = __builtin_fmaf(dx, __builtin_fmaf(g0.z, dx, g0.w * dy), g1.x * dy * dy);
                const float alpha = fminf(kAlphaMax, g1.y * __builtin_amdgcn_exp2f(p2));
                // a running pixel's entry with power <= 0 and alpha >= 1/255
                const uint64_t hitm = __builtin_amdgcn_ballot_w64(!(p2 > 0.0f)) &
                                      __builtin_amdgcn_ballot_w64(alpha >= kAlphaMin) & ~done;
                const bool hit = __builtin_amdgcn_inverse_ballot_w64(hitm);
                // transmittance through the four entries in list order, one
                // product at a time (the fp32 products of a sequential walk;
                // an entry that is no hit multiplies by exactly 1)
                const float f = hit ? 1.0f - alpha : 1.0f;
                const float t1 = T * quad_bcast<0>(f);
                const float t2 = t1 * quad_bcast<1>(f);
                const float t3 = t2 * quad_bcast<2>(f);
                const float t4 = t3 * quad_bcast<3>(f);
                // the pixel stops at the first entry whose product falls
                // below 1e-4 (a hit; that entry is not composited)
                const int ks = !(t1 >= kTMin) ? 0 : !(t2 >= kTMin) ? 1 : !(t3 >= kTMin) ? 2
                             : !(t4 >= kTMin) ? 3 : 4;
                const float Tin = k == 0 ? T : k == 1 ? t1 : k == 2 ? t2 : t3;
                const bool inc = hit && k < ks;
                const float w = inc ? alpha * Tin : 0.0f;
                const float4 c = *reinterpret_cast<const float4 *>(reinterpret_cast<const char *>(s.col) + jo);
                cr = __builtin_fmaf(w, c.x, cr);
                cg = __builtin_fmaf(w, c.y, cg);
                cb = __builtin_fmaf(w, c.z, cb);
                const bool stopping = ks < 4;
                T = ks == 0 ? T : ks == 1 ? t1 : ks == 2 ? t2 : ks == 3 ? t3 : t4;
                if (COUNT) {
                    n_hit += (hit && k <= ks) ? 1u : 0u;
                    if (stopping) {
                        const uint32_t jk = ks == 0 ? quad_bcast_u<0>(j) : ks == 1 ? quad_bcast_u<1>(j)
                                          : ks == 2 ? quad_bcast_u<2>(j) : quad_bcast_u<3>(j);
                        stop_pos = b + jk;
                    }
                }
                if (CAPTURE) {
                    const float dep = g1.z;
                    // the pivot: depth of the pixel's first composited entry
                    if (__builtin_amdgcn_ballot_w64(inc && !pivot)) {
                        const int km0 = inc ? k : 4;
                        int km = min(km0, (int)__builtin_amdgcn_mov_dpp(km0, 0xb1, 0xf, 0xf, false));
                        km = min(km, (int)__builtin_amdgcn_mov_dpp(km, 0x4e, 0xf, 0xf, false));
                        const float dk = km == 0 ? quad_bcast<0>(dep) : km == 1 ? quad_bcast<1>(dep)
                                       : km == 2 ? quad_bcast<2>(dep) : quad_bcast<3>(dep);
                        d0 = (!pivot && km < 4) ? dk : d0;
                        pivot = pivot || km < 4;
                    }
                    const float dd = dep - d0;
                    sw += w;
                    s1 = __builtin_fmaf(w, dd, s1);
                    s2 = __builtin_fmaf(w * dd, dd, s2);
                    if (inc) *reinterpret_cast<float *>(reinterpret_cast<char *>(s.g1) + jo + 12) = 1.0f;
                    if (CONTRIB) {
                        // max weight of this lane's entry over the wave's 16 pixels
                        float mw = w;
#pragma unroll
                        for (int o = 4; o <= 32; o <<= 1) mw = fmaxf(mw, __shfl_xor(mw, o));
                        if (lane < 4 && mw > 0.0f)
                            atomicMax(reinterpret_cast<unsigned int *>(a.contrib + s.idx[j]),
                                      __float_as_uint(mw));
                    }
                }
                done |= __builtin_amdgcn_ballot_w64(stopping);
                if (done == ~0ull) break;
            }
        } else {
            // list slots are read four at a time (one aligned 32-bit LDS load
            // per four entries, each slot's byte offset taken with constant
            // shifts): three entries in four wait for one LDS round trip (the
            // staged record) instead of two.  The walk runs to the wave's
            // longest list rounded up to four: the slots past every list's
            // end hold the sentinel (alpha 0)
            bool stopped = false;
            for (uint32_t e = 0; e < n_run && !stopped; e += 4) {
              const uint32_t quad = *reinterpret_cast<const uint32_t *>(&s.list[my_list][e]);
#pragma unroll
              for (int u = 0; u < 4; ++u) {
                // byte offset into the staged arrays (16-byte slots)
                const uint32_t jo = u == 0 ? (quad << 4) & 0xff0u : (quad >> (8 * u - 4)) & 0xff0u;
                const uint32_t j = jo >> 4;
                const float4 g0 = *reinterpret_cast<const float4 *>(reinterpret_cast<const char *>(s.g0) + jo);
                const float4 g1 = *reinterpret_cast<const float4 *>(reinterpret_cast<const char *>(s.g1) + jo);
                const float dx = g0.x - fpx, dy = g0.y - fpy;
                // log2 of exp(power) with power = -(A dx^2 + 2B dx dy + C dy^2)/2
                const float p2 = __builtin_fmaf(dx, __builtin_fmaf(g0.z, dx, g0.w * dy), g1.x * dy * dy);
                const float alpha = fminf(kAlphaMax, g1.y * __builtin_amdgcn_exp2f(p2));
                // composited or stopping: an entry of a running pixel with power
                // <= 0 and alpha >= 1/255.  The decisions are wave masks
                // (compares straight into scalar registers, combined there)
                const uint64_t hitm = __builtin_amdgcn_ballot_w64(!(p2 > 0.0f)) &
                                      __builtin_amdgcn_ballot_w64(alpha >= kAlphaMin) & ~done;
                const float Tn = T * (1.0f - alpha);
                // T stays above 1e-4 (Tn is never NaN)
                const uint64_t keepm = __builtin_amdgcn_ballot_w64(Tn >= kTMin);
                const bool hit = __builtin_amdgcn_inverse_ballot_w64(hitm);
                const bool inc = __builtin_amdgcn_inverse_ballot_w64(hitm & keepm);
                const bool stop = __builtin_amdgcn_inverse_ballot_w64(hitm & ~keepm);
                const float w = inc ? alpha * T : 0.0f;
                const float4 c = *reinterpret_cast<const float4 *>(reinterpret_cast<const char *>(s.col) + jo);
                cr = __builtin_fmaf(w, c.x, cr);
                cg = __builtin_fmaf(w, c.y, cg);
                cb = __builtin_fmaf(w, c.z, cb);
                T = inc ? Tn : T;
                done |= hitm & ~keepm;
                if (COUNT) {
                    n_hit += hit ? 1u : 0u;
                    if (stop) stop_pos = b + j;
                }
                if (CAPTURE) {
                    const float dep = g1.z;
                    d0 = (inc && !pivot) ? dep : d0;
                    pivot = pivot || inc;
                    const float dd = dep - d0;
                    sw += w;
                    s1 = __builtin_fmaf(w, dd, s1);
                    s2 = __builtin_fmaf(w * dd, dd, s2);
                    // the pixel composites the Gaussian (w = alpha T > 0); the
                    // lanes of a group write the same flag, in the slot's
                    // staged record (no index to form)
                    if (inc) *reinterpret_cast<float *>(reinterpret_cast<char *>(s.g1) + jo + 12) = 1.0f;
                    if (CONTRIB) {
                        // max weight over the group's 16 lanes (one Gaussian)
                        float mw = w;
#pragma unroll
                        for (int o = 8; o >= 1; o >>= 1) mw = fmaxf(mw, __shfl_xor(mw, o));
                        if ((lane & 15) == 0 && mw > 0.0f)
                            atomicMax(reinterpret_cast<unsigned int *>(a.contrib + s.idx[j]),
                                      __float_as_uint(mw));
                    }
                }
                if (done == ~0ull) {
                    stopped = true;
                    break;
                }
              }
            }
        }
        __syncthreads();
        if (CAPTURE && a.g_flag && tid < kBatch && kb < range.y && s.g1[tid].w != 0.0f)
            a.g_flag[s.idx[tid]] = 1u;
    }

    if (QUAD) {
        // a pixel's sums over its four lanes
        cr = quad_sum(cr);
        cg = quad_sum(cg);
        cb = quad_sum(cb);
        if (CAPTURE) {
            sw = quad_sum(sw);
            s1 = quad_sum(s1);
            s2 = quad_sum(s2);
        }
    }
    if (COUNT) {
        // evaluated list entries: up to and including the stopping one (one
        // lane per pixel), and the hits (every lane its own entries)
        unsigned long long e = (inside && (!QUAD || k == 0))
            ? (unsigned long long)(stop_pos < range.y ? stop_pos + 1 : range.y) - range.x : 0ull;
        unsigned long long h = n_hit;
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) {
            e += __shfl_xor(e, o);
            h += __shfl_xor(h, o);
        }
        if (lane == 0 && e) atomicAdd(a.pairs, e);
        if (lane == 0 && h) atomicAdd(a.hits, h);
    }
    // Eq. 1 / Eq. 2 of the pixel
    float D = a.empty_depth, S = 0.0f;
    if (CAPTURE && sw > 0.0f) {
        const float m1 = s1 / sw;
        D = d0 + m1;
        S = sqrtf(fmaxf(0.0f, s2 / sw - m1 * m1));
    }
    if (CAPTURE && a.tgbh_depth) {
        // Eq. 1/2 over each 2x2 block of the tile taken as one pixel: its
        // composited weights are the union of its pixels', so with
        // A = 1 - T (the pixel's summed weight) the block has the pooled
        // D_h = sum A D / sum A and sigma_h^2 = sum A (sigma^2 + (D - D_h)^2)
        // / sum A.  The blocks lie inside the block's region (the tile or
        // the quadrant, PW pixels wide): pooled through LDS (the staging
        // arrays are free once every wave has left the batch loop).
        constexpr int PW = QUAD ? 8 : kTile, NB = PW / 2;
        const int ox = QUAD ? 8 * (q & 1) : 0, oy = QUAD ? 8 * (q >> 1) : 0;
        __syncthreads();
        float *s_pa = reinterpret_cast<float *>(s.g0);   // 3 x 256 floats
        float *s_pd = s_pa + 256, *s_ps = s_pa + 512;
        const int lp = (py - ty * kTile - oy) * PW + (px - tx * kTile - ox);
        s_pa[lp] = inside ? 1.0f - T : 0.0f;
        s_pd[lp] = D;
        s_ps[lp] = S;
        __syncthreads();
        const int Wg = (a.W + 1) >> 1, Hg = (a.H + 1) >> 1;
        const int gx = tx * (kTile / 2) + ox / 2 + tid % NB, gy = ty * (kTile / 2) + oy / 2 + tid / NB;
        if (tid < NB * NB && gx < Wg && gy < Hg) {
            const int l0 = 2 * (tid / NB) * PW + 2 * (tid % NB);
            const int ls[4] = {l0, l0 + 1, l0 + PW, l0 + PW + 1};
            float sa = 0.0f, sad = 0.0f;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float ak = s_pa[ls[i]];
                if (ak > 0.0f) {
                    sa += ak;
                    sad += ak * s_pd[ls[i]];
                }
            }
            float dh = a.empty_depth, sh = 0.0f;
            if (sa > 0.0f) {
                dh = sad / sa;
                float sv = 0.0f;
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const float ak = s_pa[ls[i]];
                    if (ak > 0.0f) {
                        const float sk = s_ps[ls[i]], ek = s_pd[ls[i]] - dh;
                        sv += ak * (sk * sk + ek * ek);
                    }
                }
                sh = sqrtf(sv / sa);
            }
            a.tgbh_depth[(size_t)gy * Wg + gx] = dh;
            a.tgbh_sigma[(size_t)gy * Wg + gx] = sh;
        }
    }
    // the background seen through the remaining transmittance
    cr = __builtin_fmaf(T, a.bg[0], cr);
    cg = __builtin_fmaf(T, a.bg[1], cg);
    cb = __builtin_fmaf(T, a.bg[2], cb);
    const size_t HW = (size_t)a.W * a.H;
    if (!QUAD) {
        // A wave holds an 8x8 quadrant, so its own stores would write the
        // 32-byte halves of the tile's 64-byte rows.  The outputs go through
        // LDS instead (the staging arrays are free once every wave has left
        // the batch loop) and each wave stores four whole rows of 16 pixels
        // per plane: every store instruction writes whole cache lines.
        constexpr int kPlanes = CAPTURE ? 6 : 3;
        float *sv = reinterpret_cast<float *>(s.g0);   // kPlanes x 256 floats
        __syncthreads();
        const int lp = (py - ty * kTile) * kTile + (px - tx * kTile);
        sv[lp] = cr;
        sv[256 + lp] = cg;
        sv[512 + lp] = cb;
        if (CAPTURE) {
            sv[768 + lp] = D;
            sv[1024 + lp] = S;
            sv[1280 + lp] = 1.0f - T;
        }
        __syncthreads();
        const int qx = tx * kTile + (tid & 15), qy = ty * kTile + (tid >> 4);
        if (qx >= a.W || qy >= a.H) return;
        const size_t o = (size_t)qy * a.W + qx;
        const float vr = sv[tid], vg = sv[256 + tid], vb = sv[512 + tid];
        a.rgb[o] = vr;
        a.rgb[HW + o] = vg;
        a.rgb[2 * HW + o] = vb;
        if (a.tab) {
            a.tab[o] = vr;
            a.tab[HW + o] = vg;
            a.tab[2 * HW + o] = vb;
        }
        if (CAPTURE && kPlanes == 6) {
            const float vd = sv[768 + tid], vs = sv[1024 + tid];
            if (a.depth) a.depth[o] = vd;
            if (a.sigma) a.sigma[o] = vs;
            if (a.alpha) a.alpha[o] = sv[1280 + tid];
            if (a.tgb_depth) a.tgb_depth[o] = vd;
            if (a.tgb_sigma) a.tgb_sigma[o] = vs;
        }
        return;
    }
    if (!inside || k != 0) return;
    const size_t o = (size_t)py * a.W + px;
    a.rgb[o] = cr;
    a.rgb[HW + o] = cg;
    a.rgb[2 * HW + o] = cb;
    if (a.tab) {
        a.tab[o] = cr;
        a.tab[HW + o] = cg;
        a.tab[2 * HW + o] = cb;
    }
    if (CAPTURE) {
        if (a.depth) a.depth[o] = D;
        if (a.sigma) a.sigma[o] = S;
        if (a.alpha) a.alpha[o] = 1.0f - T;
        if (a.tgb_depth) a.tgb_depth[o] = D;
        if (a.tgb_sigma) a.tgb_sigma[o] = S;
    }
}

// Eight waves per SIMD (64 VGPRs); the capture variants, which carry the
// Eq. 1/2 sums as well, at seven (72 VGPRs) so that nothing spills to
// scratch.
template <bool CAPTURE, bool CONTRIB, bool COUNT>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(CAPTURE ? 7 : 8))) void blend_kernel(BlendArgs a) {
    __shared__ BlendLds s;
    // block roles (block-uniform): with a split count ns, the first
    // nq = 4 ceil8(ns) blocks take the quadrants of the first ns tiles of the
    // blend order, the rest shift down by nq - ns; then the tiles, then (TGS
    // frames) the stitched tiles.  Blocks are dealt to the eight XCDs in
    // turn (block b on XCD b mod 8), so block b takes quadrant (b >> 3) & 3
    // of split tile 8 (b >> 5) + (b & 7): the four blocks of a tile, which
    // stage the same records, share one XCD's L2.
    int blk = (int)blockIdx.x;
    if (a.n_split_dev) {
        const int ns = (int)*a.n_split_dev;
        const int nq = 4 * ((ns + 7) & ~7);
        if (blk < nq) {
            const int t = 8 * (blk >> 5) + (blk & 7);
            if (t < ns) blend_block<CAPTURE, CONTRIB, COUNT, true>(a, s, a.tile_list[t], (blk >> 3) & 3);
            return;
        }
        blk -= nq - ns;
        if (blk >= a.n_grid) return;
    }
    if (a.n_tiles_dev && blk >= (int)*a.n_tiles_dev) {
        if (a.stitch_list) {
            const int t = a.stitch_list[blk];
            if (a.stitch_mode == 2)
                stitch_tile_depth(a.sw, a.stitch_wg, t, a.stitch_tab, a.stitch_dfill, a.rgb);
            else
                stitch_tile_uv(a.sw, t, a.stitch_tab, a.stitch_uv, a.rgb);
        }
        return;
    }
    blend_block<CAPTURE, CONTRIB, COUNT, false>(a, s, a.tile_list ? a.tile_list[blk] : blk, 0);
}

// Adaptive frustum (Sec. III-D): min / max NDC of the projected means of the
// temporal Gaussian buffer.  Two levels: a fixed grid of blocks reduces
// grid-strided slices into partials, one block reduces the partials (no
// contended atomics; min / max are exact, so the result is deterministic).
constexpr int kAfcBlocks = kAfcPartials;

__global__ __launch_bounds__(256) void afc_partial_kernel(int n, const uint8_t *g_flag,
                                                          const float4 *g, int W, int H,
                                                          int *partial) {
    __shared__ int s_red[4][4];
    int v[4] = {float_to_ordered(__builtin_inff()), float_to_ordered(__builtin_inff()),
                float_to_ordered(-__builtin_inff()), float_to_ordered(-__builtin_inff())};
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) {
        if (!g_flag[i]) continue;
        const float4 r = g[4 * (size_t)i];
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

void launch_blend(const BlendArgs &a0, int n_blocks, hipStream_t st, hipEvent_t start,
                  hipEvent_t stop) {
    if (n_blocks <= 0) return;
    BlendArgs a = a0;
    a.n_grid = n_blocks;
    // the quadrant blocks: 4 ceil8(n_split) <= 3 split_cap + 28 more than the tiles
    const int cap = a.split_cap < kMaxSplit ? (a.split_cap > 0 ? a.split_cap : 0) : kMaxSplit;
    if (a.n_split_dev && a.tile_list && cap > 0) n_blocks += 3 * cap + 28;
    else a.n_split_dev = nullptr;
    const bool capture = a.depth || a.sigma || a.alpha || a.tgb_depth || a.tgb_sigma ||
                         a.tgbh_depth || a.g_flag || a.contrib;
    if (a.contrib)
        launch_blend_v<true, true>(a, n_blocks, st, start, stop);
    else if (capture)
        launch_blend_v<true, false>(a, n_blocks, st, start, stop);
    else
        launch_blend_v<false, false>(a, n_blocks, st, start, stop);
}

void launch_afc_bounds(int n, const uint8_t *g_flag, const float4 *g, int W, int H, int *fbox,
                       hipStream_t st) {
    // fbox[0..3] is the result; fbox[4..] holds kAfcBlocks x 4 partials
    int *partial = fbox + 4;
    afc_partial_kernel<<<kAfcBlocks, 256, 0, st>>>(n, g_flag, g, W, H, partial);
    afc_final_kernel<<<1, 64, 0, st>>>(partial, kAfcBlocks, fbox);
}

}  // namespace tgs
