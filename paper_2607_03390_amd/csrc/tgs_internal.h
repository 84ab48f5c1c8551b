// Internal declarations shared by the HIP translation units of libtgs.
// Kernel argument structs and the host-side launchers each .hip file exports.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include "tgs.h"

namespace tgs {

constexpr float kNoHit = 1001.0f;           // z_far (1000) + epsilon (1)
constexpr float kZFar = 1000.0f;            // far plane
constexpr float kAlphaMin = 1.0f / 255.0f;
constexpr float kAlphaMax = 0.99f;
constexpr float kTMin = 1e-4f;
constexpr int kTile = 16;
// Key positions are 32-bit; the limit leaves headroom so that block bases
// (partition * tile, block * 1024) and loop strides never wrap.
constexpr uint32_t kMaxKeys = 0xffff0000u;

// Camera constants as the kernels consume them.
struct CamK {
    float V[12];              // rows 0..2 of world->camera
    float fx, fy, cx, cy;
    int W, H, TX, TY;
    float limx, limy;         // 1.3 * tan(half fov) guards of the Jacobian
    float campos[3];          // camera centre in world space
};

// Device scene.  Means and opacities are one float4 per Gaussian in their own
// array (every Gaussian's is read each frame, one coalesced 1 KB request per
// wave).  The rest is read only for Gaussians that survive the culls, often
// a scattered minority of a wave, so each Gaussian's bytes are contiguous:
// two geometry float4s (32 bytes) and sh_slots SH float4s (192 bytes, three
// whole 64-byte lines, at degree 3), and a culled Gaussian's lines are
// never fetched.
struct SceneDev {
    int n, deg, ncoef, sh_slots;
    const float4 *mean_op;    // x, y, z, opacity
    const float4 *geo;        // [2i] = (sx, sy, sz, qw), [2i + 1] = (qx, qy, qz, 0)
    const float4 *sh;         // [i * sh_slots + j]: coefficient-major (k*3 + channel) floats
};

// Per-Gaussian records written by the preprocess.
struct Records {
    // One 64-byte record per Gaussian (one aligned line per gather):
    // g[4i] = (u, v, conic a, conic b), g[4i + 1] = (conic c, opacity,
    // depth, hy), g[4i + 2] = (r, g, b, hx), g[4i + 3] = (qa, qb, qc, k):
    // the blend's constants, computed once per Gaussian instead of once per
    // (Gaussian, tile): q* = conic pre-scaled by -log2(e) (1/2 on the
    // squares), and hx, hy = half extents of the box of the alpha >= 1/255
    // ellipse enlarged by 0.2% + 0.05 px (negative: alpha < 1/255 everywhere);
    // g[4i + 3].w = k >= 2 ln(255 o), the ellipse's bound on the conic form.
    float4 *g;
    ushort4 *rect;            // tile rectangle x0, y0, x1, y1 (x0 > x1: empty)
    uint8_t *status;          // bit0 survivor, bit1 newly visible
    uint32_t *count;          // keys of the Gaussian (tiles of its rectangle)
    uint32_t *dkey;           // float bits of the depth (depth-sort key)
    uint32_t *partial;        // per 256-Gaussian block: survivors, newly visible
};

// Temporal dynamic culling inputs of the preprocess.
struct CullK {
    float z_near;
    int afc, toc;
    const int *fbox;          // ordered-int encoded F_min.x, F_min.y, F_max.x, F_max.y
    const float *dmin, *smax; // warped TGB
    const uint8_t *g_rendered;
    float lambda1, lambda2;
    int footprint;            // tile rectangle: 0 = 3-sigma square, 1 = alpha footprint box
    int tgb_shift;            // dmin/smax grid = image >> tgb_shift (0, or 1: 2x2 blocks)
    int tgb_w;                // width of that grid
    uint8_t *clear_flag;      // optional (reference frames): set to 0 for every Gaussian
                              // (the temporal Gaussian buffer the blend then fills)
};

// Frame counters on the device (read back once per frame).
struct Counters {
    uint32_t n_keys;
    uint32_t n_survivors;
    uint32_t n_newly;
    uint32_t n_selected;
    uint32_t n_visible;       // Gaussians with at least one key
    uint32_t n_sorted;        // keys emitted and sorted: n_keys, or 0 past the key capacity
    uint32_t n_split;         // tiles the blend splits into quadrants (the blend order's first)
    uint32_t pad;
};

// The frame's counters as the host reads them: written by the last counting
// kernel straight into coherent pinned host memory (16-byte aligned), tag
// last (after a system-scope fence), so the host waits for the tag instead of
// a copy.
struct HostCounters {
    uint32_t n_keys, n_survivors, n_newly, n_selected, n_visible, n_sorted;
    uint32_t pad;
    uint32_t tag;
};

// Writes the frame's counters to the host: the six values as two vector
// stores, a system-scope fence (they are complete and visible), then the tag
// as a relaxed store that nothing waits for.  (A volatile store would wait
// for its own round trip to host memory, one after another.)
__device__ inline void publish_host(HostCounters *h, uint32_t n_keys, uint32_t n_survivors,
                                    uint32_t n_newly, uint32_t n_selected, uint32_t n_visible,
                                    uint32_t n_sorted, uint32_t tag) {
    reinterpret_cast<uint4 *>(h)[0] = make_uint4(n_keys, n_survivors, n_newly, n_selected);
    reinterpret_cast<uint2 *>(h)[2] = make_uint2(n_visible, n_sorted);
    __threadfence_system();
    __hip_atomic_store(&h->tag, tag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
}

// Ordered-int encoding of a float: signed-int order equals float order, so
// integer atomic min/max give exact float min/max.
__device__ inline int float_to_ordered(float f) {
    int i = __float_as_int(f);
    return i >= 0 ? i : i ^ 0x7fffffff;
}
__device__ inline float ordered_to_float(int i) {
    return __int_as_float(i >= 0 ? i : i ^ 0x7fffffff);
}

// Key count of a Gaussian in a selective-rendering frame: the selected tiles
// of its rectangle, from per-row prefix sums of the tile mask (rowpre, TY
// rows of TX + 1 entries; one subtraction per row).
__device__ inline uint32_t masked_count(ushort4 r, const uint32_t *rowpre, int TX) {
    if (r.x > r.z || r.y > r.w) return 0u;
    uint32_t c = 0;
    int y = r.y;
    // four rows per step: all eight loads are in flight before the first use
    for (; y + 3 <= (int)r.w; y += 4) {
        const uint32_t *row = rowpre + (size_t)y * (TX + 1);
        const size_t s = (size_t)(TX + 1);
        const uint32_t a0 = row[r.z + 1], b0 = row[r.x];
        const uint32_t a1 = row[s + r.z + 1], b1 = row[s + r.x];
        const uint32_t a2 = row[2 * s + r.z + 1], b2 = row[2 * s + r.x];
        const uint32_t a3 = row[3 * s + r.z + 1], b3 = row[3 * s + r.x];
        c += (a0 - b0) + (a1 - b1) + (a2 - b2) + (a3 - b3);
    }
    for (; y <= (int)r.w; ++y) {
        const uint32_t *row = rowpre + (size_t)y * (TX + 1);
        c += row[r.z + 1] - row[r.x];
    }
    return c;
}

// ---- launchers (k_preprocess.hip) ----
// Writes the records and, per 256-Gaussian block, the survivor and
// newly-visible counts (summed into cnt by the last depth-sort pass).
// fill (optional): the depth fill / correspondence query of a TemporalGS
// frame (full-resolution geometry buffer) run by blocks of the same launch
// past the Gaussians' (independent work: both read only the forward warp).
// start / stop (may be NULL): events attached to the preprocess dispatch.
struct FillK;
void launch_preprocess(const SceneDev &s, const CamK &cam, const CullK &cull, Records rec,
                       Counters *cnt, const FillK *fill, hipStream_t st, hipEvent_t start = nullptr,
                       hipEvent_t stop = nullptr);
inline int preprocess_blocks(int n) { return (n + 255) / 256; }

// Keys are emitted in blocks of kKeyBlock consecutive positions; kfirst[B]
// (written by whichever kernel produces the key offsets) is the sorted
// position of the Gaussian that owns key B * kKeyBlock, for every block below
// the key capacity.
constexpr int kKeyBlock = 1024;
__host__ __device__ inline size_t key_blocks(size_t cap) { return (cap + kKeyBlock - 1) / kKeyBlock; }
// Records, for a sorted Gaussian at position s with keys [o, o + c), s as
// the owner of every key block that starts inside that range (below nb).
__device__ inline void mark_key_blocks(uint32_t *kfirst, uint32_t nb, uint32_t s, uint64_t o,
                                       uint32_t c) {
    for (uint64_t b = (o + kKeyBlock - 1) / kKeyBlock; b < nb && b * kKeyBlock < o + c; ++b)
        kfirst[b] = s;
}

// ---- launchers (k_keys.hip) ----
// Emits the cnt->n_sorted keys of the cnt->n_visible depth-ordered Gaussians
// (cap bounds n_sorted for the grid; nothing is emitted past the key
// capacity) and clears the tile ranges (filled by launch_ranges after the
// tile sort).  rowpre / sel_cols are NULL in frames that render every tile.
// rows (optional): per block of kKeyBlock keys, the counts of the tile
// sort's first digit (key bits [0, row_bits)) in row b of rows[b][256] (see
// launch_sort_u32).
void launch_duplicate(int n, uint32_t cap, const Counters *cnt, const uint32_t *didx,
                      const uint32_t *offs, const uint32_t *kfirst, const ushort4 *rect,
                      const uint32_t *rowpre, const int *sel_cols, int TX, int n_tiles,
                      uint32_t *tkey, uint32_t *tval, uint2 *ranges, uint32_t *rows,
                      int row_bits, hipStream_t st);
// Ranges of the cnt->n_sorted tile-sorted keys; cap bounds n_sorted for the grid.
void launch_ranges(uint32_t cap, const Counters *cnt, const uint32_t *keys, uint2 *ranges,
                   hipStream_t st);
// Tiles to rasterise (tile_in[0..m), or 0..m-1 when tile_in is NULL; m =
// *n_dev when n_dev is given, else n) in blend order, longest lists first,
// into tile_out[0..m).
// max_bucket (optional, host-visible memory) receives floor(log2 of the
// longest list length) + 1 (0: all lists empty).
struct OrderK {
    int n_host;
    const uint32_t *n_dev;
    const int *tile_in;
    const uint2 *ranges;
    int *tile_out;
    uint32_t *max_bucket;
    // optional: the number of tiles the blend splits, the first of the
    // order: those whose list length bucket is at least split_bucket, or, if
    // more than max_split (<= kMaxSplit) are, at least the lowest higher
    // bucket that leaves at most max_split (0: no split)
    uint32_t *n_split;
    int split_bucket;
    int max_split;
};
void launch_order_tiles(const OrderK &o, hipStream_t st);

// ---- launchers (k_sort.hip) ----
int sort_passes_for_bits(int bits);
// Scratch words of a sort of at most max_keys keys (either kind below).
size_t sort_scratch_words(uint32_t max_keys);
// Stable LSD sort of (key, value) pairs on key bits [begin_bit, begin_bit +
// bits), in ceil(bits / 8) passes of (nearly) equal width; every key must be
// below 2^(begin_bit + bits).  The key count is *n_dev if n_dev is not NULL
// (n_max bounds it), else n_max.  Returns 1 if the result is in the alt buffers.
// n_hint: the expected key count (e.g. a recent frame's); it picks the
// partition size (small partitions fill the chip for small sorts).
// counted: the first pass's digit counts of every kKeyBlock keys are
// already in sort_count_rows(scratch) (written by the key emission), so that
// pass has no counting launch; allowed only where sort_takes_rows says so.
int launch_sort_u32(const uint32_t *n_dev, uint32_t n_max, uint32_t n_hint, int begin_bit,
                    int bits, uint32_t *keys, uint32_t *vals, uint32_t *keys_alt,
                    uint32_t *vals_alt, uint32_t *scratch, bool counted, hipStream_t st);
// Whether launch_sort_u32 with these sizes can take counted rows, and the
// width of its first digit; where the rows go in its scratch.
bool sort_takes_rows(uint32_t n_max, uint32_t n_hint, int begin_bit, int bits);
int sort_first_digit_bits(int bits);
uint32_t *sort_count_rows(uint32_t *scratch);
// Depth order of the Gaussians with count[i] > 0 among i < n, stable by index
// (keys dkey[i], the depth's float bits): four passes (dkey -> a -> b -> a ->
// v_b; k_b may alias dkey).  With rowpre (a selective-rendering frame) the
// first pass first replaces count[i] by the masked count of rect[i].  Writes cnt->n_visible (Gaussians kept), the
// sorted indices to v_b[0..n_visible), offs[s] = exclusive prefix of their
// counts and the key-block owners kfirst[0 .. key_blocks(cap)), then
// cnt->n_keys, cnt->n_sorted (n_keys if <= cap, else 0),
// cnt->n_survivors / n_newly (from the preprocess partials) and, tag last,
// the same counters to `host`.
void launch_depth_sort(int n, uint32_t *count, const ushort4 *rect, const uint32_t *rowpre, int TX,
                       const uint32_t *dkey, uint32_t *k_a, uint32_t *v_a, uint32_t *k_b,
                       uint32_t *v_b, uint32_t *offs, uint32_t *kfirst, uint32_t *scratch,
                       Counters *cnt, uint32_t cap, const uint32_t *pre_partial, int n_pre,
                       HostCounters *host, uint32_t tag, hipStream_t st);

// ---- launchers (k_segsort.hip) ----
// Per-tile depth order without the global depth sort: key counts scanned in
// index order (part: 2 words per 1024-Gaussian block), the
// Gaussians with keys compacted in index order into vidx / voffs (the
// duplication's input), the frame's counters published as the depth sort
// does; after the tile sort, each tile's list sorted by (depth bits, index)
// in place (tmp: scratch of the same size as vals).
int count_scan_blocks(int n);
void launch_count_scan(int n, uint32_t *count, const ushort4 *rect, const uint32_t *rowpre, int TX,
                       uint32_t *part, uint32_t *vidx, uint32_t *voffs, uint32_t *kfirst,
                       Counters *cnt, uint32_t cap, const uint32_t *pre_partial, int n_pre,
                       HostCounters *host, uint32_t tag, hipStream_t st);
// long_lists: lists above 2048 entries are expected (a launch of their own
// for them); otherwise the few there are take a slower in-block path.
// order (optional): the blend order of the tiles is computed by one more
// block of the short-list launch, beside the sorting blocks.
void launch_segment_sort(int n_tiles, const uint2 *ranges, uint32_t *vals, uint32_t *tmp,
                         const uint32_t *dkey, bool long_lists, const OrderK *order,
                         hipStream_t st);
// Length bucket (floor(log2 len) + 1) from which a recent frame's lists make
// the long-list launch worth its cost: lists of 2048 entries and more.
constexpr int kSegLongBucket = 12;
// Longest list the per-tile sort handles in LDS; longer ones take its slower
// in-block path.  Lists of bucket <= kSegBucketMax (floor(log2 len) + 1)
// fit.
constexpr int kSegBucketMax = 12;

// ---- launchers (k_blend.hip) ----
// View pair of a TemporalGS frame (reference -> current) for the temporal
// kernels and stitching.
struct WarpK {
    float M[12];              // reference camera -> current camera
    float Minv[12];           // current camera -> reference camera
    float kref[4], kcur[4];   // fx, fy, cx, cy
    float z_near;
    int W, H, TX, TY;         // grid size (image, or the geometry buffer's) and tiles
    int tp;                   // pixels per tile side on this grid (16, or 8 at half resolution)
};

// Operands of the depth fill / backward query: one block of tp x tp threads
// per tile; also clears oc[tile] and resets this tile's cells of the other
// warp pair (dmin_next = empty depth, smax_next = 0) for the next frame.
struct FillK {
    WarpK w;
    const float *dmin;
    float *dfill;
    float2 *uv;
    uint8_t *um, *oc;
    float *dmin_next, *smax_next;
};

struct BlendArgs {
    int W, H, TX, TY;
    const int *tile_list;     // NULL: blockIdx = tile
    const uint32_t *n_tiles_dev;  // optional: blocks at or past *n_tiles_dev do nothing
    // optional (with tile_list): the first *n_split_dev (<= split_cap) tiles
    // of tile_list are blended as four quadrant blocks each; the launch adds
    // 3 split_cap + 28 blocks (4 ceil8(n_split) quadrant blocks replace
    // n_split tile blocks; n_grid: the launch's tile blocks, set by
    // launch_blend)
    const uint32_t *n_split_dev;
    int split_cap;            // with n_split_dev: *n_split_dev <= split_cap <= kMaxSplit
    int n_grid;
    const uint2 *ranges;
    const uint32_t *vals;
    const float4 *g;          // 64-byte records (Records::g)
    float *rgb;               // [3][H][W]
    float *tab;               // optional second copy of rgb
    float *depth, *sigma, *alpha;       // optional outputs
    float *tgb_depth, *tgb_sigma;       // optional second copies
    float *tgbh_depth, *tgbh_sigma;     // optional: Eq. 1/2 pooled over 2x2 blocks
                                        // (grid ceil(W/2) x ceil(H/2))
    uint8_t *g_flag;          // optional: Gaussian composited somewhere
    float *contrib;           // optional: max weight per Gaussian
    unsigned long long *pairs;  // optional: count of evaluated pixel-Gaussian pairs
    unsigned long long *hits;   // with pairs: count of pairs with alpha >= 1/255 (composited or stopping)
    float empty_depth;        // depth written where no Gaussian is composited
    float bg[3];              // background: rgb = sum of w c + T bg
    uint8_t *mark_sel, *mark_mask;   // optional: set to 1 for every blended tile
    // optional (TGS frames): blocks at or past *n_tiles_dev stitch tile
    // stitch_list[block] from the reference image stitch_tab (Eq. 4)
    // instead of blending, so that stitching overlaps the blend's tail:
    // stitch_mode 1 samples at the per-pixel correspondences stitch_uv,
    // 2 unprojects with the half-resolution repaired depth stitch_dfill
    // (grid width stitch_wg); sw is the full-resolution view pair
    const int *stitch_list;
    int stitch_mode, stitch_wg;
    const float *stitch_tab;
    const float2 *stitch_uv;
    const float *stitch_dfill;
    WarpK sw;
};
// Longest lists split into quadrant blocks by the blend: at most kMaxSplit
// tiles (a scene's cap; the launch adds 3 cap + 28 blocks, for 4 ceil8(n_split)
// quadrant blocks, those without a quadrant exit at once; none when the
// scene does not split), by default those of kSplitBucket (lists of
// 2^(kSplitBucket-1) entries) and up.
constexpr int kMaxSplit = TGS_BLEND_SPLIT_MAX;
constexpr int kSplitBucket = TGS_BLEND_SPLIT_DEFAULT + 1;
// start/stop (may be NULL) are attached to the dispatch itself
// (hipExtLaunchKernelGGL): kernel timing without extra barrier packets.
void launch_blend(const BlendArgs &a, int n_blocks, hipStream_t st, hipEvent_t start = nullptr,
                  hipEvent_t stop = nullptr);
// fbox must hold 4 + 4 * kAfcPartials ints (result, then partials).
constexpr int kAfcPartials = 256;
void launch_afc_bounds(int n, const uint8_t *g_flag, const float4 *g, int W, int H, int *fbox,
                       hipStream_t st);

// ---- launchers (k_temporal.hip) ----
// dmin = empty depth, smax = 0 over n_px cells
void launch_temporal_init(int n_px, float *dmin, float *smax, hipStream_t st);
void launch_forward_warp(const WarpK &w, const float *D, const float *S, float *dmin, float *smax,
                         hipStream_t st);
// Also oc[tile] = 0 and dmin_next / smax_next reset to their initial values
// (the other warp pair, for the next frame).
void launch_fill_query(const FillK &f, hipStream_t st);
void launch_occluded(const WarpK &w, int n, const uint8_t *status, const float4 *g,
                     const ushort4 *rect, uint8_t *oc, hipStream_t st);
// sel_list: the selected tiles ascending in [0, n_selected), the others
// descending from the end (a permutation of all tiles);
// sel_cols[ty * TX + k] = column of the k-th selected tile of row ty
void launch_select(int TX, int TY, int mode, const uint8_t *oc, const uint8_t *um, uint8_t *sel,
                   int *sel_list, uint32_t *rowpre, int *sel_cols, uint8_t *mask_out,
                   Counters *cnt, hipStream_t st);
void launch_fill_u8(uint8_t *p, size_t n, uint8_t v, hipStream_t st);
void launch_fill_f32(float *p, size_t n, float v, hipStream_t st);
void launch_fill_i32(int *p, size_t n, int v, hipStream_t st);

}  // namespace tgs
