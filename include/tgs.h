/*
 * tgs.h -- C-ABI of the TemporalGS hot path on MI355X (gfx950).
 *
 * TemporalGS (arxiv 2607.03390) renders a stream of camera views of a 3D
 * Gaussian Splatting scene.  Reference frames are rendered by the full
 * tile-based 3DGS pipeline (Sec. III-A: preprocess, Gaussian-tile key
 * duplication, per-tile depth sort, front-to-back alpha blending) and build
 * temporal priors (Sec. III-C: the temporal geometry buffer of Eq. 1/2, the
 * temporal appearance buffer, the temporal Gaussian buffer).  The frames in
 * between use them to drop Gaussians (temporal dynamic culling, Sec. III-D)
 * and to re-render only the tiles the warped priors cannot supply (selective
 * rendering, Sec. III-E, Eq. 3/4), with pseudo reference frames inserted by
 * interval and by the eta rule (Sec. III-E, Sec. IV-B).
 *
 * Conventions shared by every entry point:
 *  - Status codes only; nothing is thrown across the ABI.  On error the
 *    caller's outputs are left untouched (unless stated) and tgs_last_error()
 *    returns a message (thread-local, valid until the next call on the thread).
 *  - "host" pointers are read during the call only; "device" pointers are
 *    HIP device memory owned by the caller (for example torch tensors) and
 *    must stay valid until the enqueued work completes.
 *  - Work is enqueued on the caller's HIP stream (hipStream_t passed as
 *    void*, NULL = the null stream).  Every render call synchronises that
 *    stream once per frame to read the key and tile counts back, so the
 *    scalar fields of tgs_frame_out are valid on return and the device
 *    outputs are complete once the stream is synchronised.
 *  - Camera: world_to_cam is a row-major rigid 4x4 matrix (camera x right, y
 *    down, z forward); pinhole intrinsics fx, fy, cx, cy in pixels with pixel
 *    centres at integer coordinates.  Images are planar float32: rgb is
 *    [3][H][W], single-channel maps are [H][W].  Tiles are 16x16 pixels,
 *    TX = ceil(W/16), TY = ceil(H/16), numbered row-major.
 *  - A scene or a state is not thread-safe; distinct states may share a scene
 *    but calls on one scene or state must not overlap.
 */
#ifndef TGS_H
#define TGS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    TGS_OK = 0,
    TGS_ERR_INVALID_ARG = 1,     /* bad pointer, size, NaN, non-rigid pose ... */
    TGS_ERR_OUT_OF_MEMORY = 2,   /* a device or host allocation failed        */
    TGS_ERR_DEVICE = 3,          /* a HIP call or kernel launch failed        */
    TGS_ERR_STATE_MISMATCH = 4,  /* camera size differs from the state's      */
    TGS_ERR_CAPACITY = 5         /* more than 0xffff0000 keys in one frame     */
} tgs_status;

/* Frame kinds reported in tgs_frame_out.frame_kind (Sec. III-B, III-E). */
enum {
    TGS_FRAME_TRUE_REF = 0,   /* full render, no culling; refreshes all priors  */
    TGS_FRAME_PSEUDO_REF = 1, /* full render with adaptive frustum culling      */
    TGS_FRAME_TGS = 2,        /* AFC + TOC + selective rendering + stitching    */
    TGS_FRAME_FULL = 3        /* tgs_render_full (no temporal state)            */
};

/* Opaque device-resident scene (structure-of-arrays copy) and temporal state. */
typedef struct tgs_scene tgs_scene;
typedef struct tgs_state tgs_state;

/* Scene description (Sec. III-A: mean, covariance from scale and rotation,
 * opacity, SH colour).  All arrays are HOST memory in array-of-structs order,
 * already activated: scales are linear, opacities in [0,1], rotations are
 * quaternions (w,x,y,z) that need not be normalised (they must not be zero),
 * sh holds (sh_degree+1)^2 coefficients x 3 channels per Gaussian,
 * coefficient-major. */
typedef struct {
    int32_t n;            /* number of Gaussians, >= 0 (0 renders background) */
    int32_t sh_degree;    /* 0..3                                             */
    const float *means;   /* [n][3]                                           */
    const float *scales;  /* [n][3]                                           */
    const float *rotations; /* [n][4]                                         */
    const float *opacities; /* [n]                                            */
    const float *sh;      /* [n][(sh_degree+1)^2][3]                          */
} tgs_scene_desc;

typedef struct {
    float world_to_cam[16];   /* row-major rigid transform                    */
    float fx, fy, cx, cy;     /* pinhole intrinsics (pixels), fx, fy > 0      */
    int32_t width, height;    /* image size, 1..16384                         */
    float bg[3];              /* background colour (finite): front-to-back    */
                              /*    blending ends with RGB = C + T bg, T the  */
                              /*    transmittance left after the pixel's last */
                              /*    composited Gaussian (Sec. III-A)          */
} tgs_camera;

/* Method parameters: lambda_TDC, lambda_SR (Sec. III-B, IV-B), eta
 * (Sec. III-E), lambda1/lambda2 of the surface range (Sec. III-C), the near
 * plane of the 3DGS preprocess, and the ablation switches of Table IV.
 * Fixed, not parameters: the far plane z_far = 1000 and its margin eps = 1
 * (the empty depth z_far + eps of Sec. III-C is the value 1001, tested by
 * equality), and the 3DGS blending constants (alpha cap 0.99, alpha_min =
 * 1/255, termination below T = 1e-4): they define the full render that the
 * method approximates, and the occluded-tile test of Sec. III-E reuses the
 * same 1/255. */
typedef struct {
    int32_t lambda_tdc;       /* 50: interval between true references          */
    int32_t lambda_sr;        /* 5: interval between references of any kind    */
    float eta;                /* 0.40: selected-tile share that forces a pseudo reference */
    float lambda1;            /* 3: surface range below the warped depth       */
    float lambda2;            /* 0: surface range above the warped depth       */
    float z_near;             /* 0.2                                           */
    int32_t enable_afc;       /* 1: adaptive frustum culling                   */
    int32_t enable_toc;       /* 1: temporal occlusion culling                 */
    int32_t enable_sr;        /* 1: selective rendering (0 = render every tile)*/
    int32_t force_all_dirty;  /* 1: select every tile in TGS frames (testing)  */
    int32_t empty_far;        /* 1: a reference pixel where no Gaussian is      */
                              /*    composited gets depth z_far (1000) in the   */
                              /*    geometry buffer and the depth output, so it */
                              /*    warps and is stitched like a far surface;   */
                              /*    0 (default): NOHIT, never warped, its tile  */
                              /*    is re-rendered (Eq. 1 has no value there)   */
    int32_t tgb_downscale;    /* 1 (default), or 2: the temporal geometry       */
                              /*    buffer on the half-resolution grid, the     */
                              /*    paper's large-scene setting (Sec. IV-B):    */
                              /*    cell (i,j) is the 2x2 pixel block {2i,2i+1} */
                              /*    x {2j,2j+1} with Eq. 1/2 pooled over it;    */
                              /*    warp, fill and correspondences run on that  */
                              /*    grid (intrinsics f/2, (c-1/2)/2), the       */
                              /*    occlusion tests read the block of the       */
                              /*    mean's pixel, and stitching unprojects each */
                              /*    pixel with its block's repaired depth       */
} tgs_params;

/* Outputs of one rendered frame.  rgb is required; the other pointers may be
 * NULL.  depth/sigma/alpha are written on reference frames and by
 * tgs_render_full only (Eq. 1, Eq. 2 and 1-T; depth is 1001 = z_far+eps and
 * sigma 0 where no Gaussian was composited); contrib (per Gaussian, the
 * largest blending weight over the image, Sec. III-C) likewise.  tile_mask
 * receives 1 for every tile that was rasterised this frame. */
typedef struct {
    float *rgb;               /* device [3][H][W]                              */
    float *depth;             /* device [H][W] or NULL                         */
    float *sigma;             /* device [H][W] or NULL                         */
    float *alpha;             /* device [H][W] or NULL                         */
    float *contrib;           /* device [n] or NULL                            */
    uint8_t *tile_mask;       /* device [TY][TX] or NULL                       */
    /* scalars written by the library on success */
    int32_t frame_kind;       /* TGS_FRAME_*                                   */
    int32_t n_selected;       /* tiles rasterised                              */
    int32_t n_survivors;      /* Gaussians past the near plane and the culls   */
    int32_t n_newly_visible;  /* newly visible Gaussians (TGS frames)          */
    int64_t n_keys;           /* Gaussian-tile keys sorted                     */
} tgs_frame_out;

/* Fills *p with the paper's defaults (lambda_TDC 50, lambda_SR 5, eta 0.40,
 * lambda1 3, lambda2 0, near 0.2, all accelerations on). */
void tgs_params_default(tgs_params *p);

/* Copies a host scene to the device (Sec. III-A parameters) as
 * structure-of-arrays, on `stream`; synchronous on return.  *out is owned by
 * the caller and released with tgs_scene_free.  Errors: INVALID_ARG for NULL
 * arrays with n > 0, sh_degree outside 0..3, non-finite values or zero
 * quaternions; OUT_OF_MEMORY; DEVICE. */
tgs_status tgs_scene_upload(const tgs_scene_desc *desc, void *stream, tgs_scene **out);
void tgs_scene_free(tgs_scene *scene);
int32_t tgs_scene_count(const tgs_scene *scene);

/* Which tiles a Gaussian is duplicated into (Sec. III-A: the tiles it
 * intersects), for every later render of `scene` (full and temporal):
 *  TGS_TILES_3SIGMA (default, the 3DGS rule): the tiles whose pixel-centre
 *    span meets the square of half side ceil(3 sqrt(lambda_max(Sigma'))).
 *  TGS_TILES_FOOTPRINT: the tiles meeting the bounding box of the ellipse
 *    where the Gaussian can reach alpha >= 1/255 (an upper bound of
 *    2 ln(255 o) computed without transcendentals, enlarged 0.1% + 0.01 px);
 *    opacity below 1/255 gives no tiles.  Every pixel it leaves out has
 *    alpha < 1/255, so the image equals a tile-free blend of all Gaussians;
 *    it differs from the 3-sigma rule only where 3 sigma clips a Gaussian
 *    that still reaches 1/255.
 * Errors: INVALID_ARG for a NULL scene or an unknown rule. */
enum { TGS_TILES_3SIGMA = 0, TGS_TILES_FOOTPRINT = 1 };
tgs_status tgs_scene_set_tile_bound(tgs_scene *scene, int32_t bound);

/* Renders one frame with the full 3DGS pipeline (Sec. III-A), no temporal
 * state.  frame_kind = TGS_FRAME_FULL.  The scene holds the frame's
 * workspace, so calls on one scene must not overlap. */
tgs_status tgs_render_full(tgs_scene *scene, const tgs_camera *cam, tgs_frame_out *out,
                           void *stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the frame
 * of tgs_render_full, computed by the same kernels, with its whole
 * workspace (records, keys, sort tables, tile ranges, counters) in a fixed
 * array of TGS_NOALLOC_SCRATCH_BYTES that the library holds on each device
 * it runs on until the process ends.  The call allocates and frees nothing;
 * the caller passes the outputs as for tgs_render_full.  Every call on one
 * device shares that device's array: calls that overlap on a device race
 * (the stream must belong to the current device).  The scene's sort path
 * and blend split apply; profiling and tgs_debug_dump do not cover it.
 * Errors: CAPACITY when n Gaussians at width x height leave no room for
 * keys, or when the frame needs more Gaussian-tile keys than the array
 * holds after them (the outputs are then incomplete); otherwise as
 * tgs_render_full. */
#define TGS_NOALLOC_SCRATCH_BYTES (64u << 20)
tgs_status tgs_render_full_noalloc(const tgs_scene *scene, const tgs_camera *cam,
                                   tgs_frame_out *out, void *stream);

/* Creates the temporal state for `scene` at width x height (Sec. III-B..E):
 * priors, warp buffers and the frame schedule.  params may be NULL
 * (defaults).  The scene must outlive the state. */
tgs_status tgs_state_create(tgs_scene *scene, int32_t width, int32_t height,
                            const tgs_params *params, tgs_state **out);
/* Forgets all priors: the next tgs_render_temporal renders a true reference. */
tgs_status tgs_state_reset(tgs_state *state);
void tgs_state_free(tgs_state *state);

/* Renders the next frame of the stream (Sec. III-B..E).  The schedule picks
 * the kind: a true reference on the first frame and every lambda_tdc frames;
 * a pseudo reference every lambda_sr frames or after a TGS frame whose
 * selected tiles exceeded eta of all tiles; otherwise a TGS frame (adaptive
 * frustum + occlusion culling, selected tiles rasterised, the others stitched
 * from the reference image warped by Eq. 3/4).  cam->width/height must equal
 * the state's (STATE_MISMATCH otherwise). */
tgs_status tgs_render_temporal(tgs_state *state, const tgs_camera *cam, tgs_frame_out *out,
                               void *stream);

/* Host layout of an exported state: this header followed by
 *   float depth[Hg*Wg], float sigma[Hg*Wg] (temporal geometry buffer, Eq. 1/2,
 *                                        on its grid: Wg = ceil(W/s),
 *                                        Hg = ceil(H/s), s = tgb_downscale)
 *   float tab[3*H*W]                     (temporal appearance buffer)
 *   uint8_t g_rendered[n]                (temporal Gaussian buffer)        */
typedef struct {
    uint32_t magic;           /* 0x54475331 'TGS1'                             */
    int32_t width, height, n;
    int32_t frame_index;      /* frames rendered since the last reset          */
    int32_t since_true_ref;   /* frames since the last true reference          */
    int32_t since_ref;        /* frames since the last reference of any kind   */
    int32_t force_pseudo;     /* the eta rule fired on the last frame          */
    int32_t has_reference;    /* priors are valid                              */
    float fbox[4];            /* adaptive frustum F_min.xy, F_max.xy (NDC)     */
    float ref_world_to_cam[16];
    float ref_intrinsics[4];  /* fx, fy, cx, cy of the reference frame         */
    int32_t tgb_width, tgb_height;   /* grid of the geometry buffer (Wg, Hg)   */
} tgs_state_header;

/* Export: with host == NULL, *nbytes receives the blob size; otherwise the
 * blob is written (synchronous) if *nbytes is large enough (INVALID_ARG
 * otherwise).  Import: replaces the priors and counters (INVALID_ARG on a
 * size or magic mismatch, STATE_MISMATCH on other sizes).  Used for
 * checkpoint / resume and state-injection testing. */
tgs_status tgs_state_export(const tgs_state *state, void *host, size_t *nbytes);
tgs_status tgs_state_import(tgs_state *state, const void *host, size_t nbytes);

/* Intermediate buffers of the last frame rendered through `scene`
 * (tgs_render_full, state == NULL) or through `state`, copied to host
 * memory (synchronous).  host == NULL queries the size into *nbytes. */
enum {
    TGS_DUMP_SORTED_VALUES = 0,  /* uint32 [n_keys] Gaussian index per sorted key   */
    TGS_DUMP_SORTED_KEYS = 1,    /* uint32 [n_keys] tile id per sorted entry         */
    TGS_DUMP_TILE_RANGES = 2,    /* uint32 [TX*TY][2] start, end into the sorted keys */
    TGS_DUMP_RECORDS = 3,        /* float [n][12]: u, v, conic a, b | conic c, opacity, depth, 0 | r, g, b, 0 */
    TGS_DUMP_RECTS = 4,          /* uint16 [n][4] tile rectangle x0,y0,x1,y1 (x0 > x1: none) */
    TGS_DUMP_STATUS = 5,         /* uint8 [n] bit0 survivor, bit1 newly visible     */
    TGS_DUMP_WARP_DEPTH = 6,     /* float [Hg*Wg] warped min depth (Eq. 3), TGB grid */
    TGS_DUMP_WARP_SIGMA = 7,     /* float [Hg*Wg] warped max sigma                  */
    TGS_DUMP_FILLED_DEPTH = 8,   /* float [Hg*Wg] repaired depth                     */
    TGS_DUMP_CORRESPONDENCE = 9, /* float [Hg*Wg][2] reference (u,v) on the grid, -1 if unmatched */
    TGS_DUMP_UNMATCHED = 10,     /* uint8 [TX*TY] unmatched tiles                    */
    TGS_DUMP_OCCLUDED = 11,      /* uint8 [TX*TY] occluded tiles                     */
    TGS_DUMP_SELECTED = 12       /* uint8 [TX*TY] selected tiles                     */
};
tgs_status tgs_debug_dump(const tgs_scene *scene, const tgs_state *state, int32_t what,
                          void *host, size_t *nbytes);
/* Elements [first, first + count) of TGS_DUMP_SORTED_VALUES or
 * TGS_DUMP_SORTED_KEYS (uint32 each) into host (count * 4 bytes,
 * synchronous): the lists of a few tiles of a frame whose sorted keys are
 * too many to copy whole (their positions come from TGS_DUMP_TILE_RANGES).
 * INVALID_ARG for another buffer, a NULL host with count > 0, or a range
 * past the frame's keys. */
tgs_status tgs_debug_dump_range(const tgs_scene *scene, const tgs_state *state, int32_t what,
                                size_t first, size_t count, void *host);

/* Kernel timing for benchmarking.  Between tgs_profile_start and
 * tgs_profile_stop the blend dispatches carry HIP start/stop events attached
 * to the dispatch itself (no extra queue packets, so timing does not perturb
 * the frame); with TGS_PROFILE_STAGES every other stage is also bracketed by
 * separately recorded events on its stream (each such record adds a queue
 * barrier of several microseconds: use it in untimed passes).  With
 * TGS_PROFILE_COUNT_PAIRS the blend kernels also count the (pixel, Gaussian)
 * list entries their pixels evaluate up to termination (pairs) and, among
 * them, those whose alpha reaches 1/255, i.e. that are composited or stop the
 * pixel (hits: the pairs whose blending arithmetic cannot be skipped).  tgs_profile_stop synchronises the device and returns, per stage,
 * the summed event time and the number of timed launches.  Process-wide,
 * not thread-safe; renders must not overlap with start/stop. */
enum { TGS_PROFILE_COUNT_PAIRS = 1, TGS_PROFILE_STAGES = 2 };
enum {
    TGS_PROF_PREPROCESS = 0,  /* per-Gaussian stage (incl. counter reset)     */
    TGS_PROF_SCAN = 1,        /* key counts + exclusive scan                  */
    TGS_PROF_READBACK = 2,    /* unused: counters reach the host without a copy */
    TGS_PROF_DUPLICATE = 3,
    TGS_PROF_SORT = 4,        /* clear + histogram + all digit passes         */
    TGS_PROF_RANGES = 5,
    TGS_PROF_BLEND_FULL = 6,  /* tgs_render_full                              */
    TGS_PROF_BLEND_REF = 7,   /* reference frames (with prior capture)        */
    TGS_PROF_BLEND_TGS = 8,   /* TemporalGS frames: selected tiles blended,   */
                              /*    the others stitched, in one launch        */
    TGS_PROF_WARP = 9,        /* buffer init + forward warp                   */
    TGS_PROF_FILL_QUERY = 10,
    TGS_PROF_OCCLUDED = 11,
    TGS_PROF_SELECT = 12,
    TGS_PROF_STITCH = 13,     /* unused: stitching runs in the TGS blend      */
    TGS_PROF_CAPTURE = 14,    /* adaptive frustum, flag/mask resets           */
    TGS_PROF_STAGES = 16
};
typedef struct {
    double ms[TGS_PROF_STAGES];
    int64_t launches[TGS_PROF_STAGES];
    int64_t pairs[TGS_PROF_STAGES];   /* blend stages only, if counted        */
    int64_t hits[TGS_PROF_STAGES];    /* blend stages only, if counted        */
} tgs_profile;
tgs_status tgs_profile_start(int32_t flags);
tgs_status tgs_profile_stop(tgs_profile *out);

/* How each tile's front-to-back order (Sec. III-A: sort by depth within a
 * tile) is produced, for every later render through `scene` (tgs_render_full
 * and the temporal states bound to it).  Both ways give identical per-tile
 * lists (depth bits, then Gaussian index):
 *   TGS_SORT_DEPTH_FIRST: the Gaussians with keys are radix-sorted by depth
 *     (four passes of at most 8 bits over them), keys are emitted in that order and
 *     stably radix-sorted by tile;
 *   TGS_SORT_PER_TILE: key counts are scanned in index order, keys emitted
 *     in index order and stably sorted by tile, then one block per tile
 *     sorts its list by (depth bits, index) in LDS (lists above 4096 entries
 *     take a slower in-block path);
 *   TGS_SORT_AUTO (default): per frame, the per-tile sort for TemporalGS
 *     frames (keys on the selected tiles only), and for every frame of a
 *     scene with fewer than 131072 Gaussians, when the longest tile list of
 *     a recent frame of the same kind has fewer than 4096 entries; else the
 *     depth-first sort.
 * INVALID_ARG for a NULL scene or another value.  Like every call on a
 * scene, it must not overlap with renders through it. */
enum { TGS_SORT_AUTO = 0, TGS_SORT_DEPTH_FIRST = 1, TGS_SORT_PER_TILE = 2 };
tgs_status tgs_scene_set_sort_path(tgs_scene *scene, int32_t mode);

/* Which tiles the blend (Sec. III-A) splits, for every later render through
 * `scene`: a tile whose sorted list has at least 2^log2_min entries is
 * blended by four blocks, one per 8x8 quadrant, each taking four list
 * entries per pixel at a time (composited in list order: the result is the
 * unsplit blend's up to the order of the colour and moment sums).  If more
 * than max_tiles tiles qualify, the threshold is doubled until at most
 * max_tiles do (whole length classes, so a frame's result never depends on
 * scheduling).  The few longest lists set the blend's tail; a quadrant
 * block re-reads the whole list, so shorter ones are cheaper unsplit.
 * log2_min in [0, 31], or -1 for no split; max_tiles in [0,
 * TGS_BLEND_SPLIT_MAX].  Defaults: TGS_BLEND_SPLIT_DEFAULT,
 * TGS_BLEND_SPLIT_MAX.  INVALID_ARG for a NULL scene or other values. */
enum { TGS_BLEND_SPLIT_DEFAULT = 12, TGS_BLEND_SPLIT_MAX = 1024 };
tgs_status tgs_scene_set_blend_split(tgs_scene *scene, int32_t log2_min, int32_t max_tiles);

/* Message of the last failed call on this thread ("" if none). */
const char *tgs_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* TGS_H */
