// Host side of libtgs: the C-ABI of include/tgs.h, device memory, the frame
// schedule of TemporalGS (Sec. III-B, III-E last paragraph, Sec. IV-B) and
// the launch sequences of full, reference and TemporalGS frames.
//
// Every frame is enqueued on the caller's stream; the only host round trip
// is one read-back of four counters after the key scan (the key count sizes
// the sort and the selected-tile count drives the eta rule).
#include <math.h>
#include <string.h>

#include <atomic>
#include <mutex>
#include <string>
#include <vector>

#include "tgs.h"
#include "tgs_internal.h"

using namespace tgs;

namespace {

thread_local std::string g_err;

tgs_status fail(tgs_status s, const std::string &msg) {
    g_err = msg;
    return s;
}

#define TGS_HIP(call)                                                                        \
    do {                                                                                     \
        hipError_t e_ = (call);                                                              \
        if (e_ != hipSuccess)                                                                \
            return fail(e_ == hipErrorOutOfMemory ? TGS_ERR_OUT_OF_MEMORY : TGS_ERR_DEVICE, \
                        std::string(#call) + ": " + hipGetErrorString(e_));                  \
    } while (0)

#define TGS_LAUNCHED(what)                                                                   \
    do {                                                                                     \
        hipError_t e_ = hipGetLastError();                                                   \
        if (e_ != hipSuccess)                                                                \
            return fail(TGS_ERR_DEVICE, std::string(what) + ": " + hipGetErrorString(e_));   \
    } while (0)

#define TGS_TRY(expr)                   \
    do {                                \
        tgs_status s_ = (expr);         \
        if (s_ != TGS_OK) return s_;    \
    } while (0)

// A growable device allocation, or (borrowed) a view of memory it does not own.
struct DevBuf {
    void *p = nullptr;
    size_t bytes = 0;
    bool borrowed = false;
    ~DevBuf() {
        if (p && !borrowed) (void)hipFree(p);
    }
    void borrow(void *q, size_t b) {
        p = q;
        bytes = b;
        borrowed = true;
    }
    tgs_status ensure(size_t want) {
        if (borrowed) return fail(TGS_ERR_CAPACITY, "a borrowed buffer cannot grow");
        if (want <= bytes && p) return TGS_OK;
        if (p) {
            (void)hipFree(p);
            p = nullptr;
            bytes = 0;
        }
        const size_t alloc = want > 0 ? want : 16;
        hipError_t e = hipMalloc(&p, alloc);
        if (e != hipSuccess) {
            p = nullptr;
            return fail(TGS_ERR_OUT_OF_MEMORY, "hipMalloc of " + std::to_string(alloc) + " bytes failed");
        }
        bytes = alloc;
        return TGS_OK;
    }
    template <typename T>
    T *as() const { return static_cast<T *>(p); }
};

// Per-frame scratch of one render path (a scene's tgs_render_full, or a state).
struct Workspace {
    DevBuf g, rect, status, count, partial;
    DevBuf dkey, didx, dkey_alt, didx_alt, offs;
    DevBuf tkey, tval, tkey_alt, tval_alt, sort, kfirst;
    DevBuf ranges, sel, sel_list, sel_cols, rowpre, cnt, tile_order;
    HostCounters *host_cnt = nullptr;     // coherent pinned memory, written by the device
    HostCounters *host_cnt_dev = nullptr; // its device-side address
    // pinned: longest tile list's log2 bucket of some recent frame, [0] of
    // frames that render every tile, [1] of selective-rendering frames
    uint32_t *host_maxb = nullptr;
    uint32_t *host_maxb_dev = nullptr;
    bool frame_seg = false;               // this frame orders tiles by the per-tile sort
    uint32_t seq = 0;                     // tag of the last frame's counters
    int n = -1, W = 0, H = 0;
    size_t key_cap = 0;
    // last frame, for tgs_debug_dump
    uint32_t last_K = 0;
    uint32_t recent_K[2] = {0xffffffffu, 0xffffffffu};   // keys of the last frame per kind
                                                        // ([1]: selective rendering)
    const uint32_t *last_keys = nullptr, *last_vals = nullptr;
    bool has_frame = false;

    ~Workspace() {
        if (host_cnt) (void)hipHostFree(host_cnt);
        if (host_maxb) (void)hipHostFree(host_maxb);
    }

    tgs_status prepare(int n_, int W_, int H_) {
        const int TX = (W_ + 15) / 16, TY = (H_ + 15) / 16;
        const size_t nn = (size_t)(n_ > 0 ? n_ : 1);
        if (!host_cnt) {
            TGS_HIP(hipHostMalloc((void **)&host_cnt, sizeof(HostCounters),
                                  hipHostMallocCoherent | hipHostMallocMapped));
            memset(host_cnt, 0, sizeof(HostCounters));
            TGS_HIP(hipHostGetDevicePointer((void **)&host_cnt_dev, host_cnt, 0));
        }
        if (!host_maxb) {
            TGS_HIP(hipHostMalloc((void **)&host_maxb, 2 * sizeof(uint32_t),
                                  hipHostMallocCoherent | hipHostMallocMapped));
            // unknown: the first frame takes the depth-sorted path
            host_maxb[0] = host_maxb[1] = 0xffffffffu;
            TGS_HIP(hipHostGetDevicePointer((void **)&host_maxb_dev, host_maxb, 0));
        }
        if (n_ != n) {
            TGS_TRY(g.ensure(nn * 4 * sizeof(float4)));
            TGS_TRY(rect.ensure(nn * sizeof(ushort4)));
            TGS_TRY(status.ensure(nn));
            TGS_TRY(count.ensure((nn + 4) * sizeof(uint32_t)));
            TGS_TRY(partial.ensure((size_t)(2 * preprocess_blocks(n_ > 0 ? n_ : 1)) * sizeof(uint32_t)));
            TGS_TRY(dkey.ensure(nn * sizeof(uint32_t)));
            TGS_TRY(didx.ensure(nn * sizeof(uint32_t)));
            TGS_TRY(dkey_alt.ensure(nn * sizeof(uint32_t)));
            TGS_TRY(didx_alt.ensure(nn * sizeof(uint32_t)));
            TGS_TRY(offs.ensure(nn * sizeof(uint32_t)));
            // the depth sort runs over at most n keys
            TGS_TRY(sort.ensure(sort_scratch_words((uint32_t)nn) * sizeof(uint32_t)));
            n = n_;
        }
        if (W_ != W || H_ != H) {
            const size_t nt = (size_t)TX * TY;
            TGS_TRY(ranges.ensure(nt * sizeof(uint2)));
            TGS_TRY(sel.ensure(nt));
            TGS_TRY(sel_list.ensure(nt * sizeof(int)));
            TGS_TRY(tile_order.ensure(nt * sizeof(int)));
            TGS_TRY(sel_cols.ensure(nt * sizeof(int)));
            TGS_TRY(rowpre.ensure((size_t)TY * (TX + 1) * sizeof(uint32_t)));
            W = W_;
            H = H_;
        }
        TGS_TRY(cnt.ensure(sizeof(Counters)));
        return TGS_OK;
    }

    // Key buffers and sort scratch for at least `want` keys (capped at the
    // key limit).  Called before a frame is enqueued, or after an overflowed
    // frame has drained: the stream holds no work that uses them.
    tgs_status ensure_keys(size_t want, int passes) {
        if (want > (size_t)kMaxKeys) want = kMaxKeys;
        if (want > key_cap || !tkey.p) {
            const size_t cap = want;
            TGS_TRY(tkey.ensure(cap * sizeof(uint32_t)));
            TGS_TRY(tval.ensure(cap * sizeof(uint32_t)));
            TGS_TRY(tkey_alt.ensure(cap * sizeof(uint32_t)));
            TGS_TRY(tval_alt.ensure(cap * sizeof(uint32_t)));
            TGS_TRY(kfirst.ensure(key_blocks(cap) * sizeof(uint32_t)));
            key_cap = cap;
        }
        const size_t nn = (size_t)(n > 0 ? n : 1);
        const size_t words = sort_scratch_words((uint32_t)key_cap);
        const size_t words_depth = sort_scratch_words((uint32_t)nn);
        TGS_TRY(sort.ensure((words > words_depth ? words : words_depth) * sizeof(uint32_t)));
        return TGS_OK;
    }

    Records records() const {
        return Records{g.as<float4>(),
                       rect.as<ushort4>(),   status.as<uint8_t>(),  count.as<uint32_t>(),
                       dkey.as<uint32_t>(),  partial.as<uint32_t>()};
    }
};

bool finite(float x) { return isfinite(x) != 0; }

tgs_status check_camera(const tgs_camera *c) {
    if (!c) return fail(TGS_ERR_INVALID_ARG, "camera is NULL");
    if (c->width < 1 || c->height < 1 || c->width > 16384 || c->height > 16384)
        return fail(TGS_ERR_INVALID_ARG, "image size must be within 1..16384");
    if (!(finite(c->fx) && finite(c->fy) && c->fx > 0.0f && c->fy > 0.0f && finite(c->cx) &&
          finite(c->cy)))
        return fail(TGS_ERR_INVALID_ARG, "intrinsics must be finite with fx, fy > 0");
    if (!(finite(c->bg[0]) && finite(c->bg[1]) && finite(c->bg[2])))
        return fail(TGS_ERR_INVALID_ARG, "background colour must be finite");
    const float *m = c->world_to_cam;
    for (int i = 0; i < 16; ++i)
        if (!finite(m[i])) return fail(TGS_ERR_INVALID_ARG, "world_to_cam has a non-finite entry");
    if (fabsf(m[12]) > 1e-6f || fabsf(m[13]) > 1e-6f || fabsf(m[14]) > 1e-6f ||
        fabsf(m[15] - 1.0f) > 1e-6f)
        return fail(TGS_ERR_INVALID_ARG, "world_to_cam last row must be (0,0,0,1)");
    double R[3][3];
    for (int i = 0; i < 3; ++i)
        for (int j = 0; j < 3; ++j) R[i][j] = m[i * 4 + j];
    for (int i = 0; i < 3; ++i)
        for (int j = 0; j < 3; ++j) {
            double s = R[0][i] * R[0][j] + R[1][i] * R[1][j] + R[2][i] * R[2][j];
            if (fabs(s - (i == j ? 1.0 : 0.0)) > 1e-4)
                return fail(TGS_ERR_INVALID_ARG, "world_to_cam rotation is not orthonormal");
        }
    const double det = R[0][0] * (R[1][1] * R[2][2] - R[1][2] * R[2][1]) -
                       R[0][1] * (R[1][0] * R[2][2] - R[1][2] * R[2][0]) +
                       R[0][2] * (R[1][0] * R[2][1] - R[1][1] * R[2][0]);
    if (fabs(det - 1.0) > 1e-4) return fail(TGS_ERR_INVALID_ARG, "world_to_cam is not a rotation");
    return TGS_OK;
}

CamK make_camk(const tgs_camera *c) {
    CamK k;
    for (int i = 0; i < 12; ++i) k.V[i] = c->world_to_cam[i];
    k.fx = c->fx;
    k.fy = c->fy;
    k.cx = c->cx;
    k.cy = c->cy;
    k.W = c->width;
    k.H = c->height;
    k.TX = (c->width + 15) / 16;
    k.TY = (c->height + 15) / 16;
    const float tanfx = (0.5f * (float)c->width) / c->fx;
    const float tanfy = (0.5f * (float)c->height) / c->fy;
    k.limx = 1.3f * tanfx;
    k.limy = 1.3f * tanfy;
    // camera centre -R^T t, formed in double
    const float *m = c->world_to_cam;
    for (int i = 0; i < 3; ++i) {
        const double s = (double)m[0 * 4 + i] * (double)m[3] + (double)m[1 * 4 + i] * (double)m[7] +
                         (double)m[2 * 4 + i] * (double)m[11];
        k.campos[i] = (float)(-s);
    }
    return k;
}

// Relative pose of Eq. 3 in double: M = W_cur W_ref^-1 and its inverse,
// both rounded to fp32 3x4 row-major.
void relative_pose(const float *ref, const float *cur, float *M, float *Minv) {
    double a[16], b[16], ainv[16], binv[16];
    for (int i = 0; i < 16; ++i) {
        a[i] = ref[i];
        b[i] = cur[i];
    }
    a[12] = a[13] = a[14] = 0.0;
    a[15] = 1.0;
    b[12] = b[13] = b[14] = 0.0;
    b[15] = 1.0;
    auto rigid_inv = [](const double *x, double *xi) {
        for (int i = 0; i < 3; ++i) {
            for (int j = 0; j < 3; ++j) xi[i * 4 + j] = x[j * 4 + i];
            xi[i * 4 + 3] = -(x[0 * 4 + i] * x[3] + x[1 * 4 + i] * x[7] + x[2 * 4 + i] * x[11]);
        }
        xi[12] = xi[13] = xi[14] = 0.0;
        xi[15] = 1.0;
    };
    auto mul = [](const double *x, const double *y, float *out) {
        for (int i = 0; i < 3; ++i)
            for (int j = 0; j < 4; ++j) {
                double s = 0.0;
                for (int k = 0; k < 4; ++k) s += x[i * 4 + k] * y[k * 4 + j];
                out[i * 4 + j] = (float)s;
            }
    };
    rigid_inv(a, ainv);
    rigid_inv(b, binv);
    mul(b, ainv, M);
    mul(a, binv, Minv);
}


// Event timing of every launch while profiling is on (tgs_profile_start/stop).
struct Profiler {
    bool on = false, count = false, stages = false;
    std::vector<hipEvent_t> pool;
    size_t used = 0;
    struct Rec {
        int stage;
        hipEvent_t a, b;
    };
    std::vector<Rec> recs;
    unsigned long long *d_pairs = nullptr;

    hipEvent_t event() {
        if (used == pool.size()) {
            hipEvent_t e = nullptr;
            if (hipEventCreate(&e) != hipSuccess) return nullptr;
            pool.push_back(e);
        }
        return pool[used++];
    }
    // d_pairs: [0, STAGES) evaluated pairs, [STAGES, 2 STAGES) pairs that reach alpha >= 1/255
    unsigned long long *pairs(int stage) { return on && count ? d_pairs + stage : nullptr; }
    unsigned long long *hits(int stage) {
        return on && count ? d_pairs + TGS_PROF_STAGES + stage : nullptr;
    }
    // events attached to one kernel dispatch (no extra packets)
    void kernel_events(int stage, hipEvent_t *a, hipEvent_t *b) {
        *a = *b = nullptr;
        if (!on) return;
        *a = event();
        *b = event();
        if (*a && *b) recs.push_back({stage, *a, *b});
        else *a = *b = nullptr;
    }
};
Profiler g_prof;

// Set for the duration of an allocation-free call on this thread: no
// profiling events (creating one allocates).
thread_local bool t_no_alloc = false;

// Brackets the launches of one stage with events recorded on their stream
// (detail mode only: each separate event record costs a barrier packet).
struct ProfScope {
    int stage;
    hipStream_t st;
    hipEvent_t a = nullptr;
    ProfScope(int stage_, hipStream_t st_) : stage(stage_), st(st_) {
        if (!t_no_alloc && g_prof.on && g_prof.stages && (a = g_prof.event()) != nullptr)
            (void)hipEventRecord(a, st);
    }
    ~ProfScope() {
        if (!a) return;
        hipEvent_t b = g_prof.event();
        if (!b) return;
        (void)hipEventRecord(b, st);
        g_prof.recs.push_back({stage, a, b});
    }
};

}  // namespace

// ---------------------------------------------------------------------------
// opaque objects
// ---------------------------------------------------------------------------

struct tgs_scene {
    int n = 0, deg = 0, ncoef = 1;
    int tile_bound = TGS_TILES_3SIGMA;
    // how each tile's depth order is produced: 0 = per frame (the per-tile
    // sort in selective-rendering frames when the longest tile list of a
    // recent frame fits its LDS bound, else the global depth sort), 1 =
    // always the global depth sort, 2 = always the per-tile sort
    int sort_path = TGS_SORT_AUTO;
    // list length bucket from which the blend splits tiles into quadrants
    // (0: never), and the most tiles split
    int split_bucket = tgs::kSplitBucket;
    int split_max = tgs::kMaxSplit;
    DevBuf data;
    SceneDev view{};
    Workspace ws;
    int last_W = 0, last_H = 0;
};

struct tgs_state {
    tgs_scene *scene = nullptr;
    int W = 0, H = 0, TX = 0, TY = 0;
    int Wg = 0, Hg = 0;               // grid of the geometry buffer (image / tgb_downscale)
    tgs_params p{};
    Workspace ws;
    DevBuf tgb_d, tgb_s, tab, g_flag, fbox, dfill, uv, um, oc;
    // forward-warp targets (Eq. 3), two pairs: a frame warps into pair
    // warp_next while its fill / query kernel resets the other pair for the
    // next frame, so no launch of its own clears them (warp_clean: pair
    // warp_next holds its initial values; warp_last: the pair of the last
    // frame, for the debug dumps)
    DevBuf dmin[2], smax[2];
    int warp_next = 0, warp_last = 0;
    bool warp_clean = false;
    int frame_index = 0, since_true = 0, since_ref = 0, force_pseudo = 0, has_ref = 0;
    float fbox_host[4] = {0, 0, 0, 0};
    float ref_w2c[16] = {0};
    float ref_intr[4] = {0};
};

// ---------------------------------------------------------------------------
// shared frame steps
// ---------------------------------------------------------------------------

namespace {

struct FrameResult {
    uint32_t K = 0, V = 0, n_surv = 0, n_newly = 0, n_sel = 0;
};

// Zero the counters and run the per-Gaussian stage.
tgs_status step_preprocess(const tgs_scene *sc, Workspace &ws, const CamK &cam, const CullK &cull,
                           hipStream_t st, const FillK *fill = nullptr) {
    ProfScope ps(TGS_PROF_PREPROCESS, st);
    CullK c = cull;
    c.footprint = sc->tile_bound == TGS_TILES_FOOTPRINT ? 1 : 0;
    // the dispatch carries its own timing events (outside the stage mode,
    // whose scope brackets the stage instead)
    hipEvent_t ev0 = nullptr, ev1 = nullptr;
    if (!t_no_alloc && !g_prof.stages) g_prof.kernel_events(TGS_PROF_PREPROCESS, &ev0, &ev1);
    launch_preprocess(sc->view, cam, c, ws.records(), ws.cnt.as<Counters>(), fill, st, ev0, ev1);
    TGS_LAUNCHED("preprocess");
    return TGS_OK;
}

constexpr int kSegSmallScene = 131072;

// The Gaussians that have keys and the start of their keys, in the order the
// keys are emitted: depth order (global depth sort; the last pass publishes
// the frame's counters to the host, tag ws.seq) or index order (count scan,
// each tile's list sorted by depth after the tile sort).  Nothing here waits.
tgs_status step_scan(const tgs_scene *sc, Workspace &ws, const uint32_t *rowpre, int TX,
                     hipStream_t st, const uint32_t **sorted_didx) {
    const int n = sc->n;
    // per frame: the per-tile sort pays off in selective-rendering frames
    // (keys only on the selected tiles) whose lists fit its LDS bound; a
    // frame rendering every tile sorts 3-4 times as many keys per tile as
    // the depth sort sorts Gaussians, and takes the global depth sort
    // (and in every frame of a small scene: below kSegSmallScene Gaussians the
    // four depth passes are launch latency, not work)
    const uint32_t maxb = ws.host_maxb ? reinterpret_cast<volatile uint32_t *>(ws.host_maxb)[rowpre ? 1 : 0]
                                       : 0xffffffffu;
    ws.frame_seg = sc->sort_path == TGS_SORT_PER_TILE ||
                   (sc->sort_path == TGS_SORT_AUTO && (rowpre != nullptr || n < kSegSmallScene) &&
                    maxb <= (uint32_t)kSegBucketMax);
    if (ws.frame_seg) {
        ProfScope ps(TGS_PROF_SORT, st);
        ws.seq += 1;
        uint32_t *part = ws.sort.as<uint32_t>();
        launch_count_scan(n, ws.count.as<uint32_t>(), ws.rect.as<ushort4>(), rowpre, TX, part,
                          ws.didx.as<uint32_t>(), ws.offs.as<uint32_t>(), ws.kfirst.as<uint32_t>(),
                          ws.cnt.as<Counters>(), (uint32_t)ws.key_cap, ws.partial.as<uint32_t>(),
                          n > 0 ? preprocess_blocks(n) : 0, ws.host_cnt_dev, ws.seq, st);
        TGS_LAUNCHED("count scan");
        *sorted_didx = ws.didx.as<uint32_t>();
        return TGS_OK;
    }
    {
        ProfScope ps(TGS_PROF_SORT, st);
        ws.seq += 1;
        launch_depth_sort(n, ws.count.as<uint32_t>(), ws.rect.as<ushort4>(), rowpre, TX,
                          ws.dkey.as<uint32_t>(),
                          ws.dkey_alt.as<uint32_t>(), ws.didx_alt.as<uint32_t>(),
                          ws.dkey.as<uint32_t>(), ws.didx.as<uint32_t>(), ws.offs.as<uint32_t>(),
                          ws.kfirst.as<uint32_t>(), ws.sort.as<uint32_t>(), ws.cnt.as<Counters>(),
                          (uint32_t)ws.key_cap,
                          ws.partial.as<uint32_t>(), n > 0 ? preprocess_blocks(n) : 0,
                          ws.host_cnt_dev, ws.seq, st);
        TGS_LAUNCHED("depth sort");
    }
    *sorted_didx = ws.didx.as<uint32_t>();
    return TGS_OK;
}

// Waits (spinning: a blocking wait adds tens of microseconds of wake-up) for
// the counters of the frame enqueued last; the stream keeps working on the
// rest of the frame meanwhile.  *overflow: the frame needed more keys than
// the buffers hold (it rendered without keys; grow and render it again).
tgs_status step_wait_counters(Workspace &ws, hipStream_t st, FrameResult &fr, bool *overflow) {
    HostCounters copy{};
    if (!ws.host_cnt) {
        // counters in device memory (allocation-free calls): copied back once
        // the frame has drained
        TGS_HIP(hipMemcpyAsync(&copy, ws.host_cnt_dev, sizeof(copy), hipMemcpyDeviceToHost, st));
        TGS_HIP(hipStreamSynchronize(st));
        if (copy.tag != ws.seq) return fail(TGS_ERR_DEVICE, "frame counters missing after the frame");
    }
    volatile HostCounters *h = ws.host_cnt ? ws.host_cnt : &copy;
    for (uint32_t spins = 1; h->tag != ws.seq; ++spins) {
        if ((spins & 4095u) == 0u) {
            const hipError_t q = hipStreamQuery(st);
            if (q == hipSuccess && h->tag != ws.seq)
                return fail(TGS_ERR_DEVICE, "frame counters missing after the stream drained");
            if (q != hipSuccess && q != hipErrorNotReady)
                return fail(TGS_ERR_DEVICE, std::string("frame read-back: ") + hipGetErrorString(q));
        }
    }
    std::atomic_thread_fence(std::memory_order_acquire);
    fr.K = h->n_keys;
    fr.V = h->n_visible;
    fr.n_surv = h->n_survivors;
    fr.n_newly = h->n_newly;
    fr.n_sel = h->n_selected;
    *overflow = fr.K > 0 && h->n_sorted == 0;
    if (*overflow && fr.K > kMaxKeys)
        return fail(TGS_ERR_CAPACITY, "frame needs " + std::to_string(fr.K) +
                                          " or more Gaussian-tile keys; the limit is " +
                                          std::to_string(kMaxKeys));
    if (!*overflow) ws.last_K = fr.K;
    return TGS_OK;
}

// After an overflow: let the frame drain, then grow the key buffers.
tgs_status grow_after_overflow(Workspace &ws, const FrameResult &fr, int passes, hipStream_t st) {
    TGS_HIP(hipStreamSynchronize(st));
    const size_t want = (size_t)fr.K + fr.K / 4 + 65536;
    return ws.ensure_keys(want, passes);
}

// Key bits of a tile id on a TX x TY grid.
int tile_id_bits(int TX, int TY) {
    int bits = 0;
    while ((1 << bits) < TX * TY) ++bits;
    return bits;
}

int tile_sort_passes(int TX, int TY) { return sort_passes_for_bits(tile_id_bits(TX, TY)); }

// Emit the keys in depth order, sort them by tile (stable), find tile ranges;
// returns the per-tile lists of Gaussian indices.
tgs_status step_keys(const tgs_scene *sc, Workspace &ws, int TX, int TY, const uint32_t *rowpre,
                     const int *sel_cols, const uint32_t *didx, hipStream_t st,
                     const uint32_t **sorted_vals) {
    const int n = sc->n;
    const uint32_t cap = (uint32_t)ws.key_cap;
    Counters *cnt = ws.cnt.as<Counters>();
    const int bits = tile_id_bits(TX, TY);
    const uint32_t hint = ws.recent_K[rowpre ? 1 : 0];
    // the emission counts the tile sort's first digit per block of keys
    // (where the sort's partitions are whole blocks), in place of that
    // pass's counting launch
    const bool counted = sort_takes_rows(cap, hint, 0, bits);
    {
        ProfScope ps(TGS_PROF_DUPLICATE, st);
        launch_duplicate(n, cap, cnt, didx, ws.offs.as<uint32_t>(), ws.kfirst.as<uint32_t>(),
                         ws.rect.as<ushort4>(), rowpre, sel_cols, TX, TX * TY,
                         ws.tkey.as<uint32_t>(), ws.tval.as<uint32_t>(), ws.ranges.as<uint2>(),
                         sort_count_rows(ws.sort.as<uint32_t>()),
                         counted ? sort_first_digit_bits(bits) : 0, st);
        TGS_LAUNCHED("duplicate");
    }
    int alt = 0;
    {
        ProfScope ps(TGS_PROF_SORT, st);
        alt = launch_sort_u32(&cnt->n_sorted, cap, hint, 0, bits, ws.tkey.as<uint32_t>(),
                              ws.tval.as<uint32_t>(), ws.tkey_alt.as<uint32_t>(),
                              ws.tval_alt.as<uint32_t>(), ws.sort.as<uint32_t>(), counted, st);
        TGS_LAUNCHED("tile sort");
    }
    const uint32_t *skeys = alt ? ws.tkey_alt.as<uint32_t>() : ws.tkey.as<uint32_t>();
    uint32_t *svals = alt ? ws.tval_alt.as<uint32_t>() : ws.tval.as<uint32_t>();
    {
        ProfScope ps(TGS_PROF_RANGES, st);
        launch_ranges(cap, cnt, skeys, ws.ranges.as<uint2>(), st);
        TGS_LAUNCHED("ranges");
    }
    // blend order: the selected tiles, or all of them, longest lists first
    OrderK order{};
    order.n_host = TX * TY;
    order.n_dev = rowpre ? &cnt->n_selected : nullptr;
    order.tile_in = rowpre ? ws.sel_list.as<int>() : nullptr;
    order.ranges = ws.ranges.as<uint2>();
    order.tile_out = ws.tile_order.as<int>();
    order.max_bucket = ws.host_maxb_dev + (rowpre ? 1 : 0);
    order.n_split = &cnt->n_split;
    order.split_bucket = sc->split_bucket;
    order.max_split = sc->split_max;
    if (ws.frame_seg) {
        // each tile's list, emitted in index order, by (depth bits, index)
        ProfScope ps(TGS_PROF_SORT, st);
        // lists above 2048 entries get a launch of their own when a recent
        // frame of the same kind had any (the longest list's bucket, from the
        // host copy)
        // the blend order (below) is computed by one more block of this launch
        const uint32_t maxb = ws.host_maxb
            ? reinterpret_cast<volatile uint32_t *>(ws.host_maxb)[rowpre ? 1 : 0] : 0xffffffffu;
        launch_segment_sort(TX * TY, ws.ranges.as<uint2>(), svals,
                            alt ? ws.tval.as<uint32_t>() : ws.tval_alt.as<uint32_t>(),
                            ws.dkey.as<uint32_t>(), maxb >= (uint32_t)kSegLongBucket, &order, st);
        TGS_LAUNCHED("per-tile sort and tile order");
    } else {
        ProfScope ps(TGS_PROF_RANGES, st);
        launch_order_tiles(order, st);
        TGS_LAUNCHED("tile order");
    }
    *sorted_vals = alt ? ws.tval_alt.as<uint32_t>() : ws.tval.as<uint32_t>();
    ws.last_keys = skeys;
    ws.last_vals = *sorted_vals;
    ws.has_frame = true;
    return TGS_OK;
}

// The blend order of the tiles and the split of the longest ones into
// quadrant blocks (per frame, from the frame's own lists; off when the scene
// does not split, and then the launch takes no spare blocks for it).
void set_blend_order(BlendArgs &a, const Workspace &ws, const tgs_scene *sc) {
    a.tile_list = ws.tile_order.as<int>();
    a.n_split_dev = &ws.cnt.as<Counters>()->n_split;
    a.split_cap = sc->split_max;
    if (sc->split_bucket <= 0 || sc->split_max <= 0) a.n_split_dev = nullptr;
}

BlendArgs blend_args(const Workspace &ws, const tgs_camera *cam, const uint32_t *vals) {
    const int W = cam->width, H = cam->height;
    BlendArgs a{};
    a.bg[0] = cam->bg[0];
    a.bg[1] = cam->bg[1];
    a.bg[2] = cam->bg[2];
    a.W = W;
    a.H = H;
    a.TX = (W + 15) / 16;
    a.TY = (H + 15) / 16;
    a.ranges = ws.ranges.as<uint2>();
    a.vals = vals;
    a.g = ws.g.as<float4>();
    a.empty_depth = kNoHit;
    return a;
}

CullK no_cull(float z_near, Workspace &ws) {
    CullK c{};
    c.z_near = z_near;
    c.lambda1 = 3.0f;
    return c;
}

tgs_status check_params(const tgs_params *p) {
    if (p->lambda_tdc < 1 || p->lambda_sr < 1)
        return fail(TGS_ERR_INVALID_ARG, "lambda_tdc and lambda_sr must be >= 1");
    if (!(finite(p->eta) && p->eta >= 0.0f))
        return fail(TGS_ERR_INVALID_ARG, "eta must be finite and >= 0");
    if (!(finite(p->lambda1) && finite(p->lambda2)))
        return fail(TGS_ERR_INVALID_ARG, "lambda1, lambda2 must be finite");
    if (!(finite(p->z_near) && p->z_near > 0.0f))
        return fail(TGS_ERR_INVALID_ARG, "z_near must be finite and > 0");
    if (p->empty_far != 0 && p->empty_far != 1)
        return fail(TGS_ERR_INVALID_ARG, "empty_far must be 0 or 1");
    if (p->tgb_downscale != 1 && p->tgb_downscale != 2)
        return fail(TGS_ERR_INVALID_ARG, "tgb_downscale must be 1 or 2");
    return TGS_OK;
}

}  // namespace

// ---------------------------------------------------------------------------
// C-ABI
// ---------------------------------------------------------------------------

extern "C" {

const char *tgs_last_error(void) { return g_err.c_str(); }

tgs_status tgs_scene_set_sort_path(tgs_scene *scene, int32_t mode) {
    g_err.clear();
    if (!scene) return fail(TGS_ERR_INVALID_ARG, "scene is NULL");
    if (mode != TGS_SORT_AUTO && mode != TGS_SORT_DEPTH_FIRST && mode != TGS_SORT_PER_TILE)
        return fail(TGS_ERR_INVALID_ARG, "sort path must be 0, 1 or 2");
    scene->sort_path = mode;
    return TGS_OK;
}

tgs_status tgs_scene_set_blend_split(tgs_scene *scene, int32_t log2_min, int32_t max_tiles) {
    g_err.clear();
    if (!scene) return fail(TGS_ERR_INVALID_ARG, "scene is NULL");
    if (log2_min < -1 || log2_min > 31) return fail(TGS_ERR_INVALID_ARG, "log2_min must be in [-1, 31]");
    if (max_tiles < 0 || max_tiles > kMaxSplit)
        return fail(TGS_ERR_INVALID_ARG, "max_tiles must be in [0, " + std::to_string(kMaxSplit) + "]");
    scene->split_bucket = log2_min + 1;
    scene->split_max = max_tiles;
    return TGS_OK;
}

tgs_status tgs_profile_start(int32_t flags) {
    g_err.clear();
    if (!g_prof.d_pairs)
        TGS_HIP(hipMalloc((void **)&g_prof.d_pairs, 2 * TGS_PROF_STAGES * sizeof(unsigned long long)));
    TGS_HIP(hipDeviceSynchronize());
    TGS_HIP(hipMemset(g_prof.d_pairs, 0, 2 * TGS_PROF_STAGES * sizeof(unsigned long long)));
    g_prof.used = 0;
    g_prof.recs.clear();
    g_prof.count = (flags & TGS_PROFILE_COUNT_PAIRS) != 0;
    g_prof.stages = (flags & TGS_PROFILE_STAGES) != 0;
    g_prof.on = true;
    return TGS_OK;
}

tgs_status tgs_profile_stop(tgs_profile *out) {
    g_err.clear();
    if (!g_prof.on) return fail(TGS_ERR_INVALID_ARG, "profiling was not started");
    g_prof.on = false;
    TGS_HIP(hipDeviceSynchronize());
    tgs_profile r{};
    for (const auto &rec : g_prof.recs) {
        float ms = 0.0f;
        TGS_HIP(hipEventElapsedTime(&ms, rec.a, rec.b));
        r.ms[rec.stage] += ms;
        r.launches[rec.stage] += 1;
    }
    unsigned long long pairs[2 * TGS_PROF_STAGES];
    TGS_HIP(hipMemcpy(pairs, g_prof.d_pairs, sizeof(pairs), hipMemcpyDeviceToHost));
    for (int k = 0; k < TGS_PROF_STAGES; ++k) {
        r.pairs[k] = g_prof.count ? (int64_t)pairs[k] : 0;
        r.hits[k] = g_prof.count ? (int64_t)pairs[TGS_PROF_STAGES + k] : 0;
    }
    g_prof.recs.clear();
    g_prof.used = 0;
    if (out) *out = r;
    return TGS_OK;
}

void tgs_params_default(tgs_params *p) {
    if (!p) return;
    p->lambda_tdc = 50;
    p->lambda_sr = 5;
    p->eta = 0.40f;
    p->lambda1 = 3.0f;
    p->lambda2 = 0.0f;
    p->z_near = 0.2f;
    p->enable_afc = 1;
    p->enable_toc = 1;
    p->enable_sr = 1;
    p->force_all_dirty = 0;
    p->empty_far = 0;
    p->tgb_downscale = 1;
}

tgs_status tgs_scene_upload(const tgs_scene_desc *d, void *stream, tgs_scene **out) {
    g_err.clear();
    if (!d || !out) return fail(TGS_ERR_INVALID_ARG, "desc and out must not be NULL");
    if (d->n < 0) return fail(TGS_ERR_INVALID_ARG, "n must be >= 0");
    if (d->sh_degree < 0 || d->sh_degree > 3)
        return fail(TGS_ERR_INVALID_ARG, "sh_degree must be within 0..3");
    const int n = d->n, ncoef = (d->sh_degree + 1) * (d->sh_degree + 1);
    if (n > 0 && (!d->means || !d->scales || !d->rotations || !d->opacities || !d->sh))
        return fail(TGS_ERR_INVALID_ARG, "scene arrays must not be NULL when n > 0");
    for (size_t k = 0; k < (size_t)n * 3; ++k)
        if (!finite(d->means[k]) || !finite(d->scales[k]))
            return fail(TGS_ERR_INVALID_ARG, "non-finite mean or scale");
    for (int i = 0; i < n; ++i) {
        const float *q = d->rotations + 4 * (size_t)i;
        if (!(finite(q[0]) && finite(q[1]) && finite(q[2]) && finite(q[3])))
            return fail(TGS_ERR_INVALID_ARG, "non-finite rotation");
        if (q[0] == 0.0f && q[1] == 0.0f && q[2] == 0.0f && q[3] == 0.0f)
            return fail(TGS_ERR_INVALID_ARG, "zero quaternion at Gaussian " + std::to_string(i));
        if (!finite(d->opacities[i])) return fail(TGS_ERR_INVALID_ARG, "non-finite opacity");
    }
    for (size_t k = 0; k < (size_t)n * ncoef * 3; ++k)
        if (!finite(d->sh[k])) return fail(TGS_ERR_INVALID_ARG, "non-finite SH coefficient");

    tgs_scene *sc = new (std::nothrow) tgs_scene();
    if (!sc) return fail(TGS_ERR_OUT_OF_MEMORY, "host allocation failed");
    sc->n = n;
    sc->deg = d->sh_degree;
    sc->ncoef = ncoef;
    const int slots = (3 * ncoef + 3) / 4;
    const size_t n_pad = ((size_t)(n > 0 ? n : 1) + 63) / 64 * 64;
    const size_t n_vec = n_pad * (3 + (size_t)slots);   // float4 count: mean, 2 geometry, SH
    tgs_status s = sc->data.ensure(n_vec * sizeof(float4));
    if (s != TGS_OK) {
        delete sc;
        return s;
    }
    float4 *base = sc->data.as<float4>();
    hipStream_t st = (hipStream_t)stream;
    std::vector<float4> stage;
    hipError_t e = hipSuccess;
    try {
        stage.assign(n_pad, make_float4(0.0f, 0.0f, 0.0f, 0.0f));
    } catch (...) {
        delete sc;
        return fail(TGS_ERR_OUT_OF_MEMORY, "host staging allocation failed");
    }
    auto put = [&](float4 *dst) -> hipError_t {
        hipError_t err = hipMemcpyAsync(dst, stage.data(), n_pad * sizeof(float4),
                                        hipMemcpyHostToDevice, st);
        if (err != hipSuccess) return err;
        return hipStreamSynchronize(st);
    };
    for (int i = 0; i < n; ++i)
        stage[i] = make_float4(d->means[3 * (size_t)i], d->means[3 * (size_t)i + 1],
                               d->means[3 * (size_t)i + 2], d->opacities[i]);
    e = put(base);
    // geometry: (sx, sy, sz, qw), (qx, qy, qz, 0) side by side per Gaussian
    if (e == hipSuccess) {
        std::vector<float4> geo;
        try {
            geo.assign(2 * n_pad, make_float4(0.0f, 0.0f, 0.0f, 0.0f));
        } catch (...) {
            delete sc;
            return fail(TGS_ERR_OUT_OF_MEMORY, "host staging allocation failed");
        }
        for (int i = 0; i < n; ++i) {
            geo[2 * (size_t)i] = make_float4(d->scales[3 * (size_t)i], d->scales[3 * (size_t)i + 1],
                                             d->scales[3 * (size_t)i + 2], d->rotations[4 * (size_t)i]);
            geo[2 * (size_t)i + 1] =
                make_float4(d->rotations[4 * (size_t)i + 1], d->rotations[4 * (size_t)i + 2],
                            d->rotations[4 * (size_t)i + 3], 0.0f);
        }
        e = hipMemcpyAsync(base + n_pad, geo.data(), geo.size() * sizeof(float4),
                           hipMemcpyHostToDevice, st);
        if (e == hipSuccess) e = hipStreamSynchronize(st);
    }
    // SH: each Gaussian's slots contiguous
    if (e == hipSuccess) {
        const size_t per = (size_t)ncoef * 3;
        std::vector<float4> sh;
        try {
            sh.assign(n_pad * slots, make_float4(0.0f, 0.0f, 0.0f, 0.0f));
        } catch (...) {
            delete sc;
            return fail(TGS_ERR_OUT_OF_MEMORY, "host staging allocation failed");
        }
        for (int i = 0; i < n; ++i) {
            const float *src = d->sh + (size_t)i * per;
            for (int j = 0; j < slots; ++j) {
                float v[4];
                for (int c = 0; c < 4; ++c) {
                    const size_t f = 4 * (size_t)j + c;
                    v[c] = f < per ? src[f] : 0.0f;
                }
                sh[(size_t)i * slots + j] = make_float4(v[0], v[1], v[2], v[3]);
            }
        }
        e = hipMemcpyAsync(base + 3 * n_pad, sh.data(), sh.size() * sizeof(float4),
                           hipMemcpyHostToDevice, st);
        if (e == hipSuccess) e = hipStreamSynchronize(st);
    }
    if (e != hipSuccess) {
        delete sc;
        return fail(TGS_ERR_DEVICE, std::string("scene upload: ") + hipGetErrorString(e));
    }
    SceneDev &v = sc->view;
    v.n = n;
    v.deg = sc->deg;
    v.ncoef = ncoef;
    v.sh_slots = slots;
    v.mean_op = base;
    v.geo = base + n_pad;
    v.sh = base + 3 * n_pad;
    *out = sc;
    return TGS_OK;
}

void tgs_scene_free(tgs_scene *scene) { delete scene; }

int32_t tgs_scene_count(const tgs_scene *scene) { return scene ? scene->n : 0; }

tgs_status tgs_scene_set_tile_bound(tgs_scene *scene, int32_t bound) {
    g_err.clear();
    if (!scene) return fail(TGS_ERR_INVALID_ARG, "scene is NULL");
    if (bound != TGS_TILES_3SIGMA && bound != TGS_TILES_FOOTPRINT)
        return fail(TGS_ERR_INVALID_ARG, "tile bound must be TGS_TILES_3SIGMA or TGS_TILES_FOOTPRINT");
    scene->tile_bound = bound;
    return TGS_OK;
}

tgs_status tgs_render_full(tgs_scene *sc, const tgs_camera *cam, tgs_frame_out *out,
                           void *stream) {
    g_err.clear();
    if (!sc || !out || !out->rgb) return fail(TGS_ERR_INVALID_ARG, "scene, out and out->rgb are required");
    TGS_TRY(check_camera(cam));
    hipStream_t st = (hipStream_t)stream;
    const int W = cam->width, H = cam->height, TX = (W + 15) / 16, TY = (H + 15) / 16;
    Workspace &ws = sc->ws;
    TGS_TRY(ws.prepare(sc->n, W, H));
    const CamK ck = make_camk(cam);
    const int passes = tile_sort_passes(TX, TY);
    TGS_TRY(ws.ensure_keys(ws.key_cap ? ws.key_cap : 4 * (size_t)sc->n + 65536, passes));
    FrameResult fr;
    for (;;) {
        TGS_TRY(step_preprocess(sc, ws, ck, no_cull(0.2f, ws), st));
        const uint32_t *didx = nullptr, *vals = nullptr;
        TGS_TRY(step_scan(sc, ws, nullptr, TX, st, &didx));
        TGS_TRY(step_keys(sc, ws, TX, TY, nullptr, nullptr, didx, st, &vals));
        if (out->contrib) launch_fill_f32(out->contrib, (size_t)sc->n, 0.0f, st);
        BlendArgs a = blend_args(ws, cam, vals);
        set_blend_order(a, ws, sc);
        a.rgb = out->rgb;
        a.depth = out->depth;
        a.sigma = out->sigma;
        a.alpha = out->alpha;
        a.contrib = out->contrib;
        a.mark_mask = out->tile_mask;   // every tile is rendered
        a.pairs = g_prof.pairs(TGS_PROF_BLEND_FULL);
        a.hits = g_prof.hits(TGS_PROF_BLEND_FULL);
        {
            hipEvent_t ev0, ev1;
            g_prof.kernel_events(TGS_PROF_BLEND_FULL, &ev0, &ev1);
            launch_blend(a, TX * TY, st, ev0, ev1);
            TGS_LAUNCHED("blend");
        }
        bool overflow = false;
        TGS_TRY(step_wait_counters(ws, st, fr, &overflow));
        ws.recent_K[0] = fr.K;
        if (!overflow) break;
        TGS_TRY(grow_after_overflow(ws, fr, passes, st));
    }
    sc->last_W = W;
    sc->last_H = H;
    out->frame_kind = TGS_FRAME_FULL;
    out->n_selected = TX * TY;
    out->n_survivors = (int32_t)fr.n_surv;
    out->n_newly_visible = 0;
    out->n_keys = fr.K;
    return TGS_OK;
}

}  // extern "C"

// ---------------------------------------------------------------------------
// allocation-free full render
// ---------------------------------------------------------------------------

// The frame workspace of tgs_render_full_noalloc: one array per device, held
// by the library until the process ends and shared by every such call on
// that device.  In host code `scratch` names a host-side stand-in, not the
// device array: every host use goes through the address hipGetSymbolAddress
// returns for the current device.
static __device__ __align__(256) unsigned char scratch[TGS_NOALLOC_SCRATCH_BYTES];

namespace {

constexpr size_t kNoAllocBytes = (size_t)TGS_NOALLOC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
char *g_scratch_ptr[kMaxDevices] = {};

// The scratch array's address on the current device, looked up on the first
// call there (with that device current) and kept.
tgs_status scratch_address(char **out) {
    int dev = -1;
    TGS_HIP(hipGetDevice(&dev));
    if (dev < 0 || dev >= kMaxDevices) return fail(TGS_ERR_DEVICE, "device index out of range");
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return fail(TGS_ERR_DEVICE, std::string("hipGetSymbolAddress(scratch): ") +
                                            hipGetErrorString(e));
        g_scratch_ptr[dev] = static_cast<char *>(p);
    }
    *out = g_scratch_ptr[dev];
    return TGS_OK;
}

// 256-byte aligned pieces of [base, base + cap), handed out in order.
struct Carve {
    char *base;
    size_t cap, off;
    void *raw(size_t bytes) {
        off = (off + 255) & ~(size_t)255;
        if (off > cap || bytes > cap - off) return nullptr;
        void *p = base + off;
        off += bytes > 0 ? bytes : 1;
        return p;
    }
    bool take(DevBuf &b, size_t bytes) {
        void *p = raw(bytes);
        if (p) b.borrow(p, bytes);
        return p != nullptr;
    }
};

// Lays the workspace of a full render (n Gaussians, W x H, key_cap keys) over
// [base, base + cap); false if it does not fit.
bool layout_full(Workspace &ws, char *base, size_t cap, int n, int W, int H, size_t key_cap) {
    Carve c{base, cap, 0};
    const size_t nn = (size_t)(n > 0 ? n : 1);
    const int TX = (W + 15) / 16, TY = (H + 15) / 16;
    const size_t nt = (size_t)TX * TY;
    const size_t sort_words = std::max(sort_scratch_words((uint32_t)key_cap),
                                       sort_scratch_words((uint32_t)nn));
    bool ok = c.take(ws.g, nn * 4 * sizeof(float4)) && c.take(ws.rect, nn * sizeof(ushort4)) &&
              c.take(ws.status, nn) && c.take(ws.count, (nn + 4) * sizeof(uint32_t)) &&
              c.take(ws.partial, (size_t)(2 * preprocess_blocks((int)nn)) * sizeof(uint32_t)) &&
              c.take(ws.dkey, nn * 4) && c.take(ws.didx, nn * 4) && c.take(ws.dkey_alt, nn * 4) &&
              c.take(ws.didx_alt, nn * 4) && c.take(ws.offs, nn * 4) &&
              c.take(ws.ranges, nt * sizeof(uint2)) && c.take(ws.sel, nt) &&
              c.take(ws.sel_list, nt * sizeof(int)) && c.take(ws.tile_order, nt * sizeof(int)) &&
              c.take(ws.sel_cols, nt * sizeof(int)) &&
              c.take(ws.rowpre, (size_t)TY * (TX + 1) * sizeof(uint32_t)) &&
              c.take(ws.cnt, sizeof(Counters)) && c.take(ws.sort, sort_words * sizeof(uint32_t)) &&
              c.take(ws.tkey, key_cap * 4) && c.take(ws.tval, key_cap * 4) &&
              c.take(ws.tkey_alt, key_cap * 4) && c.take(ws.tval_alt, key_cap * 4) &&
              c.take(ws.kfirst, key_blocks(key_cap) * sizeof(uint32_t));
    void *hc = ok ? c.raw(sizeof(HostCounters)) : nullptr;
    void *mb = hc ? c.raw(2 * sizeof(uint32_t)) : nullptr;
    if (!mb) return false;
    // counters and the longest-list bucket stay in device memory: read back
    // by a copy, never through pinned host memory
    ws.host_cnt = nullptr;
    ws.host_cnt_dev = static_cast<HostCounters *>(hc);
    ws.host_maxb = nullptr;
    ws.host_maxb_dev = static_cast<uint32_t *>(mb);
    ws.n = n;
    ws.W = W;
    ws.H = H;
    ws.key_cap = key_cap;
    return true;
}

}  // namespace

extern "C" {

tgs_status tgs_render_full_noalloc(const tgs_scene *sc, const tgs_camera *cam, tgs_frame_out *out,
                                   void *stream) {
    g_err.clear();
    if (!sc || !out || !out->rgb) return fail(TGS_ERR_INVALID_ARG, "scene, out and out->rgb are required");
    TGS_TRY(check_camera(cam));
    hipStream_t st = (hipStream_t)stream;
    const int W = cam->width, H = cam->height, TX = (W + 15) / 16, TY = (H + 15) / 16;
    char *base = nullptr;
    TGS_TRY(scratch_address(&base));
    // the largest key capacity the scratch array leaves (host arithmetic only)
    Workspace ws;
    size_t lo = 0, hi = kNoAllocBytes / 16;
    {
        Workspace probe;
        if (!layout_full(probe, base, kNoAllocBytes, sc->n, W, H, kKeyBlock))
            return fail(TGS_ERR_CAPACITY, std::to_string(sc->n) + " Gaussians at " + std::to_string(W) +
                                              "x" + std::to_string(H) + " do not fit the " +
                                              std::to_string(kNoAllocBytes >> 20) +
                                              " MiB scratch array of the allocation-free render");
        lo = kKeyBlock;
    }
    while (lo < hi) {
        const size_t mid = lo + (hi - lo + 1) / 2;
        Workspace probe;
        if (layout_full(probe, base, kNoAllocBytes, sc->n, W, H, mid)) lo = mid;
        else hi = mid - 1;
    }
    if (!layout_full(ws, base, kNoAllocBytes, sc->n, W, H, lo))
        return fail(TGS_ERR_DEVICE, "scratch layout failed");
    // no profiling events in this call (creating one allocates)
    struct NoAllocScope {
        NoAllocScope() { t_no_alloc = true; }
        ~NoAllocScope() { t_no_alloc = false; }
    } scope;
    // the counters read back must start clear: the array keeps the last
    // call's contents
    launch_fill_u8(reinterpret_cast<uint8_t *>(ws.host_cnt_dev), sizeof(HostCounters), 0, st);
    TGS_LAUNCHED("clear counters");
    const CamK ck = make_camk(cam);
    TGS_TRY(step_preprocess(sc, ws, ck, no_cull(0.2f, ws), st));
    const uint32_t *didx = nullptr, *vals = nullptr;
    TGS_TRY(step_scan(sc, ws, nullptr, TX, st, &didx));
    TGS_TRY(step_keys(sc, ws, TX, TY, nullptr, nullptr, didx, st, &vals));
    if (out->contrib) launch_fill_f32(out->contrib, (size_t)sc->n, 0.0f, st);
    BlendArgs a = blend_args(ws, cam, vals);
    set_blend_order(a, ws, sc);
    a.rgb = out->rgb;
    a.depth = out->depth;
    a.sigma = out->sigma;
    a.alpha = out->alpha;
    a.contrib = out->contrib;
    a.mark_mask = out->tile_mask;
    launch_blend(a, TX * TY, st, nullptr, nullptr);
    TGS_LAUNCHED("blend");
    FrameResult fr;
    bool overflow = false;
    TGS_TRY(step_wait_counters(ws, st, fr, &overflow));
    if (overflow)
        return fail(TGS_ERR_CAPACITY, "frame needs " + std::to_string(fr.K) +
                                          " Gaussian-tile keys; the allocation-free render holds " +
                                          std::to_string(ws.key_cap) + " at this size");
    out->frame_kind = TGS_FRAME_FULL;
    out->n_selected = TX * TY;
    out->n_survivors = (int32_t)fr.n_surv;
    out->n_newly_visible = 0;
    out->n_keys = fr.K;
    return TGS_OK;
}

tgs_status tgs_state_create(tgs_scene *scene, int32_t width, int32_t height,
                            const tgs_params *params, tgs_state **out) {
    g_err.clear();
    if (!scene || !out) return fail(TGS_ERR_INVALID_ARG, "scene and out must not be NULL");
    if (width < 1 || height < 1 || width > 16384 || height > 16384)
        return fail(TGS_ERR_INVALID_ARG, "image size must be within 1..16384");
    tgs_params p;
    tgs_params_default(&p);
    if (params) p = *params;
    TGS_TRY(check_params(&p));
    tgs_state *s = new (std::nothrow) tgs_state();
    if (!s) return fail(TGS_ERR_OUT_OF_MEMORY, "host allocation failed");
    s->scene = scene;
    s->W = width;
    s->H = height;
    s->TX = (width + 15) / 16;
    s->TY = (height + 15) / 16;
    s->p = p;
    s->Wg = (width + p.tgb_downscale - 1) / p.tgb_downscale;
    s->Hg = (height + p.tgb_downscale - 1) / p.tgb_downscale;
    const size_t px = (size_t)width * height, nt = (size_t)s->TX * s->TY;
    const size_t pg = (size_t)s->Wg * s->Hg;
    const size_t nn = (size_t)(scene->n > 0 ? scene->n : 1);
    tgs_status st = TGS_OK;
    if (st == TGS_OK) st = s->tgb_d.ensure(pg * 4);
    if (st == TGS_OK) st = s->tgb_s.ensure(pg * 4);
    if (st == TGS_OK) st = s->tab.ensure(3 * px * 4);
    if (st == TGS_OK) st = s->g_flag.ensure(nn);
    if (st == TGS_OK) st = s->fbox.ensure((4 + 4 * kAfcPartials) * sizeof(int));
    for (int b = 0; b < 2; ++b) {
        if (st == TGS_OK) st = s->dmin[b].ensure(pg * 4);
        if (st == TGS_OK) st = s->smax[b].ensure(pg * 4);
    }
    if (st == TGS_OK) st = s->dfill.ensure(pg * 4);
    if (st == TGS_OK) st = s->uv.ensure(pg * 8);
    if (st == TGS_OK) st = s->um.ensure(nt);
    if (st == TGS_OK) st = s->oc.ensure(nt);
    if (st == TGS_OK) st = s->ws.prepare(scene->n, width, height);
    if (st != TGS_OK) {
        delete s;
        return st;
    }
    *out = s;
    return TGS_OK;
}

tgs_status tgs_state_reset(tgs_state *s) {
    g_err.clear();
    if (!s) return fail(TGS_ERR_INVALID_ARG, "state is NULL");
    s->frame_index = s->since_true = s->since_ref = s->force_pseudo = s->has_ref = 0;
    return TGS_OK;
}

void tgs_state_free(tgs_state *s) { delete s; }

tgs_status tgs_render_temporal(tgs_state *s, const tgs_camera *cam, tgs_frame_out *out,
                               void *stream) {
    g_err.clear();
    if (!s || !out || !out->rgb) return fail(TGS_ERR_INVALID_ARG, "state, out and out->rgb are required");
    TGS_TRY(check_camera(cam));
    if (cam->width != s->W || cam->height != s->H)
        return fail(TGS_ERR_STATE_MISMATCH, "camera size differs from the state's");
    hipStream_t st = (hipStream_t)stream;
    tgs_scene *sc = s->scene;
    const int W = s->W, H = s->H, TX = s->TX, TY = s->TY, nt = TX * TY;
    Workspace &ws = s->ws;
    TGS_TRY(ws.prepare(sc->n, W, H));
    const CamK ck = make_camk(cam);
    const tgs_params &p = s->p;

    // schedule (Sec. III-B, III-E, IV-B)
    int kind;
    if (!s->has_ref || s->frame_index == 0 || s->since_true >= p.lambda_tdc)
        kind = TGS_FRAME_TRUE_REF;
    else if (s->force_pseudo || s->since_ref >= p.lambda_sr)
        kind = TGS_FRAME_PSEUDO_REF;
    else
        kind = TGS_FRAME_TGS;

    const int passes = tile_sort_passes(TX, TY);
    TGS_TRY(ws.ensure_keys(ws.key_cap ? ws.key_cap : 4 * (size_t)sc->n + 65536, passes));
    FrameResult fr;
    for (;;) {
        const uint32_t *vals = nullptr;
        if (kind == TGS_FRAME_TGS) {
            // full-resolution view pair (occluded tiles, stitching) and the
            // same on the geometry buffer's grid (warp, fill, correspondences)
            WarpK w{};
            relative_pose(s->ref_w2c, cam->world_to_cam, w.M, w.Minv);
            for (int k = 0; k < 4; ++k) w.kref[k] = s->ref_intr[k];
            w.kcur[0] = cam->fx;
            w.kcur[1] = cam->fy;
            w.kcur[2] = cam->cx;
            w.kcur[3] = cam->cy;
            w.z_near = p.z_near;
            w.W = W;
            w.H = H;
            w.TX = TX;
            w.TY = TY;
            w.tp = kTile;
            const bool half = p.tgb_downscale == 2;
            WarpK wg = w;
            if (half) {
                // cell (i, j) = pixels {2i, 2i+1} x {2j, 2j+1}: f / 2, (c - 1/2) / 2
                for (int k = 0; k < 2; ++k) {
                    wg.kref[k] = w.kref[k] * 0.5f;
                    wg.kcur[k] = w.kcur[k] * 0.5f;
                    wg.kref[2 + k] = (w.kref[2 + k] - 0.5f) * 0.5f;
                    wg.kcur[2 + k] = (w.kcur[2 + k] - 0.5f) * 0.5f;
                }
                wg.W = s->Wg;
                wg.H = s->Hg;
                wg.tp = kTile / 2;
            }
            const int wb = s->warp_next;
            float *dmin = s->dmin[wb].as<float>(), *smax = s->smax[wb].as<float>();
            {
                ProfScope ps(TGS_PROF_WARP, st);
                if (!s->warp_clean) launch_temporal_init(s->Wg * s->Hg, dmin, smax, st);
                s->warp_clean = false;
                launch_forward_warp(wg, s->tgb_d.as<float>(), s->tgb_s.as<float>(), dmin, smax, st);
                TGS_LAUNCHED("warp");
            }
            // depth fill and backward query; it also clears the occluded-tile
            // flags of this frame and resets the other warp pair for the next
            // one.  Run by the preprocess launch (blocks past the Gaussians'),
            // or by a launch of its own on the half-resolution grid.
            FillK fq{};
            fq.w = wg;
            fq.dmin = dmin;
            fq.dfill = s->dfill.as<float>();
            fq.uv = s->uv.as<float2>();
            fq.um = s->um.as<uint8_t>();
            fq.oc = s->oc.as<uint8_t>();
            fq.dmin_next = s->dmin[wb ^ 1].as<float>();
            fq.smax_next = s->smax[wb ^ 1].as<float>();
            s->warp_last = wb;
            s->warp_next = wb ^ 1;
            s->warp_clean = true;
            CullK cull = no_cull(p.z_near, ws);
            cull.afc = p.enable_afc;
            cull.fbox = s->fbox.as<int>();
            cull.toc = p.enable_toc;
            cull.dmin = dmin;
            cull.smax = smax;
            cull.g_rendered = s->g_flag.as<uint8_t>();
            cull.lambda1 = p.lambda1;
            cull.lambda2 = p.lambda2;
            cull.tgb_shift = half ? 1 : 0;
            cull.tgb_w = s->Wg;
            TGS_TRY(step_preprocess(sc, ws, ck, cull, st, &fq));
            {
                ProfScope ps(TGS_PROF_OCCLUDED, st);
                launch_occluded(w, sc->n, ws.status.as<uint8_t>(), ws.g.as<float4>(),
                                ws.rect.as<ushort4>(), s->oc.as<uint8_t>(), st);
                TGS_LAUNCHED("occluded tiles");
            }
            const int mode = (!p.enable_sr || p.force_all_dirty) ? 1 : 0;
            {
                ProfScope ps(TGS_PROF_SELECT, st);
                launch_select(TX, TY, mode, s->oc.as<uint8_t>(), s->um.as<uint8_t>(),
                              ws.sel.as<uint8_t>(), ws.sel_list.as<int>(), ws.rowpre.as<uint32_t>(),
                              ws.sel_cols.as<int>(), out->tile_mask, ws.cnt.as<Counters>(), st);
                TGS_LAUNCHED("tile selection");
            }
            const uint32_t *didx = nullptr;
            TGS_TRY(step_scan(sc, ws, ws.rowpre.as<uint32_t>(), TX, st, &didx));
            TGS_TRY(step_keys(sc, ws, TX, TY, ws.rowpre.as<uint32_t>(), ws.sel_cols.as<int>(), didx,
                              st, &vals));
            BlendArgs a = blend_args(ws, cam, vals);
            set_blend_order(a, ws, sc);
            a.n_tiles_dev = &ws.cnt.as<Counters>()->n_selected;
            a.rgb = out->rgb;
            a.pairs = g_prof.pairs(TGS_PROF_BLEND_TGS);
        a.hits = g_prof.hits(TGS_PROF_BLEND_TGS);
            // the blocks past the selected tiles stitch the others (Eq. 4)
            a.stitch_list = ws.sel_list.as<int>();
            a.stitch_mode = half ? 2 : 1;
            a.stitch_wg = s->Wg;
            a.stitch_tab = s->tab.as<float>();
            a.stitch_uv = s->uv.as<float2>();
            a.stitch_dfill = s->dfill.as<float>();
            a.sw = w;
            {
                hipEvent_t ev0, ev1;
                g_prof.kernel_events(TGS_PROF_BLEND_TGS, &ev0, &ev1);
                launch_blend(a, nt, st, ev0, ev1);
                TGS_LAUNCHED("blend and stitch");
            }
        } else {
            CullK cull = no_cull(p.z_near, ws);
            cull.afc = (kind == TGS_FRAME_PSEUDO_REF && p.enable_afc) ? 1 : 0;
            cull.fbox = s->fbox.as<int>();
            // the preprocess clears the temporal Gaussian buffer the blend fills
            cull.clear_flag = s->g_flag.as<uint8_t>();
            TGS_TRY(step_preprocess(sc, ws, ck, cull, st));
            const uint32_t *didx = nullptr;
            TGS_TRY(step_scan(sc, ws, nullptr, TX, st, &didx));
            TGS_TRY(step_keys(sc, ws, TX, TY, nullptr, nullptr, didx, st, &vals));
            if (out->contrib) launch_fill_f32(out->contrib, (size_t)sc->n, 0.0f, st);
            BlendArgs a = blend_args(ws, cam, vals);
            set_blend_order(a, ws, sc);
            a.rgb = out->rgb;
            a.tab = s->tab.as<float>();
            a.depth = out->depth;
            a.sigma = out->sigma;
            a.alpha = out->alpha;
            a.empty_depth = p.empty_far ? kZFar : kNoHit;
            if (p.tgb_downscale == 2) {
                a.tgbh_depth = s->tgb_d.as<float>();   // pooled over 2x2 blocks
                a.tgbh_sigma = s->tgb_s.as<float>();
            } else {
                a.tgb_depth = s->tgb_d.as<float>();
                a.tgb_sigma = s->tgb_s.as<float>();
            }
            a.g_flag = s->g_flag.as<uint8_t>();
            a.contrib = out->contrib;
            // every tile is rendered: the blend marks them
            a.mark_sel = ws.sel.as<uint8_t>();
            a.mark_mask = out->tile_mask;
            a.pairs = g_prof.pairs(TGS_PROF_BLEND_REF);
            a.hits = g_prof.hits(TGS_PROF_BLEND_REF);
            {
                hipEvent_t ev0, ev1;
                g_prof.kernel_events(TGS_PROF_BLEND_REF, &ev0, &ev1);
                launch_blend(a, nt, st, ev0, ev1);
                TGS_LAUNCHED("blend");
            }
            {
                ProfScope ps(TGS_PROF_CAPTURE, st);
                if (kind == TGS_FRAME_TRUE_REF) {
                    launch_afc_bounds(sc->n, s->g_flag.as<uint8_t>(), ws.g.as<float4>(), W, H,
                                      s->fbox.as<int>(), st);
                    TGS_LAUNCHED("adaptive frustum");
                }
            }
        }
        bool overflow = false;
        TGS_TRY(step_wait_counters(ws, st, fr, &overflow));
        ws.recent_K[kind == TGS_FRAME_TGS ? 1 : 0] = fr.K;
        if (!overflow) break;
        TGS_TRY(grow_after_overflow(ws, fr, passes, st));
    }
    if (kind != TGS_FRAME_TGS) {
        memcpy(s->ref_w2c, cam->world_to_cam, sizeof(s->ref_w2c));
        s->ref_intr[0] = cam->fx;
        s->ref_intr[1] = cam->fy;
        s->ref_intr[2] = cam->cx;
        s->ref_intr[3] = cam->cy;
        s->has_ref = 1;
        fr.n_sel = (uint32_t)nt;
    }

    // counters (Sec. III-B) and adaptive reference insertion (Sec. III-E)
    s->frame_index += 1;
    if (kind == TGS_FRAME_TRUE_REF) {
        s->since_true = 1;
        s->since_ref = 1;
        s->force_pseudo = 0;
    } else if (kind == TGS_FRAME_PSEUDO_REF) {
        s->since_true += 1;
        s->since_ref = 1;
        s->force_pseudo = 0;
    } else {
        s->since_true += 1;
        s->since_ref += 1;
        if (p.enable_sr) s->force_pseudo = (double)fr.n_sel > (double)p.eta * (double)nt ? 1 : 0;
    }
    out->frame_kind = kind;
    out->n_selected = (int32_t)fr.n_sel;
    out->n_survivors = (int32_t)fr.n_surv;
    out->n_newly_visible = kind == TGS_FRAME_TGS ? (int32_t)fr.n_newly : 0;
    out->n_keys = fr.K;
    return TGS_OK;
}

tgs_status tgs_state_export(const tgs_state *s, void *host, size_t *nbytes) {
    g_err.clear();
    if (!s || !nbytes) return fail(TGS_ERR_INVALID_ARG, "state and nbytes must not be NULL");
    const size_t px = (size_t)s->W * s->H, pg = (size_t)s->Wg * s->Hg, n = (size_t)s->scene->n;
    const size_t need = sizeof(tgs_state_header) + (2 * pg + 3 * px) * sizeof(float) + n;
    if (!host) {
        *nbytes = need;
        return TGS_OK;
    }
    if (*nbytes < need) return fail(TGS_ERR_INVALID_ARG, "export buffer too small");
    TGS_HIP(hipDeviceSynchronize());
    tgs_state_header h{};
    h.magic = 0x54475331u;
    h.width = s->W;
    h.height = s->H;
    h.n = s->scene->n;
    h.frame_index = s->frame_index;
    h.since_true_ref = s->since_true;
    h.since_ref = s->since_ref;
    h.force_pseudo = s->force_pseudo;
    h.has_reference = s->has_ref;
    int fb[4];
    TGS_HIP(hipMemcpy(fb, s->fbox.p, sizeof(fb), hipMemcpyDeviceToHost));
    for (int k = 0; k < 4; ++k) {
        const int i = fb[k] >= 0 ? fb[k] : fb[k] ^ 0x7fffffff;
        memcpy(&h.fbox[k], &i, 4);
    }
    memcpy(h.ref_world_to_cam, s->ref_w2c, sizeof(h.ref_world_to_cam));
    memcpy(h.ref_intrinsics, s->ref_intr, sizeof(h.ref_intrinsics));
    h.tgb_width = s->Wg;
    h.tgb_height = s->Hg;
    char *dst = static_cast<char *>(host);
    memcpy(dst, &h, sizeof(h));
    dst += sizeof(h);
    TGS_HIP(hipMemcpy(dst, s->tgb_d.p, pg * 4, hipMemcpyDeviceToHost));
    dst += pg * 4;
    TGS_HIP(hipMemcpy(dst, s->tgb_s.p, pg * 4, hipMemcpyDeviceToHost));
    dst += pg * 4;
    TGS_HIP(hipMemcpy(dst, s->tab.p, 3 * px * 4, hipMemcpyDeviceToHost));
    dst += 3 * px * 4;
    if (n) TGS_HIP(hipMemcpy(dst, s->g_flag.p, n, hipMemcpyDeviceToHost));
    *nbytes = need;
    return TGS_OK;
}

tgs_status tgs_state_import(tgs_state *s, const void *host, size_t nbytes) {
    g_err.clear();
    if (!s || !host) return fail(TGS_ERR_INVALID_ARG, "state and host must not be NULL");
    const size_t px = (size_t)s->W * s->H, pg = (size_t)s->Wg * s->Hg, n = (size_t)s->scene->n;
    const size_t need = sizeof(tgs_state_header) + (2 * pg + 3 * px) * sizeof(float) + n;
    if (nbytes != need) return fail(TGS_ERR_INVALID_ARG, "blob size does not match the state");
    tgs_state_header h;
    memcpy(&h, host, sizeof(h));
    if (h.magic != 0x54475331u) return fail(TGS_ERR_INVALID_ARG, "bad blob magic");
    if (h.width != s->W || h.height != s->H || h.n != s->scene->n || h.tgb_width != s->Wg ||
        h.tgb_height != s->Hg)
        return fail(TGS_ERR_STATE_MISMATCH, "blob sizes differ from the state's");
    TGS_HIP(hipDeviceSynchronize());
    const char *src = static_cast<const char *>(host) + sizeof(h);
    TGS_HIP(hipMemcpy(s->tgb_d.p, src, pg * 4, hipMemcpyHostToDevice));
    src += pg * 4;
    TGS_HIP(hipMemcpy(s->tgb_s.p, src, pg * 4, hipMemcpyHostToDevice));
    src += pg * 4;
    TGS_HIP(hipMemcpy(s->tab.p, src, 3 * px * 4, hipMemcpyHostToDevice));
    src += 3 * px * 4;
    if (n) TGS_HIP(hipMemcpy(s->g_flag.p, src, n, hipMemcpyHostToDevice));
    int fb[4];
    for (int k = 0; k < 4; ++k) {
        int i;
        memcpy(&i, &h.fbox[k], 4);
        fb[k] = i >= 0 ? i : i ^ 0x7fffffff;
    }
    TGS_HIP(hipMemcpy(s->fbox.p, fb, sizeof(fb), hipMemcpyHostToDevice));
    s->frame_index = h.frame_index;
    s->since_true = h.since_true_ref;
    s->since_ref = h.since_ref;
    s->force_pseudo = h.force_pseudo;
    s->has_ref = h.has_reference;
    memcpy(s->ref_w2c, h.ref_world_to_cam, sizeof(s->ref_w2c));
    memcpy(s->ref_intr, h.ref_intrinsics, sizeof(s->ref_intr));
    return TGS_OK;
}

tgs_status tgs_debug_dump(const tgs_scene *scene, const tgs_state *state, int32_t what, void *host,
                          size_t *nbytes) {
    g_err.clear();
    if (!nbytes || (!scene && !state))
        return fail(TGS_ERR_INVALID_ARG, "nbytes and one of scene/state are required");
    const Workspace &ws = state ? state->ws : scene->ws;
    const int n = state ? state->scene->n : scene->n;
    const int W = state ? state->W : scene->last_W, H = state ? state->H : scene->last_H;
    const size_t nt = (size_t)((W + 15) / 16) * ((H + 15) / 16);
    const size_t pg = state ? (size_t)state->Wg * state->Hg : 0;   // geometry buffer grid
    const void *src = nullptr;
    size_t size = 0;
    if (!ws.has_frame) return fail(TGS_ERR_INVALID_ARG, "no frame has been rendered yet");
    switch (what) {
        case TGS_DUMP_SORTED_VALUES: src = ws.last_vals; size = (size_t)ws.last_K * 4; break;
        case TGS_DUMP_SORTED_KEYS: src = ws.last_keys; size = (size_t)ws.last_K * 4; break;
        case TGS_DUMP_TILE_RANGES: src = ws.ranges.p; size = nt * 8; break;
        case TGS_DUMP_RECTS: src = ws.rect.p; size = (size_t)n * 8; break;
        case TGS_DUMP_STATUS: src = ws.status.p; size = (size_t)n; break;
        case TGS_DUMP_SELECTED: src = ws.sel.p; size = nt; break;
        case TGS_DUMP_RECORDS: size = (size_t)n * 48; break;
        default:
            if (!state) return fail(TGS_ERR_INVALID_ARG, "this buffer exists only for a state");
            switch (what) {
                case TGS_DUMP_WARP_DEPTH: src = state->dmin[state->warp_last].p; size = pg * 4; break;
                case TGS_DUMP_WARP_SIGMA: src = state->smax[state->warp_last].p; size = pg * 4; break;
                case TGS_DUMP_FILLED_DEPTH: src = state->dfill.p; size = pg * 4; break;
                case TGS_DUMP_CORRESPONDENCE: src = state->uv.p; size = pg * 8; break;
                case TGS_DUMP_UNMATCHED: src = state->um.p; size = nt; break;
                case TGS_DUMP_OCCLUDED: src = state->oc.p; size = nt; break;
                default: return fail(TGS_ERR_INVALID_ARG, "unknown dump id");
            }
    }
    if (!host) {
        *nbytes = size;
        return TGS_OK;
    }
    if (*nbytes < size) return fail(TGS_ERR_INVALID_ARG, "dump buffer too small");
    TGS_HIP(hipDeviceSynchronize());
    if (what == TGS_DUMP_RECORDS) {
        float *dst = static_cast<float *>(host);
        std::vector<float4> tmp((size_t)n * 4);
        if (n) TGS_HIP(hipMemcpy(tmp.data(), ws.g.p, (size_t)n * 64, hipMemcpyDeviceToHost));
        for (int i = 0; i < n; ++i) {
            // (u, v, conic a, b), (conic c, opacity, depth, 0), (r, g, b, 0)
            memcpy(dst + (size_t)i * 12, &tmp[4 * (size_t)i], 48);
            dst[(size_t)i * 12 + 7] = 0.0f;
            dst[(size_t)i * 12 + 11] = 0.0f;
        }
    } else if (size) {
        TGS_HIP(hipMemcpy(host, src, size, hipMemcpyDeviceToHost));
    }
    *nbytes = size;
    return TGS_OK;
}

tgs_status tgs_debug_dump_range(const tgs_scene *scene, const tgs_state *state, int32_t what,
                                size_t first, size_t count, void *host) {
    g_err.clear();
    if (!scene && !state) return fail(TGS_ERR_INVALID_ARG, "one of scene/state is required");
    if (what != TGS_DUMP_SORTED_VALUES && what != TGS_DUMP_SORTED_KEYS)
        return fail(TGS_ERR_INVALID_ARG, "ranges exist for the sorted values and keys only");
    if (!host && count > 0) return fail(TGS_ERR_INVALID_ARG, "host is NULL");
    const Workspace &ws = state ? state->ws : scene->ws;
    if (!ws.has_frame) return fail(TGS_ERR_INVALID_ARG, "no frame has been rendered yet");
    if (first > (size_t)ws.last_K || count > (size_t)ws.last_K - first)
        return fail(TGS_ERR_INVALID_ARG, "range past the frame's keys");
    if (count == 0) return TGS_OK;
    const uint32_t *src = what == TGS_DUMP_SORTED_VALUES ? ws.last_vals : ws.last_keys;
    TGS_HIP(hipDeviceSynchronize());
    TGS_HIP(hipMemcpy(host, src + first, count * sizeof(uint32_t), hipMemcpyDeviceToHost));
    return TGS_OK;
}

}  // extern "C"
