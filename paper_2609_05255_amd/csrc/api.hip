// C-ABI entry points of gsraster (declared in include/gsraster.h): argument
// validation on the host, workspace layout, kernel launches on the caller's
// stream, error reporting, and optional per-kernel timing with HIP events.
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <mutex>
#include <string>
#include <vector>

#include "gs_internal.h"

using namespace gsr;

namespace {

thread_local std::string g_error;

gs_status fail(gs_status st, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
gs_status fail(gs_status st, const char* fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_error = buf;
    return st;
}

gs_status ok()
{
    g_error.clear();
    return GS_OK;
}

#define GS_HIP(expr)                                                                            \
    do {                                                                                        \
        hipError_t e_ = (expr);                                                                 \
        if (e_ != hipSuccess)                                                                   \
            return fail(GS_ERR_DEVICE, "%s failed: %s", #expr, hipGetErrorString(e_));          \
    } while (0)

#define GS_CHECK(cond, ...)                                  \
    do {                                                     \
        if (!(cond)) return fail(GS_ERR_INVALID_ARG, __VA_ARGS__); \
    } while (0)

gs_status check_camera(const gs_camera* c)
{
    GS_CHECK(c != nullptr, "camera is NULL");
    GS_CHECK(c->width > 0 && c->height > 0, "image size %dx%d must be positive", c->width, c->height);
    GS_CHECK((int64_t)c->width * c->height <= ((int64_t)1 << 31), "image of %dx%d pixels is too large",
             c->width, c->height);
    GS_CHECK((c->width + kTile - 1) / kTile <= 32767 && (c->height + kTile - 1) / kTile <= 32767,
             "tile grid exceeds the 16-bit rectangle fields");
    GS_CHECK(c->fx > 0.f && c->fy > 0.f, "focal lengths must be positive");
    GS_CHECK(c->near_plane >= 0.f, "near plane must be >= 0");
    for (int i = 0; i < 12; ++i) GS_CHECK(c->viewmat[i] == c->viewmat[i], "view matrix holds NaN");
    return GS_OK;
}

gs_status check_gaussians(const gs_gaussians* g)
{
    GS_CHECK(g != nullptr, "gaussians is NULL");
    GS_CHECK(g->n >= 0 && g->n < ((int64_t)1 << 31), "n = %lld out of range [0, 2^31)", (long long)g->n);
    if (g->n > 0)
        GS_CHECK(g->means && g->log_scales && g->quats && g->opacity_logits, "a Gaussian parameter array is NULL");
    return GS_OK;
}

gs_status check_appearance(const gs_appearance* a, int64_t n)
{
    GS_CHECK(a != nullptr, "appearance is NULL");
    if (a->kind == GS_APP_SH3) {
        GS_CHECK(a->sh_degree >= 0 && a->sh_degree <= 3, "sh_degree %d outside 0..3", a->sh_degree);
        GS_CHECK(n == 0 || a->sh != nullptr, "sh is NULL");
    } else if (a->kind == GS_APP_LATENT_MLP) {
        GS_CHECK(n == 0 || (a->latent != nullptr && a->mlp_w != nullptr), "latent or mlp_w is NULL");
    } else if (a->kind == GS_APP_NEURAL) {
        GS_CHECK(a->sh_degree >= 0 && a->sh_degree <= 3, "sh_degree %d outside 0..3", a->sh_degree);
        GS_CHECK(a->neural_layers >= 0 && a->neural_layers <= 3, "neural_layers %d outside 0..3", a->neural_layers);
        GS_CHECK(a->neural_raw16 == 0 || a->neural_raw16 == 1, "neural_raw16 must be 0 or 1");
        GS_CHECK(a->neural_width == 0 || a->neural_width == 16 || a->neural_width == 32,
                 "neural_width %d: 16 or 32 neurons per layer", a->neural_width);
        if (a->neural_width == 32 && ((a->neural_layers != 0 && a->neural_layers != 2) || a->neural_raw16))
            return fail(GS_ERR_UNSUPPORTED, "32 neurons per layer are built for the table's 32-32-32-3 decoder only");
        GS_CHECK(n == 0 || a->base_color != nullptr, "base_color is NULL");
        GS_CHECK(n == 0 || a->sh_degree == 0 || (a->features != nullptr && a->mlp_w != nullptr),
                 "features or mlp_w is NULL");
    } else if (a->kind == GS_APP_NEURAL_FOLDED) {
        GS_CHECK(a->sh_degree >= 0 && a->sh_degree <= 3, "sh_degree %d outside 0..3", a->sh_degree);
        GS_CHECK((a->neural_layers == 0 || a->neural_layers == 2) && (a->neural_width == 0 || a->neural_width == 16) &&
                     a->neural_raw16 == 0,
                 "the folded form takes the paper's default decoder only");
        GS_CHECK(n == 0 || a->base_color != nullptr, "base_color is NULL");
        GS_CHECK(n == 0 || a->sh_degree == 0 || (a->preact != nullptr && a->mlp_w != nullptr),
                 "preact or mlp_w is NULL");
        GS_CHECK(((uintptr_t)a->preact & 7) == 0, "preact must be 8-byte aligned");
    } else if (a->kind == GS_APP_NASG || a->kind == GS_APP_NASGABOR) {
        GS_CHECK(a->sh_degree >= 0 && a->sh_degree <= 3, "sh_degree %d outside 0..3", a->sh_degree);
        GS_CHECK(n == 0 || a->base_color != nullptr, "base_color is NULL");
        GS_CHECK(n == 0 || a->sh_degree == 0 || a->lobes != nullptr, "lobes is NULL");
    } else {
        return fail(GS_ERR_INVALID_ARG, "unknown appearance kind %d", a->kind);
    }
    return GS_OK;
}

gs_status check_pre(const gs_preprocessed* p, int64_t n)
{
    GS_CHECK(p != nullptr, "preprocessed is NULL");
    GS_CHECK(p->num_pairs != nullptr, "num_pairs is NULL");
    if (n > 0) GS_CHECK(p->splats && p->tiles_touched && p->depth_key, "a preprocess output array is NULL");
    return GS_OK;
}

gs_status check_workspace(void* ws, size_t bytes, const Workspace& need)
{
    GS_CHECK(ws != nullptr || need.bytes == 0, "workspace is NULL");
    GS_CHECK(((uintptr_t)ws & 255) == 0, "workspace must be 256-byte aligned");
    if (bytes < need.bytes)
        return fail(GS_ERR_CAPACITY, "workspace of %zu bytes is too small: %zu needed", bytes, need.bytes);
    return GS_OK;
}

// ---- timing --------------------------------------------------------------------
struct TimedLaunch {
    int id;
    hipEvent_t a, b;
};

void resolve_pending(gs_timer* t);

}  // namespace

// A caller-owned timing context (gs_timer_create). The library itself keeps
// only the calling thread's pointer to the timer attached to it.
struct gs_timer {
    std::vector<hipEvent_t> free_events;
    std::vector<TimedLaunch> pending;
    std::vector<TimedLaunch> open;
    double ms[GS_KERNEL_COUNT];
    int64_t launches[GS_KERNEL_COUNT];
};

namespace {

thread_local gs_timer* t_timer = nullptr;

void resolve_pending(gs_timer* t)
{
    for (auto& l : t->pending) {
        float ms = 0.f;
        (void)hipEventSynchronize(l.b);
        if (hipEventElapsedTime(&ms, l.a, l.b) == hipSuccess) {
            t->ms[l.id] += ms;
            t->launches[l.id] += 1;
        }
        t->free_events.push_back(l.a);
        t->free_events.push_back(l.b);
    }
    t->pending.clear();
}

const char* const kKernelNames[GS_KERNEL_COUNT] = {
    "preprocess", "pair_count", "depth_sort", "entry_offsets", "block_entries", "block_sort", "tile_lists",
    "blend_fwd", "bwd_prep", "blend_bwd", "preprocess_bwd", "mlp_reduce", "adam", "neural_fold"};

}  // namespace

namespace gsr {

void timing_begin(int id, hipStream_t s)
{
    gs_timer* t = t_timer;
    if (!t) return;
    if (t->free_events.size() < 2) resolve_pending(t);
    if (t->free_events.size() < 2) return;
    TimedLaunch l;
    l.id = id;
    l.a = t->free_events.back();
    t->free_events.pop_back();
    l.b = t->free_events.back();
    t->free_events.pop_back();
    (void)hipEventRecord(l.a, s);
    t->open.push_back(l);
}

void timing_end(int id, hipStream_t s)
{
    gs_timer* t = t_timer;
    if (!t) return;
    for (size_t k = t->open.size(); k-- > 0;) {
        if (t->open[k].id == id) {
            (void)hipEventRecord(t->open[k].b, s);
            t->pending.push_back(t->open[k]);
            t->open.erase(t->open.begin() + (long)k);
            return;
        }
    }
}

Workspace layout_workspace(void* base, int64_t n, uint64_t capacity, int32_t kind, const Cam* cam)
{
    Workspace w;
    memset(&w, 0, sizeof(w));
    size_t off = 0;
    auto take = [&](size_t bytes) -> char* {
        char* p = base ? static_cast<char*>(base) + off : nullptr;
        off += align_up(bytes, 256);
        return p;
    };
    const int64_t nn = n > 0 ? n : 1;
    const int64_t cap = capacity > 0 ? (int64_t)capacity : 1;
    const int64_t n_blocks = cam ? (int64_t)blocks_x_of(*cam) * blocks_y_of(*cam) : 1;
    const int64_t segs = cam ? segment_bound(*cam, (uint64_t)cap) : 1;
    w.block_pairs = (uint32_t*)take(sizeof(uint32_t) * pair_count_slots(nn));
    w.keys_a = (uint32_t*)take(sizeof(uint32_t) * nn);
    w.keys_b = (uint32_t*)take(sizeof(uint32_t) * nn);
    w.vals_a = (uint32_t*)take(sizeof(uint32_t) * nn);
    w.vals_b = (uint32_t*)take(sizeof(uint32_t) * nn);
    // the depth sort's 8-bit digits over n keys; the block sort's up to 9-bit
    // digits over up to `capacity` entries
    w.hist = (uint32_t*)take(sizeof(uint32_t) * std::max(kRadix * div_up(nn, kSortTile),
                                                         2 * kRadix * div_up(cap, kBlock * kBlockSortItems)));
    w.digit_tot = (uint32_t*)take(sizeof(uint32_t) * kRadix * 4);
    w.scan_part = (uint32_t*)take(sizeof(uint32_t) * (div_up(nn, kDupChunk) + 1));
    w.sorted_rect = (uint2*)take(sizeof(uint2) * nn);
    w.entry_count = (uint64_t*)take(sizeof(uint64_t));
    w.entry_keys_a = (uint32_t*)take(sizeof(uint32_t) * cap);
    w.entry_vals_a = (uint32_t*)take(sizeof(uint32_t) * cap);
    w.entry_keys_b = (uint32_t*)take(sizeof(uint32_t) * cap);
    w.entry_vals_b = (uint32_t*)take(sizeof(uint32_t) * cap);
    w.block_ranges = (uint32_t*)take(sizeof(uint32_t) * 2 * n_blocks);
    w.seg_base = (uint32_t*)take(sizeof(uint32_t) * (n_blocks + 1));
    w.seg_block = (uint32_t*)take(sizeof(uint32_t) * segs);
    w.seg_cnt = (uint32_t*)take(sizeof(uint32_t) * 16 * 4 * segs);
    w.list_counters = (uint32_t*)take(sizeof(uint32_t) * 2);
    w.acc = (float*)take(sizeof(float) * kAccStride * nn);
    const int64_t n_tiles = cam ? (int64_t)cam->tiles_x * cam->tiles_y : 1;
    w.walk_cls = (uint32_t*)take(sizeof(uint32_t) * n_tiles);
    w.tile_order = (uint32_t*)take(sizeof(uint32_t) * n_tiles);
    w.mlp_part = (float*)take(kind == GS_APP_LATENT_MLP ? sizeof(float) * GS_MLP_WEIGHTS * kMlpPartials
                              : kind == GS_APP_NEURAL ? sizeof(float) * GS_NEURAL_MAX_WEIGHTS * kMlpPartials : 0);
    w.bytes = off;
    return w;
}

}  // namespace gsr

extern "C" {

const char* gs_last_error(void) { return g_error.c_str(); }

const char* gs_version(void) { return "gsraster 0.1.0 (gfx950)"; }

gs_status gs_adam_step(const gs_adam_tensor* tensors, int32_t count, float beta1, float eps, int64_t step,
                       void* stream)
{
    GS_CHECK(tensors != nullptr, "tensors is NULL");
    GS_CHECK(count >= 1 && count <= GS_ADAM_MAX_TENSORS, "count %d outside [1, %d]", count, GS_ADAM_MAX_TENSORS);
    GS_CHECK(step >= 1, "step %lld must be at least 1", (long long)step);
    GS_CHECK(beta1 >= 0.f && beta1 < 1.f, "beta1 must lie in [0, 1)");
    GS_CHECK(eps > 0.f, "eps must be positive");
    int64_t rows = 0;
    for (int k = 0; k < count; ++k) {
        const gs_adam_tensor& t = tensors[k];
        GS_CHECK(t.rows >= 1, "tensor %d: rows must be positive", k);
        GS_CHECK(t.n >= 0 && t.n < ((int64_t)1 << 31), "tensor %d: n out of range", k);
        GS_CHECK(t.beta2 >= 0.f && t.beta2 < 1.f, "tensor %d: beta2 must lie in [0, 1)", k);
        GS_CHECK(t.lr != nullptr, "tensor %d: lr is NULL", k);
        GS_CHECK(t.n == 0 || (t.param && t.grad && t.exp_avg && t.exp_avg_sq), "tensor %d: a buffer is NULL", k);
        rows += t.rows;
    }
    GS_CHECK(rows <= GS_ADAM_MAX_ROWS, "%lld rows in total exceed %d", (long long)rows, GS_ADAM_MAX_ROWS);
    hipStream_t s = static_cast<hipStream_t>(stream);
    timing_begin(GS_KERNEL_ADAM, s);
    GS_HIP(launch_adam(tensors, count, beta1, eps, step, s));
    timing_end(GS_KERNEL_ADAM, s);
    return ok();
}

const char* gs_kernel_name(int32_t id) { return (id >= 0 && id < GS_KERNEL_COUNT) ? kKernelNames[id] : "unknown"; }

gs_status gs_workspace_size(int64_t n, int32_t width, int32_t height, uint64_t capacity, int32_t kind, size_t* bytes)
{
    GS_CHECK(bytes != nullptr, "bytes is NULL");
    GS_CHECK(n >= 0 && n < ((int64_t)1 << 31), "n out of range");
    GS_CHECK(width > 0 && height > 0, "image size must be positive");
    GS_CHECK(capacity < ((uint64_t)1 << 32), "capacity must be below 2^32");
    GS_CHECK(kind >= GS_APP_SH3 && kind <= GS_APP_NASGABOR, "unknown appearance kind %d", kind);
    Cam grid;
    grid.tiles_x = (width + kTile - 1) / kTile;
    grid.tiles_y = (height + kTile - 1) / kTile;
    *bytes = layout_workspace(nullptr, n, capacity, kind, &grid).bytes;
    return ok();
}

}  // extern "C"

namespace {

// Checks and launches of gs_preprocess with the scratch memory already placed:
// `ws` needs only block_pairs (one tile sum per preprocess workgroup or wave,
// every one written before the pair count reads it).
gs_status preprocess_run(const gs_camera* cam, const gs_gaussians* g, const gs_appearance* app,
                         const gs_preprocessed* out, uint64_t* num_pairs_host, const Workspace& ws, hipStream_t s)
{
    const Cam c = make_cam(*cam);
    if (g->n > 0) {
        timing_begin(GS_KERNEL_PREPROCESS, s);
        int slots = 0;
        GS_HIP(launch_preprocess(c, *g, *app, *out, ws, &slots, s));
        timing_end(GS_KERNEL_PREPROCESS, s);
        timing_begin(GS_KERNEL_PAIR_COUNT, s);
        GS_HIP(launch_pair_count(slots, ws, out->num_pairs, s));
        timing_end(GS_KERNEL_PAIR_COUNT, s);
    } else {
        GS_HIP(launch_fill_u32(reinterpret_cast<uint32_t*>(out->num_pairs), 2, 0u, s));
    }
    if (num_pairs_host) {
        GS_HIP(hipMemcpyAsync(num_pairs_host, out->num_pairs, sizeof(uint64_t), hipMemcpyDeviceToHost, s));
        GS_HIP(hipStreamSynchronize(s));
    }
    return ok();
}

gs_status preprocess_checks(const gs_camera* cam, const gs_gaussians* g, const gs_appearance* app,
                            const gs_preprocessed* out)
{
    gs_status st;
    if ((st = check_camera(cam)) != GS_OK) return st;
    if ((st = check_gaussians(g)) != GS_OK) return st;
    if ((st = check_appearance(app, g->n)) != GS_OK) return st;
    return check_pre(out, g->n);
}

}  // namespace

// The preprocess's scratch for callers that cannot allocate: the tile sums
// (one per workgroup, or per wave of a decoder grid) of up to
// GS_NOALLOC_MAX_GAUSSIANS Gaussians (1 MiB), one copy per GPU for the life of
// the process. Host code reaches it only through the device address
// hipGetSymbolAddress returns for the current device.
static __device__ __align__(256) uint32_t scratch[GS_NOALLOC_MAX_GAUSSIANS / kWave];
static_assert(GS_NOALLOC_MAX_GAUSSIANS / kWave >= (GS_NOALLOC_MAX_GAUSSIANS / kBlock) * (kBlock / kWave),
              "the scratch holds pair_count_slots(GS_NOALLOC_MAX_GAUSSIANS) sums");

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
uint32_t* g_scratch_ptr[kMaxDevices] = {};

// The current device's address of `scratch`, looked up once per device.
gs_status scratch_of_current_device(uint32_t** ptr)
{
    int dev = -1;
    GS_HIP(hipGetDevice(&dev));
    GS_CHECK(dev >= 0 && dev < kMaxDevices, "device %d beyond the %d this library tracks", dev, kMaxDevices);
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || p == nullptr)
            return fail(GS_ERR_DEVICE, "hipGetSymbolAddress(scratch) failed on device %d: %s", dev,
                        hipGetErrorString(e));
        g_scratch_ptr[dev] = static_cast<uint32_t*>(p);
    }
    *ptr = g_scratch_ptr[dev];
    return GS_OK;
}

}  // namespace

extern "C" {

gs_status gs_preprocess(const gs_camera* cam, const gs_gaussians* g, const gs_appearance* app,
                        const gs_preprocessed* out, uint64_t* num_pairs_host, void* workspace, size_t workspace_bytes,
                        void* stream)
{
    gs_status st;
    if ((st = preprocess_checks(cam, g, app, out)) != GS_OK) return st;
    const Workspace need = layout_workspace(nullptr, g->n, 0, app->kind, nullptr);
    if ((st = check_workspace(workspace, workspace_bytes, need)) != GS_OK) return st;
    const Workspace ws = layout_workspace(workspace, g->n, 0, app->kind, nullptr);
    return preprocess_run(cam, g, app, out, num_pairs_host, ws, static_cast<hipStream_t>(stream));
}

gs_status gs_preprocess_noalloc(const gs_camera* cam, const gs_gaussians* g, const gs_appearance* app,
                                const gs_preprocessed* out, uint64_t* num_pairs_host, void* stream)
{
    gs_status st;
    if ((st = preprocess_checks(cam, g, app, out)) != GS_OK) return st;
    if (g->n > GS_NOALLOC_MAX_GAUSSIANS)
        return fail(GS_ERR_CAPACITY, "gs_preprocess_noalloc takes at most %d Gaussians, got %lld",
                    GS_NOALLOC_MAX_GAUSSIANS, (long long)g->n);
    uint32_t* scr = nullptr;
    if ((st = scratch_of_current_device(&scr)) != GS_OK) return st;
    Workspace ws;
    memset(&ws, 0, sizeof(ws));
    ws.block_pairs = scr;
    return preprocess_run(cam, g, app, out, num_pairs_host, ws, static_cast<hipStream_t>(stream));
}

gs_status gs_bin_sort(const gs_camera* cam, const gs_preprocessed* pre, int64_t n, uint64_t num_pairs,
                      uint64_t capacity, uint32_t* values, uint32_t* tile_ids, uint32_t* tile_ranges, void* workspace,
                      size_t workspace_bytes, void* stream)
{
    gs_status st;
    if ((st = check_camera(cam)) != GS_OK) return st;
    GS_CHECK(n >= 0 && n < ((int64_t)1 << 31), "n out of range");
    if ((st = check_pre(pre, n)) != GS_OK) return st;
    GS_CHECK(capacity < ((uint64_t)1 << 32), "capacity must be below 2^32");
    const bool on_device = num_pairs == GS_PAIRS_ON_DEVICE;
    if (!on_device && num_pairs > capacity)
        return fail(GS_ERR_CAPACITY, "%llu pairs exceed the capacity %llu", (unsigned long long)num_pairs,
                    (unsigned long long)capacity);
    GS_CHECK(tile_ranges != nullptr, "tile_ranges is NULL");
    GS_CHECK((on_device ? capacity : num_pairs) == 0 || values != nullptr, "values is NULL");
    const Cam c = make_cam(*cam);
    if (!blocks_supported(c))
        return fail(GS_ERR_UNSUPPORTED, "%dx%d tiles exceed 65536 blocks of 4x4 tiles", c.tiles_x, c.tiles_y);
    const Workspace need = layout_workspace(nullptr, n, capacity, GS_APP_SH3, &c);
    if ((st = check_workspace(workspace, workspace_bytes, need)) != GS_OK) return st;
    const Workspace ws = layout_workspace(workspace, n, capacity, GS_APP_SH3, &c);
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int n_tiles = c.tiles_x * c.tiles_y;
    if (n == 0 || (on_device ? capacity : num_pairs) == 0) {
        // no pair can be listed (in device mode a positive count then exceeds
        // the capacity; it stays in num_pairs for the caller to see)
        GS_HIP(launch_fill_u32(tile_ranges, 2 * (int64_t)n_tiles, 0u, s));
        return ok();
    }
    // device mode: the kernels read P from pre->num_pairs and size nothing by it
    const PairCount pairs = on_device ? PairCount{pre->num_pairs, capacity, capacity}
                                      : PairCount{nullptr, num_pairs, capacity};
    // block entries: at most one per pair, counted on the device (the grids
    // are sized for the capacity in both modes)
    const PairCount entries{ws.entry_count, capacity, capacity};
    const uint32_t* order = nullptr;
    BlockEntries ent{nullptr, nullptr};
    timing_begin(GS_KERNEL_DEPTH_SORT, s);
    GS_HIP(launch_depth_sort(n, pre->depth_key, pre->splats, ws, &order, s));
    timing_end(GS_KERNEL_DEPTH_SORT, s);
    timing_begin(GS_KERNEL_ENTRY_OFFSETS, s);
    GS_HIP(launch_entry_offsets(n, pairs, ws, s));
    timing_end(GS_KERNEL_ENTRY_OFFSETS, s);
    timing_begin(GS_KERNEL_BLOCK_ENTRIES, s);
    GS_HIP(launch_block_entries(c, n, order, entries, ws, s));
    timing_end(GS_KERNEL_BLOCK_ENTRIES, s);
    timing_begin(GS_KERNEL_BLOCK_SORT, s);
    GS_HIP(launch_block_sort(c, entries, ws, &ent, s));
    timing_end(GS_KERNEL_BLOCK_SORT, s);
    timing_begin(GS_KERNEL_TILE_LISTS, s);
    GS_HIP(launch_tile_lists(c, pairs, capacity, ws, ent, values, tile_ids, tile_ranges, s));
    timing_end(GS_KERNEL_TILE_LISTS, s);
    return ok();
}

gs_status gs_render_fwd(const gs_camera* cam, const gs_preprocessed* pre, int64_t n, const uint32_t* values,
                        const uint32_t* tile_ranges, float* image, float* final_T, uint32_t* n_contrib, void* stream)
{
    gs_status st;
    if ((st = check_camera(cam)) != GS_OK) return st;
    if ((st = check_pre(pre, n)) != GS_OK) return st;
    GS_CHECK(tile_ranges && image && final_T && n_contrib, "an output or range array is NULL");
    GS_CHECK(n == 0 || values != nullptr, "values is NULL");
    hipStream_t s = static_cast<hipStream_t>(stream);
    const Cam c = make_cam(*cam);
    timing_begin(GS_KERNEL_BLEND_FWD, s);
    GS_HIP(launch_blend_fwd(c, pre->splats, values, tile_ranges, image, final_T, n_contrib, s));
    timing_end(GS_KERNEL_BLEND_FWD, s);
    return ok();
}

gs_status gs_render_work(const gs_camera* cam, const gs_preprocessed* pre, int64_t n, const uint32_t* values,
                         const uint32_t* tile_ranges, uint64_t* counts, void* stream)
{
    gs_status st;
    if ((st = check_camera(cam)) != GS_OK) return st;
    if ((st = check_pre(pre, n)) != GS_OK) return st;
    GS_CHECK(tile_ranges && counts, "tile_ranges or counts is NULL");
    GS_CHECK(n == 0 || values != nullptr, "values is NULL");
    GS_CHECK(((uintptr_t)counts & 7) == 0, "counts must be 8-byte aligned");
    GS_HIP(launch_blend_count(make_cam(*cam), pre->splats, values, tile_ranges, counts,
                              static_cast<hipStream_t>(stream)));
    return ok();
}

}  // extern "C"

namespace {

// gs_render_bwd, and gs_render_bwd_adam when `adam` is not NULL (checked by the caller).
gs_status render_bwd(const gs_camera* cam, const gs_gaussians* g, const gs_appearance* app, const gs_preprocessed* pre,
                     const uint32_t* values, const uint32_t* tile_ranges, const float* final_T,
                     const uint32_t* n_contrib, const float* dL_dimage, const gs_grads* grads, void* workspace,
                     size_t workspace_bytes, void* stream, const gs_adam_tensor* adam, float beta1, float eps,
                     int64_t step)
{
    gs_status st;
    if ((st = check_camera(cam)) != GS_OK) return st;
    if ((st = check_gaussians(g)) != GS_OK) return st;
    if ((st = check_appearance(app, g->n)) != GS_OK) return st;
    GS_CHECK(app->kind != GS_APP_NEURAL_FOLDED,
             "the folded neural appearance renders only: differentiate GS_APP_NEURAL instead");
    if ((st = check_pre(pre, g->n)) != GS_OK) return st;
    GS_CHECK(tile_ranges && final_T && n_contrib && dL_dimage, "a render input array is NULL");
    GS_CHECK(grads != nullptr, "grads is NULL");
    if (g->n > 0 && !adam) {
        GS_CHECK(grads->dmeans && grads->dlog_scales && grads->dquats && grads->dopacity_logits,
                 "a geometry gradient array is NULL");
        if (app->kind == GS_APP_SH3) GS_CHECK(grads->dsh != nullptr, "dsh is NULL");
        else if (app->kind == GS_APP_NEURAL)
            GS_CHECK(grads->dbase_color && grads->dfeatures && grads->dmlp_w,
                     "dbase_color, dfeatures or dmlp_w is NULL");
        else if (app->kind == GS_APP_NASG || app->kind == GS_APP_NASGABOR)
            GS_CHECK(grads->dbase_color && grads->dlobes, "dbase_color or dlobes is NULL");
        else GS_CHECK(grads->dlatent && grads->dmlp_w, "dlatent or dmlp_w is NULL");
    }
    const Cam c = make_cam(*cam);
    const Workspace need = layout_workspace(nullptr, g->n, 0, app->kind, &c);
    if ((st = check_workspace(workspace, workspace_bytes, need)) != GS_OK) return st;
    const Workspace ws = layout_workspace(workspace, g->n, 0, app->kind, &c);
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (g->n == 0) {
        if (app->kind == GS_APP_LATENT_MLP) GS_HIP(launch_clear(grads->dmlp_w, GS_MLP_WEIGHTS, s));
        if (app->kind == GS_APP_NEURAL && grads->dmlp_w) GS_HIP(launch_clear(grads->dmlp_w, neural_weights(*app), s));
        return ok();
    }
    const bool ordered = tile_order_supported(c);
    timing_begin(GS_KERNEL_BWD_PREP, s);
    GS_HIP(launch_bwd_prep(c, tile_ranges, n_contrib, ws.acc, (int64_t)kAccStride * g->n, ws.walk_cls,
                           ordered ? ws.tile_order : nullptr, s));
    timing_end(GS_KERNEL_BWD_PREP, s);
    timing_begin(GS_KERNEL_BLEND_BWD, s);
    GS_HIP(launch_blend_bwd(c, pre->splats, values, tile_ranges, final_T, n_contrib, dL_dimage,
                            ordered ? ws.tile_order : nullptr, ws.acc, s));
    timing_end(GS_KERNEL_BLEND_BWD, s);
    timing_begin(GS_KERNEL_PREPROCESS_BWD, s);
    GS_HIP(launch_preprocess_bwd(c, *g, *app, *pre, ws, *grads, s, adam, beta1, eps, step));
    timing_end(GS_KERNEL_PREPROCESS_BWD, s);
    if (app->kind == GS_APP_LATENT_MLP || app->kind == GS_APP_NEURAL) {
        timing_begin(GS_KERNEL_MLP_REDUCE, s);
        GS_HIP(launch_mlp_reduce(g->n, *app, ws, grads->dmlp_w, s));
        timing_end(GS_KERNEL_MLP_REDUCE, s);
    }
    return ok();
}

}  // namespace

extern "C" {

gs_status gs_render_bwd(const gs_camera* cam, const gs_gaussians* g, const gs_appearance* app,
                        const gs_preprocessed* pre, const uint32_t* values, const uint32_t* tile_ranges,
                        const float* final_T, const uint32_t* n_contrib, const float* dL_dimage, const gs_grads* grads,
                        void* workspace, size_t workspace_bytes, void* stream)
{
    return render_bwd(cam, g, app, pre, values, tile_ranges, final_T, n_contrib, dL_dimage, grads, workspace,
                      workspace_bytes, stream, nullptr, 0.f, 0.f, 0);
}

gs_status gs_render_bwd_adam(const gs_camera* cam, const gs_gaussians* g, const gs_appearance* app,
                             const gs_preprocessed* pre, const uint32_t* values, const uint32_t* tile_ranges,
                             const float* final_T, const uint32_t* n_contrib, const float* dL_dimage,
                             const gs_grads* grads, const gs_adam_tensor* adam, float beta1, float eps, int64_t step,
                             void* workspace, size_t workspace_bytes, void* stream)
{
    gs_status st;
    if ((st = check_gaussians(g)) != GS_OK) return st;
    GS_CHECK(app != nullptr, "appearance is NULL");
    if (app->kind != GS_APP_SH3)
        return fail(GS_ERR_UNSUPPORTED, "gs_render_bwd_adam: appearance kind %d (SH3 only)", app->kind);
    GS_CHECK(adam != nullptr, "adam is NULL");
    GS_CHECK(step >= 1, "step %lld must be at least 1", (long long)step);
    GS_CHECK(beta1 >= 0.f && beta1 < 1.f, "beta1 must lie in [0, 1)");
    GS_CHECK(eps > 0.f, "eps must be positive");
    const float* params[GS_RENDER_ADAM_TENSORS] = {g->means, g->log_scales, g->quats, g->opacity_logits, app->sh};
    const int rows[GS_RENDER_ADAM_TENSORS] = {3, 3, 4, 1, GS_SH_COEFFS};
    for (int k = 0; k < GS_RENDER_ADAM_TENSORS; ++k) {
        const gs_adam_tensor& t = adam[k];
        GS_CHECK(t.param == params[k], "adam[%d].param is not the parameter array it updates", k);
        GS_CHECK(t.rows == rows[k] && t.n == g->n, "adam[%d]: rows %d, n %lld (%d rows of %lld expected)", k, t.rows,
                 (long long)t.n, rows[k], (long long)g->n);
        GS_CHECK(g->n == 0 || (t.exp_avg && t.exp_avg_sq), "adam[%d]: a moment array is NULL", k);
        GS_CHECK(t.lr != nullptr, "adam[%d].lr is NULL", k);
        GS_CHECK(t.beta2 >= 0.f && t.beta2 < 1.f, "adam[%d]: beta2 must lie in [0, 1)", k);
    }
    return render_bwd(cam, g, app, pre, values, tile_ranges, final_T, n_contrib, dL_dimage, grads, workspace,
                      workspace_bytes, stream, adam, beta1, eps, step);
}

gs_status gs_mlp_eval(const uint16_t* x, int64_t rows, const uint16_t* mlp_w, float* colors, void* stream)
{
    GS_CHECK(rows >= 0 && rows < ((int64_t)1 << 31), "rows = %lld out of range", (long long)rows);
    GS_CHECK(rows == 0 || (x && mlp_w && colors), "an array is NULL");
    if (rows == 0) return ok();
    GS_HIP(launch_mlp_eval(x, rows, mlp_w, colors, static_cast<hipStream_t>(stream)));
    return ok();
}

gs_status gs_neural_fold(const uint16_t* features, const uint16_t* mlp_w, int64_t n, uint16_t* preact, void* stream)
{
    GS_CHECK(n >= 0 && n < ((int64_t)1 << 31), "n = %lld out of range [0, 2^31)", (long long)n);
    GS_CHECK(n == 0 || (features && mlp_w && preact), "an array is NULL");
    GS_CHECK(((uintptr_t)preact & 7) == 0, "preact must be 8-byte aligned");
    if (n == 0) return ok();
    hipStream_t s = static_cast<hipStream_t>(stream);
    timing_begin(GS_KERNEL_NEURAL_FOLD, s);
    GS_HIP(launch_neural_fold(features, mlp_w, n, preact, s));
    timing_end(GS_KERNEL_NEURAL_FOLD, s);
    return ok();
}

gs_status gs_timer_create(gs_timer** out)
{
    GS_CHECK(out != nullptr, "out is NULL");
    gs_timer* t = new gs_timer();
    for (int k = 0; k < GS_KERNEL_COUNT; ++k) { t->ms[k] = 0.0; t->launches[k] = 0; }
    for (int k = 0; k < 2048; ++k) {
        hipEvent_t e;
        if (hipEventCreate(&e) != hipSuccess) {
            gs_timer_destroy(t);
            return fail(GS_ERR_DEVICE, "hipEventCreate failed");
        }
        t->free_events.push_back(e);
    }
    *out = t;
    return ok();
}

gs_status gs_timer_destroy(gs_timer* t)
{
    if (!t) return ok();
    if (t_timer == t) t_timer = nullptr;
    resolve_pending(t);
    for (auto& l : t->open) t->free_events.insert(t->free_events.end(), {l.a, l.b});
    for (hipEvent_t e : t->free_events) (void)hipEventDestroy(e);
    delete t;
    return ok();
}

gs_status gs_timer_attach(gs_timer* t)
{
    t_timer = t;
    return ok();
}

gs_status gs_timer_reset(gs_timer* t)
{
    GS_CHECK(t != nullptr, "timer is NULL");
    resolve_pending(t);
    for (int k = 0; k < GS_KERNEL_COUNT; ++k) { t->ms[k] = 0.0; t->launches[k] = 0; }
    return ok();
}

gs_status gs_timer_read(gs_timer* t, double* ms, int64_t* launches, int32_t count)
{
    GS_CHECK(t != nullptr, "timer is NULL");
    GS_CHECK(ms != nullptr && launches != nullptr, "output arrays are NULL");
    resolve_pending(t);
    for (int k = 0; k < count && k < GS_KERNEL_COUNT; ++k) { ms[k] = t->ms[k]; launches[k] = t->launches[k]; }
    return ok();
}

}  // extern "C"
