// Internal declarations of the gsraster HIP library (gfx950 / CDNA4).
// Kernels are launched only from the C-ABI entry points in api.hip.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <algorithm>

#include "../../include/gsraster.h"

namespace gsr {

constexpr int kTile = GS_TILE;
constexpr int kBlock = 256;               // 4 wave64 per workgroup
constexpr int kWave = 64;

// Camera as the kernels see it (by value in kernel arguments).
struct Cam {
    float V[12];          // row-major [R|t]
    float campos[3];
    float fx, fy, cx, cy;
    int width, height;
    int tiles_x, tiles_y;
    float near_plane;
    float bg[3];
};

inline Cam make_cam(const gs_camera& c) {
    Cam k;
    for (int i = 0; i < 12; ++i) k.V[i] = c.viewmat[i];
    for (int i = 0; i < 3; ++i) { k.campos[i] = c.campos[i]; k.bg[i] = c.bg[i]; }
    k.fx = c.fx; k.fy = c.fy; k.cx = c.cx; k.cy = c.cy;
    k.width = c.width; k.height = c.height;
    k.tiles_x = (c.width + kTile - 1) / kTile;
    k.tiles_y = (c.height + kTile - 1) / kTile;
    k.near_plane = c.near_plane;
    return k;
}

// Splat record as four 16-byte words (layout of gs_splat).
//  w0 = mean_x, mean_y, conic_a, conic_b
//  w1 = conic_c, opacity, color r, color g
//  w2 = color b, power_min, ext_x, ext_y
//  w3 = rect (x0 | y0 << 16), rect (x1 | y1 << 16), depth, 0
static_assert(sizeof(gs_splat) == 64, "splat record must be 64 bytes");
constexpr int kSplatRectWord = 12;   // float offset of the packed rectangle
static_assert(offsetof(gs_splat, rect) == 4 * kSplatRectWord, "rectangle offset");
static_assert(offsetof(gs_splat, power_min) == 36 && offsetof(gs_splat, depth) == 56, "record layout");

// Per-Gaussian screen-space gradient accumulator written by the blend backward.
// Stride 9 floats: dmean_x, dmean_y, dconic_a, dconic_b, dconic_c, dopacity, dcolor rgb.
constexpr int kAccStride = 9;

// Radix-sort geometry: 256 threads x 16 keys per workgroup and digits of at
// most 8 bits for the depth sort (n keys); x 32 keys and 9 bits for the block
// sort (the entries).
constexpr int kSortItems = 16;
constexpr int kBlockSortItems = 32;
constexpr int kSortTile = kBlock * kSortItems;   // 4096
constexpr int kRadix = 256;
constexpr int kDupChunk = 1024;   // depth-ordered Gaussians per workgroup in entry emission
constexpr int kBlockDim = 4;      // a block is kBlockDim x kBlockDim tiles
// Tile order of the blend backward: classes of walk length (16 per octave of a
// u32) and the largest image it is taken for (larger images keep the plain order).
constexpr int kWalkClasses = 512;
constexpr int kMaxOrderedTiles = 32768;

// Workgroups of the decoder preprocess backward (grid-stride), one partial
// weight gradient each: as many as are resident at once, 3 per compute unit
// (2 for the 32-neuron decoder, whose registers allow only 2).
constexpr int kMlpPartials = 768;
constexpr int kMlpPartials32 = 512;

__host__ __device__ inline int64_t div_up(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline size_t align_up(size_t a, size_t b) { return (a + b - 1) / b * b; }

// ---- workspace layout -------------------------------------------------------
// One layout serves every call; gs_workspace_size returns its total.
struct Workspace {
    uint32_t* block_pairs;   // [pair_count_slots] tile sums per preprocess workgroup or wave
    uint32_t* keys_a;        // [n]               depth-sort ping-pong keys
    uint32_t* keys_b;        // [n]
    uint32_t* vals_a;        // [n]               depth-sort values
    uint32_t* vals_b;        // [n]
    uint32_t* hist;          // [digits][workgroups] of a radix pass (256 x n / 4096, 512 x capacity / 8192)
    uint32_t* digit_tot;     // [4 passes][256]   digit totals of each pass
    uint32_t* scan_part;     // [n / kDupChunk + 1] chunk sums of the entry-offset scan
    uint2* sorted_rect;      // [n]               tile rectangles in depth order (empty for culled)
    uint64_t* entry_count;   // [1]               block entries (0 when the pairs exceed the capacity)
    uint32_t* entry_keys_a;  // [capacity]        entry keys: block id << 16 | tile mask
    uint32_t* entry_vals_a;  // [capacity]        entry values: Gaussian index
    uint32_t* entry_keys_b;  // [capacity]
    uint32_t* entry_vals_b;  // [capacity]
    uint32_t* block_ranges;  // [blocks][2]       each block's entries
    uint32_t* seg_base;      // [blocks + 1]      first segment of each block
    uint32_t* seg_block;     // [segments]        block of each segment
    uint32_t* seg_cnt;       // [segments][4][16] per-tile counts, then offsets, of each wave's sub-segment
    uint32_t* list_counters; // [2]               segments; tile lists over capacity
    float* acc;              // [n][9]            blend-backward accumulators
    uint32_t* walk_cls;      // [tiles]           walk-length class of each tile (blend backward)
    uint32_t* tile_order;    // [tiles]           tiles, longest walk first (blend backward)
    float* mlp_part;         // [kMlpPartials][1664] per-workgroup decoder weight gradients
    size_t bytes;
};

// `cam` (NULL for calls that bin nothing) sizes the per-block buffers.
Workspace layout_workspace(void* base, int64_t n, uint64_t capacity, int32_t kind, const struct Cam* cam);

// Number of (tile, Gaussian) pairs as the bin-sort kernels see it. Host mode:
// `host` is P itself. Device mode: P is read on the device from the
// preprocess's count `dev`, `host` is the capacity the grids are sized for,
// and a count above the capacity reads as 0 (no pairs are emitted and every
// tile range comes out empty; the count itself stays in place for the caller).
struct PairCount {
    const uint64_t* dev;
    uint64_t host;
    uint64_t cap;
    __device__ __forceinline__ uint64_t get() const
    {
        if (!dev) return host;
        const uint64_t p = *dev;
        return p <= cap ? p : 0;
    }
    __device__ __forceinline__ bool overflow() const { return dev && *dev > cap; }
};

// ---- launch helpers (defined in the kernel files) ---------------------------
// *slots: the number of tile sums it leaves in ws.block_pairs for the pair count
hipError_t launch_preprocess(const Cam& cam, const gs_gaussians& g, const gs_appearance& app,
                             const gs_preprocessed& out, const Workspace& ws, int* slots, hipStream_t s);
hipError_t launch_pair_count(int slots, const Workspace& ws, uint64_t* num_pairs, hipStream_t s);
hipError_t launch_depth_sort(int64_t n, const uint32_t* depth_key, const gs_splat* splats, const Workspace& ws,
                             const uint32_t** order_out, hipStream_t s);
hipError_t launch_entry_offsets(int64_t n, PairCount pairs, const Workspace& ws, hipStream_t s);
int blocks_x_of(const Cam& cam);
int blocks_y_of(const Cam& cam);
int64_t segment_bound(const Cam& cam, uint64_t capacity);   // segments the tile-list kernels can meet
bool blocks_supported(const Cam& cam);   // at most 65536 blocks: the block id shares a u32 key with a tile mask
hipError_t launch_block_entries(const Cam& cam, int64_t n, const uint32_t* order, PairCount entries,
                                const Workspace& ws, hipStream_t s);
struct BlockEntries {
    const uint32_t* key;   // block id << 16 | mask of the block's tiles the Gaussian meets
    const uint32_t* gid;   // Gaussian index
};
hipError_t launch_block_sort(const Cam& cam, PairCount entries, const Workspace& ws, BlockEntries* out, hipStream_t s);
hipError_t launch_tile_lists(const Cam& cam, PairCount pairs, uint64_t capacity, const Workspace& ws,
                             const BlockEntries& ent, uint32_t* values, uint32_t* tile_ids, uint32_t* tile_ranges,
                             hipStream_t s);
hipError_t launch_fill_u32(uint32_t* p, int64_t count, uint32_t value, hipStream_t s);
hipError_t launch_blend_fwd(const Cam& cam, const gs_splat* splats, const uint32_t* values,
                            const uint32_t* tile_ranges, float* image, float* final_T, uint32_t* n_contrib,
                            hipStream_t s);
hipError_t launch_clear(float* p, int64_t count, hipStream_t s);
hipError_t launch_blend_count(const Cam& cam, const gs_splat* splats, const uint32_t* values,
                              const uint32_t* tile_ranges, uint64_t* counts, hipStream_t s);
bool tile_order_supported(const Cam& cam);   // at most kMaxOrderedTiles tiles
// The backward's preparation: acc[0, acc_count) cleared and, when `order` is
// given, the tiles' launch order, longest walk first (walk_cls: n_tiles scratch).
hipError_t launch_bwd_prep(const Cam& cam, const uint32_t* tile_ranges, const uint32_t* n_contrib, float* acc,
                           int64_t acc_count, uint32_t* walk_cls, uint32_t* order, hipStream_t s);
// tile_order: NULL for the plain tile order
hipError_t launch_blend_bwd(const Cam& cam, const gs_splat* splats, const uint32_t* values,
                            const uint32_t* tile_ranges, const float* final_T, const uint32_t* n_contrib,
                            const float* dL_dimage, const uint32_t* tile_order, float* acc, hipStream_t s);
// adam: NULL, or the gs_adam_tensor of each per-Gaussian parameter in the order of
// gs_render_bwd_adam, whose step is then applied in place (SH3 only)
hipError_t launch_preprocess_bwd(const Cam& cam, const gs_gaussians& g, const gs_appearance& app,
                                 const gs_preprocessed& pre, const Workspace& ws, const gs_grads& gr,
                                 hipStream_t s, const gs_adam_tensor* adam = nullptr, float beta1 = 0.f,
                                 float eps = 0.f, int64_t step = 0);
hipError_t launch_mlp_reduce(int64_t n, const gs_appearance& app, const Workspace& ws, float* dmlp_w, hipStream_t s);
hipError_t launch_adam(const gs_adam_tensor* tensors, int count, float beta1, float eps, int64_t step, hipStream_t s);
hipError_t launch_mlp_eval(const uint16_t* x, int64_t rows, const uint16_t* w, float* out, hipStream_t s);
hipError_t launch_neural_fold(const uint16_t* features, const uint16_t* w, int64_t n, uint16_t* preact,
                              hipStream_t s);

// Kernel timing hooks (api.hip): bracket one logical kernel id.
void timing_begin(int kernel_id, hipStream_t s);
void timing_end(int kernel_id, hipStream_t s);

inline int preprocess_blocks(int64_t n) { return (int)div_up(n > 0 ? n : 1, kBlock); }
// Slots for the preprocess tile sums: one per workgroup, or one per wave of a
// decoder grid (at most one workgroup per 256 Gaussians).
inline int pair_count_slots(int64_t n) { return preprocess_blocks(n) * (kBlock / kWave); }

// Hidden layers of the neural decoder (0 in the struct: the paper's default, 2)
// and its weight count.
inline int neural_layers(const gs_appearance& a) { return a.neural_layers > 0 ? a.neural_layers : 2; }
inline int neural_weights(const gs_appearance& a)
{
    const int L = neural_layers(a), W = a.neural_width == 32 ? 32 : 16;
    return W * 32 + (L - 1) * W * W + 3 * W;
}

}  // namespace gsr
