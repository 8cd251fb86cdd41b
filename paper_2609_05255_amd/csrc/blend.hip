// Tile blend (Sec. 3.1) and its reverse. One 256-thread workgroup (4 wave64)
// per 16x16 tile, one pixel per thread; the tile's depth-sorted list is walked
// in batches of 256 splats staged in LDS. Workgroup ids are mapped to tiles so
// that each XCD (workgroups are dealt round-robin over the 8 XCDs) renders one
// contiguous band of tiles, whose lists share most of their splats in that
// XCD's L2.
#include "gs_internal.h"

namespace gsr {

namespace {

constexpr int kXcds = 8;

__device__ __forceinline__ int tile_of_block(int block, int n_tiles)
{
    const int per = (n_tiles + kXcds - 1) / kXcds;
    return (block % kXcds) * per + block / kXcds;
}

inline int blend_grid(int n_tiles) { return (int)div_up(n_tiles, kXcds) * kXcds; }

struct SplatLds {
    float2 xy[kBlock];
    float4 co[kBlock];     // conic a, b, c, opacity
    float4 rgb[kBlock];    // colour, w unused
    uint32_t id[kBlock];
};

__device__ __forceinline__ void stage_splat(SplatLds& s, int slot, const gs_splat* __restrict__ splats, uint32_t g)
{
    const float4* p = reinterpret_cast<const float4*>(splats + g);
    const float4 w0 = p[0];
    const float4 w1 = p[1];
    const float cb = reinterpret_cast<const float*>(splats + g)[8];
    s.xy[slot] = make_float2(w0.x, w0.y);
    s.co[slot] = make_float4(w0.z, w0.w, w1.x, w1.y);
    s.rgb[slot] = make_float4(w1.z, w1.w, cb, 0.f);
    s.id[slot] = g;
}

// The quadratic form and alpha of one (pixel, splat) pair; identical code in
// the forward and the backward so both take the same skip/stop decisions.
__device__ __forceinline__ float splat_power(const float2 xy, const float4 co, float px, float py, float& dx,
                                             float& dy)
{
    dx = px - xy.x;
    dy = py - xy.y;
    return __fmaf_rn(-0.5f, __fmaf_rn(co.x * dx, dx, co.z * dy * dy), -(co.y * dx) * dy);
}

constexpr float kAlphaMin = 1.0f / 255.0f;
constexpr float kAlphaMax = 0.99f;
constexpr float kTMin = 0.0001f;
constexpr float kLog2e = 1.4426950408889634f;

__device__ __forceinline__ float exp_fast(float x) { return __builtin_amdgcn_exp2f(x * kLog2e); }

}  // namespace

__global__ __launch_bounds__(kBlock) void k_blend_fwd(Cam cam, const gs_splat* __restrict__ splats,
                                                      const uint32_t* __restrict__ values,
                                                      const uint32_t* __restrict__ ranges, float* __restrict__ image,
                                                      float* __restrict__ final_T, uint32_t* __restrict__ n_contrib)
{
    __shared__ SplatLds s;
    const int n_tiles = cam.tiles_x * cam.tiles_y;
    const int tile = tile_of_block(blockIdx.x, n_tiles);
    if (tile >= n_tiles) return;
    const int tx = tile % cam.tiles_x, ty = tile / cam.tiles_x;
    const int x = tx * kTile + (threadIdx.x & 15), y = ty * kTile + (threadIdx.x >> 4);
    const bool inside = x < cam.width && y < cam.height;
    const float px = (float)x + 0.5f, py = (float)y + 0.5f;
    const uint32_t start = ranges[2 * tile], end = ranges[2 * tile + 1];

    float T = 1.f, C0 = 0.f, C1 = 0.f, C2 = 0.f;
    uint32_t last = 0;
    bool done = !inside;
    for (uint32_t b = start; b < end; b += kBlock) {
        if (__syncthreads_count(done) == kBlock) break;
        const uint32_t idx = b + threadIdx.x;
        if (idx < end) stage_splat(s, threadIdx.x, splats, values[idx]);
        __syncthreads();
        const int cnt = (int)min((uint32_t)kBlock, end - b);
        if (!done) {
            for (int j = 0; j < cnt; ++j) {
                float dx, dy;
                const float4 co = s.co[j];
                const float power = splat_power(s.xy[j], co, px, py, dx, dy);
                if (power > 0.f) continue;
                const float alpha = fminf(kAlphaMax, co.w * exp_fast(power));
                if (alpha < kAlphaMin) continue;
                const float Tn = T * (1.f - alpha);
                if (Tn < kTMin) { done = true; break; }
                const float w = alpha * T;
                const float4 c = s.rgb[j];
                C0 = __fmaf_rn(c.x, w, C0);
                C1 = __fmaf_rn(c.y, w, C1);
                C2 = __fmaf_rn(c.z, w, C2);
                T = Tn;
                last = b - start + (uint32_t)j + 1;
            }
        }
        __syncthreads();
    }
    if (inside) {
        const int64_t pix = (int64_t)y * cam.width + x;
        const int64_t hw = (int64_t)cam.width * cam.height;
        image[pix] = __fmaf_rn(T, cam.bg[0], C0);
        image[hw + pix] = __fmaf_rn(T, cam.bg[1], C1);
        image[2 * hw + pix] = __fmaf_rn(T, cam.bg[2], C2);
        final_T[pix] = T;
        n_contrib[pix] = last;
    }
}

hipError_t launch_blend_fwd(const Cam& cam, const gs_splat* splats, const uint32_t* values,
                            const uint32_t* tile_ranges, float* image, float* final_T, uint32_t* n_contrib,
                            hipStream_t s)
{
    const int n_tiles = cam.tiles_x * cam.tiles_y;
    hipLaunchKernelGGL(k_blend_fwd, dim3(blend_grid(n_tiles)), dim3(kBlock), 0, s, cam, splats, values, tile_ranges,
                       image, final_T, n_contrib);
    return hipGetLastError();
}

// ---- backward -----------------------------------------------------------------
// Per pixel, back to front from its last blended splat, with T recovered as
// T_i = T_{i+1} / (1 - alpha_i) and S the suffix sum of colour * alpha * T plus
// T_final * bg:  dL/dcolour_i = alpha_i T_i g,  dL/dalpha_i = sum_ch
// (T_i c_i - S / (1 - alpha_i)) g_ch. Each wave sums its 64 pixels' gradients of a
// splat before one set of float atomics per splat.

__device__ __forceinline__ float wave_sum(float v)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    return v;
}

__global__ __launch_bounds__(kBlock) void k_blend_bwd(Cam cam, const gs_splat* __restrict__ splats,
                                                      const uint32_t* __restrict__ values,
                                                      const uint32_t* __restrict__ ranges,
                                                      const float* __restrict__ final_T,
                                                      const uint32_t* __restrict__ n_contrib,
                                                      const float* __restrict__ dL_dimage, float* __restrict__ acc)
{
    __shared__ SplatLds s;
    __shared__ uint32_t max_last;
    const int n_tiles = cam.tiles_x * cam.tiles_y;
    const int tile = tile_of_block(blockIdx.x, n_tiles);
    if (tile >= n_tiles) return;
    const int tx = tile % cam.tiles_x, ty = tile / cam.tiles_x;
    const int x = tx * kTile + (threadIdx.x & 15), y = ty * kTile + (threadIdx.x >> 4);
    const bool inside = x < cam.width && y < cam.height;
    const float px = (float)x + 0.5f, py = (float)y + 0.5f;
    const uint32_t start = ranges[2 * tile], len = ranges[2 * tile + 1] - start;
    const int64_t pix = (int64_t)y * cam.width + x;
    const int64_t hw = (int64_t)cam.width * cam.height;

    float T = 1.f, g0 = 0.f, g1 = 0.f, g2 = 0.f;
    uint32_t last = 0;
    if (inside) {
        T = final_T[pix];
        last = min(n_contrib[pix], len);
        g0 = dL_dimage[pix];
        g1 = dL_dimage[hw + pix];
        g2 = dL_dimage[2 * hw + pix];
    }
    float S0 = T * cam.bg[0], S1 = T * cam.bg[1], S2 = T * cam.bg[2];
    if (threadIdx.x == 0) max_last = 0;
    __syncthreads();
    atomicMax(&max_last, last);
    __syncthreads();
    const uint32_t stop = max_last;   // list positions [0, stop) can contribute
    if (stop == 0) return;
    const int lane = __lane_id();
    const int nbatch = (int)((stop + kBlock - 1) / kBlock);
    for (int bi = nbatch - 1; bi >= 0; --bi) {
        const uint32_t b = (uint32_t)bi * kBlock;   // position of the batch within the tile list
        const uint32_t cnt = min((uint32_t)kBlock, stop - b);
        __syncthreads();
        if ((uint32_t)threadIdx.x < cnt) stage_splat(s, threadIdx.x, splats, values[start + b + threadIdx.x]);
        __syncthreads();
        for (int j = (int)cnt - 1; j >= 0; --j) {
            const uint32_t pos = b + (uint32_t)j;
            bool contrib = pos < last;
            float dx = 0.f, dy = 0.f, alpha = 0.f, G = 0.f;
            const float4 co = s.co[j];
            if (contrib) {
                const float power = splat_power(s.xy[j], co, px, py, dx, dy);
                contrib = power <= 0.f;
                if (contrib) {
                    G = exp_fast(power);
                    alpha = fminf(kAlphaMax, co.w * G);
                    contrib = alpha >= kAlphaMin;
                }
            }
            if (__ballot(contrib) == 0) continue;
            float dm_x = 0.f, dm_y = 0.f, dca = 0.f, dcb = 0.f, dcc = 0.f, dop = 0.f, dc0 = 0.f, dc1 = 0.f,
                  dc2 = 0.f;
            if (contrib) {
                const float oma = 1.f - alpha;
                T = T / oma;                        // transmittance in front of this splat
                const float4 c = s.rgb[j];
                const float w = alpha * T;
                dc0 = w * g0;
                dc1 = w * g1;
                dc2 = w * g2;
                const float inv = 1.f / oma;
                const float dalpha = (T * c.x - S0 * inv) * g0 + (T * c.y - S1 * inv) * g1 + (T * c.z - S2 * inv) * g2;
                S0 = __fmaf_rn(c.x, w, S0);
                S1 = __fmaf_rn(c.y, w, S1);
                S2 = __fmaf_rn(c.z, w, S2);
                if (co.w * G < kAlphaMax) {         // below the cap alpha = o G
                    dop = G * dalpha;
                    const float dpow = alpha * dalpha;
                    dm_x = dpow * (co.x * dx + co.y * dy);
                    dm_y = dpow * (co.z * dy + co.y * dx);
                    dca = -0.5f * dpow * dx * dx;
                    dcb = -dpow * dx * dy;
                    dcc = -0.5f * dpow * dy * dy;
                }
            }
            dm_x = wave_sum(dm_x);
            dm_y = wave_sum(dm_y);
            dca = wave_sum(dca);
            dcb = wave_sum(dcb);
            dcc = wave_sum(dcc);
            dop = wave_sum(dop);
            dc0 = wave_sum(dc0);
            dc1 = wave_sum(dc1);
            dc2 = wave_sum(dc2);
            if (lane == 0) {
                float* a = acc + (size_t)s.id[j] * kAccStride;
                atomicAdd(a + 0, dm_x);
                atomicAdd(a + 1, dm_y);
                atomicAdd(a + 2, dca);
                atomicAdd(a + 3, dcb);
                atomicAdd(a + 4, dcc);
                atomicAdd(a + 5, dop);
                atomicAdd(a + 6, dc0);
                atomicAdd(a + 7, dc1);
                atomicAdd(a + 8, dc2);
            }
        }
    }
}

hipError_t launch_blend_bwd(const Cam& cam, const gs_splat* splats, const uint32_t* values,
                            const uint32_t* tile_ranges, const float* final_T, const uint32_t* n_contrib,
                            const float* dL_dimage, float* acc, hipStream_t s)
{
    const int n_tiles = cam.tiles_x * cam.tiles_y;
    hipLaunchKernelGGL(k_blend_bwd, dim3(blend_grid(n_tiles)), dim3(kBlock), 0, s, cam, splats, values, tile_ranges,
                       final_T, n_contrib, dL_dimage, acc);
    return hipGetLastError();
}

// Zero fill of `count` floats; p must be 16-byte aligned. Body in float4, tail
// in scalars. A kernel rather than a memset so that it behaves the same inside
// a captured graph.
__global__ __launch_bounds__(kBlock) void k_clear(float* __restrict__ p, int64_t count)
{
    const int64_t c4 = count >> 2;
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    float4* p4 = reinterpret_cast<float4*>(p);
    for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < c4; i += stride)
        p4[i] = make_float4(0.f, 0.f, 0.f, 0.f);
    if (blockIdx.x == 0 && threadIdx.x < (count & 3)) p[(c4 << 2) + threadIdx.x] = 0.f;
}

hipError_t launch_clear(float* p, int64_t count, hipStream_t s)
{
    const int blocks = (int)std::min<int64_t>(std::max<int64_t>(div_up(count >> 2, kBlock), 1), 4096);
    hipLaunchKernelGGL(k_clear, dim3(blocks), dim3(kBlock), 0, s, p, count);
    return hipGetLastError();
}

__global__ __launch_bounds__(kBlock) void k_fill_u32(uint32_t* __restrict__ p, int64_t count, uint32_t v)
{
    const int64_t stride = (int64_t)gridDim.x * kBlock;
    for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < count; i += stride) p[i] = v;
}

hipError_t launch_fill_u32(uint32_t* p, int64_t count, uint32_t value, hipStream_t s)
{
    const int blocks = (int)std::min<int64_t>(std::max<int64_t>(div_up(count, kBlock), 1), 4096);
    hipLaunchKernelGGL(k_fill_u32, dim3(blocks), dim3(kBlock), 0, s, p, count, value);
    return hipGetLastError();
}

}  // namespace gsr
