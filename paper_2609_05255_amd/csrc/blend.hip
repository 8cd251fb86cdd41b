// Tile blend (Sec. 3.1) and its reverse. A 16x16 tile is covered by 4/PIX
// independent wave64s (PIX = 2 in the forward, 4 in the backward); wave w owns
// the 4 PIX contiguous rows from 4 PIX w, and every lane PIX pixels of one
// column (rows 4k apart), so a lane's pixels share dx and the quadratic form
// costs two fused multiply-adds per pixel. Each wave walks the tile's
// depth-sorted list in batches of 64 splats: every lane gathers one record
// (the next batch is fetched while the current one is blended) and tests it
// against the wave's pixels, the batch is staged in the wave's own LDS slot,
// and each splat that passes is then read back by the whole wave from one
// address (a broadcast read). No workgroup barriers; a wave stops when its own
// pixels are done.
//
// Workgroup ids are mapped to tiles so that each XCD (workgroups are dealt
// round-robin over the 8 XCDs) renders a contiguous band of tiles, whose lists
// share most splats in that XCD's L2; the backward of images up to 32768 tiles
// takes them longest walk first instead (the tile order below).
#include "gs_internal.h"

namespace gsr {

namespace {

constexpr int kXcds = 8;

// Pixels per lane of the forward and the backward (1, 2 or 4). The forward's
// two waves per tile halve the longest walks' time, which sets its end (its
// tiles' walks differ by 3x and cannot be ordered before blending).
#ifndef GS_FWD_PIX
#define GS_FWD_PIX 2
#endif
#ifndef GS_BWD_PIX
#define GS_BWD_PIX 4
#endif

__device__ __forceinline__ int tile_of_block(int block, int n_tiles)
{
    const int per = (n_tiles + kXcds - 1) / kXcds;
    return (block % kXcds) * per + block / kXcds;
}

inline int blend_grid(int n_tiles) { return (int)div_up(n_tiles, kXcds) * kXcds; }

constexpr float kAlphaMin = 1.0f / 255.0f;
constexpr float kAlphaMax = 0.99f;
constexpr float kTMin = 0.0001f;
constexpr float kLog2e = 1.4426950408889634f;


// One splat record in registers (the fields the blend needs).
struct SplatReg {
    float mx, my, ca, cb, cc, op, r, g, b, pmin, ex, ey;
    uint32_t id;
};

// power(dy) = -(a dx^2 + c dy^2)/2 - b dx dy for one column, in base-2 units
// (times log2 e) so that exp(power) is one hardware exp2:
// power log2 e = q0 + dy (q1 + dy q2).
struct Quad {
    float q0, q1, q2;
};

__device__ __forceinline__ Quad column_quad(const SplatReg& s, float dx)
{
    Quad q;
    q.q0 = (-0.5f * kLog2e) * s.ca * dx * dx;
    q.q1 = (-kLog2e * dx) * s.cb;
    q.q2 = (-0.5f * kLog2e) * s.cc;
    return q;
}

__device__ __forceinline__ float quad_power(const Quad& q, float dy)
{
    return __fmaf_rn(__fmaf_rn(q.q2, dy, q.q1), dy, q.q0);
}

template <int kCtrl>
__device__ __forceinline__ float dpp_f32(float v)
{
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), kCtrl, 0xF, 0xF, false));
}

// Sum over the 16 lanes of each row, in every lane of the row.
__device__ __forceinline__ float row_sum(float v)
{
    v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xF, 0xF, false));
    v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4E, 0xF, 0xF, false));
    v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x141, 0xF, 0xF, false));
    v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x140, 0xF, 0xF, false));
    return v;
}

// Whether the splat's alpha >= 1/255 region (power >= power_min, i.e. the
// conic's quadratic form q(u, v) = a u^2 + 2 b u v + c v^2 at most
// r2 = -2 power_min) meets the box [x_lo, x_hi] x [y_lo, y_hi] of the wave's
// pixel centres. The least q over the box is 0 when the mean lies inside it,
// else it is on an edge, where q is a parabola in the free coordinate: its
// vertex, clamped to the edge. The margin, 1e-3 plus 1e-5 of the largest sum
// of the three terms' magnitudes over the box, is far above the rounding of
// this evaluation and of the per-pixel power (a few ulp of that sum), so a
// splat found apart from the box reaches power_min at none of its pixels.
__device__ __forceinline__ bool ellipse_meets_box(float mx, float my, float a, float b, float c, float pmin,
                                                  float x_lo, float x_hi, float y_lo, float y_hi)
{
    const float r2 = -2.f * pmin;
    const float u0 = x_lo - mx, u1 = x_hi - mx, v0 = y_lo - my, v1 = y_hi - my;
    const float ia = __builtin_amdgcn_rcpf(a), ic = __builtin_amdgcn_rcpf(c);
    auto q = [&](float u, float v) { return a * u * u + 2.f * b * u * v + c * v * v; };
    auto on_u = [&](float u) { return q(u, fminf(fmaxf(-b * u * ic, v0), v1)); };   // edge of fixed u
    auto on_v = [&](float v) { return q(fminf(fmaxf(-b * v * ia, u0), u1), v); };   // edge of fixed v
    const bool inside = u0 <= 0.f && u1 >= 0.f && v0 <= 0.f && v1 >= 0.f;
    const float qmin = inside ? 0.f : fminf(fminf(on_u(u0), on_u(u1)), fminf(on_v(v0), on_v(v1)));
    const float um = fmaxf(fabsf(u0), fabsf(u1)), vm = fmaxf(fabsf(v0), fabsf(v1));
    const float terms = a * um * um + c * vm * vm + 2.f * fabsf(b) * um * vm;
    return qmin <= r2 + (1e-3f + 1e-5f * terms);
}

}  // namespace

template <int kPix>
__global__ __launch_bounds__(kTile * kTile / kPix) void k_blend_fwd(Cam cam, const gs_splat* __restrict__ splats,
                                                                    const uint32_t* __restrict__ values,
                                                                    const uint32_t* __restrict__ ranges,
                                                                    float* __restrict__ image,
                                                                    float* __restrict__ final_T,
                                                                    uint32_t* __restrict__ n_contrib)
{
    constexpr int kRowStep = 4;   // pixel k of a lane lies 4k rows below its first
    const int n_tiles = cam.tiles_x * cam.tiles_y;
    const int tile = tile_of_block(blockIdx.x, n_tiles);
    if (tile >= n_tiles) return;
    const int lane = __lane_id();
    const int tx = tile % cam.tiles_x, ty = tile / cam.tiles_x;
    // wave w covers the 4 kPix contiguous rows starting at 4 kPix w
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int x = tx * kTile + (lane & 15);
    const int y0 = ty * kTile + 4 * kPix * wave + (lane >> 4);
    const float px = (float)x + 0.5f;
    const uint32_t start = ranges[2 * tile], end = ranges[2 * tile + 1];
    // box of this wave's pixel centres: 16 columns, 4 kPix rows
    const float box_cx = (float)(tx * kTile) + 8.f, box_hx = 7.5f;
    const float box_lo = (float)(ty * kTile + 4 * kPix * wave) + 0.5f;
    const float box_hi = box_lo + (float)(4 * kPix - 1);
    const float box_cy = 0.5f * (box_lo + box_hi), box_hy = 0.5f * (box_hi - box_lo);

    // T > 0 while the pixel still blends; the stop rule (and a pixel outside
    // the image) makes it negative, |T| keeping the final transmittance
    float T[kPix], C0[kPix], C1[kPix], C2[kPix], py[kPix];
    uint32_t last[kPix];
#pragma unroll
    for (int k = 0; k < kPix; ++k) {
        C0[k] = C1[k] = C2[k] = 0.f;
        last[k] = 0;
        py[k] = (float)(y0 + kRowStep * k) + 0.5f;
        T[k] = (x < cam.width && (y0 + kRowStep * k) < cam.height) ? 1.f : -1.f;
    }
    bool any = false;
#pragma unroll
    for (int k = 0; k < kPix; ++k) any = any || T[k] > 0.f;
    // each batch of 64 list entries is staged in LDS; the wave then reads one
    // record per step at a uniform address (a broadcast read: no vector
    // instructions, unlike a lane-by-lane readlane broadcast)
    __shared__ float4 stage[kTile * kTile / kPix / kWave][3][kWave];
    float4 (*st)[kWave] = stage[wave];
    float4 c0 = make_float4(0.f, 0.f, 0.f, 0.f), c1 = c0, c2 = c0;
    if (start + lane < end) {
        const float4* p = reinterpret_cast<const float4*>(splats + values[start + lane]);
        c0 = p[0]; c1 = p[1]; c2 = p[2];
    }
    // the list entry of the batch after the prefetched one, loaded a batch early
    uint32_t nid = start + kWave + lane < end ? values[start + kWave + lane] : 0u;
    for (uint32_t b = start; b < end && __ballot(any) != 0; b += kWave) {
        st[0][lane] = c0; st[1][lane] = c1; st[2][lane] = c2;
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        // skip the splats that reach alpha >= 1/255 nowhere in this wave's
        // pixels: each lane tests the record it holds (before the next batch
        // replaces it; the bounding box first, then the ellipse), and the walk
        // below visits only the others, in order
        const int cnt = (int)min((uint32_t)kWave, end - b);
        const bool meets = lane < cnt && fabsf(c0.x - box_cx) <= c2.z + box_hx &&
                           fabsf(c0.y - box_cy) <= c2.w + box_hy &&
                           ellipse_meets_box(c0.x, c0.y, c0.z, c0.w, c1.x, c2.y, box_cx - box_hx, box_cx + box_hx,
                                             box_lo, box_hi);
        uint64_t todo = __ballot(meets);
        if (b + kWave + lane < end) {
            const float4* p = reinterpret_cast<const float4*>(splats + nid);
            c0 = p[0]; c1 = p[1]; c2 = p[2];
        }
        if (b + 2 * kWave + lane < end) nid = values[b + 2 * kWave + lane];
        while (todo != 0) {
            const int j = (int)__builtin_ctzll(todo);
            todo &= todo - 1;
            SplatReg s;
            const float4 w0 = st[0][j], w1 = st[1][j], w2 = st[2][j];
            s.mx = w0.x; s.my = w0.y;
            s.ca = w0.z; s.cb = w0.w; s.cc = w1.x; s.op = w1.y; s.r = w1.z; s.g = w1.w; s.b = w2.x; s.pmin = w2.y;
            const float dx = px - s.mx;
            const Quad q = column_quad(s, dx);
            const float pmin2 = s.pmin * kLog2e;
#pragma unroll
            for (int k = 0; k < kPix; ++k) {
                // one branch per pixel; the alpha floor and the stop rule are
                // selects inside it (the same decisions, fewer exec-mask changes)
                const float power2 = quad_power(q, py[k] - s.my);
                if (T[k] > 0.f && power2 <= 0.f && power2 >= pmin2) {
                    const float alpha = fminf(kAlphaMax, s.op * __builtin_amdgcn_exp2f(power2));
                    const float Tn = T[k] * (1.f - alpha);
                    const bool on = alpha >= kAlphaMin;
                    const bool stop = on && Tn < kTMin;
                    const bool blend = on && !stop;
                    const float w = blend ? alpha * T[k] : 0.f;
                    C0[k] = __fmaf_rn(s.r, w, C0[k]);
                    C1[k] = __fmaf_rn(s.g, w, C1[k]);
                    C2[k] = __fmaf_rn(s.b, w, C2[k]);
                    last[k] = blend ? b - start + (uint32_t)j + 1 : last[k];
                    T[k] = stop ? -T[k] : (blend ? Tn : T[k]);
                }
            }
            // a pixel can only stop on a splat that reaches it. T > 0 is tested
            // on its bits (T is never NaN): an integer maximum, where a float
            // one would first be canonicalised
            int tmax = __float_as_int(T[0]);
#pragma unroll
            for (int k = 1; k < kPix; ++k) tmax = max(tmax, __float_as_int(T[k]));
            any = tmax > 0;
            if (__ballot(any) == 0) break;
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
    const int64_t hw = (int64_t)cam.width * cam.height;
#pragma unroll
    for (int k = 0; k < kPix; ++k) {
        const int y = y0 + kRowStep * k;
        if (x >= cam.width || y >= cam.height) continue;
        const int64_t pix = (int64_t)y * cam.width + x;
        const float Tf = fabsf(T[k]);
        image[pix] = __fmaf_rn(Tf, cam.bg[0], C0[k]);
        image[hw + pix] = __fmaf_rn(Tf, cam.bg[1], C1[k]);
        image[2 * hw + pix] = __fmaf_rn(Tf, cam.bg[2], C2[k]);
        final_T[pix] = Tf;
        n_contrib[pix] = last[k];
    }
}

hipError_t launch_blend_fwd(const Cam& cam, const gs_splat* splats, const uint32_t* values,
                            const uint32_t* tile_ranges, float* image, float* final_T, uint32_t* n_contrib,
                            hipStream_t s)
{
    const int n_tiles = cam.tiles_x * cam.tiles_y;
    hipLaunchKernelGGL(k_blend_fwd<GS_FWD_PIX>, dim3(blend_grid(n_tiles)), dim3(kTile * kTile / GS_FWD_PIX), 0, s,
                       cam, splats, values, tile_ranges, image, final_T, n_contrib);
    return hipGetLastError();
}

// ---- backward -----------------------------------------------------------------
// Per pixel, back to front from its last blended splat, with T recovered as
// T_i = T_{i+1} / (1 - alpha_i) and S the suffix sum of colour * alpha * T plus
// T_final * bg:  dL/dcolour_i = alpha_i T_i g,  dL/dalpha_i = sum_ch
// (T_i c_i - S / (1 - alpha_i)) g_ch. The alpha and skip decisions reuse the
// forward's code, so the same splats are found contributing. Each lane sums
// its pixels, the wave sums its lanes, and lane 63 issues one set of float
// atomics per (wave, splat).

template <int kPix>
__global__ __launch_bounds__(kTile * kTile / kPix) void k_blend_bwd(Cam cam, const gs_splat* __restrict__ splats,
                                                                    const uint32_t* __restrict__ values,
                                                                    const uint32_t* __restrict__ ranges,
                                                                    const float* __restrict__ final_T,
                                                                    const uint32_t* __restrict__ n_contrib,
                                                                    const float* __restrict__ dL_dimage,
                                                                    const uint32_t* __restrict__ order,
                                                                    float* __restrict__ acc)
{
    constexpr int kRowStep = 4;   // pixel k of a lane lies 4k rows below its first
    const int n_tiles = cam.tiles_x * cam.tiles_y;
    const int tile = order ? (blockIdx.x < (unsigned)n_tiles ? (int)order[blockIdx.x] : n_tiles)
                           : tile_of_block(blockIdx.x, n_tiles);
    if (tile >= n_tiles) return;
    const int lane = __lane_id();
    const int tx = tile % cam.tiles_x, ty = tile / cam.tiles_x;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int row_lane = lane & 15;
    // lane bits of the butterfly reduction and the accumulator entry this lane adds
    const bool b0 = lane & 1, b1 = lane & 2, b2 = lane & 4;
    const int entry = (row_lane & 8) ? 8 : 4 * (lane & 1) + 2 * ((lane >> 1) & 1) + ((lane >> 2) & 1);
    const int x = tx * kTile + row_lane;
    const int y0 = ty * kTile + 4 * kPix * wave + (lane >> 4);
    const float px = (float)x + 0.5f;
    const uint32_t start = ranges[2 * tile], len = ranges[2 * tile + 1] - start;
    const int64_t hw = (int64_t)cam.width * cam.height;
    // box of this wave's pixel centres, for the same early skip as the forward
    const float box_cx = (float)(tx * kTile) + 8.f, box_hx = 7.5f;
    const float box_lo = (float)(ty * kTile + 4 * kPix * wave) + 0.5f;
    const float box_hi = box_lo + (float)(4 * kPix - 1);
    const float box_cy = 0.5f * (box_lo + box_hi), box_hy = 0.5f * (box_hi - box_lo);

    // Sg: the suffix sum S projected on the pixel's upstream gradient g, the
    // only form of S the gradient needs
    float T[kPix], py[kPix], g0[kPix], g1[kPix], g2[kPix], Sg[kPix];
    uint32_t last[kPix];
    uint32_t stop = 0;
#pragma unroll
    for (int k = 0; k < kPix; ++k) {
        const int y = y0 + kRowStep * k;
        py[k] = (float)y + 0.5f;
        T[k] = 1.f;
        g0[k] = g1[k] = g2[k] = 0.f;
        last[k] = 0;
        if (x < cam.width && y < cam.height) {
            const int64_t pix = (int64_t)y * cam.width + x;
            T[k] = final_T[pix];
            last[k] = min(n_contrib[pix], len);
            g0[k] = dL_dimage[pix];
            g1[k] = dL_dimage[hw + pix];
            g2[k] = dL_dimage[2 * hw + pix];
        }
        Sg[k] = T[k] * __fmaf_rn(cam.bg[2], g2[k], __fmaf_rn(cam.bg[1], g1[k], cam.bg[0] * g0[k]));
        stop = max(stop, last[k]);
    }
    // list positions [0, stop) can contribute
    for (int o = 32; o > 0; o >>= 1) stop = max(stop, (uint32_t)__shfl_xor((int)stop, o));
    if (stop == 0) return;
    const int nbatch = (int)((stop + kWave - 1) / kWave);
    // each batch of 64 list entries is staged in LDS and read back one record
    // per step at a uniform address (broadcast), as in the forward
    __shared__ float4 stage[kTile * kTile / kPix / kWave][3][kWave];
    __shared__ uint32_t stage_id[kTile * kTile / kPix / kWave][kWave];
    float4 (*st)[kWave] = stage[wave];
    uint32_t* sid = stage_id[wave];
    float4 c0 = make_float4(0.f, 0.f, 0.f, 0.f), c1 = c0, c2 = c0;
    uint32_t cid = 0, nid = 0;   // nid: the list entry of the batch after the prefetched one, loaded a batch early
    {
        const uint32_t p = (uint32_t)(nbatch - 1) * kWave + lane;
        if (p < stop) {
            cid = values[start + p];
            const float4* r = reinterpret_cast<const float4*>(splats + cid);
            c0 = r[0]; c1 = r[1]; c2 = r[2];
        }
        if (nbatch >= 2) nid = values[start + (uint32_t)(nbatch - 2) * kWave + lane];
    }
    for (int bi = nbatch - 1; bi >= 0; --bi) {
        const uint32_t b = (uint32_t)bi * kWave;
        st[0][lane] = c0; st[1][lane] = c1; st[2][lane] = c2;
        sid[lane] = cid;
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        const int cnt = (int)min((uint32_t)kWave, stop - b);
        // a splat that reaches alpha >= 1/255 nowhere in this wave's pixels
        // passes nothing back: each lane tests the record it holds (the
        // conservative bounding box, then the ellipse), and the walk visits only
        // the others, back to front
        uint64_t todo = __ballot(lane < cnt && fabsf(c0.x - box_cx) <= c2.z + box_hx &&
                                 fabsf(c0.y - box_cy) <= c2.w + box_hy &&
                                 ellipse_meets_box(c0.x, c0.y, c0.z, c0.w, c1.x, c2.y, box_cx - box_hx,
                                                   box_cx + box_hx, box_lo, box_hi));
        if (bi > 0) {
            cid = nid;
            const float4* r = reinterpret_cast<const float4*>(splats + cid);
            c0 = r[0]; c1 = r[1]; c2 = r[2];
            if (bi > 1) nid = values[start + b - 2 * kWave + lane];
        }
        while (todo != 0) {
            const int j = 63 - (int)__builtin_clzll(todo);
            todo ^= 1ull << j;
            const uint32_t pos = b + (uint32_t)j;
            SplatReg s;
            {
                const float4 w0 = st[0][j], w1 = st[1][j], w2 = st[2][j];
                s.mx = w0.x; s.my = w0.y; s.ca = w0.z; s.cb = w0.w;
                s.cc = w1.x; s.op = w1.y; s.r = w1.z; s.g = w1.w;
                s.b = w2.x; s.pmin = w2.y;
                s.id = sid[j];
            }
            const float dx = px - s.mx;
            const Quad q = column_quad(s, dx);
            const float pmin2 = s.pmin * kLog2e;
            // per-lane sums over its pixels: colour gradient, opacity gradient, and
            // dL/dpower times 1, dy, dy^2 (the lane's pixels share dx), from which
            // the moments dpow dx, dpow dy, dpow dx^2, dpow dx dy, dpow dy^2 and
            // then dmean2d and dconic follow once per splat
            float a_c0 = 0.f, a_c1 = 0.f, a_c2 = 0.f, a_dop = 0.f;
            float p0 = 0.f, p1 = 0.f, p2 = 0.f;
            bool any = false;
#pragma unroll
            for (int k = 0; k < kPix; ++k) {
                // one branch per pixel; the alpha floor and the cap are selects
                // inside it (the same decisions, fewer exec-mask changes)
                const float dy = py[k] - s.my;
                const float power2 = quad_power(q, dy);
                if (!(pos < last[k] && power2 <= 0.f && power2 >= pmin2)) continue;
                const float G = __builtin_amdgcn_exp2f(power2);
                const float oG = s.op * G;
                const bool on = oG >= kAlphaMin;             // alpha >= 1/255
                const float alpha = on ? fminf(kAlphaMax, oG) : 0.f;
                any = any || on;
                // hardware reciprocal (1 ulp): T is recovered over a few hundred
                // splats, so its relative error stays near 1e-5
                const float inv = __builtin_amdgcn_rcpf(1.f - alpha);
                T[k] *= inv;                                // transmittance in front of this splat
                const float w = alpha * T[k];
                a_c0 = __fmaf_rn(w, g0[k], a_c0);
                a_c1 = __fmaf_rn(w, g1[k], a_c1);
                a_c2 = __fmaf_rn(w, g2[k], a_c2);
                const float cg = __fmaf_rn(s.b, g2[k], __fmaf_rn(s.g, g1[k], s.r * g0[k]));
                const float dalpha = __fmaf_rn(T[k], cg, -inv * Sg[k]);
                Sg[k] = __fmaf_rn(w, cg, Sg[k]);
                // below the cap alpha = o G; capped (or skipped) entries pass nothing
                const bool unc = on && oG < kAlphaMax;
                a_dop = unc ? __fmaf_rn(G, dalpha, a_dop) : a_dop;
                const float dpow = unc ? alpha * dalpha : 0.f;
                const float pdy = dpow * dy;
                p0 += dpow;
                p1 += pdy;
                p2 = __fmaf_rn(pdy, dy, p2);
            }
            if (__ballot(any) == 0) continue;
            // the lane's share of the nine accumulator entries; power = -(a dx^2
            // + c dy^2)/2 - b dx dy with dx = px - mean_x, so dmean2d = (a m_x +
            // b m_y, c m_y + b m_x) and dconic = -(m_xx / 2, m_xy, m_yy / 2)
            const float m_x = dx * p0;
            float v[kAccStride];
            v[0] = __fmaf_rn(s.ca, m_x, s.cb * p1);
            v[1] = __fmaf_rn(s.cc, p1, s.cb * m_x);
            v[2] = -0.5f * dx * m_x;
            v[3] = -dx * p1;
            v[4] = -0.5f * p2;
            v[5] = a_dop;
            v[6] = a_c0;
            v[7] = a_c1;
            v[8] = a_c2;
            // Row sums by butterfly: entries 0..7 halve per exchange (partner
            // lane ^ 1, then ^ 2: each lane keeps half and adds the partner's
            // copy of it), then the four lanes of a row with the same lane % 4
            // are added (rotations by 4 and 8); entry 8 is summed plainly. Lane
            // l < 8 of a row then holds entry bsel(l), lane 8 entry 8, and the
            // four rows are added across.
            float u[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const float keep = b0 ? v[4 + i] : v[i], give = b0 ? v[i] : v[4 + i];
                u[i] = keep + dpp_f32<0xB1>(give);
            }
            float w2[2];
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                const float keep = b1 ? u[2 + i] : u[i], give = b1 ? u[i] : u[2 + i];
                w2[i] = keep + dpp_f32<0x4E>(give);
                w2[i] += dpp_f32<0x124>(w2[i]);
                w2[i] += dpp_f32<0x128>(w2[i]);
            }
            // (the DPP row sum must run in every lane: a disabled source lane
            // reads as zero, so it stays outside any condition)
            const float s8 = row_sum(v[8]);
            float t = b2 ? w2[1] : w2[0];
            t = (row_lane & 8) ? s8 : t;
            t += __shfl_xor(t, 16);
            t += __shfl_xor(t, 32);
            if (lane < kAccStride) atomicAdd(acc + (size_t)s.id * kAccStride + entry, t);
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
}

hipError_t launch_blend_bwd(const Cam& cam, const gs_splat* splats, const uint32_t* values,
                            const uint32_t* tile_ranges, const float* final_T, const uint32_t* n_contrib,
                            const float* dL_dimage, const uint32_t* tile_order, float* acc, hipStream_t s)
{
    const int n_tiles = cam.tiles_x * cam.tiles_y;
    hipLaunchKernelGGL(k_blend_bwd<GS_BWD_PIX>, dim3(tile_order ? n_tiles : blend_grid(n_tiles)),
                       dim3(kTile * kTile / GS_BWD_PIX), 0, s, cam, splats, values, tile_ranges, final_T, n_contrib,
                       dL_dimage, tile_order, acc);
    return hipGetLastError();
}

// ---- tile order of the backward -----------------------------------------------
// The backward's work in a tile follows the longest walk among its pixels (the
// list up to the last entry any of them blended), and that walk differs by a
// factor of 3 or more between tiles. Workgroups are dispatched in launch order
// and every tile's workgroup is resident at once, so each SIMD gets every
// 1024th tile of the launch order: in list order its share of long walks
// varies, and the SIMD with the most sets the kernel's duration. Launching
// the tiles longest walk first deals each SIMD one tile of every length class.
// The order is taken by a counting sort over 16 classes per octave of the walk
// length; tiles of one class come out in no fixed order (the results do not
// depend on it, beyond the float atomics' summation order).

__device__ __forceinline__ uint32_t walk_class(uint32_t walk)
{
    // exponent and the 4 leading mantissa bits of the walk length as a float:
    // 16 classes per octave, 0 .. kWalkClasses - 1 (walks of 0 and 1 share class 0)
    const uint32_t b = __float_as_uint((float)max(walk, 1u)) >> 19;
    return min(b - (127u << 4), (uint32_t)kWalkClasses - 1);   // 2^32 - 1 rounds up to 2^32
}

// Walk class of each tile, one wave per tile (workgroup `blk` of the walk).
__device__ __forceinline__ void tile_walk(const Cam& cam, const uint32_t* __restrict__ ranges,
                                          const uint32_t* __restrict__ n_contrib, uint32_t* __restrict__ walk_cls,
                                          int blk)
{
    const int n_tiles = cam.tiles_x * cam.tiles_y;
    const int tile = blk * (kBlock / kWave) + (int)(threadIdx.x / kWave);
    if (tile >= n_tiles) return;   // whole waves
    const int lane = __lane_id();
    const int tx = tile % cam.tiles_x, ty = tile / cam.tiles_x;
    const int x = tx * kTile + (lane & 15);
    uint32_t walk = 0;
#pragma unroll
    for (int k = 0; k < kTile / 4; ++k) {
        const int y = ty * kTile + (lane >> 4) + 4 * k;
        if (x < cam.width && y < cam.height) walk = max(walk, n_contrib[(int64_t)y * cam.width + x]);
    }
    for (int o = 32; o > 0; o >>= 1) walk = max(walk, (uint32_t)__shfl_xor((int)walk, o));
    if (lane == 0) walk_cls[tile] = walk_class(min(walk, ranges[2 * tile + 1] - ranges[2 * tile]));
}

// Zeroes p[0, count) as workgroup `blk` of `nblk` (16-byte stores, grid-stride).
__device__ __forceinline__ void clear_part(float* __restrict__ p, int64_t count, int blk, int nblk)
{
    const int64_t c4 = count >> 2;
    const int64_t stride = (int64_t)nblk * kBlock;
    float4* p4 = reinterpret_cast<float4*>(p);
    for (int64_t i = (int64_t)blk * kBlock + threadIdx.x; i < c4; i += stride) p4[i] = make_float4(0.f, 0.f, 0.f, 0.f);
    if (blk == 0 && threadIdx.x < (count & 3)) p[(c4 << 2) + threadIdx.x] = 0.f;
}

// The backward's preparation in one launch: the first walk_blocks workgroups
// take the tiles' walk classes (none when the tiles are not ordered), the
// others clear the screen-space accumulators.
__global__ __launch_bounds__(kBlock) void k_walk_clear(Cam cam, const uint32_t* __restrict__ ranges,
                                                       const uint32_t* __restrict__ n_contrib,
                                                       uint32_t* __restrict__ walk_cls, int walk_blocks,
                                                       float* __restrict__ acc, int64_t count)
{
    const int blk = (int)blockIdx.x;
    if (blk < walk_blocks)
        tile_walk(cam, ranges, n_contrib, walk_cls, blk);
    else
        clear_part(acc, count, blk - walk_blocks, (int)gridDim.x - walk_blocks);
}

constexpr int kOrderThreads = 1024;

__global__ __launch_bounds__(kOrderThreads) void k_tile_order(int n_tiles, const uint32_t* __restrict__ walk_cls,
                                                              uint32_t* __restrict__ order)
{
    __shared__ uint32_t cnt[kWalkClasses];
    __shared__ uint32_t scan[2][kWalkClasses];
    const int t = threadIdx.x;
    for (int c = t; c < kWalkClasses; c += kOrderThreads) cnt[c] = 0;
    __syncthreads();
    for (int i = t; i < n_tiles; i += kOrderThreads) atomicAdd(&cnt[walk_cls[i]], 1u);
    __syncthreads();
    // first position of each class, the longest class first: the sum of the
    // counts of all longer classes (inclusive scan over the reversed classes)
    int src = 0;
    for (int c = t; c < kWalkClasses; c += kOrderThreads) scan[0][c] = cnt[kWalkClasses - 1 - c];
    __syncthreads();
    for (int d = 1; d < kWalkClasses; d <<= 1) {
        for (int c = t; c < kWalkClasses; c += kOrderThreads)
            scan[src ^ 1][c] = scan[src][c] + (c >= d ? scan[src][c - d] : 0u);
        __syncthreads();
        src ^= 1;
    }
    for (int c = t; c < kWalkClasses; c += kOrderThreads) {
        const int r = kWalkClasses - 1 - c;   // reversed index of class c
        cnt[c] = scan[src][r] - cnt[c];       // counts of the classes above c
    }
    __syncthreads();
    for (int i = t; i < n_tiles; i += kOrderThreads) order[atomicAdd(&cnt[walk_cls[i]], 1u)] = (uint32_t)i;
}

bool tile_order_supported(const Cam& cam) { return (int64_t)cam.tiles_x * cam.tiles_y <= kMaxOrderedTiles; }

hipError_t launch_bwd_prep(const Cam& cam, const uint32_t* tile_ranges, const uint32_t* n_contrib, float* acc,
                           int64_t acc_count, uint32_t* walk_cls, uint32_t* order, hipStream_t s)
{
    const int n_tiles = cam.tiles_x * cam.tiles_y;
    const int walk_blocks = order ? (int)div_up(n_tiles, kBlock / kWave) : 0;
    const int clear_blocks = (int)std::min<int64_t>(std::max<int64_t>(div_up(acc_count >> 2, kBlock), 1), 4096);
    hipLaunchKernelGGL(k_walk_clear, dim3((unsigned)(walk_blocks + clear_blocks)), dim3(kBlock), 0, s, cam,
                       tile_ranges, n_contrib, walk_cls, walk_blocks, acc, acc_count);
    if (order) hipLaunchKernelGGL(k_tile_order, dim3(1), dim3(kOrderThreads), 0, s, n_tiles, walk_cls, order);
    return hipGetLastError();
}

// ---- work counts (measurement) ------------------------------------------------
// Walks every pixel's list with the forward's decisions (the same fp32
// operations as k_blend_fwd) and counts, per pixel: entries blended; entries
// evaluated in the forward (up to the stop entry, or the list's end, whose
// alpha >= 1/255 box meets the tile: the blend kernels skip the others for
// the whole tile without a per-pixel test); evaluated entries before the last
// blended one (those the backward evaluates); that last position
// (n_contrib); and the entries the method visits in the forward (up to and
// including the stop entry, or the whole list). One wave per tile, 4 pixels
// per lane; per-wave sums, then one 64-bit atomic per wave and counter.
__global__ __launch_bounds__(kWave) void k_blend_count(Cam cam, const gs_splat* __restrict__ splats,
                                                       const uint32_t* __restrict__ values,
                                                       const uint32_t* __restrict__ ranges,
                                                       unsigned long long* __restrict__ counts)
{
    constexpr int kPix = 4, kRowStep = 4;
    const int n_tiles = cam.tiles_x * cam.tiles_y;
    const int tile = blockIdx.x;
    if (tile >= n_tiles) return;
    const int lane = __lane_id();
    const int tx = tile % cam.tiles_x, ty = tile / cam.tiles_x;
    const int x = tx * kTile + (lane & 15);
    const int y0 = ty * kTile + (lane >> 4);
    const float px = (float)x + 0.5f;
    const uint32_t start = ranges[2 * tile], end = ranges[2 * tile + 1];
    const float box_cx = (float)(tx * kTile) + 8.f, box_hx = 7.5f;
    const float box_cy = (float)(ty * kTile) + 8.f, box_hy = 7.5f;
    float T[kPix], py[kPix];
    uint32_t blended[kPix], eval_fwd[kPix], eval_bwd[kPix], pending[kPix], last[kPix], walked[kPix];
#pragma unroll
    for (int k = 0; k < kPix; ++k) {
        py[k] = (float)(y0 + kRowStep * k) + 0.5f;
        T[k] = (x < cam.width && (y0 + kRowStep * k) < cam.height) ? 1.f : -1.f;
        blended[k] = eval_fwd[k] = eval_bwd[k] = pending[k] = last[k] = walked[k] = 0;
    }
    for (uint32_t p = start; p < end; ++p) {
#pragma unroll
        for (int k = 0; k < kPix; ++k) walked[k] += T[k] > 0.f ? 1u : 0u;   // visited while blending
        const float4* rec = reinterpret_cast<const float4*>(splats + values[p]);
        const float4 w0 = rec[0], w1 = rec[1], w2 = rec[2];
        SplatReg s;
        s.mx = w0.x; s.my = w0.y; s.ca = w0.z; s.cb = w0.w; s.cc = w1.x; s.op = w1.y;
        s.pmin = w2.y; s.ex = w2.z; s.ey = w2.w;
        if (!(fabsf(s.mx - box_cx) <= s.ex + box_hx && fabsf(s.my - box_cy) <= s.ey + box_hy)) continue;
        const float dx = px - s.mx;
        const Quad q = column_quad(s, dx);
        const float pmin2 = s.pmin * kLog2e;
#pragma unroll
        for (int k = 0; k < kPix; ++k) {
            if (!(T[k] > 0.f)) continue;
            ++eval_fwd[k];
            const float power2 = quad_power(q, py[k] - s.my);
            if (!(power2 <= 0.f && power2 >= pmin2)) { ++pending[k]; continue; }
            const float alpha = fminf(kAlphaMax, s.op * __builtin_amdgcn_exp2f(power2));
            if (!(alpha >= kAlphaMin)) { ++pending[k]; continue; }
            const float Tn = T[k] * (1.f - alpha);
            if (Tn < kTMin) { T[k] = -T[k]; continue; }
            T[k] = Tn;
            ++blended[k];
            eval_bwd[k] += pending[k] + 1;
            pending[k] = 0;
            last[k] = p - start + 1;
        }
    }
    unsigned long long c[5] = {0, 0, 0, 0, 0};
#pragma unroll
    for (int k = 0; k < kPix; ++k) {
        if (x >= cam.width || y0 + kRowStep * k >= cam.height) continue;
        c[0] += blended[k];
        c[1] += last[k];
        c[2] += eval_bwd[k];
        c[3] += eval_fwd[k];
        c[4] += walked[k];
    }
#pragma unroll
    for (int i = 0; i < 5; ++i) {
        unsigned long long v = c[i];
        for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
        if (lane == 0) atomicAdd(counts + i, v);
    }
}

hipError_t launch_blend_count(const Cam& cam, const gs_splat* splats, const uint32_t* values,
                              const uint32_t* tile_ranges, uint64_t* counts, hipStream_t s)
{
    hipError_t e = launch_fill_u32(reinterpret_cast<uint32_t*>(counts), 10, 0u, s);
    if (e != hipSuccess) return e;
    const int n_tiles = cam.tiles_x * cam.tiles_y;
    hipLaunchKernelGGL(k_blend_count, dim3(n_tiles), dim3(kWave), 0, s, cam, splats, values, tile_ranges,
                       reinterpret_cast<unsigned long long*>(counts));
    return hipGetLastError();
}

// Zero fill of `count` floats; p must be 16-byte aligned. Body in float4, tail
// in scalars. A kernel rather than a memset so that it behaves the same inside
// a captured graph.
__global__ __launch_bounds__(kBlock) void k_clear(float* __restrict__ p, int64_t count)
{
    clear_part(p, count, (int)blockIdx.x, (int)gridDim.x);
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
