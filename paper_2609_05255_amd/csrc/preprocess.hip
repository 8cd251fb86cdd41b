// Preprocess (Sec. 3.1) with the appearance fused in (appendix, fused rasterizer):
// one thread per Gaussian, planar coalesced parameter reads, culling, EWA
// projection, tile rectangle, colour for survivors only, and the per-block tile
// counts from which the number of pairs follows.
//
// The whole file is compiled without floating-point contraction: the tile
// rectangle and the depth key are integers decided by this fp32 arithmetic,
// and they must not depend on which multiply-adds the compiler fuses.
#include <type_traits>

#include "gs_internal.h"
#include "mlp.h"
#include "lobe.h"
#include "neural.h"
#include "sh.h"

#pragma clang fp contract(off)

namespace gsr {

namespace {

struct Geo {
    bool visible, clamp_x, clamp_y;
    float mx, my, ca, cb, cc, op, depth;
    float var_x, var_y;     // diagonal of the screen-space covariance (with the low-pass)
    int x0, y0, x1, y1;
    uint32_t tiles;
};

__device__ __forceinline__ float clampf(float v, float lo, float hi) { return v < lo ? lo : (v > hi ? hi : v); }

// Activation, projection, EWA covariance with a 0.3 px^2 low-pass, 3-sigma
// rectangle. Operation order is fixed (see the file comment).
__device__ __forceinline__ void geometry(const Cam& c, const float mu[3], const float ls[3], const float q[4],
                                         float logit, Geo& g)
{
    g.visible = false;
    g.clamp_x = g.clamp_y = false;
    g.tiles = 0;
    float s[3];
    for (int j = 0; j < 3; ++j) s[j] = (float)exp((double)ls[j]);
    const float op = (float)(1.0 / (1.0 + exp(-(double)logit)));

    const float qn = sqrtf(((q[0] * q[0] + q[1] * q[1]) + q[2] * q[2]) + q[3] * q[3]);
    const float w = q[0] / qn, x = q[1] / qn, y = q[2] / qn, z = q[3] / qn;
    float R[9];
    R[0] = 1.f - 2.f * (y * y + z * z); R[1] = 2.f * (x * y - w * z);       R[2] = 2.f * (x * z + w * y);
    R[3] = 2.f * (x * y + w * z);       R[4] = 1.f - 2.f * (x * x + z * z); R[5] = 2.f * (y * z - w * x);
    R[6] = 2.f * (x * z - w * y);       R[7] = 2.f * (y * z + w * x);       R[8] = 1.f - 2.f * (x * x + y * y);
    float M[9];
#pragma unroll
    for (int r = 0; r < 3; ++r)
#pragma unroll
        for (int k = 0; k < 3; ++k) M[3 * r + k] = R[3 * r + k] * s[k];
    float S[9];
#pragma unroll
    for (int r = 0; r < 3; ++r)
#pragma unroll
        for (int k = 0; k < 3; ++k)
            S[3 * r + k] = (M[3 * r + 0] * M[3 * k + 0] + M[3 * r + 1] * M[3 * k + 1]) + M[3 * r + 2] * M[3 * k + 2];

    float t[3];
#pragma unroll
    for (int r = 0; r < 3; ++r) t[r] = ((c.V[4 * r + 0] * mu[0] + c.V[4 * r + 1] * mu[1]) + c.V[4 * r + 2] * mu[2]) + c.V[4 * r + 3];
    if (!(t[2] > c.near_plane)) return;

    const float limx = 1.3f * ((0.5f * (float)c.width) / c.fx);
    const float limy = 1.3f * ((0.5f * (float)c.height) / c.fy);
    const float txtz = t[0] / t[2], tytz = t[1] / t[2];
    float ux = txtz, uy = tytz;
    if (ux < -limx) { ux = -limx; g.clamp_x = true; }
    if (ux > limx) { ux = limx; g.clamp_x = true; }
    if (uy < -limy) { uy = -limy; g.clamp_y = true; }
    if (uy > limy) { uy = limy; g.clamp_y = true; }
    ux = ux * t[2];
    uy = uy * t[2];
    const float tz2 = t[2] * t[2];
    const float j00 = c.fx / t[2], j02 = -(c.fx * ux) / tz2;
    const float j11 = c.fy / t[2], j12 = -(c.fy * uy) / tz2;
    float T[6];
#pragma unroll
    for (int k = 0; k < 3; ++k) {
        T[k] = j00 * c.V[0 + k] + j02 * c.V[8 + k];
        T[3 + k] = j11 * c.V[4 + k] + j12 * c.V[8 + k];
    }
    float A[6];
#pragma unroll
    for (int r = 0; r < 2; ++r)
#pragma unroll
        for (int k = 0; k < 3; ++k)
            A[3 * r + k] = (T[3 * r + 0] * S[0 + k] + T[3 * r + 1] * S[3 + k]) + T[3 * r + 2] * S[6 + k];
    float c00 = (A[0] * T[0] + A[1] * T[1]) + A[2] * T[2];
    const float c01 = (A[0] * T[3] + A[1] * T[4]) + A[2] * T[5];
    float c11 = (A[3] * T[3] + A[4] * T[4]) + A[5] * T[5];
    c00 = c00 + 0.3f;
    c11 = c11 + 0.3f;
    const float det = c00 * c11 - c01 * c01;
    if (!(det > 0.f)) return;
    g.ca = c11 / det;
    g.cb = -c01 / det;
    g.cc = c00 / det;
    g.var_x = c00;
    g.var_y = c11;

    const float mid = 0.5f * (c00 + c11);
    float disc = mid * mid - det;
    if (disc < 0.1f) disc = 0.1f;
    const float lam = mid + sqrtf(disc);
    const float rad = ceilf(3.f * sqrtf(lam));

    const float px = c.fx * txtz + c.cx, py = c.fy * tytz + c.cy;
    const float tx = (float)c.tiles_x, ty = (float)c.tiles_y;
    const float fx0 = clampf(floorf((px - rad) / 16.f), 0.f, tx);
    const float fx1 = clampf(ceilf((px + rad) / 16.f), 0.f, tx);
    const float fy0 = clampf(floorf((py - rad) / 16.f), 0.f, ty);
    const float fy1 = clampf(ceilf((py + rad) / 16.f), 0.f, ty);
    g.x0 = (int)fx0; g.x1 = (int)fx1; g.y0 = (int)fy0; g.y1 = (int)fy1;
    const int tiles = (g.x1 - g.x0) * (g.y1 - g.y0);
    if (tiles <= 0) return;
    g.tiles = (uint32_t)tiles;
    g.visible = true;
    g.mx = px;
    g.my = py;
    g.op = op;
    g.depth = t[2];
}

struct PreArgs {
    Cam cam;
    int n;
    const float* means;
    const float* log_scales;
    const float* quats;
    const float* logits;
    int sh_degree;
    const float* sh;
    const uint16_t* latent;
    const uint16_t* mlp_w;
    const float* base_color;
    const uint16_t* features;
    const uint16_t* preact;
    const float* lobes;
    int sh_y0_folded;
    gs_splat* splats;
    float* color_jac;
    uint32_t* tiles_touched;
    uint32_t* depth_key;
    uint32_t* block_pairs;
};

// Early-skip fields of the blend: alpha = min(0.99, o e^power) stays below
// 1/255 wherever power < -ln(255 o), so power_min takes that bound less a
// margin of 1e-3 (far above the rounding of either side); the pixels with
// power >= power_min lie in the ellipse d^T Q d <= -2 power_min, whose bounding
// box has half extents sqrt(-2 power_min Sigma_xx), sqrt(-2 power_min Sigma_yy),
// enlarged by 0.1% + 0.01 px.
__device__ __forceinline__ void skip_fields(const Geo& g, float& pmin, float& ex, float& ey)
{
    if (!(255.f * g.op > 1.f)) {
        pmin = __builtin_inff();
        ex = ey = -1e30f;
        return;
    }
    pmin = -logf(255.f * g.op) - 1e-3f;
    const float r2 = -2.f * pmin;
    ex = sqrtf(r2 * g.var_x) * 1.001f + 0.01f;
    ey = sqrtf(r2 * g.var_y) * 1.001f + 0.01f;
}

// Per-wave staging of the 64 splat records of a wave (4 KB).
struct SplatStage {
    float4 q[kWave * 4];
};

// Writes the wave's 64 consecutive records (Gaussians first .. first + 63)
// through LDS, so that each store instruction covers 1 KB of contiguous
// memory instead of 16 bytes at a 64-byte stride. Culled Gaussians get a zero
// record. Called by all lanes of the wave.
__device__ __forceinline__ void store_splats_wave(gs_splat* __restrict__ splats, int64_t n, int64_t first,
                                                  SplatStage& st, const Geo& g, const float col[3])
{
    const int l = __lane_id();
    float4 r0 = make_float4(0.f, 0.f, 0.f, 0.f), r1 = r0, r2 = r0, r3 = r0;
    if (g.visible) {
        float pmin, ex, ey;
        skip_fields(g, pmin, ex, ey);
        r0 = make_float4(g.mx, g.my, g.ca, g.cb);
        r1 = make_float4(g.cc, g.op, col[0], col[1]);
        r2 = make_float4(col[2], pmin, ex, ey);
        const uint32_t r01 = (uint32_t)(g.x0 & 0xFFFF) | ((uint32_t)g.y0 << 16);
        const uint32_t r23 = (uint32_t)(g.x1 & 0xFFFF) | ((uint32_t)g.y1 << 16);
        r3 = make_float4(__uint_as_float(r01), __uint_as_float(r23), g.depth, 0.f);
    }
    st.q[4 * l] = r0;
    st.q[4 * l + 1] = r1;
    st.q[4 * l + 2] = r2;
    st.q[4 * l + 3] = r3;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    float4* dst = reinterpret_cast<float4*>(splats + first);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const int e = kWave * k + l;          // 16-byte piece of the wave's 4 KB
        if (first + (e >> 2) < n) dst[e] = st.q[e];
    }
}

// Sum of a u32 over the wave, in every lane.
__device__ __forceinline__ uint32_t wave_sum_u32(uint32_t v)
{
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    return v;
}

// Sum of a u32 over the workgroup; result valid in thread 0.
__device__ __forceinline__ uint32_t block_sum_u32(uint32_t v, uint32_t* lds4)
{
    v = wave_sum_u32(v);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    if (lane == 0) lds4[wave] = v;
    __syncthreads();
    uint32_t r = 0;
    if (threadIdx.x == 0) r = lds4[0] + lds4[1] + lds4[2] + lds4[3];
    return r;
}

// Read once per frame: non-temporal loads, which leave the caches to the data
// that the sort and the blend read again.
__device__ __forceinline__ void load_geometry_params(const PreArgs& a, int i, float mu[3], float ls[3], float q[4],
                                                     float& logit)
{
    const int64_t n = a.n;
    for (int j = 0; j < 3; ++j) mu[j] = __builtin_nontemporal_load(&a.means[j * n + i]);
    for (int j = 0; j < 3; ++j) ls[j] = __builtin_nontemporal_load(&a.log_scales[j * n + i]);
    for (int j = 0; j < 4; ++j) q[j] = __builtin_nontemporal_load(&a.quats[j * n + i]);
    logit = __builtin_nontemporal_load(&a.logits[i]);
}

__device__ __forceinline__ void view_dir(const Cam& c, const float mu[3], float d[3])
{
    const float vx = mu[0] - c.campos[0], vy = mu[1] - c.campos[1], vz = mu[2] - c.campos[2];
    const float len = sqrtf(vx * vx + vy * vy + vz * vz);
    d[0] = vx / len;
    d[1] = vy / len;
    d[2] = vz / len;
}

}  // namespace

// eq. sh_color_eval: c = max(0, 0.5 + sum over bands <= kDeg of Y_k(d) sh_k),
// with Y_0 = 1 when the stored DC coefficients have Y0 folded in.
// All coefficient loads are issued together, before the sums need them; the
// sums are explicit fused multiply-adds so that sh_color_jac matches them.
template <int kDeg>
__device__ __forceinline__ void sh_color(const float* __restrict__ sh, int64_t n, int i, const float d[3],
                                         bool y0_folded, float col[3])
{
    constexpr int nb = (kDeg + 1) * (kDeg + 1);
    float c[3 * nb];
#pragma unroll
    for (int k = 0; k < 3 * nb; ++k) c[k] = __builtin_nontemporal_load(sh + (int64_t)k * n + i);
    float Y[16];
    sh_basis16(d[0], d[1], d[2], Y);
    if (y0_folded) Y[0] = 1.f;
#pragma unroll
    for (int ch = 0; ch < 3; ++ch) {
        float acc = 0.5f;
#pragma unroll
        for (int k = 0; k < nb; ++k) acc = fmaf(Y[k], c[3 * k + ch], acc);
        col[ch] = acc > 0.f ? acc : 0.f;
    }
}

// sh_color, and with it what the backward needs of the colour's dependence on
// the view direction: jac[3 c + j] = d(0.5 + sum_k Y_k sh_k[c]) / d d_j over
// the active bands, and the channels above zero as bits of `unclamped`.
template <int kDeg>
__device__ __forceinline__ void sh_color_jac(const float* __restrict__ sh, int64_t n, int i, const float d[3],
                                             bool y0_folded, float col[3], float jac[9], uint32_t& unclamped)
{
    constexpr int nb = (kDeg + 1) * (kDeg + 1);
    float c[3 * nb];
#pragma unroll
    for (int k = 0; k < 3 * nb; ++k) c[k] = __builtin_nontemporal_load(sh + (int64_t)k * n + i);
    float Y[16];
    sh_basis16(d[0], d[1], d[2], Y);
    if (y0_folded) Y[0] = 1.f;
    unclamped = 0u;
#pragma unroll
    for (int ch = 0; ch < 3; ++ch) {
        float acc = 0.5f;
#pragma unroll
        for (int k = 0; k < nb; ++k) acc = fmaf(Y[k], c[3 * k + ch], acc);   // as sh_color, bit for bit
        col[ch] = acc > 0.f ? acc : 0.f;
        unclamped |= acc > 0.f ? 1u << ch : 0u;
    }
    sh_color_jacobian(d[0], d[1], d[2], c, nb, jac);   // Y_0 is constant: k >= 1 only
}

template <int kDeg>
__global__ __launch_bounds__(kBlock) void k_preprocess_sh3(PreArgs a)
{
    __shared__ uint32_t red[4];
    __shared__ SplatStage stage[kBlock / kWave];
    const int i = blockIdx.x * kBlock + threadIdx.x;
    uint32_t tiles = 0;
    Geo g;
    g.visible = false;
    float col[3] = {0.f, 0.f, 0.f};
    if (i < a.n) {
        float mu[3], ls[3], q[4], logit;
        load_geometry_params(a, i, mu, ls, q, logit);
        geometry(a.cam, mu, ls, q, logit, g);
        if (g.visible) {
            float d[3];
            view_dir(a.cam, mu, d);
            if (a.color_jac) {
                float jac[9];
                uint32_t unclamped;
                sh_color_jac<kDeg>(a.sh, a.n, i, d, a.sh_y0_folded != 0, col, jac, unclamped);
                const int64_t n = a.n;
#pragma unroll
                for (int r = 0; r < 9; ++r) __builtin_nontemporal_store(jac[r], a.color_jac + r * n + i);
                __builtin_nontemporal_store(__uint_as_float(unclamped), a.color_jac + 9 * n + i);
            } else {
                sh_color<kDeg>(a.sh, a.n, i, d, a.sh_y0_folded != 0, col);
            }
            tiles = g.tiles;
        }
        a.tiles_touched[i] = tiles;
        a.depth_key[i] = g.visible ? __float_as_uint(g.depth) : 0xFFFFFFFFu;
    }
    store_splats_wave(a.splats, a.n, (int64_t)i - __lane_id(), stage[threadIdx.x >> 6], g, col);
    const uint32_t total = block_sum_u32(tiles, red);
    if (threadIdx.x == 0) a.block_pairs[blockIdx.x] = total;
}

// NASG / NASGabor (eq. nasg, lobe.h): one thread per Gaussian, colour
// max(0, c0 + G(d) tanh(amplitude) + 0.5), or max(0, c0 + 0.5) while the
// active degree is 0; a culled Gaussian reads no appearance.
template <bool kGabor>
__global__ __launch_bounds__(kBlock) void k_preprocess_lobe(PreArgs a)
{
    __shared__ uint32_t red[4];
    __shared__ SplatStage stage[kBlock / kWave];
    const int i = blockIdx.x * kBlock + threadIdx.x;
    uint32_t tiles = 0;
    Geo g;
    g.visible = false;
    float col[3] = {0.f, 0.f, 0.f};
    if (i < a.n) {
        float mu[3], ls[3], q[4], logit;
        load_geometry_params(a, i, mu, ls, q, logit);
        geometry(a.cam, mu, ls, q, logit, g);
        if (g.visible) {
            const int64_t n = a.n;
            float c0[3], res[3] = {0.f, 0.f, 0.f};
#pragma unroll
            for (int ch = 0; ch < 3; ++ch) c0[ch] = a.base_color[ch * n + i];
            if (a.sh_degree >= 1) {
                float r[6], amp[3];
#pragma unroll
                for (int k = 0; k < 5; ++k) r[k] = a.lobes[k * n + i];
#pragma unroll
                for (int ch = 0; ch < 3; ++ch) amp[ch] = a.lobes[(5 + ch) * n + i];
                r[5] = kGabor ? a.lobes[8 * n + i] : 0.f;
                float d[3];
                view_dir(a.cam, mu, d);
                LobeEval f;
                lobe_setup<kGabor>(r, f);
                const float G = lobe_value<kGabor>(f, d);
#pragma unroll
                for (int ch = 0; ch < 3; ++ch) res[ch] = G * tanhf(amp[ch]);
            }
#pragma unroll
            for (int ch = 0; ch < 3; ++ch) {
                const float v = c0[ch] + res[ch] + 0.5f;
                col[ch] = v > 0.f ? v : 0.f;
            }
            tiles = g.tiles;
        }
        a.tiles_touched[i] = tiles;
        a.depth_key[i] = g.visible ? __float_as_uint(g.depth) : 0xFFFFFFFFu;
    }
    store_splats_wave(a.splats, a.n, (int64_t)i - __lane_id(), stage[threadIdx.x >> 6], g, col);
    const uint32_t total = block_sum_u32(tiles, red);
    if (threadIdx.x == 0) a.block_pairs[blockIdx.x] = total;
}

// Latent + MLP: geometry per thread, then each wave decodes the colours of its
// visible Gaussians on the matrix cores, 16 at a time (mlp.h); tiles of 16
// lanes without a visible Gaussian are skipped. Each wave loops over chunks of
// 64 Gaussians on its own (no workgroup barrier after the weight fragments are
// staged), and issues a chunk's latent loads before its geometry, so that
// their latency hides behind the projection arithmetic.
__global__ __launch_bounds__(kBlock, 4) void k_preprocess_latent(PreArgs a)
{
    __shared__ MlpFrags W;
    __shared__ SplatStage stage[kBlock / kWave];
    mlp_load_frags(a.mlp_w, W, false);
    const int lane = __lane_id(), wave = threadIdx.x >> 6;
    const int64_t nchunks = div_up((int64_t)a.n, kWave);
    const int64_t stride = (int64_t)gridDim.x * (kBlock / kWave);
    uint64_t wave_tiles = 0;   // the pairs of this wave's chunks
    for (int64_t chunk = (int64_t)blockIdx.x * (kBlock / kWave) + wave; chunk < nchunks; chunk += stride) {
        const int64_t base = chunk * kWave;
        const int i = (int)(base + lane);
        MlpLatentRaw raw;
        mlp_latent_raw(a.latent, a.n, base, raw);
        uint32_t tiles = 0;
        Geo g;
        g.visible = false;
        float d[3] = {0.f, 0.f, 0.f};
        if (i < a.n) {
            float mu[3], ls[3], q[4], logit;
            load_geometry_params(a, i, mu, ls, q, logit);
            geometry(a.cam, mu, ls, q, logit, g);
            if (g.visible) {
                tiles = g.tiles;
                view_dir(a.cam, mu, d);
            }
            a.tiles_touched[i] = tiles;
            a.depth_key[i] = g.visible ? __float_as_uint(g.depth) : 0xFFFFFFFFu;
        }
        const uint64_t vis = __ballot(g.visible);
        float col[3] = {0.f, 0.f, 0.f};
        for (int t = 0; t < kWave / 16; ++t) {
            if (((vis >> (16 * t)) & 0xFFFFull) == 0) continue;
            const half8_t x = mlp_frag_from_raw(raw, t, d);
            float4_t h1[2], h2[2], o;
            half8_t a1, a2;
            mlp_tile_fwd(W, x, h1, a1, h2, a2, o);
            mlp_tile_colors(o, t, col);
        }
        store_splats_wave(a.splats, a.n, base, stage[wave], g, col);
        wave_tiles += __builtin_amdgcn_readfirstlane(wave_sum_u32(tiles));   // uniform: kept in scalar registers
    }
    // one tile sum per wave of the grid (zero for a wave without a chunk),
    // saturated: 2^32 - 1 stands for that many pairs or more
    if (lane == 0) a.block_pairs[blockIdx.x * (kBlock / kWave) + wave] = (uint32_t)min(wave_tiles, (uint64_t)0xFFFFFFFFu);
}

// The paper's neural appearance (neural.h): geometry per thread; each lane
// stages its decoder input (SH basis of its direction up to the active degree,
// sin and cos of its 8 features); the wave decodes its visible Gaussians 16 at
// a time on the matrix cores; colour max(0, c0 + tanh(MLP(x)) + 0.5), or
// max(0, c0 + 0.5) while the active degree is 0. Waves loop over 64-Gaussian
// chunks on their own, the base colour and feature loads issued before the
// geometry. kFolded: the render-only folded form, whose first layer adds the
// stored pre-activations of the view-independent inputs to the direction
// columns' product (no features, no sin/cos). L hidden layers; kRaw: 16 raw
// features as the feature inputs (the architecture table's configurations).
template <bool kFolded, int L, bool kRaw, int kW = 16>
__global__ __launch_bounds__(kBlock, kW == 32 ? 3 : 4) void k_preprocess_neural(PreArgs a)
{
    static_assert(kW == 16 || (kW == 32 && L == 2 && !kRaw && !kFolded), "the 32-neuron configuration is 32-32-32-3");
    constexpr int kF = kRaw ? 16 : GS_NEURAL_FEATURES;
    using Frags = std::conditional_t<kW == 32, MlpFrags, NeuralFrags<L>>;
    __shared__ Frags W;
    __shared__ NeuralInStage XS[kBlock / kWave];
    __shared__ SplatStage stage[kBlock / kWave];
    const bool resid = a.sh_degree >= 1;
    if (resid) neural_load_frags(a.mlp_w, W, false, kFolded);
    const int lane = __lane_id(), wave = threadIdx.x >> 6;
    const int64_t nchunks = div_up((int64_t)a.n, kWave);
    const int64_t stride = (int64_t)gridDim.x * (kBlock / kWave);
    uint64_t wave_tiles = 0;   // the pairs of this wave's chunks
    for (int64_t chunk = (int64_t)blockIdx.x * (kBlock / kWave) + wave; chunk < nchunks; chunk += stride) {
        const int64_t base = chunk * kWave;
        const int i = (int)(base + lane);
        // appearance loads first, so that they overlap the projection
        float c0[3] = {0.f, 0.f, 0.f}, f[kF];
        half4_t p4[kWave / 16];   // folded: neurons 4g..4g+3 of Gaussian base + 16t + c
#pragma unroll
        for (int j = 0; j < kF; ++j) f[j] = 0.f;
#pragma unroll
        for (int t = 0; t < kWave / 16; ++t) p4[t] = half4_t{0, 0, 0, 0};
        if (i < a.n) {
#pragma unroll
            for (int ch = 0; ch < 3; ++ch) c0[ch] = a.base_color[(int64_t)ch * a.n + i];
            if (resid && !kFolded)
#pragma unroll
                for (int j = 0; j < kF; ++j) f[j] = (float)half_of_bits(a.features[(int64_t)j * a.n + i]);
        }
        if (resid && kFolded) {
            const int g4 = lane >> 4, c = lane & 15;
#pragma unroll
            for (int t = 0; t < kWave / 16; ++t) {
                const int64_t gi = base + 16 * t + c;
                if (gi < a.n) p4[t] = *reinterpret_cast<const half4_t*>(a.preact + gi * 16 + 4 * g4);
            }
        }
        uint32_t tiles = 0;
        Geo g;
        g.visible = false;
        float d[3] = {0.f, 0.f, 0.f};
        if (i < a.n) {
            float mu[3], ls[3], q[4], logit;
            load_geometry_params(a, i, mu, ls, q, logit);
            geometry(a.cam, mu, ls, q, logit, g);
            if (g.visible) {
                tiles = g.tiles;
                view_dir(a.cam, mu, d);
            }
            a.tiles_touched[i] = tiles;
            a.depth_key[i] = g.visible ? __float_as_uint(g.depth) : 0xFFFFFFFFu;
        }
        float res[3] = {0.f, 0.f, 0.f};
        if (resid) {
            if (kFolded) {
                neural_stage_dir(XS[wave].x, g.visible, d, a.sh_degree);
            } else {
                half4_t fq[4];
                if (kRaw) {
                    neural_raw_inputs(f, fq);
                } else {
                    float sf[GS_NEURAL_FEATURES], cf[GS_NEURAL_FEATURES];
                    neural_encode_features(f, sf, cf);
                    neural_feature_inputs(sf, cf, fq);
                }
                neural_stage_inputs(XS[wave].x, g.visible, d, a.sh_degree, fq);
            }
            wave_lds_sync();
            const uint64_t vis = __ballot(g.visible);
            float o[3] = {0.f, 0.f, 0.f};
#pragma unroll
            for (int t = 0; t < kWave / 16; ++t) {
                if (((vis >> (16 * t)) & 0xFFFFull) == 0) continue;
                float4_t ot;
                if constexpr (kFolded) ot = neural_tile_out_folded(W, XS[wave].x, t, p4[t]);
                else ot = neural_tile_out(W, neural_stage_frag(XS[wave].x, t));
                neural_tile_gather(ot, t, o);
            }
            wave_lds_sync();   // the stage is read before the next chunk overwrites it
#pragma unroll
            for (int ch = 0; ch < 3; ++ch) res[ch] = tanhf(o[ch]);
        }
        float col[3];
#pragma unroll
        for (int ch = 0; ch < 3; ++ch) {
            const float v = c0[ch] + res[ch] + 0.5f;
            col[ch] = v > 0.f ? v : 0.f;
        }
        store_splats_wave(a.splats, a.n, base, stage[wave], g, col);
        wave_tiles += __builtin_amdgcn_readfirstlane(wave_sum_u32(tiles));   // uniform: kept in scalar registers
    }
    // one tile sum per wave of the grid (zero for a wave without a chunk),
    // saturated: 2^32 - 1 stands for that many pairs or more
    if (lane == 0) a.block_pairs[blockIdx.x * (kBlock / kWave) + wave] = (uint32_t)min(wave_tiles, (uint64_t)0xFFFFFFFFu);
}

// Workgroups of the latent preprocess: the number resident at once on 256 CUs
// (four per CU at the kernel's register budget), each wave looping over chunks.
constexpr int kLatentBlocks = 1024;
// and of the neural one (three per CU for the 32-neuron decoder)
constexpr int kNeuralBlocks = 1024;
constexpr int kNeuralBlocks32 = 768;

hipError_t launch_preprocess(const Cam& cam, const gs_gaussians& g, const gs_appearance& app,
                             const gs_preprocessed& out, const Workspace& ws, int* slots, hipStream_t s)
{
    PreArgs a;
    a.cam = cam;
    a.n = (int)g.n;
    a.means = g.means;
    a.log_scales = g.log_scales;
    a.quats = g.quats;
    a.logits = g.opacity_logits;
    a.sh_degree = app.sh_degree;
    a.sh = app.sh;
    a.latent = app.latent;
    a.mlp_w = app.mlp_w;
    a.base_color = app.base_color;
    a.features = app.features;
    a.preact = app.preact;
    a.lobes = app.lobes;
    a.sh_y0_folded = app.sh_y0_folded;
    a.splats = out.splats;
    a.color_jac = app.kind == GS_APP_SH3 ? out.color_jac : nullptr;
    a.tiles_touched = out.tiles_touched;
    a.depth_key = out.depth_key;
    a.block_pairs = ws.block_pairs;
    const int blocks = preprocess_blocks(g.n);
    // the SH3 and lobe kernels leave one tile sum per workgroup, the decoders
    // one per wave of their (capped) grid
    constexpr int kWaves = kBlock / kWave;
    *slots = blocks;
    if (app.kind == GS_APP_SH3) {
        switch (app.sh_degree) {
        case 0: hipLaunchKernelGGL(k_preprocess_sh3<0>, dim3(blocks), dim3(kBlock), 0, s, a); break;
        case 1: hipLaunchKernelGGL(k_preprocess_sh3<1>, dim3(blocks), dim3(kBlock), 0, s, a); break;
        case 2: hipLaunchKernelGGL(k_preprocess_sh3<2>, dim3(blocks), dim3(kBlock), 0, s, a); break;
        default: hipLaunchKernelGGL(k_preprocess_sh3<3>, dim3(blocks), dim3(kBlock), 0, s, a); break;
        }
    }
    else if (app.kind == GS_APP_NEURAL) {
        const dim3 grid(std::min(blocks, app.neural_width == 32 ? kNeuralBlocks32 : kNeuralBlocks));
        *slots = (int)grid.x * kWaves;
        const int layers = neural_layers(app);
        if (app.neural_width == 32) {
            hipLaunchKernelGGL((k_preprocess_neural<false, 2, false, 32>), grid, dim3(kBlock), 0, s, a);
        } else if (app.neural_raw16) {
            if (layers == 1) hipLaunchKernelGGL((k_preprocess_neural<false, 1, true>), grid, dim3(kBlock), 0, s, a);
            else if (layers == 3) hipLaunchKernelGGL((k_preprocess_neural<false, 3, true>), grid, dim3(kBlock), 0, s, a);
            else hipLaunchKernelGGL((k_preprocess_neural<false, 2, true>), grid, dim3(kBlock), 0, s, a);
        } else {
            if (layers == 1) hipLaunchKernelGGL((k_preprocess_neural<false, 1, false>), grid, dim3(kBlock), 0, s, a);
            else if (layers == 3) hipLaunchKernelGGL((k_preprocess_neural<false, 3, false>), grid, dim3(kBlock), 0, s, a);
            else hipLaunchKernelGGL((k_preprocess_neural<false, 2, false>), grid, dim3(kBlock), 0, s, a);
        }
    }
    else if (app.kind == GS_APP_NASG)
        hipLaunchKernelGGL(k_preprocess_lobe<false>, dim3(blocks), dim3(kBlock), 0, s, a);
    else if (app.kind == GS_APP_NASGABOR)
        hipLaunchKernelGGL(k_preprocess_lobe<true>, dim3(blocks), dim3(kBlock), 0, s, a);
    else if (app.kind == GS_APP_NEURAL_FOLDED) {
        *slots = std::min(blocks, kNeuralBlocks) * kWaves;
        hipLaunchKernelGGL((k_preprocess_neural<true, 2, false>), dim3(std::min(blocks, kNeuralBlocks)), dim3(kBlock), 0,
                           s, a);
    } else {
        *slots = std::min(blocks, kLatentBlocks) * kWaves;
        hipLaunchKernelGGL(k_preprocess_latent, dim3(std::min(blocks, kLatentBlocks)), dim3(kBlock), 0, s, a);
    }
    return hipGetLastError();
}

// Total pairs = sum of the per-workgroup or per-wave tile counts (fixed
// order, one workgroup). The counts sit at the 256-byte-aligned start of their
// workspace slice, so each thread reads runs of four with 16-byte loads, all
// issued before the sums. A saturated count (2^32 - 1, "that many or more")
// adds one more, so that the total then exceeds any capacity.
__global__ __launch_bounds__(1024) void k_pair_count(const uint32_t* block_pairs, int nslots, uint64_t* out)
{
    constexpr int kPer = 8;   // 16-byte loads in flight per thread and round
    __shared__ uint64_t red[16];
    const uint4* v4 = reinterpret_cast<const uint4*>(block_pairs);
    const int nvec = nslots >> 2;
    uint64_t v = 0;
    for (int b0 = 0; b0 < nvec; b0 += 1024 * kPer) {
        uint4 q[kPer];
#pragma unroll
        for (int k = 0; k < kPer; ++k) {
            const int b = b0 + k * 1024 + (int)threadIdx.x;
            q[k] = b < nvec ? v4[b] : make_uint4(0u, 0u, 0u, 0u);
        }
#pragma unroll
        for (int k = 0; k < kPer; ++k)
            v += (uint64_t)q[k].x + q[k].y + q[k].z + q[k].w + (q[k].x == ~0u) + (q[k].y == ~0u) + (q[k].z == ~0u) +
                 (q[k].w == ~0u);
    }
    const int rest = (nvec << 2) + (int)threadIdx.x;
    if (rest < nslots) v += (uint64_t)block_pairs[rest] + (block_pairs[rest] == ~0u);
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint64_t t = 0;
        for (int w = 0; w < 16; ++w) t += red[w];
        out[0] = t;
    }
}

hipError_t launch_pair_count(int slots, const Workspace& ws, uint64_t* num_pairs, hipStream_t s)
{
    hipLaunchKernelGGL(k_pair_count, dim3(1), dim3(1024), 0, s, ws.block_pairs, slots, num_pairs);
    return hipGetLastError();
}

// Decoder on caller-given inputs: x is [rows][17] binary16 (latent, then the
// view direction), out is [rows][3] fp32 colours.
__global__ __launch_bounds__(kBlock) void k_mlp_eval(const uint16_t* __restrict__ x, int64_t rows,
                                                     const uint16_t* __restrict__ w, float* __restrict__ out)
{
    __shared__ MlpFrags W;
    mlp_load_frags(w, W, false);
    const int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x;
    const int lane = __lane_id(), g = lane >> 4, c = lane & 15;
    const int64_t base = i - lane;
    const uint64_t vis = __ballot(i < rows);
    float col[3] = {0.f, 0.f, 0.f};
    for (int t = 0; t < kWave / 16; ++t) {
        if (((vis >> (16 * t)) & 0xFFFFull) == 0) continue;
        // B fragment: features s(g, 0..7) of row 16 t + c
        half8_t xb = {0, 0, 0, 0, 0, 0, 0, 0};
        const int src = 16 * t + c;
        if ((vis >> src) & 1) {
            const uint16_t* row = x + (base + src) * GS_MLP_IN;
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const int f = kslot(g, j);
                if (f < GS_MLP_IN) xb[j] = half_of_bits(row[f]);
            }
        }
        float4_t h1[2], h2[2], o;
        half8_t a1, a2;
        mlp_tile_fwd(W, xb, h1, a1, h2, a2, o);
        mlp_tile_colors(o, t, col);
    }
    if (i < rows)
        for (int ch = 0; ch < 3; ++ch) out[i * 3 + ch] = col[ch];
}

hipError_t launch_mlp_eval(const uint16_t* x, int64_t rows, const uint16_t* w, float* out, hipStream_t s)
{
    hipLaunchKernelGGL(k_mlp_eval, dim3((unsigned)div_up(rows, kBlock)), dim3(kBlock), 0, s, x, rows, w, out);
    return hipGetLastError();
}

// First-layer folding of the neural decoder: one wave per 64 Gaussians stages
// the unfolded input with every direction input but the constant Y_0 zero, so
// the first layer's product is exactly the pre-activation of the view-
// independent inputs; each tile's fp32 result is rounded to binary16 and
// stored Gaussian-major, 8 bytes per lane (neurons 4g..4g+3 of Gaussian c).
__global__ __launch_bounds__(kBlock) void k_neural_fold(const uint16_t* __restrict__ features,
                                                        const uint16_t* __restrict__ w, int n,
                                                        uint16_t* __restrict__ preact)
{
    __shared__ NeuralFrags<2> W;
    __shared__ NeuralInStage XS[kBlock / kWave];
    neural_load_frags(w, W, false);
    const int lane = __lane_id(), wave = threadIdx.x >> 6, g = lane >> 4, c = lane & 15;
    const int64_t base = ((int64_t)blockIdx.x * (kBlock / kWave) + wave) * kWave;
    const int64_t i = base + lane;
    float f[GS_NEURAL_FEATURES], sf[GS_NEURAL_FEATURES], cf[GS_NEURAL_FEATURES];
#pragma unroll
    for (int j = 0; j < GS_NEURAL_FEATURES; ++j) f[j] = i < n ? (float)half_of_bits(features[j * (int64_t)n + i]) : 0.f;
    neural_encode_features(f, sf, cf);
    half4_t fq[4];
    neural_feature_inputs(sf, cf, fq);
    const float d[3] = {0.f, 0.f, 1.f};   // unused at degree 0: only the constant Y_0 enters
    neural_stage_inputs(XS[wave].x, i < n, d, 0, fq);
    wave_lds_sync();
    const float4_t zero = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int t = 0; t < kWave / 16; ++t) {
        const int64_t gi = base + 16 * t + c;
        const float4_t h = mfma32(frag8(W.w1a), neural_stage_frag(XS[wave].x, t), zero);
        const half4_t hv = {(_Float16)h[0], (_Float16)h[1], (_Float16)h[2], (_Float16)h[3]};
        if (gi < n) *reinterpret_cast<half4_t*>(preact + gi * 16 + 4 * g) = hv;
    }
}

hipError_t launch_neural_fold(const uint16_t* features, const uint16_t* w, int64_t n, uint16_t* preact,
                              hipStream_t s)
{
    hipLaunchKernelGGL(k_neural_fold, dim3((unsigned)div_up(n, (int64_t)kBlock)), dim3(kBlock), 0, s, features, w,
                       (int)n, preact);
    return hipGetLastError();
}

}  // namespace gsr
