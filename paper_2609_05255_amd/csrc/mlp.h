// The latent decoder c = sigmoid(W3 relu(W2 relu(W1 [z, d]))) (no biases;
// 17 -> 32 -> 32 -> 3) on the matrix cores, for 16 Gaussians at a time, and its
// backward pass. Half-precision operands, fp32 accumulation (Sec. 4 and the
// appendix on the fused rasterizer: the decoder runs in half precision).
//
// Matrix-core fragments (wave64, l = lane, g = l/16, c = l%16):
//   v_mfma_f32_16x16x16_f16: A[c][4g + j], B[4g + j][c] (j = 0..3);
//   v_mfma_f32_16x16x32_f16: A[c][s(g, j)], B[s(g, j)][c] (j = 0..7);
//   both: D[4g + i][c] (i = 0..3).
// The 32-deep product pairs A's element j of lane group g with B's element j of
// the same group, so which K index a slot carries does not matter as long as A
// and B agree; this code gives slot (g, j) the index
//   s(g, j) = 4g + j (j < 4),  16 + 4g + (j - 4) (j >= 4),
// which makes the two D fragments of neurons 0..15 and 16..31 (lane l holds
// neurons 4g + i and 16 + 4g + i of Gaussian c), concatenated, the B fragment
// of the next layer: activations stay in registers from layer to layer.
//
// Two orientations. "Neuron-major" products put neurons on the M side
// (D[neuron][Gaussian]); they chain from layer to layer. Swapping the A and B
// registers of a product gives its transpose in the same D layout
// (D[Gaussian][neuron], "Gaussian-major"): there the Gaussians sit on the rows
// 4g + i, exactly where a 16-deep product over the tile's Gaussians wants its
// K index. The weight gradients (sums over Gaussians) therefore take
// Gaussian-major fragments straight from registers, with no transposes.
#pragma once

#include "gs_internal.h"

namespace gsr {

typedef _Float16 half4_t __attribute__((ext_vector_type(4)));
typedef _Float16 half8_t __attribute__((ext_vector_type(8)));
typedef float float4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float4_t mfma16(half4_t a, half4_t b, float4_t c)
{
    return __builtin_amdgcn_mfma_f32_16x16x16f16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float4_t mfma32(half8_t a, half8_t b, float4_t c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

// K index of slot j of lane group g in a 32-deep fragment.
__host__ __device__ constexpr int kslot(int g, int j) { return j < 4 ? 4 * g + j : 16 + 4 * g + (j - 4); }

// Per-workgroup weight fragments, one 8- (or 4-) half vector per lane, so that
// each operand is one aligned LDS read. Zero-padded outside the real sizes.
struct MlpFrags {
    alignas(16) _Float16 w1a[2][kWave][8];   // A of W1:   rows n1 = 16b + c,  K = input s(g, j)
    alignas(16) _Float16 w2a[2][kWave][8];   // A of W2:   rows n2 = 16b + c,  K = n1 s(g, j)
    alignas(16) _Float16 w3a[kWave][8];      // A of W3:   rows o = c (< 3),   K = n2 s(g, j)
    alignas(16) _Float16 w1t[2][kWave][8];   // A of W1^T: rows f = 16b + c (< 17), K = n1 s(g, j)
    alignas(16) _Float16 w2t[2][kWave][8];   // A of W2^T: rows n1 = 16b + c,  K = n2 s(g, j)
    alignas(8) _Float16 w3t[2][kWave][4];    // A of W3^T: rows n2 = 16b + c,  K = o = 4g + j (< 3)
};

// Loads the binary16 weights (W1[32][17], W2[32][32], W3[3][32], packed) into
// the fragments; the transposed ones only if `backward`. Called by every thread
// of the workgroup; ends with a barrier.
__device__ __forceinline__ void mlp_load_frags(const uint16_t* __restrict__ w, MlpFrags& s, bool backward)
{
    const _Float16* W1 = reinterpret_cast<const _Float16*>(w);
    const _Float16* W2 = W1 + 32 * GS_MLP_IN;
    const _Float16* W3 = W2 + 32 * 32;
    const _Float16 z = (_Float16)0.f;
    for (int e = threadIdx.x; e < kWave * 8; e += blockDim.x) {
        const int l = e >> 3, j = e & 7, g = l >> 4, c = l & 15;
        const int k = kslot(g, j);
        for (int b = 0; b < 2; ++b) {
            const int row = 16 * b + c;
            s.w1a[b][l][j] = k < GS_MLP_IN ? W1[row * GS_MLP_IN + k] : z;
            s.w2a[b][l][j] = W2[row * 32 + k];
            if (backward) {
                s.w1t[b][l][j] = row < GS_MLP_IN ? W1[k * GS_MLP_IN + row] : z;
                s.w2t[b][l][j] = W2[k * 32 + row];
                if (j < 4) s.w3t[b][l][j] = 4 * g + j < GS_MLP_OUT ? W3[(4 * g + j) * 32 + row] : z;
            }
        }
        s.w3a[l][j] = c < GS_MLP_OUT ? W3[c * 32 + k] : z;
    }
    __syncthreads();
}

__device__ __forceinline__ half8_t frag8(const _Float16 (*p)[8]) { return *reinterpret_cast<const half8_t*>(p[__lane_id()]); }
__device__ __forceinline__ half4_t frag4(const _Float16 (*p)[4]) { return *reinterpret_cast<const half4_t*>(p[__lane_id()]); }

// relu, then binary16: rounding to nearest keeps the sign, so rounding first
// and taking the maximum with zero on the packed halves gives the same values.
__device__ __forceinline__ half4_t relu_half4(const float4_t& v)
{
    typedef _Float16 half2_t __attribute__((ext_vector_type(2)));
    const half2_t z = {0, 0};
    half2_t a = {(_Float16)v[0], (_Float16)v[1]}, b = {(_Float16)v[2], (_Float16)v[3]};
    a = __builtin_elementwise_max(a, z);
    b = __builtin_elementwise_max(b, z);
    return half4_t{a[0], a[1], b[0], b[1]};
}

__device__ __forceinline__ half8_t relu_cat(const float4_t& lo, const float4_t& hi)
{
    const half4_t a = relu_half4(lo), b = relu_half4(hi);
    return half8_t{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
}

__device__ __forceinline__ _Float16 half_of_bits(uint16_t b) { return __builtin_bit_cast(_Float16, b); }

// B fragment (K = input feature, N = Gaussian) of the decoder input of tile t of
// the wave's 64 Gaussians (index base + lane): features s(g, 0..7) of Gaussian
// 16t + c, i.e. latent 4g..4g+3 (g < 3) or 12, 13, then d_x, d_y (g = 3), and
// d_z in slot 4 of group 0, with the view direction rounded to binary16 (round
// to nearest even). In two steps, so the loads can be issued long before the
// view direction is known: mlp_latent_raw loads the lane's latent entries of
// each tile (zeros past n), mlp_frag_from_raw completes a fragment with `d`,
// the calling lane's own direction.
struct MlpLatentRaw {
    half4_t v[kWave / 16];
};

__device__ __forceinline__ void mlp_latent_raw(const uint16_t* __restrict__ latent, int64_t n, int64_t base,
                                               MlpLatentRaw& r)
{
    const int l = __lane_id(), g = l >> 4, c = l & 15;
#pragma unroll
    for (int t = 0; t < kWave / 16; ++t) {
        const int64_t gi = base + 16 * t + c;
        const uint16_t* p = latent + (int64_t)(4 * g) * n + gi;
#pragma unroll
        for (int j = 0; j < 4; ++j)
            r.v[t][j] = (gi < n && (g < 3 || j < 2)) ? half_of_bits(p[(int64_t)j * n]) : (_Float16)0.f;
    }
}

__device__ __forceinline__ half8_t mlp_frag_from_raw(const MlpLatentRaw& r, int t, const float d[3])
{
    const int l = __lane_id(), g = l >> 4, c = l & 15;
    const int src = 16 * t + c;
    const float dx = __shfl(d[0], src), dy = __shfl(d[1], src), dz = __shfl(d[2], src);
    half8_t x = {r.v[t][0], r.v[t][1], r.v[t][2], r.v[t][3], 0, 0, 0, 0};
    if (g == 3) {
        x[2] = (_Float16)dx;
        x[3] = (_Float16)dy;
    }
    if (g == 0) x[4] = (_Float16)dz;
    return x;
}

// Neuron-major forward of one tile from its input fragment: h1[b], h2[b] hold
// the fp32 pre-activations of neurons 16b + 4g + i of Gaussian c, o the output
// pre-activations (channel i of Gaussian c in lanes 0..15, i < 3); a1, a2 the
// binary16 activations as next-layer fragments.
__device__ __forceinline__ void mlp_tile_fwd(const MlpFrags& W, const half8_t& x, float4_t h1[2], half8_t& a1,
                                             float4_t h2[2], half8_t& a2, float4_t& o)
{
    const float4_t zero = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int b = 0; b < 2; ++b) h1[b] = mfma32(frag8(W.w1a[b]), x, zero);
    a1 = relu_cat(h1[0], h1[1]);
#pragma unroll
    for (int b = 0; b < 2; ++b) h2[b] = mfma32(frag8(W.w2a[b]), a1, zero);
    a2 = relu_cat(h2[0], h2[1]);
    o = mfma32(frag8(W.w3a), a2, zero);
}

// Logistic function with the hardware exp2 and reciprocal (about 1 ulp each).
__device__ __forceinline__ float sigmoid_fast(float x)
{
    return __builtin_amdgcn_rcpf(1.f + __builtin_amdgcn_exp2f(-x * 1.4426950408889634f));
}

// Moves the tile's colours (lanes 0..15 of the neuron-major output) to the
// lanes that own the Gaussians (16 t .. 16 t + 15).
__device__ __forceinline__ void mlp_tile_colors(const float4_t& o, int t, float col[3])
{
    const int lane = __lane_id();
    const int src = lane & 15;
#pragma unroll
    for (int ch = 0; ch < 3; ++ch) {
        const float v = __shfl(sigmoid_fast(o[ch]), src);
        if ((lane >> 4) == t) col[ch] = v;
    }
}

// v = hi + lo with both parts binary16: gradients enter the matrix cores as two
// parts, so the chain keeps about 22 bits of precision instead of 11.
__device__ __forceinline__ _Float16 half_hi(float v) { return (_Float16)v; }
__device__ __forceinline__ _Float16 half_lo(float v) { return (_Float16)(v - (float)(_Float16)v); }

__device__ __forceinline__ void split4(const float4_t& v, half4_t& hi, half4_t& lo)
{
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        hi[i] = half_hi(v[i]);
        lo[i] = half_lo(v[i]);
    }
}

__device__ __forceinline__ void split_cat(const float4_t& a, const float4_t& b, half8_t& hi, half8_t& lo)
{
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        hi[i] = half_hi(a[i]);
        lo[i] = half_lo(a[i]);
        hi[4 + i] = half_hi(b[i]);
        lo[4 + i] = half_lo(b[i]);
    }
}

__device__ __forceinline__ float4_t relu_mask(const float4_t& v, const float4_t& pre)
{
    float4_t r;
#pragma unroll
    for (int i = 0; i < 4; ++i) r[i] = pre[i] > 0.f ? v[i] : 0.f;
    return r;
}

// Running sums of the weight gradients, Gaussian-major products in fp32, in
// units of 2^-se (se: the current chunk's gradient scale exponent, below):
// w1[mb][fb] rows n1 = 16mb + 4g + i, columns f = 16fb + c; w2[mb][nb] rows
// n2 = 16mb + 4g + i, columns n1 = 16nb + c; w3[nb] rows o = 4g + i, columns
// n2 = 16nb + c.
struct MlpGradAcc {
    float4_t w1[2][2], w2[2][2], w3[2];
    int se;
};

__device__ __forceinline__ void mlp_grad_zero(MlpGradAcc& a)
{
    const float4_t z = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        a.w3[u] = z;
#pragma unroll
        for (int v = 0; v < 2; ++v) a.w1[u][v] = a.w2[u][v] = z;
    }
    a.se = 0;
}

__device__ __forceinline__ float4_t ldexp4(const float4_t& v, int e)
{
    float4_t r;
#pragma unroll
    for (int i = 0; i < 4; ++i) r[i] = ldexpf(v[i], e);
    return r;
}

// Brings the running sums to units of 2^-se (exact: powers of two).
__device__ __forceinline__ void mlp_grad_rescale(MlpGradAcc& a, int se)
{
    if (se == a.se) return;
    const int e = se - a.se;
#pragma unroll
    for (int u = 0; u < 2; ++u) {
        a.w3[u] = ldexp4(a.w3[u], e);
#pragma unroll
        for (int v = 0; v < 2; ++v) {
            a.w1[u][v] = ldexp4(a.w1[u][v], e);
            a.w2[u][v] = ldexp4(a.w2[u][v], e);
        }
    }
    a.se = se;
}

// Maximum over the wave, returned to every lane.
__device__ __forceinline__ float wave_max(float v)
{
    v = fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xF, 0xF, false)));
    v = fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4E, 0xF, 0xF, false)));
    v = fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x141, 0xF, 0xF, false)));
    v = fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x140, 0xF, 0xF, false)));
    const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
    const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
    const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
    const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
    return fmaxf(fmaxf(r0, r1), fmaxf(r2, r3));
}

// Largest factor by which the backward can grow the output gradient on its
// way to the first hidden layer: dH_L = Wout^T delta and dH_(l-1) = W_l^T dH_l,
// so |dH_l| <= C_out C_L ... C_(l+1) max|delta| with C the largest column sum of
// |W| (the infinity norm of W^T). Returns the largest of 1 and these products,
// for weights stored [out][in] as binary16: W1 [width][n_in], `hidden`
// matrices [width][width], Wout [3][width]. The workgroup's first wave reads
// the weights; every thread returns the value (one barrier).
__device__ __forceinline__ float decoder_chain_bound(const uint16_t* __restrict__ w, int n_in, int width, int hidden,
                                                     float* slot)
{
    if (threadIdx.x < kWave) {
        const int u = __lane_id();
        const uint16_t* wo = w + width * n_in + hidden * width * width;
        float cs = 0.f;
        if (u < width)
            for (int o = 0; o < 3; ++o) cs += fabsf((float)half_of_bits(wo[o * width + u]));
        float prod = wave_max(cs), best = fmaxf(1.f, prod);
        for (int h = hidden - 1; h >= 0; --h) {
            const uint16_t* wh = w + width * n_in + h * width * width;
            cs = 0.f;
            if (u < width)
                for (int r = 0; r < width; ++r) cs += fabsf((float)half_of_bits(wh[r * width + u]));
            prod *= wave_max(cs);
            best = fmaxf(best, prod);
        }
        if (u == 0) *slot = best;
    }
    __syncthreads();
    return *slot;
}

// Scale exponent of a chunk whose largest colour-gradient magnitude, times the
// decoder's chain bound, is m: the output gradients delta3 = dL/dc s (1 - s)
// and the hidden-layer gradients they produce then stay below 2^9 after
// scaling by 2^se (binary16 overflows above 65504), and the largest output
// gradient lies within a factor 4 s (1 - s) and the chain bound of it, far
// from the binary16 subnormals. m = 0 keeps the previous exponent.
__device__ __forceinline__ int mlp_chunk_exponent(float m, int prev)
{
    if (!(m > 0.f)) return prev;
    int ex = 0;
    frexpf(m, &ex);
    return min(11 - ex, 100);
}

// Row pitch (halves) of the staged decoder inputs: 8-byte aligned rows whose
// fragment reads spread over the LDS banks.
constexpr int kXPitch = 36;

// Per-wave staging of what the backward needs across lanes: each Gaussian's
// decoder input (latent 0..13, binary16 direction 14..16, zeros up to 32), its
// output-colour gradient, and the gradient into its direction that the tiles
// produce.
struct MlpWaveStage {
    alignas(16) _Float16 x[kWave][kXPitch];
    float dc[kWave][4];
    float dd[kWave][4];
};

// Writes the calling lane's row of the stage (all lanes; zeros when !valid).
__device__ __forceinline__ void mlp_stage_row(MlpWaveStage& st, bool valid, const uint16_t* __restrict__ latent,
                                              int64_t n, int64_t i, const float d[3], const float dc[3])
{
    const int l = __lane_id();
    half4_t v[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) v[q] = half4_t{0, 0, 0, 0};
    if (valid) {
#pragma unroll
        for (int f = 0; f < GS_LATENT_DIM; ++f) v[f >> 2][f & 3] = half_of_bits(latent[(int64_t)f * n + i]);
        v[3][2] = (_Float16)d[0];
        v[3][3] = (_Float16)d[1];
        v[4][0] = (_Float16)d[2];
    }
#pragma unroll
    for (int q = 0; q < 8; ++q) *reinterpret_cast<half4_t*>(&st.x[l][4 * q]) = v[q];
#pragma unroll
    for (int ch = 0; ch < 3; ++ch) st.dc[l][ch] = valid ? dc[ch] : 0.f;
    st.dc[l][3] = 0.f;   // padding column: fragments read it where a channel 3 would sit
}

// B fragment of tile t from the stage: features s(g, 0..7) of Gaussian 16t + c.
__device__ __forceinline__ half8_t mlp_stage_frag(const MlpWaveStage& st, int t)
{
    const int l = __lane_id(), g = l >> 4, c = l & 15;
    const half4_t lo = *reinterpret_cast<const half4_t*>(&st.x[16 * t + c][4 * g]);
    const half4_t hi = *reinterpret_cast<const half4_t*>(&st.x[16 * t + c][16 + 4 * g]);
    return half8_t{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
}

// Backward of one tile (Gaussians 16t .. 16t + 15 of the wave), from the
// staged inputs and colour gradients, with the chunk's gradient scale 2^se
// (acc.se): delta3 = dL/dc s (1 - s) enters the matrix cores scaled, dH2, dH1
// and dX are chained neuron-major, the Gaussian-major copies give
//   dW3 = sum_G delta3 h2^T, dW2 = sum_G dh2 h1^T, dW1 = sum_G dh1 x^T
// accumulated in place into `acc` (units 2^-se). Writes the latent gradients of
// the tile's valid Gaussians to dlatent ([14][n], Gaussian base + 16t + c) and
// their direction gradients to st.dd.
//
// Precision: along the chain to dX each gradient operand is a binary16 hi+lo
// pair, since a rounding there is carried through two more layers into every
// input gradient. The weight gradients take each gradient operand as one
// binary16 value: each product then carries its own rounding (relative 2^-12
// at most), and these independent errors stay at that level in the sums.
__device__ __forceinline__ void mlp_tile_bwd(const MlpFrags& W, MlpWaveStage& st, int t, uint64_t valid,
                                             float* __restrict__ dlatent, int64_t n, int64_t base, float scale,
                                             float inv, MlpGradAcc& acc)
{
    const int l = __lane_id(), g = l >> 4, c = l & 15;
    const float4_t zero = {0.f, 0.f, 0.f, 0.f};
    const half8_t x = mlp_stage_frag(st, t);
    // Gaussian-major input fragment: feature 16fb + c of Gaussians 16t + 4g + j
    // (rows of culled Gaussians are zero)
    half4_t xg[2];
#pragma unroll
    for (int fb = 0; fb < 2; ++fb)
#pragma unroll
        for (int j = 0; j < 4; ++j) xg[fb][j] = st.x[16 * t + 4 * g + j][16 * fb + c];
    // forward, both orientations
    float4_t h1n[2], h2n[2], on;
    half8_t a1, a2;
    mlp_tile_fwd(W, x, h1n, a1, h2n, a2, on);
    float4_t h1g[2], h2g[2];
#pragma unroll
    for (int b = 0; b < 2; ++b) h1g[b] = mfma32(x, frag8(W.w1a[b]), zero);      // h1[G = 4g+i][16b + c]
#pragma unroll
    for (int b = 0; b < 2; ++b) h2g[b] = mfma32(a1, frag8(W.w2a[b]), zero);     // h2[G = 4g+i][16b + c]
    const float4_t og = mfma32(a2, frag8(W.w3a), zero);                          // o[G = 4g+i][channel c]

    // scaled output gradients: neuron-major (channel 4g + i of Gaussian c, only
    // g = 0 carries channels) and Gaussian-major (Gaussian 4g + i, channel c);
    // a culled Gaussian's staged colour gradient is zero
    float4_t d3n = zero, d3g;
    const int cn = min(c, 3);
#pragma unroll
    for (int i = 0; i < GS_MLP_OUT; ++i) {
        const float sn = sigmoid_fast(on[i]);
        const float dcn = st.dc[16 * t + c][i];
        d3n[i] = g == 0 ? dcn * scale * (sn * (1.f - sn)) : 0.f;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const float sg = sigmoid_fast(og[i]);
        const float dcg = st.dc[16 * t + 4 * g + i][cn];
        d3g[i] = c < GS_MLP_OUT ? dcg * scale * (sg * (1.f - sg)) : 0.f;
    }
    half4_t d3n_hi, d3n_lo;
    split4(d3n, d3n_hi, d3n_lo);
    const half4_t d3g_h = half4_t{(_Float16)d3g[0], (_Float16)d3g[1], (_Float16)d3g[2], (_Float16)d3g[3]};

    // dH2 = W3^T delta3, masked by relu'(h2)
    float4_t g2n[2], g2g[2];
#pragma unroll
    for (int b = 0; b < 2; ++b) {
        const half4_t w = frag4(W.w3t[b]);
        g2n[b] = relu_mask(mfma16(w, d3n_lo, mfma16(w, d3n_hi, zero)), h2n[b]);
        g2g[b] = relu_mask(mfma16(d3n_lo, w, mfma16(d3n_hi, w, zero)), h2g[b]);
    }
    half8_t g2n_hi, g2n_lo;
    split_cat(g2n[0], g2n[1], g2n_hi, g2n_lo);
    // dH1 = W2^T dH2, masked by relu'(h1)
    float4_t g1n[2], g1g[2];
#pragma unroll
    for (int b = 0; b < 2; ++b) {
        const half8_t w = frag8(W.w2t[b]);
        g1n[b] = relu_mask(mfma32(w, g2n_lo, mfma32(w, g2n_hi, zero)), h1n[b]);
        g1g[b] = relu_mask(mfma32(g2n_lo, w, mfma32(g2n_hi, w, zero)), h1g[b]);
    }
    half8_t g1n_hi, g1n_lo;
    split_cat(g1n[0], g1n[1], g1n_hi, g1n_lo);
    // dX = W1^T dH1: lane l holds features 16b + 4g + i of Gaussian c
    float4_t dx[2];
#pragma unroll
    for (int b = 0; b < 2; ++b) {
        const half8_t w = frag8(W.w1t[b]);
        dx[b] = mfma32(w, g1n_lo, mfma32(w, g1n_hi, zero)) * inv;
    }
    if ((valid >> (16 * t + c)) & 1) {
        float* p = dlatent + (int64_t)(4 * g) * n + base + 16 * t + c;
        p[0] = dx[0][0];
        p[n] = dx[0][1];
        if (g < 3) {
            p[2 * n] = dx[0][2];
            p[3 * n] = dx[0][3];
        } else {
            st.dd[16 * t + c][0] = dx[0][2];
            st.dd[16 * t + c][1] = dx[0][3];
        }
        if (g == 0) st.dd[16 * t + c][2] = dx[1][0];
    }

    // weight gradients from the Gaussian-major fragments, accumulated in place
    half4_t r1g[2], r2g[2];
#pragma unroll
    for (int b = 0; b < 2; ++b) {
        r1g[b] = relu_half4(h1g[b]);
        r2g[b] = relu_half4(h2g[b]);
    }
    // dW3[o][n2] = sum_G delta3[G][o] h2[G][n2]
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) acc.w3[nb] = mfma16(d3g_h, r2g[nb], acc.w3[nb]);
    // dW2[n2][n1] = sum_G dh2[G][n2] h1[G][n1]
#pragma unroll
    for (int mb = 0; mb < 2; ++mb) {
        const half4_t h = {(_Float16)g2g[mb][0], (_Float16)g2g[mb][1], (_Float16)g2g[mb][2], (_Float16)g2g[mb][3]};
#pragma unroll
        for (int nb = 0; nb < 2; ++nb) acc.w2[mb][nb] = mfma16(h, r1g[nb], acc.w2[mb][nb]);
    }
    // dW1[n1][f] = sum_G dh1[G][n1] x[G][f]
#pragma unroll
    for (int mb = 0; mb < 2; ++mb) {
        const half4_t h = {(_Float16)g1g[mb][0], (_Float16)g1g[mb][1], (_Float16)g1g[mb][2], (_Float16)g1g[mb][3]};
#pragma unroll
        for (int fb = 0; fb < 2; ++fb) acc.w1[mb][fb] = mfma16(h, xg[fb], acc.w1[mb][fb]);
    }
}

// Orders this wave's LDS writes before its following LDS reads by other lanes.
__device__ __forceinline__ void wave_lds_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

}  // namespace gsr
