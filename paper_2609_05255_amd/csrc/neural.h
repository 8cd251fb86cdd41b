// The paper's neural appearance decoder (Sec. 4, eq. mlp_input and
// eq. neural_color_eval) on the matrix cores, 16 Gaussians at a time: input
// x = (SH basis of the view direction up to the active degree, zero above it;
// (sin f_j, cos f_j) of the 8 features), a 32 -> 16 -> 16 -> 3 network without
// biases and with ReLU hidden units, residual tanh(MLP(x)), colour
// max(0, c0 + residual + 0.5) (eq. common_appearance with the baseline
// activation). Inputs and hidden activations are binary16 operands, sums fp32.
//
// The configurations of the paper's architecture table with 16 neurons per
// layer are the template parameter L (1..3 hidden layers): W1[16][32], then
// L - 1 matrices [16][16], then Wout[3][16]; 2 is the paper's default.
//
// Fragment layouts and the two orientations are those of mlp.h: layer 1 is one
// 32-deep product (slot s(g, j) carries input s(g, j)), layers 2 and 3 and every
// backward product are 16-deep, whose D fragment of one layer is the B fragment
// of the next. Swapping the A and B registers of a product gives its transpose
// (Gaussian-major), which the weight gradients take as operands.
#pragma once

#include "mlp.h"
#include "sh.h"

namespace gsr {

constexpr int kNeuralIn = 32, kNeuralHidden = 16;

constexpr int neural_weight_count(int layers) { return kNeuralHidden * kNeuralIn + (layers - 1) * kNeuralHidden * kNeuralHidden + GS_MLP_OUT * kNeuralHidden; }

// Per-workgroup weight fragments of a decoder with L hidden layers (binary16).
template <int L>
struct NeuralFrags {
    static constexpr int kH = L > 1 ? L - 1 : 1;   // hidden-to-hidden matrices (at least one slot)
    alignas(16) _Float16 w1a[kWave][8];     // A of W1:   rows n1 = c,             K = input s(g, j)
    alignas(8) _Float16 wha[kH][kWave][4];  // A of W_l:  rows n_l = c,            K = n_(l-1) = 4g + j
    alignas(8) _Float16 w3a[kWave][4];      // A of Wout: rows o = c (< 3),        K = n_L = 4g + j
    alignas(8) _Float16 w1t[2][kWave][4];   // A of W1^T: rows input = 16b + c,   K = n1 = 4g + j
    alignas(8) _Float16 wht[kH][kWave][4];  // A of W_l^T: rows n_(l-1) = c,       K = n_l = 4g + j
    alignas(8) _Float16 w3t[kWave][4];      // A of Wout^T: rows n_L = c,          K = o = 4g + j (< 3)
    alignas(8) _Float16 w1d[kWave][4];      // A of W1's direction columns 1..15 (folded form):
                                            //            rows n1 = c, K = 4g + j -> column 1 + 4g + j (< 16)
};

// Loads the weights into the fragments (the transposed ones only if
// `backward`, the direction columns only if `folded`). Called by every thread
// of the workgroup; ends with a barrier.
template <int L>
__device__ __forceinline__ void neural_load_frags(const uint16_t* __restrict__ w, NeuralFrags<L>& s, bool backward,
                                                  bool folded = false)
{
    const _Float16* W1 = reinterpret_cast<const _Float16*>(w);
    const _Float16* Wh = W1 + kNeuralHidden * kNeuralIn;                       // [L-1][16][16]
    const _Float16* W3 = Wh + (L - 1) * kNeuralHidden * kNeuralHidden;         // [3][16]
    const _Float16 z = (_Float16)0.f;
    for (int e = threadIdx.x; e < kWave * 8; e += blockDim.x) {
        const int l = e >> 3, j = e & 7, g = l >> 4, c = l & 15;
        s.w1a[l][j] = W1[c * kNeuralIn + kslot(g, j)];
        if (j < 4) {
            const int k = 4 * g + j;
#pragma unroll
            for (int h = 0; h < L - 1; ++h) {
                const _Float16* Wl = Wh + h * kNeuralHidden * kNeuralHidden;
                s.wha[h][l][j] = Wl[c * kNeuralHidden + k];
                if (backward) s.wht[h][l][j] = Wl[k * kNeuralHidden + c];
            }
            s.w3a[l][j] = c < GS_MLP_OUT ? W3[c * kNeuralHidden + k] : z;
            if (folded) s.w1d[l][j] = k < 15 ? W1[c * kNeuralIn + 1 + k] : z;
            if (backward) {
                for (int b = 0; b < 2; ++b) s.w1t[b][l][j] = W1[k * kNeuralIn + 16 * b + c];
                s.w3t[l][j] = k < GS_MLP_OUT ? W3[k * kNeuralHidden + c] : z;
            }
        }
    }
    __syncthreads();
}

// Per-wave staging: each Gaussian's 32 binary16 inputs (rows of kXPitch
// halves). The backward also stages each Gaussian's output gradient delta3
// (channel 3 zero) and receives from the tiles the gradients of its 16 feature
// inputs and, in its input row once the tile has read it, the gradients of its
// 16 direction inputs as fp32.
struct NeuralInStage {
    alignas(16) _Float16 x[kWave][kXPitch];
};

struct NeuralBwdStage {
    alignas(16) _Float16 x[kWave][kXPitch];
    float d3[kWave][4];
    float dxf[kWave][16];
};
static_assert(kXPitch * sizeof(_Float16) >= 16 * sizeof(float), "a row holds 16 fp32 direction gradients");

// The direction-input gradients that tile backward left in row r.
__device__ __forceinline__ const float* neural_dir_grad_row(const NeuralBwdStage& st, int r)
{
    return reinterpret_cast<const float*>(&st.x[r][0]);
}

// sin f and cos f of a binary16 value f, without branches. Cody-Waite
// reduction r = f - k pi/2 with k = rint(2f/pi) (|k| < 2^16 for binary16
// arguments) against pi/2 split into three fp32 parts, each product exact
// inside an FMA; Taylor polynomials of sin through r^9 and cos through r^10 on
// |r| <= pi/4 (truncation below 2e-9); the quadrant k mod 4 swaps and negates.
// Over every finite binary16 argument the error is at most 6.1e-8 absolute
// (1.3 ulp), as measured against fp64 sin and cos.
__device__ __forceinline__ void sincos_half_arg(float f, float* s, float* c)
{
    const float k = rintf(f * 0x1.45f306p-1f);           // 2/pi
    float r = fmaf(-k, 0x1.921fb6p+0f, f);                // pi/2 = p1 + p2 + p3
    r = fmaf(-k, -0x1.777a5cp-25f, r);
    r = fmaf(-k, -0x1.ee59dap-50f, r);
    const float r2 = r * r;
    float ps = fmaf(r2, 1.f / 362880.f, -1.f / 5040.f);
    ps = fmaf(r2, ps, 1.f / 120.f);
    ps = fmaf(r2, ps, -1.f / 6.f);
    const float sr = fmaf(r * r2, ps, r);
    float pc = fmaf(r2, -1.f / 3628800.f, 1.f / 40320.f);
    pc = fmaf(r2, pc, -1.f / 720.f);
    pc = fmaf(r2, pc, 1.f / 24.f);
    pc = fmaf(r2, pc, -0.5f);
    const float cr = fmaf(r2, pc, 1.f);
    const int q = (int)k & 3;
    const float a = (q & 1) ? cr : sr, b = (q & 1) ? sr : cr;
    *s = (q & 2) ? -a : a;
    *c = ((q + 1) & 2) ? -b : b;
}

// sin f_j and cos f_j of the calling lane's features (the frequency encoding
// with k = 1).
__device__ __forceinline__ void neural_encode_features(const float f[GS_NEURAL_FEATURES], float sf[GS_NEURAL_FEATURES],
                                                       float cf[GS_NEURAL_FEATURES])
{
#pragma unroll
    for (int j = 0; j < GS_NEURAL_FEATURES; ++j) sincos_half_arg(f[j], &sf[j], &cf[j]);
}

// The 16 feature inputs in input order, rounded to binary16: q[k] holds
// (sin f_2k, cos f_2k, sin f_2k+1, cos f_2k+1).
__device__ __forceinline__ void neural_feature_inputs(const float sf[GS_NEURAL_FEATURES],
                                                      const float cf[GS_NEURAL_FEATURES], half4_t q[4])
{
#pragma unroll
    for (int k = 0; k < 4; ++k)
        q[k] = half4_t{(_Float16)sf[2 * k], (_Float16)cf[2 * k], (_Float16)sf[2 * k + 1], (_Float16)cf[2 * k + 1]};
}

// The 16 raw features as the feature inputs (the table's F = 16 configuration).
__device__ __forceinline__ void neural_raw_inputs(const float f[16], half4_t q[4])
{
#pragma unroll
    for (int k = 0; k < 4; ++k)
        q[k] = half4_t{(_Float16)f[4 * k], (_Float16)f[4 * k + 1], (_Float16)f[4 * k + 2], (_Float16)f[4 * k + 3]};
}

// The calling lane's decoder input: SH basis values of d for bands <= degree
// (zero above), then the feature inputs `fq` (neural_feature_inputs), in
// binary16 (zeros when !valid).
__device__ __forceinline__ void neural_stage_inputs(_Float16 (*x)[kXPitch], bool valid, const float d[3], int degree,
                                                    const half4_t fq[4])
{
    const int l = __lane_id();
    half4_t v[8];
#pragma unroll
    for (int q = 0; q < 8; ++q) v[q] = half4_t{0, 0, 0, 0};
    if (valid) {
        float Y[16];
        sh_basis16(d[0], d[1], d[2], Y);
        const int nb = (degree + 1) * (degree + 1);
#pragma unroll
        for (int k = 0; k < 16; ++k) v[k >> 2][k & 3] = k < nb ? (_Float16)Y[k] : (_Float16)0.f;
#pragma unroll
        for (int q = 0; q < 4; ++q) v[4 + q] = fq[q];
    }
#pragma unroll
    for (int q = 0; q < 8; ++q) *reinterpret_cast<half4_t*>(&x[l][4 * q]) = v[q];
}

// The folded form's per-view decoder input: Y_1..15(d) for bands <= degree (zero
// above), then a zero pad, in binary16 (zeros when !valid), in row `lane`.
__device__ __forceinline__ void neural_stage_dir(_Float16 (*x)[kXPitch], bool valid, const float d[3], int degree)
{
    const int l = __lane_id();
    half4_t v[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) v[q] = half4_t{0, 0, 0, 0};
    if (valid) {
        float Y[16];
        sh_basis16(d[0], d[1], d[2], Y);
        const int nb = (degree + 1) * (degree + 1);
#pragma unroll
        for (int k = 1; k < 16; ++k) v[(k - 1) >> 2][(k - 1) & 3] = k < nb ? (_Float16)Y[k] : (_Float16)0.f;
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) *reinterpret_cast<half4_t*>(&x[l][4 * q]) = v[q];
}

// Output pre-activations of tile t in the folded form: h1 = p + W1d xd with the
// Gaussians' pre-activations p as the accumulator input (p4: neurons 4g + i of
// Gaussian 16t + c, this lane's share), then layers 2 and 3 as unfolded.
template <int L>
__device__ __forceinline__ float4_t neural_tile_out_folded(const NeuralFrags<L>& W, const _Float16 (*x)[kXPitch],
                                                           int t, const half4_t& p4)
{
    const int l = __lane_id(), g = l >> 4, c = l & 15;
    const float4_t zero = {0.f, 0.f, 0.f, 0.f};
    const half4_t xd = *reinterpret_cast<const half4_t*>(&x[16 * t + c][4 * g]);
    const float4_t p = {(float)p4[0], (float)p4[1], (float)p4[2], (float)p4[3]};
    half4_t a = relu_half4(mfma16(frag4(W.w1d), xd, p));
#pragma unroll
    for (int h = 0; h < L - 1; ++h) a = relu_half4(mfma16(frag4(W.wha[h]), a, zero));
    return mfma16(frag4(W.w3a), a, zero);
}

// B fragment of tile t: inputs s(g, 0..7) of Gaussian 16t + c.
__device__ __forceinline__ half8_t neural_stage_frag(const _Float16 (*x)[kXPitch], int t)
{
    const int l = __lane_id(), g = l >> 4, c = l & 15;
    const half4_t lo = *reinterpret_cast<const half4_t*>(&x[16 * t + c][4 * g]);
    const half4_t hi = *reinterpret_cast<const half4_t*>(&x[16 * t + c][16 + 4 * g]);
    return half8_t{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
}

// Hands the output pre-activations o of tile t to the lanes that own its
// Gaussians (lane 16t + c takes Gaussian c's three channels from lane c).
__device__ __forceinline__ void neural_tile_gather(const float4_t& o, int t, float own[3])
{
    const int lane = __lane_id();
    const int src = lane & 15;
#pragma unroll
    for (int ch = 0; ch < 3; ++ch) {
        const float v = __shfl(o[ch], src);
        if ((lane >> 4) == t) own[ch] = v;
    }
}

// Output pre-activations of one tile (channel i of Gaussian c in lanes g = 0).
template <int L>
__device__ __forceinline__ float4_t neural_tile_out(const NeuralFrags<L>& W, const half8_t& x)
{
    const float4_t zero = {0.f, 0.f, 0.f, 0.f};
    half4_t a = relu_half4(mfma32(frag8(W.w1a), x, zero));
#pragma unroll
    for (int h = 0; h < L - 1; ++h) a = relu_half4(mfma16(frag4(W.wha[h]), a, zero));
    return mfma16(frag4(W.w3a), a, zero);
}

// Running sums of the weight gradients (Gaussian-major products, fp32, in
// units of 2^-se): w1[fb] rows n1 = 4g + i, columns input 16fb + c; wh[h] rows
// n_(h+2) = 4g + i, columns n_(h+1) = c; w3 rows o = 4g + i, columns n_L = c.
template <int L>
struct NeuralGradAcc {
    float4_t w1[2], wh[NeuralFrags<L>::kH], w3;
    int se;
};

template <int L>
__device__ __forceinline__ void neural_grad_zero(NeuralGradAcc<L>& a)
{
    const float4_t z = {0.f, 0.f, 0.f, 0.f};
    a.w1[0] = a.w1[1] = a.w3 = z;
#pragma unroll
    for (int h = 0; h < NeuralFrags<L>::kH; ++h) a.wh[h] = z;
    a.se = 0;
}

template <int L>
__device__ __forceinline__ void neural_grad_rescale(NeuralGradAcc<L>& a, int se)
{
    if (se == a.se) return;
    const int e = se - a.se;
    a.w1[0] = ldexp4(a.w1[0], e);
    a.w1[1] = ldexp4(a.w1[1], e);
#pragma unroll
    for (int h = 0; h < L - 1; ++h) a.wh[h] = ldexp4(a.wh[h], e);
    a.w3 = ldexp4(a.w3, e);
    a.se = se;
}

// Scale exponent of a chunk whose largest output gradient dL/dc [c > 0]
// (1 - tanh^2), times the decoder's chain bound (decoder_chain_bound), is m:
// the output gradients and the hidden-layer gradients they produce then stay
// below 2^10 after scaling by 2^se, far below the binary16 overflow at 65504;
// the largest output gradient lies within the chain bound of 2^10, far from
// the subnormals. m = 0 keeps the previous exponent.
__device__ __forceinline__ int neural_chunk_exponent(float m, int prev)
{
    if (!(m > 0.f)) return prev;
    int ex = 0;
    frexpf(m, &ex);
    return min(10 - ex, 100);
}

// Backward of tile t (Gaussians 16t .. 16t + 15 of the wave) from the staged
// inputs and output gradients delta3 = dL/dc [c0 + res + 0.5 > 0] (1 - res^2),
// with the chunk's gradient scale 2^se (acc.se): delta3 enters the matrix
// cores scaled; the hidden-layer gradients and dX are chained neuron-major
// (binary16 hi + lo operands); the Gaussian-major copies give
//   dWout = sum_G delta3 h_L^T, dW_l = sum_G dh_l h_(l-1)^T, dW1 = sum_G dh_1 x^T
// accumulated into `acc`. Leaves the gradients of the 16 feature inputs in
// st.dxf and, once the tile's reads of its input rows are issued, those of the
// 16 direction inputs in the same rows (fp32, every band; the caller masks).
template <int L>
__device__ __forceinline__ void neural_tile_bwd(const NeuralFrags<L>& W, NeuralBwdStage& st, int t, float scale,
                                                float inv, NeuralGradAcc<L>& acc)
{
    const int l = __lane_id(), g = l >> 4, c = l & 15;
    const float4_t zero = {0.f, 0.f, 0.f, 0.f};
    const half8_t x = neural_stage_frag(st.x, t);
    // Gaussian-major inputs: input 16fb + c of Gaussians 16t + 4g + j
    half4_t xg[2];
#pragma unroll
    for (int fb = 0; fb < 2; ++fb)
#pragma unroll
        for (int j = 0; j < 4; ++j) xg[fb][j] = st.x[16 * t + 4 * g + j][16 * fb + c];
    // forward of the hidden layers, both orientations (the output layer is not
    // needed again): hn[l] neurons 4g + i of Gaussian c, hg[l] Gaussian 4g + i,
    // neuron c
    float4_t hn[L], hg[L];
    half4_t an[L];
    hn[0] = mfma32(frag8(W.w1a), x, zero);
    hg[0] = mfma32(x, frag8(W.w1a), zero);
    an[0] = relu_half4(hn[0]);
#pragma unroll
    for (int h = 1; h < L; ++h) {
        hn[h] = mfma16(frag4(W.wha[h - 1]), an[h - 1], zero);
        hg[h] = mfma16(an[h - 1], frag4(W.wha[h - 1]), zero);
        an[h] = relu_half4(hn[h]);
    }

    // output gradients: neuron-major (channel i of Gaussian c, in lanes g = 0)
    // and Gaussian-major (Gaussian 4g + i, channel c < 3; column 3 is zero)
    float4_t d3n = zero, d3g;
    const int Gn = 16 * t + c;
    if (g == 0)
#pragma unroll
        for (int i = 0; i < GS_MLP_OUT; ++i) d3n[i] = st.d3[Gn][i] * scale;
    const int cn = min(c, 3);
#pragma unroll
    for (int i = 0; i < 4; ++i) d3g[i] = st.d3[16 * t + 4 * g + i][cn] * scale;
    half4_t hi, lo;
    split4(d3n, hi, lo);
    acc.w3 = mfma16(half4_t{(_Float16)d3g[0], (_Float16)d3g[1], (_Float16)d3g[2], (_Float16)d3g[3]},
                    relu_half4(hg[L - 1]), acc.w3);                                   // dWout[o][n_L]

    // dH_L = Wout^T delta3, masked by relu'(h_L)
    const half4_t w3t = frag4(W.w3t);
    float4_t gn = relu_mask(mfma16(w3t, lo, mfma16(w3t, hi, zero)), hn[L - 1]);
    float4_t gg = relu_mask(mfma16(lo, w3t, mfma16(hi, w3t, zero)), hg[L - 1]);
    // dH_(l-1) = W_l^T dH_l, masked by relu'(h_(l-1)); dW_l from the Gaussian-major copies
#pragma unroll
    for (int h = L - 1; h >= 1; --h) {
        acc.wh[h - 1] = mfma16(half4_t{(_Float16)gg[0], (_Float16)gg[1], (_Float16)gg[2], (_Float16)gg[3]},
                               relu_half4(hg[h - 1]), acc.wh[h - 1]);                 // dW_h[n_h][n_(h-1)]
        split4(gn, hi, lo);
        const half4_t wt = frag4(W.wht[h - 1]);
        gn = relu_mask(mfma16(wt, lo, mfma16(wt, hi, zero)), hn[h - 1]);
        gg = relu_mask(mfma16(lo, wt, mfma16(hi, wt, zero)), hg[h - 1]);
    }
    split4(gn, hi, lo);
    // dX = W1^T dH1: dx[b] holds inputs 16b + 4g + i of Gaussian c
    float4_t dx[2];
#pragma unroll
    for (int b = 0; b < 2; ++b) {
        const half4_t w = frag4(W.w1t[b]);
        dx[b] = mfma16(w, lo, mfma16(w, hi, zero)) * inv;
    }
    // the tile's input rows have been read: they now take the direction-input
    // gradients
    wave_lds_sync();
    float* row = reinterpret_cast<float*>(&st.x[Gn][0]);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        row[4 * g + i] = dx[0][i];
        st.dxf[Gn][4 * g + i] = dx[1][i];
    }

    // dW1 from the Gaussian-major dH1 and inputs, accumulated in place
    const half4_t h1d = {(_Float16)gg[0], (_Float16)gg[1], (_Float16)gg[2], (_Float16)gg[3]};
#pragma unroll
    for (int fb = 0; fb < 2; ++fb) acc.w1[fb] = mfma16(h1d, xg[fb], acc.w1[fb]);   // dW1[n1][input]
}

// ---- the table's 32-neuron configuration ----------------------------------------
// 32 -> 32 -> 32 -> 3 has the shape of the latent decoder (mlp.h), so it takes
// that decoder's fragments, forward tile and weight-gradient sums, loaded from
// W1[32][32], W2[32][32], Wout[3][32]; only the input staging, the tanh
// residual and the input-gradient hand-off are the neural model's.
constexpr int kNeural32Weights = 32 * 32 + 32 * 32 + GS_MLP_OUT * 32;   // 2144

__device__ __forceinline__ void neural_load_frags(const uint16_t* __restrict__ w, MlpFrags& s, bool backward,
                                                  bool folded = false)
{
    (void)folded;   // the folded form takes the 16-neuron default only
    const _Float16* W1 = reinterpret_cast<const _Float16*>(w);
    const _Float16* W2 = W1 + 32 * 32;
    const _Float16* W3 = W2 + 32 * 32;
    const _Float16 z = (_Float16)0.f;
    for (int e = threadIdx.x; e < kWave * 8; e += blockDim.x) {
        const int l = e >> 3, j = e & 7, g = l >> 4, c = l & 15;
        const int k = kslot(g, j);
        for (int b = 0; b < 2; ++b) {
            const int row = 16 * b + c;
            s.w1a[b][l][j] = W1[row * 32 + k];
            s.w2a[b][l][j] = W2[row * 32 + k];
            if (backward) {
                s.w1t[b][l][j] = W1[k * 32 + row];
                s.w2t[b][l][j] = W2[k * 32 + row];
                if (j < 4) s.w3t[b][l][j] = 4 * g + j < GS_MLP_OUT ? W3[(4 * g + j) * 32 + row] : z;
            }
        }
        s.w3a[l][j] = c < GS_MLP_OUT ? W3[c * 32 + k] : z;
    }
    __syncthreads();
}

__device__ __forceinline__ float4_t neural_tile_out(const MlpFrags& W, const half8_t& x)
{
    float4_t h1[2], h2[2], o;
    half8_t a1, a2;
    mlp_tile_fwd(W, x, h1, a1, h2, a2, o);
    return o;
}

__device__ __forceinline__ void neural_grad_zero(MlpGradAcc& a) { mlp_grad_zero(a); }
__device__ __forceinline__ void neural_grad_rescale(MlpGradAcc& a, int se) { mlp_grad_rescale(a, se); }

// Backward of tile t for the 32-neuron decoder, with the contract of
// neural_tile_bwd<L>: delta3 from st.d3 (scaled by 2^se), the hidden gradients
// chained neuron-major with binary16 hi + lo operands, the Gaussian-major copies
// for dWout, dW2, dW1, and the input gradients left in st.dxf and the input rows.
__device__ __forceinline__ void neural_tile_bwd(const MlpFrags& W, NeuralBwdStage& st, int t, float scale,
                                                float inv, MlpGradAcc& acc)
{
    const int l = __lane_id(), g = l >> 4, c = l & 15;
    const float4_t zero = {0.f, 0.f, 0.f, 0.f};
    const half8_t x = neural_stage_frag(st.x, t);
    half4_t xg[2];
#pragma unroll
    for (int fb = 0; fb < 2; ++fb)
#pragma unroll
        for (int j = 0; j < 4; ++j) xg[fb][j] = st.x[16 * t + 4 * g + j][16 * fb + c];
    // forward of the hidden layers, both orientations
    float4_t h1n[2], h2n[2], on;
    half8_t a1, a2;
    mlp_tile_fwd(W, x, h1n, a1, h2n, a2, on);
    float4_t h1g[2], h2g[2];
#pragma unroll
    for (int b = 0; b < 2; ++b) h1g[b] = mfma32(x, frag8(W.w1a[b]), zero);      // h1[G = 4g+i][16b + c]
#pragma unroll
    for (int b = 0; b < 2; ++b) h2g[b] = mfma32(a1, frag8(W.w2a[b]), zero);     // h2[G = 4g+i][16b + c]

    // output gradients, neuron-major (lanes g = 0) and Gaussian-major
    float4_t d3n = zero, d3g;
    const int Gn = 16 * t + c;
    if (g == 0)
#pragma unroll
        for (int i = 0; i < GS_MLP_OUT; ++i) d3n[i] = st.d3[Gn][i] * scale;
    const int cn = min(c, 3);
#pragma unroll
    for (int i = 0; i < 4; ++i) d3g[i] = st.d3[16 * t + 4 * g + i][cn] * scale;
    half4_t d3n_hi, d3n_lo;
    split4(d3n, d3n_hi, d3n_lo);
    const half4_t d3g_h = half4_t{(_Float16)d3g[0], (_Float16)d3g[1], (_Float16)d3g[2], (_Float16)d3g[3]};

    // dH2 = Wout^T delta3, masked by relu'(h2)
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
    // dX = W1^T dH1: dx[b] holds inputs 16b + 4g + i of Gaussian c
    float4_t dx[2];
#pragma unroll
    for (int b = 0; b < 2; ++b) {
        const half8_t w = frag8(W.w1t[b]);
        dx[b] = mfma32(w, g1n_lo, mfma32(w, g1n_hi, zero)) * inv;
    }
    // the tile's input rows have been read: they now take the direction-input gradients
    wave_lds_sync();
    float* row = reinterpret_cast<float*>(&st.x[Gn][0]);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        row[4 * g + i] = dx[0][i];
        st.dxf[Gn][4 * g + i] = dx[1][i];
    }

    // weight gradients from the Gaussian-major fragments, accumulated in place
    half4_t r1g[2], r2g[2];
#pragma unroll
    for (int b = 0; b < 2; ++b) {
        r1g[b] = relu_half4(h1g[b]);
        r2g[b] = relu_half4(h2g[b]);
    }
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) acc.w3[nb] = mfma16(d3g_h, r2g[nb], acc.w3[nb]);          // dWout[o][n2]
#pragma unroll
    for (int mb = 0; mb < 2; ++mb) {
        const half4_t h = {(_Float16)g2g[mb][0], (_Float16)g2g[mb][1], (_Float16)g2g[mb][2], (_Float16)g2g[mb][3]};
#pragma unroll
        for (int nb = 0; nb < 2; ++nb) acc.w2[mb][nb] = mfma16(h, r1g[nb], acc.w2[mb][nb]);   // dW2[n2][n1]
    }
#pragma unroll
    for (int mb = 0; mb < 2; ++mb) {
        const half4_t h = {(_Float16)g1g[mb][0], (_Float16)g1g[mb][1], (_Float16)g1g[mb][2], (_Float16)g1g[mb][3]};
#pragma unroll
        for (int fb = 0; fb < 2; ++fb) acc.w1[mb][fb] = mfma16(h, xg[fb], acc.w1[mb][fb]);    // dW1[n1][input]
    }
}

// Adds a wave's weight-gradient sums into the workgroup buffer `red` in the
// weights' order (16-neuron decoder with L hidden layers, or the 32-neuron one).
template <int L>
__device__ __forceinline__ void neural_grad_add(const NeuralGradAcc<L>& acc, float* red)
{
    const int l = __lane_id(), g = l >> 4, c = l & 15;
    for (int e = 0; e < 4; ++e) {
        const int row = 4 * g + e;
        for (int fb = 0; fb < 2; ++fb) red[row * kNeuralIn + 16 * fb + c] += acc.w1[fb][e];
        for (int h = 0; h < L - 1; ++h)
            red[kNeuralHidden * kNeuralIn + h * kNeuralHidden * kNeuralHidden + row * kNeuralHidden + c] +=
                acc.wh[h][e];
        if (row < GS_MLP_OUT)
            red[kNeuralHidden * kNeuralIn + (L - 1) * kNeuralHidden * kNeuralHidden + row * kNeuralHidden + c] +=
                acc.w3[e];
    }
}

__device__ __forceinline__ void neural_grad_add(const MlpGradAcc& acc, float* red)
{
    const int l = __lane_id(), g = l >> 4, c = l & 15;
    for (int e = 0; e < 4; ++e) {
        for (int mb = 0; mb < 2; ++mb) {
            const int row = 16 * mb + 4 * g + e;
            for (int fb = 0; fb < 2; ++fb) red[row * 32 + 16 * fb + c] += acc.w1[mb][fb][e];
            for (int nb = 0; nb < 2; ++nb) red[32 * 32 + row * 32 + 16 * nb + c] += acc.w2[mb][nb][e];
        }
        const int o = 4 * g + e;
        if (o < GS_MLP_OUT)
            for (int nb = 0; nb < 2; ++nb) red[2 * 32 * 32 + o * 32 + 16 * nb + c] += acc.w3[nb][e];
    }
}

}  // namespace gsr
