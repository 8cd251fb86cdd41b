// The latent decoder c = sigmoid(W3 relu(W2 relu(W1 [z, d]))) (no biases;
// 17 -> 32 -> 32 -> 3) on the matrix cores, for 16 Gaussians at a time, and its
// backward pass. Half-precision operands, fp32 accumulation (Sec. 4 and the
// appendix on the fused rasterizer: the decoder runs in half precision).
//
// Everything is computed transposed, neurons x Gaussians, with
// v_mfma_f32_16x16x16_f16:  D[m][n] = sum_k A[m][k] B[k][n] + C[m][n], where
// lane l holds A[l%16][4(l/16) + j], B[4(l/16) + j][l%16] (j = 0..3) and
// D[4(l/16) + i][l%16] (i = 0..3). A layer's D fragment for neurons 16b..16b+15
// is therefore exactly the B fragment of the next layer's K-half b, so the
// activations stay in registers from layer to layer.
#pragma once

#include "gs_internal.h"

namespace gsr {

typedef _Float16 half4_t __attribute__((ext_vector_type(4)));
typedef float float4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float4_t mfma16(half4_t a, half4_t b, float4_t c)
{
    return __builtin_amdgcn_mfma_f32_16x16x16f16(a, b, c, 0, 0, 0);
}

// Row pitches (in halves) chosen so that the 16 rows an MFMA fragment reads
// fall into distinct LDS banks.
constexpr int kP32 = 36;   // rows of 32 values
constexpr int kP16 = 20;   // rows of 16 values

// Shared (per workgroup) copies of the weights, zero-padded, in the four
// orientations the products need. Row-major [rows][cols].
struct MlpWeights {
    _Float16 w1[32][kP32];    // W1[n][k], k < 17
    _Float16 w1t[32][kP32];   // W1^T[k][n], k < 17
    _Float16 w2[32][kP32];
    _Float16 w2t[32][kP32];
    _Float16 w3[16][kP32];    // W3[o][n], o < 3
    _Float16 w3t[32][kP16];   // W3^T[n][o], o < 3
};

// Loads the binary16 weights (W1[32][17], W2[32][32], W3[3][32]) into LDS.
// Called by every thread of the workgroup; ends with a barrier.
__device__ __forceinline__ void mlp_load_weights(const uint16_t* __restrict__ w, MlpWeights& s)
{
    const _Float16* src = reinterpret_cast<const _Float16*>(w);
    for (int e = threadIdx.x; e < 32 * 32; e += blockDim.x) {
        const int r = e >> 5, c = e & 31;
        s.w1[r][c] = c < GS_MLP_IN ? src[r * GS_MLP_IN + c] : (_Float16)0.f;
        s.w1t[r][c] = r < GS_MLP_IN ? src[c * GS_MLP_IN + r] : (_Float16)0.f;
        s.w2[r][c] = src[32 * GS_MLP_IN + r * 32 + c];
        s.w2t[r][c] = src[32 * GS_MLP_IN + c * 32 + r];
    }
    for (int e = threadIdx.x; e < 16 * 32; e += blockDim.x) {
        const int r = e >> 5, c = e & 31;
        s.w3[r][c] = r < GS_MLP_OUT ? src[32 * GS_MLP_IN + 32 * 32 + r * 32 + c] : (_Float16)0.f;
        const int n = e >> 4, o = e & 15;
        s.w3t[n][o] = o < GS_MLP_OUT ? src[32 * GS_MLP_IN + 32 * 32 + o * 32 + n] : (_Float16)0.f;
    }
    __syncthreads();
}

// Decoder inputs of the wave's 64 Gaussians, row = lane: latent 0..13,
// direction 14..16, zeros up to 32.
struct MlpInputs {
    _Float16 x[64][kP32];
};

// Per-wave scratch of the backward for one tile of 16 Gaussians. Gradients
// enter the matrix cores as a high and a low binary16 part (v = hi + lo), so
// the chain keeps about 22 bits of precision instead of 11.
struct MlpBwdTile {
    _Float16 h1t[32][kP16];   // hidden activations, transposed (neuron x Gaussian)
    _Float16 h2t[32][kP16];
    _Float16 g1t[2][32][kP16];   // masked, scaled gradients of the hidden layers, transposed (hi, lo)
    _Float16 g2t[2][32][kP16];
    _Float16 d3t[2][16][kP16];   // scaled output gradients, transposed (hi, lo; rows 3..15 zero)
    float dx[16][GS_MLP_IN];  // input gradients, row = Gaussian
};

// v = hi + lo with both parts binary16.
__device__ __forceinline__ _Float16 half_hi(float v) { return (_Float16)v; }
__device__ __forceinline__ _Float16 half_lo(float v) { return (_Float16)(v - (float)(_Float16)v); }

// Orders this wave's LDS writes before its following LDS reads by other lanes.
__device__ __forceinline__ void wave_lds_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ half4_t lds_half4(const _Float16* p)
{
    return *reinterpret_cast<const half4_t*>(p);
}

__device__ __forceinline__ half4_t relu_half4(float4_t v)
{
    half4_t h;
    for (int i = 0; i < 4; ++i) h[i] = (_Float16)(v[i] > 0.f ? v[i] : 0.f);
    return h;
}

// Forward of tile `tile` (rows 16 tile .. 16 tile + 15 of in.x). On return
// h1[b], h2[b] hold the fp32 pre-activations of neurons 16b + 4(l/16) + i of
// Gaussian l%16 of the tile, and o the output pre-activations 4(l/16) + i
// (outputs are lanes 0..15, i < 3).
__device__ __forceinline__ void mlp_tile_forward(const MlpWeights& W, const MlpInputs& in, int tile, float4_t h1[2],
                                                 float4_t h2[2], float4_t& o)
{
    const int lane = __lane_id(), r = lane & 15, kq = 4 * (lane >> 4);
    const float4_t zero = {0.f, 0.f, 0.f, 0.f};
    half4_t xb[2];
    xb[0] = lds_half4(&in.x[16 * tile + r][kq]);
    xb[1] = lds_half4(&in.x[16 * tile + r][16 + kq]);
    half4_t a1[2];
    for (int b = 0; b < 2; ++b) {
        float4_t acc = zero;
        acc = mfma16(lds_half4(&W.w1[16 * b + r][kq]), xb[0], acc);
        acc = mfma16(lds_half4(&W.w1[16 * b + r][16 + kq]), xb[1], acc);
        h1[b] = acc;
        a1[b] = relu_half4(acc);
    }
    half4_t a2[2];
    for (int b = 0; b < 2; ++b) {
        float4_t acc = zero;
        acc = mfma16(lds_half4(&W.w2[16 * b + r][kq]), a1[0], acc);
        acc = mfma16(lds_half4(&W.w2[16 * b + r][16 + kq]), a1[1], acc);
        h2[b] = acc;
        a2[b] = relu_half4(acc);
    }
    float4_t acc = zero;
    acc = mfma16(lds_half4(&W.w3[r][kq]), a2[0], acc);
    acc = mfma16(lds_half4(&W.w3[r][16 + kq]), a2[1], acc);
    o = acc;
}

__device__ __forceinline__ float sigmoid_fast(float x)
{
    return 1.f / (1.f + __builtin_amdgcn_exp2f(-x * 1.4426950408889634f));
}

// Stages this lane's decoder input into row `lane` of in.x: the binary16 latent
// as stored, then the view direction rounded to binary16 (round to nearest
// even), zeros elsewhere and for culled lanes.
__device__ __forceinline__ void mlp_stage_lane(MlpInputs& in, bool valid, const uint16_t* __restrict__ latent,
                                               int64_t n, int64_t i, const float d[3])
{
    const int row = __lane_id();
    for (int c = 0; c < 32; ++c) {
        _Float16 v = (_Float16)0.f;
        if (valid) {
            if (c < GS_LATENT_DIM) {
                const uint16_t bits = latent[c * n + i];
                v = __builtin_bit_cast(_Float16, bits);
            } else if (c < GS_MLP_IN) {
                v = (_Float16)d[c - GS_LATENT_DIM];
            }
        }
        in.x[row][c] = v;
    }
}

// Moves the tile's colours (lanes 0..15 after mlp_tile_forward) to the lanes
// that own the Gaussians (16 tile .. 16 tile + 15).
__device__ __forceinline__ void mlp_tile_colors(const float4_t& o, int tile, float col[3])
{
    const int lane = __lane_id();
    const int src = lane & 15;
    for (int c = 0; c < 3; ++c) {
        const float v = __shfl(sigmoid_fast(o[c]), src);
        if ((lane >> 4) == tile) col[c] = v;
    }
}

}  // namespace gsr
