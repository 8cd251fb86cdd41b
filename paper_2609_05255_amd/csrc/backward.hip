// Preprocess backward: one thread per Gaussian chains the screen-space
// gradients accumulated by the blend backward (projected mean, conic, opacity,
// colour) back to the parameters: through the EWA covariance and the pinhole
// Jacobian (with the guard-band clamp), the rotation and scale activations, the
// opacity logistic, and the appearance model -- including the colour gradient
// through the view direction into the mean (Sec. 4 fused backward). Gradients
// of culled Gaussians are written as zeros, so every output is dense.
#include "gs_internal.h"
#include "mlp.h"
#include "sh.h"

namespace gsr {

namespace {

struct BwdArgs {
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
    const uint32_t* tiles_touched;
    const float* acc;
    float* dmeans;
    float* dlog_scales;
    float* dquats;
    float* dlogits;
    float* dsh;
    float* dlatent;
    float* mlp_part;
    float* dmean2d;
};

struct GeoGrad {
    float dmu[3];
    float dls[3];
    float dq[4];
    float dlogit;
};

// Derivative of the geometry part of the preprocess (everything except colour).
__device__ __forceinline__ void geometry_bwd(const Cam& c, const float mu[3], const float ls[3], const float qraw[4],
                                             float logit, const float* g9, GeoGrad& out)
{
    float s[3];
    for (int j = 0; j < 3; ++j) s[j] = __expf(ls[j]);
    const float qn = sqrtf(qraw[0] * qraw[0] + qraw[1] * qraw[1] + qraw[2] * qraw[2] + qraw[3] * qraw[3]);
    const float iqn = 1.f / qn;
    const float w = qraw[0] * iqn, x = qraw[1] * iqn, y = qraw[2] * iqn, z = qraw[3] * iqn;
    const float R[9] = {1.f - 2.f * (y * y + z * z), 2.f * (x * y - w * z), 2.f * (x * z + w * y),
                        2.f * (x * y + w * z), 1.f - 2.f * (x * x + z * z), 2.f * (y * z - w * x),
                        2.f * (x * z - w * y), 2.f * (y * z + w * x), 1.f - 2.f * (x * x + y * y)};
    float M[9], S[9];
    for (int r = 0; r < 3; ++r)
        for (int k = 0; k < 3; ++k) M[3 * r + k] = R[3 * r + k] * s[k];
    for (int r = 0; r < 3; ++r)
        for (int k = 0; k < 3; ++k) S[3 * r + k] = M[3 * r] * M[3 * k] + M[3 * r + 1] * M[3 * k + 1] + M[3 * r + 2] * M[3 * k + 2];
    const float* V = c.V;
    float t[3];
    for (int r = 0; r < 3; ++r) t[r] = V[4 * r] * mu[0] + V[4 * r + 1] * mu[1] + V[4 * r + 2] * mu[2] + V[4 * r + 3];
    const float limx = 1.3f * ((0.5f * (float)c.width) / c.fx);
    const float limy = 1.3f * ((0.5f * (float)c.height) / c.fy);
    const float tz = t[2], itz = 1.f / tz, itz2 = itz * itz;
    const float txtz = t[0] * itz, tytz = t[1] * itz;
    const bool clx = txtz < -limx || txtz > limx;
    const bool cly = tytz < -limy || tytz > limy;
    const float ux = (clx ? (txtz < 0.f ? -limx : limx) : txtz) * tz;
    const float uy = (cly ? (tytz < 0.f ? -limy : limy) : tytz) * tz;
    const float j00 = c.fx * itz, j02 = -c.fx * ux * itz2, j11 = c.fy * itz, j12 = -c.fy * uy * itz2;
    float T[6];
    for (int k = 0; k < 3; ++k) {
        T[k] = j00 * V[k] + j02 * V[8 + k];
        T[3 + k] = j11 * V[4 + k] + j12 * V[8 + k];
    }
    float TS[6];
    for (int r = 0; r < 2; ++r)
        for (int k = 0; k < 3; ++k) TS[3 * r + k] = T[3 * r] * S[k] + T[3 * r + 1] * S[3 + k] + T[3 * r + 2] * S[6 + k];
    const float A = TS[0] * T[0] + TS[1] * T[1] + TS[2] * T[2] + 0.3f;
    const float B = TS[0] * T[3] + TS[1] * T[4] + TS[2] * T[5];
    const float C = TS[3] * T[3] + TS[4] * T[4] + TS[5] * T[5] + 0.3f;
    const float idet = 1.f / (A * C - B * B);
    const float qa = C * idet, qb = -B * idet, qc = A * idet;     // conic
    // dL/dcov = -Q GQ Q with GQ = [[da, db/2], [db/2, dc]]
    const float ga = g9[2], gb = 0.5f * g9[3], gc = g9[4];
    const float m00 = qa * ga + qb * gb, m01 = qa * gb + qb * gc;
    const float m10 = qb * ga + qc * gb, m11 = qb * gb + qc * gc;
    const float G00 = -(m00 * qa + m01 * qb), G01 = -(m00 * qb + m01 * qc);
    const float G11 = -(m10 * qb + m11 * qc);
    // cov = T S T^T: dT = 2 G2 T S, dS = T^T G2 T
    float dT[6];
    for (int k = 0; k < 3; ++k) {
        dT[k] = 2.f * (G00 * TS[k] + G01 * TS[3 + k]);
        dT[3 + k] = 2.f * (G01 * TS[k] + G11 * TS[3 + k]);
    }
    float dS[9];
    for (int r = 0; r < 3; ++r)
        for (int k = 0; k < 3; ++k)
            dS[3 * r + k] = T[r] * (G00 * T[k] + G01 * T[3 + k]) + T[3 + r] * (G01 * T[k] + G11 * T[3 + k]);
    // T = J W with J = [[j00, 0, j02], [0, j11, j12]]
    const float dj00 = dT[0] * V[0] + dT[1] * V[1] + dT[2] * V[2];
    const float dj02 = dT[0] * V[8] + dT[1] * V[9] + dT[2] * V[10];
    const float dj11 = dT[3] * V[4] + dT[4] * V[5] + dT[5] * V[6];
    const float dj12 = dT[3] * V[8] + dT[4] * V[9] + dT[5] * V[10];
    float dt[3] = {0.f, 0.f, 0.f};
    dt[2] += -c.fx * itz2 * dj00 - c.fy * itz2 * dj11;
    if (clx) dt[2] += c.fx * (ux * itz) * itz2 * dj02;                 // j02 = -fx (+-limx) / tz
    else { dt[0] += -c.fx * itz2 * dj02; dt[2] += 2.f * c.fx * t[0] * itz2 * itz * dj02; }
    if (cly) dt[2] += c.fy * (uy * itz) * itz2 * dj12;
    else { dt[1] += -c.fy * itz2 * dj12; dt[2] += 2.f * c.fy * t[1] * itz2 * itz * dj12; }
    // projected mean px = fx tx / tz + cx
    dt[0] += c.fx * itz * g9[0];
    dt[1] += c.fy * itz * g9[1];
    dt[2] += -(c.fx * t[0] * g9[0] + c.fy * t[1] * g9[1]) * itz2;
    for (int k = 0; k < 3; ++k) out.dmu[k] = V[k] * dt[0] + V[4 + k] * dt[1] + V[8 + k] * dt[2];
    // Sigma = M M^T: dM = 2 dS M (dS symmetric)
    float dR[9];
    for (int k = 0; k < 3; ++k) {
        float ds = 0.f;
        for (int r = 0; r < 3; ++r) {
            const float dm = 2.f * (dS[3 * r] * M[k] + dS[3 * r + 1] * M[3 + k] + dS[3 * r + 2] * M[6 + k]);
            ds += R[3 * r + k] * dm;
            dR[3 * r + k] = dm * s[k];
        }
        out.dls[k] = ds * s[k];
    }
    // rotation of the unit quaternion (w, x, y, z)
    float dqn[4];
    dqn[0] = 2.f * (z * (dR[3] - dR[1]) + y * (dR[2] - dR[6]) + x * (dR[7] - dR[5]));
    dqn[1] = 2.f * (y * (dR[1] + dR[3]) + z * (dR[2] + dR[6]) + w * (dR[7] - dR[5])) - 4.f * x * (dR[4] + dR[8]);
    dqn[2] = 2.f * (x * (dR[1] + dR[3]) + w * (dR[2] - dR[6]) + z * (dR[5] + dR[7])) - 4.f * y * (dR[0] + dR[8]);
    dqn[3] = 2.f * (w * (dR[3] - dR[1]) + x * (dR[2] + dR[6]) + y * (dR[5] + dR[7])) - 4.f * z * (dR[0] + dR[4]);
    const float qd = w * dqn[0] + x * dqn[1] + y * dqn[2] + z * dqn[3];
    out.dq[0] = (dqn[0] - w * qd) * iqn;
    out.dq[1] = (dqn[1] - x * qd) * iqn;
    out.dq[2] = (dqn[2] - y * qd) * iqn;
    out.dq[3] = (dqn[3] - z * qd) * iqn;
    const float o = 1.f / (1.f + __expf(-logit));
    out.dlogit = g9[5] * o * (1.f - o);
}

__device__ __forceinline__ void write_zero_grads(const BwdArgs& a, int i)
{
    const int64_t n = a.n;
    for (int j = 0; j < 3; ++j) { a.dmeans[j * n + i] = 0.f; a.dlog_scales[j * n + i] = 0.f; }
    for (int j = 0; j < 4; ++j) a.dquats[j * n + i] = 0.f;
    a.dlogits[i] = 0.f;
    if (a.dmean2d) { a.dmean2d[i] = 0.f; a.dmean2d[n + i] = 0.f; }
}

}  // namespace

__global__ __launch_bounds__(kBlock) void k_preprocess_bwd_sh3(BwdArgs a)
{
    const int i = blockIdx.x * kBlock + threadIdx.x;
    if (i >= a.n) return;
    const int64_t n = a.n;
    // Culled Gaussians take the same store instructions with zeros, so every
    // gradient plane is written once per wave with whole lines.
    const bool vis = a.tiles_touched[i] != 0;
    GeoGrad gg;
    for (int j = 0; j < 3; ++j) { gg.dmu[j] = 0.f; gg.dls[j] = 0.f; }
    for (int j = 0; j < 4; ++j) gg.dq[j] = 0.f;
    gg.dlogit = 0.f;
    float g9[kAccStride];
    for (int k = 0; k < kAccStride; ++k) g9[k] = 0.f;
    float Y[16], gc[3] = {0.f, 0.f, 0.f};
    for (int k = 0; k < 16; ++k) Y[k] = 0.f;
    const int nb = (a.sh_degree + 1) * (a.sh_degree + 1);
    if (vis) {
        float mu[3], ls[3], q[4];
        for (int j = 0; j < 3; ++j) mu[j] = a.means[j * n + i];
        for (int j = 0; j < 3; ++j) ls[j] = a.log_scales[j * n + i];
        for (int j = 0; j < 4; ++j) q[j] = a.quats[j * n + i];
        const float* ap = a.acc + (size_t)i * kAccStride;
        for (int k = 0; k < kAccStride; ++k) g9[k] = ap[k];
        geometry_bwd(a.cam, mu, ls, q, a.logits[i], g9, gg);

        // appearance: eq. sh_color_eval with its ReLU
        const float vx = mu[0] - a.cam.campos[0], vy = mu[1] - a.cam.campos[1], vz = mu[2] - a.cam.campos[2];
        const float len = sqrtf(vx * vx + vy * vy + vz * vz);
        const float il = 1.f / len;
        const float d0 = vx * il, d1 = vy * il, d2 = vz * il;
        sh_basis16(d0, d1, d2, Y);
        float coef[GS_SH_COEFFS];
        float pre[3] = {0.5f, 0.5f, 0.5f};
        for (int k = 0; k < 16; ++k)
            for (int c = 0; c < 3; ++c) {
                coef[3 * k + c] = k < nb ? a.sh[(3 * k + c) * n + i] : 0.f;
                pre[c] += Y[k] * coef[3 * k + c];
            }
        for (int c = 0; c < 3; ++c) gc[c] = pre[c] > 0.f ? g9[6 + c] : 0.f;
        float dY[16];
        for (int k = 0; k < 16; ++k) dY[k] = coef[3 * k] * gc[0] + coef[3 * k + 1] * gc[1] + coef[3 * k + 2] * gc[2];
        float dd[3] = {0.f, 0.f, 0.f};
        sh_basis16_vjp(d0, d1, d2, dY, dd);
        // d = v / |v|: dv = (dd - d (d . dd)) / |v|
        const float dot = d0 * dd[0] + d1 * dd[1] + d2 * dd[2];
        gg.dmu[0] += (dd[0] - d0 * dot) * il;
        gg.dmu[1] += (dd[1] - d1 * dot) * il;
        gg.dmu[2] += (dd[2] - d2 * dot) * il;
    }
    for (int k = 0; k < 16; ++k) {
        const bool on = k < nb;
        for (int c = 0; c < 3; ++c) a.dsh[(3 * k + c) * n + i] = on ? Y[k] * gc[c] : 0.f;
    }
    for (int j = 0; j < 3; ++j) { a.dmeans[j * n + i] = gg.dmu[j]; a.dlog_scales[j * n + i] = gg.dls[j]; }
    for (int j = 0; j < 4; ++j) a.dquats[j * n + i] = gg.dq[j];
    a.dlogits[i] = gg.dlogit;
    if (a.dmean2d) { a.dmean2d[i] = g9[0]; a.dmean2d[n + i] = g9[1]; }
}

// Latent + MLP backward. Grid-stride over chunks of 256 Gaussians so that the
// workgroup count, and with it the number of partial weight gradients, stays
// bounded. Per wave and tile of 16 Gaussians: recompute the decoder, delta3 =
// dL/dc * s (1 - s), scale it by a power of two so that its largest magnitude
// lies in [2^9, 2^10) (exact, removed again in fp32), then dH2, dH1 and dX on
// the matrix cores in registers and dW3, dW2, dW1 from LDS-transposed
// fragments with the tile's Gaussians as the reduction dimension. Every
// gradient operand is passed as two binary16 parts (hi + lo).
__global__ __launch_bounds__(kBlock) void k_preprocess_bwd_latent(BwdArgs a)
{
    __shared__ MlpWeights W;
    __shared__ MlpInputs X[kBlock / kWave];
    __shared__ MlpBwdTile TT[kBlock / kWave];
    mlp_load_weights(a.mlp_w, W);
    const int wave = threadIdx.x >> 6, lane = __lane_id();
    const int r = lane & 15, g4 = lane >> 4, kq = 4 * g4;
    MlpInputs& XI = X[wave];
    MlpBwdTile& T = TT[wave];
    for (int e = lane; e < 2 * 16 * kP16; e += kWave) (&T.d3t[0][0][0])[e] = (_Float16)0.f;
    const float4_t zero = {0.f, 0.f, 0.f, 0.f};
    float4_t aw1[2][2], aw2[2][2], aw3[2];
    for (int u = 0; u < 2; ++u) {
        aw3[u] = zero;
        for (int v = 0; v < 2; ++v) { aw1[u][v] = zero; aw2[u][v] = zero; }
    }
    const int64_t n = a.n;
    const int64_t nchunks = div_up(n, kBlock);
    for (int64_t chunk = blockIdx.x; chunk < nchunks; chunk += gridDim.x) {
        const int64_t i = chunk * kBlock + threadIdx.x;
        const bool inb = i < n;
        const bool valid = inb && a.tiles_touched[i] != 0;
        if (inb && !valid) {
            write_zero_grads(a, (int)i);
            for (int c = 0; c < GS_LATENT_DIM; ++c) a.dlatent[c * n + i] = 0.f;
        }
        float mu[3] = {0.f, 0.f, 0.f}, d[3] = {0.f, 0.f, 0.f}, g9[kAccStride];
        float len = 1.f;
        GeoGrad gg;
        if (valid) {
            float ls[3], q[4];
            for (int j = 0; j < 3; ++j) mu[j] = a.means[j * n + i];
            for (int j = 0; j < 3; ++j) ls[j] = a.log_scales[j * n + i];
            for (int j = 0; j < 4; ++j) q[j] = a.quats[j * n + i];
            const float* ap = a.acc + (size_t)i * kAccStride;
            for (int k = 0; k < kAccStride; ++k) g9[k] = ap[k];
            geometry_bwd(a.cam, mu, ls, q, a.logits[i], g9, gg);
            const float vx = mu[0] - a.cam.campos[0], vy = mu[1] - a.cam.campos[1], vz = mu[2] - a.cam.campos[2];
            len = sqrtf(vx * vx + vy * vy + vz * vz);
            d[0] = vx / len;
            d[1] = vy / len;
            d[2] = vz / len;
        } else {
            for (int k = 0; k < kAccStride; ++k) g9[k] = 0.f;
        }
        mlp_stage_lane(XI, valid, a.latent, n, i, d);
        wave_lds_sync();
        float dxo[GS_MLP_IN];
        for (int c = 0; c < GS_MLP_IN; ++c) dxo[c] = 0.f;
        const uint64_t vis = __ballot(valid);
        for (int t = 0; t < kWave / 16; ++t) {
            if (((vis >> (16 * t)) & 0xFFFFull) == 0) continue;
            float4_t h1[2], h2[2], o;
            mlp_tile_forward(W, XI, t, h1, h2, o);
            // output gradient of the tile's Gaussian r, in lanes 0..15
            const int src = 16 * t + r;
            float del[3];
            for (int c = 0; c < 3; ++c) {
                const float dc = __shfl(g9[6 + c], src);
                const float sgm = sigmoid_fast(o[c]);
                del[c] = lane < 16 ? dc * sgm * (1.f - sgm) : 0.f;
            }
            float m = fmaxf(fabsf(del[0]), fmaxf(fabsf(del[1]), fabsf(del[2])));
            for (int off = 32; off > 0; off >>= 1) m = fmaxf(m, __shfl_xor(m, off));
            int ex = 0;
            if (m > 0.f) frexpf(m, &ex);
            const int se = min(10 - ex, 100);
            const float scale = m > 0.f ? ldexpf(1.f, se) : 1.f;
            const float inv = m > 0.f ? ldexpf(1.f, -se) : 1.f;
            half4_t d3b[2];
            for (int c = 0; c < 3; ++c) {
                d3b[0][c] = half_hi(del[c] * scale);
                d3b[1][c] = half_lo(del[c] * scale);
            }
            d3b[0][3] = d3b[1][3] = (_Float16)0.f;
            if (lane < 16)
                for (int p = 0; p < 2; ++p)
                    for (int c = 0; c < 3; ++c) T.d3t[p][c][r] = d3b[p][c];
            // dH2^T = W3^T delta3^T, masked by relu'(h2)
            half4_t g2h[2][2], g1h[2][2];   // [hi/lo][K-half]
            for (int b = 0; b < 2; ++b) {
                const half4_t w = lds_half4(&W.w3t[16 * b + r][kq]);
                float4_t v = mfma16(w, d3b[0], zero);
                v = mfma16(w, d3b[1], v);
                for (int e = 0; e < 4; ++e) {
                    const float m2 = h2[b][e] > 0.f ? v[e] : 0.f;
                    g2h[0][b][e] = half_hi(m2);
                    g2h[1][b][e] = half_lo(m2);
                }
            }
            // dH1^T = W2^T dH2^T, masked by relu'(h1)
            for (int b = 0; b < 2; ++b) {
                const half4_t w0 = lds_half4(&W.w2t[16 * b + r][kq]), w1 = lds_half4(&W.w2t[16 * b + r][16 + kq]);
                float4_t v = zero;
                for (int p = 0; p < 2; ++p) {
                    v = mfma16(w0, g2h[p][0], v);
                    v = mfma16(w1, g2h[p][1], v);
                }
                for (int e = 0; e < 4; ++e) {
                    const float m1 = h1[b][e] > 0.f ? v[e] : 0.f;
                    g1h[0][b][e] = half_hi(m1);
                    g1h[1][b][e] = half_lo(m1);
                }
            }
            // dX^T = W1^T dH1^T
            for (int b = 0; b < 2; ++b) {
                const half4_t w0 = lds_half4(&W.w1t[16 * b + r][kq]), w1 = lds_half4(&W.w1t[16 * b + r][16 + kq]);
                float4_t v = zero;
                for (int p = 0; p < 2; ++p) {
                    v = mfma16(w0, g1h[p][0], v);
                    v = mfma16(w1, g1h[p][1], v);
                }
                for (int e = 0; e < 4; ++e) {
                    const int c = 16 * b + kq + e;
                    if (c < GS_MLP_IN) T.dx[r][c] = v[e] * inv;
                }
            }
            // transposed fragments for the weight gradients
            for (int b = 0; b < 2; ++b)
                for (int e = 0; e < 4; ++e) {
                    const int nn = 16 * b + kq + e;
                    T.h1t[nn][r] = (_Float16)(h1[b][e] > 0.f ? h1[b][e] : 0.f);
                    T.h2t[nn][r] = (_Float16)(h2[b][e] > 0.f ? h2[b][e] : 0.f);
                    for (int p = 0; p < 2; ++p) {
                        T.g1t[p][nn][r] = g1h[p][b][e];
                        T.g2t[p][nn][r] = g2h[p][b][e];
                    }
                }
            wave_lds_sync();
            // dW3[o][n] += sum_G delta3[G][o] h2[G][n]
            for (int nb = 0; nb < 2; ++nb) {
                const half4_t h2b = lds_half4(&T.h2t[16 * nb + r][kq]);
                float4_t p = mfma16(lds_half4(&T.d3t[0][r][kq]), h2b, zero);
                p = mfma16(lds_half4(&T.d3t[1][r][kq]), h2b, p);
                aw3[nb] += p * inv;
            }
            // dW2[n][k] += sum_G dh2[G][n] h1[G][k];  dW1[n][k] += sum_G dh1[G][n] x[G][k]
            for (int nb = 0; nb < 2; ++nb) {
                half4_t xb;
                for (int j = 0; j < 4; ++j) xb[j] = XI.x[16 * t + kq + j][16 * nb + r];
                const half4_t h1b = lds_half4(&T.h1t[16 * nb + r][kq]);
                for (int mb = 0; mb < 2; ++mb) {
                    float4_t p2 = mfma16(lds_half4(&T.g2t[0][16 * mb + r][kq]), h1b, zero);
                    p2 = mfma16(lds_half4(&T.g2t[1][16 * mb + r][kq]), h1b, p2);
                    aw2[mb][nb] += p2 * inv;
                    float4_t p1 = mfma16(lds_half4(&T.g1t[0][16 * mb + r][kq]), xb, zero);
                    p1 = mfma16(lds_half4(&T.g1t[1][16 * mb + r][kq]), xb, p1);
                    aw1[mb][nb] += p1 * inv;
                }
            }
            if (g4 == t)
                for (int c = 0; c < GS_MLP_IN; ++c) dxo[c] = T.dx[r][c];
            wave_lds_sync();
        }
        if (valid) {
            for (int c = 0; c < GS_LATENT_DIM; ++c) a.dlatent[c * n + i] = dxo[c];
            // the binary16 rounding of d passes the gradient; d = v / |v|
            const float dd0 = dxo[14], dd1 = dxo[15], dd2 = dxo[16];
            const float dot = d[0] * dd0 + d[1] * dd1 + d[2] * dd2;
            const float il = 1.f / len;
            gg.dmu[0] += (dd0 - d[0] * dot) * il;
            gg.dmu[1] += (dd1 - d[1] * dot) * il;
            gg.dmu[2] += (dd2 - d[2] * dot) * il;
            for (int j = 0; j < 3; ++j) { a.dmeans[j * n + i] = gg.dmu[j]; a.dlog_scales[j * n + i] = gg.dls[j]; }
            for (int j = 0; j < 4; ++j) a.dquats[j * n + i] = gg.dq[j];
            a.dlogits[i] = gg.dlogit;
            if (a.dmean2d) { a.dmean2d[i] = g9[0]; a.dmean2d[n + i] = g9[1]; }
        }
    }
    // workgroup sum of the four waves' weight gradients, in wave order
    __syncthreads();
    float* red = reinterpret_cast<float*>(&X[0]);
    for (int k = threadIdx.x; k < GS_MLP_WEIGHTS; k += kBlock) red[k] = 0.f;
    __syncthreads();
    for (int w = 0; w < kBlock / kWave; ++w) {
        if (wave == w) {
            for (int mb = 0; mb < 2; ++mb)
                for (int nb = 0; nb < 2; ++nb)
                    for (int e = 0; e < 4; ++e) {
                        const int nn = 16 * mb + kq + e, k = 16 * nb + r;
                        if (k < GS_MLP_IN) red[nn * GS_MLP_IN + k] += aw1[mb][nb][e];
                        red[32 * GS_MLP_IN + nn * 32 + k] += aw2[mb][nb][e];
                    }
            for (int nb = 0; nb < 2; ++nb)
                for (int e = 0; e < 4; ++e) {
                    const int o = kq + e, k = 16 * nb + r;
                    if (o < GS_MLP_OUT) red[32 * GS_MLP_IN + 32 * 32 + o * 32 + k] += aw3[nb][e];
                }
        }
        __syncthreads();
    }
    for (int k = threadIdx.x; k < GS_MLP_WEIGHTS; k += kBlock)
        a.mlp_part[(size_t)blockIdx.x * GS_MLP_WEIGHTS + k] = red[k];
}

// dW = sum of the per-workgroup partials in workgroup order.
__global__ __launch_bounds__(kBlock) void k_mlp_reduce(const float* __restrict__ part, int nparts,
                                                       float* __restrict__ dw)
{
    const int k = blockIdx.x * kBlock + threadIdx.x;
    if (k >= GS_MLP_WEIGHTS) return;
    float s = 0.f;
    for (int b = 0; b < nparts; ++b) s += part[(size_t)b * GS_MLP_WEIGHTS + k];
    dw[k] = s;
}

inline int latent_bwd_grid(int64_t n) { return (int)std::min<int64_t>(div_up(n, kBlock), kMlpPartials); }

hipError_t launch_preprocess_bwd(const Cam& cam, const gs_gaussians& g, const gs_appearance& app,
                                 const gs_preprocessed& pre, const Workspace& ws, const gs_grads& gr, hipStream_t s)
{
    BwdArgs a;
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
    a.tiles_touched = pre.tiles_touched;
    a.acc = ws.acc;
    a.dmeans = gr.dmeans;
    a.dlog_scales = gr.dlog_scales;
    a.dquats = gr.dquats;
    a.dlogits = gr.dopacity_logits;
    a.dsh = gr.dsh;
    a.dlatent = gr.dlatent;
    a.mlp_part = ws.mlp_part;
    a.dmean2d = gr.dmean2d;
    if (app.kind == GS_APP_SH3)
        hipLaunchKernelGGL(k_preprocess_bwd_sh3, dim3(preprocess_blocks(g.n)), dim3(kBlock), 0, s, a);
    else
        hipLaunchKernelGGL(k_preprocess_bwd_latent, dim3(latent_bwd_grid(g.n)), dim3(kBlock), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_mlp_reduce(int64_t n, const Workspace& ws, float* dmlp_w, hipStream_t s)
{
    hipLaunchKernelGGL(k_mlp_reduce, dim3((unsigned)div_up(GS_MLP_WEIGHTS, kBlock)), dim3(kBlock), 0, s, ws.mlp_part,
                       latent_bwd_grid(n), dmlp_w);
    return hipGetLastError();
}

}  // namespace gsr
