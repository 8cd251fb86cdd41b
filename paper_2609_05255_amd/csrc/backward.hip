// Preprocess backward: one thread per Gaussian chains the screen-space
// gradients accumulated by the blend backward (projected mean, conic, opacity,
// colour) back to the parameters: through the EWA covariance and the pinhole
// Jacobian (with the guard-band clamp), the rotation and scale activations, the
// opacity logistic, and the appearance model -- including the colour gradient
// through the view direction into the mean (Sec. 4 fused backward). Gradients
// of culled Gaussians are written as zeros, so every output is dense.
#include "gs_internal.h"
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
    const uint32_t* tiles_touched;
    const float* acc;
    float* dmeans;
    float* dlog_scales;
    float* dquats;
    float* dlogits;
    float* dsh;
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
    if (a.tiles_touched[i] == 0) {
        write_zero_grads(a, i);
        for (int k = 0; k < GS_SH_COEFFS; ++k) a.dsh[k * n + i] = 0.f;
        return;
    }
    float mu[3], ls[3], q[4];
    for (int j = 0; j < 3; ++j) mu[j] = a.means[j * n + i];
    for (int j = 0; j < 3; ++j) ls[j] = a.log_scales[j * n + i];
    for (int j = 0; j < 4; ++j) q[j] = a.quats[j * n + i];
    const float logit = a.logits[i];
    float g9[kAccStride];
    const float* ap = a.acc + (size_t)i * kAccStride;
    for (int k = 0; k < kAccStride; ++k) g9[k] = ap[k];
    GeoGrad gg;
    geometry_bwd(a.cam, mu, ls, q, logit, g9, gg);

    // appearance: eq. sh_color_eval with its ReLU
    const float vx = mu[0] - a.cam.campos[0], vy = mu[1] - a.cam.campos[1], vz = mu[2] - a.cam.campos[2];
    const float len = sqrtf(vx * vx + vy * vy + vz * vz);
    const float il = 1.f / len;
    const float d0 = vx * il, d1 = vy * il, d2 = vz * il;
    float Y[16];
    sh_basis16(d0, d1, d2, Y);
    const int nb = (a.sh_degree + 1) * (a.sh_degree + 1);
    float coef[48];
    float pre0 = 0.5f, pre1 = 0.5f, pre2 = 0.5f;
    for (int k = 0; k < 16; ++k) {
        if (k < nb) {
            coef[3 * k] = a.sh[(3 * k) * n + i];
            coef[3 * k + 1] = a.sh[(3 * k + 1) * n + i];
            coef[3 * k + 2] = a.sh[(3 * k + 2) * n + i];
            pre0 += Y[k] * coef[3 * k];
            pre1 += Y[k] * coef[3 * k + 1];
            pre2 += Y[k] * coef[3 * k + 2];
        } else {
            coef[3 * k] = coef[3 * k + 1] = coef[3 * k + 2] = 0.f;
        }
    }
    const float gc0 = pre0 > 0.f ? g9[6] : 0.f;
    const float gc1 = pre1 > 0.f ? g9[7] : 0.f;
    const float gc2 = pre2 > 0.f ? g9[8] : 0.f;
    float G[48];
    sh_basis16_grad(d0, d1, d2, G);
    float dd0 = 0.f, dd1 = 0.f, dd2 = 0.f;
    for (int k = 0; k < 16; ++k) {
        const bool on = k < nb;
        a.dsh[(3 * k) * n + i] = on ? Y[k] * gc0 : 0.f;
        a.dsh[(3 * k + 1) * n + i] = on ? Y[k] * gc1 : 0.f;
        a.dsh[(3 * k + 2) * n + i] = on ? Y[k] * gc2 : 0.f;
        const float dY = coef[3 * k] * gc0 + coef[3 * k + 1] * gc1 + coef[3 * k + 2] * gc2;
        dd0 += dY * G[3 * k];
        dd1 += dY * G[3 * k + 1];
        dd2 += dY * G[3 * k + 2];
    }
    // d = v / |v|: dv = (dd - d (d . dd)) / |v|
    const float dot = d0 * dd0 + d1 * dd1 + d2 * dd2;
    gg.dmu[0] += (dd0 - d0 * dot) * il;
    gg.dmu[1] += (dd1 - d1 * dot) * il;
    gg.dmu[2] += (dd2 - d2 * dot) * il;

    for (int j = 0; j < 3; ++j) { a.dmeans[j * n + i] = gg.dmu[j]; a.dlog_scales[j * n + i] = gg.dls[j]; }
    for (int j = 0; j < 4; ++j) a.dquats[j * n + i] = gg.dq[j];
    a.dlogits[i] = gg.dlogit;
    if (a.dmean2d) { a.dmean2d[i] = g9[0]; a.dmean2d[n + i] = g9[1]; }
}

hipError_t launch_preprocess_bwd(const Cam& cam, const gs_gaussians& g, const gs_appearance& app,
                                 const gs_preprocessed& pre, const Workspace& ws, const gs_grads& gr, hipStream_t s)
{
    if (app.kind != GS_APP_SH3) return hipErrorNotSupported;
    BwdArgs a;
    a.cam = cam;
    a.n = (int)g.n;
    a.means = g.means;
    a.log_scales = g.log_scales;
    a.quats = g.quats;
    a.logits = g.opacity_logits;
    a.sh_degree = app.sh_degree;
    a.sh = app.sh;
    a.tiles_touched = pre.tiles_touched;
    a.acc = ws.acc;
    a.dmeans = gr.dmeans;
    a.dlog_scales = gr.dlog_scales;
    a.dquats = gr.dquats;
    a.dlogits = gr.dopacity_logits;
    a.dsh = gr.dsh;
    a.dmean2d = gr.dmean2d;
    hipLaunchKernelGGL(k_preprocess_bwd_sh3, dim3(preprocess_blocks(g.n)), dim3(kBlock), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_mlp_reduce(int64_t, const Workspace&, float*, hipStream_t) { return hipErrorNotSupported; }

}  // namespace gsr
