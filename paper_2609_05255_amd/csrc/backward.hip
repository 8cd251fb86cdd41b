// Preprocess backward: one thread per Gaussian chains the screen-space
// gradients accumulated by the blend backward (projected mean, conic, opacity,
// colour) back to the parameters: through the EWA covariance and the pinhole
// Jacobian (with the guard-band clamp), the rotation and scale activations, the
// opacity logistic, and the appearance model -- including the colour gradient
// through the view direction into the mean (Sec. 4 fused backward). Gradients
// of culled Gaussians are written as zeros, so every output is dense.
#include <cstring>
#include <type_traits>

#include "adam_update.h"
#include "gs_internal.h"
#include "mlp.h"
#include "lobe.h"
#include "neural.h"
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
    const float* base_color;
    const uint16_t* features;
    const uint32_t* tiles_touched;
    const float* color_jac;
    const float* acc;
    float* dmeans;
    float* dlog_scales;
    float* dquats;
    float* dlogits;
    float* dsh;
    float* dlatent;
    float* mlp_part;
    float* dmean2d;
    float* dbase_color;
    float* dfeatures;
    const float* lobes;
    float* dlobes;
    int sh_y0_folded;
};

// The Adam step of gs_render_bwd_adam, applied where each gradient is computed.
// Tensors in the order means, log_scales, quats, opacity_logits, then the
// appearance's per-Gaussian parameters (SH3: sh).
constexpr int kFusedTensors = 5;
struct AdamFused {
    float* p[kFusedTensors];
    float* m[kFusedTensors];
    float* v[kFusedTensors];
    uint16_t* h[kFusedTensors];
    AdamStep c;
};

// A batch of K elements (t[k], row[k], Gaussian i): p[k] is the parameter as
// read before the update (the caller reads those the backward did not). All
// the batch's moments are read before any element is written, so that their
// reads are in flight together (the compiler cannot move a read past a write
// it cannot tell apart).
template <int K>
__device__ __forceinline__ void adam_apply(const AdamFused& f, const int (&t)[K], const int (&row)[K], int64_t n,
                                           int64_t i, float (&p)[K], const float (&g)[K])
{
    float m[K], v[K];
#pragma unroll
    for (int k = 0; k < K; ++k) {
        const int64_t e = (int64_t)row[k] * n + i;
        m[k] = __builtin_nontemporal_load(f.m[t[k]] + e);
        v[k] = __builtin_nontemporal_load(f.v[t[k]] + e);
    }
#pragma unroll
    for (int k = 0; k < K; ++k) {
        const int tk = t[k];
        const int64_t e = (int64_t)row[k] * n + i;
        adam_update(p[k], m[k], v[k], g[k], f.c.b1, f.c.omb1, f.c.b2[tk], f.c.omb2[tk], f.c.inv_sqrt_bc2[tk],
                    f.c.eps, f.c.step_size[f.c.row0[tk] + row[k]]);
        __builtin_nontemporal_store(m[k], f.m[tk] + e);
        __builtin_nontemporal_store(v[k], f.v[tk] + e);
        __builtin_nontemporal_store(p[k], f.p[tk] + e);
        if (f.h[tk]) __builtin_nontemporal_store(__builtin_bit_cast(uint16_t, (_Float16)p[k]), f.h[tk] + e);
    }
}

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
    // gradient plane is written once per wave with whole lines. Parameters,
    // accumulators and gradients are touched once: non-temporal accesses.
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
        for (int j = 0; j < 3; ++j) mu[j] = __builtin_nontemporal_load(&a.means[j * n + i]);
        for (int j = 0; j < 3; ++j) ls[j] = __builtin_nontemporal_load(&a.log_scales[j * n + i]);
        for (int j = 0; j < 4; ++j) q[j] = __builtin_nontemporal_load(&a.quats[j * n + i]);
        const float* ap = a.acc + (size_t)i * kAccStride;
        for (int k = 0; k < kAccStride; ++k) g9[k] = __builtin_nontemporal_load(ap + k);
        geometry_bwd(a.cam, mu, ls, q, a.logits[i], g9, gg);

        // appearance: eq. sh_color_eval with its ReLU
        const float vx = mu[0] - a.cam.campos[0], vy = mu[1] - a.cam.campos[1], vz = mu[2] - a.cam.campos[2];
        const float len = sqrtf(vx * vx + vy * vy + vz * vz);
        const float il = 1.f / len;
        const float d0 = vx * il, d1 = vy * il, d2 = vz * il;
        sh_basis16(d0, d1, d2, Y);
        if (a.sh_y0_folded) Y[0] = 1.f;   // constant either way: no direction gradient
        float dd[3] = {0.f, 0.f, 0.f};
        if (a.color_jac) {
            // the forward's direction Jacobian of the colour sums and their clamp
            float J[9];
            for (int r = 0; r < 9; ++r) J[r] = __builtin_nontemporal_load(a.color_jac + r * n + i);
            const uint32_t up = __float_as_uint(__builtin_nontemporal_load(a.color_jac + 9 * n + i));
            for (int c = 0; c < 3; ++c) gc[c] = (up >> c) & 1u ? g9[6 + c] : 0.f;
            for (int j = 0; j < 3; ++j) dd[j] = gc[0] * J[j] + gc[1] * J[3 + j] + gc[2] * J[6 + j];
        } else {
            float coef[GS_SH_COEFFS];
            float pre[3] = {0.5f, 0.5f, 0.5f};
            for (int k = 0; k < 16; ++k)
                for (int c = 0; c < 3; ++c) {
                    coef[3 * k + c] = k < nb ? __builtin_nontemporal_load(a.sh + (3 * k + c) * n + i) : 0.f;
                    pre[c] += Y[k] * coef[3 * k + c];
                }
            for (int c = 0; c < 3; ++c) gc[c] = pre[c] > 0.f ? g9[6 + c] : 0.f;
            float dY[16];
            for (int k = 0; k < 16; ++k)
                dY[k] = coef[3 * k] * gc[0] + coef[3 * k + 1] * gc[1] + coef[3 * k + 2] * gc[2];
            sh_basis16_vjp(d0, d1, d2, dY, dd);
        }
        // d = v / |v|: dv = (dd - d (d . dd)) / |v|
        const float dot = d0 * dd[0] + d1 * dd[1] + d2 * dd[2];
        gg.dmu[0] += (dd[0] - d0 * dot) * il;
        gg.dmu[1] += (dd[1] - d1 * dot) * il;
        gg.dmu[2] += (dd[2] - d2 * dot) * il;
    }
    for (int k = 0; k < 16; ++k) {
        const bool on = k < nb;
        for (int c = 0; c < 3; ++c)
            __builtin_nontemporal_store(on ? Y[k] * gc[c] : 0.f, a.dsh + (3 * k + c) * n + i);
    }
    for (int j = 0; j < 3; ++j) {
        __builtin_nontemporal_store(gg.dmu[j], &a.dmeans[j * n + i]);
        __builtin_nontemporal_store(gg.dls[j], &a.dlog_scales[j * n + i]);
    }
    for (int j = 0; j < 4; ++j) __builtin_nontemporal_store(gg.dq[j], &a.dquats[j * n + i]);
    __builtin_nontemporal_store(gg.dlogit, &a.dlogits[i]);
    if (a.dmean2d) {
        __builtin_nontemporal_store(g9[0], &a.dmean2d[i]);
        __builtin_nontemporal_store(g9[1], &a.dmean2d[n + i]);
    }
}

// gs_render_bwd_adam for SH3: the backward above, with the Adam step applied
// to every parameter element where its gradient is computed (culled Gaussians'
// and inactive bands' elements with a zero gradient, as the standalone step
// steps them); a gradient array of `a` that is not NULL still receives the
// gradient. The SH rows are stepped as soon as the colour gradient is known,
// so that the coefficients are not kept past them.
__global__ __launch_bounds__(kBlock) void k_preprocess_bwd_sh3_adam(BwdArgs a, AdamFused f)
{
    const int i = blockIdx.x * kBlock + threadIdx.x;
    if (i >= a.n) return;
    const int64_t n = a.n;
    const bool vis = a.tiles_touched[i] != 0;
    GeoGrad gg;
    for (int j = 0; j < 3; ++j) { gg.dmu[j] = 0.f; gg.dls[j] = 0.f; }
    for (int j = 0; j < 4; ++j) gg.dq[j] = 0.f;
    gg.dlogit = 0.f;
    float g9[kAccStride];
    for (int k = 0; k < kAccStride; ++k) g9[k] = 0.f;
    float Y[16], gc[3] = {0.f, 0.f, 0.f}, dY[16];
    for (int k = 0; k < 16; ++k) Y[k] = dY[k] = 0.f;
    const int nb = (a.sh_degree + 1) * (a.sh_degree + 1);
    float mu[3], ls[3], q[4];
    for (int j = 0; j < 3; ++j) mu[j] = __builtin_nontemporal_load(&a.means[j * n + i]);
    for (int j = 0; j < 3; ++j) ls[j] = __builtin_nontemporal_load(&a.log_scales[j * n + i]);
    for (int j = 0; j < 4; ++j) q[j] = __builtin_nontemporal_load(&a.quats[j * n + i]);
    const float logit = __builtin_nontemporal_load(&a.logits[i]);
    float coef[GS_SH_COEFFS];
    for (int k = 0; k < GS_SH_COEFFS; ++k) coef[k] = 0.f;
    float d0 = 0.f, d1 = 0.f, d2 = 0.f, il = 0.f;
    if (vis) {
        const float* ap = a.acc + (size_t)i * kAccStride;
        for (int k = 0; k < kAccStride; ++k) g9[k] = __builtin_nontemporal_load(ap + k);
        geometry_bwd(a.cam, mu, ls, q, logit, g9, gg);
        const float vx = mu[0] - a.cam.campos[0], vy = mu[1] - a.cam.campos[1], vz = mu[2] - a.cam.campos[2];
        const float len = sqrtf(vx * vx + vy * vy + vz * vz);
        il = 1.f / len;
        d0 = vx * il;
        d1 = vy * il;
        d2 = vz * il;
        sh_basis16(d0, d1, d2, Y);
        if (a.sh_y0_folded) Y[0] = 1.f;
        float pre[3] = {0.5f, 0.5f, 0.5f};
        for (int k = 0; k < 16; ++k)
            for (int c = 0; c < 3; ++c) {
                coef[3 * k + c] = k < nb ? __builtin_nontemporal_load(a.sh + (3 * k + c) * n + i) : 0.f;
                pre[c] += Y[k] * coef[3 * k + c];
            }
        for (int c = 0; c < 3; ++c) gc[c] = pre[c] > 0.f ? g9[6 + c] : 0.f;
        for (int k = 0; k < 16; ++k) dY[k] = coef[3 * k] * gc[0] + coef[3 * k + 1] * gc[1] + coef[3 * k + 2] * gc[2];
    }
    // the SH rows, two bands (6 rows) per batch
    constexpr int kShBatch = 6;
#pragma unroll
    for (int r0 = 0; r0 < GS_SH_COEFFS; r0 += kShBatch) {
        int tb[kShBatch], rb[kShBatch];
        float pb[kShBatch], gb[kShBatch];
#pragma unroll
        for (int j = 0; j < kShBatch; ++j) {
            const int r = r0 + j, k = r / 3, c = r % 3;
            tb[j] = 4;
            rb[j] = r;
            gb[j] = k < nb ? Y[k] * gc[c] : 0.f;
            // coefficients the backward did not read are read here
            pb[j] = vis && k < nb ? coef[r] : __builtin_nontemporal_load(a.sh + r * n + i);
            if (a.dsh) __builtin_nontemporal_store(gb[j], a.dsh + r * n + i);
        }
        adam_apply(f, tb, rb, n, i, pb, gb);
    }
    if (vis) {
        float dd[3] = {0.f, 0.f, 0.f};
        sh_basis16_vjp(d0, d1, d2, dY, dd);
        // d = v / |v|: dv = (dd - d (d . dd)) / |v|
        const float dot = d0 * dd[0] + d1 * dd[1] + d2 * dd[2];
        gg.dmu[0] += (dd[0] - d0 * dot) * il;
        gg.dmu[1] += (dd[1] - d1 * dot) * il;
        gg.dmu[2] += (dd[2] - d2 * dot) * il;
    }
    for (int j = 0; j < 3; ++j) {
        if (a.dmeans) __builtin_nontemporal_store(gg.dmu[j], &a.dmeans[j * n + i]);
        if (a.dlog_scales) __builtin_nontemporal_store(gg.dls[j], &a.dlog_scales[j * n + i]);
    }
    for (int j = 0; j < 4; ++j)
        if (a.dquats) __builtin_nontemporal_store(gg.dq[j], &a.dquats[j * n + i]);
    if (a.dlogits) __builtin_nontemporal_store(gg.dlogit, &a.dlogits[i]);
    // the geometry rows in one batch: means, log-scales, quaternion, opacity logit
    const int tg[11] = {0, 0, 0, 1, 1, 1, 2, 2, 2, 2, 3};
    const int rg[11] = {0, 1, 2, 0, 1, 2, 0, 1, 2, 3, 0};
    float pg[11] = {mu[0], mu[1], mu[2], ls[0], ls[1], ls[2], q[0], q[1], q[2], q[3], logit};
    const float gg11[11] = {gg.dmu[0], gg.dmu[1], gg.dmu[2], gg.dls[0], gg.dls[1], gg.dls[2],
                            gg.dq[0], gg.dq[1], gg.dq[2], gg.dq[3], gg.dlogit};
    adam_apply(f, tg, rg, n, i, pg, gg11);
    if (a.dmean2d) {
        __builtin_nontemporal_store(g9[0], &a.dmean2d[i]);
        __builtin_nontemporal_store(g9[1], &a.dmean2d[n + i]);
    }
}

// NASG / NASGabor backward (eq. nasg, lobe.h): geometry as for SH3; the colour
// gradient g (zero where the ReLU clamps) gives dc0 = g, d amp = g G (1 - tanh^2),
// and (g . tanh(amp)) times the kernel's gradient for the raw lobe parameters
// and the view direction (chained into the mean). Culled Gaussians and an
// inactive lobe get zeros.
template <bool kGabor>
__global__ __launch_bounds__(kBlock) void k_preprocess_bwd_lobe(BwdArgs a)
{
    constexpr int kRows = kGabor ? 9 : 8;
    const int i = blockIdx.x * kBlock + threadIdx.x;
    if (i >= a.n) return;
    const int64_t n = a.n;
    const bool vis = a.tiles_touched[i] != 0;
    GeoGrad gg;
    for (int j = 0; j < 3; ++j) { gg.dmu[j] = 0.f; gg.dls[j] = 0.f; }
    for (int j = 0; j < 4; ++j) gg.dq[j] = 0.f;
    gg.dlogit = 0.f;
    float g9[kAccStride];
    for (int k = 0; k < kAccStride; ++k) g9[k] = 0.f;
    float gc[3] = {0.f, 0.f, 0.f}, dl[kRows];
    for (int k = 0; k < kRows; ++k) dl[k] = 0.f;
    if (vis) {
        float mu[3], ls[3], q[4], c0[3];
        for (int j = 0; j < 3; ++j) mu[j] = __builtin_nontemporal_load(&a.means[j * n + i]);
        for (int j = 0; j < 3; ++j) ls[j] = __builtin_nontemporal_load(&a.log_scales[j * n + i]);
        for (int j = 0; j < 4; ++j) q[j] = __builtin_nontemporal_load(&a.quats[j * n + i]);
        for (int c = 0; c < 3; ++c) c0[c] = a.base_color[c * n + i];
        const float* ap = a.acc + (size_t)i * kAccStride;
        for (int k = 0; k < kAccStride; ++k) g9[k] = __builtin_nontemporal_load(ap + k);
        geometry_bwd(a.cam, mu, ls, q, a.logits[i], g9, gg);
        if (a.sh_degree >= 1) {
            float r[6], T[3];
            for (int k = 0; k < 5; ++k) r[k] = a.lobes[k * n + i];
            for (int c = 0; c < 3; ++c) T[c] = tanhf(a.lobes[(5 + c) * n + i]);
            r[5] = kGabor ? a.lobes[8 * n + i] : 0.f;
            const float vx = mu[0] - a.cam.campos[0], vy = mu[1] - a.cam.campos[1], vz = mu[2] - a.cam.campos[2];
            const float len = sqrtf(vx * vx + vy * vy + vz * vz);
            const float il = 1.f / len;
            const float d[3] = {vx * il, vy * il, vz * il};
            LobeEval f;
            lobe_setup<kGabor>(r, f);
            float draw[6], dd[3];
            const float G = lobe_grad<kGabor>(f, d, draw, dd);
            float sgt = 0.f;
            for (int c = 0; c < 3; ++c) {
                gc[c] = c0[c] + G * T[c] + 0.5f > 0.f ? g9[6 + c] : 0.f;
                sgt += gc[c] * T[c];
                dl[5 + c] = gc[c] * G * (1.f - T[c] * T[c]);
            }
            for (int k = 0; k < 5; ++k) dl[k] = sgt * draw[k];
            if constexpr (kGabor) dl[8] = sgt * draw[5];
            // d = v / |v|: dv = (dd - d (d . dd)) / |v|
            const float dot = d[0] * dd[0] + d[1] * dd[1] + d[2] * dd[2];
            for (int j = 0; j < 3; ++j) gg.dmu[j] += sgt * (dd[j] - d[j] * dot) * il;
        } else {
            for (int c = 0; c < 3; ++c) gc[c] = c0[c] + 0.5f > 0.f ? g9[6 + c] : 0.f;
        }
    }
    for (int c = 0; c < 3; ++c) __builtin_nontemporal_store(gc[c], &a.dbase_color[c * n + i]);
    for (int k = 0; k < kRows; ++k) __builtin_nontemporal_store(dl[k], &a.dlobes[k * n + i]);
    for (int j = 0; j < 3; ++j) {
        __builtin_nontemporal_store(gg.dmu[j], &a.dmeans[j * n + i]);
        __builtin_nontemporal_store(gg.dls[j], &a.dlog_scales[j * n + i]);
    }
    for (int j = 0; j < 4; ++j) __builtin_nontemporal_store(gg.dq[j], &a.dquats[j * n + i]);
    __builtin_nontemporal_store(gg.dlogit, &a.dlogits[i]);
    if (a.dmean2d) {
        __builtin_nontemporal_store(g9[0], &a.dmean2d[i]);
        __builtin_nontemporal_store(g9[1], &a.dmean2d[n + i]);
    }
}

// The geometry backward's per-Gaussian inputs that the decoder kernels read
// before their matrix-core phase (the mean, for the view direction, and the
// screen-space accumulator entries 0..5, read with the colour entries), kept
// per wave in LDS across that phase so that each is read from memory once.
// Each lane reads back only what it wrote: no barrier is needed.
struct GeoStage {
    float v[3 + 6][kWave];
};

__device__ __forceinline__ void geo_stage_put(GeoStage& gs, const float mu[3], const float* ap)
{
    const int l = __lane_id();
#pragma unroll
    for (int j = 0; j < 3; ++j) gs.v[j][l] = mu[j];
#pragma unroll
    for (int k = 0; k < 6; ++k) gs.v[3 + k][l] = ap[k];
}

__device__ __forceinline__ void geo_stage_get(const GeoStage& gs, float mu[3], float g9[kAccStride])
{
    const int l = __lane_id();
#pragma unroll
    for (int j = 0; j < 3; ++j) mu[j] = gs.v[j][l];
#pragma unroll
    for (int k = 0; k < 6; ++k) g9[k] = gs.v[3 + k][l];
#pragma unroll
    for (int k = 6; k < kAccStride; ++k) g9[k] = 0.f;   // the colour entries are the decoder's
}

// Latent + MLP backward: geometry as for SH3, then per tile of 16 Gaussians
// the decoder is recomputed and differentiated on the matrix cores (mlp.h):
// the latent gradient, the gradient into the view direction (chained into the
// mean), and this workgroup's sum of the weight gradients, written as one
// partial per workgroup (summed in a fixed order by k_mlp_reduce).
__global__ __launch_bounds__(kBlock, 3) void k_preprocess_bwd_latent(BwdArgs a)
{
    __shared__ MlpFrags W;
    __shared__ MlpWaveStage ST[kBlock / kWave];
    __shared__ GeoStage GS[kBlock / kWave];
    __shared__ float chain_slot;
    mlp_load_frags(a.mlp_w, W, true);
    const float chain = decoder_chain_bound(a.mlp_w, GS_MLP_IN, GS_MLP_HIDDEN, 1, &chain_slot);
    const int wave = threadIdx.x >> 6, lane = __lane_id();
    MlpWaveStage& st = ST[wave];
    MlpGradAcc acc;
    mlp_grad_zero(acc);
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
        // decoder part first: it needs the view direction and the colour gradient
        float d[3] = {0.f, 0.f, 0.f}, dc[3] = {0.f, 0.f, 0.f};
        float len = 1.f;
        if (valid) {
            float mu[3];
            for (int j = 0; j < 3; ++j) mu[j] = a.means[j * n + i];
            const float vx = mu[0] - a.cam.campos[0], vy = mu[1] - a.cam.campos[1], vz = mu[2] - a.cam.campos[2];
            len = sqrtf(vx * vx + vy * vy + vz * vz);
            d[0] = vx / len;
            d[1] = vy / len;
            d[2] = vz / len;
            const float* ap = a.acc + (size_t)i * kAccStride;
            float g9[kAccStride];
            for (int k = 0; k < kAccStride; ++k) g9[k] = ap[k];
            for (int ch = 0; ch < 3; ++ch) dc[ch] = g9[6 + ch];
            geo_stage_put(GS[wave], mu, g9);
        }
        mlp_stage_row(st, valid, a.latent, n, i, d, dc);
        // the chunk's gradient scale (a power of two, see mlp_chunk_exponent)
        const float m = wave_max(fmaxf(fmaxf(fabsf(dc[0]), fabsf(dc[1])), fabsf(dc[2])));
        mlp_grad_rescale(acc, mlp_chunk_exponent(m * chain, acc.se));
        const float scale = ldexpf(1.f, acc.se), inv = ldexpf(1.f, -acc.se);
        wave_lds_sync();
        const uint64_t vis = __ballot(valid);
        const int64_t base = chunk * kBlock + (threadIdx.x & ~(kWave - 1));
        for (int t = 0; t < kWave / 16; ++t) {
            if (((vis >> (16 * t)) & 0xFFFFull) == 0) continue;
            mlp_tile_bwd(W, st, t, vis, a.dlatent, n, base, scale, inv, acc);
        }
        wave_lds_sync();
        if (valid) {
            float mu[3], ls[3], q[4], g9[kAccStride];
            for (int j = 0; j < 3; ++j) ls[j] = a.log_scales[j * n + i];
            for (int j = 0; j < 4; ++j) q[j] = a.quats[j * n + i];
            geo_stage_get(GS[wave], mu, g9);
            GeoGrad gg;
            geometry_bwd(a.cam, mu, ls, q, a.logits[i], g9, gg);
            // the binary16 rounding of d passes the gradient; d = v / |v|
            const float dd0 = st.dd[lane][0], dd1 = st.dd[lane][1], dd2 = st.dd[lane][2];
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
        wave_lds_sync();   // st.dd is read before the next chunk restages
    }
    // workgroup sum of the four waves' weight gradients, in wave order, in the
    // LDS of the (no longer needed) weight fragments
    static_assert(sizeof(MlpFrags) >= GS_MLP_WEIGHTS * sizeof(float), "reduction buffer");
    __syncthreads();
    float* red = reinterpret_cast<float*>(&W);
    for (int k = threadIdx.x; k < GS_MLP_WEIGHTS; k += kBlock) red[k] = 0.f;
    __syncthreads();
    const int g = lane >> 4, c = lane & 15;
    mlp_grad_rescale(acc, 0);   // back to plain units
    for (int w = 0; w < kBlock / kWave; ++w) {
        if (wave == w) {
            for (int mb = 0; mb < 2; ++mb)
                for (int fb = 0; fb < 2; ++fb)
                    for (int e = 0; e < 4; ++e) {
                        const int row = 16 * mb + 4 * g + e, col = 16 * fb + c;
                        if (col < GS_MLP_IN) red[row * GS_MLP_IN + col] += acc.w1[mb][fb][e];
                        red[32 * GS_MLP_IN + row * 32 + col] += acc.w2[mb][fb][e];
                    }
            for (int nb = 0; nb < 2; ++nb)
                for (int e = 0; e < 4; ++e) {
                    const int o = 4 * g + e, col = 16 * nb + c;
                    if (o < GS_MLP_OUT) red[32 * GS_MLP_IN + 32 * 32 + o * 32 + col] += acc.w3[nb][e];
                }
        }
        __syncthreads();
    }
    for (int k = threadIdx.x; k < GS_MLP_WEIGHTS; k += kBlock)
        a.mlp_part[(size_t)blockIdx.x * GS_MLP_WEIGHTS + k] = red[k];
}

// Neural appearance backward (neural.h): as the latent one -- per wave chunk of
// 64 Gaussians the decoder inputs, colour gradients, base colours, features and
// directions are staged, each tile of 16 is recomputed and differentiated on
// the matrix cores (base-colour and feature gradients, the direction gradient
// of the active bands, the weight-gradient sums), then the geometry backward.
// While the active degree is 0 only the base colour takes a gradient. L hidden
// layers; kRaw: 16 raw features as the feature inputs.
template <int L, bool kRaw, int kW = 16>
__global__ __launch_bounds__(kBlock, kW == 32 ? 2 : 3) void k_preprocess_bwd_neural(BwdArgs a)
{
    static_assert(kW == 16 || (kW == 32 && L == 2 && !kRaw), "the 32-neuron configuration is 32-32-32-3");
    constexpr int kF = kRaw ? 16 : GS_NEURAL_FEATURES;
    constexpr int kNW = kW == 32 ? kNeural32Weights : neural_weight_count(L);
    using Frags = std::conditional_t<kW == 32, MlpFrags, NeuralFrags<L>>;
    using Acc = std::conditional_t<kW == 32, MlpGradAcc, NeuralGradAcc<L>>;
    __shared__ Frags W;
    __shared__ NeuralBwdStage ST[kBlock / kWave];
    __shared__ GeoStage GS[kBlock / kWave];
    __shared__ float chain_slot;
    const bool resid = a.sh_degree >= 1;
    if (resid) neural_load_frags(a.mlp_w, W, true);
    const float chain = resid ? decoder_chain_bound(a.mlp_w, 32, kW, L - 1, &chain_slot) : 1.f;
    const int wave = threadIdx.x >> 6, lane = __lane_id();
    NeuralBwdStage& st = ST[wave];
    Acc acc;
    neural_grad_zero(acc);
    const int64_t n = a.n;
    const int64_t nchunks = div_up(n, kBlock);
    for (int64_t chunk = blockIdx.x; chunk < nchunks; chunk += gridDim.x) {
        const int64_t i = chunk * kBlock + threadIdx.x;
        const bool inb = i < n;
        const bool valid = inb && a.tiles_touched[i] != 0;
        if (inb && !valid) {
            write_zero_grads(a, (int)i);
            for (int ch = 0; ch < 3; ++ch) a.dbase_color[ch * n + i] = 0.f;
            for (int j = 0; j < kF; ++j) a.dfeatures[j * n + i] = 0.f;
        }
        float d[3] = {0.f, 0.f, 0.f}, dc[3] = {0.f, 0.f, 0.f}, c0[3] = {0.f, 0.f, 0.f};
        float len = 1.f;
        if (valid) {
            float mu[3];
            for (int j = 0; j < 3; ++j) mu[j] = a.means[j * n + i];
            const float vx = mu[0] - a.cam.campos[0], vy = mu[1] - a.cam.campos[1], vz = mu[2] - a.cam.campos[2];
            len = sqrtf(vx * vx + vy * vy + vz * vz);
            d[0] = vx / len;
            d[1] = vy / len;
            d[2] = vz / len;
            const float* ap = a.acc + (size_t)i * kAccStride;
            float g9[kAccStride];
            for (int k = 0; k < kAccStride; ++k) g9[k] = ap[k];
            for (int ch = 0; ch < 3; ++ch) dc[ch] = g9[6 + ch];
            for (int ch = 0; ch < 3; ++ch) c0[ch] = a.base_color[ch * n + i];
            geo_stage_put(GS[wave], mu, g9);
        }
        float dd[3] = {0.f, 0.f, 0.f};
        if (resid) {
            float f[kF], sf[GS_NEURAL_FEATURES], cf[GS_NEURAL_FEATURES];
            for (int j = 0; j < kF; ++j) f[j] = valid ? (float)half_of_bits(a.features[j * n + i]) : 0.f;
            half4_t fq[4];
            if (kRaw) {
                neural_raw_inputs(f, fq);
            } else {
                neural_encode_features(f, sf, cf);
                neural_feature_inputs(sf, cf, fq);
            }
            neural_stage_inputs(st.x, valid, d, a.sh_degree, fq);
            wave_lds_sync();
            const uint64_t vis = __ballot(valid);
            // first pass: each lane's output pre-activations, then its residual
            // tanh(o), base-colour gradient and delta3 = dL/dc [c > 0] (1 - res^2)
            float o[3] = {0.f, 0.f, 0.f};
            for (int t = 0; t < kWave / 16; ++t) {
                if (((vis >> (16 * t)) & 0xFFFFull) == 0) continue;
                neural_tile_gather(neural_tile_out(W, neural_stage_frag(st.x, t)), t, o);
            }
            float m = 0.f;
            for (int ch = 0; ch < 3; ++ch) {
                const float r = tanhf(o[ch]);
                const float dcm = c0[ch] + r + 0.5f > 0.f ? dc[ch] : 0.f;   // dc = 0 when !valid
                if (valid) a.dbase_color[ch * n + i] = dcm;
                const float d3 = dcm * (1.f - r * r);
                st.d3[lane][ch] = d3;
                m = fmaxf(m, fabsf(d3));
            }
            st.d3[lane][3] = 0.f;
            // the chunk's gradient scale (a power of two, see neural_chunk_exponent)
            neural_grad_rescale(acc, neural_chunk_exponent(wave_max(m) * chain, acc.se));
            const float scale = ldexpf(1.f, acc.se), inv = ldexpf(1.f, -acc.se);
            wave_lds_sync();
            for (int t = 0; t < kWave / 16; ++t) {
                if (((vis >> (16 * t)) & 0xFFFFull) == 0) continue;
                neural_tile_bwd(W, st, t, scale, inv, acc);
            }
            wave_lds_sync();
            if (valid) {
                // direction: the active bands' input gradients through the SH basis
                const int nb = (a.sh_degree + 1) * (a.sh_degree + 1);
                const float* row = neural_dir_grad_row(st, lane);
                float dY[16];
                for (int k = 0; k < 16; ++k) dY[k] = k < nb ? row[k] : 0.f;
                sh_basis16_vjp(d[0], d[1], d[2], dY, dd);
                // features: raw ones take their inputs' gradients; encoded ones
                // d(sin f)/df = cos f, d(cos f)/df = -sin f
                if (kRaw) {
                    for (int j = 0; j < 16; ++j) a.dfeatures[j * n + i] = st.dxf[lane][j];
                } else {
                    for (int j = 0; j < GS_NEURAL_FEATURES; ++j)
                        a.dfeatures[j * n + i] = st.dxf[lane][2 * j] * cf[j] - st.dxf[lane][2 * j + 1] * sf[j];
                }
            }
        } else if (valid) {
            // no residual: c = max(0, c0 + 0.5)
            for (int ch = 0; ch < 3; ++ch) a.dbase_color[ch * n + i] = c0[ch] + 0.5f > 0.f ? dc[ch] : 0.f;
            for (int j = 0; j < kF; ++j) a.dfeatures[j * n + i] = 0.f;
        }
        if (valid) {
            float mu[3], ls[3], q[4], g9[kAccStride];
            for (int j = 0; j < 3; ++j) ls[j] = a.log_scales[j * n + i];
            for (int j = 0; j < 4; ++j) q[j] = a.quats[j * n + i];
            geo_stage_get(GS[wave], mu, g9);
            GeoGrad gg;
            geometry_bwd(a.cam, mu, ls, q, a.logits[i], g9, gg);
            if (resid) {
                // the binary16 rounding of the SH inputs passes the gradient; d = v / |v|
                const float dd0 = dd[0], dd1 = dd[1], dd2 = dd[2];
                const float dot = d[0] * dd0 + d[1] * dd1 + d[2] * dd2;
                const float il = 1.f / len;
                gg.dmu[0] += (dd0 - d[0] * dot) * il;
                gg.dmu[1] += (dd1 - d[1] * dot) * il;
                gg.dmu[2] += (dd2 - d[2] * dot) * il;
            }
            for (int j = 0; j < 3; ++j) { a.dmeans[j * n + i] = gg.dmu[j]; a.dlog_scales[j * n + i] = gg.dls[j]; }
            for (int j = 0; j < 4; ++j) a.dquats[j * n + i] = gg.dq[j];
            a.dlogits[i] = gg.dlogit;
            if (a.dmean2d) { a.dmean2d[i] = g9[0]; a.dmean2d[n + i] = g9[1]; }
        }
        if (resid) wave_lds_sync();   // the stage is read before the next chunk restages
    }
    // workgroup sum of the four waves' weight gradients, in wave order, in the
    // LDS of the (no longer needed) stage
    static_assert(sizeof(ST) >= kNW * sizeof(float), "reduction buffer");
    __syncthreads();
    float* red = reinterpret_cast<float*>(&ST[0]);
    for (int k = threadIdx.x; k < kNW; k += kBlock) red[k] = 0.f;
    __syncthreads();
    neural_grad_rescale(acc, 0);   // back to plain units
    for (int w = 0; w < kBlock / kWave; ++w) {
        if (wave == w && resid) neural_grad_add(acc, red);
        __syncthreads();
    }
    for (int k = threadIdx.x; k < kNW; k += kBlock) a.mlp_part[(size_t)blockIdx.x * kNW + k] = red[k];
}

// dW = sum of the per-workgroup partials, in a fixed order. One workgroup per
// 64 weights: thread (row, column) sums every 16th partial starting at its row,
// then the 16 row sums are added in row order.
constexpr int kReduceRows = 16, kReduceCols = 64;
__global__ __launch_bounds__(kReduceRows * kReduceCols) void k_mlp_reduce(const float* __restrict__ part, int nparts,
                                                                          int nw, float* __restrict__ dw)
{
    __shared__ float rows[kReduceRows][kReduceCols];
    const int c = threadIdx.x % kReduceCols, r = threadIdx.x / kReduceCols;
    const int k = blockIdx.x * kReduceCols + c;
    float s = 0.f;
    if (k < nw) {
        int b = r;
        for (; b + 3 * kReduceRows < nparts; b += 4 * kReduceRows) {
            const float v0 = part[(size_t)b * nw + k];
            const float v1 = part[(size_t)(b + kReduceRows) * nw + k];
            const float v2 = part[(size_t)(b + 2 * kReduceRows) * nw + k];
            const float v3 = part[(size_t)(b + 3 * kReduceRows) * nw + k];
            s = (((s + v0) + v1) + v2) + v3;
        }
        for (; b < nparts; b += kReduceRows) s += part[(size_t)b * nw + k];
    }
    rows[r][c] = s;
    __syncthreads();
    if (r == 0 && k < nw) {
        float t = 0.f;
        for (int j = 0; j < kReduceRows; ++j) t += rows[j][c];
        dw[k] = t;
    }
}

inline int decoder_bwd_grid(int64_t n, const gs_appearance& app)
{
    const int parts = app.kind == GS_APP_NEURAL && app.neural_width == 32 ? kMlpPartials32 : kMlpPartials;
    return (int)std::min<int64_t>(div_up(n, kBlock), parts);
}

hipError_t launch_preprocess_bwd(const Cam& cam, const gs_gaussians& g, const gs_appearance& app,
                                 const gs_preprocessed& pre, const Workspace& ws, const gs_grads& gr, hipStream_t s,
                                 const gs_adam_tensor* adam, float beta1, float eps, int64_t step)
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
    a.base_color = app.base_color;
    a.features = app.features;
    a.tiles_touched = pre.tiles_touched;
    a.color_jac = app.kind == GS_APP_SH3 ? pre.color_jac : nullptr;
    a.acc = ws.acc;
    a.dmeans = gr.dmeans;
    a.dlog_scales = gr.dlog_scales;
    a.dquats = gr.dquats;
    a.dlogits = gr.dopacity_logits;
    a.dsh = gr.dsh;
    a.dlatent = gr.dlatent;
    a.mlp_part = ws.mlp_part;
    a.dmean2d = gr.dmean2d;
    a.dbase_color = gr.dbase_color;
    a.dfeatures = gr.dfeatures;
    a.lobes = app.lobes;
    a.dlobes = gr.dlobes;
    a.sh_y0_folded = app.sh_y0_folded;
    AdamFused f;
    memset(&f, 0, sizeof(f));
    if (adam) {
        if (app.kind != GS_APP_SH3) return hipErrorInvalidValue;   // the entry point rejects it first
        adam_step_constants(adam, kFusedTensors, beta1, eps, step, f.c);
        for (int t = 0; t < kFusedTensors; ++t) {
            f.p[t] = adam[t].param;
            f.m[t] = adam[t].exp_avg;
            f.v[t] = adam[t].exp_avg_sq;
            f.h[t] = adam[t].param_half;
        }
    }
    if (app.kind == GS_APP_SH3) {
        if (adam)
            hipLaunchKernelGGL(k_preprocess_bwd_sh3_adam, dim3(preprocess_blocks(g.n)), dim3(kBlock), 0, s, a, f);
        else
            hipLaunchKernelGGL(k_preprocess_bwd_sh3, dim3(preprocess_blocks(g.n)), dim3(kBlock), 0, s, a);
    }
    else if (app.kind == GS_APP_NASG)
        hipLaunchKernelGGL(k_preprocess_bwd_lobe<false>, dim3(preprocess_blocks(g.n)), dim3(kBlock), 0, s, a);
    else if (app.kind == GS_APP_NASGABOR)
        hipLaunchKernelGGL(k_preprocess_bwd_lobe<true>, dim3(preprocess_blocks(g.n)), dim3(kBlock), 0, s, a);
    else if (app.kind == GS_APP_NEURAL)
    {
        const dim3 grid(decoder_bwd_grid(g.n, app));
        const int layers = neural_layers(app);
        if (app.neural_width == 32) {
            hipLaunchKernelGGL((k_preprocess_bwd_neural<2, false, 32>), grid, dim3(kBlock), 0, s, a);
        } else if (app.neural_raw16) {
            if (layers == 1) hipLaunchKernelGGL((k_preprocess_bwd_neural<1, true>), grid, dim3(kBlock), 0, s, a);
            else if (layers == 3) hipLaunchKernelGGL((k_preprocess_bwd_neural<3, true>), grid, dim3(kBlock), 0, s, a);
            else hipLaunchKernelGGL((k_preprocess_bwd_neural<2, true>), grid, dim3(kBlock), 0, s, a);
        } else {
            if (layers == 1) hipLaunchKernelGGL((k_preprocess_bwd_neural<1, false>), grid, dim3(kBlock), 0, s, a);
            else if (layers == 3) hipLaunchKernelGGL((k_preprocess_bwd_neural<3, false>), grid, dim3(kBlock), 0, s, a);
            else hipLaunchKernelGGL((k_preprocess_bwd_neural<2, false>), grid, dim3(kBlock), 0, s, a);
        }
    }
    else
        hipLaunchKernelGGL(k_preprocess_bwd_latent, dim3(decoder_bwd_grid(g.n, app)), dim3(kBlock), 0, s, a);
    return hipGetLastError();
}

hipError_t launch_mlp_reduce(int64_t n, const gs_appearance& app, const Workspace& ws, float* dmlp_w, hipStream_t s)
{
    const int nw = app.kind == GS_APP_NEURAL ? neural_weights(app) : GS_MLP_WEIGHTS;
    hipLaunchKernelGGL(k_mlp_reduce, dim3((unsigned)div_up(nw, kReduceCols)), dim3(kReduceRows * kReduceCols), 0, s,
                       ws.mlp_part, decoder_bwd_grid(n, app), nw, dmlp_w);
    return hipGetLastError();
}

}  // namespace gsr
