// One NASG or NASGabor lobe (eq. nasg): the residual G(d) tanh(a) of the lobe
// appearances, with G the normalized anisotropic spherical Gaussian of Huang et
// al. and the activations the paper describes for the NASGabor work's kernel:
//   frame   cos(theta) = tanh(r0); the half angles of the azimuth phi and the
//           twist gamma have cosines tanh(r1), tanh(r2), so phi and gamma cover
//           (0, 2 pi); z = (sin th cos ph, sin th sin ph, cos th),
//           e1 = dz/dth, e2 = (-sin ph, cos ph, 0), x = cos ga e1 + sin ga e2,
//           y = -sin ga e1 + cos ga e2 (the ZYZ Euler rotation's columns);
//   shape   lambda = exp(clamp(r3, -8, 8)), a = exp(clamp(r4, -8, 8));
//   kernel  u = (d.z + 1)/2, rho = (d.x)^2 / ((d.x)^2 + (d.y)^2), psi = a rho,
//           G = exp(2 lambda (u^(1+psi) - 1)) u^psi / K,
//           K = 2 pi (1 - exp(-2 lambda)) / (lambda sqrt(1 + a)) (unit integral);
//   Gabor   G~ = G (1 + cos(omega d.x)) / 2, omega = 20 (tanh(r5) + 1).
// fp32 throughout; sin(theta) = sech(r0), sin(phi/2) = sech(r1), sin(gamma/2) = sech(r2).
// u = (d.z + 1)/2 is evaluated as |d + z|^2 / 4 (equal for unit vectors), which
// keeps its relative accuracy where d approaches -z instead of cancelling.
#pragma once

namespace gsr {

constexpr float kLobeClamp = 8.f;
constexpr float kTwoPi = 6.28318530717958648f;

struct LobeEval {
    float x[3], y[3], z[3], e1[3], e2[3];
    float ct, st, cg, sg, sh1, sh2;
    float lam, an, dlam, dan, om, dom;
};

__device__ __forceinline__ float sech_f(float r) { return 1.f / coshf(r); }

// Frame and shape of the raw parameters r[0..4] (r[5]: the Gabor frequency).
template <bool kGabor>
__device__ __forceinline__ void lobe_setup(const float r[6], LobeEval& f)
{
    const float ct = tanhf(r[0]), st = sech_f(r[0]);
    const float ch = tanhf(r[1]), sh = sech_f(r[1]);
    const float cgh = tanhf(r[2]), sgh = sech_f(r[2]);
    const float cp = ch * ch - sh * sh, sp = 2.f * sh * ch;
    const float cg = cgh * cgh - sgh * sgh, sg = 2.f * sgh * cgh;
    f.ct = ct; f.st = st; f.cg = cg; f.sg = sg; f.sh1 = sh; f.sh2 = sgh;
    f.z[0] = st * cp; f.z[1] = st * sp; f.z[2] = ct;
    f.e1[0] = ct * cp; f.e1[1] = ct * sp; f.e1[2] = -st;
    f.e2[0] = -sp; f.e2[1] = cp; f.e2[2] = 0.f;
#pragma unroll
    for (int j = 0; j < 3; ++j) {
        f.x[j] = cg * f.e1[j] + sg * f.e2[j];
        f.y[j] = -sg * f.e1[j] + cg * f.e2[j];
    }
    const bool lin = r[3] > -kLobeClamp && r[3] < kLobeClamp, ain = r[4] > -kLobeClamp && r[4] < kLobeClamp;
    f.lam = expf(fminf(fmaxf(r[3], -kLobeClamp), kLobeClamp));
    f.an = expf(fminf(fmaxf(r[4], -kLobeClamp), kLobeClamp));
    f.dlam = lin ? f.lam : 0.f;
    f.dan = ain ? f.an : 0.f;
    if (kGabor) {
        const float t = tanhf(r[5]);
        f.om = 20.f * (t + 1.f);
        f.dom = 20.f * (1.f - t * t);
    } else {
        f.om = f.dom = 0.f;
    }
}

__device__ __forceinline__ float dot3f(const float a[3], const float b[3]) { return a[0] * b[0] + a[1] * b[1] + a[2] * b[2]; }

// (d.z + 1)/2 as |d + z|^2 / 4
__device__ __forceinline__ float lobe_u(const float d[3], const float z[3])
{
    const float s0 = d[0] + z[0], s1 = d[1] + z[1], s2 = d[2] + z[2];
    return fmaxf(0.25f * (s0 * s0 + s1 * s1 + s2 * s2), 1e-30f);
}

// Kernel value at unit direction d.
template <bool kGabor>
__device__ __forceinline__ float lobe_value(const LobeEval& f, const float d[3])
{
    const float px = dot3f(d, f.x), py = dot3f(d, f.y);
    const float u = lobe_u(d, f.z), q = px * px + py * py;
    const float psi = q > 0.f ? f.an * (px * px / q) : 0.f;
    const float L = logf(u);
    const float w = expf((1.f + psi) * L);
    const float invK = f.lam * sqrtf(1.f + f.an) / (kTwoPi * -expm1f(-2.f * f.lam));
    float G = expf(2.f * f.lam * (w - 1.f) + psi * L) * invK;
    if (kGabor) G *= 0.5f * (1.f + cosf(f.om * px));
    return G;
}

// Kernel value, its gradient w.r.t. the raw parameters (draw[0..4], draw[5] for
// Gabor) and w.r.t. the direction (dd), by the chain rule through the frame:
// d th/dr0 = -sin th, d ph/dr1 = -2 sin(ph/2), d ga/dr2 = -2 sin(ga/2);
// dz/dth = e1, dz/dph = sin th e2, dx/dth = -cos ga z, dx/dph = cos ga cos th e2
// + sin ga e3, dx/dga = y, dy/dth = sin ga z, dy/dph = -sin ga cos th e2 +
// cos ga e3, dy/dga = -x, with e3 = de2/dph = (-cos ph, -sin ph, 0).
template <bool kGabor>
__device__ __forceinline__ float lobe_grad(const LobeEval& f, const float d[3], float draw[6], float dd[3])
{
    const float px = dot3f(d, f.x), py = dot3f(d, f.y), pz = dot3f(d, f.z);
    const float u = lobe_u(d, f.z), q = px * px + py * py;
    const float rho = q > 0.f ? px * px / q : 0.f;
    const float psi = f.an * rho;
    const float L = logf(u);
    const float upsi = expf(psi * L);
    const float w = upsi * u;
    const float em = -expm1f(-2.f * f.lam);
    const float invK = f.lam * sqrtf(1.f + f.an) / (kTwoPi * em);
    const float G0 = expf(2.f * f.lam * (w - 1.f)) * upsi * invK;
    float C = 1.f, dC_dpx = 0.f, dC_dom = 0.f;
    if (kGabor) {
        float sn, cs;
        sincosf(f.om * px, &sn, &cs);
        C = 0.5f * (1.f + cs);
        dC_dpx = -0.5f * f.om * sn;
        dC_dom = -0.5f * px * sn;
    }
    const float dG0_du = G0 * (2.f * f.lam * (1.f + psi) * upsi + psi / u);
    const float dG0_dpsi = G0 * (2.f * f.lam * w * L + L);
    const float dlnK_dlam = 2.f * (1.f - em) / em - 1.f / f.lam;
    const float dG0_dlam = G0 * (2.f * (w - 1.f) - dlnK_dlam);
    const float dG0_da = G0 / (2.f * (1.f + f.an)) + dG0_dpsi * rho;
    const float iq2 = q > 0.f ? 1.f / (q * q) : 0.f;
    const float drho_dpx = 2.f * px * py * py * iq2, drho_dpy = -2.f * py * px * px * iq2;
    const float Dz = C * dG0_du * 0.5f;
    const float Dx = C * dG0_dpsi * f.an * drho_dpx + G0 * dC_dpx;
    const float Dy = C * dG0_dpsi * f.an * drho_dpy;
    const float ve1 = dot3f(d, f.e1), ve2 = dot3f(d, f.e2);
    const float ve3 = -(d[0] * f.e2[1]) + d[1] * f.e2[0];   // e3 = (-cos ph, -sin ph, 0) = (-e2.y, e2.x, 0)
    const float dth = Dz * ve1 + pz * (Dy * f.sg - Dx * f.cg);
    const float dph = Dz * f.st * ve2 + Dx * (f.cg * f.ct * ve2 + f.sg * ve3) + Dy * (f.cg * ve3 - f.sg * f.ct * ve2);
    const float dga = Dx * py - Dy * px;
    draw[0] = -dth * f.st;
    draw[1] = -2.f * dph * f.sh1;
    draw[2] = -2.f * dga * f.sh2;
    draw[3] = C * dG0_dlam * f.dlam;
    draw[4] = C * dG0_da * f.dan;
    draw[5] = kGabor ? G0 * dC_dom * f.dom : 0.f;
#pragma unroll
    for (int j = 0; j < 3; ++j) dd[j] = Dz * f.z[j] + Dx * f.x[j] + Dy * f.y[j];
    return G0 * C;
}

}  // namespace gsr
