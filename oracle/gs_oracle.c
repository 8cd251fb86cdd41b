/*
 * CPU oracle -- TEST INFRASTRUCTURE ONLY (see gs_oracle.h).
 *
 * Precision-independent helpers live here; the preprocess, blend and their
 * derivatives are in gs_oracle_body.inc, compiled once with the decision
 * precision REAL = float (suffix _f32) and once with REAL = double (_f64).
 * Build: gcc -O2 -std=c11 -ffp-contract=off -fno-fast-math -fopenmp -shared -fPIC.
 * Loops over Gaussians, pixels and tiles run on OpenMP threads; every sum is
 * taken in an order fixed by the data (pairs, blocks of Gaussians), so the
 * results do not depend on the number of threads.
 */
#include "gs_oracle.h"

#include <math.h>
#include <omp.h>
#include <stdlib.h>
#include <string.h>

void orc_set_threads(int32_t k) { omp_set_num_threads(k > 0 ? k : 1); }

int32_t orc_get_threads(void) { return (int32_t)omp_get_max_threads(); }

#ifndef M_PI
#define M_PI 3.14159265358979323846
#endif

double orc_round_half(double x)
{
    /* binary16: 10 fraction bits, smallest normal exponent -14, subnormal step 2^-24 */
    if (x == 0.0 || !isfinite(x)) return x;
    int e;
    frexp(fabs(x), &e);
    int lead = e - 1;                  /* exponent of the leading bit */
    if (lead < -14) lead = -14;
    double ulp = ldexp(1.0, lead - 10);
    double q = nearbyint(x / ulp) * ulp;   /* current rounding mode: nearest, ties to even */
    if (fabs(q) > 65504.0) return copysign(INFINITY, x);
    return q;
}

/* ---- real spherical harmonics from the Legendre definition ------------------
 * Y_l^0       = N_l0 P_l(z)
 * Y_l^m (m>0) = sqrt2 N_lm (-1)^m P_l^(m)(z) Re((x+iy)^m)
 * Y_l^-m      = sqrt2 N_lm (-1)^m P_l^(m)(z) Im((x+iy)^m)
 * with N_lm = sqrt((2l+1)/(4 pi) (l-m)!/(l+m)!), P_l^(m) the m-th derivative of
 * the Legendre polynomial and (-1)^m the Condon-Shortley phase. On the unit
 * sphere (x+iy)^m = sin^m(theta) e^{i m phi}, so this is the usual real basis;
 * off the sphere it is one polynomial extension of it. Index k = l^2 + l + m.
 */
static double fact(int k) { double r = 1; for (int i = 2; i <= k; ++i) r *= i; return r; }

static double binom(int n, int k) { return fact(n) / (fact(k) * fact(n - k)); }

/* m-th derivative of P_l evaluated at z */
static double legendre_deriv(int l, int m, double z)
{
    /* P_l(z) = 2^-l sum_k (-1)^k C(l,k) C(2l-2k,l) z^(l-2k) */
    double acc = 0.0;
    for (int k = 0; 2 * k <= l; ++k) {
        int p = l - 2 * k;
        if (p < m) continue;
        double c = ((k & 1) ? -1.0 : 1.0) * binom(l, k) * binom(2 * l - 2 * k, l) / ldexp(1.0, l);
        acc += c * fact(p) / fact(p - m) * pow(z, p - m);
    }
    return acc;
}

void orc_sh_basis(const double d[3], double Y[16], double dY[48])
{
    const double x = d[0], y = d[1], z = d[2];
    for (int l = 0; l <= 3; ++l) {
        for (int m = -l; m <= l; ++m) {
            int am = m < 0 ? -m : m;
            int k = l * l + l + m;
            double N = sqrt((2 * l + 1) / (4.0 * M_PI) * fact(l - am) / fact(l + am));
            if (m != 0) N *= sqrt(2.0) * ((am & 1) ? -1.0 : 1.0);
            /* (x+iy)^am and am*(x+iy)^(am-1) */
            double pr = 1, pi = 0, qr = 0, qi = 0;
            for (int i = 0; i < am; ++i) {
                if (i == am - 1) { qr = am * pr; qi = am * pi; }
                double nr = pr * x - pi * y, ni = pr * y + pi * x;
                pr = nr; pi = ni;
            }
            double P = legendre_deriv(l, am, z);
            double Pz = legendre_deriv(l, am + 1, z);
            double ang, dang_dx, dang_dy;
            if (m >= 0) { ang = pr; dang_dx = qr; dang_dy = -qi; }
            else        { ang = pi; dang_dx = qi; dang_dy = qr; }
            if (m == 0) { ang = 1; dang_dx = 0; dang_dy = 0; }
            Y[k] = N * P * ang;
            if (dY) {
                dY[3 * k + 0] = N * P * dang_dx;
                dY[3 * k + 1] = N * P * dang_dy;
                dY[3 * k + 2] = N * Pz * ang;
            }
        }
    }
}

/* ---- pair list -------------------------------------------------------------- */
typedef struct { int32_t tile; int32_t idx; double depth; } orc_pair;

static int pair_depth_cmp(const void* pa, const void* pb)
{
    const orc_pair* a = (const orc_pair*)pa;
    const orc_pair* b = (const orc_pair*)pb;
    if (a->depth != b->depth) return a->depth < b->depth ? -1 : 1;
    if (a->idx != b->idx) return a->idx < b->idx ? -1 : 1;
    return 0;
}

/* Sorted by (tile, depth, index): the pairs are bucketed by tile (a counting
 * sort), then each tile's bucket is sorted by (depth, index) on its own. */
int64_t orc_bin_sort(int64_t n, const int32_t* rect, const double* depth, const int32_t* tiles,
                     int32_t tiles_x, int32_t tiles_y, int64_t capacity, int32_t* values,
                     int32_t* tile_of, int64_t* ranges)
{
    int64_t total = 0;
    for (int64_t i = 0; i < n; ++i) total += tiles[i] > 0 ? tiles[i] : 0;
    if (total > capacity) return -1;
    const int64_t n_tiles = (int64_t)tiles_x * tiles_y;
    int64_t* cnt = (int64_t*)calloc((size_t)(n_tiles + 1), sizeof(int64_t));
    for (int64_t i = 0; i < n; ++i) {
        if (tiles[i] <= 0) continue;
        int x0 = rect[0 * n + i], y0 = rect[1 * n + i], x1 = rect[2 * n + i], y1 = rect[3 * n + i];
        for (int ty = y0; ty < y1; ++ty)
            for (int tx = x0; tx < x1; ++tx) cnt[ty * tiles_x + tx] += 1;
    }
    int64_t start = 0;
    for (int64_t t = 0; t < n_tiles; ++t) {
        ranges[2 * t] = start;
        ranges[2 * t + 1] = start;       /* fill position */
        start += cnt[t];
    }
    orc_pair* pairs = (orc_pair*)malloc(sizeof(orc_pair) * (size_t)(total > 0 ? total : 1));
    for (int64_t i = 0; i < n; ++i) {
        if (tiles[i] <= 0) continue;
        int x0 = rect[0 * n + i], y0 = rect[1 * n + i], x1 = rect[2 * n + i], y1 = rect[3 * n + i];
        for (int ty = y0; ty < y1; ++ty)
            for (int tx = x0; tx < x1; ++tx) {
                const int64_t t = (int64_t)ty * tiles_x + tx;
                orc_pair* q = &pairs[ranges[2 * t + 1]++];
                q->tile = (int32_t)t;
                q->idx = (int32_t)i;
                q->depth = depth[i];
            }
    }
#pragma omp parallel for schedule(dynamic, 16)
    for (int64_t t = 0; t < n_tiles; ++t)
        qsort(pairs + ranges[2 * t], (size_t)(ranges[2 * t + 1] - ranges[2 * t]), sizeof(orc_pair), pair_depth_cmp);
    for (int64_t p = 0; p < total; ++p) {
        values[p] = pairs[p].idx;
        if (tile_of) tile_of[p] = pairs[p].tile;
    }
    free(pairs);
    free(cnt);
    return total;
}

/* ---- the precision-templated stages ------------------------------------------ */
#define REAL float
#define SFX _f32
#include "gs_oracle_body.inc"
#undef REAL
#undef SFX

#define REAL double
#define SFX _f64
#include "gs_oracle_body.inc"
#undef REAL
#undef SFX

/* The latent decoder alone on caller-given inputs (fp64 on binary16 values):
 * x [rows][17], out [rows][3]. */
void orc_mlp_eval(const double* x, int64_t rows, const double* w, double* out, int32_t half_act)
{
    for (int64_t r = 0; r < rows; ++r) {
        double h1[32], h2[32], o[3];
        mlp_forward_f64(w, x + 17 * r, h1, h2, o, half_act);
        for (int c = 0; c < 3; ++c) out[3 * r + c] = 1.0 / (1.0 + exp(-o[c]));
    }
}

/* ---- NASG / NASGabor lobe (eq. nasg) ------------------------------------------
 * The paper takes the kernel from the NASGabor work without restating it; this
 * is the normalized anisotropic spherical Gaussian of Huang et al. (2024), with
 * the parametrisation read from the paper's description of the activations:
 *   frame   cos(theta) = tanh(r0), and the half angles of the azimuth phi and the
 *           twist gamma have cosines tanh(r1), tanh(r2) (so that phi and gamma
 *           cover (0, 2 pi)); z = (sin th cos ph, sin th sin ph, cos th),
 *           e1 = dz/dth, e2 = (-sin ph, cos ph, 0), x = cos ga e1 + sin ga e2,
 *           y = -sin ga e1 + cos ga e2;
 *   shape   lambda = exp(clamp(r3, -8, 8)) (sharpness), a = exp(clamp(r4, -8, 8))
 *           (anisotropy);
 *   kernel  u = (v.z + 1)/2, rho = (v.x)^2 / ((v.x)^2 + (v.y)^2), psi = a rho,
 *           G(v) = exp(2 lambda (u^(1+psi) - 1)) u^psi / K,
 *           K = 2 pi (1 - exp(-2 lambda)) / (lambda sqrt(1 + a)),
 *           which integrates to 1 over the sphere;
 *   Gabor   G~(v) = G(v) (1 + cos(omega v.x)) / 2, omega = 20 (tanh(r5) + 1),
 *           a non-negative cosine carrier along the anisotropy axis.
 * raw[0..4] (and raw[5] with gabor) are the raw lobe parameters. The frame is
 * evaluated with sin(theta) = sech(r0), sin(phi/2) = sech(r1), sin(gamma/2) = sech(r2).
 */
typedef struct lobe_frame {
    double x[3], y[3], z[3], e1[3], e2[3], e3[3];
    double ct, st, cg, sg, sh1, sh2, lam, an, om, dlam, dan, dom;
} lobe_frame;

static double dot3(const double a[3], const double b[3]) { return a[0] * b[0] + a[1] * b[1] + a[2] * b[2]; }

static double clampd(double v, double lo, double hi) { return v < lo ? lo : v > hi ? hi : v; }

static void lobe_setup(const double* raw, int gabor, lobe_frame* f)
{
    const double ct = tanh(raw[0]), st = 1.0 / cosh(raw[0]);
    const double ch = tanh(raw[1]), sh = 1.0 / cosh(raw[1]);
    const double cgh = tanh(raw[2]), sgh = 1.0 / cosh(raw[2]);
    const double cp = ch * ch - sh * sh, sp = 2.0 * sh * ch;      /* phi = 2 (phi/2) */
    const double cg = cgh * cgh - sgh * sgh, sg = 2.0 * sgh * cgh;
    f->ct = ct; f->st = st; f->cg = cg; f->sg = sg; f->sh1 = sh; f->sh2 = sgh;
    const double z[3] = {st * cp, st * sp, ct}, e1[3] = {ct * cp, ct * sp, -st}, e2[3] = {-sp, cp, 0.0};
    const double e3[3] = {-cp, -sp, 0.0};
    for (int j = 0; j < 3; ++j) {
        f->z[j] = z[j]; f->e1[j] = e1[j]; f->e2[j] = e2[j]; f->e3[j] = e3[j];
        f->x[j] = cg * e1[j] + sg * e2[j];
        f->y[j] = -sg * e1[j] + cg * e2[j];
    }
    f->lam = exp(clampd(raw[3], -8.0, 8.0));
    f->an = exp(clampd(raw[4], -8.0, 8.0));
    f->dlam = (raw[3] > -8.0 && raw[3] < 8.0) ? f->lam : 0.0;
    f->dan = (raw[4] > -8.0 && raw[4] < 8.0) ? f->an : 0.0;
    f->om = gabor ? 20.0 * (tanh(raw[5]) + 1.0) : 0.0;
    f->dom = gabor ? 20.0 * (1.0 - tanh(raw[5]) * tanh(raw[5])) : 0.0;
}

double orc_lobe_eval(const double* raw, int32_t gabor, const double v[3])
{
    lobe_frame f;
    lobe_setup(raw, gabor, &f);
    const double px = dot3(v, f.x), py = dot3(v, f.y), pz = dot3(v, f.z);
    const double u = (pz + 1.0) / 2.0, q = px * px + py * py;
    const double psi = f.an * (q > 0 ? px * px / q : 0.0);
    const double K = 2.0 * M_PI * (-expm1(-2.0 * f.lam)) / (f.lam * sqrt(1.0 + f.an));
    double G = exp(2.0 * f.lam * (pow(u, 1.0 + psi) - 1.0)) * pow(u, psi) / K;
    if (gabor) G *= (1.0 + cos(f.om * px)) / 2.0;
    return G;
}

void orc_lobe_eval_many(const double* raw, int32_t gabor, int64_t m, const double* v, double* out)
{
    for (int64_t k = 0; k < m; ++k) out[k] = orc_lobe_eval(raw, gabor, v + 3 * k);
}

/* dG/draw (5 or 6 values) and dG/dv of the lobe above, by the chain rule through
 * the frame: d theta/dr0 = -sin th, d phi/dr1 = -2 sin(phi/2), d gamma/dr2 =
 * -2 sin(gamma/2); dz/dth = e1, dz/dph = sin th e2, dx/dth = -cos ga z,
 * dx/dph = cos ga cos th e2 + sin ga e3, dx/dga = y, dy/dth = sin ga z,
 * dy/dph = -sin ga cos th e2 + cos ga e3, dy/dga = -x, e3 = de2/dph. */
double orc_lobe_grad(const double* raw, int32_t gabor, const double v[3], double* draw, double dv[3])
{
    lobe_frame f;
    lobe_setup(raw, gabor, &f);
    const double px = dot3(v, f.x), py = dot3(v, f.y), pz = dot3(v, f.z);
    const double u = (pz + 1.0) / 2.0, q = px * px + py * py;
    const double rho = q > 0 ? px * px / q : 0.0;
    const double psi = f.an * rho;
    const double em = -expm1(-2.0 * f.lam);
    const double K = 2.0 * M_PI * em / (f.lam * sqrt(1.0 + f.an));
    const double w = pow(u, 1.0 + psi), L = log(u);
    const double G0 = exp(2.0 * f.lam * (w - 1.0)) * pow(u, psi) / K;
    const double C = gabor ? (1.0 + cos(f.om * px)) / 2.0 : 1.0;
    /* partial derivatives of G0 */
    const double dG0_du = G0 * (2.0 * f.lam * (1.0 + psi) * pow(u, psi) + psi / u);
    const double dG0_dpsi = G0 * (2.0 * f.lam * w * L + L);
    const double dlnK_dlam = 2.0 * exp(-2.0 * f.lam) / em - 1.0 / f.lam;
    const double dG0_dlam = G0 * (2.0 * (w - 1.0) - dlnK_dlam);
    const double dG0_da = G0 / (2.0 * (1.0 + f.an)) + dG0_dpsi * rho;
    const double drho_dpx = q > 0 ? 2.0 * px * py * py / (q * q) : 0.0;
    const double drho_dpy = q > 0 ? -2.0 * py * px * px / (q * q) : 0.0;
    const double dC_dpx = gabor ? -f.om * sin(f.om * px) / 2.0 : 0.0;
    const double dC_dom = gabor ? -px * sin(f.om * px) / 2.0 : 0.0;
    const double Dz = C * dG0_du * 0.5;
    const double Dx = C * dG0_dpsi * f.an * drho_dpx + G0 * dC_dpx;
    const double Dy = C * dG0_dpsi * f.an * drho_dpy;
    const double ve1 = dot3(v, f.e1), ve2 = dot3(v, f.e2), ve3 = dot3(v, f.e3);
    const double dth = Dz * ve1 + Dx * (-f.cg * pz) + Dy * (f.sg * pz);
    const double dph = Dz * f.st * ve2 + Dx * (f.cg * f.ct * ve2 + f.sg * ve3) + Dy * (-f.sg * f.ct * ve2 + f.cg * ve3);
    const double dga = Dx * py - Dy * px;
    draw[0] = dth * (-f.st);
    draw[1] = dph * (-2.0 * f.sh1);
    draw[2] = dga * (-2.0 * f.sh2);
    draw[3] = C * dG0_dlam * f.dlam;
    draw[4] = C * dG0_da * f.dan;
    if (gabor) draw[5] = G0 * dC_dom * f.dom;
    for (int j = 0; j < 3; ++j) dv[j] = Dz * f.z[j] + Dx * f.x[j] + Dy * f.y[j];
    return G0 * C;
}
