/*
 * CPU oracle -- TEST INFRASTRUCTURE ONLY (see gs_oracle.h).
 *
 * Precision-independent helpers live here; the preprocess, blend and their
 * derivatives are in gs_oracle_body.inc, compiled once with the decision
 * precision REAL = float (suffix _f32) and once with REAL = double (_f64).
 * Build: gcc -O2 -std=c11 -ffp-contract=off -fno-fast-math -shared -fPIC.
 */
#include "gs_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

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

static int pair_cmp(const void* pa, const void* pb)
{
    const orc_pair* a = (const orc_pair*)pa;
    const orc_pair* b = (const orc_pair*)pb;
    if (a->tile != b->tile) return a->tile < b->tile ? -1 : 1;
    if (a->depth != b->depth) return a->depth < b->depth ? -1 : 1;
    if (a->idx != b->idx) return a->idx < b->idx ? -1 : 1;
    return 0;
}

int64_t orc_bin_sort(int64_t n, const int32_t* rect, const double* depth, const int32_t* tiles,
                     int32_t tiles_x, int32_t tiles_y, int64_t capacity, int32_t* values,
                     int32_t* tile_of, int64_t* ranges)
{
    int64_t total = 0;
    for (int64_t i = 0; i < n; ++i) total += tiles[i] > 0 ? tiles[i] : 0;
    if (total > capacity) return -1;
    orc_pair* pairs = (orc_pair*)malloc(sizeof(orc_pair) * (size_t)(total > 0 ? total : 1));
    int64_t k = 0;
    for (int64_t i = 0; i < n; ++i) {
        if (tiles[i] <= 0) continue;
        int x0 = rect[0 * n + i], y0 = rect[1 * n + i], x1 = rect[2 * n + i], y1 = rect[3 * n + i];
        for (int ty = y0; ty < y1; ++ty)
            for (int tx = x0; tx < x1; ++tx) {
                pairs[k].tile = ty * tiles_x + tx;
                pairs[k].idx = (int32_t)i;
                pairs[k].depth = depth[i];
                ++k;
            }
    }
    qsort(pairs, (size_t)total, sizeof(orc_pair), pair_cmp);
    int64_t n_tiles = (int64_t)tiles_x * tiles_y;
    for (int64_t t = 0; t < n_tiles; ++t) { ranges[2 * t] = 0; ranges[2 * t + 1] = 0; }
    for (int64_t p = 0; p < total; ++p) {
        values[p] = pairs[p].idx;
        if (tile_of) tile_of[p] = pairs[p].tile;
        ranges[2 * pairs[p].tile + 1] += 1;          /* count first */
    }
    int64_t start = 0;
    for (int64_t t = 0; t < n_tiles; ++t) {
        int64_t cnt = ranges[2 * t + 1];
        ranges[2 * t] = start;
        ranges[2 * t + 1] = start + cnt;
        start += cnt;
    }
    free(pairs);
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
