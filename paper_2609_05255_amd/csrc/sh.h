// Real spherical harmonics of degree <= 3 for the appearance model of
// eq. sh_color_eval, as homogeneous polynomials of the unit direction (x, y, z).
// Basis k = l^2 + l + m (m = -l..l), Condon-Shortley phase kept, so band 1 is
// sqrt(3/(4 pi)) (-y, z, -x). Each constant is N_lm * sqrt(2) (for m != 0)
// times the factor that the m-th derivative of the Legendre polynomial P_l and
// (x + iy)^m contribute, N_lm = sqrt((2l+1)/(4 pi) (l-m)!/(l+m)!).
#pragma once

namespace gsr {

constexpr float kSH0 = 0.28209479177387814f;    // 1/(2 sqrt(pi))
constexpr float kSH1 = 0.48860251190291992f;    // sqrt(3/(4 pi))
constexpr float kSH2a = 1.0925484305920792f;    // sqrt(15/pi)/2
constexpr float kSH2b = 0.31539156525252005f;   // sqrt(5/pi)/4
constexpr float kSH2c = 0.54627421529603959f;   // sqrt(15/pi)/4
constexpr float kSH3a = -0.59004358992664352f;  // -sqrt(35/(2 pi))/4
constexpr float kSH3b = 2.8906114426405538f;    // sqrt(105/pi)/2
constexpr float kSH3c = -0.45704579946446572f;  // -sqrt(21/(2 pi))/4
constexpr float kSH3d = 0.37317633259011546f;   // sqrt(7/pi)/4
constexpr float kSH3e = 1.4453057213202769f;    // sqrt(105/pi)/4

// Taken without fused multiply-adds, so that every kernel that inlines it gets
// the same bits whatever else it computes from x, y, z beside it.
__device__ __forceinline__ void sh_basis16(float x, float y, float z, float Y[16])
{
#pragma clang fp contract(off)
    const float xx = x * x, yy = y * y, zz = z * z;
    Y[0] = kSH0;
    Y[1] = -kSH1 * y;
    Y[2] = kSH1 * z;
    Y[3] = -kSH1 * x;
    Y[4] = kSH2a * x * y;
    Y[5] = -kSH2a * y * z;
    Y[6] = kSH2b * (2.f * zz - xx - yy);
    Y[7] = -kSH2a * x * z;
    Y[8] = kSH2c * (xx - yy);
    Y[9] = kSH3a * y * (3.f * xx - yy);
    Y[10] = kSH3b * x * y * z;
    Y[11] = kSH3c * y * (4.f * zz - xx - yy);
    Y[12] = kSH3d * z * (2.f * zz - 3.f * xx - 3.f * yy);
    Y[13] = kSH3c * x * (4.f * zz - xx - yy);
    Y[14] = kSH3e * z * (xx - yy);
    Y[15] = kSH3a * x * (xx - 3.f * yy);
}

// Gradient of each basis polynomial w.r.t. (x, y, z): G[3k + j] = dY_k/dx_j.
__device__ __forceinline__ void sh_basis16_grad(float x, float y, float z, float G[48])
{
    const float xx = x * x, yy = y * y, zz = z * z;
    G[0] = 0.f; G[1] = 0.f; G[2] = 0.f;
    G[3] = 0.f; G[4] = -kSH1; G[5] = 0.f;
    G[6] = 0.f; G[7] = 0.f; G[8] = kSH1;
    G[9] = -kSH1; G[10] = 0.f; G[11] = 0.f;
    G[12] = kSH2a * y; G[13] = kSH2a * x; G[14] = 0.f;
    G[15] = 0.f; G[16] = -kSH2a * z; G[17] = -kSH2a * y;
    G[18] = -2.f * kSH2b * x; G[19] = -2.f * kSH2b * y; G[20] = 4.f * kSH2b * z;
    G[21] = -kSH2a * z; G[22] = 0.f; G[23] = -kSH2a * x;
    G[24] = 2.f * kSH2c * x; G[25] = -2.f * kSH2c * y; G[26] = 0.f;
    G[27] = 6.f * kSH3a * x * y; G[28] = 3.f * kSH3a * (xx - yy); G[29] = 0.f;
    G[30] = kSH3b * y * z; G[31] = kSH3b * x * z; G[32] = kSH3b * x * y;
    G[33] = -2.f * kSH3c * x * y; G[34] = kSH3c * (4.f * zz - xx - 3.f * yy); G[35] = 8.f * kSH3c * y * z;
    G[36] = -6.f * kSH3d * x * z; G[37] = -6.f * kSH3d * y * z; G[38] = kSH3d * (6.f * zz - 3.f * xx - 3.f * yy);
    G[39] = kSH3c * (4.f * zz - 3.f * xx - yy); G[40] = -2.f * kSH3c * x * y; G[41] = 8.f * kSH3c * x * z;
    G[42] = 2.f * kSH3e * x * z; G[43] = -2.f * kSH3e * y * z; G[44] = kSH3e * (xx - yy);
    G[45] = 3.f * kSH3a * (xx - yy); G[46] = -6.f * kSH3a * x * y; G[47] = 0.f;
}

// dd += sum_k dY[k] * grad Y_k(x, y, z), without materialising the 16x3 gradient.
__device__ __forceinline__ void sh_basis16_vjp(float x, float y, float z, const float dY[16], float dd[3])
{
    const float xx = x * x, yy = y * y, zz = z * z;
    float gx = 0.f, gy = 0.f, gz = 0.f;
    gy += -kSH1 * dY[1];
    gz += kSH1 * dY[2];
    gx += -kSH1 * dY[3];
    gx += kSH2a * y * dY[4];               gy += kSH2a * x * dY[4];
    gy += -kSH2a * z * dY[5];              gz += -kSH2a * y * dY[5];
    gx += -2.f * kSH2b * x * dY[6];        gy += -2.f * kSH2b * y * dY[6];       gz += 4.f * kSH2b * z * dY[6];
    gx += -kSH2a * z * dY[7];              gz += -kSH2a * x * dY[7];
    gx += 2.f * kSH2c * x * dY[8];         gy += -2.f * kSH2c * y * dY[8];
    gx += 6.f * kSH3a * x * y * dY[9];     gy += 3.f * kSH3a * (xx - yy) * dY[9];
    gx += kSH3b * y * z * dY[10];          gy += kSH3b * x * z * dY[10];         gz += kSH3b * x * y * dY[10];
    gx += -2.f * kSH3c * x * y * dY[11];   gy += kSH3c * (4.f * zz - xx - 3.f * yy) * dY[11];
    gz += 8.f * kSH3c * y * z * dY[11];
    gx += -6.f * kSH3d * x * z * dY[12];   gy += -6.f * kSH3d * y * z * dY[12];
    gz += kSH3d * (6.f * zz - 3.f * xx - 3.f * yy) * dY[12];
    gx += kSH3c * (4.f * zz - 3.f * xx - yy) * dY[13];
    gy += -2.f * kSH3c * x * y * dY[13];   gz += 8.f * kSH3c * x * z * dY[13];
    gx += 2.f * kSH3e * x * z * dY[14];    gy += -2.f * kSH3e * y * z * dY[14];  gz += kSH3e * (xx - yy) * dY[14];
    gx += 3.f * kSH3a * (xx - yy) * dY[15]; gy += -6.f * kSH3a * x * y * dY[15];
    dd[0] += gx;
    dd[1] += gy;
    dd[2] += gz;
}

// jac[3 c + j] = sum over the bands below nb (k >= 1) of coef[3 k + c] dY_k/dx_j:
// the direction Jacobian of the three colour sums, one pass over the basis.
// Only the gradient components that are not identically zero are multiplied
// in (band 1 has one per basis function, and sets each of the nine entries
// first); for nb = 1 the Jacobian is zero.
__device__ __forceinline__ void sh_color_jacobian(float x, float y, float z, const float* coef, int nb,
                                                  float jac[9])
{
    if (nb < 4) {
        for (int r = 0; r < 9; ++r) jac[r] = 0.f;
        return;
    }
    const float xx = x * x, yy = y * y, zz = z * z;
    // component j of basis k's gradient is g: jac[3 c + j] += coef[3 k + c] g
    auto add = [&](int k, int j, float g) {
        if (k >= nb) return;
        for (int c = 0; c < 3; ++c) jac[3 * c + j] = fmaf(coef[3 * k + c], g, jac[3 * c + j]);
    };
    for (int c = 0; c < 3; ++c) {
        jac[3 * c + 0] = coef[9 + c] * -kSH1;   // Y_3 = -K1 x
        jac[3 * c + 1] = coef[3 + c] * -kSH1;   // Y_1 = -K1 y
        jac[3 * c + 2] = coef[6 + c] * kSH1;    // Y_2 = K1 z
    }
    add(4, 0, kSH2a * y);               add(4, 1, kSH2a * x);
    add(5, 1, -kSH2a * z);              add(5, 2, -kSH2a * y);
    add(6, 0, -2.f * kSH2b * x);        add(6, 1, -2.f * kSH2b * y);      add(6, 2, 4.f * kSH2b * z);
    add(7, 0, -kSH2a * z);              add(7, 2, -kSH2a * x);
    add(8, 0, 2.f * kSH2c * x);         add(8, 1, -2.f * kSH2c * y);
    add(9, 0, 6.f * kSH3a * x * y);     add(9, 1, 3.f * kSH3a * (xx - yy));
    add(10, 0, kSH3b * y * z);          add(10, 1, kSH3b * x * z);        add(10, 2, kSH3b * x * y);
    add(11, 0, -2.f * kSH3c * x * y);   add(11, 1, kSH3c * (4.f * zz - xx - 3.f * yy));
    add(11, 2, 8.f * kSH3c * y * z);
    add(12, 0, -6.f * kSH3d * x * z);   add(12, 1, -6.f * kSH3d * y * z);
    add(12, 2, kSH3d * (6.f * zz - 3.f * xx - 3.f * yy));
    add(13, 0, kSH3c * (4.f * zz - 3.f * xx - yy));
    add(13, 1, -2.f * kSH3c * x * y);   add(13, 2, 8.f * kSH3c * x * z);
    add(14, 0, 2.f * kSH3e * x * z);    add(14, 1, -2.f * kSH3e * y * z); add(14, 2, kSH3e * (xx - yy));
    add(15, 0, 3.f * kSH3a * (xx - yy)); add(15, 1, -6.f * kSH3a * x * y);
}

}  // namespace gsr
