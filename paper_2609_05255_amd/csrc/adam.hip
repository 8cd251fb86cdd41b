// Fused Adam step over several planar [rows][n] fp32 parameter tensors in one
// launch (Kingma and Ba, Algorithm 1, with the bias corrections folded into
// the step size and the denominator; one learning rate per row). A pure
// streaming kernel: per element it reads param, grad, m, v and writes param,
// m, v (and optionally the binary16 copy), so it is bound by HBM bandwidth.
//
// Workgroups are dealt to (tensor, row, chunk of kChunk elements): the tensor
// and row are uniform per workgroup, so the row's step size is a kernel
// argument read through the scalar unit, and consecutive lanes touch
// consecutive elements.
#include <cmath>
#include <cstring>

#include "adam_update.h"
#include "gs_internal.h"

#pragma clang fp contract(off)

namespace gsr {

namespace {

constexpr int kItems = 4;
constexpr int kChunk = kBlock * kItems;

struct AdamTensorArgs {
    float* p;
    const float* g;
    float* m;
    float* v;
    uint16_t* h;
    int64_t n;
    int64_t chunk0;        // first workgroup of this tensor
    int32_t chunks_per_row;
};

struct AdamArgs {
    int32_t count;
    AdamTensorArgs t[GS_ADAM_MAX_TENSORS];
    AdamStep c;
};

__global__ __launch_bounds__(kBlock) void k_adam(AdamArgs a)
{
    const int64_t b = blockIdx.x;
    int k = 0;
    while (k + 1 < a.count && b >= a.t[k + 1].chunk0) ++k;
    const AdamTensorArgs& T = a.t[k];
    const int64_t local = b - T.chunk0;
    const int row = (int)(local / T.chunks_per_row);
    const int64_t c = local - (int64_t)row * T.chunks_per_row;
    const float step = a.c.step_size[a.c.row0[k] + row];
    const float b2 = a.c.b2[k], omb2 = a.c.omb2[k], isbc2 = a.c.inv_sqrt_bc2[k];
    const int64_t e0 = c * kChunk + threadIdx.x;
    const int64_t rbase = (int64_t)row * T.n;
    float g[kItems], m[kItems], v[kItems], p[kItems];
    // all loads first; every element is streamed once: non-temporal accesses
#pragma unroll
    for (int j = 0; j < kItems; ++j) {
        const int64_t e = e0 + (int64_t)j * kBlock;
        if (e < T.n) {
            const int64_t i = rbase + e;
            g[j] = __builtin_nontemporal_load(T.g + i);
            m[j] = __builtin_nontemporal_load(T.m + i);
            v[j] = __builtin_nontemporal_load(T.v + i);
            p[j] = __builtin_nontemporal_load(T.p + i);
        }
    }
#pragma unroll
    for (int j = 0; j < kItems; ++j) {
        const int64_t e = e0 + (int64_t)j * kBlock;
        if (e >= T.n) continue;
        const int64_t i = rbase + e;
        adam_update(p[j], m[j], v[j], g[j], a.c.b1, a.c.omb1, b2, omb2, isbc2, a.c.eps, step);
        __builtin_nontemporal_store(m[j], T.m + i);
        __builtin_nontemporal_store(v[j], T.v + i);
        __builtin_nontemporal_store(p[j], T.p + i);
        if (T.h) __builtin_nontemporal_store(__builtin_bit_cast(uint16_t, (_Float16)p[j]), T.h + i);
    }
}

}  // namespace

void adam_step_constants(const gs_adam_tensor* ts, int count, float beta1, float eps, int64_t step, AdamStep& c)
{
    memset(&c, 0, sizeof(c));
    c.b1 = beta1;
    c.omb1 = 1.f - beta1;
    c.eps = eps;
    const double bc1 = 1.0 - std::pow((double)beta1, (double)step);
    int rows = 0;
    for (int k = 0; k < count; ++k) {
        const gs_adam_tensor& t = ts[k];
        c.row0[k] = rows;
        c.b2[k] = t.beta2;
        c.omb2[k] = 1.f - t.beta2;
        const double bc2 = 1.0 - std::pow((double)t.beta2, (double)step);
        c.inv_sqrt_bc2[k] = (float)(1.0 / std::sqrt(bc2));
        for (int r = 0; r < t.rows; ++r) c.step_size[rows + r] = (float)((double)t.lr[r] / bc1);
        rows += t.rows;
    }
}

hipError_t launch_adam(const gs_adam_tensor* ts, int count, float beta1, float eps, int64_t step, hipStream_t s)
{
    AdamArgs a;
    memset(&a, 0, sizeof(a));
    a.count = count;
    adam_step_constants(ts, count, beta1, eps, step, a.c);
    int64_t chunks = 0;
    for (int k = 0; k < count; ++k) {
        const gs_adam_tensor& t = ts[k];
        AdamTensorArgs& T = a.t[k];
        T.p = t.param;
        T.g = t.grad;
        T.m = t.exp_avg;
        T.v = t.exp_avg_sq;
        T.h = t.param_half;
        T.n = t.n;
        T.chunk0 = chunks;
        T.chunks_per_row = (int32_t)div_up(t.n, kChunk);
        chunks += (int64_t)t.rows * T.chunks_per_row;
    }
    if (chunks == 0) return hipSuccess;
    hipLaunchKernelGGL(k_adam, dim3((unsigned)chunks), dim3(kBlock), 0, s, a);
    return hipGetLastError();
}

}  // namespace gsr
