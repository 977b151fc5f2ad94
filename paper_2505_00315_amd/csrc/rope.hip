// Rotary position encoding: the (cos, sin) table and the backward rotation
// of dQ and dK (paper Section 2.2, "Positional encodings"; rope.h).
//
// Forward: the QKV projection epilogues rotate q and k in fp32 before they
// are stored (proj.hip).  Backward: the attention kernels give dQ and dK
// with respect to the rotated q and k; the projections need R(p)^T dQ and
// R(p)^T dK, applied here in place on the dQ | dK | dV rows.
#include "kernels.h"
#include "rope.h"
#include "gemm.h"

namespace mosa {

namespace {

// tab[t][j] = (cos, sin)(t theta_j), theta_j = base^(-2j/R), R = dh/2, in fp64.
__global__ __launch_bounds__(256) void rope_table_kernel(int T, int dh, double base, float2* __restrict__ tab) {
    const int q = dh / 4, e = blockIdx.x * 256 + threadIdx.x;
    if (e >= T * q) return;
    const int t = e / q, j = e % q;
    const double ang = (double)t * pow(base, -2.0 * j / (double)(dh / 2));
    double s, c;
    sincos(ang, &s, &c);
    tab[e] = make_float2((float)c, (float)s);
}

// One thread per 8-column vector of the rotated part of dQ or dK of a row
// (row = (b, h, i); position I[row], or i for dense heads, I == nullptr).
template <typename ST, int DH>
__global__ __launch_bounds__(256) void rope_grad_kernel(ST* __restrict__ dQKV, const int32_t* __restrict__ I,
                                                        const float2* __restrict__ tab, int rows, int n) {
    constexpr int VR = DH / 16;  // vectors in the rotated half of dQ (and of dK)
    const int e = blockIdx.x * 256 + threadIdx.x;
    if (e >= rows * 2 * VR) return;
    const int row = e / (2 * VR), v = e % (2 * VR), part = v / VR, c0 = 8 * (v % VR);
    const int pos = I ? I[row] : row % n;
    ST* p = dQKV + (size_t)row * (3 * DH) + part * DH + c0;
    float x[8];
    vec8_to_f32<ST>(vec8_load<ST>(p), x);
    rope8<DH>(x, c0, tab, pos, -1.f);
    vec8_store<ST>(p, vec8_from_f32<ST>(x));
}

}  // namespace

int launch_rope_table(int T, int dh, float base, float2* tab, hipStream_t stream) {
    const int total = T * (dh / 4);
    hipLaunchKernelGGL(rope_table_kernel, dim3((total + 255) / 256), dim3(256), 0, stream, T, dh, (double)base, tab);
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

int launch_rope_grad(int dtype, void* dQKV, const int32_t* I, const float2* tab, int rows, int n, int dh,
                     hipStream_t stream) {
    if (rows <= 0) return 0;
    const dim3 grid((rows * (dh / 8) + 255) / 256);
    if (dtype == kBF16) {
        auto k = dh == 64 ? rope_grad_kernel<uint16_t, 64> : rope_grad_kernel<uint16_t, 32>;
        hipLaunchKernelGGL(k, grid, dim3(256), 0, stream, (uint16_t*)dQKV, I, tab, rows, n);
    } else {
        auto k = dh == 64 ? rope_grad_kernel<float, 64> : rope_grad_kernel<float, 32>;
        hipLaunchKernelGGL(k, grid, dim3(256), 0, stream, (float*)dQKV, I, tab, rows, n);
    }
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

}  // namespace mosa
