// Rotary position encoding: the (cos, sin) table (paper Section 2.2,
// "Positional encodings"; rope.h).
//
// Forward: the QKV projection epilogues rotate q and k in fp32 before they
// are stored (proj.hip).  Backward: the attention-backward kernels turn dQ
// and dK back through the rotation, R(p)^T, before storing them
// (attn_bwd.hip), so the projections see the gradients of the unrotated q, k.
#include "kernels.h"

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

}  // namespace

int launch_rope_table(int T, int dh, float base, float2* tab, hipStream_t stream) {
    const int total = T * (dh / 4);
    hipLaunchKernelGGL(rope_table_kernel, dim3((total + 255) / 256), dim3(256), 0, stream, T, dh, (double)base, tab);
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

}  // namespace mosa
