// Rotary position encoding (paper Section 2.2, "Positional encodings") at a
// token's ORIGINAL position p: the first DH/2 dimensions of q and k are
// rotated in adjacent pairs (2j, 2j+1) by the angle p theta_j with
// theta_j = base^(-2j/(DH/2)); the other half is left unchanged.  The
// (cos, sin) pairs come from a table [T][DH/4] of float2 built in fp64
// (rope.hip), so that the angle of a large position is exact to fp32.
#pragma once

#include "common.h"

namespace mosa {

// 8 consecutive columns c0 .. c0 + 7 (c0 % 8 == 0, c0 < DH/2) of a q or k
// row at position pos: the 4 pairs they hold, rotated by +angle (sign 1) or
// by -angle (sign -1, the transpose used by the backward pass).
template <int DH>
__device__ __forceinline__ void rope8(float (&x)[8], int c0, const float2* __restrict__ tab, int pos, float sign) {
    const float2* t = tab + (size_t)pos * (DH / 4) + c0 / 2;
    const float4 a = *reinterpret_cast<const float4*>(t), b = *reinterpret_cast<const float4*>(t + 2);
    const float cs[4] = {a.x, a.z, b.x, b.z}, sn[4] = {a.y, a.w, b.y, b.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const float u = x[2 * i], v = x[2 * i + 1], s = sign * sn[i];
        x[2 * i] = u * cs[i] - v * s;
        x[2 * i + 1] = u * s + v * cs[i];
    }
}

// 4 consecutive columns d0 .. d0 + 3 (d0 % 4 == 0) of a dQ or dK row at
// position pos: the two pairs turned back by R(p)^T if they lie in the
// rotated half (the gradient with respect to the unrotated q or k).
template <int DH>
__device__ __forceinline__ void rope4_back(float (&x)[4], int d0, const float2* __restrict__ tab, int pos) {
    if (d0 >= DH / 2) return;
    const float4 t = *reinterpret_cast<const float4*>(tab + (size_t)pos * (DH / 4) + d0 / 2);
    const float u0 = x[0], v0 = x[1], u1 = x[2], v1 = x[3];
    x[0] = u0 * t.x + v0 * t.y;
    x[1] = v0 * t.x - u0 * t.y;
    x[2] = u1 * t.z + v1 * t.w;
    x[3] = v1 * t.z - u1 * t.w;
}

}  // namespace mosa
