// LDS tile helpers shared by the attention kernels: raw elements of a
// packed 8-vector (for transposed staging) and MFMA operands assembled from
// two 4-element runs of a transposed tile.
#pragma once

#include "gemm.h"

namespace mosa {

// Element j of 8 packed storage elements, as raw storage.
template <typename ST> __device__ __forceinline__ ST vec8_elem(const Vec8<ST>& v, int j);
template <> __device__ __forceinline__ uint16_t vec8_elem<uint16_t>(const Vec8<uint16_t>& v, int j) {
    const uint32_t w = j < 2 ? v.v.x : j < 4 ? v.v.y : j < 6 ? v.v.z : v.v.w;
    return (uint16_t)((j & 1) ? (w >> 16) : (w & 0xffffu));
}
template <> __device__ __forceinline__ float vec8_elem<float>(const Vec8<float>& v, int j) {
    return j == 0 ? v.a.x : j == 1 ? v.a.y : j == 2 ? v.a.z : j == 3 ? v.a.w
         : j == 4 ? v.b.x : j == 5 ? v.b.y : j == 6 ? v.b.z : v.b.w;
}

// Four consecutive storage elements from LDS as MFMA operand halves.
template <typename ST> struct Quad;
template <> struct Quad<uint16_t> { uint2 v; };
template <> struct Quad<float> { float4 v; };
template <typename ST> __device__ __forceinline__ Quad<ST> quad_load(const ST* p) {
    Quad<ST> q;
    q.v = *reinterpret_cast<const decltype(q.v)*>(p);
    return q;
}
// Frag8 from two quads (slots 0..3 and 4..7 of the lane).
template <typename ST> __device__ __forceinline__ Frag8<ST> frag8_from_quads(const Quad<ST>& lo, const Quad<ST>& hi);
template <> __device__ __forceinline__ Frag8<uint16_t> frag8_from_quads<uint16_t>(const Quad<uint16_t>& lo,
                                                                                const Quad<uint16_t>& hi) {
    Frag8<uint16_t> f;
    f.v = __builtin_bit_cast(bf16x8, make_uint4(lo.v.x, lo.v.y, hi.v.x, hi.v.y));
    return f;
}
template <> __device__ __forceinline__ Frag8<float> frag8_from_quads<float>(const Quad<float>& lo,
                                                                          const Quad<float>& hi) {
    Frag8<float> f;
    f.v[0] = lo.v.x; f.v[1] = lo.v.y; f.v[2] = lo.v.z; f.v[3] = lo.v.w;
    f.v[4] = hi.v.x; f.v[5] = hi.v.y; f.v[6] = hi.v.z; f.v[7] = hi.v.w;
    return f;
}

}  // namespace mosa
