// Deterministic head-ordered combination of per-head rows into a [B, T, d]
// output tile (used by the epilogues of out_combine and dx_combine).
//
// The output tile is 64 tokens x 128 columns; 4 threads own one token row, 32
// columns each, starting from the fp32 tile value the GEMM left in LDS.  The
// MoSA heads that selected token t are found from the slot map
// slot[b, h, t] (position of t among head h's selected tokens, or -1): the
// map for 64 tokens x 256 heads is staged in LDS token-major (16-byte loads
// of 8 tokens when T % 8 == 0), each thread
// scans its token's heads 8 at a time, and the rows of the hits are fetched
// four at a time (16 loads in flight) and added in ascending head order.
// Every output element is thus produced by one thread in a fixed order
// (bitwise reproducible, no atomics), and tokens no head selected keep the
// GEMM value exactly.
#pragma once

#include "gemm.h"

namespace mosa {

constexpr int kCombineHeads = 256;              // heads staged per pass
constexpr int kCombineLdh = kCombineHeads + 8;  // padded LDS row (int16)
constexpr size_t kCombineLds = (size_t)64 * kCombineLdh * sizeof(int16_t);

template <typename ST>
__device__ __forceinline__ void combine_tile(const float* Cs, int ldc, int tid, int b, int m0, int n0, int T, int d,
                                             int H, int k, const int16_t* __restrict__ slot,
                                             const ST* __restrict__ rows, ST* __restrict__ out, int accumulate,
                                             int16_t* s_slot) {
    const int ml = tid >> 2, cq = (tid & 3) * 32;
    const int t = m0 + ml;
    const bool active = t < T && n0 + cq < d;  // d is a multiple of 64: 32-column groups are all in or all out
    float acc[32];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        float x[8];
        cs_load8(Cs, ldc, ml, cq + 8 * c, x);
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[8 * c + e] = active ? x[e] : 0.f;
    }

    const ST* rbase = rows + (size_t)b * H * k * d + n0 + cq;
    // Queue of up to 4 pending hits as a shift register (newest in qh3/qs3),
    // so that every access uses a fixed register and nothing spills to
    // scratch memory; the valid entries are the last q.
    int q = 0, qh0 = 0, qh1 = 0, qh2 = 0, qh3 = 0, qs0 = 0, qs1 = 0, qs2 = 0, qs3 = 0;
    auto flush = [&]() {
        const int hh[4] = {qh0, qh1, qh2, qh3}, ss[4] = {qs0, qs1, qs2, qs3};
        Vec8<ST> v[4][4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const ST* p = j >= 4 - q ? rbase + ((size_t)hh[j] * k + ss[j]) * d : rbase;
#pragma unroll
            for (int c = 0; c < 4; ++c) v[j][c] = vec8_load<ST>(p + 8 * c);
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            if (j >= 4 - q) {
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    float x[8];
                    vec8_to_f32<ST>(v[j][c], x);
#pragma unroll
                    for (int e = 0; e < 8; ++e) acc[8 * c + e] += x[e];
                }
            }
        }
        q = 0;
    };
    auto push = [&](int h, int s) {
        qh0 = qh1; qh1 = qh2; qh2 = qh3; qh3 = h;
        qs0 = qs1; qs1 = qs2; qs2 = qs3; qs3 = s;
        if (++q == 4) flush();
    };

    for (int h0 = 0; h0 < H; h0 += kCombineHeads) {
        const int hn = min(kCombineHeads, H - h0);
        __syncthreads();  // the previous pass's readers are done with s_slot
        if ((T & 7) == 0) {
            // 8 tokens of one head per 16-byte load (rows of the map are
            // 16-byte aligned when T % 8 == 0); up to 8 loads in flight per
            // thread, then transposed into the token-major table.
            for (int e0 = 0; e0 < hn * 8; e0 += 8 * 256) {
                uint4 v[8];
#pragma unroll
                for (int u = 0; u < 8; ++u) {
                    const int e = e0 + u * 256 + tid, hh = e >> 3, q = e & 7;
                    const bool in = e < hn * 8 && m0 + 8 * q < T;
                    const size_t off = in ? ((size_t)b * H + h0 + hh) * T + m0 + 8 * q : 0;
                    v[u] = *reinterpret_cast<const uint4*>(slot + off);
                    if (!in) v[u] = make_uint4(0xffffffffu, 0xffffffffu, 0xffffffffu, 0xffffffffu);
                }
#pragma unroll
                for (int u = 0; u < 8; ++u) {
                    const int e = e0 + u * 256 + tid, hh = e >> 3, q = e & 7;
                    if (e < hn * 8) {
                        const uint32_t w[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
                        int16_t* dst = s_slot + (8 * q) * kCombineLdh + hh;
#pragma unroll
                        for (int j = 0; j < 8; ++j)
                            dst[j * kCombineLdh] = (int16_t)((j & 1) ? (w[j >> 1] >> 16) : (w[j >> 1] & 0xffffu));
                    }
                }
            }
        } else {
            for (int e = tid; e < hn * 64; e += 256) {
                const int hh = e >> 6, tl = e & 63;
                const int tt = m0 + tl;
                s_slot[tl * kCombineLdh + hh] = tt < T ? slot[((size_t)b * H + h0 + hh) * T + tt] : (int16_t)-1;
            }
        }
        __syncthreads();
        if (active) {
            const int16_t* mine = s_slot + ml * kCombineLdh;
            for (int hh = 0; hh < hn; hh += 8) {
                uint4 u;
                if (hh + 8 <= hn) {
                    u = *reinterpret_cast<const uint4*>(mine + hh);
                } else {
                    uint32_t w[4];
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        const uint32_t lo = hh + 2 * j < hn ? (uint16_t)mine[hh + 2 * j] : 0xffffu;
                        const uint32_t hi = hh + 2 * j + 1 < hn ? (uint16_t)mine[hh + 2 * j + 1] : 0xffffu;
                        w[j] = lo | (hi << 16);
                    }
                    u = make_uint4(w[0], w[1], w[2], w[3]);
                }
                // bit j set: head hh + j selected the token (slot >= 0)
                const uint32_t words[4] = {u.x, u.y, u.z, u.w};
                uint32_t mask = 0;
#pragma unroll
                for (int j = 0; j < 8; ++j) mask |= ((words[j >> 1] >> (16 * (j & 1) + 15)) & 1u ? 0u : 1u) << j;
                const uint64_t lo64 = ((uint64_t)u.y << 32) | u.x, hi64 = ((uint64_t)u.w << 32) | u.z;
                while (mask) {
                    const int j = __builtin_ctz(mask);
                    mask &= mask - 1;
                    const int sl = (int)(((j < 4 ? lo64 : hi64) >> (16 * (j & 3))) & 0xffffu);
                    push(h0 + hh + j, sl);
                }
            }
        }
    }
    if (active) {
        if (q > 0) flush();
        ST* y = out + ((size_t)b * T + t) * d + n0 + cq;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            float x[8];
            if (accumulate) {
                vec8_to_f32<ST>(vec8_load<ST>(y + 8 * c), x);
#pragma unroll
                for (int e = 0; e < 8; ++e) x[e] += acc[8 * c + e];
            } else {
#pragma unroll
                for (int e = 0; e < 8; ++e) x[e] = acc[8 * c + e];
            }
            vec8_store<ST>(y + 8 * c, vec8_from_f32<ST>(x));
        }
    }
}

}  // namespace mosa
