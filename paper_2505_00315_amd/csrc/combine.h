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

// The same combination as a kernel of its own: out[b, t] (+)= base[b, t] +
// sum over MoSA heads h (ascending) of rows[b, h, slot[b, h, t]], where base
// (storage type, like the rows; optional) holds the dense heads' part.  A
// workgroup takes 16 tokens of one batch element and stages their slot
// entries for every head in LDS (head-major, padded rows); each of its 16
// waves then handles one token, with the whole d-wide row spread over its
// lanes (8 consecutive columns per lane and 64-lane group, so every hit is
// one coalesced d-element load).  The hits of a token are taken 4 at a time
// in ascending head order (the lanes of a 64-head group ballot their slot
// entries); the sum starts from 0 and is added to the old output value at
// the end when accumulating, so every element is produced by one lane in a
// fixed order: the dense part, then the MoSA heads in ascending order.
constexpr int kCombineTokens = 16;               // one per wave
constexpr int kCombineThreads = 64 * kCombineTokens;
constexpr int kCombineLdt = kCombineTokens + 2;  // padded LDS row (int16) per head

// CH: 8-column groups per lane (d <= 512 CH).  USE only names the caller
// (0: the layer output, 1: dX) so that profiles tell the two launches apart.
template <typename ST, int CH, int USE>
__global__ __launch_bounds__(kCombineThreads) void combine_rows_kernel(const int16_t* __restrict__ slot,
                                                           const ST* __restrict__ rows,
                                                           const ST* __restrict__ base, ST* __restrict__ out,
                                                           int T, int d, int H, int k, int accumulate,
                                                           int tiles_per_b) {
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
    int16_t* s_slot = reinterpret_cast<int16_t*>(smem);  // [H][kCombineLdt]
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int logical = xcd_logical_id(blockIdx.x, gridDim.x);
    const int b = logical / tiles_per_b, t0 = (logical % tiles_per_b) * kCombineTokens;

    if ((T & 7) == 0) {
        for (int e = tid; e < H * 2; e += kCombineThreads) {
            const int h = e >> 1, q = e & 1, tt = t0 + 8 * q;
            uint4 v = make_uint4(0xffffffffu, 0xffffffffu, 0xffffffffu, 0xffffffffu);
            if (tt < T) v = *reinterpret_cast<const uint4*>(slot + ((size_t)b * H + h) * T + tt);
            uint32_t* dst = reinterpret_cast<uint32_t*>(s_slot + h * kCombineLdt + 8 * q);
            dst[0] = v.x;
            dst[1] = v.y;
            dst[2] = v.z;
            dst[3] = v.w;
        }
    } else {
        for (int e = tid; e < H * kCombineTokens; e += kCombineThreads) {
            const int h = e / kCombineTokens, tl = e % kCombineTokens, tt = t0 + tl;
            s_slot[h * kCombineLdt + tl] = tt < T ? slot[((size_t)b * H + h) * T + tt] : (int16_t)-1;
        }
    }
    __syncthreads();

    const ST* rb = rows + (size_t)b * H * k * d;
    {
        const int tl = wave, t = t0 + tl;
        if (t >= T) return;
        float acc[CH][8];
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            const int col = 8 * (lane + 64 * c);
            if (base && col < d) {
                vec8_to_f32<ST>(vec8_load<ST>(base + ((size_t)b * T + t) * d + col), acc[c]);
            } else {
#pragma unroll
                for (int e = 0; e < 8; ++e) acc[c][e] = 0.f;
            }
        }
        for (int hc = 0; hc < H; hc += 64) {
            const int h = hc + lane;
            const int sl = h < H ? s_slot[h * kCombineLdt + tl] : -1;
            uint64_t mask = __ballot(sl >= 0);
            while (mask) {
                int hh[4], ss[4], n = 0;
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    if (mask) {
                        const int bit = __builtin_ctzll(mask);
                        mask &= mask - 1;
                        hh[j] = hc + bit;
                        ss[j] = __builtin_amdgcn_readlane(sl, bit);
                        n = j + 1;
                    } else {  // reload the first hit; not added
                        hh[j] = hh[0];
                        ss[j] = ss[0];
                    }
                }
                Vec8<ST> v[4][CH];
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const ST* p = rb + ((size_t)hh[j] * k + ss[j]) * d;
#pragma unroll
                    for (int c = 0; c < CH; ++c) {
                        const int col = 8 * (lane + 64 * c);
                        v[j][c] = col < d ? vec8_load<ST>(p + col) : vec8_zero<ST>();
                    }
                }
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    if (j < n) {
#pragma unroll
                        for (int c = 0; c < CH; ++c) {
                            float x[8];
                            vec8_to_f32<ST>(v[j][c], x);
#pragma unroll
                            for (int e = 0; e < 8; ++e) acc[c][e] += x[e];
                        }
                    }
                }
            }
        }
        ST* y = out + ((size_t)b * T + t) * d;
#pragma unroll
        for (int c = 0; c < CH; ++c) {
            const int col = 8 * (lane + 64 * c);
            if (col >= d) continue;
            float x[8];
            if (accumulate) {
                vec8_to_f32<ST>(vec8_load<ST>(y + col), x);
#pragma unroll
                for (int e = 0; e < 8; ++e) x[e] += acc[c][e];
            } else {
#pragma unroll
                for (int e = 0; e < 8; ++e) x[e] = acc[c][e];
            }
            vec8_store<ST>(y + col, vec8_from_f32<ST>(x));
        }
    }
}

// out (+)= base + head-ordered sum of the MoSA rows; d a multiple of 8, base
// [B, T, d] in the storage type, or nullptr.
inline bool combine_rows_fits(int d, int H) {
    return d % 8 == 0 && d <= 2048 && (size_t)(H > 0 ? H : 1) * kCombineLdt * sizeof(int16_t) <= 64 * 1024;
}
template <typename ST, int USE>
int launch_combine_rows(const int16_t* slot, const ST* rows, const ST* base, ST* out, int B, int T, int d, int H,
                        int k, int accumulate, hipStream_t stream) {
    if (B == 0 || T == 0) return 0;
    if (!combine_rows_fits(d, H)) return -1;
    const int tiles = (T + kCombineTokens - 1) / kCombineTokens;
    const size_t lds = (size_t)(H > 0 ? H : 1) * kCombineLdt * sizeof(int16_t);
    if (lds > 64 * 1024) return -1;
    const dim3 grid(B * tiles), block(kCombineThreads);
    if (d <= 512)
        hipLaunchKernelGGL((combine_rows_kernel<ST, 1, USE>), grid, block, lds, stream, slot, rows, base, out, T, d, H,
                           k, accumulate, tiles);
    else if (d <= 1024)
        hipLaunchKernelGGL((combine_rows_kernel<ST, 2, USE>), grid, block, lds, stream, slot, rows, base, out, T, d, H,
                           k, accumulate, tiles);
    else
        hipLaunchKernelGGL((combine_rows_kernel<ST, 4, USE>), grid, block, lds, stream, slot, rows, base, out, T, d, H,
                           k, accumulate, tiles);
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

}  // namespace mosa
