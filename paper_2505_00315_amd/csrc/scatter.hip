// Router-scaled output projection with a deterministic scatter-add
// (paper Section 2.2: X^o = diag(r) A W^O, Y_{I_i} = X^o_i, and Eq. 3:
// the layer output is the sum of all heads; dense heads, Eq. 2, add
// A W^O over every token).
//
// A workgroup owns an output tile Y[b, t0 : t0+TT, c0 : c0+CT] as fp32 in LDS
// (TT * CT * 4 bytes, up to 128 KB) and visits the heads in ascending order,
// then the dense heads.  Each wave owns a disjoint 16-column x token-range
// part of the tile, so no two waves ever add into the same element and each
// element receives its contributions in head order: the result is bitwise
// reproducible without atomics.  For head h, the slots whose tokens fall in
// the wave's token range are a contiguous slot range (I is ascending), read
// from the per-64-token segment table.  Per block of 16 slots:
//   D = (r * A)[16 x dh] * W^O_h[dh x 16 cols]   (MFMA, K = dh)
// and each D element is added to the LDS row I[slot] - t0.  The tile is
// written to HBM once.  Rows no head selects stay exactly 0.
#include "common.h"
#include "kernels.h"

namespace mosa {

namespace {

template <typename ST, int DH, int CGROUPS>
__global__ __launch_bounds__(512) void out_scatter_kernel(int B, int T, int d, int H, int k,
                                                          const int32_t* __restrict__ I, const float* __restrict__ r,
                                                          const int32_t* __restrict__ seg, int nseg,
                                                          const ST* __restrict__ A, const ST* __restrict__ Wo, int Hd,
                                                          const ST* __restrict__ Ad, const ST* __restrict__ Wod,
                                                          ST* __restrict__ Y, int accumulate, int TT, int ntt) {
    constexpr int CT = 16 * CGROUPS;
    constexpr int NTR = 8 / CGROUPS;  // token ranges per column group
    extern __shared__ float s_acc[];   // [TT][CT]

    const int nct = d / CT;
    const int logical = xcd_logical_id(blockIdx.x, gridDim.x);
    const int ct = logical / (B * ntt), rem = logical % (B * ntt);
    const int b = rem / ntt, tt = rem % ntt;
    const int t0 = tt * TT, c0 = ct * CT;
    (void)nct;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, c16 = lane & 15;
    const int cg = wave % CGROUPS, tr = wave / CGROUPS;
    const int TR = TT / NTR;
    const int tA = min(T, t0 + tr * TR), tB = min(T, t0 + (tr + 1) * TR);
    const int col = c0 + cg * 16 + c16;  // this lane's output column

    for (int e = tid; e < TT * CT; e += 512) s_acc[e] = 0.f;
    __syncthreads();

    if (tA < tB) {
        const int jA = tA / kSegWidth, jB = (tB + kSegWidth - 1) / kSegWidth;
        // MoSA heads, ascending
        for (int h = 0; h < H; ++h) {
            const size_t bh = (size_t)b * H + h;
            const int s_lo = seg[bh * nseg + jA], s_hi = seg[bh * nseg + jB];
            if (s_lo >= s_hi) continue;
            // W^O_h fragment for this lane's column: k-slots = d_head index
            Frag8<ST> wf[DH / 32];
#pragma unroll
            for (int st = 0; st < DH / 32; ++st) {
                float x[8];
#pragma unroll
                for (int j = 0; j < 8; ++j) x[j] = ld1<ST>(Wo + ((size_t)h * DH + st * 32 + 8 * g + j) * d + col);
                wf[st] = frag8_from<ST>(x);
            }
            for (int s0 = s_lo; s0 < s_hi; s0 += 16) {
                const int slot = s0 + c16;
                const bool ok = slot < s_hi;
                const int tok = ok ? I[bh * k + slot] : 0;
                const float rv = ok ? r[bh * k + slot] : 0.f;
                f32x4 acc = zero4();
#pragma unroll
                for (int st = 0; st < DH / 32; ++st) {
                    float x[8];
                    if (ok) {
                        frag8_to_f32<ST>(frag8_load<ST>(A + (bh * k + slot) * DH + st * 32 + 8 * g), x);
#pragma unroll
                        for (int j = 0; j < 8; ++j) x[j] *= rv;
                    } else {
#pragma unroll
                        for (int j = 0; j < 8; ++j) x[j] = 0.f;
                    }
                    mma8(acc, frag8_from<ST>(x), wf[st]);
                }
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int rr = 4 * g + i;
                    const int t = __shfl(tok, rr, 64);
                    if (s0 + rr < s_hi) s_acc[(t - t0) * CT + cg * 16 + c16] += acc[i];
                }
            }
        }
        // dense heads: every token, r = 1
        for (int h = 0; h < Hd; ++h) {
            const size_t bh = (size_t)b * Hd + h;
            Frag8<ST> wf[DH / 32];
#pragma unroll
            for (int st = 0; st < DH / 32; ++st) {
                float x[8];
#pragma unroll
                for (int j = 0; j < 8; ++j) x[j] = ld1<ST>(Wod + ((size_t)h * DH + st * 32 + 8 * g + j) * d + col);
                wf[st] = frag8_from<ST>(x);
            }
            for (int s0 = tA; s0 < tB; s0 += 16) {
                const int t = s0 + c16;
                const bool ok = t < tB;
                f32x4 acc = zero4();
#pragma unroll
                for (int st = 0; st < DH / 32; ++st) {
                    const Frag8<ST> a = ok ? frag8_load<ST>(Ad + (bh * T + t) * DH + st * 32 + 8 * g) : frag8_zero<ST>();
                    mma8(acc, a, wf[st]);
                }
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int tt2 = s0 + 4 * g + i;
                    if (tt2 < tB) s_acc[(tt2 - t0) * CT + cg * 16 + c16] += acc[i];
                }
            }
        }
    }
    __syncthreads();

    // write the tile once
    const int rows = min(TT, T - t0);
    for (int e = tid; e < rows * CT; e += 512) {
        const int rrow = e / CT, cc = e % CT;
        ST* yp = Y + ((size_t)b * T + t0 + rrow) * d + c0 + cc;
        float v = s_acc[e];
        if (accumulate) v += ld1<ST>(yp);
        st1<ST>(yp, v);
    }
}

template <typename ST, int DH, int CG>
int launch_cfg(int B, int T, int d, int H, int k, const int32_t* I, const float* r, const int32_t* seg,
               const ST* A, const ST* Wo, int Hd, const ST* Ad, const ST* Wod, ST* Y, int accumulate,
               hipStream_t stream) {
    constexpr int CT = 16 * CG, NTR = 8 / CG;
    constexpr int kMaxLds = 128 * 1024;
    const int quantum = NTR * kSegWidth;                       // token ranges align with segments
    const int tt_max = (kMaxLds / (CT * 4)) / quantum * quantum;
    int TT = ((T + quantum - 1) / quantum) * quantum;
    if (TT > tt_max) TT = tt_max;
    const int ntt = (T + TT - 1) / TT;
    const size_t lds = (size_t)TT * CT * sizeof(float);
    auto kern = out_scatter_kernel<ST, DH, CG>;
    if (hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess)
        return -1;
    dim3 grid(B * ntt * (d / CT)), block(512);
    hipLaunchKernelGGL(kern, grid, block, lds, stream, B, T, d, H, k, I, r, seg, seg_count(T), A, Wo, Hd, Ad, Wod, Y,
                       accumulate, TT, ntt);
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

template <typename ST>
int launch_out_scatter_t(int B, int T, int d, int dh, int H, int k, const int32_t* I, const float* r,
                         const int32_t* seg, const ST* A, const ST* Wo, int Hd, const ST* Ad, const ST* Wod, ST* Y,
                         int accumulate, hipStream_t stream) {
    // two 16-column groups per workgroup unless that leaves too few workgroups
    const bool wide = (size_t)B * (d / 32) * ((T + 1023) / 1024) >= 256;
    if (dh == 64)
        return wide ? launch_cfg<ST, 64, 2>(B, T, d, H, k, I, r, seg, A, Wo, Hd, Ad, Wod, Y, accumulate, stream)
                    : launch_cfg<ST, 64, 1>(B, T, d, H, k, I, r, seg, A, Wo, Hd, Ad, Wod, Y, accumulate, stream);
    return wide ? launch_cfg<ST, 32, 2>(B, T, d, H, k, I, r, seg, A, Wo, Hd, Ad, Wod, Y, accumulate, stream)
                : launch_cfg<ST, 32, 1>(B, T, d, H, k, I, r, seg, A, Wo, Hd, Ad, Wod, Y, accumulate, stream);
}

}  // namespace

int launch_out_scatter(int dtype, int B, int T, int d, int dh, int H, int k, const int32_t* I, const float* r,
                       const int32_t* seg, const void* A, const void* Wo, int Hd, const void* Ad, const void* Wo_d,
                       void* Y, int accumulate, hipStream_t stream) {
    if (dtype == kBF16)
        return launch_out_scatter_t<uint16_t>(B, T, d, dh, H, k, I, r, seg, (const uint16_t*)A, (const uint16_t*)Wo,
                                              Hd, (const uint16_t*)Ad, (const uint16_t*)Wo_d, (uint16_t*)Y, accumulate,
                                              stream);
    return launch_out_scatter_t<float>(B, T, d, dh, H, k, I, r, seg, (const float*)A, (const float*)Wo, Hd,
                                       (const float*)Ad, (const float*)Wo_d, (float*)Y, accumulate, stream);
}

}  // namespace mosa
