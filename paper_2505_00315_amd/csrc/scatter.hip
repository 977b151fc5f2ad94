// Deterministic head-ordered scatter-add of per-head row contributions into
// a [B, T, d] tensor.  Two uses:
//   forward (paper Section 2.2 and Eq. 3):  Y[b, I_i] += (r_i A_i) W^O_h
//       for every MoSA head in ascending order, then every dense head
//       (Eq. 2, all tokens, r = 1);
//   backward (chain rule through Q, K, V = X^s W^{Q,K,V} and s = X^s W^r):
//       dX[b, I_i] += dQ_i W^Q_h^T + dK_i W^K_h^T + dV_i W^V_h^T + dz_i W^r_h.
//
// A workgroup owns an output tile [b, t0 : t0+TT, c0 : c0+CT] as fp32 in LDS
// (TT * CT * 4 bytes, up to 128 KB) and visits the heads in a fixed order.
// Each wave owns a disjoint 16-column x token-range part of the tile, so no
// two waves ever add into the same element and each element receives its
// contributions in head order: bitwise reproducible without atomics.  The
// slots of head h whose tokens fall in the wave's token range form a
// contiguous range (I is ascending), read from the per-64-token segment
// table.  Per block of 16 slots one MFMA tile
//   D[16 slots x 16 cols] = U[16 x K] W_h[K x 16 cols]
// is added into LDS row I[slot] - t0.  The tile is written to HBM once; rows
// no head touches stay exactly 0 (or keep the old value when accumulating).
#include "common.h"
#include "kernels.h"

namespace mosa {

namespace {

enum { kModeForward = 0, kModeBackward = 1 };

template <typename ST, int DH, int CGROUPS, int MODE>
__global__ __launch_bounds__(512) void scatter_kernel(int B, int T, int d, int H, int k,
                                                      const int32_t* __restrict__ I, const float* __restrict__ r,
                                                      const int32_t* __restrict__ seg, int nseg,
                                                      const ST* __restrict__ U0, const ST* __restrict__ U1,
                                                      const ST* __restrict__ U2, const float* __restrict__ dz,
                                                      const ST* __restrict__ W0, const ST* __restrict__ W1,
                                                      const ST* __restrict__ W2, const ST* __restrict__ Wr, int Hd,
                                                      const ST* __restrict__ Ud0, const ST* __restrict__ Ud1,
                                                      const ST* __restrict__ Ud2, const ST* __restrict__ Wd0,
                                                      const ST* __restrict__ Wd1, const ST* __restrict__ Wd2,
                                                      ST* __restrict__ Y, int accumulate, int TT, int ntt) {
    constexpr int CT = 16 * CGROUPS;
    constexpr int NTR = 8 / CGROUPS;                      // token ranges per column group
    constexpr int NMAT = MODE == kModeForward ? 1 : 3;    // K = NMAT * DH
    constexpr int NST = NMAT * DH / 32;                   // K = 32 steps
    extern __shared__ float s_acc[];                      // [TT][CT]

    const int logical = xcd_logical_id(blockIdx.x, gridDim.x);
    const int ct = logical / (B * ntt), rem = logical % (B * ntt);
    const int b = rem / ntt, tt = rem % ntt;
    const int t0 = tt * TT, c0 = ct * CT;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, c16 = lane & 15;
    const int cg = wave % CGROUPS, tr = wave / CGROUPS;
    const int TR = TT / NTR;
    const int tA = min(T, t0 + tr * TR), tB = min(T, t0 + (tr + 1) * TR);
    const int col = c0 + cg * 16 + c16;  // this lane's output column
    float* acc_col = s_acc + cg * 16 + c16;

    for (int e = tid; e < TT * CT; e += 512) s_acc[e] = 0.f;
    __syncthreads();

    // B operand of head h for this lane's column: k-slots 8g..8g+7 of K step st.
    auto load_w = [&](const ST* w0, const ST* w1, const ST* w2, int h, Frag8<ST> (&wf)[NST]) {
#pragma unroll
        for (int st = 0; st < NST; ++st) {
            if (MODE == kModeForward) {  // W^O_h[e][col], e = st*32 + 8g + j (stride d)
                float x[8];
#pragma unroll
                for (int j = 0; j < 8; ++j) x[j] = ld1<ST>(w0 + ((size_t)h * DH + st * 32 + 8 * g + j) * d + col);
                wf[st] = frag8_from<ST>(x);
            } else {  // W^m_h[col][e]: contiguous along e
                const int m = (st * 32) / DH, e0 = (st * 32) % DH + 8 * g;
                const ST* wm = m == 0 ? w0 : (m == 1 ? w1 : w2);
                wf[st] = frag8_load<ST>(wm + ((size_t)h * d + col) * DH + e0);
            }
        }
    };
    // A operand row `ridx` (one slot): r * A (forward) or dQ | dK | dV (backward)
    auto load_u = [&](const ST* u0, const ST* u1, const ST* u2, size_t ridx, float rv, bool ok, int st) {
        if (!ok) return frag8_zero<ST>();
        if (MODE == kModeForward) {
            float x[8];
            frag8_to_f32<ST>(frag8_load<ST>(u0 + ridx * DH + st * 32 + 8 * g), x);
#pragma unroll
            for (int j = 0; j < 8; ++j) x[j] *= rv;
            return frag8_from<ST>(x);
        } else {
            const int m = (st * 32) / DH, e0 = (st * 32) % DH + 8 * g;
            const ST* um = m == 0 ? u0 : (m == 1 ? u1 : u2);
            return frag8_load<ST>(um + ridx * DH + e0);
        }
    };

    if (tA < tB) {
        const int jA = tA / kSegWidth, jB = (tB + kSegWidth - 1) / kSegWidth;
        for (int h = 0; h < H; ++h) {  // MoSA heads, ascending
            const size_t bh = (size_t)b * H + h;
            const int s_lo = seg[bh * nseg + jA], s_hi = seg[bh * nseg + jB];
            if (s_lo >= s_hi) continue;
            Frag8<ST> wf[NST];
            load_w(W0, W1, W2, h, wf);
            const float wr = (MODE == kModeBackward) ? ld1<ST>(Wr + (size_t)h * d + col) : 0.f;
            for (int s0 = s_lo; s0 < s_hi; s0 += 16) {
                const int slot = s0 + c16;
                const bool ok = slot < s_hi;
                const size_t ridx = bh * k + (ok ? slot : 0);
                const int tok = ok ? I[ridx] : 0;
                const float rv = (MODE == kModeForward && ok) ? r[ridx] : 0.f;
                const float dzv = (MODE == kModeBackward && ok) ? dz[ridx] : 0.f;
                f32x4 acc = zero4();
#pragma unroll
                for (int st = 0; st < NST; ++st) mma8(acc, load_u(U0, U1, U2, ridx, rv, ok, st), wf[st]);
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int rr = 4 * g + i;
                    const int t = __shfl(tok, rr, 64);
                    float v = acc[i];
                    if (MODE == kModeBackward) v += __shfl(dzv, rr, 64) * wr;
                    if (s0 + rr < s_hi) acc_col[(t - t0) * CT] += v;
                }
            }
        }
        for (int h = 0; h < Hd; ++h) {  // dense heads: every token, r = 1
            const size_t bh = (size_t)b * Hd + h;
            Frag8<ST> wf[NST];
            load_w(Wd0, Wd1, Wd2, h, wf);
            for (int s0 = tA; s0 < tB; s0 += 16) {
                const int t = s0 + c16;
                const bool ok = t < tB;
                const size_t ridx = bh * T + (ok ? t : 0);
                f32x4 acc = zero4();
#pragma unroll
                for (int st = 0; st < NST; ++st) mma8(acc, load_u(Ud0, Ud1, Ud2, ridx, 1.f, ok, st), wf[st]);
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int t2 = s0 + 4 * g + i;
                    if (t2 < tB) acc_col[(t2 - t0) * CT] += acc[i];
                }
            }
        }
    }
    __syncthreads();

    const int rows = min(TT, T - t0);
    for (int e = tid; e < rows * CT; e += 512) {
        const int rrow = e / CT, cc = e % CT;
        ST* yp = Y + ((size_t)b * T + t0 + rrow) * d + c0 + cc;
        float v = s_acc[e];
        if (accumulate) v += ld1<ST>(yp);
        st1<ST>(yp, v);
    }
}

struct ScatterArgs {
    int B, T, d, dh, H, k, Hd;
    const int32_t* I;
    const float* r;
    const int32_t* seg;
    const void *U0, *U1, *U2;
    const float* dz;
    const void *W0, *W1, *W2, *Wr;
    const void *Ud0, *Ud1, *Ud2, *Wd0, *Wd1, *Wd2;
    void* Y;
    int accumulate;
};

template <typename ST, int DH, int CG, int MODE>
int launch_cfg(const ScatterArgs& a, hipStream_t stream) {
    constexpr int CT = 16 * CG, NTR = 8 / CG;
    constexpr int kMaxLds = 128 * 1024;
    const int quantum = NTR * kSegWidth;  // token ranges align with segment boundaries
    const int tt_max = (kMaxLds / (CT * 4)) / quantum * quantum;
    int TT = ((a.T + quantum - 1) / quantum) * quantum;
    if (TT > tt_max) TT = tt_max;
    const int ntt = (a.T + TT - 1) / TT;
    const size_t lds = (size_t)TT * CT * sizeof(float);
    auto kern = scatter_kernel<ST, DH, CG, MODE>;
    static bool attr_set = false;  // the attribute is per kernel; setting it once suffices
    if (!attr_set) {
        if (hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, kMaxLds) != hipSuccess)
            return -1;
        attr_set = true;
    }
    dim3 grid(a.B * ntt * (a.d / CT)), block(512);
    hipLaunchKernelGGL(kern, grid, block, lds, stream, a.B, a.T, a.d, a.H, a.k, a.I, a.r, a.seg, seg_count(a.T),
                       (const ST*)a.U0, (const ST*)a.U1, (const ST*)a.U2, a.dz, (const ST*)a.W0, (const ST*)a.W1,
                       (const ST*)a.W2, (const ST*)a.Wr, a.Hd, (const ST*)a.Ud0, (const ST*)a.Ud1, (const ST*)a.Ud2,
                       (const ST*)a.Wd0, (const ST*)a.Wd1, (const ST*)a.Wd2, (ST*)a.Y, a.accumulate, TT, ntt);
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

template <typename ST, int MODE>
int launch_mode(const ScatterArgs& a, hipStream_t stream) {
    // two 16-column groups per workgroup unless that leaves fewer than 256 workgroups
    const bool wide = (size_t)a.B * (a.d / 32) * ((a.T + 1023) / 1024) >= 256;
    if (a.dh == 64)
        return wide ? launch_cfg<ST, 64, 2, MODE>(a, stream) : launch_cfg<ST, 64, 1, MODE>(a, stream);
    return wide ? launch_cfg<ST, 32, 2, MODE>(a, stream) : launch_cfg<ST, 32, 1, MODE>(a, stream);
}

}  // namespace

int launch_out_scatter(int dtype, int B, int T, int d, int dh, int H, int k, const int32_t* I, const float* r,
                       const int32_t* seg, const void* A, const void* Wo, int Hd, const void* Ad, const void* Wo_d,
                       void* Y, int accumulate, hipStream_t stream) {
    ScatterArgs a{B, T, d, dh, H, k, Hd, I, r, seg, A, nullptr, nullptr, nullptr, Wo, nullptr, nullptr, nullptr,
                  Ad, nullptr, nullptr, Wo_d, nullptr, nullptr, Y, accumulate};
    return dtype == kBF16 ? launch_mode<uint16_t, kModeForward>(a, stream) : launch_mode<float, kModeForward>(a, stream);
}

int launch_dx_scatter(int dtype, int B, int T, int d, int dh, int H, int k, const int32_t* I, const int32_t* seg,
                      const void* dQ, const void* dK, const void* dV, const float* dz, const void* Wq, const void* Wk,
                      const void* Wv, const void* Wr, int Hd, const void* dQd, const void* dKd, const void* dVd,
                      const void* Wq_d, const void* Wk_d, const void* Wv_d, void* dX, int accumulate,
                      hipStream_t stream) {
    ScatterArgs a{B, T, d, dh, H, k, Hd, I, nullptr, seg, dQ, dK, dV, dz, Wq, Wk, Wv, Wr,
                  dQd, dKd, dVd, Wq_d, Wk_d, Wv_d, dX, accumulate};
    return dtype == kBF16 ? launch_mode<uint16_t, kModeBackward>(a, stream)
                          : launch_mode<float, kModeBackward>(a, stream);
}

}  // namespace mosa
