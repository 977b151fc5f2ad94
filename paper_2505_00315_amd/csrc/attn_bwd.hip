// Backward of the attention among the selected tokens (Eq. 1, index-aware
// causal mask = lower triangle in slot order), recomputing P from the saved
// log-sum-exp:
//   P_ij  = exp(S_ij / sqrt(dh) - lse_i)            (0 where masked)
//   dV_j  = sum_i P_ij dA_i
//   dP_ij = <dA_i, V_j>,  dS_ij = P_ij (dP_ij - D_i),  D_i = <dA_i, A_i>
//   dK_j  = sum_i dS_ij Q_i / sqrt(dh),  dQ_i = sum_j dS_ij K_j / sqrt(dh)
// Two passes so that no value is ever accumulated by atomics (results are
// bitwise reproducible):
//   kv pass: one wave per block of 16 keys, loop over the query blocks that
//            may attend to them; S and dP tiles come out with the key in the
//            lane (lane % 16) and queries in rows, i.e. already in the K = 16
//            operand layout for dV^T += dA^T P and dK^T += Q^T dS;
//   q pass:  one wave per block of 16 queries, loop over allowed key blocks;
//            S^T and dP^T tiles (query in the lane) feed dQ^T += K^T dS^T.
#include "common.h"
#include "kernels.h"
#include "tiles.h"

namespace mosa {

namespace {

template <typename ST, int DH>
__global__ __launch_bounds__(256) void attn_bwd_kv_kernel(const ST* __restrict__ QKV, const ST* __restrict__ dA,
                                                          const float* __restrict__ lse, const float* __restrict__ D,
                                                          int BH, int n, int causal, float scale,
                                                          ST* __restrict__ dQKV) {
    constexpr int RS = 3 * DH;  // row stride of the packed Q | K | V (and dQ | dK | dV) rows
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int g = lane >> 4, c16 = lane & 15;
    const int nb = (n + 15) / 16;
    const int task = blockIdx.x * 4 + wave;
    if (task >= BH * nb) return;
    const int bh = task / nb, j0 = (task % nb) * 16;
    const size_t base = (size_t)bh * n;
    const ST* Qp = QKV + base * RS;
    const ST* Kp = Qp + DH;
    const ST* Vp = Qp + 2 * DH;
    const ST* dAp = dA + base * DH;

    const int key = j0 + c16;  // this lane's key (as MFMA column)
    Frag8<ST> kf[DH / 32], vf[DH / 32];
#pragma unroll
    for (int s = 0; s < DH / 32; ++s) {
        kf[s] = key < n ? frag8_load<ST>(Kp + (size_t)key * RS + s * 32 + 8 * g) : frag8_zero<ST>();
        vf[s] = key < n ? frag8_load<ST>(Vp + (size_t)key * RS + s * 32 + 8 * g) : frag8_zero<ST>();
    }
    f32x4 dKt[DH / 16], dVt[DH / 16];
#pragma unroll
    for (int db = 0; db < DH / 16; ++db) dKt[db] = dVt[db] = zero4();

    for (int i0 = causal ? j0 : 0; i0 < n; i0 += 16) {
        const int qa = i0 + c16;  // query this lane feeds as MFMA A row
        f32x4 s = zero4(), dp = zero4();
#pragma unroll
        for (int st = 0; st < DH / 32; ++st) {
            const Frag8<ST> qa_f = qa < n ? frag8_load<ST>(Qp + (size_t)qa * RS + st * 32 + 8 * g) : frag8_zero<ST>();
            const Frag8<ST> da_f = qa < n ? frag8_load<ST>(dAp + (size_t)qa * DH + st * 32 + 8 * g) : frag8_zero<ST>();
            mma8(s, qa_f, kf[st]);
            mma8(dp, da_f, vf[st]);
        }
        // lane: key column c16, query rows 4g + i
        float p[4], ds[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int q = i0 + 4 * g + i;
            const bool ok = q < n && key < n && (!causal || key <= q);
            const float l = q < n ? lse[base + q] : 0.f;
            const float dd = q < n ? D[base + q] : 0.f;
            p[i] = ok ? expf(s[i] * scale - l) : 0.f;
            ds[i] = p[i] * (dp[i] - dd);
        }
        const Frag4<ST> pf = frag4_from<ST>(p);
        const Frag4<ST> dsf = frag4_from<ST>(ds);
#pragma unroll
        for (int db = 0; db < DH / 16; ++db) {
            float at[4], qt[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int q = i0 + 4 * g + i;
                at[i] = q < n ? ld1<ST>(dAp + (size_t)q * DH + db * 16 + c16) : 0.f;
                qt[i] = q < n ? ld1<ST>(Qp + (size_t)q * RS + db * 16 + c16) : 0.f;
            }
            mma4(dVt[db], frag4_from<ST>(at), pf);
            mma4(dKt[db], frag4_from<ST>(qt), dsf);
        }
        mfma_drain();  // the loop may exit right here
    }
    if (key < n) {
        // lane: key column c16, d_head rows db*16 + 4g + i
#pragma unroll
        for (int db = 0; db < DH / 16; ++db)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                st1<ST>(dQKV + (base + key) * RS + 2 * DH + db * 16 + 4 * g + i, dVt[db][i]);
                st1<ST>(dQKV + (base + key) * RS + DH + db * 16 + 4 * g + i, dKt[db][i] * scale);
            }
    }
}

template <typename ST, int DH>
__global__ __launch_bounds__(256) void attn_bwd_q_kernel(const ST* __restrict__ QKV, const ST* __restrict__ dA,
                                                         const float* __restrict__ lse, const float* __restrict__ D,
                                                         int BH, int n, int causal, float scale,
                                                         ST* __restrict__ dQKV) {
    constexpr int RS = 3 * DH;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int g = lane >> 4, c16 = lane & 15;
    const int nb = (n + 15) / 16;
    const int task = blockIdx.x * 4 + wave;
    if (task >= BH * nb) return;
    const int bh = task / nb, i0 = (task % nb) * 16;
    const size_t base = (size_t)bh * n;
    const ST* Qp = QKV + base * RS;
    const ST* Kp = Qp + DH;
    const ST* Vp = Qp + 2 * DH;
    const ST* dAp = dA + base * DH;

    const int q = i0 + c16;  // this lane's query (MFMA column)
    Frag8<ST> qf[DH / 32], daf[DH / 32];
#pragma unroll
    for (int s = 0; s < DH / 32; ++s) {
        qf[s] = q < n ? frag8_load<ST>(Qp + (size_t)q * RS + s * 32 + 8 * g) : frag8_zero<ST>();
        daf[s] = q < n ? frag8_load<ST>(dAp + (size_t)q * DH + s * 32 + 8 * g) : frag8_zero<ST>();
    }
    const float lq = q < n ? lse[base + q] : 0.f;
    const float dq = q < n ? D[base + q] : 0.f;
    f32x4 dQt[DH / 16];
#pragma unroll
    for (int db = 0; db < DH / 16; ++db) dQt[db] = zero4();

    const int kv_end = causal ? min(n, i0 + 16) : n;
    for (int j0 = 0; j0 < kv_end; j0 += 16) {
        const int kr = j0 + c16;
        f32x4 s = zero4(), dp = zero4();
#pragma unroll
        for (int st = 0; st < DH / 32; ++st) {
            const Frag8<ST> k_f = kr < n ? frag8_load<ST>(Kp + (size_t)kr * RS + st * 32 + 8 * g) : frag8_zero<ST>();
            const Frag8<ST> v_f = kr < n ? frag8_load<ST>(Vp + (size_t)kr * RS + st * 32 + 8 * g) : frag8_zero<ST>();
            mma8(s, k_f, qf[st]);
            mma8(dp, v_f, daf[st]);
        }
        // lane: query column c16, key rows 4g + i
        float ds[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int j = j0 + 4 * g + i;
            const bool ok = q < n && j < n && (!causal || j <= q);
            const float p = ok ? expf(s[i] * scale - lq) : 0.f;
            ds[i] = p * (dp[i] - dq);
        }
        const Frag4<ST> dsf = frag4_from<ST>(ds);
#pragma unroll
        for (int db = 0; db < DH / 16; ++db) {
            float kt[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int j = j0 + 4 * g + i;
                kt[i] = j < n ? ld1<ST>(Kp + (size_t)j * RS + db * 16 + c16) : 0.f;
            }
            mma4(dQt[db], frag4_from<ST>(kt), dsf);
        }
        mfma_drain();  // the loop may exit right here
    }
    if (q < n) {
#pragma unroll
        for (int db = 0; db < DH / 16; ++db)
#pragma unroll
            for (int i = 0; i < 4; ++i) st1<ST>(dQKV + (base + q) * RS + db * 16 + 4 * g + i, dQt[db][i] * scale);
    }
}

// Tiled passes for n > 32 (bf16 storage): a workgroup owns 64 keys (kv
// pass) or 64 queries (q pass) of one (b,h), 16 per wave, and walks the other
// side in tiles of 64 rows staged once in LDS for all four waves, row-major
// for the score MFMAs and transposed for the MFMAs that contract over rows
// (32 rows per MFMA, P and dS straight from registers).  The next tile's
// global loads overlap the current tile's MFMAs.
template <typename ST, int DH>
struct BwdTile {
    static constexpr int TB = 64, RS = 3 * DH;
    static constexpr int LDR = DH + 16 / (int)sizeof(ST);  // row-major rows
    static constexpr int LDT = TB + 4;                      // transposed rows
    static constexpr int VPR = DH / 8;
    static constexpr int PER = TB * VPR / 256;
    static_assert(PER >= 1 && TB * VPR % 256 == 0, "tile shape");
};

template <typename ST, int DH>
__global__ __launch_bounds__(256) void attn_bwd_kv_tiled_kernel(const ST* __restrict__ QKV, const ST* __restrict__ dA,
                                                                const float* __restrict__ lse,
                                                                const float* __restrict__ D, int BH, int n, int causal,
                                                                float scale, ST* __restrict__ dQKV) {
    using TL = BwdTile<ST, DH>;
    constexpr int TB = TL::TB, RS = TL::RS, LDR = TL::LDR, LDT = TL::LDT, VPR = TL::VPR, PER = TL::PER;
    __shared__ __attribute__((aligned(16))) ST Qs[TB * LDR];
    __shared__ __attribute__((aligned(16))) ST dAs[TB * LDR];
    __shared__ __attribute__((aligned(16))) ST QT[DH * LDT];
    __shared__ __attribute__((aligned(16))) ST dAT[DH * LDT];
    __shared__ float ls[TB], Dsh[TB];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, c16 = lane & 15;
    const int nkb = (n + TB - 1) / TB;
    const int bh = blockIdx.x / nkb, kb = blockIdx.x % nkb;  // causal: low kb has the most query tiles
    const int k0 = kb * TB, wk0 = k0 + 16 * wave;
    const size_t base = (size_t)bh * n;
    const ST* Qp = QKV + base * RS;
    const ST* Kp = Qp + DH;
    const ST* Vp = Qp + 2 * DH;
    const ST* dAp = dA + base * DH;

    const int key = wk0 + c16;  // this lane's key (MFMA column)
    const size_t krow = (size_t)min(key, n - 1);
    Frag8<ST> kf[DH / 32], vf[DH / 32];
#pragma unroll
    for (int st = 0; st < DH / 32; ++st) {
        kf[st] = frag8_load<ST>(Kp + krow * RS + st * 32 + 8 * g);
        vf[st] = frag8_load<ST>(Vp + krow * RS + st * 32 + 8 * g);
    }
    f32x4 dKt[DH / 16], dVt[DH / 16];
#pragma unroll
    for (int db = 0; db < DH / 16; ++db) dKt[db] = dVt[db] = zero4();

    const int it0 = causal ? kb : 0;
    Vec8<ST> qreg[PER], areg[PER];
    float lreg = 0.f, dreg = 0.f;
    // query rows past n are clamped to row n-1 (their scores are masked)
    auto load_tile = [&](int i0) {
#pragma unroll
        for (int p = 0; p < PER; ++p) {
            const int v = tid + 256 * p, r = v / VPR, dc = (v % VPR) * 8;
            const size_t row = (size_t)min(i0 + r, n - 1);
            qreg[p] = vec8_load<ST>(Qp + row * RS + dc);
            areg[p] = vec8_load<ST>(dAp + row * DH + dc);
        }
        const size_t rq = (size_t)min(i0 + lane, n - 1);
        lreg = lse[base + rq];
        dreg = D[base + rq];
    };
    auto store_tile = [&]() {
#pragma unroll
        for (int p = 0; p < PER; ++p) {
            const int v = tid + 256 * p, r = v / VPR, dc = (v % VPR) * 8;
            vec8_store<ST>(Qs + r * LDR + dc, qreg[p]);
            vec8_store<ST>(dAs + r * LDR + dc, areg[p]);
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                QT[(dc + j) * LDT + r] = vec8_elem<ST>(qreg[p], j);
                dAT[(dc + j) * LDT + r] = vec8_elem<ST>(areg[p], j);
            }
        }
        if (tid < TB) {
            ls[tid] = lreg;
            Dsh[tid] = dreg;
        }
    };

    load_tile(it0 * TB);
    for (int it = it0; it < nkb; ++it) {
        const int i0 = it * TB;
        __syncthreads();
        store_tile();
        __syncthreads();
        load_tile(min(it + 1, nkb - 1) * TB);
        // S and dP for 4 sub-blocks of 16 queries: lane = key c16, rows = queries 4g + i
        float p[4][4], ds[4][4];
#pragma unroll
        for (int sb = 0; sb < 4; ++sb) {
            f32x4 s = zero4(), dp = zero4();
#pragma unroll
            for (int st = 0; st < DH / 32; ++st) {
                mma8(s, frag8_load<ST>(Qs + (sb * 16 + c16) * LDR + st * 32 + 8 * g), kf[st]);
                mma8(dp, frag8_load<ST>(dAs + (sb * 16 + c16) * LDR + st * 32 + 8 * g), vf[st]);
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int ql = sb * 16 + 4 * g + i, q = i0 + ql;
                const bool ok = q < n && key < n && (!causal || key <= q);
                p[sb][i] = ok ? expf(s[i] * scale - ls[ql]) : 0.f;
                ds[sb][i] = p[sb][i] * (dp[i] - Dsh[ql]);
            }
        }
        // dV^T += dA^T P and dK^T += Q^T dS over 32 queries per MFMA
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            const float pv[8] = {p[2 * u][0], p[2 * u][1], p[2 * u][2], p[2 * u][3],
                                 p[2 * u + 1][0], p[2 * u + 1][1], p[2 * u + 1][2], p[2 * u + 1][3]};
            const float dv[8] = {ds[2 * u][0], ds[2 * u][1], ds[2 * u][2], ds[2 * u][3],
                                 ds[2 * u + 1][0], ds[2 * u + 1][1], ds[2 * u + 1][2], ds[2 * u + 1][3]};
            const Frag8<ST> pf = frag8_from<ST>(pv), dsf = frag8_from<ST>(dv);
#pragma unroll
            for (int db = 0; db < DH / 16; ++db) {
                const ST* ar = dAT + (db * 16 + c16) * LDT + 32 * u + 4 * g;
                const ST* qr = QT + (db * 16 + c16) * LDT + 32 * u + 4 * g;
                mma8(dVt[db], frag8_from_quads<ST>(quad_load<ST>(ar), quad_load<ST>(ar + 16)), pf);
                mma8(dKt[db], frag8_from_quads<ST>(quad_load<ST>(qr), quad_load<ST>(qr + 16)), dsf);
            }
        }
        mfma_drain();  // the loop may exit right here
    }

    // dK, dV rows (lane: key c16, d rows db*16 + 4g + i) through LDS to 16-byte stores
    __syncthreads();
    ST* Ks_out = Qs + wave * 16 * LDR;
    ST* Vs_out = dAs + wave * 16 * LDR;
#pragma unroll
    for (int db = 0; db < DH / 16; ++db)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int e = c16 * LDR + db * 16 + 4 * g + i;
            if constexpr (sizeof(ST) == 2) {
                Ks_out[e] = f32_to_bf16(dKt[db][i] * scale);
                Vs_out[e] = f32_to_bf16(dVt[db][i]);
            } else {
                Ks_out[e] = dKt[db][i] * scale;
                Vs_out[e] = dVt[db][i];
            }
        }
    __syncthreads();
#pragma unroll
    for (int e = lane; e < 16 * VPR; e += 64) {
        const int r = e / VPR, dc = (e % VPR) * 8;
        if (wk0 + r < n) {
            ST* out = dQKV + (base + wk0 + r) * RS;
            vec8_store<ST>(out + DH + dc, vec8_load<ST>(Ks_out + r * LDR + dc));
            vec8_store<ST>(out + 2 * DH + dc, vec8_load<ST>(Vs_out + r * LDR + dc));
        }
    }
}

template <typename ST, int DH>
__global__ __launch_bounds__(256) void attn_bwd_q_tiled_kernel(const ST* __restrict__ QKV, const ST* __restrict__ dA,
                                                               const float* __restrict__ lse,
                                                               const float* __restrict__ D, int BH, int n, int causal,
                                                               float scale, ST* __restrict__ dQKV) {
    using TL = BwdTile<ST, DH>;
    constexpr int TB = TL::TB, RS = TL::RS, LDR = TL::LDR, LDT = TL::LDT, VPR = TL::VPR, PER = TL::PER;
    __shared__ __attribute__((aligned(16))) ST Ks[TB * LDR];
    __shared__ __attribute__((aligned(16))) ST Vs[TB * LDR];
    __shared__ __attribute__((aligned(16))) ST KT[DH * LDT];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, c16 = lane & 15;
    const int nqb = (n + TB - 1) / TB;
    const int bh = blockIdx.x / nqb;
    const int qb = causal ? nqb - 1 - blockIdx.x % nqb : blockIdx.x % nqb;
    const int q0 = qb * TB, wq0 = q0 + 16 * wave;
    const size_t base = (size_t)bh * n;
    const ST* Qp = QKV + base * RS;
    const ST* Kp = Qp + DH;
    const ST* Vp = Qp + 2 * DH;
    const ST* dAp = dA + base * DH;

    const int q = wq0 + c16;  // this lane's query (MFMA column)
    const size_t qrow = (size_t)min(q, n - 1);
    Frag8<ST> qf[DH / 32], af[DH / 32];
#pragma unroll
    for (int st = 0; st < DH / 32; ++st) {
        qf[st] = frag8_load<ST>(Qp + qrow * RS + st * 32 + 8 * g);
        af[st] = frag8_load<ST>(dAp + qrow * DH + st * 32 + 8 * g);
    }
    const float lq = lse[base + qrow], dq = D[base + qrow];
    f32x4 dQt[DH / 16];
#pragma unroll
    for (int db = 0; db < DH / 16; ++db) dQt[db] = zero4();

    const int kv_end = causal ? min(n, q0 + TB) : n;
    const int ntiles = (kv_end + TB - 1) / TB;
    Vec8<ST> kreg[PER], vreg[PER];
    auto load_tile = [&](int j0) {
#pragma unroll
        for (int p = 0; p < PER; ++p) {
            const int v = tid + 256 * p, r = v / VPR, dc = (v % VPR) * 8;
            const size_t row = (size_t)min(j0 + r, n - 1);
            kreg[p] = vec8_load<ST>(Kp + row * RS + dc);
            vreg[p] = vec8_load<ST>(Vp + row * RS + dc);
        }
    };
    auto store_tile = [&]() {
#pragma unroll
        for (int p = 0; p < PER; ++p) {
            const int v = tid + 256 * p, r = v / VPR, dc = (v % VPR) * 8;
            vec8_store<ST>(Ks + r * LDR + dc, kreg[p]);
            vec8_store<ST>(Vs + r * LDR + dc, vreg[p]);
#pragma unroll
            for (int j = 0; j < 8; ++j) KT[(dc + j) * LDT + r] = vec8_elem<ST>(kreg[p], j);
        }
    };

    load_tile(0);
    for (int t = 0; t < ntiles; ++t) {
        const int j0 = t * TB;
        __syncthreads();
        store_tile();
        __syncthreads();
        load_tile(min(t + 1, ntiles - 1) * TB);
        // S^T and dP^T for 4 sub-blocks of 16 keys: lane = query c16, rows = keys 4g + i
        float ds[4][4];
#pragma unroll
        for (int sb = 0; sb < 4; ++sb) {
            f32x4 s = zero4(), dp = zero4();
#pragma unroll
            for (int st = 0; st < DH / 32; ++st) {
                mma8(s, frag8_load<ST>(Ks + (sb * 16 + c16) * LDR + st * 32 + 8 * g), qf[st]);
                mma8(dp, frag8_load<ST>(Vs + (sb * 16 + c16) * LDR + st * 32 + 8 * g), af[st]);
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int j = j0 + sb * 16 + 4 * g + i;
                const bool ok = j < n && q < n && (!causal || j <= q);
                const float pp = ok ? expf(s[i] * scale - lq) : 0.f;
                ds[sb][i] = pp * (dp[i] - dq);
            }
        }
        // dQ^T += K^T dS^T over 32 keys per MFMA
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            const float dv[8] = {ds[2 * u][0], ds[2 * u][1], ds[2 * u][2], ds[2 * u][3],
                                 ds[2 * u + 1][0], ds[2 * u + 1][1], ds[2 * u + 1][2], ds[2 * u + 1][3]};
            const Frag8<ST> dsf = frag8_from<ST>(dv);
#pragma unroll
            for (int db = 0; db < DH / 16; ++db) {
                const ST* kr = KT + (db * 16 + c16) * LDT + 32 * u + 4 * g;
                mma8(dQt[db], frag8_from_quads<ST>(quad_load<ST>(kr), quad_load<ST>(kr + 16)), dsf);
            }
        }
        mfma_drain();  // the loop may exit right here
    }

    __syncthreads();
    ST* Qs_out = Ks + wave * 16 * LDR;
#pragma unroll
    for (int db = 0; db < DH / 16; ++db)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int e = c16 * LDR + db * 16 + 4 * g + i;
            if constexpr (sizeof(ST) == 2) Qs_out[e] = f32_to_bf16(dQt[db][i] * scale);
            else Qs_out[e] = dQt[db][i] * scale;
        }
    __syncthreads();
#pragma unroll
    for (int e = lane; e < 16 * VPR; e += 64) {
        const int r = e / VPR, dc = (e % VPR) * 8;
        if (wq0 + r < n) vec8_store<ST>(dQKV + (base + wq0 + r) * RS + dc, vec8_load<ST>(Qs_out + r * LDR + dc));
    }
}

template <typename ST>
int launch_t(const ST* QKV, const ST* dA, const float* lse, const float* D, int BH, int n, int dh, int causal,
             ST* dQKV, int pass, hipStream_t stream) {
    const float scale = 1.0f / sqrtf((float)dh);
    if constexpr (sizeof(ST) == 2) {
      if (n > 32) {
        const dim3 grid(BH * ((n + 63) / 64)), block(256);
#define MOSA_ATTN_BWD_T(KERN, DHV) \
    hipLaunchKernelGGL((KERN<ST, DHV>), grid, block, 0, stream, QKV, dA, lse, D, BH, n, causal, scale, dQKV)
        if (pass == 0) {
            if (dh == 64) MOSA_ATTN_BWD_T(attn_bwd_kv_tiled_kernel, 64);
            else MOSA_ATTN_BWD_T(attn_bwd_kv_tiled_kernel, 32);
        } else {
            if (dh == 64) MOSA_ATTN_BWD_T(attn_bwd_q_tiled_kernel, 64);
            else MOSA_ATTN_BWD_T(attn_bwd_q_tiled_kernel, 32);
        }
#undef MOSA_ATTN_BWD_T
        return hipGetLastError() == hipSuccess ? 0 : -1;
      }
    }
    const int tasks = BH * ((n + 15) / 16);
    dim3 grid((tasks + 3) / 4), block(256);
#define MOSA_ATTN_BWD(KERN, DHV) \
    hipLaunchKernelGGL((KERN<ST, DHV>), grid, block, 0, stream, QKV, dA, lse, D, BH, n, causal, scale, dQKV)
    if (pass == 0) {
        if (dh == 64) MOSA_ATTN_BWD(attn_bwd_kv_kernel, 64);
        else MOSA_ATTN_BWD(attn_bwd_kv_kernel, 32);
    } else {
        if (dh == 64) MOSA_ATTN_BWD(attn_bwd_q_kernel, 64);
        else MOSA_ATTN_BWD(attn_bwd_q_kernel, 32);
    }
#undef MOSA_ATTN_BWD
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

}  // namespace

int launch_attn_bwd(int dtype, const void* QKV, const void* dA, const float* lse, const float* D, int BH, int n,
                    int dh, int causal, void* dQKV, int pass, hipStream_t stream) {
    if (dtype == kBF16)
        return launch_t<uint16_t>((const uint16_t*)QKV, (const uint16_t*)dA, lse, D, BH, n, dh, causal,
                                  (uint16_t*)dQKV, pass, stream);
    return launch_t<float>((const float*)QKV, (const float*)dA, lse, D, BH, n, dh, causal, (float*)dQKV, pass,
                           stream);
}

}  // namespace mosa
