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

template <typename ST>
int launch_t(const ST* QKV, const ST* dA, const float* lse, const float* D, int BH, int n, int dh, int causal,
             ST* dQKV, int pass, hipStream_t stream) {
    const int tasks = BH * ((n + 15) / 16);
    dim3 grid((tasks + 3) / 4), block(256);
    const float scale = 1.0f / sqrtf((float)dh);
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
