// Attention of one block of 16 queries against keys held in LDS (paper
// Eq. 1 with the index-aware causal mask, in slot order), shared by the
// single-workgroup attention kernel and the fused QKV + attention kernel.
//
// K is a row-major tile with the 16-byte units of each row XOR-permuted
// (kswz, read with ds_read_b128), V a row-major tile with units permuted by
// vt_swz (read transposed with ds_read_b64_tr_b16).  The wave keeps the
// scores of all keys of its block in registers (S^T = K Q^T, lane = query),
// takes the row maximum and sum once, and accumulates O^T += V^T P^T 32 keys
// per MFMA with V^T read in the key order of the P^T registers.  It writes
// A = r O / l (storage type) and lse = m + log l.
#pragma once

#include "gemm2.h"

namespace mosa {

constexpr int kAttnLdsMaxN = 128;

template <int U>
__device__ __forceinline__ int vt_swz(int k) {  // V tile unit permutation (an involution per row)
    if constexpr (U == 8) return 2 * ((k >> 1) & 3);
    else return 2 * ((k >> 2) & 1);
}

// Query block qb (local rows 16 qb ..) of a group of n rows whose keys are
// LDS rows kbase .. kbase + n - 1 (kbase a multiple of 16); qf: the lane's query row (16 qb + lane % 16,
// clamped) as B operand fragments; rw, A, lse: the group's r (or nullptr),
// output rows and log-sum-exp.
template <int DH>
__device__ __forceinline__ void attn_lds_block(const unsigned char* Ks, const unsigned char* Vs, int kbase,
                                               const Frag8<uint16_t> (&qf)[DH / 32], int n, int causal, float scale,
                                               int qb, const float* rw, uint16_t* A, float* lse) {
    using ST = uint16_t;
    constexpr int NMAX = kAttnLdsMaxN, U = DH / 8;
    const int lane = threadIdx.x & 63, g = lane >> 4, c16 = lane & 15;
    const int nqb = (n + 15) / 16, nkb = causal ? qb + 1 : nqb, q = 16 * qb + c16;

    // S^T for every key block: lane = query c16, rows = keys 16 sb + 4 g + i;
    // keys past n and (causal) past the query are masked (to -inf, also the
    // blocks past the diagonal), and the maximum is taken over the unscaled
    // scores (scale > 0).  Both swizzles depend on the low 4 bits of the row
    // only, so each lane's LDS addresses advance by whole blocks.
    const int lim = causal ? min(q, n - 1) : n - 1;  // last allowed key
    const unsigned char* kp[DH / 32];
#pragma unroll
    for (int st = 0; st < DH / 32; ++st) {
        const int row = kbase + c16, u = 4 * st + g;
        kp[st] = Ks + (row * U + (u ^ kswz(row, U))) * 16;
    }
    f32x4 s[NMAX / 16];
    float m = -__builtin_inff();
#pragma unroll
    for (int sb = 0; sb < NMAX / 16; ++sb) {
        s[sb] = f32x4{-__builtin_inff(), -__builtin_inff(), -__builtin_inff(), -__builtin_inff()};
        if (sb < nkb) {
            f32x4 acc = zero4();
#pragma unroll
            for (int st = 0; st < DH / 32; ++st) {
                Frag8<ST> kf;
                kf.v = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(kp[st] + sb * 16 * U * 16));
                mma8(acc, kf, qf[st]);
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) s[sb][i] = 16 * sb + 4 * g + i <= lim ? acc[i] : -__builtin_inff();
            m = fmaxf(m, fmaxf(fmaxf(s[sb][0], s[sb][1]), fmaxf(s[sb][2], s[sb][3])));
        }
    }
    m = fmaxf(m, __shfl_xor(m, 16, 64));
    m = fmaxf(m, __shfl_xor(m, 32, 64));
    // p = exp(scale (s - m)) = 2^(s c - m c), c = scale log2(e); key 0 is
    // allowed for every query, so m is finite
    const float c = scale * 1.44269504088896341f, mc = m * c;
    float l = 0.f;
#pragma unroll
    for (int sb = 0; sb < NMAX / 16; ++sb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            s[sb][i] = __builtin_amdgcn_exp2f(fmaf(s[sb][i], c, -mc));
            l += s[sb][i];
        }
    l += __shfl_xor(l, 16, 64);
    l += __shfl_xor(l, 32, 64);

    // O^T += V^T P^T, 32 keys per MFMA: slots 0..3 = keys 32 u + 4 g + i,
    // slots 4..7 = keys 32 u + 16 + 4 g + i (the P^T registers as they are).
    // Lane reads for d columns 16 db + 4 (c16 % 4) .. + 3, keys k0 and k0 + 16
    const unsigned char* vp[DH / 16];
    {
        const int k0 = kbase + 4 * g + (c16 >> 2);
#pragma unroll
        for (int db = 0; db < DH / 16; ++db) {
            const int mcol = 16 * db + 4 * (c16 & 3), un = mcol >> 3, half = (mcol >> 2) & 1;
            vp[db] = Vs + (k0 * U + (un ^ vt_swz<U>(k0))) * 16 + 8 * half;
        }
    }
    f32x4 o[DH / 16];
#pragma unroll
    for (int db = 0; db < DH / 16; ++db) o[db] = zero4();
    static_for<0, NMAX / 32>([&](auto uuc) {
        constexpr int uu = decltype(uuc)::value;
        if (2 * uu < nkb) {
            const float pv[8] = {s[2 * uu][0], s[2 * uu][1], s[2 * uu][2], s[2 * uu][3],
                                 s[2 * uu + 1][0], s[2 * uu + 1][1], s[2 * uu + 1][2], s[2 * uu + 1][3]};
            const Frag8<ST> pf = frag8_from<ST>(pv);
            u32x4 vt[DH / 16];
#pragma unroll
            for (int db = 0; db < DH / 16; ++db) {
                const u32x2 lo = lds_read_tr16_at<32 * U * 16 * uu>(vp[db]);
                const u32x2 hi = lds_read_tr16_at<32 * U * 16 * uu + 16 * U * 16>(vp[db]);
                vt[db] = u32x4{lo.x, lo.y, hi.x, hi.y};
            }
            lds_wait();
#pragma unroll
            for (int db = 0; db < DH / 16; ++db) {
                lds_ready(vt[db]);
                Frag8<ST> vf;
                vf.v = __builtin_bit_cast(bf16x8, vt[db]);
                mma8(o[db], vf, pf);
            }
        }
    });
    mfma_drain();
    // lane: query c16, d = 16 db + 4 g + i
    if (q < n) {
        const float inv = (rw ? rw[q] : 1.f) / l;
        ST* Ap = A + (size_t)q * DH;
#pragma unroll
        for (int db = 0; db < DH / 16; ++db)
            *reinterpret_cast<uint2*>(Ap + 16 * db + 4 * g) =
                make_uint2(pack_bf16x2(o[db][0] * inv, o[db][1] * inv), pack_bf16x2(o[db][2] * inv, o[db][3] * inv));
        if (g == 0) lse[q] = m * scale + logf(l);
    }
}

}  // namespace mosa
