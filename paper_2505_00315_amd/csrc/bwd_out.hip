// Backward of the output side of a head (chain rule through Section 2.2's
// X^o = diag(r) A W^O and the scatter Y_{I_i} = X^o_i, with I held fixed):
//   dX^o_i   = dY[b, I_i]                      (gather)
//   dA~_i    = dX^o_i W^O^T                    (GEMM, K = d)
//   dr_i     = <dA~_i, A_i>                    (router gradient through r)
//   dA_i     = r_i dA~_i                       (into the attention backward)
//   D_i      = <dA_i, A_i> = r_i dr_i          (softmax row term of Eq. 1's backward)
//   dz_i     = dr_i r_i (1 - r_i)              (sigma'(s) = r (1 - r))
// The forward saved the scaled rows S_i = r_i A_i, so D_i = <dA~_i, S_i> and
// dz_i = D_i (1 - r_i): no division by r, and r = 0 gives dz = D = 0.
// Dense heads are the case I = identity, r = 1 (no dz).
//
// One GEMM per head on the tiled MFMA engine: M = B*n gathered dY rows,
// N = dh, K = d; W^O_h rows are contiguous along d (the K index), so both
// operands are staged without transposes.  The epilogue holds whole rows of
// dA~ and finishes dr, dA, D, dz there; dz is also written as a 16-wide row
// (dz, 0, ..., 0) so the weight-gradient GEMM can treat W^r as a 16-column
// block of its B operand.
#include "gemm.h"
#include "gemm2.h"
#include "kernels.h"

namespace mosa {

namespace {

template <typename ST, int DH>
struct BwdOutPolicy {
    static constexpr int MT = 64, NT = DH, KC = sizeof(ST) == 2 ? 64 : 32, WM = 4, WN = 1;
    static constexpr size_t EPI_LDS = 0;
    static constexpr bool A_KCONTIG = true, B_KCONTIG = true, A_SCALED = false;
    struct Args {
        const ST* dY;
        const int32_t* I;  // nullptr: dense head
        const float* r;    // nullptr: dense head
        const ST* Wo;      // [H, DH, d]
        const ST* A;       // [B, H, n, DH], rows scaled by r
        ST* dA;
        float* D;
        float* dz;         // nullptr: dense head
        ST* dz16;          // [B, H, n, 16]
        int T, d, H, n, M, mtiles;
    };
    struct ARef {
        const ST* p;
    };
    struct BRef {
        const ST* p;
    };
    struct RowInfo {
        int unused;
    };
    __device__ static const ST* a_fallback(const Args& a) { return a.dY; }
    __device__ static const ST* b_fallback(const Args& a) { return a.Wo; }
    __device__ static void tile(const Args& a, int logical, int& h, int& m0, int& n0) {
        if (a.I) {  // a head's row tiles side by side: they share its W^O rows
            h = logical / a.mtiles;
            m0 = (logical % a.mtiles) * MT;
        } else {  // dense heads: the heads of a row tile side by side (its dY rows)
            h = logical % a.H;
            m0 = (logical / a.H) * MT;
        }
        n0 = 0;
    }
    __device__ static int k_size(const Args& a, int) { return a.d; }
    __device__ static ARef a_row(const Args& a, int h, int m, float&) {
        if (m < 0 || m >= a.M) return {nullptr};
        const int b = m / a.n, i = m % a.n;
        const int t = a.I ? a.I[((size_t)b * a.H + h) * a.n + i] : i;
        return {a.dY + ((size_t)b * a.T + t) * a.d};
    }
    __device__ static const ST* a_elem(const Args&, int, const ARef& r, int k) { return r.p ? r.p + k : nullptr; }
    __device__ static BRef b_row(const Args& a, int h, int n) {
        return {n >= 0 && n < DH ? a.Wo + ((size_t)h * DH + n) * a.d : nullptr};
    }
    __device__ static const ST* b_elem(const Args&, int, const BRef& r, int k) { return r.p ? r.p + k : nullptr; }
    __device__ static RowInfo row_info(const Args&, int, int) { return {0}; }
    __device__ static const ST* a_kaddr(const Args& a, int, const RowInfo&, int) { return a_fallback(a); }
    __device__ static bool a_kok(const Args&, int, const RowInfo&, int) { return false; }
    __device__ static float a_kscale(const Args&, int, const RowInfo&) { return 1.f; }
    __device__ static const ST* b_kaddr(const Args& a, int, const RowInfo&, int) { return b_fallback(a); }
    __device__ static bool b_kok(const Args&, int, const RowInfo&, int) { return false; }

    // 4 threads per row, DH / 4 columns each.
    __device__ static void epilogue(const Args& a, int h, int m0, int, const float* Cs, int ldc, int tid, unsigned char*) {
        constexpr int CW = DH / 4;
        const int ml = tid >> 2, cq = (tid & 3) * CW;
        const int m = m0 + ml;
        const bool ok = m < a.M;
        size_t ri = 0;
        float c[CW], part = 0.f;
        if (ok) {
            ri = ((size_t)(m / a.n) * a.H + h) * a.n + (m % a.n);
#pragma unroll
            for (int q = 0; q < CW / 8; ++q) {
                float x[8];
                vec8_to_f32<ST>(vec8_load<ST>(a.A + ri * DH + cq + 8 * q), x);
                float cv[8];
                cs_load8(Cs, ldc, ml, cq + 8 * q, cv);
#pragma unroll
                for (int j = 0; j < 8; ++j) {
                    c[8 * q + j] = cv[j];
                    part += c[8 * q + j] * x[j];
                }
            }
        }
        part += __shfl_xor(part, 1, 64);
        part += __shfl_xor(part, 2, 64);
        if (!ok) return;
        const float rr = a.r ? a.r[ri] : 1.f;
#pragma unroll
        for (int q = 0; q < CW / 8; ++q) {
            float x[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) x[j] = rr * c[8 * q + j];
            vec8_store<ST>(a.dA + ri * DH + cq + 8 * q, vec8_from_f32<ST>(x));
        }
        if ((tid & 3) == 0) {
            a.D[ri] = part;
            if (a.dz) {
                const float dzv = part * (1.f - rr);
                a.dz[ri] = dzv;
                float x[8] = {dzv, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f}, zz[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
                vec8_store<ST>(a.dz16 + ri * 16, vec8_from_f32<ST>(x));
                vec8_store<ST>(a.dz16 + ri * 16 + 8, vec8_from_f32<ST>(zz));
            }
        }
    }
};

// bf16 storage: the multi-stage engine (gemm2.h); both operands k-contiguous,
// the gathered dY rows clamped to the last row past M.
template <int DH>
struct BwdOutPolicy2 {
    using ST = uint16_t;
    using P1 = BwdOutPolicy<ST, DH>;
    static constexpr int MT = 64, NT = DH, KC = 64, WM = 4, WN = 1, STAGES = 4;
    static constexpr size_t EPI_LDS = 0;
    static constexpr bool A_KCONTIG = true, B_KCONTIG = true;
    using Args = typename P1::Args;
    using ARef = typename P1::ARef;
    using BRef = typename P1::BRef;
    __device__ static void tile(const Args& a, int logical, int& h, int& m0, int& n0) { P1::tile(a, logical, h, m0, n0); }
    __device__ static int k_size(const Args& a, int) { return a.d; }
    __device__ static ARef a_row(const Args& a, int h, int m) {
        float unused;
        return P1::a_row(a, h, min(m, a.M - 1), unused);
    }
    __device__ static const ST* a_elem(const Args&, int, const ARef& r, int k) { return r.p + k; }
    __device__ static BRef b_row(const Args& a, int h, int n) { return {a.Wo + ((size_t)h * DH + n) * a.d}; }
    __device__ static const ST* b_elem(const Args&, int, const BRef& r, int k) { return r.p + k; }
    __device__ static void epilogue(const Args& a, int h, int m0, int n0, const float* Cs, int ldc, int tid,
                                    unsigned char* extra) {
        P1::epilogue(a, h, m0, n0, Cs, ldc, tid, extra);
    }
};

template <typename ST, int DH>
int run(const ST* dY, const int32_t* I, const float* r, const ST* Wo, const ST* A, int B, int T, int d, int H, int n,
        ST* dA, float* D, float* dz, ST* dz16, hipStream_t stream) {
    using P = BwdOutPolicy<ST, DH>;
    const int M = B * n;
    typename P::Args a{dY, I, r, Wo, A, dA, D, dz, dz16, T, d, H, n, M, (M + P::MT - 1) / P::MT};
    if constexpr (sizeof(ST) == 2) {
        if (d % BwdOutPolicy2<DH>::KC == 0) return launch_gemm2<BwdOutPolicy2<DH>>(a, H * a.mtiles, stream);
    }
    return launch_gemm<ST, P>(a, H * a.mtiles, stream);
}

}  // namespace

int launch_dattn_out(int dtype, const void* dY, const int32_t* I, const float* r, const void* Wo, const void* A,
                     int B, int T, int d, int H, int dh, int n, void* dA, float* D, float* dz, void* dz16,
                     hipStream_t stream) {
    if (H == 0) return 0;
    if (dtype == kBF16) {
        auto f = dh == 64 ? run<uint16_t, 64> : run<uint16_t, 32>;
        return f((const uint16_t*)dY, I, r, (const uint16_t*)Wo, (const uint16_t*)A, B, T, d, H, n, (uint16_t*)dA, D,
                 dz, (uint16_t*)dz16, stream);
    }
    auto f = dh == 64 ? run<float, 64> : run<float, 32>;
    return f((const float*)dY, I, r, (const float*)Wo, (const float*)A, B, T, d, H, n, (float*)dA, D, dz,
             (float*)dz16, stream);
}

}  // namespace mosa
