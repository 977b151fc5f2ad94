// Weight gradients of the heads (chain rule through Section 2.2 with I held
// fixed), each a sum over every selected row r = (b, i) in a fixed order:
//   dW^Q_h = sum_r X[b, I_r]^T dQ_r   (likewise W^K, W^V)    [d x dh]
//   dW^r_h = sum_r dz_r X[b, I_r]                             [d]
//   dW^O_h = sum_r (r_r A_r)^T dY[b, I_r]                     [dh x d]
//            (the forward saved the rows r_r A_r already scaled)
// Dense heads: the same with I = identity and r = 1 (no W^r).
//
// On the tiled MFMA engine the contraction index K is the row r, which is
// contiguous in neither operand: both are staged with the engine's 8x8
// register transpose.  wgrad_qkv: M = d, N = 3 dh (+ a 16-column block whose
// first column is dz, so dW^r falls out of the same MFMAs), one workgroup per
// (head, 64 rows of d).  wgrad_o: M = dh, N = d.  The K loop runs over the rows
// in order, so the sums are bitwise reproducible.
#include "gemm.h"
#include "kernels.h"

namespace mosa {

namespace {

template <typename ST, int DH, bool ROUTER, bool GATHER>
struct WgradQkvPolicy {
    static constexpr int MT = 64, NT = 3 * DH + (ROUTER ? 16 : 0), KC = sizeof(ST) == 2 ? 64 : 32, WM = 4, WN = 1;
    static constexpr size_t EPI_LDS = 0;
    static constexpr bool A_KCONTIG = false, B_KCONTIG = false, A_SCALED = false;
    struct Args {
        const ST* X;
        const int32_t* I;
        const ST* dQKV;  // [B, H, n, 3*DH]
        const ST* dz16;  // [B, H, n, 16]
        ST* dWq;
        ST* dWk;
        ST* dWv;         // [H, d, DH]
        ST* dWr;         // [H, d]
        int T, d, H, n, R, mtiles;
        FastDiv nd;
    };
    struct ARef {};
    struct BRef {};
    // Row r = (b, i) of head h.  The token index t is kept as loaded (the
    // address arithmetic happens in a_kaddr), so the gather load is waited
    // for only when the row infos are stored to LDS, after the chunk's MFMAs.
    struct RowInfo {
        int b;   // batch element, or -1 past the last row
        int t;   // token I_r (gathered) or i (dense)
        int ri;  // selected-row index (b*H + h)*n + i
    };
    __device__ static const ST* a_fallback(const Args& a) { return a.X; }
    __device__ static const ST* b_fallback(const Args& a) { return a.dQKV; }
    __device__ static void tile(const Args& a, int logical, int& h, int& m0, int& n0) {
        h = logical / a.mtiles;
        m0 = (logical % a.mtiles) * MT;
        n0 = 0;
    }
    __device__ static int k_size(const Args& a, int) { return a.R; }
    __device__ static ARef a_row(const Args&, int, int, float&) { return {}; }
    __device__ static const ST* a_elem(const Args&, int, const ARef&, int) { return nullptr; }
    __device__ static BRef b_row(const Args&, int, int) { return {}; }
    __device__ static const ST* b_elem(const Args&, int, const BRef&, int) { return nullptr; }
    __device__ static RowInfo row_info(const Args& a, int h, int r) {
        int b, i;
        fast_divmod(a.nd, r < 0 ? 0 : r, b, i);
        const int ri = (b * a.H + h) * a.n + i;
        return {r < 0 ? -1 : b, GATHER ? a.I[ri] : i, ri};
    }
    // A[c][r] = X[b, I_r, c]: row r of the gathered input, c contiguous
    __device__ static const ST* a_kaddr(const Args& a, int, const RowInfo& r, int m8) {
        return a.X + ((size_t)max(r.b, 0) * a.T + r.t) * a.d + min(m8, a.d - 8);
    }
    __device__ static bool a_kok(const Args& a, int, const RowInfo& r, int m8) { return r.b >= 0 && m8 < a.d; }
    __device__ static float a_kscale(const Args&, int, const RowInfo&) { return 1.f; }
    // B[r][n] = dQ | dK | dV | (dz, 0...) of row r
    __device__ static const ST* b_kaddr(const Args& a, int, const RowInfo& r, int n8) {
        return n8 < 3 * DH ? a.dQKV + (size_t)r.ri * (3 * DH) + n8 : a.dz16 + (size_t)r.ri * 16 + (n8 - 3 * DH);
    }
    __device__ static bool b_kok(const Args&, int, const RowInfo& r, int) { return r.b >= 0; }
    __device__ static void epilogue(const Args& a, int h, int m0, int, const float* Cs, int ldc, int tid, unsigned char*) {
        constexpr int VPR = 3 * DH / 8;
        for (int v = tid; v < MT * VPR; v += 256) {
            const int ml = v / VPR, nn = (v % VPR) * 8;
            const int c = m0 + ml;
            if (c >= a.d) continue;
            float x[8];
            cs_load8(Cs, ldc, ml, nn, x);
            ST* W = nn < DH ? a.dWq : (nn < 2 * DH ? a.dWk : a.dWv);
            vec8_store<ST>(W + ((size_t)h * a.d + c) * DH + (nn % DH), vec8_from_f32<ST>(x));
        }
        if (ROUTER && tid < MT && m0 + tid < a.d) st1<ST>(a.dWr + (size_t)h * a.d + m0 + tid, Cs[tid * ldc + 3 * DH]);
    }
};

template <typename ST, int DH, bool GATHER>
struct WgradOPolicy {
    static constexpr int MT = DH, NT = 128, KC = sizeof(ST) == 2 ? 64 : 32, WM = 2, WN = 2;
    static constexpr size_t EPI_LDS = 0;
    static constexpr bool A_KCONTIG = false, B_KCONTIG = false, A_SCALED = false;
    struct Args {
        const ST* dY;
        const int32_t* I;
        const ST* A;      // [B, H, n, DH], rows scaled by r
        ST* dWo;          // [H, DH, d]
        int T, d, H, n, R, ntiles;
        FastDiv nd;
    };
    struct ARef {};
    struct BRef {};
    struct RowInfo {
        int b;   // batch element, or -1 past the last row
        int t;   // token I_r (gathered) or i (dense), as loaded
        int ri;  // selected-row index
    };
    __device__ static const ST* a_fallback(const Args& a) { return a.A; }
    __device__ static const ST* b_fallback(const Args& a) { return a.dY; }
    __device__ static void tile(const Args& a, int logical, int& h, int& m0, int& n0) {
        h = logical / a.ntiles;
        m0 = 0;
        n0 = (logical % a.ntiles) * NT;
    }
    __device__ static int k_size(const Args& a, int) { return a.R; }
    __device__ static ARef a_row(const Args&, int, int, float&) { return {}; }
    __device__ static const ST* a_elem(const Args&, int, const ARef&, int) { return nullptr; }
    __device__ static BRef b_row(const Args&, int, int) { return {}; }
    __device__ static const ST* b_elem(const Args&, int, const BRef&, int) { return nullptr; }
    __device__ static RowInfo row_info(const Args& a, int h, int r) {
        int b, i;
        fast_divmod(a.nd, r < 0 ? 0 : r, b, i);
        const int ri = (b * a.H + h) * a.n + i;
        return {r < 0 ? -1 : b, GATHER ? a.I[ri] : i, ri};
    }
    // A[e][r] = (r_r A_r)[e]
    __device__ static const ST* a_kaddr(const Args& a, int, const RowInfo& r, int m8) {
        return a.A + (size_t)r.ri * DH + m8;
    }
    __device__ static bool a_kok(const Args&, int, const RowInfo& r, int) { return r.b >= 0; }
    __device__ static float a_kscale(const Args&, int, const RowInfo&) { return 1.f; }
    // B[r][c] = dY[b, I_r, c]
    __device__ static const ST* b_kaddr(const Args& a, int, const RowInfo& r, int n8) {
        return a.dY + ((size_t)max(r.b, 0) * a.T + r.t) * a.d + min(n8, a.d - 8);
    }
    __device__ static bool b_kok(const Args& a, int, const RowInfo& r, int n8) { return r.b >= 0 && n8 < a.d; }
    __device__ static void epilogue(const Args& a, int h, int, int n0, const float* Cs, int ldc, int tid, unsigned char*) {
        constexpr int VPR = NT / 8;
        for (int v = tid; v < MT * VPR; v += 256) {
            const int e = v / VPR, c = (v % VPR) * 8;
            if (n0 + c >= a.d) continue;
            float x[8];
            cs_load8(Cs, ldc, e, c, x);
            vec8_store<ST>(a.dWo + ((size_t)h * DH + e) * a.d + n0 + c, vec8_from_f32<ST>(x));
        }
    }
};

template <typename ST, int DH>
int run_qkv(const ST* X, const int32_t* I, const ST* dQKV, const ST* dz16, int B, int T, int d, int H, int n, ST* dWq,
            ST* dWk, ST* dWv, ST* dWr, hipStream_t stream) {
    const int mtiles = (d + 63) / 64;
    const FastDiv nd = make_fastdiv(n);
    if (I) {  // MoSA heads: gathered rows and the router column
        using P = WgradQkvPolicy<ST, DH, true, true>;
        typename P::Args a{X, I, dQKV, dz16, dWq, dWk, dWv, dWr, T, d, H, n, B * n, mtiles, nd};
        return launch_gemm<ST, P>(a, H * mtiles, stream);
    }
    using P = WgradQkvPolicy<ST, DH, false, false>;
    typename P::Args a{X, I, dQKV, dz16, dWq, dWk, dWv, dWr, T, d, H, n, B * n, mtiles, nd};
    return launch_gemm<ST, P>(a, H * mtiles, stream);
}

template <typename ST, int DH>
int run_o(const ST* dY, const int32_t* I, const ST* A, int B, int T, int d, int H, int n, ST* dWo,
          hipStream_t stream) {
    const FastDiv nd = make_fastdiv(n);
    if (I) {
        using P = WgradOPolicy<ST, DH, true>;
        const int ntiles = (d + P::NT - 1) / P::NT;
        typename P::Args a{dY, I, A, dWo, T, d, H, n, B * n, ntiles, nd};
        return launch_gemm<ST, P>(a, H * ntiles, stream);
    }
    using P = WgradOPolicy<ST, DH, false>;
    const int ntiles = (d + P::NT - 1) / P::NT;
    typename P::Args a{dY, I, A, dWo, T, d, H, n, B * n, ntiles, nd};
    return launch_gemm<ST, P>(a, H * ntiles, stream);
}

}  // namespace

int launch_wgrad(int dtype, const void* X, const void* dY, const int32_t* I, const void* A,
                 const void* dQKV, const void* dz16, int B, int T, int d, int H, int dh, int n, void* dWq, void* dWk,
                 void* dWv, void* dWr, void* dWo, int which, hipStream_t stream) {
    if (H == 0) return 0;
    if (dtype == kBF16) {
        using ST = uint16_t;
        if (which == 0) {
            auto f = dh == 64 ? run_qkv<ST, 64> : run_qkv<ST, 32>;
            return f((const ST*)X, I, (const ST*)dQKV, (const ST*)dz16, B, T, d, H, n, (ST*)dWq, (ST*)dWk, (ST*)dWv,
                     (ST*)dWr, stream);
        }
        auto f = dh == 64 ? run_o<ST, 64> : run_o<ST, 32>;
        return f((const ST*)dY, I, (const ST*)A, B, T, d, H, n, (ST*)dWo, stream);
    }
    using ST = float;
    if (which == 0) {
        auto f = dh == 64 ? run_qkv<ST, 64> : run_qkv<ST, 32>;
        return f((const ST*)X, I, (const ST*)dQKV, (const ST*)dz16, B, T, d, H, n, (ST*)dWq, (ST*)dWk, (ST*)dWv,
                 (ST*)dWr, stream);
    }
    auto f = dh == 64 ? run_o<ST, 64> : run_o<ST, 32>;
    return f((const ST*)dY, I, (const ST*)A, B, T, d, H, n, (ST*)dWo, stream);
}

}  // namespace mosa
