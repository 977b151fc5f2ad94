// dX of the layer (chain rule through Q, K, V = X^s W^{Q,K,V} and the router
// logit s = X^s W^r of Section 2.2, I held fixed; the gather X^s = X[I]
// turns into a scatter-add over heads):
//   dX^s_i   = dQ_i W^Q_h^T + dK_i W^K_h^T + dV_i W^V_h^T + dz_i W^r_h
//   dX[b, t] = sum over heads h (ascending) of dX^s at the slot of t in head h
//              + the dense heads' dQ W^Q^T + dK W^K^T + dV W^V^T.
// Two GEMMs on the tiled MFMA engine, the same structure as the forward's
// output side:
//   dx_proj    per MoSA head: rows dQ | dK | dV (packed, K = 3 dh) times the
//              three weights read along their rows (k-contiguous, no
//              transpose), plus the rank-1 router term in the epilogue;
//   dx_combine per batch element: dense heads as one GEMM with
//              K = Hd * 3 dh, then the MoSA rows of each token added in head
//              order from the slot map (bitwise reproducible), then written.
#include "combine.h"
#include "gemm2.h"
#include "dxrow.h"
#include "gemm.h"
#include "kernels.h"

namespace mosa {

namespace {

template <typename ST, int DH>
struct DxProjPolicy {
    static constexpr int MT = 64, NT = 128, KC = (sizeof(ST) == 2 && DH == 64) ? 64 : 32, WM = 2, WN = 2;
    static constexpr size_t EPI_LDS = 0;
    static constexpr bool A_KCONTIG = true, B_KCONTIG = true, A_SCALED = false;
    struct Args {
        const ST* dQKV;  // [B, H, k, 3*DH]
        const float* dz; // [B, H, k]
        const ST* Wq;
        const ST* Wk;
        const ST* Wv;    // [H, d, DH]
        const ST* Wr;    // [H, d]
        ST* dXs;         // [B, H, k, d]
        int d, H, k, M, mtiles, ntiles;
    };
    struct ARef {
        const ST* p;
    };
    struct BRef {
        int c;
    };
    struct RowInfo {
        int unused;
    };
    __device__ static const ST* a_fallback(const Args& a) { return a.dQKV; }
    __device__ static const ST* b_fallback(const Args& a) { return a.Wq; }
    __device__ static void tile(const Args& a, int logical, int& h, int& m0, int& n0) {
        const int per = a.mtiles * a.ntiles;
        h = logical / per;
        const int rem = logical % per;
        m0 = (rem / a.ntiles) * MT;
        n0 = (rem % a.ntiles) * NT;
    }
    __device__ static int k_size(const Args&, int) { return 3 * DH; }
    __device__ static size_t ridx(const Args& a, int h, int m) {
        return ((size_t)(m / a.k) * a.H + h) * a.k + (m % a.k);
    }
    __device__ static ARef a_row(const Args& a, int h, int m, float&) {
        if (m < 0 || m >= a.M) return {nullptr};
        return {a.dQKV + ridx(a, h, m) * (3 * DH)};
    }
    __device__ static const ST* a_elem(const Args&, int, const ARef& r, int k) { return r.p ? r.p + k : nullptr; }
    __device__ static BRef b_row(const Args& a, int, int n) { return {n >= 0 && n < a.d ? n : -1}; }
    // B[k][c] = W^{k / DH}_h[c][k % DH]
    __device__ static const ST* b_elem(const Args& a, int h, const BRef& r, int k) {
        if (r.c < 0) return nullptr;
        const ST* W = k < DH ? a.Wq : (k < 2 * DH ? a.Wk : a.Wv);
        return W + ((size_t)h * a.d + r.c) * DH + (k % DH);
    }
    __device__ static RowInfo row_info(const Args&, int, int) { return {0}; }
    __device__ static const ST* a_kaddr(const Args& a, int, const RowInfo&, int) { return a_fallback(a); }
    __device__ static bool a_kok(const Args&, int, const RowInfo&, int) { return false; }
    __device__ static float a_kscale(const Args&, int, const RowInfo&) { return 1.f; }
    __device__ static const ST* b_kaddr(const Args& a, int, const RowInfo&, int) { return b_fallback(a); }
    __device__ static bool b_kok(const Args&, int, const RowInfo&, int) { return false; }
    __device__ static void epilogue(const Args& a, int h, int m0, int n0, const float* Cs, int ldc, int tid, unsigned char*) {
        constexpr int VPR = NT / 8;
        for (int v = tid; v < MT * VPR; v += 256) {
            const int ml = v / VPR, c = (v % VPR) * 8;
            const int m = m0 + ml;
            if (m >= a.M || n0 + c >= a.d) continue;
            const size_t ri = ridx(a, h, m);
            const float dzv = a.dz[ri];
            float wr[8], x[8];
            vec8_to_f32<ST>(vec8_load<ST>(a.Wr + (size_t)h * a.d + n0 + c), wr);
#pragma unroll
            for (int j = 0; j < 8; ++j) x[j] = Cs[ml * ldc + c + j] + dzv * wr[j];
            vec8_store<ST>(a.dXs + ri * a.d + n0 + c, vec8_from_f32<ST>(x));
        }
    }
};

template <typename ST, int DH>
struct DxCombinePolicy {
    static constexpr int MT = 64, NT = 128, KC = 32, WM = 2, WN = 2;
    static constexpr size_t EPI_LDS = kCombineLds;
    static constexpr bool A_KCONTIG = true, B_KCONTIG = true, A_SCALED = false;
    struct Args {
        const ST* dQKVd;      // [B, Hd, T, 3*DH]
        const ST* Wq;
        const ST* Wk;
        const ST* Wv;         // dense weights [Hd, d, DH]
        const int16_t* slot;  // [B, H, T]
        const ST* dXs;        // [B, H, k, d]
        ST* dX;
        int T, d, H, k, Hd, accumulate, mtiles, ntiles;
    };
    struct ARef {
        const ST* p;
    };
    struct BRef {
        int c;
    };
    struct RowInfo {
        int unused;
    };
    __device__ static const ST* a_fallback(const Args& a) { return a.dQKVd; }
    __device__ static const ST* b_fallback(const Args& a) { return a.Wq; }
    __device__ static void tile(const Args& a, int logical, int& b, int& m0, int& n0) {
        const int per = a.mtiles * a.ntiles;
        b = logical / per;
        const int rem = logical % per;
        m0 = (rem / a.ntiles) * MT;
        n0 = (rem % a.ntiles) * NT;
    }
    __device__ static int k_size(const Args& a, int) { return a.Hd * 3 * DH; }
    __device__ static ARef a_row(const Args& a, int b, int t, float&) {
        if (t < 0 || t >= a.T) return {nullptr};
        return {a.dQKVd + ((size_t)b * a.Hd * a.T + t) * (3 * DH)};
    }
    // K index = hd * 3 DH + j
    __device__ static const ST* a_elem(const Args& a, int, const ARef& r, int k) {
        return r.p ? r.p + (size_t)(k / (3 * DH)) * a.T * (3 * DH) + (k % (3 * DH)) : nullptr;
    }
    __device__ static BRef b_row(const Args& a, int, int n) { return {n >= 0 && n < a.d ? n : -1}; }
    __device__ static const ST* b_elem(const Args& a, int, const BRef& r, int k) {
        if (r.c < 0) return nullptr;
        const int hd = k / (3 * DH), j = k % (3 * DH);
        const ST* W = j < DH ? a.Wq : (j < 2 * DH ? a.Wk : a.Wv);
        return W + ((size_t)hd * a.d + r.c) * DH + (j % DH);
    }
    __device__ static RowInfo row_info(const Args&, int, int) { return {0}; }
    __device__ static const ST* a_kaddr(const Args& a, int, const RowInfo&, int) { return a_fallback(a); }
    __device__ static bool a_kok(const Args&, int, const RowInfo&, int) { return false; }
    __device__ static float a_kscale(const Args&, int, const RowInfo&) { return 1.f; }
    __device__ static const ST* b_kaddr(const Args& a, int, const RowInfo&, int) { return b_fallback(a); }
    __device__ static bool b_kok(const Args&, int, const RowInfo&, int) { return false; }
    __device__ static void epilogue(const Args& a, int b, int m0, int n0, const float* Cs, int ldc, int tid,
                                    unsigned char* extra) {
        combine_tile<ST>(Cs, ldc, tid, b, m0, n0, a.T, a.d, a.H, a.k, a.slot, a.dXs, a.dX, a.accumulate,
                         reinterpret_cast<int16_t*>(extra));
    }
};

// The dense heads' part alone ([B, T, d] in the storage type, here fp32) for
// combine_rows_kernel to start from.
template <typename ST, int DH>
struct DxDensePolicy : DxCombinePolicy<ST, DH> {
    using Base = DxCombinePolicy<ST, DH>;
    static constexpr size_t EPI_LDS = 0;
    struct Args : Base::Args {
        float* base;
    };
    __device__ static void epilogue(const Args& a, int b, int m0, int n0, const float* Cs, int ldc, int tid,
                                    unsigned char*) {
        constexpr int VPR = Base::NT / 4;
        for (int v = tid; v < Base::MT * VPR; v += 256) {
            const int ml = v / VPR, c = (v % VPR) * 4, t = m0 + ml;
            if (t >= a.T || n0 + c >= a.d) continue;
            *reinterpret_cast<float4*>(a.base + ((size_t)b * a.T + t) * a.d + n0 + c) =
                *reinterpret_cast<const float4*>(Cs + ml * ldc + c);
        }
    }
};

// The same on the multi-stage engine (gemm2.h), bf16: 128 tokens x 128
// columns per workgroup.  K runs over (head, Q|K|V, e): A = the dense heads'
// dQ|dK|dV rows of token t, head after head; B[k][n] = W^{Q|K|V}_d[hd][n][e]
// (k-contiguous, one of three weights per chunk, reached by its element
// offset from W^Q_d).
template <int DH>
struct DxDensePolicy2 {
    using ST = uint16_t;
    static constexpr int MT = 128, NT = 128, KC = 32, WM = 2, WN = 2, STAGES = 4;
    static constexpr size_t EPI_LDS = 0;
    static constexpr bool A_KCONTIG = true, B_KCONTIG = true;
    static_assert(DH % KC == 0, "chunks within one weight of one head");
    struct Args {
        const ST* dQKVd;  // [B, Hd, T, 3 DH]
        const ST* Wq;     // [Hd, d, DH]
        ptrdiff_t dk, dv; // W^K_d - W^Q_d, W^V_d - W^Q_d (elements)
        ST* base;         // [B, T, d], the dense heads' part in the storage type
        int T, d, Hd, mtiles, ntiles;
    };
    struct ARef {
        const ST* p;
    };
    struct BRef {
        const ST* p;
    };
    __device__ static void tile(const Args& a, int logical, int& b, int& m0, int& n0) {
        const int per = a.mtiles * a.ntiles, rem = logical % per;
        b = logical / per;
        m0 = (rem / a.ntiles) * MT;
        n0 = (rem % a.ntiles) * NT;
    }
    __device__ static int k_size(const Args& a, int) { return a.Hd * 3 * DH; }
    __device__ static ARef a_row(const Args& a, int b, int t) {
        return {a.dQKVd + ((size_t)b * a.Hd * a.T + min(t, a.T - 1)) * (3 * DH)};
    }
    __device__ static const ST* a_elem(const Args&, int, const ARef& r, int k) { return r.p + k; }
    __device__ static ptrdiff_t a_koff(const Args& a, int, int c) {
        const int k = c * KC;
        return (ptrdiff_t)(k / (3 * DH)) * a.T * (3 * DH) + k % (3 * DH);
    }
    __device__ static BRef b_row(const Args& a, int, int n) { return {a.Wq + (size_t)min(n, a.d - 1) * DH}; }
    __device__ static const ST* b_elem(const Args&, int, const BRef& r, int k) { return r.p + k; }
    __device__ static ptrdiff_t b_koff(const Args& a, int, int c) {
        const int k = c * KC, hd = k / (3 * DH), j = k % (3 * DH), w = j / DH;
        return (w == 0 ? 0 : (w == 1 ? a.dk : a.dv)) + (ptrdiff_t)hd * a.d * DH + j % DH;
    }
    __device__ static void epilogue(const Args& a, int b, int m0, int n0, const float* Cs, int ldc, int tid,
                                    unsigned char*) {
        constexpr int VPR = NT / 8;
        for (int v = tid; v < MT * VPR; v += 256) {
            const int ml = v / VPR, c = (v % VPR) * 8, t = m0 + ml;
            if (t >= a.T || n0 + c >= a.d) continue;
            float x[8];
            cs_load8(Cs, ldc, ml, c, x);
            vec8_store<ST>(a.base + ((size_t)b * a.T + t) * a.d + n0 + c, vec8_from_f32<ST>(x));
        }
    }
};

template <typename ST, int DH>
int run_proj(const ST* dQKV, const float* dz, const ST* Wq, const ST* Wk, const ST* Wv, const ST* Wr, int B, int d,
             int H, int k, ST* dXs, hipStream_t stream) {
    using P = DxProjPolicy<ST, DH>;
    const int M = B * k;
    if constexpr (sizeof(ST) == 2) {
        using R = DxProjRowPolicy<DH>;
        typename R::Args ra;
        int nblocks;
        if (dx_row_args<DH>(dQKV, dz, Wq, Wk, Wv, Wr, B, d, H, k, dXs, ra, nblocks))
            return launch_rowgemm<R>(ra, nblocks, stream);
    }
    typename P::Args a{dQKV, dz, Wq, Wk, Wv, Wr, dXs, d, H, k, M, (M + P::MT - 1) / P::MT, (d + P::NT - 1) / P::NT};
    return launch_gemm<ST, P>(a, H * a.mtiles * a.ntiles, stream);
}

template <typename ST, int DH>
int run_combine(const ST* dQKVd, const ST* Wq, const ST* Wk, const ST* Wv, const int16_t* slot, const ST* dXs, int B,
                int T, int d, int H, int k, int Hd, ST* dX, int accumulate, ST* base, int part, const Marker& mk, hipStream_t stream) {
    using P = DxCombinePolicy<ST, DH>;
    typename P::Args a{dQKVd, Wq, Wk, Wv, slot, dXs, dX, T, d, H, k, Hd, accumulate, (T + P::MT - 1) / P::MT,
                       (d + P::NT - 1) / P::NT};
    if (combine_rows_fits(d, H) && (Hd == 0 || base)) {
        // dense heads first (into base), then the per-token combination
        // (part 1: the first only, part 2: the second only, 0: both)
        if (Hd > 0 && part != 2) {
            int e;
            if constexpr (sizeof(ST) == 2) {
                using P2 = DxDensePolicy2<DH>;
                const int mt = (T + P2::MT - 1) / P2::MT, nt = (d + P2::NT - 1) / P2::NT;
                auto dist = [&](const ST* p) {  // element distance from W^Q_d
                    return (ptrdiff_t)(((intptr_t)p - (intptr_t)Wq) / (intptr_t)sizeof(ST));
                };
                typename P2::Args a2{(const uint16_t*)dQKVd, (const uint16_t*)Wq, dist(Wk), dist(Wv), base, T, d, Hd,
                                     mt, nt};
                e = launch_gemm2<P2>(a2, B * mt * nt, stream);
            } else {
                using PD = DxDensePolicy<ST, DH>;
                typename PD::Args ad{};
                static_cast<typename P::Args&>(ad) = a;
                ad.base = base;
                e = launch_gemm<ST, PD>(ad, B * a.mtiles * a.ntiles, stream);
            }
            if (e | mk("dx_dense")) return -1;
        }
        if (part == 1) return 0;
        return launch_combine_rows<ST, 1>(slot, dXs, Hd > 0 ? base : nullptr, dX, B, T, d, H, k, accumulate, stream) |
               mk("dx_combine");
    }
    if (part != 0) return 1;  // the one-kernel form cannot be split
    return launch_gemm<ST, P>(a, B * a.mtiles * a.ntiles, stream) | mk("dx_combine");
}

}  // namespace

int launch_dx_proj(int dtype, const void* dQKV, const float* dz, const void* Wq, const void* Wk, const void* Wv,
                   const void* Wr, int B, int d, int H, int dh, int k, void* dXs, hipStream_t stream) {
    if (H == 0) return 0;
    if (dtype == kBF16) {
        auto f = dh == 64 ? run_proj<uint16_t, 64> : run_proj<uint16_t, 32>;
        return f((const uint16_t*)dQKV, dz, (const uint16_t*)Wq, (const uint16_t*)Wk, (const uint16_t*)Wv,
                 (const uint16_t*)Wr, B, d, H, k, (uint16_t*)dXs, stream);
    }
    auto f = dh == 64 ? run_proj<float, 64> : run_proj<float, 32>;
    return f((const float*)dQKV, dz, (const float*)Wq, (const float*)Wk, (const float*)Wv, (const float*)Wr, B, d, H,
             k, (float*)dXs, stream);
}

int launch_dx_combine(int dtype, const void* dQKVd, const void* Wq_d, const void* Wk_d, const void* Wv_d,
                      const int16_t* slot, const void* dXs, int B, int T, int d, int H, int dh, int k, int Hd,
                      void* dX, int accumulate, void* base, int part, const Marker& mk, hipStream_t stream) {
    if (dtype == kBF16) {
        auto f = dh == 64 ? run_combine<uint16_t, 64> : run_combine<uint16_t, 32>;
        return f((const uint16_t*)dQKVd, (const uint16_t*)Wq_d, (const uint16_t*)Wk_d, (const uint16_t*)Wv_d, slot,
                 (const uint16_t*)dXs, B, T, d, H, k, Hd, (uint16_t*)dX, accumulate, (uint16_t*)base, part, mk, stream);
    }
    auto f = dh == 64 ? run_combine<float, 64> : run_combine<float, 32>;
    return f((const float*)dQKVd, (const float*)Wq_d, (const float*)Wk_d, (const float*)Wv_d, slot,
             (const float*)dXs, B, T, d, H, k, Hd, (float*)dX, accumulate, (float*)base, part, mk, stream);
}

}  // namespace mosa
