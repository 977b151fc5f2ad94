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
                int T, int d, int H, int k, int Hd, ST* dX, int accumulate, hipStream_t stream) {
    using P = DxCombinePolicy<ST, DH>;
    if (Hd == 0 && d % 8 == 0 && d <= 2048 && (size_t)H * kCombineLdt * 2 <= 64 * 1024)
        return launch_combine_rows<ST, 1>(slot, dXs, dX, B, T, d, H, k, accumulate, stream);
    typename P::Args a{dQKVd, Wq, Wk, Wv, slot, dXs, dX, T, d, H, k, Hd, accumulate, (T + P::MT - 1) / P::MT,
                       (d + P::NT - 1) / P::NT};
    return launch_gemm<ST, P>(a, B * a.mtiles * a.ntiles, stream);
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
                      void* dX, int accumulate, hipStream_t stream) {
    if (dtype == kBF16) {
        auto f = dh == 64 ? run_combine<uint16_t, 64> : run_combine<uint16_t, 32>;
        return f((const uint16_t*)dQKVd, (const uint16_t*)Wq_d, (const uint16_t*)Wk_d, (const uint16_t*)Wv_d, slot,
                 (const uint16_t*)dXs, B, T, d, H, k, Hd, (uint16_t*)dX, accumulate, stream);
    }
    auto f = dh == 64 ? run_combine<float, 64> : run_combine<float, 32>;
    return f((const float*)dQKVd, (const float*)Wq_d, (const float*)Wk_d, (const float*)Wv_d, slot,
             (const float*)dXs, B, T, d, H, k, Hd, (float*)dX, accumulate, stream);
}

}  // namespace mosa
