// Router-scaled output projection and the deterministic head-ordered
// combination into the T-long output (paper Section 2.2:
// X^o = diag(r) A W^O, Y_{I_i} = X^o_i; Eq. 3: the layer is the sum of its
// heads; Eq. 2: dense heads add A W^O over every token).
//
// Two GEMMs on the tiled MFMA engine (gemm.h):
//   out_proj    per MoSA head h: X^o[b,h,i,:] = (r_i A_i) W^O_h, M = B*k
//               selected rows, N = d, K = dh, written once (storage type);
//               the attention kernel already stored the rows as r_i A_i;
//   out_combine per batch element b: a tile of 64 tokens x 128 columns of
//               Y = A_dense W^O_dense (dense heads concatenated along K,
//               K = Hd*dh, possibly 0) and then, in the epilogue, the MoSA
//               rows of that tile added in ascending head order: for token t
//               and head h the slot is slot[b,h,t] (-1: not selected).  Each
//               output element is produced by one thread in a fixed order, so
//               the result is bitwise reproducible and unselected rows are
//               exactly the dense part (0 without dense heads).
#include "combine.h"
#include "gemm2.h"
#include "gemm.h"
#include "kernels.h"
#include "rowgemm.h"

namespace mosa {

namespace {

template <typename ST, int DH>
struct OutProjPolicy {
    static constexpr int MT = 64, NT = 128, KC = sizeof(ST) == 2 ? DH : 32, WM = 2, WN = 2;
    static constexpr size_t EPI_LDS = 0;
    static constexpr bool A_KCONTIG = true, B_KCONTIG = false, A_SCALED = false;
    struct Args {
        const ST* A;   // [B, H, k, DH], rows scaled by r
        const ST* Wo;  // [H, DH, d]
        ST* Xo;        // [B, H, k, d]
        int d, H, k, M, mtiles, ntiles;
    };
    struct ARef {
        const ST* p;
    };
    struct BRef {};
    struct RowInfo {
        int k;
    };
    __device__ static const ST* a_fallback(const Args& a) { return a.A; }
    __device__ static const ST* b_fallback(const Args& a) { return a.Wo; }
    __device__ static void tile(const Args& a, int logical, int& h, int& m0, int& n0) {
        const int per = a.mtiles * a.ntiles;
        h = logical / per;
        const int rem = logical % per;
        m0 = (rem / a.ntiles) * MT;
        n0 = (rem % a.ntiles) * NT;
    }
    __device__ static int k_size(const Args&, int) { return DH; }
    __device__ static size_t ridx(const Args& a, int h, int m) {
        return ((size_t)(m / a.k) * a.H + h) * a.k + (m % a.k);
    }
    __device__ static ARef a_row(const Args& a, int h, int m, float&) {
        if (m < 0 || m >= a.M) return {nullptr};
        return {a.A + ridx(a, h, m) * DH};
    }
    __device__ static const ST* a_elem(const Args&, int, const ARef& r, int k) { return r.p ? r.p + k : nullptr; }
    __device__ static BRef b_row(const Args&, int, int) { return {}; }
    __device__ static const ST* b_elem(const Args&, int, const BRef&, int) { return nullptr; }
    __device__ static RowInfo row_info(const Args&, int, int k) { return {k}; }
    __device__ static const ST* a_kaddr(const Args& a, int, const RowInfo&, int) { return a_fallback(a); }
    __device__ static bool a_kok(const Args&, int, const RowInfo&, int) { return false; }
    __device__ static float a_kscale(const Args&, int, const RowInfo&) { return 1.f; }
    __device__ static const ST* b_kaddr(const Args& a, int h, const RowInfo& r, int n8) {
        return a.Wo + ((size_t)h * DH + max(r.k, 0)) * a.d + min(n8, a.d - 8);
    }
    __device__ static bool b_kok(const Args& a, int, const RowInfo& r, int n8) { return r.k >= 0 && n8 < a.d; }
    __device__ static void epilogue(const Args& a, int h, int m0, int n0, const float* Cs, int ldc, int tid, unsigned char*) {
        constexpr int VPR = NT / 8;
        for (int v = tid; v < MT * VPR; v += 256) {
            const int ml = v / VPR, c = (v % VPR) * 8;
            const int m = m0 + ml;
            if (m >= a.M || n0 + c >= a.d) continue;
            float x[8];
            cs_load8(Cs, ldc, ml, c, x);
            vec8_store<ST>(a.Xo + ridx(a, h, m) * a.d + n0 + c, vec8_from_f32<ST>(x));
        }
    }
};

template <typename ST, int DH>
struct OutCombinePolicy {
    static constexpr int MT = 64, NT = 128, KC = 32, WM = 2, WN = 2;
    static constexpr size_t EPI_LDS = kCombineLds;
    static constexpr bool A_KCONTIG = true, B_KCONTIG = false, A_SCALED = false;
    struct Args {
        const ST* Ad;        // [B, Hd, T, DH]
        const ST* Wod;       // [Hd, DH, d] = [Hd*DH, d]
        const int16_t* slot; // [B, H, T]
        const ST* Xo;        // [B, H, k, d]
        ST* Y;               // [B, T, d]
        int T, d, H, k, Hd, accumulate, mtiles, ntiles;
    };
    struct ARef {
        const ST* p;
    };
    struct BRef {};
    struct RowInfo {
        int k;
    };
    __device__ static const ST* a_fallback(const Args& a) { return a.Ad; }
    __device__ static const ST* b_fallback(const Args& a) { return a.Wod; }
    __device__ static void tile(const Args& a, int logical, int& b, int& m0, int& n0) {
        const int per = a.mtiles * a.ntiles;
        b = logical / per;
        const int rem = logical % per;
        m0 = (rem / a.ntiles) * MT;
        n0 = (rem % a.ntiles) * NT;
    }
    __device__ static int k_size(const Args& a, int) { return a.Hd * DH; }
    __device__ static ARef a_row(const Args& a, int b, int t, float&) {
        if (t < 0 || t >= a.T) return {nullptr};
        return {a.Ad + ((size_t)b * a.Hd * a.T + t) * DH};
    }
    // K index = hd * DH + e: row t of dense head hd
    __device__ static const ST* a_elem(const Args& a, int, const ARef& r, int k) {
        return r.p ? r.p + (size_t)(k / DH) * a.T * DH + (k % DH) : nullptr;
    }
    __device__ static BRef b_row(const Args&, int, int) { return {}; }
    __device__ static const ST* b_elem(const Args&, int, const BRef&, int) { return nullptr; }
    __device__ static RowInfo row_info(const Args&, int, int k) { return {k}; }
    __device__ static const ST* a_kaddr(const Args& a, int, const RowInfo&, int) { return a_fallback(a); }
    __device__ static bool a_kok(const Args&, int, const RowInfo&, int) { return false; }
    __device__ static float a_kscale(const Args&, int, const RowInfo&) { return 1.f; }
    __device__ static const ST* b_kaddr(const Args& a, int, const RowInfo& r, int n8) {
        return a.Wod + (size_t)max(r.k, 0) * a.d + min(n8, a.d - 8);
    }
    __device__ static bool b_kok(const Args& a, int, const RowInfo& r, int n8) { return r.k >= 0 && n8 < a.d; }

    // 4 threads per token row, 32 columns each; MoSA rows added in head order.
    __device__ static void epilogue(const Args& a, int b, int m0, int n0, const float* Cs, int ldc, int tid,
                                    unsigned char* extra) {
        combine_tile<ST>(Cs, ldc, tid, b, m0, n0, a.T, a.d, a.H, a.k, a.slot, a.Xo, a.Y, a.accumulate,
                         reinterpret_cast<int16_t*>(extra));
    }
};

// The dense heads' part alone ([B, T, d] in the storage type, here fp32) for
// combine_rows_kernel to start from.
template <typename ST, int DH>
struct OutDensePolicy : OutCombinePolicy<ST, DH> {
    using Base = OutCombinePolicy<ST, DH>;
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
// columns per workgroup; A = the dense heads' rows of token t, head after
// head (chunks of KC stay within a head), B = W^O_d as one [Hd DH, d]
// m-contiguous operand.
template <int DH>
struct OutDensePolicy2 {
    using ST = uint16_t;
    static constexpr int MT = 128, NT = 128, KC = 32, WM = 2, WN = 2, STAGES = 4;
    static constexpr size_t EPI_LDS = 0;
    static constexpr bool A_KCONTIG = true, B_KCONTIG = false;
    static_assert(DH % KC == 0, "chunks within a head");
    struct Args {
        const ST* Ad;   // [B, Hd, T, DH]
        const ST* Wod;  // [Hd DH, d]
        ST* base;       // [B, T, d], the dense heads' part in the storage type
        int T, d, Hd, mtiles, ntiles;
    };
    struct ARef {
        const ST* p;
    };
    __device__ static void tile(const Args& a, int logical, int& b, int& m0, int& n0) {
        const int per = a.mtiles * a.ntiles, rem = logical % per;
        b = logical / per;
        m0 = (rem / a.ntiles) * MT;
        n0 = (rem % a.ntiles) * NT;
    }
    __device__ static int k_size(const Args& a, int) { return a.Hd * DH; }
    __device__ static ARef a_row(const Args& a, int b, int t) {
        return {a.Ad + ((size_t)b * a.Hd * a.T + min(t, a.T - 1)) * DH};
    }
    __device__ static const ST* a_elem(const Args&, int, const ARef& r, int k) { return r.p + k; }
    __device__ static ptrdiff_t a_koff(const Args& a, int, int c) {
        const int k = c * KC;
        return (ptrdiff_t)(k / DH) * a.T * DH + k % DH;
    }
    __device__ static size_t b_kstride(const Args& a, int) { return a.d; }
    __device__ static const ST* b_maddr(const Args& a, int, int k, int n8) {
        return a.Wod + (size_t)k * a.d + min(n8, a.d - 8);
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

// bf16 storage, d a multiple of the column block: the row-streaming kernel (rowgemm.h),
// W^O_h[:, n0:n0+256] held in registers, the r-scaled rows streamed.
template <int DH>
struct OutProjRowPolicy {
    using ST = uint16_t;
    static constexpr int K = DH, NPAIR = 2, STAGES = 4;
    static constexpr bool W_KCONTIG = false, ROW_SCALAR = false;
    struct Args {
        const ST* A;   // [B, H, k, DH], rows scaled by r
        const ST* Wo;  // [H, DH, d]
        ST* Xo;        // [B, H, k, d]
        int d, H, k, M, ntiles, tiles, per, splits, out_bytes;
    };
    __device__ static void tile(const Args& a, int logical, int& h, int& n0, int& s_beg, int& s_end) {
        const int unit = logical / a.splits, sp = logical % a.splits;
        h = unit / a.ntiles;
        n0 = (unit % a.ntiles) * (128 * NPAIR);
        s_beg = sp * a.per;
        s_end = min(a.tiles, s_beg + a.per);
    }
    __device__ static int rows(const Args& a) { return a.M; }
    __device__ static size_t ridx(const Args& a, int h, int m) {
        return ((size_t)(m / a.k) * a.H + h) * a.k + (m % a.k);
    }
    __device__ static const ST* a_row(const Args& a, int h, int m) { return a.A + ridx(a, h, m) * DH; }
    __device__ static const ST* w_mptr(const Args& a, int h, int k, int n) { return a.Wo + ((size_t)h * DH + k) * a.d + n; }
    __device__ static void col_init(const Args&, int, int, float (&)[8]) {}
    __device__ static __amdgpu_buffer_rsrc_t out_rsrc(const Args& a, int) {
        return __builtin_amdgcn_make_buffer_rsrc(a.Xo, 0, a.out_bytes, 0x00020000);
    }
    __device__ static int out_row(const Args& a, int h, int m) { return (int)(ridx(a, h, m) * a.d * 2); }
    __device__ static void finish(float (&)[8], float, const float (&)[8]) {}
};

template <typename ST, int DH>
int run_proj(const ST* A, const ST* Wo, int B, int d, int H, int k, ST* Xo, hipStream_t stream) {
    using P = OutProjPolicy<ST, DH>;
    const int M = B * k;
    if constexpr (sizeof(ST) == 2) {
        const long long out_bytes = (long long)M * H * d * 2;
        using R = OutProjRowPolicy<DH>;
        if (d % (128 * R::NPAIR) == 0 && out_bytes < (1ll << 31)) {
            const int ntiles = d / (128 * R::NPAIR), tiles = (M + 63) / 64;
            const int per = rowgemm_tiles_per_wg(H * ntiles, tiles, 512), splits = (tiles + per - 1) / per;
            typename R::Args ra{A, Wo, Xo, d, H, k, M, ntiles, tiles, per, splits, (int)out_bytes};
            return launch_rowgemm<R>(ra, H * ntiles * splits, stream);
        }
    }
    typename P::Args a{A, Wo, Xo, d, H, k, M, (M + P::MT - 1) / P::MT, (d + P::NT - 1) / P::NT};
    return launch_gemm<ST, P>(a, H * a.mtiles * a.ntiles, stream);
}

template <typename ST, int DH>
int run_combine(const ST* Ad, const ST* Wod, const int16_t* slot, const ST* Xo, int B, int T, int d, int H, int k,
                int Hd, ST* Y, int accumulate, ST* base, int part, const Marker& mk, hipStream_t stream) {
    using P = OutCombinePolicy<ST, DH>;
    typename P::Args a{Ad, Wod, slot, Xo, Y, T, d, H, k, Hd, accumulate, (T + P::MT - 1) / P::MT,
                       (d + P::NT - 1) / P::NT};
    if (combine_rows_fits(d, H) && (Hd == 0 || base)) {
        // dense heads first (into base), then the per-token combination
        // (part 1: the first only, part 2: the second only, 0: both)
        if (Hd > 0 && part != 2) {
            int e;
            if constexpr (sizeof(ST) == 2) {
                using P2 = OutDensePolicy2<DH>;
                const int mt = (T + P2::MT - 1) / P2::MT, nt = (d + P2::NT - 1) / P2::NT;
                typename P2::Args a2{(const uint16_t*)Ad, (const uint16_t*)Wod, base, T, d, Hd, mt, nt};
                e = launch_gemm2<P2>(a2, B * mt * nt, stream);
            } else {
                using PD = OutDensePolicy<ST, DH>;
                typename PD::Args ad{};
                static_cast<typename P::Args&>(ad) = a;
                ad.base = base;
                e = launch_gemm<ST, PD>(ad, B * a.mtiles * a.ntiles, stream);
            }
            if (e | mk("out_dense")) return -1;
        }
        if (part == 1) return 0;
        return launch_combine_rows<ST, 0>(slot, Xo, Hd > 0 ? base : nullptr, Y, B, T, d, H, k, accumulate, stream) |
               mk("out_combine");
    }
    if (part != 0) return 1;  // the one-kernel form cannot be split
    return launch_gemm<ST, P>(a, B * a.mtiles * a.ntiles, stream) | mk("out_combine");
}

}  // namespace

bool combine_split_ok(int d, int H) { return combine_rows_fits(d, H); }

int launch_out_proj(int dtype, const void* A, const void* Wo, int B, int d, int H, int dh, int k, void* Xo,
                    hipStream_t stream) {
    if (H == 0) return 0;
    if (dtype == kBF16) {
        auto f = dh == 64 ? run_proj<uint16_t, 64> : run_proj<uint16_t, 32>;
        return f((const uint16_t*)A, (const uint16_t*)Wo, B, d, H, k, (uint16_t*)Xo, stream);
    }
    auto f = dh == 64 ? run_proj<float, 64> : run_proj<float, 32>;
    return f((const float*)A, (const float*)Wo, B, d, H, k, (float*)Xo, stream);
}

int launch_out_combine(int dtype, const void* Ad, const void* Wo_d, const int16_t* slot, const void* Xo, int B,
                       int T, int d, int H, int dh, int k, int Hd, void* Y, int accumulate, void* base,
                       int part, const Marker& mk, hipStream_t stream) {
    if (dtype == kBF16) {
        auto f = dh == 64 ? run_combine<uint16_t, 64> : run_combine<uint16_t, 32>;
        return f((const uint16_t*)Ad, (const uint16_t*)Wo_d, slot, (const uint16_t*)Xo, B, T, d, H, k, Hd,
                 (uint16_t*)Y, accumulate, (uint16_t*)base, part, mk, stream);
    }
    auto f = dh == 64 ? run_combine<float, 64> : run_combine<float, 32>;
    return f((const float*)Ad, (const float*)Wo_d, slot, (const float*)Xo, B, T, d, H, k, Hd, (float*)Y, accumulate,
             (float*)base, part, mk, stream);
}

}  // namespace mosa
