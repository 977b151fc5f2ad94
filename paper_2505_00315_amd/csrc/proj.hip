// Gather + grouped Q/K/V projection (paper Section 2.2: X^s = X[I];
// Q = X^s W^Q, K = X^s W^K, V = X^s W^V, computed only for the k selected
// tokens of every head; a dense head is the case I = 0..T-1).
//
// One GEMM per head on the tiled MFMA engine (gemm.h): M = B*n gathered rows
// (b, i) -> token I[b,h,i], N = 3*dh (Q | K | V side by side), K = d.  The A
// rows are gathered once per thread before the K loop; the weights
// W^{Q,K,V}_h [d, dh] are n-contiguous and are transposed 8x8 in registers on
// their way into LDS.  The output is one packed row [Q | K | V] per selected
// token, so the attention kernels read each token's q, k, v from one row.
// Workgroups of one head are numbered consecutively on one XCD so the head's
// weights are fetched from HBM once into that XCD's L2.
#include "attn_lds.h"
#include "gemm.h"
#include "gemm2.h"
#include "kernels.h"
#include "rope.h"

namespace mosa {

namespace {

template <typename ST, int DH>
struct QkvPolicy {
    static constexpr int MT = 64, NT = 3 * DH, KC = sizeof(ST) == 2 ? 64 : 32, WM = 2, WN = 2;
    static constexpr size_t EPI_LDS = 0;
    static constexpr bool A_KCONTIG = true, B_KCONTIG = false, A_SCALED = false;
    struct Args {
        const ST* X;
        const int32_t* I;  // nullptr: identity (dense heads)
        const ST* W0;
        const ST* W1;
        const ST* W2;
        ST* out;  // [B, H, n, 3*DH]
        int T, d, H, n, M, mtiles;
        const float2* rope;  // rotary table [T, DH/4] or nullptr
    };
    struct ARef {
        const ST* p;
    };
    struct BRef {};
    struct RowInfo {
        int k;
    };
    __device__ static const ST* a_fallback(const Args& a) { return a.X; }
    __device__ static const ST* b_fallback(const Args& a) { return a.W0; }

    __device__ static void tile(const Args& a, int logical, int& batch, int& m0, int& n0) {
        batch = logical / a.mtiles;
        m0 = (logical % a.mtiles) * MT;
        n0 = 0;
    }
    __device__ static int k_size(const Args& a, int) { return a.d; }
    __device__ static ARef a_row(const Args& a, int h, int m, float&) {
        if (m < 0 || m >= a.M) return {nullptr};
        const int b = m / a.n, i = m % a.n;
        const int t = a.I ? a.I[((size_t)b * a.H + h) * a.n + i] : i;
        return {a.X + ((size_t)b * a.T + t) * a.d};
    }
    __device__ static const ST* a_elem(const Args&, int, const ARef& r, int k) { return r.p ? r.p + k : nullptr; }
    __device__ static BRef b_row(const Args&, int, int) { return {}; }
    __device__ static const ST* b_elem(const Args&, int, const BRef&, int) { return nullptr; }
    __device__ static RowInfo row_info(const Args&, int, int k) { return {k}; }
    __device__ static const ST* a_kaddr(const Args& a, int, const RowInfo&, int) { return a_fallback(a); }
    __device__ static bool a_kok(const Args&, int, const RowInfo&, int) { return false; }
    __device__ static float a_kscale(const Args&, int, const RowInfo&) { return 1.f; }
    // B[k][n] = W^{n / DH}_h[k][n % DH]: row k of the [d, DH] weight, n contiguous
    __device__ static const ST* b_kaddr(const Args& a, int h, const RowInfo& r, int n8) {
        const ST* W = n8 < DH ? a.W0 : (n8 < 2 * DH ? a.W1 : a.W2);
        return W + ((size_t)h * a.d + max(r.k, 0)) * DH + (n8 % DH);
    }
    __device__ static bool b_kok(const Args&, int, const RowInfo& r, int) { return r.k >= 0; }
    __device__ static void epilogue(const Args& a, int h, int m0, int, const float* Cs, int ldc, int tid, unsigned char*) {
        epilogue_rows<MT>(a, h, m0, Cs, ldc, tid);
    }
    // rows m0 .. m0 + ROWS - 1 of the C tile to their packed Q | K | V rows
    // (tab_s: the rotary rows of the tile staged by rope_stage, or nullptr)
    template <int ROWS>
    __device__ static void epilogue_rows(const Args& a, int h, int m0, const float* Cs, int ldc, int tid,
                                         const float2* tab_s = nullptr) {
        constexpr int VPR = NT / 8;  // vectors per row
        for (int v = tid; v < ROWS * VPR; v += 256) {
            const int ml = v / VPR, c = (v % VPR) * 8;
            const int m = m0 + ml;
            if (m >= a.M) continue;
            const int b = m / a.n, i = m % a.n;
            float x[8];
            cs_load8(Cs, ldc, ml, c, x);
            if (tab_s) rope_cols_at(tab_s, ml, c, x);
            else rope_cols(a, h, b, i, c, x);
            vec8_store<ST>(a.out + (((size_t)b * a.H + h) * a.n + i) * NT + c, vec8_from_f32<ST>(x));
        }
    }
    // columns c .. c + 7 of row (b, h, i): the rotary encoding of q and k
    __device__ static void rope_cols(const Args& a, int h, int b, int i, int c, float (&x)[8]) {
        if (!a.rope) return;
        const int cq = c < DH ? c : c - DH;  // column within q or k
        if (c >= 2 * DH || cq >= DH / 2) return;
        const int pos = a.I ? a.I[((size_t)b * a.H + h) * a.n + i] : i;
        rope8<DH>(x, cq, a.rope, pos, 1.f);
    }
    // the same from a staged table row (row ml of the tile)
    __device__ static void rope_cols_at(const float2* tab_s, int ml, int c, float (&x)[8]) {
        const int cq = c < DH ? c : c - DH;
        if (c >= 2 * DH || cq >= DH / 2) return;
        rope8<DH>(x, cq, tab_s, ml, 1.f);
    }
    // The (cos, sin) rows of the tile's ROWS rows (positions I, or i for dense
    // heads; rows past M take the last row's) into LDS, all loads issued
    // before any is used; ends with a barrier.
    template <int ROWS>
    __device__ static void rope_stage(const Args& a, int h, int m0, int tid, float2* tab_s) {
        constexpr int Q4 = DH / 8, PER = ROWS * Q4 / 256;  // float4 units per row / per thread
        static_assert(ROWS * Q4 % 256 == 0, "table tile");
        float4 t[PER];
#pragma unroll
        for (int j = 0; j < PER; ++j) {
            const int e = tid + 256 * j, ml = e / Q4, q4 = e % Q4, m = min(m0 + ml, a.M - 1);
            const int b = m / a.n, i = m % a.n;
            const int pos = a.I ? a.I[((size_t)b * a.H + h) * a.n + i] : i;
            t[j] = reinterpret_cast<const float4*>(a.rope + (size_t)pos * (DH / 4))[q4];
        }
#pragma unroll
        for (int j = 0; j < PER; ++j) reinterpret_cast<float4*>(tab_s)[tid + 256 * j] = t[j];
        __syncthreads();
    }
};

// bf16 storage: the multi-stage engine with direct-to-LDS loads (gemm2.h).
// A: gathered token rows (k-contiguous, clamped to the last row past M);
// B: the three weights as one m-contiguous [d][3 DH] operand.
template <int DH, int MT_ = 128>
struct QkvPolicy2 {
    using ST = uint16_t;
    static constexpr int MT = MT_, NT = 3 * DH, KC = DH == 64 ? 32 : 64, WM = 2, WN = 2, STAGES = 4;
    static constexpr size_t TAB_LDS = (size_t)MT * (DH / 4) * 8;  // staged rotary rows
    static constexpr size_t EPI_LDS = TAB_LDS;
    static constexpr bool A_KCONTIG = true, B_KCONTIG = false;
    using Args = typename QkvPolicy<ST, DH>::Args;
    struct ARef {
        const ST* p;
    };
    static int mtiles(int M) { return (M + MT - 1) / MT; }
    __device__ static void tile(const Args& a, int logical, int& batch, int& m0, int& n0) {
        const int mt = (a.M + MT - 1) / MT;
        if (a.I) {  // a head's row tiles side by side: they share its weights
            batch = logical / mt;
            m0 = (logical % mt) * MT;
        } else {  // dense heads: the heads of a row tile side by side (its X rows)
            batch = logical % a.H;
            m0 = (logical / a.H) * MT;
        }
        n0 = 0;
    }
    __device__ static int k_size(const Args& a, int) { return a.d; }
    __device__ static ARef a_row(const Args& a, int h, int m) {
        m = min(m, a.M - 1);
        const int b = m / a.n, i = m % a.n;
        const int t = a.I ? a.I[((size_t)b * a.H + h) * a.n + i] : i;
        return {a.X + ((size_t)b * a.T + t) * a.d};
    }
    __device__ static const ST* a_elem(const Args&, int, const ARef& r, int k) { return r.p + k; }
    __device__ static size_t b_kstride(const Args&, int) { return DH; }
    // B[k][n] = W^{n / DH}_h[k][n % DH]
    __device__ static const ST* b_maddr(const Args& a, int h, int k, int n8) {
        const ST* W = n8 < DH ? a.W0 : (n8 < 2 * DH ? a.W1 : a.W2);
        return W + ((size_t)h * a.d + k) * DH + (n8 % DH);
    }
    __device__ static void epilogue(const Args& a, int h, int m0, int, const float* Cs, int ldc, int tid,
                                    unsigned char* extra) {
        float2* tab_s = nullptr;
        if (a.rope) {
            tab_s = reinterpret_cast<float2*>(extra);
            QkvPolicy<ST, DH>::template rope_stage<MT>(a, h, m0, tid, tab_s);
        }
        QkvPolicy<ST, DH>::template epilogue_rows<MT>(a, h, m0, Cs, ldc, tid, tab_s);
    }
};

// QKV projection and attention in one kernel, for groups of n | 128 rows
// (n = 16, 32, 64 or 128): every 128-row tile holds whole (b, h) groups, so
// after the epilogue has written the packed Q | K | V rows (kept for the
// backward pass), the same workgroup copies the tile's K and V in bf16 into
// LDS, takes Q from the C tile, and runs the attention of its groups
// (attn_lds.h, bit-identical to the separate attention kernel).
template <int DH, int MT_ = 128>
struct QkvAttnPolicy : QkvPolicy2<DH, MT_> {
    using ST = uint16_t;
    using Base = QkvPolicy2<DH, MT_>;
    static constexpr int MT = Base::MT, U = DH / 8, KROWS = MT, VROWS = MT + 16;
    // bf16 K tile, then the V tile with 16 zero rows after it (the last
    // group's odd key block reads 16 rows past its end, at weight zero)
    static constexpr size_t KV_LDS = (size_t)(KROWS + VROWS) * DH * 2;
    static constexpr size_t EPI_LDS = KV_LDS + Base::TAB_LDS;  // then the staged rotary rows
    static_assert((MT == 128 || MT == 64) && Base::WM * Base::WN == 4, "one or two query blocks per wave");
    static constexpr int QBW = MT / 64;  // query blocks of 16 rows per wave
    struct Args : QkvPolicy<ST, DH>::Args {
        const float* r;  // [B, H, n] router weights of the selected rows
        ST* A;           // [B, H, n, DH]
        float* lse;      // [B, H, n]
        int causal;
        float scale;
    };
    __device__ static void epilogue(const Args& a, int h, int m0, int, const float* Cs, int ldc, int tid,
                                    unsigned char* extra) {
        constexpr int VPR = 3 * U;  // 16-byte vectors per packed row
        unsigned char* Ks = extra;
        unsigned char* Vs = extra + (size_t)KROWS * DH * 2;
        float2* tab_s = reinterpret_cast<float2*>(extra + KV_LDS);
        if (a.rope) QkvPolicy<ST, DH>::template rope_stage<MT>(a, h, m0, tid, tab_s);
        for (int v = tid; v < MT * VPR; v += 256) {
            const int ml = v / VPR, u = v % VPR, m = m0 + ml;
            float x[8];
            cs_load8(Cs, ldc, ml, 8 * u, x);
            if (a.rope && u < 2 * U) {
                // rotated q stays in the C tile for the attention below
                QkvPolicy<ST, DH>::rope_cols_at(tab_s, ml, 8 * u, x);
                if (u < U) {  // the C tile is this workgroup's LDS; each vector has one owner
                    float* cq = const_cast<float*>(Cs) + ml * ldc + 8 * u;
                    *reinterpret_cast<float4*>(cq) = make_float4(x[0], x[1], x[2], x[3]);
                    *reinterpret_cast<float4*>(cq + 4) = make_float4(x[4], x[5], x[6], x[7]);
                }
            }
            const uint4 y = vec8_from_f32<ST>(x).v;
            if (m < a.M) {
                const int b = m / a.n, i = m % a.n;
                *reinterpret_cast<uint4*>(a.out + (((size_t)b * a.H + h) * a.n + i) * (3 * DH) + 8 * u) = y;
            }
            // rows past M hold the clamped last row's values: finite, never used
            if (u >= 2 * U)
                *reinterpret_cast<uint4*>(Vs + (ml * U + ((u - 2 * U) ^ vt_swz<U>(ml))) * 16) = y;
            else if (u >= U)
                *reinterpret_cast<uint4*>(Ks + (ml * U + ((u - U) ^ kswz(ml, U))) * 16) = y;
        }
        for (int v = tid; v < (VROWS - MT) * U; v += 256)
            *reinterpret_cast<uint4*>(Vs + (size_t)(MT * U + v) * 16) = make_uint4(0, 0, 0, 0);
        __syncthreads();

        // MT / 16 query blocks over 4 waves: 128 rows, blocks w and 7 - w, so
        // that every wave's causal key blocks add up to the same count; 64
        // rows, block w
        const int wave = tid >> 6, lane = tid & 63, g = lane >> 4, c16 = lane & 15;
        const int n = a.n, nqb = n / 16;
        for (int j2 = 0; j2 < QBW; ++j2) {
            const int j = j2 ? 7 - wave : wave, gi = j / nqb, qb = j % nqb, mg = m0 + gi * n;
            if (mg >= a.M) continue;
            const size_t bh = (size_t)(mg / n) * a.H + h;
            Frag8<ST> qf[DH / 32];
#pragma unroll
            for (int st = 0; st < DH / 32; ++st) {
                float x[8];
                cs_load8(Cs, ldc, gi * n + 16 * qb + c16, 32 * st + 8 * g, x);
                qf[st] = frag8_from<ST>(x);
            }
            attn_lds_block<DH>(Ks, Vs, gi * n, qf, n, a.causal, a.scale, qb, a.r ? a.r + bh * n : nullptr,
                               a.A + bh * n * DH, a.lse + bh * n);
        }
    }
};

template <typename ST, int DH>
int run(const ST* X, const int32_t* I, const ST* Wq, const ST* Wk, const ST* Wv, int B, int T, int d, int H, int n,
        ST* out, const float2* rope, int narrow, hipStream_t stream) {
    using P = QkvPolicy<ST, DH>;
    typename P::Args a{X, I, Wq, Wk, Wv, out, T, d, H, n, B * n, (B * n + P::MT - 1) / P::MT, rope};
    if constexpr (sizeof(ST) == 2) {
        using N2 = QkvPolicy2<DH, 64>;
        if (narrow && d % N2::KC == 0) return launch_gemm2<N2>(a, N2::mtiles(B * n) * H, stream);
        if (d % QkvPolicy2<DH>::KC == 0) return launch_gemm2<QkvPolicy2<DH>>(a, QkvPolicy2<DH>::mtiles(B * n) * H, stream);
    }
    return launch_gemm<ST, P>(a, a.mtiles * H, stream);
}

}  // namespace

int launch_qkv_attn(int dtype, const void* X, const int32_t* I, const void* Wq, const void* Wk, const void* Wv,
                    int B, int T, int d, int H, int dh, int n, void* QKV, const float2* rope, const float* r,
                    int causal, void* A, float* lse, hipStream_t stream) {
    if (dtype != kBF16 || n < 16 || n % 16 || 128 % n || (dh != 64 && dh != 32)) return 1;
    const float scale = 1.0f / sqrtf((float)dh);
    auto go = [&](auto tag, auto mt) {
        constexpr int DH = decltype(tag)::value;
        using P = QkvAttnPolicy<DH, decltype(mt)::value>;
        if (d % P::KC) return 1;
        typename P::Args a{};
        static_cast<typename QkvPolicy<uint16_t, DH>::Args&>(a) = {
            (const uint16_t*)X, I, (const uint16_t*)Wq, (const uint16_t*)Wk, (const uint16_t*)Wv, (uint16_t*)QKV,
            T, d, H, n, B * n, 0, rope};
        a.r = r;
        a.A = (uint16_t*)A;
        a.lse = lse;
        a.causal = causal;
        a.scale = scale;
        return launch_gemm2<P>(a, P::mtiles(B * n) * H, stream);
    };
    // at most 64 rows per head (B n <= 64): 64-row tiles instead of half-empty
    // 128-row ones (measured equal or slower for more rows)
    if ((long long)B * n <= 64)
        return dh == 64 ? go(std::integral_constant<int, 64>{}, std::integral_constant<int, 64>{})
                        : go(std::integral_constant<int, 32>{}, std::integral_constant<int, 64>{});
    return dh == 64 ? go(std::integral_constant<int, 64>{}, std::integral_constant<int, 128>{})
                    : go(std::integral_constant<int, 32>{}, std::integral_constant<int, 128>{});
}

int launch_qkv(int dtype, const void* X, const int32_t* I, const void* Wq, const void* Wk, const void* Wv, int B,
               int T, int d, int H, int dh, int n, void* QKV, const float2* rope, int narrow, hipStream_t stream) {
    if (dtype == kBF16) {
        auto f = dh == 64 ? run<uint16_t, 64> : run<uint16_t, 32>;
        return f((const uint16_t*)X, I, (const uint16_t*)Wq, (const uint16_t*)Wk, (const uint16_t*)Wv, B, T, d, H, n,
                 (uint16_t*)QKV, rope, narrow, stream);
    }
    auto f = dh == 64 ? run<float, 64> : run<float, 32>;
    return f((const float*)X, I, (const float*)Wq, (const float*)Wk, (const float*)Wv, B, T, d, H, n, (float*)QKV,
             rope, 0, stream);
}

}  // namespace mosa
