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
// in order, so the sums are bitwise reproducible.  When there are too few
// (head, tile) pairs to fill the chip the rows are split into S contiguous
// ranges: each workgroup writes an fp32 partial tile and a second kernel adds
// the S partials in range order (still reproducible).
#include <algorithm>

#include "dxrow.h"
#include "gemm.h"
#include "gemm2.h"
#include "group.h"
#include "kernels.h"

namespace mosa {

namespace {

template <typename ST, int DH, bool ROUTER, bool GATHER>
struct WgradQkvPolicy {
    static constexpr int MT = 64, NT = 3 * DH + (ROUTER ? 16 : 0), KC = sizeof(ST) == 2 ? 64 : 32, WM = 4, WN = 1;
    static constexpr size_t EPI_LDS = 0;
    static constexpr bool A_KCONTIG = false, B_KCONTIG = false, A_SCALED = false, SPLITK = true;
    struct Args {
        const ST* X;
        const int32_t* I;
        const ST* dQKV;  // [B, H, n, 3*DH]
        const ST* dz16;  // [B, H, n, 16]
        ST* dWq;
        ST* dWk;
        ST* dWv;         // [H, d, DH]
        ST* dWr;         // [H, d]
        float* part;     // [S, H, d, NT] fp32 partial sums (S > 1)
        int T, d, H, n, R, mtiles, S, cps;
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
    __device__ static void tile_split(const Args& a, int logical, int& h, int& m0, int& n0, int& split) {
        const int per = a.H * a.mtiles;
        split = logical / per;
        const int rem = logical % per;
        h = rem / a.mtiles;
        m0 = (rem % a.mtiles) * MT;
        n0 = 0;
    }
    __device__ static void k_range(const Args& a, int split, int K, int& kbeg, int& kend) {
        kbeg = split * a.cps * KC;
        kend = min(K, kbeg + a.cps * KC);
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
    __device__ static void epilogue_split(const Args& a, int h, int split, int m0, int n0, const float* Cs, int ldc,
                                          int tid) {
        if (a.S == 1) {
            epilogue(a, h, m0, n0, Cs, ldc, tid, nullptr);
            return;
        }
        constexpr int VPR = NT / 4;  // float4 per row
        for (int v = tid; v < MT * VPR; v += 256) {
            const int ml = v / VPR, nn = (v % VPR) * 4;
            const int c = m0 + ml;
            if (c >= a.d) continue;
            const float4 x = *reinterpret_cast<const float4*>(Cs + ml * ldc + nn);
            *reinterpret_cast<float4*>(a.part + (((size_t)split * a.H + h) * a.d + c) * NT + nn) = x;
        }
    }
};

// Sum of the S partial tiles in split order, then the final stores.
template <typename ST, int DH, bool ROUTER>
__global__ __launch_bounds__(256) void wgrad_qkv_reduce_kernel(const float* __restrict__ part, int S, int H, int d,
                                                               ST* dWq, ST* dWk, ST* dWv, ST* dWr) {
    constexpr int NT = 3 * DH + (ROUTER ? 16 : 0);
    constexpr int G = 3 * DH / 8 + (ROUTER ? 1 : 0);  // 8-column groups written
    const int idx = blockIdx.x * 256 + threadIdx.x;
    if (idx >= H * d * G) return;
    const int gq = idx % G, hc = idx / G;  // hc = h * d + c
    float x[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    for (int sp = 0; sp < S; ++sp) {
        const float* p = part + ((size_t)sp * H * d + hc) * NT + gq * 8;
        const float4 u = reinterpret_cast<const float4*>(p)[0], w = reinterpret_cast<const float4*>(p)[1];
        x[0] += u.x; x[1] += u.y; x[2] += u.z; x[3] += u.w;
        x[4] += w.x; x[5] += w.y; x[6] += w.z; x[7] += w.w;
    }
    const int nn = gq * 8;
    if (nn < 3 * DH) {
        ST* W = nn < DH ? dWq : (nn < 2 * DH ? dWk : dWv);
        vec8_store<ST>(W + (size_t)hc * DH + (nn % DH), vec8_from_f32<ST>(x));
    } else {
        st1<ST>(dWr + hc, x[0]);
    }
}

template <typename ST, int DH, bool GATHER>
struct WgradOPolicy {
    static constexpr int MT = DH, NT = 128, KC = sizeof(ST) == 2 ? 64 : 32, WM = 2, WN = 2;
    static constexpr size_t EPI_LDS = 0;
    static constexpr bool A_KCONTIG = false, B_KCONTIG = false, A_SCALED = false, SPLITK = true;
    struct Args {
        const ST* dY;
        const int32_t* I;
        const ST* A;      // [B, H, n, DH], rows scaled by r
        ST* dWo;          // [H, DH, d]
        float* part;      // [S, H, DH, d] fp32 partial sums (S > 1)
        int T, d, H, n, R, ntiles, S, cps;
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
    __device__ static void tile_split(const Args& a, int logical, int& h, int& m0, int& n0, int& split) {
        const int per = a.H * a.ntiles;
        split = logical / per;
        const int rem = logical % per;
        h = rem / a.ntiles;
        m0 = 0;
        n0 = (rem % a.ntiles) * NT;
    }
    __device__ static void k_range(const Args& a, int split, int K, int& kbeg, int& kend) {
        kbeg = split * a.cps * KC;
        kend = min(K, kbeg + a.cps * KC);
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
    __device__ static void epilogue_split(const Args& a, int h, int split, int m0, int n0, const float* Cs, int ldc,
                                          int tid) {
        if (a.S == 1) {
            epilogue(a, h, m0, n0, Cs, ldc, tid, nullptr);
            return;
        }
        constexpr int VPR = NT / 4;
        for (int v = tid; v < MT * VPR; v += 256) {
            const int e = v / VPR, c = (v % VPR) * 4;
            if (n0 + c >= a.d) continue;
            const float4 x = *reinterpret_cast<const float4*>(Cs + e * ldc + c);
            *reinterpret_cast<float4*>(a.part + (((size_t)split * a.H + h) * DH + e) * a.d + n0 + c) = x;
        }
    }
};

template <typename ST>
__global__ __launch_bounds__(256) void wgrad_o_reduce_kernel(const float* __restrict__ part, int S, size_t n8,
                                                             ST* dWo) {
    const size_t idx = (size_t)blockIdx.x * 256 + threadIdx.x;
    if (idx >= n8) return;
    float x[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    for (int sp = 0; sp < S; ++sp) {
        const float* p = part + ((size_t)sp * n8 + idx) * 8;
        const float4 u = reinterpret_cast<const float4*>(p)[0], w = reinterpret_cast<const float4*>(p)[1];
        x[0] += u.x; x[1] += u.y; x[2] += u.z; x[3] += u.w;
        x[4] += w.x; x[5] += w.y; x[6] += w.z; x[7] += w.w;
    }
    vec8_store<ST>(dWo + idx * 8, vec8_from_f32<ST>(x));
}

// bf16 storage, MoSA heads: the multi-stage engine (gemm2.h) with the rows
// gathered through an LDS table, k = r in order over the whole range (no
// split: one workgroup owns its output tile, so the sums are reproducible
// without partials).  Table entry of row r = (b, i): x = b T + I_r (the
// token row of X or dY), y = (b H + h) n + i (the selected-row index), y = -1
// past the last row (that operand then reads zeros).  The MFMA's A operand
// is the one whose output index is contiguous in memory, interleaved so the
// accumulators go straight to 16-byte stores.
__device__ __forceinline__ int2 wgrad_k_row(const int32_t* I, const FastDiv& nd, int T, int H, int n, int h, int k,
                                            int K) {
    int b, i;
    fast_divmod(nd, min(k, K - 1), b, i);
    const int ri = (b * H + h) * n + i;
    return make_int2(b * T + I[ri], k < K ? ri : -1);
}

// dW^{Q,K,V}_h and dW^r_h: M = the 3 dh + 64 output columns [dQ | dK | dV |
// dz, 0 ...] (dz16 holds dz and 15 zeros; the rest reads the zero row),
// N = 64 rows c of d per workgroup.
template <int DH>
struct WgradQkvPolicy2 {
    using ST = uint16_t;
    static constexpr int MT = DH == 64 ? 256 : 128, NT = 64, KC = 32, WM = 2, WN = 2, STAGES = 3;
    static constexpr size_t EPI_LDS = 0;
    static constexpr bool A_KCONTIG = false, B_KCONTIG = false, KGATHER = true, A_INTERLEAVE = true, EPI_REGS = true;
    static constexpr int A_TAB = 1, B_TAB = 0, MIN_WAVES = 2;
    using Args = typename WgradQkvPolicy<ST, DH, true, true>::Args;
    __device__ static void tile(const Args& a, int logical, int& h, int& m0, int& n0) {
        h = logical / a.mtiles;
        m0 = 0;
        n0 = (logical % a.mtiles) * NT;
    }
    __device__ static int k_size(const Args& a, int) { return a.R; }
    __device__ static int2 k_row(const Args& a, int h, int k, int K) {
        return wgrad_k_row(a.I, a.nd, a.T, a.H, a.n, h, k, K);
    }
    __device__ static void a_mlane(const Args& a, int, int m8, const ST*& base, uint32_t& stride) {
        if (m8 < 3 * DH) {
            base = a.dQKV + m8;
            stride = 3 * DH;
        } else if (m8 < 3 * DH + 16) {
            base = a.dz16 + (m8 - 3 * DH);
            stride = 16;
        } else {
            base = g2_zero;
            stride = 0;
        }
    }
    __device__ static void b_mlane(const Args& a, int, int n8, const ST*& base, uint32_t& stride) {
        base = a.X + n8;
        stride = a.d;
    }
    // columns m .. m + 7 of row c = n
    __device__ static void store8(const Args& a, int h, int m, int n, const float (&x)[8]) {
        if (m < 3 * DH) {
            ST* W = m < DH ? a.dWq : (m < 2 * DH ? a.dWk : a.dWv);
            vec8_store<ST>(W + ((size_t)h * a.d + n) * DH + (m % DH), vec8_from_f32<ST>(x));
        } else if (m == 3 * DH) {
            st1<ST>(a.dWr + (size_t)h * a.d + n, x[0]);
        }
    }
};

// dW^O_h: M = 64 columns c of d per workgroup (dY rows), N = dh (the scaled
// attention rows).
template <int DH>
struct WgradOPolicy2 {
    using ST = uint16_t;
    static constexpr int MT = 64, NT = DH, KC = 64, WM = 2, WN = 2, STAGES = 4;
    static constexpr size_t EPI_LDS = 0;
    static constexpr bool A_KCONTIG = false, B_KCONTIG = false, KGATHER = true, A_INTERLEAVE = true, EPI_REGS = true;
    static constexpr int A_TAB = 0, B_TAB = 1;
    using Args = typename WgradOPolicy<ST, DH, true>::Args;
    __device__ static void tile(const Args& a, int logical, int& h, int& m0, int& n0) {
        h = logical / a.ntiles;
        m0 = (logical % a.ntiles) * MT;
        n0 = 0;
    }
    __device__ static int k_size(const Args& a, int) { return a.R; }
    __device__ static int2 k_row(const Args& a, int h, int k, int K) {
        return wgrad_k_row(a.I, a.nd, a.T, a.H, a.n, h, k, K);
    }
    __device__ static void a_mlane(const Args& a, int, int m8, const ST*& base, uint32_t& stride) {
        base = a.dY + m8;
        stride = a.d;
    }
    __device__ static void b_mlane(const Args& a, int, int n8, const ST*& base, uint32_t& stride) {
        base = a.A + n8;
        stride = DH;
    }
    // columns c = m .. m + 7 of row e = n
    __device__ static void store8(const Args& a, int h, int m, int n, const float (&x)[8]) {
        vec8_store<ST>(a.dWo + ((size_t)h * DH + n) * a.d + m, vec8_from_f32<ST>(x));
    }
};

// Dense heads (bf16) on the same engine: R = B T rows split into S ranges of
// up to 4096 rows (the row table), one fp32 partial tile per range, summed in
// range order by the reduce kernels.  "batch" = h S + s.  Row r of range s:
// x = r' = s KS + r (the row of X or dY), y = (b Hd + h) T + t (the head's
// row), y = -1 past the range.
__device__ __forceinline__ int2 wgrad_dense_k_row(const FastDiv& Td, int R, int KS, int T, int H, int batch, int S,
                                                  int k, int K) {
    const int h = batch / S, s = batch % S, r = min(s * KS + min(k, K - 1), R - 1);
    int b, t;
    fast_divmod(Td, r, b, t);
    return make_int2(r, k < K ? (b * H + h) * T + t : -1);
}

template <int DH>
struct WgradQkvDensePolicy2 : WgradQkvPolicy2<DH> {
    using ST = uint16_t;
    static constexpr int MT = DH == 64 ? 192 : 128;  // [dQ | dK | dV] (DH 32: zero rows past 96)
    using Args = typename WgradQkvPolicy2<DH>::Args;  // I unused, cps = rows per range
    __device__ static void tile(const Args& a, int logical, int& batch, int& m0, int& n0) {
        // the heads of one (row range, column tile) side by side (its X block)
        const int h = logical % a.H, rest = logical / a.H;
        batch = h * a.S + rest / a.mtiles;  // h S + s
        m0 = 0;
        n0 = (rest % a.mtiles) * WgradQkvPolicy2<DH>::NT;
    }
    __device__ static int k_size(const Args& a, int batch) { return min(a.cps, a.R - (batch % a.S) * a.cps); }
    __device__ static int2 k_row(const Args& a, int batch, int k, int K) {
        return wgrad_dense_k_row(a.nd, a.R, a.cps, a.T, a.H, batch, a.S, k, K);
    }
    __device__ static void a_mlane(const Args& a, int, int m8, const ST*& base, uint32_t& stride) {
        if (m8 < 3 * DH) {
            base = a.dQKV + m8;
            stride = 3 * DH;
        } else {
            base = g2_zero;
            stride = 0;
        }
    }
    __device__ static void b_mlane(const Args& a, int, int n8, const ST*& base, uint32_t& stride) {
        base = a.X + n8;
        stride = a.d;
    }
    // fp32 partial: part[s][h][c][3 DH], columns m .. m + 7 of row c = n
    __device__ static void store8(const Args& a, int batch, int m, int n, const float (&x)[8]) {
        if (m >= 3 * DH) return;
        const int h = batch / a.S, s = batch % a.S;
        float* p = a.part + (((size_t)s * a.H + h) * a.d + n) * (3 * DH) + m;
        reinterpret_cast<float4*>(p)[0] = make_float4(x[0], x[1], x[2], x[3]);
        reinterpret_cast<float4*>(p)[1] = make_float4(x[4], x[5], x[6], x[7]);
    }
};

template <int DH>
struct WgradODensePolicy2 : WgradOPolicy2<DH> {
    using ST = uint16_t;
    using Args = typename WgradOPolicy2<DH>::Args;  // I unused, cps = rows per range
    __device__ static void tile(const Args& a, int logical, int& batch, int& m0, int& n0) {
        // the heads of one (row range, column tile) side by side (its dY block)
        const int h = logical % a.H, rest = logical / a.H;
        batch = h * a.S + rest / a.ntiles;  // h S + s
        m0 = (rest % a.ntiles) * WgradOPolicy2<DH>::MT;
        n0 = 0;
    }
    __device__ static int k_size(const Args& a, int batch) { return min(a.cps, a.R - (batch % a.S) * a.cps); }
    __device__ static int2 k_row(const Args& a, int batch, int k, int K) {
        return wgrad_dense_k_row(a.nd, a.R, a.cps, a.T, a.H, batch, a.S, k, K);
    }
    // fp32 partial: part[s][h][e][c], columns c = m .. m + 7 of row e = n
    __device__ static void store8(const Args& a, int batch, int m, int n, const float (&x)[8]) {
        const int h = batch / a.S, s = batch % a.S;
        float* p = a.part + (((size_t)s * a.H + h) * DH + n) * a.d + m;
        reinterpret_cast<float4*>(p)[0] = make_float4(x[0], x[1], x[2], x[3]);
        reinterpret_cast<float4*>(p)[1] = make_float4(x[4], x[5], x[6], x[7]);
    }
};

// Row ranges of the dense-head split: about one workgroup per CU (256 for
// `tiles` output tiles per range), each range at most 4096 rows.  Fewer
// ranges mean fewer fp32 partials to write and sum; with 4 dense heads,
// d = 1024 and B T = 8192 rows, 4 ranges beat 2 and 8 (the hybrid layer's
// step: 0.428, 0.406 and 0.410 ms cold), 16 were slower still.
inline int dense_ranges(int R, int tiles, int kc, int& rows) {
    int S = std::max(1, (256 + tiles - 1) / tiles);
    S = std::max(S, (R + 4095) / 4096);
    rows = (R + S - 1) / S;
    rows = (rows + kc - 1) / kc * kc;
    if (rows > 4096) return 0;
    return (R + rows - 1) / rows;
}

// Rows of the k-row table for a gathered range of R rows (0: not usable).
template <class P2>
int wgrad2_table_rows(int R, int d) {
    const int rows = (R + P2::KC - 1) / P2::KC * P2::KC;
    if (R <= 0 || rows > 4096 || d % 64 != 0) return 0;
    return rows;
}

// Split of the row range: enough workgroups to fill the chip (about 512),
// at least 4 chunks per split.
int choose_splits(int base_tiles, int nchunks, int& cps) {
    int sp = (512 + base_tiles - 1) / base_tiles;
    sp = std::min(sp, std::max(1, nchunks / 4));
    sp = std::max(1, std::min(sp, 64));
    cps = (nchunks + sp - 1) / sp;
    return nchunks > 0 ? (nchunks + cps - 1) / cps : 1;
}

// Stage names of the weight-gradient kernels (MoSA heads / dense heads).
inline const char* wname(bool dense, int which, bool reduce) {
    static const char* const names[2][2][2] = {
        {{"wgrad_qkv", "wgrad_qkv_reduce"}, {"wgrad_o", "wgrad_o_reduce"}},
        {{"wgrad_qkv_dense", "wgrad_qkv_dense_reduce"}, {"wgrad_o_dense", "wgrad_o_dense_reduce"}}};
    return names[dense][which][reduce];
}

template <typename ST, int DH, bool ROUTER, bool GATHER>
int run_qkv_t(const ST* X, const int32_t* I, const ST* dQKV, const ST* dz16, int B, int T, int d, int H, int n,
              ST* dWq, ST* dWk, ST* dWv, ST* dWr, float* part, const Marker& mk, hipStream_t stream) {
    using P = WgradQkvPolicy<ST, DH, ROUTER, GATHER>;
    const bool dense = !GATHER;
    const int mtiles = (d + P::MT - 1) / P::MT, R = B * n;
    if constexpr (sizeof(ST) == 2 && ROUTER && GATHER) {
        using P2 = WgradQkvPolicy2<DH>;
        if (const int rows = wgrad2_table_rows<P2>(R, d)) {
            typename P::Args a{X, I, dQKV, dz16, dWq, dWk, dWv, dWr, part, T, d, H, n, R, d / 64, 1, 0, make_fastdiv(n)};
            return launch_gemm2<P2>(a, H * (d / 64), stream, rows) | mk(wname(dense, 0, false));
        }
    }
    if constexpr (sizeof(ST) == 2 && !ROUTER && !GATHER) {
        using P2 = WgradQkvDensePolicy2<DH>;
        int rows;
        const int S = dense_ranges(R, H * (d / 64), P2::KC, rows);
        if (S > 0 && d % 64 == 0) {
            typename P2::Args a{X, I, dQKV, dz16, dWq, dWk, dWv, dWr, part, T, d, H, n, R, d / 64, S, rows,
                                make_fastdiv(n)};
            int e = launch_gemm2<P2>(a, S * H * (d / 64), stream, rows);
            e |= mk(wname(dense, 0, false));
            if (e == 0) {
                const int total = H * d * (3 * DH / 8);
                hipLaunchKernelGGL((wgrad_qkv_reduce_kernel<ST, DH, false>), dim3((total + 255) / 256), dim3(256), 0,
                                   stream, part, S, H, d, dWq, dWk, dWv, dWr);
                e = hipGetLastError() == hipSuccess ? 0 : -1;
                e |= mk(wname(dense, 0, true));
            }
            return e;
        }
    }
    int cps;
    const int S = choose_splits(H * mtiles, (R + P::KC - 1) / P::KC, cps);
    typename P::Args a{X, I, dQKV, dz16, dWq, dWk, dWv, dWr, part, T, d, H, n, R, mtiles, S, cps, make_fastdiv(n)};
    int e = launch_gemm<ST, P>(a, S * H * mtiles, stream);
    e |= mk(wname(dense, 0, false));
    if (S > 1 && e == 0) {
        const int total = H * d * (3 * DH / 8 + (ROUTER ? 1 : 0));
        hipLaunchKernelGGL((wgrad_qkv_reduce_kernel<ST, DH, ROUTER>), dim3((total + 255) / 256), dim3(256), 0, stream,
                           part, S, H, d, dWq, dWk, dWv, dWr);
        e = hipGetLastError() == hipSuccess ? 0 : -1;
        e |= mk(wname(dense, 0, true));
    }
    return e;
}

template <typename ST, int DH>
int run_qkv(const ST* X, const int32_t* I, const ST* dQKV, const ST* dz16, int B, int T, int d, int H, int n, ST* dWq,
            ST* dWk, ST* dWv, ST* dWr, float* part, const Marker& mk, hipStream_t stream) {
    if (I)  // MoSA heads: gathered rows and the router column
        return run_qkv_t<ST, DH, true, true>(X, I, dQKV, dz16, B, T, d, H, n, dWq, dWk, dWv, dWr, part, mk, stream);
    return run_qkv_t<ST, DH, false, false>(X, I, dQKV, dz16, B, T, d, H, n, dWq, dWk, dWv, dWr, part, mk, stream);
}

template <typename ST, int DH, bool GATHER>
int run_o_t(const ST* dY, const int32_t* I, const ST* A, int B, int T, int d, int H, int n, ST* dWo, float* part,
            const Marker& mk, hipStream_t stream) {
    using P = WgradOPolicy<ST, DH, GATHER>;
    const bool dense = !GATHER;
    const int ntiles = (d + P::NT - 1) / P::NT, R = B * n;
    if constexpr (sizeof(ST) == 2 && GATHER) {
        using P2 = WgradOPolicy2<DH>;
        if (const int rows = wgrad2_table_rows<P2>(R, d)) {
            typename P::Args a{dY, I, A, dWo, part, T, d, H, n, R, d / 64, 1, 0, make_fastdiv(n)};
            return launch_gemm2<P2>(a, H * (d / 64), stream, rows) | mk(wname(dense, 1, false));
        }
    }
    if constexpr (sizeof(ST) == 2 && !GATHER) {
        using P2 = WgradODensePolicy2<DH>;
        int rows;
        const int S = dense_ranges(R, H * (d / 64), P2::KC, rows);
        if (S > 0 && d % 64 == 0) {
            typename P2::Args a{dY, I, A, dWo, part, T, d, H, n, R, d / 64, S, rows, make_fastdiv(n)};
            int e = launch_gemm2<P2>(a, S * H * (d / 64), stream, rows);
            e |= mk(wname(dense, 1, false));
            if (e == 0) {
                const size_t n8 = (size_t)H * DH * d / 8;
                hipLaunchKernelGGL((wgrad_o_reduce_kernel<ST>), dim3((unsigned)((n8 + 255) / 256)), dim3(256), 0,
                                   stream, part, S, n8, dWo);
                e = hipGetLastError() == hipSuccess ? 0 : -1;
                e |= mk(wname(dense, 1, true));
            }
            return e;
        }
    }
    int cps;
    const int S = choose_splits(H * ntiles, (R + P::KC - 1) / P::KC, cps);
    typename P::Args a{dY, I, A, dWo, part, T, d, H, n, R, ntiles, S, cps, make_fastdiv(n)};
    int e = launch_gemm<ST, P>(a, S * H * ntiles, stream);
    e |= mk(wname(dense, 1, false));
    if (S > 1 && e == 0) {
        const size_t n8 = (size_t)H * DH * d / 8;
        hipLaunchKernelGGL((wgrad_o_reduce_kernel<ST>), dim3((unsigned)((n8 + 255) / 256)), dim3(256), 0, stream, part,
                           S, n8, dWo);
        e = hipGetLastError() == hipSuccess ? 0 : -1;
        e |= mk(wname(dense, 1, true));
    }
    return e;
}

template <typename ST, int DH>
int run_o(const ST* dY, const int32_t* I, const ST* A, int B, int T, int d, int H, int n, ST* dWo, float* part,
          const Marker& mk, hipStream_t stream) {
    if (I) return run_o_t<ST, DH, true>(dY, I, A, B, T, d, H, n, dWo, part, mk, stream);
    return run_o_t<ST, DH, false>(dY, I, A, B, T, d, H, n, dWo, part, mk, stream);
}

// dW^{Q,K,V,r} and dW^O of the MoSA heads in one launch of the gathered-row
// engine (the two kinds of workgroups share the CUs); 1: not applicable.
template <int DH>
int run_both(const uint16_t* X, const uint16_t* dY, const int32_t* I, const uint16_t* A, const uint16_t* dQKV,
             const uint16_t* dz16, int B, int T, int d, int H, int n, uint16_t* dWq, uint16_t* dWk, uint16_t* dWv,
             uint16_t* dWr, uint16_t* dWo, hipStream_t stream) {
    using ST = uint16_t;
    using PQ = WgradQkvPolicy2<DH>;
    using PO = WgradOPolicy2<DH>;
    const int R = B * n;
    const int rq = wgrad2_table_rows<PQ>(R, d), ro = wgrad2_table_rows<PO>(R, d);
    if (!rq || !ro) return 1;
    typename PQ::Args aq{X, I, dQKV, dz16, dWq, dWk, dWv, dWr, nullptr, T, d, H, n, R, d / 64, 1, 0, make_fastdiv(n)};
    typename PO::Args ao{dY, I, A, dWo, nullptr, T, d, H, n, R, d / 64, 1, 0, make_fastdiv(n)};
    const int e = launch_gemm2_dual<PQ, PO>(aq, H * (d / 64), rq, ao, H * (d / 64), ro, stream);
    return e == -1 ? 1 : e;  // a shape the grouped launch cannot take falls back to two launches
}

// The three products after the attention backward in one launch: dW^{Q,K,V,r},
// dW^O and the per-head dX rows; 1: not applicable.
template <int DH>
int run_bwd_proj(const uint16_t* X, const uint16_t* dY, const int32_t* I, const uint16_t* A, const uint16_t* dQKV,
                 const uint16_t* dz16, const float* dz, const uint16_t* Wq, const uint16_t* Wk, const uint16_t* Wv,
                 const uint16_t* Wr, int B, int T, int d, int H, int n, uint16_t* dWq, uint16_t* dWk, uint16_t* dWv,
                 uint16_t* dWr, uint16_t* dWo, uint16_t* dXs, hipStream_t stream) {
    using PQ = WgradQkvPolicy2<DH>;
    using PO = WgradOPolicy2<DH>;
    using PX = DxProjRowPolicy<DH>;
    const int R = B * n;
    const int rq = wgrad2_table_rows<PQ>(R, d), ro = wgrad2_table_rows<PO>(R, d);
    typename PX::Args ax;
    int nx;
    if (!rq || !ro || !dx_row_args<DH>(dQKV, dz, Wq, Wk, Wv, Wr, B, d, H, n, dXs, ax, nx)) return 1;
    typename PQ::Args aq{X, I, dQKV, dz16, dWq, dWk, dWv, dWr, nullptr, T, d, H, n, R, d / 64, 1, 0, make_fastdiv(n)};
    typename PO::Args ao{dY, I, A, dWo, nullptr, T, d, H, n, R, d / 64, 1, 0, make_fastdiv(n)};
    return launch_group3<Gemm2Job<PQ>, Gemm2Job<PO>, RowGemmJob<PX>>(
        aq, H * (d / 64), Gemm2Job<PQ>::lds(rq), ao, H * (d / 64), Gemm2Job<PO>::lds(ro), ax, nx,
        RowGemmJob<PX>::lds(0), stream);
}

// Bytes of fp32 partial sums the two launches of one head group need.
template <typename ST, int DH>
size_t partial_bytes(int B, int d, int H, int n, bool router) {
    using PQ = WgradQkvPolicy<ST, DH, true, true>;
    using PO = WgradOPolicy<ST, DH, true>;
    const int R = B * n;
    if constexpr (sizeof(ST) == 2) {  // MoSA heads on the gathered-row engine: no partials
        if (router && wgrad2_table_rows<WgradQkvPolicy2<DH>>(R, d) && wgrad2_table_rows<WgradOPolicy2<DH>>(R, d))
            return 0;
    }
    int cps;
    const int mtiles = (d + PQ::MT - 1) / PQ::MT, ntiles = (d + PO::NT - 1) / PO::NT;
    const int sq = choose_splits(H * mtiles, (R + PQ::KC - 1) / PQ::KC, cps);
    const int so = choose_splits(H * ntiles, (R + PO::KC - 1) / PO::KC, cps);
    const size_t nq = 3 * DH + (router ? 16 : 0);
    size_t bq = sq > 1 ? (size_t)sq * H * d * nq * 4 : 0;
    size_t bo = so > 1 ? (size_t)so * H * DH * d * 4 : 0;
    if constexpr (sizeof(ST) == 2) {
        if (!router && d % 64 == 0) {  // dense heads on the multi-stage engine: one partial per row range
            int rows;
            const int sd = dense_ranges(R, H * (d / 64), WgradQkvDensePolicy2<DH>::KC, rows);
            const int so2 = dense_ranges(R, H * (d / 64), WgradODensePolicy2<DH>::KC, rows);
            bq = std::max(bq, (size_t)sd * H * d * 3 * DH * 4);
            bo = std::max(bo, (size_t)so2 * H * DH * d * 4);
        }
    }
    return bq > bo ? bq : bo;
}

}  // namespace

int launch_wgrad(int dtype, const void* X, const void* dY, const int32_t* I, const void* A, const void* dQKV,
                 const void* dz16, int B, int T, int d, int H, int dh, int n, void* dWq, void* dWk, void* dWv,
                 void* dWr, void* dWo, float* part, int which, const Marker& mk, hipStream_t stream) {
    if (H == 0) return 0;
    if (which == 2) {
        // both: one launch on the gathered-row engine where it applies
        if (dtype == kBF16 && I) {
            using ST = uint16_t;
            auto both = dh == 64 ? run_both<64> : run_both<32>;
            const int e = both((const ST*)X, (const ST*)dY, I, (const ST*)A, (const ST*)dQKV, (const ST*)dz16, B, T, d,
                               H, n, (ST*)dWq, (ST*)dWk, (ST*)dWv, (ST*)dWr, (ST*)dWo, stream);
            if (e != 1) return e | mk("wgrad");
        }
        const int e0 = launch_wgrad(dtype, X, dY, I, A, dQKV, dz16, B, T, d, H, dh, n, dWq, dWk, dWv, dWr, dWo, part,
                                    0, mk, stream);
        return e0 | launch_wgrad(dtype, X, dY, I, A, dQKV, dz16, B, T, d, H, dh, n, dWq, dWk, dWv, dWr, dWo, part, 1,
                                 mk, stream);
    }
    if (dtype == kBF16) {
        using ST = uint16_t;
        if (which == 0) {
            auto f = dh == 64 ? run_qkv<ST, 64> : run_qkv<ST, 32>;
            return f((const ST*)X, I, (const ST*)dQKV, (const ST*)dz16, B, T, d, H, n, (ST*)dWq, (ST*)dWk, (ST*)dWv,
                     (ST*)dWr, part, mk, stream);
        }
        auto f = dh == 64 ? run_o<ST, 64> : run_o<ST, 32>;
        return f((const ST*)dY, I, (const ST*)A, B, T, d, H, n, (ST*)dWo, part, mk, stream);
    }
    using ST = float;
    if (which == 0) {
        auto f = dh == 64 ? run_qkv<ST, 64> : run_qkv<ST, 32>;
        return f((const ST*)X, I, (const ST*)dQKV, (const ST*)dz16, B, T, d, H, n, (ST*)dWq, (ST*)dWk, (ST*)dWv,
                 (ST*)dWr, part, mk, stream);
    }
    auto f = dh == 64 ? run_o<ST, 64> : run_o<ST, 32>;
    return f((const ST*)dY, I, (const ST*)A, B, T, d, H, n, (ST*)dWo, part, mk, stream);
}

int launch_bwd_proj(int dtype, const void* X, const void* dY, const int32_t* I, const void* A, const void* dQKV,
                    const void* dz16, const float* dz, const void* Wq, const void* Wk, const void* Wv, const void* Wr,
                    int B, int T, int d, int H, int dh, int n, void* dWq, void* dWk, void* dWv, void* dWr, void* dWo,
                    void* dXs, hipStream_t stream) {
    if (dtype != kBF16 || H == 0 || !I) return 1;
    // few selected rows per head: the per-head streaming kernel
    const int e = launch_bwd_head(dtype, X, dY, I, A, dQKV, dz16, dz, Wq, Wk, Wv, Wr, B, T, d, H, dh, n, dWq, dWk, dWv,
                                  dWr, dWo, dXs, stream);
    if (e != 1) return e;
    using ST = uint16_t;
    auto f = dh == 64 ? run_bwd_proj<64> : run_bwd_proj<32>;
    return f((const ST*)X, (const ST*)dY, I, (const ST*)A, (const ST*)dQKV, (const ST*)dz16, dz, (const ST*)Wq,
             (const ST*)Wk, (const ST*)Wv, (const ST*)Wr, B, T, d, H, n, (ST*)dWq, (ST*)dWk, (ST*)dWv, (ST*)dWr,
             (ST*)dWo, (ST*)dXs, stream);
}

size_t wgrad_partial_bytes(int dtype, int B, int d, int H, int dh, int n, int router) {
    if (H == 0 || n == 0) return 0;
    if (dtype == kBF16)
        return dh == 64 ? partial_bytes<uint16_t, 64>(B, d, H, n, router)
                        : partial_bytes<uint16_t, 32>(B, d, H, n, router);
    return dh == 64 ? partial_bytes<float, 64>(B, d, H, n, router) : partial_bytes<float, 32>(B, d, H, n, router);
}

}  // namespace mosa
