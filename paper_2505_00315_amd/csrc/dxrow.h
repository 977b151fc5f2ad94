// The per-head dX rows of the backward on the row-streaming kernel
// (rowgemm.h), shared by the dX projection and the grouped launch of the
// backward's projections:
//   dX^s_i = dQ_i W^Q_h^T + dK_i W^K_h^T + dV_i W^V_h^T + dz_i W^r_h
// (chain rule through Q, K, V = X^s W^{Q,K,V} and s = X^s W^r, Section 2.2).
#pragma once

#include "rowgemm.h"

namespace mosa {

// bf16 storage, d a multiple of the column block: the row-streaming kernel (rowgemm.h);
// the three weights' rows for 128 columns of dX held in registers, the packed
// dQ | dK | dV rows streamed, dz through LDS for the rank-1 router term.
template <int DH>
struct DxProjRowPolicy {
    using ST = uint16_t;
    static constexpr int K = 3 * DH, NPAIR = 1, STAGES = 3;
    static constexpr bool W_KCONTIG = true, ROW_SCALAR = true;
    struct Args {
        const ST* dQKV;  // [B, H, k, 3*DH]
        const float* dz; // [B, H, k]
        const ST* Wq;
        const ST* Wk;
        const ST* Wv;    // [H, d, DH]
        const ST* Wr;    // [H, d]
        ST* dXs;         // [B, H, k, d]
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
    __device__ static const ST* a_row(const Args& a, int h, int m) { return a.dQKV + ridx(a, h, m) * (3 * DH); }
    // W[k][n] = W^{k / DH}_h[n][k % DH]: 8 consecutive k of column n
    __device__ static const ST* w_kptr(const Args& a, int h, int n, int k) {
        const ST* W = k < DH ? a.Wq : (k < 2 * DH ? a.Wk : a.Wv);
        return W + ((size_t)h * a.d + n) * DH + (k % DH);
    }
    __device__ static const float* z_ptr(const Args& a, int h, int m) { return a.dz + ridx(a, h, m); }
    __device__ static void col_init(const Args& a, int h, int n, float (&cv)[8]) {
        vec8_to_f32<ST>(vec8_load<ST>(a.Wr + (size_t)h * a.d + n), cv);
    }
    __device__ static __amdgpu_buffer_rsrc_t out_rsrc(const Args& a, int) {
        return __builtin_amdgcn_make_buffer_rsrc(a.dXs, 0, a.out_bytes, 0x00020000);
    }
    __device__ static int out_row(const Args& a, int h, int m) { return (int)(ridx(a, h, m) * a.d * 2); }
    __device__ static void finish(float (&x)[8], float z, const float (&cv)[8]) {
#pragma unroll
        for (int j = 0; j < 8; ++j) x[j] += z * cv[j];
    }
};

// Arguments and workgroup count of the dX rows for bf16 storage; false when
// the shape does not suit the kernel (d not a multiple of its column block,
// or an output past 2^31 bytes).
template <int DH>
inline bool dx_row_args(const uint16_t* dQKV, const float* dz, const uint16_t* Wq, const uint16_t* Wk,
                        const uint16_t* Wv, const uint16_t* Wr, int B, int d, int H, int k, uint16_t* dXs,
                        typename DxProjRowPolicy<DH>::Args& ra, int& nblocks) {
    using R = DxProjRowPolicy<DH>;
    const int M = B * k;
    const long long out_bytes = (long long)M * H * d * 2;
    if (d % (128 * R::NPAIR) != 0 || out_bytes >= (1ll << 31)) return false;
    const int ntiles = d / (128 * R::NPAIR), tiles = (M + 63) / 64;
    const int per = rowgemm_tiles_per_wg(H * ntiles, tiles, 512), splits = (tiles + per - 1) / per;
    ra = typename R::Args{dQKV, dz, Wq, Wk, Wv, Wr, dXs, d, H, k, M, ntiles, tiles, per, splits, (int)out_bytes};
    nblocks = H * ntiles * splits;
    return true;
}

}  // namespace mosa
