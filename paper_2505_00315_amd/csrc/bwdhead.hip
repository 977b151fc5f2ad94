// The backward's three products of the MoSA heads that follow the attention
// backward, for heads with few selected rows (R = B k <= 128), one launch:
//
//   W1  dW^{Q,K,V}_h[c, j] = sum_r X^s[r, c] G[r, j],  dW^r_h[c] = sum_r X^s[r, c] dz_r
//   W2  dW^O_h[e, c]       = sum_r (r A)[r, e] dY^s[r, c]
//   W3  dX^s_h[r, c]       = sum_j G[r, j] W_h[c, j] + dz_r W^r_h[c]
//
// with G = [dQ | dK | dV | dz, 0 ..] the gradient rows of the head's selected
// rows r = (b, i) in order, X^s = X[b, I_r], dY^s = dY[b, I_r], and
// W_h = [W^Q | W^K | W^V]_h (the chain rule through Q, K, V = X^s W and
// s = X^s W^r, Section 2.2; the rows r are summed in order, so every sum is
// reproducible).
//
// With so few rows, a tile of these products has a contraction of only R and
// a workgroup per output tile spends most of its life filling and draining
// its pipeline.  Here a workgroup owns one (job, head, range of 64-column
// tiles of d): the operand that is the same for every tile -- G^T (W1), r A
// (W2) or G (W3) -- is taken into registers once, and the tiles of the other
// operand -- X^s, dY^s or W_h -- stream through a 3-stage LDS ring filled by
// direct global->LDS loads, so the loads of the next tiles are in flight
// while a tile is multiplied and stored.  Results go from the accumulators to
// memory as 16-byte stores: each MFMA pair's output rows are interleaved
// (block 2p row i is M index 32 p + 8 (i / 4) + i % 4, block 2p + 1 the same
// + 4) so that a lane holds 8 consecutive columns of one output row.  Every
// wave issues the same number of loads and stores per tile (buffer stores
// with out-of-range offsets for the outputs that do not exist), which keeps
// the pipeline's wait counts exact.
#include "gemm2.h"
#include "kernels.h"

namespace mosa {

namespace {

constexpr int kBhDH = 64, kBhJ = 3 * kBhDH, kBhStages = 3;

struct BhArgs {
    const uint16_t* X;      // [B, T, d]
    const uint16_t* dY;     // [B, T, d]
    const int32_t* I;       // [B, H, k]
    const uint16_t* A;      // [B, H, k, 64] rows scaled by r
    const uint16_t* dQKV;   // [B, H, k, 192]
    const uint16_t* dz16;   // [B, H, k, 16]: dz and 15 zeros
    const float* dz;        // [B, H, k]
    const uint16_t* Wq;     // [H, d, 64]
    const uint16_t* Wk;
    const uint16_t* Wv;
    const uint16_t* Wr;     // [H, d]
    uint16_t* dWq;          // [H, d, 64]
    uint16_t* dWk;
    uint16_t* dWv;
    uint16_t* dWr;          // [H, d]
    uint16_t* dWo;          // [H, 64, d]
    uint16_t* dXs;          // [B, H, k, d]
    int T, d, H, k, R;      // R = B k rows per head
    int tpw, nsplit;        // 64-column tiles per workgroup; workgroups per (job, head)
};

// Selected row r of head h: its index in the [B, H, k] tensors, or -1 past R.
__device__ __forceinline__ int bh_row(const BhArgs& a, int h, int r) {
    if (r >= a.R) return -1;
    const int b = r / a.k, i = r - b * a.k;
    return (b * a.H + h) * a.k + i;
}

// Unit permutations: rows of 8 or 32 16-byte units read by transposed reads of
// 4 consecutive rows (the pairs of units of those rows land on distinct banks),
// and rows of 24 units read by 16-byte reads of the interleaved rows.
__device__ __forceinline__ int tr_swz(int r) { return 2 * (r & 3); }
__device__ __forceinline__ int il_swz(int c) { return (c & 3) | (((c >> 3) & 1) << 2); }

// Transposed fragment (8 consecutive k of one M / N index per lane) from an
// LDS tile of rows of `upr` units: source lane s reads row kb + s / 4 (and
// + 4), 4 columns starting at col0(s % 4).
__device__ __forceinline__ u32x4 bh_frag_tr(const unsigned char* tile, int upr, int kb, int col) {
    const int lane = threadIdx.x & 63, g = lane >> 4, s = lane & 15;
    const int r0 = kb + 8 * g + (s >> 2), r1 = r0 + 4;
    const int gu = col >> 3, half = (col >> 2) & 1;
    const int su0 = (gu & ~7) | ((gu & 7) ^ tr_swz(r0)), su1 = (gu & ~7) | ((gu & 7) ^ tr_swz(r1));
    const u32x2 lo = lds_read_tr16(tile + (r0 * upr + su0) * 16 + 8 * half);
    const u32x2 hi = lds_read_tr16(tile + (r1 * upr + su1) * 16 + 8 * half);
    return u32x4{lo.x, lo.y, hi.x, hi.y};
}

// Column of the interleaved M block (p, odd) that source lane s supplies.
__device__ __forceinline__ int il_col(int base, int p, int odd, int s) { return base + 32 * p + 8 * (s & 3) + 4 * odd; }

// wait_vmcnt<L (STG - 2) + min(s, STG - 1) S>() for the loads (L) and stores
// (S) one wave issues per tile.
template <int L, int S>
__device__ __forceinline__ void bh_wait(int s) {
    constexpr int base = L * (kBhStages - 2);
    if (s >= kBhStages - 1) wait_vmcnt<base + (kBhStages - 1) * S>();
    else if (s == 1) wait_vmcnt<base + S>();
    else wait_vmcnt<base>();
}

template <int NR>
struct BhShape {
    static constexpr int NROWS = 32 * NR;                 // R padded to the MFMA k steps
    static constexpr int ROWTILE = NROWS * 8 * 16;        // an X^s / dY^s tile: NROWS x 64 columns
    static constexpr int WTILE = 64 * 24 * 16;            // a W_h tile: 64 columns c x 192 j
    static constexpr size_t lds_w1 = (size_t)kBhStages * ROWTILE > 128u * 32 * 16 ? (size_t)kBhStages * ROWTILE
                                                                                   : 128u * 32 * 16;
    static constexpr size_t lds_w2 = (size_t)kBhStages * ROWTILE;
    static size_t lds_w3(int d) { return (size_t)kBhStages * WTILE + (size_t)d * 2; }
    static size_t lds(int d) {
        size_t m = lds_w1 > lds_w2 ? lds_w1 : lds_w2;
        return m > lds_w3(d) ? m : lds_w3(d);
    }
};

// The gathered rows of one ring tile (X^s or dY^s, 64 columns from c0): each
// lane's NR units, row p / 8 of the tile, stored unit p % 8.
template <int NR>
struct RowTileLoader {
    const uint16_t* src[NR];  // row start + the lane's column offset, or the zero row
    int step[NR];             // 1 for real rows, 0 for the zero row
    __device__ void init(const BhArgs& a, const uint16_t* base, int h) {
        const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
        for (int jj = 0; jj < NR; ++jj) {
            const int p = 64 * (wave + 4 * jj) + lane, r = p >> 3, su = p & 7;
            const int ri = bh_row(a, h, r);
            if (ri >= 0) {
                const int b = (r / a.k);
                src[jj] = base + ((size_t)b * a.T + a.I[ri]) * a.d + 8 * (su ^ tr_swz(r));
                step[jj] = 1;
            } else {
                src[jj] = g2_zero;
                step[jj] = 0;
            }
        }
    }
    __device__ void issue(int c0, uint32_t lds_wave) const {
#pragma unroll
        for (int jj = 0; jj < NR; ++jj) lds_load16(src[jj] + (size_t)c0 * step[jj], lds_wave + 4096 * jj);
    }
};

// W1: dW^{Q,K,V} and dW^r.  M = j (wave w: j in [64 w, 64 w + 64); wave 3 holds
// dz at j = 192 and zero rows after it), N = c (4 blocks of 16), K = r.
template <int NR>
__device__ void bh_job_w1(const BhArgs& a, int h, int t0, int t1, unsigned char* smem) {
    using S = BhShape<NR>;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, g = lane >> 4, c16 = lane & 15;
    const uint32_t lbase = __builtin_amdgcn_readfirstlane(lds_addr(smem));
    const int wave_s = __builtin_amdgcn_readfirstlane(wave);

    // G^T fragments, staged through LDS 128 rows (4 k steps) at a time
    // (rows of 32 units: dQ | dK | dV, dz16, zeros; zero rows past R).
    u32x4 af[2][2][NR];
#pragma unroll
    for (int half = 0; half < (NR + 3) / 4; ++half) {
        constexpr int UPR = 32;
#pragma unroll
        for (int jj = 0; jj < 16; ++jj) {  // 128 rows x 32 units = 16 loads per wave
            const int p = 64 * (wave + 4 * jj) + lane, rl = p >> 5, su = p & 31, r = 128 * half + rl;
            const int gu = (su & ~7) | ((su & 7) ^ tr_swz(r));
            const int ri = bh_row(a, h, r);
            const uint16_t* src = g2_zero;
            if (ri >= 0 && gu < 24) src = a.dQKV + (size_t)ri * kBhJ + 8 * gu;
            else if (ri >= 0 && gu < 26) src = a.dz16 + (size_t)ri * 16 + 8 * (gu - 24);
            lds_load16(src, lbase + 1024 * wave_s + 4096 * jj);
        }
        wait_vmcnt<0>();
        __syncthreads();
#pragma unroll
        for (int ks = 4 * half; ks < 4 * half + 4 && ks < NR; ++ks)
#pragma unroll
            for (int p = 0; p < 2; ++p)
#pragma unroll
                for (int odd = 0; odd < 2; ++odd)
                    af[p][odd][ks] = bh_frag_tr(smem, UPR, 32 * (ks - 4 * half), il_col(64 * wave, p, odd, c16));
        lds_wait();
#pragma unroll
        for (int ks = 4 * half; ks < 4 * half + 4 && ks < NR; ++ks)
#pragma unroll
            for (int p = 0; p < 2; ++p)
#pragma unroll
                for (int odd = 0; odd < 2; ++odd) lds_ready(af[p][odd][ks]);
        __syncthreads();  // the ring below reuses this LDS
    }

    RowTileLoader<NR> ld;
    ld.init(a, a.X, h);
    // outputs: wave w < 3 writes W^{Q,K,V}[w] (16-byte rows of 8 j), wave 3 the
    // dz column as dW^r (2 bytes) where j = 192, nothing for the zero rows
    uint16_t* const outs[4] = {a.dWq, a.dWk, a.dWv, a.dWr};
    const __amdgpu_buffer_rsrc_t out = __builtin_amdgcn_make_buffer_rsrc(
        outs[wave_s], 0, wave_s < 3 ? a.H * a.d * kBhDH * 2 : a.H * a.d * 2, 0x00020000);

    const int ntile = t1 - t0;
#pragma unroll
    for (int s = 0; s < kBhStages - 1; ++s)
        ld.issue(64 * (t0 + min(s, ntile - 1)), lbase + s * S::ROWTILE + 1024 * wave_s);
    for (int s = 0; s < ntile; ++s) {
        bh_wait<NR, 8>(s);
        __syncthreads();  // tile s is in LDS; the buffer of tile s - 1 is free
        ld.issue(64 * (t0 + min(s + kBhStages - 1, ntile - 1)),
                 lbase + ((s + kBhStages - 1) % kBhStages) * S::ROWTILE + 1024 * wave_s);
        const unsigned char* tile = smem + (s % kBhStages) * S::ROWTILE;
        f32x4 acc[2][2][4];
#pragma unroll
        for (int p = 0; p < 2; ++p)
#pragma unroll
            for (int odd = 0; odd < 2; ++odd)
#pragma unroll
                for (int nb = 0; nb < 4; ++nb) acc[p][odd][nb] = zero4();
#pragma unroll
        for (int ks = 0; ks < NR; ++ks) {
            u32x4 bf[4];
#pragma unroll
            for (int nb = 0; nb < 4; ++nb) bf[nb] = bh_frag_tr(tile, 8, 32 * ks, 16 * nb + 4 * (c16 & 3));
            lds_wait();
#pragma unroll
            for (int nb = 0; nb < 4; ++nb) {
                lds_ready(bf[nb]);
                Frag8<uint16_t> fb;
                fb.v = __builtin_bit_cast(bf16x8, bf[nb]);
#pragma unroll
                for (int p = 0; p < 2; ++p)
#pragma unroll
                    for (int odd = 0; odd < 2; ++odd) {
                        Frag8<uint16_t> fa;
                        fa.v = __builtin_bit_cast(bf16x8, af[p][odd][ks]);
                        mma8(acc[p][odd][nb], fa, fb);
                    }
            }
        }
        mfma_drain();
        const int c0 = 64 * (t0 + s);
#pragma unroll
        for (int p = 0; p < 2; ++p)
#pragma unroll
            for (int nb = 0; nb < 4; ++nb) {
                const int c = c0 + 16 * nb + c16, j = 64 * wave + 32 * p + 8 * g;
                float x[8];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    x[e] = acc[p][0][nb][e];
                    x[4 + e] = acc[p][1][nb][e];
                }
                if (wave < 3) {
                    const uint4 v = make_uint4(pack_bf16x2(x[0], x[1]), pack_bf16x2(x[2], x[3]),
                                               pack_bf16x2(x[4], x[5]), pack_bf16x2(x[6], x[7]));
                    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), out,
                                                           (int)(((size_t)h * a.d + c) * kBhDH + (j & 63)) * 2, 0, 0);
                } else {
                    const int off = j == 3 * kBhDH ? (h * a.d + c) * 2 : INT32_MIN;
                    __builtin_amdgcn_raw_buffer_store_b16(f32_to_bf16(x[0]), out, off, 0, 0);
                }
            }
    }
    wait_vmcnt<0>();
}

// W2: dW^O.  M = c (interleaved, 2 pairs), N = e (wave w: e in [16 w, 16 w + 16)), K = r.
template <int NR>
__device__ void bh_job_w2(const BhArgs& a, int h, int t0, int t1, unsigned char* smem) {
    using S = BhShape<NR>;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, g = lane >> 4, c16 = lane & 15;
    const uint32_t lbase = __builtin_amdgcn_readfirstlane(lds_addr(smem));
    const int wave_s = __builtin_amdgcn_readfirstlane(wave);

    // (r A) rows through LDS (rows of 8 units, zero rows past R), then this
    // wave's fragments of columns e = 16 w .. + 15
    u32x4 bfr[NR];
#pragma unroll
    for (int jj = 0; jj < NR; ++jj) {
        const int p = 64 * (wave + 4 * jj) + lane, r = p >> 3, su = p & 7;
        const int ri = bh_row(a, h, r);
        const uint16_t* src = ri >= 0 ? a.A + (size_t)ri * kBhDH + 8 * (su ^ tr_swz(r)) : g2_zero;
        lds_load16(src, lbase + 1024 * wave_s + 4096 * jj);
    }
    wait_vmcnt<0>();
    __syncthreads();
#pragma unroll
    for (int ks = 0; ks < NR; ++ks) bfr[ks] = bh_frag_tr(smem, 8, 32 * ks, 16 * wave + 4 * (c16 & 3));
    lds_wait();
#pragma unroll
    for (int ks = 0; ks < NR; ++ks) lds_ready(bfr[ks]);
    __syncthreads();

    RowTileLoader<NR> ld;
    ld.init(a, a.dY, h);
    const int ntile = t1 - t0;
#pragma unroll
    for (int s = 0; s < kBhStages - 1; ++s)
        ld.issue(64 * (t0 + min(s, ntile - 1)), lbase + s * S::ROWTILE + 1024 * wave_s);
    for (int s = 0; s < ntile; ++s) {
        bh_wait<NR, 2>(s);
        __syncthreads();
        ld.issue(64 * (t0 + min(s + kBhStages - 1, ntile - 1)),
                 lbase + ((s + kBhStages - 1) % kBhStages) * S::ROWTILE + 1024 * wave_s);
        const unsigned char* tile = smem + (s % kBhStages) * S::ROWTILE;
        f32x4 acc[2][2];
#pragma unroll
        for (int p = 0; p < 2; ++p)
#pragma unroll
            for (int odd = 0; odd < 2; ++odd) acc[p][odd] = zero4();
#pragma unroll
        for (int ks = 0; ks < NR; ++ks) {
            u32x4 af[2][2];
#pragma unroll
            for (int p = 0; p < 2; ++p)
#pragma unroll
                for (int odd = 0; odd < 2; ++odd) af[p][odd] = bh_frag_tr(tile, 8, 32 * ks, il_col(0, p, odd, c16));
            lds_wait();
            Frag8<uint16_t> fb;
            fb.v = __builtin_bit_cast(bf16x8, bfr[ks]);
#pragma unroll
            for (int p = 0; p < 2; ++p)
#pragma unroll
                for (int odd = 0; odd < 2; ++odd) {
                    lds_ready(af[p][odd]);
                    Frag8<uint16_t> fa;
                    fa.v = __builtin_bit_cast(bf16x8, af[p][odd]);
                    mma8(acc[p][odd], fa, fb);
                }
        }
        mfma_drain();
        const int c0 = 64 * (t0 + s), e = 16 * wave + c16;
#pragma unroll
        for (int p = 0; p < 2; ++p) {
            float x[8];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                x[i] = acc[p][0][i];
                x[4 + i] = acc[p][1][i];
            }
            *reinterpret_cast<uint4*>(a.dWo + ((size_t)h * kBhDH + e) * a.d + c0 + 32 * p + 8 * g) =
                make_uint4(pack_bf16x2(x[0], x[1]), pack_bf16x2(x[2], x[3]), pack_bf16x2(x[4], x[5]),
                           pack_bf16x2(x[6], x[7]));
        }
    }
    wait_vmcnt<0>();
}

// W3: the per-head dX rows.  M = c (interleaved, 2 pairs), N = r (wave w: rows
// [8 NR w, 8 NR (w + 1)), NR / 2 blocks), K = j < 192; the dz W^r term is
// added in the epilogue from W^r_h staged in LDS.
template <int NR>
__device__ void bh_job_w3(const BhArgs& a, int h, int t0, int t1, unsigned char* smem) {
    using S = BhShape<NR>;
    constexpr int NB = NR / 2, KS = kBhJ / 32;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, g = lane >> 4, c16 = lane & 15;
    const uint32_t lbase = __builtin_amdgcn_readfirstlane(lds_addr(smem));
    const int wave_s = __builtin_amdgcn_readfirstlane(wave);
    uint16_t* wr_s = reinterpret_cast<uint16_t*>(smem + kBhStages * S::WTILE);

    // G fragments (B operand: row r = 8 NR w + 16 nb + c16, j = 32 ks + 8 g ..)
    // straight from memory, dz of the lane's rows, and W^r_h into LDS.
    u32x4 gf[NB][KS];
    float dzr[NB];
    int rix[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
        const int r = 8 * NR * wave + 16 * nb + c16, ri = bh_row(a, h, r);
        rix[nb] = ri;
        dzr[nb] = ri >= 0 ? a.dz[ri] : 0.f;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
            gf[nb][ks] = ri >= 0 ? *reinterpret_cast<const u32x4*>(a.dQKV + (size_t)ri * kBhJ + 32 * ks + 8 * g)
                                 : u32x4{0u, 0u, 0u, 0u};
    }
    for (int v = tid; v < a.d / 8; v += 256)
        *reinterpret_cast<uint4*>(wr_s + 8 * v) = *reinterpret_cast<const uint4*>(a.Wr + (size_t)h * a.d + 8 * v);
    // take the fragments now (a first use inside the pipeline would wait for
    // every load in flight there)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
        asm volatile("" : "+v"(dzr[nb]));
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) asm volatile("" : "+v"(gf[nb][ks]));
    }
    __syncthreads();

    // W_h tile: 64 rows c x 24 units ([W^Q | W^K | W^V] row c0 + c), stored
    // unit of row c = global unit ^ il_swz(c) within its group of 8
    const uint16_t* wsrc[6];
#pragma unroll
    for (int jj = 0; jj < 6; ++jj) {
        const int p = 64 * (wave + 4 * jj) + lane, c = p / 24, su = p % 24;
        const int gu = (su & ~7) | ((su & 7) ^ il_swz(c));
        const uint16_t* W = gu < 8 ? a.Wq : (gu < 16 ? a.Wk : a.Wv);
        wsrc[jj] = W + ((size_t)h * a.d + c) * kBhDH + 8 * (gu & 7);
    }
    auto issue = [&](int t, int buf) {
        const size_t off = (size_t)64 * t * kBhDH;
#pragma unroll
        for (int jj = 0; jj < 6; ++jj) lds_load16(wsrc[jj] + off, lbase + buf * S::WTILE + 1024 * wave_s + 4096 * jj);
    };
    const __amdgpu_buffer_rsrc_t out = __builtin_amdgcn_make_buffer_rsrc(a.dXs, 0, a.R * a.H * a.d * 2, 0x00020000);

    const int ntile = t1 - t0;
#pragma unroll
    for (int s = 0; s < kBhStages - 1; ++s) issue(t0 + min(s, ntile - 1), s);
    for (int s = 0; s < ntile; ++s) {
        bh_wait<6, NB * 2>(s);
        __syncthreads();
        issue(t0 + min(s + kBhStages - 1, ntile - 1), (s + kBhStages - 1) % kBhStages);
        const unsigned char* tile = smem + (s % kBhStages) * S::WTILE;
        f32x4 acc[2][2][NB];
#pragma unroll
        for (int p = 0; p < 2; ++p)
#pragma unroll
            for (int odd = 0; odd < 2; ++odd)
#pragma unroll
                for (int nb = 0; nb < NB; ++nb) acc[p][odd][nb] = zero4();
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            Frag8<uint16_t> fa[2][2];
#pragma unroll
            for (int p = 0; p < 2; ++p)
#pragma unroll
                for (int odd = 0; odd < 2; ++odd) {
                    const int c = 32 * p + 8 * (c16 >> 2) + (c16 & 3) + 4 * odd, gu = 4 * ks + g;
                    const int su = (gu & ~7) | ((gu & 7) ^ il_swz(c));
                    fa[p][odd].v = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(tile + (c * 24 + su) * 16));
                }
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) {
                Frag8<uint16_t> fb;
                fb.v = __builtin_bit_cast(bf16x8, gf[nb][ks]);
#pragma unroll
                for (int p = 0; p < 2; ++p)
#pragma unroll
                    for (int odd = 0; odd < 2; ++odd) mma8(acc[p][odd][nb], fa[p][odd], fb);
            }
        }
        mfma_drain();
        const int c0 = 64 * (t0 + s);
#pragma unroll
        for (int p = 0; p < 2; ++p) {
            const int c = c0 + 32 * p + 8 * g;
            float w8[8];
            vec8_to_f32<uint16_t>(vec8_load<uint16_t>(wr_s + c), w8);
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) {
                float x[8];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    x[i] = acc[p][0][nb][i] + dzr[nb] * w8[i];
                    x[4 + i] = acc[p][1][nb][i] + dzr[nb] * w8[4 + i];
                }
                const uint4 v = make_uint4(pack_bf16x2(x[0], x[1]), pack_bf16x2(x[2], x[3]), pack_bf16x2(x[4], x[5]),
                                           pack_bf16x2(x[6], x[7]));
                const int off = rix[nb] >= 0 ? (int)(((size_t)rix[nb] * a.d + c) * 2) : INT32_MIN;
                __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), out, off, 0, 0);
            }
        }
    }
    wait_vmcnt<0>();
}

// Workgroups in three equal ranges: W1, then W2, then W3 (head and tile
// range from the position in the range).  The dX rows come last so that they
// are the freshest in the memory-side cache when the head-ordered sum reads
// them back (hybrid_d1024: 86 -> 80 us here and 28 -> 22 us for that sum,
// against the three jobs interleaved).
template <int NR>
__global__ __launch_bounds__(256) void bwd_head_kernel(const BhArgs a) {
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
    const int nu = gridDim.x / 3, j = blockIdx.x, job = j / nu, u = j % nu;
    const int h = u / a.nsplit, sp = u % a.nsplit;
    const int ntiles = a.d / 64, t0 = sp * a.tpw, t1 = min(ntiles, t0 + a.tpw);
    if (job == 0) bh_job_w1<NR>(a, h, t0, t1, smem);
    else if (job == 1) bh_job_w2<NR>(a, h, t0, t1, smem);
    else bh_job_w3<NR>(a, h, t0, t1, smem);
}

template <int NR>
int launch_nr(const BhArgs& a, hipStream_t stream) {
    const size_t lds = BhShape<NR>::lds(a.d);
    if (lds > 160 * 1024) return 1;
    auto kern = bwd_head_kernel<NR>;
    if (allow_lds((const void*)kern, lds)) return -1;
    hipLaunchKernelGGL(kern, dim3(3 * a.H * a.nsplit), dim3(256), lds, stream, a);
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

}  // namespace

int launch_bwd_head(int dtype, const void* X, const void* dY, const int32_t* I, const void* A, const void* dQKV,
                    const void* dz16, const float* dz, const void* Wq, const void* Wk, const void* Wv, const void* Wr,
                    int B, int T, int d, int H, int dh, int k, void* dWq, void* dWk, void* dWv, void* dWr, void* dWo,
                    void* dXs, hipStream_t stream) {
    const long long R = (long long)B * k;
    // up to 128 rows (measured: 86 us instead of 125 us for 256 heads of 128
    // rows; at 256 rows the grouped tile kernel is faster, 84 us instead of 93)
    if (dtype != kBF16 || dh != kBhDH || H == 0 || !I || R > 128 || d % 64 != 0 || d > 16384) return 1;
    // buffer-store ranges (32-bit byte offsets)
    if ((long long)H * d * kBhDH * 2 >= (1ll << 31) || R * H * d * 2 >= (1ll << 31)) return 1;
    using ST = uint16_t;
    BhArgs a{(const ST*)X, (const ST*)dY, I, (const ST*)A, (const ST*)dQKV, (const ST*)dz16, dz, (const ST*)Wq,
             (const ST*)Wk, (const ST*)Wv, (const ST*)Wr, (ST*)dWq, (ST*)dWk, (ST*)dWv, (ST*)dWr, (ST*)dWo, (ST*)dXs,
             T, d, H, k, (int)R, 0, 0};
    // tiles per workgroup: about 3 workgroups per CU over the three jobs
    const int ntiles = d / 64;
    int nsplit = (768 + 3 * H - 1) / (3 * H);
    nsplit = nsplit < 1 ? 1 : (nsplit > ntiles ? ntiles : nsplit);
    a.tpw = (ntiles + nsplit - 1) / nsplit;
    a.nsplit = (ntiles + a.tpw - 1) / a.tpw;
    return R <= 64 ? launch_nr<2>(a, stream) : launch_nr<4>(a, stream);
}

}  // namespace mosa
