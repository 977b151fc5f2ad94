// Backward of the attention among the selected tokens (Eq. 1, index-aware
// causal mask = lower triangle in slot order), recomputing P from the saved
// log-sum-exp:
//   P_ij  = exp(S_ij / sqrt(dh) - lse_i)            (0 where masked)
//   dV_j  = sum_i P_ij dA_i
//   dP_ij = <dA_i, V_j>,  dS_ij = P_ij (dP_ij - D_i),  D_i = <dA_i, A_i>
//   dK_j  = sum_i dS_ij Q_i / sqrt(dh),  dQ_i = sum_j dS_ij K_j / sqrt(dh)
// Two passes so that no value is ever accumulated by atomics (results are
// bitwise reproducible):
//   kv pass: one wave per block of 16 keys, loop over the query blocks that
//            may attend to them; S and dP tiles come out with the key in the
//            lane (lane % 16) and queries in rows, i.e. already in the K = 16
//            operand layout for dV^T += dA^T P and dK^T += Q^T dS;
//   q pass:  one wave per block of 16 queries, loop over allowed key blocks;
//            S^T and dP^T tiles (query in the lane) feed dQ^T += K^T dS^T.
#include "common.h"
#include "gemm2.h"
#include "kernels.h"
#include "rope.h"
#include "tiles.h"

namespace mosa {

namespace {

template <typename ST, int DH, bool WIN>
__global__ __launch_bounds__(256) void attn_bwd_kv_kernel(const ST* __restrict__ QKV, const ST* __restrict__ dA,
                                                          const float* __restrict__ lse, const float* __restrict__ D,
                                                          int BH, int n, int causal, int lb, float scale,
                                                          ST* __restrict__ dQKV, const int32_t* __restrict__ rI,
                                                          const float2* __restrict__ rtab) {
    constexpr int RS = 3 * DH;  // row stride of the packed Q | K | V (and dQ | dK | dV) rows
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int g = lane >> 4, c16 = lane & 15;
    const int nb = (n + 15) / 16;
    const int task = blockIdx.x * 4 + wave;
    if (task >= BH * nb) return;
    const int bh = task / nb, j0 = (task % nb) * 16;
    const size_t base = (size_t)bh * n;
    const ST* Qp = QKV + base * RS;
    const ST* Kp = Qp + DH;
    const ST* Vp = Qp + 2 * DH;
    const ST* dAp = dA + base * DH;

    const int key = j0 + c16;  // this lane's key (as MFMA column)
    Frag8<ST> kf[DH / 32], vf[DH / 32];
#pragma unroll
    for (int s = 0; s < DH / 32; ++s) {
        kf[s] = key < n ? frag8_load<ST>(Kp + (size_t)key * RS + s * 32 + 8 * g) : frag8_zero<ST>();
        vf[s] = key < n ? frag8_load<ST>(Vp + (size_t)key * RS + s * 32 + 8 * g) : frag8_zero<ST>();
    }
    f32x4 dKt[DH / 16], dVt[DH / 16];
#pragma unroll
    for (int db = 0; db < DH / 16; ++db) dKt[db] = dVt[db] = zero4();

    // causal with a window: queries up to lb past the block's last key see it
    const int i_end = WIN && causal ? min(n, j0 + 16 + lb) : n;
    for (int i0 = causal ? j0 : 0; i0 < i_end; i0 += 16) {
        const int qa = i0 + c16;  // query this lane feeds as MFMA A row
        f32x4 s = zero4(), dp = zero4();
#pragma unroll
        for (int st = 0; st < DH / 32; ++st) {
            const Frag8<ST> qa_f = qa < n ? frag8_load<ST>(Qp + (size_t)qa * RS + st * 32 + 8 * g) : frag8_zero<ST>();
            const Frag8<ST> da_f = qa < n ? frag8_load<ST>(dAp + (size_t)qa * DH + st * 32 + 8 * g) : frag8_zero<ST>();
            mma8(s, qa_f, kf[st]);
            mma8(dp, da_f, vf[st]);
        }
        // lane: key column c16, query rows 4g + i
        float p[4], ds[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int q = i0 + 4 * g + i;
            const bool ok = q < n && key < n && (!causal || (key <= q && (!WIN || q - key <= lb)));
            const float l = q < n ? lse[base + q] : 0.f;
            const float dd = q < n ? D[base + q] : 0.f;
            p[i] = ok ? expf(s[i] * scale - l) : 0.f;
            ds[i] = p[i] * (dp[i] - dd);
        }
        const Frag4<ST> pf = frag4_from<ST>(p);
        const Frag4<ST> dsf = frag4_from<ST>(ds);
#pragma unroll
        for (int db = 0; db < DH / 16; ++db) {
            float at[4], qt[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int q = i0 + 4 * g + i;
                at[i] = q < n ? ld1<ST>(dAp + (size_t)q * DH + db * 16 + c16) : 0.f;
                qt[i] = q < n ? ld1<ST>(Qp + (size_t)q * RS + db * 16 + c16) : 0.f;
            }
            mma4(dVt[db], frag4_from<ST>(at), pf);
            mma4(dKt[db], frag4_from<ST>(qt), dsf);
        }
        mfma_drain();  // the loop may exit right here
    }
    if (key < n) {
        // lane: key column c16, d_head rows db*16 + 4g + i
        const int pos = rtab ? (rI ? rI[base + key] : key) : 0;
#pragma unroll
        for (int db = 0; db < DH / 16; ++db) {
            float x[4] = {dKt[db][0] * scale, dKt[db][1] * scale, dKt[db][2] * scale, dKt[db][3] * scale};
            if (rtab) rope4_back<DH>(x, db * 16 + 4 * g, rtab, pos);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                st1<ST>(dQKV + (base + key) * RS + 2 * DH + db * 16 + 4 * g + i, dVt[db][i]);
                st1<ST>(dQKV + (base + key) * RS + DH + db * 16 + 4 * g + i, x[i]);
            }
        }
    }
}

template <typename ST, int DH, bool WIN>
__global__ __launch_bounds__(256) void attn_bwd_q_kernel(const ST* __restrict__ QKV, const ST* __restrict__ dA,
                                                         const float* __restrict__ lse, const float* __restrict__ D,
                                                         int BH, int n, int causal, int lb, float scale,
                                                         ST* __restrict__ dQKV, const int32_t* __restrict__ rI,
                                                         const float2* __restrict__ rtab) {
    constexpr int RS = 3 * DH;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int g = lane >> 4, c16 = lane & 15;
    const int nb = (n + 15) / 16;
    const int task = blockIdx.x * 4 + wave;
    if (task >= BH * nb) return;
    const int bh = task / nb, i0 = (task % nb) * 16;
    const size_t base = (size_t)bh * n;
    const ST* Qp = QKV + base * RS;
    const ST* Kp = Qp + DH;
    const ST* Vp = Qp + 2 * DH;
    const ST* dAp = dA + base * DH;

    const int q = i0 + c16;  // this lane's query (MFMA column)
    Frag8<ST> qf[DH / 32], daf[DH / 32];
#pragma unroll
    for (int s = 0; s < DH / 32; ++s) {
        qf[s] = q < n ? frag8_load<ST>(Qp + (size_t)q * RS + s * 32 + 8 * g) : frag8_zero<ST>();
        daf[s] = q < n ? frag8_load<ST>(dAp + (size_t)q * DH + s * 32 + 8 * g) : frag8_zero<ST>();
    }
    const float lq = q < n ? lse[base + q] : 0.f;
    const float dq = q < n ? D[base + q] : 0.f;
    f32x4 dQt[DH / 16];
#pragma unroll
    for (int db = 0; db < DH / 16; ++db) dQt[db] = zero4();

    const int kv_end = causal ? min(n, i0 + 16) : n;
    for (int j0 = WIN && causal ? max(0, i0 - lb) / 16 * 16 : 0; j0 < kv_end; j0 += 16) {
        const int kr = j0 + c16;
        f32x4 s = zero4(), dp = zero4();
#pragma unroll
        for (int st = 0; st < DH / 32; ++st) {
            const Frag8<ST> k_f = kr < n ? frag8_load<ST>(Kp + (size_t)kr * RS + st * 32 + 8 * g) : frag8_zero<ST>();
            const Frag8<ST> v_f = kr < n ? frag8_load<ST>(Vp + (size_t)kr * RS + st * 32 + 8 * g) : frag8_zero<ST>();
            mma8(s, k_f, qf[st]);
            mma8(dp, v_f, daf[st]);
        }
        // lane: query column c16, key rows 4g + i
        float ds[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int j = j0 + 4 * g + i;
            const bool ok = q < n && j < n && (!causal || (j <= q && (!WIN || q - j <= lb)));
            const float p = ok ? expf(s[i] * scale - lq) : 0.f;
            ds[i] = p * (dp[i] - dq);
        }
        const Frag4<ST> dsf = frag4_from<ST>(ds);
#pragma unroll
        for (int db = 0; db < DH / 16; ++db) {
            float kt[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int j = j0 + 4 * g + i;
                kt[i] = j < n ? ld1<ST>(Kp + (size_t)j * RS + db * 16 + c16) : 0.f;
            }
            mma4(dQt[db], frag4_from<ST>(kt), dsf);
        }
        mfma_drain();  // the loop may exit right here
    }
    if (q < n) {
        const int pos = rtab ? (rI ? rI[base + q] : q) : 0;
#pragma unroll
        for (int db = 0; db < DH / 16; ++db) {
            float x[4] = {dQt[db][0] * scale, dQt[db][1] * scale, dQt[db][2] * scale, dQt[db][3] * scale};
            if (rtab) rope4_back<DH>(x, db * 16 + 4 * g, rtab, pos);
#pragma unroll
            for (int i = 0; i < 4; ++i) st1<ST>(dQKV + (base + q) * RS + db * 16 + 4 * g + i, x[i]);
        }
    }
}

// Tiled passes for n > 32 (bf16 storage): a workgroup owns OB = 16 CB NWV
// keys (kv pass) or queries (q pass) of one (b,h), 16 CB per wave, and walks
// the other side in tiles of 64 rows staged once in LDS for all its waves,
// row-major; the MFMAs that contract over rows (32 rows per MFMA, P and dS
// straight from registers) read their operands transposed with
// ds_read_b64_tr_b16.  Every fragment read from LDS feeds the CB column
// blocks of the wave, so CB = 2 halves the LDS traffic per MFMA (the passes
// are bound by it).  The next tile's global loads overlap the current tile's
// MFMAs.  The result does not depend on CB or NWV: every output element is
// one lane's fp32 accumulation over the tiles in order.
template <typename ST, int DH>
struct BwdTile {
    static constexpr int TB = 64, RS = 3 * DH;
    static constexpr int LDR = DH + 16 / (int)sizeof(ST);  // row-major rows
    static constexpr int VPR = DH / 8;
    // LDS of the two passes for OB owned rows; a kernel that may run either
    // pass takes the larger
    static constexpr size_t kv_lds(int ob) {
        const int sr = ob > TB ? ob : TB;
        return 2 * (size_t)sr * LDR * sizeof(ST) + 2 * TB * sizeof(float);
    }
    static constexpr size_t q_lds(int ob) {
        const int sr = ob > TB ? ob : TB;
        return (size_t)(sr + TB) * LDR * sizeof(ST);
    }
    static constexpr size_t both_lds(int ob) { return kv_lds(ob) > q_lds(ob) ? kv_lds(ob) : q_lds(ob); }
    // The 64-row tiles the loop walks are stored without padding, the 16-byte
    // units of row r XOR-permuted by swz(r), so that the three access patterns
    // are free of bank conflicts: 16-byte reads of one unit of 16 consecutive
    // rows (2 or 4 rows share a 256-byte line: swz takes distinct values on the
    // rows that share a line position), transposed 8-byte reads of two
    // adjacent units of 8 consecutive rows (swz even and distinct on those, up
    // to a common low bit, so the unit pairs stay distinct), and 16-byte row
    // writes.  (The output rows after the loop keep the padded stride LDR.)
    static constexpr int U = DH / 8, L = 16 / U;
    __device__ static int swz(int r) { return 2 * ((r / L) % (U / 2)) + ((r >> 3) & 1); }
    // element offset of (row r, column c) in such a tile
    __device__ static int off(int r, int c) { return r * DH + ((((c >> 3) ^ swz(r))) << 3) + (c & 7); }
};

template <typename ST, int DH, bool WIN, int NWV, int CB>
__device__ __forceinline__ void attn_bwd_kv_tiled_body(unsigned char* smem, int blk, const ST* __restrict__ QKV,
                                                       const ST* __restrict__ dA, const float* __restrict__ lse,
                                                       const float* __restrict__ D, int BH, int n, int causal, int lb,
                                                       float scale, ST* __restrict__ dQKV,
                                                       const int32_t* __restrict__ rI,
                                                       const float2* __restrict__ rtab) {
    using TL = BwdTile<ST, DH>;
    // OB keys owned by the workgroup (16 CB per wave), query tiles of TB rows
    constexpr int TB = TL::TB, RS = TL::RS, LDR = TL::LDR, VPR = TL::VPR, NT = 64 * NWV, OB = 16 * CB * NWV;
    constexpr int PER = TB * VPR / NT, SR = OB > TB ? OB : TB;
    static_assert(PER >= 1 && TB * VPR % NT == 0, "tile shape");
    static_assert(sizeof(ST) == 2, "bf16: transposed operands by ds_read_b64_tr_b16");
    ST* Qs = reinterpret_cast<ST*>(smem);  // query tile, then the dK rows
    ST* dAs = Qs + SR * LDR;               // dA tile, then the dV rows
    float* ls = reinterpret_cast<float*>(dAs + SR * LDR);
    float* Dsh = ls + TB;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, c16 = lane & 15;
    const int nqt = (n + TB - 1) / TB;
    // block order: the owned key blocks with the most query tiles (causal:
    // low kb) first, over all (b, h)
    const int bh = blk % BH, kb = blk / BH;
    const int k0 = kb * OB, wk0 = k0 + 16 * CB * wave;
    const size_t base = (size_t)bh * n;
    const ST* Qp = QKV + base * RS;
    const ST* Kp = Qp + DH;
    const ST* Vp = Qp + 2 * DH;
    const ST* dAp = dA + base * DH;

    int key[CB];  // this lane's keys (MFMA column of each column block)
    Frag8<ST> kf[CB][DH / 32], vf[CB][DH / 32];
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) {
        key[cb] = wk0 + 16 * cb + c16;
        const size_t krow = (size_t)min(key[cb], n - 1);
#pragma unroll
        for (int st = 0; st < DH / 32; ++st) {
            kf[cb][st] = frag8_load<ST>(Kp + krow * RS + st * 32 + 8 * g);
            vf[cb][st] = frag8_load<ST>(Vp + krow * RS + st * 32 + 8 * g);
        }
    }
    f32x4 dKt[CB][DH / 16], dVt[CB][DH / 16];
#pragma unroll
    for (int cb = 0; cb < CB; ++cb)
#pragma unroll
        for (int db = 0; db < DH / 16; ++db) dKt[cb][db] = dVt[cb][db] = zero4();

    // causal: query tiles from the block's own; with a window only those
    // within lb of its last key
    const int it0 = causal ? k0 / TB : 0, it_end = WIN && causal ? min(nqt, (k0 + OB - 1 + lb) / TB + 1) : nqt;
    const float c2 = scale * 1.44269504088896341f;  // P = 2^(s c2 - lse log2 e)
    Vec8<ST> qreg[PER], areg[PER];
    float lreg = 0.f, dreg = 0.f;
    // query rows past n are clamped to row n-1 (their scores are masked)
    auto load_tile = [&](int i0) {
#pragma unroll
        for (int p = 0; p < PER; ++p) {
            const int v = tid + NT * p, r = v / VPR, dc = (v % VPR) * 8;
            const size_t row = (size_t)min(i0 + r, n - 1);
            qreg[p] = vec8_load<ST>(Qp + row * RS + dc);
            areg[p] = vec8_load<ST>(dAp + row * DH + dc);
        }
        const size_t rq = (size_t)min(i0 + lane, n - 1);
        lreg = lse[base + rq] * 1.44269504088896341f;  // log2 e
        dreg = D[base + rq];
    };
    auto store_tile = [&]() {
#pragma unroll
        for (int p = 0; p < PER; ++p) {
            const int v = tid + NT * p, r = v / VPR, dc = (v % VPR) * 8;
            vec8_store<ST>(Qs + TL::off(r, dc), qreg[p]);
            vec8_store<ST>(dAs + TL::off(r, dc), areg[p]);
        }
        if (tid < TB) {
            ls[tid] = lreg;
            Dsh[tid] = dreg;
        }
    };

    load_tile(it0 * TB);
    const int kmax = wk0 + 16 * CB - 1;  // this wave's last key
    for (int it = it0; it < it_end; ++it) {
        const int i0 = it * TB;
        // every (query, key) pair of the tile and this wave is allowed: all
        // rows exist and, causal, the first query follows the wave's last key
        // (within the window)
        const bool full = i0 + TB <= n && kmax < n &&
                          (!causal || (i0 >= kmax && (!WIN || i0 + TB - 1 - wk0 <= lb)));
        __syncthreads();
        store_tile();
        __syncthreads();
        load_tile(min(it + 1, it_end - 1) * TB);
        // S and dP for 4 sub-blocks of 16 queries: lane = key c16 of each
        // column block, rows = queries 4g + i
        float p[CB][4][4], ds[CB][4][4];
#pragma unroll
        for (int sb = 0; sb < 4; ++sb) {
            f32x4 sv[CB], dp[CB];
#pragma unroll
            for (int cb = 0; cb < CB; ++cb) sv[cb] = dp[cb] = zero4();
#pragma unroll
            for (int st = 0; st < DH / 32; ++st) {
                const Frag8<ST> qa = frag8_load<ST>(Qs + TL::off(sb * 16 + c16, st * 32 + 8 * g));
                const Frag8<ST> aa = frag8_load<ST>(dAs + TL::off(sb * 16 + c16, st * 32 + 8 * g));
#pragma unroll
                for (int cb = 0; cb < CB; ++cb) {
                    mma8(sv[cb], qa, kf[cb][st]);
                    mma8(dp[cb], aa, vf[cb][st]);
                }
            }
            // no per-element mask where the whole tile is allowed for this wave
            auto scores = [&](auto all_allowed) {
#pragma unroll
                for (int cb = 0; cb < CB; ++cb)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int ql = sb * 16 + 4 * g + i, q = i0 + ql, kk = key[cb];
                        const bool ok = decltype(all_allowed)::value ||
                                        (q < n && kk < n && (!causal || (kk <= q && (!WIN || q - kk <= lb))));
                        p[cb][sb][i] = ok ? __builtin_amdgcn_exp2f(fmaf(sv[cb][i], c2, -ls[ql])) : 0.f;
                        ds[cb][sb][i] = p[cb][sb][i] * (dp[cb][i] - Dsh[ql]);
                    }
            };
            if (full) scores(std::true_type{});
            else scores(std::false_type{});
        }
        // dV^T += dA^T P and dK^T += Q^T dS over 32 queries per MFMA
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            Frag8<ST> pf[CB], dsf[CB];
#pragma unroll
            for (int cb = 0; cb < CB; ++cb) {
                const float pv[8] = {p[cb][2 * u][0], p[cb][2 * u][1], p[cb][2 * u][2], p[cb][2 * u][3],
                                     p[cb][2 * u + 1][0], p[cb][2 * u + 1][1], p[cb][2 * u + 1][2], p[cb][2 * u + 1][3]};
                const float dv[8] = {ds[cb][2 * u][0], ds[cb][2 * u][1], ds[cb][2 * u][2], ds[cb][2 * u][3],
                                     ds[cb][2 * u + 1][0], ds[cb][2 * u + 1][1], ds[cb][2 * u + 1][2],
                                     ds[cb][2 * u + 1][3]};
                pf[cb] = frag8_from<ST>(pv);
                dsf[cb] = frag8_from<ST>(dv);
            }
            // dA^T and Q^T over the queries of those slots, read transposed
            // from the row-major tiles: lane d columns 16 db + 4 (c16 % 4) ..
            // + 3 at query rows r0 and r0 + 16
            const int r0 = 32 * u + 4 * g + (c16 >> 2);
            u32x4 at[DH / 16], qt[DH / 16];
#pragma unroll
            for (int db = 0; db < DH / 16; ++db) {
                const int mcol = 16 * db + 4 * (c16 & 3);
                const int o0 = TL::off(r0, mcol), o1 = TL::off(r0 + 16, mcol);
                const u32x2 alo = lds_read_tr16(reinterpret_cast<const unsigned char*>(dAs + o0));
                const u32x2 ahi = lds_read_tr16(reinterpret_cast<const unsigned char*>(dAs + o1));
                const u32x2 qlo = lds_read_tr16(reinterpret_cast<const unsigned char*>(Qs + o0));
                const u32x2 qhi = lds_read_tr16(reinterpret_cast<const unsigned char*>(Qs + o1));
                at[db] = u32x4{alo.x, alo.y, ahi.x, ahi.y};
                qt[db] = u32x4{qlo.x, qlo.y, qhi.x, qhi.y};
            }
            lds_wait();
#pragma unroll
            for (int db = 0; db < DH / 16; ++db) {
                lds_ready(at[db]);
                lds_ready(qt[db]);
                Frag8<ST> fa, fq;
                fa.v = __builtin_bit_cast(bf16x8, at[db]);
                fq.v = __builtin_bit_cast(bf16x8, qt[db]);
#pragma unroll
                for (int cb = 0; cb < CB; ++cb) {
                    mma8(dVt[cb][db], fa, pf[cb]);
                    mma8(dKt[cb][db], fq, dsf[cb]);
                }
            }
        }
        mfma_drain();  // the loop may exit right here
    }

    // dK, dV rows (lane: key c16 of block cb, d rows db*16 + 4g + i) through
    // LDS to 16-byte stores
    __syncthreads();
    ST* Ks_out = Qs + wave * 16 * CB * LDR;
    ST* Vs_out = dAs + wave * 16 * CB * LDR;
#pragma unroll
    for (int cb = 0; cb < CB; ++cb)
#pragma unroll
        for (int db = 0; db < DH / 16; ++db)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int e = (16 * cb + c16) * LDR + db * 16 + 4 * g + i;
                if constexpr (sizeof(ST) == 2) {
                    Ks_out[e] = f32_to_bf16(dKt[cb][db][i] * scale);
                    Vs_out[e] = f32_to_bf16(dVt[cb][db][i]);
                } else {
                    Ks_out[e] = dKt[cb][db][i] * scale;
                    Vs_out[e] = dVt[cb][db][i];
                }
            }
    __syncthreads();
#pragma unroll
    for (int e = lane; e < 16 * CB * VPR; e += 64) {
        const int r = e / VPR, dc = (e % VPR) * 8;
        if (wk0 + r < n) {
            ST* out = dQKV + (base + wk0 + r) * RS;
            Vec8<ST> kv = vec8_load<ST>(Ks_out + r * LDR + dc);
            if (rtab && dc < DH / 2) {  // back through the rotation
                float x[8];
                vec8_to_f32<ST>(kv, x);
                rope8<DH>(x, dc, rtab, rI ? rI[base + wk0 + r] : wk0 + r, -1.f);
                kv = vec8_from_f32<ST>(x);
            }
            vec8_store<ST>(out + DH + dc, kv);
            vec8_store<ST>(out + 2 * DH + dc, vec8_load<ST>(Vs_out + r * LDR + dc));
        }
    }
}

template <typename ST, int DH, bool WIN, int NWV, int CB>
__device__ __forceinline__ void attn_bwd_q_tiled_body(unsigned char* smem, int blk, const ST* __restrict__ QKV,
                                                      const ST* __restrict__ dA, const float* __restrict__ lse,
                                                      const float* __restrict__ D, int BH, int n, int causal, int lb,
                                                      float scale, ST* __restrict__ dQKV,
                                                      const int32_t* __restrict__ rI,
                                                      const float2* __restrict__ rtab) {
    using TL = BwdTile<ST, DH>;
    // OB queries owned by the workgroup (16 CB per wave), key tiles of TB rows
    constexpr int TB = TL::TB, RS = TL::RS, LDR = TL::LDR, VPR = TL::VPR, NT = 64 * NWV, OB = 16 * CB * NWV;
    constexpr int PER = TB * VPR / NT, SR = OB > TB ? OB : TB;
    static_assert(PER >= 1 && TB * VPR % NT == 0, "tile shape");
    static_assert(sizeof(ST) == 2, "bf16: transposed operands by ds_read_b64_tr_b16");
    ST* Ks = reinterpret_cast<ST*>(smem);  // key tile, then the dQ rows
    ST* Vs = Ks + SR * LDR;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, c16 = lane & 15;
    const int nqb = (n + OB - 1) / OB;
    // block order: the owned query blocks with the most key tiles (causal:
    // high qb) first, over all (b, h)
    const int bh = blk % BH;
    const int qb = causal ? nqb - 1 - blk / BH : blk / BH;
    const int q0 = qb * OB, wq0 = q0 + 16 * CB * wave;
    const size_t base = (size_t)bh * n;
    const ST* Qp = QKV + base * RS;
    const ST* Kp = Qp + DH;
    const ST* Vp = Qp + 2 * DH;
    const ST* dAp = dA + base * DH;

    int q[CB];  // this lane's queries (MFMA column of each column block)
    Frag8<ST> qf[CB][DH / 32], af[CB][DH / 32];
    float lq[CB], dq[CB];
#pragma unroll
    for (int cb = 0; cb < CB; ++cb) {
        q[cb] = wq0 + 16 * cb + c16;
        const size_t qrow = (size_t)min(q[cb], n - 1);
#pragma unroll
        for (int st = 0; st < DH / 32; ++st) {
            qf[cb][st] = frag8_load<ST>(Qp + qrow * RS + st * 32 + 8 * g);
            af[cb][st] = frag8_load<ST>(dAp + qrow * DH + st * 32 + 8 * g);
        }
        lq[cb] = lse[base + qrow] * 1.44269504088896341f;  // lse in log2 units
        dq[cb] = D[base + qrow];
    }
    const float c2 = scale * 1.44269504088896341f;  // P = 2^(s c2 - lq)
    f32x4 dQt[CB][DH / 16];
#pragma unroll
    for (int cb = 0; cb < CB; ++cb)
#pragma unroll
        for (int db = 0; db < DH / 16; ++db) dQt[cb][db] = zero4();

    const int kv_end = causal ? min(n, q0 + OB) : n;
    const int ntiles = (kv_end + TB - 1) / TB, t0 = WIN && causal ? max(0, q0 - lb) / TB : 0;
    Vec8<ST> kreg[PER], vreg[PER];
    auto load_tile = [&](int j0) {
#pragma unroll
        for (int p = 0; p < PER; ++p) {
            const int v = tid + NT * p, r = v / VPR, dc = (v % VPR) * 8;
            const size_t row = (size_t)min(j0 + r, n - 1);
            kreg[p] = vec8_load<ST>(Kp + row * RS + dc);
            vreg[p] = vec8_load<ST>(Vp + row * RS + dc);
        }
    };
    auto store_tile = [&]() {
#pragma unroll
        for (int p = 0; p < PER; ++p) {
            const int v = tid + NT * p, r = v / VPR, dc = (v % VPR) * 8;
            vec8_store<ST>(Ks + TL::off(r, dc), kreg[p]);
            vec8_store<ST>(Vs + TL::off(r, dc), vreg[p]);
        }
    };

    load_tile(t0 * TB);
    const int qmax = wq0 + 16 * CB - 1;  // this wave's last query
    for (int t = t0; t < ntiles; ++t) {
        const int j0 = t * TB;
        // every (query, key) pair of the tile and this wave is allowed: all
        // rows exist and, causal, the tile's last key precedes the wave's
        // first query (the last query within the window of the first key)
        const bool full = j0 + TB <= n && qmax < n &&
                          (!causal || (j0 + TB - 1 <= wq0 && (!WIN || qmax - j0 <= lb)));
        __syncthreads();
        store_tile();
        __syncthreads();
        load_tile(min(t + 1, ntiles - 1) * TB);
        // S^T and dP^T for 4 sub-blocks of 16 keys: lane = query c16 of each
        // column block, rows = keys 4g + i
        float ds[CB][4][4];
#pragma unroll
        for (int sb = 0; sb < 4; ++sb) {
            f32x4 sv[CB], dp[CB];
#pragma unroll
            for (int cb = 0; cb < CB; ++cb) sv[cb] = dp[cb] = zero4();
#pragma unroll
            for (int st = 0; st < DH / 32; ++st) {
                const Frag8<ST> kk = frag8_load<ST>(Ks + TL::off(sb * 16 + c16, st * 32 + 8 * g));
                const Frag8<ST> vv = frag8_load<ST>(Vs + TL::off(sb * 16 + c16, st * 32 + 8 * g));
#pragma unroll
                for (int cb = 0; cb < CB; ++cb) {
                    mma8(sv[cb], kk, qf[cb][st]);
                    mma8(dp[cb], vv, af[cb][st]);
                }
            }
            // no per-element mask where the whole tile is allowed for this wave
            auto scores = [&](auto all_allowed) {
#pragma unroll
                for (int cb = 0; cb < CB; ++cb)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int j = j0 + sb * 16 + 4 * g + i, qq = q[cb];
                        const bool ok = decltype(all_allowed)::value ||
                                        (j < n && qq < n && (!causal || (j <= qq && (!WIN || qq - j <= lb))));
                        const float pp = ok ? __builtin_amdgcn_exp2f(fmaf(sv[cb][i], c2, -lq[cb])) : 0.f;
                        ds[cb][sb][i] = pp * (dp[cb][i] - dq[cb]);
                    }
            };
            if (full) scores(std::true_type{});
            else scores(std::false_type{});
        }
        // dQ^T += K^T dS^T over 32 keys per MFMA
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            Frag8<ST> dsf[CB];
#pragma unroll
            for (int cb = 0; cb < CB; ++cb) {
                const float dv[8] = {ds[cb][2 * u][0], ds[cb][2 * u][1], ds[cb][2 * u][2], ds[cb][2 * u][3],
                                     ds[cb][2 * u + 1][0], ds[cb][2 * u + 1][1], ds[cb][2 * u + 1][2],
                                     ds[cb][2 * u + 1][3]};
                dsf[cb] = frag8_from<ST>(dv);
            }
            // K^T over the keys of those slots, read transposed from the row-major tile
            const int r0 = 32 * u + 4 * g + (c16 >> 2);
            u32x4 kt[DH / 16];
#pragma unroll
            for (int db = 0; db < DH / 16; ++db) {
                const int mcol = 16 * db + 4 * (c16 & 3);
                const u32x2 lo = lds_read_tr16(reinterpret_cast<const unsigned char*>(Ks + TL::off(r0, mcol)));
                const u32x2 hi = lds_read_tr16(reinterpret_cast<const unsigned char*>(Ks + TL::off(r0 + 16, mcol)));
                kt[db] = u32x4{lo.x, lo.y, hi.x, hi.y};
            }
            lds_wait();
#pragma unroll
            for (int db = 0; db < DH / 16; ++db) {
                lds_ready(kt[db]);
                Frag8<ST> fk;
                fk.v = __builtin_bit_cast(bf16x8, kt[db]);
#pragma unroll
                for (int cb = 0; cb < CB; ++cb) mma8(dQt[cb][db], fk, dsf[cb]);
            }
        }
        mfma_drain();  // the loop may exit right here
    }

    __syncthreads();
    ST* Qs_out = Ks + wave * 16 * CB * LDR;
#pragma unroll
    for (int cb = 0; cb < CB; ++cb)
#pragma unroll
        for (int db = 0; db < DH / 16; ++db)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int e = (16 * cb + c16) * LDR + db * 16 + 4 * g + i;
                if constexpr (sizeof(ST) == 2) Qs_out[e] = f32_to_bf16(dQt[cb][db][i] * scale);
                else Qs_out[e] = dQt[cb][db][i] * scale;
            }
    __syncthreads();
#pragma unroll
    for (int e = lane; e < 16 * CB * VPR; e += 64) {
        const int r = e / VPR, dc = (e % VPR) * 8;
        if (wq0 + r < n) {
            Vec8<ST> qv = vec8_load<ST>(Qs_out + r * LDR + dc);
            if (rtab && dc < DH / 2) {  // back through the rotation
                float x[8];
                vec8_to_f32<ST>(qv, x);
                rope8<DH>(x, dc, rtab, rI ? rI[base + wq0 + r] : wq0 + r, -1.f);
                qv = vec8_from_f32<ST>(x);
            }
            vec8_store<ST>(dQKV + (base + wq0 + r) * RS + dc, qv);
        }
    }
}

#define MOSA_BWD_TILED_PARAMS                                                                                    \
    const ST *__restrict__ QKV, const ST *__restrict__ dA, const float *__restrict__ lse,                          \
        const float *__restrict__ D, int BH, int n, int causal, int lb, float scale, ST *__restrict__ dQKV,       \
        const int32_t *__restrict__ rI, const float2 *__restrict__ rtab
#define MOSA_BWD_TILED_ARGS QKV, dA, lse, D, BH, n, causal, lb, scale, dQKV, rI, rtab

// Both passes in one launch (they are independent): blocks of even rank take
// the dK, dV pass, odd ranks the dQ pass, each in its longest-first order, so
// the short blocks of one pass fill the CUs beside the long blocks of the
// other.  Ranks go to workgroups in rounds of one per CU (the dispatcher
// hands workgroup b and b + 256 to the same CU), every second round in reverse,
// so that the blocks a CU receives add up to about the same number of tiles
// (causal, hybrid_d1024: 32 per CU instead of 24 to 40; 54 -> 48 us).
// Register budget: 3 waves per SIMD with one column block per wave (more of
// the MoSA heads' waves fit beside it in the hybrid layer's backward, 0.435 ->
// 0.431 ms per step), 2 with two (254 registers, no spills).
template <typename ST, int DH, bool WIN, int NWV, int CB>
__global__ __launch_bounds__(64 * NWV, CB == 1 ? 3 : 2) void attn_bwd_tiled_both_kernel(MOSA_BWD_TILED_PARAMS) {
    // one LDS buffer for whichever pass the block runs
    __shared__ __attribute__((aligned(16))) unsigned char smem[BwdTile<ST, DH>::both_lds(16 * CB * NWV)];
    constexpr int kRound = 256;
    const int b = blockIdx.x, m = b / kRound;
    const int s = ((m & 1) && (m + 1) * kRound <= (int)gridDim.x) ? m * kRound + (kRound - 1 - b % kRound) : b;
    if (s & 1) attn_bwd_q_tiled_body<ST, DH, WIN, NWV, CB>(smem, s >> 1, MOSA_BWD_TILED_ARGS);
    else attn_bwd_kv_tiled_body<ST, DH, WIN, NWV, CB>(smem, s >> 1, MOSA_BWD_TILED_ARGS);
}
#undef MOSA_BWD_TILED_PARAMS
#undef MOSA_BWD_TILED_ARGS

// bf16, n <= 128: both passes in one workgroup of 8 waves per (b, h).  Q, K,
// V and dA of all n rows go into LDS once (direct global->LDS loads, rows
// with XOR-permuted 16-byte units), with lse and D.  Phase 1, wave w owns key
// block w: S and dP with the key in the lane (B operands K and V from
// registers), P and dS, dV^T += dA^T P and dK^T += Q^T dS 32 queries per MFMA
// (dA^T and Q^T by transposed LDS reads in the query order of the P and dS
// registers), and dS (bf16, the MFMA operand value) into an LDS tile
// [query][key].  Phase 2, wave w owns query block w: dQ^T += K^T dS^T 32 keys
// per MFMA from that tile.  No value is accumulated by more than one lane, so
// the result is reproducible; the roundings are those of the two-pass kernels
// (P and dS enter the MFMAs as bf16).
constexpr int kAttnBwdLdsMaxN = 128;

template <int DH>
struct AttnBwdLds {
    static constexpr int NMAX = kAttnBwdLdsMaxN, LPR = DH / 8, NW = NMAX / 16;
    static constexpr int TILE = NMAX * DH * 2;           // Q, K, V, dA tiles
    static constexpr int DS_BYTES = NMAX * NMAX * 2;     // dS [query][key], 16 units per row
    static constexpr size_t lds = 4 * (size_t)TILE + DS_BYTES + 2 * NMAX * 4;
};

template <int DH>
__global__ __launch_bounds__(512) void attn_bwd_lds_kernel(const uint16_t* __restrict__ QKV,
                                                           const uint16_t* __restrict__ dA,
                                                           const float* __restrict__ lse, const float* __restrict__ D,
                                                           int BH, int n, int causal, float scale,
                                                           uint16_t* __restrict__ dQKV, const int32_t* __restrict__ rI,
                                                           const float2* __restrict__ rtab) {
    using ST = uint16_t;
    using L = AttnBwdLds<DH>;
    constexpr int RS = 3 * DH, NMAX = L::NMAX, LPR = L::LPR, NW = L::NW, TILE = L::TILE;
    constexpr int PER = NMAX * LPR / (64 * NW);  // DMA instructions per wave per tile
    static_assert(PER >= 1 && NMAX * LPR % (64 * NW) == 0, "tile shape");
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
    unsigned char* const Qs = smem;
    unsigned char* const Ks = smem + TILE;
    unsigned char* const Vs = smem + 2 * TILE;
    unsigned char* const dAs = smem + 3 * TILE;
    unsigned char* const dSs = smem + 4 * TILE;
    float* const lse_s = reinterpret_cast<float*>(dSs + L::DS_BYTES);
    float* const D_s = lse_s + NMAX;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, c16 = lane & 15;
    const int bh = xcd_logical_id(blockIdx.x, gridDim.x);
    const size_t base = (size_t)bh * n;
    const ST* Qp = QKV + base * RS;
    const ST* dAp = dA + base * DH;

    {
        const uint32_t lb = __builtin_amdgcn_readfirstlane(lds_addr(smem)) + 1024 * __builtin_amdgcn_readfirstlane(wave);
#pragma unroll
        for (int j = 0; j < PER; ++j) {
            const int p = 64 * (wave + NW * j) + lane, row = p / LPR, pos = p % LPR;
            const int col = 8 * (pos ^ kswz(row, LPR));
            const size_t r = (size_t)min(row, n - 1);
            const uint32_t off = lb + 1024 * NW * j;
            lds_load16(Qp + r * RS + col, off);
            lds_load16(Qp + r * RS + DH + col, off + TILE);
            lds_load16(Qp + r * RS + 2 * DH + col, off + 2 * TILE);
            lds_load16(dAp + r * DH + col, off + 3 * TILE);
        }
    }
    if (tid < NMAX) {
        const size_t r = base + min(tid, n - 1);
        lse_s[tid] = lse[r] * 1.44269504088896341f;  // log2 e: P = 2^(s c - lse log2 e)
        D_s[tid] = D[r];
    }
    wait_vmcnt<0>();
    __syncthreads();

    // k-contiguous operand: row `row`, d = 32 st + 8 g .. + 7
    auto frag_k = [&](const unsigned char* t, int row, int st) {
        const int u = 4 * st + g;
        Frag8<ST> f;
        f.v = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(t + (row * LPR + (u ^ kswz(row, LPR))) * 16));
        return f;
    };
    // transposed read of 4 rows k .. k + 3 (k = kb0 + (c16 >> 2) per source lane) at columns mcol .. + 3
    auto tr4 = [&](const unsigned char* t, int k, int mcol) {
        const int un = mcol >> 3, half = (mcol >> 2) & 1;
        return lds_read_tr16(t + (k * LPR + (un ^ kswz(k, LPR))) * 16 + 8 * half);
    };
    // A operand X^T (rows d = dbase + c16) over rows {kb + 4 g + i, kb + 16 + 4 g + i}
    // of a row-major tile: the order of two D-layout register blocks
    auto trA_pair = [&](const unsigned char* t, int dbase, int kb) {
        const int k0 = kb + 4 * g + (c16 >> 2), mcol = dbase + 4 * (c16 & 3);
        const u32x2 lo = tr4(t, k0, mcol), hi = tr4(t, k0 + 16, mcol);
        return u32x4{lo.x, lo.y, hi.x, hi.y};
    };
    // A operand X^T over consecutive rows kb + 8 g .. + 7
    auto trA_run = [&](const unsigned char* t, int dbase, int kb) {
        const int k0 = kb + 8 * g + (c16 >> 2), mcol = dbase + 4 * (c16 & 3);
        const u32x2 lo = tr4(t, k0, mcol), hi = tr4(t, k0 + 4, mcol);
        return u32x4{lo.x, lo.y, hi.x, hi.y};
    };
    auto ds_unit = [](int q, int key8) { return q * 16 + ((key8 >> 3) ^ (q & 15)); };  // dS tile, 16-byte unit

    const int nb = (n + 15) / 16;
    // With 8 blocks the causal work of block b is 8 - b (phase 1) or b + 1
    // (phase 2); waves w and w + 4 share a SIMD, so they take blocks s and
    // 7 - s: every SIMD gets the same work.
    const int blk = nb == 8 && causal && wave >= 4 ? 11 - wave : wave;
    const float c2 = scale * 1.44269504088896341f;
    // Phase 1: key block kb.
    if (blk < nb) {
        const int kb = blk, key = 16 * kb + c16;
        const int qmin = key >= n ? n : (causal ? key : 0);  // first query that sees this key
        Frag8<ST> kf[DH / 32], vf[DH / 32];
#pragma unroll
        for (int st = 0; st < DH / 32; ++st) {
            kf[st] = frag_k(Ks, key, st);
            vf[st] = frag_k(Vs, key, st);
        }
        f32x4 dKt[DH / 16], dVt[DH / 16];
#pragma unroll
        for (int db = 0; db < DH / 16; ++db) dKt[db] = dVt[db] = zero4();
        for (int u = causal ? kb / 2 : 0; 2 * u < nb; ++u) {
            float p[2][4], ds[2][4];
#pragma unroll
            for (int hq = 0; hq < 2; ++hq) {
                const int qb = 2 * u + hq;
                f32x4 s = zero4(), dp = zero4();
                if (qb < nb) {
#pragma unroll
                    for (int st = 0; st < DH / 32; ++st) {
                        mma8(s, frag_k(Qs, 16 * qb + c16, st), kf[st]);
                        mma8(dp, frag_k(dAs, 16 * qb + c16, st), vf[st]);
                    }
                }
                mfma_drain();
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int q = 16 * qb + 4 * g + i;
                    const bool ok = qb < nb && q >= qmin && q < n;
                    const float pv = ok ? __builtin_amdgcn_exp2f(fmaf(s[i], c2, -lse_s[q & (NMAX - 1)])) : 0.f;
                    const float dsv = pv * (dp[i] - D_s[q & (NMAX - 1)]);
                    p[hq][i] = pv;
                    ds[hq][i] = dsv;
                    if (qb < nb) {
                        ST* dst = reinterpret_cast<ST*>(dSs + ds_unit(q, key) * 16) + (key & 7);
                        *dst = f32_to_bf16(dsv);
                    }
                }
            }
            // dV^T += dA^T P, dK^T += Q^T dS over the 32 queries 32 u + {4 g + i, 16 + 4 g + i}
            const float pv8[8] = {p[0][0], p[0][1], p[0][2], p[0][3], p[1][0], p[1][1], p[1][2], p[1][3]};
            const float ds8[8] = {ds[0][0], ds[0][1], ds[0][2], ds[0][3], ds[1][0], ds[1][1], ds[1][2], ds[1][3]};
            const Frag8<ST> pf = frag8_from<ST>(pv8), dsf = frag8_from<ST>(ds8);
            u32x4 at[DH / 16], qt[DH / 16];
#pragma unroll
            for (int db = 0; db < DH / 16; ++db) {
                at[db] = trA_pair(dAs, 16 * db, 32 * u);
                qt[db] = trA_pair(Qs, 16 * db, 32 * u);
            }
            lds_wait();
#pragma unroll
            for (int db = 0; db < DH / 16; ++db) {
                lds_ready(at[db]);
                lds_ready(qt[db]);
                Frag8<ST> fa, fq;
                fa.v = __builtin_bit_cast(bf16x8, at[db]);
                fq.v = __builtin_bit_cast(bf16x8, qt[db]);
                mma8(dVt[db], fa, pf);
                mma8(dKt[db], fq, dsf);
            }
        }
        mfma_drain();
        if (key < n) {
            ST* out = dQKV + (base + key) * RS;
            const int pos = rtab ? (rI ? rI[base + key] : key) : 0;
#pragma unroll
            for (int db = 0; db < DH / 16; ++db) {
                // lane: key c16, d = 16 db + 4 g + i
                float x[4] = {dKt[db][0] * scale, dKt[db][1] * scale, dKt[db][2] * scale, dKt[db][3] * scale};
                if (rtab) rope4_back<DH>(x, 16 * db + 4 * g, rtab, pos);
                *reinterpret_cast<uint2*>(out + DH + 16 * db + 4 * g) =
                    make_uint2(pack_bf16x2(x[0], x[1]), pack_bf16x2(x[2], x[3]));
                *reinterpret_cast<uint2*>(out + 2 * DH + 16 * db + 4 * g) =
                    make_uint2(pack_bf16x2(dVt[db][0], dVt[db][1]), pack_bf16x2(dVt[db][2], dVt[db][3]));
            }
        }
    }
    __syncthreads();  // the dS tile is complete
    // Phase 2: query block qb = blk: dQ^T += K^T dS^T over 32 keys per MFMA.
    if (blk < nb) {
        const int qb = blk, q = 16 * qb + c16;
        f32x4 dQt[DH / 16];
#pragma unroll
        for (int db = 0; db < DH / 16; ++db) dQt[db] = zero4();
        const int nk = causal ? 16 * (qb + 1) : 16 * nb;
        for (int u = 0; 32 * u < nk; ++u) {
            // dS^T[keys 32 u + 8 g .. + 7][q] = dS[q][...]; key blocks past the
            // last one were never written and count as zero
            const int k8 = 32 * u + 8 * g;
            Frag8<ST> sf;
            sf.v = __builtin_bit_cast(bf16x8, k8 < 16 * nb ? *reinterpret_cast<const uint4*>(dSs + ds_unit(q, k8) * 16)
                                                           : make_uint4(0u, 0u, 0u, 0u));
            u32x4 kt[DH / 16];
#pragma unroll
            for (int db = 0; db < DH / 16; ++db) kt[db] = trA_run(Ks, 16 * db, 32 * u);
            lds_wait();
#pragma unroll
            for (int db = 0; db < DH / 16; ++db) {
                lds_ready(kt[db]);
                Frag8<ST> fk;
                fk.v = __builtin_bit_cast(bf16x8, kt[db]);
                mma8(dQt[db], fk, sf);
            }
        }
        mfma_drain();
        if (q < n) {
            ST* out = dQKV + (base + q) * RS;
            const int pos = rtab ? (rI ? rI[base + q] : q) : 0;
#pragma unroll
            for (int db = 0; db < DH / 16; ++db) {
                float x[4] = {dQt[db][0] * scale, dQt[db][1] * scale, dQt[db][2] * scale, dQt[db][3] * scale};
                if (rtab) rope4_back<DH>(x, 16 * db + 4 * g, rtab, pos);
                *reinterpret_cast<uint2*>(out + 16 * db + 4 * g) =
                    make_uint2(pack_bf16x2(x[0], x[1]), pack_bf16x2(x[2], x[3]));
            }
        }
    }
}

// bf16, at most 16 rows per (b, h) (one 16-row block): both passes in one
// wave per (b, h), no loop.  The wave loads the rows of Q, K, V and dA as
// MFMA fragments (lane: row c16, 8 consecutive head columns), computes S and
// dP (lane: query 4g + i, key c16), P and dS (rounded to bf16 as MFMA
// operands, as in the other kernels), and keeps Q, K, dA and dS ([query][key])
// in its own LDS region, from which the transposed operands of
// dV^T += dA^T P, dK^T += Q^T dS and dQ^T += K^T dS^T are read (16 rows per
// MFMA).  A lane ends with 4 consecutive head columns of one row of dQ, dK
// and dV, stored 8 bytes at a time.  No value is accumulated by more than one
// lane: reproducible.
template <int DH>
__global__ __launch_bounds__(256) void attn_bwd_small_kernel(const uint16_t* __restrict__ QKV,
                                                             const uint16_t* __restrict__ dA,
                                                             const float* __restrict__ lse,
                                                             const float* __restrict__ D, int BH, int n, int causal,
                                                             float scale, uint16_t* __restrict__ dQKV,
                                                             const int32_t* __restrict__ rI,
                                                             const float2* __restrict__ rtab) {
    using ST = uint16_t;
    using TL = BwdTile<ST, DH>;  // 16-byte units of a row XOR-permuted (conflict-free transposed reads)
    constexpr int RS = 3 * DH, NS = DH / 32, NDB = DH / 16, TILE = 16 * DH;
    __shared__ __attribute__((aligned(16))) ST lds[4][3 * TILE + 16 * 16];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int g = lane >> 4, c16 = lane & 15;
    const int bh = blockIdx.x * 4 + wave;
    if (bh >= BH) return;
    ST* Qs = lds[wave];
    ST* Ks = Qs + TILE;
    ST* As = Ks + TILE;
    ST* dSs = As + TILE;
    const size_t base = (size_t)bh * n;
    const ST* Qp = QKV + base * RS;
    const ST* dAp = dA + base * DH;
    const bool rv = c16 < n;  // this lane's row (fragment row c16) exists

    Frag8<ST> qf[NS], kf[NS], vf[NS], af[NS];
#pragma unroll
    for (int st = 0; st < NS; ++st) {
        const size_t o = (size_t)c16 * RS + st * 32 + 8 * g;
        qf[st] = rv ? frag8_load<ST>(Qp + o) : frag8_zero<ST>();
        kf[st] = rv ? frag8_load<ST>(Qp + DH + o) : frag8_zero<ST>();
        vf[st] = rv ? frag8_load<ST>(Qp + 2 * DH + o) : frag8_zero<ST>();
        af[st] = rv ? frag8_load<ST>(dAp + (size_t)c16 * DH + st * 32 + 8 * g) : frag8_zero<ST>();
    }
    float l[4], dd[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int q = 4 * g + i;
        l[i] = q < n ? lse[base + q] : 0.f;
        dd[i] = q < n ? D[base + q] : 0.f;
    }
    // Q, K, dA rows into the wave's tiles (rows past n hold zeros)
#pragma unroll
    for (int st = 0; st < NS; ++st) {
        const int o = TL::off(c16, st * 32 + 8 * g);
        *reinterpret_cast<uint4*>(Qs + o) = __builtin_bit_cast(uint4, qf[st].v);
        *reinterpret_cast<uint4*>(Ks + o) = __builtin_bit_cast(uint4, kf[st].v);
        *reinterpret_cast<uint4*>(As + o) = __builtin_bit_cast(uint4, af[st].v);
    }

    f32x4 sv = zero4(), dp = zero4();
#pragma unroll
    for (int st = 0; st < NS; ++st) {
        mma8(sv, qf[st], kf[st]);
        mma8(dp, af[st], vf[st]);
    }
    // lane: key c16, queries 4g + i
    float p[4], ds[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int q = 4 * g + i;
        const bool ok = q < n && rv && (!causal || c16 <= q);
        p[i] = ok ? expf(sv[i] * scale - l[i]) : 0.f;
        ds[i] = p[i] * (dp[i] - dd[i]);
    }
    const Frag4<ST> pf = frag4_from<ST>(p), dsf = frag4_from<ST>(ds);
    // dS as rounded for the MFMAs, [query][key], for its transposed use in dQ
    {
        const uint2 w = __builtin_bit_cast(uint2, dsf.v);
        dSs[(4 * g + 0) * 16 + c16] = (ST)(w.x & 0xffffu);
        dSs[(4 * g + 1) * 16 + c16] = (ST)(w.x >> 16);
        dSs[(4 * g + 2) * 16 + c16] = (ST)(w.y & 0xffffu);
        dSs[(4 * g + 3) * 16 + c16] = (ST)(w.y >> 16);
    }
    // B operand of dQ^T: dS[query c16][keys 4g .. 4g + 3] (the wave's own LDS
    // writes above complete before this read)
    Frag4<ST> dstf;
    dstf.v = __builtin_bit_cast(s16x4, *reinterpret_cast<const uint2*>(dSs + c16 * 16 + 4 * g));

    f32x4 dVt[NDB], dKt[NDB], dQt[NDB];
    // transposed reads: source lane supplies row 4g + c16 / 4, 4 columns from
    // 16 db + 4 (c16 % 4); lane receives rows 4g .. 4g + 3 of column 16 db + c16
    const int rr = 4 * g + (c16 >> 2);
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
        const int o = TL::off(rr, 16 * db + 4 * (c16 & 3));
        u32x2 at = lds_read_tr16(reinterpret_cast<const unsigned char*>(As + o));
        u32x2 qt = lds_read_tr16(reinterpret_cast<const unsigned char*>(Qs + o));
        u32x2 kt = lds_read_tr16(reinterpret_cast<const unsigned char*>(Ks + o));
        lds_wait();
        // the values exist only after the wait: tie their uses to it
        asm volatile("" : "+v"(at), "+v"(qt), "+v"(kt));
        Frag4<ST> fa, fq, fk;
        fa.v = __builtin_bit_cast(s16x4, at);
        fq.v = __builtin_bit_cast(s16x4, qt);
        fk.v = __builtin_bit_cast(s16x4, kt);
        dVt[db] = dKt[db] = dQt[db] = zero4();
        mma4(dVt[db], fa, pf);
        mma4(dKt[db], fq, dsf);
        mma4(dQt[db], fk, dstf);
    }
    mfma_drain();
    if (rv) {
        // lane: row c16 (key for dK, dV; query for dQ), head columns 16 db + 4g .. + 3
        const int pos = rtab ? (rI ? rI[base + c16] : c16) : 0;
        ST* out = dQKV + (base + c16) * RS;
#pragma unroll
        for (int db = 0; db < NDB; ++db) {
            const int d0 = 16 * db + 4 * g;
            float xq[4] = {dQt[db][0] * scale, dQt[db][1] * scale, dQt[db][2] * scale, dQt[db][3] * scale};
            float xk[4] = {dKt[db][0] * scale, dKt[db][1] * scale, dKt[db][2] * scale, dKt[db][3] * scale};
            if (rtab) {  // back through the rotation
                rope4_back<DH>(xq, d0, rtab, pos);
                rope4_back<DH>(xk, d0, rtab, pos);
            }
            *reinterpret_cast<uint2*>(out + d0) = make_uint2(pack_bf16x2(xq[0], xq[1]), pack_bf16x2(xq[2], xq[3]));
            *reinterpret_cast<uint2*>(out + DH + d0) =
                make_uint2(pack_bf16x2(xk[0], xk[1]), pack_bf16x2(xk[2], xk[3]));
            *reinterpret_cast<uint2*>(out + 2 * DH + d0) =
                make_uint2(pack_bf16x2(dVt[db][0], dVt[db][1]), pack_bf16x2(dVt[db][2], dVt[db][3]));
        }
    }
}

template <typename ST>
int launch_t(const ST* QKV, const ST* dA, const float* lse, const float* D, int BH, int n, int dh, int causal,
             int window, ST* dQKV, const int32_t* rI, const float2* rtab, int pass, hipStream_t stream) {
    const float scale = 1.0f / sqrtf((float)dh);
    const int lb = window > 0 ? window - 1 : n;  // keys a query may look back
    if constexpr (sizeof(ST) == 2) {
      if (n <= 16 && window == 0 && (dh == 64 || dh == 32)) {
        // both passes in one launch: the call for the dQ pass has nothing left to do
        if (pass == 1 || BH == 0) return 0;
        auto kern = dh == 64 ? attn_bwd_small_kernel<64> : attn_bwd_small_kernel<32>;
        hipLaunchKernelGGL(kern, dim3((BH + 3) / 4), dim3(256), 0, stream, QKV, dA, lse, D, BH, n, causal, scale,
                           dQKV, rI, rtab);
        return hipGetLastError() == hipSuccess ? 0 : -1;
      }
      if (n > 32 && n <= kAttnBwdLdsMaxN && window == 0) {
        // both passes in one launch: the call for the dQ pass has nothing left to do
        if (pass == 1) return 0;
        auto kern = dh == 64 ? attn_bwd_lds_kernel<64> : attn_bwd_lds_kernel<32>;
        const size_t lds = dh == 64 ? AttnBwdLds<64>::lds : AttnBwdLds<32>::lds;
        if (allow_lds((const void*)kern, lds)) return -1;
        hipLaunchKernelGGL(kern, dim3(BH), dim3(512), lds, stream, QKV, dA, lse, D, BH, n, causal, scale, dQKV, rI,
                           rtab);
        return hipGetLastError() == hipSuccess ? 0 : -1;
      }
      if (n > 32 || window > 0) {
        // 4 waves per workgroup, 16 CB owned rows per wave.  Two column
        // blocks (half the LDS reads per MFMA, 2 waves per SIMD) where the
        // rows are long (n >= 1024, no window) and the blocks still give
        // every CU two workgroups (4 dense heads, B = 8, T = 1024: 44 -> 39.5 us); one
        // otherwise (measured slower with two: n = 512 MoSA heads, local
        // windows, a single head of T = 8192 that fills half the chip).
        if (pass != 2) return -1;  // both passes are one launch here
#define MOSA_ATTN_BWD_T(DHV, CBV)                                                                      \
    do {                                                                                                \
        constexpr int NWV = 4, CB = CBV, OB = 16 * CB * NWV;                                            \
        auto kern = window > 0 ? attn_bwd_tiled_both_kernel<ST, DHV, true, NWV, CB>                     \
                               : attn_bwd_tiled_both_kernel<ST, DHV, false, NWV, CB>;                   \
        const dim3 grid(2 * BH * ((n + OB - 1) / OB)), block(64 * NWV);                                 \
        hipLaunchKernelGGL(kern, grid, block, 0, stream, QKV, dA, lse, D, BH, n, causal, lb, scale, dQKV, rI, rtab); \
    } while (0)
#define MOSA_ATTN_BWD_TD(CBV)                                                                          \
    do {                                                                                                \
        if (dh == 64) MOSA_ATTN_BWD_T(64, CBV);                                                         \
        else MOSA_ATTN_BWD_T(32, CBV);                                                                  \
    } while (0)
        const bool wide = window == 0 && n >= 1024 && 2LL * BH * ((n + 127) / 128) >= 512;
        if (wide) MOSA_ATTN_BWD_TD(2);
        else MOSA_ATTN_BWD_TD(1);
#undef MOSA_ATTN_BWD_TD
#undef MOSA_ATTN_BWD_T
        return hipGetLastError() == hipSuccess ? 0 : -1;
      }
    }
    if (pass == 2)
        return launch_t<ST>(QKV, dA, lse, D, BH, n, dh, causal, window, dQKV, rI, rtab, 0, stream) |
               launch_t<ST>(QKV, dA, lse, D, BH, n, dh, causal, window, dQKV, rI, rtab, 1, stream);
    const int tasks = BH * ((n + 15) / 16);
    dim3 grid((tasks + 3) / 4), block(256);
#define MOSA_ATTN_BWD(KERN, DHV)                                                                     \
    do {                                                                                              \
        auto kern = window > 0 ? KERN<ST, DHV, true> : KERN<ST, DHV, false>;                          \
        hipLaunchKernelGGL(kern, grid, block, 0, stream, QKV, dA, lse, D, BH, n, causal, lb, scale, dQKV, rI, rtab); \
    } while (0)
    if (pass == 0) {
        if (dh == 64) MOSA_ATTN_BWD(attn_bwd_kv_kernel, 64);
        else MOSA_ATTN_BWD(attn_bwd_kv_kernel, 32);
    } else {
        if (dh == 64) MOSA_ATTN_BWD(attn_bwd_q_kernel, 64);
        else MOSA_ATTN_BWD(attn_bwd_q_kernel, 32);
    }
#undef MOSA_ATTN_BWD
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

}  // namespace

// One launch for both passes where a kernel does both (bf16: the one-wave
// kernel for n <= 16, the LDS kernel for 32 < n <= its limit, the tiled
// kernels otherwise), else the two passes.
template <typename ST>
bool both_in_one(int n, int window) {
    if constexpr (sizeof(ST) == 2) return n > 32 || window > 0 || n <= 16;
    return false;
}

int launch_attn_bwd(int dtype, const void* QKV, const void* dA, const float* lse, const float* D, int BH, int n,
                    int dh, int causal, int window, void* dQKV, const int32_t* rope_I, const float2* rope,
                    int dense, const Marker& mk, hipStream_t stream) {
    auto run = [&](auto tag, int pass) {
        using ST = decltype(tag);
        return launch_t<ST>((const ST*)QKV, (const ST*)dA, lse, D, BH, n, dh, causal, window, (ST*)dQKV, rope_I,
                            rope, pass, stream);
    };
    auto go = [&](auto tag) {
        using ST = decltype(tag);
        if (both_in_one<ST>(n, window)) {
            const int e = run(tag, 2);
            return e | mk(dense ? "attn_bwd_dense" : "attn_bwd");
        }
        int e = run(tag, 0);
        e |= mk(dense ? "attn_bwd_kv_dense" : "attn_bwd_kv");
        e |= run(tag, 1);
        return e | mk(dense ? "attn_bwd_q_dense" : "attn_bwd_q");
    };
    return dtype == kBF16 ? go(uint16_t{}) : go(float{});
}

}  // namespace mosa
