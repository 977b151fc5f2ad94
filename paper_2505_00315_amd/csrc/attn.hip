// Attention among the selected tokens of one head (paper Eq. 1 with the
// index-aware mask of Section 2.2: M_ij = 0 iff I_i >= I_j).  I is ascending,
// so the mask is the ordinary lower triangle in slot order; without the
// causal flag every pair is allowed.  The same kernel runs the dense heads
// (n = T).
//
// Flash-style, one wave per task of 16 query rows; a workgroup of 4 waves
// runs 4 independent tasks.  Per block of 16 keys:
//   S^T = K Q^T        MFMA K = 32 over d_head (A = K rows, B = Q rows),
//                      the lane then holds query (lane % 16) and keys 4g+i;
//   online softmax     row max / row sum reduced across the 4 lane groups
//                      with two xor-shuffles;
//   O^T += V^T P^T     MFMA K = 16 over the 16 keys: the S^T tile is already
//                      in the K = 16 operand layout, so P never leaves the
//                      registers.
// Outputs A = r_i O_i / l_i (storage type; the router value r_i of the row
// applied once here, as Section 2.2's diag(r), so later stages read a scaled
// row; r = 1 for dense heads) and lse = m + log(l) (fp32, natural log).
#include "common.h"
#include "gemm.h"
#include "attn_lds.h"
#include "gemm2.h"
#include "kernels.h"
#include "tiles.h"

namespace mosa {

namespace {

template <typename ST, int DH>
__global__ __launch_bounds__(256) void attn_fwd_kernel(const ST* __restrict__ QKV, int BH, int n, int causal,
                                                       float scale, const float* __restrict__ rw, ST* __restrict__ A,
                                                       float* __restrict__ lse) {
    constexpr int RS = 3 * DH;  // row stride of the packed Q | K | V rows
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int g = lane >> 4, c16 = lane & 15;
    const int nqb = (n + 15) / 16;
    const int task = blockIdx.x * 4 + wave;
    if (task >= BH * nqb) return;
    const int bh = task / nqb, q0 = (task % nqb) * 16;
    const ST* Qp = QKV + (size_t)bh * n * RS;
    const ST* Kp = Qp + DH;
    const ST* Vp = Qp + 2 * DH;

    const int q = q0 + c16;  // this lane's query
    Frag8<ST> qf[DH / 32];
#pragma unroll
    for (int s = 0; s < DH / 32; ++s)
        qf[s] = q < n ? frag8_load<ST>(Qp + (size_t)q * RS + s * 32 + 8 * g) : frag8_zero<ST>();

    float m_run = -__builtin_inff(), l_run = 0.f;
    f32x4 o[DH / 16];
#pragma unroll
    for (int db = 0; db < DH / 16; ++db) o[db] = zero4();

    const int kv_end = causal ? min(n, q0 + 16) : n;
    for (int j0 = 0; j0 < kv_end; j0 += 16) {
        f32x4 s = zero4();
        const int kr = j0 + c16;
#pragma unroll
        for (int st = 0; st < DH / 32; ++st) {
            const Frag8<ST> kf = kr < n ? frag8_load<ST>(Kp + (size_t)kr * RS + st * 32 + 8 * g) : frag8_zero<ST>();
            mma8(s, kf, qf[st]);
        }
        float sc[4], mloc = -__builtin_inff();
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int j = j0 + 4 * g + i;
            const bool ok = j < n && (!causal || j <= q);
            sc[i] = ok ? s[i] * scale : -__builtin_inff();
            mloc = fmaxf(mloc, sc[i]);
        }
        mloc = fmaxf(mloc, __shfl_xor(mloc, 16, 64));
        mloc = fmaxf(mloc, __shfl_xor(mloc, 32, 64));
        const float m_new = fmaxf(m_run, mloc);
        // Every query row has at least one allowed key (j = 0), so m_new is finite.
        const float alpha = expf(m_run - m_new);
        float p[4], lsum = 0.f;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            p[i] = expf(sc[i] - m_new);
            lsum += p[i];
        }
        lsum += __shfl_xor(lsum, 16, 64);
        lsum += __shfl_xor(lsum, 32, 64);
        l_run = l_run * alpha + lsum;
        m_run = m_new;
        const Frag4<ST> pf = frag4_from<ST>(p);
#pragma unroll
        for (int db = 0; db < DH / 16; ++db) {
            o[db] *= alpha;
            float vv[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int j = j0 + 4 * g + i;
                vv[i] = j < n ? ld1<ST>(Vp + (size_t)j * RS + db * 16 + c16) : 0.f;
            }
            const Frag4<ST> vf = frag4_from<ST>(vv);
            mma4(o[db], vf, pf);
        }
        mfma_drain();  // the loop may exit right here
    }
    if (q < n) {
        const float inv = (rw ? rw[(size_t)bh * n + q] : 1.f) / l_run;
        ST* Ap = A + ((size_t)bh * n + q) * DH;
#pragma unroll
        for (int db = 0; db < DH / 16; ++db)
#pragma unroll
            for (int i = 0; i < 4; ++i) st1<ST>(Ap + db * 16 + 4 * g + i, o[db][i] * inv);
        if (g == 0) lse[(size_t)bh * n + q] = m_run + logf(l_run);
    }
}

// Tiled variant for n > 32 (and every local-window head): a workgroup owns
// 16 NWV query rows of one (b,h), 16 per wave (128 rows for bf16 with
// 64-wide heads, else 64), and walks the keys in tiles of 64 staged in LDS
// once for all its waves: K row-major (A operand of S^T = K Q^T) and V
// (A operand of O^T += V^T P^T, K = 32 keys per MFMA, P^T straight from the
// S^T registers; bf16 keeps V row-major and reads it transposed).  Online
// softmax in log2 units.  The next tile's global loads are in flight while
// the current one is processed.  Causal blocks are launched heaviest first.
template <typename ST, int DH, bool WIN, int NWV>
__global__ __launch_bounds__(64 * NWV) void attn_fwd_tiled_kernel(const ST* __restrict__ QKV, int BH, int n, int causal,
                                                             int lb, float scale, const float* __restrict__ rw,
                                                             ST* __restrict__ A, float* __restrict__ lse) {
    constexpr int NT = 64 * NWV, QB = 16 * NWV, KB = 64, RS = 3 * DH;
    constexpr int PAD = 16 / (int)sizeof(ST);
    constexpr int LDR = DH + PAD;   // row-major K rows (and the output staging)
    constexpr int LDT = KB + 4;     // transposed V rows (keys), quad reads stay aligned
    constexpr int VPR = DH / 8;     // Vec8 per row
    constexpr int PER = KB * VPR / NT;
    static_assert(PER >= 1 && KB * VPR % NT == 0, "tile shape");
    __shared__ __attribute__((aligned(16))) ST Ks[(KB > QB ? KB : QB) * LDR];  // K tile, then the output rows
    __shared__ __attribute__((aligned(16))) ST Vt[DH * LDT];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, c16 = lane & 15;
    const int nqb = (n + QB - 1) / QB;
    const int bh = blockIdx.x / nqb;
    const int qb = causal ? nqb - 1 - blockIdx.x % nqb : blockIdx.x % nqb;
    const int q0 = qb * QB, wq0 = q0 + 16 * wave;
    const ST* Qp = QKV + (size_t)bh * n * RS;
    const ST* Kp = Qp + DH;
    const ST* Vp = Qp + 2 * DH;

    const int q = wq0 + c16;  // this lane's query (MFMA column)
    Frag8<ST> qf[DH / 32];
#pragma unroll
    for (int st = 0; st < DH / 32; ++st) qf[st] = frag8_load<ST>(Qp + (size_t)min(q, n - 1) * RS + st * 32 + 8 * g);

    float m_run = -__builtin_inff(), l_run = 0.f;  // running max in log2 units
    const float c2 = scale * 1.44269504088896341f;
    f32x4 o[DH / 16];
#pragma unroll
    for (int db = 0; db < DH / 16; ++db) o[db] = zero4();

    // causal with a local window (lb = window - 1 keys back): the block's keys
    // start at q0 - lb
    const int kv_end = causal ? min(n, q0 + QB) : n;
    const int ntiles = (kv_end + KB - 1) / KB, t0 = WIN && causal ? max(0, q0 - lb) / KB : 0;
    Vec8<ST> kreg[PER], vreg[PER];
    // rows past n are clamped to row n-1 (finite values whose scores are masked)
    auto load_tile = [&](int j0) {
#pragma unroll
        for (int p = 0; p < PER; ++p) {
            const int v = tid + NT * p, key = v / VPR, dc = (v % VPR) * 8;
            const size_t row = (size_t)min(j0 + key, n - 1);
            kreg[p] = vec8_load<ST>(Kp + row * RS + dc);
            vreg[p] = vec8_load<ST>(Vp + row * RS + dc);
        }
    };
    // bf16: V rows stay row-major (16-byte units permuted per key row by
    // vt_swz) and are read transposed (ds_read_b64_tr_b16), as in attn_lds.h
    unsigned char* const Vs = reinterpret_cast<unsigned char*>(Vt);
    static_assert(sizeof(ST) != 2 || DH * LDT * 2 >= KB * DH * 2, "V tile fits");
    auto store_tile = [&]() {
#pragma unroll
        for (int p = 0; p < PER; ++p) {
            const int v = tid + NT * p, key = v / VPR, dc = (v % VPR) * 8;
            vec8_store<ST>(Ks + key * LDR + dc, kreg[p]);
            if constexpr (sizeof(ST) == 2) {
                *reinterpret_cast<uint4*>(Vs + (key * VPR + ((dc >> 3) ^ vt_swz<VPR>(key))) * 16) = vreg[p].v;
            } else {
#pragma unroll
                for (int j = 0; j < 8; ++j) Vt[(dc + j) * LDT + key] = vec8_elem<ST>(vreg[p], j);
            }
        }
    };

    load_tile(t0 * KB);
    for (int t = t0; t < ntiles; ++t) {
        const int j0 = t * KB;
        __syncthreads();  // every wave is done with the previous tile
        store_tile();
        __syncthreads();
        load_tile(min(t + 1, ntiles - 1) * KB);  // the last tile is simply loaded again

        // S^T for the 4 sub-blocks of 16 keys: lane = query c16, rows = keys 4g + i
        f32x4 s[4];
#pragma unroll
        for (int sb = 0; sb < 4; ++sb) {
            s[sb] = zero4();
#pragma unroll
            for (int st = 0; st < DH / 32; ++st)
                mma8(s[sb], frag8_load<ST>(Ks + (sb * 16 + c16) * LDR + st * 32 + 8 * g), qf[st]);
        }
        float mloc = -__builtin_inff();
#pragma unroll
        for (int sb = 0; sb < 4; ++sb)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int key = j0 + sb * 16 + 4 * g + i;
                const bool ok = key < n && (!causal || (key <= q && (!WIN || q - key <= lb)));
                // scores in log2 units: s scale log2(e), so that p = 2^(s - m)
                s[sb][i] = ok ? s[sb][i] * c2 : -__builtin_inff();
                mloc = fmaxf(mloc, s[sb][i]);
            }
        mloc = fmaxf(mloc, __shfl_xor(mloc, 16, 64));
        mloc = fmaxf(mloc, __shfl_xor(mloc, 32, 64));
        // With a window a query may have no allowed key in this tile yet
        // (m_new = -inf): it then adds nothing.  Its own key comes later.
        const float m_new = fmaxf(m_run, mloc);
        const float m_use = WIN && m_new == -__builtin_inff() ? 0.f : m_new;
        const float alpha = __builtin_amdgcn_exp2f(m_run - m_use);
        float p[4][4], lsum = 0.f;
#pragma unroll
        for (int sb = 0; sb < 4; ++sb)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                p[sb][i] = __builtin_amdgcn_exp2f(s[sb][i] - m_use);
                lsum += p[sb][i];
            }
        lsum += __shfl_xor(lsum, 16, 64);
        lsum += __shfl_xor(lsum, 32, 64);
        l_run = l_run * alpha + lsum;
        m_run = m_new;
#pragma unroll
        for (int db = 0; db < DH / 16; ++db) o[db] *= alpha;
        // O^T += V^T P^T, 32 keys per MFMA: lane slots 0..3 = keys 4g+i of
        // sub-block 2u, slots 4..7 = the same of sub-block 2u+1
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            const float pv[8] = {p[2 * u][0], p[2 * u][1], p[2 * u][2], p[2 * u][3],
                                 p[2 * u + 1][0], p[2 * u + 1][1], p[2 * u + 1][2], p[2 * u + 1][3]};
            const Frag8<ST> pf = frag8_from<ST>(pv);
            if constexpr (sizeof(ST) == 2) {
                // lane reads d columns 16 db + 4 (c16 % 4) .. + 3 at keys k0 and k0 + 16
                u32x4 vt[DH / 16];
                const int k0 = 32 * u + 4 * g + (c16 >> 2), k1 = k0 + 16;
#pragma unroll
                for (int db = 0; db < DH / 16; ++db) {
                    const int mcol = 16 * db + 4 * (c16 & 3), un = mcol >> 3, half = (mcol >> 2) & 1;
                    const u32x2 lo = lds_read_tr16(Vs + (k0 * VPR + (un ^ vt_swz<VPR>(k0))) * 16 + 8 * half);
                    const u32x2 hi = lds_read_tr16(Vs + (k1 * VPR + (un ^ vt_swz<VPR>(k1))) * 16 + 8 * half);
                    vt[db] = u32x4{lo.x, lo.y, hi.x, hi.y};
                }
                lds_wait();
#pragma unroll
                for (int db = 0; db < DH / 16; ++db) {
                    lds_ready(vt[db]);
                    Frag8<ST> vf;
                    vf.v = __builtin_bit_cast(bf16x8, vt[db]);
                    mma8(o[db], vf, pf);
                }
            } else {
#pragma unroll
                for (int db = 0; db < DH / 16; ++db) {
                    const ST* vrow = Vt + (db * 16 + c16) * LDT + 32 * u + 4 * g;
                    mma8(o[db], frag8_from_quads<ST>(quad_load<ST>(vrow), quad_load<ST>(vrow + 16)), pf);
                }
            }
        }
        mfma_drain();  // the loop may exit right here
    }

    // O^T (lane: query c16, d rows db*16 + 4g + i) through LDS to 16-byte row stores
    __syncthreads();
    const float inv = (rw && q < n ? rw[(size_t)bh * n + q] : 1.f) / l_run;
    ST* Os = Ks + wave * 16 * LDR;
#pragma unroll
    for (int db = 0; db < DH / 16; ++db)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float x = o[db][i] * inv;
            if constexpr (sizeof(ST) == 2) Os[c16 * LDR + db * 16 + 4 * g + i] = f32_to_bf16(x);
            else Os[c16 * LDR + db * 16 + 4 * g + i] = x;
        }
    if (g == 0 && q < n) lse[(size_t)bh * n + q] = m_run * 0.69314718055994531f + logf(l_run);  // ln 2
    __syncthreads();
#pragma unroll
    for (int e = lane; e < 16 * VPR; e += 64) {
        const int r = e / VPR, dc = (e % VPR) * 8;
        if (wq0 + r < n)
            vec8_store<ST>(A + ((size_t)bh * n + wq0 + r) * DH + dc, vec8_load<ST>(Os + r * LDR + dc));
    }
}

// bf16, n <= 128: one workgroup of 8 waves per (b, h), one block of 16
// queries per wave (attn_lds.h).  K and V of all n keys go into LDS once, by
// direct global->LDS loads (K rows with XOR-permuted 16-byte units for
// ds_read_b128, V rows as in memory, units permuted per key row, for
// transposed reads); each wave's Q rows are loaded meanwhile.
template <int DH>
__global__ __launch_bounds__(512) void attn_fwd_lds_kernel(const uint16_t* __restrict__ QKV, int BH, int n, int causal,
                                                           float scale, const float* __restrict__ rw,
                                                           uint16_t* __restrict__ A, float* __restrict__ lse) {
    using ST = uint16_t;
    constexpr int RS = 3 * DH, NMAX = kAttnLdsMaxN, U = DH / 8;  // 16-byte units per row
    constexpr int TILE = NMAX * DH * 2;                          // bytes of one K or V tile
    constexpr int NW = NMAX / 16;                                // waves, one query block each
    constexpr int PER = NMAX * U / (64 * NW);                    // DMA instructions per wave per tile
    static_assert(PER >= 1 && NMAX * U % (64 * NW) == 0, "tile shape");
    __shared__ __attribute__((aligned(16))) unsigned char smem[2 * TILE];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, c16 = lane & 15;
    const int bh = xcd_logical_id(blockIdx.x, gridDim.x);
    const ST* Qp = QKV + (size_t)bh * n * RS;
    const ST* Kp = Qp + DH;
    const ST* Vp = Qp + 2 * DH;

    // K and V rows (clamped to n - 1; those keys are masked) into LDS.
    {
        const uint32_t base = __builtin_amdgcn_readfirstlane(lds_addr(smem)) + 1024 * __builtin_amdgcn_readfirstlane(wave);
#pragma unroll
        for (int j = 0; j < PER; ++j) {
            const int p = 64 * (wave + NW * j) + lane, key = p / U, pos = p % U;
            const size_t row = (size_t)min(key, n - 1) * RS;
            lds_load16(Kp + row + 8 * (pos ^ kswz(key, U)), base + 1024 * NW * j);
            lds_load16(Vp + row + 8 * (pos ^ vt_swz<U>(key)), base + TILE + 1024 * NW * j);
        }
    }
    // causal work of query block b is b + 1; waves w and w + 4 share a SIMD,
    // so with 8 blocks they take blocks s and 7 - s
    const int nqb = (n + 15) / 16, qb = nqb == 8 && causal && wave >= 4 ? 11 - wave : wave, q = 16 * qb + c16;
    Frag8<ST> qf[DH / 32];
#pragma unroll
    for (int st = 0; st < DH / 32; ++st) qf[st] = frag8_load<ST>(Qp + (size_t)min(q, n - 1) * RS + st * 32 + 8 * g);
    wait_vmcnt<0>();
    __syncthreads();
    if (qb >= nqb) return;
    attn_lds_block<DH>(smem, smem + TILE, 0, qf, n, causal, scale, qb, rw ? rw + (size_t)bh * n : nullptr,
                       A + (size_t)bh * n * DH, lse + (size_t)bh * n);
}

// ---------------------------------------------------------------------------
// bf16 with 64-wide heads, n > 128 or a local window: flash-style attention
// with 32 queries per wave -- two 16-query MFMA column blocks that share every
// K and V fragment read from LDS, so each LDS byte feeds twice the MFMA work
// of a 16-query wave -- and 4 waves, 128 queries, per workgroup.  Keys go in
// tiles of 64 through a 4-stage LDS ring filled by direct global->LDS loads
// (K rows with XOR-permuted 16-byte units for ds_read_b128, V rows with the
// vt_swz permutation for transposed reads), 3 tiles in flight.  S^T = K Q^T
// (lane = query), online softmax in log2 units, O^T += V^T P^T 32 keys per
// MFMA from the P^T registers.
//
// A (b, h) has nqb blocks of 128 queries; block qb covers key tiles
// [lo, lo + nt) (causal: up to its last query; local window: from its first
// query's window start).  Blocks are taken heaviest first, and a block of more
// than `tps` tiles is cut into splits of tps tiles: each split writes an fp32
// partial (unnormalised O, running max m in log2 units, sum l) and
// attn_fa_merge_kernel combines the splits of a block in split order, so the
// result is reproducible.  Unsplit blocks write A and lse directly.
// ---------------------------------------------------------------------------
constexpr int kFaQB = 128, kFaKB = 64, kFaStages = 4;
constexpr int kFaPart = kFaQB * 64 + 2 * kFaQB;  // floats per partial: O [128][64], m [128], l [128]

struct FaGeom {
    int n, causal, win, lb, nqb, tps, wph;  // wph: workgroups per (b, h)
};

__host__ __device__ inline void fa_range(const FaGeom& G, int qb, int& lo, int& nt) {
    const int q0 = qb * kFaQB;
    const int hi = G.causal ? min(G.n, q0 + kFaQB) : G.n;
    lo = G.win ? (max(0, q0 - G.lb) / kFaKB) * kFaKB : 0;
    nt = (hi - lo + kFaKB - 1) / kFaKB;
}
__host__ __device__ inline int fa_nsplit(const FaGeom& G, int qb) {
    int lo, nt;
    fa_range(G, qb, lo, nt);
    return (nt + G.tps - 1) / G.tps;
}
// query block at position p of the launch order (causal: heaviest first)
__host__ __device__ inline int fa_qb_at(const FaGeom& G, int p) { return G.causal ? G.nqb - 1 - p : p; }

template <bool WIN>
__global__ __launch_bounds__(256) void attn_fa_fwd_kernel(const uint16_t* __restrict__ QKV, FaGeom G, float scale,
                                                          const float* __restrict__ rw, uint16_t* __restrict__ A,
                                                          float* __restrict__ lse, float* __restrict__ part) {
    using ST = uint16_t;
    constexpr int DH = 64, RS = 3 * DH, U = DH / 8, KB = kFaKB, QB = kFaQB, STG = kFaStages;
    constexpr int TILE = KB * DH * 2, STAGE = 2 * TILE;  // K then V
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, c16 = lane & 15;
    const int logical = xcd_logical_id(blockIdx.x, gridDim.x);  // the blocks of a (b, h) share an XCD
    const int bh = logical / G.wph, j = logical % G.wph;
    // (block, split) of this workgroup
    int qb = 0, sp = 0, first = 0;
    for (int p = 0, acc = 0; p < G.nqb; ++p) {
        const int q = fa_qb_at(G, p), ns = fa_nsplit(G, q);
        if (j < acc + ns) {
            qb = q;
            sp = j - acc;
            first = acc;
            break;
        }
        acc += ns;
    }
    int lo, nt;
    fa_range(G, qb, lo, nt);
    const int nsplit = (nt + G.tps - 1) / G.tps;
    const int tbeg = sp * G.tps, tend = min(nt, tbeg + G.tps), ntile = tend - tbeg;
    const int n = G.n, q0 = qb * QB, wq0 = q0 + 32 * wave;
    const ST* Qp = QKV + (size_t)bh * n * RS;
    const ST* Kp = Qp + DH;
    const ST* Vp = Qp + 2 * DH;

    // query fragments (B operand of S^T = K Q^T): query wq0 + 16 qs + c16,
    // d_head 32 st + 8 g .. + 7 (rows past n clamped; never written)
    Frag8<ST> qf[2][2];
#pragma unroll
    for (int qs = 0; qs < 2; ++qs)
#pragma unroll
        for (int st = 0; st < 2; ++st)
            qf[qs][st] = frag8_load<ST>(Qp + (size_t)min(wq0 + 16 * qs + c16, n - 1) * RS + 32 * st + 8 * g);
    // Take the query rows now: a first use inside the pipeline would make the
    // compiler wait for every load in flight there, the next tiles' included.
#pragma unroll
    for (int qs = 0; qs < 2; ++qs)
#pragma unroll
        for (int st = 0; st < 2; ++st) asm volatile("" : "+v"(qf[qs][st].v));

    // DMA slots: 16-byte unit p = 64 (wave + 4 jj) + lane of a tile is row
    // p / 8, stored unit p % 8, which holds global unit (p % 8) ^ perm(row)
    const uint32_t lbase = __builtin_amdgcn_readfirstlane(lds_addr(smem)) +
                           1024 * (uint32_t)__builtin_amdgcn_readfirstlane(wave);
    int drow[2], kcol[2], vcol[2];
#pragma unroll
    for (int jj = 0; jj < 2; ++jj) {
        const int p = 64 * (wave + 4 * jj) + lane, r = p >> 3, u = p & 7;
        drow[jj] = r;
        kcol[jj] = 8 * (u ^ kswz(r, U));
        vcol[jj] = 8 * (u ^ vt_swz<U>(r));
    }
    // tile t of this split (clamped: tiles past the end reload the last one
    // into a buffer nobody reads); rows past n are clamped to n - 1 (masked)
    auto issue = [&](int t, int buf) {
        const int j0 = lo + KB * (tbeg + min(t, ntile - 1));
        const uint32_t b = lbase + buf * STAGE;
#pragma unroll
        for (int jj = 0; jj < 2; ++jj) {
            const size_t row = (size_t)min(j0 + drow[jj], n - 1) * RS;
            lds_load16(Kp + row + kcol[jj], b + 4096 * jj);
            lds_load16(Vp + row + vcol[jj], b + TILE + 4096 * jj);
        }
    };

    const float c2 = scale * 1.44269504088896341f;  // scores in log2 units
    float m_run[2] = {-__builtin_inff(), -__builtin_inff()}, l_run[2] = {0.f, 0.f};
    f32x4 o[2][DH / 16];
#pragma unroll
    for (int qs = 0; qs < 2; ++qs)
#pragma unroll
        for (int db = 0; db < DH / 16; ++db) o[qs][db] = zero4();

#pragma unroll
    for (int s0 = 0; s0 < STG - 1; ++s0) issue(s0, s0);
    // LDS byte offsets (within a V tile) of this lane's transposed V reads:
    // keys k0 = 32 u + 4 g + c16 / 4 and k0 + 16, columns 16 db + 4 (c16 % 4)
    int voff[2][DH / 16][2];
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int db = 0; db < DH / 16; ++db)
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const int kk = 32 * u + 4 * g + (c16 >> 2) + 16 * h;
                const int mcol = 16 * db + 4 * (c16 & 3), un = mcol >> 3, half = (mcol >> 2) & 1;
                voff[u][db][h] = (kk * U + (un ^ vt_swz<U>(kk))) * 16 + 8 * half;
            }
    // The loop is unrolled by STG so that every ring buffer has a constant
    // LDS offset (immediate offsets in the LDS reads, no address arithmetic).
    auto tile_step = [&](int it, auto bufc) {
        constexpr int BUF = decltype(bufc)::value;
        wait_vmcnt<(STG - 2) * 4>();  // tile it is in LDS (4 loads per tile and wave)
        __syncthreads();              // for every wave; the buffer of tile it - 1 is free
        issue(it + STG - 1, (BUF + STG - 1) % STG);
        const unsigned char* Kb = smem + BUF * STAGE;
        const unsigned char* Vb = Kb + TILE;
        const int j0 = lo + KB * (tbeg + it);

        // Every LDS read of the tile first (the V^T fragments are needed only
        // after the softmax, so their latency hides behind it).
        Frag8<ST> kf[4][2];
#pragma unroll
        for (int sb = 0; sb < 4; ++sb) {
            const int row = 16 * sb + c16;
#pragma unroll
            for (int st = 0; st < 2; ++st)
                kf[sb][st].v = __builtin_bit_cast(
                    bf16x8, *reinterpret_cast<const uint4*>(Kb + (row * U + ((4 * st + g) ^ kswz(row, U))) * 16));
        }
        u32x4 vt[2][DH / 16];
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
            for (int db = 0; db < DH / 16; ++db) {
                const u32x2 a = lds_read_tr16_at<BUF * STAGE + TILE>(smem + voff[u][db][0]);
                const u32x2 b = lds_read_tr16_at<BUF * STAGE + TILE>(smem + voff[u][db][1]);
                vt[u][db] = u32x4{a.x, a.y, b.x, b.y};
            }
        // S^T for 4 blocks of 16 keys: lane = query c16, rows = keys 16 sb + 4 g
        // + i; the two d_head halves in separate passes, so that no MFMA waits
        // for the one just before it
        f32x4 s[2][4];
#pragma unroll
        for (int sb = 0; sb < 4; ++sb)
#pragma unroll
            for (int qs = 0; qs < 2; ++qs) {
                s[qs][sb] = zero4();
                mma8(s[qs][sb], kf[sb][0], qf[qs][0]);
            }
#pragma unroll
        for (int sb = 0; sb < 4; ++sb)
#pragma unroll
            for (int qs = 0; qs < 2; ++qs) mma8(s[qs][sb], kf[sb][1], qf[qs][1]);
        // a tile needs the per-element mask where it reaches past a query of
        // this wave (causal), past n, or before a query's window
        const bool need = (G.causal && j0 + KB - 1 > wq0) || j0 + KB > n || (WIN && wq0 + 31 - j0 > G.lb);
        if (need) {  // one wave-uniform branch; selects without branches inside
#pragma unroll
            for (int qs = 0; qs < 2; ++qs) {
                const int q = wq0 + 16 * qs + c16;
#pragma unroll
                for (int sb = 0; sb < 4; ++sb)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int key = j0 + 16 * sb + 4 * g + i;
                        bool ok = key < n;
                        if (G.causal) ok &= key <= q;
                        if (WIN) ok &= q - key <= G.lb;
                        s[qs][sb][i] = ok ? s[qs][sb][i] : -__builtin_inff();
                    }
            }
        }
        float p[2][4][4];
#pragma unroll
        for (int qs = 0; qs < 2; ++qs) {
            float mloc = -__builtin_inff();  // over the raw scores (the scale is positive)
#pragma unroll
            for (int sb = 0; sb < 4; ++sb)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    p[qs][sb][i] = s[qs][sb][i];
                    mloc = fmaxf(mloc, s[qs][sb][i]);
                }
            mloc = rows4_max(mloc) * c2;
            // Lazy rescaling: the reference max m moves only when the tile's
            // max exceeds it by more than 8 (log2 units), so p <= 2^8 and the
            // O and l rescaling runs only when some query of the wave moved.
            // A query with no allowed key yet keeps m = -inf and adds nothing.
            const float m_new = mloc > m_run[qs] + 8.f ? mloc : m_run[qs];
            const float m_use = m_new == -__builtin_inff() ? 0.f : m_new;
            if (__builtin_amdgcn_ballot_w64(m_new != m_run[qs])) {
                const float alpha = __builtin_amdgcn_exp2f(m_run[qs] - m_use);
                l_run[qs] *= alpha;
#pragma unroll
                for (int db = 0; db < DH / 16; ++db) o[qs][db] *= alpha;
                m_run[qs] = m_new;
            }
            float lsum = 0.f;
#pragma unroll
            for (int sb = 0; sb < 4; ++sb)
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    p[qs][sb][i] = __builtin_amdgcn_exp2f(__builtin_fmaf(p[qs][sb][i], c2, -m_use));
                    lsum += p[qs][sb][i];
                }
            l_run[qs] += rows4_sum(lsum);
        }
        // O^T += V^T P^T, 32 keys per MFMA: lane slots 0..3 = keys 4g+i of
        // block 2u, slots 4..7 = the same of block 2u+1 (V^T read in that order)
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            Frag8<ST> pf[2];
#pragma unroll
            for (int qs = 0; qs < 2; ++qs) {
                const float pv[8] = {p[qs][2 * u][0],     p[qs][2 * u][1],     p[qs][2 * u][2],     p[qs][2 * u][3],
                                     p[qs][2 * u + 1][0], p[qs][2 * u + 1][1], p[qs][2 * u + 1][2], p[qs][2 * u + 1][3]};
                pf[qs] = frag8_from<ST>(pv);
            }
            if (u == 0) lds_wait();  // the V^T fragments (issued with the K reads)
#pragma unroll
            for (int db = 0; db < DH / 16; ++db) {
                lds_ready(vt[u][db]);
                Frag8<ST> vf;
                vf.v = __builtin_bit_cast(bf16x8, vt[u][db]);
#pragma unroll
                for (int qs = 0; qs < 2; ++qs) mma8(o[qs][db], vf, pf[qs]);
            }
        }
    };
    for (int it0 = 0;; it0 += STG) {
        bool last = false;
        static_for<0, STG>([&](auto u) {
            if (last) return;
            const int it = it0 + decltype(u)::value;
            tile_step(it, u);
            last = it + 1 >= ntile;
        });
        if (last) break;
    }
    mfma_drain();      // the MFMA results are read below
    wait_vmcnt<0>();   // the trailing (clamped) loads still write into the ring
    __syncthreads();

    if (nsplit > 1) {
        // fp32 partial of this split: O^T rows straight from the accumulators
        float* pp = part + ((size_t)bh * G.wph + first + sp) * kFaPart;
#pragma unroll
        for (int qs = 0; qs < 2; ++qs) {
            const int ql = 32 * wave + 16 * qs + c16;
#pragma unroll
            for (int db = 0; db < DH / 16; ++db)
                *reinterpret_cast<float4*>(pp + ql * DH + 16 * db + 4 * g) =
                    make_float4(o[qs][db][0], o[qs][db][1], o[qs][db][2], o[qs][db][3]);
            if (g == 0) {
                pp[QB * DH + ql] = m_run[qs];
                pp[QB * DH + QB + ql] = l_run[qs];
            }
        }
        return;
    }
    // whole block: A = r O / l through LDS to 16-byte row stores, lse = m ln 2 + log l
    constexpr int LDO = DH + 8;
    ST* Os = reinterpret_cast<ST*>(smem) + wave * 32 * LDO;
#pragma unroll
    for (int qs = 0; qs < 2; ++qs) {
        const int q = wq0 + 16 * qs + c16;
        const float inv = (rw && q < n ? rw[(size_t)bh * n + q] : 1.f) / l_run[qs];
#pragma unroll
        for (int db = 0; db < DH / 16; ++db) {
            const uint2 v = make_uint2(pack_bf16x2(o[qs][db][0] * inv, o[qs][db][1] * inv),
                                       pack_bf16x2(o[qs][db][2] * inv, o[qs][db][3] * inv));
            *reinterpret_cast<uint2*>(Os + (16 * qs + c16) * LDO + 16 * db + 4 * g) = v;
        }
        if (g == 0 && q < n) lse[(size_t)bh * n + q] = m_run[qs] * 0.69314718055994531f + logf(l_run[qs]);
    }
    __syncthreads();
#pragma unroll
    for (int e = lane; e < 32 * U; e += 64) {
        const int r = e / U, dc = (e % U) * 8;
        if (wq0 + r < n)
            *reinterpret_cast<uint4*>(A + ((size_t)bh * n + wq0 + r) * DH + dc) =
                *reinterpret_cast<const uint4*>(Os + r * LDO + dc);
    }
}

// The splits of every split block, in split order: M = max m_s,
// L = sum l_s 2^(m_s - M), A = r sum O_s 2^(m_s - M) / L, lse = M ln 2 + log L.
// One workgroup per (b, h, block, quarter of the columns), one thread per query.
__global__ __launch_bounds__(128) void attn_fa_merge_kernel(FaGeom G, const float* __restrict__ part,
                                                            const float* __restrict__ rw, uint16_t* __restrict__ A,
                                                            float* __restrict__ lse) {
    constexpr int DH = 64, QB = kFaQB, NC = DH / 4;
    const int cq = blockIdx.x & 3, bp = blockIdx.x >> 2;
    const int bh = bp / G.nqb, pos = bp % G.nqb;
    int first = 0;
    for (int p = 0; p < pos; ++p) first += fa_nsplit(G, fa_qb_at(G, p));
    const int qb = fa_qb_at(G, pos), ns = fa_nsplit(G, qb);
    if (ns <= 1) return;
    const int ql = threadIdx.x, q = qb * QB + ql;
    if (q >= G.n) return;
    const float* p0 = part + ((size_t)bh * G.wph + first) * kFaPart;
    float M = -__builtin_inff();
    for (int s = 0; s < ns; ++s) M = fmaxf(M, p0[(size_t)s * kFaPart + QB * DH + ql]);
    float L = 0.f, acc[NC];
#pragma unroll
    for (int c = 0; c < NC; ++c) acc[c] = 0.f;
#pragma unroll 4
    for (int s = 0; s < ns; ++s) {
        const float* ps = p0 + (size_t)s * kFaPart;
        const float ms = ps[QB * DH + ql], ls = ps[QB * DH + QB + ql];
        float4 v[NC / 4];
        const float4* src = reinterpret_cast<const float4*>(ps + ql * DH + NC * cq);
#pragma unroll
        for (int c = 0; c < NC / 4; ++c) v[c] = src[c];
        const float wgt = ms == -__builtin_inff() ? 0.f : __builtin_amdgcn_exp2f(ms - M);
        L += ls * wgt;
#pragma unroll
        for (int c = 0; c < NC / 4; ++c) {
            acc[4 * c] += v[c].x * wgt;
            acc[4 * c + 1] += v[c].y * wgt;
            acc[4 * c + 2] += v[c].z * wgt;
            acc[4 * c + 3] += v[c].w * wgt;
        }
    }
    const float inv = (rw ? rw[(size_t)bh * G.n + q] : 1.f) / L;
    uint4* dst = reinterpret_cast<uint4*>(A + ((size_t)bh * G.n + q) * DH + NC * cq);
#pragma unroll
    for (int c = 0; c < NC / 8; ++c)
        dst[c] = make_uint4(pack_bf16x2(acc[8 * c] * inv, acc[8 * c + 1] * inv),
                            pack_bf16x2(acc[8 * c + 2] * inv, acc[8 * c + 3] * inv),
                            pack_bf16x2(acc[8 * c + 4] * inv, acc[8 * c + 5] * inv),
                            pack_bf16x2(acc[8 * c + 6] * inv, acc[8 * c + 7] * inv));
    if (cq == 0) lse[(size_t)bh * G.n + q] = M * 0.69314718055994531f + logf(L);
}

// Geometry of the flash kernel for BH heads of n rows; when there are fewer
// query blocks than CUs, the split length is chosen so that about 512
// workgroups run.  Returns false when the kernel does not apply.
bool fa_geom(int dtype, int BH, int n, int dh, int causal, int window, FaGeom& G) {
    if (dtype != kBF16 || dh != 64 || !(n > kAttnLdsMaxN || window > 0)) return false;
    G.n = n;
    G.causal = causal;
    G.win = window > 0 && causal;
    G.lb = window > 0 ? window - 1 : n;
    G.nqb = (n + kFaQB - 1) / kFaQB;
    G.tps = 1 << 30;
    long long total = 0;
    int maxt = 0;
    for (int qb = 0; qb < G.nqb; ++qb) {
        int lo, nt;
        fa_range(G, qb, lo, nt);
        total += nt;
        maxt = nt > maxt ? nt : maxt;
    }
    // split only when the blocks alone leave CUs idle: the partials and the
    // merge cost more than the causal imbalance they remove otherwise
    // (measured on 32 heads of 1024 rows: 23.2 us unsplit, 31.2 us with
    // splits of 8 tiles including the merge)
    if ((long long)BH * G.nqb < 256) {
        const long long want = (total * BH + 511) / 512;
        G.tps = (int)(want > 8 ? want : 8);
        if (G.tps >= maxt) G.tps = 1 << 30;
    }
    G.wph = 0;
    for (int qb = 0; qb < G.nqb; ++qb) G.wph += fa_nsplit(G, qb);
    return true;
}

template <typename ST>
int launch_attn_fwd_t(const ST* QKV, const float* r, int BH, int n, int dh, int causal, int window, ST* A,
                      float* lse, float* part, int dense, const Marker& mk, hipStream_t stream) {
    const float scale = 1.0f / sqrtf((float)dh);
    const int lb = window > 0 ? window - 1 : n;  // keys a query may look back
    if constexpr (sizeof(ST) == 2) {
        FaGeom G;
        if (fa_geom(kBF16, BH, n, dh, causal, window, G)) {
            const size_t lds = (size_t)kFaStages * 2 * kFaKB * 64 * 2;
            auto kern = G.win ? attn_fa_fwd_kernel<true> : attn_fa_fwd_kernel<false>;
            if (allow_lds((const void*)kern, lds)) return -1;
            const bool split = G.wph > G.nqb;
            if (split && !part) return -1;
            hipLaunchKernelGGL(kern, dim3(BH * G.wph), dim3(256), lds, stream, (const uint16_t*)QKV, G, scale, r,
                               (uint16_t*)A, lse, part);
            if (hipGetLastError() != hipSuccess || mk(dense ? "attn_dense" : "attn")) return -1;
            if (split) {
                hipLaunchKernelGGL(attn_fa_merge_kernel, dim3(4 * BH * G.nqb), dim3(128), 0, stream, G, part, r,
                                   (uint16_t*)A, lse);
                if (hipGetLastError() != hipSuccess || mk(dense ? "attn_dense_merge" : "attn_merge")) return -1;
            }
            return 0;
        }
        if (n > 32 && n <= kAttnLdsMaxN && window == 0) {
            if (dh == 64)
                hipLaunchKernelGGL((attn_fwd_lds_kernel<64>), dim3(BH), dim3(512), 0, stream, QKV, BH, n, causal, scale,
                                   r, A, lse);
            else
                hipLaunchKernelGGL((attn_fwd_lds_kernel<32>), dim3(BH), dim3(512), 0, stream, QKV, BH, n, causal, scale,
                                   r, A, lse);
            return hipGetLastError() == hipSuccess ? 0 : -1;
        }
    }
    if (n > 32 || window > 0) {
        // bf16 with 64-wide heads: 128 queries (8 waves) per workgroup share each K/V tile
        constexpr int W64 = sizeof(ST) == 2 ? 8 : 4;
        auto kern = window > 0 ? (dh == 64 ? attn_fwd_tiled_kernel<ST, 64, true, W64>
                                           : attn_fwd_tiled_kernel<ST, 32, true, 4>)
                               : (dh == 64 ? attn_fwd_tiled_kernel<ST, 64, false, W64>
                                           : attn_fwd_tiled_kernel<ST, 32, false, 4>);
        const int qbw = 16 * (dh == 64 ? W64 : 4);
        const dim3 grid(BH * ((n + qbw - 1) / qbw)), block(4 * qbw);
        hipLaunchKernelGGL(kern, grid, block, 0, stream, QKV, BH, n, causal, lb, scale, r, A, lse);
        return hipGetLastError() == hipSuccess ? 0 : -1;
    }
    const int tasks = BH * ((n + 15) / 16);
    dim3 grid((tasks + 3) / 4), block(256);
    if (dh == 64)
        hipLaunchKernelGGL((attn_fwd_kernel<ST, 64>), grid, block, 0, stream, QKV, BH, n, causal, scale, r, A, lse);
    else
        hipLaunchKernelGGL((attn_fwd_kernel<ST, 32>), grid, block, 0, stream, QKV, BH, n, causal, scale, r, A, lse);
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

}  // namespace

int launch_attn_fwd(int dtype, const void* QKV, const float* r, int BH, int n, int dh, int causal, int window,
                    void* A, float* lse, float* part, int dense, const Marker& mk, hipStream_t stream) {
    FaGeom G;
    if (fa_geom(dtype, BH, n, dh, causal, window, G))  // marks its own launches
        return launch_attn_fwd_t<uint16_t>((const uint16_t*)QKV, r, BH, n, dh, causal, window, (uint16_t*)A, lse,
                                           part, dense, mk, stream);
    const int e = dtype == kBF16 ? launch_attn_fwd_t<uint16_t>((const uint16_t*)QKV, r, BH, n, dh, causal, window,
                                                               (uint16_t*)A, lse, part, dense, mk, stream)
                                 : launch_attn_fwd_t<float>((const float*)QKV, r, BH, n, dh, causal, window,
                                                            (float*)A, lse, part, dense, mk, stream);
    return e | mk(dense ? "attn_dense" : "attn");
}

size_t attn_fwd_part_bytes(int dtype, int BH, int n, int dh, int causal, int window) {
    FaGeom G;
    if (BH <= 0 || n <= 0 || !fa_geom(dtype, BH, n, dh, causal, window, G) || G.wph == G.nqb) return 0;
    return (size_t)BH * G.wph * kFaPart * sizeof(float);
}

}  // namespace mosa
