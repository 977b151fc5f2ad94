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

template <typename ST>
int launch_attn_fwd_t(const ST* QKV, const float* r, int BH, int n, int dh, int causal, int window, ST* A,
                      float* lse, hipStream_t stream) {
    const float scale = 1.0f / sqrtf((float)dh);
    const int lb = window > 0 ? window - 1 : n;  // keys a query may look back
    if constexpr (sizeof(ST) == 2) {
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
                    void* A, float* lse, hipStream_t stream) {
    if (dtype == kBF16)
        return launch_attn_fwd_t<uint16_t>((const uint16_t*)QKV, r, BH, n, dh, causal, window, (uint16_t*)A, lse,
                                           stream);
    return launch_attn_fwd_t<float>((const float*)QKV, r, BH, n, dh, causal, window, (float*)A, lse, stream);
}

}  // namespace mosa
