// Row-streaming MFMA kernel for bf16 products with a short contraction and a
// wide output (the per-head output projection and the per-head dX rows):
//
//   Y[m, n0 + c] = sum_{k < K} A[m, k] W[k, n0 + c],   c < NC = 128 NPAIR,
//
// for a run of 64-row tiles of A.  K is small (32 .. 192), so the workgroup
// keeps its whole NC-column block of W in registers (each of the four waves
// owns 32 NPAIR columns) and streams the A tiles through an LDS ring filled by
// direct global->LDS loads (the scheme of gemm2.h: one barrier per tile,
// STAGES - 1 tiles in flight).  The work is write-bound (M x NC outputs per
// K x NC weights), so results go from the accumulators straight to memory:
//
// The MFMA computes the transposed tile, D[i = column][j = row], so a lane
// holds four consecutive columns of one row; the columns of each pair of
// 16-column blocks are interleaved (MFMA row i of the first block is column
// 8 (i / 4) + i % 4, of the second 8 (i / 4) + 4 + i % 4) so that a lane
// holds 8 consecutive columns and writes them with one 16-byte store.  The
// stores are buffer stores whose addresses for rows past the end lie outside
// the buffer range and are dropped by the hardware: every wave issues the same
// number of memory instructions per tile, which keeps the constant wait counts
// of the pipeline exact.
//
// Policy P:
//   K, NPAIR, STAGES, W_KCONTIG, ROW_SCALAR, Args;
//   tile(args, logical, h, n0, s_beg, s_end): head, first column, 64-row tiles;
//   rows(args): M;  a_row(args, h, m) -> K contiguous elements (m < M);
//   W_KCONTIG:  w_kptr(args, h, n, k) -> W[k .. k + 7, n] contiguous;
//   otherwise:  w_mptr(args, h, k, n) -> W[k, n .. n + 7] contiguous;
//   ROW_SCALAR: z_ptr(args, h, m) -> one float per row, handed to store();
//   col_init(args, h, n, cv[8]): per-column values for columns n .. n + 7;
//   out_rsrc(args, h): buffer over the output (under 2^31 bytes);
//   out_row(args, h, m): byte offset of Y[m, 0];
//   finish(x[8], z, cv[8]): final values of 8 columns.
#pragma once

#include "gemm2.h"

namespace mosa {

// One wave's 256 bytes of LDS from 64 lanes x 4 bytes (lane l writes base + 4 l).
__device__ __forceinline__ void lds_load4(const void* g, uint32_t base) {
    asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dword %0, off" : : "v"(g), "s"(base) : "memory", "m0");
}

// wait_vmcnt<BASE + u * STEP>() for a u that is a constant after unrolling.
template <int BASE, int STEP, int I = 0>
__device__ __forceinline__ void wait_vmcnt_at(int u) {
    if constexpr (I < 8 && BASE + I * STEP <= 63) {
        if (u == I) {
            wait_vmcnt<BASE + I * STEP>();
            return;
        }
        wait_vmcnt_at<BASE, STEP, I + 1>(u);
    } else {
        wait_vmcnt<0>();
    }
}

template <class P>
struct RowGemmShape {
    static constexpr int K = P::K, STG = P::STAGES, NPAIR = P::NPAIR, NB = 2 * NPAIR, NC = 128 * NPAIR;
    static constexpr int SLAB = K % 64 == 0 ? 64 : 32;  // k columns per swizzled slab
    static constexpr int LPR = SLAB / 8;                // 16-byte units per slab row
    static constexpr int KS = K / 32;                   // MFMA k steps
    static constexpr int IA = 64 * K / 8 / 256;         // A loads per wave per tile
    static constexpr int IZ = P::ROW_SCALAR ? 1 : 0;    // row-scalar loads per wave per tile
    static constexpr int NS = 4 * NPAIR;                // stores per wave per tile
    static constexpr int A_BYTES = 64 * K * 2;
    static constexpr int STAGE_BYTES = A_BYTES + IZ * 1024;
    static constexpr int W_BYTES = P::W_KCONTIG ? 0 : K * NC * 2;
    // loads and stores issued after the loads of the tile about to be used
    static constexpr int WAIT = (STG - 2) * (IA + IZ + NS) + NS;
    static_assert(K % 32 == 0 && (64 * K / 8) % 256 == 0 && (K * NC / 8) % 256 == 0, "K");
    static_assert(STG >= 2 && WAIT <= 63, "vmcnt range");
    // LDS: the ring of STG tile buffers, then (m-contiguous W) the W block,
    // apart so that the first tiles' loads are in flight while W is staged
    static constexpr int W_OFF = STG * STAGE_BYTES;
    static constexpr size_t lds_bytes() { return (size_t)STG * STAGE_BYTES + W_BYTES; }
};

// One workgroup's run of row tiles, logical index `logical`.
template <class P>
__device__ __forceinline__ void rowgemm_body(const typename P::Args& args, int logical, unsigned char* smem) {
    using ST = uint16_t;
    using S = RowGemmShape<P>;
    constexpr int K = S::K, LPR = S::LPR, SLAB = S::SLAB, KS = S::KS, STG = S::STG, NB = S::NB, NC = S::NC;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, c16 = lane & 15;
    int h, n0, s_beg, s_end;
    P::tile(args, logical, h, n0, s_beg, s_end);
    const int nsteps = s_end - s_beg, M = P::rows(args);
    const int wcol = n0 + 32 * S::NPAIR * wave;            // this wave's columns
    const int icol = 8 * (c16 >> 2) + (c16 & 3);           // column of MFMA row c16 in a block pair

    // This lane's slot in each A load: row r of the tile, 16-byte unit.
    int arow[S::IA], acol[S::IA];
#pragma unroll
    for (int j = 0; j < S::IA; ++j) {
        const int p = 64 * (wave + 4 * j) + lane;
        const int slab = p / (64 * LPR), q = p % (64 * LPR), r = q / LPR, pos = q % LPR;
        arow[j] = r;
        acol[j] = slab * SLAB + 8 * (pos ^ kswz(r, LPR));
    }
    const uint32_t lds_base = __builtin_amdgcn_readfirstlane(lds_addr(smem));
    const int wave_s = __builtin_amdgcn_readfirstlane(wave);  // uniform copy for LDS bases

    // Loads of tile s (clamped to the last tile: past the end they refill a
    // buffer nobody reads) into stage buffer bidx.
    auto issue = [&](int s, int bidx) {
        const int m0 = (s_beg + min(s, nsteps - 1)) * 64;
        const uint32_t buf = lds_base + bidx * S::STAGE_BYTES + 1024 * wave_s;
#pragma unroll
        for (int j = 0; j < S::IA; ++j) lds_load16(P::a_row(args, h, min(m0 + arow[j], M - 1)) + acol[j], buf + 4096 * j);
        if constexpr (P::ROW_SCALAR)
            lds_load4(P::z_ptr(args, h, min(m0 + lane, M - 1)), lds_base + bidx * S::STAGE_BYTES + S::A_BYTES + 256 * wave_s);
    };
    // The first STG - 1 tiles are requested before the weights, so that the
    // two latencies overlap (the weights' own waits then also cover these
    // loads: vector memory operations complete in issue order).
    if (nsteps > 0) {
#pragma unroll
        for (int s = 0; s < STG - 1; ++s) issue(s, s);
    }
    // W fragments: wf[nb][ks] for 16-column block nb (pair nb / 2, half nb % 2)
    // and k = 32 ks + 8 g .. + 7, MFMA row c16.
    bf16x8 wf[NB][KS];
    if constexpr (P::W_KCONTIG) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
            for (int ks = 0; ks < KS; ++ks)
                wf[nb][ks] = __builtin_bit_cast(
                    bf16x8, *reinterpret_cast<const uint4*>(
                                P::w_kptr(args, h, wcol + 32 * (nb >> 1) + 4 * (nb & 1) + icol, 32 * ks + 8 * g)));
    } else {
        // W[0:K][n0:n0+NC] row-major in LDS (after the ring), then the fragments from there.
        ST* wl = reinterpret_cast<ST*>(smem + S::W_OFF);
        constexpr int UPR = NC / 8;  // 16-byte units per W row
#pragma unroll
        for (int i = 0; i < K * UPR / 256; ++i) {
            const int u = tid + 256 * i, k = u / UPR, c8 = (u % UPR) * 8;
            *reinterpret_cast<uint4*>(wl + k * NC + c8) = *reinterpret_cast<const uint4*>(P::w_mptr(args, h, k, n0 + c8));
        }
        __syncthreads();
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
            for (int ks = 0; ks < KS; ++ks) {
                const int col = 32 * S::NPAIR * wave + 32 * (nb >> 1) + 4 * (nb & 1) + icol;
                uint16_t e[8];
#pragma unroll
                for (int j = 0; j < 8; ++j) e[j] = wl[(32 * ks + 8 * g + j) * NC + col];
                const uint4 u = make_uint4(e[0] | ((uint32_t)e[1] << 16), e[2] | ((uint32_t)e[3] << 16),
                                           e[4] | ((uint32_t)e[5] << 16), e[6] | ((uint32_t)e[7] << 16));
                wf[nb][ks] = __builtin_bit_cast(bf16x8, u);
            }
        __syncthreads();
    }
    float cv[S::NPAIR][8];
#pragma unroll
    for (int p = 0; p < S::NPAIR; ++p) P::col_init(args, h, wcol + 32 * p + 8 * g, cv[p]);
    const __amdgpu_buffer_rsrc_t out = P::out_rsrc(args, h);
    // Take the weights now: a first use inside the pipeline would make the
    // compiler wait for every load in flight there.
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) asm volatile("" : "+v"(wf[nb][ks]));
#pragma unroll
    for (int p = 0; p < S::NPAIR; ++p)
#pragma unroll
        for (int j = 0; j < 8; ++j) asm volatile("" : "+v"(cv[p][j]));


    auto tile_step = [&](int s, int bidx) {
        const unsigned char* ta = smem + bidx * S::STAGE_BYTES;
        f32x4 acc[NB][4];
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
            for (int jb = 0; jb < 4; ++jb) acc[nb][jb] = zero4();
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            bf16x8 af[4];
#pragma unroll
            for (int jb = 0; jb < 4; ++jb) {
                const int row = 16 * jb + c16, slab = (32 * ks) / SLAB, u = ((32 * ks) % SLAB) / 8 + g;
                af[jb] = __builtin_bit_cast(
                    bf16x8, *reinterpret_cast<const uint4*>(ta + (slab * 64 * LPR + row * LPR + (u ^ kswz(row, LPR))) * 16));
            }
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
#pragma unroll
                for (int jb = 0; jb < 4; ++jb)
                    acc[nb][jb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[nb][ks], af[jb], acc[nb][jb], 0, 0, 0);
        }
        const int m0 = (s_beg + s) * 64;
        const float* zl = reinterpret_cast<const float*>(ta + S::A_BYTES + 256 * wave);
#pragma unroll
        for (int jb = 0; jb < 4; ++jb) {
            const int m = m0 + 16 * jb + c16;
            const float z = P::ROW_SCALAR ? zl[16 * jb + c16] : 0.f;
            // byte offset of the row; rows past the end get one past 2^31
            const int ro = P::out_row(args, h, min(m, M - 1));
            const int rbase = m < M ? ro : INT32_MIN;
#pragma unroll
            for (int p = 0; p < S::NPAIR; ++p) {
                float x[8];
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    x[r] = acc[2 * p][jb][r];
                    x[4 + r] = acc[2 * p + 1][jb][r];
                }
                P::finish(x, z, cv[p]);
                const uint4 v = make_uint4(pack_bf16x2(x[0], x[1]), pack_bf16x2(x[2], x[3]), pack_bf16x2(x[4], x[5]),
                                           pack_bf16x2(x[6], x[7]));
                __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), out,
                                                       rbase + 2 * (wcol + 32 * p + 8 * g), 0, 0);
            }
        }
    };

    // Pipeline as in gemm2.h, over row tiles.  The stores make the number of
    // memory instructions issued after the loads of tile s grow over the first
    // STAGES - 1 tiles: (STAGES - 2) (IA + IZ) + min(s, STAGES - 1) NS, the
    // steady-state value being S::WAIT; the first pass waits with the smaller
    // counts.  The only way out is through mfma_drain() (see gemm2.h).
    auto pass = [&](int s0, auto first) -> bool {
#pragma unroll
        for (int u = 0; u < STG; ++u) {
            const int s = s0 + u;
            if constexpr (decltype(first)::value) wait_vmcnt_at<(STG - 2) * (S::IA + S::IZ), S::NS>(u);
            else wait_vmcnt<S::WAIT>();
            __syncthreads();  // tile s is in LDS; the buffer of tile s - 1 is free
            issue(s + STG - 1, (u + STG - 1) % STG);
            __builtin_amdgcn_sched_barrier(0);
            tile_step(s, u);
            if (s + 1 == nsteps) {
                mfma_drain();
                return true;
            }
        }
        return false;
    };
    if (nsteps > 0) {
        if (!pass(0, std::true_type{}))
            for (int s0 = STG;; s0 += STG)
                if (pass(s0, std::false_type{})) break;
    }
    wait_vmcnt<0>();
}

template <class P>
__global__ __launch_bounds__(256) void rowgemm_kernel(const typename P::Args args) {
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
    rowgemm_body<P>(args, xcd_logical_id(blockIdx.x, gridDim.x), smem);
}

// Splits the row tiles of every (head, column block) over workgroups so that
// about `target` workgroups run; returns the tiles per workgroup.
inline int rowgemm_tiles_per_wg(int units, int tiles, int target) {
    int per = (int)(((long long)units * tiles + target - 1) / target);
    if (per < 1) per = 1;
    if (per > tiles) per = tiles;
    return per;
}

template <class P>
int launch_rowgemm(const typename P::Args& args, int nblocks, hipStream_t stream) {
    if (nblocks <= 0) return 0;
    constexpr size_t lds = RowGemmShape<P>::lds_bytes();
    auto kern = rowgemm_kernel<P>;
    if (allow_lds((const void*)kern, lds)) return -1;
    hipLaunchKernelGGL(kern, dim3(nblocks), dim3(256), lds, stream, args);
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

}  // namespace mosa
