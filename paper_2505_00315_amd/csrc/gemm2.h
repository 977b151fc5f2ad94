// Multi-stage MFMA GEMM engine for bf16 storage with direct global->LDS loads.
//
//   C[M x N] = sum_k A[M x K] B[K x N]   (fp32 accumulation), one problem per
//   "batch" index, tiles of MT x NT, four waves, K in chunks of KC.
//
// Operands are copied from global memory straight into LDS with 16-byte
// global_load_lds instructions (no register staging): one instruction of a
// wave fills 1 KB of LDS, lane l writing bytes 16 l .. 16 l + 15, and each
// lane chooses the global 16 bytes that belong at its slot.  STAGES chunk
// buffers are in flight; one barrier per chunk.
//
// A k-contiguous operand (rows along M or N, 8 consecutive k per 16 bytes) is
// stored row-major [rows][KC] with the 16-byte units of a row XOR-permuted
// (f(r) below) so that the ds_read_b128 of an MFMA fragment (16 rows, same
// k) hits distinct banks.  An m-contiguous operand (rows along K, e.g. a
// weight W[k][n]) is stored [KC][R] as in memory, units permuted by h(k), and
// its MFMA fragments are read with ds_read_b64_tr_b16, which transposes 4 x 4
// blocks of 16-bit elements across the lanes of a 16-lane group: source lane
// s supplies the address of row kbase + s/4, columns m0 + 4 (s % 4) .. +3, and
// lane i receives rows kbase .. kbase + 3 of column m0 + i.  Two such reads give
// the 8 consecutive k of an MFMA operand, in the same k order as the
// k-contiguous reads.
//
// Policy P (all addresses must be valid for any k in [0, K) and any row; rows
// past the problem are clamped by the policy and their results discarded):
//   MT, NT, KC, WM, WN, STAGES, EPI_LDS; A_KCONTIG, B_KCONTIG;
//   tile(args, logical, batch, m0, n0), k_size(args, batch) (a multiple of KC);
//   k-contiguous: a_row(args, batch, m) -> ARef, a_elem(args, batch, ARef, k)
//                 (likewise b_row / b_elem);
//   m-contiguous: a_maddr(args, batch, k, m8) / b_maddr(args, batch, k, n8) and
//                 a_kstride(args, batch) / b_kstride(args, batch), the element
//                 distance between consecutive k (addresses move linearly in k);
//   epilogue(args, batch, m0, n0, Cs, ldc, tid, extra) as in gemm.h.
//
// Optional (all off by default):
//   KGATHER: the rows along k are gathered (both operands m-contiguous).  The
//     workgroup first fills an LDS table with k_row(args, batch, k, K) -> int2
//     for every k of its range (K need not be a multiple of KC; the table
//     covers the padded range), and a lane's address for row k is
//     base + tab[k].{x|y} * stride with base and stride from
//     a_mlane(args, batch, m8, base, stride) (A_TAB picks x or y; likewise
//     b_mlane / B_TAB).  A negative table entry reads zeros.
//   A_INTERLEAVE: an m-contiguous A operand whose 16-row MFMA blocks are taken
//     in pairs with interleaved columns (block 2p row i is M index
//     32 p + 8 (i / 4) + i % 4, block 2p + 1 row i is 32 p + 8 (i / 4) + 4 + i % 4),
//     so that a lane's accumulators of a block pair are 8 consecutive M.
//   MIN_WAVES: waves per SIMD the register allocation must allow.
//   CHUNK_ADD (k-contiguous A and B): each MFMA from zero, then one add.
//   EPI_REGS (needs A_INTERLEAVE): no C tile; the engine calls
//     store8(args, batch, m, n, x[8]) for M indices m .. m + 7 at column n.
//   a_tile_hook(args, m0, n0, a_tile, tid, state) / a_hook_done(args, m0, n0,
//     tid, state): called by every thread after the MFMAs of each k chunk with
//     that chunk's A tile in LDS (k-contiguous layout above), and once after
//     the last chunk; `state` is one double per thread, zero at the start.
#pragma once

#include "gemm.h"

namespace mosa {

typedef __attribute__((address_space(3))) unsigned char lds_u8;

// One wave's 1 KB of LDS from 64 lanes x 16 bytes of global memory
// (global_load_lds_dwordx4: the LDS base goes in M0, lane l writes base +
// 16 l).  Issued as inline assembly so that the compiler does not treat the
// asynchronous LDS write as aliasing every later LDS read and wait for all
// loads in flight; the engine waits for these loads itself (wait_vmcnt).
// `base` is the wave-uniform LDS byte address of the 1 KB block.
__device__ __forceinline__ void lds_load16(const void* g, uint32_t base) {
    asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" : : "v"(g), "s"(base) : "memory", "m0");
}
__device__ __forceinline__ uint32_t lds_addr(const void* p) { return (uint32_t)(size_t)(const lds_u8*)p; }

// Four 16-bit elements of a transposed 4 x 4 block (see above), issued as
// inline assembly: the compiler cannot tell which LDS bytes the builtin form
// reads and would wait for every direct-to-LDS load in flight before it.  The
// result is not ready until lds_wait() below; nothing may read it earlier.
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ u32x2 lds_read_tr16(const unsigned char* p) {
    const uint32_t off = (uint32_t)(size_t)(lds_u8*)p;
    u32x2 r;
    asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(r) : "v"(off) : "memory");
    return r;
}
// The same at p + OFF bytes (the instruction's immediate offset).
template <int OFF>
__device__ __forceinline__ u32x2 lds_read_tr16_at(const unsigned char* p) {
    static_assert(OFF >= 0 && OFF < 65536, "ds offset field");
    const uint32_t off = (uint32_t)(size_t)(lds_u8*)p;
    u32x2 r;
    asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(r) : "v"(off), "i"(OFF) : "memory");
    return r;
}
// Wait for every outstanding LDS read of this wave.
__device__ __forceinline__ void lds_wait() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }
// Wait until at most N LDS operations of this wave are outstanding (LDS
// operations complete in issue order).
template <int N>
__device__ __forceinline__ void lds_wait_n() {
    static_assert(N >= 0 && N <= 15, "lgkmcnt range");
    asm volatile("s_waitcnt lgkmcnt(%0)" ::"n"(N) : "memory");
}
// lds_wait_n<n>() for an n that is a constant after unrolling.
template <int I = 0>
__device__ __forceinline__ void lds_wait_le(int n) {
    if constexpr (I < 15) {
        if (n == I) {
            lds_wait_n<I>();
            return;
        }
        lds_wait_le<I + 1>(n);
    } else {
        lds_wait_n<15>();
    }
}
// Make x depend on the preceding lds_wait() (an empty volatile statement that
// claims to modify x keeps its consumers after the wait).
__device__ __forceinline__ void lds_ready(u32x4& x) { asm volatile("" : "+v"(x)); }

// Unit permutations (both are involutions within a row).
__device__ __forceinline__ int kswz(int r, int lpr) {
    return lpr == 8 ? ((r & 7) ^ ((r >> 3) & 1)) : ((r & 3) ^ ((r >> 2) & 3));
}
template <int U>  // units per m-contiguous row
__device__ __forceinline__ int mswz(int k, int u) {
    if constexpr (U % 16 == 0) return u ^ (2 * ((k & 3) | (((k >> 3) & 1) << 2)));
    else if constexpr (U % 8 == 0) return u ^ (2 * (((k >> 1) & 1) | (((k >> 3) & 1) << 1)));
    else return u;
}

template <class P, class = void> struct G2Gather : std::false_type {};
template <class P> struct G2Gather<P, std::void_t<decltype(P::KGATHER)>> : std::bool_constant<P::KGATHER> {};
template <class P, class = void> struct G2Interleave : std::false_type {};
template <class P>
struct G2Interleave<P, std::void_t<decltype(P::A_INTERLEAVE)>> : std::bool_constant<P::A_INTERLEAVE> {};
template <class P, class = void> struct G2MinWaves : std::integral_constant<int, 1> {};
template <class P>
struct G2MinWaves<P, std::void_t<decltype(P::MIN_WAVES)>> : std::integral_constant<int, P::MIN_WAVES> {};
// CHUNK_ADD: every MFMA (32 k) starts from a zero accumulator and is added to
// the running sum with one fp32 add per element (a summation whose error
// bound does not depend on the MFMA's internal accumulation).
template <class P, class = void> struct G2ChunkAdd : std::false_type {};
template <class P> struct G2ChunkAdd<P, std::void_t<decltype(P::CHUNK_ADD)>> : std::bool_constant<P::CHUNK_ADD> {};
template <class P, class = void> struct G2AHook : std::false_type {};
template <class P> struct G2AHook<P, std::void_t<decltype(&P::a_tile_hook)>> : std::true_type {};
template <class P, class = void> struct G2EpiRegs : std::false_type {};
template <class P> struct G2EpiRegs<P, std::void_t<decltype(P::EPI_REGS)>> : std::bool_constant<P::EPI_REGS> {};

// a_koff(args, batch, c) / b_koff(args, batch, c): element offset of k chunk c
// from chunk 0 (k-contiguous operands whose k axis is made of segments, e.g.
// heads, that are not adjacent in memory; the policy keeps KC within one
// segment).  Default: c * KC (times the k-stride of an m-contiguous operand).
template <class P, class = void> struct G2AKoff : std::false_type {};
template <class P>
struct G2AKoff<P, std::void_t<decltype(P::a_koff(std::declval<const typename P::Args&>(), 0, 0))>> : std::true_type {};
template <class P, class = void> struct G2BKoff : std::false_type {};
template <class P>
struct G2BKoff<P, std::void_t<decltype(P::b_koff(std::declval<const typename P::Args&>(), 0, 0))>> : std::true_type {};

// Zeros for the rows past the end of a gathered range.
static __device__ __attribute__((aligned(16))) const uint16_t g2_zero[8] = {0, 0, 0, 0, 0, 0, 0, 0};

template <class P>
struct Gemm2Shape {
    static constexpr int MT = P::MT, NT = P::NT, KC = P::KC, WM = P::WM, WN = P::WN, STAGES = P::STAGES;
    static constexpr int WTM = MT / WM, WTN = NT / WN, FM = WTM / 16, FN = WTN / 16;
    static constexpr int LPR = KC / 8;  // units per k-contiguous row
    static constexpr int A_UNITS = P::A_KCONTIG ? MT * LPR : KC * (MT / 8);
    static constexpr int B_UNITS = P::B_KCONTIG ? NT * LPR : KC * (NT / 8);
    static constexpr int IA = A_UNITS / 256, IB = B_UNITS / 256;  // instructions per wave per chunk
    static constexpr int A_BYTES = A_UNITS * 16, B_BYTES = B_UNITS * 16;
    static constexpr int STAGE_BYTES = A_BYTES + B_BYTES;
    static_assert(WM * WN == 4 && WTM % 16 == 0 && WTN % 16 == 0 && KC % 32 == 0, "tile shape");
    static_assert(A_UNITS % 256 == 0 && B_UNITS % 256 == 0, "whole instructions per wave");
    static_assert((STAGES - 2) * (IA + IB) <= 63, "vmcnt range");
    static constexpr bool KG = G2Gather<P>::value, IL = G2Interleave<P>::value, ER = G2EpiRegs<P>::value;
    static constexpr bool CA = G2ChunkAdd<P>::value;
    static_assert(!KG || (!P::A_KCONTIG && !P::B_KCONTIG), "gathered k needs m-contiguous operands");
    static_assert(!IL || (!P::A_KCONTIG && FM % 2 == 0), "interleaved A needs m-contiguous pairs of blocks");
    static_assert(!ER || IL, "register epilogue needs interleaved A");
    static constexpr size_t ctile_bytes = ER ? 0 : (size_t)MT * (NT + 4) * sizeof(float);
    // LDS bytes; the k-row table of a gathered range (8 bytes per row of the
    // padded range) follows the stage buffers.
    static constexpr size_t lds_bytes(int ktab_rows = 0) {
        const size_t ops = (size_t)STAGES * STAGE_BYTES + (KG ? (size_t)ktab_rows * 8 : 0);
        const size_t epi = ER ? 0 : ctile_bytes + P::EPI_LDS;
        return ops > epi ? ops : epi;
    }
};

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N <= 63, "vmcnt");
    // gfx9 s_waitcnt: vmcnt [3:0] and [15:14], expcnt [6:4] = 7, lgkmcnt [11:8] = 15
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x0F70);
}

// One workgroup's tile of logical index `logical`.
template <class P>
__device__ __forceinline__ void gemm2_body(const typename P::Args& args, int logical, unsigned char* smem) {
    using ST = uint16_t;
    using S = Gemm2Shape<P>;
    constexpr int MT = S::MT, NT = S::NT, KC = S::KC, LPR = S::LPR, STG = S::STAGES;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, c16 = lane & 15;
    int batch, m0, n0;
    P::tile(args, logical, batch, m0, n0);
    const int K = P::k_size(args, batch);
    const int nchunks = S::KG ? (K + KC - 1) / KC : K / KC;
    int2* ktab = reinterpret_cast<int2*>(smem + STG * S::STAGE_BYTES);
    if constexpr (S::KG) {
        for (int i = tid; i < nchunks * KC; i += 256) ktab[i] = P::k_row(args, batch, i, K);
        __syncthreads();
    }

    // Where this lane's 16 bytes of each load instruction come from for chunk
    // 0, and how far they move per chunk (KC elements along k).  Computed once
    // so that the loop does plain pointer arithmetic.
    const ST* asrc[S::IA > 0 ? S::IA : 1];
    const ST* bsrc[S::IB > 0 ? S::IB : 1];
    uint32_t astr[S::IA > 0 ? S::IA : 1], bstr[S::IB > 0 ? S::IB : 1];  // gathered: element stride per table unit
    int akr[S::IA > 0 ? S::IA : 1], bkr[S::IB > 0 ? S::IB : 1];         // gathered: k row within the chunk
#pragma unroll
    for (int j = 0; j < S::IA; ++j) {
        const int p = 64 * (wave + 4 * j) + lane;  // unit of the tile
        if constexpr (P::A_KCONTIG) {
            const int r = p / LPR, pos = p % LPR;
            asrc[j] = P::a_elem(args, batch, P::a_row(args, batch, m0 + r), 8 * (pos ^ kswz(r, LPR)));
        } else {
            constexpr int U = MT / 8;
            const int kr = p / U, pos = p % U;
            if constexpr (S::KG) {
                P::a_mlane(args, batch, m0 + 8 * mswz<U>(kr, pos), asrc[j], astr[j]);
                akr[j] = kr;
            } else {
                asrc[j] = P::a_maddr(args, batch, kr, m0 + 8 * mswz<U>(kr, pos));
            }
        }
    }
#pragma unroll
    for (int j = 0; j < S::IB; ++j) {
        const int p = 64 * (wave + 4 * j) + lane;
        if constexpr (P::B_KCONTIG) {
            const int r = p / LPR, pos = p % LPR;
            bsrc[j] = P::b_elem(args, batch, P::b_row(args, batch, n0 + r), 8 * (pos ^ kswz(r, LPR)));
        } else {
            constexpr int U = NT / 8;
            const int kr = p / U, pos = p % U;
            if constexpr (S::KG) {
                P::b_mlane(args, batch, n0 + 8 * mswz<U>(kr, pos), bsrc[j], bstr[j]);
                bkr[j] = kr;
            } else {
                bsrc[j] = P::b_maddr(args, batch, kr, n0 + 8 * mswz<U>(kr, pos));
            }
        }
    }
    size_t astep = KC, bstep = KC;
    if constexpr (!P::A_KCONTIG && !S::KG) astep *= P::a_kstride(args, batch);
    if constexpr (!P::B_KCONTIG && !S::KG) bstep *= P::b_kstride(args, batch);

    // LDS address of this wave's first 1 KB block of a stage (scalar).
    const uint32_t lds_wave = __builtin_amdgcn_readfirstlane(lds_addr(smem) + 1024 * wave);

    // Gathered k: this lane's table entries for the next chunk to issue, read
    // one iteration ahead so that the LDS latency stays off the issue path.
    int arv[S::IA > 0 ? S::IA : 1], brv[S::IB > 0 ? S::IB : 1];
    auto load_rows = [&](int c) {
        if constexpr (S::KG) {
            const int cc = min(c, nchunks - 1);
#pragma unroll
            for (int j = 0; j < S::IA; ++j) {
                const int2 e = ktab[cc * KC + akr[j]];
                arv[j] = P::A_TAB ? e.y : e.x;
            }
#pragma unroll
            for (int j = 0; j < S::IB; ++j) {
                const int2 e = ktab[cc * KC + bkr[j]];
                brv[j] = P::B_TAB ? e.y : e.x;
            }
        }
    };
    // base + rv * stride, or the zero row for rv < 0 (branch-free)
    auto gathered = [](const ST* base, uint32_t stride, int rv) {
        const ST* p = base + (size_t)(uint32_t)max(rv, 0) * stride;
        return rv >= 0 ? p : g2_zero;
    };

    // Issue the loads of chunk c into its stage buffer (chunks past the end
    // load valid, clamped addresses into a buffer nobody reads).  Gathered k:
    // the table entries of chunk c must be in arv / brv (load_rows(c)).
    auto issue_buf = [&](int c, int bidx) {
        const uint32_t buf = lds_wave + bidx * S::STAGE_BYTES;
        const size_t kc = (size_t)min(c, nchunks - 1);
        ptrdiff_t aoff = 0, boff = 0;
        if constexpr (!S::KG) {
            if constexpr (G2AKoff<P>::value) aoff = P::a_koff(args, batch, (int)kc);
            else aoff = (ptrdiff_t)(kc * astep);
            if constexpr (G2BKoff<P>::value) boff = P::b_koff(args, batch, (int)kc);
            else boff = (ptrdiff_t)(kc * bstep);
        }
#pragma unroll
        for (int j = 0; j < S::IA; ++j) {
            if constexpr (S::KG) lds_load16(gathered(asrc[j], astr[j], arv[j]), buf + 4096 * j);
            else lds_load16(asrc[j] + aoff, buf + 4096 * j);
        }
#pragma unroll
        for (int j = 0; j < S::IB; ++j) {
            if constexpr (S::KG) lds_load16(gathered(bsrc[j], bstr[j], brv[j]), buf + S::A_BYTES + 4096 * j);
            else lds_load16(bsrc[j] + boff, buf + S::A_BYTES + 4096 * j);
        }
    };

    const int wm = wave / S::WN, wn = wave % S::WN;
    double hook_state = 0.0;
    f32x4 acc[S::FM][S::FN];
#pragma unroll
    for (int i = 0; i < S::FM; ++i)
#pragma unroll
        for (int j = 0; j < S::FN; ++j) acc[i][j] = zero4();

    // Fragment of 8 consecutive k at ks + 8g for operand row `row` (the
    // MFMA's M or N index) from a stage buffer.
    auto frag_k = [&](const unsigned char* t, int row, int ks) {
        const int s = (ks >> 3) + g;
        Frag8<ST> f;
        f.v = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(t + (row * LPR + (s ^ kswz(row, LPR))) * 16));
        return f;
    };
    // m-contiguous fragment: two transposed reads, raw (see lds_read_tr16)
    // (colstep 8 and odd: the interleaved pairs of A_INTERLEAVE)
    auto frag_m = [&](const unsigned char* t, int mbase, int ks, auto u_tag, int colstep = 4, int odd = 0) {
        constexpr int U = decltype(u_tag)::value;
        const int mcol = mbase + colstep * (c16 & 3) + 4 * odd;
        const int u = mcol >> 3, half = (mcol >> 2) & 1;
        const int k0r = ks + 8 * g + (c16 >> 2);
        const u32x2 lo = lds_read_tr16(t + (k0r * U + mswz<U>(k0r, u)) * 16 + 8 * half);
        const int k1r = k0r + 4;
        const u32x2 hi = lds_read_tr16(t + (k1r * U + mswz<U>(k1r, u)) * 16 + 8 * half);
        return u32x4{lo.x, lo.y, hi.x, hi.y};
    };
    auto mfma_buf = [&](int bidx) {
        const unsigned char* ta = smem + bidx * S::STAGE_BYTES;
        const unsigned char* tb = ta + S::A_BYTES;
#pragma unroll
        for (int ks = 0; ks < KC; ks += 32) {
            Frag8<ST> fa[S::FM], fb[S::FN];
            u32x4 ma[S::FM], mb[S::FN];  // raw m-contiguous fragments
            if constexpr (!P::A_KCONTIG && !P::B_KCONTIG) {
#pragma unroll
                for (int j = 0; j < S::FN; ++j)
                    mb[j] = frag_m(tb, wn * S::WTN + j * 16, ks, std::integral_constant<int, NT / 8>{});
            }
#pragma unroll
            for (int i = 0; i < S::FM; ++i) {
                if constexpr (P::A_KCONTIG) fa[i] = frag_k(ta, wm * S::WTM + i * 16 + c16, ks);
                else if constexpr (S::IL)
                    ma[i] = frag_m(ta, wm * S::WTM + 32 * (i >> 1), ks, std::integral_constant<int, MT / 8>{}, 8, i & 1);
                else ma[i] = frag_m(ta, wm * S::WTM + i * 16, ks, std::integral_constant<int, MT / 8>{});
            }
#pragma unroll
            for (int j = 0; j < S::FN; ++j) {
                if constexpr (P::B_KCONTIG) fb[j] = frag_k(tb, wn * S::WTN + j * 16 + c16, ks);
                else if constexpr (P::A_KCONTIG)
                    mb[j] = frag_m(tb, wn * S::WTN + j * 16, ks, std::integral_constant<int, NT / 8>{});
            }
            if constexpr (!P::A_KCONTIG && !P::B_KCONTIG) {
                // Both operands by transposed reads: B's were issued first, so
                // after the wait for A fragment i (2 reads each) the MFMAs of
                // that row block can start while later reads are in flight.
                static_assert(2 * (S::FM - 1) <= 15, "lgkmcnt range");
#pragma unroll
                for (int i = 0; i < S::FM; ++i) {
                    lds_wait_le(2 * (S::FM - 1 - i));
                    if (i == 0) {
#pragma unroll
                        for (int j = 0; j < S::FN; ++j) {
                            lds_ready(mb[j]);
                            fb[j].v = __builtin_bit_cast(bf16x8, mb[j]);
                        }
                    }
                    lds_ready(ma[i]);
                    fa[i].v = __builtin_bit_cast(bf16x8, ma[i]);
#pragma unroll
                    for (int j = 0; j < S::FN; ++j) mma8(acc[i][j], fa[i], fb[j]);
                    __builtin_amdgcn_sched_barrier(0);  // keep these MFMAs before the next wait
                }
                continue;
            }
            if constexpr (!P::A_KCONTIG || !P::B_KCONTIG) {
                lds_wait();
#pragma unroll
                for (int i = 0; i < S::FM; ++i)
                    if constexpr (!P::A_KCONTIG) {
                        lds_ready(ma[i]);
                        fa[i].v = __builtin_bit_cast(bf16x8, ma[i]);
                    }
#pragma unroll
                for (int j = 0; j < S::FN; ++j)
                    if constexpr (!P::B_KCONTIG) {
                        lds_ready(mb[j]);
                        fb[j].v = __builtin_bit_cast(bf16x8, mb[j]);
                    }
            }
#pragma unroll
            for (int i = 0; i < S::FM; ++i)
#pragma unroll
                for (int j = 0; j < S::FN; ++j) {
                    if constexpr (S::CA) {
                        f32x4 part = zero4();
                        mma8(part, fa[i], fb[j]);
                        acc[i][j] += part;
                    } else {
                        mma8(acc[i][j], fa[i], fb[j]);
                    }
                }
        }
    };

    // Pipeline: STAGES - 1 chunks in flight; per chunk one wait, one barrier,
    // the loads of chunk c + STAGES - 1, then the MFMAs of chunk c.  Every
    // wave issues exactly IA + IB loads per chunk, so the wait count is a
    // constant.  An empty K range (no dense heads) issues nothing.
    // The loop is unrolled by STAGES so that every stage buffer has a constant
    // LDS offset: the compiler then sees that the loads in flight write other
    // buffers than the one being read and does not wait for them.
    // The only way out is after the MFMAs of the last chunk, through
    // mfma_drain(): the compiler misses the MFMA result hazard on loop-exit
    // edges, where it moves the accumulators to other registers.
    if (nchunks > 0) {
#pragma unroll
        for (int s = 0; s < STG - 1; ++s) {
            load_rows(s);
            issue_buf(s, s);
        }
        load_rows(STG - 1);
        for (int c0 = 0;; c0 += STG) {
#pragma unroll
            for (int u = 0; u < STG; ++u) {
                const int c = c0 + u;
                wait_vmcnt<(STG - 2) * (S::IA + S::IB)>();
                __syncthreads();  // chunk c is in LDS for every wave; chunk c-1's buffer is free
                issue_buf(c + STG - 1, (u + STG - 1) % STG);
                load_rows(c + STG);
                __builtin_amdgcn_sched_barrier(0);
                mfma_buf(u);
                if constexpr (G2AHook<P>::value) P::a_tile_hook(args, m0, n0, smem + u * S::STAGE_BYTES, tid, hook_state);
                if (c + 1 == nchunks) {
                    mfma_drain();
                    goto pipeline_done;
                }
            }
        }
    }
pipeline_done:
    if constexpr (G2AHook<P>::value) P::a_hook_done(args, m0, n0, tid, hook_state);
    wait_vmcnt<0>();  // the trailing loads write into the buffers the C tile reuses
    if constexpr (S::ER) {
        // lane: M indices 32 p + 8 g .. + 7 of the wave's rows, column c16 of block j
#pragma unroll
        for (int p = 0; p < S::FM / 2; ++p)
#pragma unroll
            for (int j = 0; j < S::FN; ++j) {
                float x[8];
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    x[r] = acc[2 * p][j][r];
                    x[4 + r] = acc[2 * p + 1][j][r];
                }
                P::store8(args, batch, m0 + wm * S::WTM + 32 * p + 8 * g, n0 + wn * S::WTN + 16 * j + c16, x);
            }
    } else {
        __syncthreads();

        // C tile to LDS: Cs[m][n], row stride NT + 4 floats
        float* Cs = reinterpret_cast<float*>(smem);
        constexpr int LDC = NT + 4;
#pragma unroll
        for (int i = 0; i < S::FM; ++i)
#pragma unroll
            for (int j = 0; j < S::FN; ++j)
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    Cs[(wm * S::WTM + i * 16 + 4 * g + r) * LDC + wn * S::WTN + j * 16 + c16] = acc[i][j][r];
        __syncthreads();
        P::epilogue(args, batch, m0, n0, Cs, LDC, tid, smem + S::ctile_bytes);
    }
}

template <class P>
__global__ __launch_bounds__(256, G2MinWaves<P>::value) void gemm2_kernel(const typename P::Args args) {
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
    gemm2_body<P>(args, xcd_logical_id(blockIdx.x, gridDim.x), smem);
}

// Two independent GEMMs in one launch (n1 workgroups of P1, the rest P2),
// mixed on every XCD so that both kinds share its CUs: the blocks an XCD
// receives (every eighth) are its share of P1 first, in index order, then
// its share of P2.
__device__ __forceinline__ void xcd_dual_id(int b, int nb, int n1, int& which, int& idx) {
    const int x = b % 8, j = b / 8;
    const int q = nb / 8, r = nb % 8, q1 = n1 / 8, r1 = n1 % 8;
    const int cnt1 = q1 + (x < r1 ? 1 : 0);
    const int s1 = x * q1 + (x < r1 ? x : r1);                // P1 blocks on lower XCDs
    const int sall = x * q + (x < r ? x : r);                // all blocks on lower XCDs
    if (j < cnt1) {
        which = 0;
        idx = s1 + j;
    } else {
        which = 1;
        idx = (sall - s1) + (j - cnt1);
    }
}

template <class P1, class P2>
__global__ __launch_bounds__(256, (G2MinWaves<P1>::value > G2MinWaves<P2>::value ? G2MinWaves<P1>::value
                                                                                  : G2MinWaves<P2>::value))
void gemm2_dual_kernel(const typename P1::Args a1, const typename P2::Args a2, int n1) {
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
    int which, idx;
    xcd_dual_id(blockIdx.x, gridDim.x, n1, which, idx);
    if (which == 0) gemm2_body<P1>(a1, idx, smem);
    else gemm2_body<P2>(a2, idx, smem);
}

// ktab_rows: rows of the k-row table (gathered k: the padded k range).
template <class P>
int launch_gemm2(const typename P::Args& args, int nblocks, hipStream_t stream, int ktab_rows = 0) {
    if (nblocks <= 0) return 0;
    const size_t lds = Gemm2Shape<P>::lds_bytes(ktab_rows);
    if (lds > 160 * 1024) return -1;
    auto kern = gemm2_kernel<P>;
    if (allow_lds((const void*)kern, lds)) return -1;
    hipLaunchKernelGGL(kern, dim3(nblocks), dim3(256), lds, stream, args);
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

// Both GEMMs in one launch (see gemm2_dual_kernel); requires every XCD's
// share of the blocks to hold its share of P1.
template <class P1, class P2>
int launch_gemm2_dual(const typename P1::Args& a1, int n1, int rows1, const typename P2::Args& a2, int n2, int rows2,
                      hipStream_t stream) {
    if (n1 <= 0) return launch_gemm2<P2>(a2, n2, stream, rows2);
    if (n2 <= 0) return launch_gemm2<P1>(a1, n1, stream, rows1);
    const size_t l1 = Gemm2Shape<P1>::lds_bytes(rows1), l2 = Gemm2Shape<P2>::lds_bytes(rows2);
    const size_t lds = l1 > l2 ? l1 : l2;
    if (lds > 160 * 1024) return -1;
    const int nb = n1 + n2;
    for (int x = 0; x < 8; ++x)  // xcd_dual_id's assumption
        if (nb / 8 + (x < nb % 8 ? 1 : 0) < n1 / 8 + (x < n1 % 8 ? 1 : 0)) return -1;
    auto kern = gemm2_dual_kernel<P1, P2>;
    if (allow_lds((const void*)kern, lds)) return -1;
    hipLaunchKernelGGL(kern, dim3(nb), dim3(256), lds, stream, a1, a2, n1);
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

}  // namespace mosa
