// Tiled MFMA GEMM engine shared by the projection-shaped stages of the layer.
//
//   C[M x N] = sum_k A[M x K] B[K x N]   (fp32 accumulation), one problem per
//   "batch" index (a head or a batch element), tiles of MT x NT.
//
// Operands are staged through LDS in a k-contiguous layout (As[m][k],
// Bs[n][k]) because the MFMA operand of every lane is 8 consecutive k values.
// A policy class P says where the 8-element vectors live in memory:
//   P::A_KCONTIG: a_row(m) returns a row reference (P::ARef, computed once per
//                thread, e.g. after a token-index gather) and a_elem(ref, k)
//                the address of elements k..k+7 (nullptr: zeros); likewise
//                P::B_KCONTIG with BRef / b_row / b_elem;
//   otherwise    the source is m- (or n-) contiguous: "row" k of the operand
//                is described by P::RowInfo = P::row_info(k) (e.g. a gathered
//                token row and a router value), computed one chunk ahead into
//                LDS so that the data loads of a chunk depend on LDS only;
//                a_kaddr(info, m8) / b_kaddr(info, n8) give an address of 8
//                consecutive elements that is always safe to load (clamped),
//                a_kok / b_kok whether they are real (else zeros) and
//                a_kscale(info) an optional scale.
//                The engine transposes 8x8 blocks in registers so that LDS
//                stores stay 16-byte wide.
// a_fallback / b_fallback give a valid address that is loaded (and then
// zeroed) in place of out-of-range k-contiguous vectors, so that every load of
// a chunk is issued without a branch and waited for only at the commit.
// Rows may be gathered (token indices), scaled (router values) or come from
// concatenated matrices; out-of-range vectors are nullptr and read as zero.
// The K loop is double-buffered: the global loads of chunk c+1 are issued
// before the MFMAs of chunk c.  After the loop the fp32 C tile is written to
// LDS (reusing the operand buffers) and P::epilogue writes it out with wide,
// coalesced stores and any fused elementwise work (P::EPI_LDS extra bytes of
// LDS after the C tile are the epilogue's own).
#pragma once

#include <type_traits>

#include "common.h"

namespace mosa {

// 8 consecutive storage elements.
template <typename ST> struct Vec8;
template <> struct Vec8<uint16_t> { uint4 v; };
template <> struct Vec8<float> { float4 a, b; };

template <typename ST> __device__ __forceinline__ Vec8<ST> vec8_zero();
template <> __device__ __forceinline__ Vec8<uint16_t> vec8_zero<uint16_t>() { return {make_uint4(0, 0, 0, 0)}; }
template <> __device__ __forceinline__ Vec8<float> vec8_zero<float>() {
    return {make_float4(0.f, 0.f, 0.f, 0.f), make_float4(0.f, 0.f, 0.f, 0.f)};
}

template <typename ST> __device__ __forceinline__ Vec8<ST> vec8_load(const ST* p);
template <> __device__ __forceinline__ Vec8<uint16_t> vec8_load<uint16_t>(const uint16_t* p) {
    return {*reinterpret_cast<const uint4*>(p)};
}
template <> __device__ __forceinline__ Vec8<float> vec8_load<float>(const float* p) {
    return {reinterpret_cast<const float4*>(p)[0], reinterpret_cast<const float4*>(p)[1]};
}

template <typename ST> __device__ __forceinline__ void vec8_store(ST* p, const Vec8<ST>& v);
template <> __device__ __forceinline__ void vec8_store<uint16_t>(uint16_t* p, const Vec8<uint16_t>& v) {
    *reinterpret_cast<uint4*>(p) = v.v;
}
template <> __device__ __forceinline__ void vec8_store<float>(float* p, const Vec8<float>& v) {
    reinterpret_cast<float4*>(p)[0] = v.a;
    reinterpret_cast<float4*>(p)[1] = v.b;
}

template <typename ST> __device__ __forceinline__ void vec8_to_f32(const Vec8<ST>& v, float (&x)[8]);
template <> __device__ __forceinline__ void vec8_to_f32<uint16_t>(const Vec8<uint16_t>& v, float (&x)[8]) {
    x[0] = __uint_as_float(v.v.x << 16); x[1] = __uint_as_float(v.v.x & 0xffff0000u);
    x[2] = __uint_as_float(v.v.y << 16); x[3] = __uint_as_float(v.v.y & 0xffff0000u);
    x[4] = __uint_as_float(v.v.z << 16); x[5] = __uint_as_float(v.v.z & 0xffff0000u);
    x[6] = __uint_as_float(v.v.w << 16); x[7] = __uint_as_float(v.v.w & 0xffff0000u);
}
template <> __device__ __forceinline__ void vec8_to_f32<float>(const Vec8<float>& v, float (&x)[8]) {
    x[0] = v.a.x; x[1] = v.a.y; x[2] = v.a.z; x[3] = v.a.w;
    x[4] = v.b.x; x[5] = v.b.y; x[6] = v.b.z; x[7] = v.b.w;
}

template <typename ST> __device__ __forceinline__ Vec8<ST> vec8_from_f32(const float (&x)[8]);
template <> __device__ __forceinline__ Vec8<uint16_t> vec8_from_f32<uint16_t>(const float (&x)[8]) {
    uint4 u;
    u.x = pack_bf16x2(x[0], x[1]);
    u.y = pack_bf16x2(x[2], x[3]);
    u.z = pack_bf16x2(x[4], x[5]);
    u.w = pack_bf16x2(x[6], x[7]);
    return {u};
}
template <> __device__ __forceinline__ Vec8<float> vec8_from_f32<float>(const float (&x)[8]) {
    return {make_float4(x[0], x[1], x[2], x[3]), make_float4(x[4], x[5], x[6], x[7])};
}

template <typename ST> __device__ __forceinline__ Vec8<ST> vec8_scale(const Vec8<ST>& v, float s) {
    float x[8];
    vec8_to_f32<ST>(v, x);
#pragma unroll
    for (int j = 0; j < 8; ++j) x[j] *= s;
    return vec8_from_f32<ST>(x);
}

// out[j] holds element j of every in[i] (an 8 x 8 transpose).
__device__ __forceinline__ void transpose8(const Vec8<uint16_t> (&in)[8], Vec8<uint16_t> (&out)[8]) {
    uint32_t w[8][4];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        w[i][0] = in[i].v.x; w[i][1] = in[i].v.y; w[i][2] = in[i].v.z; w[i][3] = in[i].v.w;
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        uint32_t o[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const uint32_t lo = w[2 * q][j >> 1], hi = w[2 * q + 1][j >> 1];
            // low halves (j even) or high halves (j odd) of the two words
            o[q] = (j & 1) ? __builtin_amdgcn_perm(hi, lo, 0x07060302u) : __builtin_amdgcn_perm(hi, lo, 0x05040100u);
        }
        out[j].v = make_uint4(o[0], o[1], o[2], o[3]);
    }
}
__device__ __forceinline__ void transpose8(const Vec8<float> (&in)[8], Vec8<float> (&out)[8]) {
    float x[8][8];
#pragma unroll
    for (int i = 0; i < 8; ++i) vec8_to_f32<float>(in[i], x[i]);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        float y[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) y[i] = x[i][j];
        out[j] = vec8_from_f32<float>(y);
    }
}

template <class P>
struct GemmShape {
    static constexpr int MT = P::MT, NT = P::NT, KC = P::KC, WM = P::WM, WN = P::WN;
    static constexpr int LDK = KC + 8;  // padded row (elements)
    static constexpr int WTM = MT / WM, WTN = NT / WN;
    static constexpr int FM = WTM / 16, FN = WTN / 16;
    static constexpr int A_VECS = MT * KC / 8;         // k-contiguous staging
    static constexpr int B_VECS = NT * KC / 8;
    static constexpr int A_BLKS = (MT / 8) * (KC / 8);  // transposed staging
    static constexpr int B_BLKS = (NT / 8) * (KC / 8);
    static constexpr int A_PER = P::A_KCONTIG ? (A_VECS + 255) / 256 : (A_BLKS + 255) / 256;
    static constexpr int B_PER = P::B_KCONTIG ? (B_VECS + 255) / 256 : (B_BLKS + 255) / 256;
    static_assert(WM * WN == 4, "4 waves");
    static_assert(WTM % 16 == 0 && WTN % 16 == 0 && KC % 32 == 0, "tile shape");
    static constexpr bool ROWS = !P::A_KCONTIG || !P::B_KCONTIG;  // row-info table needed
    static constexpr size_t ctile_bytes = (size_t)MT * (NT + 4) * sizeof(float);
    template <typename ST>
    static constexpr size_t ops_bytes() { return (size_t)2 * (MT + NT) * LDK * sizeof(ST); }
    static constexpr size_t rows_bytes = ROWS ? (size_t)2 * KC * sizeof(typename P::RowInfo) : 0;
    template <typename ST>
    static constexpr size_t lds_bytes() {
        const size_t ops = ops_bytes<ST>() + rows_bytes;
        const size_t epi = ctile_bytes + P::EPI_LDS;  // C tile + the epilogue's own LDS
        return ops > epi ? ops : epi;
    }
};

// Staging registers for one operand tile (raw loads plus validity and scale;
// masking and scaling are applied when the tile is committed to LDS).
template <typename ST, bool KCONTIG, int PER> struct Stage;
template <typename ST, int PER> struct Stage<ST, true, PER> {
    Vec8<ST> v[PER];
    bool ok[PER];
};
template <typename ST, int PER> struct Stage<ST, false, PER> {
    Vec8<ST> v[PER][8];
    float sc[PER][8];
    uint32_t ok[PER];  // bit i: row i of the 8 x 8 block is valid
};

// Vectorised read of 8 floats of the C tile (row stride ldc, 16-byte aligned).
__device__ __forceinline__ void cs_load8(const float* Cs, int ldc, int row, int col, float (&x)[8]) {
    const float4 a = *reinterpret_cast<const float4*>(Cs + row * ldc + col);
    const float4 b = *reinterpret_cast<const float4*>(Cs + row * ldc + col + 4);
    x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w;
    x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
}

// Split-K policies (P::SPLITK defined) map a workgroup to (batch, tile,
// split) with tile_split, restrict it to k_range(split) (a multiple of KC
// wide) and finish with epilogue_split, which writes an fp32 partial tile;
// a separate pass adds the partials in split order, so the result stays
// bitwise reproducible.
template <class P, class = void> struct SplitKTrait { static constexpr bool value = false; };
template <class P> struct SplitKTrait<P, std::void_t<decltype(P::SPLITK)>> { static constexpr bool value = P::SPLITK; };
template <class P> constexpr bool kSplitK = SplitKTrait<P>::value;

// s_waitcnt immediate for vmcnt(0) with expcnt and lgkmcnt left at their
// maxima (gfx9 encoding: vmcnt [3:0] and [15:14], expcnt [6:4], lgkmcnt [11:8]).
constexpr int kWaitVm0 = 0x0F70;

template <typename ST, class P>
__global__ __launch_bounds__(256) void gemm_kernel(const typename P::Args args) {
    using S = GemmShape<P>;
    constexpr int MT = S::MT, NT = S::NT, KC = S::KC, LDK = S::LDK;
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
    ST* As = reinterpret_cast<ST*>(smem);   // [2][MT][LDK]
    ST* Bs = As + 2 * MT * LDK;             // [2][NT][LDK]

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, c16 = lane & 15;
    int batch, m0, n0, split = 0;
    const int logical = xcd_logical_id(blockIdx.x, gridDim.x);
    if constexpr (kSplitK<P>) P::tile_split(args, logical, batch, m0, n0, split);
    else P::tile(args, logical, batch, m0, n0);
    const int K = P::k_size(args, batch);
    // this workgroup's share of the K range (the whole range unless split)
    int kbeg = 0, kend = K;
    if constexpr (kSplitK<P>) P::k_range(args, split, K, kbeg, kend);
    const int nchunks = kend > kbeg ? (kend - kbeg + KC - 1) / KC : 0;

    // Per-thread row references of the k-contiguous operands (fixed across chunks).
    typename P::ARef arow[S::A_PER > 0 ? S::A_PER : 1];
    float ascale[S::A_PER > 0 ? S::A_PER : 1];
    typename P::BRef brow[S::B_PER > 0 ? S::B_PER : 1];
    if constexpr (P::A_KCONTIG) {
#pragma unroll
        for (int j = 0; j < S::A_PER; ++j) {
            const int v = tid + 256 * j;
            ascale[j] = 1.f;
            arow[j] = P::a_row(args, batch, v < S::A_VECS ? m0 + v / (KC / 8) : -1, ascale[j]);
        }
    }
    if constexpr (P::B_KCONTIG) {
#pragma unroll
        for (int j = 0; j < S::B_PER; ++j) {
            const int v = tid + 256 * j;
            brow[j] = P::b_row(args, batch, v < S::B_VECS ? n0 + v / (KC / 8) : -1);
        }
    }

    Stage<ST, P::A_KCONTIG, S::A_PER> sa;
    Stage<ST, P::B_KCONTIG, S::B_PER> sb;
    // row infos of chunks (m/n-contiguous operands), double-buffered in LDS
    typename P::RowInfo* rinfo =
        reinterpret_cast<typename P::RowInfo*>(smem + S::template ops_bytes<ST>());
    // row_info may issue global loads (a token gather): it is called before
    // the chunk's data loads and its result stored to LDS only after the MFMAs,
    // so waiting for it never waits for the (younger) data loads.
    // Loads and the instructions that consume them are kept outside divergent
    // branches (threads past the end duplicate a neighbour's work and only
    // their stores are skipped), so the compiler's waits stay where the data
    // is consumed instead of being merged conservatively round the loop.
    auto rows_load = [&](int k0) {
        typename P::RowInfo info{};
        if constexpr (S::ROWS) {
            const int kk = k0 + (tid & (KC - 1));
            info = P::row_info(args, batch, kk < kend ? kk : -1);
        }
        return info;
    };
    auto rows_store = [&](const typename P::RowInfo& info, int buf) {
        if constexpr (S::ROWS) {
            if (tid < KC) rinfo[buf * KC + tid] = info;
        }
    };

    auto fetch = [&](int k0, int rbuf) {
        if constexpr (P::A_KCONTIG) {
#pragma unroll
            for (int j = 0; j < S::A_PER; ++j) {
                const int v = tid + 256 * j;
                const int kk = k0 + (v % (KC / 8)) * 8;
                const ST* p = (v < S::A_VECS && kk < kend) ? P::a_elem(args, batch, arow[j], kk) : nullptr;
                sa.ok[j] = p != nullptr;
                sa.v[j] = vec8_load<ST>(p ? p : P::a_fallback(args));
            }
        } else {
#pragma unroll
            for (int j = 0; j < S::A_PER; ++j) {
                const int blk = (tid + 256 * j) % S::A_BLKS;
                {
                    const int mb = blk / (KC / 8), kb = blk % (KC / 8);
                    const int m8 = m0 + mb * 8;
                    typename P::RowInfo ri[8];
#pragma unroll
                    for (int i = 0; i < 8; ++i) ri[i] = rinfo[rbuf * KC + kb * 8 + i];
                    uint32_t ok = 0;
#pragma unroll
                    for (int i = 0; i < 8; ++i) {
                        ok |= (uint32_t)P::a_kok(args, batch, ri[i], m8) << i;
                        sa.sc[j][i] = P::a_kscale(args, batch, ri[i]);
                        sa.v[j][i] = vec8_load<ST>(P::a_kaddr(args, batch, ri[i], m8));
                    }
                    sa.ok[j] = ok;
                }
            }
        }
        if constexpr (P::B_KCONTIG) {
#pragma unroll
            for (int j = 0; j < S::B_PER; ++j) {
                const int v = tid + 256 * j;
                const int kk = k0 + (v % (KC / 8)) * 8;
                const ST* p = (v < S::B_VECS && kk < kend) ? P::b_elem(args, batch, brow[j], kk) : nullptr;
                sb.ok[j] = p != nullptr;
                sb.v[j] = vec8_load<ST>(p ? p : P::b_fallback(args));
            }
        } else {
#pragma unroll
            for (int j = 0; j < S::B_PER; ++j) {
                const int blk = (tid + 256 * j) % S::B_BLKS;
                {
                    const int nb = blk / (KC / 8), kb = blk % (KC / 8);
                    const int n8 = n0 + nb * 8;
                    typename P::RowInfo ri[8];
#pragma unroll
                    for (int i = 0; i < 8; ++i) ri[i] = rinfo[rbuf * KC + kb * 8 + i];
                    uint32_t ok = 0;
#pragma unroll
                    for (int i = 0; i < 8; ++i) {
                        ok |= (uint32_t)P::b_kok(args, batch, ri[i], n8) << i;
                        sb.v[j][i] = vec8_load<ST>(P::b_kaddr(args, batch, ri[i], n8));
                    }
                    sb.ok[j] = ok;
                }
            }
        }
    };
    auto commit = [&](int buf) {
        // Every load still in flight belongs to this chunk (or is the older
        // row-info load): wait for all of them here, explicitly, so that the
        // compiler's wait tracking does not carry them round the loop.
        __builtin_amdgcn_s_waitcnt(kWaitVm0);
        ST* a = As + buf * MT * LDK;
        ST* b = Bs + buf * NT * LDK;
        if constexpr (P::A_KCONTIG) {
#pragma unroll
            for (int j = 0; j < S::A_PER; ++j) {
                const int v = tid + 256 * j;
                if (v < S::A_VECS) {
                    Vec8<ST> x = sa.ok[j] ? sa.v[j] : vec8_zero<ST>();
                    if (P::A_SCALED) x = vec8_scale<ST>(x, ascale[j]);
                    vec8_store<ST>(a + (v / (KC / 8)) * LDK + (v % (KC / 8)) * 8, x);
                }
            }
        } else {
#pragma unroll
            for (int j = 0; j < S::A_PER; ++j) {
                const int blk = (tid + 256 * j) % S::A_BLKS;
                const int mb = blk / (KC / 8), kb = blk % (KC / 8);
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    if (!((sa.ok[j] >> i) & 1u)) sa.v[j][i] = vec8_zero<ST>();
                    else if (P::A_SCALED) sa.v[j][i] = vec8_scale<ST>(sa.v[j][i], sa.sc[j][i]);
                }
                Vec8<ST> t[8];
                transpose8(sa.v[j], t);
                if (tid + 256 * j < S::A_BLKS) {
#pragma unroll
                    for (int i = 0; i < 8; ++i) vec8_store<ST>(a + (mb * 8 + i) * LDK + kb * 8, t[i]);
                }
            }
        }
        if constexpr (P::B_KCONTIG) {
#pragma unroll
            for (int j = 0; j < S::B_PER; ++j) {
                const int v = tid + 256 * j;
                if (v < S::B_VECS)
                    vec8_store<ST>(b + (v / (KC / 8)) * LDK + (v % (KC / 8)) * 8, sb.ok[j] ? sb.v[j] : vec8_zero<ST>());
            }
        } else {
#pragma unroll
            for (int j = 0; j < S::B_PER; ++j) {
                const int blk = (tid + 256 * j) % S::B_BLKS;
                const int nb = blk / (KC / 8), kb = blk % (KC / 8);
#pragma unroll
                for (int i = 0; i < 8; ++i)
                    if (!((sb.ok[j] >> i) & 1u)) sb.v[j][i] = vec8_zero<ST>();
                Vec8<ST> t[8];
                transpose8(sb.v[j], t);
                if (tid + 256 * j < S::B_BLKS) {
#pragma unroll
                    for (int i = 0; i < 8; ++i) vec8_store<ST>(b + (nb * 8 + i) * LDK + kb * 8, t[i]);
                }
            }
        }
    };

    const int wm = wave / S::WN, wn = wave % S::WN;
    f32x4 acc[S::FM][S::FN];
#pragma unroll
    for (int i = 0; i < S::FM; ++i)
#pragma unroll
        for (int j = 0; j < S::FN; ++j) acc[i][j] = zero4();

    // Pipeline: row infos of chunk c+2 and data of chunk c+1 are in flight
    // while the MFMAs of chunk c run.
    // The MFMAs of the last chunk below run unconditionally: the accumulators
    // are read right after them, and no branch may separate an MFMA from the
    // VALU reads of its result (the compiler's wait-state insertion for that
    // hazard has been seen to miss a path through such a branch).  An empty
    // K range (e.g. no dense heads, whose operand pointers are then null)
    // issues no global load at all: buffer 0 is cleared in LDS instead.
    if (nchunks > 0) {
        rows_store(rows_load(kbeg), 0);
        __syncthreads();
        const typename P::RowInfo r1 = rows_load(kbeg + KC);
        fetch(kbeg, 0);
        rows_store(r1, 1);
        commit(0);
        __syncthreads();
    } else {
        // both operand buffers (A at As, B at Bs = As + 2 MT LDK), all in LDS
        for (int e = tid; e < 2 * (MT + NT) * LDK / 8; e += 256) vec8_store<ST>(As + 8 * e, vec8_zero<ST>());
        __syncthreads();
    }
    auto mfma_chunk = [&](int buf) {
        const ST* a = As + buf * MT * LDK;
        const ST* b = Bs + buf * NT * LDK;
#pragma unroll
        for (int ks = 0; ks < KC; ks += 32) {
            Frag8<ST> fa[S::FM], fb[S::FN];
#pragma unroll
            for (int i = 0; i < S::FM; ++i)
                fa[i] = frag8_load<ST>(a + (wm * S::WTM + i * 16 + c16) * LDK + ks + 8 * g);
#pragma unroll
            for (int j = 0; j < S::FN; ++j)
                fb[j] = frag8_load<ST>(b + (wn * S::WTN + j * 16 + c16) * LDK + ks + 8 * g);
#pragma unroll
            for (int i = 0; i < S::FM; ++i)
#pragma unroll
                for (int j = 0; j < S::FN; ++j) mma8(acc[i][j], fa[i], fb[j]);
        }
    };
    // Every chunk but the last: the loop body has no conditional load, so the
    // waits for the loads of chunk c+1 stay at the commit.  The last chunk's
    // MFMAs are peeled off below.
    for (int c = 0; c < nchunks - 1; ++c) {
        const int buf = c & 1;
        const typename P::RowInfo r2 = rows_load(kbeg + (c + 2) * KC);
        // keep the compiler from sinking these loads towards their uses: the
        // row-info load goes first, the chunk's data loads before the MFMAs
        __builtin_amdgcn_sched_barrier(0);
        fetch(kbeg + (c + 1) * KC, buf ^ 1);
        __builtin_amdgcn_sched_barrier(0);
        mfma_chunk(buf);
        rows_store(r2, buf);  // rows of chunk c were consumed by fetch(c) one step earlier
        commit(buf ^ 1);
        __syncthreads();
    }
    mfma_chunk(nchunks > 0 ? (nchunks - 1) & 1 : 0);
    mfma_drain();  // explicit wait states before the accumulators are read
    __syncthreads();  // the C tile below reuses the operand buffers

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
    if constexpr (kSplitK<P>) P::epilogue_split(args, batch, split, m0, n0, Cs, LDC, tid);
    else P::epilogue(args, batch, m0, n0, Cs, LDC, tid, smem + S::ctile_bytes);
}

template <typename ST, class P>
int launch_gemm(const typename P::Args& args, int nblocks, hipStream_t stream) {
    if (nblocks <= 0) return 0;
    constexpr size_t lds = GemmShape<P>::template lds_bytes<ST>();
    auto kern = gemm_kernel<ST, P>;
    if (allow_lds((const void*)kern, lds)) return -1;
    hipLaunchKernelGGL(kern, dim3(nblocks), dim3(256), lds, stream, args);
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

}  // namespace mosa
