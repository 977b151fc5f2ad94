// Certified expert-choice top-k (paper Section 2.2: each head keeps the k
// tokens with the highest router score; Section 2.1 footnote: chosen
// separately for every batch element).
//
// Contract: the selected set equals the k tokens that come first under
// (exact logit s_t rounded once to double, descending; token index,
// ascending), returned in ascending index order.  The router kernel gives an
// fp32 logit z~_t with a proven bound |z~_t - s_t| <= beta_t, so every token
// has an interval [lo_t, hi_t] that contains its key.  One workgroup of
// several waves per (b, h) row:
//   1. radix-select (4 passes of 8 bits over order-preserving uint32 keys held
//      in registers, LDS histograms) the k-th largest lo, A, and the (k+1)-th
//      largest hi, B;
//   2. hi_t < A  => at least k tokens certainly beat t: t is out;
//      lo_t > B  => at most k-1 tokens can beat t: t is in;
//      the rest (typically none or two tokens at the threshold) is uncertain;
//   3. the uncertain tokens are re-scored in fp64 (exact products, bounded
//      summation error), which orders them unless their keys (nearly) tie;
//      only then is the exact key computed with a long accumulator
//      (exact_dot.h; lanes add integer digits with LDS atomics, which is
//      order-independent); the k - #in best of them under (key desc, index
//      asc) are chosen;
//   4. the chosen tokens are compacted in index order: I ascending,
//      r = sigmoid(z~), and the token -> slot map (slot of t in I, or -1).
//
// The error bound of z~ (router.hip): every K = 32 MFMA chunk starts from
// zero; its result is taken to differ from the exact chunk sum by at most
// (K+1) units in the last place of the largest term for any aligned-and-
// truncated adder, doubled for margin, and covering the rounded fp32
// products of the fp32 variant: 96 u32 sum|x_i w_i|.  The n_c chunk results
// are added by sequential fp32 adds: at most 1.01 n_c u sum|chunk|.
// sum|x_i w_i| <= ||x|| ||w|| (Cauchy-Schwarz).  Denormal flushing of inputs,
// products or partial sums adds at most (d + n_c) 2^-126 (1 + ||x|| + ||w||).
// The total is inflated by 2^-10 to absorb the fp64 evaluation of the bound.
#include "common.h"
#include "exact_dot.h"
#include "gemm.h"
#include "kernels.h"

namespace mosa {

namespace {

// Order-preserving map float -> uint32 (-0.0 is first made +0.0).
__device__ __forceinline__ uint32_t order_key(float f) {
    uint32_t u = __float_as_uint(f);
    if (u == 0x80000000u) u = 0u;
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float f32_down(double x) {
    float f = (float)x;
    if ((double)f > x) f = next_down(f);
    return f;
}
__device__ __forceinline__ float f32_up(double x) {
    float f = (float)x;
    if ((double)f < x) f = next_up(f);
    return f;
}

template <typename ST> __device__ __forceinline__ void split_elem(const ST* p, uint32_t& s, uint32_t& M, int& E);
template <> __device__ __forceinline__ void split_elem<uint16_t>(const uint16_t* p, uint32_t& s, uint32_t& M, int& E) {
    split_bf16(*p, s, M, E);
}
template <> __device__ __forceinline__ void split_elem<float>(const float* p, uint32_t& s, uint32_t& M, int& E) {
    split_f32(__float_as_uint(*p), s, M, E);
}

__device__ __forceinline__ uint64_t lanes_below() {
    return (1ull << (threadIdx.x & 63)) - 1ull;
}

// NW waves per row, EPT tokens per thread (token t = e * 64 NW + tid, so loads
// and stores are coalesced).  Both selections share one packed 32-bit block
// scan per radix pass; the in-order positions come from per-wave, per-stripe
// ballot counts; the uncertain tokens (if any) are re-scored one per wave in
// parallel, their list kept in LDS when short.
constexpr int kSelectLdsUnc = 64;  // uncertain tokens held in LDS (more: the global scratch arrays)

template <int NW>
__device__ __forceinline__ uint32_t block_exclusive_scan_u32(uint32_t v, uint32_t* tmp, uint32_t& total) {
    // inclusive wave scan (DPP), then the wave totals through LDS
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const uint32_t inc = wave_inclusive_scan_u32(v);
    if (lane == 63) tmp[w] = inc;
    __syncthreads();
    uint32_t base = 0, all = 0;
#pragma unroll
    for (int i = 0; i < NW; ++i) {
        const uint32_t t = tmp[i];
        base += i < w ? t : 0u;
        all += t;
    }
    __syncthreads();
    total = all;
    return base + inc - v;
}

template <typename ST, int NW, int EPT>
__global__ __launch_bounds__(64 * NW) void select_rows_kernel(
    const float* __restrict__ z, const float* __restrict__ xnorm, const ST* __restrict__ X,
    const ST* __restrict__ Wr, int T, int d, int H, int k, int first, int32_t* __restrict__ I, float* __restrict__ r,
    int16_t* __restrict__ slot, int32_t* __restrict__ unc_tok, double* __restrict__ unc_key,
    int32_t* __restrict__ unc_sel, int32_t* __restrict__ status) {
    constexpr int NT = 64 * NW;
    static_assert(NT >= 256, "one thread per histogram bin");
    __shared__ uint32_t s_hist[256];   // packed counts: A in bits 0..15, B in 16..31
    __shared__ uint32_t s_tmp[NW];
    __shared__ double s_red[NW];
    __shared__ int s_dig[4];
    __shared__ int s_cnt[NW][EPT];
    __shared__ int s_utok[kSelectLdsUnc];
    __shared__ double s_ukey[kSelectLdsUnc];
    __shared__ int s_usel[kSelectLdsUnc];
    __shared__ int s_flag;
    __shared__ int64_t s_long[NW][kLongDigits];

    const int row = blockIdx.x, b = row / H, h = row % H;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const size_t rowT = (size_t)row * T;
    const float* zr = z + rowT;
    const float* xn = xnorm + (size_t)b * T;
    const ST* w = Wr + (size_t)h * d;

    // All loads first: the logits and ||x|| of this thread's tokens, a share of w.
    float zv[EPT], xv[EPT];
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
        const int tc = min(e * NT + tid, T - 1);
        zv[e] = zr[tc];
        xv[e] = xn[tc];
    }
    double ss = 0.0;
    for (int c = tid; c < d; c += NT) {
        const double v = (double)ld1<ST>(w + c);
        ss += v * v;
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) ss += __shfl_xor(ss, o, 64);
    if (lane == 0) s_red[wave] = ss;
    __syncthreads();
    ss = 0.0;
#pragma unroll
    for (int i = 0; i < NW; ++i) ss += s_red[i];
    const double wn = sqrt(ss) * (1.0 + 0x1p-30);
    const int nc = d / 32;
    const double coef = (96.0 * 0x1p-23 + 1.01 * (double)nc * 0x1p-24) * (1.0 + 0x1p-10);
    const double absterm = (double)(d + nc) * 0x1p-126 * (1.0 + 0x1p-10);

    uint32_t lo[EPT], hi[EPT];
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
        const bool ok = e * NT + tid < T;
        const double x = (double)xv[e];
        const double beta = coef * x * wn + absterm * (1.0 + x + wn);
        lo[e] = ok ? order_key(f32_down((double)zv[e] - beta)) : 0u;  // 0: below every real key
        hi[e] = ok ? order_key(f32_up((double)zv[e] + beta)) : 0u;
    }
    // forced first token: token 0 above every real key, so it is certainly in
    // and the other k - 1 are the best of t >= 1 (r_0 still from its logit)
    if (first && tid == 0) lo[0] = hi[0] = 0xffffffffu;

    // k-th largest lo (A) and (k+1)-th largest hi (B): 8 bits per pass.
    const bool all = k >= T;
    uint32_t A = 0u, Bk = 0u;
    if (!all) {
        uint32_t prefA = 0u, prefB = 0u;
        int remA = k, remB = k + 1;
#pragma unroll
        for (int pass = 0; pass < 4; ++pass) {
            const int shift = 24 - 8 * pass;
            const uint32_t himask = pass == 0 ? 0u : (0xffffffffu << (shift + 8));
            if (tid < 256) s_hist[tid] = 0u;
            __syncthreads();
#pragma unroll
            for (int e = 0; e < EPT; ++e) {
                if (e * NT + tid < T) {
                    if (((lo[e] ^ prefA) & himask) == 0u) atomicAdd(&s_hist[(lo[e] >> shift) & 255u], 1u);
                    if (((hi[e] ^ prefB) & himask) == 0u) atomicAdd(&s_hist[(hi[e] >> shift) & 255u], 1u << 16);
                }
            }
            __syncthreads();
            // thread i looks at bin 255 - i: the exclusive scan in thread order
            // counts the candidates in higher bins (both selections packed)
            const uint32_t cnt = tid < 256 ? s_hist[255 - tid] : 0u;
            uint32_t tot;
            const uint32_t above = block_exclusive_scan_u32<NW>(cnt, s_tmp, tot);
            if (tid < 256) {
                const int ca = (int)(cnt & 0xffffu), cb = (int)(cnt >> 16);
                const int aa = (int)(above & 0xffffu), ab = (int)(above >> 16);
                if (aa < remA && aa + ca >= remA) {
                    s_dig[0] = 255 - tid;
                    s_dig[1] = remA - aa;
                }
                if (ab < remB && ab + cb >= remB) {
                    s_dig[2] = 255 - tid;
                    s_dig[3] = remB - ab;
                }
            }
            __syncthreads();
            prefA |= (uint32_t)s_dig[0] << shift;
            remA = s_dig[1];
            prefB |= (uint32_t)s_dig[2] << shift;
            remB = s_dig[3];
            __syncthreads();  // s_dig and s_hist are rewritten by the next pass
        }
        A = prefA;
        Bk = prefB;
    }

    // Classify; in-order positions of the uncertain tokens from per-wave,
    // per-stripe counts (stripe e holds tokens e NT .. e NT + NT - 1 in thread order).
    uint32_t inm = 0u, uncm = 0u;
    uint64_t ub[EPT];
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
        const bool ok = e * NT + tid < T;
        const bool in = ok && (all || lo[e] > Bk);
        const bool unc = ok && !in && !(hi[e] < A);
        inm |= (uint32_t)in << e;
        uncm |= (uint32_t)unc << e;
        const uint64_t bi = __ballot(in);
        ub[e] = __ballot(unc);
        if (lane == 0) s_cnt[wave][e] = __popcll(bi) | (__popcll(ub[e]) << 16);
    }
    __syncthreads();
    int tot_in = 0, tot_unc = 0, upos[EPT];
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
        int below = 0;
#pragma unroll
        for (int i = 0; i < NW; ++i) {
            const int c = s_cnt[i][e];
            if (i < wave) below += c >> 16;
            tot_in += c & 0xffff;
        }
        upos[e] = tot_unc + below + __popcll(ub[e] & lanes_below());
#pragma unroll
        for (int i = 0; i < NW; ++i) tot_unc += s_cnt[i][e] >> 16;
    }
    __syncthreads();  // s_cnt is reused for the selection counts
    int need = k - tot_in;  // 0 <= need <= tot_unc when the bound holds
    if (need < 0) need = 0;
    if (need > tot_unc) need = tot_unc;
    const bool resolve = need > 0 && need < tot_unc;

    const bool small = tot_unc <= kSelectLdsUnc;
    int* utok = small ? s_utok : unc_tok + rowT;
    double* ukey = small ? s_ukey : unc_key + rowT;
    int* usel = small ? s_usel : unc_sel + rowT;
    if (resolve) {
#pragma unroll
        for (int e = 0; e < EPT; ++e)
            if ((uncm >> e) & 1u) utok[upos[e]] = e * NT + tid;
        __threadfence_block();
        __syncthreads();
        // Second level, one token per wave: the logit in fp64.  Products of
        // two stored values are exact in fp64; any order of the d - 1
        // additions errs by at most (d - 1) u64 sum|x_i w_i| <= that times
        // ||x|| ||w||, and the key RN64(s) is within half an ulp of s.
        for (int u = wave; u < tot_unc; u += NW) {
            const ST* xr = X + ((size_t)b * T + utok[u]) * d;
            double acc = 0.0;
            for (int c0 = 0; c0 < d; c0 += 8 * 64) {
                const int c = min(c0 + 8 * lane, d - 8);
                float xv8[8], wv8[8];
                vec8_to_f32<ST>(vec8_load<ST>(xr + c), xv8);
                vec8_to_f32<ST>(vec8_load<ST>(w + c), wv8);
                if (c0 + 8 * lane < d) {
#pragma unroll
                    for (int j = 0; j < 8; ++j) acc += (double)xv8[j] * (double)wv8[j];
                }
            }
#pragma unroll
            for (int o = 32; o >= 1; o >>= 1) acc += __shfl_xor(acc, o, 64);
            if (lane == 0) ukey[u] = acc;
        }
        if (tid == 0) s_flag = 0;
        __threadfence_block();
        __syncthreads();
        // Decide from the fp64 intervals where they separate.
        for (int u = tid; u < tot_unc; u += NT) {
            const double vu = ukey[u];
            const double bu = 1.01 * (double)d * 0x1p-53 * (double)xn[utok[u]] * wn + fabs(vu) * 0x1p-51;
            int above = 0, maybe = 0;
            for (int v = 0; v < tot_unc; ++v) {
                if (v == u) continue;
                const double vv = ukey[v];
                const double bv = 1.01 * (double)d * 0x1p-53 * (double)xn[utok[v]] * wn + fabs(vv) * 0x1p-51;
                if (vv - bv > vu + bu) ++above;         // certainly above u
                else if (!(vv + bv < vu - bu)) ++maybe;  // order unknown
            }
            int sel = -1;
            if (above + maybe < need) sel = 1;
            else if (above >= need) sel = 0;
            else s_flag = 1;
            usel[u] = sel;
        }
        __threadfence_block();
        __syncthreads();
        if (s_flag) {
            // Exact keys, one token per wave (long accumulator in the wave's LDS digits).
            for (int u0 = 0; u0 < tot_unc; u0 += NW) {
                const int u = u0 + wave;
                if (lane < kLongDigits) s_long[wave][lane] = 0;
                __threadfence_block();
                __builtin_amdgcn_wave_barrier();
                if (u < tot_unc) {
                    const ST* xr = X + ((size_t)b * T + utok[u]) * d;
                    for (int c = lane; c < d; c += 64) {
                        uint32_t sx, Mx, sw, Mw;
                        int Ex, Ew;
                        split_elem<ST>(xr + c, sx, Mx, Ex);
                        split_elem<ST>(w + c, sw, Mw, Ew);
                        const ProductParts p = product_parts(sx, Mx, Ex, sw, Mw, Ew);
                        if (!p.zero) {
#pragma unroll
                            for (int q = 0; q < 3; ++q) {
                                if (p.v[q]) {
                                    const uint64_t add = p.negative ? (uint64_t)(-(int64_t)p.v[q]) : p.v[q];
                                    atomicAdd(reinterpret_cast<unsigned long long*>(&s_long[wave][p.j + q]),
                                              (unsigned long long)add);
                                }
                            }
                        }
                    }
                }
                __threadfence_block();
                __builtin_amdgcn_wave_barrier();
                if (u < tot_unc && lane == 0) ukey[u] = long_accumulator_round(&s_long[wave][0]);
                __threadfence_block();
                __builtin_amdgcn_wave_barrier();
            }
            __threadfence_block();
            __syncthreads();
            // exact rank among the uncertain tokens (key desc, index asc)
            for (int u = tid; u < tot_unc; u += NT) {
                const double ku = ukey[u];
                const int tu = utok[u];
                int rank = 0;
                for (int v = 0; v < tot_unc; ++v) {
                    const double kv = ukey[v];
                    const int tv = utok[v];
                    rank += (kv > ku) || (kv == ku && tv < tu);
                }
                usel[u] = rank < need;
            }
            __threadfence_block();
            __syncthreads();
        }
    }

    // Compact the chosen tokens in index order: I ascending, r, and the slot map.
    uint32_t selm = inm;
#pragma unroll
    for (int e = 0; e < EPT; ++e)
        if ((uncm >> e) & 1u)
            if (resolve ? (usel[upos[e]] > 0) : (need == tot_unc)) selm |= 1u << e;
    uint64_t sb[EPT];
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
        sb[e] = __ballot((selm >> e) & 1u);
        if (lane == 0) s_cnt[wave][e] = __popcll(sb[e]);
    }
    __syncthreads();
    int pos0 = 0;
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
        int below = 0, stripe = 0;
#pragma unroll
        for (int i = 0; i < NW; ++i) {
            const int c = s_cnt[i][e];
            if (i < wave) below += c;
            stripe += c;
        }
        const int t = e * NT + tid;
        const int pos = pos0 + below + __popcll(sb[e] & lanes_below());
        int16_t sl = -1;
        if (((selm >> e) & 1u) && pos < k) {
            I[(size_t)row * k + pos] = t;
            r[(size_t)row * k + pos] = 1.0f / (1.0f + expf(-zv[e]));
            sl = (int16_t)pos;
        }
        if (t < T) slot[rowT + t] = sl;
        pos0 += stripe;
    }
    // Exactly k tokens unless the logit error bound was violated.  Then the
    // row is flagged for the caller, and every slot is kept defined (token 0,
    // r = 0) so that the kernels downstream stay in bounds.
    if (tid == 0) status[row] = pos0 == k ? 0 : 1;
    for (int pos = pos0 + tid; pos < k; pos += NT) {
        I[(size_t)row * k + pos] = 0;
        r[(size_t)row * k + pos] = 0.f;
    }
}

template <typename ST>
int launch_select_t(const float* z, const float* xnorm, const ST* X, const ST* Wr, int B, int T, int d, int H,
                    int k, int first, int32_t* I, float* r, int16_t* slot, int32_t* unc_tok, double* unc_key,
                    int32_t* unc_sel, int32_t* status, hipStream_t stream) {
    const dim3 grid(B * H);
#define MOSA_SELECT_ROWS(NW, E)                                                                                \
    hipLaunchKernelGGL((select_rows_kernel<ST, NW, E>), grid, dim3(64 * NW), 0, stream, z, xnorm, X, Wr, T, d, H, \
                       k, first, I, r, slot, unc_tok, unc_key, unc_sel, status)
    if (T <= 256) MOSA_SELECT_ROWS(4, 1);
    else if (T <= 512) MOSA_SELECT_ROWS(4, 2);
    // many rows: the chip is full with smaller workgroups, and 4 waves pass
    // the per-row barriers faster than 8
    else if (T <= 1024 && B * H >= 1024) MOSA_SELECT_ROWS(4, 4);
    else if (T <= 1024) MOSA_SELECT_ROWS(8, 2);
    else if (T <= 2048) MOSA_SELECT_ROWS(4, 8);
    else if (T <= 8192) MOSA_SELECT_ROWS(16, 8);
    else if (T <= 16384) MOSA_SELECT_ROWS(16, 16);
    else return -1;
#undef MOSA_SELECT_ROWS
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

// Fixed sparse attention (paper Section 3.1, as a special case of MoSA):
// I = 0, stride, 2 stride, ..., r = 1; one workgroup per (b, h) row.
__global__ __launch_bounds__(256) void fixed_select_kernel(int T, int k, int stride, int32_t* __restrict__ I,
                                                           float* __restrict__ r, int16_t* __restrict__ slot,
                                                           int32_t* __restrict__ status) {
    const size_t row = blockIdx.x;
    if (threadIdx.x == 0) status[row] = 0;
    for (int i = threadIdx.x; i < k; i += 256) {
        I[row * k + i] = i * stride;
        r[row * k + i] = 1.0f;
    }
    for (int t = threadIdx.x; t < T; t += 256)
        slot[row * T + t] = (t % stride == 0 && t / stride < k) ? (int16_t)(t / stride) : (int16_t)-1;
}

}  // namespace

int launch_fixed_select(int B, int T, int H, int k, int stride, int32_t* I, float* r, int16_t* slot,
                        int32_t* status, hipStream_t stream) {
    if (B * H == 0) return 0;
    if (stride < 1 || (long long)(k - 1) * stride > T - 1) return -1;
    hipLaunchKernelGGL(fixed_select_kernel, dim3(B * H), dim3(256), 0, stream, T, k, stride, I, r, slot, status);
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

int launch_select(int dtype, const float* z, const float* xnorm, const void* X, const void* Wr, int B, int T,
                  int d, int H, int k, int first_token, int32_t* I, float* r, int16_t* slot, int32_t* unc_tok,
                  double* unc_key, int32_t* unc_sel, int32_t* status, hipStream_t stream) {
    if (dtype == kBF16)
        return launch_select_t<uint16_t>(z, xnorm, (const uint16_t*)X, (const uint16_t*)Wr, B, T, d, H, k,
                                         first_token, I, r, slot, unc_tok, unc_key, unc_sel, status, stream);
    return launch_select_t<float>(z, xnorm, (const float*)X, (const float*)Wr, B, T, d, H, k, first_token, I, r,
                                  slot, unc_tok, unc_key, unc_sel, status, stream);
}

}  // namespace mosa
