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
//   1. locate tau, the (k+1)-th largest z~, to within 1024 consecutive
//      order-preserving uint32 keys (2 radix passes of 11 bits over keys held
//      in registers; LDS histograms).  With b the largest beta_t of the row,
//      A = (lower end - b) rounded down is at most the k-th largest lo, and
//      B = (upper end + b) rounded up at least the (k+1)-th largest hi;
//   2. hi_t < A  => at least k tokens certainly beat t: t is out;
//      lo_t > B  => at most k-1 tokens can beat t: t is in;
//      the rest (typically the (k+1)-th token alone) is uncertain;
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

constexpr int kBins = 2048;  // radix histogram bins (11-bit digits)

// LDS word of radix bin b: descending position p = kBins - 1 - b, lane
// p / 32 of the scanning wave, entry j = p % 32 of that lane at word
// 256 (j / 4) + 4 (p / 32) + j % 4, so that the wave's 16-byte reads of its
// 32 entries each cover 1 KB without bank conflicts.
__device__ __forceinline__ int bin_slot(uint32_t b) {
    const int p = kBins - 1 - (int)b, l = p >> 5, j = p & 31;
    return 256 * (j >> 2) + 4 * l + (j & 3);
}

// Inverse of order_key.
__device__ __forceinline__ float key_float(uint32_t k) {
    return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
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
// and stores are coalesced).  One histogram per radix pass, scanned by
// wave 0; the in-order positions come
// from per-wave, per-stripe ballot counts; the uncertain tokens (if any) are
// re-scored one per wave in parallel, their list kept in LDS when short.
constexpr int kSelectLdsUnc = 64;  // uncertain tokens held in LDS (more: the global scratch arrays)

template <typename ST, int NW, int EPT>
__global__ __launch_bounds__(64 * NW) void select_rows_kernel(
    const float* __restrict__ z, const float* __restrict__ xnorm, const ST* __restrict__ X,
    const ST* __restrict__ Wr, int T, int d, int H, int k, int first, int32_t* __restrict__ I, float* __restrict__ r,
    int16_t* __restrict__ slot, int32_t* __restrict__ unc_tok, double* __restrict__ unc_key,
    int32_t* __restrict__ unc_sel, int32_t* __restrict__ status) {
    constexpr int NT = 64 * NW;
    __shared__ __attribute__((aligned(16))) uint32_t s_hist[2][kBins];  // one per pass
    __shared__ double s_red[NW];
    __shared__ int s_dig[2][2];
    __shared__ float s_xmax[NW];
    __shared__ int s_cnt[NW][EPT];
    __shared__ int s_cnt2[NW][EPT];
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
    // The radix select runs on the order keys of z~ itself; lo and hi
    // (z~ -+ beta_t, rounded outwards) classify the tokens afterwards, once
    // ||w|| is known, so the loads of w and ||x|| overlap the radix passes.
    uint32_t key[EPT];
#pragma unroll
    for (int e = 0; e < EPT; ++e) key[e] = e * NT + tid < T ? order_key(zv[e]) : 0u;
    // forced first token: token 0 above every real key, so it is certainly in
    // and the other k - 1 are the best of t >= 1 (r_0 still from its logit)
    if (first && tid == 0) key[0] = 0xffffffffu;
    for (int i = tid; i < kBins; i += NT) s_hist[0][i] = 0u;  // the first pass's histogram
    __syncthreads();
    // per-wave ||w||^2 and largest ||x_t|| bound (every xv is a real token's),
    // published before the first barrier that follows
    auto publish_norms = [&]() {
        float xm = xv[0];
#pragma unroll
        for (int e = 1; e < EPT; ++e) xm = fmaxf(xm, xv[e]);
        ss = wave_sum_f64(ss);
        xm = wave_max_nonneg_f32(xm);
        if (lane == 0) {
            s_red[wave] = ss;
            s_xmax[wave] = xm;
        }
    };

    // tau = the (k+1)-th largest z~, located by two radix passes over the
    // top 22 bits of the keys (11 bits each) to within the 1024 keys
    // [pref, pref + 1023].  With tlo <= tau <= thi the ends of that range,
    //   A = down(tlo - bmax) <= the k-th largest lo: the k + 1 tokens with
    //       z~ >= tau all have lo >= A;
    //   B = up(thi + bmax) >= the (k+1)-th largest hi: a token with hi > B has
    //       z~ > tau, and at most k tokens do;
    // so "lo > B: in" and "hi < A: out" below are sound.  The range widens
    // the uncertain band by at most 1023 units in the last place of tau.
    const bool all = k >= T;
    uint32_t pref = 0u;
    if (!all) {
        int rem = k + 1;
        // Two barriers per pass: the histograms alternate between two
        // buffers, so the second is cleared while wave 0 scans the first.
#pragma unroll
        for (int pass = 0; pass < 2; ++pass) {
            const int shift = 21 - 11 * pass;
            const uint32_t himask = pass == 0 ? 0u : 0xffe00000u;
            uint32_t* hist = s_hist[pass];
#pragma unroll
            for (int e = 0; e < EPT; ++e)
                if (e * NT + tid < T && ((key[e] ^ pref) & himask) == 0u)
                    atomicAdd(&hist[bin_slot((key[e] >> shift) & (kBins - 1))], 1u);
            if (pass == 0) publish_norms();
            __syncthreads();  // this pass's histogram is complete
            if (wave == 0) {
                // lane l's 32 bins (descending positions 32 l .. 32 l + 31)
                // in 8 conflict-free 16-byte reads; the lane whose range holds
                // the rem-th candidate from the top, then within its range the
                // bin, each found by a scan and a ballot
                const uint4* hv = reinterpret_cast<const uint4*>(hist);
                uint32_t csum = 0u;
#pragma unroll
                for (int q = 0; q < 8; ++q) {
                    const uint4 v = hv[64 * q + lane];
                    csum += v.x + v.y + v.z + v.w;
                }
                const uint32_t incl = wave_inclusive_scan_u32(csum), excl = incl - csum;
                // (one lane qualifies: rem never exceeds the candidates counted)
                const uint64_t mL = __ballot(excl < (uint32_t)rem && incl >= (uint32_t)rem);
                const int L = mL ? __builtin_ctzll(mL) : 0;
                const uint32_t exL = __builtin_amdgcn_readlane(excl, L);
                const uint32_t c = lane < 32 ? hist[256 * (lane >> 2) + 4 * L + (lane & 3)] : 0u;
                const uint32_t ci = wave_inclusive_scan_u32(c) + exL;
                const uint64_t mj = __ballot(lane < 32 && ci - c < (uint32_t)rem && ci >= (uint32_t)rem);
                if (mj && lane == __builtin_ctzll(mj)) {
                    s_dig[pass][0] = kBins - 1 - (32 * L + lane);
                    s_dig[pass][1] = rem - (int)(ci - c);
                }
            }
            if (pass == 0 && wave == (NW > 1 ? 1 : 0)) {
                uint4* hz = reinterpret_cast<uint4*>(s_hist[1]);
                for (int i = lane; i < kBins / 4; i += 64) hz[i] = make_uint4(0u, 0u, 0u, 0u);
            }
            __syncthreads();  // digit found, second histogram cleared
            pref |= (uint32_t)s_dig[pass][0] << shift;
            rem = s_dig[pass][1];
        }
    } else {
        publish_norms();
        __syncthreads();
    }

    double wss = 0.0;
    float xm = 0.f;
#pragma unroll
    for (int i = 0; i < NW; ++i) {
        wss += s_red[i];
        xm = fmaxf(xm, s_xmax[i]);
    }
    const double wn = sqrt(wss) * (1.0 + 0x1p-30);
    const int nc = d / 32;
    const double coef = (96.0 * 0x1p-23 + 1.01 * (double)nc * 0x1p-24) * (1.0 + 0x1p-10);
    const double absterm = (double)(d + nc) * 0x1p-126 * (1.0 + 0x1p-10);
    // beta grows with ||x||, and so does its fp64 evaluation: bmax >= every beta_t
    const double bmax = coef * (double)xm * wn + absterm * (1.0 + (double)xm + wn);
    uint32_t lo[EPT], hi[EPT];
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
        const bool ok = e * NT + tid < T;
        const double x = (double)xv[e];
        const double beta = coef * x * wn + absterm * (1.0 + x + wn);
        lo[e] = ok ? order_key(f32_down((double)zv[e] - beta)) : 0u;  // 0: below every real key
        hi[e] = ok ? order_key(f32_up((double)zv[e] + beta)) : 0u;
    }
    if (first && tid == 0) lo[0] = hi[0] = 0xffffffffu;
    uint32_t A = 0u, Bk = 0u;
    if (!all) {
        const float tlo = key_float(pref), thi = key_float(pref | 0x3ffu);
        // ends that are not finite numbers give no bound (A = 0: nothing is
        // out, B = max: nothing but a forced token is in)
        A = isfinite(tlo) ? order_key(f32_down((double)tlo - bmax)) : 0u;
        Bk = isfinite(thi) ? order_key(f32_up((double)thi + bmax)) : 0xffffffffu;
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
            acc = wave_sum_f64(acc);
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
        if (lane == 0) s_cnt2[wave][e] = __popcll(sb[e]);
    }
    __syncthreads();
    int pos0 = 0;
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
        int below = 0, stripe = 0;
#pragma unroll
        for (int i = 0; i < NW; ++i) {
            const int c = s_cnt2[i][e];
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

// One wave per (b, h) row for T <= 64 EPL (EPL tokens per lane at t = 64 e +
// lane): the same certified selection as select_rows_kernel without an LDS
// histogram or a workgroup barrier.  tau, the (k+1)-th largest key, is
// located to within 1024 keys as there, here by a binary search over its top
// 22 bits (each step counts the keys at or above a candidate: one compare per
// key and a wave sum).  Most tokens are classified by one compare of their
// key against row-wide thresholds; counts and in-order positions come from
// wave sums and ballots.  The uncertain tokens are re-scored as there, one
// token at a time by the whole wave (fp64, then the long accumulator where
// the fp64 intervals overlap).  The waves of a workgroup take independent
// rows and never wait for each other.
constexpr int kSelectWaveRows = 4;  // rows (waves) per workgroup

template <typename ST, int EPL>
__global__ __launch_bounds__(64 * kSelectWaveRows) void select_wave_kernel(
    const float* __restrict__ z, const float* __restrict__ xnorm, const ST* __restrict__ X,
    const ST* __restrict__ Wr, int rows, int T, int d, int H, int k, int first, int32_t* __restrict__ I,
    float* __restrict__ r, int16_t* __restrict__ slot, int32_t* __restrict__ unc_tok, double* __restrict__ unc_key,
    int32_t* __restrict__ unc_sel, int32_t* __restrict__ status) {
    __shared__ int s_utok[kSelectWaveRows][kSelectLdsUnc];
    __shared__ double s_ukey[kSelectWaveRows][kSelectLdsUnc];
    __shared__ int s_usel[kSelectWaveRows][kSelectLdsUnc];
    __shared__ int64_t s_long[kSelectWaveRows][kLongDigits];
    static_assert(EPL >= 1 && EPL <= 32 && kLongDigits <= 64, "shape");

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int row = blockIdx.x * kSelectWaveRows + wave;
    if (row >= rows) return;  // the whole wave; no other wave waits for it
    const int b = row / H, h = row % H;
    const size_t rowT = (size_t)row * T;
    const float* zr = z + rowT;
    const float* xn = xnorm + (size_t)b * T;
    const ST* w = Wr + (size_t)h * d;

    // All loads first: the logits and ||x|| of this lane's tokens, a share of w.
    float zv[EPL], xv[EPL];
#pragma unroll
    for (int e = 0; e < EPL; ++e) {
        const int tc = min(64 * e + lane, T - 1);
        zv[e] = zr[tc];
        xv[e] = xn[tc];
    }
    double ss = 0.0;
    for (int c = 8 * lane; c < d; c += 8 * 64) {  // d is a multiple of 64
        float wv8[8];
        vec8_to_f32<ST>(vec8_load<ST>(w + c), wv8);
#pragma unroll
        for (int j = 0; j < 8; ++j) ss += (double)wv8[j] * (double)wv8[j];
    }
    const bool all = k >= T;
    uint32_t key[EPL];
#pragma unroll
    for (int e = 0; e < EPL; ++e) key[e] = 64 * e + lane < T ? order_key(zv[e]) : 0u;  // 0: below every real key
    // forced first token: above every real key (see select_rows_kernel)
    if (first && lane == 0) key[0] = 0xffffffffu;

    // tau, the largest key v with at least k + 1 keys >= v, to within 1024
    // consecutive keys: its top 22 bits, bit by bit (a compare per key and a
    // wave sum per bit); tlo <= tau <= thi are the ends of that range
    uint32_t pref = 0u;
    if (!all) {
        for (int bit = 31; bit >= 10; --bit) {
            const uint32_t cand = pref | (1u << bit);
            uint32_t c = 0u;
#pragma unroll
            for (int e = 0; e < EPL; ++e) c += key[e] >= cand ? 1u : 0u;
            if (wave_sum_u32(c) >= (uint32_t)(k + 1)) pref = cand;
        }
    }

    // ||w|| and the largest ||x_t|| (every xv is a real token's); the bound,
    // A and B as in select_rows_kernel
    ss = wave_sum_f64(ss);
    float xm = xv[0];
#pragma unroll
    for (int e = 1; e < EPL; ++e) xm = fmaxf(xm, xv[e]);
    xm = wave_max_nonneg_f32(xm);
    const double wn = sqrt(ss) * (1.0 + 0x1p-30);
    const int nc = d / 32;
    const double coef = (96.0 * 0x1p-23 + 1.01 * (double)nc * 0x1p-24) * (1.0 + 0x1p-10);
    const double absterm = (double)(d + nc) * 0x1p-126 * (1.0 + 0x1p-10);
    const double bmax = coef * (double)xm * wn + absterm * (1.0 + (double)xm + wn);
    uint32_t A = 0u, Bk = 0u;
    if (!all) {
        const float tlo = key_float(pref), thi = key_float(pref | 0x3ffu);
        A = isfinite(tlo) ? order_key(f32_down((double)tlo - bmax)) : 0u;
        Bk = isfinite(thi) ? order_key(f32_up((double)thi + bmax)) : 0xffffffffu;
    }

    // Classify: in (lo > B), out (hi < A) or uncertain.  Most tokens are
    // decided by one key compare against the row's thresholds with bmax in
    // place of their own beta: z~ <= Lo (the float below next_down(A) - bmax,
    // one float lower for the fp64 rounding of the difference) gives
    // hi <= next_down(A) < A, and z~ >= Hi (likewise above next_up(B) +
    // bmax) gives lo >= next_up(B) > B.  The others (and a forced token)
    // take the per-token bounds.
    uint32_t lo_key = 0u, hi_key = 0xffffffffu;
    bool lo_ok = false, hi_ok = false;
    if (!all) {
        const float af = key_float(A), bf = key_float(Bk);
        if (A != 0u && isfinite(af)) {
            const float lf = next_down(f32_down((double)next_down(af) - bmax));
            lo_ok = isfinite(lf);
            lo_key = order_key(lf);
        }
        if (Bk != 0xffffffffu && isfinite(bf)) {
            const float hf = next_up(f32_up((double)next_up(bf) + bmax));
            hi_ok = isfinite(hf);
            hi_key = order_key(hf);
        }
    }
    uint32_t inm = 0u, uncm = 0u, bandm = 0u;
#pragma unroll
    for (int e = 0; e < EPL; ++e) {
        const bool ok = 64 * e + lane < T;
        const bool forced = first && lane == 0 && e == 0;
        const bool fin = ok && !forced && (all || (hi_ok && key[e] >= hi_key));
        const bool fout = ok && !forced && !all && lo_ok && key[e] <= lo_key;
        inm |= (uint32_t)fin << e;
        bandm |= (uint32_t)(ok && !fin && !fout) << e;
    }
    if (__ballot(bandm != 0u)) {
#pragma unroll
        for (int e = 0; e < EPL; ++e) {
            if ((bandm >> e) & 1u) {
                const double x = (double)xv[e];
                const double beta = coef * x * wn + absterm * (1.0 + x + wn);
                uint32_t lo = order_key(f32_down((double)zv[e] - beta));
                uint32_t hi = order_key(f32_up((double)zv[e] + beta));
                if (first && lane == 0 && e == 0) lo = hi = 0xffffffffu;
                const bool in = all || lo > Bk;
                inm |= (uint32_t)in << e;
                uncm |= (uint32_t)(!in && !(hi < A)) << e;
            }
        }
    }
    const int tot_in = (int)wave_sum_u32((uint32_t)__popc(inm));
    const int tot_unc = (int)wave_sum_u32((uint32_t)__popc(uncm));
    int need = k - tot_in;  // 0 <= need <= tot_unc when the bound holds
    if (need < 0) need = 0;
    if (need > tot_unc) need = tot_unc;
    const bool resolve = need > 0 && need < tot_unc;

    const bool small = tot_unc <= kSelectLdsUnc;
    int* utok = small ? s_utok[wave] : unc_tok + rowT;
    double* ukey = small ? s_ukey[wave] : unc_key + rowT;
    int* usel = small ? s_usel[wave] : unc_sel + rowT;
    if (resolve) {
        // the uncertain tokens in index order
        int base = 0;
#pragma unroll
        for (int e = 0; e < EPL; ++e) {
            const uint64_t ub = __ballot((uncm >> e) & 1u);
            if ((uncm >> e) & 1u) utok[base + __popcll(ub & lanes_below())] = 64 * e + lane;
            base += __popcll(ub);
        }
        __threadfence_block();
        __builtin_amdgcn_wave_barrier();
        // their logits in fp64 (bound as in select_rows_kernel)
        for (int u = 0; u < tot_unc; ++u) {
            const ST* xr = X + ((size_t)b * T + utok[u]) * d;
            double acc = 0.0;
            for (int c = 8 * lane; c < d; c += 8 * 64) {
                float xv8[8], wv8[8];
                vec8_to_f32<ST>(vec8_load<ST>(xr + c), xv8);
                vec8_to_f32<ST>(vec8_load<ST>(w + c), wv8);
#pragma unroll
                for (int j = 0; j < 8; ++j) acc += (double)xv8[j] * (double)wv8[j];
            }
            acc = wave_sum_f64(acc);
            if (lane == 0) ukey[u] = acc;
        }
        __threadfence_block();
        __builtin_amdgcn_wave_barrier();
        // decide from the fp64 intervals where they separate
        bool unknown = false;
        for (int u = lane; u < tot_unc; u += 64) {
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
            else unknown = true;
            usel[u] = sel;
        }
        const bool exact = __ballot(unknown) != 0ull;
        __threadfence_block();
        __builtin_amdgcn_wave_barrier();
        if (exact) {
            // exact keys, one token at a time (long accumulator in the wave's LDS digits)
            for (int u = 0; u < tot_unc; ++u) {
                if (lane < kLongDigits) s_long[wave][lane] = 0;
                __threadfence_block();
                __builtin_amdgcn_wave_barrier();
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
                __threadfence_block();
                __builtin_amdgcn_wave_barrier();
                if (lane == 0) ukey[u] = long_accumulator_round(&s_long[wave][0]);
                __threadfence_block();
                __builtin_amdgcn_wave_barrier();
            }
            // exact rank among the uncertain tokens (key desc, index asc)
            for (int u = lane; u < tot_unc; u += 64) {
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
            __builtin_amdgcn_wave_barrier();
        }
    }

    // Compact the chosen tokens in index order: I ascending, r, and the slot map.
    uint32_t selm = inm;
    if (!resolve) {
        if (need == tot_unc) selm |= uncm;
    } else {
        int base = 0;
#pragma unroll
        for (int e = 0; e < EPL; ++e) {
            const bool unc = (uncm >> e) & 1u;
            const uint64_t ub = __ballot(unc);
            if (unc && usel[base + __popcll(ub & lanes_below())] > 0) selm |= 1u << e;
            base += __popcll(ub);
        }
    }
    int pos0 = 0;
#pragma unroll
    for (int e = 0; e < EPL; ++e) {
        const bool sel = (selm >> e) & 1u;
        const uint64_t sb = __ballot(sel);
        const int t = 64 * e + lane;
        const int pos = pos0 + __popcll(sb & lanes_below());
        int16_t sl = -1;
        if (sel && pos < k) {
            I[(size_t)row * k + pos] = t;
            r[(size_t)row * k + pos] = 1.0f / (1.0f + expf(-zv[e]));
            sl = (int16_t)pos;
        }
        if (t < T) slot[rowT + t] = sl;
        pos0 += __popcll(sb);
    }
    // exactly k tokens unless the logit error bound was violated (then as in
    // select_rows_kernel: the row is flagged and every slot kept defined)
    if (lane == 0) status[row] = pos0 == k ? 0 : 1;
    for (int pos = pos0 + lane; pos < k; pos += 64) {
        I[(size_t)row * k + pos] = 0;
        r[(size_t)row * k + pos] = 0.f;
    }
}

template <typename ST>
int launch_select_t(const float* z, const float* xnorm, const ST* X, const ST* Wr, int B, int T, int d, int H,
                    int k, int first, int32_t* I, float* r, int16_t* slot, int32_t* unc_tok, double* unc_key,
                    int32_t* unc_sel, int32_t* status, hipStream_t stream) {
    if (T <= 1024 && B * H >= 2048) {
        // one wave per row where the rows give every SIMD two waves: each row
        // then takes longer than with the workgroup kernel (one wave does all
        // of its steps), but the launch as a whole does not, and it holds a
        // quarter of the LDS, which leaves more room to the dense QKV GEMM
        // beside it (hybrid_d1024's 2048 rows: the two-stream step 0.400 ->
        // 0.398 ms cold; with 256 or 512 rows it is slower, 11 -> 22 and 13
        // -> 25 us)
        const int rows = B * H;
        const dim3 g((rows + kSelectWaveRows - 1) / kSelectWaveRows), blk(64 * kSelectWaveRows);
#define MOSA_SELECT_WAVE(E)                                                                                    \
    hipLaunchKernelGGL((select_wave_kernel<ST, E>), g, blk, 0, stream, z, xnorm, X, Wr, rows, T, d, H, k, first, I, \
                       r, slot, unc_tok, unc_key, unc_sel, status)
        if (T <= 256) MOSA_SELECT_WAVE(4);
        else if (T <= 512) MOSA_SELECT_WAVE(8);
        else MOSA_SELECT_WAVE(16);
#undef MOSA_SELECT_WAVE
        return hipGetLastError() == hipSuccess ? 0 : -1;
    }
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
