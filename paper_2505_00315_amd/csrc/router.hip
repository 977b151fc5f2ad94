// Router logits z = X W^r^T for every MoSA head (paper Section 2.2: the
// router of head h is a vector W^r_h in R^d and scores token t by X_t . W^r_h;
// sigma is applied where the score is used).
//
// One workgroup (4 waves) owns 32 consecutive tokens of the flattened [B*T]
// token axis and up to 256 heads.  X is read from HBM once; W^r (H x d) is
// small and served from L2.  The contraction runs on MFMA
// (v_mfma_f32_16x16x32_bf16, or 16x16x4_f32 for fp32 storage) in K chunks of
// 32.  Each chunk starts from a zero accumulator and is added to the running
// fp32 sum with one VALU add: the error of the result then has the bound
// that the top-k certification relies on (see select.hip):
//   |z~ - s| <= (96 u32 + 1.01 n_c u) ||x|| ||w|| + small absolute term,
// with u = 2^-24, u32 = 2^-23 and n_c = d / 32 chunks.
//
// The kernel also writes an upper bound of ||x_t||_2 for every token
// (fp64 sum of squares, rounded up to fp32) used by that error bound.
#include "common.h"
#include "gemm2.h"
#include "kernels.h"

namespace mosa {

namespace {

constexpr int kRouterTokens = 32;
constexpr int kRouterHeads = 256;  // heads per workgroup (grid.y covers more)

// Round a non-negative double up to float.
__device__ __forceinline__ float f32_round_up(double x) {
    float f = (float)x;
    if ((double)f < x) f = next_up(f);
    return f;
}

template <typename ST>
__global__ __launch_bounds__(256) void router_kernel(const ST* __restrict__ X, const ST* __restrict__ Wr,
                                                     int BT, int T, int d, int H,
                                                     float* __restrict__ z, float* __restrict__ xnorm) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int g = lane >> 4, c16 = lane & 15;
    const int tok0 = blockIdx.x * kRouterTokens;
    const int h0 = blockIdx.y * kRouterHeads;
    const int nhb = min(16, (H - h0 + 15) / 16);  // head blocks of 16 in this workgroup

    // wave -> token block tb (16 tokens) and every other head block
    const int tb = wave & 1;
    const int tok = tok0 + tb * 16 + c16;  // token whose row this lane feeds as B
    const bool tok_ok = tok < BT;
    const ST* xrow = X + (size_t)(tok_ok ? tok : 0) * d;

    f32x4 acc[8];
#pragma unroll
    for (int m = 0; m < 8; ++m) acc[m] = zero4();

    // ||x_t||^2 in fp64 from the same fragments (waves 0 and 1 of the first
    // head group see every token of the workgroup exactly once).
    const bool do_norm = blockIdx.y == 0 && (wave >> 1) == 0;
    double ss = 0.0;
    // Groups of U chunks: all loads of a group are issued before its MFMAs;
    // out-of-range rows and chunks load a clamped address and are zeroed.
    constexpr int U = 8;
    for (int kc0 = 0; kc0 < d; kc0 += 32 * U) {
        Frag8<ST> bx[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int kc = min(kc0 + 32 * u, d - 32);
            const Frag8<ST> v = frag8_load<ST>(xrow + kc + 8 * g);
            bx[u] = (tok_ok && kc0 + 32 * u < d) ? v : frag8_zero<ST>();
        }
        if (do_norm) {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                float x[8];
                frag8_to_f32<ST>(bx[u], x);
#pragma unroll
                for (int j = 0; j < 8; ++j) ss += (double)x[j] * (double)x[j];
            }
        }
#pragma unroll
        for (int m = 0; m < 8; ++m) {
            const int hb = (wave >> 1) + 2 * m;
            if (hb < nhb) {
                const int h = h0 + hb * 16 + c16;
                const ST* wrow = Wr + (size_t)min(h, H - 1) * d;
                Frag8<ST> aw[U];
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    const int kc = min(kc0 + 32 * u, d - 32);
                    const Frag8<ST> v = frag8_load<ST>(wrow + kc + 8 * g);
                    aw[u] = (h < H && kc0 + 32 * u < d) ? v : frag8_zero<ST>();
                }
                // every chunk starts from zero and is added with one fp32 add
#pragma unroll
                for (int u = 0; u < U; ++u) {
                    f32x4 part = zero4();
                    mma8(part, aw[u], bx[u]);
                    acc[m] += part;
                }
            }
        }
    }
    // D[head][token]: lane holds token column c16, head rows 4g + i.
    if (tok_ok) {
        const int b = tok / T, t = tok % T;
#pragma unroll
        for (int m = 0; m < 8; ++m) {
            const int hb = (wave >> 1) + 2 * m;
            if (hb < nhb) {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int h = h0 + hb * 16 + 4 * g + i;
                    if (h < H) z[((size_t)b * H + h) * T + t] = acc[m][i];
                }
            }
        }
    }

    // ||x_t||_2 upper bound (lanes g = 0..3 hold disjoint quarters of the row)
    if (do_norm) {
        ss += __shfl_xor(ss, 16, 64);
        ss += __shfl_xor(ss, 32, 64);
        if (g == 0 && tok_ok) {
            // fp64 rounding of <= d squares and the sqrt: far below 2^-30 relative.
            xnorm[tok] = f32_round_up(sqrt(ss) * (1.0 + 0x1p-30));
        }
    }
}

// bf16: the same contraction on the multi-stage engine (gemm2.h), MT tokens x
// NT heads per workgroup with both operands staged through LDS, so that each
// W^r row is fetched once per workgroup rather than once per wave.  Every
// 32-k MFMA starts from zero and is added to the running sum (CHUNK_ADD): the
// same summation, and the same error bound, as router_kernel.  The workgroups
// of the first head tile also write the ||x_t|| bounds of their tokens,
// summed from the X tiles in LDS as they pass.
template <int MT_, int NT_>
struct RouterPolicy2 {
    using ST = uint16_t;
    static constexpr int MT = MT_, NT = NT_, KC = 64, WM = 2, WN = 2, STAGES = MT * NT >= 64 * 128 ? 3 : 4;
    static constexpr size_t EPI_LDS = 0;
    static constexpr bool A_KCONTIG = true, B_KCONTIG = true, CHUNK_ADD = true;
    struct Args {
        const ST* X;   // [BT, d]
        const ST* Wr;  // [H, d]
        float* z;      // [B, H, T]
        float* xnorm;  // [BT]
        int BT, T, d, H, ntiles;
    };
    struct ARef {
        const ST* p;
    };
    struct BRef {
        const ST* p;
    };
    // the head tiles of one token tile are consecutive (one XCD, X from its L2)
    __device__ static void tile(const Args& a, int logical, int& batch, int& m0, int& n0) {
        batch = 0;
        m0 = (logical / a.ntiles) * MT;
        n0 = (logical % a.ntiles) * NT;
    }
    __device__ static int k_size(const Args& a, int) { return a.d; }
    __device__ static ARef a_row(const Args& a, int, int m) { return {a.X + (size_t)min(m, a.BT - 1) * a.d}; }
    __device__ static const ST* a_elem(const Args&, int, const ARef& r, int k) { return r.p + k; }
    __device__ static BRef b_row(const Args& a, int, int n) { return {a.Wr + (size_t)min(n, a.H - 1) * a.d}; }
    __device__ static const ST* b_elem(const Args&, int, const BRef& r, int k) { return r.p + k; }
    // ||x_t||_2 bounds, by the workgroups of the first head tile, from the
    // X rows of every k chunk while they are in LDS: TPR threads per token,
    // each summing the squares of UPT 16-byte units (fp64, exact products)
    static constexpr int TPR = 256 / MT, UPT = (KC / 8) / TPR;
    static_assert(TPR * MT == 256 && UPT * TPR == KC / 8 && (TPR & (TPR - 1)) == 0, "norm threads");
    __device__ static void a_tile_hook(const Args&, int, int n0, const unsigned char* ta, int tid, double& ss) {
        if (n0 != 0) return;
        const int r = tid / TPR, u0 = (tid % TPR) * UPT;
#pragma unroll
        for (int i = 0; i < UPT; ++i) {
            const int u = u0 + i;
            const uint4 v = *reinterpret_cast<const uint4*>(ta + (r * (KC / 8) + (u ^ kswz(r, KC / 8))) * 16);
            float x[8];
            vec8_to_f32<ST>(Vec8<ST>{v}, x);
#pragma unroll
            for (int e = 0; e < 8; ++e) ss += (double)x[e] * (double)x[e];
        }
    }
    __device__ static void a_hook_done(const Args& a, int m0, int n0, int tid, double ss) {
        if (n0 != 0) return;
#pragma unroll
        for (int o = 1; o < TPR; o <<= 1) ss += __shfl_xor(ss, o, 64);
        const int tok = m0 + tid / TPR;
        // fp64 rounding of <= d squares and the sqrt: far below 2^-30 relative
        if (tid % TPR == 0 && tok < a.BT) a.xnorm[tok] = f32_round_up(sqrt(ss) * (1.0 + 0x1p-30));
    }
    __device__ static void epilogue(const Args& a, int, int m0, int n0, const float* Cs, int ldc, int tid,
                                    unsigned char*) {
        for (int v = tid; v < MT * NT; v += 256) {
            const int nl = v / MT, ml = v % MT, tok = m0 + ml, h = n0 + nl;
            if (tok < a.BT && h < a.H) {
                const int b = tok / a.T, t = tok % a.T;
                a.z[((size_t)b * a.H + h) * a.T + t] = Cs[ml * ldc + nl];
            }
        }
    }
};

template <int MT, int NT>
int run_router2(const uint16_t* X, const uint16_t* Wr, int BT, int T, int d, int H, float* z, float* xnorm,
                hipStream_t stream) {
    using P = RouterPolicy2<MT, NT>;
    const int mt = (BT + MT - 1) / MT, nt = (H + NT - 1) / NT;
    typename P::Args a{X, Wr, z, xnorm, BT, T, d, H, nt};
    return launch_gemm2<P>(a, mt * nt, stream);
}

}  // namespace

int launch_router(int dtype, const void* X, const void* Wr, int B, int T, int d, int H, float* z,
                  float* xnorm, hipStream_t stream) {
    const int BT = B * T;
    if (dtype == kBF16 && d % 64 == 0) {
        // tile: enough workgroups to fill the chip (about 256), as large as allows
        auto f = run_router2<32, 32>;
        if (H > 64) f = (size_t)((BT + 63) / 64) * ((H + 127) / 128) >= 256 ? run_router2<64, 128> : run_router2<32, 64>;
        else if (H > 32) f = run_router2<32, 64>;
        return f((const uint16_t*)X, (const uint16_t*)Wr, BT, T, d, H, z, xnorm, stream);
    }
    dim3 grid((BT + kRouterTokens - 1) / kRouterTokens, (H + kRouterHeads - 1) / kRouterHeads);
    if (dtype == kBF16)
        hipLaunchKernelGGL(router_kernel<uint16_t>, grid, dim3(256), 0, stream, (const uint16_t*)X,
                           (const uint16_t*)Wr, BT, T, d, H, z, xnorm);
    else
        hipLaunchKernelGGL(router_kernel<float>, grid, dim3(256), 0, stream, (const float*)X,
                           (const float*)Wr, BT, T, d, H, z, xnorm);
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

}  // namespace mosa
