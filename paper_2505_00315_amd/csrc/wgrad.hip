// Weight gradients of the MoSA heads (chain rule through Section 2.2 with I
// held fixed), summed over every selected row r = (b, i) in a fixed order:
//   dW^Q_h = sum_r X[b, I_r]^T dQ_r   (likewise W^K, W^V)    [d x dh]
//   dW^r_h = sum_r dz_r X[b, I_r]                             [d]
//   dW^O_h = sum_r (r_r A_r)^T dY[b, I_r]                     [dh x d]
// Dense heads: the same with I = identity and r = 1 (no W^r).
//
// The contraction index is the row r, which is not contiguous in any
// operand, so each workgroup stages 32-row chunks of both operands in LDS
// transposed (row index contiguous) and feeds MFMA K = 32 fragments from
// there.  One workgroup per (head, 64-wide slice of d); the sum over rows is
// a plain loop, so the result is bitwise reproducible.
#include "common.h"
#include "kernels.h"

namespace mosa {

namespace {

constexpr int kRowsChunk = 32;
constexpr int kLdr = kRowsChunk + 8;  // padded LDS row length

// Gathered row r of a [B, T, d] tensor for head h (I == nullptr: identity).
__device__ __forceinline__ size_t gathered_row(const int32_t* I, int r, int n, int H, int h, int T) {
    const int b = r / n, i = r % n;
    const int t = I ? I[((size_t)b * H + h) * n + i] : i;
    return (size_t)b * T + t;
}

template <typename ST, int DH, bool ROUTER>
__global__ __launch_bounds__(256) void wgrad_qkv_kernel(const ST* __restrict__ X, const int32_t* __restrict__ I,
                                                        const ST* __restrict__ dQ, const ST* __restrict__ dK,
                                                        const ST* __restrict__ dV, const float* __restrict__ dz,
                                                        int T, int d, int H, int n, int R, int nct,
                                                        ST* __restrict__ dWq, ST* __restrict__ dWk,
                                                        ST* __restrict__ dWv, ST* __restrict__ dWr) {
    constexpr int NS = 3 * DH + (ROUTER ? 16 : 0);  // small-operand columns
    constexpr int NCB = NS / 16;
    __shared__ __attribute__((aligned(16))) ST s_big[64 * kLdr];
    __shared__ __attribute__((aligned(16))) ST s_small[NS * kLdr];

    const int logical = xcd_logical_id(blockIdx.x, gridDim.x);
    const int h = logical / nct, ct = logical % nct;
    const int c0 = ct * 64;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, c16 = lane & 15;
    const size_t hb = (size_t)h * n;  // row r of head h lives at ((b*H + h)*n + i)

    f32x4 acc[NCB];
#pragma unroll
    for (int c = 0; c < NCB; ++c) acc[c] = zero4();

    const ST* Sm[3] = {dQ, dK, dV};
    for (int r0 = 0; r0 < R; r0 += kRowsChunk) {
        {  // X rows -> s_big[c][r]
            const int rl = tid >> 3, cv = (tid & 7) * 8;
            const int r = r0 + rl;
            float x[8];
            if (r < R) {
                frag8_to_f32<ST>(frag8_load<ST>(X + gathered_row(I, r, n, H, h, T) * d + c0 + cv), x);
            } else {
#pragma unroll
                for (int j = 0; j < 8; ++j) x[j] = 0.f;
            }
#pragma unroll
            for (int j = 0; j < 8; ++j) st1<ST>(&s_big[(cv + j) * kLdr + rl], x[j]);
        }
        // dQ | dK | dV rows -> s_small[m*DH + e][r]
        for (int v = tid; v < 3 * kRowsChunk * (DH / 8); v += 256) {
            const int m = v / (kRowsChunk * (DH / 8)), rem = v % (kRowsChunk * (DH / 8));
            const int rl = rem / (DH / 8), ev = (rem % (DH / 8)) * 8;
            const int r = r0 + rl;
            float x[8];
            if (r < R) {
                const int b = r / n, i = r % n;
                frag8_to_f32<ST>(frag8_load<ST>(Sm[m] + (((size_t)b * H * n + hb + i) * DH) + ev), x);
            } else {
#pragma unroll
                for (int j = 0; j < 8; ++j) x[j] = 0.f;
            }
#pragma unroll
            for (int j = 0; j < 8; ++j) st1<ST>(&s_small[(m * DH + ev + j) * kLdr + rl], x[j]);
        }
        if (ROUTER) {  // column 3*DH holds dz, the next 15 columns zeros
            for (int v = tid; v < 16 * kRowsChunk; v += 256) {
                const int col = v / kRowsChunk, rl = v % kRowsChunk;
                const int r = r0 + rl;
                float x = 0.f;
                if (col == 0 && r < R) {
                    const int b = r / n, i = r % n;
                    x = dz[(size_t)b * H * n + hb + i];
                }
                st1<ST>(&s_small[(3 * DH + col) * kLdr + rl], x);
            }
        }
        __syncthreads();
        const Frag8<ST> a = frag8_load<ST>(&s_big[(wave * 16 + c16) * kLdr + 8 * g]);
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) {
            const Frag8<ST> bs = frag8_load<ST>(&s_small[(cb * 16 + c16) * kLdr + 8 * g]);
            mma8(acc[cb], a, bs);
        }
        __syncthreads();
    }
    // lane: small column cb*16 + c16, d rows c0 + wave*16 + 4g + i
    ST* Wm[3] = {dWq, dWk, dWv};
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
        const int col = cb * 16 + c16;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int c = c0 + wave * 16 + 4 * g + i;
            if (col < 3 * DH) {
                const int m = col / DH, e = col % DH;
                st1<ST>(Wm[m] + ((size_t)h * d + c) * DH + e, acc[cb][i]);
            } else if (ROUTER && col == 3 * DH) {
                st1<ST>(dWr + (size_t)h * d + c, acc[cb][i]);
            }
        }
    }
}

template <typename ST, int DH>
__global__ __launch_bounds__(256) void wgrad_o_kernel(const ST* __restrict__ dY, const int32_t* __restrict__ I,
                                                      const float* __restrict__ rw, const ST* __restrict__ A, int T,
                                                      int d, int H, int n, int R, int nct, ST* __restrict__ dWo) {
    constexpr int NRB = DH / 16;  // row blocks (d_head)
    __shared__ __attribute__((aligned(16))) ST s_a[DH * kLdr];
    __shared__ __attribute__((aligned(16))) ST s_y[64 * kLdr];

    const int logical = xcd_logical_id(blockIdx.x, gridDim.x);
    const int h = logical / nct, ct = logical % nct;
    const int c0 = ct * 64;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, c16 = lane & 15;
    const size_t hb = (size_t)h * n;

    f32x4 acc[NRB];
#pragma unroll
    for (int m = 0; m < NRB; ++m) acc[m] = zero4();

    for (int r0 = 0; r0 < R; r0 += kRowsChunk) {
        {  // dY rows -> s_y[c][r]
            const int rl = tid >> 3, cv = (tid & 7) * 8;
            const int r = r0 + rl;
            float x[8];
            if (r < R) {
                frag8_to_f32<ST>(frag8_load<ST>(dY + gathered_row(I, r, n, H, h, T) * d + c0 + cv), x);
            } else {
#pragma unroll
                for (int j = 0; j < 8; ++j) x[j] = 0.f;
            }
#pragma unroll
            for (int j = 0; j < 8; ++j) st1<ST>(&s_y[(cv + j) * kLdr + rl], x[j]);
        }
        // r * A rows -> s_a[e][r]
        for (int v = tid; v < kRowsChunk * (DH / 8); v += 256) {
            const int rl = v / (DH / 8), ev = (v % (DH / 8)) * 8;
            const int r = r0 + rl;
            float x[8];
            if (r < R) {
                const int b = r / n, i = r % n;
                const size_t ridx = (size_t)b * H * n + hb + i;
                frag8_to_f32<ST>(frag8_load<ST>(A + ridx * DH + ev), x);
                const float rv = rw ? rw[ridx] : 1.f;
#pragma unroll
                for (int j = 0; j < 8; ++j) x[j] *= rv;
            } else {
#pragma unroll
                for (int j = 0; j < 8; ++j) x[j] = 0.f;
            }
#pragma unroll
            for (int j = 0; j < 8; ++j) st1<ST>(&s_a[(ev + j) * kLdr + rl], x[j]);
        }
        __syncthreads();
#pragma unroll
        for (int m = 0; m < NRB; ++m) {
            const int p = wave * NRB + m;  // (row block, col block) pair
            const int rb = p / 4, cb = p % 4;
            const Frag8<ST> a = frag8_load<ST>(&s_a[(rb * 16 + c16) * kLdr + 8 * g]);
            const Frag8<ST> y = frag8_load<ST>(&s_y[(cb * 16 + c16) * kLdr + 8 * g]);
            mma8(acc[m], a, y);
        }
        __syncthreads();
    }
#pragma unroll
    for (int m = 0; m < NRB; ++m) {
        const int p = wave * NRB + m;
        const int rb = p / 4, cb = p % 4;
        const int c = c0 + cb * 16 + c16;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int e = rb * 16 + 4 * g + i;
            st1<ST>(dWo + ((size_t)h * DH + e) * d + c, acc[m][i]);
        }
    }
}

template <typename ST>
int launch_t(const ST* X, const ST* dY, const int32_t* I, const float* r, const ST* A, const ST* dQ, const ST* dK,
             const ST* dV, const float* dz, int B, int T, int d, int H, int dh, int n, ST* dWq, ST* dWk, ST* dWv,
             ST* dWr, ST* dWo, int which, hipStream_t stream) {
    const int R = B * n, nct = d / 64;
    dim3 grid(H * nct), block(256);
    const bool router = dWr != nullptr;
    if (which == 0) {
#define MOSA_WQKV(DHV, RT)                                                                                    \
    hipLaunchKernelGGL((wgrad_qkv_kernel<ST, DHV, RT>), grid, block, 0, stream, X, I, dQ, dK, dV, dz, T, d, H, n, \
                       R, nct, dWq, dWk, dWv, dWr)
        if (dh == 64) {
            if (router) MOSA_WQKV(64, true);
            else MOSA_WQKV(64, false);
        } else {
            if (router) MOSA_WQKV(32, true);
            else MOSA_WQKV(32, false);
        }
#undef MOSA_WQKV
    } else {
        if (dh == 64)
            hipLaunchKernelGGL((wgrad_o_kernel<ST, 64>), grid, block, 0, stream, dY, I, r, A, T, d, H, n, R, nct, dWo);
        else
            hipLaunchKernelGGL((wgrad_o_kernel<ST, 32>), grid, block, 0, stream, dY, I, r, A, T, d, H, n, R, nct, dWo);
    }
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

}  // namespace

int launch_wgrad(int dtype, const void* X, const void* dY, const int32_t* I, const float* r, const void* A,
                 const void* dQ, const void* dK, const void* dV, const float* dz, int B, int T, int d, int H, int dh,
                 int n, void* dWq, void* dWk, void* dWv, void* dWr, void* dWo, int which, hipStream_t stream) {
    if (dtype == kBF16)
        return launch_t<uint16_t>((const uint16_t*)X, (const uint16_t*)dY, I, r, (const uint16_t*)A,
                                  (const uint16_t*)dQ, (const uint16_t*)dK, (const uint16_t*)dV, dz, B, T, d, H, dh, n,
                                  (uint16_t*)dWq, (uint16_t*)dWk, (uint16_t*)dWv, (uint16_t*)dWr, (uint16_t*)dWo,
                                  which, stream);
    return launch_t<float>((const float*)X, (const float*)dY, I, r, (const float*)A, (const float*)dQ,
                           (const float*)dK, (const float*)dV, dz, B, T, d, H, dh, n, (float*)dWq, (float*)dWk,
                           (float*)dWv, (float*)dWr, (float*)dWo, which, stream);
}

}  // namespace mosa
