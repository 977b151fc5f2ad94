// Backward of the output side of a head (chain rule through Section 2.2's
// X^o = diag(r) A W^O and the scatter Y_{I_i} = X^o_i, with I held fixed):
//   dX^o_i   = dY[b, I_i]                      (gather)
//   dA~_i    = dX^o_i W^O^T                    (MFMA, K = d)
//   dr_i     = <dA~_i, A_i>                    (router gradient through r)
//   dA_i     = r_i dA~_i                       (into the attention backward)
//   D_i      = <dA_i, A_i> = r_i dr_i          (softmax row term of Eq. 1's backward)
//   dz_i     = dr_i r_i (1 - r_i)              (sigma'(s) = r (1 - r))
// Dense heads are the case I = identity, r = 1 (no dz).
//
// Workgroup = 64 gathered rows of one head (4 waves x 16 rows) x all dh
// columns.  W^O rows are contiguous along d, which is the K index here, so
// both MFMA operands are read straight from memory as 16-byte fragments.
#include "common.h"
#include "kernels.h"

namespace mosa {

namespace {

template <typename ST, int DH>
__global__ __launch_bounds__(256) void dattn_out_kernel(const ST* __restrict__ dY, const int32_t* __restrict__ I,
                                                        const float* __restrict__ r, const ST* __restrict__ Wo,
                                                        const ST* __restrict__ A, int T, int d, int H, int n,
                                                        int nrows, int ntiles, ST* __restrict__ dA,
                                                        float* __restrict__ D, float* __restrict__ dz) {
    constexpr int NCB = DH / 16;
    const int logical = xcd_logical_id(blockIdx.x, gridDim.x);
    const int tile = logical % ntiles, h = logical / ntiles;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int g = lane >> 4, c16 = lane & 15;

    const int arow = tile * 64 + wave * 16 + c16;
    const bool arow_ok = arow < nrows;
    const ST* yrow = dY;
    if (arow_ok) {
        const int b = arow / n, i = arow % n;
        const int t = I ? I[((size_t)b * H + h) * n + i] : i;
        yrow = dY + ((size_t)b * T + t) * d;
    }
    const ST* Wh = Wo + (size_t)h * DH * d;

    f32x4 acc[NCB];
#pragma unroll
    for (int c = 0; c < NCB; ++c) acc[c] = zero4();
    for (int kc = 0; kc < d; kc += 32) {
        const Frag8<ST> a = arow_ok ? frag8_load<ST>(yrow + kc + 8 * g) : frag8_zero<ST>();
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) {
            const Frag8<ST> bw = frag8_load<ST>(Wh + (size_t)(cb * 16 + c16) * d + kc + 8 * g);
            mma8(acc[cb], a, bw);
        }
    }

    // lane holds dA~[row 4g+i][col cb*16 + c16]
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int row = tile * 64 + wave * 16 + 4 * g + i;
        const bool ok = row < nrows;
        size_t ridx = 0;
        if (ok) {
            const int b = row / n, ii = row % n;
            ridx = ((size_t)b * H + h) * n + ii;
        }
        float part = 0.f;
        if (ok) {
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb) part += acc[cb][i] * ld1<ST>(A + ridx * DH + cb * 16 + c16);
        }
        part += __shfl_xor(part, 1, 64);
        part += __shfl_xor(part, 2, 64);
        part += __shfl_xor(part, 4, 64);
        part += __shfl_xor(part, 8, 64);
        if (ok) {
            const float rr = r ? r[ridx] : 1.f;
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb) st1<ST>(dA + ridx * DH + cb * 16 + c16, rr * acc[cb][i]);
            if (c16 == 0) {
                D[ridx] = rr * part;
                if (dz) dz[ridx] = part * rr * (1.f - rr);
            }
        }
    }
}

template <typename ST>
int launch_t(const ST* dY, const int32_t* I, const float* r, const ST* Wo, const ST* A, int B, int T, int d, int H,
             int dh, int n, ST* dA, float* D, float* dz, hipStream_t stream) {
    const int nrows = B * n, ntiles = (nrows + 63) / 64;
    dim3 grid(ntiles * H), block(256);
    if (dh == 64)
        hipLaunchKernelGGL((dattn_out_kernel<ST, 64>), grid, block, 0, stream, dY, I, r, Wo, A, T, d, H, n, nrows,
                           ntiles, dA, D, dz);
    else
        hipLaunchKernelGGL((dattn_out_kernel<ST, 32>), grid, block, 0, stream, dY, I, r, Wo, A, T, d, H, n, nrows,
                           ntiles, dA, D, dz);
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

}  // namespace

int launch_dattn_out(int dtype, const void* dY, const int32_t* I, const float* r, const void* Wo, const void* A,
                     int B, int T, int d, int H, int dh, int n, void* dA, float* D, float* dz, hipStream_t stream) {
    if (dtype == kBF16)
        return launch_t<uint16_t>((const uint16_t*)dY, I, r, (const uint16_t*)Wo, (const uint16_t*)A, B, T, d, H, dh,
                                  n, (uint16_t*)dA, D, dz, stream);
    return launch_t<float>((const float*)dY, I, r, (const float*)Wo, (const float*)A, B, T, d, H, dh, n, (float*)dA,
                           D, dz, stream);
}

}  // namespace mosa
