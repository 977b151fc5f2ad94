// Gather + grouped Q/K/V projection (paper Section 2.2: X^s = X[I];
// Q = X^s W^Q, K = X^s W^K, V = X^s W^V, computed only for the k selected
// tokens of every head; a dense head is the case I = 0..T-1).
//
// One workgroup (4 waves) owns 64 rows of one head's B*n gathered rows and
// all 3*dh output columns, so each weight byte of the head is fetched by
// ceil(B*n/64) workgroups, which the XCD-aware numbering places on one XCD
// (one L2).  K loop over d in chunks of 64: the three [64 x dh] weight
// slices are read with 16-byte coalesced loads and written transposed into
// LDS (k contiguous), from where every wave reads its MFMA B fragments.  The
// gathered X rows are read straight from HBM as A fragments (k contiguous in
// X).  MFMA: v_mfma_f32_16x16x32_bf16 (bf16) / 16x16x4_f32 (fp32).
#include "common.h"
#include "kernels.h"

namespace mosa {

namespace {

constexpr int kRowsPerWG = 64;
constexpr int kChunk = 64;
constexpr int kLdsPad = 8;

template <typename ST, int DH>
__global__ __launch_bounds__(256) void qkv_kernel(const ST* __restrict__ X, const int32_t* __restrict__ I,
                                                  const ST* __restrict__ Wq, const ST* __restrict__ Wk,
                                                  const ST* __restrict__ Wv, int T, int d, int H, int n,
                                                  int nrows, int ntiles, ST* __restrict__ Q, ST* __restrict__ K,
                                                  ST* __restrict__ V) {
    constexpr int NCOL = 3 * DH;
    constexpr int NCB = NCOL / 16;
    constexpr int LDW = kChunk + kLdsPad;
    __shared__ __attribute__((aligned(16))) ST s_w[NCOL * LDW];

    const int logical = xcd_logical_id(blockIdx.x, gridDim.x);
    const int tile = logical % ntiles, h = logical / ntiles;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, c16 = lane & 15;

    // the row this lane feeds as A
    const int arow = tile * kRowsPerWG + wave * 16 + c16;
    const bool arow_ok = arow < nrows;
    const ST* xrow = X;
    if (arow_ok) {
        const int b = arow / n, i = arow % n;
        const int t = I ? I[((size_t)b * H + h) * n + i] : i;
        xrow = X + ((size_t)b * T + t) * d;
    }

    const ST* Wm[3] = {Wq + (size_t)h * d * DH, Wk + (size_t)h * d * DH, Wv + (size_t)h * d * DH};

    f32x4 acc[NCB];
#pragma unroll
    for (int c = 0; c < NCB; ++c) acc[c] = zero4();

    for (int kc = 0; kc < d; kc += kChunk) {
        // stage W[kc:kc+64, :] of q, k, v transposed: s_w[m*DH + col][kr]
        constexpr int VEC = 8;
        constexpr int PER_M = kChunk * DH / VEC;
        for (int v = tid; v < 3 * PER_M; v += 256) {
            const int m = v / PER_M, rem = v % PER_M;
            const int kr = rem / (DH / VEC), c0 = (rem % (DH / VEC)) * VEC;
            const Frag8<ST> f = frag8_load<ST>(Wm[m] + (size_t)(kc + kr) * DH + c0);
            float x[8];
            frag8_to_f32<ST>(f, x);
#pragma unroll
            for (int j = 0; j < VEC; ++j) st1<ST>(&s_w[(m * DH + c0 + j) * LDW + kr], x[j]);
        }
        __syncthreads();
#pragma unroll
        for (int ks = 0; ks < kChunk; ks += 32) {
            const Frag8<ST> a = arow_ok ? frag8_load<ST>(xrow + kc + ks + 8 * g) : frag8_zero<ST>();
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb) {
                const Frag8<ST> bw = frag8_load<ST>(&s_w[(cb * 16 + c16) * LDW + ks + 8 * g]);
                mma8(acc[cb], a, bw);
            }
        }
        __syncthreads();
    }

    // D: lane holds column c16 of block cb, rows 4g + i of this wave's 16 rows.
    ST* outm[3] = {Q, K, V};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int row = tile * kRowsPerWG + wave * 16 + 4 * g + i;
        if (row < nrows) {
            const int b = row / n, ii = row % n;
            const size_t base = (((size_t)b * H + h) * n + ii) * DH;
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb) {
                const int m = cb / (DH / 16), col = (cb % (DH / 16)) * 16 + c16;
                st1<ST>(outm[m] + base + col, acc[cb][i]);
            }
        }
    }
}

template <typename ST>
int launch_qkv_t(const ST* X, const int32_t* I, const ST* Wq, const ST* Wk, const ST* Wv, int B, int T, int d,
                 int H, int dh, int n, ST* Q, ST* K, ST* V, hipStream_t stream) {
    const int nrows = B * n;
    const int ntiles = (nrows + kRowsPerWG - 1) / kRowsPerWG;
    dim3 grid(ntiles * H), block(256);
    if (dh == 64)
        hipLaunchKernelGGL((qkv_kernel<ST, 64>), grid, block, 0, stream, X, I, Wq, Wk, Wv, T, d, H, n, nrows,
                           ntiles, Q, K, V);
    else
        hipLaunchKernelGGL((qkv_kernel<ST, 32>), grid, block, 0, stream, X, I, Wq, Wk, Wv, T, d, H, n, nrows,
                           ntiles, Q, K, V);
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

}  // namespace

int launch_qkv(int dtype, const void* X, const int32_t* I, const void* Wq, const void* Wk, const void* Wv, int B,
               int T, int d, int H, int dh, int n, void* Q, void* K, void* V, hipStream_t stream) {
    if (dtype == kBF16)
        return launch_qkv_t<uint16_t>((const uint16_t*)X, I, (const uint16_t*)Wq, (const uint16_t*)Wk,
                                      (const uint16_t*)Wv, B, T, d, H, dh, n, (uint16_t*)Q, (uint16_t*)K,
                                      (uint16_t*)V, stream);
    return launch_qkv_t<float>((const float*)X, I, (const float*)Wq, (const float*)Wk, (const float*)Wv, B, T, d,
                               H, dh, n, (float*)Q, (float*)K, (float*)V, stream);
}

}  // namespace mosa
