// Independent GEMM-engine jobs in one launch: every workgroup runs one job's
// tile, and every XCD receives its share of each job (the blocks an XCD gets,
// every eighth, are its share of job 0 first, then job 1, then the rest), so
// the different kinds of workgroups share the CUs and the launch has one
// tail instead of one per job.
#pragma once

#include "gemm2.h"
#include "rowgemm.h"

namespace mosa {

template <class P>
struct Gemm2Job {
    using Args = typename P::Args;
    static constexpr int MIN_WAVES = G2MinWaves<P>::value;
    static size_t lds(int ktab_rows) { return Gemm2Shape<P>::lds_bytes(ktab_rows); }
    __device__ static void run(const Args& a, int logical, unsigned char* smem) { gemm2_body<P>(a, logical, smem); }
};

template <class P>
struct RowGemmJob {
    using Args = typename P::Args;
    static constexpr int MIN_WAVES = 1;
    static size_t lds(int) { return RowGemmShape<P>::lds_bytes(); }
    __device__ static void run(const Args& a, int logical, unsigned char* smem) { rowgemm_body<P>(a, logical, smem); }
};

// Share of n blocks on XCD x (of 8) and the number on lower XCDs.
__host__ __device__ __forceinline__ int xcd_share(int n, int x, int& before) {
    before = x * (n / 8) + (x < n % 8 ? x : n % 8);
    return n / 8 + (x < n % 8 ? 1 : 0);
}

__device__ __forceinline__ void xcd_split3(int b, int nb, int n0, int n1, int& which, int& idx) {
    const int x = b % 8, j = b / 8;
    int s0, s1, sall;
    const int c0 = xcd_share(n0, x, s0), c1 = xcd_share(n1, x, s1);
    (void)xcd_share(nb, x, sall);
    if (j < c0) {
        which = 0;
        idx = s0 + j;
    } else if (j < c0 + c1) {
        which = 1;
        idx = s1 + (j - c0);
    } else {
        which = 2;
        idx = (sall - s0 - s1) + (j - c0 - c1);
    }
}

template <class J0, class J1, class J2>
constexpr int group_min_waves() {
    int m = J0::MIN_WAVES;
    if (J1::MIN_WAVES > m) m = J1::MIN_WAVES;
    if (J2::MIN_WAVES > m) m = J2::MIN_WAVES;
    return m;
}

template <class J0, class J1, class J2>
__global__ __launch_bounds__(256, (group_min_waves<J0, J1, J2>())) void group3_kernel(
    const typename J0::Args a0, const typename J1::Args a1, const typename J2::Args a2, int n0, int n1) {
    extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
    int which, idx;
    xcd_split3(blockIdx.x, gridDim.x, n0, n1, which, idx);
    if (which == 0) J0::run(a0, idx, smem);
    else if (which == 1) J1::run(a1, idx, smem);
    else J2::run(a2, idx, smem);
}

// Launch of three jobs (n0, n1, n2 workgroups; lds0..2: their LDS bytes).
// Returns 1, launching nothing, when an XCD's share of the blocks could not
// hold its shares of jobs 0 and 1 (the split above needs that) or the LDS
// does not fit.
template <class J0, class J1, class J2>
int launch_group3(const typename J0::Args& a0, int n0, size_t lds0, const typename J1::Args& a1, int n1, size_t lds1,
                  const typename J2::Args& a2, int n2, size_t lds2, hipStream_t stream) {
    const int nb = n0 + n1 + n2;
    if (n0 <= 0 || n1 <= 0 || n2 <= 0) return 1;
    for (int x = 0; x < 8; ++x) {
        int t;
        if (xcd_share(nb, x, t) < xcd_share(n0, x, t) + xcd_share(n1, x, t)) return 1;
    }
    size_t lds = lds0 > lds1 ? lds0 : lds1;
    if (lds2 > lds) lds = lds2;
    if (lds > 160 * 1024) return 1;
    auto kern = group3_kernel<J0, J1, J2>;
    if (allow_lds((const void*)kern, lds)) return -1;
    hipLaunchKernelGGL(kern, dim3(nb), dim3(256), lds, stream, a0, a1, a2, n0, n1);
    return hipGetLastError() == hipSuccess ? 0 : -1;
}

}  // namespace mosa
