// Device helpers shared by the MoSA kernels (gfx950 / CDNA4 only).
//
// Storage types: `bf16` values travel as uint16_t bit patterns, fp32 as float.
// Matrix-core fragments: a 16x16 output tile is produced by MFMA from
//   A  (16 rows x K)   lane l supplies row l % 16,
//   B  (K x 16 cols)   lane l supplies column l % 16,
// and lane group g = l / 16 supplies a fixed subset of the K index.  Every
// kernel here feeds A and B with the SAME k-subset per lane group, so the
// product only relies on the row/column placement, which is the same for
// v_mfma_f32_16x16x32_bf16, v_mfma_f32_16x16x16_bf16 and v_mfma_f32_16x16x4_f32:
//   D (16x16, fp32)    lane l holds column l % 16, rows 4 g + i (i = 0..3).
#pragma once

#include <type_traits>

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mosa {

// f(std::integral_constant<int, I>) for I = B .. E - 1, each I a constant
// expression in f (immediate offsets, template arguments).
template <int B, int E, class F>
__device__ __forceinline__ void static_for(F&& f) {
    if constexpr (B < E) {
        f(std::integral_constant<int, B>{});
        static_for<B + 1, E>(f);
    }
}

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;

__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// Round to nearest, ties to even (NaN stays NaN).
// Round to nearest even (gfx950 converts in hardware: v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }
// Two floats to a packed pair of bf16 (lo in bits 0..15), one instruction.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    const f32x2 f = {lo, hi};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2));
}

// Neighbouring floats of a finite value (toward +inf / -inf).
__device__ __forceinline__ float next_up(float f) {
    uint32_t u = __float_as_uint(f);
    if (u == 0x80000000u) u = 0u;
    return (int32_t)u >= 0 ? __uint_as_float(u + 1u) : __uint_as_float(u - 1u);
}
__device__ __forceinline__ float next_down(float f) { return -next_up(-f); }

template <typename ST> __device__ __forceinline__ float ld1(const ST* p);
template <> __device__ __forceinline__ float ld1<uint16_t>(const uint16_t* p) { return bf16_to_f32(*p); }
template <> __device__ __forceinline__ float ld1<float>(const float* p) { return *p; }

template <typename ST> __device__ __forceinline__ void st1(ST* p, float v);
template <> __device__ __forceinline__ void st1<uint16_t>(uint16_t* p, float v) { *p = f32_to_bf16(v); }
template <> __device__ __forceinline__ void st1<float>(float* p, float v) { *p = v; }

// ---------------------------------------------------------------------------
// K = 32 fragments: 8 k-values per lane (lane group g holds slots 8g .. 8g+7)
// ---------------------------------------------------------------------------
template <typename ST> struct Frag8;
template <> struct Frag8<uint16_t> { bf16x8 v; };
template <> struct Frag8<float> { float v[8]; };

template <typename ST> __device__ __forceinline__ Frag8<ST> frag8_zero();
template <> __device__ __forceinline__ Frag8<uint16_t> frag8_zero<uint16_t>() {
    Frag8<uint16_t> f;
    uint4 z = make_uint4(0, 0, 0, 0);
    f.v = __builtin_bit_cast(bf16x8, z);
    return f;
}
template <> __device__ __forceinline__ Frag8<float> frag8_zero<float>() {
    Frag8<float> f;
#pragma unroll
    for (int j = 0; j < 8; ++j) f.v[j] = 0.f;
    return f;
}

// 8 contiguous elements (16-byte aligned for bf16, 32-byte for fp32).
template <typename ST> __device__ __forceinline__ Frag8<ST> frag8_load(const ST* p);
template <> __device__ __forceinline__ Frag8<uint16_t> frag8_load<uint16_t>(const uint16_t* p) {
    Frag8<uint16_t> f;
    f.v = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(p));
    return f;
}
template <> __device__ __forceinline__ Frag8<float> frag8_load<float>(const float* p) {
    Frag8<float> f;
    float4 a = reinterpret_cast<const float4*>(p)[0];
    float4 b = reinterpret_cast<const float4*>(p)[1];
    f.v[0] = a.x; f.v[1] = a.y; f.v[2] = a.z; f.v[3] = a.w;
    f.v[4] = b.x; f.v[5] = b.y; f.v[6] = b.z; f.v[7] = b.w;
    return f;
}

template <typename ST> __device__ __forceinline__ Frag8<ST> frag8_from(const float (&x)[8]);
template <> __device__ __forceinline__ Frag8<uint16_t> frag8_from<uint16_t>(const float (&x)[8]) {
    uint4 u;
    u.x = pack_bf16x2(x[0], x[1]);
    u.y = pack_bf16x2(x[2], x[3]);
    u.z = pack_bf16x2(x[4], x[5]);
    u.w = pack_bf16x2(x[6], x[7]);
    Frag8<uint16_t> f;
    f.v = __builtin_bit_cast(bf16x8, u);
    return f;
}
template <> __device__ __forceinline__ Frag8<float> frag8_from<float>(const float (&x)[8]) {
    Frag8<float> f;
#pragma unroll
    for (int j = 0; j < 8; ++j) f.v[j] = x[j];
    return f;
}

template <typename ST> __device__ __forceinline__ void frag8_to_f32(const Frag8<ST>& f, float (&x)[8]);
template <> __device__ __forceinline__ void frag8_to_f32<uint16_t>(const Frag8<uint16_t>& f, float (&x)[8]) {
    uint4 u = __builtin_bit_cast(uint4, f.v);
    x[0] = __uint_as_float(u.x << 16); x[1] = __uint_as_float(u.x & 0xffff0000u);
    x[2] = __uint_as_float(u.y << 16); x[3] = __uint_as_float(u.y & 0xffff0000u);
    x[4] = __uint_as_float(u.z << 16); x[5] = __uint_as_float(u.z & 0xffff0000u);
    x[6] = __uint_as_float(u.w << 16); x[7] = __uint_as_float(u.w & 0xffff0000u);
}
template <> __device__ __forceinline__ void frag8_to_f32<float>(const Frag8<float>& f, float (&x)[8]) {
#pragma unroll
    for (int j = 0; j < 8; ++j) x[j] = f.v[j];
}

// acc += A * B over one K = 32 step.
__device__ __forceinline__ void mma8(f32x4& acc, const Frag8<uint16_t>& a, const Frag8<uint16_t>& b) {
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a.v, b.v, acc, 0, 0, 0);
}
__device__ __forceinline__ void mma8(f32x4& acc, const Frag8<float>& a, const Frag8<float>& b) {
#pragma unroll
    for (int j = 0; j < 8; ++j) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.v[j], b.v[j], acc, 0, 0, 0);
}

// ---------------------------------------------------------------------------
// K = 16 fragments: 4 k-values per lane (lane group g holds slots 4g .. 4g+3),
// the row placement of a 16x16 MFMA result, so a D tile feeds the next MFMA
// as a K = 16 operand without moving data between lanes.
// ---------------------------------------------------------------------------
template <typename ST> struct Frag4;
template <> struct Frag4<uint16_t> { s16x4 v; };
template <> struct Frag4<float> { float v[4]; };

template <typename ST> __device__ __forceinline__ Frag4<ST> frag4_from(const float (&x)[4]);
template <> __device__ __forceinline__ Frag4<uint16_t> frag4_from<uint16_t>(const float (&x)[4]) {
    const uint32_t lo = pack_bf16x2(x[0], x[1]), hi = pack_bf16x2(x[2], x[3]);
    Frag4<uint16_t> f;
    f.v = __builtin_bit_cast(s16x4, make_uint2(lo, hi));
    return f;
}
template <> __device__ __forceinline__ Frag4<float> frag4_from<float>(const float (&x)[4]) {
    Frag4<float> f;
#pragma unroll
    for (int j = 0; j < 4; ++j) f.v[j] = x[j];
    return f;
}

__device__ __forceinline__ void mma4(f32x4& acc, const Frag4<uint16_t>& a, const Frag4<uint16_t>& b) {
    acc = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a.v, b.v, acc, 0, 0, 0);
}
__device__ __forceinline__ void mma4(f32x4& acc, const Frag4<float>& a, const Frag4<float>& b) {
#pragma unroll
    for (int j = 0; j < 4; ++j) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.v[j], b.v[j], acc, 0, 0, 0);
}

__device__ __forceinline__ f32x4 zero4() { return f32x4{0.f, 0.f, 0.f, 0.f}; }

// Max / sum over the four rows of 16 lanes (lanes c, c + 16, c + 32, c + 48)
// with the gfx950 row-swap moves (no LDS traffic): v_permlane16_swap gives
// every lane the values of both rows of its row pair, v_permlane32_swap those
// of both halves.  Every lane gets the same result, (x0 op x1) op (x2 op x3).
__device__ __forceinline__ float rows4_max(float x) {
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    x = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
    const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float rows4_sum(float x) {
    const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    x = __uint_as_float(a[0]) + __uint_as_float(a[1]);
    const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// Allows a kernel more than the default 64 KB of dynamic LDS on the current
// device.  Called before every such launch (the attribute is cheap to set),
// so the library keeps no record of which kernels were raised where.
inline int allow_lds(const void* kern, size_t bytes) {
    if (bytes <= 64 * 1024) return 0;
    return hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes) == hipSuccess ? 0 : -1;
}

// Explicit wait states between the last MFMA of a loop and the first VALU
// read of its accumulators after the loop: the compiler's hazard insertion
// has been seen to miss the path that leaves a loop (or skips a block) right
// after an MFMA, so kernels call this once after such loops.
__device__ __forceinline__ void mfma_drain() {
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");
}

// Division of non-negative x < 2^24 by a runtime n via a float reciprocal and
// a one-step correction (exact in that range).
struct FastDiv {
    int n;
    float inv;
};
inline FastDiv make_fastdiv(int n) { return {n, 1.0f / (float)n}; }
__device__ __forceinline__ void fast_divmod(const FastDiv& f, int x, int& q, int& r) {
    q = (int)((float)x * f.inv);
    r = x - q * f.n;
    if (r < 0) {
        --q;
        r += f.n;
    } else if (r >= f.n) {
        ++q;
        r -= f.n;
    }
}

// ---------------------------------------------------------------------------
// Launch-order helper: the hardware dispatches workgroup b to XCD b % 8.
// Renumber so that consecutive logical ids run on the same XCD and share
// its L2: logical = (#blocks on lower XCDs) + b / 8.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int xcd_logical_id(int b, int n) {
    const int q = n / 8, r = n % 8, x = b % 8;
    return x * q + (x < r ? x : r) + b / 8;
}

// ---------------------------------------------------------------------------
// Inclusive scan of a 32-bit value over the 64 lanes of a wave (lane i gets
// the sum over lanes 0..i) with DPP row shifts (1, 2, 4, 8 within rows of 16
// lanes) and row broadcasts (lane 15 into rows 1 and 3, lane 31 into rows 2
// and 3), after which lane 63 holds the total; wave_sum_u32 returns that total
// to every lane.  The whole wave must be active.
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t wave_inclusive_scan_u32(uint32_t x) {
    x += __builtin_amdgcn_update_dpp(0u, x, 0x111, 0xf, 0xf, false);  // row_shr:1
    x += __builtin_amdgcn_update_dpp(0u, x, 0x112, 0xf, 0xf, false);  // row_shr:2
    x += __builtin_amdgcn_update_dpp(0u, x, 0x114, 0xf, 0xf, false);  // row_shr:4
    x += __builtin_amdgcn_update_dpp(0u, x, 0x118, 0xf, 0xf, false);  // row_shr:8
    x += __builtin_amdgcn_update_dpp(0u, x, 0x142, 0xa, 0xf, false);  // row_bcast:15
    x += __builtin_amdgcn_update_dpp(0u, x, 0x143, 0xc, 0xf, false);  // row_bcast:31
    return x;
}
__device__ __forceinline__ uint32_t wave_sum_u32(uint32_t x) {
    return __builtin_amdgcn_readlane(wave_inclusive_scan_u32(x), 63);
}

// The same DPP moves on a double (both 32-bit halves; lanes without a source
// get 0.0).
template <int CTRL, int ROWS>
__device__ __forceinline__ double dpp_f64(double x) {
    const uint64_t u = (uint64_t)__double_as_longlong(x);
    const uint32_t lo = __builtin_amdgcn_update_dpp(0u, (uint32_t)u, CTRL, ROWS, 0xf, false);
    const uint32_t hi = __builtin_amdgcn_update_dpp(0u, (uint32_t)(u >> 32), CTRL, ROWS, 0xf, false);
    return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}
// Sum over the wave of a double, in every lane (register moves only).
__device__ __forceinline__ double wave_sum_f64(double x) {
    x += dpp_f64<0x111, 0xf>(x);
    x += dpp_f64<0x112, 0xf>(x);
    x += dpp_f64<0x114, 0xf>(x);
    x += dpp_f64<0x118, 0xf>(x);
    x += dpp_f64<0x142, 0xa>(x);
    x += dpp_f64<0x143, 0xc>(x);
    const uint64_t u = (uint64_t)__double_as_longlong(x);
    const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)u, 63), hi = __builtin_amdgcn_readlane((uint32_t)(u >> 32), 63);
    return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}
// Maximum over the wave of non-negative floats, in every lane.
template <int CTRL, int ROWS>
__device__ __forceinline__ float dpp_f32(float x) {
    return __uint_as_float(__builtin_amdgcn_update_dpp(0u, __float_as_uint(x), CTRL, ROWS, 0xf, false));
}
__device__ __forceinline__ float wave_max_nonneg_f32(float x) {
    x = fmaxf(x, dpp_f32<0x111, 0xf>(x));
    x = fmaxf(x, dpp_f32<0x112, 0xf>(x));
    x = fmaxf(x, dpp_f32<0x114, 0xf>(x));
    x = fmaxf(x, dpp_f32<0x118, 0xf>(x));
    x = fmaxf(x, dpp_f32<0x142, 0xa>(x));
    x = fmaxf(x, dpp_f32<0x143, 0xc>(x));
    return __uint_as_float(__builtin_amdgcn_readlane(__float_as_uint(x), 63));
}

// ---------------------------------------------------------------------------
// Block-wide scans for 256 threads (4 waves).
// ---------------------------------------------------------------------------
__device__ __forceinline__ int wave_inclusive_scan(int v) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        int u = __shfl_up(v, o, 64);
        if (lane >= o) v += u;
    }
    return v;
}

// Exclusive prefix sum over the 256 threads in thread order; *total gets the sum.
// `tmp` must hold 4 ints of LDS.  Contains barriers: call from all threads.
__device__ __forceinline__ int block256_exclusive_scan(int v, int* tmp, int* total) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    int inc = wave_inclusive_scan(v);
    if (lane == 63) tmp[w] = inc;
    __syncthreads();
    int base = 0, all = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        int t = tmp[i];
        if (i < w) base += t;
        all += t;
    }
    __syncthreads();
    *total = all;
    return base + inc - v;
}

__device__ __forceinline__ double block256_sum(double v, double* tmp) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
    if ((threadIdx.x & 63) == 0) tmp[threadIdx.x >> 6] = v;
    __syncthreads();
    double s = tmp[0] + tmp[1] + tmp[2] + tmp[3];
    __syncthreads();
    return s;
}

}  // namespace mosa
