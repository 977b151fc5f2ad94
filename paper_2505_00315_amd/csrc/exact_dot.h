// Exact dot product of bf16 or fp32 vectors, rounded once to binary64.
//
// Method: a fixed-point "long accumulator" (Kulisch & Miranker, "The
// arithmetic of the digital computer: a new approach", SIAM Review 1986).
// Every product x_i * w_i of two bf16 (8-bit significand) or two fp32
// (24-bit significand) numbers is an integer M times 2^E with M < 2^48 and
// E >= -298.  The products are added as integers at weight 2^-300 into
// 20 signed 64-bit digits of 32 bits each (640 bits; a product touches at
// most three digits).  Integer addition is associative, so the digits are
// the same whatever the order of the additions (GPU lanes may add them with
// LDS atomics).  The final value is normalised once and rounded to nearest,
// ties to even.
//
// The routines are plain C++ usable on the host (for tests) and the device.
#pragma once

#include <stdint.h>

#if defined(__HIPCC__)
#define MOSA_HD __host__ __device__
#else
#define MOSA_HD
#endif

namespace mosa {

constexpr int kLongDigits = 20;     // 20 x 32 bits
constexpr int kLongLsbExp = -300;   // weight of bit 0

struct ProductParts {
    uint64_t v[3];  // magnitudes added to digits j, j+1, j+2 (each < 2^33)
    int j;          // lowest digit touched
    int negative;
    int zero;
};

// value = (-1)^s * M * 2^E for one stored element.
MOSA_HD inline void split_bf16(uint16_t bits, uint32_t& s, uint32_t& M, int& E) {
    s = bits >> 15;
    uint32_t e = (bits >> 7) & 0xffu, m = bits & 0x7fu;
    M = e ? (m | 0x80u) : m;
    E = (e ? (int)e : 1) - 127 - 7;
}
MOSA_HD inline void split_f32(uint32_t bits, uint32_t& s, uint32_t& M, int& E) {
    s = bits >> 31;
    uint32_t e = (bits >> 23) & 0xffu, m = bits & 0x7fffffu;
    M = e ? (m | 0x800000u) : m;
    E = (e ? (int)e : 1) - 127 - 23;
}

// Digit contributions of the product of two split values.
MOSA_HD inline ProductParts product_parts(uint32_t sx, uint32_t Mx, int Ex, uint32_t sw, uint32_t Mw, int Ew) {
    ProductParts p;
    uint64_t P = (uint64_t)Mx * (uint64_t)Mw;  // < 2^48
    p.zero = (P == 0);
    p.negative = (int)(sx ^ sw);
    int q = Ex + Ew - kLongLsbExp;  // >= 2 for finite inputs; <= 510
    if (q < 0) q = 0;               // unreachable for finite inputs; keeps indices in range
    p.j = q >> 5;
    const int sh = q & 31;
    const uint64_t a = (P & 0xffffffffull) << sh;  // < 2^63
    const uint64_t b = (P >> 32) << sh;            // < 2^47
    p.v[0] = a & 0xffffffffull;
    p.v[1] = (a >> 32) + (b & 0xffffffffull);
    p.v[2] = b >> 32;
    return p;
}

// Round the integer held in `dig` (value = sum dig[j] 2^(32 j) * 2^kLongLsbExp,
// digits may be any signed values whose sum fits) to the nearest double.
// The digits are normalised in place (carries propagated, the magnitude's
// 32-bit words left in the slots), so no local array is needed: on the GPU the
// digits stay in LDS and the routine uses no private (scratch) memory; its
// loops stay loops (not unrolled), so that it holds few registers.
MOSA_HD inline double long_accumulator_round(int64_t* dig) {
    int64_t carry = 0;
#pragma clang loop unroll(disable)
    for (int j = 0; j < kLongDigits; ++j) {
        const int64_t v = dig[j] + carry;
        dig[j] = (int64_t)((uint64_t)v & 0xffffffffull);
        carry = v >> 32;  // arithmetic shift: floor division
    }
    const int negative = carry < 0;
    if (negative) {  // two's-complement negation of the 640-bit word
        uint64_t c = 1;
#pragma clang loop unroll(disable)
        for (int j = 0; j < kLongDigits; ++j) {
            const uint64_t v = (uint64_t)(uint32_t)~(uint32_t)dig[j] + c;
            dig[j] = (int64_t)(uint32_t)v;
            c = v >> 32;
        }
    }
    auto w = [dig](int j) { return (uint32_t)dig[j]; };
    int top = -1;
#pragma clang loop unroll(disable)
    for (int j = kLongDigits - 1; j >= 0; --j)
        if (w(j)) { top = j; break; }
    if (top < 0) return 0.0;
    int msb = 31;
    while (!((w(top) >> msb) & 1u)) --msb;
    const int bitpos = 32 * top + msb;  // position of the leading one

    // 64-bit window whose bit 63 is the leading one, plus a sticky bit.
    uint64_t win;
    int sticky = 0;
    if (bitpos < 64) {
        uint64_t all = (uint64_t)w(0) | ((uint64_t)w(1) << 32);
        win = all << (63 - bitpos);
    } else {
        const int low = bitpos - 63, wi = low >> 5, sb = low & 31;
        uint64_t lo64 = (uint64_t)w(wi) | ((wi + 1 < kLongDigits ? (uint64_t)w(wi + 1) : 0ull) << 32);
        uint64_t hi32 = (wi + 2 < kLongDigits) ? (uint64_t)w(wi + 2) : 0ull;
        win = (lo64 >> sb) | (sb ? (hi32 << (64 - sb)) : 0ull);
        if (sb && (lo64 & ((1ull << sb) - 1ull))) sticky = 1;
#pragma clang loop unroll(disable)
        for (int j = 0; j < wi; ++j)
            if (w(j)) sticky = 1;
    }
    uint64_t sig = win >> 11;          // 53 bits, leading one at bit 52
    const uint64_t rem = win & 0x7ffull;
    if (rem > 0x400ull || (rem == 0x400ull && (sticky || (sig & 1ull)))) ++sig;
    // value = sig * 2^(bitpos - 52 + kLongLsbExp); sig <= 2^53 is exact in double.
    int e = bitpos - 52 + kLongLsbExp;
    double r = (double)sig;
    // scale by 2^e with exact power-of-two multiplications (e in [-352, 300])
    while (e > 0) { int s = e > 60 ? 60 : e; r *= (double)(1ull << s); e -= s; }
    while (e < 0) { int s = -e > 60 ? 60 : -e; r /= (double)(1ull << s); e += s; }
    return negative ? -r : r;
}

// Sequential reference use of the accumulator (host tests, single thread).
MOSA_HD inline double exact_dot_bf16(const uint16_t* x, const uint16_t* w, int n) {
    int64_t dig[kLongDigits];
    for (int j = 0; j < kLongDigits; ++j) dig[j] = 0;
    for (int i = 0; i < n; ++i) {
        uint32_t sx, Mx, sw, Mw;
        int Ex, Ew;
        split_bf16(x[i], sx, Mx, Ex);
        split_bf16(w[i], sw, Mw, Ew);
        ProductParts p = product_parts(sx, Mx, Ex, sw, Mw, Ew);
        if (p.zero) continue;
        for (int t = 0; t < 3; ++t)
            dig[p.j + t] += p.negative ? -(int64_t)p.v[t] : (int64_t)p.v[t];
    }
    return long_accumulator_round(dig);
}

MOSA_HD inline double exact_dot_f32(const uint32_t* x, const uint32_t* w, int n) {
    int64_t dig[kLongDigits];
    for (int j = 0; j < kLongDigits; ++j) dig[j] = 0;
    for (int i = 0; i < n; ++i) {
        uint32_t sx, Mx, sw, Mw;
        int Ex, Ew;
        split_f32(x[i], sx, Mx, Ex);
        split_f32(w[i], sw, Mw, Ew);
        ProductParts p = product_parts(sx, Mx, Ex, sw, Mw, Ew);
        if (p.zero) continue;
        for (int t = 0; t < 3; ++t)
            dig[p.j + t] += p.negative ? -(int64_t)p.v[t] : (int64_t)p.v[t];
    }
    return long_accumulator_round(dig);
}

}  // namespace mosa
