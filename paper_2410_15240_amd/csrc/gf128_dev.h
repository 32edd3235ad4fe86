// GF(2^128) arithmetic of GCM on the device.
//
// GHASH multiplies by the hash subkey H in GF(2^128) with the reduction
// polynomial x^128 + x^7 + x^2 + x + 1; the bit of degree 0 is the most
// significant bit of the first byte (SP 800-38D 6.3; the paper's Galois-field
// authentication, section 3.2). A multiplication by a FIXED element Y is a
// GF(2)-linear map, so it is evaluated with precomputed positional tables:
// X . Y = XOR over positions p of table[p][digit_p(X)], which needs no carries
// and no carry-less multiply instruction (CDNA has none).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "keyctx.h"

namespace fastrack {

struct u4 {
    uint32_t w[4];
};

__device__ __forceinline__ uint32_t xor3(uint32_t a, uint32_t b, uint32_t c)
{
    return __builtin_amdgcn_bitop3_b32(a, b, c, 0x96);
}

__device__ __forceinline__ uint32_t bswap32(uint32_t x)
{
    return __builtin_amdgcn_perm(0u, x, 0x00010203u);
}

// ---- big-endian-word helpers (setup only) -------------------------------
// In big-endian-word form w[0] bit 31 is degree 0 and w[3] bit 0 is degree 127.

__device__ __forceinline__ u4 to_be(const u4 &a)
{
    u4 r;
    for (int j = 0; j < 4; ++j)
        r.w[j] = bswap32(a.w[j]);
    return r;
}

__device__ __forceinline__ u4 from_be(const u4 &a) { return to_be(a); }

// Y . x^k for 0 <= k <= 64, in big-endian-word form. Multiplying by x^k moves
// every coefficient k degrees up (k bits toward the end of the string). The k
// bits that pass degree 127 form F(x) . x^128, and x^128 = 1 + x + x^2 + x^7,
// so they come back as F xor F.x xor F.x^2 xor F.x^7. For k <= 64, F has
// degree < 64 and the fold cannot overflow again.
__host__ __device__ constexpr u4 be_mul_xk(const u4 &y, int k)
{
    if (k == 0)
        return y;
    // 128-bit value v = w0:w1:w2:w3 (w0 most significant as an integer).
    uint64_t hi = ((uint64_t)y.w[0] << 32) | y.w[1];
    uint64_t lo = ((uint64_t)y.w[2] << 32) | y.w[3];
    uint64_t nhi = 0, nlo = 0, f = 0;
    if (k < 64) {
        f = lo << (64 - k);               // the k bits that fall off, left-aligned
        nlo = (lo >> k) | (hi << (64 - k));
        nhi = hi >> k;
    } else {                              // k == 64
        f = lo;
        nlo = hi;
        nhi = 0;
    }
    // f holds F left-aligned in a 64-bit word: degree d of F sits at bit 63-d,
    // which is exactly where degree d lives in the high word. Fold F.(1+x+x^2+x^7).
    uint64_t r_hi = f ^ (f >> 1) ^ (f >> 2) ^ (f >> 7);
    uint64_t r_lo = (f << 63) ^ (f << 62) ^ (f << 57);
    nhi ^= r_hi;
    nlo ^= r_lo;
    u4 r{};
    r.w[0] = (uint32_t)(nhi >> 32);
    r.w[1] = (uint32_t)nhi;
    r.w[2] = (uint32_t)(nlo >> 32);
    r.w[3] = (uint32_t)nlo;
    return r;
}

// Y . x^k for 0 <= k <= 127 (two steps of at most 64).
__host__ __device__ constexpr u4 be_mul_xk_any(const u4 &y, int k)
{
    if (k <= 64)
        return be_mul_xk(y, k);
    return be_mul_xk(be_mul_xk(y, 64), k - 64);
}

// Bit i of w moved to bit 2i + 1 of a 64-bit word (the other bits zero).
__host__ __device__ constexpr uint64_t spread_odd(uint32_t w)
{
    uint64_t x = w;
    x = (x | (x << 16)) & 0x0000FFFF0000FFFFull;
    x = (x | (x << 8)) & 0x00FF00FF00FF00FFull;
    x = (x | (x << 4)) & 0x0F0F0F0F0F0F0F0Full;
    x = (x | (x << 2)) & 0x3333333333333333ull;
    x = (x | (x << 1)) & 0x5555555555555555ull;
    return x << 1;
}

// Y^2 in big-endian-word form (setup only). Squaring is linear over GF(2): the
// coefficient of degree d moves to degree 2d. With V = w0:w1:w2:w3 as a 128-bit
// integer (degree d at bit 127 - d) the square is the 256-bit integer with bit p of
// V at bit 2p + 1; its upper half holds degrees 0..127 and its lower half F the
// degrees 128..255, which come back as F . x^128 = F . (1 + x + x^2 + x^7).
__host__ __device__ constexpr u4 be_square(const u4 &y)
{
    const uint64_t h0 = spread_odd(y.w[0]), h1 = spread_odd(y.w[1]);
    const uint64_t f0 = spread_odd(y.w[2]), f1 = spread_odd(y.w[3]);
    const u4 f = {{(uint32_t)(f0 >> 32), (uint32_t)f0, (uint32_t)(f1 >> 32), (uint32_t)f1}};
    const u4 a = be_mul_xk(f, 1), b = be_mul_xk(f, 2), c = be_mul_xk(f, 7);
    u4 r{};
    r.w[0] = (uint32_t)(h0 >> 32) ^ f.w[0] ^ a.w[0] ^ b.w[0] ^ c.w[0];
    r.w[1] = (uint32_t)h0 ^ f.w[1] ^ a.w[1] ^ b.w[1] ^ c.w[1];
    r.w[2] = (uint32_t)(h1 >> 32) ^ f.w[2] ^ a.w[2] ^ b.w[2] ^ c.w[2];
    r.w[3] = (uint32_t)h1 ^ f.w[3] ^ a.w[3] ^ b.w[3] ^ c.w[3];
    return r;
}

// XOR of x over each aligned group of 2^LL lanes, in every lane of the group: a
// butterfly of VALU moves. Quad permutes pair lanes 1 and 2 apart; once each quad
// (eight) holds one sum, the half-row (row) mirror pairs it with the neighbouring
// quad (eight); the half-row and half-wave swaps return both halves, whose XOR is
// a lane's own value xor its partner's.
template <int LL>
__device__ __forceinline__ uint32_t group_xor_sum(uint32_t x)
{
    if constexpr (LL >= 1)
        x ^= __builtin_amdgcn_update_dpp(0u, x, 0xB1, 0xF, 0xF, false);   // quad_perm [1,0,3,2]
    if constexpr (LL >= 2)
        x ^= __builtin_amdgcn_update_dpp(0u, x, 0x4E, 0xF, 0xF, false);   // quad_perm [2,3,0,1]
    if constexpr (LL >= 3)
        x ^= __builtin_amdgcn_update_dpp(0u, x, 0x141, 0xF, 0xF, false);  // row_half_mirror
    if constexpr (LL >= 4)
        x ^= __builtin_amdgcn_update_dpp(0u, x, 0x140, 0xF, 0xF, false);  // row_mirror
    if constexpr (LL >= 5) {
        const auto sw = __builtin_amdgcn_permlane16_swap(x, x, false, false);
        x = sw[0] ^ sw[1];
    }
    if constexpr (LL >= 6) {
        const auto sw = __builtin_amdgcn_permlane32_swap(x, x, false, false);
        x = sw[0] ^ sw[1];
    }
    return x;
}

// Segment weights H^(m 2^g), one nonzero base-8 digit of m at a time: digit d at
// position i is the factor H^(d 2^(g + 3i)) = H^(j 2^t), with j the odd part of d
// (1, 3, 5 or 7) and t = g + 3i + log2(d / j). The key context holds a table for
// every such factor (squares for j = 1, odd multiples otherwise).
__host__ __device__ constexpr uint32_t octal_digits(uint32_t m)   // nonzero base-8 digits of m
{
    return (uint32_t)__builtin_popcount((m | (m >> 1) | (m >> 2)) & 0x49249249u);
}

struct WeightStep {
    uint32_t j, t;   // the factor H^(j 2^t)
};

// The factor of m's lowest nonzero digit (m > 0), which is then cleared from m.
__host__ __device__ constexpr WeightStep weight_step(uint32_t &m, uint32_t g)
{
    const uint32_t i = (uint32_t)__builtin_ctz(m) / 3;
    const uint32_t d = (m >> (3 * i)) & 7u;
    const uint32_t e = (uint32_t)__builtin_ctz(d);
    m &= ~(7u << (3 * i));
    return WeightStep{d >> e, g + 3 * i + e};
}

// The columns of S^k, S(V) = V^2, for k = 1..8, in big-endian-word form:
// c[k - 1][i] = S^k(x^i). Squaring is GF(2)-linear, so V^(2^k) is the XOR of the
// columns of V's set degrees. Evaluated by the compiler (key-independent).
struct FrobTable {
    u4 c[8][128];
};

constexpr FrobTable make_frob_table()
{
    FrobTable t{};
    for (int i = 0; i < 128; ++i) {
        u4 v{};
        v.w[i >> 5] = 1u << (31 - (i & 31));
        for (int k = 0; k < 8; ++k) {
            v = be_square(v);
            t.c[k][i] = v;
        }
    }
    return t;
}

// A GF(2)-linear map M on GF(2^128) held by one wave (setup only): lane l keeps
// the columns M(x^l) and M(x^(l+64)) in big-endian-word form, and M(V) is a
// select per lane and a wave-wide XOR. All lanes must be active.
struct WaveLinear {
    u4 c0, c1;
    __device__ void load(const u4 *cols, uint32_t lane)
    {
        c0 = cols[lane];
        c1 = cols[lane + 64];
    }
    __device__ u4 apply(const u4 &v, uint32_t lane) const
    {
        const uint32_t b0 = (lane < 32 ? v.w[0] : v.w[1]) >> (31 - (lane & 31));
        const uint32_t b1 = (lane < 32 ? v.w[2] : v.w[3]) >> (31 - (lane & 31));
        const uint32_t m0 = 0u - (b0 & 1u), m1 = 0u - (b1 & 1u);
        u4 r;
#pragma unroll
        for (int j = 0; j < 4; ++j)
            r.w[j] = group_xor_sum<6>((c0.w[j] & m0) ^ (c1.w[j] & m1));
        return r;
    }
};

// ---- little-endian-word table multiplies -------------------------------

// X . Y with Y's 4-bit positional table. Word j holds bytes 4j..4j+3, and
// byte 4j+b holds nibble positions 8j+2b (high nibble) and 8j+2b+1 (low).
// Register indices stay compile-time constants so nothing is spilled to memory.
__device__ inline u4 mul_tab4(const u4 &x, const Tab4 *__restrict__ t)
{
    u4 z = {{0u, 0u, 0u, 0u}};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const uint32_t w = x.w[j];
#pragma unroll 2
        for (int b = 0; b < 4; ++b) {
            const uint32_t byte = (w >> (8 * b)) & 0xFFu;
            const int p = 8 * j + 2 * b;
            const uint4 ea = *reinterpret_cast<const uint4 *>(t->e[p][byte >> 4]);
            const uint4 eb = *reinterpret_cast<const uint4 *>(t->e[p + 1][byte & 0xFu]);
            z.w[0] = xor3(z.w[0], ea.x, eb.x);
            z.w[1] = xor3(z.w[1], ea.y, eb.y);
            z.w[2] = xor3(z.w[2], ea.z, eb.z);
            z.w[3] = xor3(z.w[3], ea.w, eb.w);
        }
    }
    return z;
}

// The same product with the eight lookups of each word in flight together
// (the scheduling barrier keeps the batches apart, so at most 32 VGPRs hold
// table entries): for latency-bound callers that run few multiplies in sequence.
__device__ inline u4 mul_tab4_b8(const u4 &x, const Tab4 *__restrict__ t)
{
    u4 z = {{0u, 0u, 0u, 0u}};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const uint32_t w = x.w[j];
        uint4 e[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            const uint32_t byte = (w >> (8 * (q >> 1))) & 0xFFu;
            const uint32_t nib = (q & 1) ? (byte & 0xFu) : (byte >> 4);
            e[q] = *reinterpret_cast<const uint4 *>(t->e[8 * j + q][nib]);
        }
#pragma unroll
        for (int q = 0; q < 8; q += 2) {
            z.w[0] = xor3(z.w[0], e[q].x, e[q + 1].x);
            z.w[1] = xor3(z.w[1], e[q].y, e[q + 1].y);
            z.w[2] = xor3(z.w[2], e[q].z, e[q + 1].z);
            z.w[3] = xor3(z.w[3], e[q].w, e[q + 1].w);
        }
        __builtin_amdgcn_sched_barrier(0);
    }
    return z;
}

// X . Y with Y's 8-bit positional table in global memory, entry (byte position k,
// value v) at t[v * 16 + k], the 16 lookups in two batches of eight: for the few
// lanes of the last levels of a lane combine.
__device__ inline u4 mul_tab8_b8(const u4 &x, const uint4 *__restrict__ t)
{
    u4 z = {{0u, 0u, 0u, 0u}};
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        uint4 e[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            const int k = 8 * h + q;
            const uint32_t v = (x.w[k >> 2] >> (8 * (k & 3))) & 0xFFu;
            e[q] = t[v * 16 + k];
        }
#pragma unroll
        for (int q = 0; q < 8; q += 2) {
            z.w[0] = xor3(z.w[0], e[q].x, e[q + 1].x);
            z.w[1] = xor3(z.w[1], e[q].y, e[q + 1].y);
            z.w[2] = xor3(z.w[2], e[q].z, e[q + 1].z);
            z.w[3] = xor3(z.w[3], e[q].w, e[q + 1].w);
        }
        __builtin_amdgcn_sched_barrier(0);
    }
    return z;
}

__device__ __forceinline__ u4 xor4(const u4 &a, const u4 &b)
{
    u4 r;
    for (int j = 0; j < 4; ++j)
        r.w[j] = a.w[j] ^ b.w[j];
    return r;
}

// XOR of a value over the 64 lanes of a wave; every lane receives the result.
__device__ inline u4 wave_xor(u4 v)
{
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1)
        for (int j = 0; j < 4; ++j)
            v.w[j] ^= __shfl_xor(v.w[j], off, 64);
    return v;
}

}  // namespace fastrack
