// Bitsliced AES-256 building blocks: 32 blocks per 32-bit lane.
//
// State layout: x[8p + b] holds bit b (b = 0 is the least significant bit) of
// state byte p (FIPS-197 byte order, p = 4c + r for column c, row r) of 32
// independent blocks, block s in bit s of every word. SubBytes is then 16
// copies of a Boolean circuit over 8 words, ShiftRows a renaming of bytes, and
// MixColumns / AddRoundKey XORs of whole words, so one 32-bit operation works
// on 32 blocks at once and no table is read.
//
// The S-box circuit is Boyar and Peralta's depth-16 circuit of 128 gates (34 AND,
// 90 XOR, 4 XNOR; J. Boyar and R. Peralta, "A depth-16 circuit for the AES
// S-box", IFIP SEC 2012): a linear top layer (T1..T27), a nonlinear middle
// (M1..M63) that inverts in the tower field GF((2^4)^2), and a linear bottom
// layer (L0..L29) that also applies the S-box's affine map.
//
// Plain C++ on uint32_t, so the same header builds for the GPU and, in the
// tests, for the host. The S-box runs as 88 three-input gates (v_bitop3_b32 on
// gfx950), a covering of the 128 two-input gates found by gen_sbox_lut3.py.
#pragma once
#include <stdint.h>

namespace fastrack {
namespace bs {

// A three-input logic gate: bit i of the result is bit (a_i*4 + b_i*2 + c_i) of
// the truth table TT (one v_bitop3_b32 on gfx950).
template <uint32_t TT>
__host__ __device__ inline uint32_t lut3(uint32_t a, uint32_t b, uint32_t c)
{
#if defined(__HIP_DEVICE_COMPILE__)
    return __builtin_amdgcn_bitop3_b32(a, b, c, TT);
#else
    uint32_t r = 0;
    for (int i = 0; i < 8; ++i)
        if ((TT >> i) & 1u)
            r |= ((i & 4) ? a : ~a) & ((i & 2) ? b : ~b) & ((i & 1) ? c : ~c);
    return r;
#endif
}

// SubBytes of one bitsliced byte in place: x[b] is bit b of 32 bytes. The
// 128-gate circuit mapped onto three-input gates by gen_sbox_lut3.py (which
// holds the gate list and checks the mapping on all 256 inputs).
__host__ __device__ inline void sbox(uint32_t *x)
{
#include "sbox_lut3.inc"
}

__host__ __device__ inline uint32_t xor3(uint32_t a, uint32_t b, uint32_t c) { return lut3<0x96>(a, b, c); }

// Bit b of a round-key word as a mask: 0 or all ones (the same key bit for every block).
__host__ __device__ inline uint32_t key_bit(uint32_t w, int b)
{
    return (uint32_t)((int32_t)(w << (31 - b)) >> 31);
}

// Output column c of ShiftRows, SubBytes, MixColumns and AddRoundKey: the four
// input bytes that ShiftRows brings into column c (row i from column c + i) go
// through the S-box circuit in place, then out[8(4c+i) + k] = bit k of row i of
// MixColumns xor the round key, kw being round-key word c (byte 4c + i in bits
// 8i .. 8i+7). With a_i the row-i byte and t_i = a_i xor a_(i+1) (indices mod 4),
// row i is {02}.t_i xor a_(i+1) xor t_(i+2) = {02}a_i xor {03}a_(i+1) xor a_(i+2)
// xor a_(i+3); multiplying by {02} moves bit k to k + 1 and folds bit 7 into bits
// 0, 1, 3 and 4 (x^8 = x^4 + x^3 + x + 1). Columns take disjoint input bytes, so
// a round can run column by column with only the bytes still unread kept.
__host__ __device__ inline void sub_mix_column(uint32_t *in, uint32_t *out, int c, uint32_t kw)
{
    uint32_t *a[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        a[i] = in + 8 * (4 * ((c + i) & 3) + i);
        sbox(a[i]);
    }
    uint32_t t[4][8];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int k = 0; k < 8; ++k)
            t[i][k] = a[i][k] ^ a[(i + 1) & 3][k];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        uint32_t *o = out + 8 * (4 * c + i);
        const uint32_t *t0 = t[i], *t2 = t[(i + 2) & 3], *a1 = a[(i + 1) & 3];
        // two three-input XORs per output bit, the key bit (a scalar) in the second
        o[0] = xor3(xor3(t0[7], a1[0], t2[0]), key_bit(kw, 8 * i + 0), 0u);
        o[1] = xor3(xor3(t0[0], t0[7], a1[1]), t2[1], key_bit(kw, 8 * i + 1));
        o[2] = xor3(xor3(t0[1], a1[2], t2[2]), key_bit(kw, 8 * i + 2), 0u);
        o[3] = xor3(xor3(t0[2], t0[7], a1[3]), t2[3], key_bit(kw, 8 * i + 3));
        o[4] = xor3(xor3(t0[3], t0[7], a1[4]), t2[4], key_bit(kw, 8 * i + 4));
        o[5] = xor3(xor3(t0[4], a1[5], t2[5]), key_bit(kw, 8 * i + 5), 0u);
        o[6] = xor3(xor3(t0[5], a1[6], t2[6]), key_bit(kw, 8 * i + 6), 0u);
        o[7] = xor3(xor3(t0[6], a1[7], t2[7]), key_bit(kw, 8 * i + 7), 0u);
    }
}

// A middle round (rounds 1..13): SubBytes, ShiftRows, MixColumns, AddRoundKey
// with the round-key words kw[0..3]; `in` is consumed.
__host__ __device__ inline void round(uint32_t *in, uint32_t *out, const uint32_t *kw)
{
#pragma unroll
    for (int c = 0; c < 4; ++c)
        sub_mix_column(in, out, c, kw[c]);
}

// The last round: SubBytes, ShiftRows and AddRoundKey (no MixColumns).
__host__ __device__ inline void final_round(uint32_t *in, uint32_t *out, const uint32_t *kw)
{
#pragma unroll
    for (int c = 0; c < 4; ++c)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            uint32_t *a = in + 8 * (4 * ((c + i) & 3) + i);
            sbox(a);
#pragma unroll
            for (int k = 0; k < 8; ++k)
                out[8 * (4 * c + i) + k] = a[k] ^ key_bit(kw[c], 8 * i + k);
        }
}

// 32 x 32 bit-matrix transpose in place: afterwards bit i of a[s] is what bit s of
// a[i] was. Five levels; level j swaps, for every pair of rows k and k + j with
// k & j == 0, the bits of row k whose index has j set with the bits of row k + j
// whose index has it clear.
__host__ __device__ inline void transpose32(uint32_t *a)
{
    constexpr uint32_t masks[5] = {0x0000FFFFu, 0x00FF00FFu, 0x0F0F0F0Fu, 0x33333333u, 0x55555555u};
#pragma unroll
    for (int lv = 0; lv < 5; ++lv) {
        const int j = 16 >> lv;
        const uint32_t m = masks[lv];
#pragma unroll
        for (int k = 0; k < 32; ++k) {
            if (k & j)
                continue;
            const uint32_t t = ((a[k] >> j) ^ a[k + j]) & m;
            a[k + j] ^= t;
            a[k] ^= t << j;
        }
    }
}

}  // namespace bs
}  // namespace fastrack
