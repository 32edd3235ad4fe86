// AES-256 on the device (FIPS-197), in the 32-bit T-table formulation.
//
// The paper's decryption kernel is AES in counter mode (section 3.2, "The AES
// block cipher", and the AES-CTR figure; section 5.2): every counter block is
// enciphered independently. One round maps column j of the state to
//   T0[s0(col j)] ^ rotl8(T0[s1(col j+1)]) ^ rotl16(T0[s2(col j+2)]) ^ rotl24(T0[s3(col j+3)]) ^ rk
// where T0 folds SubBytes and the MixColumns column (02,01,01,03) into one
// 32-bit entry, the rotations give the other three rows of MixColumns, and the
// column offsets implement ShiftRows. The final round has no MixColumns and
// takes S(x), which is byte 1 of T0[x].
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "gf128_dev.h"

namespace fastrack {

// ---- S-box and T0 (FIPS-197 5.1.1), generated on the device -------------

__device__ inline uint32_t gf8_mul_dev(uint32_t a, uint32_t b)
{
    uint32_t p = 0;
    for (int i = 0; i < 8; ++i) {
        p ^= (b & 1u) ? a : 0u;
        a = ((a << 1) ^ ((a & 0x80u) ? 0x11Bu : 0u)) & 0xFFu;
        b >>= 1;
    }
    return p;
}

// Multiplicative inverse as x^254 (x^255 = 1 for x != 0; 0 maps to 0).
__device__ inline uint32_t gf8_inv_dev(uint32_t x)
{
    uint32_t r = 1, base = x, e = 254;
    while (e) {
        if (e & 1u)
            r = gf8_mul_dev(r, base);
        base = gf8_mul_dev(base, base);
        e >>= 1;
    }
    return x ? r : 0u;
}

__device__ __forceinline__ uint32_t rotl8b(uint32_t b, int n)
{
    return ((b << n) | (b >> (8 - n))) & 0xFFu;
}

// Affine map: b ^ rotl(b,1) ^ rotl(b,2) ^ rotl(b,3) ^ rotl(b,4) ^ 0x63.
__device__ inline uint32_t sbox_entry(uint32_t x)
{
    uint32_t b = gf8_inv_dev(x);
    return b ^ rotl8b(b, 1) ^ rotl8b(b, 2) ^ rotl8b(b, 3) ^ rotl8b(b, 4) ^ 0x63u;
}

__device__ inline uint32_t t0_entry(uint32_t s)
{
    uint32_t s2 = ((s << 1) ^ ((s & 0x80u) ? 0x11Bu : 0u)) & 0xFFu;
    uint32_t s3 = s2 ^ s;
    return s2 | (s << 8) | (s << 16) | (s3 << 24);
}

// ---- key expansion (FIPS-197 5.2, Nk = 8, Nr = 14) ------------------------
// Words in the library's little-endian form: byte 0 of the word is bits 0..7.
// RotWord is a rotation right by 8 in this form; Rcon goes into byte 0.
template <class SB>
__device__ inline void expand_key_256(const uint32_t key[8], uint32_t rk[60], SB sbox)
{
    for (int i = 0; i < 8; ++i)
        rk[i] = key[i];
    uint32_t rcon = 1;
    for (int i = 8; i < 60; ++i) {
        uint32_t t = rk[i - 1];
        if ((i & 7) == 0) {
            t = (t >> 8) | (t << 24);
            t = sbox(t & 0xFF) | (sbox((t >> 8) & 0xFF) << 8) | (sbox((t >> 16) & 0xFF) << 16) |
                (sbox(t >> 24) << 24);
            t ^= rcon;
            rcon = ((rcon << 1) ^ ((rcon & 0x80u) ? 0x11Bu : 0u)) & 0xFFu;
        } else if ((i & 7) == 4) {
            t = sbox(t & 0xFF) | (sbox((t >> 8) & 0xFF) << 8) | (sbox((t >> 16) & 0xFF) << 16) |
                (sbox(t >> 24) << 24);
        }
        rk[i] = rk[i - 8] ^ t;
    }
}

__device__ __forceinline__ uint32_t rotl32(uint32_t x, int n)
{
    return (x << n) | (x >> (32 - n));
}

// Generic T-table cipher: T(x) returns T0[x] for a byte x. Used where speed is
// irrelevant (setup, per-chain tag mask); the streaming kernel has its own
// LDS-addressed copy of the round.
template <class LK>
__device__ inline u4 aes256_encrypt_tt(const u4 &in, const uint32_t *__restrict__ rk, LK T)
{
    uint32_t s0 = in.w[0] ^ rk[0], s1 = in.w[1] ^ rk[1], s2 = in.w[2] ^ rk[2], s3 = in.w[3] ^ rk[3];
    for (int r = 1; r < 14; ++r) {
        uint32_t n0 = T(s0 & 0xFF) ^ rotl32(T((s1 >> 8) & 0xFF), 8) ^ rotl32(T((s2 >> 16) & 0xFF), 16) ^
                      rotl32(T(s3 >> 24), 24) ^ rk[4 * r + 0];
        uint32_t n1 = T(s1 & 0xFF) ^ rotl32(T((s2 >> 8) & 0xFF), 8) ^ rotl32(T((s3 >> 16) & 0xFF), 16) ^
                      rotl32(T(s0 >> 24), 24) ^ rk[4 * r + 1];
        uint32_t n2 = T(s2 & 0xFF) ^ rotl32(T((s3 >> 8) & 0xFF), 8) ^ rotl32(T((s0 >> 16) & 0xFF), 16) ^
                      rotl32(T(s1 >> 24), 24) ^ rk[4 * r + 2];
        uint32_t n3 = T(s3 & 0xFF) ^ rotl32(T((s0 >> 8) & 0xFF), 8) ^ rotl32(T((s1 >> 16) & 0xFF), 16) ^
                      rotl32(T(s2 >> 24), 24) ^ rk[4 * r + 3];
        s0 = n0;
        s1 = n1;
        s2 = n2;
        s3 = n3;
    }
    auto S = [&](uint32_t x) { return (T(x) >> 8) & 0xFFu; };
    u4 o;
    o.w[0] = (S(s0 & 0xFF) | (S((s1 >> 8) & 0xFF) << 8) | (S((s2 >> 16) & 0xFF) << 16) | (S(s3 >> 24) << 24)) ^ rk[56];
    o.w[1] = (S(s1 & 0xFF) | (S((s2 >> 8) & 0xFF) << 8) | (S((s3 >> 16) & 0xFF) << 16) | (S(s0 >> 24) << 24)) ^ rk[57];
    o.w[2] = (S(s2 & 0xFF) | (S((s3 >> 8) & 0xFF) << 8) | (S((s0 >> 16) & 0xFF) << 16) | (S(s1 >> 24) << 24)) ^ rk[58];
    o.w[3] = (S(s3 & 0xFF) | (S((s0 >> 8) & 0xFF) << 8) | (S((s1 >> 16) & 0xFF) << 16) | (S(s2 >> 24) << 24)) ^ rk[59];
    return o;
}

}  // namespace fastrack
