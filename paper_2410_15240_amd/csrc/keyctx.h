// Per-key device context for multi-chain AES-256-GCM on gfx950.
//
// One KeyCtx lives in device memory per (device, key). It is produced by the
// setup kernel and read by every decrypt/encrypt launch for that key.
//
// Data layout conventions (shared by every kernel in this library):
//   * A 16-byte block is held as 4 little-endian u32 words exactly as a
//     16-byte-aligned vector load returns them: word j = bytes 4j..4j+3 with
//     byte 4j in bits 0..7. AES state column j is word j (row r in bits 8r..).
//   * GF(2^128) elements use the same little-endian-word form for storage,
//     table lookups and XOR. Only the shift-based routines used during setup
//     switch to a big-endian-word form (GCM's bit 0, the coefficient of x^0,
//     is the most significant bit of byte 0).
//   * Round key rk[4r + j] is column j of round key r in the same word form.
#pragma once
#include <stdint.h>

namespace fastrack {

constexpr int kTab4Pos = 32;    // nibble positions of a 128-bit operand
constexpr int kTab4Ent = 16;    // values of a nibble
constexpr int kSquares = 32;    // H^(2^t), t = 0..31 (chains are < 2^32 blocks)
constexpr int kOddMul = 3;      // odd multipliers j = 3, 5, 7 of the segment weights
constexpr int kOddT = 31;       // H^(j 2^t), t = 0..30 (3 . 2^30 < 2^32)

struct Tab4 {                   // 4-bit positional multiplication table of a fixed Y:
    uint32_t e[kTab4Pos][kTab4Ent][4];   // e[p][v] = (nibble v at degrees 4p..4p+3) . Y
};

struct KeyCtx {
    uint32_t rk[60];            // AES-256 round keys (FIPS-197 key expansion)
    uint32_t rk16[60];          // the same with the words of rounds 1..13 (rk[4..55]) rotated by 16 bits
    uint32_t t0[256];           // T0[x] = {02}S(x) | S(x)<<8 | S(x)<<16 | {03}S(x)<<24
    uint8_t sbox[256];
    uint32_t h[4];              // H = AES_K(0^128)
    uint32_t h8k[8][4];         // h8k[i] = H^(8 (i + 1)): H^8, H^16, ..., H^64
    uint32_t hsq[kSquares][4];        // hsq[t] = H^(2^t)
    Tab4 h1_tab;                // table of H
    Tab4 sq_tab[kSquares];      // sq_tab[t]: table of H^(2^t) (t = 0..5 also combine the lanes of an item)
    // 8-bit positional tables of H^8, H^16, ..., H^64, the 16 byte positions of one value
    // side by side: g16[i][v][k] = (byte v at byte k) . H^(8 (i + 1)). g16[L/8 - 1] is the
    // Horner multiplier H^L of L = 16, 32, 64 lanes per chain; g16[0..6] also weight the
    // partial sums of an item's eight-lane groups at the end of the lane combine.
    uint32_t g16[8][256][16][4];
    // A segment weight H^(m 2^g) is applied one nonzero base-8 digit d of m at a time:
    // H^(d 2^(g + 3i)) is a square for d = 1, 2, 4 and H^(j 2^t) with j = 3, 5, 7 otherwise
    // (6 = 3 . 2). odd_tab[i][t]: table of H^((2 i + 3) 2^t).
    Tab4 odd_tab[kOddMul][kOddT];
};

}  // namespace fastrack
