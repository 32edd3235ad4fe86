// Host build of the library's bitsliced AES building blocks
// (paper_2410_15240_amd/csrc/aes_bitslice.h) for the CPU tests: the header is
// plain C++, so with the HIP qualifiers defined away it compiles with g++.
// Slicing and unslicing here are plain bit loops (test harness code); the
// S-box circuit, the round functions and the transpose are the library's.
#define __host__
#define __device__
#include <stdint.h>
#include <string.h>

#include "aes_bitslice.h"

using namespace fastrack::bs;

extern "C" {

// The S-box circuit on every byte value: out[v] = S(v).
void bs_sbox_all(uint8_t *out)
{
    for (int g = 0; g < 8; ++g) {          // values 32g .. 32g + 31, value 32g + s in bit s
        uint32_t x[8] = {0};
        for (int s = 0; s < 32; ++s)
            for (int b = 0; b < 8; ++b)
                x[b] |= (uint32_t)(((32 * g + s) >> b) & 1) << s;
        sbox(x);
        for (int s = 0; s < 32; ++s) {
            uint8_t v = 0;
            for (int b = 0; b < 8; ++b)
                v |= (uint8_t)(((x[b] >> s) & 1) << b);
            out[32 * g + s] = v;
        }
    }
}

void bs_transpose(const uint32_t *in, uint32_t *out)
{
    uint32_t a[32];
    memcpy(a, in, sizeof a);
    transpose32(a);
    memcpy(out, a, sizeof a);
}

// AES-256 encryption of 32 blocks (in[16s .. 16s+15] is block s) with the 15
// round keys rk[16r .. 16r+15] in FIPS-197 byte order.
void bs_encrypt32(const uint8_t *rk, const uint8_t *in, uint8_t *out)
{
    uint32_t x[128] = {0}, y[128], kw[15][4];
    for (int r = 0; r < 15; ++r)
        for (int c = 0; c < 4; ++c)
            kw[r][c] = (uint32_t)rk[16 * r + 4 * c] | (uint32_t)rk[16 * r + 4 * c + 1] << 8 |
                       (uint32_t)rk[16 * r + 4 * c + 2] << 16 | (uint32_t)rk[16 * r + 4 * c + 3] << 24;
    for (int s = 0; s < 32; ++s)
        for (int j = 0; j < 128; ++j)
            x[j] |= (uint32_t)((in[16 * s + j / 8] >> (j % 8)) & 1) << s;
    for (int j = 0; j < 128; ++j)
        x[j] ^= key_bit(kw[0][j / 32], j % 32);
    for (int r = 1; r < 14; ++r) {
        round(x, y, kw[r]);
        memcpy(x, y, sizeof x);
    }
    final_round(x, y, kw[14]);
    for (int s = 0; s < 32; ++s)
        for (int p = 0; p < 16; ++p) {
            uint8_t v = 0;
            for (int b = 0; b < 8; ++b)
                v |= (uint8_t)(((y[8 * p + b] >> s) & 1) << b);
            out[16 * s + p] = v;
        }
}
}
