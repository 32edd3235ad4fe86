// Host build of the library's compile-time tables and set-up arithmetic for the
// CPU tests: the S-box and T0 table that the key set-up copies, the columns of
// the squaring map S^k (k = 1..8) that it applies to H, the GF(2^128) helpers
// they are made from (multiply by x^k, square), and the split of a segment weight
// into table factors, all evaluated on the host from the same constexpr
// functions the device code uses. Only the host
// pass is built (no device code runs).
#include <stdint.h>
#include <string.h>

#include "aes_dev.h"
#include "gf128_dev.h"

using namespace fastrack;

namespace {
constexpr SboxTables kSbox = make_sbox_tables();
constexpr FrobTable kFrob = make_frob_table();

// 16 GCM bytes (byte 0 holds degrees 0..7, degree 0 in its top bit) <-> the
// big-endian-word form of the helpers.
u4 load_be(const uint8_t *b)
{
    u4 v{};
    for (int j = 0; j < 4; ++j)
        v.w[j] = ((uint32_t)b[4 * j] << 24) | ((uint32_t)b[4 * j + 1] << 16) | ((uint32_t)b[4 * j + 2] << 8) |
                 b[4 * j + 3];
    return v;
}

void store_be(const u4 &v, uint8_t *b)
{
    for (int j = 0; j < 4; ++j)
        for (int i = 0; i < 4; ++i)
            b[4 * j + i] = (uint8_t)(v.w[j] >> (24 - 8 * i));
}
}  // namespace

extern "C" {

void tab_sbox(uint8_t *sbox, uint32_t *t0)
{
    memcpy(sbox, kSbox.sbox, 256);
    memcpy(t0, kSbox.t0, 256 * 4);
}

// out[((k - 1) * 128 + i) * 16 ..] = S^k(x^i) as GCM bytes.
void tab_frob(uint8_t *out)
{
    for (int k = 0; k < 8; ++k)
        for (int i = 0; i < 128; ++i)
            store_be(kFrob.c[k][i], out + 16 * (128 * k + i));
}

void tab_mul_xk(const uint8_t *y, int k, uint8_t *out)
{
    store_be(be_mul_xk_any(load_be(y), k), out);
}

void tab_square(const uint8_t *y, uint8_t *out)
{
    store_be(be_square(load_be(y)), out);
}

// The factors H^(j[k] 2^t[k]) that weight a segment by H^(m 2^g), in the order the
// kernel applies them; returns their count (octal_digits(m) is returned in *digits).
int tab_weight_steps(uint32_t m, uint32_t g, uint32_t *j, uint32_t *t, uint32_t *digits)
{
    *digits = octal_digits(m);
    int n = 0;
    while (m) {
        const WeightStep w = weight_step(m, g);
        j[n] = w.j;
        t[n] = w.t;
        ++n;
    }
    return n;
}

}  // extern "C"
