/*
 * gcm_oracle.c -- TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT.
 *
 * A plain, slow, obviously-correct CPU reference for multi-chain AES-256-GCM.
 * Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
 * load it. The GPU library shares no code, header, table or generator with it.
 *
 * What it computes and where each piece is defined:
 *   - AES-256 block cipher: FIPS-197 (S-box from the GF(2^8) inverse and the
 *     affine map, section 5.1.1; key expansion, section 5.2; Cipher, section 5.1;
 *     InvCipher, section 5.3, used only as a self-test). The paper uses AES with a
 *     256-bit key as the block cipher of AES-GCM (section 3.2, "The AES block
 *     cipher"; section 5.4 "Confidentiality").
 *   - GF(2^128) multiplication: SP 800-38D section 6.3, Algorithm 1 (bit-serial);
 *     a 4-bit table variant (Shoup's method) for bulk speed, checked against
 *     the bit-serial one by the tests.
 *   - GHASH: SP 800-38D section 6.4, Algorithm 2 (the Horner chain the paper
 *     draws in its GMAC figure, section 3.2 "Authentication with Galois Field").
 *   - GCTR: SP 800-38D section 6.5, Algorithm 3 (the AES-CTR keystream of
 *     section 3.2 and its figure of AES-CTR).
 *   - GCM-AE / GCM-AD with a 96-bit IV: SP 800-38D sections 7.1 and 7.2,
 *     Algorithms 4 and 5, with a full 128-bit tag (section 1.2 of the paper:
 *     "128-bit MAC tag").
 *   - Multi-chaining authentication (paper section 5.2): the buffer is split
 *     into chains of chain_bytes; chain i is an independent GCM message with
 *     its own IV, its own AAD and its own tag. Readings of what the paper leaves
 *     open:
 *       IV_i = base_IV XOR (0^32 || [i]_64)   (the chain index, big-endian, in
 *                                             IV bytes 4..11; chains are 0-based)
 *       A_i  = aad[i*aad_bytes .. (i+1)*aad_bytes)   (caller-supplied)
 *       the last chain is shorter when chain_bytes does not divide the length.
 *     On verification failure the plaintext is still produced and ok[i] = 0
 *     (the paper's eager evaluation consumes plaintext before or without the
 *     tag check, section 5.3).
 */
#include <stdint.h>
#include <stddef.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define EXPORT __attribute__((visibility("default")))

/* ------------------------------------------------------------------------ */
/* GF(2^8) with the AES polynomial x^8 + x^4 + x^3 + x + 1 (FIPS-197 4.2).   */
/* ------------------------------------------------------------------------ */

/* Multiplication by x (FIPS-197 4.2.1, "xtime"). */
static uint8_t xtime(uint8_t b)
{
    return (uint8_t)((b << 1) ^ ((b & 0x80) ? 0x1b : 0x00));
}

/* General multiplication as repeated xtime (FIPS-197 4.2.1). */
static uint8_t gf8_mul(uint8_t a, uint8_t b)
{
    uint8_t p = 0;
    for (int i = 0; i < 8; i++) {
        if (b & 1)
            p ^= a;
        a = xtime(a);
        b >>= 1;
    }
    return p;
}

/* Multiplicative inverse by exhaustive search; 0 maps to 0 (FIPS-197 5.1.1). */
static uint8_t gf8_inv(uint8_t a)
{
    if (a == 0)
        return 0;
    for (int b = 1; b < 256; b++)
        if (gf8_mul(a, (uint8_t)b) == 1)
            return (uint8_t)b;
    return 0; /* not reached: every nonzero element has an inverse */
}

static uint8_t SBOX[256];
static uint8_t INV_SBOX[256];

/*
 * S-box (FIPS-197 5.1.1): take the inverse b in GF(2^8), then apply the affine
 * map b'_i = b_i ^ b_{i+4} ^ b_{i+5} ^ b_{i+6} ^ b_{i+7} ^ c_i (indices mod 8),
 * c = 0x63.
 */
__attribute__((constructor)) static void build_sbox(void)
{
    for (int x = 0; x < 256; x++) {
        uint8_t b = gf8_inv((uint8_t)x);
        uint8_t s = 0;
        for (int i = 0; i < 8; i++) {
            int bit = ((b >> i) ^ (b >> ((i + 4) % 8)) ^ (b >> ((i + 5) % 8)) ^
                       (b >> ((i + 6) % 8)) ^ (b >> ((i + 7) % 8)) ^ (0x63 >> i)) & 1;
            s |= (uint8_t)(bit << i);
        }
        SBOX[x] = s;
        INV_SBOX[s] = (uint8_t)x;
    }
}

EXPORT void orc_sbox(uint8_t out[256], uint8_t inv_out[256])
{
    memcpy(out, SBOX, 256);
    memcpy(inv_out, INV_SBOX, 256);
}

/* ------------------------------------------------------------------------ */
/* AES-256 (FIPS-197): Nk = 8 key words, Nr = 14 rounds, Nb = 4 columns.     */
/* The state is s[r][c] = in[r + 4c].                                       */
/* ------------------------------------------------------------------------ */

#define NK 8
#define NR 14
#define NW (4 * (NR + 1)) /* 60 round-key words */

/* Key expansion (FIPS-197 5.2). Word w[i] is 4 bytes w[i][0..3]. */
static void key_expansion(const uint8_t key[32], uint8_t w[NW][4])
{
    uint8_t rcon = 0x01; /* Rcon[i/Nk] = x^(i/Nk - 1), built by xtime */
    for (int i = 0; i < NK; i++)
        memcpy(w[i], key + 4 * i, 4);
    for (int i = NK; i < NW; i++) {
        uint8_t t[4];
        memcpy(t, w[i - 1], 4);
        if (i % NK == 0) {
            /* SubWord(RotWord(temp)) xor Rcon */
            uint8_t t0 = t[0];
            t[0] = (uint8_t)(SBOX[t[1]] ^ rcon);
            t[1] = SBOX[t[2]];
            t[2] = SBOX[t[3]];
            t[3] = SBOX[t0];
            rcon = xtime(rcon);
        } else if (i % NK == 4) {
            for (int k = 0; k < 4; k++)
                t[k] = SBOX[t[k]];
        }
        for (int k = 0; k < 4; k++)
            w[i][k] = (uint8_t)(w[i - NK][k] ^ t[k]);
    }
}

EXPORT void orc_aes256_key_expansion(const uint8_t key[32], uint8_t out[NW * 4])
{
    uint8_t w[NW][4];
    key_expansion(key, w);
    memcpy(out, w, sizeof w);
}

static void add_round_key(uint8_t s[4][4], const uint8_t w[NW][4], int round)
{
    for (int c = 0; c < 4; c++)
        for (int r = 0; r < 4; r++)
            s[r][c] ^= w[4 * round + c][r];
}

static void sub_bytes(uint8_t s[4][4])
{
    for (int r = 0; r < 4; r++)
        for (int c = 0; c < 4; c++)
            s[r][c] = SBOX[s[r][c]];
}

static void inv_sub_bytes(uint8_t s[4][4])
{
    for (int r = 0; r < 4; r++)
        for (int c = 0; c < 4; c++)
            s[r][c] = INV_SBOX[s[r][c]];
}

/* Row r is rotated left by r positions (FIPS-197 5.1.2). */
static void shift_rows(uint8_t s[4][4])
{
    for (int r = 1; r < 4; r++) {
        uint8_t t[4];
        for (int c = 0; c < 4; c++)
            t[c] = s[r][(c + r) % 4];
        memcpy(s[r], t, 4);
    }
}

static void inv_shift_rows(uint8_t s[4][4])
{
    for (int r = 1; r < 4; r++) {
        uint8_t t[4];
        for (int c = 0; c < 4; c++)
            t[(c + r) % 4] = s[r][c];
        memcpy(s[r], t, 4);
    }
}

/* Each column times the fixed polynomial {03}x^3 + {01}x^2 + {01}x + {02} (FIPS-197 5.1.3). */
static void mix_columns(uint8_t s[4][4])
{
    for (int c = 0; c < 4; c++) {
        uint8_t a0 = s[0][c], a1 = s[1][c], a2 = s[2][c], a3 = s[3][c];
        /* {02}.a = xtime(a); {03}.a = xtime(a) ^ a */
        s[0][c] = (uint8_t)(xtime(a0) ^ (xtime(a1) ^ a1) ^ a2 ^ a3);
        s[1][c] = (uint8_t)(a0 ^ xtime(a1) ^ (xtime(a2) ^ a2) ^ a3);
        s[2][c] = (uint8_t)(a0 ^ a1 ^ xtime(a2) ^ (xtime(a3) ^ a3));
        s[3][c] = (uint8_t)((xtime(a0) ^ a0) ^ a1 ^ a2 ^ xtime(a3));
    }
}

/* Inverse: times {0b}x^3 + {0d}x^2 + {09}x + {0e} (FIPS-197 5.3.3). */
static void inv_mix_columns(uint8_t s[4][4])
{
    for (int c = 0; c < 4; c++) {
        uint8_t a0 = s[0][c], a1 = s[1][c], a2 = s[2][c], a3 = s[3][c];
        s[0][c] = (uint8_t)(gf8_mul(a0, 0x0e) ^ gf8_mul(a1, 0x0b) ^ gf8_mul(a2, 0x0d) ^ gf8_mul(a3, 0x09));
        s[1][c] = (uint8_t)(gf8_mul(a0, 0x09) ^ gf8_mul(a1, 0x0e) ^ gf8_mul(a2, 0x0b) ^ gf8_mul(a3, 0x0d));
        s[2][c] = (uint8_t)(gf8_mul(a0, 0x0d) ^ gf8_mul(a1, 0x09) ^ gf8_mul(a2, 0x0e) ^ gf8_mul(a3, 0x0b));
        s[3][c] = (uint8_t)(gf8_mul(a0, 0x0b) ^ gf8_mul(a1, 0x0d) ^ gf8_mul(a2, 0x09) ^ gf8_mul(a3, 0x0e));
    }
}

/* Optional count of block-cipher invocations (for the paper's cost accounting). */
static int count_enabled;
static uint64_t aes_calls;

EXPORT void orc_count_aes(int enable)
{
    __atomic_store_n(&aes_calls, 0, __ATOMIC_SEQ_CST);
    count_enabled = enable;
}

EXPORT uint64_t orc_aes_calls(void)
{
    return __atomic_load_n(&aes_calls, __ATOMIC_SEQ_CST);
}

/* Cipher (FIPS-197 5.1). */
static void cipher(const uint8_t w[NW][4], const uint8_t in[16], uint8_t out[16])
{
    uint8_t s[4][4];
    if (count_enabled)
        __atomic_fetch_add(&aes_calls, 1, __ATOMIC_RELAXED);
    for (int r = 0; r < 4; r++)
        for (int c = 0; c < 4; c++)
            s[r][c] = in[r + 4 * c];
    add_round_key(s, w, 0);
    for (int round = 1; round < NR; round++) {
        sub_bytes(s);
        shift_rows(s);
        mix_columns(s);
        add_round_key(s, w, round);
    }
    sub_bytes(s);
    shift_rows(s);
    add_round_key(s, w, NR);
    for (int r = 0; r < 4; r++)
        for (int c = 0; c < 4; c++)
            out[r + 4 * c] = s[r][c];
}

/* InvCipher (FIPS-197 5.3); only a self-test of the forward cipher. */
static void inv_cipher(const uint8_t w[NW][4], const uint8_t in[16], uint8_t out[16])
{
    uint8_t s[4][4];
    for (int r = 0; r < 4; r++)
        for (int c = 0; c < 4; c++)
            s[r][c] = in[r + 4 * c];
    add_round_key(s, w, NR);
    for (int round = NR - 1; round >= 1; round--) {
        inv_shift_rows(s);
        inv_sub_bytes(s);
        add_round_key(s, w, round);
        inv_mix_columns(s);
    }
    inv_shift_rows(s);
    inv_sub_bytes(s);
    add_round_key(s, w, 0);
    for (int r = 0; r < 4; r++)
        for (int c = 0; c < 4; c++)
            out[r + 4 * c] = s[r][c];
}

EXPORT void orc_aes256_encrypt_block(const uint8_t key[32], const uint8_t in[16], uint8_t out[16])
{
    uint8_t w[NW][4];
    key_expansion(key, w);
    cipher(w, in, out);
}

EXPORT void orc_aes256_decrypt_block(const uint8_t key[32], const uint8_t in[16], uint8_t out[16])
{
    uint8_t w[NW][4];
    key_expansion(key, w);
    inv_cipher(w, in, out);
}

/* ------------------------------------------------------------------------ */
/* GF(2^128) as used by GCM (SP 800-38D 6.3).                                */
/* A block is a 128-bit string; bit 0 is the most significant bit of byte 0 */
/* and is the coefficient of x^0. R = 11100001 || 0^120.                      */
/* ------------------------------------------------------------------------ */

/* Algorithm 1: X . Y, bit by bit. */
EXPORT void orc_gf128_mul_bitserial(const uint8_t X[16], const uint8_t Y[16], uint8_t out[16])
{
    uint8_t Z[16] = {0};
    uint8_t V[16];
    memcpy(V, Y, 16);
    for (int i = 0; i < 128; i++) {
        if ((X[i / 8] >> (7 - i % 8)) & 1)
            for (int k = 0; k < 16; k++)
                Z[k] ^= V[k];
        int lsb = V[15] & 1; /* bit 127 of V */
        for (int k = 15; k > 0; k--)
            V[k] = (uint8_t)((V[k] >> 1) | (V[k - 1] << 7));
        V[0] >>= 1;
        if (lsb)
            V[0] ^= 0xE1;
    }
    memcpy(out, Z, 16);
}

/*
 * Table variant (Shoup's 4-bit method), used for bulk GHASH so that the
 * multi-chain oracle runs in seconds. Elements are held as two big-endian
 * 64-bit halves (hi = bytes 0..7). Writing X = sum_k N_k(x) x^(4k), where N_k is
 * the nibble holding degrees 4k..4k+3, Horner from the top nibble gives
 *   Z <- Z . x^4  xor  N_k . Y.
 * M[v] = N . Y for nibble value v; RED[f] = the reduction of the 4 bits that a
 * shift by x^4 pushes past degree 127. Both tables are filled with the
 * bit-serial multiply above, so they follow from Algorithm 1.
 */
typedef struct {
    uint64_t hi, lo;
} u128;

static u128 load128(const uint8_t b[16])
{
    u128 v = {0, 0};
    for (int i = 0; i < 8; i++) {
        v.hi = (v.hi << 8) | b[i];
        v.lo = (v.lo << 8) | b[8 + i];
    }
    return v;
}

static void store128(u128 v, uint8_t b[16])
{
    for (int i = 7; i >= 0; i--) {
        b[i] = (uint8_t)v.hi;
        b[8 + i] = (uint8_t)v.lo;
        v.hi >>= 8;
        v.lo >>= 8;
    }
}

typedef struct {
    u128 M[16];
    u128 RED[16];
} gf_table;

static void gf_table_init(gf_table *t, const uint8_t Y[16])
{
    for (int v = 0; v < 16; v++) {
        /* nibble value v at degrees 0..3: bit 3 of v is degree 0 (MSB first) */
        uint8_t N[16] = {0};
        N[0] = (uint8_t)(v << 4);
        uint8_t p[16];
        orc_gf128_mul_bitserial(N, Y, p);
        t->M[v] = load128(p);
    }
    for (int f = 0; f < 16; f++) {
        /* f holds degrees 124..127 (bit 3 of f = degree 124); times x^4 */
        uint8_t F[16] = {0};
        F[15] = (uint8_t)f;
        uint8_t X4[16] = {0};
        X4[0] = 0x08; /* x^4 */
        uint8_t p[16];
        orc_gf128_mul_bitserial(F, X4, p);
        t->RED[f] = load128(p);
    }
}

static u128 gf_table_mul(const gf_table *t, u128 X)
{
    u128 Z = {0, 0};
    for (int k = 31; k >= 0; k--) {
        /* Z <- Z . x^4 : shift the bit string right by 4 and fold the overflow */
        int f = (int)(Z.lo & 0xF);
        Z.lo = (Z.lo >> 4) | (Z.hi << 60);
        Z.hi >>= 4;
        Z.hi ^= t->RED[f].hi;
        Z.lo ^= t->RED[f].lo;
        /* nibble k covers degrees 4k..4k+3 */
        uint64_t word = (k < 16) ? X.hi : X.lo;
        int shift = 60 - 4 * (k % 16);
        int v = (int)((word >> shift) & 0xF);
        Z.hi ^= t->M[v].hi;
        Z.lo ^= t->M[v].lo;
    }
    return Z;
}

EXPORT void orc_gf128_mul_table(const uint8_t X[16], const uint8_t Y[16], uint8_t out[16])
{
    gf_table t;
    gf_table_init(&t, Y);
    store128(gf_table_mul(&t, load128(X)), out);
}

/* ------------------------------------------------------------------------ */
/* GHASH (SP 800-38D 6.4, Algorithm 2): Y_0 = 0, Y_j = (Y_{j-1} xor X_j) . H */
/* ------------------------------------------------------------------------ */

typedef struct {
    uint8_t H[16];
    int bitserial; /* 1: Algorithm 1 for every product; 0: the 4-bit table */
    gf_table tab;
    uint8_t Y[16];
} ghash_state;

static void ghash_init(ghash_state *g, const uint8_t H[16], int bitserial)
{
    memcpy(g->H, H, 16);
    g->bitserial = bitserial;
    if (!bitserial)
        gf_table_init(&g->tab, H);
    memset(g->Y, 0, 16);
}

static void ghash_block(ghash_state *g, const uint8_t X[16])
{
    uint8_t t[16];
    for (int k = 0; k < 16; k++)
        t[k] = g->Y[k] ^ X[k];
    if (g->bitserial)
        orc_gf128_mul_bitserial(t, g->H, g->Y);
    else
        store128(gf_table_mul(&g->tab, load128(t)), g->Y);
}

/* Feed len bytes as ceil(len/16) blocks, the last one padded with zero bits. */
static void ghash_bytes(ghash_state *g, const uint8_t *data, uint64_t len)
{
    for (uint64_t off = 0; off < len; off += 16) {
        uint8_t blk[16] = {0};
        uint64_t n = (len - off < 16) ? len - off : 16;
        memcpy(blk, data + off, (size_t)n);
        ghash_block(g, blk);
    }
}

/* GHASH_H over whole blocks, as defined (len must be a multiple of 16). */
EXPORT int orc_ghash(const uint8_t H[16], const uint8_t *X, uint64_t nbytes, int bitserial, uint8_t out[16])
{
    if (nbytes % 16)
        return -1;
    ghash_state g;
    ghash_init(&g, H, bitserial);
    for (uint64_t off = 0; off < nbytes; off += 16)
        ghash_block(&g, X + off);
    memcpy(out, g.Y, 16);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* GCTR (SP 800-38D 6.5, Algorithm 3).                                       */
/* ------------------------------------------------------------------------ */

/* inc_32: increment the rightmost 32 bits mod 2^32 (big-endian), SP 800-38D 6.2. */
static void inc32(uint8_t cb[16])
{
    uint32_t c = ((uint32_t)cb[12] << 24) | ((uint32_t)cb[13] << 16) | ((uint32_t)cb[14] << 8) | cb[15];
    c += 1;
    cb[12] = (uint8_t)(c >> 24);
    cb[13] = (uint8_t)(c >> 16);
    cb[14] = (uint8_t)(c >> 8);
    cb[15] = (uint8_t)c;
}

static void gctr(const uint8_t w[NW][4], const uint8_t icb[16], const uint8_t *in, uint64_t len, uint8_t *out)
{
    uint8_t cb[16];
    memcpy(cb, icb, 16);
    for (uint64_t off = 0; off < len; off += 16) {
        uint8_t ks[16];
        cipher(w, cb, ks);
        /* the last partial block uses the most significant bytes of the keystream */
        uint64_t n = (len - off < 16) ? len - off : 16;
        for (uint64_t k = 0; k < n; k++)
            out[off + k] = in[off + k] ^ ks[k];
        inc32(cb);
    }
}

EXPORT void orc_gctr(const uint8_t key[32], const uint8_t icb[16], const uint8_t *in, uint64_t len, uint8_t *out)
{
    uint8_t w[NW][4];
    key_expansion(key, w);
    gctr(w, icb, in, len, out);
}

/* ------------------------------------------------------------------------ */
/* GCM with a 96-bit IV (SP 800-38D 7.1 / 7.2, Algorithms 4 and 5).           */
/* ------------------------------------------------------------------------ */

static void put_be64(uint8_t *p, uint64_t v)
{
    for (int i = 7; i >= 0; i--) {
        p[i] = (uint8_t)v;
        v >>= 8;
    }
}

/*
 * S = GHASH_H(A || 0^v || C || 0^u || [len(A)]_64 || [len(C)]_64), lengths in
 * bits; T = S xor CIPH_K(J0) (the full 128 bits: MSB_128 of GCTR(J0, S)).
 */
static void gcm_tag(const uint8_t w[NW][4], const uint8_t H[16], const uint8_t J0[16], const uint8_t *A,
                    uint64_t alen, const uint8_t *C, uint64_t clen, int bitserial, uint8_t T[16])
{
    ghash_state g;
    ghash_init(&g, H, bitserial);
    ghash_bytes(&g, A, alen);
    ghash_bytes(&g, C, clen);
    uint8_t lens[16];
    put_be64(lens, alen * 8);
    put_be64(lens + 8, clen * 8);
    ghash_block(&g, lens);
    uint8_t ej0[16];
    cipher(w, J0, ej0);
    for (int k = 0; k < 16; k++)
        T[k] = g.Y[k] ^ ej0[k];
}

static void gcm_h(const uint8_t w[NW][4], uint8_t H[16])
{
    uint8_t zero[16] = {0};
    cipher(w, zero, H); /* H = CIPH_K(0^128) */
}

static void gcm_j0(const uint8_t iv[12], uint8_t J0[16])
{
    memcpy(J0, iv, 12); /* J0 = IV || 0^31 || 1 */
    J0[12] = 0;
    J0[13] = 0;
    J0[14] = 0;
    J0[15] = 1;
}

static void gcm_ae(const uint8_t w[NW][4], const uint8_t H[16], const uint8_t iv[12], const uint8_t *P,
                   uint64_t len, const uint8_t *A, uint64_t alen, int bitserial, uint8_t *C, uint8_t T[16])
{
    uint8_t J0[16], icb[16];
    gcm_j0(iv, J0);
    memcpy(icb, J0, 16);
    inc32(icb);
    gctr(w, icb, P, len, C);
    gcm_tag(w, H, J0, A, alen, C, len, bitserial, T);
}

/* Returns 1 if the tag verifies. P is always written (see the header). */
static int gcm_ad(const uint8_t w[NW][4], const uint8_t H[16], const uint8_t iv[12], const uint8_t *C,
                  uint64_t len, const uint8_t *A, uint64_t alen, const uint8_t T[16], int bitserial, uint8_t *P)
{
    uint8_t J0[16], icb[16], Tp[16];
    gcm_j0(iv, J0);
    memcpy(icb, J0, 16);
    inc32(icb);
    gctr(w, icb, C, len, P);
    gcm_tag(w, H, J0, A, alen, C, len, bitserial, Tp);
    int diff = 0;
    for (int k = 0; k < 16; k++) /* all 16 bytes are compared */
        diff |= Tp[k] ^ T[k];
    return diff == 0;
}

EXPORT void orc_gcm_encrypt(const uint8_t key[32], const uint8_t iv[12], const uint8_t *P, uint64_t len,
                            const uint8_t *A, uint64_t alen, int bitserial, uint8_t *C, uint8_t T[16])
{
    uint8_t w[NW][4], H[16];
    key_expansion(key, w);
    gcm_h(w, H);
    gcm_ae(w, H, iv, P, len, A, alen, bitserial, C, T);
}

EXPORT int orc_gcm_decrypt(const uint8_t key[32], const uint8_t iv[12], const uint8_t *C, uint64_t len,
                           const uint8_t *A, uint64_t alen, const uint8_t T[16], int bitserial, uint8_t *P)
{
    uint8_t w[NW][4], H[16];
    key_expansion(key, w);
    gcm_h(w, H);
    return gcm_ad(w, H, iv, C, len, A, alen, T, bitserial, P);
}

/* ------------------------------------------------------------------------ */
/* Multi-chaining authentication (paper section 5.2).                        */
/* ------------------------------------------------------------------------ */

EXPORT uint64_t orc_num_chains(uint64_t len, uint64_t chain_bytes)
{
    return chain_bytes ? (len + chain_bytes - 1) / chain_bytes : 0;
}

/* IV_i = base_IV xor (0^32 || [i]_64). */
EXPORT void orc_chain_iv(const uint8_t base_iv[12], uint64_t i, uint8_t iv[12])
{
    uint8_t idx[8];
    put_be64(idx, i);
    memcpy(iv, base_iv, 12);
    for (int k = 0; k < 8; k++)
        iv[4 + k] ^= idx[k];
}

static int set_threads(int nthreads)
{
#ifdef _OPENMP
    return nthreads > 0 ? nthreads : omp_get_max_threads();
#else
    (void)nthreads;
    return 1;
#endif
}

/*
 * Encrypt every chain: ct[off_i .. off_i+len_i) and tags[16 i .. 16 i + 16).
 * Chains are independent messages, so they are spread over threads; the result
 * does not depend on the thread count.
 */
EXPORT int orc_chains_encrypt(const uint8_t key[32], const uint8_t base_iv[12], uint64_t chain_bytes,
                              const uint8_t *pt, uint64_t len, const uint8_t *aad, uint64_t aad_bytes,
                              uint8_t *ct, uint8_t *tags, int bitserial, int nthreads)
{
    if (chain_bytes == 0)
        return -1;
    uint8_t w[NW][4], H[16];
    key_expansion(key, w);
    gcm_h(w, H);
    int64_t n = (int64_t)orc_num_chains(len, chain_bytes);
    int nt = set_threads(nthreads);
    (void)nt;
#pragma omp parallel for schedule(dynamic, 1) num_threads(nt)
    for (int64_t i = 0; i < n; i++) {
        uint64_t off = (uint64_t)i * chain_bytes;
        uint64_t li = (len - off < chain_bytes) ? len - off : chain_bytes;
        uint8_t iv[12];
        orc_chain_iv(base_iv, (uint64_t)i, iv);
        gcm_ae(w, H, iv, pt + off, li, aad ? aad + (uint64_t)i * aad_bytes : NULL, aad_bytes, bitserial,
               ct + off, tags + 16 * (uint64_t)i);
    }
    return 0;
}

/* Decrypt + verify every chain; ok[i] = 1 accept / 0 reject. */
EXPORT int orc_chains_decrypt(const uint8_t key[32], const uint8_t base_iv[12], uint64_t chain_bytes,
                              const uint8_t *ct, uint64_t len, const uint8_t *tags, const uint8_t *aad,
                              uint64_t aad_bytes, uint8_t *pt, uint8_t *ok, int bitserial, int nthreads)
{
    if (chain_bytes == 0)
        return -1;
    uint8_t w[NW][4], H[16];
    key_expansion(key, w);
    gcm_h(w, H);
    int64_t n = (int64_t)orc_num_chains(len, chain_bytes);
    int nt = set_threads(nthreads);
    (void)nt;
#pragma omp parallel for schedule(dynamic, 1) num_threads(nt)
    for (int64_t i = 0; i < n; i++) {
        uint64_t off = (uint64_t)i * chain_bytes;
        uint64_t li = (len - off < chain_bytes) ? len - off : chain_bytes;
        uint8_t iv[12];
        orc_chain_iv(base_iv, (uint64_t)i, iv);
        ok[i] = (uint8_t)gcm_ad(w, H, iv, ct + off, li, aad ? aad + (uint64_t)i * aad_bytes : NULL, aad_bytes,
                                tags + 16 * (uint64_t)i, bitserial, pt + off);
    }
    return 0;
}

/*
 * Decrypt + verify a chosen subset of chains of a large buffer (for sampled
 * checks at full size). pt_out receives the chosen chains back to back, each
 * chain_bytes long (a short last chain leaves the remainder untouched). Each
 * chosen chain is the same independent GCM message (section 5.2) that
 * orc_chains_decrypt checks at its index; bitserial selects Algorithm 1 or the
 * table multiply exactly as there.
 */
EXPORT int orc_chains_decrypt_subset(const uint8_t key[32], const uint8_t base_iv[12], uint64_t chain_bytes,
                                     const uint8_t *ct, uint64_t len, const uint8_t *tags, const uint8_t *aad,
                                     uint64_t aad_bytes, const uint64_t *idx, uint64_t nidx, uint8_t *pt_out,
                                     uint8_t *ok_out, int bitserial, int nthreads)
{
    if (chain_bytes == 0)
        return -1;
    uint64_t n = orc_num_chains(len, chain_bytes);
    for (uint64_t j = 0; j < nidx; j++)
        if (idx[j] >= n)
            return -1;
    uint8_t w[NW][4], H[16];
    key_expansion(key, w);
    gcm_h(w, H);
    int nt = set_threads(nthreads);
    (void)nt;
#pragma omp parallel for schedule(dynamic, 1) num_threads(nt)
    for (int64_t j = 0; j < (int64_t)nidx; j++) {
        uint64_t i = idx[j];
        uint64_t off = i * chain_bytes;
        uint64_t li = (len - off < chain_bytes) ? len - off : chain_bytes;
        uint8_t iv[12];
        orc_chain_iv(base_iv, i, iv);
        ok_out[j] = (uint8_t)gcm_ad(w, H, iv, ct + off, li, aad ? aad + i * aad_bytes : NULL, aad_bytes,
                                    tags + 16 * i, bitserial, pt_out + (uint64_t)j * chain_bytes);
    }
    return 0;
}

/* Threads the OpenMP runtime would use by default (reported by the bench). */
EXPORT int orc_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
