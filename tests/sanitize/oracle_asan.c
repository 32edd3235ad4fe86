/* Sanitizer driver for the CPU oracle (test infrastructure): exercises its GCM and
 * multi-chain entry points on exactly sized heap buffers, so that any read or write
 * past an end, any use of uninitialised size arithmetic or any undefined integer
 * operation is reported by AddressSanitizer / UndefinedBehaviorSanitizer.
 * Exit status 0 when every round trip matches and no tamper goes unnoticed. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

void orc_gcm_encrypt(const uint8_t key[32], const uint8_t iv[12], const uint8_t *P, uint64_t len, const uint8_t *A,
                     uint64_t alen, int bitserial, uint8_t *C, uint8_t T[16]);
int orc_gcm_decrypt(const uint8_t key[32], const uint8_t iv[12], const uint8_t *C, uint64_t len, const uint8_t *A,
                    uint64_t alen, const uint8_t T[16], int bitserial, uint8_t *P);
uint64_t orc_num_chains(uint64_t len, uint64_t chain_bytes);
int orc_chains_encrypt(const uint8_t key[32], const uint8_t base_iv[12], uint64_t chain_bytes, const uint8_t *pt,
                       uint64_t len, const uint8_t *aad, uint64_t aad_bytes, uint8_t *ct, uint8_t *tags, int bitserial,
                       int nthreads);
int orc_chains_decrypt(const uint8_t key[32], const uint8_t base_iv[12], uint64_t chain_bytes, const uint8_t *ct,
                       uint64_t len, const uint8_t *tags, const uint8_t *aad, uint64_t aad_bytes, uint8_t *pt,
                       uint8_t *ok, int bitserial, int nthreads);

static uint64_t rng = 0x9E3779B97F4A7C15ull;
static uint8_t rbyte(void)
{
    rng ^= rng << 13;
    rng ^= rng >> 7;
    rng ^= rng << 17;
    return (uint8_t)rng;
}
static uint8_t *rbuf(uint64_t n)
{
    uint8_t *p = malloc(n ? n : 1);
    for (uint64_t i = 0; i < n; ++i)
        p[i] = rbyte();
    return p;
}

int main(void)
{
    uint8_t key[32], iv[12];
    for (int i = 0; i < 32; ++i)
        key[i] = rbyte();
    for (int i = 0; i < 12; ++i)
        iv[i] = rbyte();
    int fails = 0;
    /* single messages: every length class, AAD lengths, both GF multiplies */
    const uint64_t lens[] = {0, 1, 15, 16, 17, 31, 33, 255, 4095, 4096, 4097, 65536 + 7};
    const uint64_t alens[] = {0, 1, 13, 16, 32, 100};
    for (unsigned li = 0; li < sizeof lens / sizeof *lens; ++li)
        for (unsigned ai = 0; ai < sizeof alens / sizeof *alens; ++ai)
            for (int bs = 0; bs < 2; ++bs) {
                const uint64_t n = lens[li], a = alens[ai];
                if (bs && n > 4096)
                    continue;   /* the bit-serial multiply is slow */
                uint8_t *P = rbuf(n), *A = rbuf(a), *C = malloc(n ? n : 1), *Q = malloc(n ? n : 1), T[16];
                orc_gcm_encrypt(key, iv, P, n, a ? A : NULL, a, bs, C, T);
                if (!orc_gcm_decrypt(key, iv, C, n, a ? A : NULL, a, T, bs, Q) || (n && memcmp(P, Q, n)))
                    ++fails;
                T[15] ^= 1;
                if (orc_gcm_decrypt(key, iv, C, n, a ? A : NULL, a, T, bs, Q))
                    ++fails;
                free(P); free(A); free(C); free(Q);
            }
    /* multi-chain: chain sizes that divide and do not divide the length, AAD, threads */
    const uint64_t mlen[] = {1, 4096, 65536 + 48, 100000 + 5};
    const uint64_t chains[] = {16, 4096, 65536};
    for (unsigned li = 0; li < sizeof mlen / sizeof *mlen; ++li)
        for (unsigned ci = 0; ci < sizeof chains / sizeof *chains; ++ci)
            for (int nt = 1; nt <= 4; nt += 3) {
                const uint64_t n = mlen[li], c = chains[ci], k = orc_num_chains(n, c), a = 32;
                uint8_t *P = rbuf(n), *A = rbuf(k * a), *C = malloc(n), *Q = malloc(n), *T = malloc(16 * k),
                        *ok = malloc(k);
                if (orc_chains_encrypt(key, iv, c, P, n, A, a, C, T, 0, nt) ||
                    orc_chains_decrypt(key, iv, c, C, n, T, A, a, Q, ok, 0, nt) || memcmp(P, Q, n))
                    ++fails;
                for (uint64_t i = 0; i < k; ++i)
                    fails += ok[i] != 1;
                C[n - 1] ^= 0x80;   /* the last chain must fail, the others pass */
                orc_chains_decrypt(key, iv, c, C, n, T, A, a, Q, ok, 0, nt);
                for (uint64_t i = 0; i < k; ++i)
                    fails += ok[i] != (i + 1 < k);
                free(P); free(A); free(C); free(Q); free(T); free(ok);
            }
    printf("oracle sanitizer driver: %d failures\n", fails);
    return fails != 0;
}
