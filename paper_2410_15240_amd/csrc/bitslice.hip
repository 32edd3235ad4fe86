// Bitsliced AES-256-CTR keystream kernel for gfx950 (FIPS-197 rounds on 32
// blocks per lane, no tables): the keystream mode of the multi-chain
// AES-256-GCM library computed without T-table lookups. The paper's decryption
// kernel is AES-CTR (sections 3.2 and 5.2); its one-time-pad variant generates
// the keystream ahead of the ciphertext (section 5.3, "Parallel AES
// evaluation"). Built on its own, with the compiler's default scheduler.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "aes_bitslice.h"
#include "chain_dev.h"
#include "keyctx.h"
#include "launch.h"

namespace fastrack {

// ===========================================================================
// Bitsliced AES-256-CTR keystream (no tables)
// ===========================================================================
//
// The keystream mode computed with the bitsliced round functions of
// aes_bitslice.h instead of T-table lookups: every lane holds 32 blocks, one
// per bit of 128 state words. A wave pass covers 2048 consecutive data blocks
// t0 .. t0+2047 of one chain, block t0 + 64 s + l in bit s of lane l, so each of
// the 32 stores of a pass writes 64 consecutive blocks (1 KiB). Counter block
// IV_i || [t + 2]_32: with c = t0 + l + 2 fixed per lane, bits 0..5 of the
// counter are the lane's and bits 6..31 are (c >> 6) + s, added to the slice
// index in bitsliced form (a ripple-carry over 26 bits). The round keys are
// uniform, so each key bit is a scalar mask of 0 or all ones.
constexpr int kBsThreads = 256;
typedef uint32_t v4u __attribute__((ext_vector_type(4)));
constexpr uint32_t kBsPassBlocks = 2048;

__device__ __forceinline__ uint32_t bit_mask(uint32_t w, uint32_t b)
{
    return bs::key_bit(w, (int)b);   // 0 or all ones
}

// Two waves per SIMD: the 128-word state and the S-box temporaries take up to 256
// VGPRs (at 168, three waves per SIMD, the rounds spill).
constexpr int kBsWavesPerSimd = 2;

__global__ __launch_bounds__(kBsThreads, kBsWavesPerSimd) void bs_keystream_kernel(GcmLaunch p, uint32_t ppc,
                                                                     uint64_t n_passes)
{
    const KeyCtx *__restrict__ c = p.ctx;
    const uint32_t *__restrict__ rk = c->rk;
    const uint32_t lane = threadIdx.x & 63;
    const uint64_t nwaves = (uint64_t)gridDim.x * (kBsThreads / 64);
    const uint64_t full_passes = (uint64_t)(p.n_chains - 1) * ppc;
    for (uint64_t pass = __builtin_amdgcn_readfirstlane(blockIdx.x * (kBsThreads / 64) + (threadIdx.x >> 6));
         pass < n_passes; pass += nwaves) {
        uint32_t chain, k;
        if (pass < full_passes) {
            chain = (uint32_t)(pass / ppc);
            k = (uint32_t)(pass - (uint64_t)chain * ppc);
        } else {
            chain = p.n_chains - 1;
            k = (uint32_t)(pass - full_passes);
        }
        const bool last = chain == p.n_chains - 1;
        const uint32_t q = last ? p.q_last : p.qc;
        const uint32_t tail = last ? (uint32_t)(p.last_len & 15) : 0u;
        const uint32_t t0 = k * kBsPassBlocks;
        uint32_t iv[3];
        chain_iv(p, p.chain_base + chain, iv);

        // AddRoundKey of round 0 on the counter blocks, bitsliced.
        uint32_t x[128];
#pragma unroll
        for (int j = 0; j < 3; ++j) {
            const uint32_t v = iv[j] ^ rk[j];            // bytes 4j .. 4j+3, the same in every block
#pragma unroll
            for (int b = 0; b < 32; ++b)
                x[32 * j + b] = bit_mask(v, b);          // byte 4j + b/8, bit b%8
        }
        const uint32_t cl = t0 + lane + 2u;
        uint32_t cw[32];                                  // bit i of the counter, one word per bit
#pragma unroll
        for (int i = 0; i < 6; ++i)
            cw[i] = bit_mask(cl, i);
        {
            const uint32_t u = cl >> 6;
            constexpr uint32_t pat[5] = {0xAAAAAAAAu, 0xCCCCCCCCu, 0xF0F0F0F0u, 0xFF00FF00u, 0xFFFF0000u};
            uint32_t carry = 0;
#pragma unroll
            for (int j = 0; j < 26; ++j) {
                const uint32_t s = j < 5 ? pat[j] : 0u, uj = bit_mask(u, j);
                cw[6 + j] = s ^ uj ^ carry;
                carry = (s & uj) | (carry & (s ^ uj));
            }
        }
        // bytes 12..15 hold the counter big-endian: byte 15 its bits 0..7
#pragma unroll
        for (int pb = 12; pb < 16; ++pb)
#pragma unroll
            for (int b = 0; b < 8; ++b)
                x[8 * pb + b] = cw[8 * (15 - pb) + b] ^ bit_mask(rk[3], 8 * (pb - 12) + b);

        uint32_t y[128];
        bs::round(x, y, rk + 4);
#pragma unroll 1
        for (int r = 2; r < 14; r += 2) {   // two rounds per iteration: x -> y -> x, no copies
            const uint32_t k0[4] = {rk[4 * r], rk[4 * r + 1], rk[4 * r + 2], rk[4 * r + 3]};
            const uint32_t k1[4] = {rk[4 * r + 4], rk[4 * r + 5], rk[4 * r + 6], rk[4 * r + 7]};
            bs::round(y, x, k0);
            bs::round(x, y, k1);
        }
        bs::final_round(y, x, rk + 56);
        // Unslice: after the transpose, x[32 w + s] is word w of block s.
#pragma unroll
        for (int w = 0; w < 4; ++w)
            bs::transpose32(x + 32 * w);
        uint8_t *dst = p.out + (uint64_t)chain * p.chain_bytes;
#pragma unroll
        for (int sl = 0; sl < 32; ++sl) {
            const uint32_t t = t0 + 64u * sl + lane;
            if (t < q) {
                const u4 o = {{x[sl], x[32 + sl], x[64 + sl], x[96 + sl]}};
                if (tail == 0 || t + 1 < q) {   // non-temporal, as the T-table kernel stores
                    const v4u ov = {o.w[0], o.w[1], o.w[2], o.w[3]};
                    __builtin_nontemporal_store(ov, reinterpret_cast<v4u *>(dst) + t);
                }
                else
                    store_bytes(dst + 16ull * t, o, tail);
            }
        }
    }
}

hipError_t launch_bs_keystream(const GcmLaunch &p, int num_cu, hipStream_t s)
{
    if (p.n_chains == 0)
        return hipSuccess;
    const uint32_t ppc = (p.qc + kBsPassBlocks - 1) / kBsPassBlocks;
    const uint32_t ppc_last = (p.q_last + kBsPassBlocks - 1) / kBsPassBlocks;
    const uint64_t n_passes = (uint64_t)(p.n_chains - 1) * ppc + ppc_last;
    uint64_t wgs = (n_passes + kBsThreads / 64 - 1) / (kBsThreads / 64);
    if (wgs > (uint64_t)num_cu * kBsWavesPerSimd)
        wgs = (uint64_t)num_cu * kBsWavesPerSimd;
    hipLaunchKernelGGL(bs_keystream_kernel, dim3((uint32_t)wgs), dim3(kBsThreads), 0, s, p, ppc, n_passes);
    return hipGetLastError();
}

}  // namespace fastrack
