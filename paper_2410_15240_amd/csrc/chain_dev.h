// Device helpers shared by the streaming kernels (kernels.hip) and the
// bitsliced keystream kernel (bitslice.hip): the per-chain IV and partial-block
// loads and stores. Internal to the library.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "gf128_dev.h"
#include "launch.h"

namespace fastrack {

__device__ __forceinline__ u4 zero4()
{
    u4 z = {{0u, 0u, 0u, 0u}};
    return z;
}

// Little-endian word form of the 96-bit IV of global chain i:
// base_IV xor (0^32 || [i]_64), the index big-endian in IV bytes 4..11.
__device__ __forceinline__ void chain_iv(const GcmLaunch &p, uint64_t gchain, uint32_t iv[3])
{
    iv[0] = p.iv[0];
    iv[1] = p.iv[1] ^ bswap32((uint32_t)(gchain >> 32));
    iv[2] = p.iv[2] ^ bswap32((uint32_t)gchain);
}

// Load n (<= 16) bytes as a zero-padded block (constant register indices only).
__device__ inline u4 load_bytes(const uint8_t *src, uint32_t n)
{
    u4 r = zero4();
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int b = 0; b < 4; ++b)
            if ((uint32_t)(4 * j + b) < n)
                r.w[j] |= (uint32_t)src[4 * j + b] << (8 * b);
    return r;
}

__device__ inline void store_bytes(uint8_t *dst, const u4 &v, uint32_t n)
{
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
        for (int b = 0; b < 4; ++b)
            if ((uint32_t)(4 * j + b) < n)
                dst[4 * j + b] = (uint8_t)(v.w[j] >> (8 * b));
}

}  // namespace fastrack
