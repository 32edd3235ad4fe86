// gfx950 kernels for multi-chain AES-256-GCM (the paper's section 5.2,
// "Multi-chaining authentication", and its GPU decryption / authentication
// kernels of section 5.2-5.3).
//
//   key_setup_kernel   once per key: S-box, T0, round keys, H = AES_K(0),
//                      powers of H and the GF(2^128) multiplication tables.
//   gcm_kernel<ENC>    the streaming hot path: AES-256-CTR keystream XOR the
//                      data (section 3.2, AES-CTR) fused with GHASH over the
//                      AAD and ciphertext, parallel INSIDE each chain, and the
//                      per-chain tag / verification at the end of each chain.
//   seq_ghash_kernel   the paper's baseline authentication: one sequential
//                      Horner chain per tag (kept for comparison).
//
// GHASH inside a chain (GHASH definition: SP 800-38D 6.4; the paper's GMAC
// chain, section 3.2). For blocks X_1..X_m, GHASH = sum_j X_j . H^(m-j+1).
// A wave of 64 lanes takes 64 consecutive blocks per iteration (lane l gets
// block 64k + l, so loads are one coalesced 1 KiB access per wave). Each lane
// runs its own Horner chain with the fixed multiplier H^64:
//     acc_l <- acc_l . H^64  xor  X_(64k+l)
// and at the end of its segment the lanes are combined with one extra factor H:
//     G'_s = sum_l acc_l . H^(65-l)
// (lane l's last block has 63-l blocks after it), computed as a tree over the
// lanes whose level t multiplies by H^(2^t). A segment shorter than a
// multiple of 64 is padded with zero blocks at its START, which leaves GHASH
// unchanged. Segments are aligned to the end of the chain, so segment s of S
// carries the weight H^((S-1-s) . 2^seg_log2) within the chain.
// With q ciphertext blocks, G_C = GHASH over them, A the AAD and L the length
// block [len A]_64 || [len C]_64 (lengths in bits):
//     GHASH(A || C || L) = G_C . H  xor  GHASH(A) . H^(q+1)  xor  L . H
//     T = GHASH(A || C || L) xor AES_K(J0),   J0 = IV_i || 0^31 || 1.
// The AAD blocks ride in the same Horner streams (they are the blocks that
// precede the first ciphertext block), so a chain's streams sum to
// GHASH(A || C) . H = G_C . H xor GHASH(A) . H^(q+1). A chain cut into segments
// applies each segment's weight inside the chain and stores it; a second kernel
// XORs a chain's segments and adds L . H and AES_K(J0).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "aes_dev.h"
#include "chain_dev.h"
#include "gf128_dev.h"
#include "keyctx.h"
#include "launch.h"

namespace fastrack {

// ===========================================================================
// Key setup
// ===========================================================================

struct SetupArgs {
    uint32_t key[8];
};

// Entry p of the 4-bit positional table of y (little-endian form): the 16
// multiples (nibble v at degrees 4p..4p+3) . y, v's bit 3 being degree 4p.
__device__ inline void build_tab4_row(const u4 &y, int p, Tab4 *out)
{
    u4 b0 = be_mul_xk_any(to_be(y), 4 * p);
    u4 b1 = be_mul_xk(b0, 1), b2 = be_mul_xk(b1, 1), b3 = be_mul_xk(b2, 1);
    for (int v = 0; v < 16; ++v) {
        u4 e = {{0u, 0u, 0u, 0u}};
        if (v & 8) e = xor4(e, b0);
        if (v & 4) e = xor4(e, b1);
        if (v & 2) e = xor4(e, b2);
        if (v & 1) e = xor4(e, b3);
        u4 le = from_be(e);
        for (int j = 0; j < 4; ++j)
            out->e[p][v][j] = le.w[j];
    }
}

// Key setup in two launches. key_setup_kernel (one workgroup) runs the short
// dependent chain: the AES-256 key expansion, H = AES_K(0), the squares H^(2^t)
// and the powers H^8, H^16, ..., H^64. key_tables_kernel (many workgroups) then
// builds every table from those: one wave per table of an odd multiple
// H^(j 2^t) (j = 3, 5, 7), which forms its element from squares first, and one
// table row or entry per thread for the others.
//
// Key-independent parts come from tables the compiler evaluates: the S-box and
// T0, and the columns of the squaring map's powers S^k, k = 1..8.
static __constant__ const SboxTables kSboxTab = make_sbox_tables();
static __constant__ const FrobTable kFrobCols = make_frob_table();

// AES_K(0^128) by the four lanes of each quad (setup only): lane c holds state
// column c, and ShiftRows' bytes of columns c + 1, c + 2, c + 3 come by quad
// permutes. Returns column (lane & 3) of the output block. All lanes active.
__device__ inline uint32_t aes_zero_quad(const uint32_t *rk, const uint32_t *t0, uint32_t lane)
{
    const uint32_t c = lane & 3;
    uint32_t s = rk[c];   // the zero block after AddRoundKey
    uint32_t s1 = 0, s2 = 0, s3 = 0;
    auto shift = [&]() {
        s1 = __builtin_amdgcn_update_dpp(0u, s, 0x39, 0xF, 0xF, false);   // quad_perm [1,2,3,0]
        s2 = __builtin_amdgcn_update_dpp(0u, s, 0x4E, 0xF, 0xF, false);   // quad_perm [2,3,0,1]
        s3 = __builtin_amdgcn_update_dpp(0u, s, 0x93, 0xF, 0xF, false);   // quad_perm [3,0,1,2]
    };
#pragma unroll
    for (int r = 1; r < 14; ++r) {
        shift();
        s = t0[s & 0xFF] ^ rotl32(t0[(s1 >> 8) & 0xFF], 8) ^ rotl32(t0[(s2 >> 16) & 0xFF], 16) ^
            rotl32(t0[s3 >> 24], 24) ^ rk[4 * r + c];
    }
    shift();
    auto S = [&](uint32_t x) { return (t0[x] >> 8) & 0xFFu; };   // S(x) is byte 1 of T0[x]
    return (S(s & 0xFF) | (S((s1 >> 8) & 0xFF) << 8) | (S((s2 >> 16) & 0xFF) << 16) | (S(s3 >> 24) << 24)) ^
           rk[56 + c];
}

__global__ __launch_bounds__(1024) void key_setup_kernel(SetupArgs a, KeyCtx *__restrict__ ctx)
{
    __shared__ uint32_t s_sbox[256];
    __shared__ uint32_t s_t0[256];
    __shared__ uint32_t s_rk[60];
    __shared__ u4 s_hsq[kSquares];
    __shared__ u4 s_h8k[8];
    const int tid = threadIdx.x;
    const uint32_t lane = tid & 63, wave = (uint32_t)tid >> 6;

    // wave 7 + k holds the columns of S^k (k = 1..8) for the squares
    constexpr uint32_t kFrobWave0 = 8;
    WaveLinear frob;
    if (wave >= kFrobWave0)
        frob.load(kFrobCols.c[wave - kFrobWave0], lane);
    if (tid < 256) {
        const uint32_t sb = kSboxTab.sbox[tid], t = kSboxTab.t0[tid];
        s_sbox[tid] = sb;
        ctx->sbox[tid] = (uint8_t)sb;
        s_t0[tid] = t;
        ctx->t0[tid] = t;
    }
    __syncthreads();
    if (tid == 0) {
        uint32_t rk[60];
        expand_key_256(a.key, rk, [&](uint32_t x) { return s_sbox[x]; });
#pragma unroll
        for (int i = 0; i < 60; ++i) {
            s_rk[i] = rk[i];
            ctx->rk[i] = rk[i];
            ctx->rk16[i] = i >= 4 && i < 56 ? rotl32(rk[i], 16) : rk[i];
        }
    }
    __syncthreads();
    if (wave == 0) {
        const uint32_t col = aes_zero_quad(s_rk, s_t0, lane);
        u4 h;
#pragma unroll
        for (int j = 0; j < 4; ++j)
            h.w[j] = __builtin_amdgcn_readlane(col, j);
        if (lane == 0)
            s_hsq[0] = h;
        if (lane < 4)
            ctx->h[lane] = col;
    }
    __syncthreads();

    // Squares eight at a time: H^(2^(b + k)) = S^k(H^(2^b)), k = 1..8, one wave each,
    // in four rounds. The tables need H^8, H^16, ..., H^64: four are squares, and
    // the other four are products of them, formed by waves 0..2 during the rounds
    // after the first (H^24 = H^16 . H^8, H^40 = H^32 . H^8, H^48 = H^32 . H^16,
    // then H^56 = H^48 . H^8). A product by Y is one linear map whose columns the
    // wave builds (Y . x^k for its lanes k and k + 64).
    auto times = [&](const u4 &x, const u4 &y) {
        const u4 yb = to_be(y);
        WaveLinear mul;
        mul.c0 = be_mul_xk_any(yb, (int)lane);
        mul.c1 = be_mul_xk_any(yb, (int)lane + 64);
        return from_be(mul.apply(to_be(x), lane));
    };
    for (int r = 0; r < 4; ++r) {
        const int b = 8 * r;
        const int t = b + (int)(wave - kFrobWave0 + 1);
        if (wave >= kFrobWave0 && t < kSquares) {
            const u4 v = frob.apply(to_be(s_hsq[b]), lane);
            if (lane == 0)
                s_hsq[t] = from_be(v);
        }
        if (r == 1 && wave < 3) {   // H^24, H^40, H^48 (H^(2^t) for t <= 8 are in place)
            const u4 x = s_hsq[wave == 2 ? 5 : 4 + (wave & 1)], y = s_hsq[wave == 2 ? 4 : 3];
            const u4 prod = times(x, y);
            if (lane == 0)
                s_h8k[wave == 0 ? 2 : (wave == 1 ? 4 : 5)] = prod;
        }
        if (r == 2 && wave == 0) {   // H^56 = H^48 . H^8
            const u4 prod = times(s_h8k[5], s_hsq[3]);
            if (lane == 0)
                s_h8k[6] = prod;
        }
        __syncthreads();
    }
    if (tid < 8) {   // the squares among H^(8 (i + 1)): H^8, H^16, H^32, H^64
        const int sq = tid == 0 ? 3 : (tid == 1 ? 4 : (tid == 3 ? 5 : (tid == 7 ? 6 : -1)));
        const u4 v = sq >= 0 ? s_hsq[sq] : s_h8k[tid];
        for (int j = 0; j < 4; ++j)
            ctx->h8k[tid][j] = v.w[j];
    }
    for (int i = tid; i < kSquares; i += blockDim.x)
        for (int j = 0; j < 4; ++j)
            ctx->hsq[i][j] = s_hsq[i].w[j];
}

// The tables. First one wave per table of an odd multiple H^(j 2^t) (j = 3, 5, 7): the
// wave forms the element as a product of squares (H^(3 . 2^t) = H^(2^t) . H^(2^(t+1)),
// H^(5 . 2^t) = H^(2^t) . H^(2^(t+2)), H^(7 . 2^t) = H^(3 . 2^t) . H^(2^(t+2))), each a
// linear map whose columns the wave builds, and its lanes 0..31 write the table's
// nibble positions. These waves come first, as they have the longest path. Then one
// task per thread: a nibble position (16 entries) of the 4-bit tables of H and of
// every H^(2^t), or one entry of the 8-bit positional tables of H^8, H^16, ..., H^64:
// g16[i][v][k] = (byte v at byte k) . H^(8 (i + 1)), v's bit 7 = degree 8k.
constexpr uint32_t kOddThreads = kOddMul * kOddT * 64;
constexpr uint32_t kTab4Tasks = (1 + kSquares) * kTab4Pos;
constexpr uint32_t kTab8Entries = 8 * 16 * 256;
constexpr uint32_t kTableThreads = 256;
static_assert(kOddThreads % 64 == 0, "whole waves");

__device__ inline u4 times_wave(const u4 &x, const u4 &y, uint32_t lane)   // x . y, all 64 lanes
{
    const u4 yb = to_be(y);
    WaveLinear mul;
    mul.c0 = be_mul_xk_any(yb, (int)lane);
    mul.c1 = be_mul_xk_any(yb, (int)lane + 64);
    return from_be(mul.apply(to_be(x), lane));
}

__global__ __launch_bounds__(kTableThreads) void key_tables_kernel(KeyCtx *__restrict__ ctx)
{
    const uint32_t g = blockIdx.x * kTableThreads + threadIdx.x;
    if (g < kOddThreads) {   // whole waves: the branch is uniform
        const uint32_t o = g >> 6, lane = g & 63;
        const uint32_t i = o / kOddT, t = o % kOddT;   // j = 2 i + 3
        auto sq = [&](uint32_t e) {   // H^(2^e); e = 32 only for the unused H^(5 . 2^30), H^(7 . 2^30)
            const uint32_t *y = ctx->hsq[min(e, (uint32_t)kSquares - 1)];
            return u4{{y[0], y[1], y[2], y[3]}};
        };
        u4 y = times_wave(sq(t), sq(t + (i == 1 ? 2u : 1u)), lane);
        if (i == 2)
            y = times_wave(y, sq(t + 2), lane);
        if (lane < kTab4Pos)
            build_tab4_row(y, (int)lane, &ctx->odd_tab[i][t]);
        return;
    }
    const uint32_t task = g - kOddThreads;
    if (task < kTab4Tasks) {
        const uint32_t tbl = task / kTab4Pos, p = task % kTab4Pos;
        const uint32_t *y = tbl == 0 ? ctx->h : ctx->hsq[tbl - 1];
        build_tab4_row(u4{{y[0], y[1], y[2], y[3]}}, (int)p, tbl == 0 ? &ctx->h1_tab : &ctx->sq_tab[tbl - 1]);
        return;
    }
    const uint32_t ent = task - kTab4Tasks;
    if (ent >= kTab8Entries)
        return;
    const uint32_t i = ent >> 12, k = (ent >> 8) & 15, v = ent & 255;
    const uint32_t *hp = ctx->h8k[i];
    u4 b = be_mul_xk_any(to_be(u4{{hp[0], hp[1], hp[2], hp[3]}}), (int)(8 * k));   // degree 8k: v's bit 7
    u4 e = {{0u, 0u, 0u, 0u}};
    for (int bit = 7; bit >= 0; --bit) {
        if ((v >> bit) & 1u)
            e = xor4(e, b);
        b = be_mul_xk(b, 1);
    }
    const u4 le = from_be(e);
    for (int j = 0; j < 4; ++j)
        ctx->g16[i][v][k][j] = le.w[j];
}

hipError_t launch_key_setup(const uint32_t key_words[8], KeyCtx *ctx, hipStream_t s)
{
    SetupArgs a;
    for (int i = 0; i < 8; ++i)
        a.key[i] = key_words[i];
    hipLaunchKernelGGL(key_setup_kernel, dim3(1), dim3(1024), 0, s, a, ctx);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return e;
    constexpr uint32_t kTasks = kOddThreads + kTab4Tasks + kTab8Entries;
    hipLaunchKernelGGL(key_tables_kernel, dim3((kTasks + kTableThreads - 1) / kTableThreads), dim3(kTableThreads), 0, s,
                       ctx);
    return hipGetLastError();
}

// ===========================================================================
// Shared per-chain pieces
// ===========================================================================

// Position of an item: chain, segment s of S, the block range [b, e) of the
// segment in the chain's q blocks, and the chain's byte offset, length and
// final partial-block bytes.
struct ItemPos {
    uint32_t chain, s, S, q, b, e, tail;
    uint64_t off, len;
};

template <bool RAG>
__device__ __forceinline__ ItemPos item_pos(const GcmLaunch &p, uint64_t item)
{
    ItemPos r;
    if constexpr (RAG) {
        r.chain = p.ritem_chain[item];
        const RaggedChain rc = p.rchains[r.chain];
        r.s = item == rc.item0 ? 0u : (uint32_t)(item - rc.item_base);
        r.S = rc.segs;
        r.q = (uint32_t)((rc.len + 15) >> 4);
        r.off = rc.off;
        r.len = rc.len;
        r.tail = (uint32_t)(rc.len & 15);
    } else {
        const uint32_t it32 = (uint32_t)item;   // the host keeps a launch's items below 2^32
        r.chain = it32 / p.segs_full;
        r.s = it32 - r.chain * p.segs_full;
        const bool last = r.chain == p.n_chains - 1;
        r.q = last ? p.q_last : p.qc;
        r.S = last ? p.segs_last : p.segs_full;
        r.off = (uint64_t)r.chain * p.chain_bytes;
        r.len = last ? p.last_len : p.chain_bytes;
        r.tail = last ? (uint32_t)(p.last_len & 15) : 0u;
    }
    r.e = r.q - ((r.S - 1 - r.s) << p.seg_log2);
    r.b = r.s == 0 ? 0u : r.e - (1u << p.seg_log2);
    return r;
}


// ===========================================================================
// The streaming kernel
// ===========================================================================
//
// LDS layout (152 KiB + 1600 B, one 1024-thread workgroup per CU):
//   [0, 64 KiB)        row x (256 B) = T0[x] for lanes 0..31 | T1[x] for lanes 0..31
//   [64, 128 KiB)      the 8-bit table of H^L: entry (k, v) at 64 KiB + (v*16 + k)*16
//   [128, 152 KiB)     4-bit tables of H^(2^t), t = 0..2 (8 KiB each): the first levels of
//                      the lane-combine tree (the rest weights eight-lane group sums from
//                      the key's tables in global memory)
//   [152 KiB, +512 B)  per-wave segment partials and tag masks (workgroup tag combine)
//   then 1 KiB         the tag masks of the workgroup's items when wave 0 computes them all
//   then 64 B          per-wave progress counters (see the priority steps in the kernel)
// T_r[x] = rotl(T0[x], 8r), so T2[x] = rotl16(T0[x]) and T3[x] = rotl16(T1[x]): a
// round column T0[a] ^ T1[b] ^ T2[c] ^ T3[d] ^ k is T0[a] ^ T1[b] ^ rotl16(T0[c] ^
// T1[d] ^ rotl16(k)), one rotate more than with four tables, and the 64 KiB saved
// hold the tables the lane combine needs. Lanes l and l+32 share a copy: the LDS
// serves a wave's 32-bit reads 32 lanes at a time, so the 32 copies make every
// lookup conflict-free. A T0/T1 address is one v_perm_b32: byte 0 = (lane%32)*4 +
// 128*table, byte 1 = the state byte, bytes 2..3 = 0.
// GHASH multiplies by H^L as X . H^L = sum_k E_k[x_k] over the 16 byte positions k.
// The 16 entries of one byte value sit side by side in a 256-byte row, so position
// k lies in the k-th 16-byte bank group. The LDS serves a wave's 16-byte reads 16
// lanes at a time; lane l takes position k = j xor (l mod 16) at lookup j, so the 16
// lanes served together always hit 16 different bank groups, whatever the data.

constexpr int kThreads = kGcmThreads;
constexpr int kWavesPerWg = kGcmWavesPerWg;
constexpr int kTreeTabs = 6;                 // H^(2^t), t = 0..5: lanes per item up to 64
constexpr int kTreeLds = 3;                  // of which levels 0..2 in LDS (the AES modes)
constexpr uint32_t kGhBase = 4096;           // uint4 index of the GHASH table (64 KiB)
constexpr uint32_t kTreeBase = 8192;         // uint4 index of the tree tables (128 KiB)
constexpr uint32_t kWgTagBase = (128 + 8 * kTreeLds) * 1024 / 16;   // uint4 index: 16 partials, 16 masks
constexpr uint32_t kWgMaskBase = kWgTagBase + 32;                     // uint4 index: a tag mask per item (64)
static_assert(kWavesPerWg <= 16 && kWavesPerWg % 4 == 0, "one workgroup-combine slot per wave");
constexpr uint32_t kLdsBytes = (128 + 8 * kTreeLds) * 1024 + 512 + 1024 + 64;
// Modes without data AES: the GHASH table, T0 (for the J0 masks) and all six tree tables.
constexpr uint32_t kT0GhashOnly = 4096;         // uint4 index: 64 KiB
constexpr uint32_t kTreeBaseGhashOnly = 4160;   // 65 KiB
constexpr uint32_t kLdsGhashOnly = (65 + 8 * kTreeTabs) * 1024 + 64;
// Per-wave progress counters (16 words): the last 64 B of either layout.
constexpr uint32_t kProgBase = kLdsBytes / 4 - 16;
constexpr uint32_t kProgBaseGhashOnly = kLdsGhashOnly / 4 - 16;



#define FT_SEL(k) (0x0C020400u + ((uint32_t)(k) << 8))

// The streamed data blocks are read and written with non-temporal (nt) vector
// accesses: each byte is touched once, so they should not displace the key
// tables and partials from the L2 (1.4-2.2% per 64 MiB launch in an A/B run).
typedef uint32_t v4u __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint32_t tlk(const char *lds, uint32_t word, uint32_t lanec, uint32_t sel)
{
    return *reinterpret_cast<const uint32_t *>(lds + __builtin_amdgcn_perm(word, lanec, sel));
}

__device__ __forceinline__ uint32_t rotl16(uint32_t x) { return __builtin_amdgcn_alignbit(x, x, 16); }

// One output column of an AES round, T0[a.b0] ^ T1[b.b1] ^ T2[c.b2] ^ T3[d.b3] ^ k,
// with kr = rotl16(k): only T0 and T1 are in LDS.
__device__ __forceinline__ uint32_t tcol(const char *lds, uint32_t a, uint32_t b, uint32_t c, uint32_t d,
                                         uint32_t kr, uint32_t lc0, uint32_t lc1)
{
    const uint32_t u = xor3(tlk(lds, c, lc0, FT_SEL(2)), tlk(lds, d, lc1, FT_SEL(3)), kr);
    return xor3(tlk(lds, a, lc0, FT_SEL(0)), tlk(lds, b, lc1, FT_SEL(1)), rotl16(u));
}

// Final round column, S(a.b0) | S(b.b1) << 8 | S(c.b2) << 16 | S(d.b3) << 24, XOR k:
// S(x) is byte 1 of T0[x] and byte 2 of T1[x].
__device__ __forceinline__ uint32_t tlast(const char *lds, uint32_t a, uint32_t b, uint32_t c, uint32_t d,
                                          uint32_t k, uint32_t lc0, uint32_t lc1)
{
    const uint32_t a0 = tlk(lds, a, lc0, FT_SEL(0));
    const uint32_t a1 = tlk(lds, b, lc1, FT_SEL(1));
    const uint32_t a2 = tlk(lds, c, lc0, FT_SEL(2));
    const uint32_t a3 = tlk(lds, d, lc1, FT_SEL(3));
    return xor3(__builtin_amdgcn_perm(a1, a0, 0x0C0C0601u), __builtin_amdgcn_perm(a3, a2, 0x06010C0Cu), k);
}

// Lane i receives x from lane i + D (for lanes where that stays inside the
// aligned group the tree folds): DPP row shifts for D < 16, the gfx950 half-row
// and half-wave swaps for 16 and 32. VALU moves, no LDS round trip.
template <uint32_t D>
__device__ __forceinline__ uint32_t lane_down(uint32_t x)
{
    if constexpr (D < 16) {
        return __builtin_amdgcn_update_dpp(0u, x, 0x100 + D, 0xF, 0xF, false);   // row_shl:D
    } else if constexpr (D == 16) {
        return __builtin_amdgcn_permlane16_swap(x, x, false, false)[1];
    } else {
        static_assert(D == 32, "shift of 1..8, 16 or 32 lanes");
        return __builtin_amdgcn_permlane32_swap(x, x, false, false)[1];
    }
}

// Wave-wide maximum / minimum, returned uniform: VALU cross-lane moves folding
// every lane into lane 0 (no LDS permutes, which queue behind the table reads of
// the waves already streaming). All lanes must be active.
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t x)
{
    x = max(x, lane_down<32>(x));
    x = max(x, lane_down<16>(x));
    x = max(x, lane_down<8>(x));
    x = max(x, lane_down<4>(x));
    x = max(x, lane_down<2>(x));
    x = max(x, lane_down<1>(x));
    return __builtin_amdgcn_readlane(x, 0);
}

__device__ __forceinline__ int wave_min_i32(int x)
{
    x = min(x, (int)lane_down<32>((uint32_t)x));
    x = min(x, (int)lane_down<16>((uint32_t)x));
    x = min(x, (int)lane_down<8>((uint32_t)x));
    x = min(x, (int)lane_down<4>((uint32_t)x));
    x = min(x, (int)lane_down<2>((uint32_t)x));
    x = min(x, (int)lane_down<1>((uint32_t)x));
    return (int)__builtin_amdgcn_readlane((uint32_t)x, 0);
}

// The table of a segment-weight factor H^(j 2^t) (see weight_step). The exponent
// is below a chain's block count, so t stays in range (clamped all the same).
__device__ __forceinline__ const Tab4 *weight_tab(const KeyCtx *__restrict__ c, const WeightStep &w)
{
    if (w.j == 1)
        return &c->sq_tab[min(w.t, (uint32_t)kSquares - 1)];
    return &c->odd_tab[(w.j - 3) >> 1][min(w.t, (uint32_t)kOddT - 1)];
}

// X . Y where the L = 2^LL lanes of each aligned lane group hold one X (the
// groups may differ) and t points to Y's 4-bit table (it may differ per group
// as well): lane j of a group looks up the nibble positions j, j + L, ... < 32
// of X and the group XOR-sums the entries. Every lane of a group receives its
// group's product.
template <int LL>
__device__ inline u4 group_mul_tab4(const u4 &x, const Tab4 *__restrict__ t, uint32_t jl)
{
    constexpr uint32_t L = 1u << LL;
    u4 r = zero4();
#pragma unroll
    for (uint32_t rep = 0; rep < (L < 32 ? 32 / L : 1); ++rep) {
        const uint32_t pos = jl + rep * L;   // nibble position: word pos/8, byte (pos/2)%4, high nibble first
        if (pos < 32) {
            const uint32_t lo = (pos & 8) ? x.w[1] : x.w[0], hi = (pos & 8) ? x.w[3] : x.w[2];
            const uint32_t w = (pos & 16) ? hi : lo;
            const uint32_t byte = (w >> (8 * ((pos >> 1) & 3))) & 0xFFu;
            const uint32_t nib = (pos & 1) ? (byte & 0xFu) : (byte >> 4);
            const uint4 e = *reinterpret_cast<const uint4 *>(t->e[pos][nib]);
            r.w[0] ^= e.x; r.w[1] ^= e.y; r.w[2] ^= e.z; r.w[3] ^= e.w;
        }
    }
    for (int w = 0; w < 4; ++w)
        r.w[w] = group_xor_sum<LL>(r.w[w]);
    return r;
}

// AAD block u of a chain's AAD (zero-padded); one vector load when it is whole and aligned.
__device__ __forceinline__ u4 aad_block(const uint8_t *aad, uint32_t u, uint32_t aad_bytes)
{
    const uint32_t left = aad_bytes - 16u * u;
    const uint8_t *a = aad + 16u * u;
    if (left >= 16u && ((uintptr_t)a & 15) == 0) {
        const uint4 x = *reinterpret_cast<const uint4 *>(a);
        const u4 r = {{x.x, x.y, x.z, x.w}};
        return r;
    }
    return load_bytes(a, left < 16u ? left : 16u);
}

// L . H for the two length blocks of a launch, L = [len A]_64 || [len C]_64 in
// bits, with len C the full chain length (lanes 0..31) or the last chain's
// (lanes 32..63). Each lane looks up one nibble position of its L in the 4-bit
// table of H (h1), and each half of the wave XOR-sums its 32 entries.
struct LenTerms {
    u4 full, last;
};
__device__ inline LenTerms len_terms(const GcmLaunch &p, const Tab4 *h1, uint32_t lane)
{
    const uint64_t abits = (uint64_t)p.aad_bytes * 8;
    const uint64_t cbits = (lane < 32 ? p.chain_bytes : p.last_len) * 8;
    const uint32_t pos = lane & 31;                         // nibble position: degrees 4 pos .. 4 pos + 3
    const uint64_t half = pos < 16 ? abits : cbits;         // bytes 0..7 hold len A, 8..15 len C (big-endian)
    const uint32_t byte = (uint32_t)(half >> (8 * (7 - ((pos >> 1) & 7)))) & 0xFFu;
    const uint32_t nib = (pos & 1) ? (byte & 0xFu) : (byte >> 4);
    const uint4 e = *reinterpret_cast<const uint4 *>(h1->e[pos][nib]);
    u4 r = {{e.x, e.y, e.z, e.w}};
    // XOR over lanes 0..31 into lane 0 and 32..63 into lane 32 with VALU cross-lane
    // moves (DPP row shifts, the half-row swap): no LDS round trips, which queue
    // behind the table reads of the waves already streaming
    for (int w = 0; w < 4; ++w) {
        uint32_t x = r.w[w];
        x ^= lane_down<16>(x);
        x ^= lane_down<8>(x);
        x ^= lane_down<4>(x);
        x ^= lane_down<2>(x);
        x ^= lane_down<1>(x);
        r.w[w] = x;
    }
    LenTerms t;
    for (int w = 0; w < 4; ++w) {
        t.full.w[w] = __builtin_amdgcn_readlane(r.w[w], 0);
        t.last.w[w] = __builtin_amdgcn_readlane(r.w[w], 32);
    }
    return t;
}

// 16 bytes at p, read as one vector load when p is 16-byte aligned.
__device__ __forceinline__ u4 load16(const uint8_t *p)
{
    if (((uintptr_t)p & 15) == 0) {
        const uint4 x = *reinterpret_cast<const uint4 *>(p);
        const u4 r = {{x.x, x.y, x.z, x.w}};
        return r;
    }
    return load_bytes(p, 16);
}

// Encrypt: store the tag. Decrypt: ok = (tag == the received tag `got`).
template <bool ENC>
__device__ inline void emit_tag(const GcmLaunch &p, uint64_t gchain, const u4 &tag, const u4 &got)
{
    if (ENC) {
        uint8_t *dst = p.tags_out + 16 * gchain;
        if (((uintptr_t)dst & 15) == 0)
            *reinterpret_cast<uint4 *>(dst) = make_uint4(tag.w[0], tag.w[1], tag.w[2], tag.w[3]);
        else
            store_bytes(dst, tag, 16);
    } else {
        const uint32_t d = (got.w[0] ^ tag.w[0]) | (got.w[1] ^ tag.w[1]) | (got.w[2] ^ tag.w[2]) |
                           (got.w[3] ^ tag.w[3]);
        p.ok[gchain] = d == 0 ? 1 : 0;
    }
}

// Compile-time switches for the streaming kernel's iteration step: whether the
// iteration may hold AAD blocks.
struct AadSteps {
    static constexpr bool value = true;
};
struct NoAadSteps {
    static constexpr bool value = false;
};

// AES-256 of one block x (before the first AddRoundKey) with the streaming
// kernel's LDS T-tables: every lane encrypts its own block. rk holds the round
// keys of rounds 1..13 rotated by 16 bits (rk[4..55]), the others as they are.
__device__ inline u4 aes_block_lds(const char *lds, const uint32_t *rk, const u4 &x, uint32_t lc0, uint32_t lc1)
{
    uint32_t s0 = x.w[0] ^ rk[0], s1 = x.w[1] ^ rk[1], s2 = x.w[2] ^ rk[2], s3 = x.w[3] ^ rk[3];
#pragma unroll
    for (int r = 1; r < 14; ++r) {
        const uint32_t n0 = tcol(lds, s0, s1, s2, s3, rk[4 * r + 0], lc0, lc1);
        const uint32_t n1 = tcol(lds, s1, s2, s3, s0, rk[4 * r + 1], lc0, lc1);
        const uint32_t n2 = tcol(lds, s2, s3, s0, s1, rk[4 * r + 2], lc0, lc1);
        const uint32_t n3 = tcol(lds, s3, s0, s1, s2, rk[4 * r + 3], lc0, lc1);
        s0 = n0; s1 = n1; s2 = n2; s3 = n3;
    }
    u4 o;
    o.w[0] = tlast(lds, s0, s1, s2, s3, rk[56], lc0, lc1);
    o.w[1] = tlast(lds, s1, s2, s3, s0, rk[57], lc0, lc1);
    o.w[2] = tlast(lds, s2, s3, s0, s1, rk[58], lc0, lc1);
    o.w[3] = tlast(lds, s3, s0, s1, s2, rk[59], lc0, lc1);
    return o;
}

// acc . H^L xor g with the 8-bit table of H^L in LDS: byte positions 0..7
// directly, 8..15 through x^64.
// The lane constants of the GHASH lookups: l = lane mod 16.
struct GhLane {
    uint32_t sel;   // v_perm selector: byte b <- byte b xor (l mod 4) of this word (l & 4: of the paired word)
    uint32_t row;   // (l << 4) | the table's LDS byte address
    bool swap;      // l & 8: words 0,1 <-> 2,3
};

__device__ __forceinline__ GhLane ghash_lane(uint32_t lane, uint32_t table_bytes)
{
    const uint32_t l = lane & 15;
    GhLane k;
    k.sel = 0u;
    for (uint32_t b = 0; b < 4; ++b)
        k.sel |= ((b ^ (l & 3)) + (l & 4)) << (8 * b);
    k.row = (l << 4) | table_bytes;
    k.swap = (l & 8) != 0;
    return k;
}

// Horner step acc . H^L xor g: the bytes of acc are permuted so that byte j of p is
// byte j xor l of acc; lookup j then reads position j xor l, whose entry for value
// v is at row v, column (j xor l) of the table: address (v << 8 | row) xor (j << 4).
__device__ __forceinline__ u4 ghash_step(const char *lds, const u4 &acc, const u4 &g, const GhLane &k)
{
    uint32_t q[4];
#pragma unroll
    for (int w = 0; w < 4; ++w)
        q[w] = __builtin_amdgcn_perm(acc.w[w ^ 1], acc.w[w], k.sel);
    const uint32_t p[4] = {k.swap ? q[2] : q[0], k.swap ? q[3] : q[1], k.swap ? q[0] : q[2], k.swap ? q[1] : q[3]};
    u4 r = g;
#pragma unroll
    for (int j = 0; j < 16; j += 2) {
        // byte j of p into bits 8..15 (v_perm selector 0x0C: a zero byte)
        const uint32_t v0 = __builtin_amdgcn_perm(0u, p[j >> 2], 0x0C0C000Cu | ((uint32_t)(j & 3) << 8));
        const uint32_t v1 = __builtin_amdgcn_perm(0u, p[(j + 1) >> 2], 0x0C0C000Cu | ((uint32_t)((j + 1) & 3) << 8));
        const uint4 ea = *reinterpret_cast<const uint4 *>(lds + ((v0 | k.row) ^ ((uint32_t)j << 4)));
        const uint4 eb = *reinterpret_cast<const uint4 *>(lds + ((v1 | k.row) ^ ((uint32_t)(j + 1) << 4)));
        r.w[0] = xor3(r.w[0], ea.x, eb.x);
        r.w[1] = xor3(r.w[1], ea.y, eb.y);
        r.w[2] = xor3(r.w[2], ea.z, eb.z);
        r.w[3] = xor3(r.w[3], ea.w, eb.w);
    }
    return r;
}

// Lanes per item L = 2^LL. Item slot g of a wave (lanes g*L .. g*L+L-1) takes
// L consecutive blocks of its segment per iteration; each lane keeps a Horner
// accumulator with multiplier H^L, and lane j's accumulator carries the weight
// H^(L-j) in its segment (times one more H for the tag). SPLIT: chains are cut
// into segments whose weighted partials a second kernel sums. MODE is a
// GcmMode: which of keystream, data XOR and GHASH + tag the launch computes.
// RAG: chains of their own offsets and lengths from the launch's chain table.
template <bool ENC, int LL, bool SPLIT, int MODE, bool RAG>
__global__ __launch_bounds__(kThreads, gcm_wgs_per_cu(MODE) * kWavesPerWg / 4) void gcm_kernel(GcmLaunch p)
{
    constexpr bool kGhash = MODE == kFused || MODE == kVerify || MODE == kApplyKs;   // GHASH + tag
    constexpr bool kAes = MODE == kFused || MODE == kCtr || MODE == kKeystream;      // keystream by AES
    constexpr bool kRead = MODE != kKeystream;                                        // reads `in`
    constexpr bool kWrite = MODE != kVerify;                                          // writes `out`
    constexpr uint32_t L = 1u << LL;
    constexpr uint32_t G = 64u >> LL;
    // Static, so its LDS address is a compile-time constant and a v_perm result
    // can be used as the ds_read address with no further add. Modes without
    // data AES hold the GHASH table, a plain T0 (for the J0 masks) and all six
    // lane-combine tables, 113 KiB.
    constexpr uint32_t kLdsUse = kAes ? kLdsBytes : kLdsGhashOnly;
    __shared__ uint4 lds4[kLdsUse / 16];
    const char *lds = reinterpret_cast<const char *>(lds4);
    constexpr uint32_t kGh = kAes ? kGhBase : 0u;                     // uint4 index of the GHASH table
    uint32_t *t0l = reinterpret_cast<uint32_t *>(lds4 + kT0GhashOnly);   // GHASH-only modes: T0 after the table
    constexpr uint32_t kTree = kAes ? kTreeBase : kTreeBaseGhashOnly;
    constexpr int kTreeInLds = kAes ? kTreeLds : kTreeTabs;           // tree levels held in LDS
    const Tab4 *tree = reinterpret_cast<const Tab4 *>(lds4 + kTree);   // tree[t]: 4-bit table of H^(2^t)
    constexpr uint32_t kProg = kAes ? kProgBase : kProgBaseGhashOnly;
    const int tid = threadIdx.x;
    const uint32_t lane = tid & 63;
    const uint32_t jl = lane & (L - 1);      // lane within the item
    const uint32_t gs = lane >> LL;          // item slot within the wave
    const KeyCtx *__restrict__ c = p.ctx;

    {
        if (kAes) {
            // Pass k of a wave writes the 64 words (w + k W) * 64 + [0, 64) of region
            // (w + k W) / 256, all from one T0 row: lane k fetches that row up front
            // and each pass broadcasts it, so no pass waits on memory.
            uint32_t *t = reinterpret_cast<uint32_t *>(lds4);
            constexpr uint32_t kPasses = (16384 + kThreads - 1) / kThreads;
            static_assert(kPasses <= 64, "one T0 row per lane and pass");
            const uint32_t w = (uint32_t)tid >> 6;
            const uint32_t mine = c->t0[(w + kWavesPerWg * lane) & 255];
#pragma unroll 8
            for (uint32_t k = 0; k < kPasses; ++k) {
                const uint32_t ib = (w << 6) + k * kThreads;   // wave-uniform
                if (ib < 16384) {
                    const uint32_t v = __builtin_amdgcn_readlane(mine, k);
                    t[ib + lane] = lane < 32 ? v : rotl32(v, 8);
                }
            }
        } else {
            for (int i = tid; i < 256; i += kThreads)
                t0l[i] = c->t0[i];
        }
        if (tid < 16)   // slot 4 s + m: the m-th wave of SIMD s; slots no wave uses never hold anyone back
            reinterpret_cast<uint32_t *>(lds4)[kProg + tid] = (tid & 3) < kWavesPerWg / 4 ? 0u : 0xFFFFFFFFu;
        if (kGhash) {   // all loads of the 32 KiB GHASH table and the tree tables first, then the stores
            const uint4 *g = reinterpret_cast<const uint4 *>(c->g16[(L >> 3) - 1]);
            const uint4 *sq = reinterpret_cast<const uint4 *>(c->sq_tab);
            constexpr int kTreeU4 = kTreeInLds * (int)(sizeof(Tab4) / 16);
            constexpr int kPer = (4096 + kThreads - 1) / kThreads;
            constexpr int kPerT = (kTreeU4 + kThreads - 1) / kThreads;
            uint4 gv[kPer], tv[kPerT];
#pragma unroll
            for (int r = 0; r < kPer; ++r)
                gv[r] = g[min(tid + r * kThreads, 4095)];
#pragma unroll
            for (int r = 0; r < kPerT; ++r)
                tv[r] = sq[min(tid + r * kThreads, kTreeU4 - 1)];
#pragma unroll
            for (int r = 0; r < kPer; ++r)
                if (tid + r * kThreads < 4096)
                    lds4[kGh + tid + r * kThreads] = gv[r];
#pragma unroll
            for (int r = 0; r < kPerT; ++r)
                if (tid + r * kThreads < kTreeU4)
                    lds4[kTree + tid + r * kThreads] = tv[r];
        }
    }
    __syncthreads();

    const uint32_t lb = (lane & 31) << 2;
    const uint32_t lc0 = lb, lc1 = lb | 0x80u;
    const GhLane gk = ghash_lane(lane, kGh * 16);
    // The 60 round-key words are uniform: they stay in scalar registers (the XORs
    // take them as scalar operands), which keeps the kernel within the 128 VGPRs
    // that four waves per SIMD allow. Rounds 1..13 use them rotated by 16 bits (the
    // form tcol takes), precomputed per key. (Loaded after the table fill: scalar
    // loads and LDS accesses share one wait counter, so loading them earlier would
    // hold up the fill.)
    uint32_t rk[60];
#pragma unroll
    for (int i = 0; i < 60; ++i)
        rk[i] = kAes ? c->rk16[i] : 0u;

    const uint64_t nwaves = (uint64_t)gridDim.x * kWavesPerWg;
    // A launch with fewer wave-items than resident waves numbers its waves across
    // the workgroups first, which spreads the wave-items over all CUs; a full
    // launch keeps each workgroup's waves on consecutive wave-items.
    const bool spread = ((p.n_items + G - 1) / G) < nwaves;
    const uint32_t wave = __builtin_amdgcn_readfirstlane(spread ? (tid >> 6) * gridDim.x + blockIdx.x
                                                                : blockIdx.x * kWavesPerWg + (tid >> 6));
    const uint64_t n_wave_items = (p.n_items + G - 1) / G;
    const uint32_t seg = 1u << p.seg_log2;
    const uint32_t Ku_uniform = ((seg < p.qc ? seg : p.qc) + L - 1) >> LL;   // iterations per item
    // The tag mask AES_K(J0) xor L . H of the chains of this wave's next L
    // wave-items, one per lane: lane b*G + g holds the mask of slot g of the b-th
    // of them. One lane-parallel AES pass serves L wave-items.
    u4 jmask = zero4();
    uint32_t it = 0;   // wave-items done by this wave
    // The SIMD's instruction arbiter favours its oldest wave, so the waves of a SIMD
    // would finish their equal shares one after another, the last ones with the SIMD
    // to themselves. Wave w of the workgroup runs on SIMD w % 4; every wave publishes
    // its iteration count in LDS and, each iteration, takes issue priority 3 while it
    // is the slowest wave of its SIMD, 2 or 1 while it leads the slowest by one or two
    // iterations, and 0 beyond that, so the four keep pace with each other.
    // The counters are accessed through LDS-typed pointers (address space 3), with
    // compiler barriers around the accesses in place of `volatile`: a volatile access
    // through a generic pointer becomes a flat access followed by a wait for every
    // outstanding global load and store of the wave, once per iteration.
    typedef __attribute__((address_space(3))) uint32_t lds_u32;
    typedef __attribute__((address_space(3))) v4u lds_v4u;
    lds_u32 *prog = (lds_u32 *)(reinterpret_cast<uint32_t *>(lds4) + kProg);
    const uint32_t wslot = (uint32_t)tid >> 6;
    const uint32_t pidx = (wslot & 3) * 4 + (wslot >> 2);
    uint32_t iters_done = 0;
    // Workgroup tag combine (fused uniform launches of one item per wave).
    constexpr bool kWgCombine = SPLIT && LL == 6 && MODE == kFused && !RAG;
    __builtin_amdgcn_s_setprio(3);
    // The tag mask AES_K(J0) xor L . H for the item `bitem` in every lane that needs
    // one (its item exists and starts its chain, segment 0); zero in the others,
    // which stay inactive through the AES, so a pass reads the LDS for those lanes
    // only. A wave-collective (len_terms); all lanes must call it.
    auto mask_pass = [&](uint64_t bitem) {
        const ItemPos bp = item_pos<RAG>(p, bitem < p.n_items ? bitem : p.n_items - 1);
        uint32_t biv[3];
        chain_iv(p, p.chain_base + bp.chain, biv);
        const u4 j0 = {{biv[0], biv[1], biv[2], bswap32(1u)}};   // J0 = IV_i || 0^31 || 1
        const bool need = bitem < p.n_items && bp.s == 0;
        u4 lenh = zero4();
        if constexpr (!RAG) {
            const LenTerms lt = len_terms(p, &tree[0], lane);
            lenh = bp.chain == p.n_chains - 1 ? lt.last : lt.full;
        }
        u4 m = zero4();
        if (need) {
            if constexpr (RAG) {   // every chain has its own length: each lane multiplies its own
                const uint64_t abits = (uint64_t)p.aad_bytes * 8, cbits = bp.len * 8;
                const u4 lens = {{bswap32((uint32_t)(abits >> 32)), bswap32((uint32_t)abits),
                                  bswap32((uint32_t)(cbits >> 32)), bswap32((uint32_t)cbits)}};
                lenh = mul_tab4(lens, &tree[0]);
            }
            u4 e;
            if constexpr (kAes)
                e = aes_block_lds(lds, rk, j0, lc0, lc1);
            else
                e = aes256_encrypt_tt(j0, c->rk, [&](uint32_t x) { return t0l[x]; });
            m = xor4(e, lenh);
        }
        return m;
    };
    // A full uniform launch (one wave-item per wave): wave 0 computes the masks of
    // all the workgroup's items in one pass, a lane per item, and leaves them in LDS
    // for the other waves, which read them after a barrier before their tags. A pass
    // costs the LDS nearly as much with a few lanes active as with 64, so one pass
    // per workgroup instead of one per wave frees LDS time for the main loop (the 4
    // and 16 KiB chains of the 64 MiB batch have one or four items per wave).
    const bool wg_masks = MODE == kFused && !RAG && !spread && n_wave_items == nwaves;
    if (wg_masks && wslot == 0) {
        const uint64_t bitem = ((uint64_t)blockIdx.x * kWavesPerWg + lane / G) * G + lane % G;
        const u4 m = mask_pass(lane < kWavesPerWg * G ? bitem : p.n_items);
        if (lane < kWavesPerWg * G)
            lds4[kWgMaskBase + lane] = make_uint4(m.w[0], m.w[1], m.w[2], m.w[3]);
    }
    // Launches that leave waves without a wave-item (small ones) and are tagged by the
    // per-chain kernel: the idle waves compute the chains' masks, one lane per chain,
    // so the mask pass is off the working waves' path (AES of J0 is one more block
    // per chain, its position fixed by the chain index alone).
    const bool idle_masks = kGhash && SPLIT && p.idle_masks != 0;
    if (idle_masks && wave >= n_wave_items) {
        const uint64_t c0 = ((uint64_t)wave - n_wave_items) * 64;   // uniform
        if (c0 < p.n_chains) {
            const uint64_t c = c0 + lane;
            uint64_t bitem = p.n_items;   // no chain: nothing needed
            if (c < p.n_chains) {
                if constexpr (RAG)
                    bitem = p.rchains[c].item0;
                else
                    bitem = c * p.segs_full;
            }
            const u4 m = mask_pass(bitem);
            if (c < p.n_chains)
                p.masks[c] = make_uint4(m.w[0], m.w[1], m.w[2], m.w[3]);
        }
    }
    for (uint64_t wi = wave; wi < n_wave_items; wi += nwaves, ++it) {
        const uint32_t bi = it & (L - 1);
        if (kGhash && bi == 0 && !wg_masks && !idle_masks)
            jmask = mask_pass((wi + (uint64_t)(lane >> (6 - LL)) * nwaves) * G + (lane & (G - 1)));
        const uint64_t item = wi * G + gs;
        const bool valid = item < p.n_items;
        const ItemPos ip = item_pos<RAG>(p, valid ? item : p.n_items - 1);
        const uint64_t gchain = p.chain_base + ip.chain;
        // A whole-chain item checks its tag at the end: fetch the received tag now.
        u4 got = zero4();
        if constexpr (!ENC && kGhash)
            if (valid && jl == 0 && (!SPLIT || (p.wg_tag && ip.s == 0)))
                got = load16(p.tags_in + 16 * gchain);
        // Iterations of this wave-item: uniform for uniform chains; for ragged chains
        // the longest of the wave's segments (shorter ones are padded in front).
        uint32_t Ku = Ku_uniform;
        if constexpr (RAG) {
            Ku = wave_max_u32(valid ? (ip.e - ip.b + L - 1) >> LL : 0u);
        }
        uint32_t iv[3];
        chain_iv(p, gchain, iv);
        // Counter mode: columns 0..2 of the state after AddRoundKey are the IV and
        // fixed for the whole chain, so 12 of round 1's 16 lookups are too.
        uint32_t p0 = 0, p1 = 0, p2 = 0, p3 = 0;
        if constexpr (kAes) {
            // (rk[4..7] are rotated by 16 bits; T2 = rotl16(T0), T3 = rotl16(T1).)
            const uint32_t c0 = iv[0] ^ rk[0], c1 = iv[1] ^ rk[1], c2 = iv[2] ^ rk[2];
            p0 = xor3(tlk(lds, c0, lc0, FT_SEL(0)), tlk(lds, c1, lc1, FT_SEL(1)),
                      rotl16(tlk(lds, c2, lc0, FT_SEL(2)) ^ rk[4]));
            p1 = xor3(tlk(lds, c1, lc0, FT_SEL(0)), tlk(lds, c2, lc1, FT_SEL(1)),
                      rotl16(tlk(lds, c0, lc1, FT_SEL(3)) ^ rk[5]));
            p2 = tlk(lds, c2, lc0, FT_SEL(0)) ^ rotl16(xor3(tlk(lds, c0, lc0, FT_SEL(2)), tlk(lds, c1, lc1, FT_SEL(3)), rk[6]));
            p3 = tlk(lds, c0, lc1, FT_SEL(1)) ^ rotl16(xor3(tlk(lds, c1, lc0, FT_SEL(2)), tlk(lds, c2, lc1, FT_SEL(3)), rk[7]));
        }
        const uint8_t *src = kRead ? p.in + ip.off : nullptr;
        uint8_t *dst = kWrite ? p.out + ip.off : nullptr;
        const uint8_t *ksrc = MODE == kApplyKs ? p.ks + ip.off : nullptr;
        const uint32_t tail = ip.tail;   // bytes of a final partial block
        const int pad = (int)((Ku << LL) - (ip.e - ip.b));                   // zero blocks in front
        // The AAD blocks precede ciphertext block 0 of the chain in GHASH order: in
        // segment 0, AAD block u takes the slot v = u - na just before it. Lane jl
        // holds the slots v = k L + jl - pad, so its AAD blocks fall in iterations
        // k_lo..k_hi; those below 0 are extra iterations ahead of the data that only
        // feed GHASH, the others are padding slots of the first iterations.
        const int na = (kGhash && ip.s == 0 && valid) ? (int)((p.aad_bytes + 15) >> 4) : 0;
        const uint8_t *aad_c = p.aad + gchain * p.aad_bytes;
        int k_lo = 0, k_hi = -1;
        if (na) {
            k_lo = (pad - na - (int)jl + (int)L - 1) >> LL;   // ceil((pad - na - jl) / L)
            k_hi = (pad - 1 - (int)jl) >> LL;                 // floor((pad - 1 - jl) / L)
            if (k_lo > k_hi) {
                k_lo = 0;
                k_hi = -1;
            }
        }
        const int kmin = wave_min_i32(k_lo < 0 ? k_lo : 0);
        const int kmax = (int)wave_max_u32((uint32_t)(k_hi + 1)) - 1;   // k_hi >= -1
        u4 acc = zero4();
        if (kmin == -1) {
            // One extra iteration (at most L AAD blocks in front): its blocks seed the
            // accumulators directly, and the loads complete under the first iteration.
            if (k_lo == -1)
                acc = aad_block(aad_c, (uint32_t)(jl - (int)L - pad + na), p.aad_bytes);
        } else {
            for (int k = kmin; k < 0; ++k) {
                const int v = k * (int)L + (int)jl - pad;
                const u4 g = v >= -na ? aad_block(aad_c, (uint32_t)(v + na), p.aad_bytes) : zero4();
                acc = k == kmin ? g : ghash_step(lds, acc, g, gk);
            }
        }
        // The lane's slot in iteration k: v = k L + jl - pad (below 0: a padding slot),
        // block t of the chain; a final partial block holds `tail` bytes.
        struct Slot {
            int v;
            bool active, partial;
            uint32_t t;
        };
        auto slot_of = [&](uint32_t k) {
            Slot q;
            q.v = (int)(k << LL) + (int)jl - pad;
            q.active = valid && q.v >= 0;
            q.t = ip.b + (uint32_t)q.v;
            q.partial = q.active && tail != 0 && q.t == ip.q - 1;
            return q;
        };
        auto load_block = [&](const uint8_t *base, const Slot &q) {
            u4 x = zero4();
            if (q.active) {
                if (!q.partial) {
                    const v4u y = __builtin_nontemporal_load(reinterpret_cast<const v4u *>(base) + q.t);
                    x.w[0] = y.x; x.w[1] = y.y; x.w[2] = y.z; x.w[3] = y.w;
                } else {
                    x = load_bytes(base + 16ull * q.t, tail);
                }
            }
            return x;
        };
        // Counter blocks of one 256-block group (the counter's upper 24 bits fixed):
        // after round 1 only column 0 of the state varies (it takes the counter's low
        // byte), so in round 2 the three lookups of each output column that read
        // columns 1..3 are fixed too. q0..q3 cache those partial sums for the group
        // gq of the lane's current counter.
        uint32_t q0 = 0, q1 = 0, q2 = 0, q3 = 0, gq = 0xFFFFFFFFu;
        auto group_setup = [&](uint32_t ctr) {
            const uint32_t s3i = bswap32(ctr) ^ rk[3];
            const uint32_t s1 = p1 ^ rotl16(tlk(lds, s3i, lc0, FT_SEL(2)));
            const uint32_t s2 = p2 ^ tlk(lds, s3i, lc1, FT_SEL(1));
            const uint32_t s3 = p3 ^ tlk(lds, s3i, lc0, FT_SEL(0));
            q0 = tlk(lds, s1, lc1, FT_SEL(1)) ^ rotl16(xor3(tlk(lds, s2, lc0, FT_SEL(2)), tlk(lds, s3, lc1, FT_SEL(3)), rk[8]));
            q1 = xor3(tlk(lds, s1, lc0, FT_SEL(0)), tlk(lds, s2, lc1, FT_SEL(1)), rotl16(tlk(lds, s3, lc0, FT_SEL(2)) ^ rk[9]));
            q2 = xor3(tlk(lds, s2, lc0, FT_SEL(0)), tlk(lds, s3, lc1, FT_SEL(1)), rotl16(tlk(lds, s1, lc1, FT_SEL(3)) ^ rk[10]));
            q3 = tlk(lds, s3, lc0, FT_SEL(0)) ^ rotl16(xor3(tlk(lds, s1, lc0, FT_SEL(2)), tlk(lds, s2, lc1, FT_SEL(3)), rk[11]));
            gq = ctr >> 8;
        };
        const uint32_t k3 = rk[3] >> 24;   // key byte that meets the counter's low byte
        // Iteration k on the loaded data block d (and keystream block kv for kApplyKs).
        // AAD: whether iteration k may hold AAD blocks (k <= kmax); a step built
        // without them issues a fixed set of memory accesses.
        auto process = [&](auto aad, uint32_t k, const Slot &q, const u4 &d, const u4 &kv) {
            const uint32_t t = q.t;
            u4 o;
            if constexpr (kAes) {
                // Counter block IV_i || [t + 2]_32 (data blocks start at inc32(J0)).
                const uint32_t ctr = t + 2u;
                const bool stale = q.active && (ctr >> 8) != gq;
                if (__ballot(stale))
                    if (stale)
                        group_setup(ctr);
                // Round 1, column 0 (T3 of the counter's low byte), then round 2 on the
                // cached sums: each output column adds its one lookup of column 0.
                const uint32_t c0 = p0 ^ rotl16(tlk(lds, ctr ^ k3, lc1, FT_SEL(0)));
                uint32_t s0 = q0 ^ tlk(lds, c0, lc0, FT_SEL(0));
                uint32_t s1 = q1 ^ rotl16(tlk(lds, c0, lc1, FT_SEL(3)));
                uint32_t s2 = q2 ^ rotl16(tlk(lds, c0, lc0, FT_SEL(2)));
                uint32_t s3 = q3 ^ tlk(lds, c0, lc1, FT_SEL(1));
#pragma unroll
                for (int r = 3; r < 14; ++r) {
                    const uint32_t n0 = tcol(lds, s0, s1, s2, s3, rk[4 * r + 0], lc0, lc1);
                    const uint32_t n1 = tcol(lds, s1, s2, s3, s0, rk[4 * r + 1], lc0, lc1);
                    const uint32_t n2 = tcol(lds, s2, s3, s0, s1, rk[4 * r + 2], lc0, lc1);
                    const uint32_t n3 = tcol(lds, s3, s0, s1, s2, rk[4 * r + 3], lc0, lc1);
                    s0 = n0; s1 = n1; s2 = n2; s3 = n3;
                }
                // Final round, XOR the data.
                o.w[0] = tlast(lds, s0, s1, s2, s3, rk[56] ^ d.w[0], lc0, lc1);
                o.w[1] = tlast(lds, s1, s2, s3, s0, rk[57] ^ d.w[1], lc0, lc1);
                o.w[2] = tlast(lds, s2, s3, s0, s1, rk[58] ^ d.w[2], lc0, lc1);
                o.w[3] = tlast(lds, s3, s0, s1, s2, rk[59] ^ d.w[3], lc0, lc1);
            } else if constexpr (MODE == kApplyKs) {
                o = xor4(d, kv);
            } else {
                o = d;
            }
            if (kWrite && q.active) {
                if (!q.partial) {
                    const v4u ov = {o.w[0], o.w[1], o.w[2], o.w[3]};
                    __builtin_nontemporal_store(ov, reinterpret_cast<v4u *>(dst) + t);
                } else {
                    store_bytes(dst + 16ull * t, o, tail);
                }
            }
            if constexpr (kGhash) {
                u4 g = ENC ? o : d;
                if (ENC) {
                    if (!q.active) {
                        g = zero4();
                    } else if (q.partial) {                   // GHASH sees the ciphertext zero-padded
                        for (int j = 0; j < 4; ++j) {
                            const int nb = (int)tail - 4 * j;
                            const uint32_t m = nb >= 4 ? 0xFFFFFFFFu : (nb <= 0 ? 0u : ((1u << (8 * nb)) - 1u));
                            g.w[j] &= m;
                        }
                    }
                }
                if constexpr (decltype(aad)::value)
                    if ((int)k <= kmax && q.v < 0 && q.v >= -na)    // an AAD block in a padding slot
                        g = aad_block(aad_c, (uint32_t)(q.v + na), p.aad_bytes);
                acc = (k == 0 && kmin == 0) ? g : ghash_step(lds, acc, g, gk);
            }
        };
        auto pace = [&](uint32_t k) {
            const uint32_t mine = iters_done + k;
            if (lane == 0)
                prog[pidx] = mine;
            asm volatile("" ::: "memory");   // the store is made, the others' counters re-read
            const v4u g = *(const lds_v4u *)(reinterpret_cast<uint32_t *>(lds4) + kProg + (pidx & ~3u));
            const uint32_t mn = __builtin_amdgcn_readfirstlane(min(min(g.x, g.y), min(g.z, g.w)));
            const uint32_t lead = mine - (mn < mine ? mn : mine);
            if (lead == 0u)
                __builtin_amdgcn_s_setprio(3);
            else if (lead == 1u)
                __builtin_amdgcn_s_setprio(2);
            else if (lead == 2u)
                __builtin_amdgcn_s_setprio(1);
            else
                __builtin_amdgcn_s_setprio(0);
        };
        if constexpr (!kAes && kRead && !(SPLIT && LL < 6)) {
            // No AES between a load and its use to hide the memory latency: the loads
            // run up to four iterations ahead of the GHASH steps, in a queue of
            // registers. Every queued load is issued unconditionally, so the wait
            // before each use covers only the oldest one: ldq returns the raw 16 bytes
            // of slot k, or of the key context when the slot holds no whole block
            // (padding, past the item, or the chain's final partial block), and take()
            // decides at the use whether they count, so the load itself is never made
            // conditional. The partial block, if this lane has one, is read before
            // the loop.
            auto ldq = [&](const uint8_t *base, uint32_t k) {
                const Slot q = slot_of(k);
                const bool whole = k < Ku && q.active && !q.partial;
                const v4u *a = whole ? reinterpret_cast<const v4u *>(base) + q.t : reinterpret_cast<const v4u *>(c);
                return __builtin_nontemporal_load(a);
            };
            auto take = [&](const Slot &q, const v4u &y, const u4 &part) {
                return q.partial ? part : (q.active ? u4{{y.x, y.y, y.z, y.w}} : zero4());
            };
            u4 pd = zero4(), pk = zero4();   // this lane's partial block (data, keystream)
            if (tail != 0 && valid && ip.e == ip.q) {
                const int v = (int)(ip.q - 1 - ip.b) + pad;   // its slot: iteration v / L, lane v % L
                if ((uint32_t)(v & (int)(L - 1)) == jl) {
                    pd = load_bytes(src + 16ull * (ip.q - 1), tail);
                    if constexpr (MODE == kApplyKs)
                        pk = load_bytes(ksrc + 16ull * (ip.q - 1), tail);
                }
            }
            // Iterations that may hold AAD blocks (segment 0's first ones) run first,
            // with their loads in line.
            const uint32_t k0 = kmax < 0 ? 0u : min((uint32_t)kmax + 1u, Ku);
            for (uint32_t k = 0; k < k0; ++k) {
                pace(k);
                const Slot q = slot_of(k);
                process(AadSteps{}, k, q, load_block(src, q), MODE == kApplyKs ? load_block(ksrc, q) : zero4());
            }
            // Everything loaded so far has arrived: the queue below then waits only
            // for its own oldest load.
            __builtin_amdgcn_s_waitcnt(0);
            // Queue depth: four for verifying whole chains; two when a keystream block
            // and an output store come with each block, and for 64-lane segments of
            // split chains, whose items carry more state. (Keystream-apply on split
            // chains and split items of 16 or 32 lanes would exceed 128 VGPRs with a
            // queue and spill: they keep the loop below.)
            constexpr uint32_t kAhead = SPLIT ? (MODE == kApplyKs ? 1u : 2u) : (MODE == kApplyKs ? 2u : 4u);
            v4u dq[kAhead], eq[kAhead];
#pragma unroll
            for (uint32_t j = 0; j < kAhead; ++j) {
                dq[j] = ldq(src, k0 + j);
                if constexpr (MODE == kApplyKs)
                    eq[j] = ldq(ksrc, k0 + j);
            }
            // Iteration k uses the slot loaded kAhead iterations earlier and refills it
            // for iteration k + kAhead; unrolled by kAhead, so each slot stays in its
            // registers (moving a register whose load is in flight would wait for it).
            // The scheduling barrier keeps the steps from interleaving, which would
            // hold several iterations' registers at once.
            for (uint32_t k = k0; k < Ku; k += kAhead) {
#pragma unroll
                for (uint32_t j = 0; j < kAhead; ++j) {
                    __builtin_amdgcn_sched_barrier(0);
                    const uint32_t kk = k + j;
                    if (kk < Ku) {
                        pace(kk);
                        const Slot q = slot_of(kk);
                        const u4 dv = take(q, dq[j], pd), kv = MODE == kApplyKs ? take(q, eq[j], pk) : zero4();
                        dq[j] = ldq(src, kk + kAhead);
                        if constexpr (MODE == kApplyKs)
                            eq[j] = ldq(ksrc, kk + kAhead);
                        process(NoAadSteps{}, kk, q, dv, kv);
                    }
                }
            }
        } else {
            for (uint32_t k = 0; k < Ku; ++k) {
                pace(k);
                const Slot q = slot_of(k);
                process(AadSteps{}, k, q, kRead ? load_block(src, q) : zero4(),
                        MODE == kApplyKs ? load_block(ksrc, q) : zero4());
            }
        }
        iters_done += Ku;
        if constexpr (kGhash) {
            __builtin_amdgcn_s_setprio(3);   // the tail is a short latency-bound chain
            // Lane j's stream carries the weight H^(L+1-j) in its segment (one H of it
            // for the tag). sum_j acc_j H^(L-1-j) is a tree over the lanes: level t folds
            // lane j + 2^t into lane j with the factor H^(2^t), every lane active at a
            // level reading the same LDS table; then one multiply by H^2 in lane 0.
            auto fold_in = [&](uint32_t lv) {   // lane j takes lane j + 2^lv's sum
                u4 right;
                for (int w = 0; w < 4; ++w) {
                    const uint32_t x = acc.w[w];
                    switch (lv) {   // uniform: the VALU cross-lane move for this distance
                    case 0: right.w[w] = lane_down<1>(x); break;
                    case 1: right.w[w] = lane_down<2>(x); break;
                    case 2: right.w[w] = lane_down<4>(x); break;
                    case 3: right.w[w] = lane_down<8>(x); break;
                    case 4: right.w[w] = lane_down<16>(x); break;
                    default: right.w[w] = lane_down<32>(x); break;
                    }
                }
                return right;
            };
            constexpr uint32_t kLvLds = (uint32_t)LL < (uint32_t)kTreeInLds ? (uint32_t)LL : (uint32_t)kTreeInLds;
#pragma unroll 1
            for (uint32_t lv = 0; lv < kLvLds; ++lv) {
                const u4 right = fold_in(lv);
                if ((jl & ((2u << lv) - 1)) == 0)
                    acc = xor4(mul_tab4_b8(acc, &tree[lv]), right);
            }
            if constexpr (kTreeInLds == 3) {
                // After the three LDS levels, lane 8m of an item holds the sum C_m of its
                // eight-lane group m (of M = L/8). The remaining levels would multiply these
                // by H^8, H^16, H^32 one level after another; instead lane 8m multiplies C_m
                // by its own weight H^(8 (M-1-m)) from the key's 8-bit tables in global
                // memory (all groups at once, one multiply's latency), and the M products
                // are XOR-folded into lane 0 by VALU cross-lane moves.
                constexpr uint32_t M = L >> 3;
                const uint32_t m = jl >> 3;
                if ((jl & 7u) == 0 && m + 1 < M)   // M = 2: one group multiplies, by H^8 (a uniform table)
                    acc = mul_tab8_b8(acc, reinterpret_cast<const uint4 *>(c->g16[M == 2 ? 0u : M - 2 - m]));
                if constexpr (LL >= 6)
                    for (int w = 0; w < 4; ++w)
                        acc.w[w] ^= lane_down<32>(acc.w[w]);
                if constexpr (LL >= 5)
                    for (int w = 0; w < 4; ++w)
                        acc.w[w] ^= lane_down<16>(acc.w[w]);
                for (int w = 0; w < 4; ++w)
                    acc.w[w] ^= lane_down<8>(acc.w[w]);
            }
            if (jl == 0)
                acc = mul_tab4_b8(acc, &tree[1]);
            if (SPLIT)   // the segment weights below take the sum in every lane of the group
                for (int w = 0; w < 4; ++w)
                    acc.w[w] = LL == 6 ? __builtin_amdgcn_readlane(acc.w[w], 0) : __shfl(acc.w[w], (int)(lane - jl), 64);
            if (SPLIT) {
                // A chain cut into S segments: segment s carries the weight
                // H^((S-1-s) . 2^seg_log2) inside its chain, one multiply per nonzero
                // base-8 digit of S-1-s, shared by the item's lanes (a dependent
                // table multiply each, so at most 2 for up to 64 segments, 3 for 512).
                // The partials and segment 0's mask go to memory; the chain kernel
                // sums them.
                uint32_t m = valid ? ip.S - 1 - ip.s : 0u;
                const uint32_t rounds = wave_max_u32(octal_digits(m));
                for (uint32_t r = 0; r < rounds; ++r) {
                    uint32_t rest = m;
                    const WeightStep w = m ? weight_step(rest, p.seg_log2) : WeightStep{1u, 0u};
                    const u4 prod = group_mul_tab4<LL>(acc, weight_tab(c, w), jl);
                    if (m) {
                        acc = prod;
                        m = rest;
                    }
                }
                const uint32_t src_lane = bi * G + gs;
                u4 e;
                if (wg_masks) {   // wave 0's masks of this workgroup's items
                    __syncthreads();
                    const uint4 m = lds4[kWgMaskBase + wslot * G + gs];
                    e = u4{{m.x, m.y, m.z, m.w}};
                } else {
                    for (int w = 0; w < 4; ++w)   // one item per wave: the mask's lane bi is uniform
                        e.w[w] = LL == 6 ? __builtin_amdgcn_readlane(jmask.w[w], bi)
                                         : __shfl(jmask.w[w], (int)src_lane, 64);
                }
                if (kWgCombine && p.wg_tag) {   // the workgroup tags the chain after its barrier
                    if (valid && jl == 0) {
                        lds4[kWgTagBase + wslot] = make_uint4(acc.w[0], acc.w[1], acc.w[2], acc.w[3]);
                        if (ip.s == 0)   // decrypt: the mask xor the received tag, so a good chain sums to 0
                            lds4[kWgTagBase + 16 + wslot] = make_uint4(e.w[0] ^ got.w[0], e.w[1] ^ got.w[1],
                                                                       e.w[2] ^ got.w[2], e.w[3] ^ got.w[3]);
                    }
                } else if (valid && jl == 0) {
                    p.partials[item] = make_uint4(acc.w[0], acc.w[1], acc.w[2], acc.w[3]);
                    if (ip.s == 0 && !idle_masks)
                        p.masks[ip.chain] = make_uint4(e.w[0], e.w[1], e.w[2], e.w[3]);
                }
            } else {
                // The slot holds its chain's whole GHASH(A || C) . H:
                // T = GHASH(A || C) . H xor L . H xor AES_K(J0).
                u4 e;
                if (wg_masks) {   // wave 0's masks of this workgroup's items
                    __syncthreads();
                    const uint4 m = lds4[kWgMaskBase + wslot * G + gs];
                    e = u4{{m.x, m.y, m.z, m.w}};
                } else {
                    for (int w = 0; w < 4; ++w)
                        e.w[w] = LL == 6 ? __builtin_amdgcn_readlane(jmask.w[w], bi)
                                         : __shfl(jmask.w[w], (int)(bi * G + gs), 64);
                }
                if (valid && jl == 0)
                    emit_tag<ENC>(p, gchain, xor4(acc, e), got);
            }
        }
    }
    if (lane == 0)   // a finished wave no longer holds the others of its SIMD back
        prog[pidx] = 0xFFFFFFFFu;
    if constexpr (kWgCombine) {
        // Every wave took exactly one item (the item index is the wave index) and a
        // chain's S segments sit on waves w .. w+S-1 of this workgroup: the wave with
        // segment 0 XORs their partials into its mask (decrypt: mask xor received tag,
        // so the chain verifies when the sum is 0) and tags the chain.
        if (p.wg_tag) {
            __syncthreads();
            const uint32_t chain = (uint32_t)wave / p.segs_full;
            if ((uint64_t)wave < p.n_items && (uint32_t)wave == chain * p.segs_full && lane == 0) {
                const uint32_t S = chain == p.n_chains - 1 ? p.segs_last : p.segs_full;
                uint4 m = lds4[kWgTagBase + 16 + wslot];
                for (uint32_t s = 0; s < S; ++s) {
                    const uint4 g = lds4[kWgTagBase + wslot + s];
                    m.x ^= g.x; m.y ^= g.y; m.z ^= g.z; m.w ^= g.w;
                }
                emit_tag<ENC>(p, p.chain_base + chain, u4{{m.x, m.y, m.z, m.w}}, zero4());
            }
        }
    }
}

// Chains cut into segments: T = mask xor the XOR of the chain's weighted
// partials. One wave per chain: the lanes load the partials side by side and
// the wave XOR-sums them.
constexpr int kTagThreads = 256;

template <bool ENC, bool RAG>
__global__ __launch_bounds__(kTagThreads) void chain_tag_kernel(GcmLaunch p)
{
    const uint32_t chain = __builtin_amdgcn_readfirstlane(blockIdx.x * (kTagThreads / 64) + (threadIdx.x >> 6));
    const uint32_t lane = threadIdx.x & 63;
    if (chain >= p.n_chains)
        return;
    const uint64_t gchain = p.chain_base + chain;
    uint32_t S;
    uint64_t base, item0;   // segment s >= 1 has partial slot base + s; segment 0 has item0
    if constexpr (RAG) {
        const RaggedChain rc = p.rchains[chain];
        S = rc.segs;
        base = rc.item_base;
        item0 = rc.item0;
    } else {
        S = chain == p.n_chains - 1 ? p.segs_last : p.segs_full;
        base = (uint64_t)chain * p.segs_full;
        item0 = base;
    }
    u4 t = zero4();
    for (uint32_t s = lane; s < S; s += 64) {
        const uint4 g = p.partials[s == 0 ? item0 : base + s];
        t.w[0] ^= g.x; t.w[1] ^= g.y; t.w[2] ^= g.z; t.w[3] ^= g.w;
    }
    t = wave_xor(t);
    if (lane == 0) {
        const uint4 m = p.masks[chain];
        t.w[0] ^= m.x; t.w[1] ^= m.y; t.w[2] ^= m.z; t.w[3] ^= m.w;
        emit_tag<ENC>(p, gchain, t, ENC ? zero4() : load16(p.tags_in + 16 * gchain));
    }
}

template <class LK>
__device__ inline u4 j0_mask(const GcmLaunch &p, uint64_t gchain, LK T)
{
    uint32_t iv[3];
    chain_iv(p, gchain, iv);
    const u4 j0 = {{iv[0], iv[1], iv[2], bswap32(1u)}};
    return aes256_encrypt_tt(j0, p.ctx->rk, T);
}

// The paper's baseline authentication: one thread per chain, Horner with H over
// A, then every ciphertext block in order, then the length block. Each step
// multiplies by H through an 8-bit table of H in LDS (16 lookups), laid out and
// read like the streaming kernel's table of H^L (value-major, the lanes' byte
// positions rotated so that 16 lanes read 16 different bank groups), so the
// baseline gets the same table machinery as the multi-chain path and differs
// only in being one sequential chain per tag.
template <bool ENC>
__global__ __launch_bounds__(256) void seq_ghash_kernel(GcmLaunch p)
{
    __shared__ uint4 s_tab[4096];   // entry (position k, value v) at v * 16 + k: (byte v at byte k) . H
    __shared__ uint32_t s_t0[256];
    const KeyCtx *__restrict__ c = p.ctx;
    const Tab4 *h1 = &c->h1_tab;
    for (uint32_t e = threadIdx.x; e < 4096; e += 256) {
        const uint32_t v = e >> 4, k = e & 15;   // byte k: nibble positions 2k (high) and 2k+1 (low)
        const uint4 hi = *reinterpret_cast<const uint4 *>(h1->e[2 * k][v >> 4]);
        const uint4 lo = *reinterpret_cast<const uint4 *>(h1->e[2 * k + 1][v & 15]);
        s_tab[e] = make_uint4(hi.x ^ lo.x, hi.y ^ lo.y, hi.z ^ lo.z, hi.w ^ lo.w);
    }
    s_t0[threadIdx.x] = c->t0[threadIdx.x];
    __syncthreads();
    const uint32_t chain = blockIdx.x * blockDim.x + threadIdx.x;
    if (chain >= p.n_chains)
        return;
    const char *lds = reinterpret_cast<const char *>(s_tab);
    const GhLane gk = ghash_lane(threadIdx.x & 63, 0u);
    auto mul_h = [&](const u4 &x) { return ghash_step(lds, x, zero4(), gk); };   // x . H
    const uint64_t gchain = p.chain_base + chain;
    const bool last = chain == p.n_chains - 1;
    const uint64_t len_i = last ? p.last_len : p.chain_bytes;
    u4 y = zero4();
    const uint8_t *a = p.aad + gchain * p.aad_bytes;
    for (uint32_t off = 0; off < p.aad_bytes; off += 16) {
        const uint32_t n = p.aad_bytes - off < 16 ? p.aad_bytes - off : 16;
        y = mul_h(xor4(y, load_bytes(a + off, n)));
    }
    const uint8_t *ct = (ENC ? p.out : p.in) + (uint64_t)chain * p.chain_bytes;
    const uint64_t whole = len_i / 16;
    for (uint64_t t = 0; t < whole; ++t) {
        const uint4 x = reinterpret_cast<const uint4 *>(ct)[t];
        const u4 xv = {{x.x, x.y, x.z, x.w}};
        y = mul_h(xor4(y, xv));
    }
    if (len_i & 15)
        y = mul_h(xor4(y, load_bytes(ct + 16 * whole, (uint32_t)(len_i & 15))));
    const uint64_t abits = (uint64_t)p.aad_bytes * 8, cbits = len_i * 8;
    const u4 lens = {{bswap32((uint32_t)(abits >> 32)), bswap32((uint32_t)abits), bswap32((uint32_t)(cbits >> 32)),
                      bswap32((uint32_t)cbits)}};
    y = mul_h(xor4(y, lens));
    const u4 tag = xor4(y, j0_mask(p, gchain, [&](uint32_t x) { return s_t0[x]; }));
    emit_tag<ENC>(p, gchain, tag, ENC ? zero4() : load16(p.tags_in + 16 * gchain));
}

template <bool ENC, int MODE, bool RAG>
static hipError_t launch_mode(const GcmLaunch &p, int num_cu, hipStream_t s)
{
    constexpr bool ghash = MODE == kFused || MODE == kVerify || MODE == kApplyKs;
    if (p.n_items == 0)
        return hipSuccess;
    const uint64_t per_wave = 64u >> p.lanes_log2;
    const uint64_t waves = (p.n_items + per_wave - 1) / per_wave;
    // One workgroup per CU (or per wave when there are fewer waves than CUs):
    // the kernel numbers waves across workgroups, so small launches use every CU.
    uint64_t wgs = waves;
    if (wgs > (uint64_t)num_cu * gcm_wgs_per_cu(MODE))
        wgs = (uint64_t)num_cu * gcm_wgs_per_cu(MODE);
    const bool split = ghash && p.split;
    // One item per wave with every chain's segments inside one workgroup: the
    // workgroup tags the chains itself and the per-chain tag kernel is not needed.
    GcmLaunch q = p;
    q.wg_tag = MODE == kFused && !RAG && split && p.lanes_log2 == 6 && p.n_items == wgs * kWavesPerWg &&
               p.segs_full <= (uint32_t)kWavesPerWg && kWavesPerWg % p.segs_full == 0;
    q.idle_masks = split && !q.wg_tag && wgs * kWavesPerWg >= waves + (p.n_chains + 63) / 64;
    if (p.lanes_log2 == 4 && !split)
        hipLaunchKernelGGL((gcm_kernel<ENC, 4, false, MODE, RAG>), dim3((uint32_t)wgs), dim3(kThreads), 0, s, q);
    else if (p.lanes_log2 == 4)
        hipLaunchKernelGGL((gcm_kernel<ENC, 4, ghash, MODE, RAG>), dim3((uint32_t)wgs), dim3(kThreads), 0, s, q);
    else if (p.lanes_log2 == 5 && !split)
        hipLaunchKernelGGL((gcm_kernel<ENC, 5, false, MODE, RAG>), dim3((uint32_t)wgs), dim3(kThreads), 0, s, q);
    else if (p.lanes_log2 == 5)
        hipLaunchKernelGGL((gcm_kernel<ENC, 5, ghash, MODE, RAG>), dim3((uint32_t)wgs), dim3(kThreads), 0, s, q);
    else if (!split)
        hipLaunchKernelGGL((gcm_kernel<ENC, 6, false, MODE, RAG>), dim3((uint32_t)wgs), dim3(kThreads), 0, s, q);
    else
        hipLaunchKernelGGL((gcm_kernel<ENC, 6, ghash, MODE, RAG>), dim3((uint32_t)wgs), dim3(kThreads), 0, s, q);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || !ghash || !p.split || q.wg_tag)
        return e;
    constexpr uint32_t per_block = kTagThreads / 64;
    hipLaunchKernelGGL((chain_tag_kernel<ENC, RAG>), dim3((p.n_chains + per_block - 1) / per_block), dim3(kTagThreads),
                       0, s, p);
    return hipGetLastError();
}

hipError_t launch_gcm(const GcmLaunch &p, bool encrypt, GcmMode mode, int num_cu, hipStream_t s)
{
    if (p.rchains) {   // ragged chains: the fused path only
        if (mode != kFused)
            return hipErrorInvalidValue;
        return encrypt ? launch_mode<true, kFused, true>(p, num_cu, s) : launch_mode<false, kFused, true>(p, num_cu, s);
    }
    switch (mode) {
    case kFused:
        return encrypt ? launch_mode<true, kFused, false>(p, num_cu, s) : launch_mode<false, kFused, false>(p, num_cu, s);
    case kCtr:
        return launch_mode<false, kCtr, false>(p, num_cu, s);   // CTR is its own inverse
    case kVerify:
        return launch_mode<false, kVerify, false>(p, num_cu, s);
    case kKeystream:
        return launch_mode<false, kKeystream, false>(p, num_cu, s);
    case kApplyKs:
        return launch_mode<false, kApplyKs, false>(p, num_cu, s);
    }
    return hipErrorInvalidValue;
}

// Copies n16 16-byte words from a pinned host buffer (read over the host link)
// to device memory: the upload of a ragged launch's chain and item tables as a
// kernel, which enqueues like any launch instead of holding the calling thread.
// It runs beside the streaming kernel of the call before, so it is a few large
// workgroups with four loads in flight per thread: a grid of ~200 small
// workgroups (one 16-byte word per thread) slowed that kernel by ~15% whenever
// the two overlapped, while 2 to 32 workgroups of 1024 threads made no
// measurable difference to it (1024 samples x 16 chains: 230 -> 206 us per call).
constexpr uint32_t kUploadThreads = 1024;
constexpr uint64_t kUploadMaxWgs = 8;

__global__ __launch_bounds__(kUploadThreads) void upload_kernel(const uint4 *__restrict__ src, uint4 *__restrict__ dst,
                                                                uint64_t n16)
{
    const uint64_t stride = (uint64_t)gridDim.x * kUploadThreads;
    uint64_t i = (uint64_t)blockIdx.x * kUploadThreads + threadIdx.x;
    for (; i + 3 * stride < n16; i += 4 * stride) {
        const uint4 a = src[i], b = src[i + stride], c = src[i + 2 * stride], d = src[i + 3 * stride];
        dst[i] = a;
        dst[i + stride] = b;
        dst[i + 2 * stride] = c;
        dst[i + 3 * stride] = d;
    }
    for (; i < n16; i += stride)
        dst[i] = src[i];
}

hipError_t launch_upload(const void *h_src, void *d_dst, uint64_t bytes, hipStream_t s)
{
    const uint64_t n16 = bytes / 16;
    if (n16 == 0)
        return hipSuccess;
    uint64_t wgs = (n16 + 4 * kUploadThreads - 1) / (4 * kUploadThreads);
    if (wgs > kUploadMaxWgs)
        wgs = kUploadMaxWgs;
    hipLaunchKernelGGL(upload_kernel, dim3((uint32_t)wgs), dim3(kUploadThreads), 0, s,
                       static_cast<const uint4 *>(h_src), static_cast<uint4 *>(d_dst), n16);
    return hipGetLastError();
}

// Measurement helper (not part of the method): the shader clock over a window
// of real time. One wave per workgroup; lane 0 reads the shader-cycle counter
// (s_memtime) and the fixed 100 MHz counter (s_memrealtime) at both ends of a
// sleep loop that lasts `ticks` of the 100 MHz counter (or at most 2^26
// polls), so it ends whatever else runs. Workgroups go to the XCDs in turn.
__global__ __launch_bounds__(64) void clock_probe_kernel(uint64_t ticks, uint64_t *__restrict__ out)
{
    if (threadIdx.x != 0)
        return;
    const uint64_t c0 = __builtin_amdgcn_s_memtime();
    const uint64_t r0 = __builtin_amdgcn_s_memrealtime();
    uint64_t r1 = r0;
    for (uint32_t i = 0; i < (1u << 26) && r1 - r0 < ticks; ++i) {
        __builtin_amdgcn_s_sleep(20);
        r1 = __builtin_amdgcn_s_memrealtime();
    }
    const uint64_t c1 = __builtin_amdgcn_s_memtime();
    out[2 * blockIdx.x] = c1 - c0;
    out[2 * blockIdx.x + 1] = r1 - r0;
}

hipError_t launch_clock_probe(uint64_t ticks, uint32_t n_wg, uint64_t *out, hipStream_t s)
{
    hipLaunchKernelGGL(clock_probe_kernel, dim3(n_wg), dim3(64), 0, s, ticks, out);
    return hipGetLastError();
}

hipError_t launch_seq_ghash(const GcmLaunch &p, bool encrypt, hipStream_t s)
{
    const uint32_t wgs = (p.n_chains + 255) / 256;
    if (encrypt)
        hipLaunchKernelGGL(seq_ghash_kernel<true>, dim3(wgs), dim3(256), 0, s, p);
    else
        hipLaunchKernelGGL(seq_ghash_kernel<false>, dim3(wgs), dim3(256), 0, s, p);
    return hipGetLastError();
}

}  // namespace fastrack
