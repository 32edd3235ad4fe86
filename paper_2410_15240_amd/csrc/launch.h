// Host-side launch interface between the C ABI (api.hip) and the kernels
// (kernels.hip). Internal to the library.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "keyctx.h"

namespace fastrack {

// Threads per workgroup of the streaming kernel. Its 160 KiB of LDS allow one
// workgroup per CU, so this is also the number of resident threads per CU:
// 16 waves, four per SIMD, which the kernel's register use (at most 128 VGPRs)
// allows. More waves per SIMD hide more of the LDS latency of the table lookups.
#ifndef FT_GCM_THREADS
#define FT_GCM_THREADS 1024
#endif
constexpr int kGcmThreads = FT_GCM_THREADS;
constexpr int kGcmWavesPerWg = kGcmThreads / 64;

// What a launch of the streaming kernel computes.
enum GcmMode : int {
    kFused = 0,       // AES-CTR XOR the data and GHASH over the ciphertext, then the tag
    kCtr = 1,         // AES-CTR XOR the data only (plaintext released before verification)
    kVerify = 2,      // GHASH over the ciphertext and the tag check only (no data written)
    kKeystream = 3,   // the CTR keystream alone, written to `out` (no data read)
    kApplyKs = 4,     // out = in XOR a precomputed keystream `ks`, GHASH over `in`, tag check
};

// Workgroups of the streaming kernel per CU: the modes with data AES take 152
// KiB of a CU's LDS; the GHASH-only modes take 113 KiB (the GHASH table, a
// plain T0 and the six lane-combine tables) and also run one 1024-thread
// workgroup, 16 waves, per CU.
constexpr int gcm_wgs_per_cu(int mode)
{
    return (mode == kVerify || mode == kApplyKs) && kGcmWavesPerWg < 16 ? 16 / kGcmWavesPerWg : 1;
}

// One chain of a ragged launch: bytes [off, off + len) of the buffers (off a
// multiple of 16), cut into `segs` segments. Items (and their partial slots) are
// ordered with every chain's segment 0 first, then the other segments chain by
// chain: segment 0 is item item0, segment s >= 1 is item item_base + s.
struct RaggedChain {
    uint64_t off;
    uint64_t len;
    uint64_t item_base;
    uint32_t segs;
    uint32_t item0;
};

// One launch of the streaming kernel over `n_chains` consecutive chains.
// The work is split into items (chain, segment); a segment is a run of
// 2^seg_log2 blocks aligned to the END of its chain (segment 0 may be short).
// Each item is handled by 2^lanes_log2 lanes of a wave; a wave takes
// 64 >> lanes_log2 consecutive items at a time.
struct GcmLaunch {
    const KeyCtx *ctx;
    const uint8_t *in;          // 16-byte aligned; chain 0 of this launch starts here
    const uint8_t *ks;          // kApplyKs: the keystream, laid out like `in`
    uint8_t *out;               // 16-byte aligned; may equal `in`
    uint64_t chain_bytes;       // multiple of 16
    uint64_t last_len;          // bytes in the last chain of this launch (1..chain_bytes)
    uint64_t chain_base;        // global index of chain 0 (IV, tag, AAD and ok indexing)
    uint64_t n_items;
    uint32_t n_chains;
    uint32_t qc;                // blocks in a full chain
    uint32_t q_last;            // blocks in the last chain (a partial block counts as one)
    uint32_t seg_log2;
    uint32_t lanes_log2;        // lanes per item: 4 (16), 5 (32) or 6 (64); the Horner stride
    uint32_t segs_full;         // segments of a full chain
    uint32_t segs_last;         // segments of the last chain
    uint32_t iv[3];             // base IV as little-endian words
    uint32_t aad_bytes;
    const uint8_t *aad;         // global chain i's AAD at aad + i * aad_bytes
    const uint8_t *tags_in;     // decrypt: received tags, global chain i at tags_in + 16 i
    uint8_t *tags_out;          // encrypt: produced tags
    uint8_t *ok;                // decrypt: ok[global chain] = 1 accept / 0 reject
    // Launches that cut chains into several segments (split = 1) leave each
    // item's weighted GHASH partial in partials[item] and, from segment 0, the
    // chain's mask AES_K(J0) xor L . H in masks[chain]; a per-chain kernel then
    // sums them into the tag. Otherwise every item is a whole chain and tags it.
    uint4 *partials;
    uint4 *masks;
    uint32_t split;
    // Fused launches whose every wave takes exactly one item, with each chain's
    // segments on consecutive waves of one workgroup (a segment count dividing 16):
    // the workgroup sums them in LDS and tags the chain itself (no second kernel).
    uint32_t wg_tag;
    // Split launches tagged by the per-chain kernel whose grid has at least
    // ceil(n_chains / 64) waves beyond its wave-items: those waves compute every
    // chain's mask (one lane per chain) and the working waves skip theirs.
    uint32_t idle_masks;
    // Ragged launches (chains of their own lengths and offsets): the chain table
    // and each item's chain; chain_bytes, qc, last_len and the segs_* fields
    // are then unused. NULL for uniform chains.
    const RaggedChain *rchains;
    const uint32_t *ritem_chain;
};

hipError_t launch_key_setup(const uint32_t key_words[8], KeyCtx *ctx, hipStream_t s);
hipError_t launch_gcm(const GcmLaunch &p, bool encrypt, GcmMode mode, int num_cu, hipStream_t s);
hipError_t launch_seq_ghash(const GcmLaunch &p, bool encrypt, hipStream_t s);
hipError_t launch_clock_probe(uint64_t ticks, uint32_t n_wg, uint64_t *out, hipStream_t s);
// Upload `bytes` (a multiple of 16) from pinned host memory to device memory with a kernel on s.
hipError_t launch_upload(const void *h_src, void *d_dst, uint64_t bytes, hipStream_t s);
// Bitsliced keystream (bitslice.hip): the keystream of every chain of p, as kKeystream computes it.
hipError_t launch_bs_keystream(const GcmLaunch &p, int num_cu, hipStream_t s);

}  // namespace fastrack
