/*
 * fastrack.h -- C ABI of the gfx950 multi-chain AES-256-GCM library.
 *
 * The library implements the GPU side of the paper's secure CPU-to-GPU path
 * (Fastrack, arXiv 2410.15240): authenticated decryption of a transfer with
 * AES-256-GCM restructured as multi-chaining authentication (section 5.2), the
 * reverse direction (encrypt + tag), and a chunked host-to-device pipeline that
 * overlaps PCIe copies with decryption and verification (section 5.3).
 *
 * Chains. A buffer of `len` bytes is split into n = ceil(len / chain_bytes)
 * chains; chain i covers bytes [i*chain_bytes, min(len, (i+1)*chain_bytes)).
 * Each chain is an independent AES-256-GCM message (SP 800-38D, 96-bit IV,
 * 128-bit tag) with
 *     IV_i = base_iv XOR (0^32 || [i]_64)   (chain index big-endian in IV bytes 4..11)
 *     A_i  = aad[i*aad_bytes .. (i+1)*aad_bytes)
 * so chain 0 with no AAD is exactly standard GCM under base_iv. Binding the
 * chain index into the IV (and, if the caller wishes, into the AAD as the
 * paper's serial number, section 5.4) makes reordered chains fail.
 *
 * Pointers. `key` and `base_iv` are HOST pointers (32 and 12 bytes). Names
 * starting with d_ are DEVICE pointers (e.g. a torch tensor's data_ptr()),
 * h_ are HOST pointers. d_ct / d_pt must be 16-byte aligned; tags, AAD and ok
 * arrays have no alignment requirement. The caller allocates and owns every
 * buffer. The library keeps a small per-(device, key) cache of key-derived
 * tables (about 0.9 MiB each) and a per-(device, stream) scratch area for
 * partial GHASH values; fastrack_shutdown() releases both.
 *
 * Asynchrony. Calls enqueue work on the given HIP stream (NULL = the null
 * stream of the current device) and return; results are valid once the stream
 * has completed that work. `stream` is a hipStream_t passed as void*.
 *
 * Errors. The return value is FASTRACK_OK (0) or a negative code; the message
 * of the last failure on the calling thread is fastrack_last_error(). Argument
 * checks happen before any work is enqueued. A failed tag is NOT an error: it
 * sets ok[i] = 0 while the plaintext of that chain is still written (the
 * paper's eager evaluation uses plaintext before authentication completes and
 * abandons it on failure, section 5.3).
 */
#ifndef FASTRACK_H
#define FASTRACK_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum fastrack_status {
    FASTRACK_OK = 0,
    FASTRACK_EINVAL = -1,      /* invalid argument (see each function) */
    FASTRACK_EHIP = -2,        /* a HIP runtime call failed */
    FASTRACK_ENOTPINNED = -3,  /* a host buffer that must be pinned is pageable */
    FASTRACK_ENOMEM = -4       /* device allocation for the key cache or scratch failed */
};

/* flags */
#define FASTRACK_F_SEQ_GHASH 1u  /* the paper's baseline authentication: one sequential
                                    GHASH chain per tag (section 5.2); same output */

/* pipeline modes (fastrack_pipeline_h2d_mode) */
#define FASTRACK_PIPE_FUSED 0u   /* decrypt + verify each chunk in one kernel */
#define FASTRACK_PIPE_EAGER 1u   /* plaintext first, the tag check beside it (section 5.3) */
#define FASTRACK_PIPE_OTP   2u   /* keystream of the next chunk while it is in flight (section 5.3) */
#define FASTRACK_PIPE_DIRECT 3u  /* the kernel reads the pinned buffer over the host link itself */

/* Number of chains, ceil(len / chain_bytes); 0 when chain_bytes is 0. */
uint64_t fastrack_num_chains(uint64_t len, uint64_t chain_bytes);

/*
 * The work plan of a uniform-chain launch, host only (nothing is enqueued, no
 * device is touched): how decrypt + verify and encrypt + tag cut the chains of
 * `len` bytes (section 5.2: each chain is one GCM message) into work items for
 * a GPU with num_cu compute units. A chain of q blocks is cut into segments of
 * 2^seg_log2 blocks aligned to its end (segment 0 takes the rest); each item is
 * one segment, run by 2^lanes_log2 lanes for `iters` iterations.
 *   out[7]  lanes_log2, seg_log2, segments of a full chain, segments of the last
 *           chain, work items, iterations per item, 1 if chains are cut into
 *           several segments (0: every item is a whole chain)
 * EINVAL: NULL out, num_cu == 0, len == 0, chain_bytes as for decrypt, more than
 * 2^32 - 1 chains.
 */
int fastrack_plan(uint64_t len, uint64_t chain_bytes, uint32_t num_cu, uint64_t *out);

/*
 * Decrypt and verify (paper section 5.2: the receiver decrypts with AES-CTR and
 * regenerates each chain's GMAC tag to compare against the received one).
 *   d_ct    [len] ciphertext on the device
 *   d_tags  [n][16] received tags
 *   d_aad   [n][aad_bytes] per-chain AAD; ignored (may be NULL) when aad_bytes == 0
 *   d_pt    [len] plaintext out; may equal d_ct exactly (in place), must not
 *           overlap it otherwise
 *   d_ok    [n] out: 1 = tag verified, 0 = rejected
 *   flags   0 or FASTRACK_F_SEQ_GHASH
 * EINVAL: NULL key/base_iv/d_ct/d_pt/d_tags/d_ok, or NULL d_aad with
 * aad_bytes > 0; chain_bytes == 0, not a multiple of 16, or above
 * (2^32 - 2) * 16; d_ct/d_pt not 16-byte aligned or partially overlapping;
 * more than 2^32 - 1 chains; unknown flags. len == 0 is a successful no-op.
 */
int fastrack_gcm_decrypt_verify(const uint8_t *key, const uint8_t *base_iv, uint64_t chain_bytes,
                                const uint8_t *d_ct, uint64_t len, const uint8_t *d_tags,
                                const uint8_t *d_aad, uint32_t aad_bytes, uint8_t *d_pt, uint8_t *d_ok,
                                uint32_t flags, void *stream);

/*
 * Allocation-free decrypt and verify, for callers that cannot allocate device
 * memory: code under HIP graph capture, serving loops and harnesses that forbid
 * hipMalloc. The same computation, arguments, outputs and errors as
 * fastrack_gcm_decrypt_verify (flags included), with no hipMalloc, hipFree or
 * other device allocation on any call.
 * Its device memory is one static array of FASTRACK_NOALLOC_SCRATCH_BYTES per
 * GPU, held until the process ends: the key tables of the last key this entry
 * point was called with on that GPU (rebuilt in place by a kernel on `stream`
 * when the key changes), then the 16-byte GHASH partials (one per work item) and
 * chain masks (one per chain) of launches that cut chains into segments.
 * Every call on one GPU shares that GPU's array and leaves its contents behind:
 * calls that overlap on one GPU (on streams not ordered with each other) race on
 * it and give wrong results; order them. fastrack_shutdown() clears the key
 * tables.
 * EINVAL as fastrack_gcm_decrypt_verify, and also when a launch would need more
 * than FASTRACK_NOALLOC_MAX_PARTIALS partial slots (items + chains); the
 * library's work planner stays below about 200,000 for every size, so this
 * limit is a guard, not a size cap callers meet.
 */
#define FASTRACK_NOALLOC_SCRATCH_BYTES (5u << 20)
#define FASTRACK_NOALLOC_MAX_PARTIALS 230240u
int fastrack_gcm_decrypt_verify_noalloc(const uint8_t *key, const uint8_t *base_iv, uint64_t chain_bytes,
                                        const uint8_t *d_ct, uint64_t len, const uint8_t *d_tags,
                                        const uint8_t *d_aad, uint32_t aad_bytes, uint8_t *d_pt, uint8_t *d_ok,
                                        uint32_t flags, void *stream);

/*
 * Encrypt and tag: the GPU-to-CPU direction (paper section 1.1: the sender
 * encrypts and generates the MAC tag). Same chain layout and checks as above.
 *   d_pt    [len] plaintext on the device
 *   d_ct    [len] ciphertext out; may equal d_pt exactly
 *   d_tags  [n][16] tags out
 */
int fastrack_gcm_encrypt_tag(const uint8_t *key, const uint8_t *base_iv, uint64_t chain_bytes,
                             const uint8_t *d_pt, uint64_t len, const uint8_t *d_aad, uint32_t aad_bytes,
                             uint8_t *d_ct, uint8_t *d_tags, uint32_t flags, void *stream);

/*
 * Eager evaluation (paper section 5.3, "Eager evaluation"): the plaintext is
 * released before the tags are checked. AES-CTR writes d_pt on decrypt_stream;
 * GHASH over d_ct and the tag comparison run on verify_stream, which first
 * waits for the work already queued on decrypt_stream. d_pt is valid when
 * decrypt_stream completes, d_ok when verify_stream completes; a caller that
 * used the plaintext discards that work for every chain with ok[i] = 0.
 * Arguments as in fastrack_gcm_decrypt_verify (no flags); d_pt may not be
 * d_ct (EINVAL), since the ciphertext is read by the verification.
 */
int fastrack_gcm_decrypt_eager(const uint8_t *key, const uint8_t *base_iv, uint64_t chain_bytes,
                               const uint8_t *d_ct, uint64_t len, const uint8_t *d_tags, const uint8_t *d_aad,
                               uint32_t aad_bytes, uint8_t *d_pt, uint8_t *d_ok, void *decrypt_stream,
                               void *verify_stream);

/*
 * One-time-pad precompute (paper section 5.3, "Parallel AES evaluation"): the
 * CTR keystream depends only on the key, the IVs and the counters, so it can
 * be generated before the ciphertext arrives.
 * fastrack_gcm_keystream writes to d_ks[len] the keystream of the chains
 * chain_base, chain_base+1, ... that cover len bytes (chain chain_base + i at
 * d_ks + i*chain_bytes; the last chain may be short). d_ks is 16-byte aligned.
 * fastrack_gcm_apply_verify then computes d_pt = d_ct XOR d_ks and verifies
 * the same chains: tags, AAD and ok flags are indexed by GLOBAL chain index,
 * d_tags + 16*(chain_base + i), d_aad + aad_bytes*(chain_base + i),
 * d_ok[chain_base + i], so they point at the arrays of the whole message.
 * d_pt may equal d_ct or d_ks exactly; partial overlaps are EINVAL.
 */
int fastrack_gcm_keystream(const uint8_t *key, const uint8_t *base_iv, uint64_t chain_bytes, uint64_t chain_base,
                           uint64_t len, uint8_t *d_ks, void *stream);
/*
 * The same keystream as fastrack_gcm_keystream (same arguments, same output,
 * same errors), computed by a bitsliced AES-256 (FIPS-197 rounds as Boolean
 * circuits on 32 blocks per 32-bit lane, no table lookups) instead of the
 * T-table kernel: the alternative AES formulation, kept to compare the two on
 * this GPU. A wave pass covers 2048 consecutive blocks of one chain, so chains
 * much shorter than 32 KiB leave most of a pass idle.
 */
int fastrack_gcm_keystream_bitsliced(const uint8_t *key, const uint8_t *base_iv, uint64_t chain_bytes,
                                     uint64_t chain_base, uint64_t len, uint8_t *d_ks, void *stream);
int fastrack_gcm_apply_verify(const uint8_t *key, const uint8_t *base_iv, uint64_t chain_bytes, uint64_t chain_base,
                              const uint8_t *d_ct, uint64_t len, const uint8_t *d_ks, const uint8_t *d_tags,
                              const uint8_t *d_aad, uint32_t aad_bytes, uint8_t *d_pt, uint8_t *d_ok,
                              void *stream);

/* Bytes of device staging that fastrack_pipeline_h2d needs for these sizes
 * (0 for an invalid depth or chain_bytes = 0). */
uint64_t fastrack_pipeline_stage_bytes(uint64_t len, uint64_t chain_bytes, uint32_t aad_bytes,
                                       uint64_t chunk_bytes, int depth);

/*
 * Pipelined host-to-device decrypt + verify (paper section 5.3, decryption
 * pipeline): ciphertext in a pinned host "bounce buffer" (section 3.1) is
 * copied in chunks of chunk_bytes on copy_stream, and each chunk's chains are
 * decrypted and verified on compute_stream while the next chunks are in flight.
 *   h_ct         [len] ciphertext, PINNED host memory: all of [h_ct, h_ct + len)
 *                inside one pinned allocation (ENOTPINNED otherwise)
 *   h_tags       [n][16] host tags; h_aad [n][aad_bytes] host AAD (or NULL)
 *   chunk_bytes  a nonzero multiple of chain_bytes
 *   depth        0: each chunk is copied to its place in d_pt and decrypted in
 *                place (no slot is reused);
 *                2..8: a ring of `depth` device staging slots in d_stage; a
 *                slot is refilled only after the decrypt that last read it
 *   d_stage      device workspace, 256-byte aligned, of
 *                stage_bytes >= fastrack_pipeline_stage_bytes(...): the ring
 *                (depth > 0), then the tags and the AAD
 *   d_pt, d_ok   device outputs as in fastrack_gcm_decrypt_verify
 * The calling thread paces the copies: before enqueueing the copy of chunk k it
 * waits until chunk k - W has been decrypted (W = depth with a ring, 4 in place),
 * so the call returns about W chunks before the transfer ends and copy_stream
 * never waits on the device for compute_stream. Results are valid once
 * compute_stream has completed (it waits on the copies).
 * EINVAL additionally covers chunk_bytes, depth and an undersized d_stage.
 */
int fastrack_pipeline_h2d(const uint8_t *key, const uint8_t *base_iv, uint64_t chain_bytes,
                          const uint8_t *h_ct, uint64_t len, const uint8_t *h_tags, const uint8_t *h_aad,
                          uint32_t aad_bytes, uint64_t chunk_bytes, int depth, uint8_t *d_stage,
                          uint64_t stage_bytes, uint8_t *d_pt, uint8_t *d_ok, void *copy_stream,
                          void *compute_stream);

/*
 * The operations fastrack_pipeline_h2d(_mode) enqueues, in order, for these sizes
 * (the paper's decryption pipeline, section 5.3): a pure host function with no
 * device access, for inspecting and checking the schedule.
 *   h_ops    host array of max_ops records of 6 int64 each, written in order:
 *            kind, stream, event, chunk, slot, aux. May be NULL (count only).
 *            kind: 0 upload tags + AAD, 1 record `event`, 2 wait for the last
 *            record of `event`, 3 copy chunk `chunk` into buffer `slot`, 4 keystream
 *            of chunk `chunk` into ring slot `slot`, 5 decrypt + verify chunk
 *            `chunk` read from buffer `slot`, 6 XOR keystream slot `aux` into chunk
 *            `chunk` read from buffer `slot` + tag check, 7 decrypt only, 8 tag
 *            check only, 9 the calling thread waits until the last record of
 *            `event` (that of chunk `chunk`) has completed, 10 decrypt + verify of
 *            the whole buffer read from host memory by the kernel. Buffer slot -1
 *            is the chunk's own place in d_pt, 0..depth-1 a staging slot.
 *            stream: 0 copy, 1 compute, 2 verify. event: -1 none.
 * Returns the number of operations (>= 0; 0 for len = 0) or FASTRACK_EINVAL for
 * the argument errors the pipeline itself rejects (chunk_bytes, depth, mode).
 */
int64_t fastrack_pipeline_plan(uint64_t len, uint64_t chain_bytes, uint64_t chunk_bytes, int depth, uint32_t mode,
                               int64_t *h_ops, uint64_t max_ops);

/*
 * fastrack_pipeline_h2d with a mode:
 *   FASTRACK_PIPE_FUSED  as fastrack_pipeline_h2d (verify_stream unused)
 *   FASTRACK_PIPE_EAGER  chunks land in a ring of depth >= 2 staging slots; each
 *                        chunk's plaintext is written on compute_stream as soon
 *                        as it has arrived, and its tags are checked on
 *                        verify_stream beside the next copies. d_pt is valid
 *                        when compute_stream completes, d_ok when verify_stream
 *                        completes.
 *   FASTRACK_PIPE_OTP    chunks are copied to their place in d_pt; the keystream
 *                        of chunk k+1 is generated on compute_stream into one of
 *                        depth >= 2 slots while chunk k+1 is in flight, so once
 *                        it lands only the XOR and the tag check remain.
 *   FASTRACK_PIPE_DIRECT no copy engine and no chunks: after the tags and AAD
 *                        are uploaded on copy_stream, one decrypt + verify
 *                        launch on compute_stream reads h_ct through its device
 *                        mapping, so the transfer and the decryption are the
 *                        same loads. Needs depth 0. The launch occupies every
 *                        compute unit for the whole transfer (PCIe-bound), where
 *                        the chunked modes leave them free between chunks.
 * d_stage is sized by fastrack_pipeline_stage_bytes(..., depth) for every mode.
 * EINVAL additionally covers an unknown mode, depth 0 with EAGER or OTP, and
 * depth > 0 with DIRECT.
 */
int fastrack_pipeline_h2d_mode(const uint8_t *key, const uint8_t *base_iv, uint64_t chain_bytes,
                               const uint8_t *h_ct, uint64_t len, const uint8_t *h_tags, const uint8_t *h_aad,
                               uint32_t aad_bytes, uint64_t chunk_bytes, int depth, uint32_t mode,
                               uint8_t *d_stage, uint64_t stage_bytes, uint8_t *d_pt, uint8_t *d_ok,
                               void *copy_stream, void *compute_stream, void *verify_stream);

/*
 * Pipelined encrypt + device-to-host copy (the reverse direction of the
 * paper's section 5.3 pipeline, for results and gradients leaving the GPU):
 * each chunk of chunk_bytes of d_pt is encrypted and tagged on compute_stream
 * into d_ct (+ the same offset; d_ct may equal d_pt), and copied to the pinned
 * host buffer h_ct on copy_stream while later chunks are encrypted. The tags
 * (d_tags, n x 16 on the device) follow to h_tags[n][16] at the end. The
 * copies are paced from the host: the call enqueues every encryption, then
 * waits on the host for each group of chunks (at least 32 MiB) to be encrypted
 * before enqueueing its copies, and returns once all copies are enqueued (the
 * encryptions are then done; the copies may still be running).
 *   d_aad        [n][aad_bytes] device AAD, or NULL with aad_bytes = 0
 *   h_ct         [len] PINNED host memory, all of it inside one pinned
 *                allocation (ENOTPINNED otherwise)
 * h_ct and h_tags are valid once copy_stream has completed.
 * EINVAL covers the checks of fastrack_gcm_encrypt_tag, chunk_bytes (a nonzero
 * multiple of chain_bytes) and NULL h_ct, h_tags or d_tags.
 */
int fastrack_pipeline_d2h(const uint8_t *key, const uint8_t *base_iv, uint64_t chain_bytes, const uint8_t *d_pt,
                          uint64_t len, const uint8_t *d_aad, uint32_t aad_bytes, uint64_t chunk_bytes,
                          uint8_t *d_ct, uint8_t *d_tags, uint8_t *h_ct, uint8_t *h_tags, void *copy_stream,
                          void *compute_stream);

/*
 * fastrack_pipeline_d2h with a mode:
 *   FASTRACK_PIPE_FUSED  as fastrack_pipeline_d2h
 *   FASTRACK_PIPE_DIRECT one encrypt + tag launch on compute_stream writes the
 *                        ciphertext straight into h_ct through its device
 *                        mapping (d_ct is not used and may be NULL); the tags
 *                        follow to h_tags on compute_stream, and copy_stream
 *                        waits for both. The launch occupies every compute unit
 *                        for the whole transfer.
 * h_ct must lie inside one pinned allocation for both modes (ENOTPINNED).
 * EINVAL additionally covers the other modes; chunk_bytes is checked as for the
 * chunked mode in both.
 */
int fastrack_pipeline_d2h_mode(const uint8_t *key, const uint8_t *base_iv, uint64_t chain_bytes,
                               const uint8_t *d_pt, uint64_t len, const uint8_t *d_aad, uint32_t aad_bytes,
                               uint64_t chunk_bytes, uint8_t *d_ct, uint8_t *d_tags, uint8_t *h_ct, uint8_t *h_tags,
                               void *copy_stream, void *compute_stream, uint32_t mode);

/*
 * Ragged chains: the paper's per-sample layout (section 5.2: every input sample
 * of a batch is cut into several chains, each with its own tag and a one-byte
 * serial number as AAD; section 5.4: the serial number exposes reordering).
 * Chain i is bytes [h_chain_off[i], h_chain_off[i] + h_chain_len[i]) of the
 * device buffers, an independent GCM message under IV_i (the chain index i as
 * above), with AAD i at d_aad + i * aad_bytes, tag i at d_tags + 16 i and
 * ok[i]. Lengths are free (0 allowed: the tag then covers the AAD alone).
 *   h_chain_off  [n_chains] HOST array: byte offsets, each a multiple of 16,
 *                increasing, chains not overlapping (gaps are left untouched)
 *   h_chain_len  [n_chains] HOST array: byte lengths, each at most (2^32-2)*16
 * d_ct and d_pt (or d_pt and d_ct) may be NULL when every chain is empty.
 * The host arrays are read during the call only. The chain table goes to the
 * device through a per-stream pinned staging buffer that the library owns; a
 * later call on the same stream reuses it once the device has read it.
 * EINVAL: as for fastrack_gcm_decrypt_verify / fastrack_gcm_encrypt_tag, plus
 * NULL h_chain_off/h_chain_len with n_chains > 0, a misaligned, decreasing or
 * overlapping offset, an oversized chain, more than 2^32-1 chains or work items.
 * n_chains == 0 is a successful no-op.
 */
int fastrack_gcm_decrypt_verify_ragged(const uint8_t *key, const uint8_t *base_iv, const uint64_t *h_chain_off,
                                       const uint64_t *h_chain_len, uint64_t n_chains, const uint8_t *d_ct,
                                       const uint8_t *d_tags, const uint8_t *d_aad, uint32_t aad_bytes,
                                       uint8_t *d_pt, uint8_t *d_ok, void *stream);

int fastrack_gcm_encrypt_tag_ragged(const uint8_t *key, const uint8_t *base_iv, const uint64_t *h_chain_off,
                                    const uint64_t *h_chain_len, uint64_t n_chains, const uint8_t *d_pt,
                                    const uint8_t *d_aad, uint32_t aad_bytes, uint8_t *d_ct, uint8_t *d_tags,
                                    void *stream);

/*
 * Host helper for the per-sample layout: samples of h_sample_len[s] bytes are
 * packed back to back, each starting 16-byte aligned, and each is cut into
 * chains_per_sample chains of equal whole-block parts (the last part shorter,
 * parts past the end of a short sample empty and placed at the sample's
 * 16-byte-rounded end, so every offset is 16-byte aligned and the layout passes
 * the ragged entry points' chain checks). Writes n_samples *
 * chains_per_sample entries to h_chain_off / h_chain_len and returns the
 * packed buffer size in bytes (0 on NULL arrays or chains_per_sample == 0).
 */
uint64_t fastrack_sample_chains(const uint64_t *h_sample_len, uint64_t n_samples, uint32_t chains_per_sample,
                                uint64_t *h_chain_off, uint64_t *h_chain_len);

/*
 * Measurement helper, not part of the method: enqueues on `stream` one wave per
 * probe (n_probes in 1..1024; probes go to the XCDs in turn) that sleeps for
 * window_us microseconds of real time (1..10^7) and writes to d_out[2p] the
 * shader-clock cycles and to d_out[2p+1] the 100 MHz real-time ticks that
 * elapsed, so cycles / (ticks / 100 MHz) is the shader clock over the window.
 * Launched on a second stream beside other work, it measures the clock that
 * work runs at (each probe holds one wave slot and almost no issue cycles).
 * EINVAL: NULL d_out, n_probes or window_us out of range.
 */
int fastrack_clock_probe(uint64_t window_us, uint32_t n_probes, uint64_t *d_out, void *stream);

/* Message of the last failure on this thread ("" if none). */
const char *fastrack_last_error(void);

/* Release the key-table cache and scratch areas (waits for the device first). */
void fastrack_shutdown(void);

#ifdef __cplusplus
}
#endif

#endif /* FASTRACK_H */
