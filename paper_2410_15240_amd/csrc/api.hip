// C ABI of the multi-chain AES-256-GCM library: argument checks, the per-key
// table cache, per-stream scratch, work planning and the H2D pipeline.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <array>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "fastrack.h"
#include "keyctx.h"
#include "launch.h"

using namespace fastrack;

#define FT_EXPORT extern "C" __attribute__((visibility("default")))

namespace {

thread_local std::string g_err;

int fail(int code, const char *fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
    return code;
}

int hip_fail(hipError_t e, const char *what)
{
    return fail(FASTRACK_EHIP, "%s: %s", what, hipGetErrorString(e));
}

constexpr uint64_t kMaxChainBlocks = 0xFFFFFFFEull;   // GCM: at most 2^32 - 2 blocks per message
constexpr size_t kMaxKeys = 8;
constexpr int kMinSegLog2 = 8;                          // segments of >= 256 blocks (4 per lane)
constexpr int kMinSmallSegLog2 = 7;                     // small launches: down to 128 blocks (2 per lane)
constexpr uint64_t kMaxSmallSegs = 512;                 // ... with at most this many segments per chain
constexpr int kMaxPipelineDepth = 8;                    // staging-ring slots
constexpr uint64_t kD2hGroupBytes = 32ull << 20;        // D2H: encrypted bytes per copy-stream wait

struct KeyEntry {
    int dev;
    std::array<uint8_t, 32> key;
    KeyCtx *ctx;
    hipEvent_t ready;
    uint64_t last_use;
    int slot;            // its slot in the device's key pool
    bool done = false;   // `ready` has been observed complete
};

// Per device, kMaxKeys key contexts in one allocation and an event per slot,
// made with the first key on that device: a new key then allocates nothing
// (a device allocation held the calling thread ~0.1 ms, more than the key
// setup itself).
constexpr size_t kKeySlotBytes = (sizeof(KeyCtx) + 255) & ~(size_t)255;   // slots 256-byte aligned

struct KeyPool {
    int dev;
    uint8_t *base = nullptr;
    hipEvent_t ready[kMaxKeys] = {};
    bool used[kMaxKeys] = {};
};

struct ScratchEntry {
    int dev;
    hipStream_t stream;
    void *ptr;
    size_t bytes;
    // two pinned host staging buffers for the tables of ragged launches, used in
    // turn, and for each the event after the copy that last read it
    void *host[2] = {nullptr, nullptr};
    void *host_dev[2] = {nullptr, nullptr};   // their device addresses
    size_t host_bytes[2] = {0, 0};
    hipEvent_t host_read[2] = {nullptr, nullptr};
    int cur = 0;
    // Ragged launches: two device table slots (written only by the uploads, read
    // only by the ragged kernels), the library's upload stream, and for each slot
    // the event after the kernels that last read it.
    void *rtab = nullptr;
    size_t rtab_slot = 0;
    hipStream_t up = nullptr;
    hipEvent_t slot_free[2] = {nullptr, nullptr};
    bool slot_used[2] = {false, false};
};

struct DevInfo {
    int dev;
    int num_cu;
};

std::mutex g_mu;
std::vector<KeyEntry> g_keys;
std::vector<KeyPool> g_pools;
std::vector<ScratchEntry> g_scratch;
std::vector<DevInfo> g_dev;
uint64_t g_tick = 0;

int num_cu_of(int dev, int *out)
{
    for (auto &d : g_dev)
        if (d.dev == dev) {
            *out = d.num_cu;
            return FASTRACK_OK;
        }
    int n = 0;
    hipError_t e = hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess)
        return hip_fail(e, "hipDeviceGetAttribute");
    g_dev.push_back({dev, n});
    *out = n;
    return FASTRACK_OK;
}

KeyPool *pool_of(int dev)
{
    for (auto &p : g_pools)
        if (p.dev == dev)
            return &p;
    return nullptr;
}

int pool_for(int dev, KeyPool **out)
{
    if ((*out = pool_of(dev)))
        return FASTRACK_OK;
    KeyPool p;
    p.dev = dev;
    hipError_t he = hipMalloc(reinterpret_cast<void **>(&p.base), kMaxKeys * kKeySlotBytes);
    if (he != hipSuccess)
        return fail(FASTRACK_ENOMEM, "hipMalloc(%zu) for the key tables: %s", kMaxKeys * kKeySlotBytes,
                    hipGetErrorString(he));
    for (size_t i = 0; i < kMaxKeys; ++i)
        if ((he = hipEventCreateWithFlags(&p.ready[i], hipEventDisableTiming)) != hipSuccess) {
            for (size_t j = 0; j < i; ++j)
                (void)hipEventDestroy(p.ready[j]);
            (void)hipFree(p.base);
            return hip_fail(he, "hipEventCreate");
        }
    g_pools.push_back(p);
    *out = &g_pools.back();
    return FASTRACK_OK;
}

// The slot is rewritten whole by the next key's setup; the pool is cleared when freed.
void free_key_entry(KeyEntry &k)
{
    if (KeyPool *p = pool_of(k.dev))
        p->used[k.slot] = false;
}

// Device tables for (current device, key); setup is enqueued on `s` the first time.
int key_ctx(const uint8_t *key, hipStream_t s, int dev, const KeyCtx **out)
{
    std::array<uint8_t, 32> k;
    std::memcpy(k.data(), key, 32);
    for (auto &e : g_keys)
        if (e.dev == dev && e.key == k) {
            e.last_use = ++g_tick;
            if (!e.done) {   // the setup may still be running on the stream it was enqueued on
                if (hipEventQuery(e.ready) == hipSuccess) {
                    e.done = true;
                } else {
                    hipError_t he = hipStreamWaitEvent(s, e.ready, 0);
                    if (he != hipSuccess)
                        return hip_fail(he, "hipStreamWaitEvent");
                }
            }
            *out = e.ctx;
            return FASTRACK_OK;
        }
    size_t same_dev = 0, victim = g_keys.size();
    for (size_t i = 0; i < g_keys.size(); ++i)
        if (g_keys[i].dev == dev) {
            ++same_dev;
            if (victim == g_keys.size() || g_keys[i].last_use < g_keys[victim].last_use)
                victim = i;
        }
    KeyPool *pool;
    int rc;
    if ((rc = pool_for(dev, &pool)))
        return rc;
    if (same_dev >= kMaxKeys) {
        // Work queued on any stream may still read the victim's tables.
        hipError_t he = hipDeviceSynchronize();
        if (he != hipSuccess)
            return hip_fail(he, "hipDeviceSynchronize");
        free_key_entry(g_keys[victim]);
        g_keys.erase(g_keys.begin() + (long)victim);
    }
    int slot = 0;
    while (slot < (int)kMaxKeys && pool->used[slot])
        ++slot;
    if (slot == (int)kMaxKeys)
        return fail(FASTRACK_EHIP, "key pool full");   // cannot happen: at most kMaxKeys entries per device
    KeyEntry e;
    e.dev = dev;
    e.key = k;
    e.last_use = ++g_tick;
    e.slot = slot;
    e.ctx = reinterpret_cast<KeyCtx *>(pool->base + (size_t)slot * kKeySlotBytes);
    e.ready = pool->ready[slot];
    uint32_t words[8];
    for (int i = 0; i < 8; ++i)
        words[i] = (uint32_t)key[4 * i] | ((uint32_t)key[4 * i + 1] << 8) | ((uint32_t)key[4 * i + 2] << 16) |
                   ((uint32_t)key[4 * i + 3] << 24);
    hipError_t he = launch_key_setup(words, e.ctx, s);
    std::memset(words, 0, sizeof words);
    if (he != hipSuccess)
        return hip_fail(he, "key setup launch");
    if ((he = hipEventRecord(e.ready, s)) != hipSuccess) {
        (void)hipStreamSynchronize(s);
        return hip_fail(he, "hipEventRecord");
    }
    pool->used[slot] = true;
    g_keys.push_back(e);
    *out = e.ctx;
    return FASTRACK_OK;
}

// Scratch of at least `bytes` private to (device, stream): work on one stream
// is ordered. Zeroed when (re)allocated; every launch rewrites what it reads.
int scratch_for(int dev, hipStream_t s, size_t bytes, void **out)
{
    ScratchEntry *e = nullptr;
    for (auto &x : g_scratch)
        if (x.dev == dev && x.stream == s)
            e = &x;
    if (e && e->bytes >= bytes) {
        *out = e->ptr;
        return FASTRACK_OK;
    }
    if (!e) {
        g_scratch.push_back(ScratchEntry{dev, s, nullptr, 0});
        e = &g_scratch.back();
    } else {
        hipError_t he = hipStreamSynchronize(s);   // earlier launches may still use the old area
        if (he != hipSuccess)
            return hip_fail(he, "hipStreamSynchronize");
        (void)hipFree(e->ptr);
        e->ptr = nullptr;
        e->bytes = 0;
    }
    hipError_t he = hipMalloc(&e->ptr, bytes);
    if (he != hipSuccess) {
        e->ptr = nullptr;
        return fail(FASTRACK_ENOMEM, "hipMalloc(%zu) for scratch: %s", bytes, hipGetErrorString(he));
    }
    he = hipMemsetAsync(e->ptr, 0, bytes, s);
    if (he != hipSuccess) {
        (void)hipFree(e->ptr);
        e->ptr = nullptr;
        return hip_fail(he, "hipMemsetAsync of scratch");
    }
    e->bytes = bytes;
    *out = e->ptr;
    return FASTRACK_OK;
}

// Pinned host staging of at least `bytes` for (device, stream), free to overwrite:
// the copy that last read it has completed. Two buffers are used in turn, so the
// tables of the next call are written while the copy of the last one is pending.
int staging_for(int dev, hipStream_t s, size_t bytes, uint8_t **out)
{
    ScratchEntry *e = nullptr;
    for (auto &x : g_scratch)
        if (x.dev == dev && x.stream == s)
            e = &x;
    if (!e) {
        g_scratch.push_back(ScratchEntry{dev, s, nullptr, 0});
        e = &g_scratch.back();
    }
    e->cur ^= 1;
    const int b = e->cur;
    hipError_t he;
    if (e->host_read[b] && (he = hipEventSynchronize(e->host_read[b])) != hipSuccess)
        return hip_fail(he, "hipEventSynchronize");
    if (!e->host_read[b] && (he = hipEventCreateWithFlags(&e->host_read[b], hipEventDisableTiming)) != hipSuccess) {
        e->host_read[b] = nullptr;
        return hip_fail(he, "hipEventCreate");
    }
    if (e->host_bytes[b] < bytes) {
        if (e->host[b])
            (void)hipHostFree(e->host[b]);
        e->host[b] = nullptr;
        e->host_bytes[b] = 0;
        if ((he = hipHostMalloc(&e->host[b], bytes, hipHostMallocMapped)) != hipSuccess) {
            e->host[b] = nullptr;
            return fail(FASTRACK_ENOMEM, "hipHostMalloc(%zu) for staging: %s", bytes, hipGetErrorString(he));
        }
        if ((he = hipHostGetDevicePointer(&e->host_dev[b], e->host[b], 0)) != hipSuccess) {
            (void)hipHostFree(e->host[b]);
            e->host[b] = nullptr;
            return hip_fail(he, "hipHostGetDevicePointer of the table staging");
        }
        e->host_bytes[b] = bytes;
    }
    *out = static_cast<uint8_t *>(e->host[b]);
    return FASTRACK_OK;
}

// Record on `rs` (the stream whose work reads it) that the staging buffer of
// (dev, s) handed out last has been read by the work queued there so far.
int staging_read(int dev, hipStream_t s, hipStream_t rs)
{
    for (auto &x : g_scratch)
        if (x.dev == dev && x.stream == s) {
            hipError_t he = hipEventRecord(x.host_read[x.cur], rs);
            return he == hipSuccess ? FASTRACK_OK : hip_fail(he, "hipEventRecord");
        }
    return fail(FASTRACK_EHIP, "no staging for this stream");
}

uint32_t ceil_log2(uint64_t x)
{
    uint32_t r = 0;
    while ((1ull << r) < x)
        ++r;
    return r;
}

// Split `len` bytes (chains chain_base ..) into (chain, segment) work items and
// pick the lanes per item. The aim is one item per resident wave-slot: short
// chains get 16 or 32 lanes each (so one wave works on several chains and the
// per-item lane combine is amortised over more blocks per lane); long chains
// get 64 lanes and are cut into segments.
void make_plan(uint64_t len, uint64_t chain_bytes, uint64_t chain_base, uint64_t slots, GcmLaunch &p)
{
    const uint64_t n = (len + chain_bytes - 1) / chain_bytes;
    const uint64_t qc = chain_bytes / 16;
    p.chain_bytes = chain_bytes;
    p.chain_base = chain_base;
    p.n_chains = (uint32_t)n;
    p.qc = (uint32_t)qc;
    p.last_len = len - (n - 1) * chain_bytes;
    p.q_last = (uint32_t)((p.last_len + 15) / 16);
    uint32_t lg = ceil_log2(qc);
    if (lg > 31)
        lg = 31;
    uint32_t ll = 0;
    for (uint32_t cand = 4; cand <= 6; ++cand)
        if (qc >= (4ull << cand) && ((n << cand) + 63) / 64 >= slots) {
            ll = cand;
            break;
        }
    if (ll == 0)   // short chains keep few lanes each; otherwise 64 lanes
        ll = qc >= 256 ? 6 : (qc >= 128 ? 5 : 4);
    auto items_at = [&](uint32_t g) { return n * ((qc + (1ull << g) - 1) >> g); };
    if (ll == 6) {   // too few whole chains to fill the GPU: cut them into segments
        while (lg > (uint32_t)kMinSegLog2 && items_at(lg) < slots)
            --lg;
        // Small launches, where even 256-block segments leave more than half of the
        // waves idle: shorter segments, down to two iterations of the 64 lanes, while
        // a chain stays at most 512 segments (the tag sums and segment weights grow
        // with the count). 1 MiB of 64 KiB chains: 21.8 us with 256-block segments,
        // 18.2 with 128, 19.5 with 64 (whose 6-bit segment weights cost more than the
        // shorter items gain); one 1 MiB chain 22.3 -> 19.6 us; 4 MiB of 1 MiB chains
        // 23.7 -> 21.4 us.
        while (lg > (uint32_t)kMinSmallSegLog2 && items_at(lg) < slots / 2 &&
               ((qc + (1ull << (lg - 1)) - 1) >> (lg - 1)) <= kMaxSmallSegs)
            --lg;
    } else {
        // A few wave-items per wave that do not divide evenly leave some waves with
        // one more than others: cut the chains until each wave has about 4 (segments
        // of at least 4 iterations). Each item ends with a latency-bound tail (the
        // lane combine, the segment weights), so more and shorter items cost more
        // than the balance gains: 4 per wave measured ≈9% faster than 8, and than 2.
        const uint64_t g = 64u >> ll;
        auto wave_items = [&](uint32_t lgv) { return (items_at(lgv) + g - 1) / g; };
        while (lg > ll + 2 && wave_items(lg) < 4 * slots && wave_items(lg) % slots != 0)
            --lg;
    }
    p.lanes_log2 = ll;
    p.seg_log2 = lg;
    p.segs_full = (uint32_t)((qc + (1ull << lg) - 1) >> lg);
    p.segs_last = (uint32_t)((p.q_last + (1ull << lg) - 1) >> lg);
    p.n_items = (n - 1) * p.segs_full + p.segs_last;
}

bool overlap_bad(const void *a, const void *b, uint64_t len)
{
    uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
    if (x == y)
        return false;
    return x < y + len && y < x + len;
}

int check_common(const uint8_t *key, const uint8_t *base_iv, uint64_t chain_bytes, uint64_t len, const void *in,
                 const void *out, const void *aad, uint32_t aad_bytes, uint32_t flags)
{
    if (!key || !base_iv)
        return fail(FASTRACK_EINVAL, "key and base_iv must be non-NULL host pointers");
    if (chain_bytes == 0 || chain_bytes % 16 != 0)
        return fail(FASTRACK_EINVAL, "chain_bytes must be a nonzero multiple of 16 (got %llu)",
                    (unsigned long long)chain_bytes);
    if (chain_bytes / 16 > kMaxChainBlocks)
        return fail(FASTRACK_EINVAL, "chain_bytes above (2^32-2)*16, the GCM message limit");
    if (flags & ~FASTRACK_F_SEQ_GHASH)
        return fail(FASTRACK_EINVAL, "unknown flags 0x%x", flags);
    if (aad_bytes && !aad)
        return fail(FASTRACK_EINVAL, "aad is NULL but aad_bytes = %u", aad_bytes);
    if (len == 0)
        return FASTRACK_OK;
    if (!in || !out)
        return fail(FASTRACK_EINVAL, "input and output buffers must be non-NULL");
    if (((uintptr_t)in & 15) || ((uintptr_t)out & 15))
        return fail(FASTRACK_EINVAL, "input and output buffers must be 16-byte aligned");
    if (overlap_bad(in, out, len))
        return fail(FASTRACK_EINVAL, "input and output overlap without being the same buffer");
    if ((len + chain_bytes - 1) / chain_bytes > 0xFFFFFFFFull)
        return fail(FASTRACK_EINVAL, "more than 2^32-1 chains");
    return FASTRACK_OK;
}

void iv_words(const uint8_t *iv, uint32_t w[3])
{
    for (int j = 0; j < 3; ++j)
        w[j] = (uint32_t)iv[4 * j] | ((uint32_t)iv[4 * j + 1] << 8) | ((uint32_t)iv[4 * j + 2] << 16) |
               ((uint32_t)iv[4 * j + 3] << 24);
}

// Enqueue one launch of `mode` over [in, in+len) covering chains chain_base.. .
int run_gcm(bool encrypt, GcmMode mode, const KeyCtx *ctx, const uint8_t *base_iv, uint64_t chain_bytes,
            uint64_t chain_base, const uint8_t *in, const uint8_t *ks, uint64_t len, uint8_t *out,
            const uint8_t *aad, uint32_t aad_bytes, const uint8_t *tags_in, uint8_t *tags_out, uint8_t *ok,
            uint32_t flags, int dev, int num_cu, hipStream_t s, uint4 *fixed_scratch = nullptr,
            uint64_t fixed_entries = 0)
{
    GcmLaunch p;
    std::memset(&p, 0, sizeof p);
    make_plan(len, chain_bytes, chain_base, (uint64_t)num_cu * kGcmWavesPerWg * gcm_wgs_per_cu(mode), p);
    if (p.n_items > 0xFFFFFFFFull)   // the kernel indexes a launch's items in 32 bits
        return fail(FASTRACK_EINVAL, "more than 2^32-1 work items in one launch");
    p.ctx = ctx;
    p.in = in;
    p.ks = ks;
    p.out = out;
    iv_words(base_iv, p.iv);
    p.aad = aad;
    p.aad_bytes = aad_bytes;
    p.tags_in = tags_in;
    p.tags_out = tags_out;
    p.ok = ok;
    hipError_t he;
    if (mode == kFused && (flags & FASTRACK_F_SEQ_GHASH)) {
        if (!encrypt) {   // tag over the ciphertext before an in-place decrypt overwrites it
            he = launch_seq_ghash(p, false, s);
            if (he != hipSuccess)
                return hip_fail(he, "sequential GHASH launch");
        }
        he = launch_gcm(p, false, kCtr, num_cu, s);
        if (he != hipSuccess)
            return hip_fail(he, "CTR launch");
        if (encrypt) {
            he = launch_seq_ghash(p, true, s);
            if (he != hipSuccess)
                return hip_fail(he, "sequential GHASH launch");
        }
        return FASTRACK_OK;
    }
    const bool ghash = mode == kFused || mode == kVerify || mode == kApplyKs;
    p.split = ghash && p.n_items > p.n_chains ? 1u : 0u;
    if (p.split) {   // chains cut into segments: per-item partials and per-chain masks
        if (fixed_scratch) {   // the caller's fixed area (allocation-free entry point)
            if (p.n_items + p.n_chains > fixed_entries)
                return fail(FASTRACK_EINVAL, "the launch needs %llu partial slots, the fixed scratch holds %llu",
                            (unsigned long long)(p.n_items + p.n_chains), (unsigned long long)fixed_entries);
            p.partials = fixed_scratch;
        } else {
            void *sc = nullptr;
            int rc = scratch_for(dev, s, (size_t)(p.n_items + p.n_chains) * 16, &sc);
            if (rc)
                return rc;
            p.partials = reinterpret_cast<uint4 *>(sc);
        }
        p.masks = p.partials + p.n_items;
    }
    he = launch_gcm(p, encrypt, mode, num_cu, s);
    if (he != hipSuccess)
        return hip_fail(he, "GCM launch");
    return FASTRACK_OK;
}

int current_device(int *dev, int *ncu)
{
    hipError_t he = hipGetDevice(dev);
    if (he != hipSuccess)
        return hip_fail(he, "hipGetDevice");
    return num_cu_of(*dev, ncu);
}

uint64_t round256(uint64_t x) { return (x + 255) & ~255ull; }

}  // namespace

FT_EXPORT uint64_t fastrack_num_chains(uint64_t len, uint64_t chain_bytes)
{
    return chain_bytes ? (len + chain_bytes - 1) / chain_bytes : 0;
}

FT_EXPORT const char *fastrack_last_error(void) { return g_err.c_str(); }

FT_EXPORT int fastrack_plan(uint64_t len, uint64_t chain_bytes, uint32_t num_cu, uint64_t *out)
{
    g_err.clear();
    if (!out || num_cu == 0)
        return fail(FASTRACK_EINVAL, "out must be non-NULL and num_cu nonzero");
    if (chain_bytes == 0 || chain_bytes % 16 != 0 || chain_bytes / 16 > kMaxChainBlocks)
        return fail(FASTRACK_EINVAL, "chain_bytes must be a nonzero multiple of 16, at most (2^32-2)*16");
    if (len == 0 || (len + chain_bytes - 1) / chain_bytes > 0xFFFFFFFFull)
        return fail(FASTRACK_EINVAL, "len must be nonzero, with at most 2^32-1 chains");
    GcmLaunch p;
    std::memset(&p, 0, sizeof p);
    make_plan(len, chain_bytes, 0, (uint64_t)num_cu * kGcmWavesPerWg * gcm_wgs_per_cu(kFused), p);
    const uint64_t L = 1ull << p.lanes_log2, seg = 1ull << p.seg_log2;
    out[0] = p.lanes_log2;
    out[1] = p.seg_log2;
    out[2] = p.segs_full;
    out[3] = p.segs_last;
    out[4] = p.n_items;
    out[5] = ((seg < p.qc ? seg : p.qc) + L - 1) >> p.lanes_log2;   // the kernel's iterations per item
    out[6] = p.n_items > p.n_chains ? 1u : 0u;
    return FASTRACK_OK;
}

FT_EXPORT int fastrack_gcm_decrypt_verify(const uint8_t *key, const uint8_t *base_iv, uint64_t chain_bytes,
                                          const uint8_t *d_ct, uint64_t len, const uint8_t *d_tags,
                                          const uint8_t *d_aad, uint32_t aad_bytes, uint8_t *d_pt, uint8_t *d_ok,
                                          uint32_t flags, void *stream)
{
    g_err.clear();
    int rc = check_common(key, base_iv, chain_bytes, len, d_ct, d_pt, d_aad, aad_bytes, flags);
    if (rc || len == 0)
        return rc;
    if (!d_tags || !d_ok)
        return fail(FASTRACK_EINVAL, "d_tags and d_ok must be non-NULL");
    std::lock_guard<std::mutex> lk(g_mu);
    int dev, ncu;
    if ((rc = current_device(&dev, &ncu)))
        return rc;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    const KeyCtx *ctx;
    if ((rc = key_ctx(key, s, dev, &ctx)))
        return rc;
    return run_gcm(false, kFused, ctx, base_iv, chain_bytes, 0, d_ct, nullptr, len, d_pt, aad_bytes ? d_aad : nullptr, aad_bytes,
                   d_tags, nullptr, d_ok, flags, dev, ncu, s);
}

// ---------------------------------------------------------------------------
// Allocation-free decrypt + verify
// ---------------------------------------------------------------------------
//
// One static device array per GPU (each GPU that loads the library holds its own
// copy until the process ends): the key tables of the last key this entry point
// was given on that GPU, then the per-item GHASH partials and per-chain masks of
// launches that cut chains into segments. Host code never passes the array's name
// to a kernel (on the host it is only a stand-in for the symbol); it uses the
// device address that hipGetSymbolAddress returns for the current device.

namespace {
constexpr size_t kNoAllocKeyBytes = (sizeof(KeyCtx) + 255) & ~(size_t)255;
constexpr uint64_t kNoAllocEntries = (FASTRACK_NOALLOC_SCRATCH_BYTES - kNoAllocKeyBytes) / 16;
static_assert(kNoAllocEntries == FASTRACK_NOALLOC_MAX_PARTIALS, "header constant matches the layout");
}  // namespace

static __device__ __align__(256) uint8_t scratch[FASTRACK_NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int kNoAllocMaxDevices = 64;
struct NoAllocDevice {
    uint8_t *ptr = nullptr;              // device address of `scratch` on this device
    bool have_key = false;               // the key tables at ptr belong to `key`
    std::array<uint8_t, 32> key{};
};
NoAllocDevice g_noalloc[kNoAllocMaxDevices];

// The device address of this device's `scratch`, looked up once per device with
// the device current.
int noalloc_area(int dev, NoAllocDevice **out)
{
    if (dev < 0 || dev >= kNoAllocMaxDevices)
        return fail(FASTRACK_EINVAL, "device %d is beyond the %d devices the allocation-free path serves", dev,
                    kNoAllocMaxDevices);
    NoAllocDevice &d = g_noalloc[dev];
    if (!d.ptr) {
        void *p = nullptr;
        hipError_t he = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (he != hipSuccess || !p)
            return hip_fail(he != hipSuccess ? he : hipErrorInvalidSymbol, "hipGetSymbolAddress(scratch)");
        d.ptr = static_cast<uint8_t *>(p);
    }
    *out = &d;
    return FASTRACK_OK;
}
}  // namespace

FT_EXPORT int fastrack_gcm_decrypt_verify_noalloc(const uint8_t *key, const uint8_t *base_iv, uint64_t chain_bytes,
                                                  const uint8_t *d_ct, uint64_t len, const uint8_t *d_tags,
                                                  const uint8_t *d_aad, uint32_t aad_bytes, uint8_t *d_pt,
                                                  uint8_t *d_ok, uint32_t flags, void *stream)
{
    g_err.clear();
    int rc = check_common(key, base_iv, chain_bytes, len, d_ct, d_pt, d_aad, aad_bytes, flags);
    if (rc || len == 0)
        return rc;
    if (!d_tags || !d_ok)
        return fail(FASTRACK_EINVAL, "d_tags and d_ok must be non-NULL");
    std::lock_guard<std::mutex> lk(g_mu);
    int dev, ncu;
    if ((rc = current_device(&dev, &ncu)))
        return rc;
    NoAllocDevice *d;
    if ((rc = noalloc_area(dev, &d)))
        return rc;
    // Size check before anything is enqueued: the same plan run_gcm makes.
    GcmLaunch probe;
    std::memset(&probe, 0, sizeof probe);
    make_plan(len, chain_bytes, 0, (uint64_t)ncu * kGcmWavesPerWg * gcm_wgs_per_cu(kFused), probe);
    if (probe.n_items > 0xFFFFFFFFull)
        return fail(FASTRACK_EINVAL, "more than 2^32-1 work items in one launch");
    const bool seq = (flags & FASTRACK_F_SEQ_GHASH) != 0;
    if (!seq && probe.n_items > probe.n_chains && probe.n_items + probe.n_chains > kNoAllocEntries)
        return fail(FASTRACK_EINVAL,
                    "the launch needs %llu partial slots; the allocation-free scratch holds %llu "
                    "(fastrack_gcm_decrypt_verify has no such limit)",
                    (unsigned long long)(probe.n_items + probe.n_chains), (unsigned long long)kNoAllocEntries);
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    KeyCtx *ctx = reinterpret_cast<KeyCtx *>(d->ptr);
    std::array<uint8_t, 32> k;
    std::memcpy(k.data(), key, 32);
    if (!d->have_key || d->key != k) {   // the key tables are rebuilt in place, on this stream
        uint32_t words[8];
        for (int i = 0; i < 8; ++i)
            words[i] = (uint32_t)key[4 * i] | ((uint32_t)key[4 * i + 1] << 8) | ((uint32_t)key[4 * i + 2] << 16) |
                       ((uint32_t)key[4 * i + 3] << 24);
        d->have_key = false;
        hipError_t he = launch_key_setup(words, ctx, s);
        std::memset(words, 0, sizeof words);
        if (he != hipSuccess)
            return hip_fail(he, "key setup launch");
        d->key = k;
        d->have_key = true;
    }
    std::memset(k.data(), 0, 32);
    return run_gcm(false, kFused, ctx, base_iv, chain_bytes, 0, d_ct, nullptr, len, d_pt,
                   aad_bytes ? d_aad : nullptr, aad_bytes, d_tags, nullptr, d_ok, flags, dev, ncu, s,
                   reinterpret_cast<uint4 *>(d->ptr + kNoAllocKeyBytes), kNoAllocEntries);
}

FT_EXPORT int fastrack_gcm_encrypt_tag(const uint8_t *key, const uint8_t *base_iv, uint64_t chain_bytes,
                                       const uint8_t *d_pt, uint64_t len, const uint8_t *d_aad, uint32_t aad_bytes,
                                       uint8_t *d_ct, uint8_t *d_tags, uint32_t flags, void *stream)
{
    g_err.clear();
    int rc = check_common(key, base_iv, chain_bytes, len, d_pt, d_ct, d_aad, aad_bytes, flags);
    if (rc || len == 0)
        return rc;
    if (!d_tags)
        return fail(FASTRACK_EINVAL, "d_tags must be non-NULL");
    std::lock_guard<std::mutex> lk(g_mu);
    int dev, ncu;
    if ((rc = current_device(&dev, &ncu)))
        return rc;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    const KeyCtx *ctx;
    if ((rc = key_ctx(key, s, dev, &ctx)))
        return rc;
    return run_gcm(true, kFused, ctx, base_iv, chain_bytes, 0, d_pt, nullptr, len, d_ct, aad_bytes ? d_aad : nullptr, aad_bytes,
                   nullptr, d_tags, nullptr, flags, dev, ncu, s);
}

FT_EXPORT int fastrack_gcm_decrypt_eager(const uint8_t *key, const uint8_t *base_iv, uint64_t chain_bytes,
                                         const uint8_t *d_ct, uint64_t len, const uint8_t *d_tags,
                                         const uint8_t *d_aad, uint32_t aad_bytes, uint8_t *d_pt, uint8_t *d_ok,
                                         void *decrypt_stream, void *verify_stream)
{
    g_err.clear();
    int rc = check_common(key, base_iv, chain_bytes, len, d_ct, d_pt, d_aad, aad_bytes, 0);
    if (rc || len == 0)
        return rc;
    if (!d_tags || !d_ok)
        return fail(FASTRACK_EINVAL, "d_tags and d_ok must be non-NULL");
    if (static_cast<const void *>(d_ct) == static_cast<const void *>(d_pt))
        return fail(FASTRACK_EINVAL, "d_pt may not be d_ct: the ciphertext is verified while it is decrypted");
    std::lock_guard<std::mutex> lk(g_mu);
    int dev, ncu;
    if ((rc = current_device(&dev, &ncu)))
        return rc;
    hipStream_t ds = reinterpret_cast<hipStream_t>(decrypt_stream);
    hipStream_t vs = reinterpret_cast<hipStream_t>(verify_stream);
    const KeyCtx *ctx;
    if ((rc = key_ctx(key, ds, dev, &ctx)))
        return rc;
    if (vs != ds) {
        // The verify stream starts after the work already queued on the decrypt stream
        // (which may be what wrote d_ct).
        hipEvent_t e;
        hipError_t he = hipEventCreateWithFlags(&e, hipEventDisableTiming);
        if (he == hipSuccess) {
            he = hipEventRecord(e, ds);
            if (he == hipSuccess)
                he = hipStreamWaitEvent(vs, e, 0);
            (void)hipEventDestroy(e);
        }
        if (he != hipSuccess)
            return hip_fail(he, "decrypt -> verify stream ordering");
        if ((rc = key_ctx(key, vs, dev, &ctx)))
            return rc;
    }
    rc = run_gcm(false, kCtr, ctx, base_iv, chain_bytes, 0, d_ct, nullptr, len, d_pt, nullptr, 0, nullptr, nullptr,
                 nullptr, 0, dev, ncu, ds);
    if (rc)
        return rc;
    return run_gcm(false, kVerify, ctx, base_iv, chain_bytes, 0, d_ct, nullptr, len, nullptr,
                   aad_bytes ? d_aad : nullptr, aad_bytes, d_tags, nullptr, d_ok, 0, dev, ncu, vs);
}

FT_EXPORT int fastrack_gcm_keystream(const uint8_t *key, const uint8_t *base_iv, uint64_t chain_bytes,
                                     uint64_t chain_base, uint64_t len, uint8_t *d_ks, void *stream)
{
    g_err.clear();
    int rc = check_common(key, base_iv, chain_bytes, len, d_ks, d_ks, nullptr, 0, 0);
    if (rc || len == 0)
        return rc;
    std::lock_guard<std::mutex> lk(g_mu);
    int dev, ncu;
    if ((rc = current_device(&dev, &ncu)))
        return rc;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    const KeyCtx *ctx;
    if ((rc = key_ctx(key, s, dev, &ctx)))
        return rc;
    return run_gcm(false, kKeystream, ctx, base_iv, chain_bytes, chain_base, nullptr, nullptr, len, d_ks, nullptr, 0,
                   nullptr, nullptr, nullptr, 0, dev, ncu, s);
}

FT_EXPORT int fastrack_gcm_keystream_bitsliced(const uint8_t *key, const uint8_t *base_iv, uint64_t chain_bytes,
                                               uint64_t chain_base, uint64_t len, uint8_t *d_ks, void *stream)
{
    g_err.clear();
    int rc = check_common(key, base_iv, chain_bytes, len, d_ks, d_ks, nullptr, 0, 0);
    if (rc || len == 0)
        return rc;
    std::lock_guard<std::mutex> lk(g_mu);
    int dev, ncu;
    if ((rc = current_device(&dev, &ncu)))
        return rc;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    const KeyCtx *ctx;
    if ((rc = key_ctx(key, s, dev, &ctx)))
        return rc;
    GcmLaunch p;
    std::memset(&p, 0, sizeof p);
    make_plan(len, chain_bytes, chain_base, (uint64_t)ncu * kGcmWavesPerWg, p);
    p.ctx = ctx;
    p.out = d_ks;
    iv_words(base_iv, p.iv);
    hipError_t he = launch_bs_keystream(p, ncu, s);
    return he == hipSuccess ? FASTRACK_OK : hip_fail(he, "bitsliced keystream launch");
}

FT_EXPORT int fastrack_gcm_apply_verify(const uint8_t *key, const uint8_t *base_iv, uint64_t chain_bytes,
                                        uint64_t chain_base, const uint8_t *d_ct, uint64_t len, const uint8_t *d_ks,
                                        const uint8_t *d_tags, const uint8_t *d_aad, uint32_t aad_bytes,
                                        uint8_t *d_pt, uint8_t *d_ok, void *stream)
{
    g_err.clear();
    int rc = check_common(key, base_iv, chain_bytes, len, d_ct, d_pt, d_aad, aad_bytes, 0);
    if (rc || len == 0)
        return rc;
    if (!d_ks || ((uintptr_t)d_ks & 15))
        return fail(FASTRACK_EINVAL, "d_ks must be a non-NULL 16-byte-aligned device pointer");
    if (overlap_bad(d_ks, d_pt, len))
        return fail(FASTRACK_EINVAL, "d_ks and d_pt overlap partially");
    if (!d_tags || !d_ok)
        return fail(FASTRACK_EINVAL, "d_tags and d_ok must be non-NULL");
    std::lock_guard<std::mutex> lk(g_mu);
    int dev, ncu;
    if ((rc = current_device(&dev, &ncu)))
        return rc;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    const KeyCtx *ctx;
    if ((rc = key_ctx(key, s, dev, &ctx)))
        return rc;
    return run_gcm(false, kApplyKs, ctx, base_iv, chain_bytes, chain_base, d_ct, d_ks, len, d_pt,
                   aad_bytes ? d_aad : nullptr, aad_bytes, d_tags, nullptr, d_ok, 0, dev, ncu, s);
}

FT_EXPORT uint64_t fastrack_pipeline_stage_bytes(uint64_t len, uint64_t chain_bytes, uint32_t aad_bytes,
                                                 uint64_t chunk_bytes, int depth)
{
    if (chain_bytes == 0 || depth < 0 || depth == 1 || depth > kMaxPipelineDepth)
        return 0;
    const uint64_t n = (len + chain_bytes - 1) / chain_bytes;
    return (uint64_t)depth * round256(chunk_bytes) + round256(16 * n) + round256((uint64_t)aad_bytes * n);
}

namespace {

// The H2D pipeline as a list of stream operations, built on the host before any
// of them is enqueued (and exported for inspection). Streams: 0 copy, 1 compute,
// 2 verify (the eager mode only; the other modes put its work on stream 1).
enum PlanKind : uint32_t {
    kOpMeta = 0,       // upload the tags and the AAD
    kOpRecord = 1,     // record `event` on the stream
    kOpWait = 2,       // the stream waits for the last record of `event`
    kOpCopy = 3,       // copy chunk `chunk` from the host into buffer `slot` (-1: its place in d_pt)
    kOpKeystream = 4,  // keystream of chunk `chunk` into ring slot `slot`
    kOpFused = 5,      // decrypt + verify chunk `chunk` from buffer `slot` into d_pt
    kOpApply = 6,      // XOR keystream slot `aux` into chunk `chunk` (read from `slot`) + tag check
    kOpCtr = 7,        // decrypt chunk `chunk` from buffer `slot` into d_pt (no tag check)
    kOpVerify = 8,     // tag check of chunk `chunk` read from buffer `slot`
    kOpHostWait = 9,   // the calling thread waits until the last record of `event` has completed
    kOpDirect = 10,    // decrypt + verify all of h_ct, read over the host link by the kernel itself
};
struct PlanOp {
    uint32_t kind;
    uint32_t stream;
    int32_t event;
    uint64_t chunk;
    int32_t slot;
    int32_t aux;
};
// Events: meta (0); copied[i] (1..P), done[i] (1+P..2P), decrypted[i] (1+2P..3P), reused modulo
// P = 8. copied[k % P] and decrypted[k % P] are waited on right after they are recorded;
// done[k % P] is waited on by the calling thread before the copy of chunk k + W, W <= 8, which
// comes before chunk k + P records it again (a wait takes the event's last record at the time).
constexpr int kPlanP = 8;
constexpr int kPlanEvents = 3 * kPlanP + 1;
// Chunks the calling thread lets the copies run ahead of the last finished chunk when no
// staging slot bounds it (in place and keystream-ahead schedules).
constexpr uint64_t kPaceChunks = 4;

// The operations of one H2D pipeline call, in the order they are enqueued. Streams:
// 0 copy, 1 compute, 2 verify (eager mode). The copy stream never waits for an event
// of another stream: a ring slot is reused only after the calling thread has seen the
// event of its last read complete (kOpHostWait). A device-side wait there would also
// be correct, but the runtime then holds the calling thread inside the next copy's
// enqueue until the event completes, which delays the launches queued behind it and
// leaves the copy engine idle between chunks; waiting explicitly, and early, keeps
// the copies back to back.
std::vector<PlanOp> h2d_plan(uint64_t len, uint64_t chunk_bytes, int depth, uint32_t mode)
{
    std::vector<PlanOp> ops;
    const uint32_t VS = mode == FASTRACK_PIPE_EAGER ? 2u : 1u;
    auto op = [&](uint32_t kind, uint32_t stream, int32_t event, uint64_t chunk, int32_t slot, int32_t aux) {
        ops.push_back(PlanOp{kind, stream, event, chunk, slot, aux});
    };
    const int32_t meta = 0, copied = 1, done = 1 + kPlanP, decrypted = 1 + 2 * kPlanP;
    op(kOpMeta, 0, -1, 0, -1, -1);
    op(kOpRecord, 0, meta, 0, -1, -1);
    op(kOpWait, 1, meta, 0, -1, -1);
    if (VS != 1)
        op(kOpWait, VS, meta, 0, -1, -1);
    if (mode == FASTRACK_PIPE_DIRECT) {   // no copies: the kernel reads the pinned buffer itself
        op(kOpDirect, 1, -1, 0, -1, -1);
        return ops;
    }
    const uint64_t nchunks = (len + chunk_bytes - 1) / chunk_bytes;
    // OTP: the keystream of chunk 0 before anything arrives; that of chunk k+1 while
    // chunk k+1 is on the bus, in ring slot (k+1) % depth. A slot is rewritten only
    // after the XOR that read it, earlier on the same stream.
    if (mode == FASTRACK_PIPE_OTP)
        op(kOpKeystream, 1, -1, 0, 0, -1);
    // depth 0 (and OTP): each chunk is copied straight to its place in d_pt and
    // decrypted there, so no buffer is reused; the calling thread still keeps the
    // copies at most kPaceChunks ahead of the decrypts. A ring of `depth` slots must
    // not overwrite slot k % depth before chunk k - depth has been read.
    const bool ring = mode != FASTRACK_PIPE_OTP && depth > 0;
    const uint64_t window = ring ? (uint64_t)depth : kPaceChunks;
    for (uint64_t k = 0; k < nchunks; ++k) {
        const int32_t buf = ring ? (int32_t)(k % (uint64_t)depth) : -1;
        const int32_t e = (int32_t)(k % kPlanP);
        if (k >= window)
            op(kOpHostWait, 0, done + (int32_t)((k - window) % kPlanP), k - window, -1, -1);
        op(kOpCopy, 0, -1, k, buf, -1);
        op(kOpRecord, 0, copied + e, 0, -1, -1);
        if (mode == FASTRACK_PIPE_OTP && k + 1 < nchunks)
            op(kOpKeystream, 1, -1, k + 1, (int32_t)((k + 1) % (uint64_t)depth), -1);
        op(kOpWait, 1, copied + e, 0, -1, -1);
        if (mode == FASTRACK_PIPE_FUSED) {
            op(kOpFused, 1, -1, k, buf, -1);
        } else if (mode == FASTRACK_PIPE_OTP) {
            op(kOpApply, 1, -1, k, buf, (int32_t)(k % (uint64_t)depth));
        } else {   // eager: plaintext on the compute stream, the tag check beside it
            op(kOpCtr, 1, -1, k, buf, -1);
            op(kOpRecord, 1, decrypted + e, 0, -1, -1);
            op(kOpWait, VS, copied + e, 0, -1, -1);
            op(kOpVerify, VS, -1, k, buf, -1);
            op(kOpWait, VS, decrypted + e, 0, -1, -1);   // the slot is free once both have read it
        }
        op(kOpRecord, VS, done + e, 0, -1, -1);
    }
    return ops;
}

int check_pipe_mode(uint32_t mode, int depth)
{
    if (mode > FASTRACK_PIPE_DIRECT)
        return fail(FASTRACK_EINVAL, "unknown pipeline mode %u", mode);
    if (depth < 0 || depth == 1 || depth > kMaxPipelineDepth)
        return fail(FASTRACK_EINVAL, "depth must be 0 (in place) or 2..%d (staging ring)", kMaxPipelineDepth);
    if ((mode == FASTRACK_PIPE_EAGER || mode == FASTRACK_PIPE_OTP) && depth == 0)
        return fail(FASTRACK_EINVAL, "the eager and keystream pipelines need depth >= 2 staging slots");
    if (mode == FASTRACK_PIPE_DIRECT && depth != 0)
        return fail(FASTRACK_EINVAL, "the direct pipeline reads the host buffer in place and takes depth 0");
    return FASTRACK_OK;
}

// [p, p + len) must lie inside one pinned host allocation: the copy engine (or, in the
// direct mode, the kernel) reads all of it through the allocation's device mapping.
// Returns the device address of p, or nullptr.
const uint8_t *pinned_range(const uint8_t *p, uint64_t len)
{
    hipPointerAttribute_t attr;
    if (hipPointerGetAttributes(&attr, p) != hipSuccess || attr.type != hipMemoryTypeHost || !attr.devicePointer) {
        (void)hipGetLastError();
        return nullptr;
    }
    hipDeviceptr_t base = 0;
    size_t size = 0;
    if (hipMemGetAddressRange(&base, &size, (hipDeviceptr_t)const_cast<uint8_t *>(p)) != hipSuccess) {
        (void)hipGetLastError();
        return nullptr;
    }
    const uintptr_t b = (uintptr_t)base, a = (uintptr_t)p;
    if (a < b || a - b > size || len > size - (a - b))
        return nullptr;
    return static_cast<const uint8_t *>(attr.devicePointer);
}

int pipeline_impl(const uint8_t *key, const uint8_t *base_iv, uint64_t chain_bytes, const uint8_t *h_ct, uint64_t len,
                  const uint8_t *h_tags, const uint8_t *h_aad, uint32_t aad_bytes, uint64_t chunk_bytes, int depth,
                  uint32_t mode, uint8_t *d_stage, uint64_t stage_bytes, uint8_t *d_pt, uint8_t *d_ok,
                  void *copy_stream, void *compute_stream, void *verify_stream)
{
    g_err.clear();
    int rc = check_common(key, base_iv, chain_bytes, len, h_ct, d_pt, h_aad, aad_bytes, 0);
    if (rc || len == 0)
        return rc;
    if (!h_tags || !d_ok || !d_stage)
        return fail(FASTRACK_EINVAL, "h_tags, d_ok and d_stage must be non-NULL");
    if (chunk_bytes == 0 || chunk_bytes % chain_bytes != 0)
        return fail(FASTRACK_EINVAL, "chunk_bytes must be a nonzero multiple of chain_bytes");
    if ((rc = check_pipe_mode(mode, depth)))
        return rc;
    if ((uintptr_t)d_stage & 255)
        return fail(FASTRACK_EINVAL, "d_stage must be 256-byte aligned");
    const uint64_t need = fastrack_pipeline_stage_bytes(len, chain_bytes, aad_bytes, chunk_bytes, depth);
    if (stage_bytes < need)
        return fail(FASTRACK_EINVAL, "d_stage holds %llu bytes, the pipeline needs %llu",
                    (unsigned long long)stage_bytes, (unsigned long long)need);

    const uint8_t *h_ct_dev = pinned_range(h_ct, len);
    if (!h_ct_dev)
        return fail(FASTRACK_ENOTPINNED, "h_ct .. h_ct + len is not inside one pinned host allocation");
    hipError_t he = hipSuccess;

    std::lock_guard<std::mutex> lk(g_mu);
    int dev, ncu;
    if ((rc = current_device(&dev, &ncu)))
        return rc;
    hipStream_t cs = reinterpret_cast<hipStream_t>(copy_stream);
    hipStream_t ks = reinterpret_cast<hipStream_t>(compute_stream);
    hipStream_t vs = mode == FASTRACK_PIPE_EAGER ? reinterpret_cast<hipStream_t>(verify_stream) : ks;
    const KeyCtx *ctx;
    if ((rc = key_ctx(key, ks, dev, &ctx)))
        return rc;
    if (vs != ks && (rc = key_ctx(key, vs, dev, &ctx)))
        return rc;

    const uint64_t n = (len + chain_bytes - 1) / chain_bytes;
    const uint64_t slot_bytes = round256(chunk_bytes);
    uint8_t *d_tags = d_stage + (uint64_t)depth * slot_bytes;
    uint8_t *d_aad = d_tags + round256(16 * n);
    const uint8_t *aad = aad_bytes ? d_aad : nullptr;
    const uint64_t cpc = chunk_bytes / chain_bytes;
    auto chunk_len = [&](uint64_t k) { return len - k * chunk_bytes < chunk_bytes ? len - k * chunk_bytes : chunk_bytes; };
    auto slot = [&](int32_t i) { return d_stage + (uint64_t)i * slot_bytes; };
    auto buf_of = [&](const PlanOp &o) { return o.slot < 0 ? d_pt + o.chunk * chunk_bytes : slot(o.slot); };

    std::vector<hipEvent_t> ev;
    auto cleanup = [&]() {
        for (auto e : ev)
            (void)hipEventDestroy(e);
    };
    for (int i = 0; i < kPlanEvents; ++i) {
        hipEvent_t e;
        he = hipEventCreateWithFlags(&e, hipEventDisableTiming);
        if (he != hipSuccess) {
            cleanup();
            return hip_fail(he, "hipEventCreate");
        }
        ev.push_back(e);
    }
    const hipStream_t streams[3] = {cs, ks, vs};
    for (const PlanOp &o : h2d_plan(len, chunk_bytes, depth, mode)) {
        const hipStream_t st = streams[o.stream];
        const uint64_t k = o.chunk;
        switch (o.kind) {
        case kOpMeta:
            he = hipMemcpyAsync(d_tags, h_tags, 16 * n, hipMemcpyHostToDevice, st);
            if (he == hipSuccess && aad_bytes)
                he = hipMemcpyAsync(d_aad, h_aad, (size_t)aad_bytes * n, hipMemcpyHostToDevice, st);
            break;
        case kOpRecord:
            he = hipEventRecord(ev[o.event], st);
            break;
        case kOpWait:
            he = hipStreamWaitEvent(st, ev[o.event], 0);
            break;
        case kOpCopy:
            he = hipMemcpyAsync(buf_of(o), h_ct + k * chunk_bytes, chunk_len(k), hipMemcpyHostToDevice, st);
            break;
        case kOpKeystream:
            rc = run_gcm(false, kKeystream, ctx, base_iv, chain_bytes, k * cpc, nullptr, nullptr, chunk_len(k),
                         buf_of(o), nullptr, 0, nullptr, nullptr, nullptr, 0, dev, ncu, st);
            break;
        case kOpFused:
            rc = run_gcm(false, kFused, ctx, base_iv, chain_bytes, k * cpc, buf_of(o), nullptr, chunk_len(k),
                         d_pt + k * chunk_bytes, aad, aad_bytes, d_tags, nullptr, d_ok, 0, dev, ncu, st);
            break;
        case kOpApply:
            rc = run_gcm(false, kApplyKs, ctx, base_iv, chain_bytes, k * cpc, buf_of(o), slot(o.aux), chunk_len(k),
                         d_pt + k * chunk_bytes, aad, aad_bytes, d_tags, nullptr, d_ok, 0, dev, ncu, st);
            break;
        case kOpCtr:
            rc = run_gcm(false, kCtr, ctx, base_iv, chain_bytes, k * cpc, buf_of(o), nullptr, chunk_len(k),
                         d_pt + k * chunk_bytes, nullptr, 0, nullptr, nullptr, nullptr, 0, dev, ncu, st);
            break;
        case kOpVerify:
            rc = run_gcm(false, kVerify, ctx, base_iv, chain_bytes, k * cpc, buf_of(o), nullptr, chunk_len(k), nullptr,
                         aad, aad_bytes, d_tags, nullptr, d_ok, 0, dev, ncu, st);
            break;
        case kOpHostWait:
            he = hipEventSynchronize(ev[o.event]);
            break;
        case kOpDirect:
            rc = run_gcm(false, kFused, ctx, base_iv, chain_bytes, 0, h_ct_dev, nullptr, len, d_pt, aad, aad_bytes,
                         d_tags, nullptr, d_ok, 0, dev, ncu, st);
            break;
        }
        if (he != hipSuccess) {
            cleanup();
            return hip_fail(he, "pipeline");
        }
        if (rc) {
            cleanup();
            return rc;
        }
    }
    cleanup();
    return FASTRACK_OK;
}

}  // namespace

FT_EXPORT int64_t fastrack_pipeline_plan(uint64_t len, uint64_t chain_bytes, uint64_t chunk_bytes, int depth,
                                         uint32_t mode, int64_t *h_ops, uint64_t max_ops)
{
    g_err.clear();
    if (chain_bytes == 0 || chain_bytes % 16 != 0)
        return fail(FASTRACK_EINVAL, "chain_bytes must be a nonzero multiple of 16");
    if (chunk_bytes == 0 || chunk_bytes % chain_bytes != 0)
        return fail(FASTRACK_EINVAL, "chunk_bytes must be a nonzero multiple of chain_bytes");
    if (int rc = check_pipe_mode(mode, depth))
        return rc;
    if (len == 0)
        return 0;
    const std::vector<PlanOp> ops = h2d_plan(len, chunk_bytes, depth, mode);
    for (uint64_t i = 0; h_ops && i < ops.size() && i < max_ops; ++i) {
        const PlanOp &o = ops[i];
        int64_t *w = h_ops + 6 * i;
        w[0] = o.kind;
        w[1] = o.stream;
        w[2] = o.event;
        w[3] = (int64_t)o.chunk;
        w[4] = o.slot;
        w[5] = o.aux;
    }
    return (int64_t)ops.size();
}

FT_EXPORT int fastrack_pipeline_h2d(const uint8_t *key, const uint8_t *base_iv, uint64_t chain_bytes,
                                    const uint8_t *h_ct, uint64_t len, const uint8_t *h_tags, const uint8_t *h_aad,
                                    uint32_t aad_bytes, uint64_t chunk_bytes, int depth, uint8_t *d_stage,
                                    uint64_t stage_bytes, uint8_t *d_pt, uint8_t *d_ok, void *copy_stream,
                                    void *compute_stream)
{
    return pipeline_impl(key, base_iv, chain_bytes, h_ct, len, h_tags, h_aad, aad_bytes, chunk_bytes, depth,
                         FASTRACK_PIPE_FUSED, d_stage, stage_bytes, d_pt, d_ok, copy_stream, compute_stream,
                         compute_stream);
}

FT_EXPORT int fastrack_pipeline_h2d_mode(const uint8_t *key, const uint8_t *base_iv, uint64_t chain_bytes,
                                         const uint8_t *h_ct, uint64_t len, const uint8_t *h_tags,
                                         const uint8_t *h_aad, uint32_t aad_bytes, uint64_t chunk_bytes, int depth,
                                         uint32_t mode, uint8_t *d_stage, uint64_t stage_bytes, uint8_t *d_pt,
                                         uint8_t *d_ok, void *copy_stream, void *compute_stream, void *verify_stream)
{
    return pipeline_impl(key, base_iv, chain_bytes, h_ct, len, h_tags, h_aad, aad_bytes, chunk_bytes, depth, mode,
                         d_stage, stage_bytes, d_pt, d_ok, copy_stream, compute_stream, verify_stream);
}

namespace {

// Direct D2H: one encrypt + tag launch writes the ciphertext through the device
// mapping of the pinned buffer; the tags follow on the same stream, and copy_stream
// is ordered after both so that the results are valid when it completes, as in the
// chunked mode.
int d2h_direct(const uint8_t *key, const uint8_t *base_iv, uint64_t chain_bytes, const uint8_t *d_pt, uint64_t len,
               const uint8_t *d_aad, uint32_t aad_bytes, uint8_t *d_tags, uint8_t *h_ct_dev, uint8_t *h_tags,
               hipStream_t cs, hipStream_t ks)
{
    const uint64_t n = (len + chain_bytes - 1) / chain_bytes;
    hipEvent_t e;
    hipError_t he = hipEventCreateWithFlags(&e, hipEventDisableTiming);
    if (he != hipSuccess)
        return hip_fail(he, "hipEventCreate");
    int rc;
    {
        std::lock_guard<std::mutex> lk(g_mu);
        int dev, ncu;
        const KeyCtx *ctx;
        if (!(rc = current_device(&dev, &ncu)) && !(rc = key_ctx(key, ks, dev, &ctx)))
            rc = run_gcm(true, kFused, ctx, base_iv, chain_bytes, 0, d_pt, nullptr, len, h_ct_dev,
                         aad_bytes ? d_aad : nullptr, aad_bytes, nullptr, d_tags, nullptr, 0, dev, ncu, ks);
    }
    if (!rc) {
        he = hipMemcpyAsync(h_tags, d_tags, 16 * n, hipMemcpyDeviceToHost, ks);
        if (he == hipSuccess)
            he = hipEventRecord(e, ks);
        if (he == hipSuccess && cs != ks)
            he = hipStreamWaitEvent(cs, e, 0);
        if (he != hipSuccess)
            rc = hip_fail(he, "direct D2H ordering");
    }
    (void)hipEventDestroy(e);
    return rc;
}

int d2h_impl(const uint8_t *key, const uint8_t *base_iv, uint64_t chain_bytes, const uint8_t *d_pt, uint64_t len,
             const uint8_t *d_aad, uint32_t aad_bytes, uint64_t chunk_bytes, uint8_t *d_ct, uint8_t *d_tags,
             uint8_t *h_ct, uint8_t *h_tags, void *copy_stream, void *compute_stream, uint32_t mode)
{
    g_err.clear();
    if (mode != FASTRACK_PIPE_FUSED && mode != FASTRACK_PIPE_DIRECT)
        return fail(FASTRACK_EINVAL, "the D2H pipeline takes FASTRACK_PIPE_FUSED or FASTRACK_PIPE_DIRECT (got %u)", mode);
    const bool direct = mode == FASTRACK_PIPE_DIRECT;
    int rc = check_common(key, base_iv, chain_bytes, len, d_pt, direct ? h_ct : d_ct, d_aad, aad_bytes, 0);
    if (rc || len == 0)
        return rc;
    if (!d_tags || !h_ct || !h_tags)
        return fail(FASTRACK_EINVAL, "d_tags, h_ct and h_tags must be non-NULL");
    if (chunk_bytes == 0 || chunk_bytes % chain_bytes != 0)
        return fail(FASTRACK_EINVAL, "chunk_bytes must be a nonzero multiple of chain_bytes");
    uint8_t *h_ct_dev = const_cast<uint8_t *>(pinned_range(h_ct, len));
    if (!h_ct_dev)
        return fail(FASTRACK_ENOTPINNED, "h_ct .. h_ct + len is not inside one pinned host allocation");
    hipError_t he = hipSuccess;
    hipStream_t cs = reinterpret_cast<hipStream_t>(copy_stream);
    hipStream_t ks = reinterpret_cast<hipStream_t>(compute_stream);
    if (direct)
        return d2h_direct(key, base_iv, chain_bytes, d_pt, len, d_aad, aad_bytes, d_tags, h_ct_dev, h_tags, cs, ks);
    const uint64_t n = (len + chain_bytes - 1) / chain_bytes;
    const uint64_t nchunks = (len + chunk_bytes - 1) / chunk_bytes;
    const uint64_t cpc = chunk_bytes / chain_bytes;
    const uint64_t group = (kD2hGroupBytes + chunk_bytes - 1) / chunk_bytes;
    const uint64_t ngroups = (nchunks + group - 1) / group;
    auto chunk_len = [&](uint64_t k) { return len - k * chunk_bytes < chunk_bytes ? len - k * chunk_bytes : chunk_bytes; };

    // A copy that waits on the compute stream's events on the GPU stalls the copy
    // engine far longer than the encryption takes, so the copies are paced from
    // the host: every encryption is enqueued first, with an event per group of
    // chunks, and the copies of a group are enqueued once its event has completed.
    // Encrypting is several times faster than copying, so the copy engine stays busy.
    std::vector<hipEvent_t> ev;
    auto cleanup = [&]() {
        for (auto e : ev)
            (void)hipEventDestroy(e);
    };
    for (uint64_t g = 0; g < ngroups; ++g) {
        hipEvent_t e;
        he = hipEventCreateWithFlags(&e, hipEventDisableTiming);
        if (he != hipSuccess) {
            cleanup();
            return hip_fail(he, "hipEventCreate");
        }
        ev.push_back(e);
    }
    {
        std::lock_guard<std::mutex> lk(g_mu);
        int dev, ncu;
        if ((rc = current_device(&dev, &ncu))) {
            cleanup();
            return rc;
        }
        const KeyCtx *ctx;
        if ((rc = key_ctx(key, ks, dev, &ctx))) {
            cleanup();
            return rc;
        }
        for (uint64_t g = 0; g < ngroups; ++g) {
            for (uint64_t k = g * group; k < (g + 1) * group && k < nchunks; ++k) {
                const uint64_t off = k * chunk_bytes;
                rc = run_gcm(true, kFused, ctx, base_iv, chain_bytes, k * cpc, d_pt + off, nullptr, chunk_len(k),
                             d_ct + off, aad_bytes ? d_aad : nullptr, aad_bytes, nullptr, d_tags, nullptr, 0, dev, ncu,
                             ks);
                if (rc) {
                    cleanup();
                    return rc;
                }
            }
            he = hipEventRecord(ev[g], ks);
            if (he != hipSuccess) {
                cleanup();
                return hip_fail(he, "hipEventRecord");
            }
        }
    }
    for (uint64_t g = 0; g < ngroups; ++g) {
        he = hipEventSynchronize(ev[g]);
        for (uint64_t k = g * group; k < (g + 1) * group && k < nchunks && he == hipSuccess; ++k) {
            const uint64_t off = k * chunk_bytes;
            he = hipMemcpyAsync(h_ct + off, d_ct + off, chunk_len(k), hipMemcpyDeviceToHost, cs);
        }
        if (he != hipSuccess) {
            cleanup();
            return hip_fail(he, "pipeline copy");
        }
    }
    he = hipMemcpyAsync(h_tags, d_tags, 16 * n, hipMemcpyDeviceToHost, cs);
    cleanup();
    if (he != hipSuccess)
        return hip_fail(he, "tag copy");
    return FASTRACK_OK;
}

}  // namespace

FT_EXPORT int fastrack_pipeline_d2h(const uint8_t *key, const uint8_t *base_iv, uint64_t chain_bytes,
                                    const uint8_t *d_pt, uint64_t len, const uint8_t *d_aad, uint32_t aad_bytes,
                                    uint64_t chunk_bytes, uint8_t *d_ct, uint8_t *d_tags, uint8_t *h_ct,
                                    uint8_t *h_tags, void *copy_stream, void *compute_stream)
{
    return d2h_impl(key, base_iv, chain_bytes, d_pt, len, d_aad, aad_bytes, chunk_bytes, d_ct, d_tags, h_ct, h_tags,
                    copy_stream, compute_stream, FASTRACK_PIPE_FUSED);
}

FT_EXPORT int fastrack_pipeline_d2h_mode(const uint8_t *key, const uint8_t *base_iv, uint64_t chain_bytes,
                                         const uint8_t *d_pt, uint64_t len, const uint8_t *d_aad, uint32_t aad_bytes,
                                         uint64_t chunk_bytes, uint8_t *d_ct, uint8_t *d_tags, uint8_t *h_ct,
                                         uint8_t *h_tags, void *copy_stream, void *compute_stream, uint32_t mode)
{
    return d2h_impl(key, base_iv, chain_bytes, d_pt, len, d_aad, aad_bytes, chunk_bytes, d_ct, d_tags, h_ct, h_tags,
                    copy_stream, compute_stream, mode);
}

namespace {

// Ragged chains: chain i = bytes [off[i], off[i] + len[i]) of in/out, IV_i, tag i,
// AAD i, ok[i]. The chains are planned on the host (lanes per item from the mean
// chain length, segments of one size for all chains) and the chain and item
// tables go to the device through the stream's pinned staging.
// The ragged table slot b of (dev, s) with room for `bytes`, the upload stream and
// events created on first use. Growing the slots waits for both streams first.
int ragged_slot(int dev, hipStream_t s, int b, size_t bytes, ScratchEntry **out_e, uint8_t **out)
{
    ScratchEntry *e = nullptr;
    for (auto &x : g_scratch)
        if (x.dev == dev && x.stream == s)
            e = &x;
    if (!e)
        return fail(FASTRACK_EHIP, "no staging for this stream");
    hipError_t he;
    if (!e->up) {
        // default priority: the library keeps every stream at the default
        if ((he = hipStreamCreateWithFlags(&e->up, hipStreamNonBlocking)) != hipSuccess) {
            e->up = nullptr;
            return hip_fail(he, "hipStreamCreate for the table uploads");
        }
        for (int k = 0; k < 2; ++k)
            if ((he = hipEventCreateWithFlags(&e->slot_free[k], hipEventDisableTiming)) != hipSuccess) {
                e->slot_free[k] = nullptr;
                return hip_fail(he, "hipEventCreate");
            }
    }
    if (e->rtab_slot < bytes) {
        if (e->rtab) {   // earlier kernels and uploads may still use the old slots
            if ((he = hipStreamSynchronize(s)) != hipSuccess || (he = hipStreamSynchronize(e->up)) != hipSuccess)
                return hip_fail(he, "hipStreamSynchronize");
            (void)hipFree(e->rtab);
            e->rtab = nullptr;
            e->rtab_slot = 0;
            e->slot_used[0] = e->slot_used[1] = false;
        }
        const size_t slot = (bytes + (1u << 20) - 1) & ~(size_t)((1u << 20) - 1);   // whole MiB, fewer regrowths
        if ((he = hipMalloc(&e->rtab, 2 * slot)) != hipSuccess) {
            e->rtab = nullptr;
            return fail(FASTRACK_ENOMEM, "hipMalloc(%zu) for the ragged tables: %s", 2 * slot, hipGetErrorString(he));
        }
        e->rtab_slot = slot;
    }
    *out_e = e;
    *out = static_cast<uint8_t *>(e->rtab) + (size_t)b * e->rtab_slot;
    return FASTRACK_OK;
}

int run_ragged(bool encrypt, const uint8_t *key, const uint8_t *base_iv, const uint64_t *h_off, const uint64_t *h_len,
               uint64_t n, const uint8_t *in, uint8_t *out, const uint8_t *aad, uint32_t aad_bytes,
               const uint8_t *tags_in, uint8_t *tags_out, uint8_t *ok, void *stream)
{
    g_err.clear();
    if (!key || !base_iv)
        return fail(FASTRACK_EINVAL, "key and base_iv must be non-NULL host pointers");
    if (n == 0)
        return FASTRACK_OK;
    if (!h_off || !h_len)
        return fail(FASTRACK_EINVAL, "h_chain_off and h_chain_len must be non-NULL host arrays");
    if (n > 0xFFFFFFFFull)
        return fail(FASTRACK_EINVAL, "more than 2^32-1 chains");
    uint64_t end = 0, blocks = 0, qmax = 0;
    // per-call work arrays, kept per thread so that calls do not allocate them
    thread_local std::vector<uint32_t> q, it0, order, cnt;
    q.resize(n);   // blocks of each chain (a partial block counts as one)
    for (uint64_t i = 0; i < n; ++i) {
        if (h_off[i] & 15)
            return fail(FASTRACK_EINVAL, "chain %llu starts at offset %llu, not a multiple of 16", (unsigned long long)i,
                        (unsigned long long)h_off[i]);
        if (h_off[i] < end)
            return fail(FASTRACK_EINVAL, "chain %llu overlaps the chain before it (chains must be in increasing order)",
                        (unsigned long long)i);
        if ((h_len[i] + 15) / 16 > kMaxChainBlocks)
            return fail(FASTRACK_EINVAL, "chain %llu is longer than (2^32-2)*16 bytes", (unsigned long long)i);
        end = h_off[i] + h_len[i];
        q[i] = (uint32_t)((h_len[i] + 15) / 16);
        blocks += q[i];
        qmax = q[i] > qmax ? q[i] : qmax;
    }
    if (aad_bytes && !aad)
        return fail(FASTRACK_EINVAL, "aad is NULL but aad_bytes = %u", aad_bytes);
    if (blocks && (!in || !out))   // NULL buffers are fine when every chain is empty
        return fail(FASTRACK_EINVAL, "input and output buffers must be non-NULL");
    if (((uintptr_t)in & 15) || ((uintptr_t)out & 15))
        return fail(FASTRACK_EINVAL, "input and output must be 16-byte aligned");
    if (blocks && overlap_bad(in, out, end))
        return fail(FASTRACK_EINVAL, "input and output overlap partially (in place means the same pointer)");
    if (encrypt ? !tags_out : (!tags_in || !ok))
        return fail(FASTRACK_EINVAL, encrypt ? "d_tags must be non-NULL" : "d_tags and d_ok must be non-NULL");

    std::lock_guard<std::mutex> lk(g_mu);
    int dev, ncu;
    int rc;
    if ((rc = current_device(&dev, &ncu)))
        return rc;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    const KeyCtx *ctx;
    if ((rc = key_ctx(key, s, dev, &ctx)))
        return rc;

    // Plan: lanes per item from the mean chain length, as for uniform chains. Chains
    // of their own lengths leave the waves unevenly loaded when a wave takes few
    // items, so chains are cut into segments of one size (2^lg blocks, at least
    // 4 iterations of the item's lanes) until every wave has about 4 wave-items (fewer
    // and longer items than that pay their tails too often; more leave waves uneven).
    const uint64_t slots = (uint64_t)ncu * kGcmWavesPerWg;
    const uint64_t qmean = (blocks + n - 1) / n;
    uint32_t ll = 0;
    for (uint32_t cand = 4; cand <= 6; ++cand)
        if (qmean >= (4ull << cand) && ((n << cand) + 63) / 64 >= slots) {
            ll = cand;
            break;
        }
    if (ll == 0)
        ll = qmean >= 256 ? 6 : (qmean >= 128 ? 5 : 4);
    uint32_t lg0 = ceil_log2(qmax > 0 ? qmax : 1);
    if (lg0 > 31)
        lg0 = 31;
    // Items of a chain of x blocks with segments of 2^g: max(1, ceil(x / 2^g)) (no overflow for x < 2^32).
    auto segs_of = [](uint32_t x, uint32_t g) {
        const uint32_t sg = (x >> g) + ((x & ((1u << g) - 1)) != 0);
        return sg ? sg : 1u;
    };
    auto items_at = [&](uint32_t g) {
        uint64_t t = 0;
        for (uint64_t i = 0; i < n; ++i)
            t += segs_of(q[i], g);
        return t;
    };
    const uint32_t lg_min = ll + 2 < lg0 ? ll + 2 : lg0;
    const uint64_t want_items = (4 * slots) << (6 - ll);   // 4 wave-items of 64 / 2^ll items per wave
    // The segment size is the largest 2^lg (lg_min <= lg <= lg0) that still gives
    // want_items items, else 2^lg_min. The item count falls as lg grows, so the
    // search starts from an estimate (a chain adds about x / 2^lg + 1/2 items) and
    // steps to the answer: one or two passes over the chains instead of one per
    // candidate size.
    uint32_t lg = lg0;
    {
        const uint64_t rest = want_items > n / 2 ? want_items - n / 2 : 1;
        uint32_t ge = 0;
        while (ge < 31 && ((uint64_t)blocks >> (ge + 1)) >= rest)
            ++ge;
        lg = ge < lg_min ? lg_min : (ge > lg0 ? lg0 : ge);
    }
    uint64_t n_items = items_at(lg);
    if (n_items >= want_items) {
        while (lg < lg0) {
            const uint64_t up = items_at(lg + 1);
            if (up < want_items)
                break;
            ++lg;
            n_items = up;
        }
    } else {
        while (lg > lg_min && n_items < want_items)
            n_items = items_at(--lg);
    }
    if (n_items > 0xFFFFFFFFull)
        return fail(FASTRACK_EINVAL, "more than 2^32-1 work items");

    // Device: chain table | item table | (split) partials | masks. Host: the two tables.
    // Tables (chain table | item table) go through pinned staging and an upload kernel
    // into a table slot; partials and masks (split launches) use the stream's scratch.
    const size_t tab_bytes = round256(n * sizeof(RaggedChain)) + round256(n_items * 4);
    const bool split = n_items > n;
    void *sc = nullptr;
    if (split && (rc = scratch_for(dev, s, (n_items + n) * 16, &sc)))
        return rc;
    uint8_t *host = nullptr;
    if ((rc = staging_for(dev, s, tab_bytes, &host)))
        return rc;
    ScratchEntry *se = nullptr;
    uint8_t *tab = nullptr;
    int slot = 0;
    for (auto &x : g_scratch)
        if (x.dev == dev && x.stream == s)
            slot = x.cur;
    if ((rc = ragged_slot(dev, s, slot, tab_bytes, &se, &tab)))
        return rc;
    RaggedChain *hc = reinterpret_cast<RaggedChain *>(host);
    uint32_t *hi = reinterpret_cast<uint32_t *>(host + round256(n * sizeof(RaggedChain)));
    // Item order: every chain's segment 0 (the short one, or the whole chain) first,
    // longest first, then the full-length segments chain by chain. A wave-item runs
    // as many iterations as its longest item, so items of like length side by side
    // waste fewer lanes (on the 1024-sample batch: 98.5% of the lane-iterations
    // useful instead of 89%).
    it0.resize(n);   // iterations of each chain's segment 0, then its item number
    uint32_t max_it0 = 0;
    const uint32_t lmask = (1u << lg) - 1, lstep = (1u << ll) - 1;
    for (uint64_t i = 0; i < n; ++i) {
        const uint32_t x = q[i];
        const uint32_t b0 = x == 0 ? 0u : ((x - 1) & lmask) + 1;   // blocks of segment 0
        it0[i] = (uint32_t)(((uint64_t)b0 + lstep) >> ll);
        max_it0 = it0[i] > max_it0 ? it0[i] : max_it0;
    }
    if (max_it0 < (1u << 16)) {   // counting sort on the iteration count, longest first
        cnt.assign((size_t)max_it0 + 1, 0);
        for (uint64_t i = 0; i < n; ++i)
            ++cnt[max_it0 - it0[i]];
        uint32_t run = 0;
        for (auto &c : cnt) {
            const uint32_t k = c;
            c = run;
            run += k;
        }
        for (uint64_t i = 0; i < n; ++i) {
            const uint32_t k = cnt[max_it0 - it0[i]]++;
            it0[i] = k;
            hi[k] = (uint32_t)i;
        }
    } else {
        order.resize(n);
        for (uint64_t i = 0; i < n; ++i)
            order[i] = (uint32_t)i;
        std::stable_sort(order.begin(), order.end(), [&](uint32_t a, uint32_t b) { return it0[a] > it0[b]; });
        for (uint64_t k = 0; k < n; ++k) {
            it0[order[k]] = (uint32_t)k;
            hi[k] = order[k];
        }
    }
    // The chain table in chain order, one sequential pass (with the full-length
    // segments' items behind the segment-0 items).
    uint64_t item = n;
    for (uint64_t i = 0; i < n; ++i) {
        const uint32_t sg = segs_of(q[i], lg);
        RaggedChain &c = hc[i];
        c.off = h_off[i];
        c.len = h_len[i];
        c.item_base = item - 1;   // segment s >= 1 is item item_base + s
        c.segs = sg;
        c.item0 = it0[i];
        for (uint32_t k = 1; k < sg; ++k)
            hi[item++] = (uint32_t)i;
    }
    // A copy kernel reads the pinned tables over the host link: hipMemcpyAsync held
    // the calling thread until the stream reached the copy, leaving the GPU idle
    // while the host then prepared the launch.
    // The upload runs on the library's upload stream, so it overlaps the kernels of
    // the call before: it waits only for the kernels that last read this slot (two
    // calls back), and the kernels of this call wait for it.
    hipError_t he;
    const void *host_dev = se->host_dev[slot];   // the staging buffer's device address
    if (se->slot_used[slot] && (he = hipStreamWaitEvent(se->up, se->slot_free[slot], 0)) != hipSuccess)
        return hip_fail(he, "hipStreamWaitEvent");
    if ((he = launch_upload(host_dev, tab, tab_bytes, se->up)) != hipSuccess)
        return hip_fail(he, "chain table upload");
    if ((rc = staging_read(dev, s, se->up)))   // the staging is read once the upload has run
        return rc;
    if ((he = hipStreamWaitEvent(s, se->host_read[slot], 0)) != hipSuccess)
        return hip_fail(he, "hipStreamWaitEvent");

    GcmLaunch p;
    std::memset(&p, 0, sizeof p);
    p.ctx = ctx;
    p.in = in;
    p.out = out;
    iv_words(base_iv, p.iv);
    p.aad = aad_bytes ? aad : nullptr;
    p.aad_bytes = aad_bytes;
    p.tags_in = tags_in;
    p.tags_out = tags_out;
    p.ok = ok;
    p.n_chains = (uint32_t)n;
    p.n_items = n_items;
    p.lanes_log2 = ll;
    p.seg_log2 = lg;
    p.qc = (uint32_t)qmax;
    p.rchains = reinterpret_cast<const RaggedChain *>(tab);
    p.ritem_chain = reinterpret_cast<const uint32_t *>(tab + round256(n * sizeof(RaggedChain)));
    p.split = split ? 1u : 0u;
    if (split) {
        p.partials = reinterpret_cast<uint4 *>(sc);
        p.masks = p.partials + n_items;
    }
    he = launch_gcm(p, encrypt, kFused, ncu, s);
    if (he != hipSuccess)
        return hip_fail(he, "GCM launch");
    if ((he = hipEventRecord(se->slot_free[slot], s)) != hipSuccess)
        return hip_fail(he, "hipEventRecord");
    se->slot_used[slot] = true;
    return FASTRACK_OK;
}

}  // namespace

FT_EXPORT int fastrack_gcm_decrypt_verify_ragged(const uint8_t *key, const uint8_t *base_iv, const uint64_t *h_chain_off,
                                                 const uint64_t *h_chain_len, uint64_t n_chains, const uint8_t *d_ct,
                                                 const uint8_t *d_tags, const uint8_t *d_aad, uint32_t aad_bytes,
                                                 uint8_t *d_pt, uint8_t *d_ok, void *stream)
{
    return run_ragged(false, key, base_iv, h_chain_off, h_chain_len, n_chains, d_ct, d_pt, d_aad, aad_bytes, d_tags,
                      nullptr, d_ok, stream);
}

FT_EXPORT int fastrack_gcm_encrypt_tag_ragged(const uint8_t *key, const uint8_t *base_iv, const uint64_t *h_chain_off,
                                              const uint64_t *h_chain_len, uint64_t n_chains, const uint8_t *d_pt,
                                              const uint8_t *d_aad, uint32_t aad_bytes, uint8_t *d_ct, uint8_t *d_tags,
                                              void *stream)
{
    return run_ragged(true, key, base_iv, h_chain_off, h_chain_len, n_chains, d_pt, d_ct, d_aad, aad_bytes, nullptr,
                      d_tags, nullptr, stream);
}

FT_EXPORT uint64_t fastrack_sample_chains(const uint64_t *h_sample_len, uint64_t n_samples, uint32_t chains_per_sample,
                                          uint64_t *h_chain_off, uint64_t *h_chain_len)
{
    if (!h_sample_len || !h_chain_off || !h_chain_len || chains_per_sample == 0)
        return 0;
    uint64_t off = 0, c = 0;
    for (uint64_t s = 0; s < n_samples; ++s) {
        const uint64_t len = h_sample_len[s];
        // equal parts rounded up to whole blocks, so every part that holds data starts
        // aligned; parts past the end are empty and sit at the sample's 16-byte-rounded end
        const uint64_t part = ((len + chains_per_sample - 1) / chains_per_sample + 15) & ~15ull;
        const uint64_t end16 = (len + 15) & ~15ull;
        for (uint32_t j = 0; j < chains_per_sample; ++j) {
            const uint64_t b = (uint64_t)j * part;
            const uint64_t l = b >= len ? 0 : (len - b < part ? len - b : part);
            h_chain_off[c] = off + (b < len ? b : end16);
            h_chain_len[c] = l;
            ++c;
        }
        off = (off + len + 15) & ~15ull;   // the next sample starts 16-byte aligned
    }
    return off;
}

FT_EXPORT int fastrack_clock_probe(uint64_t window_us, uint32_t n_probes, uint64_t *d_out, void *stream)
{
    g_err.clear();
    if (!d_out || n_probes == 0 || n_probes > 1024)
        return fail(FASTRACK_EINVAL, "d_out must be non-NULL and n_probes in 1..1024 (got %u)", n_probes);
    if (window_us == 0 || window_us > 10000000)
        return fail(FASTRACK_EINVAL, "window_us must be in 1..10^7 (got %llu)", (unsigned long long)window_us);
    hipError_t he = launch_clock_probe(window_us * 100, n_probes, d_out, reinterpret_cast<hipStream_t>(stream));
    return he == hipSuccess ? FASTRACK_OK : hip_fail(he, "clock probe launch");
}

FT_EXPORT void fastrack_shutdown(void)
{
    std::lock_guard<std::mutex> lk(g_mu);
    // Key-derived tables of the allocation-free path do not outlive the library's use.
    int cur = -1;
    if (hipGetDevice(&cur) == hipSuccess) {
        for (int dev = 0; dev < kNoAllocMaxDevices; ++dev) {
            NoAllocDevice &d = g_noalloc[dev];
            if (!d.ptr || !d.have_key)
                continue;
            if (hipSetDevice(dev) == hipSuccess && hipDeviceSynchronize() == hipSuccess)
                (void)hipMemset(d.ptr, 0, kNoAllocKeyBytes);
            d.have_key = false;
            d.key.fill(0);
        }
        (void)hipSetDevice(cur);
    }
    if (g_keys.empty() && g_scratch.empty() && g_pools.empty())
        return;
    (void)hipDeviceSynchronize();
    g_keys.clear();
    for (auto &p : g_pools) {
        // key-derived material does not outlive the library's state
        (void)hipMemset(p.base, 0, kMaxKeys * kKeySlotBytes);
        (void)hipFree(p.base);
        for (auto &ev : p.ready)
            (void)hipEventDestroy(ev);
    }
    g_pools.clear();
    for (auto &s : g_scratch) {
        (void)hipFree(s.ptr);
        (void)hipFree(s.rtab);
        for (int b = 0; b < 2; ++b) {
            if (s.host[b])
                (void)hipHostFree(s.host[b]);
            if (s.host_read[b])
                (void)hipEventDestroy(s.host_read[b]);
            if (s.slot_free[b])
                (void)hipEventDestroy(s.slot_free[b]);
        }
        if (s.up)
            (void)hipStreamDestroy(s.up);
    }
    g_scratch.clear();
}
