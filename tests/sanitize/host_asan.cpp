// Sanitizer driver for the library's host-only paths (test infrastructure): the
// pipeline planner, the per-sample chain layout, the size helpers and the argument
// checks that return before any HIP call, on exactly sized host arrays, under
// AddressSanitizer / UndefinedBehaviorSanitizer. No device is touched.
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include <vector>

#include "fastrack.h"

int main()
{
    int fails = 0;
    const uint64_t MiB = 1ull << 20;
    const uint64_t lens[] = {1, 4096, 64 * MiB, 64 * MiB + 4096, 100 * MiB + 16};
    for (uint64_t len : lens)
        for (int depth : {0, 2, 3, 8})
            for (uint32_t mode = 0; mode <= 2; ++mode) {
                const int64_t n = fastrack_pipeline_plan(len, 4096, 8 * MiB, depth, mode, nullptr, 0);
                if (n < 0)
                    continue;   // rejected combination (checked below)
                std::vector<int64_t> ops((size_t)(6 * n));   // exactly n records
                fails += fastrack_pipeline_plan(len, 4096, 8 * MiB, depth, mode, ops.data(), (uint64_t)n) != n;
                std::vector<int64_t> half((size_t)(6 * (n / 2)));   // a short buffer: only n/2 written
                fails += fastrack_pipeline_plan(len, 4096, 8 * MiB, depth, mode, half.data(), (uint64_t)(n / 2)) != n;
                fails += fastrack_pipeline_stage_bytes(len, 4096, 32, 8 * MiB, depth) == 0;
            }
    fails += fastrack_pipeline_plan(64 * MiB, 4096, 8 * MiB, 1, 0, nullptr, 0) != FASTRACK_EINVAL;
    fails += fastrack_pipeline_plan(64 * MiB, 4096, 8 * MiB, 0, 1, nullptr, 0) != FASTRACK_EINVAL;
    fails += strlen(fastrack_last_error()) == 0;
    const uint64_t nss[] = {1, 3, 100};
    for (uint64_t ns : nss)
        for (uint32_t k : {1u, 7u, 16u}) {
            std::vector<uint64_t> slen(ns), off(ns * k), ln(ns * k);
            for (uint64_t i = 0; i < ns; ++i)
                slen[i] = (i * 7919 + 5) % 70000;
            const uint64_t total = fastrack_sample_chains(slen.data(), ns, k, off.data(), ln.data());
            for (uint64_t c = 0; c < ns * k; ++c)
                fails += off[c] + ln[c] > total;
        }
    const uint64_t nlen[] = {0, 1, 16, 1ull << 40}, nch[] = {0, 16, 4096};
    for (uint64_t len : nlen)
        for (uint64_t c : nch)
            fails += fastrack_num_chains(len, c) != (c ? (len + c - 1) / c : 0);
    // argument checks that return before any HIP call (the pointers are never dereferenced)
    uint8_t key[32] = {0}, iv[12] = {0};
    uint8_t *A = reinterpret_cast<uint8_t *>(0x10000), *B = reinterpret_cast<uint8_t *>(0x90000);
    fails += fastrack_gcm_decrypt_verify(key, iv, 17, A, 4096, B, nullptr, 0, B, B, 0, nullptr) != FASTRACK_EINVAL;
    fails += fastrack_gcm_encrypt_tag(key, iv, 4096, A, 4096, nullptr, 8, B, B, 0, nullptr) != FASTRACK_EINVAL;
    fails += fastrack_gcm_decrypt_verify(key, iv, 4096, A, 4096, B, nullptr, 0, A + 16, B, 0, nullptr) != FASTRACK_EINVAL;
    const uint64_t roff[3] = {0, 4096, 100}, rlen[3] = {4096, 4096, 16};   // overlapping chains
    fails += fastrack_gcm_decrypt_verify_ragged(key, iv, roff, rlen, 3, A, B, nullptr, 0, B, B, nullptr) !=
             FASTRACK_EINVAL;
    printf("host sanitizer driver: %d failures (last error: %s)\n", fails, fastrack_last_error());
    return fails != 0;
}
