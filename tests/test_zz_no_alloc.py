"""The allocation-free decrypt + verify entry point through the C ABI: its output
equals that of fastrack_gcm_decrypt_verify on the same inputs, bit for bit, over
calls in a row that shrink the input, change the key and cut chains into
segments (so the fixed area's partial slots are used) or not."""
import ctypes
import time

import numpy as np
import pytest

import oracle
import workloads as W

pytestmark = pytest.mark.gpu

KiB, MiB = W.KiB, W.MiB


def say(*a):
    print("[%s]" % time.strftime("%H:%M:%S"), *a, flush=True)


@pytest.fixture(scope="module")
def L():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2410_15240_amd as F
    L = F.lib()
    vp, u64, u32 = ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint32
    L.fastrack_gcm_decrypt_verify_noalloc.argtypes = [vp, vp, u64, vp, u64, vp, vp, u32, vp, vp, u32, vp]
    L.fastrack_gcm_decrypt_verify_noalloc.restype = ctypes.c_int
    return L


def run(L, fn, w, chain, ct, tags, aad, abytes, flags=0):
    import torch
    key = ctypes.create_string_buffer(bytes(w.key), 32)
    iv = ctypes.create_string_buffer(bytes(w.base_iv), 12)
    out = torch.full_like(ct, 0x77)
    ok = torch.full((tags.shape[0],), 0x55, dtype=torch.uint8, device=ct.device)
    stream = torch.cuda.current_stream().cuda_stream
    rc = getattr(L, fn)(key, iv, chain, ct.data_ptr(), ct.numel(), tags.data_ptr(),
                        aad.data_ptr() if abytes else None, abytes, out.data_ptr(), ok.data_ptr(), flags, stream)
    assert rc == 0, L.fastrack_last_error()
    torch.cuda.synchronize()
    return out.cpu().numpy(), ok.cpu().numpy()


# (seed, length, chain, aad bytes): the first cuts 64 KiB chains into segments, the
# second is smaller under a new key (segments again), the third smaller still under
# the first key, whole chains only (no partial slots), the fourth one long chain.
CALLS = [(501, 8 * MiB + 48, 64 * KiB, 32), (502, MiB + 100, 16 * KiB, 13), (501, 300 * KiB + 5, 4 * KiB, 0),
         (503, 3 * MiB + 16, 4 * MiB, 1)]


def test_noalloc_matches_decrypt_verify_over_calls_in_a_row(L):
    import torch
    for seed, length, chain, abytes in CALLS:
        say("no-alloc call: seed", seed, "length", length, "chain", chain, "aad", abytes)
        w = W.random_case(seed, length, chain, abytes)
        aad = W.case_aad(w, chain)
        ct, tags = oracle.chains_encrypt(w.key, w.base_iv, chain, w.payload, aad, abytes)
        n = tags.shape[0]
        W.flip_bit(ct[(n // 2) * chain:], 3)          # one chain tampered in the middle
        d_ct = torch.from_numpy(ct).cuda()
        d_tags = torch.from_numpy(tags).cuda()
        d_aad = torch.from_numpy(np.ascontiguousarray(aad)).cuda() if abytes else None
        pt_a, ok_a = run(L, "fastrack_gcm_decrypt_verify_noalloc", w, chain, d_ct, d_tags, d_aad, abytes)
        pt_b, ok_b = run(L, "fastrack_gcm_decrypt_verify", w, chain, d_ct, d_tags, d_aad, abytes)
        assert np.array_equal(pt_a, pt_b) and np.array_equal(ok_a, ok_b)
        want_pt, want_ok = oracle.chains_decrypt(w.key, w.base_iv, chain, ct, tags, aad, abytes)
        assert np.array_equal(pt_a, want_pt) and np.array_equal(ok_a, want_ok)
        assert ok_a.tolist() == [0 if i == n // 2 else 1 for i in range(n)]


def test_noalloc_sequential_ghash_flag(L):
    import torch
    say("no-alloc call with the sequential-GHASH flag")
    w = W.random_case(504, 256 * KiB + 7, 64 * KiB, 0)
    ct, tags = oracle.chains_encrypt(w.key, w.base_iv, 64 * KiB, w.payload)
    d_ct, d_tags = torch.from_numpy(ct).cuda(), torch.from_numpy(tags).cuda()
    pt_a, ok_a = run(L, "fastrack_gcm_decrypt_verify_noalloc", w, 64 * KiB, d_ct, d_tags, None, 0, flags=1)
    pt_b, ok_b = run(L, "fastrack_gcm_decrypt_verify", w, 64 * KiB, d_ct, d_tags, None, 0)
    assert np.array_equal(pt_a, pt_b) and np.array_equal(ok_a, ok_b) and ok_a.all()
    assert np.array_equal(pt_a, w.payload)
