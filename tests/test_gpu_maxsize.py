"""GPU: the largest chain the method allows, in one launch.

A GCM message (each chain, paper section 5.2) holds at most 2^32 - 2 blocks, so
one chain of (2^32 - 2) * 16 bytes (64 GiB) is the largest input the library
accepts as a single chain. The oracle cannot run GHASH over 64 GiB in test time,
so the test pins what it can compute one block at a time and checks the rest by
properties that hold at any size:
- sampled ciphertext blocks, at the start, the middle and where the 32-bit block
  counter reaches its top (2^32 - 1 for the last block), equal the plaintext XOR
  the oracle's AES-256 of IV || [t + 2]_32;
- decrypt + verify of the GPU's own ciphertext and tag accepts the chain and
  returns the plaintext exactly;
- one flipped ciphertext bit in the last block is rejected and flips exactly
  that plaintext bit (CTR malleability).
"""
import numpy as np
import pytest

import oracle
import workloads as W

pytestmark = pytest.mark.gpu

MAX_BLOCKS = (1 << 32) - 2
GiB = 1 << 30


@pytest.fixture(scope="module")
def F():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2410_15240_amd as F
    F.lib()
    return F


def equal_in_slices(a, b):
    n = a.numel()
    return all(bool((a[i:i + GiB] == b[i:i + GiB]).all()) for i in range(0, n, GiB))


def test_largest_chain(F):
    import torch
    length = MAX_BLOCKS * 16
    free, _ = torch.cuda.mem_get_info()
    if free < 2 * length + 8 * GiB:
        pytest.skip("needs %d GiB of free device memory (two 64 GiB buffers)" % ((2 * length + 8 * GiB) >> 30))
    rng = np.random.Generator(np.random.PCG64(W.SEED_BASE + 4242))
    key, iv = W.draw_key_iv(rng)
    g = torch.Generator(device="cuda").manual_seed(4242)
    pt = torch.empty(length, dtype=torch.uint8, device="cuda")
    for i in range(0, length, GiB):
        m = min(GiB, length - i)
        pt[i:i + m] = torch.randint(0, 256, (m,), dtype=torch.uint8, device="cuda", generator=g)
    try:
        ct, tags = F.encrypt_tag(key, iv, length, pt)
        torch.cuda.synchronize()
        # sampled blocks against the oracle's keystream block AES_K(IV || [t + 2]_32)
        samples = [0, 1, 2, 255, 256, 1 << 20, 1 << 31, MAX_BLOCKS - 258, MAX_BLOCKS - 257, MAX_BLOCKS - 256,
                   MAX_BLOCKS - 2, MAX_BLOCKS - 1]
        for t in samples:
            ks = oracle.aes256_encrypt_block(key, np.frombuffer(bytes(iv) + (t + 2).to_bytes(4, "big"), np.uint8))
            p = pt[16 * t:16 * t + 16].cpu().numpy()
            c = ct[16 * t:16 * t + 16].cpu().numpy()
            assert np.array_equal(c, p ^ ks), t
        # tamper one bit of the last block: rejected, and exactly that bit differs
        bit = 8 * 16 * (MAX_BLOCKS - 1) + 77
        byte, mask = bit // 8, 0x80 >> (bit % 8)
        ct[byte] ^= mask
        out, ok = F.decrypt_verify(key, iv, length, ct, tags, out=ct)
        assert ok.cpu().tolist() == [0]
        out[byte] ^= mask
        assert equal_in_slices(out, pt)
        # encrypt again in place, then the untouched ciphertext and tag verify
        ct2, tags2 = F.encrypt_tag(key, iv, length, out, out=out)
        assert torch.equal(tags2, tags)
        pt2, ok2 = F.decrypt_verify(key, iv, length, ct2, tags2, out=ct2)
        assert ok2.cpu().tolist() == [1]
        assert equal_in_slices(pt2, pt)
    finally:
        del pt
        ct = ct2 = pt2 = out = None
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
