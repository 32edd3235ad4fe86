"""GPU parity of the eager-evaluation, keystream-precompute and pipeline-mode
paths (the paper's section 5.3 variants) through the C ABI, against the CPU
oracle. Every expected value comes from the oracle; comparisons are bit-exact."""
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
def F():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2410_15240_amd as F
    if not __import__("os").path.exists(F.library_path()):
        from paper_2410_15240_amd import build
        build.build()
    F.lib()
    return F


def dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(t):
    import torch
    torch.cuda.synchronize()
    return t.cpu().numpy()


def tampered_case(seed, length, chain, abytes):
    w = W.random_case(seed, length, chain, abytes)
    aad = W.case_aad(w, chain)
    ct, tags = oracle.chains_encrypt(w.key, w.base_iv, chain, w.payload, aad, abytes)
    n = tags.shape[0]
    W.flip_bit(ct, 5)                                         # chain 0
    if n > 2:
        W.flip_bit(tags[n - 2], 100)                          # a tag
    if n > 3 and abytes:
        W.flip_bit(aad[3], 7)                                 # an AAD bit
    want_pt, want_ok = oracle.chains_decrypt(w.key, w.base_iv, chain, ct, tags, aad, abytes)
    return w, aad, ct, tags, want_pt, want_ok


EAGER_SHAPES = [(4096 * 5 + 7, 4096, 32), (3 * 65536 + 16, 65536, 0), (2 * MiB + 100, 256 * KiB, 13),
                (8 * MiB, 1 * MiB, 32), (17, 16, 0)]


@pytest.mark.parametrize("length,chain,abytes", EAGER_SHAPES)
def test_eager_matches_oracle(F, length, chain, abytes):
    import torch
    say("eager", length, chain, abytes)
    w, aad, ct, tags, want_pt, want_ok = tampered_case(length % 997 + abytes, length, chain, abytes)
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    for vs in (s2, s1):                                       # separate and shared streams
        e = F.decrypt_eager(w.key, w.base_iv, chain, dev(ct), dev(tags), dev(aad) if abytes else None,
                            decrypt_stream=s1, verify_stream=vs)
        s1.synchronize()
        assert np.array_equal(e.plaintext.cpu().numpy(), want_pt)
        assert e.rejected() == np.nonzero(want_ok == 0)[0].tolist()
        assert e.done()
        assert e.settle(lambda: "commit", lambda bad: ("rollback", bad)) == ("rollback", e.rejected())


def test_eager_rejects_decrypting_in_place(F):
    w = W.random_case(1, 4096, 4096, 0)
    ct, tags = oracle.chains_encrypt(w.key, w.base_iv, 4096, w.payload)
    d_ct = dev(ct)
    with pytest.raises(F.FastrackError):
        F.decrypt_eager(w.key, w.base_iv, 4096, d_ct, dev(tags), out=d_ct)


KS_SHAPES = [(4096 * 5 + 7, 4096, 0), (4096 * 5 + 7, 4096, 3), (3 * 65536 + 16, 65536, 1), (1 * MiB, 1 * MiB, 0),
             (8 * MiB + 48, 1 * MiB, 2), (5, 16, 7)]


@pytest.mark.parametrize("length,chain,base", KS_SHAPES)
def test_keystream_is_the_ciphertext_of_zeros(F, length, chain, base):
    say("keystream", length, chain, base)
    w = W.random_case(length % 991 + base, 16, 16, 0)        # key and IV only
    total = base * chain + length
    zeros = np.zeros(total, np.uint8)
    ct_zero, _ = oracle.chains_encrypt(w.key, w.base_iv, chain, zeros)
    ks = F.keystream(w.key, w.base_iv, chain, length, chain_base=base)
    assert np.array_equal(host(ks), ct_zero[base * chain:])


@pytest.mark.parametrize("length,chain,abytes", EAGER_SHAPES)
def test_apply_verify_matches_oracle(F, length, chain, abytes):
    say("apply", length, chain, abytes)
    w, aad, ct, tags, want_pt, want_ok = tampered_case(length % 983 + abytes + 1, length, chain, abytes)
    d_tags, d_aad = dev(tags), (dev(aad) if abytes else None)
    ks = F.keystream(w.key, w.base_iv, chain, length)
    pt, ok = F.apply_verify(w.key, w.base_iv, chain, dev(ct), ks, d_tags, d_aad, aad_bytes=abytes or None)
    assert np.array_equal(host(pt), want_pt)
    assert np.array_equal(host(ok), want_ok)
    # a run of chains in the middle, indexed globally, decrypted in place over its keystream
    n = tags.shape[0]
    if n >= 3:
        c0, m = 1, n - 2
        sub = ct[c0 * chain:(c0 + m) * chain]
        ks2 = F.keystream(w.key, w.base_iv, chain, sub.size, chain_base=c0)
        ok2 = dev(np.full(n, 7, np.uint8))
        pt2, ok2 = F.apply_verify(w.key, w.base_iv, chain, dev(sub), ks2, d_tags, d_aad,
                                  aad_bytes=abytes or None, chain_base=c0, out=ks2, ok=ok2)
        assert np.array_equal(host(pt2), want_pt[c0 * chain:(c0 + m) * chain])
        got = host(ok2)
        assert np.array_equal(got[c0:c0 + m], want_ok[c0:c0 + m])
        assert got[0] == 7 and got[n - 1] == 7                # chains outside the run untouched


@pytest.mark.parametrize("mode,depth", [(1, 2), (1, 3), (2, 2), (2, 3), (0, 0), (0, 2)])
def test_pipeline_modes_small(F, mode, depth):
    import torch
    say("pipeline mode", mode, "depth", depth)
    chain, chunk = 64 * KiB, 1 * MiB
    length = 24 * MiB + 3 * chain + 100
    w = W.random_case(60 + 4 * mode + depth, length, chain, 32)
    aad = W.case_aad(w, chain)
    ct, tags = oracle.chains_encrypt(w.key, w.base_iv, chain, w.payload, aad, 32)
    W.flip_bit(ct[7 * chain:], 9)
    W.flip_bit(tags[300], 3)
    want_pt, want_ok = oracle.chains_decrypt(w.key, w.base_iv, chain, ct, tags, aad, 32)
    h_ct = torch.from_numpy(ct).pin_memory()
    cs, ks, vs = torch.cuda.Stream(), torch.cuda.Stream(), torch.cuda.Stream()
    pt, ok = F.pipeline_h2d(w.key, w.base_iv, chain, h_ct, torch.from_numpy(tags), torch.from_numpy(aad),
                            chunk_bytes=chunk, depth=depth, copy_stream=cs, compute_stream=ks, mode=mode,
                            verify_stream=vs)
    ks.synchronize()
    vs.synchronize()
    assert np.array_equal(host(pt), want_pt)
    assert np.array_equal(host(ok), want_ok)


@pytest.mark.parametrize("length,chain,chunk,abytes,inplace", [
    (24 * MiB + 3 * 64 * KiB + 100, 64 * KiB, 1 * MiB, 32, False),
    (5 * MiB + 16, 256 * KiB, 2 * MiB, 0, True),
    (40 * 4096 + 5, 4096, 4 * 4096, 13, False),
])
def test_pipeline_d2h_matches_oracle(F, length, chain, chunk, abytes, inplace):
    import torch
    say("d2h", length, chain, chunk, abytes, inplace)
    w = W.random_case(length % 977 + abytes, length, chain, abytes)
    aad = W.case_aad(w, chain)
    want_ct, want_tags = oracle.chains_encrypt(w.key, w.base_iv, chain, w.payload, aad, abytes)
    cs, ks = torch.cuda.Stream(), torch.cuda.Stream()
    d_pt = dev(w.payload)
    h_ct, h_tags = F.pipeline_d2h(w.key, w.base_iv, chain, d_pt, dev(aad) if abytes else None, chunk_bytes=chunk,
                                  out=d_pt if inplace else None, copy_stream=cs, compute_stream=ks)
    cs.synchronize()
    assert np.array_equal(h_tags.numpy(), want_tags)
    assert np.array_equal(h_ct.numpy()[:length], want_ct)


def test_pipeline_d2h_gradients_256mib(F):
    """The fp32-gradients workload (256 MiB, 256 KiB chains) leaving the GPU in 8 MiB chunks."""
    import torch
    say("d2h gradients generate")
    w = W.config4()
    chain = w.chain_sizes[0]
    say("d2h gradients oracle encrypt")
    want_ct, want_tags = oracle.chains_encrypt(w.key, w.base_iv, chain, w.payload)
    cs, ks = torch.cuda.Stream(), torch.cuda.Stream()
    say("d2h gradients GPU")
    h_ct, h_tags = F.pipeline_d2h(w.key, w.base_iv, chain, dev(w.payload), chunk_bytes=8 * MiB, copy_stream=cs,
                                  compute_stream=ks)
    cs.synchronize()
    assert np.array_equal(h_tags.numpy(), want_tags)
    assert np.array_equal(h_ct.numpy(), want_ct)
