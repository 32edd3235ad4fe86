"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Every expected value comes from the oracle (tests/../oracle), never from the
GPU. AES-GCM is deterministic, so plaintext, ciphertext, tags and ok flags are
compared bit for bit. Sizes: small edge shapes that still span several
segments and a ragged tail, then each workload at its full size.
"""
import time

import numpy as np
import pytest

import oracle
import workloads as W

pytestmark = pytest.mark.gpu

KiB, MiB, GiB = W.KiB, W.MiB, W.GiB


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


def check_decrypt(F, key, iv, chain, ct, tags, aad, abytes, flags=0, inplace=False, label=""):
    want_pt, want_ok = oracle.chains_decrypt(key, iv, chain, ct, tags, aad, abytes)
    d_ct = dev(ct)
    out = d_ct if inplace else None
    pt, ok = F.decrypt_verify(key, iv, chain, d_ct, dev(tags), dev(aad) if abytes else None, out=out, flags=flags)
    got_pt, got_ok = host(pt), host(ok)
    assert np.array_equal(got_ok, want_ok), (label, np.nonzero(got_ok != want_ok)[0][:10])
    if not np.array_equal(got_pt, want_pt):
        bad = np.nonzero(got_pt != want_pt)[0]
        raise AssertionError("%s: plaintext differs at %d bytes, first at %d" % (label, bad.size, bad[0]))
    return want_ok


def check_encrypt(F, key, iv, chain, pt, aad, abytes, flags=0, inplace=False, label=""):
    want_ct, want_tags = oracle.chains_encrypt(key, iv, chain, pt, aad, abytes)
    d_pt = dev(pt)
    out = d_pt if inplace else None
    ct, tags = F.encrypt_tag(key, iv, chain, d_pt, dev(aad) if abytes else None, out=out, flags=flags)
    got_ct, got_tags = host(ct), host(tags)
    assert np.array_equal(got_tags, want_tags), (label, "tags differ")
    assert np.array_equal(got_ct, want_ct), (label, "ciphertext differs")


SMALL = [
    (16, 16, 0), (17, 16, 0), (1, 1024, 0), (15, 4096, 1), (4096, 4096, 0), (1000, 64, 1), (5000, 1024, 32),
    (65536 + 48, 4096, 0), (100000 + 5, 16384, 13), (1 << 20, 65536, 0), (3 * 65536 + 16, 65536, 32),
    ((1 << 20) + 7, 1 << 20, 0), (777777, 1 << 20, 32), (2 * MiB + 100, 256 * KiB, 16),
    # AAD longer than one iteration of lanes: GHASH-only iterations ahead of the data
    (3 * 4096 + 5, 4096, 1000), (3 * 65536 + 16, 65536, 2000), (2 * MiB + 100, 256 * KiB, 5003),
    (40, 16, 100),
    # many chains with 16 and 32 lanes each whose wave-items do not divide evenly over
    # the 4096 resident waves of a 256-CU GPU: the chains are cut into segments
    (16400 * 2048 + 100, 2048, 1), (9000 * 4096 - 7, 4096, 32),
]


@pytest.mark.parametrize("length,chain,abytes", SMALL)
def test_small_shapes(F, length, chain, abytes):
    say("small", length, chain, abytes)
    w = W.random_case(length % 1000 + chain % 97 + abytes, length, chain, abytes)
    aad = W.case_aad(w, chain)
    ct, tags = oracle.chains_encrypt(w.key, w.base_iv, chain, w.payload, aad, abytes)
    for flags in (0, F.F_SEQ_GHASH):
        for inplace in (False, True):
            lab = "len=%d chain=%d aad=%d flags=%d inplace=%d" % (length, chain, abytes, flags, inplace)
            ok = check_decrypt(F, w.key, w.base_iv, chain, ct, tags, aad, abytes, flags, inplace, lab)
            assert ok.all()
            check_encrypt(F, w.key, w.base_iv, chain, w.payload, aad, abytes, flags, inplace, lab)


# Launches that leave most waves idle cut chains into short segments (down to
# 128 blocks, at most 512 per chain): two-iteration segments of 64 KiB chains,
# 128-block segments of 1 MiB chains, with AAD, tails and tampering inside
# middle segments.
SEGMENTED = [(1 * MiB, 64 * KiB, 32), (2 * MiB, 1 * MiB, 32), (4 * MiB - 16, 1 * MiB, 1000),
             (3 * MiB + 5, 1 * MiB, 13), (512 * KiB + 48, 32 * KiB, 0)]


@pytest.mark.parametrize("length,chain,abytes", SEGMENTED)
def test_short_segments(F, length, chain, abytes):
    say("short segments", length, chain, abytes)
    w = W.random_case(length % 977 + abytes, length, chain, abytes)
    aad = W.case_aad(w, chain)
    ct, tags = oracle.chains_encrypt(w.key, w.base_iv, chain, w.payload, aad, abytes)
    lab = "len=%d chain=%d aad=%d" % (length, chain, abytes)
    assert check_decrypt(F, w.key, w.base_iv, chain, ct, tags, aad, abytes, label=lab).all()
    check_encrypt(F, w.key, w.base_iv, chain, w.payload, aad, abytes, label=lab)
    n = tags.shape[0]
    c2 = ct.copy()
    bad = sorted({0, n // 2, n - 1})
    for i in bad:   # one bit in the middle of the chain, far from its first and last segment
        lo = i * chain
        hi = min(length, lo + chain)
        W.flip_bit(c2[lo:], 8 * ((hi - lo) // 2) + 3)
    ok = check_decrypt(F, w.key, w.base_iv, chain, c2, tags, aad, abytes, label=lab + " tampered")
    assert [i for i in range(n) if not ok[i]] == bad


def test_long_single_chain(F):
    """One 256 MiB chain (plus a partial block): 4097 segments of 4096 blocks, so the
    segment weights H^((S-1-s) 2^12) use the squares H^(2^t) up to t = 24, which only
    chains of millions of blocks reach."""
    length, abytes = 256 * MiB + 48, 32
    say("long single chain", length)
    w = W.random_case(77, length, length, abytes)
    aad = W.case_aad(w, length)
    ct, tags = oracle.chains_encrypt(w.key, w.base_iv, length, w.payload, aad, abytes)
    lab = "one chain of %d bytes" % length
    assert check_decrypt(F, w.key, w.base_iv, length, ct, tags, aad, abytes, label=lab).all()
    check_encrypt(F, w.key, w.base_iv, length, w.payload, aad, abytes, label=lab)
    c2 = ct.copy()
    W.flip_bit(c2, 8 * (length // 3) + 5)
    pt, ok = F.decrypt_verify(w.key, w.base_iv, length, dev(c2), dev(tags), dev(aad))
    assert not bool(ok.cpu().numpy()[0]), "a flipped bit one third into the chain was accepted"


def test_tamper_positions(F):
    say("tamper positions")
    chain, length, abytes = 8192, 20 * 8192 + 40, 32
    w = W.random_case(3, length, chain, abytes)
    aad = W.case_aad(w, chain)
    ct, tags = oracle.chains_encrypt(w.key, w.base_iv, chain, w.payload, aad, abytes)
    n = tags.shape[0]
    c2, t2, a2 = ct.copy(), tags.copy(), aad.copy()
    W.flip_bit(c2, 0)                                   # first bit of chain 0
    W.flip_bit(c2[3 * chain:], 8 * chain - 1)           # last bit of chain 3
    W.flip_bit(c2[(n - 1) * chain:], 8 * 40 - 1)        # last bit of the short last chain
    W.flip_bit(t2[5], 77)                               # a tag bit
    W.flip_bit(a2[7], 200)                              # an AAD bit
    c2[9 * chain:10 * chain], c2[11 * chain:12 * chain] = ct[11 * chain:12 * chain], ct[9 * chain:10 * chain]
    t2[[9, 11]] = tags[[11, 9]]                         # swapped chains
    for flags in (0, F.F_SEQ_GHASH):
        ok = check_decrypt(F, w.key, w.base_iv, chain, c2, t2, a2, abytes, flags, label="tamper")
        assert [i for i in range(n) if not ok[i]] == [0, 3, 5, 7, 9, 11, n - 1]


def test_config1_uniform_1mib(F):
    w = W.config1()
    for chain in w.chain_sizes:
        say("config1 chain", chain)
        ct, tags = oracle.chains_encrypt(w.key, w.base_iv, chain, w.payload)
        for flags in (0, F.F_SEQ_GHASH):
            ok = check_decrypt(F, w.key, w.base_iv, chain, ct, tags, None, 0, flags, label="config1")
            assert ok.all() and ok.size == (16 if chain == 64 * KiB else 1)


def test_config2_image_batch_chain_sweep(F):
    w = W.config2()
    for chain in w.chain_sizes:
        say("config2 chain", chain)
        aad = w.aad(chain)
        ct, tags = oracle.chains_encrypt(w.key, w.base_iv, chain, w.payload, aad, 32)
        ok = check_decrypt(F, w.key, w.base_iv, chain, ct, tags, aad, 32, label="config2 %d" % chain)
        assert ok.all()


def test_config3_weights_1gib_tamper(F):
    say("config3 generate")
    w = W.config3()
    chain = w.chain_sizes[0]
    say("config3 oracle encrypt")
    ct, tags = oracle.chains_encrypt(w.key, w.base_iv, chain, w.payload)
    for c, b in zip(w.tamper_chains, w.tamper_bits):
        W.flip_bit(ct[c * chain:(c + 1) * chain], int(b))
    say("config3 GPU decrypt + oracle decrypt")
    ok = check_decrypt(F, w.key, w.base_iv, chain, ct, tags, None, 0, label="config3")
    assert sorted(np.nonzero(ok == 0)[0].tolist()) == w.tamper_chains.tolist()
    assert len(w.tamper_chains) == 10


def test_config4_gradients_encrypt(F):
    say("config4 generate")
    w = W.config4()
    chain = w.chain_sizes[0]
    say("config4 GPU encrypt + oracle encrypt")
    check_encrypt(F, w.key, w.base_iv, chain, w.payload, None, 0, label="config4")


def test_workgroup_tag_combine_edges(F):
    """64 KiB chains over 64 MiB - 16 KiB + 100 bytes: on 256 CUs the plan cuts the 1024
    chains into 4 segments each (the short last chain, 48 KiB + 100 bytes with a partial
    last block, also into 4), 4096 items for 4096 waves, so each chain is summed and tagged
    inside its workgroup. Tampering in a middle segment, in the last partial block, in a tag
    and in an AAD is rejected exactly; decrypt (also in place) and encrypt match the oracle."""
    chain, length, abytes = 64 * KiB, 64 * MiB - 16 * KiB + 100, 32
    say("workgroup tag combine edges")
    w = W.random_case(88, length, chain, abytes)
    aad = W.case_aad(w, chain)
    n = aad.shape[0]
    ct, tags = oracle.chains_encrypt(w.key, w.base_iv, chain, w.payload, aad, abytes)
    bad, tg, ad = ct.copy(), tags.copy(), aad.copy()
    W.flip_bit(bad, 8 * (5 * chain + 2 * 16 * KiB + 77))   # chain 5, segment 2
    W.flip_bit(bad, 8 * (length - 1) + 3)                  # the last chain's partial last block
    tg[700, 3] ^= 0x10
    ad[300, 0] ^= 1
    ok = check_decrypt(F, w.key, w.base_iv, chain, bad, tg, ad, abytes, label="workgroup decrypt")
    assert int(ok.sum()) == n - 4 and not ok[[5, 300, 700, n - 1]].any()
    check_decrypt(F, w.key, w.base_iv, chain, bad, tg, ad, abytes, inplace=True, label="workgroup decrypt in place")
    check_encrypt(F, w.key, w.base_iv, chain, w.payload, aad, abytes, label="workgroup encrypt")


@pytest.mark.parametrize("depth", [0, 2, 3])
def test_config5_pipeline_small(F, depth):
    """The pipeline on 64 MiB with a ragged last chunk and AAD, vs the oracle."""
    import torch
    say("pipeline small depth", depth)
    chain, chunk = 64 * KiB, 1 * MiB
    length = 64 * MiB + 3 * chain + 100
    w = W.random_case(50 + depth, length, chain, 32)
    aad = W.case_aad(w, chain)
    ct, tags = oracle.chains_encrypt(w.key, w.base_iv, chain, w.payload, aad, 32)
    W.flip_bit(ct[5 * chain:], 3)
    want_pt, want_ok = oracle.chains_decrypt(w.key, w.base_iv, chain, ct, tags, aad, 32)
    h_ct = torch.from_numpy(ct).pin_memory()
    copy_s = torch.cuda.Stream()
    comp_s = torch.cuda.Stream()
    pt, ok = F.pipeline_h2d(w.key, w.base_iv, chain, h_ct, torch.from_numpy(tags), torch.from_numpy(aad),
                            chunk_bytes=chunk, depth=depth, copy_stream=copy_s, compute_stream=comp_s)
    comp_s.synchronize()
    assert np.array_equal(host(ok), want_ok)
    assert np.array_equal(host(pt), want_pt)


@pytest.fixture(scope="module")
def config5_data():
    import torch
    say("config5 generate 4 GiB into pinned memory")
    length = 4 * GiB
    h_pt = torch.empty(length, dtype=torch.uint8, pin_memory=True)
    w = W.config5(length, out=h_pt.numpy())
    chain = w.chain_sizes[0]
    h_ct = torch.empty(length, dtype=torch.uint8, pin_memory=True)
    say("config5 oracle encrypt 4 GiB")
    _, tags = oracle.chains_encrypt(w.key, w.base_iv, chain, w.payload, out=h_ct.numpy())
    say("config5 oracle decrypt of the 64 sampled chains")
    want, want_ok = oracle.chains_decrypt_subset(w.key, w.base_iv, chain, h_ct.numpy(), tags, w.sample_chains)
    assert want_ok.all()
    yield w, h_pt, h_ct, tags, want
    del h_pt, h_ct


@pytest.mark.parametrize("mode,depth", [(0, 0), (0, 2), (0, 3), (1, 2), (2, 2), (3, 0)])
def test_config5_pipeline_4gib(F, config5_data, mode, depth):
    import torch
    w, h_pt, h_ct, tags, want = config5_data
    chain = w.chain_sizes[0]
    say("config5 pipeline mode", mode, "depth", depth)
    copy_s, comp_s, ver_s = torch.cuda.Stream(), torch.cuda.Stream(), torch.cuda.Stream()
    pt, ok = F.pipeline_h2d(w.key, w.base_iv, chain, h_ct, torch.from_numpy(tags), None,
                            chunk_bytes=w.extra["chunk_bytes"], depth=depth, copy_stream=copy_s,
                            compute_stream=comp_s, mode=mode, verify_stream=ver_s)
    comp_s.synchronize()
    ver_s.synchronize()
    assert host(ok).all()
    idx = torch.from_numpy(w.sample_chains).cuda()
    got = pt.view(-1, chain).index_select(0, idx)
    assert np.array_equal(host(got), want)
    # every byte equals the generated plaintext (the oracle round trip of its own encryption)
    assert torch.equal(pt, h_pt.cuda())
    del pt, ok
    torch.cuda.empty_cache()
