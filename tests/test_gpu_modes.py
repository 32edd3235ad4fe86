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
             (8 * MiB + 48, 1 * MiB, 2), (5, 16, 7),
             # a chain one block past a 2048-block pass, a ragged last chain, one short chain
             (3 * 32784 + 4099, 32784, 1), (32768 * 2 + 33, 32768, 0), (100, 96, 2)]


@pytest.mark.parametrize("bitsliced", [False, True], ids=["ttable", "bitsliced"])
@pytest.mark.parametrize("length,chain,base", KS_SHAPES)
def test_keystream_is_the_ciphertext_of_zeros(F, length, chain, base, bitsliced):
    say("keystream", length, chain, base, "bitsliced" if bitsliced else "ttable")
    w = W.random_case(length % 991 + base, 16, 16, 0)        # key and IV only
    total = base * chain + length
    zeros = np.zeros(total, np.uint8)
    ct_zero, _ = oracle.chains_encrypt(w.key, w.base_iv, chain, zeros)
    ks = F.keystream(w.key, w.base_iv, chain, length, chain_base=base, bitsliced=bitsliced)
    assert np.array_equal(host(ks), ct_zero[base * chain:])


def test_bitsliced_keystream_far_chain_index(F):
    """Chain indices above 2^32 reach the upper IV word: each chain is the oracle's
    GCM encryption of zeros under its own IV_i."""
    say("bitsliced keystream, chain base 2^32 + 3")
    w = W.random_case(77, 16, 16, 0)
    chain, base = 40960, (1 << 32) + 3
    ks = host(F.keystream(w.key, w.base_iv, chain, 2 * chain, chain_base=base, bitsliced=True))
    for j in range(2):
        want, _ = oracle.gcm_encrypt(w.key, oracle.chain_iv(w.base_iv, base + j), bytes(chain))
        assert np.array_equal(ks[j * chain:(j + 1) * chain], np.frombuffer(bytes(want), np.uint8))


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


# Launches of whole chains (no segments) with 16-, 32- and 64-lane items: the verify and
# keystream-apply kernels then queue their loads four (apply: two) iterations ahead. The
# last chain ends in a partial block; 32-byte AAD puts AAD blocks in the first iterations.
WHOLE_SHAPES = [(16384 * 4096 - 9, 4096), (8192 * 8192 - 3, 8192), (4096 * 16384 - 15, 16384)]


@pytest.mark.parametrize("length,chain", WHOLE_SHAPES)
def test_verify_and_apply_whole_chains(F, length, chain):
    import torch
    say("whole-chain verify/apply", length, chain)
    w, aad, ct, tags, want_pt, want_ok = tampered_case(chain + 3, length, chain, 32)
    n = tags.shape[0]
    W.flip_bit(ct, 8 * (length - 2))                          # the last chain's partial block
    W.flip_bit(ct, 8 * (chain * (n // 2) + 16 * 7) + 3)       # a block in a middle chain
    want_pt, want_ok = oracle.chains_decrypt(w.key, w.base_iv, chain, ct, tags, aad, 32)
    assert (want_ok == 0).sum() >= 4
    d_ct, d_tags, d_aad = dev(ct), dev(tags), dev(aad)
    e = F.decrypt_eager(w.key, w.base_iv, chain, d_ct, d_tags, d_aad)
    torch.cuda.synchronize()
    assert np.array_equal(e.plaintext.cpu().numpy(), want_pt)
    assert e.rejected() == np.nonzero(want_ok == 0)[0].tolist()
    ks = F.keystream(w.key, w.base_iv, chain, length)
    pt, ok = F.apply_verify(w.key, w.base_iv, chain, d_ct, ks, d_tags, d_aad)
    assert np.array_equal(host(pt), want_pt)
    assert np.array_equal(host(ok), want_ok)


@pytest.mark.parametrize("mode,depth", [(1, 2), (1, 3), (1, 8), (2, 2), (2, 3), (0, 0), (0, 2), (0, 8), (3, 0)])
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


@pytest.mark.parametrize("length,chain,chunk,abytes,inplace,mode", [
    (24 * MiB + 3 * 64 * KiB + 100, 64 * KiB, 1 * MiB, 32, False, 0),
    (5 * MiB + 16, 256 * KiB, 2 * MiB, 0, True, 0),
    (40 * 4096 + 5, 4096, 4 * 4096, 13, False, 0),
    (24 * MiB + 3 * 64 * KiB + 100, 64 * KiB, 1 * MiB, 32, False, 3),
    (40 * 4096 + 5, 4096, 4 * 4096, 13, False, 3),
])
def test_pipeline_d2h_matches_oracle(F, length, chain, chunk, abytes, inplace, mode):
    import torch
    say("d2h", length, chain, chunk, abytes, inplace, "mode", mode)
    w = W.random_case(length % 977 + abytes, length, chain, abytes)
    aad = W.case_aad(w, chain)
    want_ct, want_tags = oracle.chains_encrypt(w.key, w.base_iv, chain, w.payload, aad, abytes)
    cs, ks = torch.cuda.Stream(), torch.cuda.Stream()
    d_pt = dev(w.payload)
    h_ct, h_tags = F.pipeline_d2h(w.key, w.base_iv, chain, d_pt, dev(aad) if abytes else None, chunk_bytes=chunk,
                                  out=d_pt if inplace else None, copy_stream=cs, compute_stream=ks, mode=mode)
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


def test_direct_modes_inside_a_larger_pinned_buffer(F):
    # h_ct is a 16-byte-aligned view inside a larger pinned allocation: the kernel
    # reads (H2D) or writes (D2H) exactly its bytes through the device mapping and
    # leaves the guard bytes on both sides alone.
    import torch
    chain, length, front, back = 64 * KiB, 3 * MiB + 5 * 16 + 7, 4096 + 48, 4096
    say("direct modes in a larger pinned buffer")
    w = W.random_case(77, length, chain, 32)
    aad = W.case_aad(w, chain)
    ct, tags = oracle.chains_encrypt(w.key, w.base_iv, chain, w.payload, aad, 32)
    W.flip_bit(ct[2 * chain:], 5)
    want_pt, want_ok = oracle.chains_decrypt(w.key, w.base_iv, chain, ct, tags, aad, 32)
    big = torch.full((front + length + back,), 0xA5, dtype=torch.uint8).pin_memory()
    big[front:front + length].copy_(torch.from_numpy(ct))
    cs, ks = torch.cuda.Stream(), torch.cuda.Stream()
    pt, ok = F.pipeline_h2d(w.key, w.base_iv, chain, big[front:front + length], torch.from_numpy(tags),
                            torch.from_numpy(aad), chunk_bytes=MiB, depth=0, copy_stream=cs, compute_stream=ks,
                            mode=F.PIPE_DIRECT)
    ks.synchronize()
    assert np.array_equal(host(pt), want_pt)
    assert np.array_equal(host(ok), want_ok)
    # D2H: encrypt the plaintext into the middle of a guarded pinned buffer
    want_ct, want_tags = oracle.chains_encrypt(w.key, w.base_iv, chain, w.payload, aad, 32)
    big.fill_(0x5A)
    h_tags = torch.empty((tags.shape[0], 16), dtype=torch.uint8).pin_memory()
    F.pipeline_d2h(w.key, w.base_iv, chain, dev(w.payload), dev(aad), chunk_bytes=MiB, h_ct=big[front:front + length],
                   h_tags=h_tags, copy_stream=cs, compute_stream=ks, mode=F.PIPE_DIRECT)
    cs.synchronize()
    b = big.numpy()
    assert np.array_equal(b[front:front + length], want_ct)
    assert np.array_equal(h_tags.numpy(), want_tags)
    assert (b[:front] == 0x5A).all() and (b[front + length:] == 0x5A).all()


def test_pipelines_reject_ranges_outside_one_pinned_allocation(F):
    # [h_ct, h_ct + len) must lie inside one pinned allocation. The check runs on the
    # host before any copy or launch: a range that runs 4 KiB past the end of a 1 MiB
    # pinned block (a power of two, so the allocator's block is exactly that) and a
    # pageable buffer are both rejected with ENOTPINNED, in both directions and modes.
    import ctypes
    import torch
    L = F.lib()
    chain, length = 64 * KiB, MiB
    h = torch.zeros(length, dtype=torch.uint8).pin_memory()
    pageable = torch.zeros(length, dtype=torch.uint8)
    tags = torch.zeros((16, 16), dtype=torch.uint8)
    d_pt = torch.empty(length, dtype=torch.uint8, device="cuda")
    d_ct = torch.empty(length, dtype=torch.uint8, device="cuda")
    d_tags = torch.empty((16, 16), dtype=torch.uint8, device="cuda")
    ok = torch.empty(16, dtype=torch.uint8, device="cuda")
    stage = torch.empty(F.stage_bytes(length, chain, 0, MiB, 0), dtype=torch.uint8, device="cuda")
    key, iv = (ctypes.c_uint8 * 32)(), (ctypes.c_uint8 * 12)()
    s = torch.cuda.current_stream().cuda_stream
    for what, ptr in (("overrun", h.data_ptr() + 4096), ("pageable", pageable.data_ptr())):
        for mode in (F.PIPE_FUSED, F.PIPE_DIRECT):
            say("reject", what, "mode", mode)
            rc = L.fastrack_pipeline_h2d_mode(key, iv, chain, ptr, length, tags.data_ptr(), None, 0, MiB, 0, mode,
                                              stage.data_ptr(), stage.numel(), d_pt.data_ptr(), ok.data_ptr(), s, s, s)
            assert rc == -3 and b"pinned" in L.fastrack_last_error(), (what, mode, rc)
            rc = L.fastrack_pipeline_d2h_mode(key, iv, chain, d_pt.data_ptr(), length, None, 0, MiB, d_ct.data_ptr(),
                                              d_tags.data_ptr(), ptr, tags.data_ptr(), s, s, mode)
            assert rc == -3 and b"pinned" in L.fastrack_last_error(), (what, mode, rc)
    torch.cuda.synchronize()


def test_internal_buffers_survive_reuse_while_side_streams_run(F):
    """The binding allocates the staging ring (H2D) and the device ciphertext and tags (D2H)
    itself and drops them on return, while the copy and compute streams still use them.
    New tensors of the same sizes, allocated and filled on the current stream right after
    the call and before any synchronisation, must not take their memory."""
    import torch
    say("internal buffers vs allocator reuse")
    chain, chunk, depth = 64 * KiB, 1 * MiB, 2
    length = 12 * MiB + 3 * chain + 100
    w = W.random_case(91, length, chain, 32)
    aad = W.case_aad(w, chain)
    ct, tags = oracle.chains_encrypt(w.key, w.base_iv, chain, w.payload, aad, 32)
    W.flip_bit(ct[5 * chain:], 17)
    want_pt, want_ok = oracle.chains_decrypt(w.key, w.base_iv, chain, ct, tags, aad, 32)
    h_ct = torch.from_numpy(ct).pin_memory()
    n = tags.shape[0]
    need = F.stage_bytes(length, chain, 32, chunk, depth)
    cs, ks = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    pt, ok = F.pipeline_h2d(w.key, w.base_iv, chain, h_ct, torch.from_numpy(tags), torch.from_numpy(aad),
                            chunk_bytes=chunk, depth=depth, copy_stream=cs, compute_stream=ks)
    junk = [torch.full((need,), 0xA5, dtype=torch.uint8, device="cuda") for _ in range(3)]
    junk += [torch.full((sz,), 0x5A, dtype=torch.uint8, device="cuda") for sz in (2 * MiB, MiB, 16 * n)]
    ks.synchronize()
    cs.synchronize()
    assert np.array_equal(host(pt), want_pt)
    assert np.array_equal(host(ok), want_ok)
    del junk
    # D2H: the device ciphertext and tags are the binding's own
    want_ct, want_tags = oracle.chains_encrypt(w.key, w.base_iv, chain, w.payload, aad, 32)
    d_pt, d_aad = dev(w.payload), dev(aad)
    torch.cuda.synchronize()
    h_out, h_tags = F.pipeline_d2h(w.key, w.base_iv, chain, d_pt, d_aad, chunk_bytes=chunk, copy_stream=cs,
                                   compute_stream=ks)
    junk = [torch.full((length,), 0xC3, dtype=torch.uint8, device="cuda") for _ in range(2)]
    junk += [torch.full((16 * n,), 0x3C, dtype=torch.uint8, device="cuda") for _ in range(2)]
    cs.synchronize()
    ks.synchronize()
    assert np.array_equal(h_tags.numpy(), want_tags)
    assert np.array_equal(h_out.numpy()[:length], want_ct)
