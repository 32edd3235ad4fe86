"""GPU parity of ragged chains (the paper's per-sample chaining) through the C ABI.

Every expected value comes from the oracle's ragged_encrypt / ragged_decrypt,
which run each chain as its own GCM message; comparisons are bit for bit.
Cases: hand-built layouts that exercise each lanes-per-item choice, chains
cut into segments next to short and empty chains, AAD longer than one
iteration, gaps between chains (left untouched), and the per-sample batch
workload with tampered and reordered chains.
"""
import time
import zlib

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


FILL = 0x5A


def check_ragged(F, w, label, inplace=False):
    off, ln = w.extra["chain_off"], w.extra["chain_len"]
    ab = w.aad_bytes
    aad = w.extra.get("aad")
    n = off.size
    say(label, "chains", n, "bytes", w.payload.size, "aad", ab)
    base = np.full(w.payload.size, FILL, np.uint8)
    want_ct, want_tags = oracle.ragged_encrypt(w.key, w.base_iv, off, ln, w.payload, aad, ab, out=base.copy())
    d_pt = dev(w.payload)
    ct, tags = F.encrypt_tag_ragged(w.key, w.base_iv, off, ln, d_pt, dev(aad) if ab else None, out=dev(base))
    got_ct, got_tags = host(ct), host(tags)
    assert np.array_equal(got_tags, want_tags), (label, "tags differ at chains",
                                                 np.nonzero((got_tags != want_tags).any(1))[0][:10])
    if not np.array_equal(got_ct, want_ct):
        bad = np.nonzero(got_ct != want_ct)[0]
        raise AssertionError("%s: ciphertext differs at %d bytes, first at %d" % (label, bad.size, bad[0]))
    # decrypt, with a few chains tampered (one flipped bit each)
    r = np.random.Generator(np.random.PCG64(len(label) * 7919 + n))
    c2 = want_ct.copy()
    nonempty = np.nonzero(ln > 0)[0]
    bad = np.sort(r.choice(nonempty, size=min(3, nonempty.size), replace=False)) if nonempty.size else []
    for i in bad:
        o, l = int(off[i]), int(ln[i])
        W.flip_bit(c2[o:o + l], int(r.integers(0, 8 * l)))
    want_pt, want_ok = oracle.ragged_decrypt(w.key, w.base_iv, off, ln, c2, want_tags, aad, ab, out=c2.copy()
                                             if inplace else base.copy())
    d_ct = dev(c2)
    pt, ok = F.decrypt_verify_ragged(w.key, w.base_iv, off, ln, d_ct, dev(want_tags), dev(aad) if ab else None,
                                     out=d_ct if inplace else dev(base))
    got_pt, got_ok = host(pt), host(ok)
    assert np.array_equal(got_ok, want_ok), (label, np.nonzero(got_ok != want_ok)[0][:10])
    assert sorted(np.nonzero(got_ok == 0)[0].tolist()) == sorted(int(i) for i in bad)
    if not np.array_equal(got_pt, want_pt):
        badb = np.nonzero(got_pt != want_pt)[0]
        raise AssertionError("%s: plaintext differs at %d bytes, first at %d" % (label, badb.size, badb[0]))


def lens_of(seed, n, lo, hi):
    r = np.random.Generator(np.random.PCG64(W.SEED_BASE + 3000 + seed))
    return r.integers(lo, hi + 1, n).tolist()


CASES = [
    # (label, chain lengths, gaps in blocks, aad bytes)
    ("tiny-mixed", [0, 1, 17, 4096, 15, 33, 1000, 16], [0, 2, 0, 1, 0, 3, 0, 0], 3),
    ("one-chain", [100000 + 7], None, 0),
    ("empty-chains-only", [0, 0, 0], [0, 1, 0], 32),
    ("empty-chains-no-aad", [0, 0], None, 0),
    ("long-aad", lens_of(1, 40, 0, 3000), None, 1000),
    ("lanes16-many", lens_of(2, 5000, 0, 3000), None, 1),
    ("lanes16-fill", lens_of(3, 9000, 1100, 1300), None, 0),
    ("lanes32", lens_of(4, 300, 2048, 4000), lens_of(5, 300, 0, 2), 32),
    ("lanes64-split", [3 * MiB + 5, MiB, 17, 0, 64 * KiB + 16], [0, 0, 1, 0, 0], 32),
    ("split-next-to-short", [2 * MiB] + lens_of(6, 100, 1000, 5000), None, 1),
    ("wave-pads-short", [16, 64 * KiB, 16, 48, 64 * KiB + 1, 0, 256, 4096] * 8, None, 0),
    # short chains only (at most 64 blocks): whole chains, tagged in the streaming kernel
    ("whole-chains", lens_of(9, 20000, 200, 1024), None, 1),
]


@pytest.mark.parametrize("label,lens,gaps,ab", CASES, ids=[c[0] for c in CASES])
def test_ragged_parity(F, label, lens, gaps, ab):
    w = W.ragged_case(zlib.crc32(label.encode()) & 0xFFFF, lens, gaps, ab)
    check_ragged(F, w, label)


def test_ragged_in_place(F):
    w = W.ragged_case(77, lens_of(7, 200, 0, 9000), lens_of(8, 200, 0, 1), 16)
    check_ragged(F, w, "in-place", inplace=True)


def test_ragged_matches_uniform_layout(F):
    """Offsets i * chain_bytes: the ragged and the uniform entry points agree with each other and the oracle."""
    w = W.random_case(90, 40 * 4096 + 100, 4096, 32)
    chain = 4096
    n = W.n_chains(w.payload.size, chain)
    off = np.arange(n, dtype=np.uint64) * chain
    ln = np.minimum(chain, w.payload.size - off.astype(np.int64)).astype(np.uint64)
    aad = w.extra["aad"]
    ct_u, tags_u = F.encrypt_tag(w.key, w.base_iv, chain, dev(w.payload), dev(aad))
    ct_r, tags_r = F.encrypt_tag_ragged(w.key, w.base_iv, off, ln, dev(w.payload), dev(aad))
    want_ct, want_tags = oracle.chains_encrypt(w.key, w.base_iv, chain, w.payload, aad, 32)
    assert np.array_equal(host(tags_u), want_tags) and np.array_equal(host(tags_r), want_tags)
    assert np.array_equal(host(ct_u), want_ct) and np.array_equal(host(ct_r), want_ct)


def sample_layout(F, w):
    off, ln, total = F.sample_chains(w.extra["sample_lens"], w.extra["chains_per_sample"])
    assert total == w.payload.size
    return off, ln


@pytest.mark.parametrize("n_samples,k", [(256, 16), (64, 8), (33, 13)])
def test_sample_batch_parity(F, n_samples, k):
    w = W.sample_batch(n_samples=n_samples, chains_per_sample=k)
    off, ln = sample_layout(F, w)
    # the layout helper: every sample is covered exactly by its k chains
    so, sl = w.extra["sample_off"], w.extra["sample_lens"]
    for s in range(n_samples):
        o, l = off[s * k:(s + 1) * k], ln[s * k:(s + 1) * k]
        assert int(o[0]) == int(so[s]) and int(l.sum()) == int(sl[s])
        assert np.all(o[1:] == o[:-1] + l[:-1])
    w.extra["chain_off"], w.extra["chain_len"] = off, ln
    check_ragged(F, w, "samples-%dx%d" % (n_samples, k))


def test_sample_batch_reorder_is_rejected(F):
    """Section 5.4: chains swapped within a sample fail through the serial-number AAD."""
    w = W.sample_batch(n_samples=16, chains_per_sample=16)
    off, ln = sample_layout(F, w)
    aad = w.extra["aad"]
    ct, tags = oracle.ragged_encrypt(w.key, w.base_iv, off, ln, w.payload, aad, 1)
    a2 = aad.copy()
    a2[[3 * 16 + 4, 3 * 16 + 9]] = aad[[3 * 16 + 9, 3 * 16 + 4]]
    _, want_ok = oracle.ragged_decrypt(w.key, w.base_iv, off, ln, ct, tags, a2, 1)
    _, ok = F.decrypt_verify_ragged(w.key, w.base_iv, off, ln, dev(ct), dev(tags), dev(a2))
    got = host(ok)
    assert np.array_equal(got, want_ok)
    assert sorted(np.nonzero(got == 0)[0].tolist()) == [3 * 16 + 4, 3 * 16 + 9]


def test_sample_batch_full_size(F):
    """The per-sample workload at its bench size (1024 samples x 16 chains, about 131 MiB): 512 sampled
    chains against the oracle one by one; every chain round-trips and exactly the tampered ones fail."""
    w = W.sample_batch(n_samples=1024, chains_per_sample=16)
    off, ln = sample_layout(F, w)
    aad = w.extra["aad"]
    n = off.size
    say("samples-1024x16 encrypt")
    ct, tags = F.encrypt_tag_ragged(w.key, w.base_iv, off, ln, dev(w.payload), dev(aad))
    got_ct, got_tags = host(ct), host(tags)
    r = np.random.Generator(np.random.PCG64(W.SEED_BASE + 4000))
    pick = np.sort(r.choice(n, size=512, replace=False))
    for i in pick.tolist():
        o, l = int(off[i]), int(ln[i])
        c, t = oracle.gcm_encrypt(w.key, oracle.chain_iv(w.base_iv, i), w.payload[o:o + l], aad[i])
        assert np.array_equal(got_ct[o:o + l], c) and np.array_equal(got_tags[i], t), i
    bad = np.sort(r.choice(np.nonzero(ln > 0)[0], size=20, replace=False))
    for i in bad.tolist():
        o, l = int(off[i]), int(ln[i])
        W.flip_bit(got_ct[o:o + l], int(r.integers(0, 8 * l)))
    say("samples-1024x16 decrypt")
    pt, ok = F.decrypt_verify_ragged(w.key, w.base_iv, off, ln, dev(got_ct), tags, dev(aad))
    got_pt, got_ok = host(pt), host(ok)
    assert np.nonzero(got_ok == 0)[0].tolist() == bad.tolist()
    good = np.zeros(w.payload.size, bool)     # the bytes of untampered chains (gaps are not written)
    for i in range(n):
        good[int(off[i]):int(off[i] + ln[i])] = True
    for i in bad.tolist():
        good[int(off[i]):int(off[i] + ln[i])] = False
    assert np.array_equal(got_pt[good], w.payload[good])
    for i in bad.tolist():     # a tampered chain still decrypts (one flipped bit), as in the oracle
        o, l = int(off[i]), int(ln[i])
        want, ok_i = oracle.gcm_decrypt(w.key, oracle.chain_iv(w.base_iv, i), got_ct[o:o + l], got_tags[i], aad[i])
        assert not ok_i and np.array_equal(got_pt[o:o + l], want)
