"""Pins of the CPU oracle against things other than itself.

Each test checks the oracle against the system crypto library (a library
routine its special cases reduce to), a closed form, an algebraic invariant,
brute force on tiny inputs, or a fact the paper states (tests/golden/). A
plausible mistake (a dropped term, a wrong sign, index or bit order, a
transposed operand) fails at least one of them.
"""
import json
import os

import numpy as np
import pytest

import libcrypto_ref as LC
import oracle
import workloads as W

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
needs_libcrypto = pytest.mark.skipif(not LC.available(), reason="system libcrypto not present")


def rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


def rbytes(r, n):
    return np.frombuffer(r.bytes(n), np.uint8).copy()


# --------------------------------------------------------------------------
# AES-256 (FIPS-197)
# --------------------------------------------------------------------------

def test_sbox_invariants():
    s, inv = oracle.sbox()
    assert sorted(s.tolist()) == list(range(256)), "S-box must be a permutation"
    assert s[0] == 0x63, "inv(0) = 0, so S(0) is the affine constant"
    x = np.arange(256, dtype=np.uint8)
    assert not np.any(s == x), "the AES S-box has no fixed points"
    assert not np.any(s == (x ^ 0xFF)), "nor opposite fixed points"
    assert np.array_equal(inv[s], x)


def test_sbox_is_affine_image_of_inverse():
    """Brute force: S(x) xor 0x63 is GF(2)-linear in inv(x), i.e. A(u xor v) = A(u) xor A(v)."""
    s, inv_s = oracle.sbox()

    def gmul(a, b):  # schoolbook carry-less product reduced by x^8+x^4+x^3+x+1
        p = 0
        for i in range(8):
            if (b >> i) & 1:
                p ^= a << i
        for d in range(14, 7, -1):
            if (p >> d) & 1:
                p ^= 0x11B << (d - 8)
        return p

    inv = [0] * 256
    for a in range(1, 256):
        for b in range(1, 256):
            if gmul(a, b) == 1:
                inv[a] = b
                break
    lin = {inv[x]: int(s[x]) ^ 0x63 for x in range(256)}
    for u in range(256):
        for v in (1, 2, 4, 8, 16, 32, 64, 128):
            assert lin[u ^ v] == lin[u] ^ lin[v]


def test_key_expansion_structure():
    r = rng(11)
    key = rbytes(r, 32)
    w = oracle.key_expansion(key).astype(np.int64)
    assert np.array_equal(w[:8].reshape(-1), key)
    for i in range(8, 60):
        if i % 8 not in (0, 4):
            # words without SubWord/RotWord are the plain XOR of w[i-8] and w[i-1]
            assert np.array_equal(w[i], w[i - 8] ^ w[i - 1])


@needs_libcrypto
def test_aes256_vs_libcrypto():
    r = rng(12)
    for _ in range(200):
        key, blk = rbytes(r, 32), rbytes(r, 16)
        assert bytes(oracle.aes256_encrypt_block(key, blk)) == LC.aes256_ecb_encrypt(key, blk)


def test_inv_cipher_roundtrip():
    r = rng(13)
    for _ in range(50):
        key, blk = rbytes(r, 32), rbytes(r, 16)
        c = oracle.aes256_encrypt_block(key, blk)
        assert np.array_equal(oracle.aes256_decrypt_block(key, c), blk)


# --------------------------------------------------------------------------
# GF(2^128) (SP 800-38D 6.3)
# --------------------------------------------------------------------------

ONE = np.array([0x80] + [0] * 15, np.uint8)


def unit(i):
    b = np.zeros(16, np.uint8)
    b[i // 8] = 0x80 >> (i % 8)
    return b


def poly_int(b):
    """Block -> integer whose bit i is the coefficient of x^i (bit 0 = MSB of byte 0)."""
    v = 0
    for i in range(128):
        if (b[i // 8] >> (7 - i % 8)) & 1:
            v |= 1 << i
    return v


def poly_block(v):
    b = np.zeros(16, np.uint8)
    for i in range(128):
        if (v >> i) & 1:
            b[i // 8] |= 0x80 >> (i % 8)
    return b


def poly_mul_textbook(x, y):
    """Carry-less polynomial product reduced modulo x^128 + x^7 + x^2 + x + 1."""
    a, b = poly_int(x), poly_int(y)
    p = 0
    while b:
        if b & 1:
            p ^= a
        a <<= 1
        b >>= 1
    mod = (1 << 128) | 0x87
    for d in range(254, 127, -1):
        if (p >> d) & 1:
            p ^= mod << (d - 128)
    return poly_block(p)


def test_gf128_identity_and_reduction_closed_form():
    r = rng(21)
    for _ in range(20):
        y = rbytes(r, 16)
        assert np.array_equal(oracle.gf128_mul_bitserial(ONE, y), y)
        assert np.array_equal(oracle.gf128_mul_bitserial(y, ONE), y)
    # x^127 . x = x^128 = x^7 + x^2 + x + 1 = R
    got = oracle.gf128_mul_bitserial(unit(127), unit(1))
    assert bytes(got) == bytes([0xE1] + [0] * 15)


def test_gf128_matches_textbook_polynomial_product():
    r = rng(22)
    for _ in range(60):
        x, y = rbytes(r, 16), rbytes(r, 16)
        assert np.array_equal(oracle.gf128_mul_bitserial(x, y), poly_mul_textbook(x, y))


def test_gf128_field_laws():
    r = rng(23)
    m = oracle.gf128_mul_bitserial
    for _ in range(30):
        a, b, c = rbytes(r, 16), rbytes(r, 16), rbytes(r, 16)
        assert np.array_equal(m(a, b), m(b, a))
        assert np.array_equal(m(m(a, b), c), m(a, m(b, c)))
        assert np.array_equal(m(a, b ^ c), m(a, b) ^ m(a, c))


def test_gf128_table_equals_bitserial():
    r = rng(24)
    for _ in range(4):
        y = rbytes(r, 16)
        for i in range(128):
            assert np.array_equal(oracle.gf128_mul_table(unit(i), y), oracle.gf128_mul_bitserial(unit(i), y))
    for _ in range(2000):
        x, y = rbytes(r, 16), rbytes(r, 16)
        assert np.array_equal(oracle.gf128_mul_table(x, y), oracle.gf128_mul_bitserial(x, y))


# --------------------------------------------------------------------------
# GHASH (SP 800-38D 6.4)
# --------------------------------------------------------------------------

def gpow(h, e):
    out = ONE.copy()
    for _ in range(e):
        out = poly_mul_textbook(out, h)
    return out


def test_ghash_horner_equals_closed_form():
    r = rng(31)
    for m in range(1, 9):
        h = rbytes(r, 16)
        xs = rbytes(r, 16 * m)
        want = np.zeros(16, np.uint8)
        for j in range(1, m + 1):  # sum X_j . H^(m-j+1)
            want ^= poly_mul_textbook(xs[16 * (j - 1):16 * j], gpow(h, m - j + 1))
        for bitserial in (True, False):
            assert np.array_equal(oracle.ghash(h, xs, bitserial), want)


def test_ghash_linearity_and_zero_prefix():
    r = rng(32)
    for m in (1, 3, 17, 64):
        h = rbytes(r, 16)
        x1, x2 = rbytes(r, 16 * m), rbytes(r, 16 * m)
        assert np.array_equal(oracle.ghash(h, x1 ^ x2, False), oracle.ghash(h, x1, False) ^ oracle.ghash(h, x2, False))
        padded = np.concatenate([np.zeros(16 * 5, np.uint8), x1])
        assert np.array_equal(oracle.ghash(h, padded, False), oracle.ghash(h, x1, False))


def test_ghash_split_identity():
    """GHASH(A || C || L) = (GHASH(A) . H^q  xor  GHASH(C)  xor  L) . H, q = number of C blocks."""
    r = rng(33)
    for a, q in ((1, 1), (2, 5), (3, 16)):
        h = rbytes(r, 16)
        A, C, L = rbytes(r, 16 * a), rbytes(r, 16 * q), rbytes(r, 16)
        whole = oracle.ghash(h, np.concatenate([A, C, L]), True)
        inner = poly_mul_textbook(oracle.ghash(h, A, True), gpow(h, q)) ^ oracle.ghash(h, C, True) ^ L
        assert np.array_equal(whole, poly_mul_textbook(inner, h))


# --------------------------------------------------------------------------
# GCTR (SP 800-38D 6.5)
# --------------------------------------------------------------------------

def test_gctr_malleability_and_roundtrip():
    r = rng(41)
    key, icb = rbytes(r, 32), rbytes(r, 16)
    pt = rbytes(r, 100)
    ct = oracle.gctr(key, icb, pt)
    assert np.array_equal(oracle.gctr(key, icb, ct), pt)
    for bit in (0, 7, 8, 333, 799):
        c2 = ct.copy()
        W.flip_bit(c2, bit)
        p2 = oracle.gctr(key, icb, c2)
        diff = np.unpackbits(p2 ^ pt)
        assert diff.sum() == 1 and diff[bit] == 1


def test_gctr_inc32_wraps_low_word_only():
    r = rng(42)
    key = rbytes(r, 32)
    icb = rbytes(r, 16)
    icb[12:] = 0xFF  # low 32 bits = 2^32 - 1
    ks = oracle.gctr(key, icb, np.zeros(32, np.uint8))
    second = icb.copy()
    second[12:] = 0  # inc32 wraps to 0 and leaves the upper 96 bits alone
    assert np.array_equal(ks[:16], oracle.aes256_encrypt_block(key, icb))
    assert np.array_equal(ks[16:], oracle.aes256_encrypt_block(key, second))


def test_gctr_partial_block_uses_keystream_msb():
    r = rng(43)
    key, icb = rbytes(r, 32), rbytes(r, 16)
    full = oracle.gctr(key, icb, np.zeros(48, np.uint8))
    for n in (1, 5, 15, 17, 31, 33, 47):
        assert np.array_equal(oracle.gctr(key, icb, np.zeros(n, np.uint8)), full[:n])


# --------------------------------------------------------------------------
# GCM (SP 800-38D 7.1 / 7.2)
# --------------------------------------------------------------------------

@needs_libcrypto
@pytest.mark.parametrize("length", [0, 1, 15, 16, 17, 4095, 4096, 65536])
@pytest.mark.parametrize("alen", [0, 1, 32])
def test_gcm_vs_libcrypto(length, alen):
    r = rng(1000 + length + alen)
    key, iv = rbytes(r, 32), rbytes(r, 12)
    pt, aad = rbytes(r, length), rbytes(r, alen)
    want_ct, want_tag = LC.gcm_encrypt(key, iv, pt, aad)
    modes = (False, True) if length <= 4096 else (False,)
    for bitserial in modes:
        ct, tag = oracle.gcm_encrypt(key, iv, pt, aad, bitserial=bitserial)
        assert bytes(ct) == want_ct and bytes(tag) == want_tag
        back, ok = oracle.gcm_decrypt(key, iv, ct, tag, aad, bitserial=bitserial)
        assert ok and np.array_equal(back, pt)


def test_gcm_rejects_every_single_bit_flip():
    r = rng(51)
    key, iv = rbytes(r, 32), rbytes(r, 12)
    pt, aad = rbytes(r, 64), rbytes(r, 16)
    ct, tag = oracle.gcm_encrypt(key, iv, pt, aad)
    for field_name, buf in (("ct", ct), ("tag", tag), ("aad", aad)):
        for bit in range(8 * buf.size):
            b = buf.copy()
            W.flip_bit(b, bit)
            args = {"ct": ct, "tag": tag, "aad": aad}
            args[field_name] = b
            p, ok = oracle.gcm_decrypt(key, iv, args["ct"], args["tag"], args["aad"])
            assert not ok, (field_name, bit)
            if field_name == "ct":  # plaintext is still produced, differing in exactly that bit
                assert np.unpackbits(p ^ pt).sum() == 1


# --------------------------------------------------------------------------
# Multi-chaining (paper section 5.2)
# --------------------------------------------------------------------------

@needs_libcrypto
@pytest.mark.parametrize("length,chain,alen", [(4096, 1024, 0), (5000, 1024, 32), (1000, 16, 1), (16 * 1024 + 7, 4096, 32),
                                               (65536, 65536, 0), (70000, 1 << 20, 0), (1, 16, 0)])
def test_each_chain_is_standard_gcm(length, chain, alen):
    r = rng(2000 + length)
    key, base_iv = rbytes(r, 32), rbytes(r, 12)
    pt = rbytes(r, length)
    n = W.n_chains(length, chain)
    aad = rbytes(r, n * alen).reshape(n, alen) if alen else None
    ct, tags = oracle.chains_encrypt(key, base_iv, chain, pt, aad, alen)
    assert tags.shape == (n, 16)
    for i in range(n):
        iv = bytearray(bytes(base_iv))
        for k in range(8):  # chain index, big-endian, into IV bytes 4..11
            iv[4 + k] ^= (i >> (8 * (7 - k))) & 0xFF
        assert bytes(oracle.chain_iv(base_iv, i)) == bytes(iv)
        seg = pt[i * chain:(i + 1) * chain]
        c, t = LC.gcm_encrypt(key, bytes(iv), seg, aad[i] if alen else b"")
        assert bytes(ct[i * chain:i * chain + seg.size]) == c and bytes(tags[i]) == t
    back, ok = oracle.chains_decrypt(key, base_iv, chain, ct, tags, aad, alen)
    assert ok.all() and np.array_equal(back, pt)


@needs_libcrypto
def test_single_chain_is_plain_gcm_under_base_iv():
    r = rng(61)
    key, base_iv = rbytes(r, 32), rbytes(r, 12)
    pt = rbytes(r, 3000)
    ct, tags = oracle.chains_encrypt(key, base_iv, 1 << 20, pt)
    c, t = LC.gcm_encrypt(key, base_iv, pt)
    assert bytes(ct) == c and bytes(tags[0]) == t


def test_bitserial_and_table_chains_agree():
    r = rng(62)
    key, base_iv = rbytes(r, 32), rbytes(r, 12)
    pt = rbytes(r, 2000)
    a = oracle.chains_encrypt(key, base_iv, 256, pt, bitserial=False)
    b = oracle.chains_encrypt(key, base_iv, 256, pt, bitserial=True)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def test_thread_count_does_not_change_results():
    r = rng(63)
    key, base_iv = rbytes(r, 32), rbytes(r, 12)
    pt = rbytes(r, 1 << 18)
    one = oracle.chains_encrypt(key, base_iv, 4096, pt, nthreads=1)
    many = oracle.chains_encrypt(key, base_iv, 4096, pt, nthreads=4)
    assert np.array_equal(one[0], many[0]) and np.array_equal(one[1], many[1])


def test_reordered_or_duplicated_chains_are_rejected():
    """Section 5.4 (reorder attacks): chains moved to another position must fail."""
    r = rng(64)
    key, base_iv = rbytes(r, 32), rbytes(r, 12)
    chain = 512
    pt = rbytes(r, 8 * chain)
    aad = W.serial_byte_aad(pt.size, chain)
    ct, tags = oracle.chains_encrypt(key, base_iv, chain, pt, aad, 1)
    c2, t2 = ct.copy(), tags.copy()
    c2[2 * chain:3 * chain], c2[5 * chain:6 * chain] = ct[5 * chain:6 * chain], ct[2 * chain:3 * chain]
    t2[[2, 5]] = tags[[5, 2]]
    _, ok = oracle.chains_decrypt(key, base_iv, chain, c2, t2, aad, 1)
    assert ok.tolist() == [1, 1, 0, 1, 1, 0, 1, 1]
    c3, t3 = ct.copy(), tags.copy()
    c3[3 * chain:4 * chain] = ct[1 * chain:2 * chain]
    t3[3] = tags[1]
    _, ok = oracle.chains_decrypt(key, base_iv, chain, c3, t3, aad, 1)
    assert ok.tolist() == [1, 1, 1, 0, 1, 1, 1, 1]
    # swapping only the AAD serial numbers is caught as well
    a4 = aad.copy()
    a4[[0, 7]] = aad[[7, 0]]
    _, ok = oracle.chains_decrypt(key, base_iv, chain, ct, tags, a4, 1)
    assert ok.tolist() == [0, 1, 1, 1, 1, 1, 1, 0]


def test_tamper_is_exact_per_chain():
    r = rng(65)
    key, base_iv = rbytes(r, 32), rbytes(r, 12)
    chain = 1024
    pt = rbytes(r, 40 * chain + 100)
    ct, tags = oracle.chains_encrypt(key, base_iv, chain, pt)
    n = tags.shape[0]
    bad = sorted(r.choice(n, size=6, replace=False).tolist())
    c2 = ct.copy()
    for i in bad:
        lo = i * chain
        hi = min(ct.size, lo + chain)
        W.flip_bit(c2[lo:hi], int(r.integers(0, 8 * (hi - lo))))
    p2, ok = oracle.chains_decrypt(key, base_iv, chain, c2, tags)
    assert [i for i in range(n) if not ok[i]] == bad
    assert np.unpackbits(p2 ^ pt).sum() == len(bad)


@needs_libcrypto
@pytest.mark.parametrize("bitserial", [False, True])
def test_decrypt_subset_rows_are_the_chains(bitserial):
    """Sampled checks (section 5.2: every chain is its own GCM message): row j of the subset
    decrypt is chain idx[j], as libcrypto decrypts it under IV_i and as chains_decrypt does,
    for index sets with a short last chain, 32-byte AAD, tampered chains and repeats."""
    r = rng(66 + int(bitserial))
    key, base_iv = rbytes(r, 32), rbytes(r, 12)
    chain, alen = 1024, 32
    pt = rbytes(r, 9 * chain + 200)   # chain 9 is 200 bytes
    n = W.n_chains(pt.size, chain)
    aad = rbytes(r, n * alen).reshape(n, alen)
    ct, tags = oracle.chains_encrypt(key, base_iv, chain, pt, aad, alen)
    bad_ct, bad_tags, bad_aad = ct.copy(), tags.copy(), aad.copy()
    W.flip_bit(bad_ct[3 * chain:4 * chain], 77)       # chain 3: ciphertext bit
    bad_tags[6, 15] ^= 0x01                            # chain 6: tag bit
    bad_aad[9, 0] ^= 0x80                              # chain 9 (short): AAD bit
    full_pt, full_ok = oracle.chains_decrypt(key, base_iv, chain, bad_ct, bad_tags, bad_aad, alen, bitserial=bitserial)
    assert full_ok.tolist() == [1, 1, 1, 0, 1, 1, 0, 1, 1, 0]
    for idx in ([9], [0, 9, 3], [6, 6, 2], list(range(n))[::-1], [3, 5, 7, 9]):
        sub_pt, sub_ok = oracle.chains_decrypt_subset(key, base_iv, chain, bad_ct, bad_tags, idx, bad_aad, alen,
                                                      bitserial=bitserial)
        assert sub_pt.shape == (len(idx), chain) and sub_ok.shape == (len(idx),)
        for j, i in enumerate(idx):
            lo, hi = i * chain, min(pt.size, (i + 1) * chain)
            want_pt, want_ok = LC.gcm_decrypt(key, oracle.chain_iv(base_iv, i), bad_ct[lo:hi], bad_tags[i],
                                              bad_aad[i])
            assert bytes(sub_pt[j, :hi - lo]) == want_pt == bytes(full_pt[lo:hi])
            assert not sub_pt[j, hi - lo:].any()       # the rest of a short chain's row stays zero
            assert int(sub_ok[j]) == int(want_ok) == int(full_ok[i])
    with pytest.raises(ValueError):
        oracle.chains_decrypt_subset(key, base_iv, chain, bad_ct, bad_tags, [n], bad_aad, alen)


def test_multichain_costs_match_the_paper():
    facts = json.load(open(os.path.join(GOLDEN, "paper_facts.json")))
    assert facts["tag_bits"]["value"] == 128 and facts["key_bits"]["value"] == 256
    r = rng(66)
    key, base_iv = rbytes(r, 32), rbytes(r, 12)
    length = 16 * 4096
    pt = rbytes(r, length)
    costs = {}
    for n in (1, 8, 16):
        chain = length // n
        aad = W.serial_byte_aad(length, chain)
        oracle.count_aes(True)
        _, tags = oracle.chains_encrypt(key, base_iv, chain, pt, aad, 1, nthreads=1)
        calls = oracle.aes_calls()
        oracle.count_aes(False)
        costs[n] = (tags.shape[0], aad.size, calls)
    for n in (8, 16):
        assert costs[n][0] - costs[1][0] == n - 1            # n-1 more tags
        assert costs[n][1] == n * facts["serial_aad_bytes"]["value"]   # n AAD bytes
        assert costs[n][2] - costs[1][2] == n - 1            # n-1 more AES blocks (one J0 per chain)


# --------------------------------------------------------------------------
# Per-sample (ragged) chains (paper sections 5.2 and 5.4)
# --------------------------------------------------------------------------

@needs_libcrypto
def test_ragged_chains_are_standard_gcm_at_their_offsets():
    w = W.ragged_case(1, [0, 1, 17, 4096, 15, 33, 1000, 16], gaps=[0, 2, 0, 1, 0, 3, 0, 0], aad_bytes=3)
    off, ln, aad = w.extra["chain_off"], w.extra["chain_len"], w.extra["aad"]
    fill = np.full(w.payload.size, 0xA5, np.uint8)
    ct, tags = oracle.ragged_encrypt(w.key, w.base_iv, off, ln, w.payload, aad, 3, out=fill.copy())
    covered = np.zeros(w.payload.size, bool)
    for i in range(off.size):
        o, l = int(off[i]), int(ln[i])
        covered[o:o + l] = True
        c, t = LC.gcm_encrypt(w.key, bytes(oracle.chain_iv(w.base_iv, i)), w.payload[o:o + l], aad[i])
        assert bytes(ct[o:o + l]) == c and bytes(tags[i]) == t, i
    assert (ct[~covered] == 0xA5).all()       # bytes outside every chain are left alone
    pt, ok = oracle.ragged_decrypt(w.key, w.base_iv, off, ln, ct, tags, aad, 3)
    assert ok.all() and np.array_equal(pt[covered], w.payload[covered])


def test_ragged_with_uniform_offsets_is_the_uniform_layout():
    r = rng(67)
    key, base_iv = rbytes(r, 32), rbytes(r, 12)
    chain, length = 1024, 9 * 1024 + 300
    pt = rbytes(r, length)
    n = W.n_chains(length, chain)
    off = np.arange(n, dtype=np.uint64) * chain
    ln = np.minimum(chain, length - off.astype(np.int64)).astype(np.uint64)
    aad = rbytes(r, n * 32).reshape(n, 32)
    want = oracle.chains_encrypt(key, base_iv, chain, pt, aad, 32)
    got = oracle.ragged_encrypt(key, base_iv, off, ln, pt, aad, 32)
    assert np.array_equal(got[0], want[0]) and np.array_equal(got[1], want[1])


def test_ragged_sample_reorder_and_tamper_are_caught_per_chain():
    """Section 5.4: the serial-number AAD exposes chains moved within a sample."""
    w = W.sample_batch(n_samples=3, chains_per_sample=4, median=3000, sigma=0.3, lo=100, hi=5000)
    lens = w.extra["sample_lens"]
    offs, cl = [], []
    for o, l in zip(w.extra["sample_off"].tolist(), lens.tolist()):
        part = ((l + 3) // 4 + 15) // 16 * 16
        for j in range(4):
            b = min(j * part, l)
            offs.append(o + b)
            cl.append(min(part, l - b))
    off, ln = np.array(offs, np.uint64), np.array(cl, np.uint64)
    aad = w.extra["aad"]
    ct, tags = oracle.ragged_encrypt(w.key, w.base_iv, off, ln, w.payload, aad, 1)
    # the same ciphertext and tag under another serial number (chain 1 presented as chain 2)
    a2 = aad.copy()
    a2[[1, 2]] = aad[[2, 1]]
    _, ok = oracle.ragged_decrypt(w.key, w.base_iv, off, ln, ct, tags, a2, 1)
    assert ok.tolist() == [1, 0, 0] + [1] * 9
    c2 = ct.copy()
    W.flip_bit(c2[int(off[6]):int(off[6] + ln[6])], 5)
    _, ok = oracle.ragged_decrypt(w.key, w.base_iv, off, ln, c2, tags, aad, 1)
    assert ok.tolist() == [1] * 6 + [0] + [1] * 5
