"""CPU oracle for multi-chain AES-256-GCM -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package. The GPU product path never imports it.

Thin ctypes wrapper over ``gcm_oracle.c``; every function takes and returns
numpy ``uint8`` arrays. See the C file for what each routine computes and the
section of FIPS-197 / SP 800-38D / the paper it follows.
"""
import ctypes as _ct
import os as _os

import numpy as _np

from . import build as _build

_lib = None


def lib():
    """Load the oracle library, building it first if nothing is built yet."""
    global _lib
    if _lib is None:
        if not _os.path.exists(_build.LIB):
            _build.build()
        L = _ct.CDLL(_build.LIB)
        u8p = _ct.POINTER(_ct.c_uint8)
        u64 = _ct.c_uint64
        L.orc_sbox.argtypes = [u8p, u8p]
        L.orc_aes256_key_expansion.argtypes = [u8p, u8p]
        L.orc_aes256_encrypt_block.argtypes = [u8p, u8p, u8p]
        L.orc_aes256_decrypt_block.argtypes = [u8p, u8p, u8p]
        L.orc_gf128_mul_bitserial.argtypes = [u8p, u8p, u8p]
        L.orc_gf128_mul_table.argtypes = [u8p, u8p, u8p]
        L.orc_ghash.argtypes = [u8p, u8p, u64, _ct.c_int, u8p]
        L.orc_ghash.restype = _ct.c_int
        L.orc_gctr.argtypes = [u8p, u8p, u8p, u64, u8p]
        L.orc_gcm_encrypt.argtypes = [u8p, u8p, u8p, u64, u8p, u64, _ct.c_int, u8p, u8p]
        L.orc_gcm_decrypt.argtypes = [u8p, u8p, u8p, u64, u8p, u64, u8p, _ct.c_int, u8p]
        L.orc_gcm_decrypt.restype = _ct.c_int
        L.orc_num_chains.argtypes = [u64, u64]
        L.orc_num_chains.restype = u64
        L.orc_chain_iv.argtypes = [u8p, u64, u8p]
        L.orc_chains_encrypt.argtypes = [u8p, u8p, u64, u8p, u64, u8p, u64, u8p, u8p, _ct.c_int, _ct.c_int]
        L.orc_chains_encrypt.restype = _ct.c_int
        L.orc_chains_decrypt.argtypes = [u8p, u8p, u64, u8p, u64, u8p, u8p, u64, u8p, u8p, _ct.c_int, _ct.c_int]
        L.orc_chains_decrypt.restype = _ct.c_int
        L.orc_chains_decrypt_subset.argtypes = [u8p, u8p, u64, u8p, u64, u8p, u8p, u64,
                                                _ct.POINTER(_ct.c_uint64), u64, u8p, u8p, _ct.c_int, _ct.c_int]
        L.orc_chains_decrypt_subset.restype = _ct.c_int
        L.orc_max_threads.restype = _ct.c_int
        L.orc_count_aes.argtypes = [_ct.c_int]
        L.orc_aes_calls.restype = u64
        _lib = L
    return _lib


def _u8(a, n=None):
    a = _np.ascontiguousarray(_np.frombuffer(a, dtype=_np.uint8) if isinstance(a, (bytes, bytearray)) else a,
                              dtype=_np.uint8).reshape(-1)
    if n is not None and a.size != n:
        raise ValueError("expected %d bytes, got %d" % (n, a.size))
    return a


def _p(a):
    if a is None:
        return None
    return a.ctypes.data_as(_ct.POINTER(_ct.c_uint8))


def sbox():
    """(S-box, inverse S-box), each a uint8[256], computed from FIPS-197 5.1.1."""
    s = _np.zeros(256, _np.uint8)
    inv = _np.zeros(256, _np.uint8)
    lib().orc_sbox(_p(s), _p(inv))
    return s, inv


def key_expansion(key):
    """The 60 round-key words of AES-256 as uint8[60, 4] (FIPS-197 5.2)."""
    out = _np.zeros(240, _np.uint8)
    lib().orc_aes256_key_expansion(_p(_u8(key, 32)), _p(out))
    return out.reshape(60, 4)


def aes256_encrypt_block(key, block):
    out = _np.zeros(16, _np.uint8)
    lib().orc_aes256_encrypt_block(_p(_u8(key, 32)), _p(_u8(block, 16)), _p(out))
    return out


def aes256_decrypt_block(key, block):
    out = _np.zeros(16, _np.uint8)
    lib().orc_aes256_decrypt_block(_p(_u8(key, 32)), _p(_u8(block, 16)), _p(out))
    return out


def gf128_mul_bitserial(x, y):
    out = _np.zeros(16, _np.uint8)
    lib().orc_gf128_mul_bitserial(_p(_u8(x, 16)), _p(_u8(y, 16)), _p(out))
    return out


def gf128_mul_table(x, y):
    out = _np.zeros(16, _np.uint8)
    lib().orc_gf128_mul_table(_p(_u8(x, 16)), _p(_u8(y, 16)), _p(out))
    return out


def ghash(h, blocks, bitserial=True):
    b = _u8(blocks)
    out = _np.zeros(16, _np.uint8)
    if lib().orc_ghash(_p(_u8(h, 16)), _p(b), b.size, int(bitserial), _p(out)) != 0:
        raise ValueError("GHASH input must be whole 16-byte blocks")
    return out


def gctr(key, icb, data):
    d = _u8(data)
    out = _np.zeros(d.size, _np.uint8)
    lib().orc_gctr(_p(_u8(key, 32)), _p(_u8(icb, 16)), _p(d), d.size, _p(out))
    return out


def gcm_encrypt(key, iv, pt, aad=b"", bitserial=False):
    """Single-message GCM-AE with a 96-bit IV: returns (ct, tag)."""
    p = _u8(pt)
    a = _u8(aad)
    ct = _np.zeros(p.size, _np.uint8)
    tag = _np.zeros(16, _np.uint8)
    lib().orc_gcm_encrypt(_p(_u8(key, 32)), _p(_u8(iv, 12)), _p(p), p.size, _p(a), a.size, int(bitserial),
                          _p(ct), _p(tag))
    return ct, tag


def gcm_decrypt(key, iv, ct, tag, aad=b"", bitserial=False):
    """Single-message GCM-AD: returns (pt, ok). pt is produced even if ok is False."""
    c = _u8(ct)
    a = _u8(aad)
    pt = _np.zeros(c.size, _np.uint8)
    ok = lib().orc_gcm_decrypt(_p(_u8(key, 32)), _p(_u8(iv, 12)), _p(c), c.size, _p(a), a.size,
                               _p(_u8(tag, 16)), int(bitserial), _p(pt))
    return pt, bool(ok)


def num_chains(length, chain_bytes):
    return int(lib().orc_num_chains(length, chain_bytes))


def chain_iv(base_iv, i):
    out = _np.zeros(12, _np.uint8)
    lib().orc_chain_iv(_p(_u8(base_iv, 12)), i, _p(out))
    return out


def chains_encrypt(key, base_iv, chain_bytes, pt, aad=None, aad_bytes=0, bitserial=False, nthreads=0, out=None):
    """Multi-chain encrypt: returns (ct uint8[len], tags uint8[n, 16])."""
    p = _u8(pt)
    n = num_chains(p.size, chain_bytes)
    a = _u8(aad, n * aad_bytes) if aad_bytes else None
    ct = out if out is not None else _np.empty(p.size, _np.uint8)
    tags = _np.zeros((n, 16), _np.uint8)
    rc = lib().orc_chains_encrypt(_p(_u8(key, 32)), _p(_u8(base_iv, 12)), chain_bytes, _p(p), p.size, _p(a),
                                  aad_bytes, _p(ct), _p(tags), int(bitserial), nthreads)
    if rc != 0:
        raise ValueError("chain_bytes must be nonzero")
    return ct, tags


def chains_decrypt(key, base_iv, chain_bytes, ct, tags, aad=None, aad_bytes=0, bitserial=False, nthreads=0,
                   out=None):
    """Multi-chain decrypt + verify: returns (pt uint8[len], ok uint8[n])."""
    c = _u8(ct)
    n = num_chains(c.size, chain_bytes)
    t = _u8(tags, 16 * n)
    a = _u8(aad, n * aad_bytes) if aad_bytes else None
    pt = out if out is not None else _np.empty(c.size, _np.uint8)
    ok = _np.zeros(n, _np.uint8)
    rc = lib().orc_chains_decrypt(_p(_u8(key, 32)), _p(_u8(base_iv, 12)), chain_bytes, _p(c), c.size, _p(t),
                                  _p(a), aad_bytes, _p(pt), _p(ok), int(bitserial), nthreads)
    if rc != 0:
        raise ValueError("chain_bytes must be nonzero")
    return pt, ok


def chains_decrypt_subset(key, base_iv, chain_bytes, ct, tags, idx, aad=None, aad_bytes=0, bitserial=False,
                          nthreads=0):
    """Decrypt + verify only the chains in idx: returns (pt uint8[len(idx), chain_bytes], ok uint8[len(idx)]).
    Row j is chain idx[j] exactly as chains_decrypt computes it (a short last chain fills the front of its row,
    the rest of the row stays zero)."""
    c = _u8(ct)
    n = num_chains(c.size, chain_bytes)
    t = _u8(tags, 16 * n)
    a = _u8(aad, n * aad_bytes) if aad_bytes else None
    ix = _np.ascontiguousarray(idx, dtype=_np.uint64).reshape(-1)
    pt = _np.zeros((ix.size, chain_bytes), _np.uint8)
    ok = _np.zeros(ix.size, _np.uint8)
    rc = lib().orc_chains_decrypt_subset(_p(_u8(key, 32)), _p(_u8(base_iv, 12)), chain_bytes, _p(c), c.size,
                                         _p(t), _p(a), aad_bytes, ix.ctypes.data_as(_ct.POINTER(_ct.c_uint64)),
                                         ix.size, _p(pt), _p(ok), int(bitserial), nthreads)
    if rc != 0:
        raise ValueError("bad chain index or chain_bytes")
    return pt, ok


def ragged_encrypt(key, base_iv, chain_off, chain_len, pt, aad=None, aad_bytes=0, out=None):
    """Chains of their own offsets and lengths (the paper's per-sample chaining, section 5.2): chain i is
    bytes [off_i, off_i + len_i) of pt, encrypted as its own GCM message under chain_iv(base_iv, i) with
    AAD aad[i]. Bytes outside every chain keep the value they have in ``out`` (zeros if out is None).
    Returns (ct uint8[len(pt)], tags uint8[n, 16])."""
    p = _u8(pt)
    off = _np.asarray(chain_off, dtype=_np.uint64).reshape(-1)
    ln = _np.asarray(chain_len, dtype=_np.uint64).reshape(-1)
    n = off.size
    a = _u8(aad, n * aad_bytes).reshape(n, aad_bytes) if aad_bytes else None
    ct = out if out is not None else _np.zeros(p.size, _np.uint8)
    tags = _np.zeros((n, 16), _np.uint8)
    for i in range(n):
        o, l = int(off[i]), int(ln[i])
        c, t = gcm_encrypt(key, chain_iv(base_iv, i), p[o:o + l], a[i] if aad_bytes else b"")
        ct[o:o + l] = c
        tags[i] = t
    return ct, tags


def ragged_decrypt(key, base_iv, chain_off, chain_len, ct, tags, aad=None, aad_bytes=0, out=None):
    """Inverse of ragged_encrypt: returns (pt uint8[len(ct)], ok uint8[n]); every chain's plaintext is
    written whether or not its tag verifies."""
    c = _u8(ct)
    off = _np.asarray(chain_off, dtype=_np.uint64).reshape(-1)
    ln = _np.asarray(chain_len, dtype=_np.uint64).reshape(-1)
    n = off.size
    t = _u8(tags, 16 * n).reshape(n, 16)
    a = _u8(aad, n * aad_bytes).reshape(n, aad_bytes) if aad_bytes else None
    pt = out if out is not None else _np.zeros(c.size, _np.uint8)
    ok = _np.zeros(n, _np.uint8)
    for i in range(n):
        o, l = int(off[i]), int(ln[i])
        p, good = gcm_decrypt(key, chain_iv(base_iv, i), c[o:o + l], t[i], a[i] if aad_bytes else b"")
        pt[o:o + l] = p
        ok[i] = int(good)
    return pt, ok


def max_threads():
    return int(lib().orc_max_threads())


def count_aes(enable):
    """Reset the block-cipher call counter and switch counting on or off."""
    lib().orc_count_aes(int(enable))


def aes_calls():
    return int(lib().orc_aes_calls())
