"""The host's system crypto library (OpenSSL libcrypto) through ctypes.

Used only by tests, as an independent pin of the oracle: a library routine the
oracle's special cases must reduce to. Neither the oracle nor the GPU library
links it. Tests that need it skip when it is absent.
"""
import ctypes
import ctypes.util

import numpy as np

_EVP_CTRL_GCM_SET_IVLEN = 0x9
_EVP_CTRL_GCM_GET_TAG = 0x10
_EVP_CTRL_GCM_SET_TAG = 0x11

_lib = None


def available() -> bool:
    return _load() is not None


def _load():
    global _lib
    if _lib is not None:
        return _lib or None
    name = ctypes.util.find_library("crypto")
    for cand in ([name] if name else []) + ["libcrypto.so.3", "libcrypto.so"]:
        try:
            L = ctypes.CDLL(cand)
            break
        except OSError:
            continue
    else:
        _lib = False
        return None
    vp = ctypes.c_void_p
    L.EVP_CIPHER_CTX_new.restype = vp
    L.EVP_CIPHER_CTX_free.argtypes = [vp]
    L.EVP_aes_256_gcm.restype = vp
    L.EVP_aes_256_ecb.restype = vp
    L.EVP_aes_256_ctr.restype = vp
    L.EVP_EncryptInit_ex.argtypes = [vp, vp, vp, ctypes.c_char_p, ctypes.c_char_p]
    L.EVP_DecryptInit_ex.argtypes = [vp, vp, vp, ctypes.c_char_p, ctypes.c_char_p]
    L.EVP_EncryptUpdate.argtypes = [vp, ctypes.c_char_p, ctypes.POINTER(ctypes.c_int), ctypes.c_char_p, ctypes.c_int]
    L.EVP_DecryptUpdate.argtypes = [vp, ctypes.c_char_p, ctypes.POINTER(ctypes.c_int), ctypes.c_char_p, ctypes.c_int]
    L.EVP_EncryptFinal_ex.argtypes = [vp, ctypes.c_char_p, ctypes.POINTER(ctypes.c_int)]
    L.EVP_DecryptFinal_ex.argtypes = [vp, ctypes.c_char_p, ctypes.POINTER(ctypes.c_int)]
    L.EVP_CIPHER_CTX_ctrl.argtypes = [vp, ctypes.c_int, ctypes.c_int, vp]
    L.EVP_CIPHER_CTX_set_padding.argtypes = [vp, ctypes.c_int]
    _lib = L
    return L


def _b(x) -> bytes:
    return bytes(np.asarray(x, dtype=np.uint8).reshape(-1)) if not isinstance(x, (bytes, bytearray)) else bytes(x)


def aes256_ecb_encrypt(key, data) -> bytes:
    L = _load()
    key, data = _b(key), _b(data)
    ctx = L.EVP_CIPHER_CTX_new()
    try:
        assert L.EVP_EncryptInit_ex(ctx, L.EVP_aes_256_ecb(), None, key, None) == 1
        L.EVP_CIPHER_CTX_set_padding(ctx, 0)
        out = ctypes.create_string_buffer(len(data) + 32)
        n = ctypes.c_int(0)
        assert L.EVP_EncryptUpdate(ctx, out, ctypes.byref(n), data, len(data)) == 1
        return out.raw[: n.value]
    finally:
        L.EVP_CIPHER_CTX_free(ctx)


def gcm_encrypt(key, iv, pt, aad=b""):
    """Returns (ct bytes, tag bytes[16])."""
    L = _load()
    key, iv, pt, aad = _b(key), _b(iv), _b(pt), _b(aad)
    ctx = L.EVP_CIPHER_CTX_new()
    try:
        assert L.EVP_EncryptInit_ex(ctx, L.EVP_aes_256_gcm(), None, None, None) == 1
        assert L.EVP_CIPHER_CTX_ctrl(ctx, _EVP_CTRL_GCM_SET_IVLEN, len(iv), None) == 1
        assert L.EVP_EncryptInit_ex(ctx, None, None, key, iv) == 1
        n = ctypes.c_int(0)
        if aad:
            assert L.EVP_EncryptUpdate(ctx, None, ctypes.byref(n), aad, len(aad)) == 1
        out = ctypes.create_string_buffer(len(pt) + 16)
        ct = b""
        if pt:
            assert L.EVP_EncryptUpdate(ctx, out, ctypes.byref(n), pt, len(pt)) == 1
            ct = out.raw[: n.value]
        fin = ctypes.create_string_buffer(16)
        assert L.EVP_EncryptFinal_ex(ctx, fin, ctypes.byref(n)) == 1
        ct += fin.raw[: n.value]
        tag = ctypes.create_string_buffer(16)
        assert L.EVP_CIPHER_CTX_ctrl(ctx, _EVP_CTRL_GCM_GET_TAG, 16, ctypes.cast(tag, ctypes.c_void_p)) == 1
        return ct, tag.raw
    finally:
        L.EVP_CIPHER_CTX_free(ctx)


def gcm_decrypt(key, iv, ct, tag, aad=b""):
    """Returns (pt bytes, ok bool)."""
    L = _load()
    key, iv, ct, tag, aad = _b(key), _b(iv), _b(ct), _b(tag), _b(aad)
    ctx = L.EVP_CIPHER_CTX_new()
    try:
        assert L.EVP_DecryptInit_ex(ctx, L.EVP_aes_256_gcm(), None, None, None) == 1
        assert L.EVP_CIPHER_CTX_ctrl(ctx, _EVP_CTRL_GCM_SET_IVLEN, len(iv), None) == 1
        assert L.EVP_DecryptInit_ex(ctx, None, None, key, iv) == 1
        n = ctypes.c_int(0)
        if aad:
            assert L.EVP_DecryptUpdate(ctx, None, ctypes.byref(n), aad, len(aad)) == 1
        out = ctypes.create_string_buffer(len(ct) + 16)
        pt = b""
        if ct:
            assert L.EVP_DecryptUpdate(ctx, out, ctypes.byref(n), ct, len(ct)) == 1
            pt = out.raw[: n.value]
        tbuf = ctypes.create_string_buffer(tag, 16)
        assert L.EVP_CIPHER_CTX_ctrl(ctx, _EVP_CTRL_GCM_SET_TAG, 16, ctypes.cast(tbuf, ctypes.c_void_p)) == 1
        fin = ctypes.create_string_buffer(16)
        ok = L.EVP_DecryptFinal_ex(ctx, fin, ctypes.byref(n)) == 1
        return pt, ok
    finally:
        L.EVP_CIPHER_CTX_free(ctx)
