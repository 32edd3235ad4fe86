"""The C ABI without a GPU: the library loads, exports every declared symbol,
and rejects invalid arguments before any HIP call is made."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fastrack.h")


@pytest.fixture(scope="module")
def L():
    import paper_2410_15240_amd as F
    if not os.path.exists(F.library_path()):
        from paper_2410_15240_amd import build
        build.build()
    return F.lib()


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^[A-Za-z_][\w \t\*]*?\b(fastrack_\w+)\s*\(", text, re.M)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for want in ("fastrack_gcm_decrypt_verify", "fastrack_gcm_encrypt_tag", "fastrack_pipeline_h2d",
                 "fastrack_num_chains", "fastrack_last_error", "fastrack_shutdown", "fastrack_pipeline_stage_bytes",
                 "fastrack_gcm_decrypt_verify_ragged", "fastrack_gcm_encrypt_tag_ragged", "fastrack_sample_chains"):
        assert want in names


def test_library_exports_every_declared_symbol(L):
    for name in declared_functions():
        assert hasattr(L, name), name


def test_num_chains_and_stage_bytes(L):
    assert L.fastrack_num_chains(0, 16) == 0
    assert L.fastrack_num_chains(1, 16) == 1
    assert L.fastrack_num_chains(1 << 20, 65536) == 16
    assert L.fastrack_num_chains(1 << 20, 1 << 20) == 1
    assert L.fastrack_num_chains((1 << 20) + 1, 1 << 20) == 2
    assert L.fastrack_num_chains(100, 0) == 0
    n = 4096
    assert L.fastrack_pipeline_stage_bytes(4 << 30, 1 << 20, 0, 8 << 20, 2) == 2 * (8 << 20) + 16 * n
    assert L.fastrack_pipeline_stage_bytes(4 << 30, 1 << 20, 32, 8 << 20, 3) == 3 * (8 << 20) + 16 * n + 32 * n


KEY = ctypes.create_string_buffer(32)
IV = ctypes.create_string_buffer(12)
A = 0x10000  # fake, 16-byte aligned "device" addresses: never dereferenced on these paths
B = 0x90000


def dec(L, chain=4096, ct=A, length=65536, tags=B + 0x100000, aad=None, abytes=0, pt=B, ok=B + 0x200000, flags=0,
        key=KEY, iv=IV):
    return L.fastrack_gcm_decrypt_verify(key, iv, chain, ct, length, tags, aad, abytes, pt, ok, flags, None)


def enc(L, chain=4096, pt=A, length=65536, aad=None, abytes=0, ct=B, tags=B + 0x100000, flags=0):
    return L.fastrack_gcm_encrypt_tag(KEY, IV, chain, pt, length, aad, abytes, ct, tags, flags, None)


@pytest.mark.parametrize("kw", [
    dict(chain=0), dict(chain=24), dict(chain=(1 << 32) * 16),
    dict(key=None), dict(iv=None),
    dict(ct=None), dict(pt=None), dict(tags=None), dict(ok=None),
    dict(ct=A + 8), dict(pt=B + 4),
    dict(pt=A + 16),                       # partial overlap of input and output
    dict(abytes=32, aad=None),
    dict(flags=2),
])
def test_decrypt_rejects_bad_arguments(L, kw):
    L.fastrack_last_error.restype = ctypes.c_char_p
    assert dec(L, **kw) == -1
    assert L.fastrack_last_error()


@pytest.mark.parametrize("kw", [dict(chain=0), dict(tags=None), dict(ct=A + 32), dict(pt=A + 1), dict(flags=8)])
def test_encrypt_rejects_bad_arguments(L, kw):
    assert enc(L, **kw) == -1


@pytest.mark.parametrize("args", [(0, 8, 0x1000), (10 ** 7 + 1, 8, 0x1000), (100, 0, 0x1000), (100, 1025, 0x1000),
                                  (100, 8, None)])
def test_clock_probe_rejects_bad_arguments(L, args):
    """The shader-clock probe checks its window, probe count and output pointer before any launch."""
    window, n, out = args
    assert L.fastrack_clock_probe(window, n, out, None) == -1


def test_zero_length_is_a_no_op(L):
    assert dec(L, length=0) == 0
    assert enc(L, length=0) == 0


def pipe(L, chain=1 << 20, length=16 << 20, chunk=8 << 20, depth=2, stage=0x100000000, stage_bytes=None,
         h_ct=0x20000, h_tags=0x40000):
    if stage_bytes is None:
        stage_bytes = L.fastrack_pipeline_stage_bytes(length, chain, 0, chunk, depth)
    return L.fastrack_pipeline_h2d(KEY, IV, chain, h_ct, length, h_tags, None, 0, chunk, depth, stage,
                                   stage_bytes, 0x300000000, 0x400000000, None, None)


@pytest.mark.parametrize("kw", [dict(depth=1), dict(depth=9), dict(depth=-1), dict(chunk=(8 << 20) + 16), dict(chunk=0),
                                dict(stage_bytes=1024), dict(stage=0x100000010), dict(stage=None),
                                dict(h_tags=None)])
def test_pipeline_rejects_bad_arguments(L, kw):
    assert pipe(L, **kw) == -1


def test_pipeline_stage_bytes(L):
    n, tags = 16, 256
    # in place: only the tags and the AAD (each rounded to 256 bytes)
    assert L.fastrack_pipeline_stage_bytes(16 << 20, 1 << 20, 0, 8 << 20, 0) == tags
    assert L.fastrack_pipeline_stage_bytes(16 << 20, 1 << 20, 32, 8 << 20, 0) == tags + 512
    # a ring of depth slots of chunk_bytes (rounded to 256) in front
    assert L.fastrack_pipeline_stage_bytes(16 << 20, 1 << 20, 0, 8 << 20, 3) == 3 * (8 << 20) + tags
    assert L.fastrack_pipeline_stage_bytes(n * 4096 - 5, 4096, 1, 4096, 2) == 2 * 4096 + 256 + 256
    for bad in (1, 9, -1):
        assert L.fastrack_pipeline_stage_bytes(16 << 20, 1 << 20, 0, 8 << 20, bad) == 0


def test_binding_fails_loudly_without_the_library(monkeypatch):
    import paper_2410_15240_amd as F
    monkeypatch.setattr(F._build, "LIB", "/nonexistent/libfastrack.so")
    monkeypatch.setattr(F, "_lib", None)
    with pytest.raises(RuntimeError):
        F.lib()


def eager(L, chain=4096, ct=A, length=65536, tags=B + 0x100000, pt=B, ok=B + 0x200000):
    return L.fastrack_gcm_decrypt_eager(KEY, IV, chain, ct, length, tags, None, 0, pt, ok, None, None)


@pytest.mark.parametrize("kw", [dict(pt=A), dict(tags=None), dict(ok=None), dict(ct=A + 4), dict(chain=24),
                                dict(pt=A + 16)])
def test_eager_rejects_bad_arguments(L, kw):
    assert eager(L, **kw) == -1


def keystream(L, chain=4096, base=0, length=65536, ks=A):
    return L.fastrack_gcm_keystream(KEY, IV, chain, base, length, ks, None)


@pytest.mark.parametrize("kw", [dict(chain=0), dict(ks=None), dict(ks=A + 8), dict(chain=(1 << 32) * 16)])
def test_keystream_rejects_bad_arguments(L, kw):
    assert keystream(L, **kw) == -1


def test_keystream_zero_length_is_a_no_op(L):
    assert keystream(L, length=0) == 0


def apply(L, chain=4096, base=0, ct=A, length=65536, ks=B + 0x400000, tags=B + 0x100000, pt=B, ok=B + 0x200000):
    return L.fastrack_gcm_apply_verify(KEY, IV, chain, base, ct, length, ks, tags, None, 0, pt, ok, None)


@pytest.mark.parametrize("kw", [dict(ks=None), dict(ks=B + 0x400004), dict(ks=B + 16), dict(tags=None),
                                dict(ok=None), dict(pt=A + 32), dict(ct=None)])
def test_apply_verify_rejects_bad_arguments(L, kw):
    assert apply(L, **kw) == -1


def pipe_mode(L, mode=1, depth=2, chain=1 << 20, length=16 << 20, chunk=8 << 20):
    stage_bytes = L.fastrack_pipeline_stage_bytes(length, chain, 0, chunk, max(depth, 2))
    return L.fastrack_pipeline_h2d_mode(KEY, IV, chain, 0x20000, length, 0x40000, None, 0, chunk, depth, mode,
                                        0x100000000, stage_bytes, 0x300000000, 0x400000000, None, None, None)


@pytest.mark.parametrize("kw", [dict(mode=3), dict(mode=1, depth=0), dict(mode=2, depth=0), dict(mode=1, depth=1),
                                dict(mode=2, depth=9)])
def test_pipeline_mode_rejects_bad_arguments(L, kw):
    assert pipe_mode(L, **kw) == -1


def d2h(L, chain=4096, pt=A, length=65536, chunk=16384, ct=B, tags=B + 0x100000, h_ct=0x20000, h_tags=0x40000):
    return L.fastrack_pipeline_d2h(KEY, IV, chain, pt, length, None, 0, chunk, ct, tags, h_ct, h_tags, None, None)


@pytest.mark.parametrize("kw", [dict(chunk=0), dict(chunk=4096 + 16), dict(tags=None), dict(h_ct=None),
                                dict(h_tags=None), dict(ct=A + 16), dict(pt=A + 4), dict(chain=0)])
def test_pipeline_d2h_rejects_bad_arguments(L, kw):
    assert d2h(L, **kw) == -1


def u64s(*v):
    return (ctypes.c_uint64 * max(len(v), 1))(*v)


def rag_dec(L, off=(0, 4096, 8192), ln=(4096, 100, 0), n=None, ct=A, tags=B + 0x100000, pt=B, ok=B + 0x200000,
            aad=None, abytes=0, key=KEY):
    n = (3 if off is None else len(off)) if n is None else n
    o = None if off is None else u64s(*off)
    l = None if ln is None else u64s(*ln)
    return L.fastrack_gcm_decrypt_verify_ragged(key, IV, o, l, n, ct, tags, aad, abytes, pt, ok, None)


def rag_enc(L, off=(0, 4096), ln=(4096, 100), pt=A, ct=B, tags=B + 0x100000):
    return L.fastrack_gcm_encrypt_tag_ragged(KEY, IV, u64s(*off), u64s(*ln), len(off), pt, None, 0, ct, tags, None)


@pytest.mark.parametrize("kw", [
    dict(off=(0, 4100, 8192)),               # misaligned chain offset
    dict(off=(0, 4096, 4096 + 64)),          # chain 2 starts inside chain 1 (100 bytes, 7 blocks)
    dict(off=(4096, 0, 8192)),               # decreasing
    dict(off=None), dict(ln=None), dict(key=None),
    dict(ln=(4096, (1 << 32) * 16, 0)),       # oversized chain
    dict(ct=None), dict(ct=A + 8), dict(pt=A + 16), dict(tags=None), dict(ok=None),
    dict(abytes=1, aad=None),
])
def test_ragged_decrypt_rejects_bad_arguments(L, kw):
    assert rag_dec(L, **kw) == -1
    assert L.fastrack_last_error()


@pytest.mark.parametrize("kw", [dict(tags=None), dict(off=(16, 0)), dict(pt=A + 4)])
def test_ragged_encrypt_rejects_bad_arguments(L, kw):
    assert rag_enc(L, **kw) == -1


def test_ragged_no_chains_is_a_no_op(L):
    assert rag_dec(L, off=(), ln=(), n=0) == 0


def test_ragged_empty_chains_need_no_data_buffers(L):
    assert rag_dec(L, off=(0, 16), ln=(0, 0), ct=None, pt=None, key=None) == -1   # still checks the rest
    assert rag_dec(L, off=(0, 16), ln=(0, 1), ct=None, pt=None) == -1


def test_sample_chains_layout(L):
    """Samples packed back to back, each 16-byte aligned, each cut into equal whole-block parts."""
    lens = [100, 0, 33, 4096, 5]
    k = 4
    n = len(lens) * k
    off, ln = (ctypes.c_uint64 * n)(), (ctypes.c_uint64 * n)()
    total = L.fastrack_sample_chains(u64s(*lens), len(lens), k, off, ln)
    want_off, want_len, pos = [], [], 0
    for s in lens:
        part = -(-(-(-s // k)) // 16) * 16          # ceil(ceil(s / k) / 16) * 16
        end16 = -(-s // 16) * 16
        for j in range(k):
            b = j * part
            want_off.append(pos + (b if b < s else end16))   # empty parts at the sample's aligned end
            want_len.append(max(0, min(part, s - b)))
        pos += end16
    assert list(off) == want_off and list(ln) == want_len and total == pos
    assert sum(want_len) == sum(lens)
    assert L.fastrack_sample_chains(u64s(*lens), len(lens), 0, off, ln) == 0


@pytest.mark.parametrize("lens,k", [([100, 0, 33, 4096, 5], 4), ([1, 17, 3800, 3801, 15], 16), ([0, 0, 16], 3),
                                    ([70000, 12345, 64], 16)])
def test_sample_chains_layout_passes_the_ragged_checks(L, lens, k):
    """Every offset the layout helper writes is accepted by the ragged entry points' chain checks
    (16-byte aligned, increasing, not overlapping). The call is given no ok buffer, so it stops at
    that last argument check, after the chain table has been checked and before any HIP call."""
    L.fastrack_last_error.restype = ctypes.c_char_p
    n = len(lens) * k
    off, ln = (ctypes.c_uint64 * n)(), (ctypes.c_uint64 * n)()
    L.fastrack_sample_chains(u64s(*lens), len(lens), k, off, ln)
    assert all(o % 16 == 0 for o in off)
    assert rag_dec(L, off=tuple(off), ln=tuple(ln), ok=None) == -1
    assert b"d_ok" in L.fastrack_last_error()
