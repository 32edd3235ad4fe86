"""Python binding of the gfx950 multi-chain AES-256-GCM library (libfastrack.so).

Argument marshalling only: every step of the path runs in the library's HIP
kernels. PyTorch supplies device memory, pinned host memory and streams. The
binding raises if the native library is missing; there is no fallback.

Chain layout, IV derivation and error behaviour are documented in
include/fastrack.h.
"""
import ctypes as _ct
import os as _os

import torch as _torch  # loads the HIP runtime that the library then shares

from . import build as _build

__all__ = ["FastrackError", "decrypt_verify", "decrypt_verify_noalloc", "encrypt_tag", "decrypt_eager", "Eager", "keystream", "apply_verify",
           "pipeline_h2d", "pipeline_d2h", "decrypt_verify_ragged", "encrypt_tag_ragged", "sample_chains", "num_chains", "stage_bytes", "shutdown", "clock_probe", "clock_ghz", "library_path", "F_SEQ_GHASH", "PIPE_FUSED",
           "PIPE_EAGER", "PIPE_OTP", "PIPE_DIRECT"]

F_SEQ_GHASH = 1
PIPE_FUSED, PIPE_EAGER, PIPE_OTP, PIPE_DIRECT = 0, 1, 2, 3

OK, EINVAL, EHIP, ENOTPINNED, ENOMEM = 0, -1, -2, -3, -4
_NAMES = {EINVAL: "EINVAL", EHIP: "EHIP", ENOTPINNED: "ENOTPINNED", ENOMEM: "ENOMEM"}


class FastrackError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__("%s (%d): %s" % (_NAMES.get(code, "error"), code, msg))
        self.code = code


_lib = None


def library_path() -> str:
    return _build.LIB


def lib():
    """The loaded native library. Raises if it has not been built."""
    global _lib
    if _lib is None:
        if not _os.path.exists(_build.LIB):
            raise RuntimeError("libfastrack.so is not built; run `python -m paper_2410_15240_amd.build` "
                               "(or __graft_entry__.build())")
        L = _ct.CDLL(_build.LIB)
        vp, u8p, u64, u32 = _ct.c_void_p, _ct.c_void_p, _ct.c_uint64, _ct.c_uint32
        L.fastrack_num_chains.argtypes = [u64, u64]
        L.fastrack_num_chains.restype = u64
        L.fastrack_gcm_decrypt_verify.argtypes = [u8p, u8p, u64, u8p, u64, u8p, u8p, u32, u8p, u8p, u32, vp]
        L.fastrack_gcm_decrypt_verify.restype = _ct.c_int
        L.fastrack_gcm_decrypt_verify_noalloc.argtypes = [u8p, u8p, u64, u8p, u64, u8p, u8p, u32, u8p, u8p, u32,
                                                          vp]
        L.fastrack_gcm_decrypt_verify_noalloc.restype = _ct.c_int
        L.fastrack_gcm_encrypt_tag.argtypes = [u8p, u8p, u64, u8p, u64, u8p, u32, u8p, u8p, u32, vp]
        L.fastrack_gcm_encrypt_tag.restype = _ct.c_int
        L.fastrack_pipeline_stage_bytes.argtypes = [u64, u64, u32, u64, _ct.c_int]
        L.fastrack_pipeline_stage_bytes.restype = u64
        L.fastrack_pipeline_h2d.argtypes = [u8p, u8p, u64, u8p, u64, u8p, u8p, u32, u64, _ct.c_int, u8p, u64, u8p,
                                            u8p, vp, vp]
        L.fastrack_pipeline_h2d.restype = _ct.c_int
        L.fastrack_pipeline_h2d_mode.argtypes = [u8p, u8p, u64, u8p, u64, u8p, u8p, u32, u64, _ct.c_int, u32, u8p,
                                                 u64, u8p, u8p, vp, vp, vp]
        L.fastrack_pipeline_h2d_mode.restype = _ct.c_int
        L.fastrack_pipeline_d2h.argtypes = [u8p, u8p, u64, u8p, u64, u8p, u32, u64, u8p, u8p, u8p, u8p, vp, vp]
        L.fastrack_pipeline_d2h.restype = _ct.c_int
        L.fastrack_pipeline_d2h_mode.argtypes = [u8p, u8p, u64, u8p, u64, u8p, u32, u64, u8p, u8p, u8p, u8p, vp, vp,
                                                 u32]
        L.fastrack_pipeline_d2h_mode.restype = _ct.c_int
        L.fastrack_gcm_decrypt_eager.argtypes = [u8p, u8p, u64, u8p, u64, u8p, u8p, u32, u8p, u8p, vp, vp]
        L.fastrack_gcm_decrypt_eager.restype = _ct.c_int
        L.fastrack_gcm_keystream.argtypes = [u8p, u8p, u64, u64, u64, u8p, vp]
        L.fastrack_gcm_keystream.restype = _ct.c_int
        L.fastrack_gcm_keystream_bitsliced.argtypes = [u8p, u8p, u64, u64, u64, u8p, vp]
        L.fastrack_gcm_keystream_bitsliced.restype = _ct.c_int
        L.fastrack_gcm_apply_verify.argtypes = [u8p, u8p, u64, u64, u8p, u64, u8p, u8p, u8p, u32, u8p, u8p, vp]
        L.fastrack_gcm_apply_verify.restype = _ct.c_int
        L.fastrack_gcm_decrypt_verify_ragged.argtypes = [u8p, u8p, vp, vp, u64, u8p, u8p, u8p, u32, u8p, u8p, vp]
        L.fastrack_gcm_decrypt_verify_ragged.restype = _ct.c_int
        L.fastrack_gcm_encrypt_tag_ragged.argtypes = [u8p, u8p, vp, vp, u64, u8p, u8p, u32, u8p, u8p, vp]
        L.fastrack_gcm_encrypt_tag_ragged.restype = _ct.c_int
        L.fastrack_sample_chains.argtypes = [vp, u64, u32, vp, vp]
        L.fastrack_sample_chains.restype = u64
        L.fastrack_clock_probe.argtypes = [u64, u32, vp, vp]
        L.fastrack_clock_probe.restype = _ct.c_int
        L.fastrack_last_error.restype = _ct.c_char_p
        L.fastrack_shutdown.restype = None
        _lib = L
    return _lib


def _check(rc):
    if rc != OK:
        raise FastrackError(rc, lib().fastrack_last_error().decode(errors="replace"))


def _host_bytes(x, n, what):
    if isinstance(x, _torch.Tensor):
        x = x.detach().to("cpu", _torch.uint8).contiguous().numpy().tobytes()
    elif not isinstance(x, (bytes, bytearray)):
        x = bytes(memoryview(x).cast("B"))
    x = bytes(x)
    if len(x) != n:
        raise ValueError("%s must be %d bytes, got %d" % (what, n, len(x)))
    return _ct.create_string_buffer(x, n)


def _dptr(t):
    return None if t is None else t.data_ptr()


def _u8(t, what, numel=None, min_numel=None, cuda=True, device=None, pinned=False):
    """Check a caller's buffer before its address reaches the library: a uint8,
    contiguous tensor of the size the call reads or writes, on the data's device
    (cuda=True) or in host memory (cuda=False; pinned where the library needs it)."""
    if not isinstance(t, _torch.Tensor):
        raise ValueError("%s must be a torch tensor" % what)
    if t.dtype != _torch.uint8:
        raise ValueError("%s must be uint8, got %s" % (what, t.dtype))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % what)
    if numel is not None and t.numel() != numel:
        raise ValueError("%s holds %d bytes, the call needs exactly %d" % (what, t.numel(), numel))
    if min_numel is not None and t.numel() < min_numel:
        raise ValueError("%s holds %d bytes, the call needs at least %d" % (what, t.numel(), min_numel))
    if cuda:
        if not t.is_cuda:
            raise ValueError("%s must be a CUDA tensor" % what)
        if device is not None and t.device != device:
            raise ValueError("%s is on %s, the data on %s" % (what, t.device, device))
    else:
        if t.device.type != "cpu":
            raise ValueError("%s must be a host (CPU) tensor" % what)
        if pinned and not t.is_pinned():
            raise ValueError("%s must be in pinned host memory" % what)
    return t


def _aad_bytes(aad, n, what="aad", aad_bytes=None, **kw):
    """AAD bytes per chain of an n-chain call: aad must hold exactly n x aad_bytes
    bytes (a (n, a) tensor, or a flat one whose size n divides)."""
    if aad is None:
        if aad_bytes:
            raise ValueError("aad_bytes = %d but no aad tensor" % aad_bytes)
        return 0
    if not isinstance(aad, _torch.Tensor):
        raise ValueError("%s must be a torch tensor" % what)
    if aad_bytes is None:
        if aad.dim() == 2 and aad.shape[0] == n:
            aad_bytes = int(aad.shape[1])
        elif n > 0 and aad.numel() % n == 0:
            aad_bytes = aad.numel() // n
        elif n == 0 and aad.numel() == 0:
            aad_bytes = 0
        else:
            raise ValueError("%s holds %d bytes, not a whole number of bytes for each of the %d chains"
                             % (what, aad.numel(), n))
    if aad_bytes < 0 or aad_bytes > 0xFFFFFFFF:
        raise ValueError("aad_bytes out of range: %d" % aad_bytes)
    _u8(aad, what, numel=n * aad_bytes, **kw)
    return aad_bytes


def _stream(s):
    if s is None:
        return _torch.cuda.current_stream().cuda_stream
    return s.cuda_stream if hasattr(s, "cuda_stream") else int(s)


def _stream_obj(s, device):
    if s is None:
        return _torch.cuda.current_stream(device)
    if isinstance(s, _torch.cuda.Stream):
        return s
    return _torch.cuda.ExternalStream(_stream(s), device=device)


def _used_on(tensors, streams, device):
    """The binding allocated `tensors` on the current stream, and the library's work
    on `streams` still reads or writes them after the call returns: tell the caching
    allocator, so that freeing one does not hand its memory to a new allocation
    while that work is in flight."""
    cur = _torch.cuda.current_stream(device)
    for s in streams:
        so = _stream_obj(s, device)
        if so.cuda_stream == cur.cuda_stream:
            continue
        for t in tensors:
            if t is not None:
                t.record_stream(so)


def num_chains(length, chain_bytes):
    return int(lib().fastrack_num_chains(length, chain_bytes))


def stage_bytes(length, chain_bytes, aad_bytes, chunk_bytes, depth):
    return int(lib().fastrack_pipeline_stage_bytes(length, chain_bytes, aad_bytes, chunk_bytes, depth))


def decrypt_verify(key, base_iv, chain_bytes, ct, tags, aad=None, out=None, ok=None, flags=0, stream=None):
    """Decrypt + verify every chain of ct (uint8 CUDA tensor). Returns (pt, ok).
    tags holds n x 16 bytes and aad (optional) n x aad_bytes bytes, n = num_chains."""
    _u8(ct, "ct")
    dev = ct.device
    n = num_chains(ct.numel(), chain_bytes)
    _u8(tags, "tags", numel=16 * n, device=dev)
    aad_bytes = _aad_bytes(aad, n, device=dev)
    new = []
    if out is None:
        out = _torch.empty_like(ct)
        new.append(out)
    if ok is None:
        ok = _torch.empty(n, dtype=_torch.uint8, device=dev)
        new.append(ok)
    _u8(out, "out", numel=ct.numel(), device=dev)
    _u8(ok, "ok", numel=n, device=dev)
    with _torch.cuda.device(dev):
        _check(lib().fastrack_gcm_decrypt_verify(_host_bytes(key, 32, "key"), _host_bytes(base_iv, 12, "base_iv"),
                                                 chain_bytes, _dptr(ct), ct.numel(), _dptr(tags), _dptr(aad),
                                                 aad_bytes, _dptr(out), _dptr(ok), flags, _stream(stream)))
        _used_on(new, [stream], dev)
    return out, ok


def decrypt_verify_noalloc(key, base_iv, chain_bytes, ct, tags, aad, out, ok, flags=0, stream=None):
    """decrypt_verify through the allocation-free entry point: the caller passes every
    buffer (out, ok) and the library allocates no device memory. Calls on one GPU
    share the library's fixed device area: order calls made on different streams."""
    _u8(ct, "ct")
    dev = ct.device
    n = num_chains(ct.numel(), chain_bytes)
    _u8(tags, "tags", numel=16 * n, device=dev)
    aad_bytes = _aad_bytes(aad, n, device=dev)
    _u8(out, "out", numel=ct.numel(), device=dev)
    _u8(ok, "ok", numel=n, device=dev)
    with _torch.cuda.device(dev):
        _check(lib().fastrack_gcm_decrypt_verify_noalloc(_host_bytes(key, 32, "key"),
                                                         _host_bytes(base_iv, 12, "base_iv"), chain_bytes, _dptr(ct),
                                                         ct.numel(), _dptr(tags), _dptr(aad), aad_bytes, _dptr(out),
                                                         _dptr(ok), flags, _stream(stream)))
    return out, ok


def encrypt_tag(key, base_iv, chain_bytes, pt, aad=None, out=None, tags=None, flags=0, stream=None):
    """Encrypt every chain of pt (uint8 CUDA tensor) and produce its tag. Returns (ct, tags)."""
    _u8(pt, "pt")
    dev = pt.device
    n = num_chains(pt.numel(), chain_bytes)
    aad_bytes = _aad_bytes(aad, n, device=dev)
    new = []
    if out is None:
        out = _torch.empty_like(pt)
        new.append(out)
    if tags is None:
        tags = _torch.empty((n, 16), dtype=_torch.uint8, device=dev)
        new.append(tags)
    _u8(out, "out", numel=pt.numel(), device=dev)
    _u8(tags, "tags", numel=16 * n, device=dev)
    with _torch.cuda.device(dev):
        _check(lib().fastrack_gcm_encrypt_tag(_host_bytes(key, 32, "key"), _host_bytes(base_iv, 12, "base_iv"),
                                              chain_bytes, _dptr(pt), pt.numel(), _dptr(aad), aad_bytes, _dptr(out),
                                              _dptr(tags), flags, _stream(stream)))
        _used_on(new, [stream], dev)
    return out, tags


class Eager:
    """Plaintext released before its tags are checked (the paper's eager evaluation).

    `plaintext` is usable once the decrypt stream has reached the launch; `ok` is
    final once `verified` (an event on the verify stream) has completed. A caller
    that already consumed the plaintext rolls back the work of rejected chains."""

    def __init__(self, plaintext, ok, verified):
        self.plaintext, self.ok, self.verified = plaintext, ok, verified

    def done(self):
        """True once the tag check has finished (does not block)."""
        return self.verified.query()

    def rejected(self):
        """Block until the tags are checked; the indices of the chains whose tag failed."""
        self.verified.synchronize()
        return _torch.nonzero(self.ok == 0).flatten().tolist()

    def settle(self, commit, rollback):
        """Block until verified, then call commit() if every chain passed, else rollback(rejected)."""
        bad = self.rejected()
        return rollback(bad) if bad else commit()


def decrypt_eager(key, base_iv, chain_bytes, ct, tags, aad=None, out=None, ok=None, decrypt_stream=None,
                  verify_stream=None):
    """Decrypt on decrypt_stream and check the tags on verify_stream. Returns an Eager."""
    _u8(ct, "ct")
    dev = ct.device
    n = num_chains(ct.numel(), chain_bytes)
    _u8(tags, "tags", numel=16 * n, device=dev)
    aad_bytes = _aad_bytes(aad, n, device=dev)
    new = []
    if out is None:
        out = _torch.empty_like(ct)
        new.append(out)
    if ok is None:
        ok = _torch.empty(n, dtype=_torch.uint8, device=dev)
        new.append(ok)
    _u8(out, "out", numel=ct.numel(), device=dev)
    _u8(ok, "ok", numel=n, device=dev)
    with _torch.cuda.device(dev):
        ds = decrypt_stream if decrypt_stream is not None else _torch.cuda.current_stream(dev)
        vs = verify_stream if verify_stream is not None else ds
        _check(lib().fastrack_gcm_decrypt_eager(_host_bytes(key, 32, "key"), _host_bytes(base_iv, 12, "base_iv"),
                                                chain_bytes, _dptr(ct), ct.numel(), _dptr(tags), _dptr(aad),
                                                aad_bytes, _dptr(out), _dptr(ok), _stream(ds), _stream(vs)))
        _used_on(new, [ds, vs], dev)
        ev = _torch.cuda.Event()
        ev.record(_stream_obj(vs, dev))
    return Eager(out, ok, ev)


def keystream(key, base_iv, chain_bytes, length, chain_base=0, out=None, stream=None, device=None, bitsliced=False):
    """The CTR keystream of chains chain_base.. covering `length` bytes (a uint8 CUDA tensor).
    bitsliced=True computes it with the bitsliced AES kernel instead of the T-table one."""
    new = []
    if out is None:
        device = _torch.device("cuda", _torch.cuda.current_device()) if device is None else _torch.device(device)
        out = _torch.empty(length, dtype=_torch.uint8, device=device)
        new.append(out)
    _u8(out, "out", min_numel=length)
    with _torch.cuda.device(out.device):
        fn = lib().fastrack_gcm_keystream_bitsliced if bitsliced else lib().fastrack_gcm_keystream
        _check(fn(_host_bytes(key, 32, "key"), _host_bytes(base_iv, 12, "base_iv"), chain_bytes, chain_base, length,
                  _dptr(out), _stream(stream)))
        _used_on(new, [stream], out.device)
    return out


def apply_verify(key, base_iv, chain_bytes, ct, ks, tags, aad=None, aad_bytes=None, chain_base=0, out=None, ok=None,
                 stream=None):
    """pt = ct XOR ks and the tag check of chains chain_base.. of ct. tags, aad and ok
    are the whole message's arrays, indexed by global chain index. Returns (pt, ok)."""
    _u8(ct, "ct")
    dev = ct.device
    _u8(ks, "ks", min_numel=ct.numel(), device=dev)
    _u8(tags, "tags", device=dev)
    if tags.numel() % 16:
        raise ValueError("tags must hold whole 16-byte tags, got %d bytes" % tags.numel())
    total = tags.numel() // 16
    n = num_chains(ct.numel(), chain_bytes)
    if chain_base + n > total:
        raise ValueError("tags hold %d chains, need %d" % (total, chain_base + n))
    aad_bytes = _aad_bytes(aad, total, aad_bytes=aad_bytes, device=dev)
    new = []
    if out is None:
        out = _torch.empty_like(ct)
        new.append(out)
    if ok is None:
        ok = _torch.empty(total, dtype=_torch.uint8, device=dev)
        new.append(ok)
    _u8(out, "out", numel=ct.numel(), device=dev)
    _u8(ok, "ok", min_numel=chain_base + n, device=dev)
    with _torch.cuda.device(dev):
        _check(lib().fastrack_gcm_apply_verify(_host_bytes(key, 32, "key"), _host_bytes(base_iv, 12, "base_iv"),
                                               chain_bytes, chain_base, _dptr(ct), ct.numel(), _dptr(ks), _dptr(tags),
                                               _dptr(aad), aad_bytes, _dptr(out), _dptr(ok), _stream(stream)))
        _used_on(new, [stream], dev)
    return out, ok


def pipeline_h2d(key, base_iv, chain_bytes, h_ct, h_tags, h_aad=None, chunk_bytes=8 << 20, depth=0, stage=None,
                 out=None, ok=None, copy_stream=None, compute_stream=None, device=None, mode=PIPE_FUSED,
                 verify_stream=None):
    """Chunked H2D copy of pinned ciphertext overlapped with decrypt + verify. Returns (pt, ok) on the device.
    mode PIPE_EAGER checks the tags on verify_stream; PIPE_OTP generates each chunk's keystream while it is
    in flight. Both need depth >= 2. PIPE_DIRECT (depth 0) has the decrypt kernel read h_ct itself.
    The call returns while the streams still work; buffers the caller passes (stage, out, ok, h_ct, h_tags,
    h_aad) must stay allocated until copy_stream and compute_stream (and verify_stream) have finished."""
    _u8(h_ct, "h_ct", cuda=False, pinned=True)
    device = _torch.device("cuda", _torch.cuda.current_device()) if device is None else _torch.device(device)
    length = h_ct.numel()
    n = num_chains(length, chain_bytes)
    _u8(h_tags, "h_tags", numel=16 * n, cuda=False)
    aad_bytes = _aad_bytes(h_aad, n, "h_aad", cuda=False)
    need = stage_bytes(length, chain_bytes, aad_bytes, chunk_bytes, depth)
    new = []
    if stage is None:
        stage = _torch.empty(max(need, 1), dtype=_torch.uint8, device=device)
        new.append(stage)
    if out is None:
        out = _torch.empty(length, dtype=_torch.uint8, device=device)
        new.append(out)
    if ok is None:
        ok = _torch.empty(n, dtype=_torch.uint8, device=device)
        new.append(ok)
    _u8(stage, "stage", min_numel=need, device=device)
    _u8(out, "out", numel=length, device=device)
    _u8(ok, "ok", numel=n, device=device)
    with _torch.cuda.device(device):
        vstream = verify_stream if verify_stream is not None else compute_stream
        _check(lib().fastrack_pipeline_h2d_mode(_host_bytes(key, 32, "key"), _host_bytes(base_iv, 12, "base_iv"),
                                                chain_bytes, h_ct.data_ptr(), length, h_tags.data_ptr(), _dptr(h_aad),
                                                aad_bytes, chunk_bytes, depth, mode, _dptr(stage), stage.numel(),
                                                _dptr(out), _dptr(ok), _stream(copy_stream), _stream(compute_stream),
                                                _stream(vstream)))
        _used_on(new, [copy_stream, compute_stream, vstream], device)
    return out, ok


def pipeline_d2h(key, base_iv, chain_bytes, pt, aad=None, chunk_bytes=8 << 20, out=None, tags=None, h_ct=None,
                 h_tags=None, copy_stream=None, compute_stream=None, mode=PIPE_FUSED):
    """Encrypt + tag pt (uint8 CUDA tensor) chunk by chunk into `out` (device; may be pt) and copy each
    chunk to the pinned host tensor h_ct while later chunks are encrypted. Returns (h_ct, h_tags).
    mode PIPE_DIRECT writes the ciphertext straight into h_ct from the kernel (`out` is not used).
    The results are valid once copy_stream has finished."""
    _u8(pt, "pt")
    dev = pt.device
    n = num_chains(pt.numel(), chain_bytes)
    aad_bytes = _aad_bytes(aad, n, device=dev)
    new = []
    if out is None and mode != PIPE_DIRECT:
        out = _torch.empty_like(pt)
        new.append(out)
    if tags is None:
        tags = _torch.empty((n, 16), dtype=_torch.uint8, device=dev)
        new.append(tags)
    if h_ct is None:
        h_ct = _torch.empty(pt.numel(), dtype=_torch.uint8, pin_memory=True)
    if h_tags is None:
        h_tags = _torch.empty((n, 16), dtype=_torch.uint8, pin_memory=True)
    if out is not None:
        _u8(out, "out", numel=pt.numel(), device=dev)
    _u8(tags, "tags", numel=16 * n, device=dev)
    _u8(h_ct, "h_ct", min_numel=pt.numel(), cuda=False, pinned=True)
    _u8(h_tags, "h_tags", numel=16 * n, cuda=False)
    with _torch.cuda.device(dev):
        _check(lib().fastrack_pipeline_d2h_mode(_host_bytes(key, 32, "key"), _host_bytes(base_iv, 12, "base_iv"),
                                                chain_bytes, _dptr(pt), pt.numel(), _dptr(aad), aad_bytes,
                                                chunk_bytes, _dptr(out), _dptr(tags), h_ct.data_ptr(),
                                                h_tags.data_ptr(), _stream(copy_stream), _stream(compute_stream),
                                                mode))
        _used_on(new, [copy_stream, compute_stream], dev)
    return h_ct, h_tags


def _u64_host(x, what):
    import numpy as np
    a = np.ascontiguousarray(np.asarray(x, dtype=np.uint64))
    if a.ndim != 1:
        raise ValueError("%s must be one-dimensional" % what)
    return a


def sample_chains(sample_lens, chains_per_sample):
    """Per-sample chain layout: samples packed 16-byte aligned, each cut into chains_per_sample chains.
    Returns (chain_off, chain_len, total_bytes) with numpy uint64 arrays."""
    import numpy as np
    if int(chains_per_sample) <= 0:
        raise ValueError("chains_per_sample must be positive")
    s = _u64_host(sample_lens, "sample_lens")
    n = s.size * int(chains_per_sample)
    off = np.zeros(max(n, 1), dtype=np.uint64)
    ln = np.zeros(max(n, 1), dtype=np.uint64)
    total = lib().fastrack_sample_chains(s.ctypes.data, s.size, chains_per_sample, off.ctypes.data, ln.ctypes.data)
    return off[:n], ln[:n], int(total)


def _ragged_layout(chain_off, chain_len, size, what):
    off, ln = _u64_host(chain_off, "chain_off"), _u64_host(chain_len, "chain_len")
    if off.size != ln.size:
        raise ValueError("chain_off and chain_len differ in length")
    if off.size and int((off + ln).max()) > size:
        raise ValueError("a chain ends past the end of %s" % what)
    return off, ln


def decrypt_verify_ragged(key, base_iv, chain_off, chain_len, ct, tags, aad=None, out=None, ok=None, stream=None):
    """Decrypt + verify chains of their own offsets and lengths in ct (uint8 CUDA tensor). Returns (pt, ok);
    bytes of pt outside every chain are left as they were."""
    _u8(ct, "ct")
    dev = ct.device
    off, ln = _ragged_layout(chain_off, chain_len, ct.numel(), "ct")
    n = off.size
    _u8(tags, "tags", numel=16 * n, device=dev)
    aad_bytes = _aad_bytes(aad, n, device=dev)
    new = []
    if out is None:
        out = _torch.empty_like(ct)
        new.append(out)
    if ok is None:
        ok = _torch.empty(n, dtype=_torch.uint8, device=dev)
        new.append(ok)
    _u8(out, "out", numel=ct.numel(), device=dev)
    _u8(ok, "ok", numel=n, device=dev)
    with _torch.cuda.device(dev):
        _check(lib().fastrack_gcm_decrypt_verify_ragged(_host_bytes(key, 32, "key"),
                                                        _host_bytes(base_iv, 12, "base_iv"), off.ctypes.data,
                                                        ln.ctypes.data, n, _dptr(ct), _dptr(tags), _dptr(aad),
                                                        aad_bytes, _dptr(out), _dptr(ok), _stream(stream)))
        _used_on(new, [stream], dev)
    return out, ok


def encrypt_tag_ragged(key, base_iv, chain_off, chain_len, pt, aad=None, out=None, tags=None, stream=None):
    """Encrypt + tag chains of their own offsets and lengths in pt (uint8 CUDA tensor). Returns (ct, tags)."""
    _u8(pt, "pt")
    dev = pt.device
    off, ln = _ragged_layout(chain_off, chain_len, pt.numel(), "pt")
    n = off.size
    aad_bytes = _aad_bytes(aad, n, device=dev)
    new = []
    if out is None:
        out = _torch.empty_like(pt)
        new.append(out)
    if tags is None:
        tags = _torch.empty((n, 16), dtype=_torch.uint8, device=dev)
        new.append(tags)
    _u8(out, "out", numel=pt.numel(), device=dev)
    _u8(tags, "tags", numel=16 * n, device=dev)
    with _torch.cuda.device(dev):
        _check(lib().fastrack_gcm_encrypt_tag_ragged(_host_bytes(key, 32, "key"), _host_bytes(base_iv, 12, "base_iv"),
                                                     off.ctypes.data, ln.ctypes.data, n, _dptr(pt), _dptr(aad),
                                                     aad_bytes, _dptr(out), _dptr(tags), _stream(stream)))
        _used_on(new, [stream], dev)
    return out, tags


def clock_probe(window_us, n_probes=8, stream=None, device=None):
    """Measurement helper: enqueue the shader-clock probe (one sleeping wave per probe
    for window_us of real time). Returns a uint64 tensor (n_probes, 2) of (shader
    cycles, 100 MHz ticks); read it once the stream is done (see clock_ghz)."""
    dev = _torch.device("cuda", _torch.cuda.current_device()) if device is None else _torch.device(device)
    out = _torch.zeros((n_probes, 2), dtype=_torch.int64, device=dev)
    with _torch.cuda.device(dev):
        _check(lib().fastrack_clock_probe(int(window_us), int(n_probes), out.data_ptr(), _stream(stream)))
    return out


def clock_ghz(probe):
    """Shader clock in GHz of each probe of a finished clock_probe result."""
    c = probe.cpu().double()
    return (c[:, 0] / (c[:, 1] / 1e8) / 1e9).tolist()


def shutdown():
    if _lib is not None:
        _lib.fastrack_shutdown()
