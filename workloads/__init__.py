"""Seeded synthetic inputs for multi-chain AES-256-GCM, shared by tests and bench.

This module holds none of the method's arithmetic: it draws keys, base IVs and
payload bytes, lays out caller-supplied AAD, and chooses tamper positions and
sample indices. Encryption, decryption and tag computation live in the oracle
(test side) and in the GPU library (product side), never here.

Every generator uses ``numpy.random.Generator(PCG64(seed))`` with a fixed draw
order: key (32 B) -> base IV (12 B) -> payload -> tamper choices -> sample
choices. The paper's workloads (ImageNet batches for ResNet-50, ogbn-products
node features, MovieLens-1M; section 6.1) are not available, so these inputs
stand in for their shapes and sizes.
"""
from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

SEED_BASE = 241015240
KiB = 1024
MiB = 1024 * KiB
GiB = 1024 * MiB


def rng_for(config: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(SEED_BASE + config))


def n_chains(length: int, chain_bytes: int) -> int:
    return (length + chain_bytes - 1) // chain_bytes


def draw_key_iv(rng: np.random.Generator):
    key = rng.integers(0, 256, 32, dtype=np.uint8)
    base_iv = rng.integers(0, 256, 12, dtype=np.uint8)
    return key, base_iv


def index_length_aad(length: int, chain_bytes: int) -> np.ndarray:
    """The 32-byte per-chain AAD of the batch workload: [i]_128 || [len_i]_128.

    Both fields are big-endian 128-bit integers: the chain index and the chain's
    length in bytes. Returned as uint8[n, 32].
    """
    n = n_chains(length, chain_bytes)
    aad = np.zeros((n, 32), np.uint8)
    idx = np.arange(n, dtype=np.uint64)
    lens = np.minimum(np.uint64(chain_bytes), np.uint64(length) - idx * np.uint64(chain_bytes))
    for b in range(8):
        aad[:, 15 - b] = ((idx >> np.uint64(8 * b)) & np.uint64(0xFF)).astype(np.uint8)
        aad[:, 31 - b] = ((lens >> np.uint64(8 * b)) & np.uint64(0xFF)).astype(np.uint8)
    return aad


def serial_byte_aad(length: int, chain_bytes: int) -> np.ndarray:
    """The paper's 1-byte chain-order AAD (section 5.4): chain i carries byte i (n <= 256)."""
    n = n_chains(length, chain_bytes)
    if n > 256:
        raise ValueError("a 1-byte serial number covers at most 256 chains")
    return np.arange(n, dtype=np.uint8).reshape(n, 1)


def f32_to_bf16_bytes(x: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 with round-to-nearest-even, returned as raw little-endian bytes."""
    u = x.astype(np.float32, copy=False).view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16).view(np.uint8)


def flip_bit(buf: np.ndarray, bit: int) -> None:
    """Flip one bit in place; bit 0 is the most significant bit of byte 0."""
    buf[bit // 8] ^= np.uint8(0x80 >> (bit % 8))


@dataclass
class Workload:
    name: str
    key: np.ndarray
    base_iv: np.ndarray
    payload: np.ndarray                 # plaintext bytes (uint8[len])
    chain_sizes: List[int]              # chain_bytes values this workload runs at
    aad_bytes: int = 0
    tamper_chains: Optional[np.ndarray] = None   # chains whose ciphertext gets one flipped bit
    tamper_bits: Optional[np.ndarray] = None     # bit index within each tampered chain
    sample_chains: Optional[np.ndarray] = None   # chains checked one by one at full size
    extra: dict = field(default_factory=dict)

    def aad(self, chain_bytes: int) -> Optional[np.ndarray]:
        if self.aad_bytes == 0:
            return None
        if self.aad_bytes == 32:
            return index_length_aad(self.payload.size, chain_bytes)
        raise ValueError("unsupported AAD layout")


def config1() -> Workload:
    """1 MiB of uniform random bytes; 16 x 64 KiB chains and a single 1 MiB chain; no AAD."""
    rng = rng_for(1)
    key, iv = draw_key_iv(rng)
    payload = np.frombuffer(rng.bytes(MiB), np.uint8).copy()
    return Workload("uniform-1MiB", key, iv, payload, [64 * KiB, MiB])


IMAGE_SHAPE = (256, 3, 224, 224)


def config2() -> Workload:
    """A 256x3x224x224 uint8 image batch, zero-padded to 64 MiB; chains 4 KiB .. 1 MiB; 32-byte AAD."""
    rng = rng_for(2)
    key, iv = draw_key_iv(rng)
    payload = np.zeros(64 * MiB, np.uint8)
    nimg = int(np.prod(IMAGE_SHAPE))
    payload[:nimg] = rng.integers(0, 256, nimg, dtype=np.uint8)
    return Workload("image-batch-64MiB", key, iv, payload, [4 * KiB, 16 * KiB, 64 * KiB, 256 * KiB, MiB],
                    aad_bytes=32)


def config3(nvalues: int = 1 << 29) -> Workload:
    """bf16 model weights drawn N(0, 0.02) (1 GiB at 2^29 values); 1 MiB chains; 1% of chains tampered."""
    rng = rng_for(3)
    key, iv = draw_key_iv(rng)
    payload = np.empty(2 * nvalues, np.uint8)
    step = 1 << 24
    for s in range(0, nvalues, step):
        e = min(nvalues, s + step)
        payload[2 * s:2 * e] = f32_to_bf16_bytes(rng.standard_normal(e - s, dtype=np.float32) * np.float32(0.02))
    chain = MiB
    n = n_chains(payload.size, chain)
    k = int(round(0.01 * n))
    tamper = np.sort(rng.choice(n, size=k, replace=False)).astype(np.int64)
    bits = np.array([int(rng.integers(0, 8 * min(chain, payload.size - c * chain))) for c in tamper], np.int64)
    return Workload("bf16-weights-1GiB", key, iv, payload, [chain], tamper_chains=tamper, tamper_bits=bits)


def config4(nvalues: int = 1 << 26) -> Workload:
    """fp32 gradients drawn N(0, 1) (256 MiB at 2^26 values); 256 KiB chains; GPU encrypt + tag."""
    rng = rng_for(4)
    key, iv = draw_key_iv(rng)
    payload = rng.standard_normal(nvalues, dtype=np.float32).view(np.uint8).copy()
    return Workload("fp32-gradients-256MiB", key, iv, payload, [256 * KiB])


def config5(length: int = 4 * GiB, out: Optional[np.ndarray] = None) -> Workload:
    """Uniform random bytes (4 GiB) for the pipelined host-to-device path; 1 MiB chains; 64 sampled chains.

    ``out`` may be a preallocated (e.g. pinned) uint8 buffer of ``length`` bytes.
    """
    rng = rng_for(5)
    key, iv = draw_key_iv(rng)
    payload = out if out is not None else np.empty(length, np.uint8)
    step = 256 * MiB
    for s in range(0, length, step):
        e = min(length, s + step)
        payload[s:e] = np.frombuffer(rng.bytes(e - s), np.uint8)
    chain = MiB
    n = n_chains(length, chain)
    sample = np.sort(rng.choice(n, size=min(64, n), replace=False)).astype(np.int64)
    return Workload("uniform-4GiB-pipelined", key, iv, payload, [chain], sample_chains=sample,
                    extra={"chunk_bytes": 8 * MiB, "depths": [2, 3]})


def random_case(seed: int, length: int, chain_bytes: int, aad_bytes: int = 0) -> Workload:
    """Small seeded case for edge-shape parity tests (uniform bytes, arbitrary AAD bytes)."""
    rng = np.random.Generator(np.random.PCG64(SEED_BASE + 1000 + seed))
    key, iv = draw_key_iv(rng)
    payload = np.frombuffer(rng.bytes(length), np.uint8).copy()
    w = Workload("random-%d" % seed, key, iv, payload, [chain_bytes], aad_bytes=aad_bytes)
    if aad_bytes:
        w.extra["aad"] = np.frombuffer(rng.bytes(n_chains(length, chain_bytes) * aad_bytes),
                                       np.uint8).reshape(-1, aad_bytes).copy()
    return w


def case_aad(w: Workload, chain_bytes: int) -> Optional[np.ndarray]:
    """The AAD array of a workload at a chain size (None when it carries none)."""
    if "aad" in w.extra:
        return w.extra["aad"]
    return w.aad(chain_bytes)


def sample_batch(n_samples: int = 256, chains_per_sample: int = 16, seed: int = 6, median: int = 110 * KiB,
                 sigma: float = 0.6, lo: int = 4 * KiB, hi: int = MiB) -> Workload:
    """A batch of variable-size samples in the paper's per-sample chain layout (sections 5.2 and 5.4).

    Sample sizes are log-normal (median ``median`` bytes, shape ``sigma``) clipped to [lo, hi] and not
    multiples of 16 in general: compressed-image-like files standing in for a batch of ImageNet JPEGs
    (the paper's ResNet-50 workload, section 6.1). Samples are packed back to back, each starting
    16-byte aligned, with zero bytes in the gaps; the payload bytes are uniform (compressed data is
    high-entropy). Each sample is cut into ``chains_per_sample`` chains (16 tags per sample as in the
    paper's evaluation, section 6.4), and each chain carries its 1-byte serial number within the sample as
    AAD. ``extra`` holds sample_lens, sample_off, chains_per_sample and the AAD array (uint8[n, 1]).
    """
    rng = rng_for(seed)
    key, iv = draw_key_iv(rng)
    lens = np.clip(np.round(median * np.exp(sigma * rng.standard_normal(n_samples))), lo, hi).astype(np.uint64)
    padded = (lens + np.uint64(15)) & ~np.uint64(15)
    offs = np.zeros(n_samples, np.uint64)
    if n_samples > 1:
        offs[1:] = np.cumsum(padded)[:-1]
    total = int(padded.sum())
    payload = np.zeros(total, np.uint8)
    for o, l in zip(offs.tolist(), lens.tolist()):
        payload[o:o + l] = np.frombuffer(rng.bytes(l), np.uint8)
    serial = np.tile(np.arange(chains_per_sample, dtype=np.uint8), n_samples).reshape(-1, 1)
    return Workload("sample-batch-%d" % n_samples, key, iv, payload, [], aad_bytes=1,
                    extra={"sample_lens": lens, "sample_off": offs, "chains_per_sample": chains_per_sample,
                           "aad": serial})


def ragged_case(seed: int, chain_lens, gaps=None, aad_bytes: int = 0) -> Workload:
    """Small seeded ragged case: chains of the given lengths laid out in order, chain i starting at the
    16-byte-aligned end of chain i-1 plus gaps[i] blocks; uniform bytes, arbitrary AAD bytes.
    ``extra`` holds chain_off and chain_len (uint64)."""
    rng = np.random.Generator(np.random.PCG64(SEED_BASE + 2000 + seed))
    key, iv = draw_key_iv(rng)
    ln = np.asarray(chain_lens, dtype=np.uint64)
    g = np.zeros(ln.size, np.uint64) if gaps is None else np.asarray(gaps, dtype=np.uint64)
    off = np.zeros(ln.size, np.uint64)
    pos = 0
    for i in range(ln.size):
        pos += 16 * int(g[i])
        off[i] = pos
        pos += (int(ln[i]) + 15) // 16 * 16
    payload = np.frombuffer(rng.bytes(pos), np.uint8).copy() if pos else np.zeros(0, np.uint8)
    w = Workload("ragged-%d" % seed, key, iv, payload, [], aad_bytes=aad_bytes,
                 extra={"chain_off": off, "chain_len": ln})
    if aad_bytes:
        w.extra["aad"] = np.frombuffer(rng.bytes(ln.size * aad_bytes), np.uint8).reshape(-1, aad_bytes).copy()
    return w
