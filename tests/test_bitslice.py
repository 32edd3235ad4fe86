"""The bitsliced AES building blocks of the GPU library, built for the host and
checked against the CPU oracle (FIPS-197) and plain definitions: the S-box
circuit on every input, the 32 x 32 bit transpose that unslices the keystream,
and a whole AES-256 encryption of 32 blocks through the circuit, MixColumns,
ShiftRows and AddRoundKey."""
import ctypes
import os
import shutil
import subprocess

import numpy as np
import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2410_15240_amd", "csrc")


@pytest.fixture(scope="module")
def B(tmp_path_factory):
    if shutil.which("g++") is None:
        pytest.skip("g++ not found")
    so = str(tmp_path_factory.mktemp("bs") / "libbs_host.so")
    r = subprocess.run(["g++", "-O2", "-std=c++17", "-fPIC", "-shared", "-I", CSRC,
                        os.path.join(ROOT, "tests", "bitslice", "bs_host.cpp"), "-o", so],
                       stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    assert r.returncode == 0, r.stdout
    L = ctypes.CDLL(so)
    for f in (L.bs_sbox_all, L.bs_transpose, L.bs_encrypt32):
        f.restype = None
    return L


def p(a):
    return a.ctypes.data_as(ctypes.c_void_p)


def test_sbox_circuit_is_the_sbox_on_every_input(B):
    out = np.zeros(256, np.uint8)
    B.bs_sbox_all(p(out))
    assert np.array_equal(out, oracle.sbox()[0])


def test_transpose32_against_a_plain_transpose(B):
    rng = np.random.default_rng(1)
    for _ in range(20):
        a = rng.integers(0, 2 ** 32, 32, dtype=np.uint64).astype(np.uint32)
        out = np.zeros(32, np.uint32)
        B.bs_transpose(p(a), p(out))
        bits = (a[:, None] >> np.arange(32, dtype=np.uint32)[None, :]) & 1   # bits[i, s] = bit s of a[i]
        want = (bits.T.astype(np.uint64) << np.arange(32, dtype=np.uint64)[None, :]).sum(axis=1).astype(np.uint32)
        assert np.array_equal(out, want)


def test_bitsliced_aes256_equals_the_oracle(B):
    rng = np.random.default_rng(2)
    for trial in range(8):
        key = rng.integers(0, 256, 32, dtype=np.uint8)
        blocks = rng.integers(0, 256, (32, 16), dtype=np.uint8)
        if trial == 0:
            blocks[:] = 0                       # all-zero blocks (H = AES_K(0))
        rk = np.ascontiguousarray(oracle.key_expansion(key).reshape(-1))
        out = np.zeros((32, 16), np.uint8)
        B.bs_encrypt32(p(rk), p(blocks), p(out))
        for s in range(32):
            assert np.array_equal(out[s], oracle.aes256_encrypt_block(key, blocks[s])), (trial, s)
