"""The compile-time tables and set-up arithmetic of the GPU library, built for the
host and checked against the CPU oracle and plain definitions:
  * the S-box against the oracle's (FIPS-197 5.1.1) and T0 against its definition,
    the MixColumns column (02, 01, 01, 03) times S(x) (FIPS-197 5.1.3), byte 0 first;
  * multiplication by x^k and squaring in GF(2^128) against the oracle's bit-serial
    multiply (the GCM field of section 3.2, SP 800-38D 6.3);
  * the columns of the squaring map S^k(x^i) = (x^i)^(2^k), k = 1..8, that the key
    set-up applies to H to reach the squares H^(2^t), against repeated oracle
    multiplies, and their linearity on random elements;
  * the split of a segment weight H^(m 2^g) into table factors H^(j 2^t) (one per
    nonzero base-8 digit of m): the exponents sum to m 2^g, every factor has a
    table, and the product of the factors is H^(m 2^g) in the oracle's field.
The header functions are constexpr and shared by the device code; only the host
pass is compiled here."""
import ctypes
import os

import numpy as np
import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2410_15240_amd", "csrc")
HIPCC = "/opt/rocm/bin/hipcc"


@pytest.fixture(scope="module")
def T(tmp_path_factory):
    import subprocess
    if not os.path.exists(HIPCC):
        pytest.skip("hipcc not found")
    so = str(tmp_path_factory.mktemp("tab") / "libtables_host.so")
    r = subprocess.run([HIPCC, "--offload-arch=gfx950", "--offload-host-only", "-O1", "-std=c++17", "-fPIC",
                        "-shared", "-I", CSRC, os.path.join(ROOT, "tests", "tables", "tables_host.hip"), "-o", so],
                       stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, timeout=300)
    assert r.returncode == 0, r.stdout[-4000:]
    L = ctypes.CDLL(so)
    for f in (L.tab_sbox, L.tab_frob, L.tab_mul_xk, L.tab_square):
        f.restype = None
    L.tab_mul_xk.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p]
    L.tab_weight_steps.argtypes = [ctypes.c_uint32, ctypes.c_uint32] + [ctypes.c_void_p] * 3
    L.tab_weight_steps.restype = ctypes.c_int
    return L


def p(a):
    return a.ctypes.data_as(ctypes.c_void_p)


def x_pow(i):
    """x^i (i < 128) as 16 GCM bytes: degree d is bit 7 - d % 8 of byte d // 8."""
    b = np.zeros(16, np.uint8)
    b[i // 8] = 0x80 >> (i % 8)
    return b


def xtime(v):
    return ((v << 1) ^ (0x1B if v & 0x80 else 0)) & 0xFF


def test_sbox_and_t0(T):
    s = np.zeros(256, np.uint8)
    t0 = np.zeros(256, np.uint32)
    T.tab_sbox(p(s), p(t0))
    want_s = oracle.sbox()[0]
    assert np.array_equal(s, want_s)
    for x in range(256):
        v = int(want_s[x])
        want = xtime(v) | (v << 8) | (v << 16) | ((xtime(v) ^ v) << 24)
        assert int(t0[x]) == want, x


def test_mul_by_x_power_against_the_oracle(T):
    rng = np.random.default_rng(11)
    out = np.zeros(16, np.uint8)
    for k in range(128):
        y = rng.integers(0, 256, 16, dtype=np.uint8)
        T.tab_mul_xk(p(y), k, p(out))
        assert np.array_equal(out, oracle.gf128_mul_bitserial(y, x_pow(k))), k
    # every bit that folds back: y = x^127 times x^k for every k
    for k in range(128):
        T.tab_mul_xk(p(x_pow(127)), k, p(out))
        assert np.array_equal(out, oracle.gf128_mul_bitserial(x_pow(127), x_pow(k))), k


def test_square_against_the_oracle(T):
    rng = np.random.default_rng(12)
    out = np.zeros(16, np.uint8)
    cases = [x_pow(i) for i in range(128)] + [rng.integers(0, 256, 16, dtype=np.uint8) for _ in range(64)]
    for y in cases:
        T.tab_square(p(y), p(out))
        assert np.array_equal(out, oracle.gf128_mul_bitserial(y, y))


def test_squaring_map_columns(T):
    cols = np.zeros(8 * 128 * 16, np.uint8)
    T.tab_frob(p(cols))
    cols = cols.reshape(8, 128, 16)
    for i in range(128):
        v = x_pow(i)
        for k in range(8):
            v = oracle.gf128_mul_bitserial(v, v)
            assert np.array_equal(cols[k, i], v), (k + 1, i)
    # applied as a linear map (XOR of the columns of the set degrees) it is V^(2^k)
    rng = np.random.default_rng(13)
    for _ in range(16):
        y = rng.integers(0, 256, 16, dtype=np.uint8)
        bits = np.unpackbits(y)                 # bit d = degree d (MSB first per byte)
        want = y.copy()
        for k in range(8):
            want = oracle.gf128_mul_bitserial(want, want)
            got = np.bitwise_xor.reduce(cols[k][bits.astype(bool)], axis=0)
            assert np.array_equal(got, want), k + 1


def weight_steps(T, m, g):
    j = np.zeros(12, np.uint32)
    t = np.zeros(12, np.uint32)
    d = np.zeros(1, np.uint32)
    n = T.tab_weight_steps(m, g, p(j), p(t), p(d))
    return [(int(a), int(b)) for a, b in zip(j[:n], t[:n])], int(d[0])


def test_segment_weight_factors(T):
    # every exponent a segment weight can have: m 2^g below 2^32 (a chain has fewer blocks)
    rng = np.random.default_rng(14)
    cases = [(m, g) for g in (0, 4, 7, 8, 10, 13) for m in range(1, 600)]
    cases += [(int(m), g) for g in range(0, 31) for m in rng.integers(1, 1 << (32 - g), 64) if m << g < 1 << 32]
    cases += [((1 << 32) - 1, 0), (0o7777777777, 0), (0o3333333333, 1), (6, 29), (3, 30), (1, 31), (4, 29)]
    for m, g in cases:
        steps, digits = weight_steps(T, m, g)
        assert digits == sum(1 for k in range(11) if (m >> (3 * k)) & 7), (m, g)
        assert len(steps) == digits, (m, g)
        assert sum(j << t for j, t in steps) == m << g, (m, g)          # the factors make up the weight
        for j, t in steps:
            assert j in (1, 3, 5, 7), (m, g, j)
            assert t < (32 if j == 1 else 31), (m, g, j, t)           # squares t <= 31, odd multiples t <= 30
    # the product of the factors, each H^(j 2^t) formed as the table kernel forms it, is H^(m 2^g)
    h = rng.integers(0, 256, 16, dtype=np.uint8)
    sq = [h]
    for _ in range(33):
        sq.append(oracle.gf128_mul_bitserial(sq[-1], sq[-1]))   # sq[t] = H^(2^t)

    def power(e):   # H^e by square-and-multiply over the squares
        r = None
        for t in range(40):
            if (e >> t) & 1:
                r = sq[t] if r is None else oracle.gf128_mul_bitserial(r, sq[t])
        return r

    def factor(j, t):   # H^(3 2^t) = H^(2^t) H^(2^(t+1)), H^(5 2^t) = H^(2^t) H^(2^(t+2)), H^(7 2^t) = H^(3 2^t) H^(2^(t+2))
        if j == 1:
            return sq[t]
        y = oracle.gf128_mul_bitserial(sq[t], sq[t + (2 if j == 5 else 1)])
        return oracle.gf128_mul_bitserial(y, sq[t + 2]) if j == 7 else y

    for m, g in [(1, 7), (6, 7), (7, 10), (63, 8), (511, 7), (0o5307, 4), (12345, 3)]:
        steps, _ = weight_steps(T, m, g)
        prod = None
        for j, t in steps:
            f = factor(j, t)
            prod = f if prod is None else oracle.gf128_mul_bitserial(prod, f)
        assert np.array_equal(prod, power(m << g)), (m, g)
