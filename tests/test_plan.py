"""The work planner on the CPU (fastrack_plan: host only, no device).

Every chain is an independent GCM message (paper section 5.2), and the kernels
split each into segments of 2^seg_log2 blocks aligned to the chain's end. What
the kernels rely on is checked here for many launch shapes: the segments of
every chain partition its blocks exactly, each item's iterations cover its
segment, the item count is what the kernels index, and small launches keep at
most 512 segments per chain. The benchmark's own launches are pinned to the
plans the design describes."""
import ctypes

import pytest

KiB, MiB, GiB = 1 << 10, 1 << 20, 1 << 30


@pytest.fixture(scope="module")
def L():
    import os
    import paper_2410_15240_amd as F
    if not os.path.exists(F.library_path()):
        from paper_2410_15240_amd import build
        build.build()
    L = F.lib()
    L.fastrack_plan.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint32, ctypes.c_void_p]
    L.fastrack_plan.restype = ctypes.c_int
    return L


def plan(L, length, chain, num_cu=256):
    out = (ctypes.c_uint64 * 7)()
    rc = L.fastrack_plan(length, chain, num_cu, out)
    assert rc == 0, rc
    keys = ("lanes_log2", "seg_log2", "segs_full", "segs_last", "items", "iters", "split")
    return dict(zip(keys, (int(v) for v in out)))


def segments(p, q, S):
    """[b, e) of segments 0..S-1 of a chain of q blocks, as the kernels place them."""
    g = 1 << p["seg_log2"]
    out = []
    for s in range(S):
        e = q - (S - 1 - s) * g
        b = 0 if s == 0 else e - g
        out.append((b, e))
    return out


SHAPES = [(16, 16), (17, 16), (1, 1024), (4096, 4096), (1000, 64), (65536 + 48, 4096), (100005, 16384),
          (MiB, 64 * KiB), (MiB, MiB), (MiB + 7, MiB), (777777, MiB), (2 * MiB + 100, 256 * KiB),
          (3 * MiB + 5, MiB), (4 * MiB - 16, MiB), (8 * MiB, MiB), (16400 * 2048 + 100, 2048),
          (9000 * 4096 - 7, 4096), (64 * MiB, 4 * KiB), (64 * MiB - 1000, 64 * KiB), (64 * MiB, 8 * KiB),
          (128 * MiB + 7, 4 * KiB), (40 * MiB + 48, 256 * KiB), (GiB, MiB), (GiB, 16 * MiB), (GiB + 16, 64 * MiB),
          (4 * GiB, GiB), (3 * GiB + 5, (1 << 32) * 16 - 32), (5 * MiB + 3, 48 * KiB), (12345678, 1008)]


@pytest.mark.parametrize("length,chain", SHAPES)
@pytest.mark.parametrize("num_cu", [256, 80, 1])
def test_segments_partition_every_chain(L, length, chain, num_cu):
    p = plan(L, length, chain, num_cu)
    n = -(-length // chain)
    qc = chain // 16
    q_last = -(-(length - (n - 1) * chain) // 16)
    lanes = 1 << p["lanes_log2"]
    assert p["lanes_log2"] in (4, 5, 6)
    assert p["items"] == (n - 1) * p["segs_full"] + p["segs_last"] < 1 << 32
    assert p["split"] == (p["items"] > n)
    g = 1 << p["seg_log2"]
    assert p["segs_full"] == -(-qc // g) and p["segs_last"] == -(-q_last // g)
    assert p["iters"] * lanes >= min(g, qc)                       # the iterations cover a full segment
    assert (p["iters"] - 1) * lanes < min(g, qc)                  # ... with no idle iteration
    for q, S in ((qc, p["segs_full"]), (q_last, p["segs_last"])):
        if S > 1 << 16:   # a huge chain: the counts above, not every segment
            continue
        segs = segments(p, q, S)
        assert segs[0][0] == 0 and segs[-1][1] == q               # from the chain's start to its end
        for (b0, e0), (b1, e1) in zip(segs, segs[1:]):
            assert e0 == b1                                       # contiguous, no block twice
        for b, e in segs:
            assert 0 <= b < e <= q and e - b <= g                 # nonempty, at most one segment long
        assert all(e - b == g for b, e in segs[1:])               # only segment 0 may be short


@pytest.mark.parametrize("length,chain", [(MiB, 64 * KiB), (MiB, MiB), (2 * MiB, MiB), (4 * MiB, MiB),
                                          (512 * KiB + 48, 32 * KiB), (4 * MiB, 64 * KiB)])
def test_small_launches_cut_within_limits(L, length, chain):
    # launches that would leave most waves idle cut chains down to 128-block segments,
    # at most 512 segments per chain
    p = plan(L, length, chain)
    assert p["split"] == 1
    assert p["seg_log2"] >= 7
    assert p["segs_full"] <= 512


def test_the_benchmark_launches(L):
    # the 64 MiB image batch at each chain size of its sweep: 16 lanes per whole 4 KiB chain,
    # 64 lanes per whole 16 KiB chain, 64 KiB to 1 MiB chains cut into 1024-block segments;
    # one wave-item of 16 iterations per resident wave (256 CUs x 16 waves) in every case
    want = {4 * KiB: (4, 0, 16384), 16 * KiB: (6, 0, 4096), 64 * KiB: (6, 1, 4096), 256 * KiB: (6, 1, 4096),
            MiB: (6, 1, 4096)}
    for chain, (ll, split, items) in want.items():
        p = plan(L, 64 * MiB, chain)
        assert (p["lanes_log2"], p["split"], p["items"], p["iters"]) == (ll, split, items, 16), (chain, p)
        assert (p["items"] << p["lanes_log2"]) // 64 == 256 * 16
    p = plan(L, MiB, 64 * KiB)   # 1 MiB of 16 chains: two-iteration segments of 64 lanes
    assert (p["lanes_log2"], p["seg_log2"], p["segs_full"], p["iters"]) == (6, 7, 32, 2)


@pytest.mark.parametrize("args", [(0, 16, 256), (16, 0, 256), (16, 24, 256), (16, 16, 0),
                                  (1 << 40, 16, 256), (16, (1 << 32) * 16, 256)])
def test_plan_rejects_bad_arguments(L, args):
    out = (ctypes.c_uint64 * 7)()
    assert L.fastrack_plan(*args, out) == -1
    assert L.fastrack_plan(16, 16, 256, None) == -1
