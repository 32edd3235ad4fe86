"""GPU parity of the library's host-side state: the per-key table cache (more
keys than it holds, so entries are evicted and rebuilt), a key whose table set-up
was queued on one stream and is used on another, and the per-stream scratch area
growing between launches. Every expected value comes from the CPU oracle;
comparisons are bit-exact."""
import numpy as np
import pytest

import oracle
import workloads as W

pytestmark = pytest.mark.gpu

KiB, MiB = W.KiB, W.MiB


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


def case(seed, length, chain, abytes):
    w = W.random_case(seed, length, chain, abytes)
    aad = W.case_aad(w, chain)
    ct, tags = oracle.chains_encrypt(w.key, w.base_iv, chain, w.payload, aad, abytes)
    return w, aad, ct, tags


def test_more_keys_than_the_cache_holds(F):
    # 12 keys, each used twice in turn: the cache keeps 8 per device, so the second
    # round finds every early key evicted and sets its tables up again.
    cases = [case(300 + i, 3 * 4096 + 100, 4096, 16) for i in range(12)]
    for rnd in range(2):
        for i, (w, aad, ct, tags) in enumerate(cases):
            pt, ok = F.decrypt_verify(w.key, w.base_iv, 4096, dev(ct), dev(tags), dev(aad))
            assert host(ok).tolist() == [1] * tags.shape[0], (rnd, i)
            assert np.array_equal(host(pt), w.payload), (rnd, i)


def test_key_set_up_on_one_stream_used_on_another(F):
    import torch
    w, aad, ct, tags = case(320, 5 * 65536 + 48, 65536, 32)
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    d_ct, d_tags, d_aad = dev(ct), dev(tags), dev(aad)
    torch.cuda.synchronize()
    # the first call with this key queues its table set-up on s1; the call on s2
    # right after it must wait for that set-up, not read the tables half-built
    pt1, ok1 = F.decrypt_verify(w.key, w.base_iv, 65536, d_ct, d_tags, d_aad, stream=s1)
    pt2, ok2 = F.decrypt_verify(w.key, w.base_iv, 65536, d_ct, d_tags, d_aad, stream=s2)
    for pt, ok in ((pt1, ok1), (pt2, ok2)):
        assert host(ok).tolist() == [1] * tags.shape[0]
        assert np.array_equal(host(pt), w.payload)


def test_scratch_grows_between_launches(F):
    # Launches that cut chains into segments keep per-item partials in the stream's
    # scratch area; a larger launch after a small one reallocates it.
    for seed, length, chain in ((330, 2 * MiB + 16, MiB), (331, 64 * MiB + 48, 4 * MiB), (332, 3 * MiB, MiB)):
        w, aad, ct, tags = case(seed, length, chain, 0)
        bad = ct.copy()
        W.flip_bit(bad, 8 * (length - 1))        # the last byte: the last chain fails
        want_pt, want_ok = oracle.chains_decrypt(w.key, w.base_iv, chain, bad, tags, None, 0)
        pt, ok = F.decrypt_verify(w.key, w.base_iv, chain, dev(bad), dev(tags))
        assert host(ok).tolist() == want_ok.tolist(), seed
        assert np.array_equal(host(pt), want_pt), seed
