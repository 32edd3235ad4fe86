"""The H2D pipeline's schedule without a GPU: fastrack_pipeline_plan returns the
operations the pipeline enqueues, in order, and a fake executor replays them with
random operation durations under the stream and event rules the pipeline relies on
(work on one stream runs in order; a wait holds its stream until the work recorded
before the most recent record of the event, as of the wait's enqueue, has finished;
a host wait holds the calling thread, and so every operation enqueued after it,
until then).
For every duration draw: a staging slot is rewritten only after every read of its
previous chunk has finished, a chunk is decrypted (and checked) only after its copy
landed, a keystream slot is overwritten only after the XOR that read it, and every
chunk is decrypted and tag-checked exactly once. A schedule with one wait removed is
caught, which shows that the checks can fail."""
import ctypes
import os
import random

import pytest

MiB = 1 << 20
FUSED, EAGER, OTP = 0, 1, 2
META, RECORD, WAIT, COPY, KEYSTREAM, DECRYPT, APPLY, CTR, VERIFY, HOST_WAIT, DIRECT = range(11)
DIRECT_MODE = 3
READS = (DECRYPT, APPLY, CTR, VERIFY)


@pytest.fixture(scope="module")
def L():
    import paper_2410_15240_amd as F
    if not os.path.exists(F.library_path()):
        from paper_2410_15240_amd import build
        build.build()
    L = F.lib()
    L.fastrack_pipeline_plan.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint64, ctypes.c_int,
                                         ctypes.c_uint32, ctypes.c_void_p, ctypes.c_uint64]
    L.fastrack_pipeline_plan.restype = ctypes.c_int64
    return L


def plan(L, length, chain, chunk, depth, mode):
    n = L.fastrack_pipeline_plan(length, chain, chunk, depth, mode, None, 0)
    assert n >= 0, n
    buf = (ctypes.c_int64 * (6 * n))()
    assert L.fastrack_pipeline_plan(length, chain, chunk, depth, mode, buf, n) == n
    return [tuple(buf[6 * i:6 * i + 6]) for i in range(n)]


def replay(ops, rng):
    """Start/end times of every operation under random durations."""
    stream_t = [0.0, 0.0, 0.0]
    event_t = {}
    times = []
    host_t = 0.0   # nothing enqueued after a host wait starts before the wait returns
    for kind, stream, event, chunk, slot, aux in ops:
        if kind == HOST_WAIT:
            host_t = max(host_t, event_t[event])
            times.append((host_t, host_t))
            continue
        stream_t[stream] = max(stream_t[stream], host_t)
        if kind == RECORD:
            event_t[event] = stream_t[stream]
            times.append((stream_t[stream], stream_t[stream]))
        elif kind == WAIT:
            stream_t[stream] = max(stream_t[stream], event_t.get(event, 0.0))
            times.append((stream_t[stream], stream_t[stream]))
        else:
            start = stream_t[stream]
            dur = rng.uniform(0.1, 10.0) if kind != COPY else rng.uniform(1.0, 20.0)
            stream_t[stream] = start + dur
            times.append((start, start + dur))
    return times


def violations(ops, times, nchunks):
    bad = []
    # per chunk: its copy, its reads, its keystream and its XOR
    copy_end, reads = {}, {}
    ks_of, apply_of = {}, {}
    for (kind, stream, event, chunk, slot, aux), (s, e) in zip(ops, times):
        if kind == COPY:
            copy_end[chunk] = (e, slot)
        elif kind in READS:
            reads.setdefault(chunk, []).append((kind, s, e, slot))
            if kind == APPLY:
                apply_of[chunk] = (s, e, aux)
        elif kind == KEYSTREAM:
            ks_of[chunk] = (s, e, slot)
    for k in range(nchunks):
        kinds = sorted(r[0] for r in reads.get(k, []))
        if kinds not in ([DECRYPT], [APPLY], [CTR, VERIFY]):
            bad.append("chunk %d decrypted/checked %s" % (k, kinds))
            continue
        cend, cslot = copy_end[k]
        for kind, s, e, slot in reads[k]:
            if s < cend:
                bad.append("chunk %d read at %.2f before its copy landed at %.2f" % (k, s, cend))
            if slot != cslot:
                bad.append("chunk %d read from slot %d, copied to %d" % (k, slot, cslot))
        if k in apply_of:
            s, e, aux = apply_of[k]
            ks, ke, kslot = ks_of[k]
            if kslot != aux or s < ke:
                bad.append("chunk %d XORed keystream slot %d before its keystream (slot %d) was written" % (k, aux, kslot))
    # a staging slot is rewritten only after every read of the chunk it held
    holders = {}
    for (kind, stream, event, chunk, slot, aux), (s, e) in zip(ops, times):
        if kind == COPY and slot >= 0:
            prev = holders.get(slot)
            if prev is not None:
                last_read = max(r[2] for r in reads.get(prev, [(0, 0, 0, 0)]))
                if s < last_read:
                    bad.append("slot %d rewritten by chunk %d at %.2f while chunk %d was read until %.2f"
                               % (slot, chunk, s, prev, last_read))
            holders[slot] = chunk
    # a keystream slot is overwritten only after the XOR that read it
    ks_holder = {}
    for (kind, stream, event, chunk, slot, aux), (s, e) in zip(ops, times):
        if kind == KEYSTREAM:
            prev = ks_holder.get(slot)
            if prev is not None and prev in apply_of and s < apply_of[prev][1]:
                bad.append("keystream slot %d rewritten for chunk %d before chunk %d's XOR finished" % (slot, chunk, prev))
            ks_holder[slot] = chunk
    return bad


SCHEDULES = [
    (64 * MiB, MiB, 8 * MiB, 0, FUSED), (64 * MiB, MiB, 8 * MiB, 2, FUSED), (64 * MiB, MiB, 8 * MiB, 3, FUSED),
    (64 * MiB + 4096, 4096, 8 * MiB, 2, FUSED), (100 * MiB + 16, MiB, 8 * MiB, 5, FUSED),
    (64 * MiB, MiB, 8 * MiB, 2, EAGER), (64 * MiB, MiB, 8 * MiB, 3, EAGER), (40 * MiB + 7, 65536, 4 * MiB, 8, EAGER),
    (64 * MiB, MiB, 8 * MiB, 2, OTP), (64 * MiB, MiB, 8 * MiB, 3, OTP), (9 * MiB, MiB, MiB, 2, OTP),
    (4096 * MiB, MiB, 8 * MiB, 2, FUSED), (4096 * MiB, MiB, 8 * MiB, 3, EAGER),
]


@pytest.mark.parametrize("length,chain,chunk,depth,mode", SCHEDULES)
def test_schedule_is_safe_under_any_timing(L, length, chain, chunk, depth, mode):
    ops = plan(L, length, chain, chunk, depth, mode)
    nchunks = (length + chunk - 1) // chunk
    rng = random.Random(length ^ (depth << 8) ^ mode)
    draws = 200 if nchunks <= 64 else 10
    for _ in range(draws):
        bad = violations(ops, replay(ops, rng), nchunks)
        assert not bad, bad[:5]


def test_a_missing_wait_is_caught(L):
    # The host's wait before reusing a ring slot is what keeps the slot safe: drop
    # the first one and some duration draw must let a copy overrun a read.
    ops = plan(L, 64 * MiB, MiB, 8 * MiB, 2, FUSED)
    first_wait = next(i for i, o in enumerate(ops) if o[0] == HOST_WAIT)
    broken = ops[:first_wait] + ops[first_wait + 1:]
    rng = random.Random(7)
    assert any(violations(broken, replay(broken, rng), 8) for _ in range(200))


@pytest.mark.parametrize("length,chain,chunk,depth,mode", SCHEDULES)
def test_copy_stream_never_waits_on_the_device(L, length, chain, chunk, depth, mode):
    # Every device-side wait is on the compute or verify stream; the copies are held
    # back only by the calling thread, at most `window` chunks ahead of the last
    # finished chunk (depth with a ring, 4 otherwise).
    ops = plan(L, length, chain, chunk, depth, mode)
    assert not [o for o in ops if o[0] == WAIT and o[1] == 0]
    window = depth if (mode != OTP and depth > 0) else 4
    waited = {}
    for i, o in enumerate(ops):
        if o[0] == HOST_WAIT:
            waited[i] = o[3]
        if o[0] == COPY and o[3] >= window:
            prev = [c for j, c in waited.items() if j < i]
            assert prev and max(prev) == o[3] - window, (o, prev[-3:])


def test_host_wait_names_the_record_of_its_chunk(L):
    # A host wait takes the last record of its event at the time of the wait: that
    # record must be the one made for the chunk the wait names.
    for depth, mode in ((2, FUSED), (8, FUSED), (0, FUSED), (2, EAGER), (8, EAGER), (3, OTP)):
        ops = plan(L, 200 * MiB, MiB, 8 * MiB, depth, mode)
        last_record = {}
        k = -1   # the chunk whose operations are being enqueued
        for o in ops:
            if o[0] == COPY:
                k = o[3]
            if o[0] == RECORD:
                last_record[o[2]] = k
            if o[0] == HOST_WAIT:
                assert last_record[o[2]] == o[3], (depth, mode, o, last_record[o[2]])


def test_direct_plan(L):
    ops = plan(L, 64 * MiB + 16, MiB, 8 * MiB, 0, DIRECT_MODE)
    assert [o[0] for o in ops] == [META, RECORD, WAIT, DIRECT]
    assert ops[2][1] == 1 and ops[3][1] == 1


def test_plan_rejects_what_the_pipeline_rejects(L):
    for args in ((64 * MiB, MiB, 3 * MiB // 2, 2, FUSED), (64 * MiB, MiB, 8 * MiB, 1, FUSED),
                 (64 * MiB, MiB, 8 * MiB, 0, EAGER), (64 * MiB, MiB, 8 * MiB, 0, OTP),
                 (64 * MiB, MiB, 8 * MiB, 9, FUSED), (64 * MiB, MiB, 8 * MiB, 2, DIRECT_MODE),
                 (64 * MiB, MiB, 8 * MiB, 0, 4), (64 * MiB, 0, 8 * MiB, 2, FUSED)):
        assert L.fastrack_pipeline_plan(*args, None, 0) == -1, args
    assert L.fastrack_pipeline_plan(0, MiB, 8 * MiB, 2, FUSED, None, 0) == 0
