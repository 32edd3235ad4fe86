"""Benchmark of the multi-chain AES-256-GCM hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--skip-pipeline] [--skip-cpu]

A timed step is one decrypt + verify pass of the 64 MiB image batch
(256x3x224x224 uint8, zero-padded, 32-byte AAD per chain) at each of the chain
sizes 4 KiB, 16 KiB, 64 KiB, 256 KiB and 1 MiB, with every input already
resident in HBM. `value` is the payload decrypted per second over the whole
timed region (GB/s, 1e9 bytes). The W warm-up steps are followed by more until
0.3 s have passed, so the timed steps run at the settled shader clock, which the
script measures during them. Outside the timed region the script also
measures encrypt + tag (256 MiB fp32 gradients, 256 KiB chains), the
sequential-GHASH baseline against the multi-chain path (1 MiB buffer), the
pipelined 4 GiB host-to-device decrypt against a plain pinned copy, and the
CPU oracle on the host cores. One JSON line is printed.
"""
import argparse
import ctypes
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0            # MI355X HBM3E peak
# Integer VALU peak: 256 CUs x 128 lanes x 2.4 GHz = 78.6 T 32-bit lane-ops/s, the lane rate
# behind the published fp32 vector peak (157.3 TFLOP/s = 128 lanes x 2 flops per FMA per CU per
# clock); a wave64 32-bit operation issues at two per CU per clock. An issue-rate probe of
# independent v_xor_b32 / v_add_u32 / v_bitop3_b32 reached 3.4 / 3.4 / 3.0 wave-instructions per
# CU per ns, above the one per clock that 64 lanes per CU would allow.
ALU_PEAK_TOPS = 256 * 128 * 2.4e9 / 1e12
# Under sustained load the shader clock dips for a few milliseconds after work
# starts (kernel traces show launches ~15% slower 2-8 ms into a burst) and then
# settles; warm-up runs at least this long so that the timed steps see the
# settled clock whatever --steps is.
WARMUP_MIN_S = 0.3
# The timed steps follow at least this long of gap-free steps: after the warm-up's
# synchronisations the clock still climbs for 20-30 ms of gap-free load (measured with
# the probe: 2.18 -> 2.22 -> 2.26 GHz in 10 ms chunks, then steady).
GAPLESS_S = 0.05
# Every other timed leg (per-size launches, encrypt sweep, the extra workloads) first
# runs its own calls gap-free for this long, at most PRE_MAX_CALLS of them.
PRE_S, PRE_MAX_CALLS = 0.05, 2000
ROTATE = 4                       # buffer sets the per-size timings cycle through
# LDS reads per 64 blocks of the streaming kernel's main loop and their measured cost
# (CU-cycles per wave instruction, conflict-free, 16 waves per CU)
LDS_T_READS, LDS_T_CYCLES = 197, 2.8
LDS_GH_READS, LDS_GH_CYCLES = 16, 5.5

KiB, MiB, GiB = 1024, 1 << 20, 1 << 30


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--skip-pipeline", action="store_true")
    ap.add_argument("--skip-cpu", action="store_true")
    ap.add_argument("--skip-extras", action="store_true", help="only the timed decrypt sweep and the encrypt sweep")
    ap.add_argument("--pipeline-only", action="store_true",
                    help="only the 4 GiB pipeline leg; prints its results as one JSON line (for tracing)")
    ap.add_argument("--formulation-only", action="store_true",
                    help="only the T-table against bitsliced keystream leg; one JSON line (for profiling)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: the path is per-GPU and shards by whole chains with no exchange "
              "(each GPU would take its own range of chains); run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2410_15240_amd as F
    import workloads as W

    if not os.path.exists(F.library_path()):
        from paper_2410_15240_amd import build
        build.build()
    F.lib()
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()
    if args.pipeline_only:
        print(json.dumps(pipeline(F, W, torch, np, dev)), flush=True)
        return
    if args.formulation_only:
        print(json.dumps(aes_formulation(F, W, torch, dev, stream)), flush=True)
        return

    # ---------------- inputs (config: image batch, chain sweep) ----------------
    w = W.config2()
    payload = torch.from_numpy(w.payload).to(dev)
    L = payload.numel()
    cases = []
    for chain in w.chain_sizes:
        aad = torch.from_numpy(w.aad(chain)).to(dev)
        ct, tags = F.encrypt_tag(w.key, w.base_iv, chain, payload, aad)
        out = torch.empty_like(ct)
        ok = torch.empty(tags.shape[0], dtype=torch.uint8, device=dev)
        cases.append((chain, ct, tags, aad, out, ok))
    torch.cuda.synchronize()

    def step(evs=None):
        for i, (chain, ct, tags, aad, out, ok) in enumerate(cases):
            if evs is not None:
                evs[i][0].record(stream)
            F.decrypt_verify(w.key, w.base_iv, chain, ct, tags, aad, out=out, ok=ok)
            if evs is not None:
                evs[i][1].record(stream)

    log("warmup", args.warmup, "steps, at least %.1f s" % WARMUP_MIN_S)
    warm_steps, warm_s = warm_up(torch, step, args.warmup, WARMUP_MIN_S)
    step_est_ms = warm_s * 1e3 / max(1, warm_steps)
    t_start, t_end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    log("timed steps", args.steps)
    # The shader clock during the timed steps: probes sleeping on a second stream
    # for about the length of the timed region (one wave each, next to the launches).
    pstream = torch.cuda.Stream()
    go = torch.cuda.Event()
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    # The last warm-up steps (GAPLESS_S of them) run straight into the timed ones, with no
    # idle gap between them: after a gap the shader clock dips for several
    # milliseconds, which would otherwise fall inside a short timed region. The
    # event pair below brackets exactly the timed steps.
    gapless = max(20, int(GAPLESS_S / max(step_est_ms * 1e-3, 1e-6)) + 1)
    for _ in range(gapless):
        step()
    go.record(stream)
    pstream.wait_event(go)
    probe = F.clock_probe(max(1, int(0.9 * args.steps * step_est_ms * 1e3)), 8, stream=pstream)
    # The timed region holds only the launches: a timing event between launches
    # costs the GPU a few microseconds each.
    t_start.record(stream)
    for s in range(args.steps):
        step()
    t_end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    total_ms = t_start.elapsed_time(t_end)
    clocks = F.clock_ghz(probe)
    for chain, ct, tags, aad, out, ok in cases:
        assert bool(ok.all()), "benchmark decrypt rejected a chain"
        assert torch.equal(out, payload), "benchmark decrypt produced wrong plaintext"
    # Per chain size: 20 back-to-back launches of that size between two events, three
    # times with no idle gap between the runs; the median of the three. The runs follow
    # 50 ms of untimed launches of the size, gap-free (the checks above leave the GPU
    # idle, and the clock dips for several milliseconds after that: after 100 launches
    # (8 ms) the first size still measured a few percent slow).
    # The launches of one size cycle through four copies of its buffers (512 MiB in all),
    # as the sweep's five sizes do (640 MiB): re-reading one 64 MiB buffer would be
    # served partly by the 256 MB Infinity Cache.
    per = []
    for i, (chain, ct, tags, aad, out, ok) in enumerate(cases):
        sets = [(ct, tags, out, ok)] + [(ct.clone(), tags.clone(), torch.empty_like(out), torch.empty_like(ok))
                                        for _ in range(ROTATE - 1)]
        turn = [0]

        def one():
            c_, t_, o_, k_ = sets[turn[0] % ROTATE]
            turn[0] += 1
            F.decrypt_verify(w.key, w.base_iv, chain, c_, t_, aad, out=o_, ok=k_)
        per.append(time_calls(torch, stream, one, 20, runs=3))
        for c_, t_, o_, k_ in sets:
            assert bool(k_.all()) and torch.equal(o_, payload), "benchmark decrypt produced wrong plaintext"
        del sets
    # The achievable HBM rate on this machine: a plain 64 MiB device-to-device copy
    # (read + write bytes over time, best of five gap-free runs of 20 copies). Under
    # rocprofv3 --pmc its FETCH_SIZE / WRITE_SIZE also calibrate the counters.
    dst, src = cases[0][4], cases[0][1]
    copy_ms = time_runs(torch, stream, lambda: dst.copy_(src), 20, 5)[0]
    copy_gbs = 2 * src.numel() / (copy_ms * 1e-3) / 1e9
    torch.cuda.synchronize()
    ms_per_step = total_ms / args.steps
    value = len(cases) * L / (ms_per_step * 1e-3) / 1e9
    sweep = {}
    alg_bytes = []
    for i, (chain, ct, tags, aad, out, ok) in enumerate(cases):
        n = tags.shape[0]
        ms = per[i]
        ab = 2 * L + n * (16 + 32 + 1)   # payload in + out, tags, AAD, ok flags
        alg_bytes.append(ab)
        sweep["%dKiB" % (chain // KiB)] = {"gbps": round(L / (ms * 1e-3) / 1e9, 1), "us": round(ms * 1e3, 1),
                                           "chains": n, "hbm_frac": round(ab / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}
    # average launch duration over the timed region (5 launches per step, one per chain size)
    launch_ms = ms_per_step / len(cases)
    per_size_mean_ms = float(np.mean(per))
    bytes_per_launch = float(np.mean(alg_bytes))
    hbm_gbs = bytes_per_launch / (launch_ms * 1e-3) / 1e9
    log("decrypt sweep %.1f GB/s, %.3f ms/step, %.1f us/launch (per-size mean %.1f us), clock %s GHz, copy %.0f GB/s"
        % (value, ms_per_step, launch_ms * 1e3, per_size_mean_ms * 1e3, ["%.2f" % c for c in clocks], copy_gbs))
    sq = sq_profile("decrypt")
    # The LDS bound of the main loop: per 64 blocks (one wave-iteration) 197 conflict-free
    # 32-bit T-table reads at 2.8 CU-cycles each and 16 conflict-free 16-byte GHASH reads
    # at 5.5 (microbenchmarks on the box), over 256 CUs at the clock the probe measured.
    lds_cycles = LDS_T_READS * LDS_T_CYCLES + LDS_GH_READS * LDS_GH_CYCLES
    clk = float(np.mean(clocks))
    bound_us = L / 16 / 64 / 256 * lds_cycles / (clk * 1e3)
    lds_bound = {"cycles_per_64_blocks": round(lds_cycles, 1), "clock_ghz": round(clk, 3),
                 "main_loop_bound_us": round(bound_us, 2), "frac": round(bound_us / (launch_ms * 1e3), 3),
                 "note": "launch time against the LDS time of the main loop alone at the measured clock; the "
                         "rest of a launch is set-up and tail"}
    valu = None
    if sq:
        insts = float(np.mean([sq[k] for k in sq]))   # VALU wave-instructions per launch, mean over the sizes
        tops = insts * 64 / (launch_ms * 1e-3) / 1e12
        valu = {"achieved": round(tops, 2), "peak": round(ALU_PEAK_TOPS, 2), "unit": "T lane-op/s",
                "frac": round(tops / ALU_PEAK_TOPS, 3), "valu_insts_per_launch": int(insts),
                "source": "SQ_INSTS_VALU (rocprofv3 --pmc) of the same launches, %s" % os.path.basename(SQ_FILE)}

    result = {
        "metric": "AES-256-GCM decrypt+verify GB/s vs chain size; % HBM peak; pipelined H2D GB/s",
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "warmup_run": {"steps": warm_steps + gapless, "seconds": round(warm_s, 3),
                       "gapless_steps": gapless},
        "ms_per_step": round(ms_per_step, 4),
        "wall_s": round(wall, 3),   # host clock: the gapless warm-up steps and the timed steps
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u8",
        "data": "synthetic (seeded uint8 image batch, zero-padded; see workloads/)",
        "config": {"workload": "image-batch-64MiB: 256x3x224x224 uint8 zero-padded to 64 MiB, decrypt+verify at "
                               "chain sizes 4K/16K/64K/256K/1M, 32-byte AAD per chain",
                   "bytes_per_step": len(cases) * L, "parallelism": "single GPU"},
        "sweep": sweep,
        "launch_us": {"timed_region_mean": round(launch_ms * 1e3, 2), "per_size_mean": round(per_size_mean_ms * 1e3, 2),
                      "ratio": round(launch_ms / per_size_mean_ms, 3)},
        "shader_clock_ghz": {"mean": round(float(np.mean(clocks)), 3), "min": round(min(clocks), 3),
                             "max": round(max(clocks), 3),
                             "how": "s_memtime cycles over s_memrealtime ticks, 8 probe waves (one per XCD) "
                                    "sleeping on a second stream during the timed steps"},
        "roofline": {"bound": "hbm", "achieved": round(hbm_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(hbm_gbs / HBM_PEAK_GBS, 4), "traffic": measured_traffic(),
                     "kernel": "gcm_kernel<decrypt> (+ chain_tag_kernel where chains are cut into segments)",
                     "alg_bytes_per_launch": int(bytes_per_launch), "launch_us": round(launch_ms * 1e3, 2),
                     "device_copy_gbps": round(copy_gbs, 1),
                     "frac_of_device_copy": round(hbm_gbs / copy_gbs, 4),
                     "limiter": "LDS table reads and integer VALU issue (the AES T-table lookups and GHASH "
                                "table lookups), not HBM",
                     "lds_bound": lds_bound,
                     "valu": valu},
    }

    result["encrypt_sweep"] = encrypt_sweep(F, W, torch, dev, stream)
    if not args.skip_extras:
        result.update(extras(F, W, torch, np, dev, stream, args))
    if not args.skip_cpu:
        result["cpu_baseline"] = cpu_baseline(W, np, cases, w)
    print(json.dumps(result), flush=True)


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "gcm_decrypt_image-batch-64MiB_traffic.txt")
# everything that shapes the kernels' machine code
KERNEL_SRCS = [os.path.join(ROOT, "paper_2410_15240_amd", *p) for p in
               (("csrc", "kernels.hip"), ("csrc", "aes_dev.h"), ("csrc", "gf128_dev.h"), ("csrc", "keyctx.h"),
                ("csrc", "launch.h"), ("csrc", "chain_dev.h"), ("build.py",))]


def kernels_sha256():
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SRCS:
        h.update(open(f, "rb").read())
    return h.hexdigest()


def measured_traffic():
    """Calibrated HBM bytes per decrypt launch from the committed rocprofv3 counter
    summary, or None when the kernel sources have changed since it was taken."""
    try:
        fields = {}
        for line in open(TRAFFIC_FILE):
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                fields[k.strip()] = v.strip()
        if fields.get("kernels_sha256") != kernels_sha256():
            return None
        return int(float(fields["traffic_bytes_per_launch"]))
    except (OSError, KeyError, ValueError):
        return None


def warm_up(torch, step, steps, min_s):
    """Run `steps` untimed steps, then more in blocks of 20 until min_s seconds have
    passed. Returns (steps run, seconds)."""
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    n = 0
    for _ in range(steps):
        step()
        n += 1
    torch.cuda.synchronize()
    while time.perf_counter() - t0 < min_s:
        for _ in range(20):
            step()
        n += 20
        torch.cuda.synchronize()
    return n, time.perf_counter() - t0


SQ_FILE = os.path.join(ROOT, "profiles", "gcm_image-batch-64MiB_valu.txt")


def sq_profile(direction):
    """VALU wave-instructions per launch of each chain size ("decrypt" or "encrypt")
    from the committed rocprofv3 counter summary, or None when the kernel sources
    have changed since it was taken."""
    try:
        fields, out = {}, {}
        for line in open(SQ_FILE):
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                fields[k.strip()] = v.strip()
        if fields.get("kernels_sha256") != kernels_sha256():
            return None
        for k, v in fields.items():
            if k.startswith(direction + "_valu_insts_"):
                out[k[len(direction) + len("_valu_insts_"):]] = float(v)
        return out or None
    except (OSError, ValueError):
        return None


def time_runs(torch, stream, fn, reps, runs):
    """Times of one call (ms, sorted): the mean over `reps` back-to-back calls between
    two events, for each of `runs` runs that follow one another with no idle gap.
    Untimed calls filling about PRE_S seconds run first, straight into the timed ones:
    after idling, the GPU runs its first milliseconds at a lower clock, which then
    keeps climbing for 20-30 ms."""
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(4):
        fn()
    torch.cuda.synchronize()
    one = max((time.perf_counter() - t0) / 4, 1e-6)
    for _ in range(min(PRE_MAX_CALLS, max(1, int(PRE_S / one)))):
        fn()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(runs)]
    for a, b in evs:
        a.record(stream)
        for _ in range(reps):
            fn()
        b.record(stream)
    torch.cuda.synchronize()
    return sorted(a.elapsed_time(b) / reps for a, b in evs)


def time_calls(torch, stream, fn, reps, runs=1):
    """Median over `runs` gap-free runs of the mean time of one call (ms) over `reps`
    back-to-back calls (see time_runs)."""
    ts = time_runs(torch, stream, fn, reps, runs)
    return ts[len(ts) // 2]


def encrypt_sweep(F, W, torch, dev, stream):
    """Encrypt + tag against chain size: the decrypt sweep's image batch and chain sizes."""
    w2s = W.config2()
    p2s = torch.from_numpy(w2s.payload).to(dev)
    o2s = torch.empty_like(p2s)
    esweep = {}
    sq = sq_profile("encrypt") or {}
    L2 = p2s.numel()
    ins = [p2s] + [p2s.clone() for _ in range(ROTATE - 1)]   # four buffer sets, as in the decrypt sweep
    outs = [o2s] + [torch.empty_like(o2s) for _ in range(ROTATE - 1)]
    for chain in w2s.chain_sizes:
        a2s = torch.from_numpy(w2s.aad(chain)).to(dev)
        n2 = F.num_chains(L2, chain)
        tgs = [torch.empty((n2, 16), dtype=torch.uint8, device=dev) for _ in range(ROTATE)]
        turn = [0]

        def enc():
            j = turn[0] % ROTATE
            turn[0] += 1
            F.encrypt_tag(w2s.key, w2s.base_iv, chain, ins[j], a2s, out=outs[j], tags=tgs[j])
        ms = time_calls(torch, stream, enc, 20, runs=3)
        name = "%dKiB" % (chain // KiB)
        e = {"gbps": round(L2 / ms / 1e6, 1), "us": round(ms * 1e3, 1),
             "hbm_frac": round((2 * L2 + n2 * (32 + 16)) / ms / 1e6 / HBM_PEAK_GBS, 4)}
        if name in sq:
            e["valu_frac"] = round(sq[name] * 64 / (ms * 1e-3) / 1e12 / ALU_PEAK_TOPS, 3)
        esweep[name] = e
    log("encrypt sweep:", esweep)
    return {"workload": "image-batch-64MiB, 32-byte AAD per chain", "sweep": esweep,
            "valu_frac_source": os.path.basename(SQ_FILE) if sq else None}


def extras(F, W, torch, np, dev, stream, args):
    res = {}
    # encrypt + tag: fp32 gradients, 256 KiB chains
    w4 = W.config4()
    pt4 = torch.from_numpy(w4.payload).to(dev)
    c4 = w4.chain_sizes[0]
    out4 = torch.empty_like(pt4)
    tags4 = torch.empty((F.num_chains(pt4.numel(), c4), 16), dtype=torch.uint8, device=dev)
    ms = time_calls(torch, stream, lambda: F.encrypt_tag(w4.key, w4.base_iv, c4, pt4, out=out4, tags=tags4), 20)
    n4 = tags4.shape[0]
    res["encrypt_tag"] = {"workload": "fp32-gradients-256MiB, 256 KiB chains", "gbps": round(pt4.numel() / ms / 1e6, 1),
                          "us": round(ms * 1e3, 1),
                          "hbm_frac": round((2 * pt4.numel() + 16 * n4) / ms / 1e6 / HBM_PEAK_GBS, 4),
                          "note": "256 MiB in + 256 MiB out partly served by the 256 MB Infinity Cache"}
    log("encrypt+tag %.1f GB/s" % res["encrypt_tag"]["gbps"])
    del pt4, out4, tags4

    # the paper's sequential GHASH vs multi-chain, 1 MiB buffer
    w1 = W.config1()
    p1 = torch.from_numpy(w1.payload).to(dev)
    seq = {}
    for chain in w1.chain_sizes:
        ct1, tg1 = F.encrypt_tag(w1.key, w1.base_iv, chain, p1)
        o1 = torch.empty_like(ct1)
        k1 = torch.empty(tg1.shape[0], dtype=torch.uint8, device=dev)
        for name, flags in (("multi_chain", 0), ("sequential_ghash", F.F_SEQ_GHASH)):
            ms = time_calls(torch, stream, lambda: F.decrypt_verify(w1.key, w1.base_iv, chain, ct1, tg1, out=o1,
                                                                   ok=k1, flags=flags), 50)
            assert bool(k1.all())
            seq["%s_%dKiB" % (name, chain // KiB)] = {"us": round(ms * 1e3, 1),
                                                      "gbps": round(p1.numel() / ms / 1e6, 2)}
    for chain in w1.chain_sizes:
        k = "%dKiB" % (chain // KiB)
        seq["sequential_over_multi_chain_%s" % k] = round(seq["sequential_ghash_" + k]["us"] / seq["multi_chain_" + k]["us"], 1)
    # The paper's own comparison: sequential GHASH per tag, one chain against 16 chains
    seq["sequential_1_chain_over_16_chains"] = round(seq["sequential_ghash_1024KiB"]["us"] /
                                                     seq["sequential_ghash_64KiB"]["us"], 1)
    seq["paper_multi_chain_gain"] = "5-15x (section 5.2; 16 tags per item up to 16x, section 6.4), context only"
    res["config1_1MiB"] = seq
    log("1 MiB:", seq)

    # bf16 weights, 1 GiB, 1 MiB chains: decrypt + verify, then the 1% tampered chains rejected exactly
    w3 = W.config3()
    p3 = torch.from_numpy(w3.payload).to(dev)
    c3 = w3.chain_sizes[0]
    ct3, tg3 = F.encrypt_tag(w3.key, w3.base_iv, c3, p3)
    o3 = torch.empty_like(ct3)
    k3 = torch.empty(tg3.shape[0], dtype=torch.uint8, device=dev)
    ms = time_calls(torch, stream, lambda: F.decrypt_verify(w3.key, w3.base_iv, c3, ct3, tg3, out=o3, ok=k3), 10)
    assert bool(k3.all()) and torch.equal(o3, p3), "1 GiB decrypt failed"
    for c, b in zip(w3.tamper_chains, w3.tamper_bits):   # one bit per chosen chain, as the parity test flips it
        byte = int(c) * c3 + int(b) // 8
        ct3[byte] ^= 0x80 >> (int(b) % 8)   # bit 0 is the most significant bit of byte 0
    F.decrypt_verify(w3.key, w3.base_iv, c3, ct3, tg3, out=o3, ok=k3)
    torch.cuda.synchronize()
    rejected = torch.nonzero(k3 == 0).flatten().cpu().tolist()
    res["weights_1GiB"] = {"workload": "bf16-weights-1GiB, 1 MiB chains, no AAD", "gbps": round(p3.numel() / ms / 1e6, 1),
                           "us": round(ms * 1e3, 1), "chains": int(tg3.shape[0]),
                           "tampered": len(w3.tamper_chains),
                           "rejected_exactly_the_tampered": rejected == [int(x) for x in w3.tamper_chains]}
    log("1 GiB weights:", res["weights_1GiB"])
    del p3, ct3, o3, w3

    # eager evaluation: plaintext released before the tag check (64 MiB image batch, 64 KiB chains)
    w2 = W.config2()
    chain2 = 64 * KiB
    p2 = torch.from_numpy(w2.payload).to(dev)
    a2 = torch.from_numpy(w2.aad(chain2)).to(dev)
    c2, t2 = F.encrypt_tag(w2.key, w2.base_iv, chain2, p2, a2)
    o2 = torch.empty_like(c2)
    k2 = torch.empty(t2.shape[0], dtype=torch.uint8, device=dev)
    vstream = torch.cuda.Stream()
    fused = lambda: F.decrypt_verify(w2.key, w2.base_iv, chain2, c2, t2, a2, out=o2, ok=k2)
    fused_ms = time_calls(torch, stream, fused, 40)
    # Eager calls back to back and warm, each one's decryption waiting (on the device)
    # for the previous call's verification: no call overlaps the next, and the GPU
    # never idles between them. Plaintext ready = the decrypt stream's part; verified
    # = through the verification on the second stream.
    n_e, pre_e = 40, 60
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(n_e)]
    torch.cuda.synchronize()
    for i in range(pre_e + n_e):
        stream.wait_stream(vstream)
        if i >= pre_e:
            ev[i - pre_e][0].record(stream)
        e = F.decrypt_eager(w2.key, w2.base_iv, chain2, c2, t2, a2, out=o2, ok=k2, decrypt_stream=stream,
                            verify_stream=vstream)
        if i >= pre_e:
            ev[i - pre_e][1].record(stream)
            ev[i - pre_e][2].record(vstream)
    torch.cuda.synchronize()
    pt_ms = [x[0].elapsed_time(x[1]) for x in ev]
    ok_ms = [x[0].elapsed_time(x[2]) for x in ev]
    assert not e.rejected() and torch.equal(o2, p2)
    res["eager"] = {"workload": "image-batch-64MiB, 64 KiB chains, 32-byte AAD",
                    "fused_us": round(fused_ms * 1e3, 1), "plaintext_ready_us": round(float(np.median(pt_ms)) * 1e3, 1),
                    "verified_us": round(float(np.median(ok_ms)) * 1e3, 1)}
    log("eager:", res["eager"])

    # one-time-pad precompute: what is left once an 8 MiB chunk (1 MiB chains) has arrived
    chunk = 8 * MiB
    p5 = p2[:chunk]
    c5, t5 = F.encrypt_tag(w2.key, w2.base_iv, MiB, p5)
    o5 = torch.empty_like(c5)
    k5 = torch.empty(t5.shape[0], dtype=torch.uint8, device=dev)
    ks5 = F.keystream(w2.key, w2.base_iv, MiB, chunk)
    ks_ms = time_calls(torch, stream, lambda: F.keystream(w2.key, w2.base_iv, MiB, chunk, out=ks5), 50)
    apply_ms = time_calls(torch, stream, lambda: F.apply_verify(w2.key, w2.base_iv, MiB, c5, ks5, t5, out=o5, ok=k5), 50)
    assert bool(k5.all()) and torch.equal(o5, p5)
    fused5_ms = time_calls(torch, stream, lambda: F.decrypt_verify(w2.key, w2.base_iv, MiB, c5, t5, out=o5, ok=k5), 50)
    res["aes_formulation"] = aes_formulation(F, W, torch, dev, stream)
    res["otp"] = {"workload": "8 MiB chunk, 1 MiB chains", "keystream_us": round(ks_ms * 1e3, 1),
                  "after_arrival_fused_us": round(fused5_ms * 1e3, 1),
                  "after_arrival_apply_us": round(apply_ms * 1e3, 1)}
    log("otp:", res["otp"])
    del p2, a2, c2, t2, o2, k2, c5, t5, o5, k5, ks5

    # per-sample chaining: 1024 variable-size samples x 16 chains, 1-byte serial AAD, against uniform
    # 8 KiB chains over the same bytes (the mean chain is about 8 KiB)
    w6 = W.sample_batch(n_samples=1024, chains_per_sample=16)
    off6, ln6, total6 = F.sample_chains(w6.extra["sample_lens"], 16)
    p6 = torch.from_numpy(w6.payload).to(dev)
    a6 = torch.from_numpy(w6.extra["aad"]).to(dev)
    c6, t6 = F.encrypt_tag_ragged(w6.key, w6.base_iv, off6, ln6, p6, a6)
    o6 = torch.empty_like(c6)
    k6 = torch.empty(off6.size, dtype=torch.uint8, device=dev)
    # 100 untimed calls first: the first calls of this leg also touch freshly allocated
    # table slots and staging (slower for the first ~50 calls on the box)
    rag_ms = time_calls(torch, stream, lambda: F.decrypt_verify_ragged(w6.key, w6.base_iv, off6, ln6, c6, t6, a6,
                                                                      out=o6, ok=k6), 40)
    assert bool(k6.all())
    enc_ms = time_calls(torch, stream, lambda: F.encrypt_tag_ragged(w6.key, w6.base_iv, off6, ln6, p6, a6, out=o6,
                                                                   tags=t6), 40)
    cu, tu = F.encrypt_tag(w6.key, w6.base_iv, 8 * KiB, p6)
    ku = torch.empty(tu.shape[0], dtype=torch.uint8, device=dev)
    uni_ms = time_calls(torch, stream, lambda: F.decrypt_verify(w6.key, w6.base_iv, 8 * KiB, cu, tu, out=o6, ok=ku), 40)
    nbytes = int(ln6.sum())
    res["ragged"] = {"workload": "sample-batch: 1024 samples (log-normal sizes, median 110 KiB) x 16 chains, "
                                 "1-byte serial AAD, %.1f MiB" % (total6 / MiB),
                     "chains": int(off6.size), "decrypt_gbps": round(nbytes / rag_ms / 1e6, 1),
                     "decrypt_us": round(rag_ms * 1e3, 1), "encrypt_gbps": round(nbytes / enc_ms / 1e6, 1),
                     "uniform_8KiB_decrypt_gbps": round(p6.numel() / uni_ms / 1e6, 1)}
    log("ragged:", res["ragged"])
    del p6, a6, c6, t6, o6, k6, cu, tu, ku

    # per-key setup: the first call with a new key (key set-up, tables, 1 MiB decrypt of 16
    # chains), the median over five keys never used before, each call after an idle GPU
    t = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ct1, tg1 = F.encrypt_tag(w1.key, w1.base_iv, 65536, p1)
    o1c = torch.empty_like(ct1)
    k1c = torch.empty(tg1.shape[0], dtype=torch.uint8, device=dev)
    cold = []
    for i in range(5):
        key2 = bytes((7 * i + j) & 255 for j in range(32))
        torch.cuda.synchronize()
        t[0].record(stream)
        F.decrypt_verify(key2, w1.base_iv, 65536, ct1, tg1, out=o1c, ok=k1c)
        t[1].record(stream)
        torch.cuda.synchronize()
        cold.append(t[0].elapsed_time(t[1]) * 1e3)
    res["cold_key_call_us"] = round(sorted(cold)[len(cold) // 2], 1)

    if not args.skip_pipeline:
        res["pipeline_h2d"] = pipeline(F, W, torch, np, dev)
    return res


def aes_formulation(F, W, torch, dev, stream):
    """The two AES formulations on the same keystream (64 MiB of the image-batch key
    and IV, 1 MiB and 64 KiB chains): T-tables in LDS against the bitsliced circuit."""
    w = W.config2()
    form = {}
    ks = torch.empty(64 * MiB, dtype=torch.uint8, device=dev)
    for chain in (MiB, 64 * KiB):
        ref = F.keystream(w.key, w.base_iv, chain, 64 * MiB)
        t_ms = time_calls(torch, stream, lambda: F.keystream(w.key, w.base_iv, chain, 64 * MiB, out=ks), 20)
        b_ms = time_calls(torch, stream, lambda: F.keystream(w.key, w.base_iv, chain, 64 * MiB, out=ks,
                                                            bitsliced=True), 20)
        assert torch.equal(ks, ref), "bitsliced keystream differs from the T-table keystream"
        form["%dKiB" % (chain // KiB)] = {"ttable_us": round(t_ms * 1e3, 1), "bitsliced_us": round(b_ms * 1e3, 1),
                                          "bitsliced_over_ttable": round(b_ms / t_ms, 3)}
    log("aes formulation:", form)
    return {"workload": "64 MiB keystream (no data read)", "by_chain": form}


def hip_runtime_path():
    """The HIP runtime this process already uses (the one torch loaded), so that ctypes
    calls go to the same runtime instance as torch's streams."""
    with open("/proc/self/maps") as f:
        for line in f:
            path = line.split()[-1]
            if os.path.basename(path).startswith("libamdhip64.so"):
                return path
    raise RuntimeError("the HIP runtime is not loaded")


def pipeline(F, W, torch, np, dev):
    length, chain, chunk = 4 * GiB, MiB, 8 * MiB
    # The 4 GiB of seeded bytes of the pipelined workload, generated straight into
    # pinned memory, then encrypted by this library's encrypt + tag (the timed legs
    # never run the CPU oracle; the parity tests check this path against the
    # oracle's own encryption of the same bytes).
    h_pt = torch.empty(length, dtype=torch.uint8, pin_memory=True)
    w5 = W.config5(length, out=h_pt.numpy())
    key, iv = w5.key, w5.base_iv
    h_ct = torch.empty(length, dtype=torch.uint8, pin_memory=True)
    n = F.num_chains(length, chain)
    h_tags = torch.empty((n, 16), dtype=torch.uint8)
    d_pt = h_pt.to(dev)
    del h_pt
    d_ct, d_tags = F.encrypt_tag(key, iv, chain, d_pt)
    h_ct.copy_(d_ct)
    h_tags.copy_(d_tags)
    del d_ct, d_tags
    torch.cuda.synchronize()
    res = {"workload": "uniform-4GiB: 4 GiB of seeded bytes in pinned memory, 1 MiB chains, 8 MiB chunks",
           "input": "the workload's bytes encrypted on the GPU by this library's encrypt+tag (the parity tests "
                    "use the oracle's encryption of the same bytes)"}
    stage = torch.empty(F.stage_bytes(length, chain, 0, chunk, 3), dtype=torch.uint8, device=dev)
    out = torch.empty(length, dtype=torch.uint8, device=dev)
    ok = torch.empty(n, dtype=torch.uint8, device=dev)
    cs, ks, vs = torch.cuda.Stream(), torch.cuda.Stream(), torch.cuda.Stream()
    def timed_s(fn, streams, reps=3):
        # one untimed pass, then `reps` timed passes (host clock, all streams the pass
        # uses drained), sorted
        fn()
        torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            fn()
            for st in streams:
                st.synchronize()
            ts.append(time.perf_counter() - t0)
        return sorted(ts)

    median_s = lambda fn, streams: timed_s(fn, streams)[1]   # the pipelines: median of three
    best_s = lambda fn, streams: timed_s(fn, streams, 5)[0]  # the copy ceiling: the best of five

    for name, mode, depth in (("depth0", 0, 0), ("depth2", 0, 2), ("depth3", 0, 3), ("eager_depth2", 1, 2),
                              ("otp_depth2", 2, 2), ("direct", 3, 0)):
        run = lambda: F.pipeline_h2d(key, iv, chain, h_ct, h_tags, None, chunk, depth, stage, out, ok, cs, ks,
                                     mode=mode, verify_stream=vs)
        ok.zero_()
        out.zero_()
        dt = median_s(run, (ks, vs, cs))
        assert bool(ok.all()) and torch.equal(out, d_pt), "pipeline produced wrong output"
        res["%s_gbps" % name] = round(length / dt / 1e9, 2)
        log("pipeline %s: %.2f GB/s" % (name, length / dt / 1e9))
    # D2H: encrypt + tag of the same 4 GiB on the device, copied out chunk by chunk
    h_out = torch.empty(length, dtype=torch.uint8, pin_memory=True)
    h_tg = torch.empty((n, 16), dtype=torch.uint8, pin_memory=True)
    d_ctb = torch.empty_like(d_pt)
    d_tg = torch.empty((n, 16), dtype=torch.uint8, device=dev)
    for name, mode in (("d2h", F.PIPE_FUSED), ("d2h_direct", F.PIPE_DIRECT)):
        h_out.zero_()
        dt = median_s(lambda: F.pipeline_d2h(key, iv, chain, d_pt, chunk_bytes=chunk, out=d_ctb, tags=d_tg,
                                             h_ct=h_out, h_tags=h_tg, copy_stream=cs, compute_stream=ks, mode=mode),
                      (cs, ks))
        assert torch.equal(h_out, h_ct) and torch.equal(h_tg, h_tags), "%s produced wrong ciphertext" % name
        res["%s_gbps" % name] = round(length / dt / 1e9, 2)
        log("pipeline %s: %.2f GB/s" % (name, res["%s_gbps" % name]))
    # plain pinned copies of the same bytes in the same chunks on one stream, through
    # the runtime's hipMemcpyAsync (the copy engine's rate, nothing else enqueued); the
    # ceiling the pipelines are compared with is the best of five passes
    hip = ctypes.CDLL(hip_runtime_path())
    hip.hipMemcpyAsync.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int, ctypes.c_void_p]
    hip.hipMemcpyAsync.restype = ctypes.c_int

    def copies(dst, src, kind):
        for off in range(0, length, chunk):
            assert hip.hipMemcpyAsync(dst + off, src + off, chunk, kind, cs.cuda_stream) == 0

    dt = best_s(lambda: copies(h_out.data_ptr(), d_ctb.data_ptr(), 2), (cs,))
    res["pinned_copy_d2h_gbps"] = round(length / dt / 1e9, 2)
    res["d2h_ratio_vs_copy"] = round(res["d2h_gbps"] / res["pinned_copy_d2h_gbps"], 3)
    res["d2h_direct_ratio_vs_copy"] = round(res["d2h_direct_gbps"] / res["pinned_copy_d2h_gbps"], 3)
    log("pinned d2h copy %.2f GB/s" % res["pinned_copy_d2h_gbps"])
    del h_out, d_ctb, d_tg
    dt = best_s(lambda: copies(out.data_ptr(), h_ct.data_ptr(), 1), (cs,))
    res["pinned_copy_gbps"] = round(length / dt / 1e9, 2)
    best = max(res["depth0_gbps"], res["depth2_gbps"], res["depth3_gbps"])
    res["ratio_vs_copy"] = round(best / res["pinned_copy_gbps"], 3)
    res["direct_ratio_vs_copy"] = round(res["direct_gbps"] / res["pinned_copy_gbps"], 3)
    log("pinned copy %.2f GB/s" % res["pinned_copy_gbps"])
    del stage, out, ok, h_ct, d_pt
    torch.cuda.empty_cache()
    return res


def cpu_baseline(W, np, cases, w):
    import oracle
    # the oracle decrypts the same image batch at every chain size of the sweep
    total = 0
    t0 = time.perf_counter()
    host = [(chain, ct.cpu().numpy(), tags.cpu().numpy(), aad.cpu().numpy()) for chain, ct, tags, aad, out, ok in cases]
    passes = 2
    for _ in range(passes):
        for chain, c, t, a in host:
            s = time.perf_counter()
            _, okc = oracle.chains_decrypt(w.key, w.base_iv, chain, c, t, a, 32)
            total += time.perf_counter() - s
            assert okc.all()
    nbytes = passes * sum(ct.numel() for _, ct, *_ in cases)
    log("cpu oracle %.3f GB/s (%.1f s)" % (nbytes / total / 1e9, time.perf_counter() - t0))
    # the same oracle on one thread (64 KiB chains), and encrypt + tag on every thread
    chain, c, t, a = host[2]
    s = time.perf_counter()
    _, okc = oracle.chains_decrypt(w.key, w.base_iv, chain, c, t, a, 32, nthreads=1)
    one = c.size / (time.perf_counter() - s) / 1e9
    assert okc.all()
    s = time.perf_counter()
    oracle.chains_encrypt(w.key, w.base_iv, chain, w.payload, a, 32)
    enc = w.payload.size / (time.perf_counter() - s) / 1e9
    log("cpu oracle one thread %.4f GB/s, encrypt %.3f GB/s" % (one, enc))
    return {"value": round(nbytes / total / 1e9, 4), "unit": "GB/s", "cores": oracle.max_threads(), "kind": "oracle",
            "sample": "the 64 MiB image batch decrypted + verified at all 5 chain sizes, twice (640 MiB), OpenMP over chains",
            "one_thread_gbps": round(one, 4), "encrypt_gbps": round(enc, 4),
            "one_thread_sample": "the same batch at 64 KiB chains, decrypted + verified on one thread",
            "encrypt_sample": "the same batch encrypted + tagged at 64 KiB chains, every thread"}


if __name__ == "__main__":
    main()
