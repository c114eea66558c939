#!/usr/bin/env python3
"""Benchmark of the triangular multiplicative update on one MI355X.

One step = one layer = the outgoing (Eq. 2) and the incoming (Eq. 3) update
of a seeded N x N x 128 bf16 pair tensor resident in HBM (N = 4096 by
default), each through the library's three kernels K1 projection -> K2
contraction -> K3 epilogue (exactly the launches tri_mul_outgoing /
tri_mul_incoming make), with HIP events between the kernels so that every
kernel's duration is measured inside the timed region on the stream it runs
on.

Prints one JSON line.  `value` is the layer throughput in TFLOP/s
(algorithmic flops of both directions / wall time of the step); the
roofline object reports the contraction kernel against the bf16 MFMA peak.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)


def cpu_baseline(N, sample):
    """The fp64 oracle (as it stands) timed on host cores on a bounded sample
    of the same workload, extrapolated per stage to the whole layer.

    Sample: one direction (outgoing) for a `sample` x `sample` block of output
    pairs of the N = 4096 problem: the projections of 2 x sample x N pairs,
    the contraction of sample^2 pairs over all N tokens and 128 channels, and
    the epilogue of sample^2 pairs.  Each stage's measured cost per unit
    (pair, pair x token) is scaled to the full layer (2 directions)."""
    import ctypes

    import numpy as np

    import oracle
    from paper_2603_14806_amd import perf, synth
    try:   # keep freed heap memory mapped: first-touch page faults otherwise dominate numpy's temporaries
        libc = ctypes.CDLL("libc.so.6")
        libc.mallopt(-3, 1 << 30)    # M_MMAP_THRESHOLD
        libc.mallopt(-1, 1 << 62)    # M_TRIM_THRESHOLD
    except Exception:
        pass
    try:
        from threadpoolctl import threadpool_info
        cores = max([p.get("num_threads", 1) for p in threadpool_info() if p.get("user_api") == "blas"] or [1])
    except Exception:
        cores = os.cpu_count()
    W = {k: oracle.f64(v) for k, v in synth.weights(dtype="bf16").items()}
    rows = synth.pair_tensor(N, dtype="bf16", shape=(2 * sample, N, 128))  # stand-in z rows, same law
    mask_rows = np.ones((2 * sample, N))
    t0 = time.perf_counter()
    a, _, _ = oracle.project(rows[:sample], mask_rows[:sample], W)
    _, b, _ = oracle.project(rows[sample:], mask_rows[sample:], W)
    t1 = time.perf_counter()
    C = oracle.contract_outgoing(a, b)
    t2 = time.perf_counter()
    zb = oracle.f64(rows[:sample, :sample])
    m = np.ones((sample, sample))
    _, _, g = oracle.project(zb, m, W)
    oracle.epilogue(C, g, m, W)
    t3 = time.perf_counter()
    per_pair_proj = (t1 - t0) / (2 * sample * N)
    per_pair_token = (t2 - t1) / (sample * sample * N)
    per_pair_epi = (t3 - t2) / (sample * sample)
    # full direction: projections of N^2 pairs, contraction over N^3, epilogue N^2
    t_dir = per_pair_proj * N * N + per_pair_token * N ** 3 + per_pair_epi * N * N
    f = perf.flops(N)["total"]
    return {"value": round(2 * f / (2 * t_dir) / 1e12, 6), "unit": "TFLOP/s", "cores": int(cores),
            "kind": "oracle", "nproc": os.cpu_count(), "cpu_model": cpu_model(),
            "implementation": "the fp64 numpy oracle (oracle/trimul.py) as it stands; its matrix products run "
                              "in the BLAS library numpy links, on `cores` threads",
            "sample": (f"outgoing update of a {sample}x{sample} block of output pairs at N={N} (c_z=c=128, fp64): "
                       f"projections of {2 * sample}x{N} pairs, contraction over {N} tokens, epilogue; "
                       f"measured {t3 - t0:.1f} s, per-stage cost extrapolated to both directions of the layer "
                       f"({2 * t_dir:.0f} s per layer)"),
            "sample_seconds": round(t3 - t0, 2)}


def cpu_model():
    """The host CPU's model name from /proc/cpuinfo (None if unreadable)."""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


class ClockSampler:
    """Samples the GPU's current graphics clock (the DPM level the amdgpu
    sysfs file marks as current) every `period` seconds on a host thread, for
    the clock-adjusted MFMA fraction.  Plain file reads, no GPU calls."""

    def __init__(self, period=0.02):
        import glob
        import threading
        self.period, self.samples, self._stop = period, [], threading.Event()
        devs = sorted(d for d in glob.glob("/sys/class/drm/card*/device") if os.path.exists(d + "/pp_dpm_sclk"))
        self.path = devs[0] + "/pp_dpm_sclk" if devs else None
        self._th = threading.Thread(target=self._run, daemon=True)

    def _read(self):
        for line in open(self.path):
            if line.rstrip().endswith("*"):
                return float(line.split(":", 1)[1].replace("*", "").strip().lower().replace("mhz", ""))
        return None

    def _run(self):
        while not self._stop.is_set():
            try:
                v = self._read()
                if v:
                    self.samples.append(v)
            except (OSError, ValueError):
                return
            self._stop.wait(self.period)

    def __enter__(self):
        if self.path:
            self._th.start()
        return self

    def __exit__(self, *exc):
        self._stop.set()
        if self.path:
            self._th.join()

    def summary(self):
        if not self.samples:
            return None
        v = sorted(self.samples)
        return {"mean_MHz": round(sum(v) / len(v), 1), "min_MHz": v[0], "max_MHz": v[-1], "samples": len(v)}

    def adjusted_basis(self, min_samples=10):
        """The mean clock for the clock-adjusted fraction, or None when the
        timed region was too short for a steady reading (a one-step run
        catches the clock still ramping and would overstate the fraction)."""
        c = self.summary()
        return None if c is None or c["samples"] < min_samples else c


def gpu_state():
    """Current graphics and memory clocks (and socket power, where exposed) of
    the first GPU, read from the amdgpu sysfs files -- plain file reads, no
    child process.  None where the files are missing or unreadable."""
    import glob

    def current(path):   # the DPM level marked '*', e.g. '1: 2100Mhz *'
        for line in open(path):
            if line.rstrip().endswith("*"):
                return line.split(":", 1)[1].replace("*", "").strip()
        return None

    try:
        dev = sorted(d for d in glob.glob("/sys/class/drm/card*/device") if os.path.exists(d + "/pp_dpm_sclk"))[0]
        out = {"sclk": current(dev + "/pp_dpm_sclk"), "mclk": current(dev + "/pp_dpm_mclk")}
        pw = glob.glob(dev + "/hwmon/hwmon*/power1_average") + glob.glob(dev + "/hwmon/hwmon*/power1_input")
        if pw:
            out["power_W"] = round(int(open(pw[0]).read()) / 1e6, 1)
        return out
    except (IndexError, OSError, ValueError):
        return None


def cpu_oracle_extras(timings):
    """The fp64 oracle on bounded samples of the untimed extras' workloads,
    extrapolated to the full workloads (each sample a few seconds):
    - layer backward: the whole update backward at N = 128 (outgoing, all
      pairs), scaled by the ratio of the flop counts of N = 4096 and N = 128;
    - outer product mean: a 128 x 128 block of pairs over all S = 4096
      sequences of the S = 4096, N = 1024 problem, scaled by the pair count;
    - triangle attention: four rows i (all 2048 queries, 4 heads) of the
      rows = n = 2048 problem, scaled by the row count."""
    import numpy as np

    import oracle
    from paper_2603_14806_amd import perf, synth
    rng = np.random.default_rng(synth.SEED)
    out = {}
    if "backward_layer" in timings:
        n = 128
        W = {k: oracle.f64(v) for k, v in synth.weights(dtype="bf16").items()}
        z, dout = rng.standard_normal((n, n, 128)), rng.standard_normal((n, n, 128))
        t0 = time.perf_counter()
        oracle.tri_mul_backward(z, np.ones(n), W, "outgoing", dout)
        t = time.perf_counter() - t0
        ms = 1e3 * t * perf.flops(4096)["total"] / perf.flops(n)["total"]
        out["backward_layer"] = {"ms_extrapolated": round(ms, 1), "sample_seconds": round(t, 2),
                                 "sample": f"tri_mul_backward (fp64) of the whole update at N={n}, scaled by the "
                                           f"flop ratio of N=4096 to N={n}"}
    if "outer_product_mean" in timings:
        S, n, blk = 4096, 1024, 128
        # the block's tokens only: the tile [0, blk) x [0, blk) reads nothing else
        a, b = rng.standard_normal((S, blk, 32)), rng.standard_normal((S, blk, 32))
        w = rng.standard_normal((128, 1024)) / 32
        t0 = time.perf_counter()
        oracle.outer_product_mean_tile(a, b, None, w, np.zeros(128), 0, blk, 0, blk)
        t = time.perf_counter() - t0
        out["outer_product_mean"] = {"ms_extrapolated": round(1e3 * t * (n / blk) ** 2, 1),
                                     "sample_seconds": round(t, 2),
                                     "sample": f"outer_product_mean_tile (fp64), a {blk}x{blk} block of pairs over "
                                               f"all S={S} sequences, scaled by the pair count ({(n // blk) ** 2}x)"}
        del a, b
    if "triangle_attention" in timings:
        n, H, rows = 2048, 4, 4
        q, k, v = (rng.standard_normal((rows, n, H, 32)) for _ in range(3))
        bias = rng.standard_normal((H, n, n))
        t0 = time.perf_counter()
        oracle.triangle_attention(q, k, v, bias, None)
        t = time.perf_counter() - t0
        out["triangle_attention"] = {"ms_extrapolated": round(1e3 * t * n / rows, 1), "sample_seconds": round(t, 2),
                                     "sample": f"triangle_attention (fp64) of {rows} rows (all {n} queries, {H} "
                                               f"heads), scaled by the row count ({n // rows}x)"}
    return out


def stream_reference(dev, gib=1, reps=5):
    """What plain streaming reaches on this GPU in this run: torch's copy of
    one buffer into another and its add of two buffers into a third, each
    buffer `gib` GiB of fp32, best of `reps` (HIP events).  Context for the
    HBM fractions of the projection and the epilogue, measured outside the
    timed region."""
    import torch
    n = int(gib * (1 << 30)) // 4
    x = torch.ones(n, device=dev)
    y = torch.ones(n, device=dev)
    z = torch.empty(n, device=dev)
    out = {}
    for name, fn, nbytes in (("copy", lambda: z.copy_(x), 8 * n), ("add", lambda: torch.add(x, y, out=z), 12 * n)):
        fn()
        best = None
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            e1.synchronize()
            ms = e0.elapsed_time(e1)
            best = ms if best is None else min(best, ms)
        out[f"{name}_GB_per_s"] = round(nbytes / (best * 1e-3) / 1e9, 1)
    del x, y, z
    torch.cuda.empty_cache()
    out["what"] = (f"torch copy (read + write) and add (two reads + one write) over {gib} GiB fp32 buffers, "
                   f"best of {reps}, outside the timed region; frac_of_stream = achieved / the better of the two")
    return out


def measured_traffic():
    """HBM-side bytes per K2 launch from the committed rocprofv3 counter runs
    (FETCH_SIZE and WRITE_SIZE, each scaled by a plain copy of known size),
    valid only while the contraction kernel source is the one measured."""
    import hashlib
    try:
        rec = json.load(open(os.path.join(ROOT, "profiles", "k2_contract_traffic.json")))
        csrc = os.path.join(ROOT, "paper_2603_14806_amd", "csrc")
        src = b"".join(open(os.path.join(csrc, f), "rb").read() for f in ("contract.hip", "common.h", "k2_addr.h"))
        if hashlib.sha256(src).hexdigest() == rec["source_sha256"]:
            return rec["traffic_bytes_per_launch"]
    except (OSError, KeyError, ValueError):
        pass
    return None


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--N", type=int, default=4096)
    ap.add_argument("--cpu-sample", type=int, default=128)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the untimed extras (the N=2048 workload, backward passes, outer product mean, "
                         "triangle attention, ring tile), e.g. for profiling runs that attribute the kernels' "
                         "statistics to the timed N=4096 layer alone")
    ap.add_argument("--copy-calibration", type=float, default=0.0,
                    help="GiB moved by one plain device-to-device copy before the run (HBM counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}): the library has no multi-GPU path; "
              "one device's tile of a sharded run is timed by the ring_tile field (tile (7,7) of an 8x8 grid at N=30000).", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2603_14806_amd import perf, synth
    from paper_2603_14806_amd import trimul as T

    N = args.N
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.copy_calibration > 0:
        n = int(args.copy_calibration * (1 << 30)) // 4
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        print(f"[bench] calibration copy of {4 * n} bytes done", file=sys.stderr, flush=True)
        del src, dst
    print(f"[bench] N={N} steps={args.steps} warmup={args.warmup}", file=sys.stderr, flush=True)
    layer = T.TriMul(synth.weights(dtype="bf16"), dtype="bf16", out_dtype="f32")
    z = synth.pair_tensor(N, dtype="bf16", device=dev)
    mask = synth.token_mask(N, 0, device=dev)
    npanel = T.tri_mul_panel_size(layer.h, N) // 2
    A = torch.empty(npanel, dtype=torch.bfloat16, device=dev)
    B = torch.empty_like(A)
    C = torch.empty(N * (-(-N // 32) * 32) * 128, dtype=torch.float32, device=dev)   # result layout
    outs = [torch.empty((N, N, 128), dtype=torch.float32, device=dev) for _ in range(2)]
    stream = torch.cuda.current_stream()
    h = layer.h
    OPPOSITE = {T.TRI_MUL_OUTGOING: T.TRI_MUL_INCOMING, T.TRI_MUL_INCOMING: T.TRI_MUL_OUTGOING}

    # The three kernels of the full calls, in their order: the projection
    # with the opposite direction's pair indexing writes the direction's
    # operands transposed, which the contraction reads transposed
    # (tri_mul_contract_transposed; bitwise the same C as the plain order).
    def step(evs):
        for d, direction in enumerate((T.TRI_MUL_OUTGOING, T.TRI_MUL_INCOMING)):
            e = [torch.cuda.Event(enable_timing=True) for _ in range(4)] if evs is not None else None
            if e: e[0].record(stream)
            T.tri_mul_project(h, z, mask, N, OPPOSITE[direction], A, B, stream)
            if e: e[1].record(stream)
            T.tri_mul_contract_transposed(h, A, B, N, C, stream)
            if e: e[2].record(stream)
            T.tri_mul_epilogue(h, C, z, mask, N, outs[d], stream)
            if e: e[3].record(stream)
            if e: evs.append(e)

    state_before = gpu_state()
    for _ in range(args.warmup):
        step(None)
    torch.cuda.synchronize()
    print("[bench] warmup done", file=sys.stderr, flush=True)

    evs = []
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    with ClockSampler() as clocks:
        t0.record(stream)
        for _ in range(args.steps):
            step(evs)
        t1.record(stream)
        torch.cuda.synchronize()
    ms_step = t0.elapsed_time(t1) / args.steps
    k_ms = {name: sum(e[i].elapsed_time(e[i + 1]) for e in evs) / len(evs)
            for i, name in enumerate(("project", "contract", "epilogue"))}
    per_step = sorted(evs[2 * i][0].elapsed_time(evs[2 * i + 1][3]) for i in range(args.steps))
    step_median = per_step[len(per_step) // 2] if len(per_step) % 2 else \
        0.5 * (per_step[len(per_step) // 2 - 1] + per_step[len(per_step) // 2])
    print(f"[bench] timed {args.steps} steps: {ms_step:.3f} ms/layer; per kernel {k_ms}", file=sys.stderr, flush=True)

    # the full entry points (one call = the same three launches), outside the timed region
    ws, need = layer.workspace(N)
    f0, f1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    f0.record(stream)
    for _ in range(2):
        T.tri_mul_outgoing(h, z, mask, N, outs[0], ws, need, stream)
        T.tri_mul_incoming(h, z, mask, N, outs[1], ws, need, stream)
    f1.record(stream)
    torch.cuda.synchronize()
    full_ms = f0.elapsed_time(f1) / 2
    stream_ref = stream_reference(dev)
    print(f"[bench] plain streams: {stream_ref}", file=sys.stderr, flush=True)
    best_stream = max(stream_ref["copy_GB_per_s"], stream_ref["add_GB_per_s"])

    # the N = 2048 workload with channel-scaled z (s_c ~ U(0.5, 2)), both
    # directions through the three kernels, outside the timed region
    c3 = None
    if N != 2048 and not args.no_extras:
        N3 = 2048
        z3 = synth.pair_tensor(N3, dtype="bf16", scale=synth.channel_scale(), device=dev)
        np3 = T.tri_mul_panel_size(h, N3) // 2
        A3, B3 = A[:np3], B[:np3]
        C3 = C[:N3 * (-(-N3 // 32) * 32) * 128]
        o3 = outs[0].view(-1)[:N3 * N3 * 128].view(N3, N3, 128)
        ev3 = {}
        for direction, code in (("outgoing", T.TRI_MUL_OUTGOING), ("incoming", T.TRI_MUL_INCOMING)):
            for _ in range(2):   # warm-up
                T.tri_mul_project(h, z3, None, N3, OPPOSITE[code], A3, B3, stream)
                T.tri_mul_contract_transposed(h, A3, B3, N3, C3, stream)
                T.tri_mul_epilogue(h, C3, z3, None, N3, o3, stream)
            es = []
            for _ in range(5):
                e = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
                e[0].record(stream)
                T.tri_mul_project(h, z3, None, N3, OPPOSITE[code], A3, B3, stream)
                e[1].record(stream)
                T.tri_mul_contract_transposed(h, A3, B3, N3, C3, stream)
                e[2].record(stream)
                T.tri_mul_epilogue(h, C3, z3, None, N3, o3, stream)
                e[3].record(stream)
                es.append(e)
            ev3[direction] = es
        torch.cuda.synchronize()
        fl3 = perf.flops(N3)
        c3 = {"what": "N=2048, z_ijc = s_c n_ijc with s_c ~ U(0.5, 2) per pair channel, n ~ N(0,1), all-ones mask, "
                      "bf16 storage, fp32 output; each direction through K1 -> K2 -> K3, 2 warm-up + 5 timed "
                      "calls; not part of ms_per_step"}
        for direction, es in ev3.items():
            k = [sum(e[i].elapsed_time(e[i + 1]) for e in es) / len(es) for i in range(3)]
            tot = sum(e[0].elapsed_time(e[3]) for e in es) / len(es)
            c3[direction] = {"ms": round(tot, 4), "TFLOP_per_s": round(fl3["total"] / (tot * 1e-3) / 1e12, 2),
                             "project_ms": round(k[0], 4), "contract_ms": round(k[1], 4),
                             "epilogue_ms": round(k[2], 4),
                             "contract_TFLOP_per_s": round(fl3["contract"] / (k[1] * 1e-3) / 1e12, 2)}
        c3["ms_per_layer"] = round(c3["outgoing"]["ms"] + c3["incoming"]["ms"], 4)
        del z3
        print(f"[bench] N=2048 channel-scaled layer {c3['ms_per_layer']:.3f} ms", file=sys.stderr, flush=True)

    bwd_ms = lbwd_ms = sbwd_ms = opm_ms = ta_ms = tile_ms = tile_pk_ms = tile_ws_ms = None
    ta_scores = 2048 * 4 * 2048 * 2048
    opm_flops = 2 * 4096 * (1024 * 32) ** 2
    if not args.no_extras:
        # the contraction backward (training), outside the timed region: both
        # gradients of one direction, with C standing in for dC
        dA, dB = torch.empty_like(C), torch.empty_like(C)
        bws_n = T.tri_mul_contract_backward_workspace_size(h, N)
        bws = torch.empty(bws_n, dtype=torch.uint8, device=dev)
        for _ in range(2):   # warm-up (clocks settle over the first calls)
            T.tri_mul_contract_backward(h, C, A, B, N, dA, dB, bws, bws_n, stream)
        b0, b1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        b0.record(stream)
        for _ in range(3):
            T.tri_mul_contract_backward(h, C, A, B, N, dA, dB, bws, bws_n, stream)
        b1.record(stream)
        torch.cuda.synchronize()
        bwd_ms = b0.elapsed_time(b1) / 3
        del dA, dB, bws
        print(f"[bench] contraction backward {bwd_ms:.3f} ms", file=sys.stderr, flush=True)

        # the whole layer backward (outgoing), outside the timed region: dz and
        # all weight gradients for an upstream gradient dout ~ N(0,1)
        dout = synth.pair_tensor(N, dtype="f32", device=dev, name="dout")
        dz = torch.empty_like(z)
        grads = {k: torch.empty(v, dtype=torch.float32, device=dev) for k, v in T.WEIGHT_SHAPES.items()}
        lws_n = T.tri_mul_backward_workspace_size(h, N)
        lws = torch.empty(lws_n, dtype=torch.uint8, device=dev)
        T.tri_mul_layer_backward(h, "outgoing", z, mask, N, dout, dz, grads, lws, lws_n, stream)
        l0, l1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        l0.record(stream)
        for _ in range(2):
            T.tri_mul_layer_backward(h, "outgoing", z, mask, N, dout, dz, grads, lws, lws_n, stream)
        l1.record(stream)
        torch.cuda.synchronize()
        lbwd_ms = l0.elapsed_time(l1) / 2
        print(f"[bench] layer backward {lbwd_ms:.3f} ms", file=sys.stderr, flush=True)
        # the same backward from the forward's saved A, B, C (training keeps them)
        T.tri_mul_project(h, z, mask, N, T.TRI_MUL_INCOMING, A, B, stream)   # the outgoing operands transposed
        T.tri_mul_contract_transposed(h, A, B, N, C, stream)
        T.tri_mul_layer_backward_saved(h, "outgoing", z, mask, N, A, B, C, dout, dz, grads, lws, lws_n, stream)
        l0.record(stream)
        for _ in range(2):
            T.tri_mul_layer_backward_saved(h, "outgoing", z, mask, N, A, B, C, dout, dz, grads, lws, lws_n, stream)
        l1.record(stream)
        torch.cuda.synchronize()
        sbwd_ms = l0.elapsed_time(l1) / 2
        del dout, dz, grads, lws
        print(f"[bench] layer backward from saved forward {sbwd_ms:.3f} ms", file=sys.stderr, flush=True)

        # the outer product mean (a second op of the same ring archetype), outside
        # the timed region: S = 4096 sequences, N = 1024 tokens, D = 32, c_z = 128
        oS, oN = 4096, 1024
        og = torch.Generator(device=dev).manual_seed(synth.SEED)
        oa = torch.randn((oS, oN, 32), generator=og, device=dev).to(torch.bfloat16)
        ob = torch.randn((oS, oN, 32), generator=og, device=dev).to(torch.bfloat16)
        ow = (torch.randn((128, 1024), generator=og, device=dev) / 32).to(torch.bfloat16)
        opm = T.OuterProductMean(ow, None, out_dtype="f32")
        oout = torch.empty((oN, oN, 128), device=dev)
        ows_n = T.opm_forward_workspace_size(opm.h, oS, oN)
        ows = torch.empty(ows_n, dtype=torch.uint8, device=dev)
        for _ in range(3):   # warm-up (clocks settle over the first calls)
            T.opm_forward(opm.h, oa, ob, None, oS, oN, oout, ows, ows_n, stream)
        o0, o1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        o0.record(stream)
        for _ in range(3):
            T.opm_forward(opm.h, oa, ob, None, oS, oN, oout, ows, ows_n, stream)
        o1.record(stream)
        torch.cuda.synchronize()
        opm_ms = o0.elapsed_time(o1) / 3
        del oa, ob, oout, ows
        opm.close()
        print(f"[bench] outer product mean {opm_ms:.3f} ms", file=sys.stderr, flush=True)

        # the triangle attention core (rows = n = 2048, 4 heads of 32), outside the timed region
        tn, tH = 2048, 4
        tq = torch.randn((tn, tn, tH, 32), generator=og, device=dev).to(torch.bfloat16)
        tk = torch.randn((tn, tn, tH, 32), generator=og, device=dev).to(torch.bfloat16)
        tv = torch.randn((tn, tn, tH, 32), generator=og, device=dev).to(torch.bfloat16)
        tb = torch.randn((tH, tn, tn), generator=og, device=dev).to(torch.bfloat16)
        tout = torch.empty((tn, tn, tH, 32), device=dev)
        for _ in range(3):   # warm-up (clocks settle over the first calls)
            T.tri_attn_forward(tq, tk, tv, tb, None, tn, tn, tH, tn, "f32", tout, stream)
        a0, a1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a0.record(stream)
        for _ in range(3):
            T.tri_attn_forward(tq, tk, tv, tb, None, tn, tn, tH, tn, "f32", tout, stream)
        a1.record(stream)
        torch.cuda.synchronize()
        ta_ms = a0.elapsed_time(a1) / 3
        # the same with bf16 output (the probabilities enter the PV product as bf16 alone)
        tout16 = torch.empty((tn, tn, tH, 32), dtype=torch.bfloat16, device=dev)
        T.tri_attn_forward(tq, tk, tv, tb, None, tn, tn, tH, tn, "bf16", tout16, stream)
        a0.record(stream)
        for _ in range(3):
            T.tri_attn_forward(tq, tk, tv, tb, None, tn, tn, tH, tn, "bf16", tout16, stream)
        a1.record(stream)
        torch.cuda.synchronize()
        ta16_ms = a0.elapsed_time(a1) / 3
        del tq, tk, tv, tb, tout, tout16
        print(f"[bench] triangle attention {ta_ms:.3f} ms (bf16 output {ta16_ms:.3f} ms)", file=sys.stderr, flush=True)

        # one device's share of the paper's 2-D ring, outside the timed region:
        # tile (7, 7) of an 8 x 8 grid at N = 30000 (3750 x 3750 pairs, the last
        # 300 tokens padded), 8 ring steps of block_accumulate over 3750-token
        # k-panels, the last running the epilogue.  Two panel pairs alternate
        # (3.6 GB each, far beyond any cache, so every step streams its panels
        # from HBM as 8 distinct ones would).
        bn, bg = 30000, 8
        bb = bn // bg
        brow, bld = 7 * bb, (bb + 7) // 8 * 8
        bmask = synth.token_mask(bn, 300, device=dev)
        bpa = [synth.pair_tensor(0, dtype="bf16", device=dev, name="a_panel", seed=synth.SEED + p,
                                 shape=(128, bb, bld)) for p in range(2)]
        bpb = [synth.pair_tensor(0, dtype="bf16", device=dev, name="b_panel", seed=synth.SEED + p,
                                 shape=(128, bb, bld)) for p in range(2)]
        bz = synth.pair_tensor(0, dtype="bf16", device=dev, name="z_tile", shape=(bb, bb, 128))
        bacc = torch.empty((128, bb, bb), dtype=torch.float32, device=dev)
        bout = torch.empty((bb, bb, 128), dtype=torch.float32, device=dev)
        tws = torch.empty(layer.block_workspace_size(T.BlockView(bn, brow, brow, bb, bb, 0, bb, bld, bld, 0, bg)),
                          dtype=torch.uint8, device=dev)

        bviews = [T.BlockView(bn, brow, brow, bb, bb, p * bb, bb, bld, bld, p, bg) for p in range(bg)]

        def ring_tile_ws():   # one stream: repack, contraction, (epilogue) per step
            for p in range(bg):
                layer.block_accumulate(bviews[p], bpa[p & 1], bpb[p & 1], bacc, bmask, bz, bout, stream, ws=tws)

        # the pipelined ring step: panel p + 1 repacked on a second stream while
        # panel p is contracted (on 32 fewer compute units) into the packed
        # accumulator; two workspaces, ordered by events
        tws2 = torch.empty_like(tws)
        pacc = torch.empty(layer.block_accumulator_size(bviews[0]) // 4, dtype=torch.float32, device=dev)
        side = torch.cuda.Stream()

        def ring_tile():
            packed = [torch.cuda.Event() for _ in range(bg)]
            done = [torch.cuda.Event() for _ in range(bg)]
            wss = (tws, tws2)
            layer.block_repack(bviews[0], bpa[0], bpb[0], bmask, wss[0], stream)
            packed[0].record(stream)
            side.wait_stream(stream)
            for p in range(bg):
                if p + 1 < bg:
                    if p >= 1:
                        side.wait_event(done[p - 1])
                    layer.block_repack(bviews[p + 1], bpa[(p + 1) & 1], bpb[(p + 1) & 1], bmask, wss[(p + 1) % 2],
                                       side)
                    packed[p + 1].record(side)
                stream.wait_event(packed[p])
                layer.block_accumulate_packed(bviews[p], wss[p % 2], pacc, bmask, bz, bout,
                                              reserve_cus=32 if p + 1 < bg else 0, stream=stream)
                done[p].record(stream)
            stream.wait_stream(side)

        # the ring with the panels in the contraction's blocked layout: the
        # device projects its own tile (the a and b panels of k-block 7 it
        # contributes to the ring) and contracts the eight panel pairs as they
        # arrive, with no repack; the other seven pairs alternate between two
        # projected tiles (made before the timed calls, as a ring delivers them)
        # The same ring in the transposed operand order (every device projects
        # its tile with the opposite direction's pair indexing, the steps read
        # both panels transposed: bitwise the same sums, the faster order) is
        # the timed one; the plain order is reported beside it.
        n_bp = layer.block_panel_size(bb, bb) // 2
        own = [torch.empty(n_bp, dtype=torch.bfloat16, device=dev) for _ in range(2)]
        arrived, arrived_t = [], []
        for p in range(2):
            zt = synth.pair_tensor(0, dtype="bf16", device=dev, name="z_tile", seed=synth.SEED + 1 + p,
                                   shape=(bb, bb, 128))
            arrived.append(layer.block_project(zt, bmask, bn, brow, p * bb, "outgoing"))
            arrived_t.append(layer.block_project(zt, bmask, bn, brow, p * bb, "incoming"))
            del zt

        def ring_tile_blocked():
            T.tri_mul_block_project(layer.h, bz, bb, bmask, bn, brow, brow, bb, bb, T.TRI_MUL_OUTGOING,
                                    own[0], own[1], stream)
            for p in range(bg):
                a_, b_ = own if p == bg - 1 else arrived[p & 1]
                layer.block_accumulate_blocked(bviews[p], a_, b_, pacc, bmask, bz, bout, stream=stream)

        def ring_tile_transposed():
            T.tri_mul_block_project(layer.h, bz, bb, bmask, bn, brow, brow, bb, bb, T.TRI_MUL_INCOMING,
                                    own[0], own[1], stream)
            for p in range(bg):
                a_, b_ = own if p == bg - 1 else arrived_t[p & 1]
                layer.block_accumulate_transposed(bviews[p], a_, b_, pacc, bmask, bz, bout, stream=stream)

        def time_ring(fn):
            fn()
            t0e, t1e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            t0e.record(stream)
            for _ in range(2):
                fn()
            t1e.record(stream)
            torch.cuda.synchronize()
            return t0e.elapsed_time(t1e) / 2

        tile_ms = time_ring(ring_tile_transposed)
        tile_plain_ms = time_ring(ring_tile_blocked)
        tile_pk_ms = time_ring(ring_tile)
        tile_ws_ms = time_ring(ring_tile_ws)
        del bpa, bpb, bz, bacc, bout, tws, tws2, pacc, own, arrived, arrived_t
        torch.cuda.empty_cache()
        print(f"[bench] ring tile {tile_ms:.3f} ms (plain operand order {tile_plain_ms:.3f} ms; "
              f"row-major panels: pipelined repack {tile_pk_ms:.3f} ms, "
              f"one-stream repacking entry point {tile_ws_ms:.3f} ms)", file=sys.stderr, flush=True)

    fl = perf.flops(N)
    by = perf.bytes_moved(N)
    bw = perf.backward_layer_work(N)
    bws_ = perf.backward_layer_work(N, recompute=False)
    opm_proj_flops = 2 * 1024 * 1024 * 1024 * 128
    tile_flops = 2.0 * 3750 * 3750 * 30000 * 128

    def mfma_roof(flop, ms):
        a = flop / (ms * 1e-3) / 1e12
        return {"bound": "mfma", "achieved": round(a, 2), "peak": perf.PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": round(a / perf.PEAK_BF16_TFLOPS, 4)}
    layer_flops = 2 * fl["total"]
    contract_tflops = fl["contract"] / (k_ms["contract"] * 1e-3) / 1e12
    clk = clocks.summary()
    clk_adj = clocks.adjusted_basis()

    def hbm_roof(nbytes, ms):
        a = nbytes / (ms * 1e-3) / 1e9
        return {"bound": "hbm", "achieved": round(a, 1), "peak": perf.PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(a / perf.PEAK_HBM_GBS, 4), "bytes_per_launch": nbytes,
                "frac_of_stream": round(a / best_stream, 4)}
    result = {
        "metric": "triangle-mult ms/layer + TFLOP/s at N=4096 bf16; % of MFMA bf16 peak",
        "value": round(layer_flops / (ms_step * 1e-3) / 1e12, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"triangle multiplicative update, outgoing + incoming (one layer), N={N}, c_z=128, "
                               f"c=128, bf16 storage / fp32 accumulation, fp32 output, all-ones mask, z~N(0,1)",
                   "N": N, "c_z": 128, "c": 128, "parallelism": "none (one GPU)"},
        "ms_per_layer": round(ms_step, 4),
        "ms_per_layer_full_calls": round(full_ms, 4),
        "ms_per_layer_median": round(step_median, 4), "ms_per_layer_min": round(per_step[0], 4),
        "gpu_state": {"before": state_before, "after": gpu_state()},
        "contract_pct_of_bf16_peak": round(100 * contract_tflops / perf.PEAK_BF16_TFLOPS, 2),
        "contract_pct_of_bf16_peak_clock_adjusted": None if clk_adj is None else
            round(100 * contract_tflops / perf.bf16_peak_at(clk_adj["mean_MHz"]), 2),
        "sclk_during_timed_steps": clk,
        "kernels": {
            "project": {"ms": round(k_ms["project"], 4),
                        "GB_per_s": round(by["project"] / (k_ms["project"] * 1e-3) / 1e9, 1),
                        "TFLOP_per_s": round(fl["project"] / (k_ms["project"] * 1e-3) / 1e12, 2),
                        "roofline": hbm_roof(by["project"], k_ms["project"])},
            "contract": {"ms": round(k_ms["contract"], 4), "TFLOP_per_s": round(contract_tflops, 2)},
            "epilogue": {"ms": round(k_ms["epilogue"], 4),
                         "GB_per_s": round(by["epilogue"] / (k_ms["epilogue"] * 1e-3) / 1e9, 1),
                         "roofline": hbm_roof(by["epilogue"], k_ms["epilogue"])},
            "stream_reference": stream_ref,
        },
        "n2048_channel_scaled": c3,
        "backward_contract": None if bwd_ms is None else {"ms": round(bwd_ms, 4),
                              "TFLOP_per_s": round(2 * fl["contract"] / (bwd_ms * 1e-3) / 1e12, 2),
                              "roofline": mfma_roof(2 * fl["contract"], bwd_ms),
                              "what": "dA = dC B and dB = dC^T A for all 128 channels (one direction), "
                                      "including the layout kernels; not part of ms_per_step"},
        "outer_product_mean": None if opm_ms is None else {"ms": round(opm_ms, 4),
                               "TFLOP_per_s": round(opm_flops / (opm_ms * 1e-3) / 1e12, 2),
                               "roofline": mfma_roof(opm_flops + opm_proj_flops, opm_ms),
                               "what": "opm_forward, S=4096 sequences x N=1024 tokens, D=32, c_z=128, bf16 in, "
                                       "fp32 out: 2*S*(N*D)^2 = 8.80 TFLOP contraction + counts + projection; "
                                       "not part of ms_per_step"},
        "triangle_attention": None if ta_ms is None else {"ms": round(ta_ms, 4), "ms_bf16_out": round(ta16_ms, 4),
                               "G_scores_per_s": round(ta_scores / (ta_ms * 1e-3) / 1e9, 1),
                               "TFLOP_per_s": round(4 * 32 * ta_scores / (ta_ms * 1e-3) / 1e12, 2),
                               "roofline": {"bound": "alu", "achieved": round(ta_scores / (ta_ms * 1e-3) / 1e12, 3),
                                            "peak": round(perf.PEAK_LANE_OPS / perf.TRIATTN_SLOTS / 1e12, 3),
                                            "unit": "T scores/s",
                                            "frac": round(ta_scores / (ta_ms * 1e-3) / (perf.PEAK_LANE_OPS
                                                                                         / perf.TRIATTN_SLOTS), 4),
                                            "peak_basis": perf.TRIATTN_BASIS},
                               "what": "tri_attn_forward, rows = n = 2048, 4 heads of 32, bf16 in, fp32 out: "
                                       "rows*H*n^2 = 34.4e9 scores (QK and PV 128 flop each); ms_bf16_out: the "
                                       "same call with bf16 output; not part of ms_per_step"},
        "ring_tile": None if tile_ms is None else {"ms": round(tile_ms, 4),
                      "TFLOP_per_s": round(tile_flops / (tile_ms * 1e-3) / 1e12, 2),
                      "roofline": mfma_roof(tile_flops, tile_ms),
                      "ms_blocked_plain_order": round(tile_plain_ms, 4),
                      "ms_rowmajor_pipelined": round(tile_pk_ms, 4),
                      "ms_one_stream_ws": round(tile_ws_ms, 4),
                      "what": "one device's share of a layer on an 8x8 grid at N=30000, tile (7,7): the projection "
                              "of its 3750x3750 z tile into blocked a, b panels written transposed "
                              "(tri_mul_block_project with the opposite direction), 8 ring steps reading them "
                              "transposed (tri_mul_block_accumulate_transposed: 3750x3750 outputs, "
                              "3750-token k-panels, 128 channels, 108.0 TFLOP contraction, packed fp32 "
                              "accumulator) and the tile epilogue on the last step, fp32 output; TFLOP/s counts "
                              "the contraction only.  ms_blocked_plain_order: the same ring on panels in the "
                              "direction's own order (tri_mul_block_accumulate_blocked).  With row-major panels "
                              "instead (no projection): "
                              "ms_rowmajor_pipelined = tri_mul_block_repack of panel p + 1 on a second stream while "
                              "panel p is contracted on 224 CUs (tri_mul_block_accumulate_packed), "
                              "ms_one_stream_ws = tri_mul_block_accumulate_ws on one stream; not part of "
                              "ms_per_step"},
        "backward_layer_saved": None if sbwd_ms is None else {"ms": round(sbwd_ms, 4),
                           "roofline": {"bound": "mfma + hbm", "floor_ms": round(bws_["floor_ms"], 3),
                                        "frac": round(bws_["floor_ms"] / sbwd_ms, 4),
                                        "basis": "floor = two N^3 bf16 products at MFMA peak + the per-pair "
                                                 "kernels' algorithmic bytes at HBM peak; frac = floor / ms"},
                           "what": "tri_mul_outgoing_backward_saved: the layer backward from the forward's saved "
                                   "A, B panels and C (no recomputation); not part of ms_per_step"},
        "backward_layer": None if lbwd_ms is None else {"ms": round(lbwd_ms, 4),
                           "roofline": {"bound": "mfma + hbm", "floor_ms": round(bw["floor_ms"], 3),
                                        "frac": round(bw["floor_ms"] / lbwd_ms, 4),
                                        "mfma_flops": bw["mfma_flops"], "hbm_bytes": bw["hbm_bytes"],
                                        "basis": "floor = three N^3 bf16 products at MFMA peak + the per-pair "
                                                 "kernels' algorithmic bytes at HBM peak; frac = floor / ms"},
                           "what": "tri_mul_outgoing_backward: recompute of the forward projections and "
                                   "contraction, dz and all ten weight gradients; not part of ms_per_step"},
        "roofline": {"bound": "mfma", "achieved": round(contract_tflops, 2), "peak": perf.PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(contract_tflops / perf.PEAK_BF16_TFLOPS, 4),
                     "frac_clock_adjusted": None if clk_adj is None else
                         round(contract_tflops / perf.bf16_peak_at(clk_adj["mean_MHz"]), 4),
                     "traffic": measured_traffic(), "kernel": "k2_contract_ws",
                     "per_launch": f"2*N^3*c = {fl['contract']:.4e} flop (128 channels of one {N}^3 product)"},
        "cpu_baseline": None,
    }
    del A, B, C, outs, z, ws
    layer.close()
    torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle on a sample", file=sys.stderr, flush=True)
        result["cpu_baseline"] = cpu_baseline(N, args.cpu_sample)
        extras = {k: result[k] for k in ("backward_layer", "outer_product_mean", "triangle_attention")
                  if result[k] is not None}
        if extras:
            print("[bench] timing the CPU oracle on samples of the extras", file=sys.stderr, flush=True)
            for k, v in cpu_oracle_extras(extras).items():
                v["gpu_speedup"] = round(v["ms_extrapolated"] / extras[k]["ms"], 1)
                extras[k]["cpu_oracle"] = v
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
