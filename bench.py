"""Decode state-update throughput of the DeltaLog HIP path on one MI355X.

    python bench.py [--workload NAME] [--steps K] [--warmup W] [--gpus 1] [--no-cpu-baseline]

Default workload: the serving-step stack -- 24 GDN delta-rule layers, each 256
sequences x 32 heads, dk = dv = 128, fp32 state, bf16 q/k/v, merge interval M = 16, with
per-sequence log fill offsets uniform in [0, M) so that merges are staggered across
sequences (every launch mixes appending and merging slots).  A step is one decode token
of all 256 sequences through all 24 layers (24 launches of dl_append_step); the value is
sequence tokens per second, 256 * K / elapsed.  Other workloads (--workload): GDN
64x32x128^2 at M = 16 (R = 8 layer states), KDA 128x32x128^2 at M in {8,16,32} (R = 4),
RWKV6 128x40x64^2 at M = 16 (R = 12), linear attention, RetNet, GLA, and the small GDN
latency case 1x2x64^2 at M = 8 (fp32 or bf16 q/k/v).  Single-layer workloads step R
independent copies of the layer's state in turn, like consecutive layers of a model, so
the working set is far larger than the 256 MB last-level cache; their value is per-layer
token-updates per second, B * R * K / elapsed.

Token inputs come from a pool of 16 seeded steps of the workload generator, cycled over
the run; initial states are drawn on the device (seeded torch normal, std 0.02).  The
values do not change the cost of any kernel.

Timing: W untimed steps, then --repeats timed rollouts of exactly K steps each, every one
bracketed by torch.cuda.synchronize() and HIP events on the launch stream (the state
keeps decoding from one rollout to the next; K is a multiple of M, so every rollout has
the same phase mix); the value is the median rollout.  The same K steps are also timed
as replays of one captured HIP graph (or as direct launches, under --graph).

Besides the contract fields the JSON line carries: the eager dense baseline
(dl_eager_step on the same states), the per-phase split (append at each live length,
merge; a separate pass with an event pair around each step's launches), the roofline entry of
the dominant kernel (algorithmic bytes of the average launch over its average duration,
the duration taken from HIP events around the timed region on the launch stream), the
HBM traffic of that kernel from the committed counter profile when the kernel sources
and build flags still match it, and the fp64 CPU oracle timed on a bounded sample on this
host, on all its cores and on one.
"""

import argparse
import glob
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "decode state-update tokens/s per GPU + achieved HBM GB/s (append, merge, eager)"
HBM_PEAK_GBS = 8000.0
POOL = 16


def workloads():
    from paper_2608_15533_amd import workloads as W
    return {
        "gdn_b1_h2_d64_m8": (W.GDN_SMALL, 1),
        "gdn_b1_h2_d64_m8_bf16": (W.GDN_SMALL.with_(name="gdn_b1_h2_d64_m8_bf16",
                                                    in_dtype="bf16"), 1),
        "gdn_b64_h32_d128_m16": (W.GDN_B64, 8),
        "kda_b128_h32_d128_m8": (W.kda_with_merge_interval(8), 4),
        "kda_b128_h32_d128_m16": (W.kda_with_merge_interval(16), 4),
        "kda_b128_h32_d128_m32": (W.kda_with_merge_interval(32), 4),
        "rwkv6_b128_h40_d64_m16": (W.RWKV6_B128, 12),
        "linattn_b64_h32_d128_m16": (W.LINATTN_B64, 8),
        "retnet_b64_h32_d128_m16": (W.RETNET_B64, 8),
        "gla_b128_h32_d128_m16": (W.GLA_B128, 4),
        "gdn_stack24_b256_h32_d128_m16": (W.GDN_STACK, 24),
    }


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--workload", default="gdn_stack24_b256_h32_d128_m16",
                    choices=sorted(workloads()))
    ap.add_argument("--steps", type=int, default=0,
                    help="timed steps per rollout (0: the workload's own decode length)")
    ap.add_argument("--warmup", type=int, default=32)
    ap.add_argument("--repeats", type=int, default=5,
                    help="timed rollouts of --steps steps; the value is their median")
    ap.add_argument("--replicas", type=int, default=0, help="layer states (0: workload default)")
    ap.add_argument("--merge-interval", type=int, default=0,
                    help="override the workload's merge interval M (0: workload default)")
    ap.add_argument("--batch", type=int, default=0,
                    help="override the workload's sequence count B (0: workload default)")
    ap.add_argument("--state-dtype", default="f32", choices=("f32", "bf16"),
                    help="dtype of the dense state (bf16: rounded on every store)")
    ap.add_argument("--tiled", type=int, default=0, choices=(0, 2, 4), metavar="NV",
                    help="time the value-tiled step (dl_append_step_tiled) with NV value tiles "
                         "per head instead of the one-workgroup-per-head kernel")
    ap.add_argument("--fused-replay", action="store_true",
                    help="with --tiled: every tile recomputes the replay coefficients "
                         "(default: split replay, prepared once per head)")
    ap.add_argument("--graph", action="store_true",
                    help="submit the timed steps as replays of one HIP graph holding 16 steps "
                         "x R launches (the same launches, captured once)")
    ap.add_argument("--phase-cycles", type=int, default=2,
                    help="merge cycles of the per-phase pass (event pair around each step)")
    ap.add_argument("--single-submission", action="store_true",
                    help="time only the chosen submission (direct launches, or --graph), "
                         "not the other one as well (counter runs)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="time budget of each of the two CPU oracle runs (all cores, one core)")
    ap.add_argument("--decode-loop", default="", metavar="MODES",
                    help="instead of the kernel bench: time the decode loop (slot allocator, "
                         "graph-captured steps) under comma-separated scheduling modes "
                         "(fused, phased, phased_concurrent; 'all'), with and without graphs")
    ap.add_argument("--layers", type=int, default=24, help="decode-loop layers")
    ap.add_argument("--merge-first", action="store_true",
                    help="decode loop, fused mode: rows of merging slots first (same as "
                         "--row-order merge_first)")
    ap.add_argument("--row-order", default="", choices=("", "slot", "merge_first", "balanced",
                                                         "interleaved"),
                    help="row order of a launch whose slots sit at different live lengths "
                         "(the staggered stack, the decode loop's fused mode): slot order, "
                         "merging slots first, or by live length, longest first "
                         "(default: balanced for the kernel bench, slot for the decode loop)")
    ap.add_argument("--uniform", action="store_true",
                    help="decode loop: admit every sequence at once (default: staggered)")
    ap.add_argument("--autotune", type=int, default=0, metavar="MAX_M",
                    help="instead of the kernel bench: measure the append cost at every live "
                         "length and the merge cost at every length up to MAX_M, predict the "
                         "amortised step time of every merge interval, and check the "
                         "prediction against timed cycles")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain device-to-device copy of MIB MiB (5 times); used to "
                         "scale the HBM byte counters of a profiler run")
    return ap.parse_args()


def copy_calibration(mib):
    """A plain copy kernel of known size: counters read on it give the scale factor
    between the profiler's FETCH_SIZE / WRITE_SIZE and bytes actually moved."""
    import torch
    n = mib * 2**20 // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes_read": n * 4, "bytes_written": n * 4,
                      "launches": 5}), flush=True)


def code_only(text):
    """C/C++ source text without comments and with every whitespace run collapsed to one
    space (string and character literals kept verbatim): what the compiler sees, up to
    layout."""
    out, i, n = [], 0, len(text)
    while i < n:
        c = text[i]
        if c in "\"'":
            j = i + 1
            while j < n and text[j] != c:
                j += 2 if text[j] == "\\" else 1
            out.append(text[i:j + 1])
            i = j + 1
        elif text.startswith("//", i):
            j = text.find("\n", i)
            i = n if j < 0 else j
        elif text.startswith("/*", i):
            j = text.find("*/", i + 2)
            i = n if j < 0 else j + 2
            out.append(" ")
        else:
            out.append(c)
            i += 1
    return " ".join("".join(out).split())


def library_build_flags():
    """The compiler flags the library in use was built with (dl_build_flags()), read with
    a bare ctypes load so that no GPU runtime state is touched; the flags a default build
    would use when no library is built."""
    import ctypes
    from paper_2608_15533_amd import build as B
    path = os.environ.get("DELTALOG_LIB") or B.LIB
    try:
        lib = ctypes.CDLL(path)
        lib.dl_build_flags.restype = ctypes.c_char_p
        return lib.dl_build_flags().decode()
    except (OSError, AttributeError):
        return B.build_flags_string()


def kernel_source_hash(build_flags=None):
    """sha256 over the code of the kernel sources and the public header, comments and
    layout excluded, and over the compiler flags of the build (``build_flags``; default:
    those of the library in use): any change to the code or to the flags invalidates
    counter figures taken earlier, an edit of a comment does not."""
    files = sorted(glob.glob(os.path.join(ROOT, "paper_2608_15533_amd", "csrc", "*")))
    files.append(os.path.join(ROOT, "include", "deltalog.h"))
    h = hashlib.sha256()
    for f in files:
        h.update(os.path.basename(f).encode())
        with open(f, encoding="utf-8", errors="surrogateescape") as fh:
            h.update(code_only(fh.read()).encode("utf-8", errors="surrogateescape"))
    flags = library_build_flags() if build_flags is None else build_flags
    h.update(b"flags:" + " ".join(flags.split()).encode())
    return h.hexdigest()[:16]


def profile_key(workload, state_dtype, tiled=0, fused_replay=False):
    key = workload + ("_bf16state" if state_dtype == "bf16" else "")
    if tiled:
        key += f"_tiled{tiled}" + ("_fused" if fused_replay else "_split")
    return key


def counter_profile(key):
    """The TRAFFIC_JSON record of the committed counter profile of ``key`` (HBM bytes per
    launch of the dominant kernel, measured state-write ratio), or None when there is
    none or the kernel code changed since it was taken; and where it came from."""
    path = os.path.join(ROOT, "profiles", f"{key}_hbm_counters.txt")
    if not os.path.exists(path):
        return None, "no counter profile"
    m = re.search(r"^TRAFFIC_JSON (\{.*\})$", open(path).read(), flags=re.M)
    if not m:
        return None, "counter profile has no TRAFFIC_JSON line"
    d = json.loads(m.group(1))
    if d.get("kernel_source_hash") != kernel_source_hash():
        return None, "kernel sources changed since the counters were taken"
    return d, os.path.relpath(path, ROOT)


def counter_traffic(key):
    """HBM bytes per launch of the dominant kernel from the committed counter profile,
    or None (see ``counter_profile``)."""
    d, src = counter_profile(key)
    return (None if d is None else d["step_kernel_bytes_per_launch"]), src


def copy_ceiling(torch, stream, gib=2, reps=5):
    """Read+write GB/s of the runtime's device-to-device copy of ``gib`` GiB (median of
    ``reps`` copies timed with HIP events on the launch stream), reported beside the
    kernel's achieved bandwidth as a reference point for read-and-write traffic."""
    n = (gib << 30) // 4
    src = torch.empty(n, dtype=torch.float32, device="cuda").fill_(1.0)
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    ms = []
    for _ in range(reps):
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record(stream)
        dst.copy_(src)
        b.record(stream)
        torch.cuda.synchronize()
        ms.append(a.elapsed_time(b))
    del src, dst
    torch.cuda.empty_cache()
    return 2 * (gib << 30) / (float(np.median(ms)) * 1e-3) / 1e9


def host_cpu():
    """Cores this process may run on, and the CPU model (from /proc/cpuinfo, else lscpu)."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    if model is None:
        try:
            import subprocess
            out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
            m = re.search(r"^Model name:\s*(.+)$", out, flags=re.M)
            model = m.group(1).strip() if m else None
        except (OSError, subprocess.SubprocessError):
            pass
    return {"affinity_cores": len(os.sched_getaffinity(0)), "cpu_count": os.cpu_count(),
            "model": model or "unknown"}


def cpu_baseline(w, budget_s):
    """The fp64 oracle eager recurrence (Eq. 3), as it stands, on a bounded sample of the
    workload: one layer of at most 64 x 32 heads of 128^2 (fewer sequences than B where
    the layer is larger), for up to the workload's decode length or ``budget_s`` seconds.
    It runs twice: on every core this process may use, the heads split into one chunk per
    core and stepped by a thread pool (NumPy releases the GIL in its array loops), and on
    one core.  The rate is in the unit of the GPU value: per-layer token-updates/s, or,
    for a layer stack, sequence tokens/s through all layers -- the one-layer rate divided
    by the layer count (an extrapolation: the layers are identical in cost)."""
    from concurrent.futures import ThreadPoolExecutor

    from oracle import eager as OE
    from paper_2608_15533_amd import workloads as W

    cap = 64 * 32 * 128 * 128
    B = w.B if w.B * w.H * w.dk * w.dv <= cap else max(1, cap // (w.H * w.dk * w.dv))
    ws = w.with_(B=B)
    N = B * w.H
    S0 = W.initial_state(ws).astype(np.float64).reshape(N, w.dk, w.dv)
    flat = lambda a: None if a is None else a.reshape((N,) + a.shape[2:])
    xs = [{k: flat(a) for k, a in W.step_inputs(ws, t).items()} for t in range(4)]
    u = W.bonus(ws)
    u = None if u is None else np.broadcast_to(u, (B,) + u.shape).reshape(N, w.dk)
    part = lambda a, lo, hi: None if a is None else a[lo:hi]

    def rollout(threads):
        S = S0.copy()
        chunks = [(i * N // threads, (i + 1) * N // threads) for i in range(threads)]

        def one(c, x):
            lo, hi = c
            S[lo:hi], _ = OE.eager_step(w.op, S[lo:hi], x["q"][lo:hi], x["k"][lo:hi],
                                        x["v"][lo:hi], part(x["beta"], lo, hi),
                                        part(x["lam"], lo, hi), u=part(u, lo, hi))

        steps = 0
        with ThreadPoolExecutor(threads) as ex:
            wall0, cpu0 = time.perf_counter(), time.process_time()
            while True:
                x = xs[steps % len(xs)]
                list(ex.map(lambda c: one(c, x), chunks))
                steps += 1
                el = time.perf_counter() - wall0
                if el >= budget_s or steps >= w.steps:
                    break
            cpu = time.process_time() - cpu0
        return steps, el, cpu

    host = host_cpu()
    cores = host["affinity_cores"]
    steps_all, el_all, cpu_all = rollout(cores)
    steps_one, el_one, _ = rollout(1)
    scale = 1.0 / w.layers                   # sequence tokens through all layers
    rate = lambda steps, el: round(B * steps / el * scale, 2)
    unit = ("sequence tokens/s (all layers)" if w.layers > 1 else "tokens/s")
    return {
        "value": rate(steps_all, el_all),
        "unit": unit,
        "cores": cores,
        "kind": "oracle",
        "sample": (f"fp64 eager oracle (Eq. 3), one layer of {B} of the {w.B} sequences x "
                   f"{w.H} heads of {w.dk}x{w.dv}: {steps_all} decode steps on {cores} cores "
                   f"({el_all:.1f} s wall, {cpu_all:.1f} s CPU; heads split into {cores} "
                   f"chunks over a thread pool) and {steps_one} steps on one core "
                   f"({el_one:.1f} s)"
                   + (f"; the {w.layers}-layer rate is the one-layer rate / {w.layers} "
                      "(extrapolated)" if w.layers > 1 else "")),
        "single_core_value": rate(steps_one, el_one),
        "cpu_model": host["model"],
        "affinity_cores": cores,
        "cpu_count": host["cpu_count"],
    }


def decode_loop(args):
    """Decode-loop throughput: a GDN stack of ``--layers`` layers, B slots x 32 heads of
    128^2, M = 16 (or the overrides), bf16 q/k/v, fp32 state.  Sequences are admitted
    B/M per step over the first M steps (staggered logs, so every step mixes appends and
    merges) or all at once (``--uniform``).  Each timed step is one plan + one decode
    token through every layer; token inputs stay in the engine's fixed buffers (their
    values do not change any kernel's cost).  Prints one JSON line with every mode."""
    import torch
    from paper_2608_15533_amd import decode
    from paper_2608_15533_amd import deltalog as D
    from paper_2608_15533_amd import traffic as T

    B = args.batch or 256
    M = args.merge_interval or 16
    layers = args.layers
    H, dk, dv = 32, 128, 128
    K, WU = args.steps or 64, args.warmup
    modes = decode.MODES if args.decode_loop == "all" else tuple(args.decode_loop.split(","))
    desc = D.make_desc("gdn", B, H, dk, dv, M, "bf16")
    torch.cuda.set_device(0)
    res = {}
    for mode in modes:
        for graphs in (True, False):
            eng = decode.DecodeEngine(desc, layers, mode=mode, graphs=graphs,
                                      merge_first=args.merge_first,
                                      row_order=args.row_order or None)
            gen = torch.Generator(device="cuda")
            gen.manual_seed(20261202)
            for layer in range(layers):
                x = eng.inputs[layer]
                qk = torch.randn((2, B, H, dk), generator=gen, device="cuda")
                qk = qk / qk.norm(dim=-1, keepdim=True)
                x.q.copy_(qk[0])
                x.k.copy_(qk[1])
                x.v.copy_(torch.randn((B, H, dv), generator=gen, device="cuda"))
                g = torch.randn((B, H), generator=gen, device="cuda")
                x.lam.copy_(torch.nn.functional.logsigmoid(3.0 + 0.5 * g))
                x.beta.copy_(torch.sigmoid(torch.randn((B, H), generator=gen, device="cuda")))
                st = eng.states[layer]
                st.S.copy_(torch.randn(st.S.shape, generator=gen, device="cuda") * 0.02)
            per_step = B if args.uniform else max(1, -(-B // M))
            steps_run = 0
            while eng.sched.free_slots:
                for _ in range(min(per_step, eng.sched.free_slots)):
                    slot = eng.sched.admit()           # the base already holds a state
                    for st in eng.states:
                        st.len[slot].zero_()
                eng.schedule()
                eng.step()
                steps_run += 1
            for _ in range(WU):
                eng.schedule()
                eng.step()
            torch.cuda.synchronize()
            # algorithmic bytes of the timed steps, from a copy of the live-length mirror
            live = list(eng.sched.live)
            C = M - 1
            nbytes = 0
            for _ in range(K):
                for s in eng.sched.active:
                    nbytes += T.step_bytes("gdn", dk, dv, M, live[s]).total
                    live[s] = 0 if live[s] >= C else live[s] + 1
            nbytes *= H * layers
            stream = torch.cuda.current_stream()
            t0 = torch.cuda.Event(enable_timing=True)
            t1 = torch.cuda.Event(enable_timing=True)
            h0 = time.perf_counter()
            t0.record(stream)
            for _ in range(K):
                eng.schedule()
                eng.step()
            t1.record(stream)
            h1 = time.perf_counter()
            torch.cuda.synchronize()
            ms = t0.elapsed_time(t1)
            n = len(eng.sched.active)
            assert eng.error_words() == [0] * layers
            res[mode + ("" if graphs else "_direct")] = {
                "seq_tokens_per_s": round(n * K / (ms * 1e-3), 1),
                "layer_token_updates_per_s": round(n * layers * K / (ms * 1e-3), 1),
                "ms_per_step": round(ms / K, 5),
                "host_ms_per_step": round((h1 - h0) * 1e3 / K, 5),
                "GB/s": round(nbytes / (ms * 1e-3) / 1e9, 1),
                "frac": round(nbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                "graphs": len(eng.graph_keys),
                "replays": eng.replays,
            }
            del eng
            torch.cuda.empty_cache()
    print(json.dumps({
        "metric": "decode-loop sequence tokens/s (all layers' state updates per token)",
        "unit": "tokens/s", "steps": K, "warmup": WU, "data": "synthetic",
        "config": {"workload": f"GDN {layers}-layer decode loop: B={B} slots, H={H}, "
                               f"dk=dv={dk}, M={M}, bf16 q/k/v, fp32 state, "
                               f"{'uniform' if args.uniform else 'staggered'} admission",
                   "batch": B, "layers": layers, "merge_interval": M,
                   "fused_row_order": (args.row_order or
                                       ("merge_first" if args.merge_first else "slot"))},
        "modes": res,
        "kernel_source_hash": kernel_source_hash(),
    }), flush=True)


def autotune(args):
    """Merge-interval selection from measured phase costs for the chosen workload shape
    (``--batch`` and ``--state-dtype`` apply), checked against timed full cycles at
    several merge intervals.  Prints one JSON line."""
    import torch
    from paper_2608_15533_amd import autotune as A
    from paper_2608_15533_amd import deltalog as D
    from paper_2608_15533_amd import traffic as T

    w, _ = workloads()[args.workload]
    if args.batch:
        w = w.with_(B=args.batch)
    sd = args.state_dtype
    max_M = args.autotune
    torch.cuda.set_device(0)
    t0 = time.perf_counter()
    cal = A.calibrate(w.op, w.B, w.H, w.dk, w.dv, w.in_dtype, sd, max_M=max_M, reps=5)
    cal_s = time.perf_counter() - t0
    best, pred = A.choose(cal["append_us"], cal["merge_us"])
    R = cal["replicas"]

    def cycle_us(M, cycles=4):
        """Mean launch time of dl_append_step over whole M-step cycles (every slot at
        the same live length, R layer states in turn)."""
        desc = D.make_desc(w.op, w.B, w.H, w.dk, w.dv, M, w.in_dtype, sd)
        gen = torch.Generator(device="cuda")
        gen.manual_seed(7)
        sts = [D.DeltaLogState(desc, 0.02 * torch.randn(w.B, w.H, w.dk, w.dv, generator=gen,
                                                        device="cuda")) for _ in range(R)]
        tok = A._token(desc, w.B, gen)
        o = torch.empty((w.B, w.H, w.dv), dtype=torch.float32, device="cuda")
        for _ in range(M):
            for st in sts:
                D.dl_append_step(desc, st, tok, o)
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(200_000)           # the host enqueues while the device is busy
        e0.record()
        for _ in range(cycles * M):
            for st in sts:
                D.dl_append_step(desc, st, tok, o)
        e1.record()
        e1.synchronize()
        assert all(int(st.err.item()) == 0 for st in sts)
        us = e0.elapsed_time(e1) * 1e3 / (cycles * M * R)
        del sts
        torch.cuda.empty_cache()
        return us

    check = sorted({M for M in (1, 2, 4, 8, 16, 32, 64, best) if M <= max_M})
    measured = {M: cycle_us(M) for M in check}
    mbest = min(measured, key=lambda M: (measured[M], M))
    res = {
        "autotune": {
            "workload": w.name, "op": w.op, "batch": w.B, "heads": w.H, "dk": w.dk,
            "dv": w.dv, "in_dtype": w.in_dtype, "state_dtype": sd, "replicas": R,
            "calibration_s": round(cal_s, 2),
            "append_us": [round(x, 3) for x in cal["append_us"]],
            "merge_us": [round(x, 3) for x in cal["merge_us"]],
            "predicted_us_per_step": {M: round(t, 3) for M, t in pred.items()},
            "chosen_M": best,
            "byte_optimal_M": T.byte_optimal_merge_interval(w.op, w.dk, w.dv, w.in_dtype, sd,
                                                            max_M=max_M),
            "measured_us_per_step": {M: round(t, 3) for M, t in measured.items()},
            "measured_best_M_of_checked": mbest,
            "chosen_vs_measured_best": round(measured[best] / measured[mbest], 4),
            "predicted_tokens_per_s": round(w.B * 1e6 / pred[best], 1),
            "measured_tokens_per_s_at_chosen": round(w.B * 1e6 / measured[best], 1),
        }
    }
    print(json.dumps(res), flush=True)


def main():
    args = parse()
    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}): the decode state "
              "update has no cross-GPU step; run with --gpus 1.", file=sys.stderr)
        sys.exit(2)
    if args.decode_loop:
        decode_loop(args)
        return
    if args.autotune:
        autotune(args)
        return

    import ctypes

    import torch
    from paper_2608_15533_amd import deltalog as D
    from paper_2608_15533_amd import traffic as T
    from paper_2608_15533_amd import workloads as W

    w, R = workloads()[args.workload]
    if args.merge_interval or args.batch:
        w = w.with_(M=args.merge_interval or w.M, B=args.batch or w.B)
        # enough layer states for a working set of at least 1 GiB (4x the last-level cache)
        per_layer = w.B * w.H * (w.dk * w.dv * (2 if args.state_dtype == "bf16" else 4)
                                 + (w.M - 1) * (w.dk + w.dv) * 4)
        R = max(2, -(-(1 << 30) // per_layer)) if w.layers == 1 else R
    R = args.replicas or R
    K, WU = args.steps or w.steps, args.warmup
    if K < 1 or WU < 0 or args.repeats < 1:
        raise SystemExit("--steps, --repeats >= 1 and --warmup >= 0")
    dev = "cuda"
    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()
    sp = stream.cuda_stream
    sd = args.state_dtype
    desc = D.make_desc(w.op, w.B, w.H, w.dk, w.dv, w.M, w.in_dtype, sd)
    heads = w.B * w.H
    it = torch.bfloat16 if w.in_dtype == "bf16" else torch.float32

    # -------------------------------------------------------------- device buffers
    gen = torch.Generator(device=dev)
    states = []
    for r in range(R):
        gen.manual_seed(20261202 + r)
        S0 = torch.randn((w.B, w.H, w.dk, w.dv), generator=gen, device=dev) * 0.02
        states.append(D.DeltaLogState(desc, S0))
        del S0
    eager_S = [s.S.clone() for s in states]
    u = W.bonus(w)
    toks = []
    for t in range(POOL):
        x = W.step_inputs(w, t)
        cv = lambda a, dt: None if a is None else torch.from_numpy(a).to(dev).to(dt).contiguous()
        toks.append(D.Token(desc, w.B, cv(x["q"], it), cv(x["k"], it), cv(x["v"], it),
                            cv(x["lam"], torch.float32), cv(x["beta"], torch.float32),
                            cv(u, torch.float32)))
    outs = [torch.empty((w.B, w.H, w.dv), dtype=torch.float32, device=dev) for _ in range(R)]

    # staggered log fill (partial-batch warm-up through slot lists)
    live = np.zeros(w.B, dtype=np.int64)                 # host mirror of every slot's L
    if w.staggered:
        for rnd, rows in W.warmup_schedule(w):
            sl = torch.from_numpy(rows.astype(np.int32)).to(dev)
            for r in range(R):
                D.dl_append_step(desc, states[r], toks[rnd % POOL], outs[r][: len(rows)], slots=sl)
            live[rows] += 1
        assert np.array_equal(live, W.fill_offsets(w))
    torch.cuda.synchronize()

    # Row order of the DeltaLog launches.  With staggered logs the slots of a launch sit
    # at different live lengths; the balanced order (longest log first, as the decode
    # scheduler plans it) gives every XCD the same mix.  The order repeats with the merge
    # interval, so one slot list per phase serves the whole run.
    row_order = args.row_order or ("balanced" if w.staggered else "slot")
    PER = POOL
    lists = None
    if row_order != "slot":
        from paper_2608_15533_amd.scheduler import balanced_order, interleaved_order
        PER = int(np.lcm(POOL, w.M))
        lists = []
        for k in range(PER):
            Lk = (live + k) % w.M
            if row_order == "balanced":
                order = balanced_order(range(w.B), Lk)
            elif row_order == "interleaved":
                order = interleaved_order(range(w.B), Lk)
            else:
                order = tuple(np.nonzero(Lk == w.M - 1)[0]) + tuple(np.nonzero(Lk < w.M - 1)[0])
            lists.append(torch.tensor(order, dtype=torch.int32, device=dev))
    dref = ctypes.byref(desc)
    app = D.lib.dl_append_step
    eag = D.lib.dl_eager_step
    sl_ptr = (lambda k: None) if lists is None else (lambda k: lists[k % PER].data_ptr())
    app_args = [[(dref, ctypes.byref(states[r].struct), ctypes.byref(toks[k % POOL].struct),
                  outs[r].data_ptr(), sl_ptr(k), w.B, sp) for k in range(PER)]
                for r in range(R)]
    if args.tiled:
        # value-tiled path: [ReplayPrep] + tiles + Finalize per layer and step; one
        # scratch buffer serves every layer (the launches are ordered on one stream)
        split = not args.fused_replay
        ws = D.tiled_workspace(desc, w.B) if split else None
        wsp, wsn = (None, 0) if ws is None else (ws.data_ptr(), ws.numel())
        app = D.lib.dl_append_step_tiled
        app_args = [[(dref, ctypes.byref(states[r].struct), ctypes.byref(toks[k % POOL].struct),
                      outs[r].data_ptr(), sl_ptr(k), w.B, args.tiled, int(split), wsp, wsn, sp)
                     for k in range(PER)] for r in range(R)]
    eag_args = [[(dref, eager_S[r].data_ptr(), ctypes.byref(toks[k % POOL].struct),
                  outs[r].data_ptr(), None, w.B, sp) for k in range(PER)] for r in range(R)]

    done = [0]                                           # steps executed so far

    def run(fn, argtab, nsteps, events=None, capture=None):
        """Launch ``nsteps`` steps (R launches each) from the next step index; with
        ``capture`` (a stream handle) the launches are recorded, not executed."""
        k0 = done[0]
        for i, k in enumerate(range(k0, k0 + nsteps)):
            if events is not None:
                events[i][0].record(stream)
            for r in range(R):
                a = argtab[r][k % PER]
                rc = fn(*(a if capture is None else a[:-1] + (capture,)))
                if rc != 0:
                    raise D.DeltaLogError(rc, fn.__name__)
            if events is not None:
                events[i][1].record(stream)
        if capture is None:
            done[0] += nsteps

    def region(body):
        """One timed region: synchronize, HIP events on the launch stream around
        ``body``, synchronize; returns elapsed ms."""
        torch.cuda.synchronize()
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        t0.record(stream)
        body()
        t1.record(stream)
        torch.cuda.synchronize()
        return t0.elapsed_time(t1)

    def timed_direct(fn, argtab, warm):
        """``warm`` untimed steps, then the timed rollouts of K steps (no per-launch
        events inside); returns (ms of each rollout, first timed step index)."""
        run(fn, argtab, warm)
        first = done[0]
        return [region(lambda: run(fn, argtab, K)) for _ in range(args.repeats)], first

    graph_possible = K % PER == 0 and WU % PER == 0

    def timed_graph(fn, argtab, warm):
        """The same rollouts submitted as replays of one captured graph of PER steps x R
        launches (the kernels loaded by PER direct steps first)."""
        run(fn, argtab, PER)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        cs = torch.cuda.Stream()
        cs.wait_stream(stream)
        with torch.cuda.stream(cs):
            with torch.cuda.graph(g, stream=cs):
                run(fn, argtab, PER, capture=cs.cuda_stream)
        stream.wait_stream(cs)

        def replays(n):
            for _ in range(n // PER):
                g.replay()
            done[0] += n

        replays(max(warm - PER, 0))
        first = done[0]
        ms = [region(lambda: replays(K)) for _ in range(args.repeats)]
        del g
        return ms, first

    def per_launch(fn, argtab, nsteps):
        """A separate pass with an event pair around each step's R launches, which share
        one live length (per-phase split): returns the mean launch time of every step, so
        the cost of recording events is spread over R launches instead of inflating each.
        The events are created beforehand so the host keeps ahead of the device."""
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(nsteps)]
        run(fn, argtab, nsteps, evs)
        torch.cuda.synchronize()
        return np.array([a.elapsed_time(b) for a, b in evs]) / R

    def launch_bytes(k):
        """Algorithmic bytes of one layer launch at step k (every slot at its own L)."""
        Ls = (live + k) % w.M
        counts = np.bincount(Ls, minlength=w.M)
        return sum(int(c) * w.H * T.step_bytes(w.op, w.dk, w.dv, w.M, L, w.in_dtype, sd).total
                   for L, c in enumerate(counts) if c)

    # ------------------------------------------------------------------ DeltaLog
    primary, secondary = (timed_graph, timed_direct) if args.graph else (timed_direct, timed_graph)
    if args.graph and not graph_possible:
        raise SystemExit(f"--graph needs --steps and --warmup to be multiples of {PER}")
    rollouts, first = primary(app, app_args, WU)
    dl_ms = float(np.median(rollouts))
    n_launch = K * R
    tokens = w.B * K if w.layers > 1 else w.B * R * K    # stack: tokens through all layers
    dl_tok = tokens / (dl_ms * 1e-3)
    # roofline: every timed launch -- all rollouts -- over the time of all rollouts
    nrep = len(rollouts)
    avg_launch_us = float(np.sum(rollouts)) * 1e3 / (n_launch * nrep)
    bytes_per_launch = float(np.mean([launch_bytes(first + k) for k in range(K * nrep)]))
    achieved = bytes_per_launch / (avg_launch_us * 1e-6) / 1e9
    other = None
    if graph_possible and not args.single_submission:
        o_ms, _ = secondary(app, app_args, PER)
        o_med = float(np.median(o_ms))
        other = {"submission": "direct launches" if args.graph else "HIP graph replay",
                 "value": round(tokens / (o_med * 1e-3), 1),
                 "us_per_step": round(o_med * 1e3 / K, 3),
                 "rollouts_ms": [round(x, 4) for x in o_ms]}

    PH = args.phase_cycles * w.M
    k0 = done[0]
    ph_durs = per_launch(app, app_args, PH)
    for s in states:
        assert int(s.err.item()) == 0
    phases = {"source": "separate pass, HIP event pair around each step's launches (one per "
                        "layer state, all at one live length), median per phase"}
    if not w.staggered:
        by_L = {}
        for L in range(w.M):
            sel = np.array([(k0 + k) % w.M == L for k in range(PH)])
            us = float(np.median(ph_durs[sel]) * 1e3)
            b = T.step_bytes(w.op, w.dk, w.dv, w.M, L, w.in_dtype, sd).total * heads
            by_L[("merge_L%d" if L == w.M - 1 else "append_L%d") % L] = {
                "us": round(us, 2), "GB/s": round(b / (us * 1e-6) / 1e9, 1)}
        app_sel = np.array([(k0 + k) % w.M < w.M - 1 for k in range(PH)])
        phases_out = []
        if app_sel.any():
            app_us = float(np.median(ph_durs[app_sel]) * 1e3)
            app_b = float(np.mean([launch_bytes(k0 + k) for k in range(PH) if app_sel[k]]))
            phases_out.append(("append", app_us, app_b))
        mrg_us = float(np.median(ph_durs[~app_sel]) * 1e3)
        mrg_b = T.merge_bytes(w.op, w.dk, w.dv, w.M - 1, w.in_dtype, sd).total * heads
        phases_out.append(("merge", mrg_us, mrg_b))
        for name, us, b in phases_out:
            gbs = b / (us * 1e-6) / 1e9
            phases[name] = {"us": round(us, 2), "GB/s": round(gbs, 1),
                            "frac": round(gbs / HBM_PEAK_GBS, 4)}
        phases["by_live_length"] = by_L
    else:
        us = float(np.median(ph_durs) * 1e3)
        b = float(np.mean([launch_bytes(k0 + k) for k in range(PH)]))
        phases["mixed"] = {"us": round(us, 2), "GB/s": round(b / (us * 1e-6) / 1e9, 1),
                           "note": "every launch mixes appending and merging slots"}

    # ------------------------------------------------------------------ eager baseline
    eg_rollouts, _ = primary(eag, eag_args, WU)
    eg_ms = float(np.median(eg_rollouts))
    eg_tok = tokens / (eg_ms * 1e-3)
    eg_bytes = T.eager_bytes(w.op, w.dk, w.dv, w.in_dtype, sd).total * heads
    eg_us = eg_ms * 1e3 / n_launch
    eg_gbs = eg_bytes / (eg_us * 1e-6) / 1e9

    if args.batch or args.merge_interval or args.replicas:
        prof, traffic_src = None, "no counter profile for this configuration (overrides given)"
    else:
        prof, traffic_src = counter_profile(profile_key(args.workload, sd, args.tiled,
                                                        args.fused_replay))
    traffic = None if prof is None else prof["step_kernel_bytes_per_launch"]
    copy_gbs = copy_ceiling(torch, stream)
    state_mib = heads * w.dk * w.dv * (2 if sd == "bf16" else 4) / 2**20
    kname = {"gdn": "GDN", "kda": "KDA", "rwkv6": "RWKV6", "linattn": "LinearAttention",
             "retnet": "RetNet", "gla": "GLA"}[w.op]
    res = {
        "metric": METRIC,
        "value": round(dl_tok, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": WU,
        "ms_per_step": round(dl_ms / K, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": (f"{kname} decode state update: B={w.B} sequences, H={w.H} heads, "
                         f"dk={w.dk}, dv={w.dv}, {'fp32' if sd == 'f32' else 'bf16'} state, "
                         f"{w.in_dtype} q/k/v, merge interval "
                         f"M={w.M}" + (f", {w.layers} layers, staggered log fill"
                                       if w.layers > 1 else "")),
            "name": args.workload + (f" M={w.M}" if args.merge_interval else "")
                    + (f" B={w.B}" if args.batch else "")
                    + (f" tiled{args.tiled}-{'fused' if args.fused_replay else 'split'}"
                       if args.tiled else ""),
            "op": w.op, "batch": w.B, "heads": w.H, "dk": w.dk,
            "dv": w.dv, "merge_interval": w.M, "in_dtype": w.in_dtype, "state_dtype": sd,
            "layer_states": R, "state_MiB_per_layer": state_mib,
            "row_order": row_order,
            "working_set_MiB": round(sum(t.numel() * t.element_size() for st in states
                                         for t in st.buffers().values()
                                         if t is not None) / 2**20, 1),
            "tokens_per_s_definition": ("per-layer token-updates/s = B*R*K/elapsed"
                                        if w.layers == 1 else
                                        "tokens through all layers = B*K/elapsed"),
        },
        "roofline": {
            "bound": "hbm",
            "kernel": (f"deltalog_kernel<{kname},{w.dk},{w.dv},STEP,{w.in_dtype},{sd} state> "
                       "(dl_append_step: append or merge)" if not args.tiled else
                       f"dl_append_step_tiled, {args.tiled} value tiles, "
                       f"{'fused' if args.fused_replay else 'split'} replay: "
                       "[replay_prep_kernel] + tile_step_kernel + finalize_kernel per call "
                       "(durations and bytes are per call)"),
            "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": None if traffic is None else round(traffic, 1),
            "traffic_unit": "bytes per launch (FETCH_SIZE + WRITE_SIZE, copy-calibrated)",
            "traffic_source": traffic_src,
            "avg_launch_us": round(avg_launch_us, 3),
            "d2d_copy_GB/s": round(copy_gbs, 1),
            "achieved_vs_d2d_copy": round(achieved / copy_gbs, 4),
            "algorithmic_bytes_per_launch": round(bytes_per_launch, 1),
            "duration_source": "HIP events around each timed rollout: summed over the "
                               "rollouts / their launches",
        },
        "timing": {
            "submission": "HIP graph replay" if args.graph else "direct launches",
            "repeats": args.repeats,
            "rollouts_ms": [round(x, 4) for x in rollouts],
            "value_from": "median rollout",
            "us_per_step": round(dl_ms * 1e3 / K, 3),
            "other_submission": other,
        },
        "phases": phases,
        "eager": {
            "tokens_per_s": round(eg_tok, 1),
            "ms_per_step": round(eg_ms / K, 5),
            "rollouts_ms": [round(x, 4) for x in eg_rollouts],
            "us_per_launch": round(eg_us, 3),
            "GB/s": round(eg_gbs, 1),
            "frac": round(eg_gbs / HBM_PEAK_GBS, 4),
        },
        "speedup_vs_eager": round(dl_tok / eg_tok, 3),
        "state_write_ratio_measured": (None if prof is None
                                       else prof.get("state_write_ratio_measured")),
        "state_write_ratio_bound": round(T.state_write_ratio(w.op, w.dk, w.dv, w.M, w.in_dtype, sd), 3),
        "state_write_ratio_layout": round(T.library_state_write_ratio(w.op, w.dk, w.dv, w.M,
                                                                     w.in_dtype, sd), 3),
        "kernel_source_hash": kernel_source_hash(),
    }
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(w, args.cpu_seconds)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
