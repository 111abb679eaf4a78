"""Decode state-update throughput of the DeltaLog HIP path on one MI355X.

    python bench.py [--steps K] [--warmup W] [--replicas R] [--gpus 1] [--no-cpu-baseline]

Workload: GDN delta-rule decode, 64 sequences x 32 heads, dk = dv = 128, fp32 state,
bf16 q/k/v, merge interval M = 16 (one merge every 16 steps).  R independent copies of
that layer's state (default 8, 1.2 GiB in all) are stepped in turn, like consecutive
layers of a model, so the working set is far larger than the 256 MB last-level cache
and every step streams its state from HBM.  A step is one decode token through all R
layer states (R launches of dl_append_step); the reported value is per-layer
token-updates per second, B * R * K / elapsed.  Token inputs come from a pool of 16
pre-generated seeded steps cycled over the run (their values do not change the cost).

The JSON line also carries: the eager dense baseline (dl_eager_step on the same
replicas), the per-phase split (append at each live length, merge), the roofline entry
of the dominant kernel (algorithmic bytes of each launch over its duration measured
with HIP events on the launch stream), and the fp64 CPU oracle timed on a bounded
sample on this host.
"""

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "decode state-update tokens/s per GPU + achieved HBM GB/s (append, merge, eager)"
HBM_PEAK_GBS = 8000.0
POOL = 16


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=256)
    ap.add_argument("--warmup", type=int, default=32)
    ap.add_argument("--replicas", type=int, default=8)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
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


def cpu_baseline(w, budget_s):
    """The fp64 oracle eager recurrence, as it stands, on a bounded sample of the same
    workload (all 64 x 32 heads, as many steps as fit the time budget)."""
    from oracle import eager as OE
    from paper_2608_15533_amd import workloads as W

    S = W.initial_state(w).astype(np.float64)
    xs = [W.step_inputs(w, t) for t in range(4)]
    wall0, cpu0 = time.perf_counter(), time.process_time()
    steps = 0
    while True:
        x = xs[steps % len(xs)]
        S, _ = OE.eager_step(w.op, S, x["q"], x["k"], x["v"], x["beta"], x["lam"])
        steps += 1
        el = time.perf_counter() - wall0
        if el >= budget_s or steps >= 256:
            break
    cpu = time.process_time() - cpu0
    return {
        "value": w.B * steps / el,
        "unit": "tokens/s",
        "cores": max(1, int(round(cpu / el))),
        "kind": "oracle",
        "sample": f"fp64 eager oracle, {w.B}x{w.H} heads {w.dk}x{w.dv}, {steps} decode steps "
                  f"({el:.1f} s wall, {cpu:.1f} s CPU) on the host of this GPU",
    }


def main():
    args = parse()
    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}): the decode state "
              "update has no cross-GPU step; run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2608_15533_amd import deltalog as D
    from paper_2608_15533_amd import traffic as T
    from paper_2608_15533_amd import workloads as W

    w = W.GDN_B64
    R, K, WU = args.replicas, args.steps, args.warmup
    dev = "cuda"
    torch.cuda.set_device(0)
    stream = torch.cuda.current_stream()
    sp = stream.cuda_stream
    desc = D.make_desc(w.op, w.B, w.H, w.dk, w.dv, w.M, w.in_dtype)

    # -------------------------------------------------------------- device buffers
    states = []
    for r in range(R):
        S0 = torch.from_numpy(W.initial_state(w, layer=r)).to(dev)
        states.append(D.DeltaLogState(desc, S0))
    eager_S = [s.S.clone() for s in states]
    toks = []
    for t in range(POOL):
        x = W.step_inputs(w, t)
        cv = lambda a, dt: torch.from_numpy(a).to(dev).to(dt).contiguous()
        toks.append(D.Token(desc, w.B, cv(x["q"], torch.bfloat16), cv(x["k"], torch.bfloat16),
                            cv(x["v"], torch.bfloat16), cv(x["lam"], torch.float32),
                            cv(x["beta"], torch.float32)))
    outs = [torch.empty((w.B, w.H, w.dv), dtype=torch.float32, device=dev) for _ in range(R)]
    torch.cuda.synchronize()

    import ctypes
    dref = ctypes.byref(desc)
    app = D.lib.dl_append_step
    eag = D.lib.dl_eager_step
    app_args = [[(dref, ctypes.byref(states[r].struct), ctypes.byref(toks[t].struct),
                  outs[r].data_ptr(), None, w.B, sp) for t in range(POOL)] for r in range(R)]
    eag_args = [[(dref, eager_S[r].data_ptr(), ctypes.byref(toks[t].struct),
                  outs[r].data_ptr(), None, w.B, sp) for t in range(POOL)] for r in range(R)]

    def run(fn, argtab, k0, nsteps, events=None):
        for k in range(k0, k0 + nsteps):
            for r in range(R):
                if events is not None:
                    a = torch.cuda.Event(enable_timing=True)
                    a.record(stream)
                rc = fn(*argtab[r][k % POOL])
                if rc != 0:
                    raise D.DeltaLogError(rc, fn.__name__)
                if events is not None:
                    b = torch.cuda.Event(enable_timing=True)
                    b.record(stream)
                    events.append((a, b))

    def timed(fn, argtab):
        """W untimed steps, then K timed steps bracketed by synchronize + HIP events on
        the launch stream; returns elapsed ms (no per-launch events inside)."""
        run(fn, argtab, 0, WU)
        torch.cuda.synchronize()
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        t0.record(stream)
        run(fn, argtab, WU, K)
        t1.record(stream)
        torch.cuda.synchronize()
        return t0.elapsed_time(t1)

    def per_launch(fn, argtab, k0, nsteps):
        """A separate pass with an event pair around every launch (per-phase split)."""
        evs = []
        run(fn, argtab, k0, nsteps, evs)
        torch.cuda.synchronize()
        return np.array([a.elapsed_time(b) for a, b in evs]).reshape(nsteps, R)

    # ------------------------------------------------------------------ DeltaLog
    dl_ms = timed(app, app_args)
    heads = w.B * w.H
    Ls = [(WU + k) % w.M for k in range(K)]           # live length at each timed step
    step_bytes = np.array([T.step_bytes(w.op, w.dk, w.dv, w.M, L, w.in_dtype).total * heads
                           for L in Ls])
    n_launch = K * R
    dl_tok = w.B * R * K / (dl_ms * 1e-3)
    avg_launch_us = dl_ms * 1e3 / n_launch
    bytes_per_launch = float(step_bytes.mean())
    achieved = bytes_per_launch / (avg_launch_us * 1e-6) / 1e9

    # per-phase split: one more full cycle per replica, every launch bracketed
    k0 = WU + K
    PH = 2 * w.M
    ph_durs = per_launch(app, app_args, k0, PH)
    for s in states:
        assert int(s.err.item()) == 0
    phases = {}
    for L in range(w.M):
        sel = np.array([(k0 + k) % w.M == L for k in range(PH)])
        us = float(ph_durs[sel].mean() * 1e3)
        b = T.step_bytes(w.op, w.dk, w.dv, w.M, L, w.in_dtype).total * heads
        name = "merge_L%d" % L if L == w.M - 1 else f"append_L{L}"
        phases[name] = {"us": round(us, 2), "GB/s": round(b / (us * 1e-6) / 1e9, 1)}
    app_sel = np.array([(k0 + k) % w.M < w.M - 1 for k in range(PH)])
    app_us = float(ph_durs[app_sel].mean() * 1e3)
    app_bytes = float(np.mean([T.step_bytes(w.op, w.dk, w.dv, w.M, (k0 + k) % w.M, w.in_dtype).total
                               for k in range(PH) if app_sel[k]]) * heads)
    mrg_us = float(ph_durs[~app_sel].mean() * 1e3)
    mrg_bytes = T.merge_bytes(w.op, w.dk, w.dv, w.M - 1, w.in_dtype).total * heads

    # ------------------------------------------------------------------ eager baseline
    eg_ms = timed(eag, eag_args)
    eg_tok = w.B * R * K / (eg_ms * 1e-3)
    eg_bytes = T.eager_bytes(w.op, w.dk, w.dv, w.in_dtype).total * heads
    eg_us = eg_ms * 1e3 / n_launch
    eg_gbs = eg_bytes / (eg_us * 1e-6) / 1e9

    state_mib = w.B * w.H * w.dk * w.dv * 4 / 2**20
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
            "workload": "GDN decode state update: B=64 sequences, H=32 heads, dk=dv=128, "
                        "fp32 state, bf16 q/k/v, merge interval M=16",
            "op": w.op, "batch": w.B, "heads": w.H, "dk": w.dk, "dv": w.dv,
            "merge_interval": w.M, "in_dtype": w.in_dtype, "state_dtype": "f32",
            "layer_replicas": R, "state_MiB_per_layer": state_mib,
            "working_set_MiB": round(sum(t.numel() * t.element_size() for st in states
                                         for t in st.buffers().values()) / 2**20, 1),
            "tokens_per_s_definition": "per-layer token-updates/s = B*R*K/elapsed",
        },
        "roofline": {
            "bound": "hbm",
            "kernel": "deltalog_kernel<GDN,128,128,STEP,bf16> (dl_append_step: append or merge)",
            "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": None,
            "avg_launch_us": round(avg_launch_us, 3),
            "algorithmic_bytes_per_launch": round(bytes_per_launch, 1),
            "duration_source": "HIP events around the timed region / launches",
        },
        "phases": {
            "source": "separate pass, HIP event pair around each launch",
            "append": {"us": round(app_us, 2), "GB/s": round(app_bytes / (app_us * 1e-6) / 1e9, 1),
                       "frac": round(app_bytes / (app_us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)},
            "merge": {"us": round(mrg_us, 2), "GB/s": round(mrg_bytes / (mrg_us * 1e-6) / 1e9, 1),
                      "frac": round(mrg_bytes / (mrg_us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)},
            "by_live_length": phases,
        },
        "eager": {
            "tokens_per_s": round(eg_tok, 1),
            "ms_per_step": round(eg_ms / K, 5),
            "us_per_launch": round(eg_us, 3),
            "GB/s": round(eg_gbs, 1),
            "frac": round(eg_gbs / HBM_PEAK_GBS, 4),
        },
        "speedup_vs_eager": round(dl_tok / eg_tok, 3),
        "state_write_ratio_model": round(T.state_write_ratio(w.op, w.dk, w.dv, w.M, w.in_dtype), 2),
    }
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(w, args.cpu_seconds)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
