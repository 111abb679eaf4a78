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
    return ap.parse_args()


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
                    events.append(torch.cuda.Event(enable_timing=True))
                    events[-1].record(stream)
                rc = fn(*argtab[r][k % POOL])
                if rc != 0:
                    raise D.DeltaLogError(rc, fn.__name__)

    def timed(fn, argtab):
        run(fn, argtab, 0, WU)
        torch.cuda.synchronize()
        evs = []
        t0 = torch.cuda.Event(enable_timing=True)
        t0.record(stream)
        run(fn, argtab, WU, K, evs)
        t1 = torch.cuda.Event(enable_timing=True)
        t1.record(stream)
        torch.cuda.synchronize()
        total_ms = t0.elapsed_time(t1)
        marks = evs + [t1]
        durs = np.array([marks[i].elapsed_time(marks[i + 1]) for i in range(len(evs))])
        return total_ms, durs.reshape(K, R)

    # ------------------------------------------------------------------ DeltaLog
    dl_ms, dl_durs = timed(app, app_args)
    for s in states:
        assert int(s.err.item()) == 0
    heads = w.B * w.H
    Ls = [(WU + k) % w.M for k in range(K)]           # live length at each timed step
    step_bytes = np.array([T.step_bytes(w.op, w.dk, w.dv, w.M, L, w.in_dtype).total * heads
                           for L in Ls])
    launch_bytes = np.repeat(step_bytes[:, None], R, axis=1)
    dl_tok = w.B * R * K / (dl_ms * 1e-3)
    achieved = launch_bytes.sum() / (dl_durs.sum() * 1e-3) / 1e9

    phases = {}
    for L in range(w.M):
        sel = np.array([l == L for l in Ls])
        if not sel.any():
            continue
        us = float(dl_durs[sel].mean() * 1e3)
        b = T.step_bytes(w.op, w.dk, w.dv, w.M, L, w.in_dtype).total * heads
        name = "merge" if L == w.M - 1 else f"append_L{L}"
        phases[name] = {"us": round(us, 2), "GB/s": round(b / (us * 1e-6) / 1e9, 1)}
    app_sel = np.array([l < w.M - 1 for l in Ls])
    app_us = float(dl_durs[app_sel].mean() * 1e3)
    app_bytes = float(launch_bytes[app_sel].mean())
    mrg_sel = ~app_sel
    mrg_us = float(dl_durs[mrg_sel].mean() * 1e3) if mrg_sel.any() else None
    mrg_bytes = float(launch_bytes[mrg_sel].mean()) if mrg_sel.any() else None

    # ------------------------------------------------------------------ eager baseline
    eg_ms, eg_durs = timed(eag, eag_args)
    eg_tok = w.B * R * K / (eg_ms * 1e-3)
    eg_bytes = T.eager_bytes(w.op, w.dk, w.dv, w.in_dtype).total * heads
    eg_gbs = eg_bytes / (eg_durs.mean() * 1e-3) / 1e9

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
            "avg_launch_us": round(float(dl_durs.mean() * 1e3), 3),
            "algorithmic_bytes_per_launch": round(float(launch_bytes.mean()), 1),
        },
        "phases": {
            "append": {"us": round(app_us, 2), "GB/s": round(app_bytes / (app_us * 1e-6) / 1e9, 1)},
            "merge": None if mrg_us is None else
            {"us": round(mrg_us, 2), "GB/s": round(mrg_bytes / (mrg_us * 1e-6) / 1e9, 1)},
            "by_live_length": phases,
        },
        "eager": {
            "tokens_per_s": round(eg_tok, 1),
            "ms_per_step": round(eg_ms / K, 5),
            "us_per_launch": round(float(eg_durs.mean() * 1e3), 3),
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
