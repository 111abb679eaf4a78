"""Helpers shared by the GPU parity tests: drive the HIP path through the C ABI and the
fp64 oracle on the same seeded inputs.  Not collected by pytest."""

import sys

import numpy as np
import torch

from oracle import eager as OE
from paper_2608_15533_amd import workloads as W

TOL_F32_STATE = 1e-4        # relative Frobenius error bar for fp32 state
TOL_BF16_STATE = 2e-2       # ... and for bf16 state (the state is rounded on every store)


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def D():
    from paper_2608_15533_amd import deltalog
    return deltalog


def to_dev(a, dtype):
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda").to(dtype).contiguous()


def token(desc, x, u=None, rows=None):
    """Device Token from a step-input dict (numpy float32 arrays, optional row subset)."""
    dl = D()
    it = torch.bfloat16 if desc.in_dtype == dl.DL_BF16 else torch.float32
    if rows is not None:
        x = W.select_rows(x, rows)
    n = x["q"].shape[0]
    beta = None if x.get("beta") is None else to_dev(x["beta"], torch.float32)
    ud = None if u is None else to_dev(u, torch.float32)
    lam = None if x.get("lam") is None else to_dev(x["lam"], torch.float32)
    return dl.Token(desc, n, to_dev(x["q"], it), to_dev(x["k"], it), to_dev(x["v"], it),
                    lam, beta, ud)


def sub(x, rows):
    """fp64 copy of rows of a step-input dict."""
    return {k: (None if a is None else np.asarray(a[rows], dtype=np.float64)) for k, a in x.items()}


def oracle_step(op, S, x, u):
    """One eager fp64 step of the oracle on [N, H, ...] arrays."""
    ub = None if u is None else np.broadcast_to(np.asarray(u, dtype=np.float64), x["k"].shape)
    return OE.eager_step(op, S, x["q"], x["k"], x["v"], x.get("beta"), x["lam"], u=ub)


def rel(x, ref):
    return OE.rel_fro(x, ref)


class Rollout:
    """A DeltaLog (or eager) rollout of workload ``w`` on the GPU, with the fp64 oracle
    following the slots in ``sample`` (all slots by default).

    Checks, per step, the sampled outputs; after each step, the dense base of every
    sampled slot that merged in it; at the end (after a flush), every sampled base.
    Returns the worst relative errors seen.
    """

    def __init__(self, w, M=None, layer=0, sample=None, eager=False, B=None, steps=None,
                 state_dtype="f32", tiled=None):
        self.dl = D()
        self.w = w if B is None else w.with_(B=B)
        self.M = w.M if M is None else M
        self.layer = layer
        self.steps = w.steps if steps is None else steps
        self.eager = eager
        self.tiled = tiled                    # None, or (value_tiles, split_replay)
        w = self.w
        self.sample = np.arange(w.B) if sample is None else np.asarray(sample)
        self.desc = self.dl.make_desc(w.op, w.B, w.H, w.dk, w.dv, self.M, w.in_dtype,
                                      state_dtype)
        S0 = W.initial_state(w, layer)
        if state_dtype == "bf16":
            S0 = W.round_bf16(S0)                   # the stored prefill state
        self.u = W.bonus(w, layer)
        st = torch.bfloat16 if state_dtype == "bf16" else torch.float32
        if eager:
            self.S = to_dev(S0, st)
        else:
            self.state = self.dl.DeltaLogState(self.desc, to_dev(S0, torch.float32))
        self.S_ref = S0[self.sample].astype(np.float64)
        self.o = torch.empty((w.B, w.H, w.dv), dtype=torch.float32, device="cuda")
        self.ws = (self.dl.tiled_workspace(self.desc, w.B)
                   if tiled is not None and tiled[1] else None)
        self.err_out = 0.0
        self.err_state = 0.0
        self.n_state_checks = 0
        self.live = np.zeros(w.B, dtype=np.int64)      # host mirror of the live length

    def base(self):
        return self.S if self.eager else self.state.S

    def _step_rows(self, x, rows, check_out=True):
        dl, w = self.dl, self.w
        n = len(rows)
        full = n == w.B and np.array_equal(rows, np.arange(w.B))
        tok = token(self.desc, x, self.u, rows=None if full else rows)
        slots = None if full else torch.from_numpy(np.asarray(rows, dtype=np.int32)).to("cuda")
        o = self.o[:n]
        if self.eager:
            dl.dl_eager_step(self.desc, self.S, tok, o, slots=slots)
        elif self.tiled is not None:
            dl.dl_append_step_tiled(self.desc, self.state, tok, o, slots=slots,
                                    value_tiles=self.tiled[0], split_replay=self.tiled[1],
                                    workspace=self.ws)
        else:
            dl.dl_append_step(self.desc, self.state, tok, o, slots=slots)
        # oracle on the sampled slots that took this step
        pos = {int(s): i for i, s in enumerate(rows)}
        mine = [j for j, s in enumerate(self.sample) if int(s) in pos]
        if not mine:
            return
        take = np.array([pos[int(self.sample[j])] for j in mine])
        xs = sub(x if full else W.select_rows(x, rows), take)
        S_new, o_ref = oracle_step(w.op, self.S_ref[mine], xs, self.u)
        self.S_ref[mine] = S_new
        if check_out:
            got = o[torch.from_numpy(take).to("cuda")].cpu().numpy()
            self.err_out = max(self.err_out, rel(got, o_ref))
        merged_now = []
        for j in mine:
            s = int(self.sample[j])
            if self.eager or self.live[s] == self.M - 1:
                merged_now.append(j)
        for s in rows:
            self.live[s] = 0 if (self.eager or self.live[s] == self.M - 1) else self.live[s] + 1
        if merged_now:
            idx = torch.from_numpy(self.sample[merged_now].astype(np.int64)).to("cuda")
            got = self.base()[idx].float().cpu().numpy()
            self.err_state = max(self.err_state, rel(got, self.S_ref[merged_now]))
            self.n_state_checks += 1

    def warmup(self):
        """Bring slot b to live length o_b (staggered workloads) with partial batches."""
        for r, rows in W.warmup_schedule(self.w):
            x = W.step_inputs(self.w, 0, self.layer, warmup=r)
            self._step_rows(x, rows[np.isin(rows, np.arange(self.w.B))])

    def run(self):
        if self.w.staggered:
            self.warmup()
        for t in range(self.steps):
            x = W.step_inputs(self.w, t, self.layer)
            self._step_rows(x, np.arange(self.w.B))
        torch.cuda.synchronize()
        return self

    def flush_and_check(self):
        if not self.eager:
            self.dl.dl_merge(self.desc, self.state)
            torch.cuda.synchronize()
        idx = torch.from_numpy(self.sample.astype(np.int64)).to("cuda")
        got = self.base()[idx].float().cpu().numpy()
        e = rel(got, self.S_ref)
        self.err_state = max(self.err_state, e)
        return e

    def device_error_word(self):
        return 0 if self.eager else int(self.state.err.item())
