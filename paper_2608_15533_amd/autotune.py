"""Merge-interval selection from measured phase costs.

Sec. 3.2 prices one DeltaLog cycle in bytes (Eq. 10): the dense write is paid once
per M steps, while the replay stream grows with the live length, so the best M is a
trade-off that depends on the operator and on the kernels.  Bytes are a proxy; what a
deployment wants to minimise is time.  This module measures on the device the two
launch kinds a cycle consists of, at every live length, and predicts the amortised
step time of every merge interval from them:

    T(M) = ( a(0) + a(1) + ... + a(M-2) + m(M-1) ) / M

    a(L)  one dl_append_step over all slots at live length L (L < C: the append branch
          of Alg. 1, Eq. 5);
    m(L)  one dl_merge with the step's token at live length L (Eq. 6 at L; the merge
          a cycle of interval L+1 ends with).

T(1) = m(0) is the eager-equivalent cost: the state read and written every step.
Launch costs do not depend on the values in the state or the log, only on the live
length, so every length is measured directly by setting the live length before the
timed launches; no cycle has to be stepped through.
"""

import math

import torch

from . import deltalog as D


def predict(append_us, merge_us):
    """Amortised microseconds per step for M = 1 .. len(merge_us) (a dict M -> T(M)).

    ``append_us[L]`` is a(L) for L = 0 .. len(append_us)-1 and ``merge_us[L]`` is m(L);
    merge intervals whose appends were not measured are left out."""
    out = {}
    for M in range(1, len(merge_us) + 1):
        if M - 1 > len(append_us):
            break
        out[M] = (sum(append_us[:M - 1]) + merge_us[M - 1]) / M
    return out


def choose(append_us, merge_us):
    """The merge interval with the smallest predicted step time (the smallest such M on
    a tie) and the full prediction."""
    T = predict(append_us, merge_us)
    best = min(T, key=lambda M: (T[M], M))
    return best, T


def _token(desc, n, gen):
    """Bounded synthetic inputs of one step (their values do not change any cost)."""
    H, dk, dv = desc.heads, desc.dk, desc.dv
    it = torch.bfloat16 if desc.in_dtype == D.DL_BF16 else torch.float32
    dev = dict(device="cuda")
    q = (torch.randn(n, H, dk, generator=gen, **dev) / math.sqrt(dk)).to(it)
    k = (torch.randn(n, H, dk, generator=gen, **dev) / math.sqrt(dk)).to(it)
    v = torch.randn(n, H, dv, generator=gen, **dev).to(it)
    dl = D.decay_width(desc)
    lam = None
    if dl:
        shape = (n, H) if dl == 1 else (n, H, dl)
        lam = (-torch.nn.functional.softplus(torch.randn(shape, generator=gen, **dev)) / 16)
    beta = torch.sigmoid(torch.randn(n, H, generator=gen, **dev))
    u = 0.1 * torch.randn(H, dk, generator=gen, **dev)
    return D.Token(desc, n, q.contiguous(), k.contiguous(), v.contiguous(),
                   None if lam is None else lam.contiguous(), beta.contiguous(), u.contiguous())


def _timed(launch, states, reps, prepare):
    """Median over ``reps`` of the mean launch time (us) of one launch per state, with
    every state prepared (outside the timed region) before each repetition."""
    times = []
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    for _ in range(reps):
        for st in states:
            prepare(st)
        # Keep the device busy while the host enqueues the timed launches, so that the
        # interval holds launches only, not the host's submission time.
        if hasattr(torch.cuda, "_sleep"):
            torch.cuda._sleep(50_000 * len(states))
        e0.record()
        for st in states:
            launch(st)
        e1.record()
        e1.synchronize()
        times.append(e0.elapsed_time(e1) * 1e3 / len(states))
    times.sort()
    return times[len(times) // 2]


def calibrate(op, B, H, dk, dv, in_dtype="bf16", state_dtype="f32", max_M=64, replicas=0,
              reps=3, min_working_set=2**30, seed=20261202):
    """Measure a(L) for L = 0 .. max_M-2 and m(L) for L = 0 .. max_M-1 on cuda.

    ``replicas`` independent layer states (0: enough for ``min_working_set`` bytes of
    dense state, at most 16) are launched in turn, so that the timing reflects states
    streamed from HBM rather than held in the last-level cache.  Returns a dict with
    the two cost lists (microseconds per launch over all B slots) and the setup."""
    if not 2 <= max_M <= 64:
        raise ValueError("max_M must lie in [2, 64]")
    desc = D.make_desc(op, B, H, dk, dv, max_M, in_dtype, state_dtype)
    state_bytes = B * H * dk * dv * (2 if state_dtype == "bf16" else 4)
    R = replicas or max(1, min(16, -(-min_working_set // state_bytes)))
    gen = torch.Generator(device="cuda")
    gen.manual_seed(seed)
    states = [D.DeltaLogState(desc, 0.02 * torch.randn(B, H, dk, dv, generator=gen,
                                                         device="cuda")) for _ in range(R)]
    tok = _token(desc, B, gen)
    o = torch.empty((B, H, dv), dtype=torch.float32, device="cuda")

    def at_length(L):
        def prep(st):
            st.len.fill_(L)
        return prep

    for st in states:                                    # warm-up of both kernels
        D.dl_append_step(desc, st, tok, o)
        D.dl_merge(desc, st, tok, o)
    torch.cuda.synchronize()
    append_us = [_timed(lambda st: D.dl_append_step(desc, st, tok, o), states, reps,
                        at_length(L)) for L in range(max_M - 1)]
    merge_us = [_timed(lambda st: D.dl_merge(desc, st, tok, o), states, reps, at_length(L))
                for L in range(max_M)]
    errs = [int(st.err.item()) for st in states]
    if any(errs):
        raise RuntimeError(f"device error word set during calibration: {errs}")
    return {"op": op, "B": B, "H": H, "dk": dk, "dv": dv, "in_dtype": in_dtype,
            "state_dtype": state_dtype, "replicas": R, "reps": reps,
            "append_us": append_us, "merge_us": merge_us}
