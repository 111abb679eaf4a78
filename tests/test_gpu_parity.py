"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle on seeded inputs.

Bar: relative Frobenius error <= 1e-4 for fp32 state, on every step's outputs, on the
dense base after every merge, and on the base after a final flush.  Mid-size cases run
every slot through the oracle; the full-size workloads (the launch configuration the
benchmark times) run every slot on the GPU and a sample of slots through the oracle."""

import numpy as np
import pytest

from paper_2608_15533_amd import workloads as W

from gpu_harness import TOL_BF16_STATE, TOL_F32_STATE, Rollout, log

pytestmark = pytest.mark.gpu


def _check(r, what, tol=TOL_F32_STATE):
    e_flush = r.flush_and_check()
    log(f"{what}: max out err {r.err_out:.2e}, max state err {r.err_state:.2e} "
        f"({r.n_state_checks} merge checks), flush {e_flush:.2e}")
    assert r.device_error_word() == 0
    assert r.err_out <= tol, what
    assert r.err_state <= tol, what


@pytest.mark.parametrize("in_dtype", ["f32", "bf16"])
@pytest.mark.parametrize("eager", [False, True], ids=["deltalog", "eager"])
def test_gdn_b1_h2_d64_m8(in_dtype, eager):
    """1 sequence, 2 heads, 64x64, M = 8, 64 steps: every output, 8 merges, flush."""
    w = W.GDN_SMALL.with_(in_dtype=in_dtype)
    r = Rollout(w, eager=eager).run()
    assert eager or r.n_state_checks == w.steps // w.M
    _check(r, f"gdn small {in_dtype} {'eager' if eager else 'deltalog'}")


MID = [
    ("gdn", W.GDN_B64, 16), ("kda", W.KDA_B128, 8), ("kda", W.KDA_B128, 16),
    ("kda", W.KDA_B128, 32), ("rwkv6", W.RWKV6_B128, 16),
    ("linattn", W.LINATTN_B64, 16), ("retnet", W.RETNET_B64, 16), ("gla", W.GLA_B128, 16),
]


@pytest.mark.parametrize("op,w,M", MID, ids=[f"{o}_m{m}" for o, _, m in MID])
@pytest.mark.parametrize("eager", [False, True], ids=["deltalog", "eager"])
def test_mid_size_all_slots(op, w, M, eager):
    """Full head shape and merge interval, 3 slots, 2M+5 steps (two merges and a ragged
    partial cycle), every slot checked."""
    r = Rollout(w, M=M, B=3, steps=2 * M + 5, eager=eager).run()
    _check(r, f"{op} mid M={M} {'eager' if eager else 'deltalog'}")


FULL = [
    ("gdn_b64_h32_d128_m16", W.GDN_B64, 16, [0, 17, 63]),
    ("kda_b128_h32_d128_m8", W.KDA_B128, 8, [1, 64, 127]),
    ("kda_b128_h32_d128_m16", W.KDA_B128, 16, [2, 77, 126]),
    ("kda_b128_h32_d128_m32", W.KDA_B128, 32, [3, 90, 125]),
    ("rwkv6_b128_h40_d64_m16", W.RWKV6_B128, 16, [0, 55, 127]),
    ("linattn_b64_h32_d128_m16", W.LINATTN_B64, 16, [0, 21, 63]),
    ("retnet_b64_h32_d128_m16", W.RETNET_B64, 16, [5, 40, 62]),
    ("gla_b128_h32_d128_m16", W.GLA_B128, 16, [4, 66, 127]),
]


@pytest.mark.parametrize("name,w,M,sample", FULL, ids=[f[0] for f in FULL])
def test_full_size_sampled(name, w, M, sample):
    """The full workload (all slots, all steps) on the GPU; the oracle follows 3 slots."""
    r = Rollout(w, M=M, sample=sample).run()
    assert r.n_state_checks == w.steps // M
    _check(r, f"{name} full")


@pytest.mark.parametrize("layer", [0, 23])
def test_serving_stack_layer_staggered(layer):
    """One layer of the 24-layer stack: 256 slots whose logs start at staggered fill
    offsets (partial-batch warm-up through slot lists), 128 steps; the oracle follows
    slots with different offsets, so merges land on different steps."""
    w = W.GDN_STACK
    off = W.fill_offsets(w)
    sample = [int(np.argmax(off == o)) for o in (0, 7, 15) if np.any(off == o)]
    r = Rollout(w, layer=layer, sample=sample).run()
    assert r.n_state_checks >= w.steps // w.M
    _check(r, f"stack layer {layer} staggered")


BF16_STATE = [("gdn", W.GDN_B64, 16), ("kda", W.KDA_B128, 16), ("rwkv6", W.RWKV6_B128, 16),
              ("linattn", W.LINATTN_B64, 16), ("retnet", W.RETNET_B64, 16),
              ("gla", W.GLA_B128, 16)]


@pytest.mark.parametrize("op,w,M", BF16_STATE, ids=[o for o, _, _ in BF16_STATE])
@pytest.mark.parametrize("eager", [False, True], ids=["deltalog", "eager"])
def test_bf16_state_mid_size(op, w, M, eager):
    """bf16 state (rounded on every store), 3 slots, 4 cycles + a ragged tail, 2e-2 bar."""
    r = Rollout(w, M=M, B=3, steps=4 * M + 5, eager=eager, state_dtype="bf16").run()
    _check(r, f"{op} bf16 state {'eager' if eager else 'deltalog'}", tol=TOL_BF16_STATE)


def test_bf16_state_full_size_gdn():
    """The full GDN 64x32x128^2 workload (256 steps) with a bf16 state; 3 sampled slots."""
    r = Rollout(W.GDN_B64, sample=[0, 31, 63], state_dtype="bf16").run()
    _check(r, "gdn full bf16 state", tol=TOL_BF16_STATE)


LONG = [("gdn", W.GDN_B64, 16), ("kda", W.KDA_B128, 16), ("rwkv6", W.RWKV6_B128, 16),
        ("linattn", W.LINATTN_B64, 16), ("retnet", W.RETNET_B64, 16), ("gla", W.GLA_B128, 16)]


@pytest.mark.parametrize("op,w,M", LONG, ids=[o for o, _, _ in LONG])
def test_long_rollout_no_drift(op, w, M):
    """1 slot at full head shape through 64 merge cycles (1024 steps): the fp32
    DeltaLog path stays within the bar against the fp64 oracle on every output and
    after every merge, and its error in the last 16 cycles is of the same order as in
    the first 16 (no growth from the repeated log replay and merge)."""
    r = Rollout(w, M=M, B=1, steps=64 * M)
    quarter, errs = 16 * M, []
    for t in range(r.steps):
        if t % quarter == 0:
            errs.append(0.0)
            r.err_out = 0.0
        x = W.step_inputs(r.w, t, r.layer)
        r._step_rows(x, np.arange(r.w.B))
        errs[-1] = max(errs[-1], r.err_out)
    r.err_out = max(errs)
    log(f"{op} long rollout, output error per 16 cycles: "
        + ", ".join(f"{e:.1e}" for e in errs))
    _check(r, f"{op} long rollout M={M} x 64 cycles")
    assert errs[-1] <= 10 * max(errs[0], 1e-7), errs


@pytest.mark.parametrize("eager", [False, True], ids=["deltalog", "eager"])
def test_deltanet_is_gdn_without_decay(eager):
    """DeltaNet (the delta rule without a gate) is GDN with lambda = 0: the GDN
    kernels, fed zero log-decays, follow the oracle on the full head shape through two
    merges and a ragged partial cycle."""
    M = 16
    r = Rollout(W.GDN_B64, M=M, B=3, steps=2 * M + 5, eager=eager)
    for t in range(r.steps):
        x = dict(W.step_inputs(r.w, t, r.layer))
        x["lam"] = np.zeros_like(x["lam"])
        r._step_rows(x, np.arange(r.w.B))
    _check(r, f"deltanet (gdn, lambda = 0) {'eager' if eager else 'deltalog'}")


CAMPAIGN = [("gdn", W.GDN_B64, 16), ("kda", W.KDA_B128, 16), ("rwkv6", W.RWKV6_B128, 16)]


@pytest.mark.parametrize("B", [64, 128, 256])
@pytest.mark.parametrize("op,w,M", CAMPAIGN, ids=[o for o, _, _ in CAMPAIGN])
def test_rollout_against_dense_eager_all_slots(op, w, M, B):
    """The numerical check of Sec. 5 at full size: 128-token rollouts at B in {64, 128,
    256}, DeltaLog against the eager dense kernel on the same inputs, every slot and
    head compared.  Reports the largest output relative error (over steps, and over
    single (slot, head) rows) and the state relative error after a flush; both paths
    are fp32, so the bar is the fp32 one."""
    import torch
    from gpu_harness import D, to_dev, token

    dl = D()
    w = w.with_(B=B)
    steps = 128
    desc = dl.make_desc(op, B, w.H, w.dk, w.dv, M, w.in_dtype)
    S0 = W.initial_state(w)
    st = dl.DeltaLogState(desc, to_dev(S0, torch.float32))
    Se = to_dev(S0, torch.float32)
    del S0
    u = W.bonus(w)
    o = torch.empty((B, w.H, w.dv), dtype=torch.float32, device="cuda")
    oe = torch.empty_like(o)
    worst_step = worst_row = 0.0
    for t in range(steps):
        tok = token(desc, W.step_inputs(w, t), u)
        dl.dl_append_step(desc, st, tok, o)
        dl.dl_eager_step(desc, Se, tok, oe)
        diff = (o - oe).double()
        ref = oe.double()
        worst_step = max(worst_step, float(diff.norm() / ref.norm()))
        row = diff.norm(dim=-1) / ref.norm(dim=-1).clamp_min(1e-30)
        worst_row = max(worst_row, float(row.max()))
    dl.dl_merge(desc, st)
    torch.cuda.synchronize()
    ds = (st.S.double() - Se.double())
    state_err = float(ds.norm() / Se.double().norm())
    state_row = float((ds.flatten(2).norm(dim=-1) / Se.double().flatten(2).norm(dim=-1)).max())
    log(f"{op} B={B} M={M}, 128 steps vs eager: output rel err max over steps {worst_step:.2e}, "
        f"max over (step, slot, head) {worst_row:.2e}; flushed state rel err {state_err:.2e}, "
        f"max over (slot, head) {state_row:.2e}")
    assert int(st.err.item()) == 0
    assert worst_row <= TOL_F32_STATE and state_row <= TOL_F32_STATE


# beta exists only for the delta rule; linear attention has no decay to vary
DEGENERATE = [(op, case) for op in ("gdn", "kda", "rwkv6", "linattn", "retnet", "gla")
              for case in ("zero_beta", "zero_keys", "strong_decay", "no_decay")
              if not (case == "zero_beta" and op not in ("gdn", "kda"))
              and not (case in ("strong_decay", "no_decay") and op == "linattn")]


@pytest.mark.parametrize("op,case", DEGENERATE, ids=[f"{o}-{c}" for o, c in DEGENERATE])
def test_degenerate_inputs(op, case):
    """Degenerate gates and factors through two merge cycles at full head shape: no write
    (beta = 0, delta rule only), zero keys (no update at all), a decay so strong that
    exp(ell) underflows within the cycle (lambda = -30 per step; every factor is an exp
    of a log-decay difference, so nothing overflows), and no decay (lambda = 0).  The
    oracle follows every slot; the bar is the fp32 one and no NaN or Inf may appear."""
    w = {"gdn": W.GDN_B64, "kda": W.KDA_B128, "rwkv6": W.RWKV6_B128,
         "linattn": W.LINATTN_B64, "retnet": W.RETNET_B64, "gla": W.GLA_B128}[op]
    M = 8
    r = Rollout(w, M=M, B=2, steps=2 * M + 3)
    for t in range(r.steps):
        x = dict(W.step_inputs(r.w, t, r.layer))
        if case == "zero_beta":
            x["beta"] = np.zeros_like(x["beta"])
        elif case == "zero_keys":
            x["k"] = np.zeros_like(x["k"])
        elif case == "strong_decay":
            x["lam"] = np.full_like(x["lam"], -30.0)
        else:
            x["lam"] = np.zeros_like(x["lam"])
        r._step_rows(x, np.arange(r.w.B))
    o = r.o.cpu().numpy()
    assert np.isfinite(o).all() and np.isfinite(r.base().float().cpu().numpy()).all()
    _check(r, f"{op} {case}")
