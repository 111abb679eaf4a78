"""GPU tests of the value-tiled step (Sec. 3.3: ReplayPrep, per-tile AppendDecode,
Finalize) through the C ABI: parity with the fp64 oracle for every operator, tile
count and replay variant; split replay bit-identical to fused replay; the shared log
metadata identical to the untiled kernel's; slot lists and the error word."""

import numpy as np
import pytest
import torch

from oracle import eager as OE
from paper_2608_15533_amd import workloads as W

from gpu_harness import TOL_F32_STATE, D, Rollout, log, to_dev, token

pytestmark = pytest.mark.gpu

WL = {"gdn": W.GDN_B64, "kda": W.KDA_B128, "rwkv6": W.RWKV6_B128,
      "linattn": W.LINATTN_B64, "retnet": W.RETNET_B64, "gla": W.GLA_B128}


def _check(r, what):
    e_flush = r.flush_and_check()
    log(f"{what}: max out err {r.err_out:.2e}, max state err {r.err_state:.2e} "
        f"({r.n_state_checks} merge checks), flush {e_flush:.2e}")
    assert r.device_error_word() == 0
    assert r.err_out <= TOL_F32_STATE, what
    assert r.err_state <= TOL_F32_STATE, what


@pytest.mark.parametrize("split", [True, False], ids=["split", "fused"])
@pytest.mark.parametrize("nv", [2, 4])
@pytest.mark.parametrize("op", list(WL))
def test_tiled_mid_size_against_oracle(op, nv, split):
    """Full head shape, M = 8, 3 slots, 2M+5 steps (two merges and a ragged cycle)."""
    w = WL[op]
    r = Rollout(w, M=8, B=3, steps=21, tiled=(nv, split)).run()
    _check(r, f"tiled {op} nv={nv} {'split' if split else 'fused'}")


def test_tiled_full_size_gdn():
    """The full GDN 64x32x128^2, M = 16 workload (256 steps) on the tiled split path."""
    r = Rollout(W.GDN_B64, sample=[0, 33, 63], tiled=(4, True)).run()
    assert r.n_state_checks == W.GDN_B64.steps // W.GDN_B64.M
    _check(r, "tiled gdn full")


def test_tiled_staggered_slot_lists():
    """Layer 0 of the staggered 24-layer stack (warm-up through partial slot lists)."""
    w = W.GDN_STACK
    off = W.fill_offsets(w)
    sample = [int(np.argmax(off == o)) for o in (0, 9, 15) if np.any(off == o)]
    r = Rollout(w, sample=sample, tiled=(2, True)).run()
    _check(r, "tiled stack layer 0")


def _run_tiled(desc, S0, xs, u, nv, split, untiled=False):
    dl = D()
    st = dl.DeltaLogState(desc, to_dev(S0, torch.float32))
    ws = dl.tiled_workspace(desc, desc.num_slots)
    outs = []
    for x in xs:
        tok = token(desc, x, u)
        o = torch.empty((desc.num_slots, desc.heads, desc.dv), dtype=torch.float32, device="cuda")
        if untiled:
            dl.dl_append_step(desc, st, tok, o)
        else:
            dl.dl_append_step_tiled(desc, st, tok, o, value_tiles=nv, split_replay=split,
                                    workspace=ws)
        outs.append(o)
    torch.cuda.synchronize()
    # bf16 buffers are widened to fp32 (exactly) for numpy
    bufs = {k: (None if v is None else
                (v.float() if v.dtype == torch.bfloat16 else v).cpu().numpy().copy())
            for k, v in st.buffers().items()}
    return [o.cpu().numpy() for o in outs], bufs


@pytest.mark.parametrize("op", list(WL))
def test_split_replay_is_bitwise_fused_replay(op):
    """The prepared coefficients are the fused tiles' own coefficients: same bits."""
    w = WL[op].with_(B=4)
    M, steps = 8, 11
    S0 = W.initial_state(w)
    xs = [W.step_inputs(w, t) for t in range(steps)]
    u = W.bonus(w)
    desc = D().make_desc(op, w.B, w.H, w.dk, w.dv, M, w.in_dtype)
    o1, b1 = _run_tiled(desc, S0, xs, u, 4, True)
    o2, b2 = _run_tiled(desc, S0, xs, u, 4, False)
    for t in range(steps):
        np.testing.assert_array_equal(o1[t], o2[t], err_msg=f"step {t}")
    for k in b1:
        if b1[k] is not None:
            np.testing.assert_array_equal(b1[k], b2[k], err_msg=k)


@pytest.mark.parametrize("op", list(WL))
def test_tiled_log_metadata_matches_untiled(op):
    """After appends, the single-writer entries (K_log, Lam_log) and the finalized L
    equal the untiled kernel's bit for bit; U_log and outputs agree to the bar (bitwise
    where U_log is a copy of v)."""
    w = WL[op].with_(B=3)
    M, steps = 8, 5
    S0 = W.initial_state(w)
    xs = [W.step_inputs(w, t) for t in range(steps)]
    u = W.bonus(w)
    desc = D().make_desc(op, w.B, w.H, w.dk, w.dv, M, w.in_dtype)
    ot, bt = _run_tiled(desc, S0, xs, u, 2, True)
    ou, bu = _run_tiled(desc, S0, xs, u, 0, False, untiled=True)
    for k in ("k_log", "lam_log", "len", "S", "err"):
        if bu[k] is not None:
            np.testing.assert_array_equal(bt[k], bu[k], err_msg=k)
    L = steps
    Ut = bt["u_log"][:, :, :L].astype(np.float64)
    Uu = bu["u_log"][:, :, :L].astype(np.float64)
    if op in OE.DELTA_OPS:
        assert OE.rel_fro(Ut, Uu) <= TOL_F32_STATE
    else:
        np.testing.assert_array_equal(Ut, Uu)
    for t in range(steps):
        assert OE.rel_fro(ot[t], ou[t]) <= TOL_F32_STATE


def test_tiled_bad_slot_sets_error_word_and_writes_nothing():
    dl = D()
    w = W.GDN_B64.with_(B=2, H=2)
    desc = dl.make_desc("gdn", w.B, w.H, w.dk, w.dv, 4, w.in_dtype)
    st = dl.DeltaLogState(desc, to_dev(W.initial_state(w), torch.float32))
    ws = dl.tiled_workspace(desc, 1)
    before = {k: v.float().cpu().numpy().copy() for k, v in st.buffers().items()
              if v is not None}
    x = W.step_inputs(w, 0)
    o = torch.zeros((1, w.H, w.dv), dtype=torch.float32, device="cuda")
    dl.dl_append_step_tiled(desc, st, token(desc, x, rows=[0]), o,
                            slots=torch.tensor([7], dtype=torch.int32, device="cuda"),
                            value_tiles=4, split_replay=True, workspace=ws)
    torch.cuda.synchronize()
    assert int(st.err.item()) == 1
    for k, v in st.buffers().items():
        if k != "err" and v is not None:
            np.testing.assert_array_equal(before[k], v.float().cpu().numpy(), err_msg=k)
