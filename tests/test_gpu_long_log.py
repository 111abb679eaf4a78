"""GPU tests of the long-log build of the STEP and MERGE kernels (capacity C = M - 1 above
one coefficient pass of 16 entries), which the host picks from the merge interval: two
merge chunks staged by the coefficient passes for one log-decay per head, later chunks
staged from global memory one chunk ahead, the next pass's keys prefetched.  Every
operator against the fp64 oracle at capacities of 16 + 1 (one entry past a pass),
31 (two whole chunks) and 47 (a third chunk from global memory), a forced merge in the
middle of a chunk through dl_merge (the MERGE kernel's long build), a bf16 state, and
bitwise equality where every intermediate is exact."""

import numpy as np
import pytest
import torch

from oracle import eager as OE
from paper_2608_15533_amd import workloads as W

from gpu_harness import TOL_BF16_STATE, TOL_F32_STATE, D, Rollout, log, to_dev, token
from test_gpu_properties import dyadic_inputs, oracle_run, rel, run_deltalog

pytestmark = pytest.mark.gpu

WL = {"gdn": W.GDN_B64, "kda": W.KDA_B128, "rwkv6": W.RWKV6_B128,
      "linattn": W.LINATTN_B64, "retnet": W.RETNET_B64, "gla": W.GLA_B128}


def _check(r, what, tol=TOL_F32_STATE):
    e_flush = r.flush_and_check()
    log(f"{what}: max out err {r.err_out:.2e}, max state err {r.err_state:.2e} "
        f"({r.n_state_checks} merge checks), flush {e_flush:.2e}")
    assert r.device_error_word() == 0
    assert r.err_out <= tol, what
    assert r.err_state <= tol, what


@pytest.mark.parametrize("M", [18, 32, 48])
@pytest.mark.parametrize("op", list(WL))
def test_long_log_mid_size(op, M):
    """Full head shape, 3 slots, 2M+5 steps: two merges of a long log and a ragged cycle,
    every slot and every step against the oracle."""
    r = Rollout(WL[op], M=M, B=3, steps=2 * M + 5).run()
    assert r.n_state_checks == 2
    _check(r, f"{op} long M={M}")


@pytest.mark.parametrize("op", list(WL))
def test_long_log_bf16_state(op):
    """The long build with a bf16 dense state (no early chunk loads), M = 32."""
    M = 32
    r = Rollout(WL[op], M=M, B=3, steps=2 * M + 5, state_dtype="bf16").run()
    _check(r, f"{op} long M={M} bf16 state", tol=TOL_BF16_STATE)


@pytest.mark.parametrize("op", list(WL))
def test_long_log_forced_merge_mid_chunk(op):
    """M = 40: 25 appends (the second chunk holds 9 entries), then dl_merge with the next
    token (Eq. 6 at L = 25 < C = 39, the MERGE kernel's long build), then 20 more steps
    and a flush, against the eager oracle."""
    dl = D()
    w = WL[op].with_(B=3)
    M = 40
    S0 = W.initial_state(w)
    xs = [W.step_inputs(w, t) for t in range(46)]
    u = W.bonus(w)
    desc = dl.make_desc(op, w.B, w.H, w.dk, w.dv, M, w.in_dtype)
    ref_o, ref_S = oracle_run(op, S0, xs, u)
    outs, st = run_deltalog(desc, S0, xs[:25], u)
    assert np.all(st.len.cpu().numpy() == 25)
    o = torch.empty((w.B, w.H, w.dv), dtype=torch.float32, device="cuda")
    dl.dl_merge(desc, st, token(desc, xs[25], u), o)
    torch.cuda.synchronize()
    e_o, e_S = rel(o.cpu().numpy(), ref_o[25]), rel(st.S.cpu().numpy(), ref_S[25])
    log(f"{op} forced merge at L = 25 of C = 39: out {e_o:.2e}, state {e_S:.2e}")
    assert e_o <= TOL_F32_STATE and e_S <= TOL_F32_STATE
    assert np.all(st.len.cpu().numpy() == 0)
    for t in range(26, 46):
        dl.dl_append_step(desc, st, token(desc, xs[t], u), o)
        torch.cuda.synchronize()
        assert rel(o.cpu().numpy(), ref_o[t]) <= TOL_F32_STATE, t
    dl.dl_merge(desc, st)
    torch.cuda.synchronize()
    assert rel(st.S.cpu().numpy(), ref_S[45]) <= TOL_F32_STATE
    assert int(st.err.item()) == 0


@pytest.mark.parametrize("dk,dv", [(128, 128), (64, 64)])
@pytest.mark.parametrize("op", OE.OPS)
def test_long_log_exact_dyadic_bitwise(op, dk, dv):
    """M = 40 on inputs where every intermediate is exact in fp32 (one-hot keys, integer
    state and values, beta = 1, lambda = 0): 45 steps through the long build, outputs of
    every step and the base after the merge and after a flush equal the oracle bit for
    bit -- any indexing slip in the staged, prefetched or global chunks shows."""
    B, H, M, steps = 2, 2, 40, 45
    S0, xs, u = dyadic_inputs(op, B, H, dk, dv, steps, seed=400 + dk + OE.OPS.index(op))
    for x in xs:
        if x["beta"] is not None:
            x["beta"][:] = 1.0          # integers stay integers over many writes
    desc = D().make_desc(op, B, H, dk, dv, M, "bf16")
    outs, st = run_deltalog(desc, S0, xs, u)
    ref_o, ref_S = oracle_run(op, S0, xs, u)
    for t in range(steps):
        np.testing.assert_array_equal(outs[t].astype(np.float64), ref_o[t], err_msg=f"step {t}")
    D().dl_merge(desc, st)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(st.S.cpu().numpy().astype(np.float64), ref_S[-1])
