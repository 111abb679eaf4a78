"""GPU properties of the HIP path, through the C ABI: exact (bitwise) results where all
arithmetic is exact, M = 1 equals the eager kernel, determinism, slot-order and batch
composition invariance, readout immutability, forced merge and flush, log contents,
device-detected corruption, every supported head shape, the largest merge interval."""

import numpy as np
import pytest
import torch

from oracle import eager as OE
from oracle.deltalog_model import DeltaLogModel
from paper_2608_15533_amd import workloads as W

from gpu_harness import TOL_BF16_STATE, TOL_F32_STATE, D, log, oracle_step, rel, to_dev, token

pytestmark = pytest.mark.gpu

OPS = OE.OPS
SHAPES = ((64, 64), (128, 128), (64, 128), (128, 64))
WL = {"gdn": W.GDN_B64, "kda": W.KDA_B128, "rwkv6": W.RWKV6_B128,
      "linattn": W.LINATTN_B64, "retnet": W.RETNET_B64, "gla": W.GLA_B128}


def lam_rows(x, N):
    """lambda of a step-input dict as [N, dl] rows (None for linear attention)."""
    return None if x["lam"] is None else x["lam"].reshape(N, -1)


def dyadic_inputs(op, B, H, dk, dv, steps, seed):
    """Inputs whose every intermediate is exact in fp32: one-hot keys, integer state and
    values, queries with 4 entries in {-1, 1}, beta in {1, 1/2}, lambda = 0 (none for
    linear attention), dyadic u."""
    rng = np.random.default_rng(seed)
    S0 = rng.integers(-3, 4, size=(B, H, dk, dv)).astype(np.float32)
    xs = []
    for _ in range(steps):
        k = np.zeros((B, H, dk), np.float32)
        idx = rng.integers(0, dk, size=(B, H))
        np.put_along_axis(k, idx[..., None], 1.0, axis=-1)
        q = np.zeros((B, H, dk), np.float32)
        for b in range(B):
            for h in range(H):
                pos = rng.choice(dk, 4, replace=False)
                q[b, h, pos] = rng.choice([-1.0, 1.0], 4)
        v = rng.integers(-4, 5, size=(B, H, dv)).astype(np.float32)
        lam = (None if op == "linattn" else
               np.zeros((B, H) if op in ("gdn", "retnet") else (B, H, dk), np.float32))
        beta = (rng.choice([1.0, 0.5], size=(B, H)).astype(np.float32)
                if op in OE.DELTA_OPS else None)
        xs.append(dict(q=q, k=k, v=v, lam=lam, beta=beta))
    u = (rng.integers(-4, 5, size=(H, dk)) / 4.0).astype(np.float32) if op == "rwkv6" else None
    return S0, xs, u


def run_deltalog(desc, S0, xs, u, slots_per_step=None):
    """Run steps through dl_append_step; returns (outputs list, state object)."""
    dl = D()
    st = dl.DeltaLogState(desc, to_dev(S0, torch.float32))
    outs = []
    for t, x in enumerate(xs):
        rows = None if slots_per_step is None else slots_per_step[t]
        n = desc.num_slots if rows is None else len(rows)
        tok = token(desc, x, u, rows=rows)
        o = torch.empty((n, desc.heads, desc.dv), dtype=torch.float32, device="cuda")
        sl = None if rows is None else torch.tensor(rows, dtype=torch.int32, device="cuda")
        dl.dl_append_step(desc, st, tok, o, slots=sl)
        outs.append(o)
    torch.cuda.synchronize()
    return [o.cpu().numpy() for o in outs], st


def run_eager(desc, S0, xs, u):
    dl = D()
    S = to_dev(S0, dl.state_torch_dtype(desc))
    outs = []
    for x in xs:
        tok = token(desc, x, u)
        o = torch.empty((desc.num_slots, desc.heads, desc.dv), dtype=torch.float32, device="cuda")
        dl.dl_eager_step(desc, S, tok, o)
        outs.append(o)
    torch.cuda.synchronize()
    return [o.cpu().numpy() for o in outs], S


def oracle_run(op, S0, xs, u):
    S = S0.astype(np.float64)
    outs, states = [], []
    for x in xs:
        S, o = oracle_step(op, S, {k: (None if a is None else a.astype(np.float64))
                                   for k, a in x.items()}, u)
        outs.append(o)
        states.append(S)
    return outs, states


@pytest.mark.parametrize("in_dtype", ["bf16", "f32"])
@pytest.mark.parametrize("dk,dv", SHAPES)
@pytest.mark.parametrize("op", OPS)
def test_exact_dyadic_bitwise(op, dk, dv, in_dtype):
    """All intermediates are exact in fp32, so the GPU must equal the oracle bit for bit
    (outputs every step, the base after each merge, the base after a flush)."""
    log(f"exact dyadic {op} {dk}x{dv} {in_dtype}")
    B, H, M, steps = 3, 2, 4, 8
    S0, xs, u = dyadic_inputs(op, B, H, dk, dv, steps, seed=dk + dv + OPS.index(op))
    desc = D().make_desc(op, B, H, dk, dv, M, in_dtype)
    outs, st = run_deltalog(desc, S0, xs, u)
    ref_o, ref_S = oracle_run(op, S0, xs, u)
    for t in range(steps):
        np.testing.assert_array_equal(outs[t].astype(np.float64), ref_o[t], err_msg=f"step {t}")
    np.testing.assert_array_equal(st.S.cpu().numpy().astype(np.float64), ref_S[M * (steps // M) - 1])
    eo, eS = run_eager(desc, S0, xs, u)
    for t in range(steps):
        np.testing.assert_array_equal(eo[t].astype(np.float64), ref_o[t], err_msg=f"eager step {t}")
    np.testing.assert_array_equal(eS.cpu().numpy().astype(np.float64), ref_S[-1])


@pytest.mark.parametrize("op", OPS)
def test_merge_interval_1_equals_eager_bitwise(op):
    """M = 1 makes every step a merge: the DeltaLog kernel must reproduce the eager
    kernel bit for bit (same arithmetic, same order)."""
    w = WL[op].with_(B=4)
    S0 = W.initial_state(w)
    xs = [W.step_inputs(w, t) for t in range(6)]
    u = W.bonus(w)
    desc = D().make_desc(op, w.B, w.H, w.dk, w.dv, 1, w.in_dtype)
    o1, st = run_deltalog(desc, S0, xs, u)
    o2, S2 = run_eager(desc, S0, xs, u)
    for a, b in zip(o1, o2):
        np.testing.assert_array_equal(a, b)
    np.testing.assert_array_equal(st.S.cpu().numpy(), S2.cpu().numpy())


def _state_arrays(st):
    """Host copies of every state buffer (bf16 buffers widened to fp32, exactly)."""
    return {k: (v.float() if v.dtype == torch.bfloat16 else v).cpu().numpy().copy()
            for k, v in st.buffers().items() if v is not None}


@pytest.mark.parametrize("op", OPS)
def test_deterministic_and_slot_order_invariant(op):
    """Two runs are bitwise identical; running the slots in a permuted order (a shuffled
    slot list) gives every slot bitwise the same state, log and outputs."""
    w = WL[op].with_(B=6)
    M, steps = 4, 7
    S0 = W.initial_state(w)
    xs = [W.step_inputs(w, t) for t in range(steps)]
    u = W.bonus(w)
    desc = D().make_desc(op, w.B, w.H, w.dk, w.dv, M, w.in_dtype)
    o1, st1 = run_deltalog(desc, S0, xs, u)
    o2, st2 = run_deltalog(desc, S0, xs, u)
    perm = [4, 1, 5, 0, 3, 2]
    o3, st3 = run_deltalog(desc, S0, xs, u, slots_per_step=[perm] * steps)
    a1, a2, a3 = _state_arrays(st1), _state_arrays(st2), _state_arrays(st3)
    for k in a1:
        np.testing.assert_array_equal(a1[k], a2[k], err_msg=k)
        np.testing.assert_array_equal(a1[k], a3[k], err_msg=k)
    for t in range(steps):
        np.testing.assert_array_equal(o1[t], o2[t])
        np.testing.assert_array_equal(o1[t][perm], o3[t])


@pytest.mark.parametrize("op", OPS)
def test_batch_composition_invariance(op):
    """A slot's result does not depend on which other slots share the launch: stepping
    slots in varying subsets equals stepping each subset's slots in full launches."""
    w = WL[op].with_(B=5)
    M, steps = 3, 6
    S0 = W.initial_state(w)
    xs = [W.step_inputs(w, t) for t in range(steps)]
    u = W.bonus(w)
    desc = D().make_desc(op, w.B, w.H, w.dk, w.dv, M, w.in_dtype)
    rng = np.random.default_rng(3)
    sets = [sorted(rng.choice(w.B, size=rng.integers(1, w.B + 1), replace=False).tolist())
            for _ in range(steps)]
    o_part, st_part = run_deltalog(desc, S0, xs, u, slots_per_step=sets)
    # Reference: the oracle model, stepping exactly the listed slots.
    model = DeltaLogModel(op, S0.reshape(-1, w.dk, w.dv), M)
    ub = None if u is None else np.broadcast_to(u, (w.B, w.H, w.dk)).reshape(-1, w.dk)
    for t, rows in enumerate(sets):
        act = np.zeros((w.B, w.H), bool)
        act[rows] = True
        x = xs[t]
        o = model.step(x["q"].reshape(-1, w.dk), x["k"].reshape(-1, w.dk), x["v"].reshape(-1, w.dv),
                       None if x["beta"] is None else x["beta"].reshape(-1),
                       lam_rows(x, w.B * w.H), u=ub, active=act.reshape(-1))
        ref = o.reshape(w.B, w.H, w.dv)[rows]
        assert rel(o_part[t], ref) <= TOL_F32_STATE
    assert rel(st_part.S.cpu().numpy(), model.Sbar.reshape(w.B, w.H, w.dk, w.dv)) <= TOL_F32_STATE
    np.testing.assert_array_equal(st_part.len.cpu().numpy(), model.L.reshape(w.B, w.H))


@pytest.mark.parametrize("op", OPS)
def test_log_contents_match_the_model(op):
    """After L appends the log holds: K_log = k bitwise (exact copies), Lam_log = the
    cumulative log-decay at each entry, its newest entry = the model's ell (none for
    linear attention), U_log = the delta-rule values b
    (GDN/KDA) or v bitwise (the others), len = L -- compared with the fp64 Alg. 1 model."""
    w = WL[op].with_(B=3)
    M, steps = 8, 5
    S0 = W.initial_state(w)
    xs = [W.step_inputs(w, t) for t in range(steps)]
    u = W.bonus(w)
    desc = D().make_desc(op, w.B, w.H, w.dk, w.dv, M, w.in_dtype)
    _, st = run_deltalog(desc, S0, xs, u)
    N = w.B * w.H
    model = DeltaLogModel(op, S0.reshape(N, w.dk, w.dv), M)
    ub = None if u is None else np.broadcast_to(u, (w.B, w.H, w.dk)).reshape(N, w.dk)
    for x in xs:
        model.step(x["q"].reshape(N, -1), x["k"].reshape(N, -1), x["v"].reshape(N, -1),
                   None if x["beta"] is None else x["beta"].reshape(N), lam_rows(x, N), u=ub)
    a = _state_arrays(st)
    L = steps
    assert np.all(a["len"] == L)
    K = a["k_log"].astype(np.float64).reshape(N, M - 1, w.dk)[:, :L]
    np.testing.assert_array_equal(K, model.K[:, :L])
    if op == "linattn":
        assert "lam_log" not in a
    else:
        lam_log = a["lam_log"]
        if lam_log.ndim == 3:               # scalar snapshots: entry-major [B, C, H]
            lam_log = lam_log.transpose(0, 2, 1)[..., None]
        lam_log = lam_log.reshape(N, M - 1, -1)
        assert rel(lam_log[:, :L], model.Lam[:, :L]) <= 1e-6
        assert rel(lam_log[:, L - 1], model.ell) <= 1e-6    # ell: the newest snapshot
    U = a["u_log"].astype(np.float64).reshape(N, M - 1, w.dv)[:, :L]
    if op not in OE.DELTA_OPS:
        np.testing.assert_array_equal(U, model.U[:, :L])
    else:
        assert rel(U, model.U[:, :L]) <= TOL_F32_STATE
    np.testing.assert_array_equal(a["S"], S0)          # appends never touch the base


@pytest.mark.parametrize("op", OPS)
def test_readout_forced_merge_flush(op):
    """dl_readout equals q^T S_eager and mutates nothing; a forced merge at L < C equals
    the eager step; a flush materialises the eager state and empties the log."""
    w = WL[op].with_(B=3)
    dl = D()
    M = 16
    S0 = W.initial_state(w)
    xs = [W.step_inputs(w, t) for t in range(9)]
    u = W.bonus(w)
    desc = dl.make_desc(op, w.B, w.H, w.dk, w.dv, M, w.in_dtype)
    ref_o, ref_S = oracle_run(op, S0, xs, u)
    _, st = run_deltalog(desc, S0, xs[:5], u)
    before = _state_arrays(st)
    it = torch.bfloat16 if w.in_dtype == "bf16" else torch.float32
    q = to_dev(xs[5]["q"], it)
    o = torch.empty((w.B, w.H, w.dv), dtype=torch.float32, device="cuda")
    dl.dl_readout(desc, st, q, o)
    torch.cuda.synchronize()
    ro_ref = np.einsum("bhi,bhij->bhj", xs[5]["q"].astype(np.float64), ref_S[4])
    assert rel(o.cpu().numpy(), ro_ref) <= TOL_F32_STATE
    after = _state_arrays(st)
    for k in before:
        np.testing.assert_array_equal(before[k], after[k], err_msg=k)
    # forced merge with the token of step 5 at L = 5 < C = 15
    tok = token(desc, xs[5], u)
    dl.dl_merge(desc, st, tok, o)
    torch.cuda.synchronize()
    assert rel(o.cpu().numpy(), ref_o[5]) <= TOL_F32_STATE
    assert rel(st.S.cpu().numpy(), ref_S[5]) <= TOL_F32_STATE
    assert np.all(st.len.cpu().numpy() == 0)
    # three appends then a flush
    for t in (6, 7, 8):
        dl.dl_append_step(desc, st, token(desc, xs[t], u), o)
    dl.dl_merge(desc, st)
    torch.cuda.synchronize()
    assert rel(st.S.cpu().numpy(), ref_S[8]) <= TOL_F32_STATE
    assert np.all(st.len.cpu().numpy() == 0)
    # a flush of an empty log changes nothing
    S_now = st.S.cpu().numpy().copy()
    dl.dl_merge(desc, st)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(st.S.cpu().numpy(), S_now)


@pytest.mark.parametrize("dk,dv", [(64, 128), (128, 64)])
@pytest.mark.parametrize("op", OPS)
def test_rectangular_heads(op, dk, dv):
    """dk != dv layouts (different thread maps) against the oracle over two merge cycles."""
    w = W.Workload("rect", 77, op, 3, 4, dk, dv, 4, 11)
    S0 = W.initial_state(w)
    xs = [W.step_inputs(w, t) for t in range(w.steps)]
    u = W.bonus(w)
    desc = D().make_desc(op, w.B, w.H, dk, dv, w.M, w.in_dtype)
    outs, st = run_deltalog(desc, S0, xs, u)
    ref_o, ref_S = oracle_run(op, S0, xs, u)
    assert max(rel(a, b) for a, b in zip(outs, ref_o)) <= TOL_F32_STATE
    D().dl_merge(desc, st)
    torch.cuda.synchronize()
    assert rel(st.S.cpu().numpy(), ref_S[-1]) <= TOL_F32_STATE


@pytest.mark.parametrize("dk,dv", [(64, 128), (128, 64), (128, 128)])
@pytest.mark.parametrize("op", ["kda", "gla", "gdn"])
def test_bf16_state_head_shapes(op, dk, dv):
    """bf16 state on every head layout that prefetches its per-key snapshots (64x128,
    128x128) or does not (128x64), two merge cycles and a flush, against the fp64 oracle
    started from the same bf16-rounded state; the bf16-state bar."""
    log(f"bf16 state {op} {dk}x{dv}")
    w = W.Workload("bf16shape", 78, op, 3, 4, dk, dv, 4, 11)
    S0 = W.round_bf16(W.initial_state(w))
    xs = [W.step_inputs(w, t) for t in range(w.steps)]
    u = W.bonus(w)
    desc = D().make_desc(op, w.B, w.H, dk, dv, w.M, w.in_dtype, "bf16")
    outs, st = run_deltalog(desc, S0, xs, u)
    ref_o, ref_S = oracle_run(op, S0, xs, u)
    assert max(rel(a, b) for a, b in zip(outs, ref_o)) <= TOL_BF16_STATE
    D().dl_merge(desc, st)
    torch.cuda.synchronize()
    assert int(st.err.item()) == 0
    assert rel(st.S.float().cpu().numpy(), ref_S[-1]) <= TOL_BF16_STATE


@pytest.mark.parametrize("op", OPS)
def test_largest_merge_interval(op):
    """M = 64 (63 live entries, merged in 4 staged chunks) over 70 steps."""
    base = WL[op]
    w = base.with_(B=2, H=2, M=64, steps=70)
    S0 = W.initial_state(w)
    xs = [W.step_inputs(w, t) for t in range(w.steps)]
    u = W.bonus(w)
    u = None if u is None else u[: w.H]
    desc = D().make_desc(op, w.B, w.H, w.dk, w.dv, w.M, w.in_dtype)
    outs, st = run_deltalog(desc, S0, xs, u)
    ref_o, ref_S = oracle_run(op, S0, xs, u)
    err = max(rel(a, b) for a, b in zip(outs, ref_o))
    log(f"{op} M=64 max out err {err:.2e}")
    assert err <= TOL_F32_STATE
    D().dl_merge(desc, st)
    torch.cuda.synchronize()
    assert rel(st.S.cpu().numpy(), ref_S[-1]) <= TOL_F32_STATE


def test_device_detected_corruption_sets_error_word():
    """A slot id outside [0, B) or a live length outside [0, C] is skipped and reported in
    the error word; nothing is written for that slot."""
    dl = D()
    w = W.GDN_B64.with_(B=2, H=2)
    desc = dl.make_desc("gdn", w.B, w.H, w.dk, w.dv, 4, w.in_dtype)
    st = dl.DeltaLogState(desc, to_dev(W.initial_state(w), torch.float32))
    x = W.step_inputs(w, 0)
    o = torch.zeros((1, w.H, w.dv), dtype=torch.float32, device="cuda")
    before = _state_arrays(st)
    dl.dl_append_step(desc, st, token(desc, x, rows=[0]), o,
                      slots=torch.tensor([5], dtype=torch.int32, device="cuda"))
    torch.cuda.synchronize()
    assert int(st.err.item()) == 1
    after = _state_arrays(st)
    for k in before:
        if k != "err":
            np.testing.assert_array_equal(before[k], after[k], err_msg=k)
    st.err.zero_()
    st.len[1, 0] = 9                                    # > C = 3
    dl.dl_append_step(desc, st, token(desc, x), torch.zeros((2, w.H, w.dv), device="cuda"))
    torch.cuda.synchronize()
    assert int(st.err.item()) == 2
    assert int(st.len[1, 0].item()) == 9                # the corrupted head was skipped
    assert int(st.len[0, 0].item()) == 1                # the others stepped


def test_zero_rows_is_a_no_op_on_device():
    dl = D()
    w = W.GDN_B64.with_(B=2, H=2)
    desc = dl.make_desc("gdn", w.B, w.H, w.dk, w.dv, 4, w.in_dtype)
    st = dl.DeltaLogState(desc, to_dev(W.initial_state(w), torch.float32))
    x = W.step_inputs(w, 0)
    tok = token(desc, x, rows=[0])
    tok.n = 0
    before = _state_arrays(st)
    dl.dl_append_step(desc, st, tok, torch.zeros((0, w.H, w.dv), device="cuda"),
                      slots=torch.zeros((0,), dtype=torch.int32, device="cuda"))
    torch.cuda.synchronize()
    after = _state_arrays(st)
    for k in before:
        np.testing.assert_array_equal(before[k], after[k], err_msg=k)


@pytest.mark.parametrize("op", OPS)
def test_exact_dyadic_bf16_state_bitwise(op):
    """bf16 state: with beta = 1 every stored value is a small integer, exact in bf16, so
    the GPU must still equal the oracle bit for bit (outputs, merged base, eager state)."""
    B, H, M, steps, dk = 3, 2, 4, 8, 128
    S0, xs, u = dyadic_inputs(op, B, H, dk, dk, steps, seed=17 + OPS.index(op))
    for x in xs:
        if x["beta"] is not None:
            x["beta"][:] = 1.0
    desc = D().make_desc(op, B, H, dk, dk, M, "bf16", "bf16")
    outs, st = run_deltalog(desc, S0, xs, u)
    ref_o, ref_S = oracle_run(op, S0, xs, u)
    for t in range(steps):
        np.testing.assert_array_equal(outs[t].astype(np.float64), ref_o[t], err_msg=f"step {t}")
    np.testing.assert_array_equal(st.S.float().cpu().numpy().astype(np.float64), ref_S[-1])
    eo, eS = run_eager(desc, S0, xs, u)
    for t in range(steps):
        np.testing.assert_array_equal(eo[t].astype(np.float64), ref_o[t], err_msg=f"eager {t}")
    np.testing.assert_array_equal(eS.float().cpu().numpy().astype(np.float64), ref_S[-1])


@pytest.mark.parametrize("M", [2, 8])
@pytest.mark.parametrize("op", OPS)
def test_embedded_2x2_bruteforce(op, M):
    """The 2x2 exact-rational brute force of the oracle pins, embedded in a 64x64 head
    (state, keys, queries and values zero outside the 2x2 block, so the block evolves
    exactly as the hand-expanded formulas say): three steps through dl_append_step (M = 2
    merges at the second step; M = 8 only appends) and a flush.  Inputs are stored in
    fp32 and the exact reference uses the stored values; the decay goes through the
    hardware exp, hence a 1e-6 bar inside the block and exact zeros outside it."""
    from fractions import Fraction as Fr

    import oracle_pins as P

    d = 64
    S = [[Fr(1, 2), Fr(-3, 4)], [Fr(5, 8), Fr(1, 4)]]
    seq = [
        dict(q=[Fr(3, 5), Fr(4, 5)], k=[Fr(4, 5), Fr(-3, 5)], v=[Fr(1), Fr(-2)],
             beta=Fr(1, 2), g=[Fr(3, 4), Fr(1, 2)]),
        dict(q=[Fr(-1, 2), Fr(1, 3)], k=[Fr(1, 3), Fr(2, 3)], v=[Fr(3, 2), Fr(1, 4)],
             beta=Fr(3, 4), g=[Fr(7, 8), Fr(5, 8)]),
        dict(q=[Fr(2), Fr(-1)], k=[Fr(-1, 2), Fr(1, 2)], v=[Fr(-1), Fr(1, 8)],
             beta=Fr(1, 4), g=[Fr(1, 2), Fr(15, 16)]),
    ]
    u2 = [Fr(1, 5), Fr(-2, 5)]
    f32 = lambda x: np.float32(float(x))
    exact = lambda x: Fr(float(np.float32(x)))          # the stored fp32 value, exactly
    S0 = np.zeros((1, 1, d, d), np.float32)
    for i in range(2):
        for j in range(2):
            S0[0, 0, i, j] = f32(S[i][j])
    S = [[exact(S0[0, 0, i, j]) for j in range(2)] for i in range(2)]
    u = None
    if op == "rwkv6":
        u = np.zeros((1, d), np.float32)
        u[0, :2] = [f32(x) for x in u2]
        u2 = [exact(x) for x in u[0, :2]]
    scalar = op in ("gdn", "retnet", "linattn")
    xs, refs = [], []
    for st in seq:
        g = [Fr(1), Fr(1)] if op == "linattn" else ([st["g"][0]] * 2 if scalar else st["g"])
        x = {n: np.zeros((1, 1, d), np.float32) for n in ("q", "k", "v")}
        for n in ("q", "k", "v"):
            x[n][0, 0, :2] = [f32(t) for t in st[n]]
        lam_vals = [np.float32(np.log(float(t))) for t in g]
        if op == "linattn":
            x["lam"] = None
        elif scalar:
            x["lam"] = np.array([[lam_vals[0]]], np.float32)
        else:
            x["lam"] = np.zeros((1, 1, d), np.float32)
            x["lam"][0, 0, :2] = lam_vals
        x["beta"] = np.array([[f32(st["beta"])]], np.float32) if op in OE.DELTA_OPS else None
        xs.append(x)
        # exact recurrence on the stored inputs; the decay factor is exp of the stored
        # lambda, taken as the nearest rational (the only non-exact quantity)
        ge = [Fr(float(np.exp(np.float64(v)))) for v in lam_vals] if op != "linattn" else g
        q2, k2, v2 = ([exact(t) for t in x[n][0, 0, :2]] for n in ("q", "k", "v"))
        b2 = exact(x["beta"][0, 0]) if x["beta"] is not None else None
        S, o = P._bf_step_fraction(op, S, q2, k2, v2, b2, ge, u2)
        refs.append(([float(t) for t in o], [[float(t) for t in row] for row in S]))
    desc = D().make_desc(op, 1, 1, d, d, M, "f32")
    outs, st = run_deltalog(desc, S0, xs, u)
    for t, (o_ref, _) in enumerate(refs):
        np.testing.assert_allclose(outs[t][0, 0, :2], o_ref, rtol=1e-6, atol=1e-6,
                                   err_msg=f"{op} M={M} step {t}")
        assert not np.any(outs[t][0, 0, 2:]), f"{op} output outside the block, step {t}"
    D().dl_merge(desc, st)
    torch.cuda.synchronize()
    Sg = st.S.cpu().numpy()[0, 0]
    np.testing.assert_allclose(Sg[:2, :2], refs[-1][1], rtol=1e-6, atol=1e-6,
                               err_msg=f"{op} M={M} flushed block")
    Sg[:2, :2] = 0.0
    assert not np.any(Sg), f"{op} M={M}: state outside the block"


@pytest.mark.parametrize("op", ["gdn", "rwkv6"])
def test_independent_states_on_two_streams(op):
    """The library keeps no state between calls: two layers stepped on two side streams
    (default priority), their launches interleaved from one host thread, end bitwise
    equal to the same layers stepped one after the other on the current stream."""
    dl = D()
    w = WL[op].with_(B=4)
    M, steps = 4, 9
    desc = dl.make_desc(op, w.B, w.H, w.dk, w.dv, M, w.in_dtype)
    u = W.bonus(w)
    S0 = [W.initial_state(w, layer) for layer in (0, 1)]
    xs = [[W.step_inputs(w, t, layer) for t in range(steps)] for layer in (0, 1)]
    toks = [[token(desc, x, u) for x in xs[layer]] for layer in (0, 1)]

    def fresh():
        return [dl.DeltaLogState(desc, to_dev(S0[layer], torch.float32)) for layer in (0, 1)]

    def outs():
        return [[torch.empty((w.B, w.H, w.dv), dtype=torch.float32, device="cuda")
                 for _ in range(steps)] for _ in (0, 1)]

    ref_st, ref_o = fresh(), outs()
    for layer in (0, 1):
        for t in range(steps):
            dl.dl_append_step(desc, ref_st[layer], toks[layer][t], ref_o[layer][t])
    torch.cuda.synchronize()

    st, o = fresh(), outs()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    for s in streams:
        s.wait_stream(torch.cuda.current_stream())
    for t in range(steps):
        for layer in (0, 1):
            dl.dl_append_step(desc, st[layer], toks[layer][t], o[layer][t], stream=streams[layer])
    for s in streams:
        torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    for layer in (0, 1):
        a, b = _state_arrays(ref_st[layer]), _state_arrays(st[layer])
        for k in a:
            np.testing.assert_array_equal(a[k], b[k], err_msg=(layer, k))
        for t in range(steps):
            assert torch.equal(ref_o[layer][t], o[layer][t]), (layer, t)
