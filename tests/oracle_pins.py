"""Pins for the fp64 oracle: closed forms, special cases, exact brute force, invariants.

Each ``pin_*`` function raises AssertionError when the implementation it is given is
wrong.  ``test_oracle_pins.py`` runs them on the real oracle; ``test_oracle_mutants.py``
runs them on deliberately broken copies (a dropped term, a wrong sign, a transposed
operand, an undecayed correction, ...) and requires every mutant to be caught, which
shows that the pins constrain every term of the recurrence.

The step interface is ``step(op, S, q, k, v, beta, lam, u) -> (S_new, o)`` over a
leading head axis N; the model interface is the ``DeltaLogModel`` class.
"""

from fractions import Fraction as Fr

import numpy as np

from paper_2608_15533_amd import workloads as W

TIGHT = 1e-12


def _close(a, b, tol=TIGHT, what=""):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    den = max(np.linalg.norm(b.ravel()), 1e-300)
    err = np.linalg.norm((a - b).ravel()) / den
    assert err <= tol, f"{what}: relative error {err:.3e} > {tol:.1e}"


def small_workload(op, N=3, d=8, M=4, steps=12, dk=None, dv=None, in_dtype="f32", cfg=91):
    """A tiny workload drawn with the shared generator (same distributions, small dims)."""
    dk = d if dk is None else dk
    dv = d if dv is None else dv
    return W.Workload(f"tiny_{op}", cfg, op, N, 1, dk, dv, M, steps, in_dtype=in_dtype)


SCALAR_DECAY_OPS = ("gdn", "retnet", "linattn")   # lambda is one value per head
DELTA_OPS = ("gdn", "kda")


def tiny_inputs(w):
    """(S0 [N,dk,dv], list of per-step dicts with [N,...] arrays, u [N,dk] or None).
    Linear attention has no decay; its lambda is given as zeros [N]."""
    S0 = W.initial_state(w)[:, 0].astype(np.float64) * 25.0   # O(0.5) entries
    steps = []
    for t in range(w.steps):
        x = W.step_inputs(w, t)
        st = {k: (None if a is None else a[:, 0].astype(np.float64)) for k, a in x.items()}
        if st["lam"] is None:
            st["lam"] = np.zeros(w.B)
        steps.append(st)
    u = W.bonus(w)
    u = None if u is None else np.broadcast_to(u[0], (w.B, w.dk)).astype(np.float64)
    return S0, steps, u


# --------------------------------------------------------------------------- eager
def _bf_step_fraction(op, S, q, k, v, beta, g, u):
    """One step on a 2x2 head in exact rationals, every element written out by hand.

    g[i] = exp(lambda_i) is given as a rational.  Table 1 / Eq. 3:
      delta rule:  S'_ij = g_i S_ij;  c_j = sum_m k_m S'_mj;  b_j = beta (v_j - c_j)
                   S_ij <- S'_ij + k_i b_j;  o_j = sum_i q_i S_ij  (post-update)
      RWKV6:       o_j = sum_i r_i S_ij + (sum_i r_i u_i k_i) v_j  (pre-update + bonus)
                   S_ij <- g_i S_ij + k_i v_j
      additive:    S_ij <- g_i S_ij + k_i v_j;  o_j = sum_i q_i S_ij  (post-update)
                   (linear attention g = 1, RetNet g_0 = g_1, GLA per key)
    """
    n = 2
    if op in ("linattn", "retnet", "gla"):
        Sn = [[g[i] * S[i][j] + k[i] * v[j] for j in range(n)] for i in range(n)]
        o = [q[0] * Sn[0][j] + q[1] * Sn[1][j] for j in range(n)]
    elif op in ("gdn", "kda"):
        Sd = [[g[i] * S[i][j] for j in range(n)] for i in range(n)]
        c = [k[0] * Sd[0][j] + k[1] * Sd[1][j] for j in range(n)]
        b = [beta * (v[j] - c[j]) for j in range(n)]
        Sn = [[Sd[i][j] + k[i] * b[j] for j in range(n)] for i in range(n)]
        o = [q[0] * Sn[0][j] + q[1] * Sn[1][j] for j in range(n)]
    else:
        bonus = q[0] * u[0] * k[0] + q[1] * u[1] * k[1]
        o = [q[0] * S[0][j] + q[1] * S[1][j] + bonus * v[j] for j in range(n)]
        Sn = [[g[i] * S[i][j] + k[i] * v[j] for j in range(n)] for i in range(n)]
    return Sn, o


def pin_bruteforce_2x2(step, op):
    """Three steps on a 2x2 head against exact rational arithmetic."""
    S = [[Fr(1, 2), Fr(-3, 4)], [Fr(5, 8), Fr(1, 4)]]
    seq = [
        dict(q=[Fr(3, 5), Fr(4, 5)], k=[Fr(4, 5), Fr(-3, 5)], v=[Fr(1), Fr(-2)],
             beta=Fr(1, 2), g=[Fr(3, 4), Fr(1, 2)]),
        dict(q=[Fr(-1, 2), Fr(1, 3)], k=[Fr(1, 3), Fr(2, 3)], v=[Fr(3, 2), Fr(1, 4)],
             beta=Fr(3, 4), g=[Fr(7, 8), Fr(5, 8)]),
        dict(q=[Fr(2), Fr(-1)], k=[Fr(-1, 2), Fr(1, 2)], v=[Fr(-1), Fr(1, 8)],
             beta=Fr(1, 4), g=[Fr(1, 2), Fr(15, 16)]),
    ]
    u = [Fr(1, 5), Fr(-2, 5)]
    Sf = np.array([[float(x) for x in row] for row in S])[None]
    for t, st in enumerate(seq):
        if op == "linattn":
            g = [Fr(1), Fr(1)]
        elif op in SCALAR_DECAY_OPS:
            g = [st["g"][0], st["g"][0]]
        else:
            g = st["g"]
        S, o = _bf_step_fraction(op, S, st["q"], st["k"], st["v"], st["beta"], g, u)
        f = lambda xs: np.array([float(x) for x in xs])[None]
        lam = np.log(np.array([float(g[0])])) if op in SCALAR_DECAY_OPS else np.log(f(g))
        Sf, of = step(op, Sf, f(st["q"]), f(st["k"]), f(st["v"]),
                      np.array([float(st["beta"])]), lam,
                      f(u) if op == "rwkv6" else None)
        exp_S = np.array([[float(x) for x in row] for row in S])[None]
        _close(Sf, exp_S, 1e-13, f"{op} 2x2 state step {t}")
        _close(of, f(o), 1e-13, f"{op} 2x2 output step {t}")


def _no_write(op, st):
    """(k, beta) of a step that writes nothing: beta = 0 (delta rule) or k = 0."""
    if op in DELTA_OPS:
        return st["k"], np.zeros_like(st["beta"])
    return np.zeros_like(st["k"]), None


def pin_identity(step, op):
    """No write (beta = 0 for the delta rule, else k = 0) and lambda = 0: S unchanged and
    o = S^T q."""
    w = small_workload(op)
    S0, steps, u = tiny_inputs(w)
    st = steps[0]
    lam = np.zeros_like(st["lam"])
    k, beta = _no_write(op, st)
    S1, o = step(op, S0, st["q"], k, st["v"], beta, lam, u)
    _close(S1, S0, 0.0, f"{op} identity state")
    _close(o, np.einsum("ni,nij->nj", st["q"], S0), 1e-14, f"{op} identity output")


def pin_decay_only(step, op):
    """n steps with no write: S_n = diag(exp(sum lambda)) S_0 (S_0 for linear attention)."""
    w = small_workload(op, steps=5)
    S0, steps, u = tiny_inputs(w)
    S = S0
    tot = np.zeros_like(steps[0]["lam"])
    for st in steps:
        k, beta = _no_write(op, st)
        S, _ = step(op, S, st["q"], k, st["v"], beta, st["lam"], u)
        tot = tot + st["lam"]
    rows = np.exp(tot)[:, None, None] if op in SCALAR_DECAY_OPS else np.exp(tot)[:, :, None]
    _close(S, rows * S0, 1e-14, f"{op} decay-only closed form")


def pin_delta_write(step, op):
    """Delta rule with beta = 1 and |k| = 1 stores v exactly under k: S_t^T k_t = v_t."""
    w = small_workload(op, steps=4)
    S, steps, u = tiny_inputs(w)
    for st in steps:
        k = st["k"] / np.linalg.norm(st["k"], axis=-1, keepdims=True)   # |k| = 1 in fp64
        S, _ = step(op, S, st["q"], k, st["v"], np.ones_like(st["beta"]), st["lam"], u)
        _close(np.einsum("ni,nij->nj", k, S), st["v"], 1e-13, f"{op} delta write")


def pin_published_delta_rule(step, op):
    """Matrix-product forms of the delta-rule operators as their authors define them.

    GDN: S_t = alpha (I - beta k k^T) S_{t-1} + beta k v^T
    KDA: S_t = (I - beta k k^T) diag(alpha) S_{t-1} + beta k v^T
    (state laid out dk x dv so that o = q^T S), with o_t = q^T S_t.
    """
    w = small_workload(op, steps=3)
    S, steps, u = tiny_inputs(w)
    N, dk = S.shape[0], S.shape[1]
    I = np.eye(dk)
    for st in steps:
        k, v, q, beta = st["k"], st["v"], st["q"], st["beta"]
        P = I[None] - beta[:, None, None] * np.einsum("ni,nj->nij", k, k)
        if op == "gdn":
            ref = np.exp(st["lam"])[:, None, None] * np.matmul(P, S)
        else:
            ref = np.matmul(P, np.exp(st["lam"])[:, :, None] * S)
        ref = ref + beta[:, None, None] * np.einsum("ni,nj->nij", k, v)
        S, o = step(op, S, q, k, v, beta, st["lam"], u)
        _close(S, ref, 1e-13, f"{op} published matrix form")
        _close(o, np.einsum("ni,nij->nj", q, ref), 1e-13, f"{op} published output")


def pin_kda_equal_keys_is_gdn(step):
    """KDA with the same log-decay on every key is GDN."""
    w = small_workload("gdn", steps=4)
    S0, steps, u = tiny_inputs(w)
    Sg, Sk = S0, S0
    for st in steps:
        lam_k = np.repeat(st["lam"][:, None], S0.shape[1], axis=1)
        Sg, og = step("gdn", Sg, st["q"], st["k"], st["v"], st["beta"], st["lam"], None)
        Sk, ok = step("kda", Sk, st["q"], st["k"], st["v"], st["beta"], lam_k, None)
        _close(Sk, Sg, 1e-15, "kda==gdn state")
        _close(ok, og, 1e-15, "kda==gdn output")


def pin_rwkv6_linear_attention(step):
    """RWKV6 with lambda = 0, u = 0 and S_0 = 0 is causal linear attention (Eq. 1 shifted):
    o_t = r_t^T sum_{s<t} k_s v_s^T; with orthonormal keys it recalls v_s exactly."""
    d, T = 8, 5
    rng = np.random.default_rng(5)
    Q, _ = np.linalg.qr(rng.standard_normal((d, d)))
    keys = Q[:T]
    vals = rng.standard_normal((T, d))
    S = np.zeros((1, d, d))
    for t in range(T):
        r = keys[t - 1][None] if t > 0 else rng.standard_normal((1, d))
        S, o = step("rwkv6", S, r, keys[t][None], vals[t][None], None, np.zeros((1, d)),
                    np.zeros((1, d)))
        ref = np.zeros(d) if t == 0 else vals[t - 1]
        if t > 0:
            _close(o[0], ref, 1e-13, "rwkv6 recall")
        else:
            assert np.allclose(o, 0.0)
    _close(S[0], keys.T @ vals, 1e-13, "rwkv6 sum of outer products")


def pin_rwkv6_bonus(step):
    """The bonus reads the current token: with S_0 = 0, o = (r . (u * k)) v."""
    d = 8
    rng = np.random.default_rng(6)
    r, k, v, u = (rng.standard_normal((1, d)) for _ in range(4))
    _, o = step("rwkv6", np.zeros((1, d, d)), r, k, v, None, -np.ones((1, d)), u)
    _close(o, np.sum(r * u * k) * v, 1e-14, "rwkv6 bonus")


def _sequence(op, T, d=8, seed=21):
    """S0 [1,d,d] and a T-step sequence of the op's inputs (shared generator)."""
    w = small_workload(op, N=1, d=d, steps=T, cfg=seed)
    S0, steps, _ = tiny_inputs(w)
    Q = np.stack([st["q"][0] for st in steps])
    K = np.stack([st["k"][0] for st in steps])
    V = np.stack([st["v"][0] for st in steps])
    return S0, steps, Q, K, V


def _run(step, op, S0, steps):
    S, outs = S0, []
    for st in steps:
        S, o = step(op, S, st["q"], st["k"], st["v"], None, st["lam"], None)
        outs.append(o[0])
    return S[0], np.stack(outs)


def pin_linear_attention_matrix_form(step):
    """Causal linear attention (Eq. 1) in matrix form: O = Q S0 + tril(Q K^T) V, and the
    final state is S0 + K^T V."""
    S0, steps, Q, K, V = _sequence("linattn", 9)
    S, O = _run(step, "linattn", S0, steps)
    _close(O, Q @ S0[0] + np.tril(Q @ K.T) @ V, 1e-13, "linear attention outputs")
    _close(S, S0[0] + K.T @ V, 1e-13, "linear attention state")


def pin_retnet_parallel_form(step):
    """RetNet's parallel retention with a fixed gamma: o_n = gamma^(n+1) q_n^T S0 +
    sum_{m<=n} gamma^(n-m) (q_n . k_m) v_m, i.e. O = (Q K^T * Dg) V + diag(gamma^(n+1)) Q S0."""
    S0, steps, Q, K, V = _sequence("retnet", 10)
    gamma = 0.9
    for st in steps:
        st["lam"] = np.full(1, np.log(gamma))
    S, O = _run(step, "retnet", S0, steps)
    n = np.arange(len(steps))
    Dg = np.where(n[:, None] >= n[None, :], gamma ** (n[:, None] - n[None, :]), 0.0)
    ref = (Q @ K.T * Dg) @ V + (gamma ** (n + 1))[:, None] * (Q @ S0[0])
    _close(O, ref, 1e-13, "retnet parallel form")


def pin_gla_parallel_form(step):
    """Gated linear attention in parallel form: with cumulative gates b_t = prod_{r<=t}
    exp(lambda_r) (per key), o_t = (q_t * b_t)^T S0 + sum_{s<=t} ((q_t * b_t) . (k_s / b_s)) v_s."""
    S0, steps, Q, K, V = _sequence("gla", 10)
    S, O = _run(step, "gla", S0, steps)
    Bc = np.exp(np.cumsum(np.stack([st["lam"][0] for st in steps]), axis=0))
    Qb, Kb = Q * Bc, K / Bc
    _close(O, np.tril(Qb @ Kb.T) @ V + Qb @ S0[0], 1e-12, "gla parallel form")
    _close(S, Bc[-1][:, None] * S0[0] + Kb.T @ V * Bc[-1][:, None], 1e-12, "gla state")


def pin_gla_equal_gates_is_retnet(step):
    """GLA whose per-key gates are all equal is RetNet with that scalar decay."""
    S0, steps, _, _, _ = _sequence("gla", 6)
    Sg = Sr = S0
    for st in steps:
        lam_s = st["lam"][:, :1]
        Sg, og = step("gla", Sg, st["q"], st["k"], st["v"], None,
                      np.broadcast_to(lam_s, st["lam"].shape), None)
        Sr, o_r = step("retnet", Sr, st["q"], st["k"], st["v"], None, lam_s[:, 0], None)
        _close(Sg, Sr, 1e-15, "gla==retnet state")
        _close(og, o_r, 1e-15, "gla==retnet output")


# --------------------------------------------------------------------------- model
def _eager_seq(step, op, S0, steps, u):
    S = S0
    outs, states = [], []
    for st in steps:
        S, o = step(op, S, st["q"], st["k"], st["v"], st.get("beta"), st["lam"], u)
        outs.append(o)
        states.append(S)
    return outs, states


def pin_model_matches_eager(Model, step, op, M, steps_n=13):
    """Eq. 7 reconstructs the eager state after every step; outputs agree; the base equals
    the eager state right after each merge (closure argument of Sec. 3.2)."""
    w = small_workload(op, M=M, steps=steps_n)
    S0, steps, u = tiny_inputs(w)
    outs, states = _eager_seq(step, op, S0, steps, u)
    m = Model(op, S0, M)
    for t, st in enumerate(steps):
        o = m.step(st["q"], st["k"], st["v"], st.get("beta"), st["lam"], u=u)
        _close(o, outs[t], TIGHT, f"{op} M={M} output step {t}")
        _close(m.logical_state(), states[t], TIGHT, f"{op} M={M} Eq.7 state step {t}")
        exp_L = (t + 1) % M
        assert np.all(m.L == exp_L), f"{op} M={M} live length {m.L} != {exp_L} at step {t}"
        if exp_L == 0:
            _close(m.Sbar, states[t], TIGHT, f"{op} M={M} base after merge step {t}")
            assert np.all(m.ell == 0.0)


def pin_model_overwrite_through_log(Model):
    """lambda = 0, beta = 1, orthonormal keys: write k1->v1, k2->v2, k1->v3 with all three
    entries still in the log.  The third write's correction must come from log entry 0:
    U_2 = v3 - v1, and afterwards S^T k1 = v3, S^T k2 = v2."""
    d = 8
    rng = np.random.default_rng(7)
    Q, _ = np.linalg.qr(rng.standard_normal((d, d)))
    k1, k2 = Q[0][None], Q[1][None]
    v1, v2, v3 = (rng.standard_normal((1, d)) for _ in range(3))
    m = Model("gdn", np.zeros((1, d, d)), 8)
    z, one = np.zeros(1), np.ones(1)
    for k, v in ((k1, v1), (k2, v2), (k1, v3)):
        m.step(k, k, v, one, z)
    assert m.L[0] == 3
    _close(m.U[0, 2], (v3 - v1)[0], 1e-13, "third entry's corrected value")
    S = m.logical_state()
    _close(np.einsum("ni,nij->nj", k1, S), v3, 1e-13, "recall k1")
    _close(np.einsum("ni,nij->nj", k2, S), v2, 1e-13, "recall k2")
    _close(m.Sbar, np.zeros((1, d, d)), 0.0, "base untouched by appends")


def pin_model_replay_readout(Model, op):
    """The factored readout (base term + one coefficient per entry) equals q^T (Eq. 7 state)."""
    w = small_workload(op, M=6, steps=4)
    S0, steps, u = tiny_inputs(w)
    m = Model(op, S0, 6)
    for st in steps:
        m.step(st["q"], st["k"], st["v"], st.get("beta"), st["lam"], u=u)
    x = steps[-1]["q"]
    _close(m.replay_readout(x), np.einsum("ni,nij->nj", x, m.logical_state()), TIGHT,
           f"{op} replay readout")


def pin_model_merge_is_gemm(Model, op):
    """A merge writes diag(e^ell') Sbar + Ktilde^T U + k b^T, with Ktilde_i = e^(ell'-Lam_i) K_i,
    computed here as one dense matrix product over the stacked log (a library GEMM)."""
    M = 5
    w = small_workload(op, M=M, steps=M)
    S0, steps, u = tiny_inputs(w)
    m = Model(op, S0, M)
    for st in steps[:-1]:
        m.step(st["q"], st["k"], st["v"], st.get("beta"), st["lam"], u=u)
    st = steps[-1]
    Sbar, ell, K, U, Lam = (x.copy() for x in (m.Sbar, m.ell, m.K, m.U, m.Lam))
    ell_new = ell + st["lam"].reshape(ell.shape)
    dk = S0.shape[1]
    e = np.exp(np.broadcast_to(ell_new, (w.B, dk)))
    Kt = np.exp(np.broadcast_to(ell_new[:, None, :] - Lam, (w.B, M - 1, dk))) * K
    if op not in DELTA_OPS:
        a, b = st["k"], st["v"]
    else:
        S_dec = e[:, :, None] * Sbar + np.matmul(Kt.transpose(0, 2, 1), U)
        b = st["beta"][:, None] * (st["v"] - np.einsum("ni,nij->nj", st["k"], S_dec))
        a = st["k"]
    Kx = np.concatenate([Kt, a[:, None, :]], axis=1)          # [N, L+1, dk]
    Ux = np.concatenate([U, b[:, None, :]], axis=1)           # [N, L+1, dv]
    ref = e[:, :, None] * Sbar + np.matmul(Kx.transpose(0, 2, 1), Ux)
    m.step(st["q"], st["k"], st["v"], st.get("beta"), st["lam"], u=u)
    assert np.all(m.L == 0)
    _close(m.Sbar, ref, TIGHT, f"{op} merge vs GEMM form")


def pin_model_flush_and_readout(Model, step, op):
    """Flush materialises Eq. 7 and clears the log; readout equals q^T S_eager; a forced
    merge at L < C equals the eager step."""
    M = 8
    w = small_workload(op, M=M, steps=6)
    S0, steps, u = tiny_inputs(w)
    outs, states = _eager_seq(step, op, S0, steps, u)
    m = Model(op, S0, M)
    for st in steps[:3]:
        m.step(st["q"], st["k"], st["v"], st.get("beta"), st["lam"], u=u)
    x = steps[3]["q"]
    _close(m.readout(x), np.einsum("ni,nij->nj", x, states[2]), TIGHT, f"{op} readout")
    m.flush()
    assert np.all(m.L == 0) and np.all(m.ell == 0.0)
    _close(m.Sbar, states[2], TIGHT, f"{op} flush")
    st = steps[3]
    m.step(st["q"], st["k"], st["v"], st.get("beta"), st["lam"], u=u)
    st = steps[4]
    o = m.step(st["q"], st["k"], st["v"], st.get("beta"), st["lam"], u=u, force_merge=True)
    assert np.all(m.L == 0)
    _close(o, outs[4], TIGHT, f"{op} forced-merge output")
    _close(m.Sbar, states[4], TIGHT, f"{op} forced-merge state")


def pin_model_partial_batch(Model, step, op):
    """Heads outside a step's slot list keep their state; the rest follow eager."""
    M = 4
    w = small_workload(op, M=M, steps=9)
    S0, steps, u = tiny_inputs(w)
    m = Model(op, S0, M)
    S = S0.copy()
    rng = np.random.default_rng(11)
    for t, st in enumerate(steps):
        act = rng.random(w.B) < 0.6
        o = m.step(st["q"], st["k"], st["v"], st.get("beta"), st["lam"], u=u, active=act)
        S1, o1 = step(op, S, st["q"], st["k"], st["v"], st.get("beta"), st["lam"], u)
        S = np.where(act[:, None, None], S1, S)
        _close(o[act], o1[act], TIGHT, f"{op} partial output step {t}")
        assert np.all(np.isnan(o[~act]))
        _close(m.logical_state(), S, TIGHT, f"{op} partial state step {t}")
