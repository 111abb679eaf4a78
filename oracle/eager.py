"""Eager dense recurrence in float64 -- the plain definition the GPU path must reproduce.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

The unified one-token decode step (Eq. 3) is

    S_t = D(lambda_t) S_{t-1} + a_t b_t^T,      D(l) = diag(exp(l))   (Eq. 2)

with the state S in R^{dk x dv}; D scales the *rows* (key dimension) of S.  Table 1
instantiates (a_t, b_t) and the decay form per operator:

    GDN      : head-wise scalar decay, a = k, b = beta (v - k^T S_old)
    KDA      : per-key (diagonal) decay, same delta-rule pair as GDN
    RWKV6    : per-key decay, a = k, b = v (no correction)
    Linear attention : no decay, a = phi(k), b = v (phi already applied to k)
    RetNet   : head-wise scalar decay gamma_t = exp(lambda_t), a = k, b = v
    GLA      : per-key (diagonal) decay, a = k, b = v

Readings taken where the text is silent or ambiguous:

* Correction state (delta rule).  Table 1 writes the old-state correction as
  ``k_t^T S_{t-1}``.  The paper states the model semantics are unchanged and that the
  correction is a *pre-update readout* (Sec. 3.1, "Append stage"); the published GDN
  and KDA recurrences apply the correction to the decayed state
  ``D(lambda_t) S_{t-1}``.  This oracle uses the decayed state by default; the literal
  undecayed form is kept behind ``correction="undecayed"`` for diagnostics only.
* Output timing.  GDN/KDA, linear attention, RetNet and GLA read out the post-update
  state ``o = q^T S_t`` (Eq. 3; Eq. 1 for linear attention).
  RWKV6 reads the pre-update state plus the per-head bonus ``u``:
  ``o = r^T (S_{t-1} + diag(u) k v^T)`` -- the standard RWKV6 readout.
* No query scaling is applied inside the step: any feature map or 1/sqrt(dk) is
  absorbed into q by the caller (Sec. 2.1 folds the query feature map into q_t).

Shapes (any leading batch dims ``...``, typically ``[N]`` heads):
    S  [..., dk, dv]   q,k,r [..., dk]   v [..., dv]   beta [...]
    lam [...] (GDN, RetNet: scalar per head) or [..., dk] (KDA, RWKV6, GLA);
        ignored for linear attention
    u  [..., dk] (RWKV6 bonus, broadcast from the per-head parameter [H, dk])
"""

import numpy as np

OPS = ("gdn", "kda", "rwkv6", "linattn", "retnet", "gla")
DELTA_OPS = ("gdn", "kda")                  # b = beta (v - correction)
PER_KEY_OPS = ("kda", "rwkv6", "gla")       # diagonal decay: lambda is [..., dk]
ADDITIVE_OPS = ("linattn", "retnet", "gla")  # pair (k, v) and post-update readout


def _f64(x):
    return np.asarray(x, dtype=np.float64)


def row_decay(lam, dk, per_key):
    """exp(lambda) as a per-row factor of shape [..., dk, 1] (Eq. 2).

    ``per_key`` False: lam has shape [...] (one log-decay per head) and the value is
    repeated over all dk rows (Sec. 2.1 represents scalar decay as a constant log-decay
    vector).  ``per_key`` True: lam has shape [..., dk].
    """
    lam = _f64(lam)
    if not per_key:
        lam = np.broadcast_to(lam[..., None], lam.shape + (dk,))
    elif lam.shape[-1] != dk:
        raise ValueError("per-key log-decay must have a trailing dimension of dk")
    return np.exp(lam)[..., :, None]


def _readout(S, q):
    """o_j = sum_i q_i S_ij  (q^T S)."""
    return np.einsum("...i,...ij->...j", q, S)


def gdn_kda_step(S, q, k, v, beta, lam, per_key, correction="decayed"):
    """One delta-rule decode step: GDN (``per_key`` False) or KDA (``per_key`` True).

    Eq. 3 with Table 1's GDN/KDA row.  Returns (S_t, o_t).
    """
    S, q, k, v, beta = map(_f64, (S, q, k, v, beta))
    dk = S.shape[-2]
    Sd = row_decay(lam, dk, per_key) * S                       # D(lambda_t) S_{t-1}
    if correction == "decayed":
        c = _readout(Sd, k)                           # k^T D(lambda_t) S_{t-1}
    elif correction == "undecayed":                   # literal Table 1 text, diagnostic only
        c = _readout(S, k)
    else:
        raise ValueError(correction)
    b = beta[..., None] * (v - c)                     # b_t = beta_t (v_t - correction)
    S_new = Sd + k[..., :, None] * b[..., None, :]    # + a_t b_t^T with a_t = k_t
    o = _readout(S_new, q)                            # post-update readout, Eq. 3
    return S_new, o


def rwkv6_step(S, r, k, v, lam, u):
    """One RWKV6 decode step: o = r^T (S_{t-1} + diag(u) k v^T); S_t = D(lambda) S + k v^T.

    Table 1's RWKV6 row (diagonal decay, pair (k, v)) with the bonus readout.
    """
    S, r, k, v, u = map(_f64, (S, r, k, v, u))
    dk = S.shape[-2]
    bonus = np.sum(r * u * k, axis=-1)                # r^T diag(u) k
    o = _readout(S, r) + bonus[..., None] * v         # pre-update readout + bonus
    S_new = row_decay(lam, dk, True) * S + k[..., :, None] * v[..., None, :]
    return S_new, o


def additive_step(S, q, k, v, lam, decay):
    """One step of the additive operators of Table 1 (pair (k_t, v_t), no correction)
    with the post-update readout of Eq. 3:  S_t = T(S_{t-1}) + k v^T,  o = q^T S_t, where
    T is the identity (``decay`` "none": linear attention, Eq. 1), gamma_t S with
    gamma_t = exp(lambda_t) (``"scalar"``: RetNet) or D(lambda_t) S (``"diagonal"``: GLA).
    """
    S, q, k, v = map(_f64, (S, q, k, v))
    dk = S.shape[-2]
    if decay == "none":
        Sd = S
    elif decay in ("scalar", "diagonal"):
        Sd = row_decay(lam, dk, decay == "diagonal") * S
    else:
        raise ValueError(decay)
    S_new = Sd + k[..., :, None] * v[..., None, :]
    return S_new, _readout(S_new, q)


def eager_step(op, S, q, k, v, beta, lam, u=None, correction="decayed"):
    """Dispatch one eager step for ``op`` in ``OPS``; returns (S_t, o_t).

    For RWKV6 ``q`` carries the receptance r.  ``beta`` is used by the delta rule only,
    ``lam`` by every operator but linear attention, ``u`` by RWKV6 only.
    """
    if op in DELTA_OPS:
        return gdn_kda_step(S, q, k, v, beta, lam, op == "kda", correction=correction)
    if op == "rwkv6":
        return rwkv6_step(S, q, k, v, lam, u)
    if op in ADDITIVE_OPS:
        decay = {"linattn": "none", "retnet": "scalar", "gla": "diagonal"}[op]
        return additive_step(S, q, k, v, lam, decay)
    raise ValueError(op)


def rel_fro(x, ref):
    """Relative Frobenius error ||x - ref|| / ||ref|| in float64 (the parity metric)."""
    x, ref = _f64(x), _f64(ref)
    den = np.linalg.norm(ref.ravel())
    num = np.linalg.norm((x - ref).ravel())
    if den == 0.0:
        return float(num)
    return float(num / den)
