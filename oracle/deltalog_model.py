"""DeltaLog base-plus-log state machine in float64 (Alg. 1, Eqs. 4-7).

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

The physical state of Sec. 3.1 for N (slot, head) pairs:

    Sbar [N, dk, dv]   dense base, last materialisation
    ell  [N, dl]       cumulative log-decay since that materialisation (dl = 1 for
                       head-wise scalar decay (GDN, RetNet) and for linear attention,
                       whose log-decay is identically zero; dk for per-key decay (KDA,
                       RWKV6, GLA))
    K    [N, C, dk]    deferred key-side factors a_i       (C = M - 1 live-log capacity)
    U    [N, C, dv]    deferred value-side factors b_i
    Lam  [N, C, dl]    log-decay snapshot taken when entry i was appended
    L    [N]           live-log length, 0 <= L <= C

The represented logical state is Eq. 7:

    S = D(ell) Sbar + sum_{i < L} D(ell - Lam_i) K_i U_i^T

and one decode step follows Alg. 1: pre-update readouts, ``ell <- ell + lambda``,
form (a, b) and any post-update output, then append (Eq. 5) if L < C, else merge
(Eq. 6) and reset.  Every quantity here is evaluated from the *logical state* of
Eq. 7 with plain dense products, so the machine can be read against the paper line by
line; ``replay_readout`` additionally writes the readout directly in factored form (the
quantity a kernel computes without materialising S) and is pinned against the dense
readout in the tests.

Readings: the delta-rule correction is taken on the decayed
state D(lambda_t) S_{t-1}, which is Eq. 7 evaluated at the already-advanced ``ell``;
the merging step is the M-th step of a cycle and consumes that step's token (Eq. 6
includes a_t b_t^T); merge and flush are also defined at any live length L < C, since
Eqs. 6 and 7 are written for general L; log slots i >= L are never read.
"""

import numpy as np

from .eager import DELTA_OPS, OPS, PER_KEY_OPS


def _f64(x):
    return np.asarray(x, dtype=np.float64)


class DeltaLogModel:
    """Alg. 1 for a batch of N independent (slot, head) pairs, each with its own L."""

    def __init__(self, op, S0, M):
        if op not in OPS:
            raise ValueError(op)
        if M < 1:
            raise ValueError("merge interval M must be >= 1")
        S0 = _f64(S0)
        if S0.ndim == 2:
            S0 = S0[None]
        self.op = op
        self.M = int(M)
        self.C = self.M - 1
        N, dk, dv = S0.shape
        self.N, self.dk, self.dv = N, dk, dv
        self.dl = dk if op in PER_KEY_OPS else 1
        # Freshly initialised slot: dense base from "prefill", empty log (Sec. 4).
        self.Sbar = S0.copy()
        self.ell = np.zeros((N, self.dl))
        self.K = np.zeros((N, self.C, dk))
        self.U = np.zeros((N, self.C, dv))
        self.Lam = np.zeros((N, self.C, self.dl))
        self.L = np.zeros(N, dtype=np.int64)
        self.last_merged = np.zeros(N, dtype=bool)

    # ----------------------------------------------------------------- helpers
    def _rows(self, l):
        """exp(l) as per-row factors [N, dk] (D of Eq. 2); l is [N, dl]."""
        return np.exp(np.broadcast_to(l, (self.N, self.dk)))

    def _live(self, i):
        """Mask of heads whose entry i is live (i < L)."""
        return i < self.L

    def logical_state(self, ell=None):
        """Eq. 7 evaluated at cumulative log-decay ``ell`` (default: the stored one)."""
        ell = self.ell if ell is None else ell
        S = self._rows(ell)[:, :, None] * self.Sbar
        for i in range(self.C):
            live = self._live(i)
            if not live.any():
                continue
            w = np.zeros((self.N, self.dk))
            w[live] = self._rows(ell - self.Lam[:, i])[live]   # D(ell - Lam_i)
            S = S + (w * self.K[:, i])[:, :, None] * self.U[:, i][:, None, :]
        return S

    def replay_readout(self, x, ell=None):
        """x^T (Eq. 7 state) without forming S: base term plus one coefficient per entry.

        x^T D(ell) Sbar + sum_{i<L} ((exp(ell - Lam_i) * x) . K_i) U_i
        """
        ell = self.ell if ell is None else ell
        x = _f64(x)
        o = np.einsum("ni,nij->nj", self._rows(ell) * x, self.Sbar)
        for i in range(self.C):
            live = self._live(i)
            if not live.any():
                continue
            gam = np.zeros(self.N)
            gam[live] = np.sum(self._rows(ell - self.Lam[:, i])[live] * x[live]
                               * self.K[live, i], axis=-1)
            o = o + gam[:, None] * self.U[:, i]
        return o

    # ------------------------------------------------------------- the cycle
    def _commit(self, a, b, ell_new, merge, active):
        """Append (Eq. 5) where ``merge`` is False, merge (Eq. 6) where it is True.

        Heads outside ``active`` are left untouched.
        """
        mi = np.nonzero(merge & active)[0]
        ai = np.nonzero(~merge & active)[0]
        # Eq. 6 (evaluated before any head of this step is modified):
        # D(ell) Sbar + sum_{i<L} D(ell - Lam_i) K_i U_i^T + a b^T, then reset.
        S_new = self.logical_state(ell_new) + a[:, :, None] * b[:, None, :] if mi.size else None
        if ai.size:
            j = self.L[ai]
            self.K[ai, j] = a[ai]
            self.U[ai, j] = b[ai]
            self.Lam[ai, j] = ell_new[ai]
            self.ell[ai] = ell_new[ai]
            self.L[ai] += 1
        if mi.size:
            self.Sbar[mi] = S_new[mi]
            self.ell[mi] = 0.0
            self.L[mi] = 0
        self.last_merged = merge & active

    def step(self, q, k, v, beta, lam, u=None, force_merge=False, active=None):
        """One decode step of Alg. 1; returns the output o [N, dv].

        ``q`` is the receptance r for RWKV6.  ``lam`` is [N] (GDN, RetNet), [N, dk]
        (KDA, RWKV6, GLA), or None for linear attention (no decay: lambda = 0).
        ``force_merge`` merges every head regardless of L (a merge at L < C).
        ``active`` (bool [N], default all) selects the heads that take this step; the
        others keep their state and get NaN outputs (a partial decode batch).
        """
        active = np.full(self.N, True) if active is None else np.asarray(active, dtype=bool)
        if self.op == "linattn":
            lam = np.zeros((self.N, self.dl))
        q, k, v, lam = map(_f64, (q, k, v, lam))
        lam = lam.reshape(self.N, self.dl)
        if np.any(self.L > self.C) or np.any(self.L < 0):
            raise ValueError("live-log length out of range")
        merge = np.full(self.N, True) if force_merge else (self.L == self.C)
        if self.op == "rwkv6":
            # Alg. 1 takes operator readouts on the pre-update state first; for RWKV6
            # that is r^T S_{t-1} plus the bonus term r^T diag(u) k v^T.
            S_prev = self.logical_state()
            bonus = np.sum(q * _f64(u) * k, axis=-1)
            o = np.einsum("ni,nij->nj", q, S_prev) + bonus[:, None] * v
            ell_new = self.ell + lam                       # Alg. 1: ell <- ell + lambda_t
            a, b = k, v                                    # Table 1: pair (k_t, v_t)
        elif self.op not in DELTA_OPS:
            # linear attention, RetNet, GLA: pair (k_t, v_t), post-update output (Eq. 3)
            ell_new = self.ell + lam                       # Alg. 1: ell <- ell + lambda_t
            a, b = k, v
            S_t = self.logical_state(ell_new) + a[:, :, None] * b[:, None, :]
            o = np.einsum("ni,nij->nj", q, S_t)
        else:
            ell_new = self.ell + lam                       # Alg. 1: ell <- ell + lambda_t
            S_dec = self.logical_state(ell_new)            # = D(lambda_t) S_{t-1}
            c = np.einsum("ni,nij->nj", k, S_dec)          # old-state correction
            b = _f64(beta).reshape(self.N)[:, None] * (v - c)
            a = k                                          # Table 1: pair (k_t, b_t)
            S_t = S_dec + a[:, :, None] * b[:, None, :]
            o = np.einsum("ni,nij->nj", q, S_t)            # post-update output (Eq. 3)
        self._commit(a, b, ell_new, merge, active)
        return np.where(active[:, None], o, np.nan)

    def flush(self):
        """Materialise Eq. 7 into the base and clear the log (no token consumed)."""
        self.Sbar = self.logical_state()
        self.ell[:] = 0.0
        self.L[:] = 0

    def readout(self, x):
        """o = x^T S for the current logical state (Eq. 7); mutates nothing."""
        return np.einsum("ni,nij->nj", _f64(x), self.logical_state())
