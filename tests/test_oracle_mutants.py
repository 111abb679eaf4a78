"""Plant plausible mistakes in copies of the oracle (on the CPU) and require the pins to
catch every one of them: a dropped term, a wrong sign, a transposed operand, a wrong
index or snapshot, a missing reset.  This is what makes the pins a pin."""

import numpy as np
import pytest

from oracle import eager
from oracle.deltalog_model import DeltaLogModel

import oracle_pins as P


def _ein(x, S):
    return np.einsum("...i,...ij->...j", x, S)


def _mut_delta(kind):
    def step(op, S, q, k, v, beta, lam, u):
        if op == "rwkv6":
            return eager.eager_step(op, S, q, k, v, beta, lam, u=u)
        S, q, k, v, beta = (np.asarray(x, dtype=np.float64) for x in (S, q, k, v, beta))
        rows = eager.row_decay(lam, S.shape[-2], op == "kda")
        Sd = rows * S
        if kind == "column_decay":
            Sd = np.swapaxes(rows, -1, -2) * S
        if kind == "negated_decay":
            Sd = S / rows
        c = _ein(k, Sd)
        if kind == "undecayed":
            c = _ein(k, S)
        if kind == "correction_with_q":
            c = _ein(q, Sd)
        b = beta[..., None] * (v - c)
        if kind == "drop_beta":
            b = v - c
        if kind == "sign":
            b = beta[..., None] * (v + c)
        if kind == "drop_correction":
            b = beta[..., None] * v
        outer = k[..., :, None] * b[..., None, :]
        if kind == "outer_transposed":
            outer = np.swapaxes(outer, -1, -2)
        S_new = Sd + outer
        o = _ein(q, S_new)
        if kind == "pre_update_output":
            o = _ein(q, Sd)
        if kind == "transposed_readout":
            o = np.einsum("...i,...ji->...j", q, S_new)
        return S_new, o
    return step


def _mut_rwkv6(kind):
    def step(op, S, q, k, v, beta, lam, u):
        if op != "rwkv6":
            return eager.eager_step(op, S, q, k, v, beta, lam, u=u)
        S, r, k, v, u = (np.asarray(x, dtype=np.float64) for x in (S, q, k, v, u))
        rows = eager.row_decay(lam, S.shape[-2], True)
        bonus = np.sum(r * u * k, axis=-1)
        if kind == "bonus_without_u":
            bonus = np.sum(r * k, axis=-1)
        S_new = rows * S + k[..., :, None] * v[..., None, :]
        o = _ein(r, S) + bonus[..., None] * v
        if kind == "no_bonus":
            o = _ein(r, S)
        if kind == "post_update_readout":
            o = _ein(r, S_new)
        if kind == "undecayed_write":
            S_new = S + k[..., :, None] * v[..., None, :]
        return S_new, o
    return step


def _mut_additive(kind):
    def step(op, S, q, k, v, beta, lam, u):
        if op not in eager.ADDITIVE_OPS:
            return eager.eager_step(op, S, q, k, v, beta, lam, u=u)
        S, q, k, v = (np.asarray(x, dtype=np.float64) for x in (S, q, k, v))
        if op == "linattn":
            rows = np.ones(S.shape[:-1] + (1,))
        else:
            rows = eager.row_decay(lam, S.shape[-2], op == "gla")
        Sd = rows * S
        if kind == "ignore_decay":
            Sd = S
        if kind == "column_decay":
            Sd = np.swapaxes(rows, -1, -2) * S
        outer = k[..., :, None] * v[..., None, :]
        if kind == "outer_transposed":
            outer = np.swapaxes(outer, -1, -2)
        S_new = Sd + outer
        if kind == "decay_after_write":
            S_new = rows * (S + outer)
        if kind == "drop_state":
            S_new = outer
        o = _ein(q, S_new)
        if kind == "pre_update_output":
            o = _ein(q, Sd)
        if kind == "transposed_readout":
            o = np.einsum("...i,...ji->...j", q, S_new)
        return S_new, o
    return step


DELTA_MUTANTS = ["column_decay", "negated_decay", "undecayed", "correction_with_q", "drop_beta",
                 "sign", "drop_correction", "outer_transposed", "pre_update_output",
                 "transposed_readout"]
RWKV6_MUTANTS = ["bonus_without_u", "no_bonus", "post_update_readout", "undecayed_write"]
ADDITIVE_MUTANTS = ["ignore_decay", "column_decay", "outer_transposed", "decay_after_write",
                    "drop_state", "pre_update_output", "transposed_readout"]


def _eager_pins(step, ops):
    for op in ops:
        yield lambda op=op: P.pin_bruteforce_2x2(step, op)
        yield lambda op=op: P.pin_identity(step, op)
        yield lambda op=op: P.pin_decay_only(step, op)
        if op in ("gdn", "kda"):
            yield lambda op=op: P.pin_delta_write(step, op)
            yield lambda op=op: P.pin_published_delta_rule(step, op)
    if "rwkv6" in ops:
        yield lambda: P.pin_rwkv6_linear_attention(step)
        yield lambda: P.pin_rwkv6_bonus(step)
    if "linattn" in ops:
        yield lambda: P.pin_linear_attention_matrix_form(step)
    if "retnet" in ops:
        yield lambda: P.pin_retnet_parallel_form(step)
    if "gla" in ops:
        yield lambda: P.pin_gla_parallel_form(step)
        yield lambda: P.pin_gla_equal_gates_is_retnet(step)


def _caught(pins):
    for pin in pins:
        try:
            pin()
        except (AssertionError, FloatingPointError):
            return True
    return False


@pytest.mark.parametrize("kind", DELTA_MUTANTS)
@pytest.mark.parametrize("op", ("gdn", "kda"))
def test_eager_delta_rule_mutant_is_caught(op, kind):
    if kind == "column_decay" and op == "gdn":
        pytest.skip("a scalar decay scales rows and columns alike: not a mistake for GDN")
    assert _caught(_eager_pins(_mut_delta(kind), (op,))), f"{op} mutant {kind} not caught"


@pytest.mark.parametrize("kind", RWKV6_MUTANTS)
def test_eager_rwkv6_mutant_is_caught(kind):
    assert _caught(_eager_pins(_mut_rwkv6(kind), ("rwkv6",))), f"rwkv6 mutant {kind} not caught"


@pytest.mark.parametrize("kind", ADDITIVE_MUTANTS)
@pytest.mark.parametrize("op", ("linattn", "retnet", "gla"))
def test_eager_additive_mutant_is_caught(op, kind):
    if op == "linattn" and kind in ("ignore_decay", "column_decay", "decay_after_write"):
        pytest.skip("linear attention has no decay: not a mistake for it")
    if op == "retnet" and kind == "column_decay":
        pytest.skip("a scalar decay scales rows and columns alike: not a mistake for RetNet")
    assert _caught(_eager_pins(_mut_additive(kind), (op,))), f"{op} mutant {kind} not caught"


# ------------------------------------------------------------------ model mutants
class SnapshotBeforeDecay(DeltaLogModel):
    """Lam_L records the cumulative log-decay *before* adding lambda_t."""
    def _commit(self, a, b, ell_new, merge, active):
        old = self.ell.copy()
        super()._commit(a, b, ell_new, merge, active)
        app = ~merge & active
        j = self.L[app] - 1
        self.Lam[np.nonzero(app)[0], j] = old[app]


class NoResetAtMerge(DeltaLogModel):
    """The cumulative log-decay is not reset after a merge."""
    def _commit(self, a, b, ell_new, merge, active):
        super()._commit(a, b, ell_new, merge, active)
        mi = merge & active
        self.ell[mi] = ell_new[mi]


class MergeDropsToken(DeltaLogModel):
    """The merge forgets the current token's a b^T."""
    def _commit(self, a, b, ell_new, merge, active):
        super()._commit(a, b * (~merge)[:, None], ell_new, merge, active)


class MergeOneLate(DeltaLogModel):
    """Merges when L == M (one step late) instead of L == C; the log grows by one slot."""
    def __init__(self, op, S0, M):
        super().__init__(op, S0, M)
        self.C = M
        self.K = np.zeros((self.N, M, self.dk))
        self.U = np.zeros((self.N, M, self.dv))
        self.Lam = np.zeros((self.N, M, self.dl))

    def step(self, *a, **kw):
        self.C = self.M
        return super().step(*a, **kw)


class DecaySumNotDifference(DeltaLogModel):
    """Replays entry i with exp(ell + Lam_i) instead of exp(ell - Lam_i)."""
    def logical_state(self, ell=None):
        saved = self.Lam
        self.Lam = -saved
        try:
            return super().logical_state(ell)
        finally:
            self.Lam = saved


class EllNotAdvancedOnAppend(DeltaLogModel):
    """An append records the entry but leaves the cumulative log-decay unchanged."""
    def _commit(self, a, b, ell_new, merge, active):
        old = self.ell.copy()
        super()._commit(a, b, ell_new, merge, active)
        app = ~merge & active
        self.ell[app] = old[app]


MODEL_MUTANTS = [SnapshotBeforeDecay, NoResetAtMerge, MergeDropsToken, MergeOneLate,
                 DecaySumNotDifference, EllNotAdvancedOnAppend]


def _real_step(op, S, q, k, v, beta, lam, u):
    return eager.eager_step(op, S, q, k, v, beta, lam, u=u)


DECAY_BOOKKEEPING = (SnapshotBeforeDecay, NoResetAtMerge, DecaySumNotDifference,
                     EllNotAdvancedOnAppend)


@pytest.mark.parametrize("Model", MODEL_MUTANTS, ids=lambda c: c.__name__)
@pytest.mark.parametrize("op", eager.OPS)
def test_model_mutant_is_caught(op, Model):
    if op == "linattn" and Model in DECAY_BOOKKEEPING:
        pytest.skip("linear attention's log-decay is identically zero: not a mistake for it")
    pins = [lambda M=M: P.pin_model_matches_eager(Model, _real_step, op, M) for M in (2, 3, 8)]
    pins.append(lambda: P.pin_model_merge_is_gemm(Model, op))
    pins.append(lambda: P.pin_model_flush_and_readout(Model, _real_step, op))
    with np.errstate(all="ignore"):
        assert _caught(pins), f"{op} model mutant {Model.__name__} not caught"
