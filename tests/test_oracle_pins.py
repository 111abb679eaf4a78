"""The fp64 oracle against what the paper and the mathematics fix (CPU only)."""

import pytest

from oracle import eager
from oracle.deltalog_model import DeltaLogModel

import oracle_pins as P

OPS = eager.OPS


def step(op, S, q, k, v, beta, lam, u):
    return eager.eager_step(op, S, q, k, v, beta, lam, u=u)


@pytest.mark.parametrize("op", OPS)
def test_bruteforce_2x2_exact_rationals(op):
    P.pin_bruteforce_2x2(step, op)


@pytest.mark.parametrize("op", OPS)
def test_identity_update(op):
    P.pin_identity(step, op)


@pytest.mark.parametrize("op", OPS)
def test_decay_only_closed_form(op):
    P.pin_decay_only(step, op)


@pytest.mark.parametrize("op", ("gdn", "kda"))
def test_delta_write_stores_value(op):
    P.pin_delta_write(step, op)


@pytest.mark.parametrize("op", ("gdn", "kda"))
def test_published_matrix_form(op):
    P.pin_published_delta_rule(step, op)


def test_kda_with_equal_keys_is_gdn():
    P.pin_kda_equal_keys_is_gdn(step)


def test_rwkv6_reduces_to_linear_attention():
    P.pin_rwkv6_linear_attention(step)


def test_rwkv6_bonus_term():
    P.pin_rwkv6_bonus(step)


def test_linear_attention_matrix_form():
    P.pin_linear_attention_matrix_form(step)


def test_retnet_parallel_retention():
    P.pin_retnet_parallel_form(step)


def test_gla_parallel_form():
    P.pin_gla_parallel_form(step)


def test_gla_with_equal_gates_is_retnet():
    P.pin_gla_equal_gates_is_retnet(step)


@pytest.mark.parametrize("op", OPS)
@pytest.mark.parametrize("M", (1, 2, 3, 8))
def test_model_matches_eager_every_step(op, M):
    P.pin_model_matches_eager(DeltaLogModel, step, op, M)


def test_model_overwrite_through_log():
    P.pin_model_overwrite_through_log(DeltaLogModel)


@pytest.mark.parametrize("op", OPS)
def test_model_replay_readout(op):
    P.pin_model_replay_readout(DeltaLogModel, op)


@pytest.mark.parametrize("op", OPS)
def test_model_merge_is_gemm(op):
    P.pin_model_merge_is_gemm(DeltaLogModel, op)


@pytest.mark.parametrize("op", OPS)
def test_model_flush_readout_forced_merge(op):
    P.pin_model_flush_and_readout(DeltaLogModel, step, op)


@pytest.mark.parametrize("op", OPS)
def test_model_partial_batch(op):
    P.pin_model_partial_batch(DeltaLogModel, step, op)


def test_undecayed_reading_is_rejected_by_the_pins():
    """The literal undecayed-correction reading of Table 1 fails the delta-write and the
    published-form pins, so the pins decide between the two readings."""
    def literal(op, S, q, k, v, beta, lam, u):
        return eager.eager_step(op, S, q, k, v, beta, lam, u=u, correction="undecayed")
    for pin in (P.pin_delta_write, P.pin_published_delta_rule):
        with pytest.raises(AssertionError):
            pin(literal, "gdn")


def test_rel_fro():
    import numpy as np
    a = np.array([3.0, 4.0])
    assert eager.rel_fro(a, a) == 0.0
    assert abs(eager.rel_fro(a + [0.0, 0.5], a) - 0.1) < 1e-15
