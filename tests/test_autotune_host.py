"""Host logic of the merge-interval selection (no GPU): the amortised step-time
prediction against its closed form for affine phase costs, and the choice against
brute force."""

import random

import pytest

from paper_2608_15533_amd import autotune as A


def _affine(alpha, beta, mu, nu, max_M):
    a = [alpha + beta * L for L in range(max_M - 1)]
    m = [mu + nu * L for L in range(max_M)]
    return a, m


def test_prediction_matches_closed_form_for_affine_costs():
    # a(L) = alpha + beta L, m(L) = mu + nu L:
    # T(M) = ((M-1) alpha + beta (M-1)(M-2)/2 + mu + nu (M-1)) / M
    alpha, beta, mu, nu = 20.0, 0.4, 50.0, 1.5
    a, m = _affine(alpha, beta, mu, nu, 64)
    T = A.predict(a, m)
    assert sorted(T) == list(range(1, 65))
    for M, t in T.items():
        ref = ((M - 1) * alpha + beta * (M - 1) * (M - 2) / 2 + mu + nu * (M - 1)) / M
        assert t == pytest.approx(ref, rel=1e-12)


def test_eager_equivalent_and_single_append():
    a, m = [3.0, 4.0], [10.0, 12.0, 15.0]
    T = A.predict(a, m)
    assert T[1] == 10.0                      # M = 1: every step merges at L = 0
    assert T[2] == pytest.approx((3.0 + 12.0) / 2)
    assert T[3] == pytest.approx((3.0 + 4.0 + 15.0) / 3)


def test_choice_is_the_brute_force_argmin():
    rng = random.Random(7)
    for _ in range(200):
        n = rng.randint(2, 64)
        a = [rng.uniform(1, 100) for _ in range(n - 1)]
        m = [rng.uniform(1, 200) for _ in range(n)]
        M, T = A.choose(a, m)
        brute = [(sum(a[:k - 1]) + m[k - 1]) / k for k in range(1, n + 1)]
        best = min(range(1, n + 1), key=lambda k: (brute[k - 1], k))
        assert M == best


def test_u_shape_optimum_near_continuous_optimum():
    # With a(L) = alpha + beta L and m(L) = mu (flat), T(M) ~ alpha + beta M / 2 +
    # (mu - alpha) / M, minimised near M* = sqrt(2 (mu - alpha) / beta).
    alpha, beta, mu = 25.0, 0.5, 75.0
    a, m = _affine(alpha, beta, mu, 0.0, 64)
    M, T = A.choose(a, m)
    cont = (2 * (mu - alpha) / beta) ** 0.5
    assert abs(M - cont) <= 1.5
    assert T[M] < T[1] and T[M] < T[64]


def test_monotone_cases_pick_the_ends():
    # merges far dearer than appends that never grow: the longest log wins
    a, m = [1.0] * 63, [100.0] * 64
    assert A.choose(a, m)[0] == 64
    # appends as dear as the merge: eager-equivalent M = 1 (ties go to the smaller M)
    a, m = [10.0] * 63, [10.0] * 64
    assert A.choose(a, m)[0] == 1


def test_unmeasured_intervals_are_left_out():
    T = A.predict([1.0, 2.0], [5.0] * 10)
    assert sorted(T) == [1, 2, 3]
