"""The seeded input generators: reproducible, correctly rounded, correctly shaped."""

import numpy as np
import pytest
import torch

from paper_2608_15533_amd import workloads as W


def test_round_bf16_matches_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(100000).astype(np.float32),
                        np.float32([0.0, -0.0, 1.0, 1.00390625, 1.005859375, 3.0e-39, 65504.0])])
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    np.testing.assert_array_equal(W.round_bf16(x), ref)


@pytest.mark.parametrize("w", list(W.WORKLOADS.values()), ids=lambda w: w.name)
def test_step_inputs_shapes_and_determinism(w):
    w = w.with_(B=min(w.B, 4))
    a, b = W.step_inputs(w, 3), W.step_inputs(w, 3)
    for key in a:
        if a[key] is None:
            assert (key == "beta" and w.op not in ("gdn", "kda")) or \
                (key == "lam" and w.op == "linattn")
            continue
        np.testing.assert_array_equal(a[key], b[key])
        assert a[key].dtype == np.float32
    assert a["q"].shape == (w.B, w.H, w.dk) and a["v"].shape == (w.B, w.H, w.dv)
    if w.op != "linattn":
        assert a["lam"].shape == ((w.B, w.H) if w.dl == 1 else (w.B, w.H, w.dk))
        assert np.all(a["lam"] <= 0.0)
    if w.in_dtype == "bf16":
        for key in ("q", "k", "v"):
            np.testing.assert_array_equal(W.round_bf16(a[key]), a[key])
    if w.op != "rwkv6":
        n = np.linalg.norm(a["k"].astype(np.float64), axis=-1)
        assert np.all(np.abs(n - 1.0) < 1e-2)
    c = W.step_inputs(w, 4)
    assert not np.array_equal(a["k"], c["k"])


def test_initial_state_per_slot_seeding():
    w = W.GDN_B64
    full = W.initial_state(w.with_(B=3))
    part = W.initial_state(w, slots=[2])
    np.testing.assert_array_equal(full[2], part[0])
    assert abs(full.std() - 0.02) < 1e-3


def test_gate_distributions():
    g = W.step_inputs(W.GDN_B64, 0)
    alpha = np.exp(g["lam"].astype(np.float64))
    assert 0.94 < alpha.mean() < 0.96          # E[sigmoid(N(3, .5))] ~ 0.95
    k = W.step_inputs(W.KDA_B128.with_(B=8), 0)
    assert abs(np.mean(-16.0 * k["lam"]) - 0.806) < 0.02   # E[softplus(N(0,1))] ~ 0.806
    r = W.step_inputs(W.RWKV6_B128.with_(B=8), 0)
    w6 = np.exp(r["lam"].astype(np.float64))
    assert 0.5 < w6.mean() < 0.6
    gl = W.step_inputs(W.GLA_B128.with_(B=8), 0)
    assert abs(np.mean(16.0 * gl["lam"]) + 0.806) < 0.02   # E[log sigmoid(N(0,1))] ~ -0.806
    rn = W.step_inputs(W.RETNET_B64.with_(B=2), 5)
    gamma = np.exp(rn["lam"][0].astype(np.float64))
    np.testing.assert_allclose(1.0 - gamma, 2.0 ** (-5.0 - 5.0 * np.arange(32) / 32), rtol=1e-5)
    assert np.array_equal(rn["lam"], W.step_inputs(W.RETNET_B64.with_(B=2), 9)["lam"])
    la = W.step_inputs(W.LINATTN_B64.with_(B=2), 0)
    assert np.all(la["q"] > 0) and np.all(la["k"] > 0)     # positive feature map


def test_staggered_warmup_reaches_offsets():
    w = W.GDN_STACK
    off = W.fill_offsets(w)
    assert off.min() >= 0 and off.max() <= w.M - 1
    taken = np.zeros(w.B, dtype=np.int64)
    for _, sl in W.warmup_schedule(w):
        taken[sl] += 1
    np.testing.assert_array_equal(taken, off)
