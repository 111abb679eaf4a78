"""GPU parity at the full launch sizes with every slot followed by the fp64 oracle.

The full-size rollouts of ``test_gpu_parity`` run all slots on the GPU but follow three
slots with the oracle, and its every-slot check compares the DeltaLog kernel with the
eager kernel of the same template.  Here the oracle follows every (slot, head) of the
launch the benchmark times, for one merge cycle and one step past it: every output of
every step, the dense base of every slot right after it merges (Eq. 6), and every base
after a final flush of the one-entry logs (Eq. 7).  The staggered serving-stack layer
runs its partial-batch warm-up first, so its 16 steps merge every slot once, at 16
different steps.  Bar: relative Frobenius error <= 1e-4 (fp32 state)."""

import pytest

from paper_2608_15533_amd import workloads as W

from gpu_harness import TOL_F32_STATE, Rollout, log

pytestmark = pytest.mark.gpu

CASES = [
    ("gdn_b64_h32_d128_m16", W.GDN_B64, 16),
    ("kda_b128_h32_d128_m16", W.KDA_B128, 16),
    ("kda_b128_h32_d128_m32", W.KDA_B128, 32),      # the long-log build (C > 16)
    ("rwkv6_b128_h40_d64_m16", W.RWKV6_B128, 16),
    ("gla_b128_h32_d128_m16", W.GLA_B128, 16),
]


@pytest.mark.parametrize("name,w,M", CASES, ids=[c[0] for c in CASES])
def test_every_slot_one_cycle(name, w, M):
    r = Rollout(w, M=M, steps=M + 1).run()
    e_flush = r.flush_and_check()
    log(f"{name} every slot, {M + 1} steps: max out err {r.err_out:.2e}, "
        f"max state err {r.err_state:.2e} ({r.n_state_checks} merge checks), flush {e_flush:.2e}")
    assert r.device_error_word() == 0
    assert r.n_state_checks == 1
    assert r.err_out <= TOL_F32_STATE, name
    assert r.err_state <= TOL_F32_STATE, name


def test_every_slot_serving_stack_layer():
    """Layer 0 of the 24-layer stack (256 slots x 32 heads, fill offsets uniform in
    [0, M)): warm-up through slot lists, then M steps in which every slot merges once."""
    w = W.GDN_STACK
    r = Rollout(w, steps=w.M).run()
    e_flush = r.flush_and_check()
    log(f"stack layer 0 every slot: max out err {r.err_out:.2e}, max state err "
        f"{r.err_state:.2e} ({r.n_state_checks} merge steps), flush {e_flush:.2e}")
    assert r.device_error_word() == 0
    assert r.n_state_checks >= w.M - 1              # one step per fill offset that merges
    assert r.err_out <= TOL_F32_STATE
    assert r.err_state <= TOL_F32_STATE
