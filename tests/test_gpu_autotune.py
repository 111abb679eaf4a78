"""GPU check of the merge-interval calibration: every live length is measured, the
costs are finite and positive, the chosen interval is valid, and the state buffers
report no device error."""

import math

import pytest

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("op,dk,dv", [("gdn", 128, 128), ("rwkv6", 64, 64), ("linattn", 64, 128)])
def test_calibration_covers_every_length(op, dk, dv):
    from paper_2608_15533_amd import autotune as A
    cal = A.calibrate(op, 4, 2, dk, dv, max_M=8, replicas=2, reps=2)
    assert len(cal["append_us"]) == 7 and len(cal["merge_us"]) == 8
    for t in cal["append_us"] + cal["merge_us"]:
        assert math.isfinite(t) and t > 0
    M, T = A.choose(cal["append_us"], cal["merge_us"])
    assert 1 <= M <= 8 and sorted(T) == list(range(1, 9))


def test_calibration_rejects_out_of_range_interval():
    from paper_2608_15533_amd import autotune as A
    with pytest.raises(ValueError):
        A.calibrate("gdn", 4, 2, 64, 64, max_M=65)
