"""The per-head traffic model (Eqs. 8-10) against the DRAM traffic the paper prints."""

import json
import os

import pytest

from paper_2608_15533_amd import traffic as T

GOLD = os.path.join(os.path.dirname(__file__), "golden", "gdn_b128_h32_d128_m8_dram_traffic.json")
GIB = float(1 << 30)


def _gold():
    with open(GOLD) as f:
        return json.load(f)


def test_read_traffic_reproduces_printed_counters():
    """Reads are what the model predicts within 1% at the three printed points (dense,
    append at live length 0 and 6, merge at 7).  Reads are not distorted by write-back
    residency in the cache, unlike the printed write figures."""
    g = _gold()
    heads = g["B"] * g["H"]
    args = (g["op"], g["dk"], g["dv"])
    pts = {                                  # the paper's representation (ell stored)
        "dense_read": T.eager_bytes(*args).read,
        "append_read_L0": T.append_bytes(*args, 0, stored_ell=True).read,
        "append_read_L6": T.append_bytes(*args, 6, stored_ell=True).read,
        "merge_read_L7": T.merge_bytes(*args, 7, stored_ell=True).read,
    }
    for key, per_head in pts.items():
        model = per_head * heads / GIB
        assert abs(model - g[key]) / g[key] < 0.01, (key, model, g[key])


def test_write_ratio_bounds_printed_reduction():
    """The model's state-write ratio M/(1+eps) for this shape is 7.39; the printed 7.83x is
    above it (the printed dense write, 0.230 GiB, sits below the 0.25 GiB state, so the
    counters miss some write-back).  The model ratio is the conservative bar."""
    g = _gold()
    r = T.state_write_ratio(g["op"], g["dk"], g["dv"], g["M"])
    assert 7.3 < r < g["write_reduction"]
    assert r < g["M"]


@pytest.mark.parametrize("op,dk,M,in_dtype,eager,app0,merge", [
    ("gdn", 64, 8, "f32", 33800, 17940, 37420),
    ("gdn", 128, 16, "bf16", 132360, 67604, 143948),
    ("kda", 128, 8, "bf16", 132868, 69636, 142852),
    ("rwkv6", 64, 16, "bf16", 33664, 18304, 41856),
])
def test_per_head_bytes(op, dk, M, in_dtype, eager, app0, merge):
    """Hand-summed per-head totals (fp32 output, fp32 state) for the tested shapes, in
    the paper's representation; this library's layout drops the cumulative log-decay
    read and write (8 bytes per step with one log-decay per head, 8 dk per key)."""
    assert T.eager_bytes(op, dk, dk, in_dtype).total == eager
    assert T.append_bytes(op, dk, dk, 0, in_dtype, stored_ell=True).total == app0
    assert T.merge_bytes(op, dk, dk, M - 1, in_dtype, stored_ell=True).total == merge
    saved = 8 * (dk if op in ("kda", "rwkv6", "gla") else 1)
    assert T.append_bytes(op, dk, dk, 0, in_dtype).total == app0 - saved
    assert T.merge_bytes(op, dk, dk, M - 1, in_dtype).total == merge - saved


def test_benefit_condition():
    """Eq. 10 benefit condition: DeltaLog moves fewer bytes than eager iff
    C_state (1 - 1/M) > C_log(M) + 2 C_decay; true for M in 2..32 at 128x128 GDN."""
    eager = T.eager_bytes("gdn", 128, 128).total
    for M in range(2, 33):
        assert T.amortized_bytes_per_token("gdn", 128, 128, M, stored_ell=True) < eager
        assert T.amortized_bytes_per_token("gdn", 128, 128, M) < eager
    # M = 1 is the eager step plus the cumulative log-decay traffic of the paper's
    # representation; this library keeps none for head-wise decay, so it equals eager
    assert T.amortized_bytes_per_token("gdn", 128, 128, 1, stored_ell=True) > eager
    assert T.amortized_bytes_per_token("gdn", 128, 128, 1) == eager


def test_byte_optimal_merge_interval():
    """Eq. 10's optimum for the tested shapes (bf16 activations, fp32 state): an interior
    minimum that is larger for head-wise scalar decay (compact metadata) than for
    per-key decay, and no larger than where the benefit condition still holds."""
    gdn = T.byte_optimal_merge_interval("gdn", 128, 128)
    kda = T.byte_optimal_merge_interval("kda", 128, 128)
    rwkv6 = T.byte_optimal_merge_interval("rwkv6", 64, 64)
    assert (gdn, kda, rwkv6) == (13, 10, 8)
    for op, d, m in (("gdn", 128, gdn), ("kda", 128, kda), ("rwkv6", 64, rwkv6)):
        a = [T.amortized_bytes_per_token(op, d, d, M) for M in range(1, 65)]
        assert a[m - 1] == min(a)
        assert a[m - 1] < T.eager_bytes(op, d, d).total


def test_library_write_ratio_against_the_bound():
    """The library writes the live length (4 bytes per head-step) where the paper's
    representation writes the cumulative log-decay (4 dl bytes): with one log-decay per
    head the implied write ratio equals the bound of Eq. 9, with per-key decay it
    exceeds it, and without decay (linear attention) the live length puts it just
    below."""
    for op, d, M in (("gdn", 128, 16), ("retnet", 128, 16), ("gdn", 64, 8)):
        assert T.library_state_write_ratio(op, d, d, M) == pytest.approx(
            T.state_write_ratio(op, d, d, M), rel=1e-12)
    for op, d, M in (("kda", 128, 16), ("rwkv6", 64, 16), ("gla", 128, 16)):
        assert T.library_state_write_ratio(op, d, d, M) > 1.05 * T.state_write_ratio(op, d, d, M)
    lib, bound = (T.library_state_write_ratio("linattn", 128, 128, 16),
                  T.state_write_ratio("linattn", 128, 128, 16))
    assert lib < bound and (bound - lib) / bound < 0.002


def test_live_length_metadata_lowers_the_write_ratio_slightly():
    """The int32 live length written every step is metadata outside Eq. 9; including it
    lowers the implied write reduction by well under 1% at the tested shapes."""
    for op, d, M in (("gdn", 128, 16), ("kda", 128, 16), ("rwkv6", 64, 16)):
        base = T.state_write_ratio(op, d, d, M)
        with_len = T.state_write_ratio(op, d, d, M, live_length_bytes=4)
        assert with_len < base
        assert (base - with_len) / base < 0.01
