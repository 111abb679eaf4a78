"""Randomised argument checks of the C ABI on a host without a GPU.

Every call here has a misaligned output pointer, which the library checks last: a call
that passes every other check stops there with DL_E_ALIGN.  So each fuzzed call must
return a negative dl_status (or DL_OK for n == 0, which is a no-op) and none may reach a
HIP call (DL_E_HIP).  For single perturbations of a valid call the status must be the
one the header documents for that argument."""

import ctypes
import random

import pytest
import torch

from paper_2608_15533_amd import deltalog as D

A = 0x10000000

# These calls hand fake device addresses to the real library and rely on its host-side
# checks to refuse every one of them; where a GPU is visible a regression in those checks
# would launch a kernel on such an address, so the module runs only where none is.
pytestmark = pytest.mark.skipif(torch.cuda.device_count() > 0,
                                reason="fake device addresses: only on a host without a GPU")
O_BAD = A + 0xB00004                                  # misaligned output: never launches


def _state():
    return D.dl_state(A, A + 0x200000, A + 0x300000, A + 0x400000, A + 0x500000, None)


def _token():
    return D.dl_token(A + 0x600000, A + 0x700000, A + 0x800000, A + 0x900000, A + 0xA00000,
                      A + 0xC00000)


def _call(entry, d, s, t, n, slots, extra):
    if entry == "append":
        return D.lib.dl_append_step(ctypes.byref(d), ctypes.byref(s), ctypes.byref(t), O_BAD,
                                    slots, n, None)
    if entry == "eager":
        return D.lib.dl_eager_step(ctypes.byref(d), A, ctypes.byref(t), O_BAD, slots, n, None)
    if entry == "merge":
        return D.lib.dl_merge(ctypes.byref(d), ctypes.byref(s), ctypes.byref(t), O_BAD, slots,
                              n, None)
    if entry == "readout":
        return D.lib.dl_readout(ctypes.byref(d), ctypes.byref(s), A + 0x600000, O_BAD, slots,
                                n, None)
    nv, split = extra
    return D.lib.dl_append_step_tiled(ctypes.byref(d), ctypes.byref(s), ctypes.byref(t), O_BAD,
                                      slots, n, nv, split, A + 0xD00000, 1 << 24, None)


DESC_FIELDS = {
    "abi_version": [1, 3, 4, 5],
    "op": [-1, 0, 1, 2, 3, 4, 5, 6],
    "num_slots": [-1, 0, 1, 4],
    "heads": [-1, 0, 1, 2],
    "dk": [0, 32, 64, 96, 128, 256],
    "dv": [0, 64, 100, 128],
    "merge_interval": [-1, 0, 1, 17, 64, 65],
    "in_dtype": [-1, 0, 1, 2],
    "u_log_dtype": [0, 1, 5],
    "state_dtype": [0, 1, 3],
}
PTR_CHOICES = [None, A, A + 2, A + 4, A + 8]


@pytest.mark.parametrize("seed", range(40))
def test_fuzzed_calls_never_launch(seed):
    rng = random.Random(seed)
    for _ in range(250):
        op = rng.choice(["gdn", "kda", "rwkv6", "linattn", "retnet", "gla"])
        d = D.make_desc(op, 4, 2, 128, 128, 16, "bf16")
        s, t = _state(), _token()
        for _ in range(rng.randint(0, 3)):
            f = rng.choice(list(DESC_FIELDS))
            setattr(d, f, rng.choice(DESC_FIELDS[f]))
        for _ in range(rng.randint(0, 2)):
            obj, fields = rng.choice([(s, [f for f, _ in D.dl_state._fields_]),
                                      (t, [f for f, _ in D.dl_token._fields_])])
            setattr(obj, rng.choice(fields), rng.choice(PTR_CHOICES))
        n = rng.choice([-1, 0, 1, 3, 4, 5])
        slots = rng.choice([None, A + 0xE00000, A + 0xE00002])
        entry = rng.choice(["append", "eager", "merge", "readout", "tiled"])
        extra = (rng.choice([0, 1, 2, 3, 4, 8]), rng.choice([0, 1]))
        rc = _call(entry, d, s, t, n, slots, extra)
        assert rc != D.DL_E_HIP, (seed, entry)
        assert rc < 0 or (rc == D.DL_OK and n == 0), (seed, entry, rc)
        assert D.dl_status_str(rc) != "unknown dl_status"


@pytest.mark.parametrize("entry", ["append", "eager", "merge", "readout", "tiled"])
def test_valid_call_stops_at_the_output_alignment(entry):
    for op in ("gdn", "kda", "rwkv6", "linattn", "retnet", "gla"):
        d = D.make_desc(op, 4, 2, 128, 128, 16, "bf16")
        assert _call(entry, d, _state(), _token(), 4, None, (4, 1)) == D.DL_E_ALIGN, op
        assert _call(entry, d, _state(), _token(), 0, None, (4, 1)) == D.DL_OK, op


@pytest.mark.parametrize("field,value,code", [
    ("abi_version", 5, D.DL_E_VERSION), ("op", 6, D.DL_E_UNSUPPORTED),
    ("dk", 96, D.DL_E_UNSUPPORTED), ("merge_interval", 65, D.DL_E_UNSUPPORTED),
    ("num_slots", 0, D.DL_E_SHAPE), ("in_dtype", 2, D.DL_E_DTYPE),
    ("state_dtype", 3, D.DL_E_DTYPE),
])
@pytest.mark.parametrize("entry", ["append", "eager", "merge", "readout", "tiled"])
def test_single_descriptor_faults_map_to_documented_codes(entry, field, value, code):
    d = D.make_desc("gdn", 4, 2, 128, 128, 16, "bf16")
    setattr(d, field, value)
    assert _call(entry, d, _state(), _token(), 4, None, (4, 1)) == code
