"""The C-ABI library on a host without a GPU: it loads, exports every symbol the header
declares, and rejects bad arguments before any HIP call (so nothing is launched).

Fake device addresses are used throughout: every call here fails validation (or has
n == 0), so no pointer is ever dereferenced and no kernel is enqueued."""

import ctypes
import os
import re
import subprocess

import pytest
import torch

from paper_2608_15533_amd import deltalog as D

HEADER = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include", "deltalog.h")

A = 0x10000000          # a fake, 256-byte aligned "device" address

# These calls hand fake device addresses to the real library and rely on its host-side
# checks to refuse every one of them; where a GPU is visible a regression in those checks
# would launch a kernel on such an address, so the module runs only where none is.
pytestmark = pytest.mark.skipif(torch.cuda.device_count() > 0,
                                reason="fake device addresses: only on a host without a GPU")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dl_[a-z_]+)\s*\(", text)))


def test_header_functions_are_exported():
    names = _declared_functions()
    assert set(names) == set(D.EXPORTED)
    out = subprocess.run(["nm", "-D", "--defined-only", D.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\bT (dl_[a-z_]+)\b", out))
    for n in names:
        assert n in exported, n
        assert hasattr(D.lib, n)


def test_version_and_status_strings():
    assert D.dl_abi_version() == D.DL_ABI_VERSION == 4
    for code in range(0, -9, -1):
        s = D.dl_status_str(code)
        assert s.startswith("DL_") and s != "unknown dl_status"
    assert D.dl_status_str(-99) == "unknown dl_status"


def desc(**kw):
    d = D.make_desc("gdn", 4, 2, 128, 128, 16, "bf16")
    for k, v in kw.items():
        setattr(d, k, v)
    return d


def state(**kw):
    s = D.dl_state(A, A + 0x200000, A + 0x300000, A + 0x400000, A + 0x500000, None)
    for k, v in kw.items():
        setattr(s, k, v)
    return s


def token(**kw):
    t = D.dl_token(A + 0x600000, A + 0x700000, A + 0x800000, A + 0x900000, A + 0xA00000, None)
    for k, v in kw.items():
        setattr(t, k, v)
    return t


def append(d, s=None, t=None, o=A + 0xB00000, slots=None, n=4):
    return D.lib.dl_append_step(ctypes.byref(d), ctypes.byref(s or state()),
                                ctypes.byref(t or token()), o, slots, n, None)


def test_null_descriptor():
    assert D.lib.dl_append_step(None, ctypes.byref(state()), ctypes.byref(token()), A, None, 4,
                                None) == D.DL_E_NULL


@pytest.mark.parametrize("field,value,code", [
    ("abi_version", 1, D.DL_E_VERSION),
    ("op", 6, D.DL_E_UNSUPPORTED),
    ("op", -1, D.DL_E_UNSUPPORTED),
    ("dk", 96, D.DL_E_UNSUPPORTED),
    ("dv", 256, D.DL_E_UNSUPPORTED),
    ("merge_interval", 0, D.DL_E_UNSUPPORTED),
    ("merge_interval", 65, D.DL_E_UNSUPPORTED),
    ("num_slots", 0, D.DL_E_SHAPE),
    ("heads", 0, D.DL_E_SHAPE),
    ("in_dtype", 7, D.DL_E_DTYPE),
    ("u_log_dtype", D.DL_BF16, D.DL_E_DTYPE),        # GDN U_log must be fp32
    ("state_dtype", 5, D.DL_E_DTYPE),
])
def test_descriptor_rejections(field, value, code):
    assert append(desc(**{field: value})) == code


def test_descriptor_layout_matches_header():
    """The ctypes mirror of dl_desc has the header's field order and size (10 int32)."""
    text = open(HEADER).read()
    body = re.search(r"typedef struct \{(.*?)\} dl_desc;", text, flags=re.S).group(1)
    body = re.sub(r"/\*.*?\*/", "", body, flags=re.S)
    names = re.findall(r"int32_t\s+([a-z_]+(?:\s*,\s*[a-z_]+)*)\s*;", body)
    fields = [n.strip() for group in names for n in group.split(",")]
    assert fields == [f for f, _ in D.dl_desc._fields_]
    assert ctypes.sizeof(D.dl_desc) == 4 * len(fields) == 40


def test_bf16_state_descriptor_is_accepted():
    """state_dtype = BF16 passes validation (the call then stops at a misaligned output)."""
    assert append(desc(state_dtype=D.DL_BF16), o=A + 4) == D.DL_E_ALIGN


def test_rwkv6_u_log_dtype_must_match_input():
    d = D.make_desc("rwkv6", 4, 2, 64, 64, 16, "bf16")
    d.u_log_dtype = D.DL_F32
    assert append(d, t=token(beta=None, u=A + 0xC00000)) == D.DL_E_DTYPE


def test_slot_list_rules():
    assert append(desc(), n=5) == D.DL_E_SHAPE              # n > B
    assert append(desc(), n=-1) == D.DL_E_SHAPE
    assert append(desc(), n=3) == D.DL_E_SHAPE              # identity needs n == B
    assert append(desc(), slots=A + 2, n=3) == D.DL_E_ALIGN


@pytest.mark.parametrize("field", ["S", "len", "k_log", "u_log", "lam_log"])
def test_state_nulls(field):
    assert append(desc(), s=state(**{field: None})) == D.DL_E_NULL


def test_state_has_no_cumulative_log_decay_buffer():
    """The cumulative log-decay is the newest Lam_log snapshot, not a buffer: dl_state
    holds S, the three log buffers, the live length and the error word."""
    assert [f for f, _ in D.dl_state._fields_] == ["S", "k_log", "u_log", "lam_log", "len",
                                                    "err"]


def test_log_buffers_optional_when_M_is_1():
    """With M == 1 there is no log: NULL log buffers pass the state checks (the call then
    stops at the misaligned output, which is checked after the state)."""
    s = state(k_log=None, u_log=None, lam_log=None)
    assert append(desc(merge_interval=1), s=s, o=A + 4) == D.DL_E_ALIGN
    assert append(desc(merge_interval=2), s=s, o=A + 4) == D.DL_E_NULL


@pytest.mark.parametrize("field", ["q", "k", "v", "lam", "beta"])
def test_token_nulls(field):
    assert append(desc(), t=token(**{field: None})) == D.DL_E_NULL


def test_rwkv6_needs_bonus():
    d = D.make_desc("rwkv6", 4, 2, 64, 64, 16, "bf16")
    assert append(d, t=token(beta=None)) == D.DL_E_NULL


def test_linear_attention_takes_no_decay_buffers():
    """Linear attention has no decay: NULL lam and lam_log (and beta) pass the checks
    (the call then stops at the misaligned output)."""
    d = D.make_desc("linattn", 4, 2, 128, 128, 16, "bf16")
    s = state(lam_log=None)
    assert append(d, s=s, t=token(lam=None, beta=None), o=A + 4) == D.DL_E_ALIGN
    assert append(d, s=state(k_log=None), t=token(lam=None, beta=None)) == D.DL_E_NULL


@pytest.mark.parametrize("op", ["retnet", "gla"])
def test_decaying_additive_operators_need_lam_not_beta(op):
    d = D.make_desc(op, 4, 2, 128, 128, 16, "bf16")
    assert append(d, t=token(beta=None), o=A + 4) == D.DL_E_ALIGN
    assert append(d, t=token(lam=None, beta=None)) == D.DL_E_NULL
    assert append(d, s=state(lam_log=None), t=token(beta=None)) == D.DL_E_NULL


@pytest.mark.parametrize("op", ["linattn", "retnet", "gla"])
def test_additive_u_log_holds_copies_of_v(op):
    """U_log of the operators without a correction holds v in the activation dtype."""
    d = D.make_desc(op, 4, 2, 128, 128, 16, "bf16")
    assert d.u_log_dtype == D.DL_BF16
    d.u_log_dtype = D.DL_F32
    assert append(d, t=token(beta=None)) == D.DL_E_DTYPE


@pytest.mark.parametrize("where,field,off", [
    ("state", "S", 8), ("state", "k_log", 4), ("state", "u_log", 8), ("state", "lam_log", 2),
    ("token", "q", 8), ("token", "k", 2), ("token", "v", 4), ("token", "lam", 1),
])
def test_alignment(where, field, off):
    if where == "state":
        s = state()
        setattr(s, field, getattr(s, field) + off)
        assert append(desc(), s=s) == D.DL_E_ALIGN
    else:
        t = token()
        setattr(t, field, getattr(t, field) + off)
        assert append(desc(), t=t) == D.DL_E_ALIGN


@pytest.mark.parametrize("op,off,code", [
    ("kda", 4, D.DL_E_ALIGN), ("rwkv6", 8, D.DL_E_ALIGN), ("gla", 12, D.DL_E_ALIGN),
    ("gdn", 4, D.DL_E_ALIGN + 100), ("retnet", 8, D.DL_E_ALIGN + 100),
])
def test_per_key_snapshots_need_16_byte_alignment(op, off, code):
    """Per-key Lam_log rows are read 16 bytes at a time: lam_log must be 16-byte aligned
    for KDA, RWKV6 and GLA; one snapshot per head (GDN, RetNet) needs 4 bytes.  (+100
    marks the calls that pass the state checks and stop at the misaligned output.)"""
    dk = 64 if op == "rwkv6" else 128
    d = D.make_desc(op, 4, 2, dk, dk, 16, "bf16")
    t = token(beta=None if op not in ("gdn", "kda") else A + 0x900000,
              u=A + 0xC00000 if op == "rwkv6" else None)
    s = state()
    s.lam_log += off
    if code == D.DL_E_ALIGN:
        assert append(d, s=s, t=t) == D.DL_E_ALIGN
    else:
        assert append(d, s=s, t=t, o=A + 4) == D.DL_E_ALIGN   # stopped at o, not at lam_log
        assert append(d, s=s, t=t, o=None) == D.DL_E_NULL


def test_output_checks():
    assert append(desc(), o=None) == D.DL_E_NULL
    assert append(desc(), o=A + 4) == D.DL_E_ALIGN


def test_zero_rows_is_a_no_op():
    """n == 0 returns DL_OK without touching the GPU (this host has none)."""
    assert append(desc(), slots=A, n=0) == D.DL_OK
    d = desc()
    assert D.lib.dl_eager_step(ctypes.byref(d), A, ctypes.byref(token()), A, A, 0, None) == D.DL_OK
    assert D.lib.dl_merge(ctypes.byref(d), ctypes.byref(state()), None, None, A, 0, None) == D.DL_OK
    assert D.lib.dl_readout(ctypes.byref(d), ctypes.byref(state()), A, A, A, 0, None) == D.DL_OK
    assert append(desc(), slots=None, n=0) == D.DL_OK      # an empty list may be NULL
    assert append(desc(), s=state(S=None), t=token(q=None), o=None, n=0) == D.DL_OK


def test_other_entry_points_validate():
    d = desc()
    assert D.lib.dl_eager_step(ctypes.byref(d), None, ctypes.byref(token()), A, None, 4, None) == D.DL_E_NULL
    assert D.lib.dl_merge(ctypes.byref(d), ctypes.byref(state()), ctypes.byref(token()), None,
                          None, 4, None) == D.DL_E_NULL          # a merge with a token needs o
    assert D.lib.dl_merge(ctypes.byref(d), None, None, None, None, 4, None) == D.DL_E_NULL
    assert D.lib.dl_readout(ctypes.byref(d), ctypes.byref(state()), None, A, None, 4, None) == D.DL_E_NULL
    assert D.lib.dl_readout(ctypes.byref(d), ctypes.byref(state()), A + 8, A, None, 4, None) == D.DL_E_ALIGN


def tiled(d, s=None, t=None, o=A + 0xB00000, slots=None, n=4, nv=4, split=1, ws=A + 0xD00000,
          wsb=1 << 20):
    return D.lib.dl_append_step_tiled(ctypes.byref(d), ctypes.byref(s or state()),
                                      ctypes.byref(t or token()), o, slots, n, nv, split, ws,
                                      wsb, None)


def test_tiled_workspace_size():
    d = desc()                                          # B=4, H=2, M=16
    assert D.dl_tiled_workspace_bytes(d, 4) == 4 * 2 * 2 * 15 * 4
    assert D.dl_tiled_workspace_bytes(d, 0) == 0
    assert D.dl_tiled_workspace_bytes(desc(merge_interval=1), 4) == 0
    out = ctypes.c_size_t(0)
    assert D.lib.dl_tiled_workspace_bytes(ctypes.byref(d), 5, ctypes.byref(out)) == D.DL_E_SHAPE
    assert D.lib.dl_tiled_workspace_bytes(ctypes.byref(d), 1, None) == D.DL_E_NULL


def test_tiled_rejections():
    """Every tiled-path check fails before any launch (misaligned output last)."""
    assert tiled(desc(), o=A + 4) == D.DL_E_ALIGN        # everything else valid
    assert tiled(desc(), nv=3) == D.DL_E_UNSUPPORTED
    assert tiled(desc(), nv=1) == D.DL_E_UNSUPPORTED
    assert tiled(desc(state_dtype=D.DL_BF16)) == D.DL_E_DTYPE
    assert tiled(desc(), ws=None) == D.DL_E_NULL          # split replay needs scratch
    assert tiled(desc(), ws=A + 8) == D.DL_E_ALIGN
    assert tiled(desc(), wsb=4 * 2 * 2 * 15 * 4 - 1) == D.DL_E_SHAPE
    assert tiled(desc(), wsb=4 * 2 * 2 * 15 * 4, o=A + 4) == D.DL_E_ALIGN   # exactly enough
    assert tiled(desc(), split=0, ws=None, wsb=0, o=A + 4) == D.DL_E_ALIGN  # fused: no scratch
    assert tiled(desc(merge_interval=1), ws=None, wsb=0, o=A + 4) == D.DL_E_ALIGN
    assert tiled(desc(), n=0, nv=4, ws=None) == D.DL_OK   # n == 0: no-op
    assert tiled(desc(), s=state(len=None)) == D.DL_E_NULL
    assert tiled(desc(), t=token(beta=None)) == D.DL_E_NULL


def test_binding_refuses_to_load_without_the_library(tmp_path):
    """No non-HIP fallback: with the library absent, importing the binding (and the
    decode engine above it) raises ImportError instead of computing anything."""
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    env = dict(os.environ, DELTALOG_LIB=str(tmp_path / "absent" / "libdeltalog.so"))
    for mod in ("paper_2608_15533_amd.deltalog", "paper_2608_15533_amd.decode"):
        r = subprocess.run([sys.executable, "-c", f"import {mod}"], cwd=root, env=env,
                           capture_output=True, text=True, timeout=300)
        assert r.returncode != 0, mod
        assert "ImportError" in r.stderr and "no non-HIP fallback" in r.stderr, r.stderr[-400:]


def noalloc(d, s=None, t=None, o=A + 0xB00000, slots=None, n=4, nv=4):
    return D.lib.dl_append_step_tiled_noalloc(ctypes.byref(d), ctypes.byref(s or state()),
                                              ctypes.byref(t or token()), o, slots, n, nv, None)


def test_noalloc_rejections_before_any_hip_call():
    """The allocation-free entry point runs the tiled step's checks first (misaligned
    output last), then refuses a call whose coefficient scratch would exceed the fixed
    array, all before its first HIP call (the scratch lookup)."""
    assert noalloc(desc(), o=A + 4) == D.DL_E_ALIGN
    assert noalloc(desc(), nv=3) == D.DL_E_UNSUPPORTED
    assert noalloc(desc(state_dtype=D.DL_BF16)) == D.DL_E_DTYPE
    assert noalloc(desc(), s=state(len=None)) == D.DL_E_NULL
    assert noalloc(desc(), t=token(beta=None)) == D.DL_E_NULL
    assert noalloc(desc(), n=0) == D.DL_OK
    assert noalloc(desc(), n=5) == D.DL_E_SHAPE
    # n * H * 2 * (M - 1) * 4 bytes: 2048 x 32 heads at M = 64 needs 31.5 MiB
    big = D.make_desc("gdn", 2048, 32, 128, 128, 64, "bf16")
    assert D.dl_tiled_workspace_bytes(big, 2048) > D.DL_NOALLOC_SCRATCH_BYTES
    assert noalloc(big, n=2048) == D.DL_E_SCRATCH
    # the largest row count that fits is accepted by the size check
    fit = D.DL_NOALLOC_SCRATCH_BYTES // (32 * 2 * 63 * 4)
    assert D.dl_tiled_workspace_bytes(big, fit) <= D.DL_NOALLOC_SCRATCH_BYTES
    assert D.dl_tiled_workspace_bytes(big, fit + 1) > D.DL_NOALLOC_SCRATCH_BYTES
    assert noalloc(big, n=fit + 1, slots=A) == D.DL_E_SCRATCH
    assert "scratch" in D.dl_status_str(D.DL_E_SCRATCH)


def test_noalloc_scratch_size_matches_the_header():
    text = open(HEADER).read()
    assert "#define DL_NOALLOC_SCRATCH_BYTES (4u << 20)" in text
    assert D.DL_NOALLOC_SCRATCH_BYTES == 4 << 20

