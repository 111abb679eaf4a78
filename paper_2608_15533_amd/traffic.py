"""Algorithmic HBM bytes of one decode step per (slot, head) -- the traffic model of Sec. 3.2.

This is host-side bookkeeping for measurement (roofline fractions, write-traffic
ratios); no kernel arithmetic lives here.  It restates Eqs. 8-10 per head and per
phase, with the precisions the library uses:

* ``T_common``: the current-token inputs both schemes read -- q (or r), k, v in the
  activation dtype, beta (fp32, delta rule only) and the step log-decay lambda (fp32,
  one value per head or one per key; none for linear attention, which has no decay).
  The RWKV6 bonus u is a per-head parameter shared by every slot and is not counted (as
  in the paper's model).
* dense state ``C_state``: p_S * dk * dv bytes per head (p_S = 4 for fp32 state, 2 for
  bf16 state).
* one log entry ``C_entry``: p_K dk + p_U dv + 4 d_lambda bytes (Eq. 9), with K_log in the
  activation dtype and U_log fp32 for the delta rule (GDN/KDA: computed values), the
  activation dtype for the others (exact copies of v).
* cumulative log-decay ``C_decay``: 4 d_lambda bytes, read and written every DeltaLog step
  in the paper's representation (d_lambda = 0 for linear attention: no decay, no
  snapshots).  This library stores no such buffer: the cumulative log-decay equals the
  newest snapshot, which the replay reads anyway, so its steps move no separate
  ``C_decay`` bytes (``stored_ell=False``, the default, is the library's layout;
  ``True`` the paper's).
* the output o: fp32, dv values.
* live-length and index metadata are omitted as lower-order, as the paper does.

Per phase (one head, one token):

    eager        read  T_common + C_state                write C_state + o
    append at L  read  T_common + C_state + C_decay + L C_entry
                 write C_entry + C_decay + o
    merge at L   read  T_common + C_state + C_decay + L C_entry
                 write C_state + C_decay + o

(C_decay counted only in the paper's representation, ``stored_ell=True``.)
"""

from dataclasses import dataclass

DTYPE_BYTES = {"bf16": 2, "f32": 4}
DELTA_OPS = ("gdn", "kda")
PER_KEY_OPS = ("kda", "rwkv6", "gla")


@dataclass(frozen=True)
class HeadTraffic:
    read: int
    write: int

    @property
    def total(self):
        return self.read + self.write


def _sizes(op, dk, dv, in_dtype, state_dtype="f32"):
    pin = DTYPE_BYTES[in_dtype]
    delta = op in DELTA_OPS
    dl = 0 if op == "linattn" else (dk if op in PER_KEY_OPS else 1)
    common = pin * (2 * dk + dv) + 4 * dl + (4 if delta else 0)
    state = DTYPE_BYTES[state_dtype] * dk * dv
    p_u = 4 if delta else pin
    entry = pin * dk + p_u * dv + 4 * dl
    decay = 4 * dl
    out = 4 * dv
    return common, state, entry, decay, out


def eager_bytes(op, dk, dv, in_dtype="bf16", state_dtype="f32"):
    """Bytes one eager dense step moves for one head (Eq. 8 plus the output)."""
    common, state, _, _, out = _sizes(op, dk, dv, in_dtype, state_dtype)
    return HeadTraffic(read=common + state, write=state + out)


def _ell(decay, stored_ell):
    return decay if stored_ell else 0


def append_bytes(op, dk, dv, L, in_dtype="bf16", state_dtype="f32", stored_ell=False):
    """Bytes of a DeltaLog append step taken at live length L."""
    common, state, entry, decay, out = _sizes(op, dk, dv, in_dtype, state_dtype)
    ell = _ell(decay, stored_ell)
    return HeadTraffic(read=common + state + ell + L * entry, write=entry + ell + out)


def merge_bytes(op, dk, dv, L, in_dtype="bf16", state_dtype="f32", stored_ell=False):
    """Bytes of a DeltaLog merge step that folds L live entries (plus the token)."""
    common, state, entry, decay, out = _sizes(op, dk, dv, in_dtype, state_dtype)
    ell = _ell(decay, stored_ell)
    return HeadTraffic(read=common + state + ell + L * entry, write=state + ell + out)


def step_bytes(op, dk, dv, M, L, in_dtype="bf16", state_dtype="f32", stored_ell=False):
    """Bytes of the Alg. 1 step at live length L: append if L < M-1, else merge."""
    if L < M - 1:
        return append_bytes(op, dk, dv, L, in_dtype, state_dtype, stored_ell)
    return merge_bytes(op, dk, dv, L, in_dtype, state_dtype, stored_ell)


def cycle_bytes(op, dk, dv, M, in_dtype="bf16", state_dtype="f32", stored_ell=False):
    """Total bytes of one full cycle (M-1 appends at L = 0..M-2, one merge at L = M-1)."""
    r = w = 0
    for L in range(M):
        t = step_bytes(op, dk, dv, M, L, in_dtype, state_dtype, stored_ell)
        r += t.read
        w += t.write
    return HeadTraffic(read=r, write=w)


def amortized_bytes_per_token(op, dk, dv, M, in_dtype="bf16", state_dtype="f32",
                              stored_ell=False):
    """Average bytes per head-token over a cycle (the Eq. 10 quantity, plus outputs)."""
    c = cycle_bytes(op, dk, dv, M, in_dtype, state_dtype, stored_ell)
    return c.total / M


def state_write_ratio(op, dk, dv, M, in_dtype="bf16", state_dtype="f32", live_length_bytes=0,
                      stored_ell=True):
    """Eager / DeltaLog state-write bytes per token, outputs excluded.  With the defaults
    this is the bound of Eq. 9, M / (1 + eps), in the paper's representation (the
    cumulative log-decay written every step).  ``live_length_bytes`` adds the per-step
    write of the live length (metadata the paper's model omits; 4 for the int32 length
    this library keeps per slot and head); ``stored_ell=False`` leaves out the
    cumulative log-decay, which this library does not store."""
    _, state, entry, decay, _ = _sizes(op, dk, dv, in_dtype, state_dtype)
    ell = _ell(decay, stored_ell)
    dl_writes = (state + (M - 1) * entry + M * (ell + live_length_bytes)) / M
    return state / dl_writes


def library_state_write_ratio(op, dk, dv, M, in_dtype="bf16", state_dtype="f32"):
    """The write ratio this library's layout implies: the log entries and the 4-byte live
    length of every head-step (no cumulative log-decay buffer)."""
    return state_write_ratio(op, dk, dv, M, in_dtype, state_dtype, live_length_bytes=4,
                             stored_ell=False)


def byte_optimal_merge_interval(op, dk, dv, in_dtype="bf16", state_dtype="f32", max_M=64):
    """The merge interval that minimises the amortised bytes per token (Eq. 10's
    trade-off: the dense write amortised over M against the growing replay)."""
    return min(range(1, max_M + 1),
               key=lambda M: amortized_bytes_per_token(op, dk, dv, M, in_dtype, state_dtype))
