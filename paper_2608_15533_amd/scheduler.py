"""Host-side decode scheduling for DeltaLog state slots: the slot allocator, a mirror of
every slot's live log length, and the per-step plan (row order, append queue, merge
queue, graph key).  Pure Python with no device or library dependency; the engine that
runs the plans is ``decode.DecodeEngine``.

Sec. 4 describes the serving integration this follows: one state slot per request and
recurrent layer; prefill initialises the dense base while the auxiliary state starts
empty; a reused slot resets only its auxiliary buffers; decode batches are split into an
append queue and a merge queue, and the captured graph for a batch is selected by a key
that encodes the phase.  The live length follows Alg. 1: it grows by one per append and
returns to zero at the step that merges (when the log already holds C = M - 1 entries).
"""

from dataclasses import dataclass

MODES = ("fused", "phased", "phased_concurrent")
ROW_ORDERS = ("slot", "merge_first", "balanced", "interleaved")


def balanced_order(slots, live):
    """Rows ordered by live length, longest first (the slots that merge in this step
    first), ties in slot order.  The kernel deals runs of 32 consecutive (row, head)
    workgroups to the eight XCDs in turn, so with 32 heads per row, row r runs on XCD
    r mod 8: dealing the rows in this order gives every XCD the same mix of merges and
    of log lengths, instead of whatever mix the slot ids happen to have."""
    return tuple(sorted(slots, key=lambda s: (-live[s], s)))


def interleaved_order(slots, live, xcds=8):
    """The balanced order's share for each XCD (every xcds-th row of it), but each XCD's
    rows taken in bit-reversed order over its dispatch sequence, so the merging and the
    long-log rows are spread over the launch instead of all starting first."""
    bal = balanced_order(slots, live)
    n = len(bal)
    per = -(-n // xcds)                       # rows per XCD (the last round may be short)
    bits = max(1, (per - 1).bit_length())
    rev = sorted(range(per), key=lambda t: int(format(t, f"0{bits}b")[::-1], 2))
    out = []
    for t in range(per):                      # dispatch round t
        for x in range(xcds):                 # row t * xcds + x runs on XCD x
            i = x + xcds * rev[t]
            if i < n:
                out.append(bal[i])
    # rounds where rev[t] pointed past the end of a short list are refilled in order
    seen = set(out)
    out += [s for s in bal if s not in seen]
    return tuple(out)


class SlotError(RuntimeError):
    pass


@dataclass(frozen=True)
class StepPlan:
    """One decode step: the row order of the launch(es), the append queue and the merge
    queue, and the graph key.  Phased modes order the append queue first, then the
    merge queue.  The fused mode (one launch; the device picks each slot's phase) keeps
    slot order (``row_order="slot"``), puts the merge queue first (``"merge_first"``) so
    the longer merging workgroups are dispatched before the appending ones, or orders the
    rows by live length, longest first (``"balanced"``, see ``balanced_order``)."""
    order: tuple
    append_slots: tuple
    merge_slots: tuple
    key: tuple

    @property
    def n(self):
        return len(self.order)

    @property
    def n_append(self):
        return len(self.append_slots)

    @property
    def n_merge(self):
        return len(self.merge_slots)

    def row_of(self, slot):
        return self.order.index(slot)


class DecodeScheduler:
    """Slot allocator and per-step planner for B slots with merge interval M."""

    def __init__(self, num_slots, merge_interval, mode="fused", merge_first=False,
                 row_order=None):
        if mode not in MODES:
            raise ValueError(f"mode must be one of {MODES}")
        if merge_interval < 1:
            raise ValueError("merge interval must be >= 1")
        row_order = row_order or ("merge_first" if merge_first else "slot")
        if row_order not in ROW_ORDERS:
            raise ValueError(f"row order must be one of {ROW_ORDERS}")
        self.B = num_slots
        self.C = merge_interval - 1
        self.mode = mode
        self.row_order = row_order
        self.merge_first = row_order == "merge_first"
        self.live = [0] * num_slots                 # host mirror of each slot's L
        self.active = []                            # admission order
        self._free = list(range(num_slots))[::-1]   # lowest slot id handed out first

    @property
    def free_slots(self):
        return len(self._free)

    def admit(self):
        if not self._free:
            raise SlotError("no free state slot")
        slot = self._free.pop()
        self.live[slot] = 0
        self.active.append(slot)
        return slot

    def release(self, slot):
        if slot not in self.active:
            raise SlotError(f"slot {slot} is not active")
        self.active.remove(slot)
        self.live[slot] = 0
        self._free.append(slot)

    def plan(self):
        """The next step's row order and its graph key."""
        act = sorted(self.active)
        app = tuple(s for s in act if self.live[s] < self.C)
        mrg = tuple(s for s in act if self.live[s] >= self.C)
        if self.mode == "fused":
            if self.row_order == "balanced":
                order = balanced_order(act, self.live)
            elif self.row_order == "interleaved":
                order = interleaved_order(act, self.live)
            else:
                order = mrg + app if self.merge_first else tuple(act)
            return StepPlan(order, app, mrg, ("fused", len(act)))
        return StepPlan(app + mrg, app, mrg, (self.mode, len(app), len(mrg)))

    def commit(self, plan):
        """Advance the mirror after the plan's step ran (Alg. 1: append, or merge and
        reset when the log was full)."""
        for s in plan.order:
            self.live[s] = 0 if self.live[s] >= self.C else self.live[s] + 1

    def flushed(self, slot):
        self.live[slot] = 0
