"""Decode loop around the library: state slots for a stack of recurrent layers, a slot
allocator, and graph-captured decode steps (the serving-side integration of Sec. 4).

Host-side orchestration only: every step of the state update runs in the HIP kernels
behind the C ABI.  Two parts:

* ``DecodeScheduler`` (``scheduler.py``) -- pure host logic, no device: the slot
  allocator (admit / release / reuse), a mirror of every slot's live log length, and the
  per-step plan (which slots run, in which row order, split into an append queue and a
  merge queue).
* ``DecodeEngine`` -- owns the per-layer ``DeltaLogState`` buffers, fixed token-input and
  output buffers, a device slot list, and a cache of captured HIP graphs keyed by the
  plan's batch descriptor.

Scheduling policies (``mode``):

``"fused"``
    One ``dl_append_step`` launch per layer over all active slots.  Every workgroup
    takes the append or merge branch of Alg. 1 for its own slot, so a batch whose slots
    sit at different points of their cycles is one launch, and one captured graph per
    batch size covers both phases.  ``row_order`` (scheduler) picks the rows' order:
    slot order; ``"merge_first"``, the rows of slots that merge in the step first, so
    the longer merging workgroups start before the appending ones; or ``"balanced"``,
    rows by live length, longest first.  The kernel deals runs of consecutive heads to
    the eight XCDs in turn, so the last two spread the merges evenly over the XCDs
    whatever slot ids the merging sequences hold.
``"phased"``
    The paper's phase-specialised scheduling (Sec. 4: an append queue and a merge queue,
    append and merge graphs selected by a key that encodes the phase).  Rows are ordered
    append queue first, then merge queue; per layer the append queue runs
    ``dl_append_step`` and the merge queue ``dl_merge`` with the token.  A batch whose
    slots are all in one phase gets the paper's append graph or merge graph.
``"phased_concurrent"``
    As ``"phased"``, but the merge launches go on a second stream, forked from and joined
    back to the caller's stream, so the small merge launch overlaps the append launch.

Correctness does not depend on the host's live-length mirror: ``dl_append_step`` merges
a slot that is full, and ``dl_merge`` with a token is Eq. 6 at any live length.  The
mirror only decides which launch a slot goes to.

Graphs: the first step with a new key runs its launches directly (which also loads the
kernels) and records the same launches into a graph for the key; later steps with that
key replay it.  A graph holds kernel launches only (no memset or copy nodes); the slot
list a graph reads is a fixed device buffer that the engine refreshes with one small
host-to-device copy, outside the graph, when the plan's row order changes.

Slot lifecycle (Sec. 4): ``admit`` writes the prefill state into the slot's dense base
and resets only the slot's live length (which also restarts the cumulative log-decay;
log rows past the live length are never read).  ``release`` frees the slot, optionally
flushing its log into the base first so the materialised state can be saved.
"""

import torch

from . import deltalog as D
from .scheduler import MODES, DecodeScheduler, SlotError, StepPlan  # noqa: F401


class LayerInputs:
    """Fixed device buffers for one layer's token rows (capacity = all slots)."""

    def __init__(self, desc, device):
        n, H, dk, dv = desc.num_slots, desc.heads, desc.dk, desc.dv
        it = torch.bfloat16 if desc.in_dtype == D.DL_BF16 else torch.float32
        f32 = dict(dtype=torch.float32, device=device)
        self.desc = desc
        self.q = torch.zeros((n, H, dk), dtype=it, device=device)
        self.k = torch.zeros((n, H, dk), dtype=it, device=device)
        self.v = torch.zeros((n, H, dv), dtype=it, device=device)
        dl = D.decay_width(desc)
        self.lam = (None if dl == 0 else
                    torch.zeros((n, H) if dl == 1 else (n, H, dl), **f32))
        self.beta = torch.zeros((n, H), **f32) if desc.op in D.DELTA_OP_IDS else None
        self.u = torch.zeros((H, dk), **f32) if desc.op == D.DL_OP_RWKV6 else None
        self._tokens = {}

    def token(self, r0, r1):
        """dl_token over rows [r0, r1) (contiguous views of the fixed buffers; cached,
        since the buffers never move)."""
        tok = self._tokens.get((r0, r1))
        if tok is None:
            tok = D.Token(self.desc, r1 - r0, self.q[r0:r1], self.k[r0:r1], self.v[r0:r1],
                          None if self.lam is None else self.lam[r0:r1],
                          None if self.beta is None else self.beta[r0:r1], self.u)
            self._tokens[(r0, r1)] = tok
        return tok

    def write(self, rows, q, k, v, lam, beta=None):
        """Write token rows ``rows`` (row indices of the current plan)."""
        idx = torch.as_tensor(rows, dtype=torch.long, device=self.q.device)
        self.q[idx] = q.to(self.q.device, self.q.dtype)
        self.k[idx] = k.to(self.k.device, self.k.dtype)
        self.v[idx] = v.to(self.v.device, self.v.dtype)
        if self.lam is not None:
            self.lam[idx] = lam.to(self.lam.device, torch.float32)
        if self.beta is not None:
            self.beta[idx] = beta.to(self.beta.device, torch.float32)


class DecodeEngine:
    """``layers`` recurrent layers, each a DeltaLog state over ``desc.num_slots`` slots,
    stepped one decode token at a time under a scheduling ``mode``."""

    def __init__(self, desc, layers, mode="fused", graphs=True, device="cuda",
                 merge_first=False, row_order=None):
        if layers < 1:
            raise ValueError("need at least one layer")
        self.desc = desc
        self.layers = layers
        self.graphs = graphs
        self.device = device
        self.sched = DecodeScheduler(desc.num_slots, desc.merge_interval, mode, merge_first,
                                     row_order)
        self.states = [D.DeltaLogState(desc, device=device) for _ in range(layers)]
        self.inputs = [LayerInputs(desc, device) for _ in range(layers)]
        self.outputs = [torch.zeros((desc.num_slots, desc.heads, desc.dv),
                                    dtype=torch.float32, device=device)
                        for _ in range(layers)]
        self.slot_list = torch.zeros((desc.num_slots,), dtype=torch.int32, device=device)
        self._list_order = None
        self._graph_cache = {}
        self._side = torch.cuda.Stream(device=device) if mode == "phased_concurrent" else None
        self.plan = None
        self.replays = 0
        self.direct_steps = 0

    @property
    def mode(self):
        return self.sched.mode

    # ------------------------------------------------------------- slot lifecycle
    def admit(self, prefill=None):
        """Take a free slot; write ``prefill`` (one [H, dk, dv] tensor per layer, or
        None for a zero state) into its dense base and start an empty log."""
        if prefill is not None and len(prefill) != self.layers:
            raise ValueError("prefill needs one state per layer")
        slot = self.sched.admit()
        for layer, st in enumerate(self.states):
            if prefill is None:
                st.S[slot].zero_()
            else:
                st.S[slot].copy_(prefill[layer])
            st.len[slot].zero_()
        self.plan = None
        return slot

    def release(self, slot, flush=False):
        """Free an active slot; with ``flush`` fold its log into the base first and
        return the materialised per-layer states ([H, dk, dv] each)."""
        if slot not in self.sched.active:
            raise SlotError(f"slot {slot} is not active")
        saved = None
        if flush:
            saved = self.flush(slot)
        self.sched.release(slot)
        self.plan = None
        return saved

    def flush(self, slot):
        """Fold the slot's log into its base (``dl_merge`` without a token) in every
        layer; returns copies of the materialised bases."""
        sl = torch.tensor([slot], dtype=torch.int32, device=self.device)
        for st in self.states:
            D.dl_merge(self.desc, st, slots=sl)
        self.sched.flushed(slot)
        return [st.S[slot].clone() for st in self.states]

    def readout(self, slot, q_per_layer):
        """q^T S (Eq. 7) of one slot in every layer, without changing any state."""
        sl = torch.tensor([slot], dtype=torch.int32, device=self.device)
        outs = []
        for st, q in zip(self.states, q_per_layer):
            o = torch.empty((1, self.desc.heads, self.desc.dv), dtype=torch.float32,
                            device=self.device)
            D.dl_readout(self.desc, st, q.reshape(1, self.desc.heads, self.desc.dk), o,
                         slots=sl)
            outs.append(o[0])
        return outs

    # ------------------------------------------------------------- decoding
    def schedule(self):
        """Plan the next step.  Returns the plan; token rows for slot ``s`` go to row
        ``plan.row_of(s)`` of every layer's inputs, and its outputs come back there."""
        self.plan = self.sched.plan()
        if self.plan.order != self._list_order and self.plan.n:
            host = torch.tensor(self.plan.order, dtype=torch.int32).pin_memory()
            self.slot_list[: self.plan.n].copy_(host, non_blocking=True)
            self._list_order = self.plan.order
        return self.plan

    def _launch(self, plan, stream):
        n, na, nm = plan.n, plan.n_append, plan.n_merge
        desc = self.desc
        if self.mode == "fused":
            for layer in range(self.layers):
                D.dl_append_step(desc, self.states[layer], self.inputs[layer].token(0, n),
                                 self.outputs[layer][:n], slots=self.slot_list[:n],
                                 stream=stream)
            return
        side = self._side
        if side is not None and nm and na:
            side.wait_stream(stream)
        for layer in range(self.layers):
            st, inp, out = self.states[layer], self.inputs[layer], self.outputs[layer]
            if na:
                D.dl_append_step(desc, st, inp.token(0, na), out[:na],
                                 slots=self.slot_list[:na], stream=stream)
            if nm:
                ms = side if (side is not None and na) else stream
                D.dl_merge(desc, st, inp.token(na, n), out[na:n],
                           slots=self.slot_list[na:n], stream=ms)
        if side is not None and nm and na:
            stream.wait_stream(side)

    def step(self):
        """Run the planned step (``schedule()`` first) through every layer."""
        plan = self.plan if self.plan is not None else self.schedule()
        if plan.n:
            cur = torch.cuda.current_stream(self.device)
            g = self._graph_cache.get(plan.key) if self.graphs else None
            if g is not None:
                g.replay()
                self.replays += 1
            else:
                self._launch(plan, cur)
                self.direct_steps += 1
                if self.graphs:
                    self._graph_cache[plan.key] = self._capture(plan)
        self.sched.commit(plan)
        self.plan = None
        return plan

    def _capture(self, plan):
        g = torch.cuda.CUDAGraph()
        s = torch.cuda.Stream(device=self.device)
        s.wait_stream(torch.cuda.current_stream(self.device))
        with torch.cuda.graph(g, stream=s):
            self._launch(plan, s)
        torch.cuda.current_stream(self.device).wait_stream(s)
        return g

    @property
    def graph_keys(self):
        return sorted(self._graph_cache)

    def output(self, layer, slot, plan):
        """Output row of ``slot`` in ``layer`` for a step that ran ``plan``."""
        return self.outputs[layer][plan.row_of(slot)]

    def error_words(self):
        return [int(st.err.item()) for st in self.states]
