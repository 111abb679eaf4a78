"""GPU tests of the decode loop (slot lifecycle, phase scheduling, graph replay).

A scripted serving trace admits requests at different steps (so their logs are
staggered and merges land on different steps), releases one with a flush (its
materialised state is checked), releases another without one, and reuses both freed
slots for new requests.  Every request's token stream and prefill state are seeded and
per request; the fp64 oracle follows each request through every layer.

Bars: relative Frobenius error <= 1e-4 against the oracle for every output row and for
flushed states; bitwise equality between scheduling modes and between graph replay and
direct launches (the same kernels on the same inputs)."""

import numpy as np
import pytest
import torch

from paper_2608_15533_amd import workloads as W

from gpu_harness import TOL_F32_STATE, log, oracle_step, rel

pytestmark = pytest.mark.gpu

LAYERS = 2
SLOTS = 4
STEPS = 16
M = 4
# step -> list of actions; ("admit", request) / ("release", request, flush)
TRACE = {
    0: [("admit", 0), ("admit", 1), ("admit", 2)],
    3: [("admit", 3)],
    5: [("release", 1, True)],
    6: [("admit", 4)],
    9: [("release", 0, False)],
    10: [("admit", 5)],
    13: [("release", 3, True), ("admit", 6)],
}
SHAPES = {"gdn": (4, 128, 128), "kda": (4, 128, 128), "rwkv6": (4, 64, 64),
          "linattn": (4, 128, 128), "retnet": (4, 64, 64), "gla": (4, 128, 64)}


def _request(op, r):
    """One request: a single-sequence workload with its own seed (cfg field)."""
    H, dk, dv = SHAPES[op]
    return W.Workload(f"req{r}", 100 + r, op, 1, H, dk, dv, M, STEPS, in_dtype="bf16")


def _D():
    from paper_2608_15533_amd import decode, deltalog
    return decode, deltalog


def run_trace(op, mode, graphs, oracle=False):
    """Drive the trace; returns (outputs per (step, request, layer), flushed states,
    engine).  With ``oracle`` the fp64 oracle follows every request and the worst
    errors are asserted."""
    decode, dl = _D()
    H, dk, dv = SHAPES[op]
    desc = dl.make_desc(op, SLOTS, H, dk, dv, M, "bf16")
    eng = decode.DecodeEngine(desc, LAYERS, mode=mode, graphs=graphs)
    shared_u = W.bonus(_request(op, 0), 0) if op == "rwkv6" else None
    if shared_u is not None:
        for layer in range(LAYERS):
            eng.inputs[layer].u.copy_(torch.from_numpy(W.bonus(_request(op, 0), layer)))
    slot_of, t_of, ref = {}, {}, {}
    outs, saved = {}, {}
    err_o = err_s = 0.0
    for t in range(STEPS):
        for act in TRACE.get(t, []):
            r = act[1]
            if act[0] == "admit":
                w = _request(op, r)
                pre = [torch.from_numpy(W.initial_state(w, layer)[0]).cuda()
                       for layer in range(LAYERS)]
                slot_of[r] = eng.admit(pre)
                t_of[r] = 0
                ref[r] = [W.initial_state(w, layer).astype(np.float64)
                          for layer in range(LAYERS)]
            else:
                flush = act[2]
                got = eng.release(slot_of[r], flush=flush)
                if flush:
                    saved[r] = [g.float().cpu().numpy() for g in got]
                    if oracle:
                        for layer in range(LAYERS):
                            err_s = max(err_s, rel(saved[r][layer][None], ref[r][layer]))
                del slot_of[r]
        plan = eng.schedule()
        live = sorted(slot_of, key=lambda r: plan.row_of(slot_of[r]))
        xs = {}
        for layer in range(LAYERS):
            rows, parts = [], {k: [] for k in ("q", "k", "v", "lam", "beta")}
            for r in live:
                x = W.step_inputs(_request(op, r), t_of[r], layer)
                xs[(r, layer)] = x
                rows.append(plan.row_of(slot_of[r]))
                for k in parts:
                    if x[k] is not None:
                        parts[k].append(torch.from_numpy(x[k]))
            cat = {k: (torch.cat(v) if v else None) for k, v in parts.items()}
            eng.inputs[layer].write(rows, cat["q"], cat["k"], cat["v"], cat["lam"], cat["beta"])
        eng.step()
        torch.cuda.synchronize()
        for layer in range(LAYERS):
            for r in live:
                o = eng.output(layer, slot_of[r], plan).cpu().numpy()
                outs[(t, r, layer)] = o
                if oracle:
                    x = {k: (None if a is None else a.astype(np.float64))
                         for k, a in xs[(r, layer)].items()}
                    u = None if shared_u is None else W.bonus(_request(op, 0), layer)
                    S_new, o_ref = oracle_step(op, ref[r][layer], x, u)
                    ref[r][layer] = S_new
                    err_o = max(err_o, rel(o[None], o_ref))
        for r in live:
            t_of[r] += 1
    # final flush of everything still active: materialised state vs oracle
    for r in sorted(slot_of):
        got = eng.flush(slot_of[r])
        saved[r] = [g.float().cpu().numpy() for g in got]
        if oracle:
            for layer in range(LAYERS):
                err_s = max(err_s, rel(saved[r][layer][None], ref[r][layer]))
    torch.cuda.synchronize()
    assert eng.error_words() == [0] * LAYERS
    if oracle:
        log(f"decode trace {op} {mode} graphs={graphs}: max out err {err_o:.2e}, "
            f"flushed state err {err_s:.2e}, graph keys {eng.graph_keys}, "
            f"replays {eng.replays}, direct {eng.direct_steps}")
        assert err_o <= TOL_F32_STATE
        assert err_s <= TOL_F32_STATE
    return outs, saved, eng


@pytest.mark.parametrize("op", list(SHAPES))
@pytest.mark.parametrize("mode", ["fused", "phased", "phased_concurrent"])
def test_trace_against_oracle(op, mode):
    _, _, eng = run_trace(op, mode, graphs=True, oracle=True)
    assert eng.replays > 0


@pytest.mark.parametrize("op", ["gdn", "rwkv6", "linattn"])
def test_modes_and_graphs_bitwise_equal(op):
    """Every scheduling mode, with and without graphs, gives bit-identical outputs and
    flushed states: the same kernel arithmetic on the same rows."""
    base_o, base_s, _ = run_trace(op, "fused", graphs=False)
    for mode in ("fused", "phased", "phased_concurrent"):
        for graphs in (True, False):
            if (mode, graphs) == ("fused", False):
                continue
            o, s, _ = run_trace(op, mode, graphs)
            assert o.keys() == base_o.keys()
            for key in base_o:
                assert np.array_equal(o[key], base_o[key]), (mode, graphs, key)
            for r in base_s:
                for layer in range(LAYERS):
                    assert np.array_equal(s[r][layer], base_s[r][layer]), (mode, graphs, r)


def test_uniform_batch_uses_one_append_and_one_merge_graph():
    """Requests admitted together: the phased engine captures exactly two graphs (the
    append graph and the merge graph of that batch descriptor) and replays them, with
    host work and synchronisations between replays."""
    decode, dl = _D()
    desc = dl.make_desc("gdn", 3, 2, 64, 64, M, "bf16")
    eng = decode.DecodeEngine(desc, LAYERS, mode="phased", graphs=True)
    ref = decode.DecodeEngine(desc, LAYERS, mode="fused", graphs=False)
    w = W.Workload("uniform", 120, "gdn", 3, 2, 64, 64, M, 3 * M, in_dtype="bf16")
    for e in (eng, ref):
        for b in range(3):
            e.admit([torch.from_numpy(W.initial_state(w, layer)[b]).cuda()
                     for layer in range(LAYERS)])
    for t in range(3 * M):
        for e in (eng, ref):
            plan = e.schedule()
            for layer in range(LAYERS):
                x = W.step_inputs(w, t, layer)
                rows = [plan.row_of(b) for b in range(3)]
                e.inputs[layer].write(rows, *(torch.from_numpy(x[k])
                                              for k in ("q", "k", "v", "lam", "beta")))
            e.step()
        torch.cuda.synchronize()
        for layer in range(LAYERS):
            assert torch.equal(eng.outputs[layer][:3][torch.tensor(
                [plan.row_of(b) for b in range(3)], device="cuda")],
                ref.outputs[layer][:3]), (t, layer)
        _ = eng.states[0].S.sum().item()       # unrelated device work between replays
    assert eng.graph_keys == [("phased", 0, 3), ("phased", 3, 0)]
    assert eng.direct_steps == 2 and eng.replays == 3 * M - 2
    for layer in range(LAYERS):
        assert torch.equal(eng.states[layer].S, ref.states[layer].S)


def test_reused_slot_matches_fresh_slot_bitwise():
    """A slot released with a non-empty log and re-admitted behaves exactly like a slot
    that was never used: admission resets its auxiliary state."""
    decode, dl = _D()
    desc = dl.make_desc("kda", 2, 2, 128, 128, 8, "bf16")
    w = W.Workload("reuse", 121, "kda", 2, 2, 128, 128, 8, 12, in_dtype="bf16")
    pre = [torch.from_numpy(W.initial_state(w, layer)[1]).cuda() for layer in range(LAYERS)]

    def drive(eng, slot, steps, t0):
        res = []
        for t in range(t0, t0 + steps):
            plan = eng.schedule()
            for layer in range(LAYERS):
                x = W.select_rows(W.step_inputs(w, t, layer), np.array([1]))
                eng.inputs[layer].write([plan.row_of(slot)], *(torch.from_numpy(x[k])
                                        for k in ("q", "k", "v", "lam", "beta")))
            eng.step()
            res.append([eng.output(layer, slot, plan).clone() for layer in range(LAYERS)])
        return res

    used = decode.DecodeEngine(desc, LAYERS, mode="fused")
    s0 = used.admit(pre)
    drive(used, s0, 5, 100)                  # L = 5 with a non-zero cumulative decay
    used.release(s0)                         # no flush: the stale log stays behind
    s1 = used.admit(pre)
    assert s1 == s0
    fresh = decode.DecodeEngine(desc, LAYERS, mode="fused")
    f0 = fresh.admit(pre)
    a = drive(used, s1, 12, 0)
    b = drive(fresh, f0, 12, 0)
    torch.cuda.synchronize()
    for x, y in zip(a, b):
        for layer in range(LAYERS):
            assert torch.equal(x[layer], y[layer])
    for layer in range(LAYERS):
        assert torch.equal(used.states[layer].S[s1], fresh.states[layer].S[f0])
