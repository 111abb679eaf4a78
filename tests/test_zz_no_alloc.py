"""The allocation-free entry point, dl_append_step_tiled_noalloc, through the C ABI: its
split-replay coefficients live in the library's fixed per-GPU scratch array instead of
a caller workspace.  Each call must give exactly what dl_append_step_tiled gives with a
workspace (same kernels, same coefficients): outputs and every state buffer bit for bit,
over consecutive calls that shrink (the scratch keeps the previous call's contents)."""

import numpy as np
import pytest
import torch

from paper_2608_15533_amd import workloads as W

from gpu_harness import D, log, to_dev, token

pytestmark = pytest.mark.gpu

WL = {"gdn": W.GDN_B64, "kda": W.KDA_B128, "rwkv6": W.RWKV6_B128}


def _host(st):
    return {k: (v.float() if v.dtype == torch.bfloat16 else v).cpu().numpy().copy()
            for k, v in st.buffers().items() if v is not None}


@pytest.mark.parametrize("op", list(WL))
def test_noalloc_equals_the_workspace_entry_point(op):
    dl = D()
    w = WL[op].with_(B=6)
    M = 8
    desc = dl.make_desc(op, w.B, w.H, w.dk, w.dv, M, w.in_dtype)
    S0 = to_dev(W.initial_state(w), torch.float32)
    u = W.bonus(w)
    st_ws = dl.DeltaLogState(desc, S0)
    st_na = dl.DeltaLogState(desc, S0)
    ws = dl.tiled_workspace(desc, w.B)
    # five identical untiled steps fill every log to L = 5, so the calls below replay
    # live entries through the prepared coefficients
    for t in range(5):
        tok = token(desc, W.step_inputs(w, t), u)
        for st in (st_ws, st_na):
            o = torch.empty((w.B, w.H, w.dv), dtype=torch.float32, device="cuda")
            dl.dl_append_step(desc, st, tok, o)
    # call 1: all 6 slots, 4 value tiles; call 2: a smaller input (3 listed slots,
    # 2 value tiles); call 3: all slots again, the listed ones now merging
    calls = [(None, 4), ([4, 1, 2], 2), (None, 4)]
    for c, (rows, nv) in enumerate(calls):
        x = W.step_inputs(w, 5 + c)
        tok = token(desc, x, u, rows=rows)
        n = w.B if rows is None else len(rows)
        sl = None if rows is None else torch.tensor(rows, dtype=torch.int32, device="cuda")
        o_ws = torch.full((n, w.H, w.dv), float("nan"), dtype=torch.float32, device="cuda")
        o_na = torch.full((n, w.H, w.dv), float("nan"), dtype=torch.float32, device="cuda")
        log(f"noalloc {op}: call {c}, n={n}, value tiles {nv}")
        dl.dl_append_step_tiled(desc, st_ws, tok, o_ws, slots=sl, value_tiles=nv,
                                split_replay=True, workspace=ws)
        dl.dl_append_step_tiled_noalloc(desc, st_na, tok, o_na, slots=sl, value_tiles=nv)
        torch.cuda.synchronize()
        assert np.isfinite(o_na.cpu().numpy()).all()
        np.testing.assert_array_equal(o_na.cpu().numpy(), o_ws.cpu().numpy(),
                                      err_msg=f"output, call {c}")
        b_ws, b_na = _host(st_ws), _host(st_na)
        for k in b_ws:
            np.testing.assert_array_equal(b_na[k], b_ws[k], err_msg=f"{k}, call {c}")
        assert int(st_na.err.item()) == 0
    lens = st_na.len.cpu().numpy()
    assert (lens[[1, 2, 4]] == 0).all() and (lens[[0, 3, 5]] == 7).all()   # merged / appended
