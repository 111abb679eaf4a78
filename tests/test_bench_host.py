"""Host-side parts of bench.py (no GPU): the one-GPU contract, the counter-profile
lookup keyed by the kernel-source hash, the algorithmic bytes the roofline divides
by, and the CPU-oracle baseline leg."""

import json
import os
import subprocess
import sys

import pytest

import bench
from paper_2608_15533_amd import traffic as T
from paper_2608_15533_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_every_workload_has_a_positive_algorithmic_step():
    for name, (w, R) in bench.workloads().items():
        assert R >= 1, name
        for L in range(w.M):
            b = T.step_bytes(w.op, w.dk, w.dv, w.M, L, w.in_dtype).total
            assert b > 0, (name, L)
        # the dense state dominates every step: read always, written at the merge
        state = w.dk * w.dv * 4
        assert T.step_bytes(w.op, w.dk, w.dv, w.M, 0, w.in_dtype).total > state
        assert T.step_bytes(w.op, w.dk, w.dv, w.M, w.M - 1, w.in_dtype).total > 2 * state


def test_counter_traffic_follows_the_kernel_source_hash(monkeypatch, tmp_path):
    key = "unit_test_workload"
    prof = tmp_path / "profiles"
    prof.mkdir()
    (prof / f"{key}_hbm_counters.txt").write_text(
        "# header\nTRAFFIC_JSON " + json.dumps({"kernel_source_hash": "abc",
                                                 "step_kernel_bytes_per_launch": 123.0}) + "\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "kernel_source_hash", lambda: "abc")
    val, src = bench.counter_traffic(key)
    assert val == 123.0 and src.endswith(f"{key}_hbm_counters.txt")
    monkeypatch.setattr(bench, "kernel_source_hash", lambda: "changed")
    val, src = bench.counter_traffic(key)
    assert val is None and "changed" in src
    val, src = bench.counter_traffic("no_such_workload")
    assert val is None and src == "no counter profile"


def test_profile_keys():
    assert bench.profile_key("gdn_b64_h32_d128_m16", "f32") == "gdn_b64_h32_d128_m16"
    assert bench.profile_key("gdn_b64_h32_d128_m16", "bf16") == "gdn_b64_h32_d128_m16_bf16state"
    assert bench.profile_key("x", "f32", tiled=2) == "x_tiled2_split"
    assert bench.profile_key("x", "f32", tiled=4, fused_replay=True) == "x_tiled4_fused"


def test_cpu_baseline_leg_reports_the_contract_fields():
    res = bench.cpu_baseline(W.GDN_SMALL, 0.2)
    assert res["kind"] == "oracle" and res["unit"] == "tokens/s"
    assert res["value"] > 0 and res["single_core_value"] > 0
    assert res["cores"] == res["affinity_cores"] == len(os.sched_getaffinity(0))
    assert res["cpu_model"]
    assert "fp64 eager oracle" in res["sample"]


def test_cpu_baseline_of_the_layer_stack_is_a_bounded_one_layer_sample():
    """The 24-layer stack is timed on one layer of 64 of its 256 sequences and reported
    in sequence tokens/s through all layers, the extrapolation stated."""
    res = bench.cpu_baseline(W.GDN_STACK, 0.01)
    assert res["unit"] == "sequence tokens/s (all layers)"
    assert "64 of the 256 sequences" in res["sample"]
    assert "rate / 24 (extrapolated)" in res["sample"]


def test_small_latency_workloads_are_benchmarked():
    wl = bench.workloads()
    for name in ("gdn_b1_h2_d64_m8", "gdn_b1_h2_d64_m8_bf16"):
        w, R = wl[name]
        assert (w.B, w.H, w.dk, w.dv, w.M, w.steps, R) == (1, 2, 64, 64, 8, 64, 1)
    assert wl["gdn_b1_h2_d64_m8"][0].in_dtype == "f32"
    assert wl["gdn_b1_h2_d64_m8_bf16"][0].in_dtype == "bf16"


def test_kernel_source_hash_is_stable():
    assert bench.kernel_source_hash() == bench.kernel_source_hash()
    assert len(bench.kernel_source_hash()) == 16


def test_code_only_drops_comments_and_layout_but_keeps_literals():
    src = ('int a = 1;   // trailing\n/* block\n comment */ const char* s = "// /* kept */";\n'
           "char q = '\\'';\n#define X  2\n")
    assert bench.code_only(src) == ('int a = 1; const char* s = "// /* kept */"; '
                                    "char q = '\\''; #define X 2")


def test_kernel_hash_ignores_comments_but_not_code(monkeypatch, tmp_path):
    import shutil
    shutil.copytree(os.path.join(ROOT, "paper_2608_15533_amd", "csrc"),
                    tmp_path / "paper_2608_15533_amd" / "csrc")
    shutil.copytree(os.path.join(ROOT, "include"), tmp_path / "include")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    h0 = bench.kernel_source_hash()
    f = tmp_path / "paper_2608_15533_amd" / "csrc" / "dl_kernel.hpp"
    text = f.read_text()
    f.write_text("// an added comment\n" + text.replace("\n\n", "\n\n\n", 1))
    assert bench.kernel_source_hash() == h0
    f.write_text(text.replace("#pragma once", "#pragma once\nstatic int dl_changed = 1;", 1))
    assert bench.kernel_source_hash() != h0


def test_kernel_hash_covers_the_build_flags():
    """A library built with other flags (e.g. a -D tuning macro) hashes differently, so a
    counter profile taken on one build is never attached to another."""
    from paper_2608_15533_amd import build as B
    h0 = bench.kernel_source_hash(B.build_flags_string())
    assert bench.kernel_source_hash(B.build_flags_string(["-DDL_XCD_CHUNK=16"])) != h0
    assert bench.kernel_source_hash(" ".join(B.DEVICE_FLAGS) + "  ") == h0   # layout only


def test_library_reports_the_flags_it_was_built_with():
    from paper_2608_15533_amd import build as B
    assert bench.library_build_flags() == B.build_flags_string()
