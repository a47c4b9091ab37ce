"""The benchmark's command-line contract that holds without a GPU: one GPU
only, the oracle's CPU baseline record, the validation of timed launches and
the host side of the measurement helpers."""

import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def run_bench(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], cwd=ROOT,
                          capture_output=True, text=True, timeout=300)


@pytest.mark.parametrize("n", ["2", "8"])
def test_more_than_one_gpu_is_refused(n):
    r = run_bench("--gpus", n)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr and r.stdout == ""


def test_cpu_baseline_record():
    """The oracle's baseline on a sample of a high-load-shaped call (here a
    small stand-in), scaled to one call, with the host's core count and CPU
    model."""
    sys.path.insert(0, ROOT)
    import bench
    from workloads import custom_shape, make_inputs
    rec = bench.cpu_baseline_highload(make_inputs(custom_shape(32, 16, 2, 64), seed=1), 0.2)
    assert rec["kind"] == "oracle" and rec["unit"] == "us/call"
    assert rec["value"] > 0 and rec["cores"] == len(os.sched_getaffinity(0))
    assert isinstance(rec["cpu_model"], str)
    assert "8 of the 32 sequences" in rec["sample"] and "scaled to one call" in rec["sample"]


def test_validation_rejects_a_wrong_output():
    """Every timed launch is checked against the oracle before it is timed
    (the paper's harness rejects invalid candidates, Section 3.2): an output
    off by a little more than the bar, or not finite, is recorded as
    invalid; the oracle's own output rounded to bf16 passes."""
    sys.path.insert(0, ROOT)
    import numpy as np
    import torch
    import bench
    from oracle import decode_attention
    from workloads import custom_shape, f32_to_bf16_bits, make_inputs
    inp = make_inputs(custom_shape(3, 16, 2, 77), seed=4)
    O, _ = decode_attention(inp.q, inp.k, inp.v)
    as_bf16 = lambda x: torch.from_numpy(f32_to_bf16_bits(x.astype(np.float32)).view(np.int16)).view(torch.bfloat16)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16)
    full = bench.OracleFull(np, inp)
    rows = bench.OracleRows(np, torch, t(inp.q), t(inp.k), t(inp.v), [0, 2])

    class Fake:
        def __init__(self, out, name):
            self.out, self.name = out, name

        def sample(self, torch):
            return self.out

    good = as_bf16(O)
    off = as_bf16(O + 0.03)
    nan = good.clone()
    nan[1, 3, 5] = float("nan")
    bench.VALIDATION.update(validated=0, invalid=[])
    bench.validate(torch, full, [Fake(good, "good"), Fake(off, "off"), Fake(nan, "nan")], "planted")
    bench.validate(torch, rows, [Fake(good, "good rows"), Fake(off, "off rows")], "planted")
    assert bench.VALIDATION["validated"] == 5
    assert sorted(x["launch"] for x in bench.VALIDATION["invalid"]) == ["nan", "off", "off rows"]


def test_read_probe_library_checks_its_arguments():
    """The HBM read probe the benchmark sets the decode kernel against is
    built beside the decode library and rejects invalid arguments before any
    device access (no GPU here)."""
    import ctypes
    path = os.path.join(ROOT, "paper_2604_00028_amd", "libhbm_probe.so")
    if not os.path.exists(path):
        pytest.skip("libhbm_probe.so is not built")
    lib = ctypes.CDLL(path)
    f = lib.hbm_read_probe
    f.restype = ctypes.c_int
    f.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_int,
                  ctypes.c_int, ctypes.c_void_p]
    p = ctypes.c_void_p(0x1000)
    assert f(None, 1 << 20, p, 1 << 20, 256, 4, 0, None) == 1              # no source
    assert f(p, 1 << 20, None, 1 << 20, 256, 4, 0, None) == 1              # no sink
    assert f(p, (1 << 20) + 8, p, 1 << 20, 256, 4, 0, None) == 1           # not whole 16-byte vectors
    assert f(p, 1 << 20, p, 256 * 256 * 4 - 4, 256, 4, 0, None) == 1       # sink too small for the grid
    assert f(p, 1 << 20, p, 1 << 20, 0, 4, 0, None) == 1                   # no workgroups
    assert f(p, 1 << 20, p, 1 << 20, 256, 4, 2, None) == 1                 # hint not 0 or 1
    for loads in (0, 2, 12, 32):
        assert f(p, 1 << 20, p, 1 << 20, 256, loads, 0, None) == 1         # loads not 4, 8 or 16
    g = lib.hbm_read_probe_waves
    g.restype = ctypes.c_int
    g.argtypes = f.argtypes
    assert g(None, 1 << 20, p, 1 << 20, 256, 8, 0, None) == 1              # no source
    assert g(p, 1 << 20, p, 1 << 20, 3, 8, 0, None) == 1                   # regions do not divide the buffer
    assert g(p, 1 << 20, p, 256 * 256 * 4 - 4, 256, 8, 0, None) == 1       # sink too small
    assert g(p, 1 << 20, p, 1 << 20, 256, 4, 0, None) == 1                 # loads not 8 or 16


def test_wave_forms_pair_each_plan_with_its_other_wave_count():
    """The wave-count sweep launches every shape with two and with four waves
    per workgroup: the planner's plan and a valid plan of the other count
    (same split, tile and merge), with the fetch path that count takes."""
    sys.path.insert(0, ROOT)
    import bench
    import paper_2604_00028_amd as da
    for B, H_Q, H_KV, L in bench.WAVES_SHAPES:
        plan = da.da_choose_splits(B, H_Q, H_KV, L, num_cus=256)
        assert plan.num_splits == 1 and plan.v_slices == 1 and plan.heads_per_tile == H_Q // H_KV
        two, four = bench.wave_forms(da, plan, H_KV)
        assert (two.group_waves, four.group_waves) == (2, 4)
        assert four.wg_per_cu == 0 and (two is plan or two.wg_per_cu == 0)
        assert plan.group_waves == 2 and two is plan or plan.group_waves == 4 and four is plan
        lone = plan.grid <= 256
        assert two.combine == 0 and two.kv_fetch == (0 if H_KV == 1 and lone else 1)
        assert plan.wg_per_cu == 0 or (plan.group_waves == 2 and plan.grid > 320)
        assert four.kv_fetch == (2 if lone else 1)
        for p in (two, four):
            assert (p.num_splits, p.grid, p.heads_per_tile, p.v_slices) == (1, plan.grid, plan.heads_per_tile, 1)


def test_waves_sweep_summary(tmp_path, monkeypatch):
    sys.path.insert(0, ROOT)
    import json
    import bench
    row = lambda grid, planned, ratio: {"B": grid // 8, "H_Q": 64, "H_KV": 8, "L_K": 1024, "grid": grid,
                                        "cus": 256, "planned_waves": planned, "two_fetch": 1, "four_fetch": 1,
                                        "two_us": 10 * ratio, "two_iqr": [9.9, 10.1], "four_us": 10.0,
                                        "four_iqr": [9.9, 10.1], "two_over_four": ratio}
    src = tmp_path / "waves.json"
    src.write_text(json.dumps({"rows": [row(256, 2, 0.96), row(320, 2, 0.99), row(512, 4, 1.01), row(576, 4, 0.995)],
                               "validated": 8, "invalid": [], "rounds": 7}))
    out = tmp_path / "waves.md"
    monkeypatch.setattr(bench, "PROFILE_WAVES", str(out))
    bench.waves_sweep_summary(str(src))
    text = out.read_text()
    assert "python3 bench.py --waves-sweep $OUT/waves.json --rounds 7" in text
    assert "| 40 | 64 | 8 | 1024 | 320 / 256 | 2 | 9.9 (9.9-10.1, registers to LDS) |" in text
    assert "up to 5/4 (the two-wave rule): two / four 0.990-0.990 over 1 shapes" in text
    assert "past 5/4, 2-16 KV heads: two / four 0.995-1.010 over 2 shapes" in text
    assert "faster one on 3 of 4 shapes" in text
