"""bench.py's contract: one GPU only, the algorithmic operation count of the
blind rotation written out by hand, the clock statistic (CPU), and the
fields of the JSON line of a short run (GPU)."""
import math
import os
import subprocess
import sys

import pytest

import bench
from paper_1911_07101_amd import workloads as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode != 0
    assert "one GPU" in r.stderr


def _lane_ops_by_stage(N, n_lwe, l, parts):
    """Per CMux, stage by stage, for the 128-bit parameters' shape: 2l forward
    transforms, the transform-domain products, 2 x parts inverse transforms
    with their twist, digit extraction, the rotation difference and the
    rounding (one VALU lane-operation per FMA, add or integer op)."""
    n = N // 2                      # complex points of the folded polynomial
    stages = int(math.log2(n))
    butterflies = n // 2 * stages
    forward = 2 * l * butterflies * 6
    products = 2 * l * (2 * parts) * n * 4
    # inverse: stage s has n/2 butterflies, of which those with twiddle 1 or
    # -i (n/2 at stage 0, n/2^(s+1) ... counted as n >> s for s >= 1) take 4
    inverse_one = 0
    for s in range(stages):
        trivial = n // 2 if s == 0 else n >> s
        inverse_one += (n // 2 - trivial) * 6 + trivial * 4
    inverse = 2 * parts * (inverse_one + 4 * n)
    digits = 2 * l * N * 4
    rotation = 2 * N * 3
    rounding = 2 * N * 2 * parts
    return n_lwe * (forward + products + inverse + digits + rotation + rounding)


def test_algorithmic_count_matches_a_stage_by_stage_count():
    for name in ("tfhe128_nand", "lut3_n2048", "toy"):
        p = wl.CONFIGS[name]["params"]
        assert bench.algorithmic_lane_ops(p, 2) == _lane_ops_by_stage(p["N"], p["n"], p["l"], 2)
    # the figure the roofline is quoted on
    assert bench.algorithmic_lane_ops(wl.CONFIGS["tfhe128_nand"]["params"], 2) == 143_871_840


def test_clock_is_read_from_the_marked_dpm_level():
    assert bench.parse_sclk("0: 500Mhz\n1: 2362Mhz *\n2: 2400Mhz\n") == 2362
    assert bench.parse_sclk("S: 100Mhz *\n0: 500Mhz\n1: 2400Mhz\n") is None  # asleep
    assert bench.parse_sclk("0: 500Mhz\n1: 2400Mhz *\n") == 2400
    assert bench.parse_sclk("") is None
    assert bench.ClockSampler(None).mhz() is None


def test_clock_is_the_median_of_the_timed_window():
    c = bench.ClockSampler(None)
    # the driver's figure ramps up while the GPU wakes (before the window),
    # then reads the running clock
    c.samples = [(0.0, 368), (0.1, 1500), (0.2, 1700), (1.0, 2310), (1.1, 2320), (1.2, 2300), (1.3, 2290),
                 (1.4, 2330), (2.0, 500)]
    assert c.window(1.0, 1.4) == [2310, 2320, 2300, 2290, 2330]
    assert c.mhz(1.0, 1.4) == 2310
    assert c.mhz(1.0, 1.3) is None  # fewer than 5 samples in the window
    assert c.mhz(1.0, 1.3, least=4) == 2310


@pytest.mark.gpu
@pytest.mark.parametrize("config", ["tfhe128_nand", "lut3_n2048"])
def test_bench_line_has_every_field(config):
    """A short run of bench.py (a child process) prints one JSON line with
    the fields its readers rely on, a roofline object against the 39.3 T
    lane-op/s VALU peak, and outputs that decrypt to the expected bits."""
    import json
    print(f"[bench-contract] bench.py --config {config} --steps 2 --warmup 1", flush=True)
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--config", config, "--steps", "2",
                        "--warmup", "1", "--no-cpu-baseline"], capture_output=True, text=True, timeout=240)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [l for l in r.stdout.splitlines() if l.strip()]
    assert len(lines) == 1
    d = json.loads(lines[0])
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better",
                "scaling", "vs_baseline", "dtype", "data", "config", "roofline"):
        assert key in d, key
    assert d["n_gpus"] == 1 and d["steps"] == 2 and d["warmup"] == 1 and d["higher_is_better"] is True
    assert d["config"]["workload"] == config and d["value"] > 0 and d["truth_table_ok"] is True
    roof = d["roofline"]
    assert roof["bound"] == "alu" and abs(roof["peak"] - 39.3216) < 1e-9
    assert 0 < roof["frac"] < 1 and abs(roof["frac"] - roof["achieved"] / roof["peak"]) < 1e-12
    # the clock over the timed window (untimed steps let it settle first);
    # a two-step window may hold too few samples for a figure
    if roof["clock_samples"] >= 5:
        assert 1000 < roof["clock_mhz"] <= 2500
        assert abs(roof["frac_at_clock"] - roof["frac"] * 2400 / roof["clock_mhz"]) < 1e-9
    hbm = d["hbm"]
    assert hbm["peak_GBps"] == 8000 and hbm["algorithmic_GBps"] > 0
    assert "gfx950" in d["device"]


@pytest.mark.gpu
def test_driver_length_run_reports_the_clock():
    """A run of 20 timed steps after 5 warm-up steps (0.6 s of timed work)
    reports the clock of its timed window and the roofline fraction at that
    clock."""
    import json
    print("[bench-contract] bench.py --steps 20 --warmup 5", flush=True)
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--steps", "20", "--warmup", "5",
                        "--no-cpu-baseline"], capture_output=True, text=True, timeout=240)
    assert r.returncode == 0, r.stderr[-2000:]
    roof = json.loads(r.stdout.strip().splitlines()[-1])["roofline"]
    if roof["clock_samples"] == 0:
        pytest.skip("the DPM table is not readable here")
    assert roof["clock_mhz"] is not None and roof["frac_at_clock"] is not None


@pytest.mark.gpu
def test_issue_rate_probe_lines():
    """bench.py --issue-rate prints one line per instruction kind; the fp64
    FMA and the conversion run at no more than the issue model's 64
    lane-operations per CU per clock and the 32-bit kinds at no more than
    twice that (CDNA4's 32-bit VALU rate), within a margin (15 %) wider than
    the driver's clock reading is ever off (about 2 %)."""
    import json
    print("[bench-contract] bench.py --issue-rate 2000", flush=True)
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--issue-rate", "2000"],
                       capture_output=True, text=True, timeout=240)
    assert r.returncode == 0, r.stderr[-2000:]
    lines = [json.loads(x) for x in r.stdout.strip().splitlines()]
    rate = {d["instruction"]: d for d in lines}
    assert sorted(rate) == sorted(("v_fma_f64", "v_add_u32", "v_cvt_f64_i32", "v_bfe_i32", "v_mul_lo_u32"))
    for d in lines:
        assert d["ms"] > 0 and d["lane_ops_per_s"] > 0
        limit = 64 if d["instruction"] in ("v_fma_f64", "v_cvt_f64_i32") else 128
        if d["lane_ops_per_cu_per_clock"] is not None:
            assert d["lane_ops_per_cu_per_clock"] <= limit * 1.15, d
