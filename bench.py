#!/usr/bin/env python3
"""Throughput of batched TFHE gate bootstrapping on one MI355X.

One step = one call of tfhe_gate_bootstrap_batch on the whole batch: gate
pre-combination and modulus switch, blind rotation (n CMux external products)
with SampleExtract, and key switching.  Default workload: 4096 NAND gate
bootstraps with the 128-bit parameters n = 630, N = 1024, l = 3, Bg = 2^7,
key switching t = 8, base 2^2.  Inputs are seeded synthetic encrypted bits,
resident in device memory before timing starts.

Prints one JSON line with the throughput, the roofline position of the
blind-rotation kernel (timed with HIP events on its own stream), and the CPU
oracle's throughput on a bounded sample of the same workload.
"""
import argparse
import hashlib
import json
import math
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "gate bootstraps/sec (n=630,N=1024) + % of int-VALU roofline, 1 MI355X"
# CDNA4 (MI355X): 256 CUs x 64 lanes x 2.4 GHz; a full-rate VALU instruction
# (32-bit integer op, fp64 add/mul/FMA) retires 64 lane-operations per CU per clock
PEAK_LANE_OPS = 256 * 64 * 2.4e9
PEAK_HBM = 8.0e12


def algorithmic_lane_ops(p, parts: int) -> float:
    """VALU lane-operations one bootstrap's blind rotation needs with the
    complex fp64 transform over n = N/2 points (FMA = 1 op; key split into
    `parts` parts, so 2*parts transform-domain outputs); address arithmetic,
    memory traffic and loop control are not counted."""
    N, n_lwe, l = p["N"], p["n"], p["l"]
    n = N // 2
    outs = 2 * parts
    bfly = n // 2 * int(math.log2(n))
    fwd = 2 * l * bfly * 8                 # complex multiply (4) + 2 complex adds (4)
    digits = 2 * l * N * 4 + 2 * N * 3     # digit extract + convert; rotation difference
    pointwise = 2 * l * outs * n * 4       # complex multiply-accumulate: 4 FMAs
    inv = outs * bfly * 8
    convert = 2 * N * 2 * parts            # round (1 add) and shift-add per part, accumulate
    return float(n_lwe * (fwd + digits + pointwise + inv + convert))


def algorithmic_bytes_br(p, B, parts) -> float:
    """Bytes the blind-rotation launch must move: the transform-domain key once,
    modulus-switched inputs in, extracted samples out."""
    bk = p["n"] * 2 * p["l"] * 2 * parts * (p["N"] // 2) * 16
    return float(bk + B * (p["n"] + 1) * 2 + B * (p["N"] + 1) * 4)


def kernel_source_digest() -> str:
    h = hashlib.sha256()
    for f in ("gt_kernels.hip", "gt_layout.hpp"):
        with open(os.path.join(ROOT, "paper_1911_07101_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(digest: str):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if it
    was taken on the current kernel source."""
    path = os.path.join(ROOT, "profiles", "blind_rotate_tfhe128_traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        rec = json.load(fh)
    if rec.get("kernel_source_digest") != digest:
        return None
    return rec.get("hbm_bytes_per_launch")


def cpu_baseline(cfg, ca, cb, gpu_out):
    import numpy as np

    import oracle
    from paper_1911_07101_amd import tfhe

    p = cfg["params"]
    threads = oracle.threads()
    count = int(min(64, max(4, 2 * threads)))
    keys = oracle.Keys(p, cfg["key_seed"])
    t0 = time.perf_counter()
    ref = oracle.gate_bootstrap(keys, cfg["gate"], ca[:count], cb[:count])
    dt = time.perf_counter() - t0
    return {
        "value": count / dt, "unit": "bootstraps/s", "cores": threads, "kind": "oracle",
        "sample": f"first {count} {cfg['gate']} gates of the batch (schoolbook products, "
                  f"OpenMP over gates), {dt:.1f} s wall",
        "host_cpu": platform.processor() or platform.machine(),
        "matches_gpu": bool(np.array_equal(ref, tfhe.to_host(gpu_out)[:count])),
    }


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="tfhe128_nand")
    ap.add_argument("--batch", type=int, default=None, help="override the batch size")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="before timing, run one plain device copy of this size (counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the bootstrap batch has no cross-GPU step on this "
              "path; run it with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_1911_07101_amd import tfhe, workloads as wl

    cfg = dict(wl.CONFIGS[args.config])
    if cfg["kind"] != "gate":
        raise SystemExit("bench.py times gate-bootstrap workloads")
    p = cfg["params"]
    B = args.batch or cfg["batch"]
    dev = torch.device("cuda:0")

    sk, ek = tfhe.tfhe_keygen_from_seed(p, cfg["key_seed"], 0)
    a, b = wl.gate_inputs(cfg["input_seed"], B)
    ca_h = tfhe.tfhe_encrypt_torus(sk, cfg["input_seed"], tfhe.encode_bits(a), 0)
    cb_h = tfhe.tfhe_encrypt_torus(sk, cfg["input_seed"], tfhe.encode_bits(b), B)
    ca, cb = tfhe.to_device(ca_h), tfhe.to_device(cb_h)
    out = torch.empty((B, p["n"] + 1), dtype=torch.int32, device=dev)
    ws = tfhe.alloc_workspace(ek, B)
    stream = torch.cuda.current_stream()

    if args.copy_probe_mib:
        src = torch.empty(args.copy_probe_mib << 18, dtype=torch.int32, device=dev).fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    for _ in range(args.warmup):
        tfhe.tfhe_gate_bootstrap_batch(ek, cfg["gate"], ca, cb, out=out, workspace=ws, stream=stream)
    torch.cuda.synchronize()

    tfhe.tfhe_stage_timing(True)
    tfhe.tfhe_stage_times()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        tfhe.tfhe_gate_bootstrap_batch(ek, cfg["gate"], ca, cb, out=out, workspace=ws, stream=stream)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    stages = tfhe.tfhe_stage_times()
    tfhe.tfhe_stage_timing(False)

    elapsed = t1 - t0
    value = B * args.steps / elapsed
    res = tfhe.to_host(out)
    dec = tfhe.tfhe_decrypt_phase(sk, res).astype(np.int64)
    dec = (np.where(dec >= 1 << 31, dec - (1 << 32), dec) > 0).astype(np.uint8)
    truth_ok = bool(np.array_equal(dec, 1 - (a & b))) if cfg["gate"] == "NAND" else None

    br_ms, br_n = stages["blind_rotate"]
    br_s = br_ms / 1e3 / max(br_n, 1)
    parts, bound = tfhe.tfhe_transform_error_bound(p)
    ops = algorithmic_lane_ops(p, parts) * B
    achieved = ops / br_s
    digest = kernel_source_digest()
    traffic = measured_traffic(digest)
    line = {
        "metric": METRIC,
        "value": value,
        "unit": "bootstraps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": elapsed / args.steps * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u32/f64",
        "data": "synthetic",
        "config": {"workload": args.config, "gate": cfg["gate"], "batch": B, "n": p["n"], "N": p["N"],
                   "l": p["l"], "bg_bit": p["bg_bit"], "ks_t": p["ks_t"], "ks_basebit": p["ks_basebit"]},
        "roofline": {
            "bound": "alu",
            "kernel": "blind_rotate_kernel",
            "achieved": achieved / 1e12,
            "peak": PEAK_LANE_OPS / 1e12,
            "unit": "T lane-op/s",
            "frac": achieved / PEAK_LANE_OPS,
            "traffic": traffic,
            "ops_per_bootstrap": algorithmic_lane_ops(p, parts),
            "launch_ms": br_s * 1e3,
        },
        "hbm": {
            "kernel": "blind_rotate_kernel",
            "algorithmic_bytes_per_launch": algorithmic_bytes_br(p, B, parts),
            "achieved_GBps": algorithmic_bytes_br(p, B, parts) / br_s / 1e9,
            "peak_GBps": PEAK_HBM / 1e9,
        },
        "stage_ms_per_step": {k: (v[0] / max(v[1], 1)) for k, v in stages.items()},
        "truth_table_ok": truth_ok,
        "transform": {"key_parts": parts, "worst_case_error": bound},
        "kernel_source_digest": digest,
        "device": torch.cuda.get_device_name(0),
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(cfg, ca_h, cb_h, out)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
