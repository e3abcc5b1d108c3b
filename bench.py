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
    fwd = 2 * l * bfly * 6                 # a = u + w v: 4 FMAs; b = 2u - a: 2 FMAs
    digits = 2 * l * N * 4 + 2 * N * 3     # digit extract + convert; rotation difference
    pointwise = 2 * l * outs * n * 4       # complex multiply-accumulate: 4 FMAs
    # cyclic inverse by decimation in time: butterflies with twiddle 1 or -i
    # (n/2 at the first stage, n/2^s at stage s >= 1) take 4 adds, the others
    # 6 FMAs; then the twist, one complex product (4 ops) per point
    trivial = n // 2 + sum(n >> s for s in range(1, int(math.log2(n))))
    inv = outs * (bfly * 6 - trivial * 2 + n * 4)
    convert = 2 * N * 2 * parts            # round (1 add) and shift-add per part, accumulate
    return float(n_lwe * (fwd + digits + pointwise + inv + convert))


def algorithmic_bytes_br(p, B, parts) -> float:
    """Bytes the blind-rotation launch must move: the transform-domain key once,
    modulus-switched inputs in, extracted samples out."""
    bk = p["n"] * 2 * p["l"] * 2 * parts * (p["N"] // 2) * 16
    return float(bk + B * (p["n"] + 1) * 2 + B * (p["N"] + 1) * 4)


def kernel_source_digest() -> str:
    """Digest of the kernel sources' code: comments (the sources hold only
    // comments) and blank lines are left out, so that editing a comment does
    not mark the committed counter summaries as taken on other kernels."""
    h = hashlib.sha256()
    for f in ("gt_kernels.hip", "gt_layout.hpp"):
        with open(os.path.join(ROOT, "paper_1911_07101_amd", "csrc", f), encoding="utf-8") as fh:
            for line in fh:
                code = line.split("//", 1)[0].rstrip()
                if code:
                    h.update(code.encode() + b"\n")
    return h.hexdigest()[:16]


TRAFFIC_FILES = {"tfhe128_nand": "blind_rotate_tfhe128_traffic.json",
                 "lut3_n2048": "blind_rotate_split_lut3_n2048_traffic.json"}


def measured_traffic(digest: str, config: str = "tfhe128_nand"):
    """HBM bytes per launch from the committed rocprofv3 counter summary of
    the workload, if it was taken on the current kernel source."""
    if config not in TRAFFIC_FILES:
        return None
    path = os.path.join(ROOT, "profiles", TRAFFIC_FILES[config])
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        rec = json.load(fh)
    if rec.get("kernel_source_digest") != digest:
        return None
    return rec.get("hbm_bytes_per_launch")


def host_cpu_model() -> str:
    """The host CPU's model name (Linux /proc/cpuinfo), else the machine type."""
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or platform.machine()


def parse_sclk(text: str):
    """Current shader clock (MHz) from the driver's DPM table (sysfs
    pp_dpm_sclk): the numbered level marked '*'; None while the GPU sleeps
    (the 'S:' line is marked) or if no level is marked."""
    import re
    for line in text.splitlines():
        m = re.match(r"\s*(\d+):\s*(\d+)\s*mhz\s*\*", line, re.I)
        if m:
            return int(m.group(2))
    return None


def sclk_path():
    """pp_dpm_sclk of cuda:0's card (matched by PCI address), else of the
    only card, else None."""
    import glob

    import torch
    cards = sorted(glob.glob("/sys/class/drm/card*/device/pp_dpm_sclk"))
    try:
        pr = torch.cuda.get_device_properties(0)
        bus = f"{pr.pci_domain_id:04x}:{pr.pci_bus_id:02x}:{pr.pci_device_id:02x}"
        for c in cards:
            if os.path.basename(os.path.realpath(os.path.dirname(c))).startswith(bus):
                return c
    except (AttributeError, RuntimeError, OSError):
        pass
    return cards[0] if len(cards) == 1 else None


class ClockSampler:
    """The GPU's shader clock while the steps run: a host thread reads the
    DPM table every 10 ms and keeps (time, MHz) pairs.  Context for the
    roofline fraction, whose peak assumes 2.4 GHz: MI355X machines run this
    kernel at 2.0 to 2.4 GHz."""

    def __init__(self, path, period=0.01):
        import threading
        self.path, self.period, self.samples = path, period, []
        self._stop = threading.Event()
        self._thread = threading.Thread(target=self._run, daemon=True) if path else None

    def _run(self):
        while not self._stop.is_set():
            try:
                with open(self.path) as fh:
                    v = parse_sclk(fh.read())
            except OSError:
                return
            if v is not None:
                self.samples.append((time.perf_counter(), v))
            self._stop.wait(self.period)

    def __enter__(self):
        if self._thread:
            self._thread.start()
        return self

    def __exit__(self, *exc):
        if self._thread:
            self._stop.set()
            self._thread.join()

    def window(self, t0=None, t1=None):
        """The samples taken in [t0, t1] (open ends: all)."""
        return [v for t, v in self.samples if (t0 is None or t >= t0) and (t1 is None or t <= t1)]

    def mhz(self, t0=None, t1=None, least=5):
        """Median of the samples taken in [t0, t1], or None with fewer than
        `least` of them.  The driver's figure takes about half a second to
        settle after the GPU wakes, so bench.py runs untimed steps for a
        second before the warm-up and reads only the timed window."""
        s = sorted(self.window(t0, t1))
        if len(s) < least:
            return None
        return s[len(s) // 2]


def cpu_baseline(cfg, ca, cb, gpu_out, testvec=None):
    """The oracle on the first gates (or lookups) of the batch.  ca, cb: the
    gate inputs; for a table-lookup workload ca holds the inputs and testvec
    the test polynomial."""
    import numpy as np

    import oracle
    from paper_1911_07101_amd import tfhe

    p = cfg["params"]
    threads = oracle.threads()
    keys = oracle.Keys(p, cfg["key_seed"])
    if testvec is None:
        count = int(min(128, max(8, 6 * threads)))  # about 15 s of oracle work on 16 cores
        what = f"{cfg['gate']} gates"
        t0 = time.perf_counter()
        ref = oracle.gate_bootstrap(keys, cfg["gate"], ca[:count], cb[:count])
    else:
        count = int(min(64, max(4, 2 * threads)))  # N = 2048: ~3x the work per bootstrap
        what = "table lookups"
        t0 = time.perf_counter()
        ref = oracle.lut_bootstrap(keys, ca[:count], testvec)
    dt = time.perf_counter() - t0
    # the same oracle on one thread, over the first one or two bootstraps
    one = 2 if testvec is None else 1
    oracle.set_threads(1)
    try:
        t1 = time.perf_counter()
        if testvec is None:
            ref1 = oracle.gate_bootstrap(keys, cfg["gate"], ca[:one], cb[:one])
        else:
            ref1 = oracle.lut_bootstrap(keys, ca[:one], testvec)
        dt1 = time.perf_counter() - t1
    finally:
        oracle.set_threads(threads)
    return {
        "value": count / dt, "unit": "bootstraps/s", "cores": threads, "kind": "oracle",
        "sample": f"first {count} {what} of the batch (schoolbook products, "
                  f"OpenMP over bootstraps), {dt:.1f} s wall",
        "host_cpu": host_cpu_model(),
        "host_nproc": os.cpu_count(),
        "single_thread_s_per_bootstrap": dt1 / one,
        "single_thread_sample": f"first {one} of the same {what} on one thread, {dt1:.1f} s",
        "matches_gpu": bool(np.array_equal(ref, tfhe.to_host(gpu_out)[:count])
                            and np.array_equal(ref1, ref[:one])),
    }


def _timed(fn, reps: int):
    """Median wall time (ms) of fn() over reps calls, each bracketed by HIP
    events on the current stream (fn launches on that stream)."""
    import torch
    times = []
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        fn()
        e1.record()
        e1.synchronize()
        times.append(e0.elapsed_time(e1))
    times.sort()
    return times[len(times) // 2]


def suite(path: str):
    """Throughput of every workload (toy latency, 128-bit NAND batch sweep, MLP
    forward ReLU and backward iReLU, the TFHE side of the BGV-to-TFHE switch
    for the MLP layer, conv ReLU resident and streamed from
    pinned host memory, the 3-bit softmax unit as a multiplexer tree and as a
    LUT bootstrap at N = 2048); one JSON record per line, also written to
    path."""
    import numpy as np
    import torch

    from paper_1911_07101_amd import tfhe, workloads as wl

    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    recs = []

    def emit(**r):
        recs.append(r)
        print(json.dumps(r), flush=True)

    def bits_of(ph):
        ph = ph.astype(np.int64)
        return (np.where(ph >= 1 << 31, ph - (1 << 32), ph) > 0).astype(np.uint8)

    # toy: latency of one 16-gate call
    cfg = wl.CONFIGS["toy"]
    p = cfg["params"]
    sk, ek = tfhe.tfhe_keygen_from_seed(p, cfg["key_seed"], 0)
    a, b = wl.gate_inputs(cfg["input_seed"], cfg["batch"])
    ca = tfhe.to_device(tfhe.tfhe_encrypt_torus(sk, cfg["input_seed"], tfhe.encode_bits(a), 0))
    cb = tfhe.to_device(tfhe.tfhe_encrypt_torus(sk, cfg["input_seed"], tfhe.encode_bits(b), len(a)))
    out = torch.empty((len(a), p["n"] + 1), dtype=torch.int32, device=dev)
    ws = tfhe.alloc_workspace(ek, len(a))
    call = lambda: tfhe.tfhe_gate_bootstrap_batch(ek, "NAND", ca, cb, out=out, workspace=ws, stream=stream)
    call()
    ms = _timed(call, 21)
    ok = np.array_equal(bits_of(tfhe.tfhe_decrypt_phase(sk, tfhe.to_host(out))), 1 - (a & b))
    emit(workload="toy", gates=len(a), ms_per_call=ms, per_s=len(a) / ms * 1e3, unit="bootstraps/s", ok=bool(ok))
    del ek, sk

    # 128-bit NAND: batch sweep (key generation, the key's transform and its
    # upload are client-side setup, timed here apart from every call)
    cfg = wl.CONFIGS["tfhe128_nand"]
    p = cfg["params"]
    t0 = time.perf_counter()
    sk, ek = tfhe.tfhe_keygen_from_seed(p, cfg["key_seed"], 0)
    emit(workload="keygen", config="tfhe128_nand", s=time.perf_counter() - t0,
         what="secret keys, bootstrapping key in the transform domain, key-switching key, uploaded")
    for B in (256, 1024, 4096, 16384, 65536):
        a, b = wl.gate_inputs(cfg["input_seed"], B)
        ca = tfhe.to_device(tfhe.tfhe_encrypt_torus(sk, cfg["input_seed"], tfhe.encode_bits(a), 0))
        cb = tfhe.to_device(tfhe.tfhe_encrypt_torus(sk, cfg["input_seed"], tfhe.encode_bits(b), B))
        out = torch.empty((B, p["n"] + 1), dtype=torch.int32, device=dev)
        ws = tfhe.alloc_workspace(ek, B)
        call = lambda: tfhe.tfhe_gate_bootstrap_batch(ek, "NAND", ca, cb, out=out, workspace=ws, stream=stream)
        call()
        ms = _timed(call, 5 if B <= 16384 else 3)
        ok = np.array_equal(bits_of(tfhe.tfhe_decrypt_phase(sk, tfhe.to_host(out))), 1 - (a & b))
        emit(workload="tfhe128_nand", gates=B, ms_per_call=ms, per_s=B / ms * 1e3, unit="bootstraps/s", ok=bool(ok))
        del ca, cb, out, ws

    # MLP ReLU: 7680 8-bit values, 53,760 gates in one call
    cfg = wl.CONFIGS["mlp_relu"]
    V = cfg["values"]
    xs = wl.int8_values(cfg["input_seed"], V)
    ct = tfhe.tfhe_encrypt_torus(sk, cfg["input_seed"], tfhe.encode_bits(wl.to_bits(xs, 8).ravel()))
    x = tfhe.to_device(ct.reshape(V, 8, p["n"] + 1))
    y = torch.empty_like(x)
    ws = tfhe.alloc_workspace(ek, V * 7)
    call = lambda: tfhe.glyph_relu_batch(ek, x, 8, y=y, workspace=ws, stream=stream)
    call()
    ms = _timed(call, 3)
    dec = bits_of(tfhe.tfhe_decrypt_phase(sk, tfhe.to_host(y).reshape(-1, p["n"] + 1))).reshape(V, 8)
    ok = np.array_equal(wl.from_bits(dec), np.maximum(xs.astype(np.int64), 0))
    emit(workload="mlp_relu", values=V, gates=V * 7, ms_per_call=ms, per_s=V * 7 / ms * 1e3,
         unit="gate bootstraps/s", ok=bool(ok))
    del x, y, ws

    # MLP backward iReLU: 7680 8-bit errors gated by the forward signs
    cfg = wl.CONFIGS["mlp_irelu"]
    V = cfg["values"]
    us = wl.int8_values(cfg["input_seed"], V)
    ds = wl.int8_values(cfg["input_seed"], V, stream=7)
    u = tfhe.to_device(tfhe.tfhe_encrypt_torus(sk, cfg["input_seed"], tfhe.encode_bits(wl.to_bits(us, 8).ravel()))
                       .reshape(V, 8, p["n"] + 1))
    d = tfhe.to_device(tfhe.tfhe_encrypt_torus(sk, cfg["input_seed"] + 1, tfhe.encode_bits(wl.to_bits(ds, 8).ravel()))
                       .reshape(V, 8, p["n"] + 1))
    y = torch.empty_like(d)
    ws = tfhe.alloc_workspace(ek, V * 8)
    call = lambda: tfhe.glyph_irelu_batch(ek, u, d, out=y, workspace=ws, stream=stream)
    call()
    ms = _timed(call, 3)
    dec = bits_of(tfhe.tfhe_decrypt_phase(sk, tfhe.to_host(y).reshape(-1, p["n"] + 1))).reshape(V, 8)
    ok = np.array_equal(wl.from_bits(dec), np.where(us >= 0, ds.astype(np.int64), 0))
    emit(workload="mlp_irelu", values=V, gates=V * 8, ms_per_call=ms, per_s=V * 8 / ms * 1e3,
         unit="gate bootstraps/s", ok=bool(ok))
    del u, d, y, ws

    # TFHE side of the BGV-to-TFHE switch for the MLP layer's 7680 values and
    # the conv layer's 207,360: LWE samples (n = 630) of 4-bit messages packed
    # 960 to a TRLWE sample (step 2), the 960 coefficients of each extracted
    # (step 3) and key-switched back to n; every value decodes to its
    # message.  Step 4 (TFHE to BGV) is a programmable bootstrap with a torus
    # test vector: the LUT bootstrap measured last.
    t0 = time.perf_counter()
    tfhe.tfhe_packing_key_upload(sk, ek)
    pk_s = time.perf_counter() - t0
    Zp = 960
    for layer in ("mlp_relu", "conv_relu"):
        cfg = wl.CONFIGS[layer]
        V, seed = cfg["values"], cfg["input_seed"] + 5
        msgs = wl.messages(seed, V, 4)
        lwe = tfhe.to_device(tfhe.tfhe_encrypt_torus(sk, seed, (msgs << 28).astype(np.uint32))
                             .reshape(V // Zp, Zp, p["n"] + 1))
        packed = torch.empty((V // Zp, 2, p["N"]), dtype=torch.int32, device=dev)
        ext = torch.empty((V // Zp, Zp, p["N"] + 1), dtype=torch.int32, device=dev)
        back = torch.empty((V, p["n"] + 1), dtype=torch.int32, device=dev)
        steps = [lambda: tfhe.tfhe_pack_keyswitch_batch(ek, lwe, out=packed, stream=stream),
                 lambda: tfhe.tfhe_sample_extract_batch(packed, Zp, out=ext, stream=stream),
                 lambda: tfhe.tfhe_keyswitch_batch(ek, ext.view(V, p["N"] + 1), out=back, stream=stream)]
        for f in steps:
            f()
        step_ms = [_timed(f, 5) for f in steps]
        ph = tfhe.tfhe_decrypt_phase(sk, tfhe.to_host(back)).astype(np.int64)
        ok = np.array_equal(((ph + (1 << 27)) >> 28) % 16, msgs)
        emit(workload="switch_bgv_to_tfhe", layer=layer, values=V, lwe_per_trlwe=Zp,
             pack_keyswitch_ms=step_ms[0], sample_extract_ms=step_ms[1], keyswitch_ms=step_ms[2],
             per_s=V / sum(step_ms) * 1e3, unit="values/s", packing_key_setup_s=pk_s, ok=bool(ok))
        del lwe, packed, ext, back

    # conv ReLU: 207,360 values, calls of 16,384 gates; inputs resident in HBM
    cfg = wl.CONFIGS["conv_relu"]
    V, step = cfg["values"], cfg["gates_per_call"]
    total = V * 7
    xs = wl.int8_values(cfg["input_seed"], V)
    ct = tfhe.tfhe_encrypt_torus(sk, cfg["input_seed"], tfhe.encode_bits(wl.to_bits(xs, 8).ravel()))
    ct = ct.reshape(V, 8, p["n"] + 1)
    x = tfhe.to_device(ct)
    y = torch.empty_like(x)
    ws = tfhe.alloc_workspace(ek, step)

    def conv_resident():
        for begin in range(0, total, step):
            tfhe.glyph_relu_batch(ek, x, 8, y=y, gate_begin=begin, gate_end=min(begin + step, total),
                                  workspace=ws, stream=stream)
    conv_resident()
    ms = _timed(conv_resident, 1)
    dec = bits_of(tfhe.tfhe_decrypt_phase(sk, tfhe.to_host(y).reshape(-1, p["n"] + 1))).reshape(V, 8)
    ok = np.array_equal(wl.from_bits(dec), np.maximum(xs.astype(np.int64), 0))
    emit(workload="conv_relu", values=V, gates=total, calls=(total + step - 1) // step, ms=ms,
         per_s=total / ms * 1e3, unit="gate bootstraps/s", inputs="resident in HBM", ok=bool(ok))
    del x, y

    # conv ReLU streamed from pinned host memory: chunks of whole values,
    # copy-in / compute / copy-out on three streams, double-buffered
    vals = step // 7
    chunks = [(v0, min(v0 + vals, V)) for v0 in range(0, V, vals)]
    hx = torch.from_numpy(ct.view(np.int32)).pin_memory()
    hy = torch.empty(hx.shape, dtype=torch.int32, pin_memory=True)
    dx = [torch.empty((vals, 8, p["n"] + 1), dtype=torch.int32, device=dev) for _ in range(2)]
    dy = [torch.empty_like(dx[0]) for _ in range(2)]
    s_in, s_out = torch.cuda.Stream(), torch.cuda.Stream()

    def conv_streamed():
        done_in = [torch.cuda.Event() for _ in chunks]
        done_comp = [torch.cuda.Event() for _ in chunks]
        done_out = [torch.cuda.Event() for _ in chunks]
        for k, (v0, v1) in enumerate(chunks):
            buf = k & 1
            with torch.cuda.stream(s_in):
                if k >= 2:
                    s_in.wait_event(done_comp[k - 2])
                dx[buf][: v1 - v0].copy_(hx[v0:v1], non_blocking=True)
                done_in[k].record(s_in)
            stream.wait_event(done_in[k])
            if k >= 2:
                stream.wait_event(done_out[k - 2])
            tfhe.glyph_relu_batch(ek, dx[buf][: v1 - v0], 8, y=dy[buf][: v1 - v0], workspace=ws, stream=stream)
            done_comp[k].record(stream)
            with torch.cuda.stream(s_out):
                s_out.wait_event(done_comp[k])
                hy[v0:v1].copy_(dy[buf][: v1 - v0], non_blocking=True)
                done_out[k].record(s_out)
        stream.wait_stream(s_out)

    torch.cuda.synchronize()
    t0 = time.perf_counter()
    conv_streamed()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3
    dec = bits_of(tfhe.tfhe_decrypt_phase(sk, hy.numpy().view(np.uint32).reshape(-1, p["n"] + 1))).reshape(V, 8)
    ok = np.array_equal(wl.from_bits(dec), np.maximum(xs.astype(np.int64), 0))
    emit(workload="conv_relu", values=V, gates=total, calls=len(chunks), ms=ms, per_s=total / ms * 1e3,
         unit="gate bootstraps/s", inputs="pinned host memory, H2D and D2H overlapped with compute",
         bytes_each_way=int(hx.numel() * 4), ok=bool(ok))
    del hx, hy, dx, dy, ws

    # the paper's 3-bit softmax unit as a multiplexer tree over bit-wise
    # encrypted inputs (same messages and table as the LUT bootstrap below)
    cfg = wl.CONFIGS["softmax_mux3"]
    V, mb, ob = cfg["values"], cfg["msg_bits"], cfg["out_bits"]
    m = wl.messages(cfg["input_seed"], V, mb)
    table = wl.lut(cfg["input_seed"], mb)
    x = tfhe.to_device(tfhe.tfhe_encrypt_torus(sk, cfg["input_seed"], tfhe.encode_bits(wl.to_bits(m, mb).ravel()))
                       .reshape(V, mb, p["n"] + 1))
    y = torch.empty((V, ob, p["n"] + 1), dtype=torch.int32, device=dev)
    ws = tfhe.alloc_mux_lut_workspace(ek, V, mb, ob)
    call = lambda: tfhe.glyph_mux_lut_batch(ek, x, table, ob, out=y, workspace=ws, stream=stream)
    call()
    ms = _timed(call, 3)
    dec = bits_of(tfhe.tfhe_decrypt_phase(sk, tfhe.to_host(y).reshape(-1, p["n"] + 1))).reshape(V, ob)
    ok = np.array_equal((dec.astype(np.int64) << np.arange(ob)).sum(axis=1), table[m])
    muxes = ((1 << (mb - 1)) - 1) * ob
    emit(workload="softmax_mux3", values=V, multiplexers_per_value=muxes, bootstraps=2 * muxes * V,
         ms_per_call=ms, per_s=V / ms * 1e3, unit="3-bit lookups/s", ok=bool(ok))
    del x, y, ws, ek, sk

    # 3-bit LUT bootstrap, N = 2048
    cfg = wl.CONFIGS["lut3_n2048"]
    p = cfg["params"]
    t0 = time.perf_counter()
    sk, ek = tfhe.tfhe_keygen_from_seed(p, cfg["key_seed"], 0)
    emit(workload="keygen", config="lut3_n2048", s=time.perf_counter() - t0,
         what="secret keys, bootstrapping key in the transform domain, key-switching key, uploaded")
    B = cfg["batch"]
    m = wl.messages(cfg["input_seed"], B, cfg["msg_bits"])
    table = wl.lut(cfg["input_seed"], cfg["msg_bits"])
    tv = tfhe.to_device(tfhe.tfhe_lut_testvec(p["N"], cfg["msg_bits"], table))
    x = tfhe.to_device(tfhe.tfhe_encrypt_torus(sk, cfg["input_seed"], (m << 28).astype(np.uint32), 0))
    out = torch.empty((B, p["n"] + 1), dtype=torch.int32, device=dev)
    ws = tfhe.alloc_workspace(ek, B)
    call = lambda: tfhe.tfhe_lut_bootstrap_batch(ek, x, tv, out=out, workspace=ws, stream=stream)
    call()
    ms = _timed(call, 5)
    ph = tfhe.tfhe_decrypt_phase(sk, tfhe.to_host(out)).astype(np.int64)
    ok = np.array_equal(((ph + (1 << 27)) >> 28) & 15, table[m])
    emit(workload="lut3_n2048", gates=B, ms_per_call=ms, per_s=B / ms * 1e3, unit="bootstraps/s = 3-bit lookups/s",
         ok=bool(ok))

    with open(path, "w") as fh:
        json.dump(recs, fh, indent=1)


def issue_rate(iters: int):
    """The VALU issue rate of each instruction kind the blind rotation uses
    (tfhe_probe_valu_rate): 8 waves per SIMD, each running iters rounds of 16
    instructions on 8 independent chains; lane-operations per CU per clock at
    the clock read over the timed launches, against the 64 (4 SIMDs x 16
    lanes) that the roofline's peak assumes.  One JSON line per kind."""
    import torch

    from paper_1911_07101_amd import tfhe

    props = torch.cuda.get_device_properties(0)
    cus = props.multi_processor_count
    waves = cus * 4 * 8
    out = torch.empty(waves * 64, dtype=torch.int32, device="cuda:0")
    stream = torch.cuda.current_stream()
    for kind in tfhe.PROBE_KINDS:
        with ClockSampler(sclk_path()) as clock:
            t_settle = time.perf_counter()
            while time.perf_counter() - t_settle < 0.5:
                tfhe.tfhe_probe_valu_rate(kind, waves, iters, out=out, stream=stream)
                torch.cuda.synchronize()
            times = []
            t0 = time.perf_counter()
            for _ in range(40):
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record(stream)
                tfhe.tfhe_probe_valu_rate(kind, waves, iters, out=out, stream=stream)
                e1.record(stream)
                e1.synchronize()
                times.append(e0.elapsed_time(e1))
            t1 = time.perf_counter()
        ms = sorted(times)[len(times) // 2]
        lane_ops = waves * 64 * iters * 16
        mhz = clock.mhz(t0, t1)
        rate = lane_ops / (ms / 1e3)
        print(json.dumps({
            "probe": "valu_issue_rate", "instruction": kind, "waves": waves, "iters": iters,
            "instructions_per_wave": iters * 16, "ms": ms, "lane_ops_per_s": rate,
            "frac_of_peak_at_2400MHz": rate / PEAK_LANE_OPS, "clock_mhz": mhz,
            "lane_ops_per_cu_per_clock": rate / cus / (mhz * 1e6) if mhz else None,
            "device": f"{props.name} ({getattr(props, 'gcnArchName', '?')}, {cus} CUs)"}), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=40)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--settle", type=float, default=1.0,
                    help="seconds of untimed steps before the warm-up (lets the clock reading settle)")
    ap.add_argument("--config", default="tfhe128_nand")
    ap.add_argument("--batch", type=int, default=None, help="override the batch size")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="before timing, run one plain device copy of this size (counter calibration)")
    ap.add_argument("--suite", metavar="PATH", default=None,
                    help="instead of the headline line, time every workload and write the records to PATH")
    ap.add_argument("--issue-rate", type=int, metavar="ITERS", default=0,
                    help="instead of the headline line, measure the VALU issue rate of each instruction kind "
                         "the blind rotation uses (ITERS rounds of 8 instructions per wave)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the bootstrap batch has no cross-GPU step on this "
              "path; run it with --gpus 1", file=sys.stderr)
        sys.exit(2)

    if args.suite:
        suite(args.suite)
        return
    if args.issue_rate:
        issue_rate(args.issue_rate)
        return

    import numpy as np
    import torch

    from paper_1911_07101_amd import tfhe, workloads as wl

    cfg = dict(wl.CONFIGS[args.config])
    if cfg["kind"] not in ("gate", "lut"):
        raise SystemExit("bench.py times gate-bootstrap and table-lookup workloads")
    p = cfg["params"]
    B = args.batch or cfg["batch"]
    dev = torch.device("cuda:0")

    sk, ek = tfhe.tfhe_keygen_from_seed(p, cfg["key_seed"], 0)
    out = torch.empty((B, p["n"] + 1), dtype=torch.int32, device=dev)
    ws = tfhe.alloc_workspace(ek, B)
    stream = torch.cuda.current_stream()
    tv_h = None
    if cfg["kind"] == "gate":
        a, b = wl.gate_inputs(cfg["input_seed"], B)
        ca_h = tfhe.tfhe_encrypt_torus(sk, cfg["input_seed"], tfhe.encode_bits(a), 0)
        cb_h = tfhe.tfhe_encrypt_torus(sk, cfg["input_seed"], tfhe.encode_bits(b), B)
        ca, cb = tfhe.to_device(ca_h), tfhe.to_device(cb_h)
        step = lambda: tfhe.tfhe_gate_bootstrap_batch(ek, cfg["gate"], ca, cb, out=out, workspace=ws, stream=stream)
    else:
        # 3-bit messages m (encoded m / 16, one padding bit) looked up in a
        # seeded random 8-entry table by one programmable bootstrap each
        m = wl.messages(cfg["input_seed"], B, cfg["msg_bits"])
        table = wl.lut(cfg["input_seed"], cfg["msg_bits"])
        tv_h = tfhe.tfhe_lut_testvec(p["N"], cfg["msg_bits"], table)
        tv = tfhe.to_device(tv_h)
        shift = 31 - cfg["msg_bits"]
        ca_h, cb_h = tfhe.tfhe_encrypt_torus(sk, cfg["input_seed"], (m << shift).astype(np.uint32), 0), None
        ca = tfhe.to_device(ca_h)
        step = lambda: tfhe.tfhe_lut_bootstrap_batch(ek, ca, tv, out=out, workspace=ws, stream=stream)

    if args.copy_probe_mib:
        src = torch.empty(args.copy_probe_mib << 18, dtype=torch.int32, device=dev).fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    with ClockSampler(sclk_path()) as clock:
        # untimed steps first, so that the clock figure has settled (and the
        # GPU left its idle state) when the timed window starts
        t_settle = time.perf_counter()
        while time.perf_counter() - t_settle < args.settle:
            step()
            torch.cuda.synchronize()
        for _ in range(args.warmup):
            step()
        torch.cuda.synchronize()

        tfhe.tfhe_stage_timing(True)
        tfhe.tfhe_stage_times()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        ev[0].record(stream)
        for k in range(args.steps):
            step()
            ev[k + 1].record(stream)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
    step_ms = sorted(ev[k].elapsed_time(ev[k + 1]) for k in range(args.steps))
    stages = tfhe.tfhe_stage_times()
    tfhe.tfhe_stage_timing(False)

    elapsed = t1 - t0
    value = B * args.steps / elapsed
    res = tfhe.to_host(out)
    ph = tfhe.tfhe_decrypt_phase(sk, res).astype(np.int64)
    if cfg["kind"] == "gate":
        dec = (np.where(ph >= 1 << 31, ph - (1 << 32), ph) > 0).astype(np.uint8)
        truth_ok = bool(np.array_equal(dec, 1 - (a & b))) if cfg["gate"] == "NAND" else None
    else:
        truth_ok = bool(np.array_equal(((ph + (1 << (shift - 1))) >> shift) & ((2 << cfg["msg_bits"]) - 1), table[m]))

    br_ms, br_n = stages["blind_rotate"]
    br_s = br_ms / 1e3 / max(br_n, 1)
    parts, bound = tfhe.tfhe_transform_error_bound(p)
    ops = algorithmic_lane_ops(p, parts) * B
    achieved = ops / br_s
    digest = kernel_source_digest()
    traffic = measured_traffic(digest, args.config)
    timed_clock = clock.window(t0, t1)
    mhz = clock.mhz(t0, t1)
    props = torch.cuda.get_device_properties(0)
    line = {
        "metric": METRIC if cfg["kind"] == "gate" and p["N"] == 1024 else
                  f"{'gate' if cfg['kind'] == 'gate' else 'table-lookup'} bootstraps/sec "
                  f"(n={p['n']},N={p['N']}) + % of VALU roofline, 1 MI355X",
        "value": value,
        "unit": "bootstraps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": elapsed / args.steps * 1e3,
        "ms_per_step_median_events": step_ms[len(step_ms) // 2],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u32/f64",
        "data": "synthetic",
        "config": {"workload": args.config, "gate": cfg.get("gate", "lut%d" % cfg.get("msg_bits", 0)), "batch": B,
                   "n": p["n"], "N": p["N"], "l": p["l"], "bg_bit": p["bg_bit"], "ks_t": p["ks_t"],
                   "ks_basebit": p["ks_basebit"]},
        "roofline": {
            "bound": "alu",
            "kernel": "blind_rotate_kernel" if p["N"] <= 1024 else "blind_rotate_split_kernel",
            "achieved": achieved / 1e12,
            "peak": PEAK_LANE_OPS / 1e12,
            "unit": "T lane-op/s",
            "frac": achieved / PEAK_LANE_OPS,
            "traffic": traffic,
            "ops_per_bootstrap": algorithmic_lane_ops(p, parts),
            "launch_ms": br_s * 1e3,
            # the GPU's clock during the timed steps (the peak assumes 2.4 GHz)
            "clock_mhz": mhz,
            "clock_samples": len(timed_clock),
            "clock_mhz_range": [min(timed_clock), max(timed_clock)] if timed_clock else None,
            "frac_at_clock": achieved / (PEAK_LANE_OPS * mhz / 2400) if mhz else None,
        },
        "hbm": {
            "kernel": "blind_rotate_kernel" if p["N"] <= 1024 else "blind_rotate_split_kernel",
            "algorithmic_bytes_per_launch": algorithmic_bytes_br(p, B, parts),
            "algorithmic_GBps": algorithmic_bytes_br(p, B, parts) / br_s / 1e9,
            # HBM bytes from the committed rocprofv3 counters of this source
            # (FETCH_SIZE + WRITE_SIZE, calibrated on a device copy)
            "measured_bytes_per_launch": traffic,
            "measured_GBps": traffic / br_s / 1e9 if traffic else None,
            "measured_frac": traffic / br_s / PEAK_HBM if traffic else None,
            "peak_GBps": PEAK_HBM / 1e9,
        },
        "stage_ms_per_step": {k: (v[0] / max(v[1], 1)) for k, v in stages.items()},
        "truth_table_ok": truth_ok,
        "transform": {"key_parts": parts, "worst_case_error": bound},
        "kernel_source_digest": digest,
        "device": f"{torch.cuda.get_device_name(0)} ({getattr(props, 'gcnArchName', '?')}, "
                  f"{props.multi_processor_count} CUs)",
        # the paper's CPU timing of the same activation path (its own TFHE
        # parameters and hardware): context, not a baseline for this metric
        "paper_context": {"relu_unit_s": 0.1, "softmax_unit_s": 3.3, "bootstraps_per_relu_unit": 7,
                          "hardware": "Intel Xeon E7-8890 v4, 2.2 GHz, 2 sockets x 12 cores, single-core runs",
                          "source": "Section 3.1 (forward/backward ReLU, forward softmax), Section 4 setup"},
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(cfg, ca_h, cb_h, out, tv_h)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
