"""The allocation-free gate bootstrap (tfhe_gate_bootstrap_batch_noalloc),
called through the C ABI, against tfhe_gate_bootstrap_batch with a caller
workspace: two calls in a row on the library's shared device array, the
second with a smaller batch, give word-for-word the results of the
workspace entry point, and a batch beyond the array is refused."""
import ctypes
import sys

import numpy as np
import pytest

from paper_1911_07101_amd import tfhe, workloads as wl

pytestmark = pytest.mark.gpu


def say(msg):
    print(f"[no-alloc] {msg}", flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def torch():
    import torch as _t
    if not _t.cuda.is_available():
        pytest.skip("no GPU")
    return _t


def _bits(phase):
    p = phase.astype(np.int64)
    return (np.where(p >= 1 << 31, p - (1 << 32), p) > 0).astype(np.uint8)


@pytest.mark.parametrize("cfg_name", ["tfhe128_nand", "lut3_n2048"])
def test_noalloc_gate_bootstrap_matches_the_workspace_entry(torch, cfg_name):
    cfg = wl.CONFIGS[cfg_name]
    p = cfg["params"]
    say(f"keygen {cfg_name}")
    sk, ek = tfhe.tfhe_keygen_from_seed(p, cfg["key_seed"], 0)
    L = tfhe.lib()
    rng = np.random.default_rng(71)
    first = {"tfhe128_nand": 4096 + 3, "lut3_n2048": 2048 + 5}[cfg_name]
    for B, gate in ((first, "NAND"), (700, "XOR")):  # the second call smaller than the first
        a, b = rng.integers(0, 2, B), rng.integers(0, 2, B)
        ca = tfhe.to_device(tfhe.tfhe_encrypt_torus(sk, 72, tfhe.encode_bits(a), 0))
        cb = tfhe.to_device(tfhe.tfhe_encrypt_torus(sk, 72, tfhe.encode_bits(b), B))
        ref = torch.empty((B, p["n"] + 1), dtype=torch.int32, device="cuda:0")
        out = torch.full((B, p["n"] + 1), 7, dtype=torch.int32, device="cuda:0")
        ws = tfhe.alloc_workspace(ek, B)
        g = tfhe.GATES[gate]
        say(f"{cfg_name}: {B} {gate} gates, workspace entry then no-allocation entry")
        assert L.tfhe_gate_bootstrap_batch(ek.handle, g, tfhe._dptr(ca), tfhe._dptr(cb), tfhe._dptr(ref), B,
                                           tfhe._dptr(ws), ws.numel(), None) == tfhe.TFHE_OK
        assert L.tfhe_gate_bootstrap_batch_noalloc(ek.handle, g, tfhe._dptr(ca), tfhe._dptr(cb), tfhe._dptr(out),
                                                   B, None) == tfhe.TFHE_OK, L.tfhe_last_error()
        torch.cuda.synchronize()
        got, want = tfhe.to_host(out), tfhe.to_host(ref)
        assert np.array_equal(got, want), f"{int((got != want).any(axis=1).sum())} of {B} gates differ"
        truth = 1 - (a & b) if gate == "NAND" else a ^ b
        assert np.array_equal(_bits(tfhe.tfhe_decrypt_phase(sk, got)), truth)
    # the largest batch the array holds, and one more
    limit = tfhe.NOALLOC_SCRATCH_BYTES
    most = limit // ((p["n"] + 1) * 2 + (p["N"] + 1) * 4) + 2  # above the largest batch that fits
    while tfhe.tfhe_workspace_bytes(ek, most) > limit:
        most -= 1
    assert tfhe.tfhe_workspace_bytes(ek, most) <= limit < tfhe.tfhe_workspace_bytes(ek, most + 1)
    assert most == {"tfhe128_nand": 12515, "lut3_n2048": 6919}[cfg_name]  # the limits the header states
    big = torch.zeros((most + 1, p["n"] + 1), dtype=torch.int32, device="cuda:0")
    dst = torch.empty_like(big)
    rc = L.tfhe_gate_bootstrap_batch_noalloc(ek.handle, 0, tfhe._dptr(big), tfhe._dptr(big), tfhe._dptr(dst),
                                             most + 1, None)
    assert rc == tfhe.TFHE_EINVAL and "workspace" in L.tfhe_last_error().decode()
    say(f"{cfg_name}: a batch of {most + 1} refused, {most} fit")


def test_noalloc_gate_bootstrap_in_a_captured_graph(torch):
    """The entry point's purpose: a call recorded into a HIP graph (torch's
    graph capture on a side stream; the call allocates nothing and records
    no memory set) and replayed three times, with eager work and new inputs
    copied into the captured buffers between the replays, gives each time
    word for word what the workspace entry point gives on the same inputs
    (128-bit parameters, 3000 NAND gates: 8-wave blocks and a one-wave
    tail)."""
    cfg = wl.CONFIGS["tfhe128_nand"]
    p = cfg["params"]
    say("keygen tfhe128_nand (graph)")
    sk, ek = tfhe.tfhe_keygen_from_seed(p, cfg["key_seed"], 0)
    L = tfhe.lib()
    B = 3000
    rng = np.random.default_rng(73)

    def inputs(seed):
        a, b = rng.integers(0, 2, B), rng.integers(0, 2, B)
        ca = tfhe.tfhe_encrypt_torus(sk, seed, tfhe.encode_bits(a), 0)
        cb = tfhe.tfhe_encrypt_torus(sk, seed, tfhe.encode_bits(b), B)
        return a, b, ca, cb

    a, b, ca_h, cb_h = inputs(80)
    ca, cb = tfhe.to_device(ca_h), tfhe.to_device(cb_h)
    out = torch.zeros((B, p["n"] + 1), dtype=torch.int32, device="cuda:0")
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    nand = tfhe.GATES["NAND"]
    with torch.cuda.stream(side):  # eager call first: the array's address is looked up outside the capture
        assert L.tfhe_gate_bootstrap_batch_noalloc(ek.handle, nand, tfhe._dptr(ca), tfhe._dptr(cb), tfhe._dptr(out),
                                                   B, ctypes.c_void_p(side.cuda_stream)) == tfhe.TFHE_OK
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    say("capture")
    with torch.cuda.graph(graph, stream=side):
        rc = L.tfhe_gate_bootstrap_batch_noalloc(ek.handle, nand, tfhe._dptr(ca), tfhe._dptr(cb), tfhe._dptr(out),
                                                 B, ctypes.c_void_p(side.cuda_stream))
    assert rc == tfhe.TFHE_OK, L.tfhe_last_error()
    for replay in range(3):
        if replay:
            a, b, ca_h, cb_h = inputs(80 + replay)
            ca.copy_(tfhe.to_device(ca_h))
            cb.copy_(tfhe.to_device(cb_h))
        out.fill_(0)  # eager work between the replays
        torch.cuda.synchronize()
        say(f"replay {replay}")
        graph.replay()
        torch.cuda.synchronize()
        ref = tfhe.to_host(tfhe.tfhe_gate_bootstrap_batch(ek, "NAND", ca, cb))
        got = tfhe.to_host(out)
        assert np.array_equal(got, ref), f"replay {replay}: {int((got != ref).any(axis=1).sum())} of {B} gates differ"
        assert np.array_equal(_bits(tfhe.tfhe_decrypt_phase(sk, got)), 1 - (a & b))
