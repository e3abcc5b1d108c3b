"""GPU parity: the HIP path, called through the C ABI, against the CPU oracle.

All arithmetic is mod 2^32 and exact, so every comparison is bit for bit.
Inputs are seeded synthetic plaintexts (paper_1911_07101_amd.workloads); each
side generates keys and ciphertexts itself from the same seeds (the library's
key generation is checked byte-identical to the oracle's on the CPU).
"""
import os
import sys
import time

import numpy as np
import pytest

import oracle
from paper_1911_07101_amd import tfhe, workloads as wl

pytestmark = pytest.mark.gpu

M32 = 1 << 32
MU = 1 << 29
TRUTH = {"NAND": lambda a, b: 1 - (a & b), "AND": lambda a, b: a & b, "OR": lambda a, b: a | b,
         "NOR": lambda a, b: 1 - (a | b), "XOR": lambda a, b: a ^ b, "XNOR": lambda a, b: 1 - (a ^ b),
         "ANDNY": lambda a, b: (1 - a) & b, "ANDYN": lambda a, b: a & (1 - b),
         "ORNY": lambda a, b: (1 - a) | b, "ORYN": lambda a, b: a | (1 - b)}


def say(msg):
    print(f"[gpu-parity] {msg}", flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def torch():
    import torch as _t
    if not _t.cuda.is_available():
        pytest.skip("no GPU")
    return _t


def s32(x):
    x = np.asarray(x, dtype=np.int64) % M32
    return np.where(x >= M32 // 2, x - M32, x)


def bits_of(phase):
    return (s32(phase) > 0).astype(np.uint8)


_KEYS = {}


def keys_for(cfg_name, torch, params=None, seed=None):
    """(library secret key, library eval key, oracle keys) for a config."""
    params = params or wl.CONFIGS[cfg_name]["params"]
    seed = seed if seed is not None else wl.CONFIGS[cfg_name]["key_seed"]
    k = (cfg_name, tuple(sorted(params.items())), seed)
    if k not in _KEYS:
        say(f"keygen {cfg_name} n={params['n']} N={params['N']} seed={seed:#x}")
        sk, ek = tfhe.tfhe_keygen_from_seed(params, seed, 0)
        ok = oracle.Keys(params, seed)
        _KEYS[k] = (sk, ek, ok)
    return _KEYS[k]


# ------------------------------------------------------------ transform

PRODUCT_PARAMS = {
    256: dict(n=4, N=256, l=3, bg_bit=7, ks_t=2, ks_basebit=2, alpha_lwe=0.0, alpha_bk=0.0),
    512: dict(n=4, N=512, l=3, bg_bit=7, ks_t=2, ks_basebit=2, alpha_lwe=0.0, alpha_bk=0.0),
    1024: dict(n=4, N=1024, l=3, bg_bit=7, ks_t=2, ks_basebit=2, alpha_lwe=0.0, alpha_bk=0.0),
    2048: dict(n=4, N=2048, l=2, bg_bit=10, ks_t=2, ks_basebit=2, alpha_lwe=0.0, alpha_bk=0.0),
}


@pytest.mark.parametrize("N", [256, 512, 1024, 2048])
def test_negacyclic_product_exact(torch, N):
    """The fp64 transform product, rounded, equals the schoolbook product mod
    2^32, including inputs at the extremes of the error bound."""
    p = PRODUCT_PARAMS[N]
    _, ek, _ = keys_for(f"product{N}", torch, p, 7)
    half = 1 << (p["bg_bit"] - 1)
    rng = np.random.default_rng(N)
    B = 7  # more than one block of polynomials and a ragged tail
    d = rng.integers(-half, half, (B, N)).astype(np.int32)
    b = rng.integers(0, M32, (B, N), dtype=np.uint64).astype(np.uint32)
    # extremes: all digits -Bg/2 against coefficients whose signed key parts
    # (16-bit halves, or 11-bit thirds where the library needs three parts)
    # are all at their largest magnitude with one sign, and alternating digit signs
    parts, _ = tfhe.tfhe_transform_error_bound(p)
    if parts == 2:
        ext_neg, ext_pos = -(1 << 31), (1 << 31) - (1 << 15)          # halves (-2^15, 0), (2^15, -2^15)
    else:
        ext_neg = -1024 - 1024 * 2**11 - 511 * 2**22                   # thirds (-1024, -1024, -511)
        ext_pos = 1023 + 1023 * 2**11 + 511 * 2**22                    # thirds (1023, 1023, 511)
    d[0] = -half
    b[0] = np.uint32(ext_neg % M32)
    d[1] = -half
    b[1] = np.uint32(ext_pos % M32)
    d[2] = np.where(np.arange(N) % 2 == 0, -half, half - 1)
    b[2] = np.where(np.arange(N) % 2 == 0, ext_neg % M32, ext_pos % M32).astype(np.uint32)
    d[3] = half - 1
    b[3] = np.uint32(ext_neg % M32)
    say(f"negacyclic product N={N} B={B}")
    out = tfhe.to_host(tfhe.tfhe_negacyclic_mul_batch(ek, torch.from_numpy(d).cuda(), tfhe.to_device(b)))
    torch.cuda.synchronize()
    for k in range(B):
        ref = oracle.negacyclic_mul((d[k].astype(np.int64) % M32).astype(np.uint32), b[k])
        assert np.array_equal(out[k], ref), f"polynomial {k}"


# ------------------------------------------------------------ stages (toy)

def test_blind_rotate_extract_parity_toy(torch):
    p = wl.CONFIGS["toy"]["params"]
    sk, ek, ok = keys_for("toy", torch)
    rng = np.random.default_rng(11)
    B = 37  # spans several blocks and a ragged tail
    x = rng.integers(0, M32, (B, p["n"] + 1), dtype=np.uint64).astype(np.uint32)
    x[0, :p["n"]] = 0  # a trivial sample (never rotated)
    x[1, :] = 0
    tv_gate = oracle.gate_testvec(p["N"])
    say(f"blind rotate + extract toy B={B} (gate polynomial)")
    got = tfhe.to_host(tfhe.tfhe_bootstrap_extract_batch(ek, tfhe.to_device(x)))
    ref = oracle.bootstrap_no_ks(ok, x, tv_gate)
    assert np.array_equal(got, ref)
    tv = rng.integers(0, M32, p["N"], dtype=np.uint64).astype(np.uint32)
    say("blind rotate + extract toy with an arbitrary test polynomial")
    got = tfhe.to_host(tfhe.tfhe_bootstrap_extract_batch(ek, tfhe.to_device(x), tfhe.to_device(tv)))
    assert np.array_equal(got, oracle.bootstrap_no_ks(ok, x, tv))


@pytest.mark.parametrize("cfg_name", ["toy", "tfhe128_nand", "lut3_n2048"])
def test_rotation_edges(torch, cfg_name):
    """Degenerate rotation amounts through blind rotation and extraction, bit
    for bit against the oracle: bodies whose switched value b is 0, 1, N - 1,
    N, N + 1 or 2N - 1 (every b in [0, 2N) at N = 256), the rotation by
    X^N = -1 flipping signs and by X^0 leaving the accumulator unchanged, and
    mask words whose switched values a_i take the same edge values."""
    p = wl.CONFIGS[cfg_name]["params"]
    n, N = p["n"], p["N"]
    sk, ek, ok = keys_for(cfg_name, torch)
    rng = np.random.default_rng(31)
    step = (1 << 32) // (2 * N)  # ms(k * step) = k
    edges = [0, 1, 2, N - 2, N - 1, N, N + 1, N + 2, 2 * N - 2, 2 * N - 1]
    bodies = list(range(2 * N)) if N <= 256 else edges + [int(v) for v in rng.integers(0, 2 * N, 6)]
    # at n = 630 and N = 2048 the edge samples sit at spread rows of a batch
    # one ragged block past a full round of the timed launch shape (blocks of
    # 8 ciphertexts at N = 1024, 4 at N = 2048); the oracle checks those rows
    B = {"toy": len(bodies), "tfhe128_nand": 2048 + 5, "lut3_n2048": 1024 + 3}[cfg_name]
    rows = np.linspace(0, B - 1, len(bodies)).astype(int)
    assert len(set(rows.tolist())) == len(bodies)
    x = rng.integers(0, M32, (B, n + 1), dtype=np.uint64).astype(np.uint32)
    for k, c in enumerate(rows):
        x[c, n] = bodies[k] * step
        for i in range(len(edges)):
            x[c, i] = edges[(i + k) % len(edges)] * step
    say(f"rotation edges {cfg_name} N={N} B={B}, {len(rows)} rows checked")
    got = tfhe.to_host(tfhe.tfhe_bootstrap_extract_batch(ek, tfhe.to_device(x)))
    assert np.array_equal(got[rows], oracle.bootstrap_no_ks(ok, x[rows], oracle.gate_testvec(N)))


@pytest.mark.parametrize("cfg_name", ["toy", "tfhe128_nand"])
def test_modulus_switch_ties(torch, cfg_name):
    """The modulus switch rounds half up: words exactly half a step of
    2^32 / 2N above a multiple (ties, which round up), one below a tie (round
    down), and 2^32 minus half a step (rounds to 2N, i.e. 0) in every mask
    word and body, through blind rotation and extraction, bit for bit against
    the oracle (timed launch shape at n = 630, oracle-checked rows)."""
    p = wl.CONFIGS[cfg_name]["params"]
    n, N = p["n"], p["N"]
    sk, ek, ok = keys_for(cfg_name, torch)
    rng = np.random.default_rng(43)
    step = (1 << 32) // (2 * N)
    B = {"toy": 61, "tfhe128_nand": 2048 + 5}[cfg_name]
    rows = np.arange(B) if B < 100 else np.linspace(0, B - 1, 8).astype(int)
    k = rng.integers(0, 2 * N, (B, n + 1))
    kind = rng.integers(0, 3, (B, n + 1))
    x = np.where(kind == 0, k * step + step // 2,                      # tie: rounds up to k + 1
                 np.where(kind == 1, k * step + step // 2 - 1,         # just below: k
                          (1 << 32) - step // 2)).astype(np.uint64).astype(np.uint32)  # wraps to 0
    say(f"modulus switch ties {cfg_name} B={B}, {len(rows)} rows checked")
    got = tfhe.to_host(tfhe.tfhe_bootstrap_extract_batch(ek, tfhe.to_device(x)))
    assert np.array_equal(got[rows], oracle.bootstrap_no_ks(ok, x[rows], oracle.gate_testvec(N)))


@pytest.mark.parametrize("cfg_name", ["tfhe128_nand", "lut3_n2048"])
def test_decomposition_edges(torch, cfg_name):
    """The signed gadget decomposition at its edges inside the blind rotation:
    with a constant test polynomial c, the accumulator starts as +-c in every
    coefficient, so the first CMux decomposes D = X^a ACC - ACC in {0, 2c, -2c}.
    c is chosen so that 2c is 2^31 (both signs alike), a rounding tie (half a
    step below the last digit, once and three times), every digit at Bg/2 - 1,
    or 2^32 minus half a step (rounds to 0).  Timed launch shape, oracle-checked
    rows, bit for bit."""
    p = wl.CONFIGS[cfg_name]["params"]
    n, N, l, bg = p["n"], p["N"], p["l"], p["bg_bit"]
    L = l * bg
    sk, ek, ok = keys_for(cfg_name, torch)
    rng = np.random.default_rng(41)
    step = (1 << 32) // (2 * N)
    top_digits = ((1 << (bg - 1)) - 1) * sum(1 << (31 - j * bg) for j in range(1, l + 1))
    cs = [1 << 30, 1 << (30 - L), 3 << (30 - L), top_digits, (1 << 31) - (1 << (30 - L))]
    B = {"tfhe128_nand": 2048 + 5, "lut3_n2048": 1024 + 3}[cfg_name]
    rows = np.linspace(0, B - 1, 6).astype(int)
    for c in cs:
        tv = np.full(N, c, np.uint32)
        x = rng.integers(0, M32, (B, n + 1), dtype=np.uint64).astype(np.uint32)
        x[:, n] = (rng.integers(0, 2 * N, B) * step).astype(np.uint32)
        say(f"decomposition edges {cfg_name}: c = {c:#010x}, B={B}, {len(rows)} rows checked")
        got = tfhe.to_host(tfhe.tfhe_bootstrap_extract_batch(ek, tfhe.to_device(x), tfhe.to_device(tv)))
        assert np.array_equal(got[rows], oracle.bootstrap_no_ks(ok, x[rows], tv)), hex(c)


# parameter sets whose transform bound needs the key in three parts: the
# three-part blind-rotation kernels (4 points per lane) at every ring size
THREE_PARTS = {
    256: dict(n=8, N=256, l=1, bg_bit=18, ks_t=8, ks_basebit=2, alpha_lwe=2**-15, alpha_bk=2**-25),
    512: dict(n=8, N=512, l=1, bg_bit=16, ks_t=8, ks_basebit=2, alpha_lwe=2**-15, alpha_bk=2**-25),
    1024: dict(n=8, N=1024, l=2, bg_bit=14, ks_t=8, ks_basebit=2, alpha_lwe=2**-15, alpha_bk=2**-25),
    2048: dict(n=8, N=2048, l=2, bg_bit=12, ks_t=8, ks_basebit=2, alpha_lwe=2**-15, alpha_bk=2**-25),
}


@pytest.mark.parametrize("N", sorted(THREE_PARTS))
def test_blind_rotate_extract_three_key_parts(torch, N):
    """Blind rotation + SampleExtract with the key split into three parts
    (one or more ciphertexts per wave at N <= 512, two waves per ciphertext at
    N = 1024, four at N = 2048): a small batch in full, and a batch large
    enough for the multi-ciphertext block shape, sampled, against the oracle."""
    p = THREE_PARTS[N]
    assert tfhe.tfhe_transform_error_bound(p)[0] == 3
    sk, ek, ok = keys_for(f"three-parts-{N}", torch, params=p, seed=0x3A3A + N)
    rng = np.random.default_rng(N)
    tv = rng.integers(0, M32, N, dtype=np.uint64).astype(np.uint32)
    for B, sample in ((5, None), (1030, np.array([0, 1, 513, 1029]))):
        x = rng.integers(0, M32, (B, p["n"] + 1), dtype=np.uint64).astype(np.uint32)
        say(f"three key parts N={N} B={B}")
        got = tfhe.to_host(tfhe.tfhe_bootstrap_extract_batch(ek, tfhe.to_device(x), tfhe.to_device(tv)))
        idx = np.arange(B) if sample is None else sample
        assert np.array_equal(got[idx], oracle.bootstrap_no_ks(ok, x[idx], tv))


@pytest.mark.parametrize("N", [256, 512, 1024])
@pytest.mark.parametrize("l,bg_bit", [(1, 10), (2, 9), (4, 6)])
def test_one_wave_kernel_ring_sizes_and_gadgets(torch, N, l, bg_bit):
    """The blind rotation with two key parts at N = 256, 512 and 1024 (N/16
    lanes per ciphertext) for gadgets other than the default: a small batch
    (every sample checked) and one that fills blocks of 8 waves on every CU
    plus a ragged block (spread rows checked), with an arbitrary test
    polynomial, bit for bit against the oracle."""
    params = dict(n=8, N=N, l=l, bg_bit=bg_bit, ks_t=8, ks_basebit=2, alpha_lwe=2 ** -15, alpha_bk=2 ** -25)
    assert tfhe.tfhe_transform_error_bound(params)[0] == 2
    sk, ek, ok = keys_for(f"ring{N}_l{l}_bg{bg_bit}", torch, params=params, seed=0x1024 + N + 16 * l + bg_bit)
    rng = np.random.default_rng(53 + N + l * bg_bit)
    tv = rng.integers(0, M32, N, dtype=np.uint64).astype(np.uint32)
    full = 256 * 8 * 64 // (N // 16) + 3  # 256 blocks of 8 waves, plus a ragged one
    for B, rows in ((7, np.arange(7)), (full, np.linspace(0, full - 1, 8).astype(int))):
        x = rng.integers(0, M32, (B, 9), dtype=np.uint64).astype(np.uint32)
        say(f"one-wave kernel N={N} l={l} bg_bit={bg_bit} B={B}")
        got = tfhe.to_host(tfhe.tfhe_bootstrap_extract_batch(ek, tfhe.to_device(x), tfhe.to_device(tv)))
        assert np.array_equal(got[rows], oracle.bootstrap_no_ks(ok, x[rows], tv)), B


@pytest.mark.parametrize("l,bg_bit", [(3, 7), (1, 10), (4, 6), (2, 11), (2, 9)])
def test_split_kernel_digit_paths(torch, l, bg_bit):
    """The two-wave blind rotation at N = 2048 with two key parts for other
    gadgets: digits recomputed from the accumulator for each digit (l != 2 or
    Bg > 2^10) and the second digit kept packed from the first (l = 2,
    Bg = 2^9), in blocks of one ciphertext (a small batch, every sample
    checked) and of four (1027 samples, spread rows checked), with an
    arbitrary test polynomial, bit for bit against the oracle."""
    params = dict(n=8, N=2048, l=l, bg_bit=bg_bit, ks_t=8, ks_basebit=2, alpha_lwe=2 ** -15, alpha_bk=2 ** -25)
    assert tfhe.tfhe_transform_error_bound(params)[0] == 2
    sk, ek, ok = keys_for(f"split_l{l}_bg{bg_bit}", torch, params=params, seed=0x5117 + 16 * l + bg_bit)
    rng = np.random.default_rng(47 + l * bg_bit)
    tv = rng.integers(0, M32, 2048, dtype=np.uint64).astype(np.uint32)
    for B, rows in ((5, np.arange(5)), (1027, np.linspace(0, 1026, 8).astype(int))):
        x = rng.integers(0, M32, (B, 9), dtype=np.uint64).astype(np.uint32)
        say(f"split kernel l={l} bg_bit={bg_bit} B={B}")
        got = tfhe.to_host(tfhe.tfhe_bootstrap_extract_batch(ek, tfhe.to_device(x), tfhe.to_device(tv)))
        assert np.array_equal(got[rows], oracle.bootstrap_no_ks(ok, x[rows], tv)), B


def test_parameter_and_batch_limits(torch):
    """The largest LWE dimension the library accepts (n = 4096, here with the
    toy ring) and a batch of 100,003 gates (many rounds of blocks and a
    ragged last block), sampled against the oracle; every output decrypts to
    its truth table."""
    p = dict(n=4096, N=256, l=3, bg_bit=7, ks_t=8, ks_basebit=2, alpha_lwe=2**-15, alpha_bk=2**-25)
    sk, ek, ok = keys_for("n-4096", torch, params=p, seed=0x4096)
    a, b = np.array([0, 1, 1, 0, 1]), np.array([1, 1, 0, 0, 1])
    ca = tfhe.tfhe_encrypt_torus(sk, 5, tfhe.encode_bits(a), 0)
    cb = tfhe.tfhe_encrypt_torus(sk, 5, tfhe.encode_bits(b), len(a))
    say("n = 4096, 5 NAND")
    got = tfhe.to_host(tfhe.tfhe_gate_bootstrap_batch(ek, "NAND", tfhe.to_device(ca), tfhe.to_device(cb)))
    assert np.array_equal(got, oracle.gate_bootstrap(ok, "NAND", ca, cb))
    assert np.array_equal(bits_of(tfhe.tfhe_decrypt_phase(sk, got)), 1 - (a & b))

    cfg = wl.CONFIGS["toy"]
    sk, ek, ok = keys_for("toy", torch)
    B = 100_003
    a, b = wl.gate_inputs(cfg["input_seed"] + 9, B)
    ca = tfhe.tfhe_encrypt_torus(sk, 9, tfhe.encode_bits(a), 0)
    cb = tfhe.tfhe_encrypt_torus(sk, 9, tfhe.encode_bits(b), B)
    say(f"toy, {B} NOR")
    got = tfhe.to_host(tfhe.tfhe_gate_bootstrap_batch(ek, "NOR", tfhe.to_device(ca), tfhe.to_device(cb)))
    assert np.array_equal(bits_of(tfhe.tfhe_decrypt_phase(sk, got)), 1 - (a | b))
    idx = np.array([0, 1, 4095, 4096, 65535, 65536, B - 2, B - 1])
    assert np.array_equal(got[idx], oracle.gate_bootstrap(ok, "NOR", ca[idx], cb[idx]))


def test_keyswitch_parity_toy(torch):
    p = wl.CONFIGS["toy"]["params"]
    sk, ek, ok = keys_for("toy", torch)
    rng = np.random.default_rng(12)
    for B in (1, 33, 70):
        x = rng.integers(0, M32, (B, p["N"] + 1), dtype=np.uint64).astype(np.uint32)
        say(f"keyswitch toy B={B}")
        got = tfhe.to_host(tfhe.tfhe_keyswitch_batch(ek, tfhe.to_device(x)))
        assert np.array_equal(got, oracle.keyswitch(ok, x))


@pytest.mark.parametrize("B", [4096 + 3, 8192 + 5])
def test_keyswitch_rounding_edges(torch, B):
    """Key switching at n = 630, N = 1024 (t = 8, base 4) on the matrix
    cores, ragged in both the sample tiles and the split of the coefficient
    range: coefficients at the rounding tie (half a step of 2^-16 rounds up),
    just below it, at 0, all digits 3, and at the wrap (2^32 - 2^15 and above
    round to 0), bit for bit against the oracle on spread rows."""
    p = wl.CONFIGS["tfhe128_nand"]["params"]
    N = p["N"]
    sk, ek, ok = keys_for("tfhe128_nand", torch)
    rng = np.random.default_rng(37)
    half = 1 << 15
    edges = [0, half, half - 1, 3 * half, (1 << 32) - half, (1 << 32) - half - 1, (1 << 32) - 1,
             0xFFFF0000, 0x55550000, 0xAAAA8000, 0x80000000, 0x7FFF8000]
    x = rng.integers(0, M32, (B, N + 1), dtype=np.uint64).astype(np.uint32)
    for c in range(0, B, 7):  # every 7th sample takes the edges at every coefficient
        x[c, :N] = np.array([edges[(i + c) % len(edges)] for i in range(N)], np.uint64).astype(np.uint32)
    rows = np.unique(np.concatenate([np.arange(0, B, 7)[:96], np.linspace(0, B - 1, 64).astype(int)]))
    say(f"keyswitch edges B={B}, {len(rows)} rows checked")
    got = tfhe.to_host(tfhe.tfhe_keyswitch_batch(ek, tfhe.to_device(x)))
    assert np.array_equal(got[rows], oracle.keyswitch(ok, x[rows]))


@pytest.mark.parametrize("B", [1, 127, 129, 1000, 8192 + 5])
def test_keyswitch_parity_n750(torch, B):
    """Key switching from N = 2048 to n = 750 (twelve 64-column tiles, the
    last holding 47 columns): every batch size the launcher splits the 2048
    coefficients differently for, from one sample (all coefficients spread
    over many blocks) to 8197; all rows up to 1000 samples, spread rows
    above."""
    p = wl.CONFIGS["lut3_n2048"]["params"]
    N = p["N"]
    sk, ek, ok = keys_for("lut3_n2048", torch)
    rng = np.random.default_rng(B)
    x = rng.integers(0, M32, (B, N + 1), dtype=np.uint64).astype(np.uint32)
    x[0, :N:5] = 0xFFFFFFFF  # all digits 3 and a wrap to 0
    rows = np.arange(B) if B <= 1000 else np.unique(np.linspace(0, B - 1, 96).astype(int))
    say(f"keyswitch n=750 B={B}, {len(rows)} rows checked")
    got = tfhe.to_host(tfhe.tfhe_keyswitch_batch(ek, tfhe.to_device(x)))
    assert got.shape == (B, p["n"] + 1)
    assert np.array_equal(got[rows], oracle.keyswitch(ok, x[rows]))


@pytest.mark.parametrize("ks_t,ks_basebit", [(4, 3), (16, 2), (2, 5)])
def test_keyswitch_parity_other_digit_sizes(torch, ks_t, ks_basebit):
    """The key switch for digit shapes other than t = 8, base 4 (the kernel's
    runtime-shaped variants, 32 and 64 key rows per coefficient)."""
    p = dict(wl.CONFIGS["toy"]["params"], n=40, ks_t=ks_t, ks_basebit=ks_basebit)
    sk, ek, ok = keys_for(f"ks{ks_t}x{ks_basebit}", torch, p, 3)
    rng = np.random.default_rng(ks_t * 10 + ks_basebit)
    x = rng.integers(0, M32, (45, p["N"] + 1), dtype=np.uint64).astype(np.uint32)
    say(f"keyswitch t={ks_t} basebit={ks_basebit}")
    got = tfhe.to_host(tfhe.tfhe_keyswitch_batch(ek, tfhe.to_device(x)))
    assert np.array_equal(got, oracle.keyswitch(ok, x))


@pytest.mark.parametrize("gate", list(TRUTH))
def test_gate_bootstrap_toy(torch, gate):
    cfg = wl.CONFIGS["toy"]
    p = cfg["params"]
    sk, ek, ok = keys_for("toy", torch)
    a, b = wl.gate_inputs(cfg["input_seed"], cfg["batch"])
    ca = tfhe.tfhe_encrypt_torus(sk, cfg["input_seed"], tfhe.encode_bits(a), 0)
    cb = tfhe.tfhe_encrypt_torus(sk, cfg["input_seed"], tfhe.encode_bits(b), len(a))
    oa = oracle.encrypt(p["n"], ok.s, cfg["input_seed"], p["alpha_lwe"], tfhe.encode_bits(a), 0)
    assert np.array_equal(ca, oa)
    say(f"gate {gate} toy B={len(a)}")
    got = tfhe.to_host(tfhe.tfhe_gate_bootstrap_batch(ek, gate, tfhe.to_device(ca), tfhe.to_device(cb)))
    ref = oracle.gate_bootstrap(ok, gate, ca, cb)
    assert np.array_equal(got, ref)
    assert np.array_equal(bits_of(oracle.phase(ok.s, got)), TRUTH[gate](a, b))


def test_not_gate(torch):
    rng = np.random.default_rng(3)
    x = rng.integers(0, M32, (9, 65), dtype=np.uint64).astype(np.uint32)
    got = tfhe.to_host(tfhe.tfhe_not_batch(tfhe.to_device(x)))
    assert np.array_equal(got, oracle.not_gate(x))


def test_determinism_and_batch_independence(torch):
    cfg = wl.CONFIGS["toy"]
    p = cfg["params"]
    sk, ek, ok = keys_for("toy", torch)
    rng = np.random.default_rng(5)
    B = 41
    a, b = rng.integers(0, 2, B), rng.integers(0, 2, B)
    ca = tfhe.to_device(tfhe.tfhe_encrypt_torus(sk, 1, tfhe.encode_bits(a), 0))
    cb = tfhe.to_device(tfhe.tfhe_encrypt_torus(sk, 1, tfhe.encode_bits(b), B))
    say("determinism toy")
    r1 = tfhe.to_host(tfhe.tfhe_gate_bootstrap_batch(ek, "XOR", ca, cb))
    r2 = tfhe.to_host(tfhe.tfhe_gate_bootstrap_batch(ek, "XOR", ca, cb))
    assert np.array_equal(r1, r2)
    parts = [tfhe.to_host(tfhe.tfhe_gate_bootstrap_batch(ek, "XOR", ca[s:e].contiguous(), cb[s:e].contiguous()))
             for s, e in [(0, 1), (1, 6), (6, 41)]]
    assert np.array_equal(np.concatenate(parts), r1)


def test_concurrent_calls_on_two_streams(torch):
    """Two calls in flight at once on two streams (default priority), each
    with its own workspace and output, give the results of the same calls
    made one after the other."""
    cfg = wl.CONFIGS["tfhe128_nand"]
    p = cfg["params"]
    sk, ek, ok = keys_for("tfhe128_nand", torch)
    rng = np.random.default_rng(23)
    B = 1024
    ins = []
    for k in range(2):
        a, b = rng.integers(0, 2, B), rng.integers(0, 2, B)
        ins.append((tfhe.to_device(tfhe.tfhe_encrypt_torus(sk, 40 + k, tfhe.encode_bits(a), 0)),
                    tfhe.to_device(tfhe.tfhe_encrypt_torus(sk, 40 + k, tfhe.encode_bits(b), B))))
    say("sequential reference, 2 x 1024 NAND")
    ref = [tfhe.to_host(tfhe.tfhe_gate_bootstrap_batch(ek, "NAND", ca, cb)) for ca, cb in ins]
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    outs = [torch.empty((B, p["n"] + 1), dtype=torch.int32, device="cuda") for _ in range(2)]
    wss = [tfhe.alloc_workspace(ek, B) for _ in range(2)]
    torch.cuda.synchronize()
    say("two streams at once")
    for k in range(2):
        with torch.cuda.stream(streams[k]):
            tfhe.tfhe_gate_bootstrap_batch(ek, "NAND", *ins[k], out=outs[k], workspace=wss[k], stream=streams[k])
    torch.cuda.synchronize()
    for k in range(2):
        assert np.array_equal(tfhe.to_host(outs[k]), ref[k])


def test_buffers_given_to_a_side_stream_are_not_reused_early(torch):
    """A buffer handed to a call on a caller-given stream is recorded on that
    stream: when Python drops it right after the call, torch's caching
    allocator does not give its memory to the next allocation on the default
    stream while the side stream still has work queued, and the call's
    result is that of the same call on the default stream."""
    p = wl.CONFIGS["toy"]["params"]
    sk, ek, ok = keys_for("toy", torch)
    B = 8
    size = tfhe.tfhe_workspace_bytes(ek, B)
    first = torch.empty(size, dtype=torch.uint8, device="cuda:0")
    ptr = first.data_ptr()
    del first
    again = torch.empty(size, dtype=torch.uint8, device="cuda:0")
    if again.data_ptr() != ptr:
        pytest.skip("the allocator does not hand a freed block of this size straight back")
    del again
    rng = np.random.default_rng(29)
    big = 16384
    busy = [tfhe.to_device(tfhe.tfhe_encrypt_torus(sk, 50, tfhe.encode_bits(rng.integers(0, 2, big)), k * big))
            for k in range(2)]
    a, b = rng.integers(0, 2, B), rng.integers(0, 2, B)
    ca = tfhe.to_device(tfhe.tfhe_encrypt_torus(sk, 51, tfhe.encode_bits(a), 0))
    cb = tfhe.to_device(tfhe.tfhe_encrypt_torus(sk, 51, tfhe.encode_bits(b), B))
    ref = tfhe.to_host(tfhe.tfhe_gate_bootstrap_batch(ek, "NAND", ca, cb))
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    say(f"side stream: {big} toy NAND gates, then {B} with a workspace dropped at once")
    tfhe.tfhe_gate_bootstrap_batch(ek, "NAND", *busy, stream=side)  # keeps the side stream busy
    ws = tfhe.alloc_workspace(ek, B)
    ptr = ws.data_ptr()
    out = tfhe.tfhe_gate_bootstrap_batch(ek, "NAND", ca, cb, workspace=ws, stream=side)
    del ws
    other = torch.empty(size, dtype=torch.uint8, device="cuda:0")
    still_busy = not side.query()
    reused = other.data_ptr() == ptr
    other.fill_(0xA5)  # a write on the default stream, where the workspace lived
    torch.cuda.synchronize()
    say(f"side stream busy at the allocation: {still_busy}; block handed back: {reused}")
    if still_busy:
        assert not reused
    assert np.array_equal(tfhe.to_host(out), ref)


def test_relu_toy_all_values(torch):
    """All 256 8-bit values through the ReLU unit on the toy parameters,
    streamed in uneven gate windows."""
    p = wl.CONFIGS["toy"]["params"]
    sk, ek, ok = keys_for("toy", torch)
    xs = np.arange(-128, 128)
    bits = wl.to_bits(xs, 8)
    ct = tfhe.tfhe_encrypt_torus(sk, 21, tfhe.encode_bits(bits.ravel())).reshape(256, 8, p["n"] + 1)
    x = tfhe.to_device(ct)
    y = torch.zeros_like(x)
    total = 256 * 7
    say("relu toy 256 values in 3 windows")
    for s, e in [(0, 5), (5, 1000), (1000, total)]:
        tfhe.glyph_relu_batch(ek, x, 8, y=y, gate_begin=s, gate_end=e)
    got = tfhe.to_host(y)
    ref = oracle.relu(ok, ct, 8)
    assert np.array_equal(got, ref)
    dec = bits_of(tfhe.tfhe_decrypt_phase(sk, got.reshape(-1, p["n"] + 1))).reshape(256, 8)
    assert np.array_equal(wl.from_bits(dec), np.maximum(xs, 0))


@pytest.mark.parametrize("bits", [2, 5, 16])
def test_relu_toy_other_widths(torch, bits):
    """The ReLU unit on values of other bit widths (the unit has bits - 1
    gates per value and a trivial sign), against the oracle and max(x, 0)."""
    p = wl.CONFIGS["toy"]["params"]
    sk, ek, ok = keys_for("toy", torch)
    rng = np.random.default_rng(200 + bits)
    lo, hi = -(1 << (bits - 1)), 1 << (bits - 1)
    xs = np.concatenate([[lo, -1, 0, hi - 1], rng.integers(lo, hi, 29)])
    ct = tfhe.tfhe_encrypt_torus(sk, 60 + bits, tfhe.encode_bits(wl.to_bits(xs, bits).ravel()))
    ct = ct.reshape(len(xs), bits, p["n"] + 1)
    say(f"relu toy {len(xs)} values of {bits} bits")
    got = tfhe.to_host(tfhe.glyph_relu_batch(ek, tfhe.to_device(ct), bits))
    assert np.array_equal(got, oracle.relu(ok, ct, bits))
    dec = bits_of(tfhe.tfhe_decrypt_phase(sk, got.reshape(-1, p["n"] + 1))).reshape(len(xs), bits)
    assert np.array_equal(wl.from_bits(dec), np.maximum(xs, 0))


def test_irelu_toy_all_4bit_pairs(torch):
    """Backward iReLU for every (4-bit u, 4-bit delta) pair on the toy
    parameters, in uneven gate windows: bit-exact with the oracle, and every
    output decrypts to delta where u >= 0, else 0."""
    p = wl.CONFIGS["toy"]["params"]
    sk, ek, ok = keys_for("toy", torch)
    us, ds = np.meshgrid(np.arange(-8, 8), np.arange(-8, 8), indexing="ij")
    us, ds = us.ravel(), ds.ravel()
    V = len(us)
    cu = tfhe.tfhe_encrypt_torus(sk, 31, tfhe.encode_bits(wl.to_bits(us, 4).ravel())).reshape(V, 4, p["n"] + 1)
    cd = tfhe.tfhe_encrypt_torus(sk, 32, tfhe.encode_bits(wl.to_bits(ds, 4).ravel())).reshape(V, 4, p["n"] + 1)
    u, d = tfhe.to_device(cu), tfhe.to_device(cd)
    y = torch.zeros_like(d)
    say(f"irelu toy {V} pairs in 3 windows")
    for s, e in [(0, 3), (3, 700), (700, V * 4)]:
        tfhe.glyph_irelu_batch(ek, u, d, out=y, gate_begin=s, gate_end=e)
    got = tfhe.to_host(y)
    assert np.array_equal(got, oracle.irelu(ok, cu, 4, cd, 4))
    dec = bits_of(tfhe.tfhe_decrypt_phase(sk, got.reshape(-1, p["n"] + 1))).reshape(V, 4)
    assert np.array_equal(wl.from_bits(dec), np.where(us >= 0, ds, 0))


def test_irelu_window_writes_only_its_gates(torch):
    """A call writes exactly the output words of its gate window."""
    p = wl.CONFIGS["toy"]["params"]
    sk, ek, ok = keys_for("toy", torch)
    V, bits = 9, 5
    rng = np.random.default_rng(5)
    cu = tfhe.tfhe_encrypt_torus(sk, 33, tfhe.encode_bits(rng.integers(0, 2, V * 3))).reshape(V, 3, p["n"] + 1)
    cd = tfhe.tfhe_encrypt_torus(sk, 34, tfhe.encode_bits(rng.integers(0, 2, V * bits))).reshape(V, bits, p["n"] + 1)
    y = torch.full((V, bits, p["n"] + 1), -1, dtype=torch.int32, device="cuda:0")
    tfhe.glyph_irelu_batch(ek, tfhe.to_device(cu), tfhe.to_device(cd), out=y, gate_begin=7, gate_end=23)
    got = tfhe.to_host(y).reshape(V * bits, p["n"] + 1)
    assert np.all(got[:7] == M32 - 1) and np.all(got[23:] == M32 - 1)
    assert np.array_equal(got[7:23], oracle.irelu_gates(ok, cu, 3, cd, bits, np.arange(7, 23)))


def test_mux_toy(torch):
    """Multiplexers on random encrypted bits: bit-exact with the oracle and
    decrypting to c ? a : b."""
    p = wl.CONFIGS["toy"]["params"]
    sk, ek, ok = keys_for("toy", torch)
    B = 37
    rng = np.random.default_rng(23)
    bits = rng.integers(0, 2, (3, B))
    cts = [tfhe.tfhe_encrypt_torus(sk, 40 + k, tfhe.encode_bits(bits[k])) for k in range(3)]
    say(f"mux toy B={B}")
    got = tfhe.to_host(tfhe.tfhe_mux_batch(ek, *[tfhe.to_device(c) for c in cts]))
    assert np.array_equal(got, oracle.mux(ok, *cts))
    assert np.array_equal(bits_of(tfhe.tfhe_decrypt_phase(sk, got)), np.where(bits[0] == 1, bits[1], bits[2]))


@pytest.mark.parametrize("msg_bits,out_bits", [(1, 3), (2, 2), (3, 3), (4, 2)])
def test_mux_lut_toy(torch, msg_bits, out_bits):
    """Multiplexer-tree table lookup over every input, repeated into a ragged
    batch: bit-exact with the oracle and decrypting to the table entry."""
    p = wl.CONFIGS["toy"]["params"]
    sk, ek, ok = keys_for("toy", torch)
    rng = np.random.default_rng(100 + msg_bits)
    table = rng.integers(0, 1 << out_bits, 1 << msg_bits).astype(np.uint32)
    xs = np.resize(np.arange(1 << msg_bits), 19)
    ct = tfhe.tfhe_encrypt_torus(sk, 50 + msg_bits, tfhe.encode_bits(wl.to_bits(xs, msg_bits).ravel()))
    ct = ct.reshape(len(xs), msg_bits, p["n"] + 1)
    say(f"mux lut toy msg_bits={msg_bits} out_bits={out_bits} V={len(xs)}")
    got = tfhe.to_host(tfhe.glyph_mux_lut_batch(ek, tfhe.to_device(ct), table, out_bits))
    assert np.array_equal(got, oracle.mux_lut(ok, ct, msg_bits, table, out_bits))
    dec = bits_of(tfhe.tfhe_decrypt_phase(sk, got.reshape(-1, p["n"] + 1))).reshape(len(xs), out_bits)
    assert np.array_equal((dec.astype(np.int64) << np.arange(out_bits)).sum(axis=1), table[xs])


def test_pack_keyswitch_toy(torch):
    """Packing key switching of B = 3 sets of LWE samples (Z = N, a ragged
    100 and 1) into TRLWE samples: bit-exact with the oracle, and coefficient
    z of the phase decodes to message z."""
    p = wl.CONFIGS["toy"]["params"]
    sk, ek, ok = keys_for("toy", torch)
    tfhe.tfhe_packing_key_upload(sk, ek)
    rng = np.random.default_rng(61)
    for Z in (p["N"], 100, 1):
        B = 3
        m = rng.integers(0, 64, (B, Z)).astype(np.uint32)
        lwe = tfhe.tfhe_encrypt_torus(sk, 60 + Z, (m.ravel() << 26).astype(np.uint32)).reshape(B, Z, p["n"] + 1)
        say(f"pack keyswitch toy B={B} Z={Z}")
        got = tfhe.to_host(tfhe.tfhe_pack_keyswitch_batch(ek, tfhe.to_device(lwe)))
        for b in range(B):
            assert np.array_equal(got[b], oracle.pack_keyswitch(ok, lwe[b])), (Z, b)
            ext = np.stack([oracle.sample_extract_at(got[b], z) for z in range(Z)])
            ph = oracle.phase(ok.S, ext).astype(np.int64)
            assert np.array_equal(((ph + (1 << 25)) >> 26) % 64, m[b])



@pytest.mark.parametrize("B,Z,check", [(9, 1000, (0, 8)), (3, 517, (2,))])
def test_pack_keyswitch_transform_128bit(torch, B, Z, check):
    """Packing key switching at the 128-bit parameters on the transform
    path: nine outputs (a block of eight and a ragged block of one) and three
    outputs in one-wave blocks, Z samples each; the checked outputs bit-exact
    with the oracle, and every coefficient z of every output decodes to
    message z."""
    p = wl.CONFIGS["tfhe128_nand"]["params"]
    sk, ek, ok = keys_for("tfhe128_nand", torch)
    tfhe.tfhe_packing_key_upload(sk, ek)
    m = np.random.default_rng(70 + B).integers(0, 16, (B, Z)).astype(np.uint32)
    lwe = tfhe.tfhe_encrypt_torus(sk, 70 + B, (m.ravel() << 28).astype(np.uint32)).reshape(B, Z, p["n"] + 1)
    say(f"pack keyswitch 128-bit B={B} Z={Z}")
    got = tfhe.tfhe_pack_keyswitch_batch(ek, tfhe.to_device(lwe))
    ext = tfhe.to_host(tfhe.tfhe_sample_extract_batch(got, Z))
    ph = tfhe.tfhe_decrypt_phase(sk, ext, key_kind=1).astype(np.int64)
    assert np.array_equal(((ph + (1 << 27)) >> 28) % 16, m)
    got = tfhe.to_host(got)
    for b in check:
        assert np.array_equal(got[b], oracle.pack_keyswitch(ok, lwe[b])), b



@pytest.mark.parametrize("N,ks_t,ks_basebit,B,Z", [(512, 4, 2, 5, 300), (1024, 12, 1, 9, 77)])
def test_pack_keyswitch_transform_shapes(torch, N, ks_t, ks_basebit, B, Z):
    """The transform path of the packing key switch at other ring sizes and
    digit shapes: one-wave blocks of two outputs at N = 512 with base-4
    digits, and blocks of eight outputs at N = 1024 with base-2 digits (one
    key entry per digit), ragged batches, every output bit-exact with the
    oracle."""
    p = dict(wl.CONFIGS["toy"]["params"], n=40, N=N, ks_t=ks_t, ks_basebit=ks_basebit)
    sk, ek, ok = keys_for(f"pack{N}t{ks_t}b{ks_basebit}", torch, p, 0x9A00 + N + ks_t)
    tfhe.tfhe_packing_key_upload(sk, ek)
    m = np.random.default_rng(N + ks_t).integers(0, 16, (B, Z)).astype(np.uint32)
    lwe = tfhe.tfhe_encrypt_torus(sk, 80 + ks_t, (m.ravel() << 28).astype(np.uint32)).reshape(B, Z, p["n"] + 1)
    say(f"pack keyswitch N={N} t={ks_t} basebit={ks_basebit} B={B} Z={Z}")
    got = tfhe.to_host(tfhe.tfhe_pack_keyswitch_batch(ek, tfhe.to_device(lwe)))
    for b in range(B):
        assert np.array_equal(got[b], oracle.pack_keyswitch(ok, lwe[b])), b

def test_pack_keyswitch_n2048(torch):
    """Packing key switching at N = 2048 (n = 750), which takes the
    coefficient-domain kernel: two outputs of 37 samples, bit-exact with the
    oracle."""
    p = wl.CONFIGS["lut3_n2048"]["params"]
    sk, ek, ok = keys_for("lut3_n2048", torch)
    tfhe.tfhe_packing_key_upload(sk, ek)
    B, Z = 2, 37
    m = np.random.default_rng(73).integers(0, 16, (B, Z)).astype(np.uint32)
    lwe = tfhe.tfhe_encrypt_torus(sk, 73, (m.ravel() << 28).astype(np.uint32)).reshape(B, Z, p["n"] + 1)
    say(f"pack keyswitch n=750 N=2048 B={B} Z={Z}")
    got = tfhe.to_host(tfhe.tfhe_pack_keyswitch_batch(ek, tfhe.to_device(lwe)))
    for b in range(B):
        assert np.array_equal(got[b], oracle.pack_keyswitch(ok, lwe[b])), b

def test_sample_extract_batch(torch):
    """SampleExtract of the first K coefficients of random TRLWE samples
    equals the oracle's extraction of each coefficient."""
    rng = np.random.default_rng(62)
    for N, B, K in [(256, 5, 256), (1024, 3, 7), (2048, 2, 1)]:
        acc = rng.integers(0, M32, (B, 2, N), dtype=np.uint64).astype(np.uint32)
        got = tfhe.to_host(tfhe.tfhe_sample_extract_batch(tfhe.to_device(acc), K))
        for b in range(B):
            ref = np.stack([oracle.sample_extract_at(acc[b], i) for i in range(K)])
            assert np.array_equal(got[b], ref), (N, b)


def test_bootstrap_onto_multiples_of_inverse_modulus_n2048(torch):
    """Step 4 of the switch with the N = 2048 parameters: a programmable
    bootstrap whose test polynomial holds multiples of 1/q (q = 257) maps
    each 3-bit message m to f(m)/q; bit-exact with the oracle on a sample and
    decoding to f(m) for all 512 inputs (before key switching)."""
    cfg = wl.CONFIGS["lut3_n2048"]
    p = cfg["params"]
    sk, ek, ok = keys_for("lut3_n2048", torch)
    q = 257
    f = np.random.default_rng(63).integers(0, q, 8)
    values = np.array([(int(v) * (1 << 32) + q // 2) // q for v in f], dtype=np.uint64).astype(np.uint32)
    tv = tfhe.tfhe_torus_testvec(p["N"], 3, values)
    assert np.array_equal(tv, oracle.torus_testvec(p["N"], 3, values))
    m = np.arange(8, dtype=np.uint32).repeat(64)
    ct = tfhe.tfhe_encrypt_torus(sk, 64, (m << 28).astype(np.uint32))
    say("bootstrap onto multiples of 1/257, N=2048, 512 samples")
    got = tfhe.to_host(tfhe.tfhe_bootstrap_extract_batch(ek, tfhe.to_device(ct), tfhe.to_device(tv)))
    ph = tfhe.tfhe_decrypt_phase(sk, got, 1).astype(np.int64)
    assert np.array_equal(((ph * q + (1 << 31)) >> 32) % q, f[m])
    idx = np.array([0, 100, 301, 511])
    assert np.array_equal(got[idx], oracle.bootstrap_no_ks(ok, ct[idx], tv))


# ---------------------------------------------------- full-size workloads

@pytest.mark.parametrize("msg_bits", [1, 2, 3])
def test_lut_bootstrap_n1024(torch, msg_bits):
    """Table-lookup bootstraps (+ key switching) at the 128-bit parameters
    (N = 1024) with 1-, 2- and 3-bit tables: bit for bit against the oracle,
    and every output decrypts to its table entry (a 3-bit output's half box,
    1/32, is ~6.7 output standard deviations at these parameters)."""
    cfg = wl.CONFIGS["tfhe128_nand"]
    p = cfg["params"]
    sk, ek, ok = keys_for("tfhe128_nand", torch)
    rng = np.random.default_rng(300 + msg_bits)
    M = 1 << msg_bits
    table = rng.integers(0, M, M).astype(np.uint32)
    m = np.resize(np.arange(M), 67).astype(np.uint32)
    tv = tfhe.tfhe_lut_testvec(p["N"], msg_bits, table)
    assert np.array_equal(tv, oracle.lut_testvec(p["N"], msg_bits, table))
    shift = 31 - msg_bits
    ct = tfhe.tfhe_encrypt_torus(sk, 70 + msg_bits, (m << shift).astype(np.uint32))
    say(f"lut bootstrap N=1024 msg_bits={msg_bits} B={len(m)}")
    got = tfhe.to_host(tfhe.tfhe_lut_bootstrap_batch(ek, tfhe.to_device(ct), tfhe.to_device(tv)))
    ph = tfhe.tfhe_decrypt_phase(sk, got).astype(np.int64)
    assert np.array_equal(((ph + (1 << (shift - 1))) >> shift) & (2 * M - 1), table[m])
    idx = np.array([0, 1, M - 1, len(m) - 1])
    assert np.array_equal(got[idx], oracle.lut_bootstrap(ok, ct[idx], tv))


@pytest.mark.parametrize("gate", list(TRUTH))
def test_gate_bootstrap_128bit(torch, gate):
    """Every gate at the 128-bit parameters: all outputs decrypt to the truth
    table, a sample matches the oracle bit for bit."""
    p = wl.CONFIGS["tfhe128_nand"]["params"]
    sk, ek, ok = keys_for("tfhe128_nand", torch)
    rng = np.random.default_rng(400 + list(TRUTH).index(gate))
    B = 96
    a, b = rng.integers(0, 2, B), rng.integers(0, 2, B)
    ca = tfhe.tfhe_encrypt_torus(sk, 80, tfhe.encode_bits(a), 0)
    cb = tfhe.tfhe_encrypt_torus(sk, 80, tfhe.encode_bits(b), B)
    say(f"{gate} 128-bit B={B}")
    got = tfhe.to_host(tfhe.tfhe_gate_bootstrap_batch(ek, gate, tfhe.to_device(ca), tfhe.to_device(cb)))
    assert np.array_equal(bits_of(tfhe.tfhe_decrypt_phase(sk, got)), TRUTH[gate](a, b))
    idx = np.array([0, 37, B - 1])
    assert np.array_equal(got[idx], oracle.gate_bootstrap(ok, gate, ca[idx], cb[idx]))


def test_tfhe128_nand_4096(torch):
    cfg = wl.CONFIGS["tfhe128_nand"]
    p = cfg["params"]
    sk, ek, ok = keys_for("tfhe128_nand", torch)
    a, b = wl.gate_inputs(cfg["input_seed"], cfg["batch"])
    ca = tfhe.tfhe_encrypt_torus(sk, cfg["input_seed"], tfhe.encode_bits(a), 0)
    cb = tfhe.tfhe_encrypt_torus(sk, cfg["input_seed"], tfhe.encode_bits(b), len(a))
    say(f"NAND n=630 N=1024 B={len(a)}")
    t0 = time.time()
    got = tfhe.to_host(tfhe.tfhe_gate_bootstrap_batch(ek, "NAND", tfhe.to_device(ca), tfhe.to_device(cb)))
    say(f"  gpu {time.time() - t0:.2f}s")
    assert np.array_equal(bits_of(tfhe.tfhe_decrypt_phase(sk, got)), 1 - (a & b))
    idx = wl.sample_indices(cfg["input_seed"], len(a), cfg["sample"])
    t0 = time.time()
    ref = oracle.gate_bootstrap(ok, "NAND", ca[idx], cb[idx])
    say(f"  oracle sample of {len(idx)} in {time.time() - t0:.1f}s")
    assert np.array_equal(got[idx], ref)


def test_block_shapes_for_small_batches(torch):
    """A batch that four one-wave blocks per CU hold (N = 1024: up to 1024
    gates) runs in blocks of one wave, a larger one in blocks of 8; at
    N = 2048 up to two one-ciphertext blocks per CU (512 lookups) run one
    wave per SIMD, up to three (768) with two, else blocks of four
    ciphertexts, whose partly filled last round runs as one-ciphertext
    blocks of either kind (1102 = 1024 + 78, 1600 = 1024 + 576).  Both sides
    of each boundary, with a ragged last block, give the same samples as the
    full batch, and the last sample of each size matches the oracle."""
    for name, sizes in (("tfhe128_nand", (2100, 1025, 1024, 600, 7)),
                        ("lut3_n2048", (1600, 1102, 769, 768, 513, 512, 100))):
        cfg = wl.CONFIGS[name]
        p = cfg["params"]
        sk, ek, ok = keys_for(name, torch)
        if name == "tfhe128_nand":
            a, b = wl.gate_inputs(cfg["input_seed"], cfg["batch"])
            ca = tfhe.tfhe_encrypt_torus(sk, cfg["input_seed"], tfhe.encode_bits(a), 0)
            cb = tfhe.tfhe_encrypt_torus(sk, cfg["input_seed"], tfhe.encode_bits(b), len(a))
            run = lambda B: tfhe.to_host(tfhe.tfhe_gate_bootstrap_batch(
                ek, "NAND", tfhe.to_device(ca[:B]), tfhe.to_device(cb[:B])))
            ref_of = lambda idx: oracle.gate_bootstrap(ok, "NAND", ca[idx], cb[idx])
        else:
            m = wl.messages(cfg["input_seed"], cfg["batch"], cfg["msg_bits"])
            tv = tfhe.tfhe_lut_testvec(p["N"], cfg["msg_bits"], wl.lut(cfg["input_seed"], cfg["msg_bits"]))
            ct = tfhe.tfhe_encrypt_torus(sk, cfg["input_seed"], (m << 28).astype(np.uint32))
            run = lambda B: tfhe.to_host(tfhe.tfhe_lut_bootstrap_batch(ek, tfhe.to_device(ct[:B]), tfhe.to_device(tv)))
            ref_of = lambda idx: oracle.lut_bootstrap(ok, ct[idx], tv)
        say(f"block shapes {name} B={max(sizes)}")
        full = run(max(sizes))
        for B in sizes:
            say(f"  B={B}")
            assert np.array_equal(run(B), full[:B])
        say("  oracle: last sample of each size")
        idx = np.array([B - 1 for B in sizes])
        assert np.array_equal(full[idx], ref_of(idx))


def test_mlp_relu_7680(torch):
    cfg = wl.CONFIGS["mlp_relu"]
    p = cfg["params"]
    sk, ek, ok = keys_for("tfhe128_nand", torch)  # same parameter set, shared keys
    xs = wl.int8_values(cfg["input_seed"], cfg["values"])
    bits = wl.to_bits(xs, 8)
    ct = tfhe.tfhe_encrypt_torus(sk, cfg["input_seed"], tfhe.encode_bits(bits.ravel()))
    ct = ct.reshape(cfg["values"], 8, p["n"] + 1)
    say(f"relu n=630 V={cfg['values']} gates={cfg['values'] * 7}")
    t0 = time.time()
    y = tfhe.to_host(tfhe.glyph_relu_batch(ek, tfhe.to_device(ct), 8))
    say(f"  gpu {time.time() - t0:.2f}s")
    dec = bits_of(tfhe.tfhe_decrypt_phase(sk, y.reshape(-1, p["n"] + 1))).reshape(-1, 8)
    assert np.array_equal(wl.from_bits(dec), np.maximum(xs.astype(np.int64), 0))
    gates = wl.sample_indices(cfg["input_seed"], cfg["values"] * 7, cfg["sample"])
    ref = oracle.relu_gates(ok, ct, 8, gates)
    got = np.stack([y[g // 7, g % 7] for g in gates])
    assert np.array_equal(got, ref)
    assert np.all(y[:, 7, :p["n"]] == 0) and np.all(y[:, 7, p["n"]] == M32 - MU)


def test_mlp_irelu_7680(torch):
    """Backward iReLU over the MLP layer: 7680 8-bit errors gated by the
    signs of the 7680 forward pre-activations, 61,440 gates in windows of
    16,384 (the last one ragged)."""
    cfg = wl.CONFIGS["mlp_irelu"]
    p = cfg["params"]
    sk, ek, ok = keys_for("tfhe128_nand", torch)  # same parameter set, shared keys
    V = cfg["values"]
    us = wl.int8_values(cfg["input_seed"], V)
    ds = wl.int8_values(cfg["input_seed"], V, stream=7)
    cu = tfhe.tfhe_encrypt_torus(sk, cfg["input_seed"], tfhe.encode_bits(wl.to_bits(us, 8).ravel()))
    cd = tfhe.tfhe_encrypt_torus(sk, cfg["input_seed"] + 1, tfhe.encode_bits(wl.to_bits(ds, 8).ravel()))
    cu, cd = cu.reshape(V, 8, p["n"] + 1), cd.reshape(V, 8, p["n"] + 1)
    u, d = tfhe.to_device(cu), tfhe.to_device(cd)
    y = torch.empty_like(d)
    total, step = V * 8, 16384
    ws = tfhe.alloc_workspace(ek, step)
    say(f"irelu n=630 V={V} gates={total}")
    t0 = time.time()
    for s in range(0, total, step):
        tfhe.glyph_irelu_batch(ek, u, d, out=y, gate_begin=s, gate_end=min(s + step, total), workspace=ws)
    got = tfhe.to_host(y)
    say(f"  gpu {time.time() - t0:.2f}s")
    dec = bits_of(tfhe.tfhe_decrypt_phase(sk, got.reshape(-1, p["n"] + 1))).reshape(V, 8)
    assert np.array_equal(wl.from_bits(dec), np.where(us >= 0, ds.astype(np.int64), 0))
    gates = wl.sample_indices(cfg["input_seed"], total, cfg["sample"])
    ref = oracle.irelu_gates(ok, cu, 8, cd, 8, gates)
    assert np.array_equal(got.reshape(-1, p["n"] + 1)[gates], ref)


def test_softmax_mux3_8192(torch):
    """The 3-bit softmax exponentiation unit by multiplexer tree on 8192
    bit-wise encrypted values (128-bit parameters, the LUT workload's
    messages and table): every output decrypts to its table entry, and a
    sample matches the oracle bit for bit."""
    cfg = wl.CONFIGS["softmax_mux3"]
    p = cfg["params"]
    sk, ek, ok = keys_for("tfhe128_nand", torch)  # same parameter set, shared keys
    V, mb, ob = cfg["values"], cfg["msg_bits"], cfg["out_bits"]
    m = wl.messages(cfg["input_seed"], V, mb)
    table = wl.lut(cfg["input_seed"], mb)
    ct = tfhe.tfhe_encrypt_torus(sk, cfg["input_seed"], tfhe.encode_bits(wl.to_bits(m, mb).ravel()))
    ct = ct.reshape(V, mb, p["n"] + 1)
    say(f"softmax mux tree n=630 V={V}")
    t0 = time.time()
    got = tfhe.to_host(tfhe.glyph_mux_lut_batch(ek, tfhe.to_device(ct), table, ob))
    say(f"  gpu {time.time() - t0:.2f}s")
    dec = bits_of(tfhe.tfhe_decrypt_phase(sk, got.reshape(-1, p["n"] + 1))).reshape(V, ob)
    assert np.array_equal((dec.astype(np.int64) << np.arange(ob)).sum(axis=1), table[m])
    idx = wl.sample_indices(cfg["input_seed"], V, cfg["sample"])
    t0 = time.time()
    ref = oracle.mux_lut(ok, ct[idx], mb, table, ob)
    say(f"  oracle sample of {len(idx)} values in {time.time() - t0:.1f}s")
    assert np.array_equal(got[idx], ref)


def test_switch_steps_128bit(torch):
    """Steps 2 and 3 of the BGV-to-TFHE switch at the 128-bit parameters:
    1024 LWE samples packed into one TRLWE sample (bit-exact with the
    oracle), then its first 64 coefficients extracted and key-switched back
    to dimension n, each decoding to its message."""
    cfg = wl.CONFIGS["tfhe128_nand"]
    p = cfg["params"]
    sk, ek, ok = keys_for("tfhe128_nand", torch)
    say("packing key n=630 N=1024 (library and oracle)")
    tfhe.tfhe_packing_key_upload(sk, ek)
    Z = p["N"]
    m = np.random.default_rng(65).integers(0, 16, Z).astype(np.uint32)
    lwe = tfhe.tfhe_encrypt_torus(sk, 65, (m << 28).astype(np.uint32)).reshape(1, Z, p["n"] + 1)
    t0 = time.time()
    acc = tfhe.tfhe_pack_keyswitch_batch(ek, tfhe.to_device(lwe))
    ext = tfhe.tfhe_sample_extract_batch(acc, 64)
    back = tfhe.to_host(tfhe.tfhe_keyswitch_batch(ek, ext.reshape(64, p["N"] + 1)))
    say(f"  gpu {time.time() - t0:.2f}s")
    ph = tfhe.tfhe_decrypt_phase(sk, back).astype(np.int64)
    assert np.array_equal(((ph + (1 << 27)) >> 28) % 16, m[:64])
    t0 = time.time()
    ref = oracle.pack_keyswitch(ok, lwe[0])
    say(f"  oracle packing in {time.time() - t0:.1f}s")
    assert np.array_equal(tfhe.to_host(acc)[0], ref)


def test_conv_relu_streamed(torch):
    """207,360 8-bit values (60 x 6 x 24 x 24), 1,451,520 ReLU gates streamed
    through calls of 16,384 gates; every output decrypts to max(x, 0) and a
    sample drawn across many calls matches the oracle bit for bit."""
    cfg = wl.CONFIGS["conv_relu"]
    p = cfg["params"]
    sk, ek, ok = keys_for("tfhe128_nand", torch)
    V, step = cfg["values"], cfg["gates_per_call"]
    total = V * 7
    xs = wl.int8_values(cfg["input_seed"], V)
    bits = wl.to_bits(xs, 8)
    say(f"conv relu: encrypting {V * 8} bits")
    ct = tfhe.tfhe_encrypt_torus(sk, cfg["input_seed"], tfhe.encode_bits(bits.ravel()))
    x = tfhe.to_device(ct.reshape(V, 8, p["n"] + 1))
    y = torch.empty_like(x)
    ws = tfhe.alloc_workspace(ek, step)
    t0 = time.time()
    calls = 0
    for begin in range(0, total, step):
        tfhe.glyph_relu_batch(ek, x, 8, y=y, gate_begin=begin, gate_end=min(begin + step, total), workspace=ws)
        calls += 1
        if calls % 16 == 0:
            torch.cuda.synchronize()
            say(f"  {calls} calls, {min(begin + step, total)} gates, {time.time() - t0:.1f}s")
    torch.cuda.synchronize()
    say(f"  gpu {calls} calls in {time.time() - t0:.1f}s")
    yh = tfhe.to_host(y)
    del x, y
    dec = bits_of(tfhe.tfhe_decrypt_phase(sk, yh.reshape(-1, p["n"] + 1))).reshape(V, 8)
    assert np.array_equal(wl.from_bits(dec), np.maximum(xs.astype(np.int64), 0))
    gates = wl.sample_indices(cfg["input_seed"], total, cfg["sample"])
    assert len(np.unique(gates // step)) > 20  # the sample spans many calls
    ref = oracle.relu_gates(ok, ct.reshape(V, 8, p["n"] + 1), 8, gates)
    got = np.stack([yh[g // 7, g % 7] for g in gates])
    assert np.array_equal(got, ref)


def test_lut3_n2048_8192(torch):
    cfg = wl.CONFIGS["lut3_n2048"]
    p = cfg["params"]
    sk, ek, ok = keys_for("lut3_n2048", torch)
    m = wl.messages(cfg["input_seed"], cfg["batch"], cfg["msg_bits"])
    lut = wl.lut(cfg["input_seed"], cfg["msg_bits"])
    tv = tfhe.tfhe_lut_testvec(p["N"], cfg["msg_bits"], lut)
    assert np.array_equal(tv, oracle.lut_testvec(p["N"], cfg["msg_bits"], lut))
    ct = tfhe.tfhe_encrypt_torus(sk, cfg["input_seed"], (m << 28).astype(np.uint32))
    say(f"lut bootstrap n=750 N=2048 B={len(m)}")
    t0 = time.time()
    got = tfhe.to_host(tfhe.tfhe_lut_bootstrap_batch(ek, tfhe.to_device(ct), tfhe.to_device(tv)))
    say(f"  gpu {time.time() - t0:.2f}s")
    ph = tfhe.tfhe_decrypt_phase(sk, got).astype(np.int64)
    assert np.array_equal(((ph + (1 << 27)) >> 28) & 15, lut[m])
    idx = wl.sample_indices(cfg["input_seed"], len(m), cfg["sample"])
    t0 = time.time()
    ref = oracle.lut_bootstrap(ok, ct[idx], tv)
    say(f"  oracle sample of {len(idx)} in {time.time() - t0:.1f}s")
    assert np.array_equal(got[idx], ref)


def test_planted_oracle_error_is_detected(torch):
    """The comparison can fail: a single flipped bit in the oracle's copy of
    the bootstrapping key (planted on the CPU) breaks bit-exact agreement."""
    cfg = wl.CONFIGS["toy"]
    p = cfg["params"]
    sk, ek, ok = keys_for("toy", torch)
    bad = oracle.Keys(p, cfg["key_seed"])
    bad.bk[12345] ^= np.uint32(1 << 20)
    a, b = wl.gate_inputs(cfg["input_seed"], cfg["batch"])
    ca = tfhe.tfhe_encrypt_torus(sk, cfg["input_seed"], tfhe.encode_bits(a), 0)
    cb = tfhe.tfhe_encrypt_torus(sk, cfg["input_seed"], tfhe.encode_bits(b), len(a))
    got = tfhe.to_host(tfhe.tfhe_gate_bootstrap_batch(ek, "NAND", tfhe.to_device(ca), tfhe.to_device(cb)))
    assert np.array_equal(got, oracle.gate_bootstrap(ok, "NAND", ca, cb))
    assert not np.array_equal(got, oracle.gate_bootstrap(bad, "NAND", ca, cb))


def test_workspace_too_small_is_rejected(torch):
    sk, ek, ok = keys_for("toy", torch)
    x = tfhe.to_device(np.zeros((8, 65), np.uint32))
    ws = torch.empty(tfhe.tfhe_workspace_bytes(ek, 8) - 256, dtype=torch.uint8, device="cuda:0")
    with pytest.raises(tfhe.TfheError) as ei:
        tfhe.tfhe_gate_bootstrap_batch(ek, "AND", x, x, workspace=ws)
    assert ei.value.rc == tfhe.TFHE_EINVAL
    with pytest.raises(tfhe.TfheError) as ei:
        tfhe.tfhe_gate_bootstrap_batch(ek, 17, x, x)
    assert ei.value.rc == tfhe.TFHE_EINVAL


def test_counts_too_large_for_one_launch_are_refused(torch):
    """Every server-side call refuses, before any launch, a count whose
    one-dimensional launch would exceed 2^32 - 256 work-items, and the size
    queries refuse counts no call accepts.  Each call passes a NULL data
    pointer, so a call that passed the count check would fail on it instead,
    with another message: no call here can reach a launch."""
    import ctypes

    p = wl.CONFIGS["toy"]["params"]  # n = 64, N = 256
    sk, ek = tfhe.tfhe_keygen_from_seed(p, 7, 0)
    tfhe.tfhe_packing_key_upload(sk, ek)
    L = tfhe.lib()
    h = ek.handle
    most = (1 << 32) - 256
    ws = tfhe.alloc_workspace(ek, 8)
    wp, wb = tfhe._dptr(ws), ws.numel()

    def refused(rc, what):
        msg = L.tfhe_last_error().decode()
        assert rc == tfhe.TFHE_EINVAL and "exceed" in msg and what in msg, (rc, msg)

    B = most // 65 + 1  # n + 1 = 65 words per ciphertext
    say(f"count limits: bootstraps of {B} ciphertexts")
    refused(L.tfhe_gate_bootstrap_batch(h, 0, None, None, None, B, wp, wb, None), "ciphertexts")
    refused(L.tfhe_lut_bootstrap_batch(h, None, None, None, B, wp, wb, None), "ciphertexts")
    refused(L.tfhe_bootstrap_extract_batch(h, None, None, None, B, wp, wb, None), "ciphertexts")
    assert L.tfhe_gate_bootstrap_batch(h, 0, None, None, None, B - 1, wp, wb, None) == tfhe.TFHE_EINVAL
    assert "NULL" in L.tfhe_last_error().decode()  # one fewer passes the count check
    refused(L.tfhe_keyswitch_batch(h, None, None, most // 257 + 1, None), "samples")
    refused(L.glyph_relu_batch(h, None, None, most // 8 + 1, 8, 0, 1, wp, wb, None), "values")
    refused(L.glyph_relu_batch(h, None, None, 10_000_000, 8, 0, most // 65 + 1, wp, wb, None), "gates")
    refused(L.glyph_irelu_batch(h, None, 8, None, None, most // 8 + 1, 8, 0, 1, wp, wb, None), "values")
    refused(L.glyph_irelu_batch(h, None, 8, None, None, 10_000_000, 8, 0, most // 65 + 1, wp, wb, None),
            "gates")
    refused(L.tfhe_mux_batch(h, None, None, None, None, most // 514 + 1, wp, wb, None), "multiplexers")
    table = (ctypes.c_uint32 * 8)(0, 1, 2, 3, 4, 5, 6, 7)
    V = most // (3 * 4 * 257) + 1
    refused(L.glyph_mux_lut_batch(h, None, 3, table, 3, None, V, wp, wb, None), "values")
    assert L.glyph_mux_lut_workspace_bytes(h, V, 3, 3) == tfhe.TFHE_EINVAL
    assert L.glyph_mux_lut_workspace_bytes(h, V - 1, 3, 3) > 0
    refused(L.tfhe_pack_keyswitch_batch(h, None, 1, None, most // 512 + 1, None), "ciphertexts")
    refused(L.tfhe_negacyclic_mul_batch(h, None, None, None, most // 256 + 1, None), "products")
    assert L.tfhe_workspace_bytes(h, most + 1) == tfhe.TFHE_EINVAL
    assert L.tfhe_workspace_bytes(h, most) > 0


def test_empty_and_invalid_calls(torch):
    """Empty batches are no-ops that leave the output untouched; gate windows
    outside the tensor, a missing packing key and bad table sizes are
    rejected before any launch."""
    p = wl.CONFIGS["toy"]["params"]
    sk, ek, ok = keys_for("toy", torch)
    row = p["n"] + 1
    x = tfhe.to_device(np.zeros((4, row), np.uint32))
    sentinel = torch.full((4, row), 7, dtype=torch.int32, device="cuda:0")
    ws = tfhe.alloc_workspace(ek, 8)
    L = tfhe.lib()
    assert L.tfhe_gate_bootstrap_batch(ek.handle, 0, tfhe._dptr(x), tfhe._dptr(x), tfhe._dptr(sentinel), 0,
                                       tfhe._dptr(ws), ws.numel(), None) == tfhe.TFHE_OK
    assert L.tfhe_keyswitch_batch(ek.handle, tfhe._dptr(x), tfhe._dptr(sentinel), 0, None) == tfhe.TFHE_OK
    assert L.tfhe_mux_batch(ek.handle, tfhe._dptr(x), tfhe._dptr(x), tfhe._dptr(x), tfhe._dptr(sentinel), 0,
                            tfhe._dptr(ws), ws.numel(), None) == tfhe.TFHE_OK
    torch.cuda.synchronize()
    assert bool((sentinel == 7).all())
    y = tfhe.to_device(np.zeros((2, 8, row), np.uint32))
    with pytest.raises(tfhe.TfheError) as ei:  # 2 values x 7 gates: window end 15 is outside
        tfhe.glyph_relu_batch(ek, y, 8, y=torch.empty_like(y), gate_begin=0, gate_end=15)
    assert ei.value.rc == tfhe.TFHE_EINVAL
    with pytest.raises(tfhe.TfheError) as ei:
        tfhe.glyph_irelu_batch(ek, y, y, out=torch.empty_like(y), gate_begin=10, gate_end=9)
    assert ei.value.rc == tfhe.TFHE_EINVAL
    x3 = tfhe.to_device(np.zeros((2, 3, row), np.uint32))
    with pytest.raises(ValueError):
        tfhe.glyph_mux_lut_batch(ek, x3, np.arange(7), 3)  # 3 selector bits need 8 entries
    with pytest.raises(tfhe.TfheError) as ei:  # entry 9 does not fit in 3 output bits
        tfhe.glyph_mux_lut_batch(ek, x3, np.array([0, 1, 2, 3, 4, 5, 6, 9]), 3)
    assert ei.value.rc == tfhe.TFHE_EINVAL
    with pytest.raises(ValueError):  # rows of n = 64 words where the key needs n + 1
        tfhe.tfhe_gate_bootstrap_batch(ek, "AND", x[:, :row - 1].contiguous(), x[:, :row - 1].contiguous())
    with pytest.raises(ValueError):  # 64-bit elements
        tfhe.tfhe_keyswitch_batch(ek, torch.zeros((4, p["N"] + 1), dtype=torch.int64, device="cuda:0"))
    sk2, ek2 = tfhe.tfhe_keygen_from_seed(p, 5, 0)  # fresh key without a packing key
    with pytest.raises(tfhe.TfheError) as ei:
        tfhe.tfhe_pack_keyswitch_batch(ek2, tfhe.to_device(np.zeros((1, 3, row), np.uint32)))
    assert ei.value.rc == tfhe.TFHE_EINVAL
    with pytest.raises(tfhe.TfheError) as ei:  # a packing key built from another secret key
        tfhe.tfhe_packing_key_upload(sk, ek2)
    assert ei.value.rc == tfhe.TFHE_EINVAL and "not made from" in str(ei.value)
    tfhe.tfhe_packing_key_upload(sk2, ek2)  # its own secret key
