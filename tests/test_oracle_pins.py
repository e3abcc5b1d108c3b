"""Pins of the CPU oracle against mathematics it does not compute itself.

Each test checks the oracle against a library routine, a closed form, an
invariant of TFHE bootstrapping, the truth semantics the paper states
(Section 3.1: gates with bootstrapping, the free NOT, the forward ReLU unit) or
an independent implementation -- chosen so that a dropped term, a wrong sign or
index, or a transposed operand anywhere in the oracle fails at least one.
"""
import math
import os

import numpy as np
import pytest

import brute_tfhe as brute
import oracle

M32 = 1 << 32
MU = 1 << 29
GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")

TOY = dict(n=64, N=256, l=3, bg_bit=7, ks_t=8, ks_basebit=2,
           alpha_lwe=2.0 ** -15, alpha_bk=2.0 ** -25, alpha_ks=2.0 ** -15)
TINY = dict(n=6, N=16, l=3, bg_bit=7, ks_t=8, ks_basebit=2,
            alpha_lwe=2.0 ** -15, alpha_bk=2.0 ** -25, alpha_ks=2.0 ** -15)
# noiseless keys with exact gadgets (l * bg_bit = 32, t * basebit = 32)
EXACT = dict(n=8, N=16, l=4, bg_bit=8, ks_t=16, ks_basebit=2,
             alpha_lwe=0.0, alpha_bk=0.0, alpha_ks=0.0)


def s32(x):
    x = np.asarray(x, dtype=np.int64) % M32
    return np.where(x >= M32 // 2, x - M32, x)


def np_negacyclic(a, b):
    """Z[X] product by numpy.convolve, folded with X^N = -1, then mod 2^32."""
    N = len(a)
    full = np.convolve(np.array([int(x) for x in a], dtype=object),
                       np.array([int(x) for x in b], dtype=object))
    out = list(full[:N])
    for k in range(N, 2 * N - 1):
        out[k - N] -= full[k]
    return np.array([int(x) % M32 for x in out], dtype=np.uint32)


# ---------------------------------------------------------------- generator

def test_splitmix64_reference_sequence():
    """The generator's stream is SplitMix64: its outputs from state 1234567
    equal the published reference sequence, and a (seed, tag, idx) word is
    output idx of the stream whose state is output tag of the seed's stream."""
    ref = [int(x) for x in open(os.path.join(GOLDEN, "splitmix64_seed1234567.txt"))
           if x.strip() and not x.startswith("#")]
    assert [oracle.stream_output(1234567, k) for k in range(len(ref))] == ref
    for tag in range(len(ref)):
        for idx in (0, 1, 77):
            assert oracle.word(1234567, tag, idx) == oracle.stream_output(ref[tag], idx)
            assert oracle.word(1234567, tag, idx) == brute.word(1234567, tag, idx)


def test_gaussian_moments():
    xs = np.array([oracle.gauss(7, 4, i) for i in range(40000)])
    assert abs(xs.mean()) < 0.03
    assert abs(xs.std() - 1.0) < 0.02
    # tail mass beyond 2 sigma of a standard normal is 4.55%
    assert abs((np.abs(xs) > 2).mean() - 0.0455) < 0.006


def test_noise_scale_and_rounding():
    alpha = 2.0 ** -15
    e = s32([oracle.noise(3, 6, i, alpha) for i in range(20000)]).astype(np.float64) / M32
    assert abs(e.std() / alpha - 1.0) < 0.03
    # alpha = 2^-45 is 2^-13 of one torus32 unit: always rounds to zero
    assert all(oracle.noise(3, 4, i, 2.0 ** -45) == 0 for i in range(2000))


# ---------------------------------------------------------------- ring arithmetic

@pytest.mark.parametrize("N", [1, 2, 4, 8, 16, 32, 64])
def test_negacyclic_product_matches_numpy(N):
    rng = np.random.default_rng(N)
    for _ in range(3):
        a = rng.integers(0, M32, N, dtype=np.uint64).astype(np.uint32)
        b = rng.integers(0, M32, N, dtype=np.uint64).astype(np.uint32)
        assert np.array_equal(oracle.negacyclic_mul(a, b), np_negacyclic(a, b))
    # small signed digits times full-range coefficients (the external product's shape)
    d = rng.integers(-64, 64, N).astype(np.int64)
    b = rng.integers(0, M32, N, dtype=np.uint64).astype(np.uint32)
    assert np.array_equal(oracle.negacyclic_mul((d % M32).astype(np.uint32), b), np_negacyclic(d, b))


def test_negacyclic_product_is_commutative_and_bilinear():
    rng = np.random.default_rng(1)
    N = 128
    a, b, c = (rng.integers(0, M32, N, dtype=np.uint64).astype(np.uint32) for _ in range(3))
    assert np.array_equal(oracle.negacyclic_mul(a, b), oracle.negacyclic_mul(b, a))
    lhs = oracle.negacyclic_mul(a, (b.astype(np.uint64) + c).astype(np.uint32))
    rhs = (oracle.negacyclic_mul(a, b).astype(np.uint64) + oracle.negacyclic_mul(a, c)).astype(np.uint32)
    assert np.array_equal(lhs, rhs)


@pytest.mark.parametrize("N", [4, 16, 256])
def test_rotation_closed_forms(N):
    rng = np.random.default_rng(N + 5)
    p = rng.integers(0, M32, N, dtype=np.uint64).astype(np.uint32)
    # X^0 = X^{2N} = 1 and X^N = -1
    assert np.array_equal(oracle.rotate(p, 0), p)
    assert np.array_equal(oracle.rotate(oracle.rotate(p, N), N), p)
    assert np.array_equal(oracle.rotate(p, N), (np.uint32(0) - p).astype(np.uint32))
    for _ in range(8):
        a, b = (int(x) for x in rng.integers(0, 2 * N, 2))
        assert np.array_equal(oracle.rotate(oracle.rotate(p, a), b), oracle.rotate(p, (a + b) % (2 * N)))
    # rotation = product with the signed monomial X^e
    for e in list(rng.integers(0, 2 * N, 6)) + [1, N - 1, N + 1, 2 * N - 1]:
        mono = np.zeros(N, np.int64)
        if e < N:
            mono[e] = 1
        else:
            mono[e - N] = -1
        assert np.array_equal(oracle.rotate(p, int(e)), np_negacyclic(mono, p))


@pytest.mark.parametrize("l,bg", [(3, 7), (2, 10), (4, 8), (1, 16), (6, 5)])
def test_decomposition_range_and_recomposition(l, bg):
    rng = np.random.default_rng(l * 100 + bg)
    xs = list(range(0, M32, 104729 * 97)) + [int(x) for x in rng.integers(0, M32, 3000)]
    xs += [0, 1, M32 - 1, M32 // 2, M32 // 2 - 1] + [(1 << (32 - l * bg)) * k + ((1 << (31 - l * bg)) if l * bg < 32 else 0)
                                                        for k in range(5)]
    half = 1 << (bg - 1)
    bound = (1 << (31 - l * bg)) if l * bg < 32 else 0
    for x in xs:
        d = oracle.decompose(l, bg, x % M32)
        assert all(-half <= v < half for v in d)
        rec = sum(v * (1 << (32 - (j + 1) * bg)) for j, v in enumerate(d))
        err = int(s32(rec - x))
        assert -bound < err <= bound or (bound == 0 and err == 0)
        assert d == brute.decompose(x % M32, l, bg)


def test_mod_switch_is_rounded_scaling():
    from fractions import Fraction
    rng = np.random.default_rng(9)
    for N in (16, 256, 1024, 2048):
        xs = [int(x) for x in rng.integers(0, M32, 500)] + [0, M32 - 1, M32 // (4 * N), M32 // (4 * N) - 1]
        for x in xs:
            f = Fraction(x * 2 * N, M32)
            expect = math.floor(f + Fraction(1, 2)) % (2 * N)
            assert oracle.mod_switch(x, N) == expect


def test_sample_extract_phase_identity():
    rng = np.random.default_rng(11)
    N = 64
    S = rng.integers(0, 2, N).astype(np.uint32)
    acc = rng.integers(0, M32, 2 * N, dtype=np.uint64).astype(np.uint32)
    A, B = acc[:N], acc[N:]
    ext = oracle.sample_extract(acc)
    poly_phase = (B.astype(np.int64) - np_negacyclic(A, S).astype(np.int64)) % M32
    assert oracle.phase(S, ext)[()] == poly_phase[0]


# ---------------------------------------------------------------- keys

def test_keys_decrypt_to_their_messages():
    p = TOY
    keys = oracle.Keys(p, 77)
    N, n, l, bg = p["N"], p["n"], p["l"], p["bg_bit"]
    bk = keys.bk_view()
    tol = 2.0 ** -25 * 7 * M32  # 7 sigma of the BK noise
    for i in (0, 13, n - 1):
        for r in range(2 * l):
            A, B = bk[i, r, 0], bk[i, r, 1]
            ph = (B.astype(np.int64) - np_negacyclic(A, keys.S).astype(np.int64)) % M32
            q, j = divmod(r, l)
            g = int(keys.s[i]) << (32 - (j + 1) * bg)
            # TRGSW row: phase = -s_i g S (mask row) or + s_i g (body row), plus noise
            if q == 0:
                expect = (-(np_negacyclic(np.array([g] + [0] * (N - 1), np.uint32), keys.S).astype(np.int64))) % M32
            else:
                expect = np.array([g] + [0] * (N - 1), np.int64)
            assert np.all(np.abs(s32(ph - expect)) < tol)
    ksk = keys.ksk_view()
    tol = 7 * 2.0 ** -15 * M32
    for i in (0, 101, N - 1):
        for j in range(p["ks_t"]):
            for v in (1, 2, 3):
                msg = (v * int(keys.S[i]) << (32 - (j + 1) * p["ks_basebit"])) % M32
                ph = int(oracle.phase(keys.s, ksk[i, j, v - 1]))
                assert abs(int(s32(ph - msg))) < tol


def test_keygen_and_bootstrap_match_brute_force():
    """Two implementations written separately agree bit for bit."""
    p = TINY
    keys = oracle.Keys(p, 4242)
    s, S, bk, ksk = brute.keygen(p, 4242)
    assert keys.s.tolist() == s and keys.S.tolist() == S
    assert keys.bk_view().tolist() == [[list(row) for row in rows] for rows in bk]
    kv = keys.ksk_view()
    for (i, j, v), row in ksk.items():
        assert kv[i, j, v - 1].tolist() == row
    rng = np.random.default_rng(3)
    for trial in range(4):
        bits = rng.integers(0, 2, 2)
        mu = np.where(bits == 1, MU, M32 - MU).astype(np.uint32)
        ct = oracle.encrypt(p["n"], keys.s, 99, p["alpha_lwe"], mu, first_index=2 * trial)
        assert ct[0].tolist() == brute.encrypt(s, 99, p["alpha_lwe"], int(mu[0]), 2 * trial)
        for g in ("NAND", "XOR", "ANDNY"):
            out = oracle.gate_bootstrap(keys, g, ct[0], ct[1])[0]
            assert out.tolist() == brute.gate(p, bk, ksk, g, ct[0].tolist(), ct[1].tolist())


# ---------------------------------------------------------------- closed forms

@pytest.mark.parametrize("p", [TOY, TINY])
def test_trivial_ciphertext_closed_form(p):
    """A trivial input (0, b) is never rotated: the bootstrap returns
    (0^N, +-v) exactly and key switching keeps it (0^n, +-v)."""
    keys = oracle.Keys(p, 5)
    N, n = p["N"], p["n"]
    tv = np.arange(1, N + 1, dtype=np.uint32) * np.uint32(977)
    for b in [0, 1, M32 // 3, M32 // 2, M32 - 1, 123456789, 3 * M32 // 4]:
        lwe = np.zeros(n + 1, np.uint32)
        lwe[n] = b
        bbar = oracle.mod_switch(b, N)
        expect = int(tv[bbar]) if bbar < N else (M32 - int(tv[bbar - N])) % M32
        acc = oracle.blind_rotate(keys, lwe, tv)
        assert not acc[0].any()
        ext = oracle.sample_extract(acc)
        assert not ext[:N].any() and int(ext[N]) == expect
        ks = oracle.keyswitch(keys, ext)[0]
        assert not ks[:n].any() and int(ks[n]) == expect


def test_noiseless_exact_gadget_gives_exact_sign():
    """With noiseless keys and exact gadgets every step is exact: the output
    phase is +1/8 when phi = bbar - sum abar_i s_i mod 2N lies in [0, N) and
    -1/8 otherwise -- checked for every phi in [0, 2N)."""
    p = EXACT
    keys = oracle.Keys(p, 8)
    n, N = p["n"], p["N"]
    rng = np.random.default_rng(21)
    tv = oracle.gate_testvec(N)
    seen = set()
    for trial in range(6 * N):
        a = rng.integers(0, M32, n, dtype=np.uint64).astype(np.uint32)
        target = trial % (2 * N)
        abar = [oracle.mod_switch(int(x), N) for x in a]
        dot = sum(x * int(s) for x, s in zip(abar, keys.s))
        bbar = (target + dot) % (2 * N)
        b = (bbar * (M32 // (2 * N)) + int(rng.integers(-M32 // (8 * N), M32 // (8 * N)))) % M32
        assert oracle.mod_switch(b, N) == bbar
        lwe = np.concatenate([a, [b]]).astype(np.uint32)
        ext = oracle.bootstrap_no_ks(keys, lwe, tv)[0]
        out = oracle.keyswitch(keys, ext)[0]
        expect = MU if target < N else M32 - MU
        assert int(oracle.phase(keys.S, ext)) == expect
        assert int(oracle.phase(keys.s, out)) == expect
        seen.add(target)
    assert seen == set(range(2 * N))


def test_noiseless_cmux_selects():
    """One CMux with a noiseless exact key multiplies the phase polynomial by
    X^{abar * s_i} exactly."""
    p = EXACT
    keys = oracle.Keys(p, 31)
    N = p["N"]
    rng = np.random.default_rng(2)
    acc = rng.integers(0, M32, 2 * N, dtype=np.uint64).astype(np.uint32).reshape(2, N)

    def poly_phase(c):
        return ((c[1].astype(np.int64) - np_negacyclic(c[0], keys.S).astype(np.int64)) % M32).astype(np.uint32)

    for i in range(p["n"]):
        for abar in (0, 1, 5, N, 2 * N - 1):
            out = oracle.cmux(keys, i, abar, acc)
            e = abar * int(keys.s[i])
            assert np.array_equal(poly_phase(out), oracle.rotate(poly_phase(acc), e % (2 * N)))


def brute_cmux(N, l, bg, row, abar, acc):
    """One CMux step written with the pure-Python pieces of brute_tfhe
    (monomial, schoolbook product, carry-based decomposition)."""
    X = brute.monomial(N, abar)
    polys = [list(map(int, acc[0])), list(map(int, acc[1]))]
    digit_polys = []
    for P in polys:
        D = [(x - y) % M32 for x, y in zip(brute.polymul_negacyclic(X, P), P)]
        per = [brute.decompose(x, l, bg) for x in D]
        digit_polys += [[per[m][j] for m in range(N)] for j in range(l)]
    out = [list(P) for P in polys]
    for r, dp in enumerate(digit_polys):
        for q in range(2):
            prod = brute.polymul_negacyclic(dp, list(map(int, row[r][q])))
            out[q] = [(x + y) % M32 for x, y in zip(out[q], prod)]
    return np.array(out, dtype=np.uint32)


@pytest.mark.parametrize("l,bg", [(3, 7), (2, 10)])
def test_cmux_with_a_given_key_row_matches_brute_force(l, bg):
    """The oracle's CMux with a caller-given key row (the form the stage check
    of one CMux uses) against the independent pure-Python CMux, with key rows
    at the largest magnitudes of both signs and accumulators whose rotation
    difference has every digit at -Bg/2 or Bg/2 - 1, and at random."""
    N = 16
    p = dict(TINY, l=l, bg_bit=bg)
    rng = np.random.default_rng(l * 100 + bg)
    half = 1 << (bg - 1)
    rnd = 1 << (31 - l * bg) if l * bg < 32 else 0

    def word_with_digits(d):
        return (sum((d + half) << (32 - j * bg) for j in range(1, l + 1))
                - sum(half << (32 - j * bg) for j in range(1, l + 1)) - rnd) % M32

    rows = [np.full((2 * l, 2, N), w, np.uint32) for w in (0x80008000, 0x7FFF7FFF, 0xFFFFFFFF, 0x80000000)]
    rows.append(rng.integers(0, M32, (2 * l, 2, N), dtype=np.uint64).astype(np.uint32))
    accs = []
    for d in (-half, half - 1):
        w = word_with_digits(d)
        assert brute.decompose(w, l, bg) == [d] * l
        # X^N acc - acc = -2 acc: acc = -w / 2 gives the difference w (w even)
        accs.append((np.full((2, N), (-(w // 2)) % M32, np.uint64).astype(np.uint32), N))
    accs.append((rng.integers(0, M32, (2, N), dtype=np.uint64).astype(np.uint32), int(rng.integers(0, 2 * N))))
    for row in rows:
        for acc, abar in accs:
            got = oracle.cmux_row(p, row, abar, acc)
            assert np.array_equal(got, brute_cmux(N, l, bg, row, abar, acc))


def test_mod_switch_array_matches_the_brute_force_rounding():
    rng = np.random.default_rng(12)
    for N in (16, 1024, 2048):
        xs = np.concatenate([rng.integers(0, M32, 300, dtype=np.uint64),
                             np.array([0, M32 - 1, M32 // (4 * N), M32 // (4 * N) - 1], dtype=np.uint64)]).astype(np.uint32)
        got = oracle.mod_switch_array(xs.reshape(4, -1), N).ravel()
        assert [int(g) for g in got] == [brute.mod_switch(int(x), N) for x in xs]


# ---------------------------------------------------------------- semantics

TRUTH = {"NAND": lambda a, b: 1 - (a & b), "AND": lambda a, b: a & b, "OR": lambda a, b: a | b,
         "NOR": lambda a, b: 1 - (a | b), "XOR": lambda a, b: a ^ b, "XNOR": lambda a, b: 1 - (a ^ b),
         "ANDNY": lambda a, b: (1 - a) & b, "ANDYN": lambda a, b: a & (1 - b),
         "ORNY": lambda a, b: (1 - a) | b, "ORYN": lambda a, b: a | (1 - b)}


def decrypt_bits(key, ct):
    return (s32(oracle.phase(key, ct)) > 0).astype(np.uint8)


def test_all_gates_truth_tables():
    p = TOY
    keys = oracle.Keys(p, 1234)
    a = np.array([0, 0, 1, 1] * 3, np.uint8)
    b = np.array([0, 1, 0, 1] * 3, np.uint8)
    enc = lambda bits, first: oracle.encrypt(p["n"], keys.s, 55, p["alpha_lwe"],
                                             np.where(bits == 1, MU, M32 - MU), first)
    ca, cb = enc(a, 0), enc(b, 100)
    assert np.array_equal(decrypt_bits(keys.s, ca), a)
    for g, f in TRUTH.items():
        out = oracle.gate_bootstrap(keys, g, ca, cb)
        assert np.array_equal(decrypt_bits(keys.s, out), f(a, b)), g
    # NOT needs no bootstrap and is exact negation
    na = oracle.not_gate(ca)
    assert np.array_equal(decrypt_bits(keys.s, na), 1 - a)
    assert np.array_equal(s32(oracle.phase(keys.s, na)), -s32(oracle.phase(keys.s, ca)))


def test_relu_3bit_golden_table():
    """The 3-bit forward ReLU unit of Section 3.1 against its truth table."""
    rows = [line.split() for line in open(os.path.join(GOLDEN, "relu_3bit.txt"))
            if line.strip() and not line.startswith("#")]
    p = TOY
    keys = oracle.Keys(p, 404)
    xs = np.array([int(r[0]) for r in rows])
    bits = np.array([[int(c) for c in r[1]] for r in rows], np.uint8)   # LSB first
    want = np.array([[int(c) for c in r[3]] for r in rows], np.uint8)
    mu = np.where(bits.ravel() == 1, MU, M32 - MU)
    x = oracle.encrypt(p["n"], keys.s, 66, p["alpha_lwe"], mu).reshape(len(rows), 3, p["n"] + 1)
    y = oracle.relu(keys, x, 3)
    got = decrypt_bits(keys.s, y.reshape(-1, p["n"] + 1)).reshape(len(rows), 3)
    assert np.array_equal(got, want)
    assert np.array_equal(np.maximum(xs, 0), [int(r[2]) for r in rows])


def test_relu_8bit_all_values():
    """Every 8-bit two's-complement input decrypts to max(x, 0) after the
    unit of 7 bootstrapped ANDs and one NOT (Section 3.1)."""
    from paper_1911_07101_amd import workloads as wl
    p = TOY
    keys = oracle.Keys(p, 808)
    xs = np.arange(-128, 128)
    bits = wl.to_bits(xs, 8)
    mu = np.where(bits.ravel() == 1, MU, M32 - MU)
    x = oracle.encrypt(p["n"], keys.s, 67, p["alpha_lwe"], mu).reshape(256, 8, p["n"] + 1)
    y = oracle.relu(keys, x, 8)
    got = decrypt_bits(keys.s, y.reshape(-1, p["n"] + 1)).reshape(256, 8)
    assert np.array_equal(wl.from_bits(got), np.maximum(xs, 0))


def test_irelu_all_4bit_pairs():
    """Backward iReLU (Section 3.1): for every 4-bit pre-activation u and
    4-bit error delta, the unit's output decrypts to delta where u >= 0 and to
    0 where u < 0 -- which needs the error's sign bit gated too."""
    from paper_1911_07101_amd import workloads as wl
    p = TOY
    keys = oracle.Keys(p, 909)
    us, ds = np.meshgrid(np.arange(-8, 8), np.arange(-8, 8), indexing="ij")
    us, ds = us.ravel(), ds.ravel()
    enc = lambda vals, seed: oracle.encrypt(
        p["n"], keys.s, seed, p["alpha_lwe"],
        np.where(wl.to_bits(vals, 4).ravel() == 1, MU, M32 - MU)).reshape(len(vals), 4, p["n"] + 1)
    u, d = enc(us, 71), enc(ds, 72)
    y = oracle.irelu(keys, u, 4, d, 4)
    got = wl.from_bits(decrypt_bits(keys.s, y.reshape(-1, p["n"] + 1)).reshape(-1, 4))
    assert np.array_equal(got, np.where(us >= 0, ds, 0))
    # a subset of gates gives the same words as the full unit
    ids = np.array([0, 5, 17, 255, 1023])
    assert np.array_equal(oracle.irelu_gates(keys, u, 4, d, 4, ids), y.reshape(-1, p["n"] + 1)[ids])


def test_mux_truth_table():
    """The multiplexer decrypts to c ? a : b for every input combination."""
    p = TOY
    keys = oracle.Keys(p, 1001)
    bits = np.array([(c, a, b) for c in (0, 1) for a in (0, 1) for b in (0, 1)] * 2)
    enc = lambda col, seed: oracle.encrypt(p["n"], keys.s, seed, p["alpha_lwe"],
                                           np.where(bits[:, col] == 1, MU, M32 - MU))
    out = oracle.mux(keys, enc(0, 81), enc(1, 82), enc(2, 83))
    assert np.array_equal(decrypt_bits(keys.s, out), np.where(bits[:, 0] == 1, bits[:, 1], bits[:, 2]))


@pytest.mark.parametrize("msg_bits,out_bits", [(1, 2), (2, 3), (3, 3)])
def test_mux_lut_all_inputs(msg_bits, out_bits):
    """The multiplexer tree returns the bits of table[x] for every input x
    (Section 3.1's 3-bit softmax unit is msg_bits = out_bits = 3)."""
    from paper_1911_07101_amd import workloads as wl
    p = TOY
    keys = oracle.Keys(p, 1002 + msg_bits)
    rng = np.random.default_rng(msg_bits)
    table = rng.integers(0, 1 << out_bits, 1 << msg_bits)
    xs = np.arange(1 << msg_bits)
    x = oracle.encrypt(p["n"], keys.s, 84, p["alpha_lwe"],
                       np.where(wl.to_bits(xs, msg_bits).ravel() == 1, MU, M32 - MU))
    out = oracle.mux_lut(keys, x.reshape(len(xs), msg_bits, p["n"] + 1), msg_bits, table, out_bits)
    got = decrypt_bits(keys.s, out.reshape(-1, p["n"] + 1)).reshape(len(xs), out_bits)
    assert np.array_equal((got << np.arange(out_bits)).sum(axis=1), table[xs])


def test_lut_bootstrap_all_messages():
    p = dict(TOY, n=64, N=512)
    keys = oracle.Keys(p, 515)
    rng = np.random.default_rng(17)
    for _ in range(2):
        lut = rng.integers(0, 8, 8).astype(np.uint32)
        tv = oracle.lut_testvec(p["N"], 3, lut)
        m = np.arange(8, dtype=np.uint32).repeat(2)
        ct = oracle.encrypt(p["n"], keys.s, 9, p["alpha_lwe"], (m << 28).astype(np.uint32))
        out = oracle.lut_bootstrap(keys, ct, tv)
        ph = oracle.phase(keys.s, out).astype(np.int64)
        dec = ((ph + (1 << 27)) >> 28) & 15
        assert np.array_equal(dec, lut[m])


def test_lut_testvec_closed_form():
    lut = np.array([3, 1, 4, 1, 5, 2, 6, 7], np.uint32)
    N = 256
    tv = oracle.lut_testvec(N, 3, lut).astype(np.int64)
    for j in range(N):
        box = (j + N // 16) // (N // 8)
        want = (lut[box] << 28) if box < 8 else (-(int(lut[0]) << 28)) % M32
        assert tv[j] == want


def test_gate_noise_matches_variance_estimate():
    """Measured output noise of NAND bootstraps on the toy parameters against
    the TFHE variance estimate (blind rotation + key switching)."""
    p = TOY
    keys = oracle.Keys(p, 2024)
    n, N, l, bg = p["n"], p["N"], p["l"], p["bg_bit"]
    cnt = 400
    rng = np.random.default_rng(8)
    a, b = rng.integers(0, 2, cnt), rng.integers(0, 2, cnt)
    enc = lambda bits, first: oracle.encrypt(n, keys.s, 77, p["alpha_lwe"],
                                             np.where(bits == 1, MU, M32 - MU), first)
    out = oracle.gate_bootstrap(keys, "NAND", enc(a, 0), enc(b, cnt))
    want = np.where((1 - (a & b)) == 1, MU, -MU)
    err = (s32(oracle.phase(keys.s, out)) - want).astype(np.float64) / M32
    Bg = 1 << bg
    e_d2 = (Bg * Bg + 2) / 12.0  # mean square of a uniform digit in [-Bg/2, Bg/2)
    var_br = n * 2 * l * N * e_d2 * p["alpha_bk"] ** 2
    var_ks = N * p["ks_t"] * 0.75 * p["alpha_ks"] ** 2 + (N / 2) * (2.0 ** -(p["ks_t"] * p["ks_basebit"] + 1)) ** 2 / 3
    sigma = math.sqrt(var_br + var_ks)
    assert 0.6 < err.std() / sigma < 1.5
    assert np.all(np.abs(err) < 0.125)


# ------------------------------------- TFHE side of the switch (Section 3.2)

def trlwe_phase(S, acc):
    """B - A*S with the product by numpy.convolve (independent of the oracle)."""
    A, B = acc[0], acc[1]
    return ((B.astype(np.int64) - np_negacyclic(A, S).astype(np.int64)) % M32).astype(np.uint32)


def test_sample_extract_at_every_coefficient():
    """The extracted sample of coefficient i decrypts, under S, to
    coefficient i of the TRLWE phase; coefficient 0 agrees with the
    gate bootstrap's SampleExtract."""
    N = 64
    rng = np.random.default_rng(3)
    S = rng.integers(0, 2, N).astype(np.uint32)
    acc = rng.integers(0, M32, (2, N), dtype=np.uint64).astype(np.uint32)
    ph = trlwe_phase(S, acc)
    for i in range(N):
        e = oracle.sample_extract_at(acc, i)
        assert oracle.phase(S, e[None])[0] == ph[i], i
    assert np.array_equal(oracle.sample_extract_at(acc, 0), oracle.sample_extract(acc))


def test_packing_key_entries_decrypt_to_their_messages():
    """Every packing-key entry (i, j, v) is a TRLWE sample under S of the
    constant v * s_i * 2^(32-(j+1)*basebit), up to the key noise."""
    p = dict(TOY, n=8, N=64)
    keys = oracle.Keys(p, 4242)
    t, bb = p["ks_t"], p["ks_basebit"]
    pks = keys.packing_key().reshape(p["n"], t, (1 << bb) - 1, 2, p["N"])
    for i in range(p["n"]):
        for j in range(t):
            for v in range(1, 1 << bb):
                ph = s32(trlwe_phase(keys.S, pks[i, j, v - 1]))
                want = np.zeros(p["N"], np.int64)
                want[0] = s32(v * int(keys.s[i]) << (32 - (j + 1) * bb))
                assert np.all(np.abs(s32(ph - want)) < 2 ** 32 * 2.0 ** -20), (i, j, v)


def test_pack_keyswitch_trivial_inputs_exact():
    """Samples with a = 0 pack into exactly (0, sum_z b_z X^z)."""
    p = dict(TOY, n=8, N=64)
    keys = oracle.Keys(p, 4243)
    Z = 40
    lwe = np.zeros((Z, p["n"] + 1), np.uint32)
    lwe[:, -1] = np.random.default_rng(4).integers(0, M32, Z, dtype=np.uint64).astype(np.uint32)
    acc = oracle.pack_keyswitch(keys, lwe)
    assert np.all(acc[0] == 0)
    assert np.array_equal(acc[1][:Z], lwe[:, -1]) and np.all(acc[1][Z:] == 0)


def test_pack_keyswitch_packs_the_phases():
    """Z fresh LWE samples of messages m_z / 64 pack into a TRLWE whose phase
    coefficient z is m_z / 64 up to rounding and noise (coefficients >= Z are
    near 0), checked with an independent product; extracting coefficient z
    again gives an LWE sample of m_z / 64."""
    p = TOY
    keys = oracle.Keys(p, 4244)
    Z = 100
    m = np.random.default_rng(5).integers(0, 64, Z).astype(np.uint32)
    lwe = oracle.encrypt(p["n"], keys.s, 91, p["alpha_lwe"], m << 26)
    acc = oracle.pack_keyswitch(keys, lwe)
    ph = trlwe_phase(keys.S, acc).astype(np.int64)
    assert np.array_equal(((ph + (1 << 25)) >> 26) % 64, np.concatenate([m, np.zeros(p["N"] - Z, np.uint32)]))
    err = s32(ph - np.concatenate([m.astype(np.int64) << 26, np.zeros(p["N"] - Z, np.int64)]))
    assert np.max(np.abs(err)) < 2 ** 32 * 2.0 ** -10  # rounding to 16 bits over n = 64 terms, plus noise
    for z in (0, 17, Z - 1):
        e = oracle.sample_extract_at(acc, z)
        assert ((int(oracle.phase(keys.S, e[None])[0]) + (1 << 25)) >> 26) % 64 == m[z]


def test_torus_testvec_generalises_lut_testvec():
    N = 256
    lut = np.random.default_rng(6).integers(0, 8, 8).astype(np.uint32)
    assert np.array_equal(oracle.torus_testvec(N, 3, lut << 28), oracle.lut_testvec(N, 3, lut))


def test_functional_bootstrap_onto_multiples_of_inverse_modulus():
    """Bootstrapping with a test vector of multiples of 1/q (q = p^r = 257)
    maps a 3-bit message m to f(m)/q (Section 3.2, step 4); the result is
    taken before key switching (the next step switches into BGV), with a
    low-noise bootstrapping key as in the N = 2048 LUT parameters: its phase
    under S times q rounds to f(m)."""
    p = dict(TOY, N=512, alpha_bk=2.0 ** -45)
    keys = oracle.Keys(p, 4245)
    q = 257
    f = np.random.default_rng(7).integers(0, q, 8)
    values = np.array([(int(v) * (1 << 32) + q // 2) // q for v in f], dtype=np.uint64).astype(np.uint32)
    tv = oracle.torus_testvec(p["N"], 3, values)
    m = np.arange(8, dtype=np.uint32).repeat(2)
    ct = oracle.encrypt(p["n"], keys.s, 92, p["alpha_lwe"], m << 28)
    out = oracle.bootstrap_no_ks(keys, ct, tv)
    ph = oracle.phase(keys.S, out).astype(np.int64)
    assert np.array_equal(((ph * q + (1 << 31)) >> 32) % q, f[m])


def test_results_do_not_depend_on_the_thread_count():
    """The oracle spreads ciphertexts over OpenMP threads; each bootstrap is
    computed by one thread from its own inputs, so one thread and all of
    them give the same bits (the CPU baseline times both)."""
    keys = oracle.Keys(TOY, 4246)
    rng = np.random.default_rng(8)
    bits = rng.integers(0, 2, (2, 12)).astype(np.uint32)
    mu = np.where(bits == 1, 1 << 29, (1 << 32) - (1 << 29)).astype(np.uint32)  # +-1/8
    ca = oracle.encrypt(TOY["n"], keys.s, 93, TOY["alpha_lwe"], mu[0])
    cb = oracle.encrypt(TOY["n"], keys.s, 94, TOY["alpha_lwe"], mu[1])
    every = oracle.gate_bootstrap(keys, "NAND", ca, cb)
    threads = oracle.threads()
    oracle.set_threads(1)
    try:
        assert oracle.threads() == 1
        one = oracle.gate_bootstrap(keys, "NAND", ca, cb)
    finally:
        oracle.set_threads(threads)
    assert oracle.threads() == threads
    assert np.array_equal(every, one)
