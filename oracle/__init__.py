"""TEST INFRASTRUCTURE ONLY: ctypes wrapper of the CPU oracle (tfhe_oracle.c).

The oracle is a plain, slow CPU implementation of TFHE gate bootstrapping
(modulus switch, blind rotation with schoolbook negacyclic products, sample
extraction, key switching), the Glyph forward ReLU and backward iReLU units,
the homomorphic multiplexer and the softmax's multiplexer-tree table lookup,
the look-up-table bootstrap, and the TFHE steps of the cryptosystem switch
(packing key switching, SampleExtract of any coefficient, bootstrapping onto
arbitrary torus values).  Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s
``cpu_baseline`` leg may import this package; the GPU library never does, and
the two share no code.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "tfhe_oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")

# gcc, no fast-math and no FP contraction: the Gaussian noise goes through
# glibc's scalar log/cos/sqrt exactly as written
CFLAGS = ["-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off",
          "-fno-fast-math", "-Wall", "-Wextra", "-Wno-unused-parameter"]

GATES = {"NAND": 0, "AND": 1, "OR": 2, "NOR": 3, "XOR": 4, "XNOR": 5,
         "ANDNY": 6, "ANDYN": 7, "ORNY": 8, "ORYN": 9}

MU = 1 << 29  # 1/8 on the torus


def build(verbose: bool = False) -> str:
    """Compile liboracle.so with gcc (always recompiles)."""
    cmd = ["gcc", *CFLAGS, "-o", _LIB_PATH + ".tmp", _SRC, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(_LIB_PATH + ".tmp", _LIB_PATH)
    return _LIB_PATH


class Params(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int32), ("N", ctypes.c_int32), ("l", ctypes.c_int32),
                ("bg_bit", ctypes.c_int32), ("ks_t", ctypes.c_int32),
                ("ks_basebit", ctypes.c_int32), ("alpha_lwe", ctypes.c_double),
                ("alpha_bk", ctypes.c_double), ("alpha_ks", ctypes.c_double)]


_lib = None
_u32p = ctypes.POINTER(ctypes.c_uint32)
_i32p = ctypes.POINTER(ctypes.c_int32)
_i64p = ctypes.POINTER(ctypes.c_int64)


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
        build()
    lib = ctypes.CDLL(_LIB_PATH)
    P = ctypes.POINTER(Params)
    sig = {
        "oracle_stream_output": (ctypes.c_uint64, [ctypes.c_uint64, ctypes.c_uint64]),
        "oracle_word": (ctypes.c_uint64, [ctypes.c_uint64, ctypes.c_uint32, ctypes.c_uint64]),
        "oracle_gauss": (ctypes.c_double, [ctypes.c_uint64, ctypes.c_uint32, ctypes.c_uint64]),
        "oracle_noise": (ctypes.c_uint32, [ctypes.c_uint64, ctypes.c_uint32, ctypes.c_uint64, ctypes.c_double]),
        "oracle_negacyclic_mul": (None, [ctypes.c_int32, _u32p, _u32p, _u32p]),
        "oracle_rotate": (None, [ctypes.c_int32, _u32p, ctypes.c_uint32, _u32p]),
        "oracle_decompose": (None, [ctypes.c_int32, ctypes.c_int32, ctypes.c_uint32, _i32p]),
        "oracle_mod_switch": (ctypes.c_uint32, [ctypes.c_uint32, ctypes.c_int32]),
        "oracle_mod_switch_batch": (None, [_u32p, ctypes.c_int64, ctypes.c_int32, _u32p]),
        "oracle_bk_words": (ctypes.c_int64, [P]),
        "oracle_ksk_words": (ctypes.c_int64, [P]),
        "oracle_keygen": (None, [P, ctypes.c_uint64, _u32p, _u32p, _u32p, _u32p]),
        "oracle_encrypt": (None, [ctypes.c_int32, _u32p, ctypes.c_uint64, ctypes.c_double, _u32p,
                                  ctypes.c_int64, ctypes.c_int64, _u32p]),
        "oracle_phase": (None, [ctypes.c_int32, _u32p, _u32p, ctypes.c_int64, _u32p]),
        "oracle_gate_combine": (None, [P, ctypes.c_int32, _u32p, _u32p, _u32p]),
        "oracle_blind_rotate": (None, [P, _u32p, _u32p, _u32p, _u32p]),
        "oracle_cmux": (None, [P, _u32p, ctypes.c_uint32, _u32p]),
        "oracle_sample_extract": (None, [ctypes.c_int32, _u32p, _u32p]),
        "oracle_keyswitch": (None, [P, _u32p, _u32p, _u32p, ctypes.c_int64]),
        "oracle_lut_testvec": (None, [ctypes.c_int32, ctypes.c_int32, _u32p, _u32p]),
        "oracle_gate_bootstrap": (None, [P, _u32p, _u32p, ctypes.c_int32, _u32p, _u32p, _u32p,
                                         ctypes.c_int64]),
        "oracle_bootstrap_no_ks": (None, [P, _u32p, _u32p, _u32p, _u32p, ctypes.c_int64]),
        "oracle_lut_bootstrap": (None, [P, _u32p, _u32p, _u32p, _u32p, _u32p, ctypes.c_int64]),
        "oracle_relu_gates": (None, [P, _u32p, _u32p, _u32p, ctypes.c_int32, _i64p, ctypes.c_int64,
                                     _u32p]),
        "oracle_not": (None, [ctypes.c_int32, _u32p, _u32p, ctypes.c_int64]),
        "oracle_threads": (ctypes.c_int, []),
        "oracle_set_threads": (None, [ctypes.c_int]),
        "oracle_pks_words": (ctypes.c_int64, [P]),
        "oracle_packing_keygen": (None, [P, ctypes.c_uint64, _u32p, _u32p, _u32p]),
        "oracle_pack_keyswitch": (None, [P, _u32p, _u32p, ctypes.c_int32, _u32p]),
        "oracle_sample_extract_at": (None, [ctypes.c_int32, _u32p, ctypes.c_int32, _u32p]),
        "oracle_torus_testvec": (None, [ctypes.c_int32, ctypes.c_int32, _u32p, _u32p]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    _lib = lib
    return lib


def _u32(a: np.ndarray):
    assert a.dtype == np.uint32 and a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(_u32p)


def params(n, N, l, bg_bit, ks_t, ks_basebit, alpha_lwe, alpha_bk, alpha_ks=None) -> Params:
    return Params(n, N, l, bg_bit, ks_t, ks_basebit, alpha_lwe, alpha_bk,
                  alpha_lwe if alpha_ks is None else alpha_ks)


def as_params(d) -> Params:
    """Params from a mapping with the keys of the config tables."""
    if isinstance(d, Params):
        return d
    return params(d["n"], d["N"], d["l"], d["bg_bit"], d["ks_t"], d["ks_basebit"],
                  d["alpha_lwe"], d["alpha_bk"], d.get("alpha_ks"))


# ---- thin functional wrappers ------------------------------------------

def stream_output(state, k):
    return _load().oracle_stream_output(state, k)


def word(seed, tag, idx):
    return _load().oracle_word(seed, tag, idx)


def gauss(seed, tag, idx):
    return _load().oracle_gauss(seed, tag, idx)


def noise(seed, tag, idx, alpha):
    return _load().oracle_noise(seed, tag, idx, alpha)


def negacyclic_mul(a, b):
    a = np.ascontiguousarray(a, dtype=np.uint32)
    b = np.ascontiguousarray(b, dtype=np.uint32)
    c = np.zeros_like(a)
    _load().oracle_negacyclic_mul(len(a), _u32(a), _u32(b), _u32(c))
    return c


def rotate(p, e):
    p = np.ascontiguousarray(p, dtype=np.uint32)
    out = np.zeros_like(p)
    _load().oracle_rotate(len(p), _u32(p), e, _u32(out))
    return out


def decompose(l, bg_bit, x):
    d = (ctypes.c_int32 * l)()
    _load().oracle_decompose(l, bg_bit, x, d)
    return list(d)


def mod_switch(x, N):
    return _load().oracle_mod_switch(x, N)


def mod_switch_array(x, N):
    """mod_switch of every word of x (any shape)."""
    x = np.ascontiguousarray(x, dtype=np.uint32)
    out = np.zeros_like(x)
    _load().oracle_mod_switch_batch(_u32(x), x.size, N, _u32(out))
    return out


class Keys:
    """Secret and evaluation keys produced by oracle_keygen."""

    def __init__(self, p, seed):
        p = as_params(p)
        lib = _load()
        self.p = p
        self.seed = seed
        self.s = np.zeros(p.n, np.uint32)
        self.S = np.zeros(p.N, np.uint32)
        self.bk = np.zeros(lib.oracle_bk_words(ctypes.byref(p)), np.uint32)
        self.ksk = np.zeros(lib.oracle_ksk_words(ctypes.byref(p)), np.uint32)
        lib.oracle_keygen(ctypes.byref(p), seed, _u32(self.s), _u32(self.S), _u32(self.bk),
                          _u32(self.ksk))

    def bk_view(self):
        p = self.p
        return self.bk.reshape(p.n, 2 * p.l, 2, p.N)

    def ksk_view(self):
        p = self.p
        return self.ksk.reshape(p.N, p.ks_t, (1 << p.ks_basebit) - 1, p.n + 1)

    def packing_key(self):
        """Packing key of the functional key switching (computed on first use)."""
        if getattr(self, "pks", None) is None:
            p = self.p
            lib = _load()
            self.pks = np.zeros(lib.oracle_pks_words(ctypes.byref(p)), np.uint32)
            lib.oracle_packing_keygen(ctypes.byref(p), self.seed, _u32(self.s), _u32(self.S), _u32(self.pks))
        return self.pks


def encrypt(dim, key, seed, alpha, mu, first_index=0):
    mu = np.ascontiguousarray(mu, dtype=np.uint32).ravel()
    key = np.ascontiguousarray(key, dtype=np.uint32)
    ct = np.zeros((len(mu), dim + 1), np.uint32)
    _load().oracle_encrypt(dim, _u32(key), seed, alpha, _u32(mu), first_index, len(mu), _u32(ct))
    return ct


def phase(key, ct):
    key = np.ascontiguousarray(key, dtype=np.uint32)
    ct = np.ascontiguousarray(ct, dtype=np.uint32)
    dim = ct.shape[-1] - 1
    count = ct.size // (dim + 1)
    out = np.zeros(count, np.uint32)
    _load().oracle_phase(dim, _u32(key), _u32(ct), count, _u32(out))
    return out.reshape(ct.shape[:-1])


def gate_combine(p, gate, ca, cb):
    p = as_params(p)
    out = np.zeros(p.n + 1, np.uint32)
    _load().oracle_gate_combine(ctypes.byref(p), GATES.get(gate, gate),
                                _u32(np.ascontiguousarray(ca, np.uint32)),
                                _u32(np.ascontiguousarray(cb, np.uint32)), _u32(out))
    return out


def blind_rotate(keys: Keys, lwe, testvec):
    p = keys.p
    acc = np.zeros(2 * p.N, np.uint32)
    _load().oracle_blind_rotate(ctypes.byref(p), _u32(keys.bk),
                                _u32(np.ascontiguousarray(lwe, np.uint32)),
                                _u32(np.ascontiguousarray(testvec, np.uint32)), _u32(acc))
    return acc.reshape(2, p.N)


def cmux(keys: Keys, i, abar, acc):
    p = keys.p
    acc = np.array(acc, dtype=np.uint32).ravel()
    bk_i = np.ascontiguousarray(keys.bk_view()[i]).ravel()
    _load().oracle_cmux(ctypes.byref(p), _u32(bk_i), abar, _u32(acc))
    return acc.reshape(2, p.N)


def cmux_row(p, bk_row, abar, acc):
    """One CMux with a given key row bk_row ([2l][2][N] words, coefficient
    domain) on the accumulator acc ([2][N]) rotated by abar."""
    p = as_params(p)
    acc = np.array(acc, dtype=np.uint32).ravel()
    bk_row = np.ascontiguousarray(bk_row, dtype=np.uint32).ravel()
    assert bk_row.size == 2 * p.l * 2 * p.N and acc.size == 2 * p.N
    _load().oracle_cmux(ctypes.byref(p), _u32(bk_row), abar, _u32(acc))
    return acc.reshape(2, p.N)


def sample_extract(acc):
    acc = np.ascontiguousarray(acc, dtype=np.uint32).ravel()
    N = len(acc) // 2
    out = np.zeros(N + 1, np.uint32)
    _load().oracle_sample_extract(N, _u32(acc), _u32(out))
    return out


def keyswitch(keys: Keys, ext):
    p = keys.p
    ext = np.ascontiguousarray(ext, dtype=np.uint32)
    count = ext.size // (p.N + 1)
    out = np.zeros((count, p.n + 1), np.uint32)
    _load().oracle_keyswitch(ctypes.byref(p), _u32(keys.ksk), _u32(ext), _u32(out), count)
    return out


def lut_testvec(N, msg_bits, lut):
    lut = np.ascontiguousarray(lut, dtype=np.uint32)
    tv = np.zeros(N, np.uint32)
    _load().oracle_lut_testvec(N, msg_bits, _u32(lut), _u32(tv))
    return tv


def gate_testvec(N):
    return np.full(N, MU, np.uint32)


def gate_bootstrap(keys: Keys, gate, ca, cb):
    p = keys.p
    ca = np.ascontiguousarray(ca, dtype=np.uint32)
    cb = np.ascontiguousarray(cb, dtype=np.uint32)
    count = ca.size // (p.n + 1)
    out = np.zeros((count, p.n + 1), np.uint32)
    _load().oracle_gate_bootstrap(ctypes.byref(p), _u32(keys.bk), _u32(keys.ksk),
                                  GATES.get(gate, gate), _u32(ca), _u32(cb), _u32(out), count)
    return out


def bootstrap_no_ks(keys: Keys, lwe, testvec):
    p = keys.p
    lwe = np.ascontiguousarray(lwe, dtype=np.uint32)
    count = lwe.size // (p.n + 1)
    out = np.zeros((count, p.N + 1), np.uint32)
    _load().oracle_bootstrap_no_ks(ctypes.byref(p), _u32(keys.bk), _u32(lwe),
                                   _u32(np.ascontiguousarray(testvec, np.uint32)), _u32(out), count)
    return out


def lut_bootstrap(keys: Keys, lwe, testvec):
    p = keys.p
    lwe = np.ascontiguousarray(lwe, dtype=np.uint32)
    count = lwe.size // (p.n + 1)
    out = np.zeros((count, p.n + 1), np.uint32)
    _load().oracle_lut_bootstrap(ctypes.byref(p), _u32(keys.bk), _u32(keys.ksk), _u32(lwe),
                                 _u32(np.ascontiguousarray(testvec, np.uint32)), _u32(out), count)
    return out


def relu_gates(keys: Keys, x, bits, gate_ids):
    """Outputs of the given gate indices of the forward ReLU over x[V][bits][n+1]."""
    p = keys.p
    x = np.ascontiguousarray(x, dtype=np.uint32)
    ids = np.ascontiguousarray(gate_ids, dtype=np.int64)
    out = np.zeros((len(ids), p.n + 1), np.uint32)
    _load().oracle_relu_gates(ctypes.byref(p), _u32(keys.bk), _u32(keys.ksk), _u32(x), bits,
                              ids.ctypes.data_as(_i64p), len(ids), _u32(out))
    return out


def relu(keys: Keys, x, bits):
    """Full forward ReLU: gates for bits < bits-1, trivial false for the sign."""
    p = keys.p
    x = np.ascontiguousarray(x, dtype=np.uint32).reshape(-1, bits, p.n + 1)
    V = x.shape[0]
    ids = np.arange(V * (bits - 1), dtype=np.int64)
    g = relu_gates(keys, x, bits, ids).reshape(V, bits - 1, p.n + 1)
    y = np.zeros_like(x)
    y[:, : bits - 1] = g
    y[:, bits - 1, p.n] = np.uint32((1 << 32) - MU)
    return y


def irelu_gates(keys: Keys, u, u_bits, delta, bits, gate_ids):
    """Outputs of the given gates of the backward iReLU (Section 3.1,
    "Backward iReLU"): gate g is bit i = g % bits of value v = g // bits,
    AND(NOT u[v][u_bits-1], delta[v][i]) -- the error bit where the forward
    pre-activation's sign is 0, else 0.  Every bit of the error is gated, the
    sign bit included."""
    p = keys.p
    u = np.ascontiguousarray(u, dtype=np.uint32).reshape(-1, u_bits, p.n + 1)
    delta = np.ascontiguousarray(delta, dtype=np.uint32).reshape(-1, bits, p.n + 1)
    ids = np.asarray(gate_ids, dtype=np.int64)
    v, i = ids // bits, ids % bits
    return gate_bootstrap(keys, "ANDNY", u[v, u_bits - 1], delta[v, i])


def irelu(keys: Keys, u, u_bits, delta, bits):
    """Full backward iReLU over delta[V][bits][n+1]."""
    p = keys.p
    V = np.asarray(delta).size // (bits * (p.n + 1))
    return irelu_gates(keys, u, u_bits, delta, bits, np.arange(V * bits)).reshape(V, bits, p.n + 1)


def mux(keys: Keys, c, a, b):
    """Homomorphic multiplexer c ? a : b on encrypted bits (the unit of the
    softmax lookup, Section 3.1 "Forward Softmax"): bootstrap AND(c, a) and
    AND(NOT c, b) to dimension N without key switching, add the two samples
    and the constant 1/8 (true + false + 1/8 = 1/8, false + false + 1/8 =
    -1/8), then key-switch once."""
    p = keys.p
    c = np.asarray(c, dtype=np.uint32).reshape(-1, p.n + 1)
    a = np.asarray(a, dtype=np.uint32).reshape(-1, p.n + 1)
    b = np.asarray(b, dtype=np.uint32).reshape(-1, p.n + 1)
    M = len(c)
    halves = [gate_combine(p, "AND", c[e], a[e]) for e in range(M)]
    halves += [gate_combine(p, "ANDNY", c[e], b[e]) for e in range(M)]
    ext = bootstrap_no_ks(keys, np.stack(halves), gate_testvec(p.N))
    s = (ext[:M].astype(np.uint64) + ext[M:].astype(np.uint64)) & 0xFFFFFFFF
    s[:, p.N] = (s[:, p.N] + MU) & 0xFFFFFFFF
    return keyswitch(keys, s.astype(np.uint32))


def mux_lut(keys: Keys, x, msg_bits, table, out_bits):
    """Table lookup by a tree of multiplexers (the paper's softmax
    exponentiation unit): x[v] holds msg_bits encrypted bits, LSB first,
    selecting entry k = sum x[v][i] 2^i of the public table; the result holds
    the out_bits bits of table[k].  Tree level 1 picks between constants with
    x[v][0] (a constant, x[v][0] or NOT x[v][0], no bootstrap); level i picks
    between the level i-1 nodes 2j (bit 0) and 2j + 1 (bit 1) with x[v][i-1]."""
    p = keys.p
    x = np.asarray(x, dtype=np.uint32).reshape(-1, msg_bits, p.n + 1)
    table = np.asarray(table, dtype=np.int64)
    V = len(x)
    triv = lambda bit: np.concatenate([np.zeros(p.n, np.uint32),
                                       np.array([MU if bit else (1 << 32) - MU], np.uint32)])
    # nodes[v][o] = list of ciphertexts of the current level
    nodes = [[None] * out_bits for _ in range(V)]
    for v in range(V):
        for o in range(out_bits):
            lvl = []
            for j in range(1 << (msg_bits - 1)):
                b0, b1 = (table[2 * j] >> o) & 1, (table[2 * j + 1] >> o) & 1
                lvl.append(triv(b0) if b0 == b1 else (x[v][0].copy() if b1 else not_gate(x[v][0])))
            nodes[v][o] = lvl
    for level in range(1, msg_bits):
        sel, ta, fb, where = [], [], [], []
        for v in range(V):
            for o in range(out_bits):
                for j in range(len(nodes[v][o]) // 2):
                    sel.append(x[v][level]); ta.append(nodes[v][o][2 * j + 1]); fb.append(nodes[v][o][2 * j])
                    where.append((v, o))
        res = mux(keys, np.stack(sel), np.stack(ta), np.stack(fb))
        new = [[[] for _ in range(out_bits)] for _ in range(V)]
        for (v, o), r in zip(where, res):
            new[v][o].append(r)
        nodes = new
    return np.stack([np.stack([nodes[v][o][0] for o in range(out_bits)]) for v in range(V)])


def pack_keyswitch(keys: Keys, lwe):
    """Functional key switching of Z LWE samples into one TRLWE sample whose
    phase is sum_z phase_z X^z (Section 3.2, step 2); returns [2][N]."""
    p = keys.p
    lwe = np.ascontiguousarray(lwe, dtype=np.uint32).reshape(-1, p.n + 1)
    out = np.zeros(2 * p.N, np.uint32)
    _load().oracle_pack_keyswitch(ctypes.byref(p), _u32(keys.packing_key()), _u32(lwe), len(lwe), _u32(out))
    return out.reshape(2, p.N)


def sample_extract_at(acc, idx):
    """LWE sample of coefficient idx of the TRLWE sample acc ([2][N])."""
    acc = np.ascontiguousarray(acc, dtype=np.uint32).ravel()
    N = len(acc) // 2
    out = np.zeros(N + 1, np.uint32)
    _load().oracle_sample_extract_at(N, _u32(acc), idx, _u32(out))
    return out


def torus_testvec(N, msg_bits, values):
    values = np.ascontiguousarray(values, dtype=np.uint32)
    tv = np.zeros(N, np.uint32)
    _load().oracle_torus_testvec(N, msg_bits, _u32(values), _u32(tv))
    return tv


def not_gate(ct):
    ct = np.ascontiguousarray(ct, dtype=np.uint32)
    return (np.uint32(0) - ct).astype(np.uint32)


def threads():
    return _load().oracle_threads()


def set_threads(n: int):
    """Threads of later oracle calls from this thread (timing only)."""
    _load().oracle_set_threads(int(n))
