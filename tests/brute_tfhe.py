"""A second, pure-Python implementation of TFHE gate bootstrapping for tiny
parameters (N <= 64, n <= 16), used only to pin the C oracle bit-exactly.

Written separately from the C oracle: polynomials are Python lists of ints,
products are formed in Z[X] first and only then reduced mod X^N + 1 and mod
2^32, rotations are expressed as products with a signed monomial, and the
gadget decomposition is computed digit by digit from the rounded value.  The
shared part is the convention (the generator, rounding rules and layouts),
which each side implements on its own.
"""
from __future__ import annotations

import math

M32 = 1 << 32
M64 = (1 << 64) - 1
GAMMA = 0x9E3779B97F4A7C15


def _mix(z: int) -> int:
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & M64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & M64
    return z ^ (z >> 31)


def word(seed: int, tag: int, idx: int) -> int:
    key = _mix((seed + (tag + 1) * GAMMA) & M64)
    return _mix((key + (idx + 1) * GAMMA) & M64)


def torus(seed, tag, idx):
    return word(seed, tag, idx) >> 32


def noise(seed, tag, idx, alpha):
    w1, w2 = word(seed, tag, 2 * idx), word(seed, tag, 2 * idx + 1)
    u1 = float((w1 >> 11) + 1) * 2.0 ** -53
    u2 = float(w2 >> 11) * 2.0 ** -53
    z = math.sqrt(-2.0 * math.log(u1)) * math.cos(6.283185307179586 * u2)
    x = z * (alpha * 4294967296.0)
    # llround: nearest, ties away from zero
    e = int(math.floor(abs(x) + 0.5)) * (1 if x >= 0 else -1)
    return e % M32


def polymul_negacyclic(a, b):
    N = len(a)
    full = [0] * (2 * N - 1)
    for i, ai in enumerate(a):
        if ai:
            for j, bj in enumerate(b):
                full[i + j] += ai * bj
    out = full[:N] + [0]
    for k in range(N, 2 * N - 1):
        out[k - N] -= full[k]
    return [x % M32 for x in out[:N]]


def monomial(N, e):
    """X^e as a coefficient list in Z[X]/(X^N+1), e in [0, 2N)."""
    m = [0] * N
    if e < N:
        m[e] = 1
    else:
        m[e - N] = -1
    return m


def mod_switch(x, N):
    # round(x * 2N / 2^32) with ties upward, then mod 2N
    num = x * 2 * N
    q, r = divmod(num, M32)
    if 2 * r >= M32:
        q += 1
    return q % (2 * N)


def signed(x):
    x %= M32
    return x - M32 if x >= M32 // 2 else x


def decompose(x, l, bg_bit):
    """Digits d_1..d_l in [-Bg/2, Bg/2) with sum d_j 2^(32-j bg) = x rounded."""
    Bg = 1 << bg_bit
    shift = 32 - l * bg_bit
    # nearest multiple of 2^shift, ties upward, as a residue in units of 2^shift
    v = ((x + ((1 << shift) >> 1)) % M32) >> shift if shift > 0 else x % M32
    digits = []
    carry = 0
    for j in range(l, 0, -1):  # least significant digit first
        d = (v & (Bg - 1)) + carry
        v >>= bg_bit
        if d >= Bg // 2:
            d -= Bg
            carry = 1
        else:
            carry = 0
        digits.append(d)
    return digits[::-1]


def keygen(p, seed):
    n, N, l, bg = p["n"], p["N"], p["l"], p["bg_bit"]
    s = [word(seed, 1, i) & 1 for i in range(n)]
    S = [word(seed, 2, j) & 1 for j in range(N)]
    bk = []
    for i in range(n):
        rows = []
        for r in range(2 * l):
            base = (i * 2 * l + r) * N
            A = [torus(seed, 3, base + m) for m in range(N)]
            AS = polymul_negacyclic(A, S)
            B = [(AS[m] + noise(seed, 4, base + m, p["alpha_bk"])) % M32 for m in range(N)]
            q, j = divmod(r, l)
            g = s[i] << (32 - (j + 1) * bg)
            if q == 0:
                A[0] = (A[0] + g) % M32
            else:
                B[0] = (B[0] + g) % M32
            rows.append((A, B))
        bk.append(rows)
    t, bb = p["ks_t"], p["ks_basebit"]
    base = 1 << bb
    ksk = {}
    u = 0
    for i in range(N):
        for j in range(t):
            for v in range(1, base):
                a = [torus(seed, 5, u * n + k) for k in range(n)]
                msg = (v * S[i] << (32 - (j + 1) * bb)) % M32
                b = (sum(x * y for x, y in zip(a, s)) + msg + noise(seed, 6, u, p["alpha_ks"])) % M32
                ksk[(i, j, v)] = a + [b]
                u += 1
    return s, S, bk, ksk


def encrypt(key, seed, alpha, mu, index):
    dim = len(key)
    a = [torus(seed, 7, index * dim + k) for k in range(dim)]
    b = (sum(x * y for x, y in zip(a, key)) + mu + noise(seed, 8, index, alpha)) % M32
    return a + [b]


def phase(key, ct):
    return (ct[-1] - sum(x * y for x, y in zip(ct[:-1], key))) % M32


GATE_TABLE = {  # (constant in units of 1/8, weight of a, weight of b)
    "NAND": (1, -1, -1), "AND": (-1, 1, 1), "OR": (1, 1, 1), "NOR": (-1, -1, -1),
    "XOR": (2, 2, 2), "XNOR": (-2, -2, -2), "ANDNY": (-1, -1, 1), "ANDYN": (-1, 1, -1),
    "ORNY": (1, -1, 1), "ORYN": (1, 1, -1),
}


def bootstrap(p, bk, ksk, lwe, testvec, keyswitch=True):
    n, N, l, bg = p["n"], p["N"], p["l"], p["bg_bit"]
    bbar = mod_switch(lwe[n], N)
    acc_a = [0] * N
    acc_b = polymul_negacyclic(monomial(N, (2 * N - bbar) % (2 * N)), testvec)
    for i in range(n):
        abar = mod_switch(lwe[i], N)
        X = monomial(N, abar)
        Da = [(x - y) % M32 for x, y in zip(polymul_negacyclic(X, acc_a), acc_a)]
        Db = [(x - y) % M32 for x, y in zip(polymul_negacyclic(X, acc_b), acc_b)]
        digit_polys = []
        for D in (Da, Db):
            per_coef = [decompose(x, l, bg) for x in D]
            for j in range(l):
                digit_polys.append([per_coef[m][j] for m in range(N)])
        new_a, new_b = list(acc_a), list(acc_b)
        for r, dp in enumerate(digit_polys):
            A, B = bk[i][r]
            pa, pb = polymul_negacyclic(dp, A), polymul_negacyclic(dp, B)
            new_a = [(x + y) % M32 for x, y in zip(new_a, pa)]
            new_b = [(x + y) % M32 for x, y in zip(new_b, pb)]
        acc_a, acc_b = new_a, new_b
    ext = [acc_a[0]] + [(-acc_a[N - j]) % M32 for j in range(1, N)] + [acc_b[0]]
    if not keyswitch:
        return ext
    t, bb = p["ks_t"], p["ks_basebit"]
    prec = t * bb
    out = [0] * n + [ext[N]]
    for i in range(N):
        x = ext[i]
        r = x if prec == 32 else ((x + (1 << (31 - prec))) % M32) >> (32 - prec)
        for j in range(t):
            v = (r >> ((t - 1 - j) * bb)) & ((1 << bb) - 1)
            if v:
                row = ksk[(i, j, v)]
                out = [(o - w) % M32 for o, w in zip(out, row)]
    return out


def gate(p, bk, ksk, name, ca, cb):
    k, wa, wb = GATE_TABLE[name]
    n = p["n"]
    comb = [(wa * x + wb * y) % M32 for x, y in zip(ca, cb)]
    comb[n] = (comb[n] + k * (1 << 29)) % M32
    return bootstrap(p, bk, ksk, comb, [1 << 29] * p["N"])
