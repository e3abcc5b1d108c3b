"""Python binding of libglyph_tfhe.so (include/glyph_tfhe.h).

Argument marshalling only: every step of the path runs in the library's HIP
kernels.  Device buffers are torch tensors on a ROCm device (int32 tensors
hold the raw uint32 torus words); streams are torch streams.  Host buffers are
numpy uint32 arrays.  The functions carry the C names.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libglyph_tfhe.so")

TFHE_OK, TFHE_EINVAL, TFHE_EUNSUPPORTED, TFHE_ENOMEM, TFHE_EHIP, TFHE_EDEVICE = 0, -1, -2, -3, -4, -5
GATES = {"NAND": 0, "AND": 1, "OR": 2, "NOR": 3, "XOR": 4, "XNOR": 5,
         "ANDNY": 6, "ANDYN": 7, "ORNY": 8, "ORYN": 9}
MU = 1 << 29


class TfheError(RuntimeError):
    def __init__(self, rc: int, msg: str):
        super().__init__(f"{msg} (rc={rc})")
        self.rc = rc


class tfhe_params(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int32), ("N", ctypes.c_int32), ("l", ctypes.c_int32),
                ("bg_bit", ctypes.c_int32), ("ks_t", ctypes.c_int32),
                ("ks_basebit", ctypes.c_int32), ("alpha_lwe", ctypes.c_double),
                ("alpha_bk", ctypes.c_double), ("alpha_ks", ctypes.c_double)]


def make_params(d) -> tfhe_params:
    if isinstance(d, tfhe_params):
        return d
    return tfhe_params(d["n"], d["N"], d["l"], d["bg_bit"], d["ks_t"], d["ks_basebit"],
                       d["alpha_lwe"], d["alpha_bk"], d.get("alpha_ks", d["alpha_lwe"]))


_lib = None
_vp = ctypes.c_void_p
_i64 = ctypes.c_int64
_i32 = ctypes.c_int32
_u64 = ctypes.c_uint64

_SIGNATURES = {
    "tfhe_strerror": (ctypes.c_char_p, [ctypes.c_int]),
    "tfhe_last_error": (ctypes.c_char_p, []),
    "tfhe_keygen_from_seed": (ctypes.c_int, [_vp, _u64, ctypes.c_int, _vp, _vp]),
    "tfhe_secret_keygen": (ctypes.c_int, [_vp, _u64, _vp]),
    "tfhe_eval_key_upload": (ctypes.c_int, [_vp, ctypes.c_int, _vp]),
    "tfhe_secret_key_free": (None, [_vp]),
    "tfhe_eval_key_free": (None, [_vp]),
    "tfhe_eval_key_params": (ctypes.c_int, [_vp, _vp]),
    "tfhe_export_keys": (ctypes.c_int, [_vp, _vp, _vp, _vp, _vp]),
    "tfhe_encrypt_torus": (ctypes.c_int, [_vp, _u64, _vp, _i64, _i64, _vp]),
    "tfhe_decrypt_phase": (ctypes.c_int, [_vp, ctypes.c_int, _vp, _i64, _vp]),
    "tfhe_lut_testvec": (ctypes.c_int, [_i32, _i32, _vp, _vp]),
    "tfhe_workspace_bytes": (_i64, [_vp, _i64]),
    "tfhe_gate_bootstrap_batch": (ctypes.c_int, [_vp, ctypes.c_int, _vp, _vp, _vp, _i64, _vp, _i64, _vp]),
    "tfhe_lut_bootstrap_batch": (ctypes.c_int, [_vp, _vp, _vp, _vp, _i64, _vp, _i64, _vp]),
    "tfhe_bootstrap_extract_batch": (ctypes.c_int, [_vp, _vp, _vp, _vp, _i64, _vp, _i64, _vp]),
    "tfhe_keyswitch_batch": (ctypes.c_int, [_vp, _vp, _vp, _i64, _vp]),
    "glyph_relu_batch": (ctypes.c_int, [_vp, _vp, _vp, _i64, _i32, _i64, _i64, _vp, _i64, _vp]),
    "glyph_irelu_batch": (ctypes.c_int, [_vp, _vp, _i32, _vp, _vp, _i64, _i32, _i64, _i64, _vp, _i64, _vp]),
    "tfhe_mux_batch": (ctypes.c_int, [_vp, _vp, _vp, _vp, _vp, _i64, _vp, _i64, _vp]),
    "glyph_mux_lut_batch": (ctypes.c_int, [_vp, _vp, _i32, _vp, _i32, _vp, _i64, _vp, _i64, _vp]),
    "glyph_mux_lut_workspace_bytes": (_i64, [_vp, _i64, _i32, _i32]),
    "tfhe_packing_key_upload": (ctypes.c_int, [_vp, _vp]),
    "tfhe_export_packing_key": (ctypes.c_int, [_vp, _vp]),
    "tfhe_pack_keyswitch_batch": (ctypes.c_int, [_vp, _vp, _i32, _vp, _i64, _vp]),
    "tfhe_sample_extract_batch": (ctypes.c_int, [_i32, _vp, _i64, _i32, _vp, _vp]),
    "tfhe_torus_testvec": (ctypes.c_int, [_i32, _i32, _vp, _vp]),
    "tfhe_not_batch": (ctypes.c_int, [_i32, _vp, _vp, _i64, _vp]),
    "tfhe_negacyclic_mul_batch": (ctypes.c_int, [_vp, _vp, _vp, _vp, _i64, _vp]),
    "tfhe_transform_error_bound": (ctypes.c_int, [_vp, _vp, _vp]),
    "tfhe_gate_bootstrap_batch_noalloc": (ctypes.c_int, [_vp, ctypes.c_int, _vp, _vp, _vp, _i64, _vp]),
    "tfhe_debug_mod_switch_batch": (ctypes.c_int, [_vp, ctypes.c_int, _vp, _vp, _vp, _i64, _vp]),
    "tfhe_debug_cmux_workspace_bytes": (_i64, [_vp, _i64]),
    "tfhe_debug_cmux_batch": (ctypes.c_int, [_vp, _vp, _vp, _vp, _vp, _i64, _vp, _i64, _vp]),
    "tfhe_stage_timing": (ctypes.c_int, [ctypes.c_int]),
    "tfhe_stage_times": (ctypes.c_int, [_vp, _vp]),
    "tfhe_probe_valu_rate": (ctypes.c_int, [ctypes.c_int, _i64, _i64, _vp, _vp]),
}


def lib():
    """The loaded library.  Raises if it has not been built: there is no
    fallback path."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() first")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGNATURES.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def _check(rc: int):
    if rc != TFHE_OK:
        raise TfheError(rc, lib().tfhe_last_error().decode() or lib().tfhe_strerror(rc).decode())


def _host_u32(a) -> np.ndarray:
    a = np.ascontiguousarray(a)
    if a.dtype != np.uint32:
        a = a.astype(np.uint32)
    return a


def _hptr(a: np.ndarray):
    return ctypes.c_void_p(a.ctypes.data)


def _dptr(t):
    """Device pointer of a torch tensor (must be contiguous and on a GPU)."""
    if not t.is_cuda:
        raise ValueError("expected a device tensor")
    if not t.is_contiguous():
        raise ValueError("expected a contiguous tensor")
    return ctypes.c_void_p(t.data_ptr())


def _dbuf(t, words: int, name: str, device=None):
    """Device pointer of a buffer of at least `words` 32-bit words: the C ABI
    takes plain pointers, so sizes, element width and device are checked
    here, before any kernel can touch memory outside the tensor."""
    if t.element_size() != 4:
        raise ValueError(f"{name}: expected 32-bit elements, got {t.dtype}")
    if t.numel() < words:
        raise ValueError(f"{name}: {t.numel()} words, the call needs {words}")
    if device is not None and t.is_cuda and t.device.index != device:
        raise ValueError(f"{name}: on cuda:{t.device.index}, the key is on cuda:{device}")
    return _dptr(t)


def _wsbuf(ws, device):
    """(pointer, size in bytes) of a workspace tensor on the key's device."""
    if ws.is_cuda and ws.device.index != device:
        raise ValueError(f"workspace: on cuda:{ws.device.index}, the key is on cuda:{device}")
    return _dptr(ws), ws.numel() * ws.element_size()


def _stream(stream, device, *tensors):
    """Handle of the HIP stream a call enqueues on: `stream`, else the
    current stream of the key's device.  The device buffers handed to a
    caller-given stream are recorded on it (torch's record_stream): once
    Python drops one (a workspace allocated here, an input the caller lets
    go), the caching allocator would otherwise give its memory to the next
    allocation on another stream while the call may still be running."""
    import torch
    if stream is None:
        return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)
    for t in tensors:
        if t is not None and t.is_cuda:
            t.record_stream(stream)
    return ctypes.c_void_p(stream.cuda_stream)


# ---------------------------------------------------------------- keys

class SecretKey:
    def __init__(self, handle, params: tfhe_params):
        self._h = handle
        self.params = params

    @property
    def handle(self):
        return self._h

    def __del__(self):
        if getattr(self, "_h", None) and _lib is not None:
            _lib.tfhe_secret_key_free(self._h)
            self._h = None


class EvalKey:
    def __init__(self, handle, params: tfhe_params, device: int):
        self._h = handle
        self.params = params
        self.device = device

    @property
    def handle(self):
        return self._h

    def free(self):
        if getattr(self, "_h", None) and _lib is not None:
            _lib.tfhe_eval_key_free(self._h)
            self._h = None

    def __del__(self):
        self.free()


def tfhe_secret_keygen(params, seed: int) -> SecretKey:
    p = make_params(params)
    h = ctypes.c_void_p()
    _check(lib().tfhe_secret_keygen(ctypes.byref(p), seed, ctypes.byref(h)))
    return SecretKey(h, p)


def tfhe_eval_key_upload(sk: SecretKey, device: int = 0) -> EvalKey:
    h = ctypes.c_void_p()
    _check(lib().tfhe_eval_key_upload(sk.handle, device, ctypes.byref(h)))
    return EvalKey(h, sk.params, device)


def tfhe_keygen_from_seed(params, seed: int, device: int = 0):
    p = make_params(params)
    hs, he = ctypes.c_void_p(), ctypes.c_void_p()
    _check(lib().tfhe_keygen_from_seed(ctypes.byref(p), seed, device, ctypes.byref(hs), ctypes.byref(he)))
    return SecretKey(hs, p), EvalKey(he, p, device)


def tfhe_transform_error_bound(params):
    """(key_parts, worst-case transform error) for a parameter set."""
    p = make_params(params)
    parts = ctypes.c_int32()
    bound = ctypes.c_double()
    _check(lib().tfhe_transform_error_bound(ctypes.byref(p), ctypes.byref(parts), ctypes.byref(bound)))
    return parts.value, bound.value


def tfhe_export_keys(sk: SecretKey) -> dict:
    p = sk.params
    base = (1 << p.ks_basebit) - 1
    s = np.zeros(p.n, np.uint32)
    S = np.zeros(p.N, np.uint32)
    bk = np.zeros(p.n * 2 * p.l * 2 * p.N, np.uint32)
    ksk = np.zeros(p.N * p.ks_t * base * (p.n + 1), np.uint32)
    _check(lib().tfhe_export_keys(sk.handle, _hptr(s), _hptr(S), _hptr(bk), _hptr(ksk)))
    return {"s": s, "S": S, "bk": bk, "ksk": ksk}


# ---------------------------------------------------------- client side

def tfhe_encrypt_torus(sk: SecretKey, seed: int, mu, first_index: int = 0) -> np.ndarray:
    mu = _host_u32(mu).ravel()
    ct = np.zeros((len(mu), sk.params.n + 1), np.uint32)
    _check(lib().tfhe_encrypt_torus(sk.handle, seed, _hptr(mu), first_index, len(mu), _hptr(ct)))
    return ct


def tfhe_decrypt_phase(sk: SecretKey, ct, key_kind: int = 0) -> np.ndarray:
    ct = _host_u32(ct)
    dim = sk.params.n if key_kind == 0 else sk.params.N
    if ct.ndim < 1 or ct.shape[-1] != dim + 1:
        raise ValueError(f"rows of {ct.shape[-1] if ct.ndim else 0} words; key_kind {key_kind} decrypts "
                         f"rows of {dim + 1}")
    count = ct.size // (dim + 1)
    out = np.zeros(count, np.uint32)
    _check(lib().tfhe_decrypt_phase(sk.handle, key_kind, _hptr(ct), count, _hptr(out)))
    return out.reshape(ct.shape[:-1])


def tfhe_lut_testvec(N: int, msg_bits: int, lut) -> np.ndarray:
    lut = _host_u32(lut)
    tv = np.zeros(N, np.uint32)
    _check(lib().tfhe_lut_testvec(N, msg_bits, _hptr(lut), _hptr(tv)))
    return tv


def encode_bits(bits) -> np.ndarray:
    """+1/8 for true, -1/8 for false."""
    b = np.asarray(bits).astype(np.int64)
    return np.where(b != 0, MU, (1 << 32) - MU).astype(np.uint32)


# ---------------------------------------------------------- server side

def to_device(a: np.ndarray, device: int = 0):
    import torch
    a = _host_u32(a)
    return torch.from_numpy(a.view(np.int32)).to(f"cuda:{device}")


def to_host(t) -> np.ndarray:
    return t.detach().cpu().numpy().view(np.uint32)


def tfhe_workspace_bytes(ek: EvalKey, batch: int) -> int:
    v = lib().tfhe_workspace_bytes(ek.handle, batch)
    if v < 0:
        _check(int(v))
    return int(v)


def _on(stream):
    """Allocation context of buffers that a call on `stream` will use: torch's
    caching allocator hands out blocks per stream, and a block last used on
    another stream may still be in use there by queued work, so buffers for
    a caller-given stream are allocated on that stream."""
    import contextlib

    import torch
    return torch.cuda.stream(stream) if stream is not None else contextlib.nullcontext()


def alloc_workspace(ek: EvalKey, batch: int, stream=None):
    import torch
    with _on(stream):
        return torch.empty(max(tfhe_workspace_bytes(ek, batch), 256), dtype=torch.uint8,
                           device=f"cuda:{ek.device}")


def _empty(shape, ek: EvalKey, stream=None):
    import torch
    with _on(stream):
        return torch.empty(shape, dtype=torch.int32, device=f"cuda:{ek.device}")


def tfhe_gate_bootstrap_batch(ek: EvalKey, gate, ca, cb, out=None, workspace=None, stream=None):
    B = ca.shape[0]
    n = ek.params.n
    out = _empty((B, n + 1), ek, stream) if out is None else out
    ws = alloc_workspace(ek, B, stream) if workspace is None else workspace
    g = GATES[gate] if isinstance(gate, str) else int(gate)
    w = B * (n + 1)
    d = ek.device
    _check(lib().tfhe_gate_bootstrap_batch(ek.handle, g, _dbuf(ca, w, "ca", d), _dbuf(cb, w, "cb", d),
                                           _dbuf(out, w, "out", d), B, *_wsbuf(ws, d), _stream(stream, d, ca, cb, out, ws)))
    return out


NOALLOC_SCRATCH_BYTES = 64 << 20  # TFHE_NOALLOC_SCRATCH_BYTES


def tfhe_gate_bootstrap_batch_noalloc(ek: EvalKey, gate, ca, cb, out, stream=None):
    """tfhe_gate_bootstrap_batch with the library's own device workspace (no
    allocation anywhere in the call): out must be given; batches up to
    tfhe_workspace_bytes(ek, B) <= NOALLOC_SCRATCH_BYTES."""
    B = ca.shape[0]
    w, d = B * (ek.params.n + 1), ek.device
    g = GATES[gate] if isinstance(gate, str) else int(gate)
    _check(lib().tfhe_gate_bootstrap_batch_noalloc(ek.handle, g, _dbuf(ca, w, "ca", d), _dbuf(cb, w, "cb", d),
                                                   _dbuf(out, w, "out", d), B, _stream(stream, d, ca, cb, out)))
    return out


def tfhe_lut_bootstrap_batch(ek: EvalKey, x, testvec, out=None, workspace=None, stream=None):
    B = x.shape[0]
    out = _empty((B, ek.params.n + 1), ek, stream) if out is None else out
    ws = alloc_workspace(ek, B, stream) if workspace is None else workspace
    w, d = B * (ek.params.n + 1), ek.device
    _check(lib().tfhe_lut_bootstrap_batch(ek.handle, _dbuf(x, w, "x", d), _dbuf(testvec, ek.params.N, "testvec", d),
                                          _dbuf(out, w, "out", d), B, *_wsbuf(ws, d), _stream(stream, d, x, testvec, out, ws)))
    return out


def tfhe_bootstrap_extract_batch(ek: EvalKey, x, testvec=None, out=None, workspace=None, stream=None):
    B = x.shape[0]
    out = _empty((B, ek.params.N + 1), ek, stream) if out is None else out
    ws = alloc_workspace(ek, B, stream) if workspace is None else workspace
    p, d = ek.params, ek.device
    tv = _dbuf(testvec, p.N, "testvec", d) if testvec is not None else ctypes.c_void_p(0)
    _check(lib().tfhe_bootstrap_extract_batch(ek.handle, _dbuf(x, B * (p.n + 1), "x", d), tv,
                                              _dbuf(out, B * (p.N + 1), "out", d), B, *_wsbuf(ws, d),
                                              _stream(stream, d, x, testvec, out, ws)))
    return out


def tfhe_keyswitch_batch(ek: EvalKey, x, out=None, stream=None):
    B = x.shape[0]
    out = _empty((B, ek.params.n + 1), ek, stream) if out is None else out
    p, d = ek.params, ek.device
    _check(lib().tfhe_keyswitch_batch(ek.handle, _dbuf(x, B * (p.N + 1), "x", d),
                                      _dbuf(out, B * (p.n + 1), "out", d), B, _stream(stream, d, x, out)))
    return out


def glyph_relu_batch(ek: EvalKey, x, bits: int, y=None, gate_begin: int = 0, gate_end=None,
                     workspace=None, stream=None):
    V = x.shape[0]
    n = ek.params.n
    y = _empty((V, bits, n + 1), ek, stream) if y is None else y
    if gate_end is None:
        gate_end = V * (bits - 1)
    ws = alloc_workspace(ek, gate_end - gate_begin, stream) if workspace is None else workspace
    w, d = V * bits * (n + 1), ek.device
    _check(lib().glyph_relu_batch(ek.handle, _dbuf(x, w, "x", d), _dbuf(y, w, "y", d), V, bits, gate_begin,
                                  gate_end, *_wsbuf(ws, d), _stream(stream, d, x, y, ws)))
    return y


def glyph_irelu_batch(ek: EvalKey, u, delta, out=None, gate_begin: int = 0, gate_end=None,
                      workspace=None, stream=None):
    """Backward iReLU: u [V][u_bits][n+1] (its sign words are read), delta and
    out [V][bits][n+1]; gates [gate_begin, gate_end) of the V*bits."""
    V, u_bits = u.shape[0], u.shape[1]
    bits = delta.shape[1]
    out = _empty(tuple(delta.shape), ek, stream) if out is None else out
    if gate_end is None:
        gate_end = V * bits
    ws = alloc_workspace(ek, gate_end - gate_begin, stream) if workspace is None else workspace
    row, d = ek.params.n + 1, ek.device
    _check(lib().glyph_irelu_batch(ek.handle, _dbuf(u, V * u_bits * row, "u", d), u_bits,
                                   _dbuf(delta, V * bits * row, "delta", d), _dbuf(out, V * bits * row, "out", d),
                                   V, bits, gate_begin, gate_end, *_wsbuf(ws, d), _stream(stream, d, u, delta, out, ws)))
    return out


def tfhe_mux_batch(ek: EvalKey, c, a, b, out=None, workspace=None, stream=None):
    """out[e] encrypts c[e] ? a[e] : b[e]; all [B][n+1] device."""
    B = c.shape[0]
    out = _empty((B, ek.params.n + 1), ek, stream) if out is None else out
    ws = alloc_workspace(ek, 2 * B, stream) if workspace is None else workspace
    w, d = B * (ek.params.n + 1), ek.device
    _check(lib().tfhe_mux_batch(ek.handle, _dbuf(c, w, "c", d), _dbuf(a, w, "a", d), _dbuf(b, w, "b", d),
                                _dbuf(out, w, "out", d), B, *_wsbuf(ws, d), _stream(stream, d, c, a, b, out, ws)))
    return out


def glyph_mux_lut_workspace_bytes(ek: EvalKey, V: int, msg_bits: int, out_bits: int) -> int:
    r = lib().glyph_mux_lut_workspace_bytes(ek.handle, V, msg_bits, out_bits)
    if r < 0:
        _check(int(r))
    return int(r)


def alloc_mux_lut_workspace(ek: EvalKey, V: int, msg_bits: int, out_bits: int, stream=None):
    import torch
    with _on(stream):
        return torch.empty(max(glyph_mux_lut_workspace_bytes(ek, V, msg_bits, out_bits), 1), dtype=torch.uint8,
                           device=f"cuda:{ek.device}")


def glyph_mux_lut_batch(ek: EvalKey, x, table, out_bits: int, out=None, workspace=None, stream=None):
    """Table lookup by a multiplexer tree: x [V][msg_bits][n+1] encrypted bits
    (LSB first) select entries of the public table (2^msg_bits values below
    2^out_bits); returns out [V][out_bits][n+1]."""
    V, msg_bits = x.shape[0], x.shape[1]
    t = _host_u32(table)
    if t.size != 1 << msg_bits:
        raise ValueError(f"table needs {1 << msg_bits} entries")
    out = _empty((V, out_bits, ek.params.n + 1), ek, stream) if out is None else out
    ws = alloc_mux_lut_workspace(ek, V, msg_bits, out_bits, stream) if workspace is None else workspace
    row, d = ek.params.n + 1, ek.device
    _check(lib().glyph_mux_lut_batch(ek.handle, _dbuf(x, V * msg_bits * row, "x", d), msg_bits, _hptr(t), out_bits,
                                     _dbuf(out, V * out_bits * row, "out", d), V, *_wsbuf(ws, d),
                                     _stream(stream, d, x, out, ws)))
    return out


def tfhe_packing_key_upload(sk: SecretKey, ek: EvalKey):
    _check(lib().tfhe_packing_key_upload(sk.handle, ek.handle))


def tfhe_export_packing_key(sk: SecretKey) -> np.ndarray:
    p = sk.params
    pks = np.zeros(p.n * p.ks_t * ((1 << p.ks_basebit) - 1) * 2 * p.N, np.uint32)
    _check(lib().tfhe_export_packing_key(sk.handle, _hptr(pks)))
    return pks


def tfhe_pack_keyswitch_batch(ek: EvalKey, lwe, out=None, stream=None):
    """lwe [B][Z][n+1] -> TRLWE samples [B][2][N] (phase sum_z phase_z X^z)."""
    B, Z = lwe.shape[0], lwe.shape[1]
    out = _empty((B, 2, ek.params.N), ek, stream) if out is None else out
    p, d = ek.params, ek.device
    _check(lib().tfhe_pack_keyswitch_batch(ek.handle, _dbuf(lwe, B * Z * (p.n + 1), "lwe", d), Z,
                                           _dbuf(out, B * 2 * p.N, "out", d), B, _stream(stream, d, lwe, out)))
    return out


def tfhe_sample_extract_batch(trlwe, K: int, out=None, stream=None):
    """TRLWE samples [B][2][N] -> LWE samples of coefficients 0..K-1, [B][K][N+1]."""
    import torch
    B, N = trlwe.shape[0], trlwe.shape[2]
    if out is None:
        with _on(stream):
            out = torch.empty((B, K, N + 1), dtype=torch.int32, device=trlwe.device)
    d = trlwe.device.index
    _check(lib().tfhe_sample_extract_batch(N, _dbuf(trlwe, B * 2 * N, "trlwe", d), B, K,
                                           _dbuf(out, B * K * (N + 1), "out", d), _stream(stream, d, trlwe, out)))
    return out


def tfhe_torus_testvec(N: int, msg_bits: int, values) -> np.ndarray:
    v = _host_u32(values)
    tv = np.zeros(N, np.uint32)
    _check(lib().tfhe_torus_testvec(N, msg_bits, _hptr(v), _hptr(tv)))
    return tv


def tfhe_not_batch(x, out=None, stream=None):
    import torch
    dim = x.shape[-1] - 1
    count = x.numel() // (dim + 1)
    if out is None:
        with _on(stream):
            out = torch.empty_like(x)
    w = count * (dim + 1)
    _check(lib().tfhe_not_batch(dim, _dbuf(x, w, "x"), _dbuf(out, w, "out", x.device.index), count,
                                _stream(stream, x.device.index, x, out)))
    return out


def tfhe_negacyclic_mul_batch(ek: EvalKey, d, b, out=None, stream=None):
    import torch
    B = d.shape[0]
    if out is None:
        with _on(stream):
            out = torch.empty_like(b)
    w, dev = B * ek.params.N, ek.device
    _check(lib().tfhe_negacyclic_mul_batch(ek.handle, _dbuf(d, w, "d", dev), _dbuf(b, w, "b", dev),
                                           _dbuf(out, w, "out", dev), B, _stream(stream, dev, d, b, out)))
    return out


# ------------------------------------------------------------ stage checks

def tfhe_debug_mod_switch_batch(ek: EvalKey, x, gate=None, cb=None, out=None, stream=None):
    """Modulus switch of x [B][n+1] (gate None), or of the pre-combination of
    (x, cb) for a gate, to Z_2N: int16 tensor [B][n+1] holding the uint16 words."""
    import torch
    B, n, d = x.shape[0], ek.params.n, ek.device
    g = -1 if gate is None else (GATES[gate] if isinstance(gate, str) else int(gate))
    if g >= 0 and cb is None:
        raise ValueError("a gate needs its second operand cb")
    if out is None:
        with _on(stream):
            out = torch.empty((B, n + 1), dtype=torch.int16, device=f"cuda:{d}")
    if out.element_size() != 2 or out.numel() < B * (n + 1):
        raise ValueError("out: expected at least B * (n + 1) 16-bit words")
    w = B * (n + 1)
    pcb = _dbuf(cb, w, "cb", d) if g >= 0 else ctypes.c_void_p(0)
    _check(lib().tfhe_debug_mod_switch_batch(ek.handle, g, _dbuf(x, w, "x", d), pcb, _dptr(out), B,
                                             _stream(stream, d, x, cb, out)))
    return out


def tfhe_debug_cmux_batch(ek: EvalKey, bk_row, abar, acc_in, out=None, workspace=None, stream=None):
    """One CMux step with a caller-given coefficient-domain key row bk_row
    ([2l][2][N] host words) on the accumulators acc_in [B][2][N] with rotation
    amounts abar [B] (device): returns acc_out [B][2][N]."""
    import torch
    p, d = ek.params, ek.device
    B = acc_in.shape[0]
    row = _host_u32(bk_row).ravel()
    if row.size != 2 * p.l * 2 * p.N:
        raise ValueError(f"bk_row: {row.size} words, a key row has {2 * p.l * 2 * p.N}")
    with _on(stream):
        if out is None:
            out = torch.empty((B, 2, p.N), dtype=torch.int32, device=f"cuda:{d}")
        if workspace is None:
            nb = lib().tfhe_debug_cmux_workspace_bytes(ek.handle, B)
            if nb < 0:
                _check(int(nb))
            workspace = torch.empty(max(int(nb), 256), dtype=torch.uint8, device=f"cuda:{d}")
    w = B * 2 * p.N
    _check(lib().tfhe_debug_cmux_batch(ek.handle, _hptr(row), _dbuf(abar, B, "abar", d), _dbuf(acc_in, w, "acc_in", d),
                                       _dbuf(out, w, "out", d), B, *_wsbuf(workspace, d),
                                       _stream(stream, d, abar, acc_in, out, workspace)))
    return out


# ---------------------------------------------------------------- profiling

STAGES = ("prep", "blind_rotate", "keyswitch")


def tfhe_stage_timing(enable: bool):
    _check(lib().tfhe_stage_timing(1 if enable else 0))


def tfhe_stage_times() -> dict:
    """{stage: (total_ms, launches)} of the launches recorded since the last read."""
    ms = (ctypes.c_double * 3)()
    n = (ctypes.c_int64 * 3)()
    _check(lib().tfhe_stage_times(ms, n))
    return {STAGES[k]: (ms[k], n[k]) for k in range(3)}


PROBE_KINDS = ("v_fma_f64", "v_add_u32", "v_cvt_f64_i32", "v_bfe_i32", "v_mul_lo_u32")


def tfhe_probe_valu_rate(kind, waves: int, iters: int, out=None, stream=None):
    """Launch the VALU issue-rate probe for one instruction kind (a name of
    PROBE_KINDS or its index) on the current device; returns the [waves * 64]
    output tensor.  The caller times the launch on `stream`."""
    import torch
    k = PROBE_KINDS.index(kind) if isinstance(kind, str) else int(kind)
    dev = torch.cuda.current_device()
    if out is None:
        with _on(stream):
            out = torch.empty(waves * 64, dtype=torch.int32, device=f"cuda:{dev}")
    _check(lib().tfhe_probe_valu_rate(k, waves, iters, _dbuf(out, waves * 64, "out", dev), _stream(stream, dev, out)))
    return out

