"""CPU checks of the GPU library: it loads, exports every symbol its header
declares, and its host-side (client) steps -- key generation, encryption,
test-polynomial construction, argument validation -- agree with the oracle,
which shares no code with it."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
from paper_1911_07101_amd import tfhe, workloads as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "glyph_tfhe.h")
TOY = wl.CONFIGS["toy"]["params"]


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"^[A-Za-z_][\w\s\*]*?\b((?:tfhe|glyph)_\w+)\s*\(", text, flags=re.M)
    return sorted(set(names))


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(tfhe.LIB_PATH)
    names = declared_functions()
    assert len(names) >= 20
    for name in names:
        assert hasattr(lib, name), name
    # and the binding covers all of them
    assert set(names) <= set(tfhe._SIGNATURES)


@pytest.mark.parametrize("cfg", ["toy", "tfhe128_nand"])
def test_secret_keygen_matches_oracle(cfg):
    p = wl.CONFIGS[cfg]["params"]
    seed = wl.CONFIGS[cfg]["key_seed"]
    sk = tfhe.tfhe_secret_keygen(p, seed)
    mine = tfhe.tfhe_export_keys(sk)
    ref = oracle.Keys(p, seed)
    assert np.array_equal(mine["s"], ref.s)
    assert np.array_equal(mine["S"], ref.S)
    assert np.array_equal(mine["bk"], ref.bk)
    assert np.array_equal(mine["ksk"], ref.ksk)


def test_secret_keygen_matches_oracle_lut_params_small():
    # the N = 2048, l = 2, Bg = 2^10 gadget and the 2^-45 noise floor, smaller n
    p = dict(wl.CONFIGS["lut3_n2048"]["params"], n=24)
    sk = tfhe.tfhe_secret_keygen(p, 99)
    mine = tfhe.tfhe_export_keys(sk)
    ref = oracle.Keys(p, 99)
    for k in ("s", "S", "bk", "ksk"):
        assert np.array_equal(mine[k], getattr(ref, k)), k


def test_encryption_and_phase_match_oracle():
    sk = tfhe.tfhe_secret_keygen(TOY, 5)
    ref = oracle.Keys(TOY, 5)
    mu = np.arange(300, dtype=np.uint32) * np.uint32(14318181)
    ct = tfhe.tfhe_encrypt_torus(sk, 77, mu, first_index=1000)
    assert np.array_equal(ct, oracle.encrypt(TOY["n"], ref.s, 77, TOY["alpha_lwe"], mu, 1000))
    assert np.array_equal(tfhe.tfhe_decrypt_phase(sk, ct), oracle.phase(ref.s, ct))
    ext = np.random.default_rng(1).integers(0, 2**32, (7, TOY["N"] + 1), dtype=np.uint64).astype(np.uint32)
    assert np.array_equal(tfhe.tfhe_decrypt_phase(sk, ext, key_kind=1), oracle.phase(ref.S, ext))


def test_lut_testvec_matches_oracle():
    rng = np.random.default_rng(4)
    for N, bits in [(256, 3), (2048, 3), (1024, 2), (512, 4)]:
        lut = rng.integers(0, 1 << bits, 1 << bits).astype(np.uint32)
        assert np.array_equal(tfhe.tfhe_lut_testvec(N, bits, lut), oracle.lut_testvec(N, bits, lut))
    with pytest.raises(tfhe.TfheError):
        tfhe.tfhe_lut_testvec(256, 3, np.array([8] * 8, np.uint32))


@pytest.mark.parametrize("change,rc", [
    (dict(N=768), tfhe.TFHE_EUNSUPPORTED),
    (dict(N=4096), tfhe.TFHE_EUNSUPPORTED),
    (dict(l=5, bg_bit=7), tfhe.TFHE_EUNSUPPORTED),         # l * bg_bit > 32
    (dict(N=2048, l=1, bg_bit=24), tfhe.TFHE_EUNSUPPORTED),  # transform error bound above 1/8
    (dict(ks_t=17, ks_basebit=2), tfhe.TFHE_EUNSUPPORTED),
    (dict(ks_basebit=9, ks_t=2), tfhe.TFHE_EUNSUPPORTED),
    (dict(ks_t=16, ks_basebit=3), tfhe.TFHE_EUNSUPPORTED),    # 128 key rows per coefficient
    (dict(n=0), tfhe.TFHE_EUNSUPPORTED),
    (dict(alpha_bk=-1.0), tfhe.TFHE_EINVAL),
])
def test_parameter_validation(change, rc):
    with pytest.raises(tfhe.TfheError) as ei:
        tfhe.tfhe_secret_keygen(dict(TOY, **change), 1)
    assert ei.value.rc == rc


def test_upload_without_gfx950_device_fails_cleanly():
    torch = pytest.importorskip("torch")
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    sk = tfhe.tfhe_secret_keygen(TOY, 1)
    with pytest.raises(tfhe.TfheError) as ei:
        tfhe.tfhe_eval_key_upload(sk, 0)
    assert ei.value.rc == tfhe.TFHE_EDEVICE


def test_transform_error_bound_covers_every_workload():
    """Every parameter set used here keeps the transform's worst-case error
    below 1/8, and the bound grows with the digit base and ring degree."""
    for name, cfg in wl.CONFIGS.items():
        parts, bound = tfhe.tfhe_transform_error_bound(cfg["params"])
        assert parts in (2, 3) and bound < 0.125, name
    _, b7 = tfhe.tfhe_transform_error_bound(dict(TOY, N=1024, bg_bit=7))
    _, b8 = tfhe.tfhe_transform_error_bound(dict(TOY, N=1024, bg_bit=8))
    _, b7n = tfhe.tfhe_transform_error_bound(dict(TOY, N=512, bg_bit=7))
    assert b7n < b7 < b8
    # 16-bit halves cover every workload; 16-bit digits at N = 2048 need the
    # 3-part split, and 24-bit digits are beyond any split
    assert all(tfhe.tfhe_transform_error_bound(c["params"])[0] == 2 for c in wl.CONFIGS.values())
    assert tfhe.tfhe_transform_error_bound(dict(TOY, N=2048, l=1, bg_bit=16))[0] == 3
    with pytest.raises(tfhe.TfheError) as ei:
        tfhe.tfhe_transform_error_bound(dict(TOY, N=2048, l=1, bg_bit=24))
    assert ei.value.rc == tfhe.TFHE_EUNSUPPORTED


def test_packing_key_matches_oracle():
    """The library's packing key (host keygen, rotated sums for A*S) is
    word-for-word the oracle's (schoolbook products)."""
    p = dict(TOY, n=12, N=256)
    sk = tfhe.tfhe_secret_keygen(p, 77)
    ok = oracle.Keys(p, 77)
    assert np.array_equal(tfhe.tfhe_export_packing_key(sk), ok.packing_key())


def test_torus_testvec_matches_oracle():
    rng = np.random.default_rng(12)
    for N, bits in [(256, 3), (1024, 3), (2048, 5)]:
        vals = rng.integers(0, 1 << 32, 1 << bits, dtype=np.uint64).astype(np.uint32)
        assert np.array_equal(tfhe.tfhe_torus_testvec(N, bits, vals), oracle.torus_testvec(N, bits, vals))


def test_binding_checks_buffers_before_any_call():
    """The C ABI takes plain pointers, so the binding checks element width,
    size and placement of every device buffer before calling it."""
    import torch
    with pytest.raises(ValueError, match="32-bit"):
        tfhe._dbuf(torch.zeros(8, dtype=torch.int64), 8, "x")
    with pytest.raises(ValueError, match="needs 8"):
        tfhe._dbuf(torch.zeros(7, dtype=torch.int32), 8, "x")
    with pytest.raises(ValueError, match="device tensor"):
        tfhe._dbuf(torch.zeros(8, dtype=torch.int32), 8, "x")


MAX_ITEMS = (1 << 32) - 256  # work-items of one launch dimension the library allows


def test_counts_too_large_for_one_launch_are_refused():
    """The calls that take no eval key refuse, before any HIP call, a count
    whose one-dimensional launch would exceed 2^32 - 256 work-items.  Their
    data pointers are NULL, so a call that passed the count check fails on
    those instead, with another message: nothing here can reach a launch."""
    L = tfhe.lib()

    def refused(rc):
        return rc == tfhe.TFHE_EINVAL and "exceed" in L.tfhe_last_error().decode()

    def null_buffer(rc):
        return rc == tfhe.TFHE_EINVAL and "NULL" in L.tfhe_last_error().decode()

    # sample extraction of all 256 coefficients at N = 256: 256 * 257 words per ciphertext
    most = MAX_ITEMS // (256 * 257)
    assert most == 65280
    assert null_buffer(L.tfhe_sample_extract_batch(256, None, most, 256, None, None))
    assert refused(L.tfhe_sample_extract_batch(256, None, most + 1, 256, None, None))
    # NOT of LWE samples of dimension 64: 65 words each
    most = MAX_ITEMS // 65
    assert null_buffer(L.tfhe_not_batch(64, None, None, most, None))
    assert refused(L.tfhe_not_batch(64, None, None, most + 1, None))
    assert refused(L.tfhe_not_batch((1 << 31) - 1, None, None, 3, None))  # no overflow in dim + 1


def test_decrypt_checks_the_row_width_of_its_key():
    """tfhe_decrypt_phase strides by the dimension of the key it decrypts
    with (n for key_kind 0, N for 1): rows of the other width are refused
    before the C call, which would otherwise read past the buffer."""
    sk = tfhe.tfhe_secret_keygen(TOY, 3)
    ct = np.zeros((4, TOY["n"] + 1), np.uint32)
    assert tfhe.tfhe_decrypt_phase(sk, ct, 0).shape == (4,)
    with pytest.raises(ValueError, match="rows of"):
        tfhe.tfhe_decrypt_phase(sk, ct, 1)
    ext = np.zeros((2, 3, TOY["N"] + 1), np.uint32)
    assert tfhe.tfhe_decrypt_phase(sk, ext, 1).shape == (2, 3)
    with pytest.raises(ValueError, match="rows of"):
        tfhe.tfhe_decrypt_phase(sk, ext, 0)


def test_issue_rate_probe_refuses_bad_arguments():
    """tfhe_probe_valu_rate checks its arguments before any HIP call (the
    output pointer is NULL or the arguments are out of range, so nothing
    here can reach a launch)."""
    L = tfhe.lib()

    def einval(rc, what):
        return rc == tfhe.TFHE_EINVAL and what in L.tfhe_last_error().decode()

    assert einval(L.tfhe_probe_valu_rate(5, 4, 1, None, None), "kind")
    assert einval(L.tfhe_probe_valu_rate(-1, 4, 1, None, None), "kind")
    assert einval(L.tfhe_probe_valu_rate(0, 6, 1, None, None), "waves")
    assert einval(L.tfhe_probe_valu_rate(0, 0, 1, None, None), "waves")
    assert einval(L.tfhe_probe_valu_rate(0, (1 << 20) + 4, 1, None, None), "waves")
    assert einval(L.tfhe_probe_valu_rate(0, 4, 0, None, None), "iters")
    assert einval(L.tfhe_probe_valu_rate(0, 4, (1 << 24) + 1, None, None), "iters")
    assert einval(L.tfhe_probe_valu_rate(0, 4, 1, None, None), "NULL")
