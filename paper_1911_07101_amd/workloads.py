"""Parameter sets and seeded synthetic plaintext inputs of the TFHE activation path.

This module holds data only -- parameter tables, seeds and plaintext generators
(random bits, 8-bit values, 3-bit messages and tables).  It performs none of the
method's arithmetic: encoding onto the torus, encryption and everything after
it belong to the GPU library on one side and to the CPU oracle on the other.
Both take their plaintext inputs from here.

The inputs stand in for the paper's encrypted activations (MNIST and
Skin-Cancer-MNIST training, Section 4 "Experimental Methodology"), whose
datasets are not used: uniform random bits for gates, uniform 8-bit
two's-complement values for the ReLU layers (the paper quantises activations to
8 bits), uniform 3-bit messages and a random 8-entry table for the table-lookup
bootstrap (the paper's 3-bit softmax table, Section 3.1).
"""
from __future__ import annotations

import numpy as np

_TFHE_1024 = dict(n=630, N=1024, l=3, bg_bit=7, ks_t=8, ks_basebit=2,
                  alpha_lwe=2.0 ** -15, alpha_bk=2.0 ** -25, alpha_ks=2.0 ** -15)

CONFIGS = {
    # insecure toy parameters for plumbing and fast parity
    "toy": dict(params=dict(n=64, N=256, l=3, bg_bit=7, ks_t=8, ks_basebit=2,
                            alpha_lwe=2.0 ** -15, alpha_bk=2.0 ** -25, alpha_ks=2.0 ** -15),
                kind="gate", gate="NAND", batch=16, key_seed=0x19110710, input_seed=0x5EED0001),
    # 128-bit TFHE parameters, batched NAND gate bootstrapping
    "tfhe128_nand": dict(params=_TFHE_1024, kind="gate", gate="NAND", batch=4096,
                         key_seed=0x19110711, input_seed=0x5EED0002, sample=64),
    # MLP ReLU layer: 60-sample mini-batch x 128 hidden neurons of 8-bit values
    "mlp_relu": dict(params=_TFHE_1024, kind="relu", values=60 * 128, bits=8,
                     key_seed=0x19110712, input_seed=0x5EED0003, sample=64),
    # conv ReLU layer: 60 samples x 6 channels x 24 x 24 of 8-bit values,
    # streamed through in calls of 16,384 gates
    "conv_relu": dict(params=_TFHE_1024, kind="relu", values=60 * 6 * 24 * 24, bits=8,
                      gates_per_call=16384, key_seed=0x19110713, input_seed=0x5EED0004,
                      sample=64),
    # backward iReLU of the MLP layer: 8-bit errors gated by the signs of the
    # forward 8-bit pre-activations
    "mlp_irelu": dict(params=_TFHE_1024, kind="irelu", values=60 * 128, bits=8,
                      key_seed=0x19110715, input_seed=0x5EED0006, sample=64),
    # the paper's 3-bit softmax exponentiation unit as a multiplexer tree on
    # bit-wise encrypted inputs (128-bit parameters), over the same messages
    # and table as the LUT bootstrap below
    "softmax_mux3": dict(params=_TFHE_1024, kind="mux_lut", values=8192, msg_bits=3, out_bits=3,
                         key_seed=0x19110716, input_seed=0x5EED0005, sample=8),
    # programmable (table-lookup) bootstrap on 3-bit messages, N = 2048
    "lut3_n2048": dict(params=dict(n=750, N=2048, l=2, bg_bit=10, ks_t=8, ks_basebit=2,
                                   alpha_lwe=2.0 ** -17, alpha_bk=2.0 ** -45,
                                   alpha_ks=2.0 ** -17),
                       kind="lut", msg_bits=3, batch=8192, key_seed=0x19110714,
                       input_seed=0x5EED0005, sample=64),
}


def _rng(seed: int, stream: int) -> np.random.Generator:
    return np.random.Generator(np.random.Philox(key=[seed & 0xFFFFFFFFFFFFFFFF, stream]))


def random_bits(seed: int, count: int, stream: int = 0) -> np.ndarray:
    """count uniform bits (uint8 0/1)."""
    return _rng(seed, stream).integers(0, 2, size=count, dtype=np.uint8)


def gate_inputs(seed: int, batch: int):
    """Two independent uniform bit vectors for a batch of two-input gates."""
    return random_bits(seed, batch, 1), random_bits(seed, batch, 2)


def int8_values(seed: int, count: int, stream: int = 3) -> np.ndarray:
    """count values uniform in [-128, 127] (stream 3: activations; another
    stream gives an independent set, e.g. 7 for backward errors)."""
    return _rng(seed, stream).integers(-128, 128, size=count, dtype=np.int64).astype(np.int8)


def to_bits(values: np.ndarray, bits: int) -> np.ndarray:
    """Two's-complement bit planes, LSB first: shape [V][bits] of 0/1."""
    v = np.asarray(values, dtype=np.int64) & ((1 << bits) - 1)
    return ((v[:, None] >> np.arange(bits)[None, :]) & 1).astype(np.uint8)


def from_bits(b: np.ndarray) -> np.ndarray:
    """Inverse of to_bits (signed)."""
    b = np.asarray(b, dtype=np.int64)
    bits = b.shape[-1]
    u = (b << np.arange(bits)).sum(axis=-1)
    return np.where(u >= (1 << (bits - 1)), u - (1 << bits), u)


def messages(seed: int, count: int, msg_bits: int) -> np.ndarray:
    """count messages uniform in [0, 2^msg_bits)."""
    return _rng(seed, 4).integers(0, 1 << msg_bits, size=count, dtype=np.uint32)


def lut(seed: int, msg_bits: int) -> np.ndarray:
    """A random table of 2^msg_bits entries, each a msg_bits-bit value."""
    return _rng(seed, 5).integers(0, 1 << msg_bits, size=1 << msg_bits, dtype=np.uint32)


def sample_indices(seed: int, total: int, count: int) -> np.ndarray:
    """count distinct sorted indices in [0, total) (always includes 0 and total-1)."""
    if count >= total:
        return np.arange(total, dtype=np.int64)
    idx = _rng(seed, 6).choice(total, size=count - 2, replace=False)
    return np.unique(np.concatenate([[0, total - 1], idx])).astype(np.int64)
