"""MI355X-native TFHE activation path of Glyph (arXiv 1911.07101).

The work is done by libglyph_tfhe.so (HIP kernels for gfx950 behind the C ABI
of include/glyph_tfhe.h); ``tfhe`` is its Python binding and ``workloads``
holds the parameter sets and seeded plaintext inputs.
"""
from . import tfhe, workloads  # noqa: F401
from .tfhe import (  # noqa: F401
    glyph_irelu_batch, glyph_mux_lut_batch, glyph_relu_batch, tfhe_bootstrap_extract_batch,
    tfhe_decrypt_phase, tfhe_encrypt_torus, tfhe_eval_key_upload, tfhe_export_keys,
    tfhe_gate_bootstrap_batch, tfhe_keygen_from_seed, tfhe_keyswitch_batch, tfhe_lut_bootstrap_batch,
    tfhe_lut_testvec, tfhe_mux_batch, tfhe_negacyclic_mul_batch, tfhe_not_batch,
    tfhe_pack_keyswitch_batch, tfhe_packing_key_upload, tfhe_sample_extract_batch, tfhe_secret_keygen,
    tfhe_torus_testvec, tfhe_workspace_bytes,
)
