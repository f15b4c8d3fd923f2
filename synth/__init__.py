"""Seeded synthetic inputs shared by the oracle tests, the GPU parity tests and the benchmark.

This package draws random numbers and rounds them to the storage formats the
calibration data uses (bf16). It contains none of the quantization method's
arithmetic: no Hessian, no quantizer, no compensation, no gradient.
"""
from .gen import (  # noqa: F401
    CONFIGS,
    DecoderBlockInputs,
    LayerInputs,
    MLPBlockInputs,
    bf16_bits,
    bf16_round,
    bf16_from_bits,
    make_decoder_block,
    make_group_weights,
    make_mlp_block,
    make_module,
    make_output_grads,
    module_names,
)
