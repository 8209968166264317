"""Seeded synthetic inputs shared by the oracle and the GPU path.

This module holds model shapes, the seeded weight generator and the seeded
prompt generator. It performs none of the method's arithmetic: it only draws
random numbers and stores them in the model's storage formats (IEEE fp32 or
bf16 bit patterns). Both the oracle and the GPU library consume exactly these
arrays; neither side's arithmetic lives here.
"""
from .configs import CONFIGS, ModelConfig, get_config
from .weights import generate_weights, tensor_names, prompts, bf16_bits_from_f32

__all__ = ["CONFIGS", "ModelConfig", "get_config", "generate_weights",
           "tensor_names", "prompts", "bf16_bits_from_f32"]
