"""Exact widening of bf16 bit patterns (oracle; test infrastructure only).

A bf16 value is the upper 16 bits of the float32 with the same sign, exponent and leading
mantissa bits, so widening is a 16-bit left shift of the pattern; every bf16 value is exactly
representable in float32 and float64."""
import numpy as np


def bf16_bits_to_f32(bits) -> np.ndarray:
    b = np.asarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def bf16_bits_to_f64(bits) -> np.ndarray:
    return bf16_bits_to_f32(bits).astype(np.float64)
