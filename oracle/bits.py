"""Exact widening of 16-bit floating-point bit patterns to float64 (test infrastructure only).

The GPU path reads bf16 (query/document token embeddings) and fp16 (pooled chunk embeddings).
The oracle works on the exact real numbers those bit patterns denote.  Both conversions below are
exact: every bf16 value is an fp32 value (bf16 is the upper half of an fp32 word), and every fp16
value, subnormals included, is representable in float64.
"""

import numpy as np


def decode_bf16(bits):
    """bf16 bit patterns (uint16 / int16 array) -> float64 array of the same shape, exactly."""
    b = np.asarray(bits).astype(np.uint16, copy=False)
    wide = b.astype(np.uint32) << np.uint32(16)
    return wide.view(np.float32).astype(np.float64)


def decode_fp16(bits):
    """IEEE binary16 bit patterns (uint16 / int16 array) -> float64 array, exactly."""
    b = np.asarray(bits).astype(np.uint16, copy=False)
    return b.view(np.float16).astype(np.float64)
