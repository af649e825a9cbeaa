"""bfloat16 storage mirroring for the oracle (test infrastructure only).

bfloat16 keeps the top 16 bits of an IEEE-754 binary32 value (1 sign, 8
exponent, 7 fraction bits).  Rounding to it is round-to-nearest, ties to even
on the discarded low 16 bits.  Pinned by tests against torch's own
``.to(torch.bfloat16)`` conversion (library special case) and against
hand-checkable values (1 + 2^-8 is a tie that rounds to 1; 1 + 3*2^-8 rounds
up to 1 + 2^-6 ... see tests).
"""
import numpy as np


def bf16_bits_to_f32(bits):
    """uint16 bf16 bit patterns -> float32 values (exact)."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32)


def round_bf16(x):
    """Round to the nearest bf16 value (ties to even); returns float64.

    float64 input is first rounded to float32 (the GPU path rounds fp32
    values), then the low 16 bits of the float32 pattern are rounded off.
    """
    f = np.asarray(x, dtype=np.float64).astype(np.float32)
    b = np.ascontiguousarray(f).view(np.uint32).astype(np.uint64)
    lsb = (b >> np.uint64(16)) & np.uint64(1)
    b = (b + np.uint64(0x7FFF) + lsb) & np.uint64(0xFFFF0000)
    return b.astype(np.uint32).view(np.float32).astype(np.float64).reshape(f.shape)
