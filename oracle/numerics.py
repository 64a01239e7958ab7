"""bf16 emulation for the oracle (rounding points of the bf16 model variant).

The paper fixes no precision.  The bf16 variant stores weights and the
cached K/V in bf16; this module rounds float64 or float32 values to the
nearest bf16 value (ties to even), returned in the input dtype, using integer
operations on the IEEE bit patterns.
"""
import numpy as np


def round_bf16(x):
    """Nearest bf16 value of each element (ties to even), same dtype as x.

    float64: keep 8 significant bits of the 53 (drop 45 mantissa bits).
    float32: keep 8 of the 24 (drop 16 mantissa bits).  Finite inputs only.
    """
    x = np.asarray(x)
    if x.dtype == np.float64:
        b = x.view(np.uint64)
        drop = np.uint64(45)
        half = np.uint64((1 << 44) - 1)
        one = np.uint64(1)
        mask = ~np.uint64((1 << 45) - 1)
        lsb = (b >> drop) & one
        with np.errstate(over="ignore"):
            r = (b + half + lsb) & mask
        return r.view(np.float64)
    if x.dtype == np.float32:
        b = x.view(np.uint32)
        lsb = (b >> np.uint32(16)) & np.uint32(1)
        r = (b + np.uint32(0x7FFF) + lsb) & np.uint32(0xFFFF0000)
        return r.view(np.float32)
    raise TypeError(f"round_bf16: unsupported dtype {x.dtype}")


def bf16_bits_to_float(bits, dtype=np.float64):
    """Decode uint16 bf16 bit patterns to floats (exact)."""
    bits = np.asarray(bits, dtype=np.uint16)
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(dtype)
