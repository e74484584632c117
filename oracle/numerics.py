"""bfloat16 decode/encode for the oracle (plain bit manipulation).

bf16 is the top 16 bits of an IEEE-754 binary32. Decoding is exact; encoding
uses round-to-nearest-even, the rounding the kernel's output uses.
Pinned in tests/test_oracle_core.py against torch's own bf16 casts.
"""
import numpy as np


def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32).astype(np.float64)


def f64_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    f = np.asarray(x, dtype=np.float64).astype(np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    nan = np.isnan(f)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16).astype(np.uint16)
    r[nan] = 0x7FC0
    return r


def torch_bf16_to_f64(t) -> np.ndarray:
    """Decode a torch bfloat16 tensor (any device) to a numpy fp64 array."""
    import torch
    bits = t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
    return bf16_bits_to_f64(bits)
