"""Counter-based random bits that come out bit-identical on CPU and GPU.

The mixing function is Chris Wellons' "lowbias32" 32-bit integer hash
(published in "Prospecting for Hash Functions", 2018):

    x ^= x >> 16;  x *= 0x7feb352d;  x ^= x >> 15;  x *= 0x846ca68b;  x ^= x >> 16

It is evaluated with int64 torch tensors holding values in [0, 2**32).  Each
32-bit product is formed from 16-bit halves so that no int64 product
overflows; the result is therefore the same on every device torch supports.
"""

import torch

_M32 = 0xFFFFFFFF
_C1 = 0x7FEB352D
_C2 = 0x846CA68B


def _mul32(x: torch.Tensor, c: int) -> torch.Tensor:
    """(x * c) mod 2**32 for int64 x in [0, 2**32) without int64 overflow."""
    lo, hi = c & 0xFFFF, c >> 16
    return (x * lo + (((x * hi) & 0xFFFF) << 16)) & _M32


def lowbias32(x: torch.Tensor) -> torch.Tensor:
    x = x ^ (x >> 16)
    x = _mul32(x, _C1)
    x = x ^ (x >> 15)
    x = _mul32(x, _C2)
    x = x ^ (x >> 16)
    return x


def _lowbias32_int(x: int) -> int:
    x &= _M32
    x ^= x >> 16
    x = (x * _C1) & _M32
    x ^= x >> 15
    x = (x * _C2) & _M32
    x ^= x >> 16
    return x


def tensor_key(seed: int, tag: int) -> tuple:
    """Two 32-bit stream keys for one tensor, from a model seed and a tensor tag."""
    k1 = _lowbias32_int(_lowbias32_int(seed) ^ _lowbias32_int(tag ^ 0x9E3779B9))
    k2 = _lowbias32_int(k1 ^ 0x85EBCA6B ^ _lowbias32_int(tag))
    return k1, k2


def hash_uniform16(counter: torch.Tensor, key: tuple) -> torch.Tensor:
    """Two independent 16-bit uniforms per counter, packed as one 32-bit value."""
    k1, k2 = key
    return lowbias32(lowbias32(counter ^ k1) ^ k2)
