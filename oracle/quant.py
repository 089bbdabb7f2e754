"""Group-wise 4-bit weights: the INT4 weight-only target.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper's phone targets are 4-bit models quantised with AutoGPTQ (§4.1,
"Models and datasets"; FP16 to INT4 in §2.2).  It fixes no format beyond
that, so this build takes GPTQ's symmetric group-wise form: a matrix W[out][in]
is stored as 4-bit codes q[out][in] in [0, 16) and one scale per output row
and group of G consecutive inputs, s[out][in / G]; the weight an entry stands
for is

    w[o][i] = s[o][i // G] * (q[o][i] - 8)

(zero point 8).  Codes travel two to a byte, the even input in the low
nibble.  The forward of a quantised model is the ordinary forward on these
weights (oracle.model), so this module only states the dequantisation.
"""

import numpy as np

ZERO_POINT = 8


def unpack_codes(packed):
    """Codes [out][in] from bytes [out][in / 2]: input 2j in the low nibble of
    byte j, input 2j + 1 in its high nibble."""
    b = np.asarray(packed, dtype=np.uint8)
    codes = np.empty(b.shape[:-1] + (2 * b.shape[-1],), dtype=np.int64)
    codes[..., 0::2] = b & 0x0F
    codes[..., 1::2] = b >> 4
    return codes


def dequantize(codes, scales, group):
    """float64 W[out][in] = scales[out][in // group] * (codes[out][in] - 8)."""
    q = np.asarray(codes, dtype=np.float64)
    s = np.asarray(scales, dtype=np.float64)
    n_out, n_in = q.shape
    if n_in % group != 0 or s.shape != (n_out, n_in // group):
        raise ValueError(f"codes {q.shape} and scales {s.shape} do not match group {group}")
    return np.repeat(s, group, axis=1) * (q - ZERO_POINT)
