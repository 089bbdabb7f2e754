"""Random bf16 weights for a LLaMA-shaped decoder, regenerated per tensor.

Every weight element is drawn from a counter-based stream keyed by
(model seed, tensor kind, layer), so any single tensor can be regenerated on
its own, on CPU or GPU, bit-identically.  The distribution is the
Irwin-Hall sum of four independent 16-bit uniforms, centred and scaled to the
requested standard deviation (0.02): a bounded, symmetric, near-normal law
with the same mean and variance as N(0, 0.02**2).  The scaled value is formed
in fp32 from an exactly representable integer and then rounded to bf16
(round-to-nearest-even).  Norm gains are 1 unless gain jitter is requested.

Plain (unpacked) layouts, all row-major with W[out][in]:
  tok_embed [V][d], lm_head [V][d], final_norm [d]
  per layer: attn_norm [d], w_qkv [3d][d] (rows: q, k, v), w_o [d][d],
             ffn_norm [d], w_gate_up [2F][d] (rows: gate, up), w_down [d][F]

4-bit models (weight_bits 4) give each layer matrix as a pair (codes, scales):
codes uint8 [out][in / 2] (input 2j in the low nibble of byte j); each code is
8 + trunc((a - b) / 2) for two independent uniform nibbles a, b, a symmetric
bell over [1, 15] centred on the zero point 8 (GPTQ's symmetric codes of
near-normal weights have that shape; uniform codes would give every weight a
mean of -s / 2); scales bf16 [out][in / 128], each uniform in [0.75, 1.25)
times weight_std / 3.067, the RMS of (code - 8), so that the weights the pairs
stand for have about the bf16 models' spread.  The embedding, LM head and norm
gains stay bf16.
"""

import math

import torch

from .configs import ModelShape
from .rng import hash_uniform16, tensor_key

KIND = {
    "tok_embed": 1,
    "final_norm": 2,
    "lm_head": 3,
    "attn_norm": 10,
    "w_qkv": 11,
    "w_o": 12,
    "ffn_norm": 13,
    "w_gate_up": 14,
    "w_down": 15,
}

_IH4_STD = math.sqrt(4.0 * (65536.0 * 65536.0 - 1.0) / 12.0)
_Q4_GROUP = 128
_Q4_CODE_STD = math.sqrt(2408.0 / 256.0)  # RMS of trunc((a - b) / 2) over uniform nibbles a, b
_SCALE_TAG = 0x40  # added to a matrix's kind for its scales' stream
_CHUNK = 1 << 24


def _draw(numel: int, key: tuple, std: float, device) -> torch.Tensor:
    out = torch.empty(numel, dtype=torch.bfloat16, device=device)
    scale = torch.tensor(std / _IH4_STD, dtype=torch.float32, device=device)
    for start in range(0, numel, _CHUNK):
        stop = min(numel, start + _CHUNK)
        e = torch.arange(start, stop, dtype=torch.int64, device=device)
        h0 = hash_uniform16(2 * e, key)
        h1 = hash_uniform16(2 * e + 1, key)
        s = (h0 & 0xFFFF) + (h0 >> 16) + (h1 & 0xFFFF) + (h1 >> 16) - 2 * 65535
        out[start:stop] = (s.to(torch.float32) * scale).to(torch.bfloat16)
    return out


def gen_tensor(shape: ModelShape, kind: str, layer: int, dims: tuple, device="cpu",
               std: float | None = None) -> torch.Tensor:
    tag = (KIND[kind] << 16) | (layer & 0xFFFF)
    key = tensor_key(shape.seed, tag)
    numel = 1
    for x in dims:
        numel *= x
    std = shape.weight_std if std is None else std
    return _draw(numel, key, std, device).view(*dims)


def _draw_codes(nbytes: int, key: tuple, device) -> torch.Tensor:
    out = torch.empty(nbytes, dtype=torch.uint8, device=device)
    for start in range(0, nbytes, _CHUNK):
        stop = min(nbytes, start + _CHUNK)
        e = torch.arange(start, stop, dtype=torch.int64, device=device)
        h = hash_uniform16(e, key)

        def code(shift):  # 8 + trunc((a - b) / 2) from the nibbles at bits shift and shift + 4
            a, b = (h >> shift) & 0xF, (h >> (shift + 4)) & 0xF
            return 8 + torch.div(a - b, 2, rounding_mode="trunc")

        out[start:stop] = (code(0) | (code(8) << 4)).to(torch.uint8)
    return out


def _draw_scales(numel: int, key: tuple, std: float, device) -> torch.Tensor:
    out = torch.empty(numel, dtype=torch.bfloat16, device=device)
    for start in range(0, numel, _CHUNK):
        stop = min(numel, start + _CHUNK)
        e = torch.arange(start, stop, dtype=torch.int64, device=device)
        u = (hash_uniform16(e, key) & 0xFFFF).to(torch.float32) * (1.0 / 65536.0)
        out[start:stop] = ((0.75 + 0.5 * u) * (std / _Q4_CODE_STD)).to(torch.bfloat16)
    return out


def gen_q4_matrix(shape: ModelShape, kind: str, layer: int, dims: tuple, device="cpu") -> tuple:
    """(codes uint8 [out][in / 2], scales bf16 [out][in / 128]) of one 4-bit matrix."""
    n_out, n_in = dims
    if n_in % _Q4_GROUP != 0:
        raise ValueError(f"4-bit matrices need inputs in multiples of {_Q4_GROUP}, got {n_in}")
    tag = (KIND[kind] << 16) | (layer & 0xFFFF)
    codes = _draw_codes(n_out * n_in // 2, tensor_key(shape.seed, tag), device).view(n_out, n_in // 2)
    stag = ((KIND[kind] + _SCALE_TAG) << 16) | (layer & 0xFFFF)
    scales = _draw_scales(n_out * (n_in // _Q4_GROUP), tensor_key(shape.seed, stag), shape.weight_std,
                          device).view(n_out, n_in // _Q4_GROUP)
    return codes, scales


class ModelWeights:
    """Lazily generated weights of one model shape on one device."""

    def __init__(self, shape: ModelShape, device="cpu", gain_jitter: float = 0.0):
        self.shape = shape
        self.device = device
        self.gain_jitter = gain_jitter

    def _gain(self, kind: str, layer: int) -> torch.Tensor:
        d = self.shape.d_model
        if self.gain_jitter == 0.0:
            return torch.ones(d, dtype=torch.bfloat16, device=self.device)
        j = gen_tensor(self.shape, kind, layer, (d,), self.device, std=self.gain_jitter)
        return (1.0 + j.float()).to(torch.bfloat16)

    def tok_embed(self) -> torch.Tensor:
        s = self.shape
        return gen_tensor(s, "tok_embed", 0, (s.vocab, s.d_model), self.device)

    def lm_head(self) -> torch.Tensor:
        s = self.shape
        return gen_tensor(s, "lm_head", 0, (s.vocab, s.d_model), self.device)

    def final_norm(self) -> torch.Tensor:
        return self._gain("final_norm", 0)

    def layer(self, l: int) -> dict:
        s = self.shape
        d, f = s.d_model, s.d_ffn
        if s.weight_bits == 4:
            return {
                "attn_norm": self._gain("attn_norm", l),
                "w_qkv": gen_q4_matrix(s, "w_qkv", l, (3 * d, d), self.device),
                "w_o": gen_q4_matrix(s, "w_o", l, (d, d), self.device),
                "ffn_norm": self._gain("ffn_norm", l),
                "w_gate_up": gen_q4_matrix(s, "w_gate_up", l, (2 * f, d), self.device),
                "w_down": gen_q4_matrix(s, "w_down", l, (d, f), self.device),
            }
        return {
            "attn_norm": self._gain("attn_norm", l),
            "w_qkv": gen_tensor(s, "w_qkv", l, (3 * d, d), self.device),
            "w_o": gen_tensor(s, "w_o", l, (d, d), self.device),
            "ffn_norm": self._gain("ffn_norm", l),
            "w_gate_up": gen_tensor(s, "w_gate_up", l, (2 * f, d), self.device),
            "w_down": gen_tensor(s, "w_down", l, (d, f), self.device),
        }


def make_weights(shape: ModelShape, device="cpu", gain_jitter: float = 0.0) -> ModelWeights:
    return ModelWeights(shape, device, gain_jitter)
