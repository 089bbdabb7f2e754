"""Test helpers: build oracle inputs from the shared seeded generators."""

import numpy as np

import oracle
import workloads


def oracle_config(shape) -> oracle.OracleConfig:
    return oracle.OracleConfig(
        n_layers=shape.n_layers, d_model=shape.d_model, n_heads=shape.n_heads,
        head_dim=shape.head_dim, d_ffn=shape.d_ffn, vocab=shape.vocab,
        rms_eps=shape.rms_eps, rope_theta=shape.rope_theta)


def to_np(t):
    return t.float().cpu().numpy().astype(np.float64)


def host_matrix(v):
    """float64 host copy of a plain weight, or the matrix a 4-bit (codes, scales) pair stands for."""
    if isinstance(v, tuple):
        codes, scales = v
        return oracle.dequantize(oracle.unpack_codes(codes.cpu().numpy()), to_np(scales), 128)
    return to_np(v)


def oracle_weights(shape, gain_jitter=0.0, cache=True) -> oracle.OracleWeights:
    gen = workloads.make_weights(shape, "cpu", gain_jitter)

    def layer_fn(l):
        return {k: host_matrix(v) for k, v in gen.layer(l).items()}

    return oracle.OracleWeights(oracle_config(shape), to_np(gen.tok_embed()),
                                to_np(gen.final_norm()), to_np(gen.lm_head()), layer_fn, cache=cache)
