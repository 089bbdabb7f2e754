"""The shared seeded input generators: determinism, shapes, and distribution."""

import numpy as np
import torch

import workloads
from workloads.rng import _lowbias32_int, lowbias32


def test_lowbias32_tensor_matches_integer_form():
    rng = np.random.default_rng(0)
    xs = rng.integers(0, 2 ** 32, 20000, dtype=np.uint64)
    got = lowbias32(torch.from_numpy(xs.astype(np.int64))).numpy()
    want = np.array([_lowbias32_int(int(x)) for x in xs], dtype=np.int64)
    np.testing.assert_array_equal(got, want)


def test_weights_are_deterministic_and_scaled():
    shape = workloads.MODELS["tiny"]
    a = workloads.make_weights(shape).layer(1)["w_qkv"]
    b = workloads.make_weights(shape).layer(1)["w_qkv"]
    assert a.dtype == torch.bfloat16 and a.shape == (3 * 256, 256)
    assert torch.equal(a, b)
    c = workloads.make_weights(shape).layer(0)["w_qkv"]
    assert not torch.equal(a, c)
    x = a.float()
    assert abs(x.mean().item()) < 1e-3
    assert abs(x.std().item() - 0.02) < 5e-4
    # Irwin-Hall(4) support: |w| <= sqrt(12) * std
    assert x.abs().max().item() <= 0.02 * 12 ** 0.5 * 1.01


def test_trees():
    p = workloads.complete_tree((2, 2, 2, 2))
    assert len(p) == 31 and p[0] == -1 and workloads.tree_depths(p).max() == 4
    p = workloads.complete_tree((4, 3, 2))
    assert len(p) == 41 and list(np.bincount(workloads.tree_depths(p))) == [1, 4, 12, 24]
    for seed in range(5):
        r = workloads.random_tree(128, 7, seed)
        d = workloads.tree_depths(r)
        assert r[0] == -1 and all(0 <= r[i] < i for i in range(1, 128))
        assert d.max() <= 8 and all(d[r[i]] <= 7 for i in range(1, 128))
    t = workloads.draw_tokens(1000, 32000, seed=1)
    assert t.dtype == np.int32 and t.min() >= 0 and t.max() < 32000


def test_q4_weights_shape_and_law():
    # 4-bit layers: (codes, scales) pairs; codes 8 + trunc((a - b) / 2) lie in
    # [1, 15], symmetric about the zero point; scales in [0.75, 1.25) x std / 3.067
    shape = workloads.MODELS["q4small"]
    lay = workloads.make_weights(shape, "cpu").layer(1)
    d, f = shape.d_model, shape.d_ffn
    dims = {"w_qkv": (3 * d, d), "w_o": (d, d), "w_gate_up": (2 * f, d), "w_down": (d, f)}
    for k, (n_out, n_in) in dims.items():
        codes, scales = lay[k]
        assert codes.dtype == torch.uint8 and tuple(codes.shape) == (n_out, n_in // 2), k
        assert scales.dtype == torch.bfloat16 and tuple(scales.shape) == (n_out, n_in // 128), k
        q = torch.stack([codes & 0xF, codes >> 4], dim=-1).flatten().long()
        hist = torch.bincount(q, minlength=16)
        assert hist[0] == 0 and q.min() >= 1 and q.max() <= 15, k
        # symmetric law: counts of 8 + j and 8 - j agree to sampling noise
        for j in range(1, 8):
            a, b = float(hist[8 + j]), float(hist[8 - j])
            assert abs(a - b) <= 5 * (a + b) ** 0.5 + 5, (k, j)
        s = scales.float() * (3.0669610365963242 / shape.weight_std)
        assert s.min() >= 0.74 and s.max() <= 1.26, k
    assert lay["attn_norm"].dtype == torch.bfloat16 and tuple(lay["attn_norm"].shape) == (d,)
    again = workloads.make_weights(shape, "cpu").layer(1)
    assert torch.equal(again["w_down"][0], lay["w_down"][0]) and torch.equal(again["w_down"][1], lay["w_down"][1])
