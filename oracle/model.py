"""Plain float64 statement of the target model's forward and the tree-masked pass.

TEST INFRASTRUCTURE ONLY (see the package docstring).

What the verification pass computes (arXiv 2309.04255, §3.2): the target
model examines every draft token of a token tree in one non-autoregressive
pass, and the result at each position equals examining that position's
branch sequentially.  So for tree node i with root-to-i chain
(i_0 = 0, i_1, ..., i_d = i):

    logits_i = last-position logits of the ordinary causal forward over
               prefix s_0..s_{P-1} followed by t_{i_0}, ..., t_{i_d},
               at positions 0 .. P+d.

`causal_forward` is that plain definition.  `tree_forward` is the one-pass
form: every node is computed once, and node i attends to the prefix plus its
ancestors and itself only (§3.2, "Tree decoder": the masking table keeps
positions of other branches from affecting a token).  Brute force pins one
against the other.

The decoder block (the paper names its layers only generically, §2.1): token
embedding; per layer RMSNorm -> Q/K/V projections -> rotary positions ->
softmax attention -> output projection + residual -> RMSNorm -> SwiGLU
feed-forward + residual; final RMSNorm -> LM head.

Precision.  All arithmetic is float64.  Weights are bf16 values.  With
rounding=True the storage precision of the verified pass is applied: the
inputs of every projection (normalised activations, attention output, SwiGLU
product) and the stored q/k/v are rounded to bf16 (round-to-nearest-even); the
residual stream, scores, softmax and logits stay float64.  With
rounding=False no activation is rounded (pure float64 on bf16 weights).
"""

from dataclasses import dataclass

import numpy as np


@dataclass(frozen=True)
class OracleConfig:
    n_layers: int
    d_model: int
    n_heads: int
    head_dim: int
    d_ffn: int
    vocab: int
    rms_eps: float = 1e-6
    rope_theta: float = 10000.0


class OracleWeights:
    """Weights as float64 arrays in the plain W[out][in] layout.

    tok_embed [V][d], final_norm [d], lm_head [V][d]; layer_fn(l) returns a
    mapping with attn_norm [d], w_qkv [3d][d] (rows q, k, v), w_o [d][d],
    ffn_norm [d], w_gate_up [2F][d] (rows gate, up), w_down [d][F].
    """

    def __init__(self, cfg: OracleConfig, tok_embed, final_norm, lm_head, layer_fn, cache=True):
        self.cfg = cfg
        self.tok_embed = np.asarray(tok_embed, dtype=np.float64)
        self.final_norm = np.asarray(final_norm, dtype=np.float64)
        self.lm_head = np.asarray(lm_head, dtype=np.float64)
        self._layer_fn = layer_fn
        self._cache = {} if cache else None

    def layer(self, l: int) -> dict:
        if self._cache is not None and l in self._cache:
            return self._cache[l]
        raw = self._layer_fn(l)
        d, f = self.cfg.d_model, self.cfg.d_ffn
        qkv = np.asarray(raw["w_qkv"], dtype=np.float64)
        gu = np.asarray(raw["w_gate_up"], dtype=np.float64)
        w = {
            "attn_norm": np.asarray(raw["attn_norm"], dtype=np.float64),
            "wq": qkv[0:d],
            "wk": qkv[d:2 * d],
            "wv": qkv[2 * d:3 * d],
            "wo": np.asarray(raw["w_o"], dtype=np.float64),
            "ffn_norm": np.asarray(raw["ffn_norm"], dtype=np.float64),
            "wg": gu[0:f],
            "wu": gu[f:2 * f],
            "wd": np.asarray(raw["w_down"], dtype=np.float64),
        }
        if self._cache is not None:
            self._cache[l] = w
        return w


# ---------------------------------------------------------------- elementary

def bf16_round(x) -> np.ndarray:
    """Nearest bfloat16 value of each float64 element, ties to even, as float64.

    bfloat16 keeps 8 significant bits (7 stored) and float32's exponent
    range, so for normal magnitudes this is rounding the 52-bit float64
    fraction to 7 bits.  (Magnitudes below 2**-126 would be bf16 subnormals,
    which this does not model; they do not arise here.)
    """
    a = np.ascontiguousarray(x, dtype=np.float64)
    u = a.view(np.uint64)
    drop = np.uint64(45)
    lsb = (u >> drop) & np.uint64(1)
    half_minus_one = np.uint64((1 << 44) - 1)
    mask = ~np.uint64((1 << 45) - 1)
    r = (u + half_minus_one + lsb) & mask
    return r.view(np.float64).reshape(np.shape(x))


def rmsnorm(x, g, eps):
    """x / sqrt(mean(x^2) + eps) * g over the last axis."""
    x = np.asarray(x, dtype=np.float64)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * g


def rope(x, pos, theta):
    """Rotary position embedding, rotate-half pairing.

    x [..., Dh], pos broadcastable to x.shape[:-1].  Dimension j < Dh/2 is
    paired with j + Dh/2 and rotated by angle pos * theta**(-2j/Dh).
    """
    x = np.asarray(x, dtype=np.float64)
    dh = x.shape[-1]
    half = dh // 2
    inv_freq = theta ** (-2.0 * np.arange(half, dtype=np.float64) / dh)
    ang = np.asarray(pos, dtype=np.float64)[..., None] * inv_freq
    c, s = np.cos(ang), np.sin(ang)
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def silu(z):
    z = np.asarray(z, dtype=np.float64)
    return z / (1.0 + np.exp(-z))


def attend(q, k, v):
    """Softmax attention of one query over an explicit key list, all heads.

    q [H, Dh]; k, v [T, H, Dh] -> [H, Dh].  Scores scaled by 1/sqrt(Dh).
    """
    dh = q.shape[-1]
    # per head h: s_h = k_h q_h / sqrt(Dh) over the T keys, then p_h^T v_h
    # (products batched over the heads)
    s = np.matmul(k.transpose(1, 0, 2), q[:, :, None])[:, :, 0] / np.sqrt(dh)
    s = s - s.max(axis=1, keepdims=True)
    p = np.exp(s)
    p = p / p.sum(axis=1, keepdims=True)
    return np.matmul(p[:, None, :], v.transpose(1, 0, 2))[:, 0, :]


def _rnd(rounding):
    return bf16_round if rounding else (lambda a: np.asarray(a, dtype=np.float64))


def _qkv(cfg, w, x, pos, R):
    n = x.shape[0]
    h, dh = cfg.n_heads, cfg.head_dim
    xn = R(rmsnorm(x, w["attn_norm"], cfg.rms_eps))
    q = (xn @ w["wq"].T).reshape(n, h, dh)
    k = (xn @ w["wk"].T).reshape(n, h, dh)
    v = (xn @ w["wv"].T).reshape(n, h, dh)
    q = R(rope(q, np.asarray(pos)[:, None], cfg.rope_theta))
    k = R(rope(k, np.asarray(pos)[:, None], cfg.rope_theta))
    v = R(v)
    return q, k, v


def _attn_residual(cfg, w, x, o, R):
    n = x.shape[0]
    o = R(o.reshape(n, cfg.d_model))
    return x + o @ w["wo"].T


def _ffn_residual(cfg, w, x, R):
    xn = R(rmsnorm(x, w["ffn_norm"], cfg.rms_eps))
    hidden = R(silu(xn @ w["wg"].T) * (xn @ w["wu"].T))
    return x + hidden @ w["wd"].T


def _after_attention(cfg, w, x, o, R):
    return _ffn_residual(cfg, w, _attn_residual(cfg, w, x, o, R), R)


def _logits(weights, x, R):
    cfg = weights.cfg
    xn = R(rmsnorm(x, weights.final_norm, cfg.rms_eps))
    return xn @ weights.lm_head.T


# ---------------------------------------------------------------- causal form

def causal_forward(weights: OracleWeights, tokens, rounding=True, past_k=None, past_v=None):
    """Ordinary causal forward: the plain definition of what is verified.

    tokens [T]; optional past_k/past_v [L, S, H, Dh] hold the keys/values of
    S earlier positions.  Token t sits at position S + t and attends to every
    earlier position and itself.  Returns (logits [T, V], k [L, T, H, Dh],
    v [L, T, H, Dh]) for the new tokens.
    """
    cfg = weights.cfg
    R = _rnd(rounding)
    tokens = np.asarray(tokens, dtype=np.int64)
    T = len(tokens)
    S = 0 if past_k is None else past_k.shape[1]
    pos = S + np.arange(T)
    x = weights.tok_embed[tokens].copy()
    ks, vs = [], []
    for l in range(cfg.n_layers):
        w = weights.layer(l)
        q, k, v = _qkv(cfg, w, x, pos, R)
        kk = k if past_k is None else np.concatenate([past_k[l], k], axis=0)
        vv = v if past_v is None else np.concatenate([past_v[l], v], axis=0)
        o = np.stack([attend(q[t], kk[: S + t + 1], vv[: S + t + 1]) for t in range(T)])
        x = _after_attention(cfg, w, x, o, R)
        ks.append(k)
        vs.append(v)
    return _logits(weights, x, R), np.stack(ks), np.stack(vs)


def prefill_kv(weights: OracleWeights, prefix_tokens, rounding=True):
    """Keys/values of the accepted prefix, [L, P, H, Dh] each, by the causal forward."""
    _, k, v = causal_forward(weights, prefix_tokens, rounding)
    return k, v


# ---------------------------------------------------------------- tree form

def _depths(parent):
    depth = np.zeros(len(parent), dtype=np.int64)
    for i in range(1, len(parent)):
        depth[i] = depth[parent[i]] + 1
    return depth


def ancestors_and_self(parent, i):
    """Root-to-i node chain (i's branch up to and including i)."""
    chain = []
    while i != -1:
        chain.append(int(i))
        i = int(parent[i])
    return chain[::-1]


def tree_forward(weights: OracleWeights, prefix_k, prefix_v, tree_tokens, parent, rounding=True):
    """One masked pass over every node of a token tree (§3.2).

    prefix_k/prefix_v [L, P, H, Dh] are the accepted prefix's keys/values.
    Node i sits at position P + depth(i) and attends to all P prefix
    positions and to its own branch: its ancestors, root first, then itself.
    Returns (logits [n, V], tree k [L, n, H, Dh], tree v [L, n, H, Dh]).
    """
    cfg = weights.cfg
    R = _rnd(rounding)
    tree_tokens = np.asarray(tree_tokens, dtype=np.int64)
    x = weights.tok_embed[tree_tokens].copy()
    ks, vs = [], []
    for l in range(cfg.n_layers):
        _, x, k, v = tree_layer(weights, l, x, prefix_k[l], prefix_v[l], parent, rounding)
        ks.append(k)
        vs.append(v)
    return _logits(weights, x, R), np.stack(ks), np.stack(vs)


def tree_layer(weights: OracleWeights, l, x, prefix_k_l, prefix_v_l, parent, rounding=True):
    """Decoder layer l of the masked pass (§3.2).

    x [n, d] is the layer's input residual stream; prefix_k_l/prefix_v_l
    [P, H, Dh] are that layer's prefix keys/values.  Node i sits at position
    P + depth(i) and attends to the P prefix positions and to its branch
    (ancestors, root first, then itself).  Returns (the residual stream after
    the attention block, after the whole layer, tree k [n, H, Dh], tree v
    [n, H, Dh]).
    """
    cfg = weights.cfg
    R = _rnd(rounding)
    parent = np.asarray(parent, dtype=np.int64)
    n = len(parent)
    P = prefix_k_l.shape[0]
    pos = P + _depths(parent)
    w = weights.layer(l)
    x = np.asarray(x, dtype=np.float64)
    q, k, v = _qkv(cfg, w, x, pos, R)
    o = np.empty_like(q)
    for i in range(n):
        branch = ancestors_and_self(parent, i)
        keys = np.concatenate([prefix_k_l, k[branch]], axis=0)
        vals = np.concatenate([prefix_v_l, v[branch]], axis=0)
        o[i] = attend(q[i], keys, vals)
    x_mid = _attn_residual(cfg, w, x, o, R)
    return x_mid, _ffn_residual(cfg, w, x_mid, R), k, v


def logits_from_stream(weights: OracleWeights, x, rounding=True):
    """Final RMSNorm and LM head of a residual stream x [n, d] -> logits [n, V]."""
    return _logits(weights, np.asarray(x, dtype=np.float64), _rnd(rounding))


def verify_tree(weights: OracleWeights, prefix_k, prefix_v, tree_tokens, parent, rounding=True):
    """Tree forward, per-node greedy target token, and the accepted path.

    Returns a dict: logits [n, V], amax [n] (lowest index among equal
    maxima), path (root first), accept_len, next_token, rectified.
    """
    from .walk import accept_walk

    logits, _, _ = tree_forward(weights, prefix_k, prefix_v, tree_tokens, parent, rounding)
    amax = np.argmax(logits, axis=1)
    path, next_token, rectified = accept_walk(parent, tree_tokens, amax)
    return {
        "logits": logits,
        "amax": amax,
        "path": path,
        "accept_len": len(path) - 1,
        "next_token": int(next_token),
        "rectified": bool(rectified),
    }
