"""Plausible mistakes planted in the oracle (on the CPU) must be caught by its pins.

Each case patches one piece of oracle.model, reruns the brute-force check of
the tree pass and asserts that it now fails.  This shows the pins can tell a
right tree pass from a wrong one.
"""

import numpy as np
import pytest

import oracle
import oracle.model as om
import workloads
from tests.util import oracle_weights

TINY = workloads.MODELS["tiny"]


@pytest.fixture(scope="module")
def setup():
    ow = oracle_weights(TINY, gain_jitter=0.1)
    ptoks = workloads.draw_tokens(16, TINY.vocab, seed=3)
    k, v = oracle.prefill_kv(ow, ptoks, rounding=False)
    parent = workloads.complete_tree((2, 2))
    tok = workloads.draw_tokens(len(parent), TINY.vocab, seed=41)
    ref = []
    for i in range(len(parent)):
        seq = np.concatenate([ptoks, tok[om.ancestors_and_self(parent, i)]])
        ref.append(oracle.causal_forward(ow, seq, rounding=False)[0][-1])
    return ow, k, v, parent, tok, np.stack(ref)


def _err(setup):
    ow, k, v, parent, tok, ref = setup
    logits, _, _ = oracle.tree_forward(ow, k, v, tok, parent, rounding=False)
    return np.abs(logits - ref).max()


def test_unmutated_passes(setup):
    assert _err(setup) < 1e-9


def test_position_by_node_index_is_caught(setup, monkeypatch):
    monkeypatch.setattr(om, "_depths", lambda parent: np.arange(len(parent)))
    assert _err(setup) > 1e-3


def test_mask_without_self_is_caught(setup, monkeypatch):
    real = om.ancestors_and_self
    monkeypatch.setattr(om, "ancestors_and_self", lambda parent, i: real(parent, i)[:-1])
    assert _err(setup) > 1e-3


def test_mask_over_all_earlier_nodes_is_caught(setup, monkeypatch):
    monkeypatch.setattr(om, "ancestors_and_self", lambda parent, i: list(range(i + 1)))
    assert _err(setup) > 1e-3


def test_rope_sign_error_is_caught(setup, monkeypatch):
    real = om.rope
    monkeypatch.setattr(om, "rope", lambda x, pos, theta: real(x, -np.asarray(pos), theta))
    ow, k, v, parent, tok, ref = setup
    # the prefix K/V were made by the unmutated forward, so any mismatch shows
    assert _err(setup) > 1e-3


def test_missing_residual_is_caught(setup, monkeypatch):
    real = om._ffn_residual

    def no_ffn_residual(cfg, w, x, R):
        y = real(cfg, w, x, R)
        return y - x  # drops the residual stream around the feed-forward block
    monkeypatch.setattr(om, "_ffn_residual", no_ffn_residual)
    assert _err(setup) > 1e-3
