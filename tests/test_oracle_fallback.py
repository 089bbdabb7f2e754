"""Pins of the oracle's self-adaptive fallback (§3.3): the Eq. 3 update worked
out by hand, its closed forms, the most matching branch on a hand-built tree,
and the fallback stop in the hand-worked pacer example (T_c after each step
worked out by hand)."""

import numpy as np
import pytest

import oracle

# Successor distributions by fed token, as in the hand-worked pacer example.
TABLE = {0: {1: .60, 2: .35}, 1: {3: .50, 4: .45}, 2: {5: .90}}


def _forward(tokens, parent):
    p = dict(TABLE.get(int(tokens[-1]), {6: .95}))
    rest = (1.0 - sum(p.values())) / (8 - len(p))
    return np.log(np.array([p.get(t, rest) for t in range(8)]))


def test_eq3_by_hand():
    assert oracle.DEFAULT_ALPHA == 0.01
    # all correct: halved
    assert oracle.update_alpha(0.01, 3, 3, 0.2) == pytest.approx(0.005, rel=1e-15)
    # half wrong, T_c = 1/4: divided by (1/4)^(1/2) = 1/2
    assert oracle.update_alpha(0.01, 2, 4, 0.25) == pytest.approx(0.02, rel=1e-15)
    # all wrong: divided by T_c itself
    assert oracle.update_alpha(0.01, 0, 4, 0.25) == pytest.approx(0.04, rel=1e-15)
    # one of three wrong, T_c = 1/8: divided by (1/8)^(1/3) = 1/2
    assert oracle.update_alpha(0.03, 2, 3, 0.125) == pytest.approx(0.06, rel=1e-14)


def test_eq3_closed_forms():
    a = 0.01
    for k in range(1, 8):
        a = oracle.update_alpha(a, 5, 5, 0.9)
        assert a == pytest.approx(0.01 * 2.0 ** -k, rel=1e-15)
    # an error never lowers alpha (T_c <= 1), and a certain tree (T_c = 1) leaves it
    assert oracle.update_alpha(0.01, 1, 4, 1.0) == 0.01
    assert oracle.update_alpha(0.01, 1, 4, 0.5) > 0.01
    assert oracle.tree_confidence([0.2, 0.7, 0.1]) == 0.7


def test_most_matching_branch():
    parent = [-1, 0, 0, 1, 1, 3]     # depths 0, 1, 1, 2, 2, 3
    assert oracle.most_matching_branch(parent, [0, 1]) == (3, 1)      # deepest leaf under 1: node 5
    assert oracle.most_matching_branch(parent, [0]) == (3, 0)
    assert oracle.most_matching_branch(parent, [0, 2]) == (1, 1)      # all correct
    assert oracle.most_matching_branch(parent, [0, 1, 4]) == (2, 2)


@pytest.mark.parametrize("alpha,fed,tokens,parents,t_c", [
    # T_c by hand: root .6; after node 1 .35; after node 2 .315; after node 3 (token 5) .30
    (0.7, 1, [0, 1, 2], [-1, 0, 0], [.6]),
    (0.36, 2, [0, 1, 2, 3, 4], [-1, 0, 0, 1, 1], [.6, .35]),
    (0.32, 3, [0, 1, 2, 3, 4, 5], [-1, 0, 0, 1, 1, 2], [.6, .35, .315]),
    (0.2, 4, [0, 1, 2, 5, 3, 4, 6], [-1, 0, 0, 2, 1, 1, 3], [.6, .35, .315, .30]),
])
def test_fallback_stop_by_hand(alpha, fed, tokens, parents, t_c):
    tok, par, info = oracle.generate_tree(None, None, None, 0, 3, threshold=0.3, forward=_forward, alpha=alpha)
    assert tok.tolist() == tokens and par.tolist() == parents
    assert info["fed"] == fed
    np.testing.assert_allclose(info["t_c"], t_c, rtol=1e-12)
