"""Pins of the oracle's draft-side tree generation (§3.1 threshold, §3.2 tree
decoder and confidence-based branch pacer, Eq. 1).

- With a threshold no probability exceeds, the tree is one chain: the draft
  model's plain greedy decoding (an independent path: the causal forward).
- A hand-worked example: fixed successor distributions per token (through
  the forward hook), the tree worked out by hand from Eq. 1 and the threshold.
"""

import numpy as np
import pytest

import oracle
import workloads
from tests.util import oracle_weights

DRAFT = workloads.ModelShape("draft_tiny", 2, 256, 4, 64, 688, 1024, weight_std=0.1, seed=0x5EEDD001)


@pytest.fixture(scope="module")
def draft():
    ow = oracle_weights(DRAFT)
    prefix = workloads.draw_tokens(24, DRAFT.vocab, seed=41)
    pk, pv = oracle.prefill_kv(ow, prefix, rounding=True)
    return ow, prefix, pk, pv


def test_no_branching_is_greedy_decoding(draft):
    ow, prefix, pk, pv = draft
    root = 17
    tok, par, info = oracle.generate_tree(ow, pk, pv, root, 6, threshold=1.0)
    greedy, _ = oracle.greedy_decode(ow, prefix, root, 7, rounding=True)
    # fed nodes root + 6 greedy tokens, then the 7th greedy token as the one pending leaf
    np.testing.assert_array_equal(tok, np.concatenate([[root], greedy]))
    np.testing.assert_array_equal(par, np.arange(-1, 7))


def test_hand_worked_pacer_example():
    # Successor distributions by the fed token (vocabulary of 8; the rest of
    # the mass spread evenly):
    #   after 0: p(1) = .60, p(2) = .35     after 1: p(3) = .50, p(4) = .45
    #   after 2: p(5) = .90                 otherwise: p(6) = .95
    # M = 3 iterations, threshold .30.  By hand (deficit M C / sum C - T):
    #   root fed; pending 1 (C .6, T 1), 2 (C .35, T 1)
    #   it 1: deficits .895, .105 -> feed 1 (node 1); pending 2, 3 (C .3, T 2), 4 (C .27, T 2)
    #   it 2: deficits .141, -1.02, -1.12 -> feed 2 (node 2); pending 3, 4, 5 (C .315, T 2)
    #   it 3: deficits -.983, -1.085, -.932 -> feed 5 (node 3); pending 3, 4, 6 (C .299, T 3)
    table = {0: {1: .60, 2: .35}, 1: {3: .50, 4: .45}, 2: {5: .90}}

    def forward(tokens, parent):
        p = dict(table.get(int(tokens[-1]), {6: .95}))
        rest = (1.0 - sum(p.values())) / (8 - len(p))
        row = np.array([p.get(t, rest) for t in range(8)])
        return np.log(row)

    tok, par, info = oracle.generate_tree(None, None, None, 0, 3, threshold=0.3, forward=forward)
    assert tok.tolist() == [0, 1, 2, 5, 3, 4, 6]
    assert par.tolist() == [-1, 0, 0, 2, 1, 1, 3]
    assert info["fed"] == 4
