"""Pins for the oracle's accept walk: the paper's worked example, hand-built cases,
and exhaustive path enumeration on small random trees."""

import json
import os

import numpy as np
import pytest

import oracle
import workloads

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_paper_worked_example():
    with open(os.path.join(GOLDEN, "paper_s3_2_verification_example.json")) as f:
        ex = json.load(f)
    parent, tok, amax = ex["parent"], ex["tree_tokens"], ex["amax"]
    seqs = oracle.correct_sequences(parent, tok, amax)
    got_tokens = [[tok[i] for i in acc] + [nxt] for acc, nxt, _ in seqs]
    assert got_tokens == ex["expected"]["branch_correct_tokens"]
    path, nxt, rect = oracle.accept_walk(parent, tok, amax)
    assert path == ex["expected"]["path"]
    assert len(path) - 1 == ex["expected"]["accept_len"]
    assert nxt == ex["expected"]["next_token"]
    assert rect == ex["expected"]["rectified"]


@pytest.mark.parametrize("case", [
    # (parent, tokens, amax, path, next, rectified)
    ([-1], [5], [7], [0], 7, False),                                   # root only: bonus token
    ([-1, 0, 1, 2, 3], [0, 1, 2, 3, 4], [1, 2, 3, 4, 9], [0, 1, 2, 3, 4], 9, False),  # chain, all match
    ([-1, 0, 1, 2, 3], [0, 1, 2, 3, 4], [1, 2, 8, 4, 9], [0, 1, 2], 8, True),         # error at depth 3
    ([-1, 0, 0, 1, 1, 2, 2], [0, 5, 6, 1, 2, 3, 4], [9, 0, 0, 0, 0, 0, 0], [0], 9, True),  # nothing matches
    ([-1, 0, 0, 1, 2, 4], [0, 3, 3, 7, 8, 1], [3, 7, 8, 0, 1, 2], [0, 2, 4, 5], 2, False),  # duplicate siblings, deeper wins
    ([-1, 0, 0, 1, 2], [0, 3, 3, 7, 8], [3, 7, 8, 5, 6], [0, 1, 3], 5, False),       # equal depth: smaller index
    ([-1, 0, 0, 0], [0, 4, 5, 6], [6, 1, 1, 1], [0, 3], 1, False),                  # third child matches
])
def test_hand_built(case):
    parent, tok, amax, want_path, want_next, want_rect = case
    path, nxt, rect = oracle.accept_walk(parent, tok, amax)
    assert (path, nxt, rect) == (want_path, want_next, want_rect)


def _enumerate(parent, tok, amax):
    """Independent statement: over every node, the root path is accepted iff each
    node's token equals the target token at its parent; keep the deepest, then
    the smallest node index."""
    n = len(parent)
    best = None
    for i in range(n):
        chain = []
        j = i
        while j != -1:
            chain.append(j)
            j = parent[j]
        chain = chain[::-1]
        ok = all(tok[chain[k]] == amax[chain[k - 1]] for k in range(1, len(chain)))
        if ok and (best is None or len(chain) > len(best)):
            best = chain
    has_child = best[-1] in set(parent[1:])
    return best, amax[best[-1]], has_child


@pytest.mark.parametrize("seed", range(60))
def test_exhaustive_small_trees(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 16))
    parent = [int(x) for x in workloads.random_tree(n, 7, seed)]
    vocab = 3  # tiny vocabulary so that matches (and duplicate siblings) are frequent
    tok = [int(x) for x in rng.integers(0, vocab, n)]
    amax = [int(x) for x in rng.integers(0, vocab, n)]
    assert oracle.accept_walk(parent, tok, amax) == _enumerate(parent, tok, amax)
