"""Pins of the oracle's generate-and-verify loop (§3.1, §3.2 rollback).

The loop must reproduce plain greedy decoding token for token, whatever the
draft trees hold (planted greedy continuations of every length, fully correct
branches, uniform noise), and after each rollback the prefix cache must equal
the causal cache of the accepted sequence.  A commit in node order instead of
path order, a plausible mistake, is caught.
"""

import numpy as np
import pytest

import oracle
import workloads
from tests.util import oracle_weights

SHAPE = workloads.MODELS["tiny"]
P = 16
STEPS = 14


@pytest.fixture(scope="module")
def setup():
    ow = oracle_weights(SHAPE, gain_jitter=0.1)
    prefix = workloads.draw_tokens(P, SHAPE.vocab, seed=11)
    first = int(workloads.draw_tokens(1, SHAPE.vocab, seed=12)[0])
    greedy, gaps = oracle.greedy_decode(ow, prefix, first, STEPS + 8, rounding=True)
    # a meaningful exact comparison: no near-tie among the greedy choices
    assert gaps.min() > 1e-9, gaps.min()
    return ow, prefix, first, greedy


def _planted(greedy, parent, schedule, leaves):
    """Drafts planting K tokens of the true greedy continuation along a leaf's branch."""
    it = [0]

    def draft(root, produced):
        i = it[0]
        it[0] += 1
        cont = greedy[len(produced):]
        return workloads.draft_tree(parent, root, cont, schedule[i % len(schedule)],
                                    leaves[i % len(leaves)], SHAPE.vocab, seed=100 + i), parent

    return draft


def test_planted_drafts_equal_greedy(setup):
    ow, prefix, first, greedy = setup
    parent = workloads.complete_tree((2, 2, 2))
    out, log, _, _ = oracle.speculative_decode(
        ow, prefix, first, STEPS, _planted(greedy, parent, [0, 1, 2, 3, 1, 3], [14, 7, 10]), rounding=True)
    np.testing.assert_array_equal(out, greedy[:STEPS])
    lens = [r["accept_len"] for r in log]
    assert lens[:4] == [0, 1, 2, 3], lens          # exactly the planted length is accepted
    assert log[3]["rectified"] is False             # a fully correct branch: bonus token
    assert log[1]["rectified"] is True


def test_random_drafts_equal_greedy(setup):
    ow, prefix, first, greedy = setup
    parent = workloads.random_tree(20, 7, 5)

    def draft(root, produced):
        tok = workloads.draw_tokens(len(parent), SHAPE.vocab, seed=500 + len(produced), stream=3)
        tok[0] = root
        return tok, parent

    out, log, _, _ = oracle.speculative_decode(ow, prefix, first, 6, draft, rounding=True)
    np.testing.assert_array_equal(out, greedy[:6])


def test_chain_bonus_equals_greedy(setup):
    ow, prefix, first, greedy = setup
    parent = workloads.chain_tree(5)
    out, log, _, _ = oracle.speculative_decode(
        ow, prefix, first, STEPS, _planted(greedy, parent, [4], [4]), rounding=True)
    np.testing.assert_array_equal(out, greedy[:STEPS])
    assert all(r["accept_len"] == 4 and not r["rectified"] for r in log)


def _cache_matches_causal(ow, prefix, first, all_tokens, cache):
    k, v = cache
    committed = [first] + list(all_tokens[:-1])  # the last next-token is not in the cache yet
    rk, rv = oracle.prefill_kv(ow, np.concatenate([prefix, committed]), rounding=False)
    return k.shape == rk.shape and np.abs(k - rk).max() < 1e-9 and np.abs(v - rv).max() < 1e-9


def test_rollback_cache_is_causal_cache(setup):
    ow, prefix, first, greedy = setup
    parent = workloads.complete_tree((2, 2, 2))
    draft = _planted(greedy, parent, [3, 2, 3], [14, 10])
    out, log, cache, all_tokens = oracle.speculative_decode(ow, prefix, first, 8, draft, rounding=False)
    assert any(r["path"] != list(range(len(r["path"]))) for r in log)  # paths not in node order
    assert _cache_matches_causal(ow, prefix, first, all_tokens, cache)


def test_commit_in_node_order_is_caught(setup):
    ow, prefix, first, greedy = setup
    parent = workloads.complete_tree((2, 2, 2))
    draft = _planted(greedy, parent, [3, 2, 3], [14, 10])

    def wrong_commit(k, v, tk, tv, path):
        return oracle.commit_path(k, v, tk, tv, list(range(len(path))))

    _, _, cache, all_tokens = oracle.speculative_decode(ow, prefix, first, 8, draft, rounding=False,
                                                        commit=wrong_commit)
    assert not _cache_matches_causal(ow, prefix, first, all_tokens, cache)
