"""Pins for the oracle's tree-masked pass.

Brute force: every node's logits must equal the last-position logits of the
ordinary causal forward over prefix + the node's branch (the paper's claim
that one non-autoregressive pass gives the same results as examining each
branch sequentially, §3.2).  Plus invariants that hold for any correct
implementation and special cases that reduce to the causal forward.
"""

import numpy as np
import pytest

import oracle
import workloads
from oracle.model import ancestors_and_self
from tests.util import oracle_weights

TINY = workloads.MODELS["tiny"]


@pytest.fixture(scope="module")
def ow():
    return oracle_weights(TINY, gain_jitter=0.1)


@pytest.fixture(scope="module")
def prefix(ow):
    toks = workloads.draw_tokens(32, TINY.vocab, seed=3)
    out = {}
    for rounding in (False, True):
        out[rounding] = oracle.prefill_kv(ow, toks, rounding)
    return toks, out


def _brute(ow, prefix_toks, tok, parent, i, rounding):
    branch = ancestors_and_self(parent, i)
    seq = np.concatenate([prefix_toks, np.asarray(tok)[branch]])
    logits, _, _ = oracle.causal_forward(ow, seq, rounding)
    return logits[-1]


TREES = {
    "binary_d3": workloads.complete_tree((2, 2, 2)),
    "branch_432": workloads.complete_tree((4, 3, 2))[:20],
    "random20": workloads.random_tree(20, 7, 5),
    "chain6": workloads.chain_tree(6),
    "single": workloads.chain_tree(1),
}


@pytest.mark.parametrize("name", sorted(TREES))
def test_brute_force_float64(ow, prefix, name):
    parent = TREES[name]
    tok = workloads.draw_tokens(len(parent), TINY.vocab, seed=17, stream=len(parent))
    ptoks, kv = prefix
    logits, _, _ = oracle.tree_forward(ow, kv[False][0], kv[False][1], tok, parent, rounding=False)
    for i in range(len(parent)):
        ref = _brute(ow, ptoks, tok, parent, i, rounding=False)
        assert np.abs(logits[i] - ref).max() < 1e-9, (name, i)


def test_brute_force_with_bf16_storage(ow, prefix):
    # Same statement with activations rounded to bf16 at the storage points.
    parent = TREES["binary_d3"]
    tok = workloads.draw_tokens(len(parent), TINY.vocab, seed=23)
    ptoks, kv = prefix
    logits, _, _ = oracle.tree_forward(ow, kv[True][0], kv[True][1], tok, parent, rounding=True)
    for i in range(len(parent)):
        ref = _brute(ow, ptoks, tok, parent, i, rounding=True)
        assert np.abs(logits[i] - ref).max() < 1e-9, i


def test_prefill_split_equals_whole(ow):
    toks = workloads.draw_tokens(40, TINY.vocab, seed=5)
    whole, kw, vw = oracle.causal_forward(ow, toks, rounding=False)
    k1, v1 = oracle.prefill_kv(ow, toks[:25], rounding=False)
    part, k2, v2 = oracle.causal_forward(ow, toks[25:], rounding=False, past_k=k1, past_v=v1)
    assert np.abs(part - whole[25:]).max() < 1e-9
    assert np.abs(np.concatenate([k1, k2], axis=1) - kw).max() < 1e-12


def test_relabelling_permutes_rows(ow, prefix):
    # Any topological relabelling of the nodes permutes the logit rows.
    parent = TREES["random20"]
    n = len(parent)
    tok = workloads.draw_tokens(n, TINY.vocab, seed=29)
    _, kv = prefix
    base, _, _ = oracle.tree_forward(ow, kv[False][0], kv[False][1], tok, parent, rounding=False)
    rng = np.random.default_rng(0)
    # random topological order: repeatedly pick a random available node
    order, avail, placed = [0], set(), {0}
    children = {i: [c for c in range(n) if parent[c] == i] for i in range(n)}
    avail.update(children[0])
    while avail:
        c = sorted(avail)[rng.integers(len(avail))]
        avail.remove(c)
        order.append(c)
        placed.add(c)
        avail.update(children[c])
    new_of = {old: new for new, old in enumerate(order)}
    parent2 = np.array([-1] + [new_of[int(parent[o])] for o in order[1:]], dtype=np.int32)
    tok2 = np.asarray(tok)[order]
    perm, _, _ = oracle.tree_forward(ow, kv[False][0], kv[False][1], tok2, parent2, rounding=False)
    assert np.abs(perm - base[order]).max() < 1e-10


def test_sibling_independence_and_duplicates(ow, prefix):
    parent = TREES["binary_d3"]
    n = len(parent)
    tok = workloads.draw_tokens(n, TINY.vocab, seed=31)
    _, kv = prefix
    K, V = kv[False]
    base, _, _ = oracle.tree_forward(ow, K, V, tok, parent, rounding=False)
    # change node 2's token: only node 2's subtree may change
    tok_b = tok.copy()
    tok_b[2] = (tok_b[2] + 1) % TINY.vocab
    alt, _, _ = oracle.tree_forward(ow, K, V, tok_b, parent, rounding=False)
    subtree = {i for i in range(n) if 2 in ancestors_and_self(parent, i)}
    for i in range(n):
        diff = np.abs(alt[i] - base[i]).max()
        if i in subtree:
            assert diff > 1e-3, i
        else:
            assert diff < 1e-12, i
    # identical sibling subtrees (nodes 1 and 2 with the same tokens below) give identical rows
    tok_c = tok.copy()
    tok_c[2] = tok_c[1]
    tok_c[5], tok_c[6] = tok_c[3], tok_c[4]
    dup, _, _ = oracle.tree_forward(ow, K, V, tok_c, parent, rounding=False)
    for a, b in ((1, 2), (3, 5), (4, 6)):
        assert np.abs(dup[a] - dup[b]).max() < 1e-12


def test_planted_tree_accepts_exactly_k(ow, prefix):
    # Plant the target's own greedy continuation along one branch: the walk
    # must accept exactly K nodes and return the target's next token.
    ptoks, kv = prefix
    parent = TREES["binary_d3"]
    tok = workloads.draw_tokens(len(parent), TINY.vocab, seed=37)
    K = 2
    seq = [int(x) for x in np.concatenate([ptoks, tok[:1]])]
    cont = []
    for _ in range(K + 1):
        logits, _, _ = oracle.causal_forward(ow, seq, rounding=True)
        cont.append(int(np.argmax(logits[-1])))
        seq.append(cont[-1])
    leaf = len(parent) - 1
    tok_p = workloads.plant_path(parent, tok, leaf, cont, TINY.vocab)
    res = oracle.verify_tree(ow, kv[True][0], kv[True][1], tok_p, parent, rounding=True)
    assert res["accept_len"] == K
    assert res["next_token"] == cont[K]
    assert res["path"] == ancestors_and_self(parent, leaf)[:K + 1]
    assert res["rectified"] is True
