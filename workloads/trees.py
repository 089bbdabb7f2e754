"""Token-tree shapes and token draws.

A tree is given as parent[n] (int32) in topological order: parent[0] = -1 for
the root (the last accepted token), 0 <= parent[i] < i otherwise.  Tokens are
tree_tokens[n]; tree_tokens[0] is the root's token.
"""

import numpy as np


def complete_tree(branching) -> np.ndarray:
    """Root plus levels where every node of level k has branching[k] children (BFS order)."""
    parent = [-1]
    level = [0]
    for b in branching:
        nxt = []
        for p in level:
            for _ in range(b):
                parent.append(p)
                nxt.append(len(parent) - 1)
        level = nxt
    return np.asarray(parent, dtype=np.int32)


def chain_tree(n: int) -> np.ndarray:
    return np.arange(-1, n - 1, dtype=np.int32)


def tree_depths(parent) -> np.ndarray:
    parent = np.asarray(parent)
    depth = np.zeros(len(parent), dtype=np.int32)
    for i in range(1, len(parent)):
        depth[i] = depth[parent[i]] + 1
    return depth


def random_tree(n: int, max_parent_depth: int, seed: int) -> np.ndarray:
    """parent[i] uniform over {j < i : depth[j] <= max_parent_depth} (numpy PCG64)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    parent = np.full(n, -1, dtype=np.int32)
    depth = np.zeros(n, dtype=np.int32)
    for i in range(1, n):
        eligible = np.nonzero(depth[:i] <= max_parent_depth)[0]
        p = int(eligible[rng.integers(0, len(eligible))])
        parent[i] = p
        depth[i] = depth[p] + 1
    return parent


def draw_tokens(count: int, vocab: int, seed: int, stream: int = 0) -> np.ndarray:
    """Uniform token ids in [0, vocab) from numpy PCG64 seeded by (seed, stream)."""
    rng = np.random.Generator(np.random.PCG64([seed, stream]))
    return rng.integers(0, vocab, size=count, dtype=np.int64).astype(np.int32)


def make_tree(recipe, vocab: int, seed: int):
    """(parent, tree_tokens) from a workload tree recipe (see configs.Workload)."""
    kind = recipe[0]
    if kind == "complete":
        parent = complete_tree(recipe[1])
    elif kind == "random":
        parent = random_tree(recipe[1], recipe[2], seed)
    elif kind == "chain":
        parent = chain_tree(recipe[1])
    else:
        raise ValueError(f"unknown tree recipe {recipe!r}")
    tokens = draw_tokens(len(parent), vocab, seed, stream=1)
    return parent, tokens


def plant_path(parent, tree_tokens, leaf: int, continuation, vocab: int):
    """Plant a greedy continuation along the root->leaf branch.

    continuation = (c_1, ..., c_{K+1}): the target's greedy tokens after the
    root, supplied by the caller.  The branch node at depth k gets c_k for
    k <= K; the branch node at depth K+1 (if any) gets a token other than
    c_{K+1}.  Any node hanging off the branch at depth k <= K+1 (a sibling of
    a branch node) that carries c_k is given another token, so that exactly
    K draft nodes can match.  Returns a new token array.
    """
    parent = np.asarray(parent)
    tok = np.array(tree_tokens, dtype=np.int32, copy=True)
    chain = []
    i = leaf
    while i != -1:
        chain.append(i)
        i = int(parent[i])
    chain = chain[::-1]  # root .. leaf
    K = len(continuation) - 1
    children = {}
    for c in range(1, len(parent)):
        children.setdefault(int(parent[c]), []).append(c)
    for k in range(1, min(len(chain), K + 2)):
        node = chain[k]
        c_k = int(continuation[k - 1])
        if k <= K:
            tok[node] = c_k
        elif tok[node] == c_k:
            tok[node] = (c_k + 1) % vocab
        for sib in children.get(int(parent[node]), []):
            if sib != node and tok[sib] == c_k:
                tok[sib] = (c_k + 1) % vocab
    return tok


def draft_tree(parent, root_token: int, continuation, K: int, leaf: int, vocab: int, seed: int):
    """Draft tokens for a tree of the given shape: the root carries root_token,
    every other node a uniform draw, and the root->leaf branch has the first K
    tokens of `continuation` (the target's greedy tokens after the root,
    supplied by the caller) planted, then a wrong token (plant_path)."""
    tok = draw_tokens(len(parent), vocab, seed, stream=2)
    tok[0] = root_token
    return plant_path(parent, tok, leaf, list(continuation)[: K + 1], vocab)
