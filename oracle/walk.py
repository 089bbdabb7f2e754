"""Greedy acceptance over a verified token tree (arXiv 2309.04255, §3.2).

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper's steps after the one-pass verification:
  1. the tree is split into branch sequences (root-to-leaf chains);
  2. each branch's *correct sequence* is its prefix up to the first position
     where the draft token differs from the target's output, followed by the
     target's token at that position (the rectified token);
  3. the correct sequences form a *correct token tree*;
  4. a depth-first search picks the longest path in it: the verified sequence.

The target's output at a node is its greedy token (the highest-probability
token is taken as the ground truth, §1 and §3.1).  Readings taken here where
the paper is silent: a branch with no error ends with the target's token
after its leaf (a "bonus" token, so every correct sequence ends with exactly
one target token); among equally long paths the one ending at the node with
the smallest index wins.
"""

import numpy as np


def _children(parent):
    ch = {i: [] for i in range(len(parent))}
    for c in range(1, len(parent)):
        ch[int(parent[c])].append(c)
    return ch


def branch_sequences(parent):
    """Root-to-leaf node chains, one per leaf, leaves in increasing index."""
    parent = np.asarray(parent)
    ch = _children(parent)
    out = []
    for leaf in range(len(parent)):
        if ch[leaf]:
            continue
        chain = []
        i = leaf
        while i != -1:
            chain.append(i)
            i = int(parent[i])
        out.append(chain[::-1])
    return out


def correct_sequences(parent, tree_tokens, amax):
    """Per branch: (accepted node chain, target token after it, stopped at an error)."""
    out = []
    for chain in branch_sequences(parent):
        acc = [chain[0]]
        error = False
        for k in range(1, len(chain)):
            if int(tree_tokens[chain[k]]) == int(amax[chain[k - 1]]):
                acc.append(chain[k])
            else:
                error = True
                break
        out.append((acc, int(amax[acc[-1]]), error))
    return out


def accept_walk(parent, tree_tokens, amax):
    """Verified sequence: longest path of the correct token tree, by DFS.

    Returns (path, next_token, rectified): path is the accepted node chain,
    root first (path[0] = 0); next_token is the target's token after the
    last accepted node; rectified is True when that node has draft children
    (all of which were rejected), False when it is a draft leaf.
    """
    parent = np.asarray(parent)
    # Correct token tree over nodes: union of the accepted chains.
    succ = {}
    for acc, _, _ in correct_sequences(parent, tree_tokens, amax):
        for a, b in zip(acc[:-1], acc[1:]):
            succ.setdefault(a, set()).add(b)
    best = (0, 0)  # (depth, node) ; larger depth wins, then smaller node index
    stack = [(0, 0)]
    while stack:
        node, depth = stack.pop()
        if depth > best[0] or (depth == best[0] and node < best[1]):
            best = (depth, node)
        for c in sorted(succ.get(node, ()), reverse=True):
            stack.append((c, depth + 1))
    last = best[1]
    path = []
    i = last
    while i != -1:
        path.append(i)
        i = int(parent[i])
    path = path[::-1]
    rectified = bool(_children(parent)[last])
    return path, int(amax[last]), rectified
