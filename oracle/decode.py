"""Greedy generation with the target model: plainly, and by token-tree verification.

TEST INFRASTRUCTURE ONLY (see the package docstring).

LLMCad's loop (§3.1 "Simplified workflow"; §3.2 "Token tree verification and
rectification"): a draft token tree rooted at the last accepted token is
verified by the target in one pass; the verified sequence -- the longest root
path whose draft tokens equal the target's greedy tokens -- is kept, the tree
is rolled back to it, and generation continues from the target's token after
its last node (a rectified token where a draft token was wrong, or the next
token after a fully correct branch).  Every kept token is the target's own
greedy choice at its position, so the output equals greedy decoding with the
target alone (§2 and §3.2: verification loses no accuracy, and examining
tokens in one non-autoregressive pass gives the same results as examining
them one by one).

`greedy_decode` is that plain definition.  `speculative_decode` runs the loop
with `tree_forward` and `accept_walk`: the accepted nodes' keys/values (the
root's included) were computed at the positions they keep, so committing them
to the prefix cache in path order is the whole rollback.
"""

import numpy as np

from .model import causal_forward, prefill_kv, tree_forward
from .walk import accept_walk


def greedy_decode(weights, prefix_tokens, first_token, steps, rounding=True):
    """Plain greedy decoding.

    The prefix is in the cache; first_token (the last accepted token) is fed
    next, then each step feeds the argmax of the previous position (lowest
    index among equal maxima).  Returns (the `steps` tokens generated after
    first_token, the top-1 minus top-2 logit gap at each step).
    """
    k, v = prefill_kv(weights, prefix_tokens, rounding)
    tok, out, gaps = int(first_token), [], []
    for _ in range(steps):
        logits, k1, v1 = causal_forward(weights, [tok], rounding, k, v)
        k = np.concatenate([k, k1], axis=1)
        v = np.concatenate([v, v1], axis=1)
        row = logits[0]
        top = np.sort(row)[-2:]
        gaps.append(float(top[1] - top[0]))
        tok = int(np.argmax(row))
        out.append(tok)
    return np.asarray(out, dtype=np.int64), np.asarray(gaps)


def commit_path(k, v, tree_k, tree_v, path):
    """Rollback after verification: the verified sequence's keys/values
    (tree nodes path[0..], root first) join the prefix cache, in path order."""
    path = list(path)
    return (np.concatenate([k, tree_k[:, path]], axis=1),
            np.concatenate([v, tree_v[:, path]], axis=1))


def speculative_decode(weights, prefix_tokens, first_token, steps, draft, rounding=True,
                       commit=commit_path):
    """Generate-and-verify loop over draft token trees.

    draft(root_token, produced) returns (tree_tokens, parent) for the next
    tree, tree_tokens[0] == root_token; produced is the list of tokens
    generated so far.  Each iteration appends the accepted draft tokens and
    the target's token after them.  Returns (the first `steps` generated
    tokens, per-iteration records with path, accept_len and rectified, the
    final cache (k, v) [L, S, H, Dh], every generated token).
    """
    k, v = prefill_kv(weights, prefix_tokens, rounding)
    root, out, log = int(first_token), [], []
    while len(out) < steps:
        tree_tokens, parent = draft(root, list(out))
        tree_tokens = np.asarray(tree_tokens, dtype=np.int64)
        assert int(tree_tokens[0]) == root
        logits, tk, tv = tree_forward(weights, k, v, tree_tokens, parent, rounding)
        amax = np.argmax(logits, axis=1)
        path, nxt, rectified = accept_walk(parent, tree_tokens, amax)
        k, v = commit(k, v, tk, tv, path)
        out += [int(tree_tokens[i]) for i in path[1:]] + [int(nxt)]
        log.append({"accept_len": len(path) - 1, "rectified": bool(rectified), "path": list(path)})
        root = int(nxt)
    return np.asarray(out[:steps], dtype=np.int64), log, (k, v), out
