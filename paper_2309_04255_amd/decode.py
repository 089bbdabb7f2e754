"""Greedy generate-and-verify loop over draft token trees (§3.1, §3.2).

Host control only: every step of a verification pass and of the rollback runs
in libllmcad's kernels (llmcad_verify_tree, llmcad_commit_path).  Each
iteration verifies the draft tree rooted at the last accepted token, rolls the
cache back to the verified sequence, and continues from the target's token
after it; the draft trees come from the caller (the draft model is not part of
this library).
"""

import numpy as np


def speculative_decode(sess, prefix_len: int, first_token: int, steps: int, draft):
    """Generate `steps` tokens after first_token with the target in `sess`
    (a binding.Session whose cache holds the accepted prefix [0, prefix_len)).

    draft(root_token, produced) returns (tree_tokens, parent), tree_tokens[0]
    == root_token.  Returns (the first `steps` generated tokens, one record
    per iteration with path and accept_len, the final prefix length).
    """
    root, out, log = int(first_token), [], []
    while len(out) < steps:
        tree_tokens, parent = draft(root, list(out))
        tree_tokens = np.asarray(tree_tokens, dtype=np.int32)
        if int(tree_tokens[0]) != root:
            raise ValueError("the draft tree's root must be the last accepted token")
        n = sess.verify_tree(prefix_len, tree_tokens, parent, want_logits=False)
        sess.commit(prefix_len, n)
        path, acc, nxt = sess.outcome()  # (synchronises: the next tree depends on it)
        out += [int(tree_tokens[i]) for i in path[1:]] + [nxt]
        log.append({"accept_len": acc, "path": path, "prefix_len": prefix_len})
        prefix_len += acc + 1
        root = nxt
    return np.asarray(out[:steps], dtype=np.int64), log, prefix_len


def draft_decode(target, drafter, prefix_len: int, first_token: int, steps: int, iterations: int = 8,
                 threshold: float = 0.3, fallback=None):
    """The generate-and-verify loop with a draft model (§3.1, §3.2, §3.3).

    `target` and `drafter` are Sessions whose caches hold the same prefix of
    length prefix_len.  Each iteration the drafter grows a tree from the
    current token (draft.generate_tree, stopped by the fallback threshold
    alpha or at `iterations` fed nodes), the target verifies it and rolls its
    cache back to the verified sequence, the drafter's cache is rolled back
    with the same accepted path, and alpha is updated (Eq. 3).  An accepted
    node that the drafter never fed (a pending candidate, always the last
    one of the path) gets its keys/values from one tree-decoder step.
    Returns (tokens, per-iteration log, final prefix length)."""
    import numpy as np

    from . import binding, draft

    fb = fallback if fallback is not None else draft.Fallback()
    out, log, root = [], [], int(first_token)
    while len(out) < steps:
        alpha = fb.alpha
        tok, par, info = draft.generate_tree(drafter, prefix_len, root, iterations, threshold, alpha=alpha)
        n = len(tok)
        target.verify_tree(prefix_len, tok, par, want_logits=False)
        target.commit(prefix_len, n)
        binding.commit_path(drafter.cfg, drafter.k_cache, drafter.v_cache, prefix_len, target.path,
                            target.accept_len, n)
        path, acc, nxt = target.outcome()  # (synchronises: the next tree depends on it)
        if path[-1] >= info["fed"]:
            chain = np.asarray([tok[i] for i in path])
            drafter.extend(prefix_len, chain, np.arange(-1, acc), acc)
            drafter.check("tree-decoder step")
        fb.update(par, path, info["t_c"][-1])
        out += [int(tok[i]) for i in path[1:]] + [nxt]
        log.append({"accept_len": acc, "nodes": n, "fed": info["fed"], "alpha": alpha,
                    "t_c": info["t_c"][-1], "prefix_len": prefix_len})
        prefix_len += acc + 1
        root = nxt
    return out[:steps], log, prefix_len
