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
        acc = int(sess.accept_len.item())  # (synchronises: the next tree depends on it)
        path = [int(x) for x in sess.path[: acc + 1].cpu()]
        nxt = int(sess.next_token.item())
        out += [int(tree_tokens[i]) for i in path[1:]] + [nxt]
        log.append({"accept_len": acc, "path": path, "prefix_len": prefix_len})
        prefix_len += acc + 1
        root = nxt
    return np.asarray(out[:steps], dtype=np.int64), log, prefix_len
