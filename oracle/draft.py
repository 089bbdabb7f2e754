"""Draft-side token-tree generation: the tree decoder and the branch pacer.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The draft model grows a token tree rooted at the last accepted token (§3.1
"Simplified workflow"; §3.2 "Token tree generation"):
- Tree decoder: one node is fed per iteration; it attends to the prefix and to
  its own branch only (the masking table), so branches do not affect each
  other.  Feeding node x gives the draft's distribution over x's successor.
- Candidates: the most likely successor always extends x's branch; every
  other token whose probability exceeds the threshold (30% in the paper)
  starts a branch of its own.  A candidate is a draft token with a known
  value; it becomes a fed node when its branch is chosen to grow.
- Branch pacer (Eq. 1): with M the number of iterations of the whole tree,
  branch x (ending at candidate x) holding T_x draft tokens with cumulative
  confidence C_x (the product of its tokens' probabilities), its deficit is
  f(x) = M C_x / sum_i C_i - T_x.  Under max-min fairness the branch with the
  largest deficit grows next (ties: the candidate created first).

Node numbering is the feeding order (a node is fed after its parent).  The
tree handed to the target holds the fed nodes and, after them, the pending
candidates as leaves.  Each iteration's forward is `tree_forward` over the
fed nodes (the last row is the new node's), which is the pinned one-pass form.
"""

import numpy as np

from .model import tree_forward


def _softmax64(row):
    z = np.asarray(row, dtype=np.float64)
    e = np.exp(z - z.max())
    return e / e.sum()


def generate_tree(weights, prefix_k, prefix_v, root_token, iterations, threshold=0.3, rounding=True,
                  forward=None, alpha=None, max_nodes=128):
    """Grow a draft tree with `iterations` fed nodes after the root.

    prefix_k/prefix_v: the draft model's prefix keys/values [L, P, H, Dh].
    forward(tokens, parent) -> the draft's logits row of the last node, by
    default the last row of tree_forward.  Returns (tree_tokens, parent, info)
    where info holds the number of fed nodes, each fed node's probability, the
    pending candidates and, per iteration, the pacer's margin (largest deficit
    minus the runner-up).

    alpha: the self-adaptive fallback threshold (§3.3); when given, growth
    stops after the first draft step whose tree-cumulative confidence T_c
    (the largest cumulative confidence of a pending candidate) is below it,
    and `iterations` is only the cap (the pacer's M).  info["t_c"] lists T_c
    after each step (the root's expansion first).

    max_nodes: the largest tree the verifier takes (the paper sets no size;
    this is a resource cap).  A candidate is added only while the tree (fed
    nodes plus pending candidates) holds fewer nodes, except the fed node's
    most likely successor, which always is; growth stops once the tree holds
    max_nodes nodes, since the next expansion would find no room.
    """
    if forward is None:
        def forward(tokens, parent):
            logits, _, _ = tree_forward(weights, prefix_k, prefix_v, tokens, parent, rounding)
            return logits[-1]

    tokens, parent, conf = [int(root_token)], [-1], [1.0]   # fed nodes
    pending = []  # candidates: (token, fed parent, probability, cumulative confidence, depth)

    def expand(node):
        prob = _softmax64(forward(np.asarray(tokens), np.asarray(parent)))
        order = np.argsort(-prob, kind="stable")  # most likely first, lowest index among ties
        best = int(order[0])
        cum = float(np.prod([conf[i] for i in _branch(parent, node)]))
        depth = len(_branch(parent, node)) + 1  # draft tokens of the candidate's branch
        pending.append((best, node, float(prob[best]), cum * float(prob[best]), depth))
        for t in order[1:]:
            if prob[t] <= threshold or len(tokens) + len(pending) >= max_nodes:
                break
            pending.append((int(t), node, float(prob[t]), cum * float(prob[t]), depth))

    def fall_back():
        t_cs.append(max(c for _, _, _, c, _ in pending))
        return alpha is not None and t_cs[-1] < alpha

    t_cs = []
    expand(0)
    stop = fall_back()
    M = iterations
    gaps = []  # per iteration: largest deficit minus the runner-up (inf with one candidate)
    for _ in range(iterations):
        if stop or len(tokens) + len(pending) >= max_nodes:
            break
        total = sum(c for _, _, _, c, _ in pending)
        deficits = [M * c / total - d for _, _, _, c, d in pending]
        k = int(np.argmax(deficits))  # first maximum: the earliest candidate
        rest = deficits[:k] + deficits[k + 1:]
        gaps.append(deficits[k] - max(rest) if rest else np.inf)
        tok, par, p, _, _ = pending.pop(k)
        tokens.append(tok)
        parent.append(par)
        conf.append(p)
        expand(len(tokens) - 1)
        stop = fall_back()
    # the tree for verification: the fed nodes, then the pending candidates as leaves
    all_tokens = tokens + [t for t, _, _, _, _ in pending]
    all_parent = parent + [q for _, q, _, _, _ in pending]
    info = {"fed": len(tokens), "conf": conf, "pending": [(t, q, p) for t, q, p, _, _ in pending],
            "deficit_gaps": gaps, "t_c": t_cs}
    return np.asarray(all_tokens, dtype=np.int64), np.asarray(all_parent, dtype=np.int64), info


def _branch(parent, node):
    """Draft nodes of node's branch (root excluded), root side first."""
    out = []
    while node > 0:
        out.append(node)
        node = int(parent[node])
    return out[::-1]
