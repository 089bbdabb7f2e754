"""Self-adaptive fallback (§3.3): when the draft stops and the target verifies.

TEST INFRASTRUCTURE ONLY (see the package docstring).

- Tree-cumulative confidence: T_c is the largest cumulative confidence over
  the tree's branches (a branch ends at a pending candidate; its cumulative
  confidence is the product of its tokens' probabilities).  After every draft
  step the draft falls back to verification when T_c < alpha.
- Self-adaptive threshold, Eq. 3: after a verification with N_correct of the
  N_all draft tokens of the most matching branch correct, alpha halves when
  all are correct and is otherwise divided by T_c ** ((N_all - N_correct) / N_all).
  The default initial alpha is 0.01.
- Most matching branch: the root-to-leaf branch that agrees with the target
  longest, i.e. one through the last accepted node; among several, the
  deepest (the first leaf in node order among equally deep ones).
"""

DEFAULT_ALPHA = 0.01


def tree_confidence(branch_confidences):
    """T_c = max_i C_i over the tree's branches."""
    return max(branch_confidences)


def update_alpha(alpha, n_correct, n_all, t_c):
    """Eq. 3."""
    if n_all <= 0:
        return alpha
    if n_correct == n_all:
        return alpha * 0.5
    return alpha / t_c ** ((n_all - n_correct) / n_all)


def most_matching_branch(parent, path):
    """(N_all, N_correct) for a verified tree: path = the accepted nodes from
    the root (path[0] = root); N_correct = len(path) - 1 accepted draft
    tokens; N_all = draft tokens on the deepest root-to-leaf branch through
    the last accepted node."""
    n = len(parent)
    depth = [0] * n
    for i in range(1, n):
        depth[i] = depth[parent[i]] + 1
    last = path[-1]
    below = [False] * n
    below[last] = True
    for i in range(last + 1, n):  # parents precede their children
        below[i] = below[parent[i]]
    n_all = max(depth[i] for i in range(n) if below[i])
    return n_all, len(path) - 1
