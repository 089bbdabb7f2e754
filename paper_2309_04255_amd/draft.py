"""Draft-side token-tree generation on the GPU (§3.1, §3.2 "Token tree generation").

A draft model (any model the library runs, in its own Session, its cache
holding the accepted prefix) grows a token tree rooted at the last accepted
token:
- tree decoder: each iteration feeds one node through llmcad_extend_tree
  (the new node's forward against the prefix and its own branch, the earlier
  nodes' keys/values read from the cache), and its logits row comes back;
- candidates: the most likely successor of the fed node always extends its
  branch, and every other token with probability above `threshold` (30% in
  the paper) starts a branch;
- branch pacer (Eq. 1, max-min fairness): with M the iteration budget and a
  candidate's branch holding T tokens of cumulative confidence C (product of
  their probabilities), the candidate with the largest M C / sum(C) - T is fed
  next (the earliest created among equal ones).

Self-adaptive fallback (§3.3): with a threshold alpha, growth stops after
the first step whose tree-cumulative confidence T_c (the largest cumulative
confidence of a pending candidate) is below alpha, and the target verifies;
`Fallback` updates alpha after each verification (Eq. 3).

Each step is one llmcad_extend_tree_candidates call: the library returns the
fed node's candidates -- its most likely token and every token whose
probability exceeds the threshold, with their probabilities (the softmax of
the node's logits, computed on the GPU in the same launch) -- so the host
reads back one small record per step, not the logits row.  Only when more
tokens exceed the threshold than a record holds (thresholds below 1/63) does
the driver read the row and take the float64 softmax itself.  The pacer's
choice is made on the host between steps (the next node depends on it).
Nodes are numbered in feeding order; the returned tree lists the fed nodes,
then the candidates not yet fed as leaves.
"""

import numpy as np


class _Tree:
    def __init__(self, root):
        self.tok = [int(root)]
        self.par = [-1]
        self.cum = [1.0]    # cumulative confidence of the node's branch
        self.depth = [0]    # draft tokens of the node's branch
        self.cand = []      # [token, fed parent, probability] in creation order

    def size(self):
        return len(self.tok) + len(self.cand)

    def add_candidates(self, node, toks, probs, max_nodes):
        # toks/probs: the most likely token (lowest index among equal maxima),
        # then every other token above the threshold, most likely first (ties:
        # lower index); added while the tree has fewer than max_nodes nodes
        for i, (t, pr) in enumerate(zip(toks, probs)):
            if i > 0 and self.size() >= max_nodes:
                break
            self.cand.append([int(t), node, float(pr)])

    def pick(self, budget):
        conf = np.array([self.cum[q] * p for _, q, p in self.cand])
        length = np.array([self.depth[q] + 1 for _, q, _ in self.cand])
        deficit = budget * conf / conf.sum() - length
        return int(np.argmax(deficit))

    def feed(self, k):
        t, q, p = self.cand.pop(k)
        self.tok.append(t)
        self.par.append(q)
        self.cum.append(self.cum[q] * p)
        self.depth.append(self.depth[q] + 1)
        return len(self.tok) - 1


def _probs(logits_row):
    z = logits_row.astype(np.float64)
    z = np.exp(z - z.max())
    return z / z.sum()


def candidates_from_row(logits_row, threshold):
    """(tokens, probabilities) of a logits row on the host: the argmax, then
    every other token whose float64 softmax probability exceeds the
    threshold, most likely first (ties: lower index)."""
    prob = _probs(logits_row)
    best = int(np.argmax(prob))
    over = np.flatnonzero(prob > threshold)
    over = over[over != best]
    over = over[np.argsort(-prob[over], kind="stable")]
    toks = [best] + [int(x) for x in over]
    return toks, [float(prob[t]) for t in toks]


def generate_tree(sess, prefix_len: int, root_token: int, iterations: int, threshold: float = 0.3,
                  alpha: float | None = None, max_nodes: int | None = None, keep_rows: bool = False):
    """Grow a draft tree with `iterations` fed nodes after the root (at most,
    when `alpha` is given: see the module docstring), on the draft model in
    `sess`.  Returns (tree_tokens, parent, info): the tree for
    verification (fed nodes, then the pending candidates), and info with the
    number of fed nodes, each fed node's probability, T_c after each step,
    every fed node's candidates (tokens, probabilities) and, with keep_rows,
    the fed nodes' logits rows ("fed", "conf", "t_c", "cands", "logits").

    The tree never exceeds max_nodes nodes (default: the session's max_n, the
    largest tree its verifier's workspace takes): candidates past the cap are
    not added (the most likely successor always is), and growth stops when a
    fed node's expansion would find no room.  Raises LlmcadPassError if a
    tree-decoder step failed on the device."""
    if max_nodes is None:
        max_nodes = getattr(sess, "max_n", 128)
    if max_nodes < 2:
        raise ValueError("a draft tree needs room for at least two nodes")
    tree = _Tree(root_token)
    rows, t_c, cands = [], [], []
    node = 0
    for it in range(iterations + 1):
        rec = sess.extend_candidates(prefix_len, np.asarray(tree.tok), np.asarray(tree.par), node, threshold)[0]
        if keep_rows or rec["count"] < 1:
            rows.append(sess.logits[0].float().cpu().numpy())
        if rec["count"] >= 1:
            toks, probs = rec["tok"], rec["prob"]
        else:  # (more tokens above the threshold than a record holds)
            toks, probs = candidates_from_row(rows[-1], threshold)
        cands.append((toks, probs))
        tree.add_candidates(node, toks, probs, max_nodes)
        t_c.append(max(tree.cum[q] * p for _, q, p in tree.cand))
        if it == iterations or (alpha is not None and t_c[-1] < alpha) or tree.size() >= max_nodes:
            break
        node = tree.feed(tree.pick(iterations))
    sess.check("tree-decoder step")
    tok = np.asarray(tree.tok + [c[0] for c in tree.cand], dtype=np.int32)
    par = np.asarray(tree.par + [c[1] for c in tree.cand], dtype=np.int32)
    conf = [1.0] + [tree.cum[i] / tree.cum[tree.par[i]] for i in range(1, len(tree.tok))]
    return tok, par, {"fed": len(tree.tok), "conf": conf, "t_c": t_c, "cands": cands,
                      "logits": np.stack(rows) if keep_rows else None}


class Fallback:
    """The self-adaptive threshold alpha of §3.3 (default 0.01)."""

    def __init__(self, alpha: float = 0.01):
        self.alpha = alpha

    def update(self, parent, path, t_c: float) -> float:
        """Eq. 3 after a verification of the tree `parent` that accepted the
        nodes `path` (root first).  The most matching branch is the deepest
        root-to-leaf branch through the last accepted node; its draft tokens
        are N_all, the accepted ones N_correct."""
        parent = np.asarray(parent)
        n = len(parent)
        depth = np.zeros(n, dtype=np.int64)
        under = np.zeros(n, dtype=bool)
        under[path[-1]] = True
        for i in range(1, n):
            depth[i] = depth[parent[i]] + 1
            under[i] |= under[parent[i]]
        n_all = int(depth[under].max())
        n_correct = len(path) - 1
        if n_all > 0:
            if n_correct == n_all:
                self.alpha *= 0.5
            else:
                self.alpha /= t_c ** ((n_all - n_correct) / n_all)
        return self.alpha
