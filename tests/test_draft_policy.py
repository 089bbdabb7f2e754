"""The GPU draft driver's host policy (branch threshold, §3.1; branch pacer,
§3.2 Eq. 1) against the oracle's generator, on the CPU: a stand-in session
serves logits rows from a table -- and, for the candidates entry point, the
record the library builds from such a row (the argmax and every token above
the threshold, by probability) -- so both sides see the same probabilities
and must make the same integer decisions (which candidates, in which order,
which branch grows)."""

import numpy as np
import pytest
import torch

import oracle
from paper_2309_04255_amd import draft


CAND_MAX = 64  # entries of one candidate record (llmcad_candidates)


class TableSession:
    """Answers a tree-decoder step for the node `first` with the row
    forward(tokens, parent): as logits (extend), or as the candidate record
    of that row (extend_candidates; float64 softmax, the argmax first, then
    the tokens above the threshold by probability, ties to the lower token;
    count -1 when more than CAND_MAX - 1 exceed it)."""

    def __init__(self, forward):
        self.forward = forward
        self.calls = 0
        self.logits = None

    def extend(self, prefix_len, tree_tokens, parent, first):
        assert first == len(tree_tokens) - 1  # one new node per step
        self.calls += 1
        row = self.forward(np.asarray(tree_tokens), np.asarray(parent))
        self.logits = torch.from_numpy(np.asarray(row, dtype=np.float32)[None, :])
        return self.logits

    def extend_candidates(self, prefix_len, tree_tokens, parent, first, threshold):
        row = self.extend(prefix_len, tree_tokens, parent, first)[0].numpy().astype(np.float64)
        e = np.exp(row - row.max())
        prob = e / e.sum()
        best = int(np.flatnonzero(row == row.max())[0])
        others = sorted((v for v in range(len(row)) if prob[v] > threshold and v != best),
                        key=lambda v: (-prob[v], v))
        toks = [best] + others
        if len(toks) > CAND_MAX:
            return [{"count": -1, "argmax": best, "tok": [], "prob": []}]
        return [{"count": len(toks), "argmax": best, "tok": toks, "prob": [float(prob[v]) for v in toks]}]

    def check(self, what=""):
        pass  # (no device: nothing can fail)


def _random_forward(vocab, seed, peak):
    """Successor logits keyed by the fed token's branch: a few large logits so
    that several tokens land near the threshold, plus exact ties."""

    def forward(tokens, parent):
        key = hash((seed, tuple(int(t) for t in tokens), tuple(int(q) for q in parent))) & 0xFFFFFFFF
        g = np.random.default_rng(key)
        row = g.normal(0, 1, vocab)
        hot = g.choice(vocab, 4, replace=False)
        row[hot] += peak * g.random(4)
        row[hot[1]] = row[hot[2]]  # an exact tie among the likely tokens
        return row.astype(np.float32)

    return forward


def test_hand_worked_example():
    table = {0: {1: .60, 2: .35}, 1: {3: .50, 4: .45}, 2: {5: .90}}

    def forward(tokens, parent):
        p = dict(table.get(int(tokens[-1]), {6: .95}))
        rest = (1.0 - sum(p.values())) / (8 - len(p))
        return np.log(np.array([p.get(t, rest) for t in range(8)]))

    tok, par, info = draft.generate_tree(TableSession(forward), 0, 0, 3, threshold=0.3)
    assert tok.tolist() == [0, 1, 2, 5, 3, 4, 6]
    assert par.tolist() == [-1, 0, 0, 2, 1, 1, 3]
    assert info["fed"] == 4


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("threshold", [0.3, 0.1, 0.02])
def test_matches_oracle_generator(seed, threshold):
    forward = _random_forward(64, seed, peak=9.0)
    sess = TableSession(forward)
    tok, par, info = draft.generate_tree(sess, 0, 5, 10, threshold=threshold)
    otok, opar, oinfo = oracle.generate_tree(None, None, None, 5, 10, threshold=threshold,
                                             forward=lambda t, p: forward(t, p).astype(np.float64))
    np.testing.assert_array_equal(tok, otok)
    np.testing.assert_array_equal(par, opar)
    np.testing.assert_allclose(info["conf"], oinfo["conf"], rtol=1e-12)
    assert sess.calls == 11


@pytest.mark.parametrize("seed", range(4))
@pytest.mark.parametrize("alpha", [0.5, 0.05, 0.005])
def test_fallback_stop_matches_oracle(seed, alpha):
    forward = _random_forward(64, seed, peak=6.0)
    tok, par, info = draft.generate_tree(TableSession(forward), 0, 5, 12, threshold=0.1, alpha=alpha)
    otok, opar, oinfo = oracle.generate_tree(None, None, None, 5, 12, threshold=0.1, alpha=alpha,
                                             forward=lambda t, p: forward(t, p).astype(np.float64))
    np.testing.assert_array_equal(tok, otok)
    np.testing.assert_array_equal(par, opar)
    np.testing.assert_allclose(info["t_c"], oinfo["t_c"], rtol=1e-12)


def test_fallback_update_matches_oracle():
    rng = np.random.default_rng(7)
    fb, alpha = draft.Fallback(), oracle.DEFAULT_ALPHA
    assert fb.alpha == alpha
    for _ in range(200):
        n = int(rng.integers(2, 20))
        parent = [-1] + [int(rng.integers(0, i)) for i in range(1, n)]
        path = [0]
        while True:  # an accepted path: a random descent that may stop anywhere
            kids = [i for i in range(n) if parent[i] == path[-1]]
            if not kids or rng.random() < 0.3:
                break
            path.append(int(rng.choice(kids)))
        t_c = float(rng.uniform(0.01, 1.0))
        n_all, n_correct = oracle.most_matching_branch(parent, path)
        alpha = oracle.update_alpha(alpha, n_correct, n_all, t_c)
        assert fb.update(parent, path, t_c) == pytest.approx(alpha, rel=1e-12)


@pytest.mark.parametrize("max_nodes", [128, 50, 2])
def test_flat_wide_rows_stay_within_the_verifier_cap(max_nodes):
    # Flat but wide successor rows: 40 tokens share ~97% of the mass, so with
    # a 2% threshold every expansion offers ~40 candidates and 6 iterations
    # would build a tree of ~240 nodes.  Both the driver and the oracle stop
    # at max_nodes, make the same decisions, and the result fits the verifier.
    vocab = 64

    def forward(tokens, parent):
        key = hash(("wide", tuple(int(t) for t in tokens), tuple(int(q) for q in parent))) & 0xFFFFFFFF
        g = np.random.default_rng(key)
        row = np.full(vocab, -8.0)
        row[g.choice(vocab, 40, replace=False)] = g.uniform(0.0, 0.2, 40)
        return row.astype(np.float32)

    sess = TableSession(forward)
    tok, par, info = draft.generate_tree(sess, 0, 5, 6, threshold=0.02, max_nodes=max_nodes)
    otok, opar, oinfo = oracle.generate_tree(None, None, None, 5, 6, threshold=0.02, max_nodes=max_nodes,
                                             forward=lambda t, p: forward(t, p).astype(np.float64))
    np.testing.assert_array_equal(tok, otok)
    np.testing.assert_array_equal(par, opar)
    assert len(tok) <= max_nodes
    assert len(tok) == max_nodes  # (these rows always fill the cap)
    assert info["fed"] == oinfo["fed"] >= 1
    # every fed node beyond the root got its most likely successor as a child
    for q in range(info["fed"]):
        assert q in set(int(x) for x in par[1:]), q


def test_record_overflow_reads_the_row():
    # More tokens above the threshold than a candidate record holds: the
    # driver takes the logits row and its own float64 softmax, and still makes
    # the oracle's decisions.
    vocab = 256

    def forward(tokens, parent):
        key = hash(("many", tuple(int(t) for t in tokens), tuple(int(q) for q in parent))) & 0xFFFFFFFF
        g = np.random.default_rng(key)
        row = np.full(vocab, -9.0)
        row[g.choice(vocab, 120, replace=False)] = g.uniform(0.0, 0.1, 120)
        return row.astype(np.float32)

    sess = TableSession(forward)
    tok, par, info = draft.generate_tree(sess, 0, 5, 2, threshold=0.005, max_nodes=128)
    otok, opar, oinfo = oracle.generate_tree(None, None, None, 5, 2, threshold=0.005, max_nodes=128,
                                             forward=lambda t, p: forward(t, p).astype(np.float64))
    assert len(info["cands"][0][0]) > CAND_MAX  # the fallback ran
    np.testing.assert_array_equal(tok, otok)
    np.testing.assert_array_equal(par, opar)
