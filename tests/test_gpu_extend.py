"""GPU tree-decoder steps (llmcad_extend_tree) against the oracle (§3.2 tree decoder).

A tree grown in chunks, or one node per call as a draft model grows it, must
give every node the logits and the cache K/V of the one-pass masked forward
over the whole tree (the oracle's tree_forward, itself pinned by brute force
to the causal forward of every branch): each step reads the earlier nodes'
keys/values from their cache slots.  Same models and prefix as the
verification tests.
"""

import types

import numpy as np
import pytest
import torch

import oracle
import workloads
from tests import parity
from tests.util import oracle_weights

pytestmark = pytest.mark.gpu

P = 100
SHAPES = {
    "tiny": workloads.MODELS["tiny"],
    "small128": workloads.ModelShape("small128", 2, 512, 4, 128, 1000, 1998, seed=0x5EED0128),
}


@pytest.fixture(scope="module", params=sorted(SHAPES))
def model(request):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2309_04255_amd import binding

    shape = SHAPES[request.param]
    print(f"\n[model] {shape.name}", flush=True)
    sess = binding.Session(shape, capacity=P + 200, max_n=128)
    binding.workspace_init(sess.cfg, 128, sess.workspace)
    sess.load_weights(workloads.make_weights(shape, "cuda", gain_jitter=0.1))
    ow = oracle_weights(shape, gain_jitter=0.1)
    prefix = workloads.draw_tokens(P, shape.vocab, seed=3)
    ok, ov = oracle.prefill_kv(ow, prefix, rounding=True)
    sess.prefill(prefix, 0)
    torch.cuda.synchronize()
    return types.SimpleNamespace(shape=shape, sess=sess, ow=ow, ok=ok, ov=ov)


def _grow(m, parent, tok, cuts):
    """Extend the tree through node counts cuts[0] < cuts[1] < ... = n; returns all logits rows."""
    rows, first = [], 0
    for upto in cuts:
        lg = m.sess.extend(P, tok[:upto], parent[:upto], first)
        rows.append(lg.float().cpu().numpy())
        first = upto
    return np.concatenate(rows, axis=0)


@pytest.mark.parametrize("tree,cuts", [
    ("binary_d3_n15", "chunks"),
    ("binary_d3_n15", "one"),
    ("random_n40", "chunks"),
    ("chain_n9", "one"),
])
def test_grown_tree_matches_one_pass(model, tree, cuts):
    m = model
    parent = {"binary_d3_n15": workloads.complete_tree((2, 2, 2)),
              "random_n40": workloads.random_tree(40, 7, 8),
              "chain_n9": workloads.chain_tree(9)}[tree]
    n = len(parent)
    tok = workloads.draw_tokens(n, m.shape.vocab, seed=31, stream=n)
    steps = list(range(1, n + 1)) if cuts == "one" else sorted({max(1, n // 3), (2 * n) // 3, n})
    logits = _grow(m, parent, tok, steps)
    ref, rk, rv = oracle.tree_forward(m.ow, m.ok, m.ov, tok, parent, rounding=True)
    what = f"{m.shape.name}/{tree}/{cuts}"
    err, rel = parity.check_logits(logits, ref, what)
    parity.check_argmax(np.argmax(logits, axis=1), ref, what)
    gk = m.sess.k_cache[:, :, P:P + n].float().cpu().numpy().transpose(0, 2, 1, 3)
    gv = m.sess.v_rows[:, :, P:P + n].float().cpu().numpy().transpose(0, 2, 1, 3)
    for g, r in ((gk, rk), (gv, rv)):
        assert np.abs(g - r).max() <= 2e-2 * np.abs(r).max()
    print(f"[{what}] {len(steps)} steps, max_abs={err:.2e} rel={rel:.2e}", flush=True)


def test_extend_from_zero_is_the_verification_forward(model):
    # first = 0 computes the whole tree: the verification pass's logits, bit for bit
    m = model
    parent = workloads.complete_tree((4, 3, 2))
    n = len(parent)
    tok = workloads.draw_tokens(n, m.shape.vocab, seed=5, stream=7)
    ext = m.sess.extend(P, tok, parent, 0).float().cpu().numpy()
    m.sess.verify_tree(P, tok, parent)
    ver = m.sess.logits[:n].float().cpu().numpy()
    np.testing.assert_array_equal(ext, ver)


def _softmax64(row):
    z = np.asarray(row, dtype=np.float64)
    z = np.exp(z - z.max())
    return z / z.sum()


@pytest.mark.parametrize("first,threshold", [(0, 0.01), (5, 0.002), (0, 0.3)])
def test_candidate_records_every_row(model, first, threshold):
    # llmcad_extend_tree_candidates over several rows at once (a binary tree of
    # 15 nodes, all of it or its nodes 5..14): each row's record is the float64
    # softmax of the logits row the same call stored -- the argmax first, then
    # every other token above the threshold (tokens within 1e-5 relative of it
    # may fall either way), higher probability first, probabilities within
    # 1e-5 relative -- and the row's max and normaliser.  The logits equal the
    # plain tree-decoder step's bit for bit.
    from paper_2309_04255_amd import binding

    parent = workloads.complete_tree((2, 2, 2))
    tok = workloads.draw_tokens(len(parent), model.shape.vocab, seed=77, stream=3)
    n = len(parent)
    plain = model.sess.extend(P, tok, parent, first).float().cpu().numpy()
    recs = model.sess.extend_candidates(P, tok, parent, first, threshold)
    rows = model.sess.logits[:n - first].float().cpu().numpy()
    np.testing.assert_array_equal(rows, plain)
    assert len(recs) == n - first
    for r, rec in enumerate(recs):
        p64 = _softmax64(rows[r])
        assert rec["argmax"] == int(np.argmax(rows[r]))
        assert rec["max_logit"] == float(rows[r].max())
        np.testing.assert_allclose(rec["sum_exp"], np.exp(rows[r].astype(np.float64) - rows[r].max()).sum(),
                                   rtol=1e-5)
        assert 1 <= rec["count"] <= binding.CAND_MAX, rec["count"]
        toks, probs = rec["tok"], rec["prob"]
        assert toks[0] == rec["argmax"]
        np.testing.assert_allclose(probs, p64[toks], rtol=1e-5)
        assert all(a > b or (a == b and s < t) for a, b, s, t in zip(probs, probs[1:], toks, toks[1:]))
        near = np.abs(p64 - threshold) <= 1e-5 * threshold
        want = set(np.flatnonzero((p64 > threshold) & ~near).tolist()) - {toks[0]}
        assert want <= set(toks[1:]) <= want | set(np.flatnonzero(near).tolist()), (r, want, toks)


def test_candidate_records_overflow(model):
    # A threshold below 1/64 on these near-uniform rows puts far more than 63
    # tokens above it: every record says so (count -1) and still carries the
    # argmax, the max and the normaliser, so a driver can fall back to the row.
    parent = workloads.complete_tree((2, 2))
    tok = workloads.draw_tokens(len(parent), model.shape.vocab, seed=78, stream=3)
    recs = model.sess.extend_candidates(P, tok, parent, 0, 1e-4)
    rows = model.sess.logits[:len(parent)].float().cpu().numpy()
    for r, rec in enumerate(recs):
        assert np.count_nonzero(_softmax64(rows[r]) > 1e-4) > 64
        assert rec["count"] == -1 and rec["tok"] == [] and rec["prob"] == []
        assert rec["argmax"] == int(np.argmax(rows[r]))
        assert rec["max_logit"] == float(rows[r].max())
