"""GPU draft-side tree generation (paper_2309_04255_amd.draft) against the
oracle's generator (§3.1 branch threshold, §3.2 tree decoder and branch
pacer, Eq. 1).

Per case:
1. forward: the logits row the GPU returned for every fed node matches the
   oracle's one-pass masked forward over the fed nodes;
2. candidates: each fed node's record from the library (its argmax and every
   token above the threshold, with fp32 softmax probabilities computed in the
   same launch) is the float64 softmax of the GPU's own row: the same argmax,
   the same tokens above the threshold (tokens within 1e-5 of it may fall
   either way), probabilities within 1e-5 relative, most likely first;
3. policy: the oracle's generator, handed the GPU's candidate probabilities
   (as a row whose softmax gives them back: their logarithms, the remaining
   mass spread evenly over the other tokens), builds the GPU's tree exactly
   (same probabilities in, integer decisions out).

The draft model is a small random LLaMA-shaped decoder whose weight scale
(std 0.3) gives next-token distributions like a trained draft's (top-1
probabilities between about 0.3 and 0.9), so that the paper's 30% threshold
branches.  Its activations are large, and bf16 rounding alone moves its
logits far more than the target models': the forward bar is twice the spread
between the oracle with and without its bf16 rounding points.  For the same
reason a tree built from the oracle's own rows may part from the GPU's at a
near tie; 1 and 2 together pin the generator.
"""

import numpy as np
import pytest
import torch

import oracle
import workloads
from tests.util import oracle_weights

pytestmark = pytest.mark.gpu

DRAFT = workloads.ModelShape("draft_tiny", 2, 256, 4, 64, 688, 1024, weight_std=0.3, seed=0x5EEDD001)
P = 24
# threshold, prefix seed, iterations, fallback threshold alpha (§3.3) or None
CASES = [(0.3, 51, 12, None), (0.15, 40, 12, None), (0.15, 45, 16, None), (0.15, 45, 16, 0.03)]


@pytest.fixture(scope="module")
def draft_model():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2309_04255_amd import binding

    sess = binding.Session(DRAFT, capacity=P + 64, max_n=128)
    binding.workspace_init(sess.cfg, 128, sess.workspace)
    sess.load_weights(workloads.make_weights(DRAFT, "cuda"))
    return sess, oracle_weights(DRAFT)


def _softmax(rows):
    z = np.asarray(rows, dtype=np.float64)
    z = np.exp(z - z.max(axis=-1, keepdims=True))
    return z / z.sum(axis=-1, keepdims=True)


@pytest.mark.parametrize("threshold,seed,iterations,alpha", CASES)
def test_draft_tree_matches_oracle(draft_model, threshold, seed, iterations, alpha):
    from paper_2309_04255_amd import draft

    sess, ow = draft_model
    prefix = workloads.draw_tokens(P, DRAFT.vocab, seed=seed)
    root = int(workloads.draw_tokens(1, DRAFT.vocab, seed=seed, stream=9)[0])
    what = f"thr={threshold} seed={seed} it={iterations} alpha={alpha}"
    print(f"\n[draft] {what}", flush=True)
    sess.prefill(prefix, 0)
    tok, par, info = draft.generate_tree(sess, P, root, iterations, threshold, alpha=alpha, keep_rows=True)
    fed = info["fed"]
    assert len(tok) > fed
    if alpha is None:
        assert fed == iterations + 1
    else:  # stopped by the fallback before the cap
        assert fed < iterations + 1 and info["t_c"][-1] < alpha <= min(info["t_c"][:-1])
    assert np.any(np.bincount(par[1:], minlength=len(par)) >= 2), "no branching"
    gpu_rows = info["logits"]

    # 1. forward parity over the fed nodes, against the model's own rounding spread
    pk, pv = oracle.prefill_kv(ow, prefix, rounding=True)
    ref, _, _ = oracle.tree_forward(ow, pk, pv, tok[:fed], par[:fed], rounding=True)
    xk, xv = oracle.prefill_kv(ow, prefix, rounding=False)
    exact, _, _ = oracle.tree_forward(ow, xk, xv, tok[:fed], par[:fed], rounding=False)
    spread = np.abs(ref - exact).max()
    spread_rel = np.linalg.norm(ref - exact) / np.linalg.norm(ref)
    err = np.abs(gpu_rows - ref).max()
    rel = np.linalg.norm(gpu_rows - ref) / np.linalg.norm(ref)
    print(f"[draft] {what}: {len(tok)} nodes, logits max_abs={err:.2e} rel={rel:.2e} "
          f"(rounding spread {spread:.2e} / {spread_rel:.2e})", flush=True)
    assert err <= 2 * spread and rel <= 2 * spread_rel, (what, err, spread, rel, spread_rel)

    # 2. the library's candidates are the float64 softmax of the GPU's rows
    for q in range(fed):
        toks, probs = info["cands"][q]
        p64 = _softmax(gpu_rows[q])
        assert toks[0] == int(np.argmax(gpu_rows[q])), (what, q)
        np.testing.assert_allclose(probs, p64[toks], rtol=1e-5)
        assert all(a >= b for a, b in zip(probs, probs[1:])), (what, q, probs)
        near = np.abs(p64 - threshold) <= 1e-5 * threshold
        want = set(np.flatnonzero((p64 > threshold) & ~near).tolist()) - {toks[0]}
        got = set(toks[1:])
        assert want <= got and got <= want | set(np.flatnonzero(near).tolist()), (what, q, want, got)

    # 3. the oracle's policy on the GPU's candidate probabilities builds the GPU's tree
    def replay(tokens, parent):
        np.testing.assert_array_equal(tokens, tok[:len(tokens)])
        np.testing.assert_array_equal(parent, par[:len(parent)])
        toks, probs = info["cands"][len(tokens) - 1]
        rest = (1.0 - sum(probs)) / (DRAFT.vocab - len(toks))
        row = np.full(DRAFT.vocab, np.log(max(rest, 1e-300)))
        row[toks] = np.log(probs)
        return row

    otok, opar, oinfo = oracle.generate_tree(None, None, None, root, iterations, threshold, forward=replay,
                                             alpha=alpha)
    np.testing.assert_array_equal(otok, tok)
    np.testing.assert_array_equal(opar, par)
    np.testing.assert_allclose(oinfo["conf"], info["conf"], rtol=1e-12)
