"""GPU rollback and the generate-and-verify loop, through the C ABI (§3.1, §3.2).

llmcad_commit_path must move exactly the verified sequence's cache rows
(bit-exact copies of what the pass wrote), leave everything else alone, and
leave the cache holding the causal keys/values of the accepted sequence.  The
loop built on it (paper_2309_04255_amd.decode) must reproduce the oracle's
plain greedy decoding token for token wherever the oracle's top-2 logit gap
exceeds 1e-2; the seeds are chosen so that no step of the compared range is
closer than that.  The degenerate one-node tree is plain greedy decoding.
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

P = 40
SEED = 31
STEPS = 18
SHAPES = {
    "tiny": workloads.MODELS["tiny"],
    "small128": workloads.ModelShape("small128", 2, 512, 4, 128, 1000, 1998, seed=0x5EED0128),
}
BINARY = workloads.complete_tree((2, 2, 2))


@pytest.fixture(scope="module", params=sorted(SHAPES))
def model(request):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2309_04255_amd import binding, decode

    shape = SHAPES[request.param]
    print(f"\n[model] {shape.name}", flush=True)
    sess = binding.Session(shape, capacity=P + 200, max_n=128)
    binding.workspace_init(sess.cfg, 128, sess.workspace)
    sess.load_weights(workloads.make_weights(shape, "cuda", gain_jitter=0.1))
    ow = oracle_weights(shape, gain_jitter=0.1)
    prefix = workloads.draw_tokens(P, shape.vocab, seed=SEED)
    first = int(workloads.draw_tokens(1, shape.vocab, seed=SEED, stream=5)[0])
    greedy, gaps = oracle.greedy_decode(ow, prefix, first, STEPS + 8, rounding=True)
    return types.SimpleNamespace(shape=shape, sess=sess, ow=ow, prefix=prefix, first=first, greedy=greedy,
                                 gaps=gaps, binding=binding, decode=decode)


def _reset(m):
    m.sess.prefill(m.prefix, 0)
    torch.cuda.synchronize()


def _planted(m, parent, schedule, leaves):
    it = [0]

    def draft(root, produced):
        i = it[0]
        it[0] += 1
        return workloads.draft_tree(parent, root, m.greedy[len(produced):], schedule[i % len(schedule)],
                                    leaves[i % len(leaves)], m.shape.vocab, seed=100 + i), parent

    return draft


def _compare_with_greedy(m, out, what):
    """Exact wherever the oracle is confident; after a near-tie the sequences may part."""
    for t, tok in enumerate(out):
        if tok != m.greedy[t]:
            assert m.gaps[t] <= parity.GAP, f"{what}: token {t}: {tok} != {m.greedy[t]} (gap {m.gaps[t]:.3g})"
            return t
    return len(out)


def test_commit_moves_path_rows(model):
    m = model
    _reset(m)
    s = m.sess
    n = len(BINARY)
    tok = workloads.draft_tree(BINARY, m.first, m.greedy, 2, 14, m.shape.vocab, seed=7)
    s.verify_tree(P, tok, BINARY, want_logits=False)
    torch.cuda.synchronize()
    k0, v0 = s.k_cache[:, :, :P + n].clone(), s.v_rows[:, :, :P + n].clone()
    s.commit(P, n)
    torch.cuda.synchronize()
    acc = int(s.accept_len.item())
    path = [int(x) for x in s.path[: acc + 1].cpu()]
    # (the fixture's seed gives the first greedy steps top-2 gaps above 1e-2 on
    # both models, so the planted acceptance is always asserted)
    assert np.all(m.gaps[:2] > parity.GAP), m.gaps[:2]
    assert acc == 2 and path == [0, 2, 6], path  # planted along root -> 2 -> 6 -> 14
    for k in range(n):
        src = path[k] if k <= acc else k
        assert torch.equal(s.k_cache[:, :, P + k], k0[:, :, P + src]), k
        assert torch.equal(s.v_rows[:, :, P + k], v0[:, :, P + src]), k
    assert torch.equal(s.k_cache[:, :, :P], k0[:, :, :P])
    assert torch.equal(s.v_rows[:, :, :P], v0[:, :, :P])
    # the cache now holds the accepted sequence's causal keys/values
    seq = np.concatenate([m.prefix, [m.first], m.greedy[:acc]])
    rk, rv = oracle.prefill_kv(m.ow, seq, rounding=True)
    gk = s.k_cache[:, :, P:P + acc + 1].float().cpu().numpy().transpose(0, 2, 1, 3)
    gv = s.v_rows[:, :, P:P + acc + 1].float().cpu().numpy().transpose(0, 2, 1, 3)
    for g, r in ((gk, rk[:, P:]), (gv, rv[:, P:])):
        assert np.abs(g - r).max() <= 2e-2 * np.abs(r).max()


def test_loop_with_planted_drafts(model):
    m = model
    _reset(m)
    out, log, plen = m.decode.speculative_decode(m.sess, P, m.first, STEPS,
                                                 _planted(m, BINARY, [0, 1, 2, 3, 1, 3], [14, 7, 10]))
    matched = _compare_with_greedy(m, out, "planted")
    assert matched == STEPS, matched
    assert [r["accept_len"] for r in log[:4]] == [0, 1, 2, 3]
    assert plen == P + sum(r["accept_len"] + 1 for r in log)
    print(f"[{m.shape.name}] {len(log)} passes for {STEPS} tokens", flush=True)


def test_loop_with_random_drafts(model):
    m = model
    _reset(m)
    parent = workloads.random_tree(20, 7, 5)

    def draft(root, produced):
        tok = workloads.draw_tokens(len(parent), m.shape.vocab, seed=500 + len(produced), stream=3)
        tok[0] = root
        return tok, parent

    out, _, _ = m.decode.speculative_decode(m.sess, P, m.first, 6, draft)
    assert _compare_with_greedy(m, out, "random") == 6


def test_loop_with_one_node_trees_is_greedy_decoding(model):
    m = model
    _reset(m)
    out, log, _ = m.decode.speculative_decode(m.sess, P, m.first, 8,
                                              lambda root, produced: (np.array([root]), np.array([-1])))
    assert _compare_with_greedy(m, out, "one-node") == 8
    assert all(r["accept_len"] == 0 for r in log)


@pytest.mark.parametrize("drafter_kind,threshold,alpha", [("self", 0.3, 1e-4), ("self", 0.03, 1e-3),
                                                          ("other", 0.03, 0.01)])
def test_draft_model_loop_is_greedy(model, drafter_kind, threshold, alpha):
    # The full loop with a draft model (§3.1-§3.3): the drafter grows each tree
    # (threshold, branch pacer, fallback), the target verifies and both caches
    # roll back.  "self" drafts with the target's own weights (most drafts are
    # accepted, and the last accepted node is often a candidate the drafter
    # never fed); "other" with a different random model (almost nothing is
    # accepted).  Either way the output is the target's greedy decoding, and
    # the drafter's cache holds the accepted sequence's keys/values.
    m = model
    from paper_2309_04255_amd import draft

    shape = m.shape if drafter_kind == "self" else workloads.ModelShape(
        m.shape.name + "_draft", m.shape.n_layers, m.shape.d_model, m.shape.n_heads, m.shape.head_dim,
        m.shape.d_ffn, m.shape.vocab, seed=m.shape.seed ^ 0xD0)
    drafter = m.binding.Session(shape, capacity=P + 200, max_n=128)
    m.binding.workspace_init(drafter.cfg, 128, drafter.workspace)
    drafter.load_weights(workloads.make_weights(shape, "cuda", gain_jitter=0.1))
    _reset(m)
    drafter.prefill(m.prefix, 0)
    what = f"{m.shape.name}/draft-{drafter_kind}/thr={threshold}/alpha={alpha}"
    print(f"[{what}]", flush=True)
    out, log, plen = m.decode.draft_decode(m.sess, drafter, P, m.first, STEPS, iterations=6,
                                           threshold=threshold, fallback=draft.Fallback(alpha))
    agree = _compare_with_greedy(m, out, what)
    accs = [e["accept_len"] for e in log]
    print(f"[{what}] {len(log)} passes, accept lengths {accs}, nodes {[e['nodes'] for e in log]}, "
          f"agree {agree}/{len(out)}", flush=True)
    if drafter_kind == "self":
        assert sum(accs) >= len(accs), accs   # self-drafting accepts on average at least one token per pass
    # the drafter's cache rows [P, plen) hold the accepted sequence's keys/values, as the target's do
    for a, b in ((drafter.k_cache, m.sess.k_cache), (drafter.v_rows, m.sess.v_rows)):
        if drafter_kind == "self":
            ga = a[:, :, P:plen].float()
            gb = b[:, :, P:plen].float()
            assert (ga - gb).abs().max().item() <= 2e-2 * gb.abs().max().item()
