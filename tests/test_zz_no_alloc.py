"""llmcad_verify_tree_noalloc (the entry point for callers that cannot
allocate) against llmcad_verify_tree, through the C ABI: on the same inputs
both run the same kernels, so every output must be bit-identical -- logits,
per-node argmax path, accept length, next token -- and the pass status must
be 0.  Two calls in a row on the library's one scratch buffer, the second on
a smaller tree, so the second starts from what the first left behind."""

import numpy as np
import pytest
import torch

import workloads

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
    sess = binding.Session(shape, capacity=P + 64, max_n=64)
    binding.workspace_init(sess.cfg, 64, sess.workspace)
    sess.load_weights(workloads.make_weights(shape, "cuda", gain_jitter=0.1))
    sess.prefill(workloads.draw_tokens(P, shape.vocab, seed=3), 0)
    sess.check("prefill")
    return shape, sess, binding


def _outputs(sess, n):
    return (sess.logits[:n].clone(), sess.path[:n].clone(), sess.accept_len.clone(), sess.next_token.clone())


@pytest.mark.parametrize("trees", [("b222_n15", "b2222_n31"), ("b2222_n31", "b222_n15")])
def test_noalloc_matches_workspace_entry_point(model, trees):
    shape, sess, binding = model
    shapes = {"b222_n15": (2, 2, 2), "b2222_n31": (2, 2, 2, 2)}
    for call, name in enumerate(trees):
        parent = workloads.complete_tree(shapes[name])
        n = len(parent)
        tok = workloads.draw_tokens(n, shape.vocab, seed=40 + call)
        tok[1] = tok[2]  # (duplicate siblings: identical rows on both sides)
        binding.verify_tree(sess.cfg, sess.packed, sess.k_cache, sess.v_cache, P, tok, parent, sess.logits,
                            sess.path, sess.accept_len, sess.next_token, sess.workspace)
        want_path, want_acc, want_next = sess.outcome()
        want = _outputs(sess, n)
        k_want = sess.k_cache[:, :, :P + n].clone()
        sess.logits.zero_()
        sess.path.fill_(-7)
        sess.accept_len.fill_(-7)
        sess.next_token.fill_(-7)
        status = torch.full((1,), -7, dtype=torch.int32, device=sess.device)
        binding.verify_tree_noalloc(sess.cfg, sess.packed, sess.k_cache, sess.v_cache, P, tok, parent,
                                    sess.logits, sess.path, sess.accept_len, sess.next_token, status)
        torch.cuda.synchronize()
        assert int(status.item()) == binding.PASS_OK
        got = _outputs(sess, n)
        for g, w, what in zip(got, want, ("logits", "path", "accept_len", "next_token")):
            assert torch.equal(g, w), f"{shape.name} call {call} ({name}): {what} differs"
        assert torch.equal(sess.k_cache[:, :, :P + n], k_want)
        assert int(got[2].item()) == want_acc and int(got[3].item()) == want_next
        assert [int(x) for x in got[1][: want_acc + 1].cpu()] == want_path


def test_noalloc_rejects_passes_beyond_its_scratch(model):
    shape, sess, binding = model
    big = binding.make_config(workloads.MODELS["llama30b"])
    parent = workloads.chain_tree(128)
    rc = binding.verify_tree_noalloc(big, sess.packed, sess.k_cache, sess.v_cache, 0, np.zeros(128), parent,
                                     sess.logits, sess.path, sess.accept_len, sess.next_token,
                                     raise_on_error=False)
    assert rc == binding.EWORKSPACE
