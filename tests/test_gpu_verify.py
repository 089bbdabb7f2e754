"""GPU parity of the HIP verification pass against the oracle (through the C ABI).

Models: the tiny 2-layer shape (head_dim 64, F = 688 not a multiple of 32), a
small head_dim-128 shape with ragged F and V (V = 1998 leaves a partial
16-column block of the LM head), and a small 4-bit model (group-quantised
layer matrices, 4 to 11 scale groups per row; the oracle runs on the weights
the codes and scales stand for).  Norm gains are jittered so that the gain path is exercised.
Trees span one to eight 16-row blocks with ragged tails (n = 1 ... 128), and
the prefix (100) is not a multiple of the 64-position attention chunk.
"""

import os
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
    "q4small": workloads.MODELS["q4small"],
}
TREES = {
    "single": workloads.chain_tree(1),
    "binary_d3_n15": workloads.complete_tree((2, 2, 2)),
    "random_n20": workloads.random_tree(20, 7, 5),
    "chain_n9": workloads.chain_tree(9),
    "binary_d4_n31": workloads.complete_tree((2, 2, 2, 2)),
    "b432_n41": workloads.complete_tree((4, 3, 2)),
    "random_n77": workloads.random_tree(77, 7, 8),
    "random_n128": workloads.random_tree(128, 7, 9),
}


def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2309_04255_amd import binding

    return binding


@pytest.fixture(scope="module", params=sorted(SHAPES))
def model(request):
    binding = _gpu()
    shape = SHAPES[request.param]
    print(f"\n[model] {shape.name}", flush=True)
    gen = workloads.make_weights(shape, "cuda", gain_jitter=0.1)
    sess = binding.Session(shape, capacity=P + 200, max_n=128)
    binding.workspace_init(sess.cfg, 128, sess.workspace)
    sess.load_weights(gen)
    ow = oracle_weights(shape, gain_jitter=0.1)
    prefix = workloads.draw_tokens(P, shape.vocab, seed=3)
    ok, ov = oracle.prefill_kv(ow, prefix, rounding=True)
    sess.prefill(prefix, 0)
    torch.cuda.synchronize()
    return types.SimpleNamespace(shape=shape, sess=sess, ow=ow, prefix=prefix, ok=ok, ov=ov,
                                 binding=binding, gen=gen)


def _gpu_amax(m, n):
    off, size = m.binding.workspace_region(m.sess.cfg, n, 4)
    return m.sess.workspace[off:off + 4 * n].view(torch.int32).cpu().numpy()


def _run(m, parent, tok):
    n = len(parent)
    m.sess.verify_tree(P, tok, parent)
    logits, path, acc, nxt = m.sess.results(n)
    return logits.numpy(), path, acc, nxt, _gpu_amax(m, n)


def _check_all(m, parent, tok, what):
    logits, path, acc, nxt, amax = _run(m, parent, tok)
    ref, _, _ = oracle.tree_forward(m.ow, m.ok, m.ov, tok, parent, rounding=True)
    err, rel = parity.check_logits(logits, ref, what)
    np.testing.assert_array_equal(amax, np.argmax(logits, axis=1))
    parity.check_argmax(amax, ref, what)
    parity.check_walk(parent, tok, amax, path, acc, nxt, ref, what)
    print(f"[{what}] max_abs={err:.2e} rel={rel:.2e}", flush=True)
    return logits


def test_weights_identical_on_cpu_and_gpu(model):
    cpu = workloads.make_weights(model.shape, "cpu", gain_jitter=0.1).layer(1)
    gpu = model.gen.layer(1)
    for k in cpu:
        pairs = zip(cpu[k], gpu[k]) if isinstance(cpu[k], tuple) else [(cpu[k], gpu[k])]
        for c, g in pairs:
            assert torch.equal(c, g.cpu()), k


@pytest.mark.parametrize("tree", list(TREES))
def test_verify_matches_oracle(model, tree):
    parent = TREES[tree]
    tok = workloads.draw_tokens(len(parent), model.shape.vocab, seed=101, stream=len(parent))
    _check_all(model, parent, tok, f"{model.shape.name}/{tree}")


def test_launch_shape_variants(model, monkeypatch):
    # One and four key splits in the attention, and smaller grids (each
    # workgroup then takes longer runs of column blocks, cut into several
    # tiles, and with 24 or 3 workgroups the attention units take several
    # rounds, the later ones with nothing fetched before the barrier) meet
    # the oracle bar too.
    parent = TREES["b432_n41"]
    tok = workloads.draw_tokens(len(parent), model.shape.vocab, seed=7)
    _check_all(model, parent, tok, "default")
    for env in ({"LLMCAD_ATTN_SPLITS": "1"}, {"LLMCAD_ATTN_SPLITS": "4"},
                {"LLMCAD_PASS_GRID": "200"}, {"LLMCAD_PASS_GRID": "24"}, {"LLMCAD_PASS_GRID": "3"}):
        for k, v in env.items():
            monkeypatch.setenv(k, v)
        _check_all(model, parent, tok, str(env))
        for k in env:
            monkeypatch.delenv(k)


def test_wide_gate_up_tiles(model, monkeypatch):
    # Passes of up to 32 rows whose gate/up runs exceed 8 blocks per
    # workgroup take tiles of up to 9 blocks (a separate kernel instance).
    # Small grids force it on the test models: 9 blocks per workgroup (one
    # tile), 10 (9 + 1) and ~43 (several tiles and a ragged last one).
    parent = TREES["binary_d4_n31"]
    tok = workloads.draw_tokens(len(parent), model.shape.vocab, seed=11)
    Fp = -(-model.shape.d_ffn // 32) * 32
    grids = sorted({-(-(Fp // 8) // 9), -(-(Fp // 8) // 10), 3})
    for G in grids:
        monkeypatch.setenv("LLMCAD_PASS_GRID", str(G))
        _check_all(model, parent, tok, f"grid {G}")
    monkeypatch.delenv("LLMCAD_PASS_GRID")


@pytest.mark.parametrize("tree", ["binary_d4_n31", "b432_n41", "random_n77", "random_n128"])
def test_split_k_variants(model, monkeypatch, tree):
    # Split-K for the O and down projections (passes of 32 or more rows):
    # groups of 2 or 4 workgroups share a group of column blocks, each over
    # a slice of the k-steps, and add their partial tiles in slice order.
    # The small models' d/16 blocks need a grid of at most 4 d/16 workgroups
    # for a block per group: 64 and 24 workgroups (with 24 and S = 4 some
    # workgroups of a group finish no block).  Each variant meets the oracle
    # bar, and (bf16 models) its logits differ from the unsplit pass's
    # somewhere (another order of fp32 additions): the split path ran.
    parent = TREES[tree]
    tok = workloads.draw_tokens(len(parent), model.shape.vocab, seed=11)
    for grid, s_o, s_down in ((64, 4, 4), (64, 2, 4), (24, 4, 2), (24, 2, 4)):
        monkeypatch.setenv("LLMCAD_PASS_GRID", str(grid))
        monkeypatch.setenv("LLMCAD_SPLIT_O", "1")
        monkeypatch.setenv("LLMCAD_SPLIT_DOWN", "1")
        base = _check_all(model, parent, tok, f"grid {grid} unsplit")
        monkeypatch.setenv("LLMCAD_SPLIT_O", str(s_o))
        monkeypatch.setenv("LLMCAD_SPLIT_DOWN", str(s_down))
        split = _check_all(model, parent, tok, f"grid {grid} split O {s_o} down {s_down}")
        if model.shape.weight_bits == 16:
            assert not np.array_equal(base, split), "the split-K path did not run"
        again = _run(model, parent, tok)[0]
        np.testing.assert_array_equal(split, again)  # bit-reproducible
        for k in ("LLMCAD_PASS_GRID", "LLMCAD_SPLIT_O", "LLMCAD_SPLIT_DOWN"):
            monkeypatch.delenv(k)


@pytest.mark.parametrize("tree", ["b432_n41", "random_n77", "random_n128"])
def test_row_split_tiles(model, monkeypatch, tree):
    # Row-split tiles (passes of 64+ rows, workgroups with more blocks than a
    # K-split tile holds: the waves split the rows and share each k-step's
    # weight fragments through LDS).  The small models' phases give a
    # workgroup that many blocks on small grids (on 3 workgroups every step
    # does; on 24 some).  With them on (the default) and off, the pass meets
    # the oracle bar and repeats bit for bit; on 3 workgroups the results
    # differ somewhere (another order of fp32 additions: the path ran, bf16
    # models).
    parent = TREES[tree]
    tok = workloads.draw_tokens(len(parent), model.shape.vocab, seed=13)
    for grid in (24, 3):
        monkeypatch.setenv("LLMCAD_PASS_GRID", str(grid))
        monkeypatch.setenv("LLMCAD_ROW_TILES", "2")
        base = _check_all(model, parent, tok, f"grid {grid} K-split tiles")
        monkeypatch.delenv("LLMCAD_ROW_TILES")
        rows = _check_all(model, parent, tok, f"grid {grid} row-split tiles")
        if model.shape.weight_bits == 16 and grid == 3:
            assert not np.array_equal(base, rows), "the row-split path did not run"
        np.testing.assert_array_equal(rows, _run(model, parent, tok)[0])
        monkeypatch.delenv("LLMCAD_PASS_GRID")


def _long_prefix_session(model, PL):
    """A session whose cache holds PL seeded random bf16 prefix keys/values
    (written straight into the cache) and the oracle's copies of them."""
    shape, binding = model.shape, model.binding
    sess = binding.Session(shape, capacity=PL + 160, max_n=128)
    binding.workspace_init(sess.cfg, 128, sess.workspace)
    sess.load_weights(model.gen)
    rng = np.random.default_rng(0x10AD)
    dims = (shape.n_layers, PL, shape.n_heads, shape.head_dim)
    pk = oracle.bf16_round(rng.standard_normal(dims) * 0.7)
    pv = oracle.bf16_round(rng.standard_normal(dims) * 0.7)
    sess.k_cache[:, :, :PL] = torch.from_numpy(pk.transpose(0, 2, 1, 3).astype(np.float32)).to(torch.bfloat16).cuda()
    sess.v_rows[:, :, :PL] = torch.from_numpy(pv.transpose(0, 2, 1, 3).astype(np.float32)).to(torch.bfloat16).cuda()
    return sess, pk, pv


@pytest.mark.parametrize("PL", [P, 600])
def test_attention_prefetch_is_exact(model, monkeypatch, PL):
    # The attention fetches the prefix part of its keys/values before its
    # phase's barrier (registers, and copies to LDS made for one wave by
    # another); fetched after the barrier instead, every output bit must be
    # the same.  Two prefix lengths: a few steps, and several per wave.
    sess = model.sess if PL == P else _long_prefix_session(model, PL)[0]
    parent = TREES["b432_n41"]
    n = len(parent)
    tok = workloads.draw_tokens(n, model.shape.vocab, seed=19)
    runs = []
    for mode in ("1", "2"):
        monkeypatch.setenv("LLMCAD_ATTN_PREFETCH", mode)
        sess.verify_tree(PL, tok, parent)
        logits, path, acc, nxt = sess.results(n)
        runs.append((logits.numpy(), path, acc, nxt))
    np.testing.assert_array_equal(runs[0][0], runs[1][0])
    assert runs[0][1:] == runs[1][1:]


@pytest.mark.parametrize("PL,splits", [(600, "default"), (600, "1"), (600, "2"), (600, "3"), (600, "4"),
                                       (2100, "default"), (2100, "1")])
def test_long_prefix_key_splits(model, monkeypatch, PL, splits):
    # Long prefixes (600 and 2100 positions; neither a multiple of the
    # attention's 32-key step, so one step holds prefix and tree keys): the
    # attention's key splits (1 to 4 per head and row block, merged in split
    # order) all meet the oracle bar, whether a split's prefix steps were all
    # fetched before the phase's barrier or (one split over a 2100-position
    # prefix) most of them stream in afterwards.  The prefix K/V are seeded
    # random bf16 values written straight into the cache and handed to the
    # oracle.
    shape, binding = model.shape, model.binding
    sess, pk, pv = _long_prefix_session(model, PL)
    if splits != "default":
        monkeypatch.setenv("LLMCAD_ATTN_SPLITS", splits)
    parent = TREES["b432_n41"]
    n = len(parent)
    tok = workloads.draw_tokens(n, shape.vocab, seed=23)
    sess.verify_tree(PL, tok, parent)
    logits, path, acc, nxt = sess.results(n)
    logits = logits.numpy()
    ref, _, _ = oracle.tree_forward(model.ow, pk, pv, tok, parent, rounding=True)
    what = f"{shape.name}/P{PL}/splits={splits}"
    err, rel = parity.check_logits(logits, ref, what)
    off, _ = binding.workspace_region(sess.cfg, n, 4)
    amax = sess.workspace[off:off + 4 * n].view(torch.int32).cpu().numpy()
    np.testing.assert_array_equal(amax, np.argmax(logits, axis=1))
    parity.check_argmax(amax, ref, what)
    parity.check_walk(parent, tok, amax, path, acc, nxt, ref, what)
    print(f"[{what}] max_abs={err:.2e} rel={rel:.2e}", flush=True)


def test_pass_status_ok(model):
    parent = TREES["binary_d3_n15"]
    tok = workloads.draw_tokens(len(parent), model.shape.vocab, seed=3)
    _run(model, parent, tok)
    off, _ = model.binding.workspace_region(model.sess.cfg, len(parent), 5)
    assert int(model.sess.workspace[off:off + 4].view(torch.int32).item()) == 0


def test_deterministic_and_prefix_untouched(model):
    parent = TREES["random_n77"]
    tok = workloads.draw_tokens(len(parent), model.shape.vocab, seed=5)
    before = model.sess.k_cache[:, :, :P].clone(), model.sess.v_rows[:, :, :P].clone()
    a = _run(model, parent, tok)
    b = _run(model, parent, tok)
    np.testing.assert_array_equal(a[0], b[0])
    assert a[1:4] == b[1:4]
    assert torch.equal(model.sess.k_cache[:, :, :P], before[0])
    assert torch.equal(model.sess.v_rows[:, :, :P], before[1])


def test_tree_kv_written_to_node_slots(model):
    parent = TREES["binary_d3_n15"]
    n = len(parent)
    tok = workloads.draw_tokens(n, model.shape.vocab, seed=9)
    _run(model, parent, tok)
    _, tk, tv = oracle.tree_forward(model.ow, model.ok, model.ov, tok, parent, rounding=True)
    # cache [L][H][cap][Dh] vs oracle [L][n][H][Dh]
    gk = model.sess.k_cache[:, :, P:P + n].float().cpu().numpy().transpose(0, 2, 1, 3)
    gv = model.sess.v_rows[:, :, P:P + n].float().cpu().numpy().transpose(0, 2, 1, 3)
    for g, r in ((gk, tk), (gv, tv)):
        scale = np.abs(r).max()
        assert np.abs(g - r).max() <= 2e-2 * scale


def test_isolated_prefix_kv(model):
    # Upload the oracle's bf16 prefix K/V instead of the GPU prefill's.
    s = model.sess
    saved = s.k_cache[:, :, :P].clone(), s.v_rows[:, :, :P].clone()
    try:
        s.k_cache[:, :, :P] = torch.from_numpy(model.ok.transpose(0, 2, 1, 3).astype(np.float32)).to(
            torch.bfloat16).cuda()
        s.v_rows[:, :, :P] = torch.from_numpy(model.ov.transpose(0, 2, 1, 3).astype(np.float32)).to(
            torch.bfloat16).cuda()
        parent = TREES["binary_d4_n31"]
        tok = workloads.draw_tokens(len(parent), model.shape.vocab, seed=13)
        _check_all(model, parent, tok, "isolated")
    finally:
        s.k_cache[:, :, :P] = saved[0]
        s.v_rows[:, :, :P] = saved[1]


def test_prefill_last_logits(model):
    binding = model.binding
    s = model.sess
    toks = workloads.draw_tokens(150, model.shape.vocab, seed=21)
    k = torch.zeros_like(s.k_cache)
    v = torch.zeros_like(s.v_cache)
    out = torch.empty(model.shape.vocab, dtype=torch.float32, device="cuda")
    binding.prefill(s.cfg, s.packed, k, v, toks, 0, out, s.workspace)
    torch.cuda.synchronize()
    ref, _, _ = oracle.causal_forward(model.ow, toks, rounding=True)
    parity.check_logits(out.cpu().numpy()[None], ref[-1:], "prefill")


def test_planted_tree(model):
    # Plant the oracle's greedy continuation along the last branch of a 41-node
    # tree; the GPU must accept exactly K nodes and return the next greedy token.
    parent = TREES["b432_n41"]
    n = len(parent)
    # (seed 53: on both models every node the oracle's walk reads has a top-2
    # gap above 5e-2, so the exact acceptance below is always asserted)
    tok = workloads.draw_tokens(n, model.shape.vocab, seed=53)
    K = 2
    seq = [int(x) for x in np.concatenate([model.prefix, tok[:1]])]
    cont = []
    for _ in range(K + 1):
        lg, _, _ = oracle.causal_forward(model.ow, seq, rounding=True)
        cont.append(int(np.argmax(lg[-1])))
        seq.append(cont[-1])
    tok_p = workloads.plant_path(parent, tok, n - 1, cont, model.shape.vocab)
    ref = oracle.verify_tree(model.ow, model.ok, model.ov, tok_p, parent, rounding=True)
    assert ref["accept_len"] == K
    logits, path, acc, nxt, amax = _run(model, parent, tok_p)
    confident = parity.check_walk(parent, tok_p, amax, path, acc, nxt, ref["logits"], "planted")
    assert confident, "the planted path's seed no longer gives confident oracle gaps"
    assert acc == K and nxt == cont[K]


def test_pass_status_failure_raises_and_recovers(model, monkeypatch):
    # The pass's waits are bounded: one that runs out sets the device status
    # to 1 and the workgroup leaves the pass.  LLMCAD_FAIL_WAITS=1 makes every
    # grid wait give up at once (every workgroup still exits normally), so
    # the failure path runs deterministically: the session must raise,
    # re-initialise the workspace, and serve a correct pass afterwards.
    binding = model.binding
    parent = TREES["binary_d3_n15"]
    tok = workloads.draw_tokens(len(parent), model.shape.vocab, seed=41)
    monkeypatch.setenv("LLMCAD_FAIL_WAITS", "1")
    model.sess.verify_tree(P, tok, parent)
    with pytest.raises(binding.LlmcadPassError) as err:
        model.sess.results(len(parent))
    assert err.value.status == binding.PASS_WAIT_TIMEOUT
    model.sess.verify_tree(P, tok, parent, want_logits=False)
    with pytest.raises(binding.LlmcadPassError):
        model.sess.outcome()
    monkeypatch.delenv("LLMCAD_FAIL_WAITS")
    assert model.sess.pass_status() == binding.PASS_OK  # (cleared by the re-initialisation)
    _check_all(model, parent, tok, "after a failed pass")
    assert model.sess.pass_status() == binding.PASS_OK


def test_host_errors_leave_cache_untouched(model):
    binding = model.binding
    s = model.sess
    before = s.k_cache.clone()
    V = model.shape.vocab
    cases = [
        ([1, 2], [0, 0], binding.ETREE),          # parent[0] != -1
        ([1, 2, 3], [-1, 0, 2], binding.ETREE),   # parent[i] >= i
        ([1, V], [-1, 0], binding.ETREE),          # token out of range
        ([], [], binding.ETREE),                   # empty tree
    ]
    for tok, par, want in cases:
        rc = binding.verify_tree(s.cfg, s.packed, s.k_cache, s.v_cache, P, tok, par, s.logits, s.path,
                                 s.accept_len, s.next_token, s.workspace, raise_on_error=False)
        assert rc == want, (tok, par, rc)
    rc = binding.verify_tree(s.cfg, s.packed, s.k_cache, s.v_cache, s.capacity - 1, [1, 2], [-1, 0],
                             s.logits, s.path, s.accept_len, s.next_token, s.workspace,
                             raise_on_error=False)
    assert rc == binding.ECAPACITY
    big = workloads.chain_tree(129)
    rc = binding.verify_tree(s.cfg, s.packed, s.k_cache, s.v_cache, P, np.zeros(129), big, s.logits,
                             s.path, s.accept_len, s.next_token, s.workspace, raise_on_error=False)
    assert rc == binding.ETREE
    torch.cuda.synchronize()
    assert torch.equal(s.k_cache, before)
