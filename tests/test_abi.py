"""The C-ABI library on the CPU: it loads, exports every declared symbol, sizes
its buffers, and rejects bad arguments on the host before touching a device."""

import ctypes
import os
import re

import numpy as np
import pytest

import workloads

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "llmcad.h")


@pytest.fixture(scope="module")
def binding():
    from paper_2309_04255_amd import binding

    return binding


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\*?\s+\*?(llmcad_\w+)\s*\(", text, re.M)))


def test_exports_every_declared_symbol(binding):
    names = declared_functions()
    assert len(names) >= 10
    lib = binding.lib()
    for name in names:
        assert hasattr(lib, name), name
    assert set(binding.SYMBOLS) == set(names)


def test_config_checks(binding):
    ok = binding.make_config(workloads.MODELS["llama7b"])
    assert binding.check_config(ok) == binding.OK
    bad = binding.make_config(workloads.MODELS["llama7b"])
    bad.head_dim = 96
    assert binding.check_config(bad) == binding.ESHAPE
    bad = binding.make_config(workloads.MODELS["llama7b"])
    bad.n_heads = 31
    assert binding.check_config(bad) == binding.ESHAPE
    bad = binding.make_config(workloads.MODELS["llama7b"])
    bad.vocab = 0
    assert binding.check_config(bad) == binding.EARG
    assert binding.packed_bytes(bad) == 0
    assert binding.lib().llmcad_check_config(None) == binding.EARG


def test_q4_config_checks(binding):
    s = workloads.MODELS["llama7b_q4"]
    cfg = binding.make_config(s)
    assert cfg.weight_bits == 4 and binding.check_config(cfg) == binding.OK
    for bits, want in ((0, binding.OK), (16, binding.OK), (8, binding.EARG), (-4, binding.EARG)):
        c = binding.make_config(s)
        c.weight_bits = bits
        assert binding.check_config(c) == want, bits
    # the scale groups need d and F in multiples of 128
    c = binding.make_config(s)
    c.d_ffn = 11000
    assert binding.check_config(c) == binding.ESHAPE
    c.weight_bits = 16
    assert binding.check_config(c) == binding.OK
    c = binding.make_config(workloads.MODELS["tiny"])  # d = 256, F = 688
    c.weight_bits = 4
    assert binding.check_config(c) == binding.ESHAPE


def test_q4_sizes(binding):
    # the packed image holds codes (half a byte per weight) and one bf16
    # scale per 16 columns and group of 128 inputs, padded to whole blocks;
    # the globals are bf16 as in the bf16 models (weight_bytes counts what a
    # pass reads, so the embedding table is added here)
    s = workloads.MODELS["llama7b_q4"]
    pb = binding.packed_bytes(binding.make_config(s))
    held = s.weight_bytes() + 2 * s.vocab * s.d_model
    assert held <= pb <= held * 1.002
    b16 = binding.packed_bytes(binding.make_config(workloads.MODELS["llama7b"]))
    assert pb < 0.3 * b16


def test_q4_pack_validation(binding):
    lib = binding.lib()
    fake = ctypes.c_void_p(0x1000)
    q = binding.LlmcadQ4Matrix(fake.value, fake.value)
    src = binding.LlmcadQ4LayerWeights(fake.value, q, q, fake.value, q, q)
    cfg = binding.make_config(workloads.MODELS["q4small"])
    pb = binding.packed_bytes(cfg)
    # a bf16 configuration does not take 4-bit layers, nor a 4-bit one bf16 layers
    c16 = binding.make_config(workloads.MODELS["q4small"])
    c16.weight_bits = 16
    assert lib.llmcad_pack_layer_q4(ctypes.byref(c16), 0, ctypes.byref(src), fake, pb, None) == binding.EARG
    plain = binding.LlmcadLayerWeights(*([fake.value] * 6))
    assert lib.llmcad_pack_layer(ctypes.byref(cfg), 0, ctypes.byref(plain), fake, pb, None) == binding.EARG
    assert lib.llmcad_pack_layer_q4(ctypes.byref(cfg), 2, ctypes.byref(src), fake, pb, None) == binding.EARG
    assert lib.llmcad_pack_layer_q4(ctypes.byref(cfg), 0, None, fake, pb, None) == binding.EARG
    missing = binding.LlmcadQ4LayerWeights(fake.value, q, binding.LlmcadQ4Matrix(fake.value, None), fake.value, q, q)
    assert lib.llmcad_pack_layer_q4(ctypes.byref(cfg), 0, ctypes.byref(missing), fake, pb, None) == binding.EARG
    assert lib.llmcad_pack_layer_q4(ctypes.byref(cfg), 0, ctypes.byref(src), fake, pb - 1, None) == binding.EWORKSPACE


def test_sizes(binding):
    s = workloads.MODELS["llama7b"]
    cfg = binding.make_config(s)
    weight_bytes = 2 * (s.n_layers * (4 * s.d_model ** 2 + 3 * s.d_model * s.d_ffn + 2 * s.d_model)
                        + 2 * s.vocab * s.d_model + s.d_model)
    pb = binding.packed_bytes(cfg)
    assert weight_bytes <= pb <= weight_bytes * 1.001
    assert binding.workspace_bytes(cfg, 31) < binding.workspace_bytes(cfg, 128)
    assert binding.workspace_bytes(cfg, 0) == 0 and binding.workspace_bytes(cfg, 129) == 0
    off, size = binding.workspace_region(cfg, 31, 0)
    assert size == 32 * s.d_model * 4 and off + size <= binding.workspace_bytes(cfg, 31)


def test_state_regions_fixed(binding, monkeypatch):
    # The regions that hold state between passes (counters with the pass
    # status, and the zero line the kernels read for absent inputs) sit at
    # offsets that depend on neither the pass's node count nor its grid, so
    # that one llmcad_workspace_init serves passes of every size.
    cfg = binding.make_config(workloads.MODELS["llama7b"])
    seen = {5: set(), 13: set()}
    for grid in (None, "3", "24", "200"):
        if grid is None:
            monkeypatch.delenv("LLMCAD_PASS_GRID", raising=False)
        else:
            monkeypatch.setenv("LLMCAD_PASS_GRID", grid)
        for n in (1, 16, 17, 31, 64, 100, 128):
            for which in seen:
                off, size = binding.workspace_region(cfg, n, which)
                seen[which].add((off, size))
                assert off + size <= binding.workspace_bytes(cfg, n)
    assert len(seen[5]) == 1 and len(seen[13]) == 1, seen
    (zoff, zsize), = seen[13]
    (soff, _), = seen[5]
    assert zsize >= 4096 and not (zoff <= soff < zoff + zsize)


def _call_verify(binding, cfg, tok, par, prefix_len=10, cap=64, ws_bytes=1 << 30, packed=16):
    lib = binding.lib()
    tok = np.ascontiguousarray(tok, dtype=np.int32)
    par = np.ascontiguousarray(par, dtype=np.int32)
    I32P = ctypes.POINTER(ctypes.c_int32)
    fake = ctypes.c_void_p(256)  # never dereferenced: every case below fails a host check
    return lib.llmcad_verify_tree(
        ctypes.byref(cfg), ctypes.c_void_p(packed) if packed else None, fake, fake, cap, prefix_len,
        tok.ctypes.data_as(I32P), par.ctypes.data_as(I32P), len(tok), fake, fake, fake, fake, fake,
        ws_bytes, None)


def test_host_validation(binding):
    cfg = binding.make_config(workloads.MODELS["tiny"])
    V = cfg.vocab
    assert _call_verify(binding, cfg, [1, 2], [0, 0]) == binding.ETREE
    assert _call_verify(binding, cfg, [1, 2, 3], [-1, 0, 2]) == binding.ETREE
    assert _call_verify(binding, cfg, [1, 2, 3], [-1, 0, -1]) == binding.ETREE
    assert _call_verify(binding, cfg, [1, V], [-1, 0]) == binding.ETREE
    assert _call_verify(binding, cfg, [-1, 3], [-1, 0]) == binding.ETREE
    assert _call_verify(binding, cfg, np.zeros(129), np.arange(-1, 128)) == binding.ETREE
    assert _call_verify(binding, cfg, [1, 2], [-1, 0], prefix_len=63, cap=64) == binding.ECAPACITY
    assert _call_verify(binding, cfg, [1, 2], [-1, 0], prefix_len=-1) == binding.ECAPACITY
    assert _call_verify(binding, cfg, [1, 2], [-1, 0], cap=96) == binding.ECAPACITY  # (not a multiple of 64)
    assert _call_verify(binding, cfg, [1, 2], [-1, 0], ws_bytes=1000) == binding.EWORKSPACE
    assert _call_verify(binding, cfg, [1, 2], [-1, 0], packed=0) == binding.EARG
    bad = binding.make_config(workloads.MODELS["tiny"])
    bad.head_dim = 32
    bad.n_heads = 8
    assert _call_verify(binding, bad, [1, 2], [-1, 0]) == binding.ESHAPE
    assert binding.status_string(binding.ETREE) == "invalid token tree"


def _call_noalloc(binding, cfg, tok, par, prefix_len=10, cap=64, packed=16):
    lib = binding.lib()
    tok = np.ascontiguousarray(tok, dtype=np.int32)
    par = np.ascontiguousarray(par, dtype=np.int32)
    I32P = ctypes.POINTER(ctypes.c_int32)
    fake = ctypes.c_void_p(256)  # never dereferenced: every case below fails a host check
    return lib.llmcad_verify_tree_noalloc(
        ctypes.byref(cfg), ctypes.c_void_p(packed) if packed else None, fake, fake, cap, prefix_len,
        tok.ctypes.data_as(I32P), par.ctypes.data_as(I32P), len(tok), fake, fake, fake, fake, None, None)


def test_noalloc_host_validation(binding):
    # the no-allocation entry point makes llmcad_verify_tree's host checks,
    # and refuses a pass whose workspace exceeds its scratch, before any
    # device call
    cfg = binding.make_config(workloads.MODELS["tiny"])
    V = cfg.vocab
    assert _call_noalloc(binding, cfg, [1, 2], [0, 0]) == binding.ETREE
    assert _call_noalloc(binding, cfg, [1, V], [-1, 0]) == binding.ETREE
    assert _call_noalloc(binding, cfg, np.zeros(129), np.arange(-1, 128)) == binding.ETREE
    assert _call_noalloc(binding, cfg, [1, 2], [-1, 0], prefix_len=63, cap=64) == binding.ECAPACITY
    assert _call_noalloc(binding, cfg, [1, 2], [-1, 0], packed=0) == binding.EARG
    big = binding.make_config(workloads.MODELS["llama30b"])
    assert binding.workspace_bytes(big, 128) > binding.SCRATCH_BYTES
    assert _call_noalloc(binding, big, np.zeros(128), np.arange(-1, 127), cap=4096) == binding.EWORKSPACE
    b7 = binding.make_config(workloads.MODELS["llama7b"])
    assert binding.workspace_bytes(b7, 32) <= binding.SCRATCH_BYTES < binding.workspace_bytes(b7, 33)


def test_prefill_validation(binding):
    cfg = binding.make_config(workloads.MODELS["tiny"])
    lib = binding.lib()
    I32P = ctypes.POINTER(ctypes.c_int32)
    fake = ctypes.c_void_p(256)
    toks = np.array([1, 2, cfg.vocab], dtype=np.int32)
    rc = lib.llmcad_prefill(ctypes.byref(cfg), fake, fake, fake, 64, toks.ctypes.data_as(I32P), 3, 0,
                            None, fake, 1 << 30, None)
    assert rc == binding.ETREE
    toks = np.array([1, 2, 3], dtype=np.int32)
    rc = lib.llmcad_prefill(ctypes.byref(cfg), fake, fake, fake, 64, toks.ctypes.data_as(I32P), 3, 62,
                            None, fake, 1 << 30, None)
    assert rc == binding.ECAPACITY
    rc = lib.llmcad_prefill(ctypes.byref(cfg), fake, fake, fake, 64, toks.ctypes.data_as(I32P), 3, 0,
                            None, fake, 100, None)
    assert rc == binding.EWORKSPACE


def test_commit_validation(binding):
    # Host-side checks of the rollback entry point; none of these calls
    # enqueues anything (n = 1 leaves the root in place and returns at once).
    cfg = binding.make_config(workloads.MODELS["tiny"])
    lib = binding.lib()
    fake = ctypes.c_void_p(256)
    assert lib.llmcad_commit_path(ctypes.byref(cfg), None, fake, 64, 10, fake, fake, 4, None) == binding.EARG
    assert lib.llmcad_commit_path(ctypes.byref(cfg), fake, fake, 64, 10, None, fake, 4, None) == binding.EARG
    assert lib.llmcad_commit_path(ctypes.byref(cfg), fake, fake, 64, 10, fake, fake, 0, None) == binding.ETREE
    assert lib.llmcad_commit_path(ctypes.byref(cfg), fake, fake, 64, 10, fake, fake, 129, None) == binding.ETREE
    assert lib.llmcad_commit_path(ctypes.byref(cfg), fake, fake, 64, 61, fake, fake, 4, None) == binding.ECAPACITY
    assert lib.llmcad_commit_path(ctypes.byref(cfg), fake, fake, 64, -1, fake, fake, 4, None) == binding.ECAPACITY
    assert lib.llmcad_commit_path(ctypes.byref(cfg), fake, fake, 64, 10, fake, fake, 1, None) == binding.OK


def test_extend_validation(binding):
    # Host-side checks of the tree-decoder step; nothing is enqueued.
    cfg = binding.make_config(workloads.MODELS["tiny"])
    lib = binding.lib()
    I32P = ctypes.POINTER(ctypes.c_int32)
    fake = ctypes.c_void_p(256)
    tok = np.array([1, 2, 3], dtype=np.int32)
    par = np.array([-1, 0, 1], dtype=np.int32)

    def call(first, n=3, prefix_len=10, cap=64, t=tok, p=par, ws=1 << 30):
        return lib.llmcad_extend_tree(ctypes.byref(cfg), fake, fake, fake, cap, prefix_len,
                                      t.ctypes.data_as(I32P), p.ctypes.data_as(I32P), n, first, None, fake, ws,
                                      None)

    assert call(3) == binding.ETREE             # first must be < n
    assert call(-1) == binding.ETREE
    assert call(1, p=np.array([-1, 0, 2], dtype=np.int32)) == binding.ETREE
    assert call(1, t=np.array([1, 2, cfg.vocab], dtype=np.int32)) == binding.ETREE
    assert call(1, prefix_len=62) == binding.ECAPACITY
    assert call(1, ws=100) == binding.EWORKSPACE


def test_extend_candidates_validation(binding):
    # Host-side checks of the tree-decoder step with candidate summaries:
    # logits and the record buffer are required, the threshold lies in (0, 1),
    # and the tree checks of llmcad_extend_tree apply; nothing is enqueued.
    cfg = binding.make_config(workloads.MODELS["tiny"])
    lib = binding.lib()
    I32P = ctypes.POINTER(ctypes.c_int32)
    fake = ctypes.c_void_p(256)
    tok = np.array([1, 2, 3], dtype=np.int32)
    par = np.array([-1, 0, 1], dtype=np.int32)

    def call(first=2, thr=0.3, logits=fake, cand=fake, t=tok, p=par, ws=1 << 30):
        return lib.llmcad_extend_tree_candidates(ctypes.byref(cfg), fake, fake, fake, 64, 10,
                                                 t.ctypes.data_as(I32P), p.ctypes.data_as(I32P), 3, first,
                                                 ctypes.c_float(thr), logits, cand, fake, ws, None)

    assert call(logits=None) == binding.EARG
    assert call(cand=None) == binding.EARG
    for thr in (0.0, 1.0, -0.5, float("nan")):
        assert call(thr=thr) == binding.EARG, thr
    assert call(first=3) == binding.ETREE
    assert call(p=np.array([-1, 0, 2], dtype=np.int32)) == binding.ETREE
    assert call(ws=100) == binding.EWORKSPACE
    # the record layout the binding parses: 4 header words, then CAND_MAX tokens and probabilities
    assert binding.CAND_WORDS == 4 + 2 * binding.CAND_MAX == 132
    w = np.zeros(binding.CAND_WORDS, dtype=np.int32)
    w[0], w[1] = 2, 7
    w[2:4] = np.array([3.5, 1.25], dtype=np.float32).view(np.int32)
    w[4:6] = [7, 9]
    w[4 + binding.CAND_MAX:6 + binding.CAND_MAX] = np.array([0.5, 0.25], dtype=np.float32).view(np.int32)
    rec = binding.parse_candidates(w)
    assert rec == {"count": 2, "argmax": 7, "max_logit": 3.5, "sum_exp": 1.25, "tok": [7, 9], "prob": [0.5, 0.25]}
