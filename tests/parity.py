"""Parity checks between the HIP path and the oracle.

Bars (the floating-point bar is the one stated for this pass):
  logits   max |gpu - oracle| <= 2e-2 and ||gpu - oracle||_2 / ||oracle||_2 <= 1e-2
  argmax   equal wherever the oracle's top-2 logit gap exceeds 1e-2
  walk     path / accept_len / next_token equal whenever every node the walk
           reads (every node reachable under the oracle's argmax) has gap
           > 1e-2; in any case the GPU's walk must be the oracle's walk
           applied to the GPU's own argmax (integer logic, bit-exact).
"""

import numpy as np

import oracle

ABS_TOL = 2e-2
REL_TOL = 1e-2
GAP = 1e-2


def top2_gap(logits):
    part = np.partition(logits, -2, axis=1)
    return part[:, -1] - part[:, -2]


def reachable(parent, tokens, amax):
    n = len(parent)
    reach = np.zeros(n, dtype=bool)
    reach[0] = True
    for i in range(1, n):
        reach[i] = reach[parent[i]] and tokens[i] == amax[parent[i]]
    return reach


def check_logits(gpu, ref, what=""):
    gpu = np.asarray(gpu, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert gpu.shape == ref.shape, (gpu.shape, ref.shape)
    assert np.all(np.isfinite(gpu)), f"{what}: non-finite GPU logits"
    err = np.abs(gpu - ref).max()
    rel = np.linalg.norm(gpu - ref) / np.linalg.norm(ref)
    assert err <= ABS_TOL, f"{what}: max abs error {err:.3e} > {ABS_TOL}"
    assert rel <= REL_TOL, f"{what}: relative L2 error {rel:.3e} > {REL_TOL}"
    return err, rel


def check_argmax(gpu_amax, ref_logits, what=""):
    ref_amax = np.argmax(ref_logits, axis=1)
    gap = top2_gap(ref_logits)
    sure = gap > GAP
    bad = np.nonzero(sure & (np.asarray(gpu_amax) != ref_amax))[0]
    assert len(bad) == 0, f"{what}: argmax differs at confident rows {bad.tolist()}"
    return int(sure.sum())


def check_walk(parent, tokens, gpu_amax, gpu_path, gpu_accept, gpu_next, ref_logits, what=""):
    parent = np.asarray(parent)
    tokens = np.asarray(tokens)
    gpu_amax = np.asarray(gpu_amax)
    # 1. the GPU's walk is the oracle's walk on the GPU's own argmax
    path, nxt, _ = oracle.accept_walk(parent, tokens, gpu_amax)
    assert list(gpu_path) == path, f"{what}: path {list(gpu_path)} != {path} (on GPU argmax)"
    assert gpu_accept == len(path) - 1
    assert gpu_next == nxt
    # 2. equal to the oracle's result when every node the walk reads is confident
    ref_amax = np.argmax(ref_logits, axis=1)
    gap = top2_gap(ref_logits)
    reach = reachable(parent, tokens, ref_amax)
    if np.all(gap[reach] > GAP):
        rpath, rnext, _ = oracle.accept_walk(parent, tokens, ref_amax)
        assert list(gpu_path) == rpath, f"{what}: path {list(gpu_path)} != oracle {rpath}"
        assert gpu_next == rnext, f"{what}: next {gpu_next} != oracle {rnext}"
        return True
    return False
