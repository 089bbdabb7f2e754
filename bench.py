#!/usr/bin/env python3
"""Token-tree verification benchmark on one MI355X.

A step is one verification pass (§3.2 of arXiv 2309.04255): the target
model's forward over every node of a draft token tree against the prefix KV
cache, the per-node argmax and the accept walk, all in libllmcad's HIP
kernels.  Default workload: LLaMA-7B shape (32 layers, d 4096, 32x128 heads,
F 11008, V 32000), random bf16 weights, 512-token prefix, 31-node tree
(root + complete binary tree of depth 4), uniform tokens.

Prints one JSON line (rank 0):
  value            passes/s over the timed steps (inputs resident in HBM)
  hbm_roofline_frac  algorithmic bytes of a pass / (time per pass * 8 TB/s)
  roofline         the dominant kernel, which is the whole pass (one
                   persistent launch): algorithmic bytes per launch / mean
                   launch time (HIP events on the pass's stream), against 8 TB/s
  cpu_baseline     the CPU oracle timed on this host on a bounded sample
Progress goes to stderr.
"""

import argparse
import hashlib
import json
import re
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK = 8.0e12  # MI355X HBM3E, bytes/s
METRIC = "tree-verify passes/sec + % HBM roofline, LLaMA-7B shape, 31-node tree"
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "pass_kernel_traffic.json")
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2309_04255_amd", "csrc", f)
                  for f in ("pass.hip", "device.h", "layout.h", "kernels.h")]


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def pass_bytes(shape, P, n):
    """Algorithmic HBM bytes of one pass: every weight byte once (layer
    matrices as stored: bf16, or 4-bit codes plus a bf16 scale per 128
    inputs; norm gains, LM head), prefix K+V read once, tree K/V written,
    the nodes' embedding rows, fp32 logits."""
    L, d, V = shape.n_layers, shape.d_model, shape.vocab
    return shape.weight_bytes() + 4 * L * P * d + 4 * L * n * d + 2 * n * d + 4 * n * V


def source_hash():
    h = hashlib.sha256()
    for path in KERNEL_SOURCES:
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def _read_traffic():
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return {}
    return t if isinstance(t, dict) else {}


def load_traffic(workload):
    """Measured HBM bytes per pass-kernel launch for this workload (FETCH_SIZE
    + WRITE_SIZE, calibrated against a copy kernel), or None when the counters
    were taken on other kernel sources or never for this workload."""
    t = _read_traffic().get(workload)
    if not t or t.get("kernel_sources_sha256_16") != source_hash():
        return None
    return t.get("bytes_per_launch")


def write_traffic(fetch_csv, write_csv, workload, copy_mib):
    """From two rocprofv3 --pmc runs of `bench.py --calibration-copy-mib N`
    (one collecting FETCH_SIZE, one WRITE_SIZE; per dispatch, in KiB), the
    pass kernel's HBM bytes per launch.  Calibration: the N MiB fill that
    precedes the copy writes a known size (write factor), and the copy's
    chunks read as much as they write (read factor).  Stores the entry for
    `workload` in TRAFFIC_FILE, tagged with the kernel sources' hash."""
    import csv

    def per_kernel(path):
        vals = {}
        with open(path, newline="") as f:
            for row in csv.DictReader(f):
                vals.setdefault(row["Kernel_Name"], []).append(float(row["Counter_Value"]))
        return vals

    fetch, write = per_kernel(fetch_csv), per_kernel(write_csv)
    copy = "__amd_rocclr_copyBuffer"
    fill = [k for k in write if "FillFunctor<float>" in k]
    if copy not in fetch or copy not in write or not fill:
        raise SystemExit(f"calibration kernels not found: {sorted(write)}")
    fill_kib = max(write[fill[0]])
    write_factor = copy_mib * 1024.0 / fill_kib
    chunk_fetch = statistics.median(v for v in fetch[copy] if v > 4096)
    chunk_write = statistics.median(v for v in write[copy] if v > 4096)
    read_factor = chunk_write * write_factor / chunk_fetch
    # The verification passes are the last launches of the pass kernel's
    # instance for the workload's row count (pass_kernel<16-row blocks, head
    # dim, wide gate/up tiles>; the prefill's 128-row chunks run before them,
    # as another instance when the tree has fewer rows): take that
    # instance's last launches.
    import workloads

    wl = workloads.get_workload(workload)
    n = len(workloads.make_tree(wl.tree, wl.shape.vocab, wl.seed)[0])
    mb = -(-n // 16)
    mb = 1 if mb <= 1 else 2 if mb <= 2 else 4 if mb <= 4 else 8
    inst = re.compile(rf"pass_kernel<{mb}, {wl.shape.head_dim}(, (true|false))?>")
    names = [k for k in fetch if inst.search(k)]
    if len(names) != 1:
        raise SystemExit(f"pass kernel instance for {workload} not found: {sorted(fetch)}")
    passk = names[0]
    f_kib, w_kib = statistics.median(fetch[passk][-3:]), statistics.median(write[passk][-3:])
    out = {
        "workload": workload, "kernel_sources_sha256_16": source_hash(), "kernel": passk[:90],
        "launches_used": 3, "fetch_kib": round(f_kib), "write_kib": round(w_kib),
        "calibration": {"fill_mib": copy_mib, "fill_write_kib": fill_kib, "write_factor": round(write_factor, 4),
                        "copy_chunk_fetch_kib": chunk_fetch, "copy_chunk_write_kib": chunk_write,
                        "read_factor": round(read_factor, 4)},
        "read_bytes": round(f_kib * 1024 * read_factor), "write_bytes": round(w_kib * 1024 * write_factor),
    }
    out["bytes_per_launch"] = out["read_bytes"] + out["write_bytes"]
    all_t = _read_traffic()
    all_t[workload] = out
    with open(TRAFFIC_FILE, "w") as f:
        json.dump(all_t, f, indent=1, sort_keys=True)
        f.write("\n")
    print(json.dumps(out, indent=1))


def cpu_baseline(gen, shape, P, parent, tok, seed, budget_s=20.0):
    """Time the CPU oracle on a pass of the workload: oracle.tree_layer layer
    by layer (float64 NumPy with the bf16 rounding points), then the final
    norm and LM head.  Layers are timed until `budget_s` seconds of oracle
    arithmetic have been spent (every layer when the whole pass fits, as at
    the LLaMA-7B shape); the per-layer mean is then scaled to all layers.
    The weights come from the seeded generator on the GPU, widened to
    float64 there and copied to the host one layer at a time; that
    preparation is not timed (it is reported apart), the oracle's arithmetic
    is.  The prefix keys/values are random bf16 values of the workload's
    shape (their values do not change the oracle's cost)."""
    import numpy as np
    import torch

    import oracle

    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:  # threadpoolctl missing: report the visible cores
        threads = os.cpu_count() or 1

    def host64(t):
        if isinstance(t, tuple):  # a 4-bit matrix: the oracle's dequantisation on the host
            codes, scales = t
            return oracle.dequantize(oracle.unpack_codes(codes.cpu().numpy()), host64(scales), 128)
        return t.double().cpu().numpy()

    cfg = oracle.OracleConfig(shape.n_layers, shape.d_model, shape.n_heads, shape.head_dim, shape.d_ffn,
                              shape.vocab, shape.rms_eps, shape.rope_theta)
    layer = {}
    t_prep = time.perf_counter()
    w = oracle.OracleWeights(cfg, np.zeros((1, shape.d_model)), host64(gen.final_norm()), host64(gen.lm_head()),
                             lambda l: layer[l], cache=False)
    x = host64(gen.tok_embed()[torch.as_tensor(np.asarray(tok, dtype=np.int64), device="cuda")])
    prep = time.perf_counter() - t_prep
    rng = np.random.default_rng(seed)
    H, Dh = shape.n_heads, shape.head_dim
    t_layers, done = 0.0, 0
    for l in range(shape.n_layers):
        t0 = time.perf_counter()
        layer.clear()
        layer[l] = {k: host64(v) for k, v in gen.layer(l).items()}
        pk = oracle.bf16_round(rng.standard_normal((P, H, Dh)))
        pv = oracle.bf16_round(rng.standard_normal((P, H, Dh)))
        t1 = time.perf_counter()
        _, x, _, _ = oracle.tree_layer(w, l, x, pk, pv, parent, rounding=True)
        t2 = time.perf_counter()
        prep += t1 - t0
        t_layers += t2 - t1
        done += 1
        if t_layers >= budget_s:
            break
    t0 = time.perf_counter()
    oracle.logits_from_stream(w, x)
    t_head = time.perf_counter() - t0
    layer.clear()
    t_calc = t_layers * shape.n_layers / done + t_head
    log(f"cpu baseline: oracle {t_layers:.1f}s over {done}/{shape.n_layers} layers + {t_head:.1f}s head "
        f"-> {t_calc:.1f}s per pass (+{prep:.1f}s of untimed weight preparation)")
    whole = done == shape.n_layers
    return {
        "value": round(1.0 / t_calc, 6),
        "unit": "passes/s",
        "cores": int(threads),
        "kind": "oracle",
        "sample": ((f"one whole pass of the workload (P={P}, n={len(parent)}): oracle.tree_layer over all "
                    f"{shape.n_layers} layers" if whole else
                    f"a pass of the workload (P={P}, n={len(parent)}) with oracle.tree_layer timed on its first "
                    f"{done} of {shape.n_layers} layers ({t_layers:.1f}s) and the mean scaled to all layers") +
                   f", then the final norm and LM head, float64 NumPy with the bf16 rounding points; weight "
                   f"conversion ({prep:.1f}s, untimed) excluded; BLAS threads {threads}, host cores visible "
                   f"{os.cpu_count()}"),
    }


def decode_loop(sess, shape, P, parent, tok, iterations=12, planted=4):
    """The generate-and-verify loop (verify, roll back, continue) on the bench
    workload's tree.  Before each iteration the target's own greedy
    continuation from the loop's current context is taken from one-node
    passes (plain greedy decoding, checked against the tree pass's argmax;
    untimed), and `planted` of its tokens are planted along one deepest
    branch of the tree, the other nodes uniform.
    Timed per iteration: the verification pass, the rollback kernel and the
    read-back of accept_len / next token that the host needs for the next
    tree.  Also times the rollback kernel alone."""
    import numpy as np
    import torch

    import workloads

    n = len(parent)
    leaf = n - 1
    chain = []  # the planted branch, root .. leaf
    i = leaf
    while i != -1:
        chain.append(i)
        i = int(parent[i])
    chain = chain[::-1]
    depth = min(planted, len(chain) - 1)

    def greedy_from(plen, root, k):
        out = []
        for t in range(k):
            sess.verify_tree(plen + t, np.array([root]), np.array([-1]), want_logits=False)
            root = sess.outcome()[2]
            out.append(root)
        return out

    def plant(plen, root, it):
        # One-node passes and the tree pass add their partial sums in
        # different orders, so at near-ties (common with random weights)
        # their greedy tokens can differ: check the planted tokens against the
        # tree pass's own argmax and fix the first that differs, until none do.
        cont = greedy_from(plen, root, planted + 1)
        for _ in range(depth + 1):
            ptok = workloads.draft_tree(parent, root, cont, planted, leaf, shape.vocab, seed=it)
            sess.verify_tree(plen, ptok, parent, want_logits=True)
            sess.outcome()
            amax = sess.logits[:n].argmax(dim=1).cpu().numpy()
            bad = [d for d in range(depth) if int(amax[chain[d]]) != int(cont[d])]
            if not bad:
                break
            cont[bad[0]] = int(amax[chain[bad[0]]])
        return ptok

    plen, root = P, int(tok[0])
    accs, t_loop, made = [], 0.0, 0
    last = None
    for it in range(iterations + 1):  # the first iteration warms up
        ptok = plant(plen, root, it)
        torch.cuda.synchronize()
        t = time.perf_counter()
        sess.verify_tree(plen, ptok, parent, want_logits=False)
        sess.commit(plen, n)
        path, acc, nxt = sess.outcome()
        dt = time.perf_counter() - t
        if it > 0:
            t_loop += dt
            made += acc + 1
            accs.append(acc)
        last = (plen, path)
        plen, root = plen + acc + 1, nxt
    # rollback kernel alone: the last tree's accepted rows, moved again
    # (the same rows, the same bytes)
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    reps = 50
    e0.record(stream)
    for _ in range(reps):
        sess.commit(last[0], n)
    e1.record(stream)
    torch.cuda.synchronize()
    commit_us = e0.elapsed_time(e1) * 1e3 / reps
    moved = sum(1 for k, i in enumerate(last[1]) if i != k)
    commit_bytes = 2 * 2 * moved * shape.n_layers * shape.n_heads * shape.head_dim * 2  # K+V, read+write
    log(f"decode loop: {made} tokens in {iterations} passes, {t_loop * 1e3:.1f} ms; rollback {commit_us:.1f} us "
        f"for {moved} rows per layer and head")
    draft_tree = draft_generation(sess, plen, root, iterations)
    return {
        "tokens_per_s": round(made / t_loop, 1),
        "passes": iterations,
        "tokens_per_pass": round(made / iterations, 3),
        "ms_per_iteration": round(t_loop * 1e3 / iterations, 4),
        "accept_lens": accs,
        "draft": (f"{n}-node tree of the workload; {planted} tokens of the target's own greedy continuation "
                  f"(one-node passes from the loop's context, checked against the tree pass's own argmax; "
                  f"untimed) planted along one depth-{planted} branch, the other nodes uniform"),
        "iteration": "verify pass + rollback kernel + read back accept_len / next token (host sync)",
        "commit_us": round(commit_us, 2),
        "commit_rows_moved": moved,
        "commit_bytes": commit_bytes,
        "draft_tree": draft_tree,
    }


def draft_generation(sess, plen, root, iterations, threshold=0.3):
    """Draft-side tree generation with this model as the draft (in the
    paper's LLaMA2 pair the 7B model drafts for the 13B): `iterations` fed
    nodes after the root, one tree-decoder step each (with the candidate
    summary: the argmax and the tokens above the threshold come back, not the
    logits row), the branch pacer run on the host between steps.  Also times
    one step alone (the step's launch on the stream, no read-back); the
    difference per step is the host's share (read-back, pacer, launch)."""
    import numpy as np
    import torch

    from paper_2309_04255_amd import binding, draft

    draft.generate_tree(sess, plen, root, iterations, threshold)  # warm-up
    torch.cuda.synchronize()
    t = time.perf_counter()
    tok, par, info = draft.generate_tree(sess, plen, root, iterations, threshold)
    dt = time.perf_counter() - t
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    reps = 20
    ftok, fpar = np.asarray(tok[:info["fed"]]), np.asarray(par[:info["fed"]])
    cand = torch.zeros((1, binding.CAND_WORDS), dtype=torch.int32, device="cuda")
    e0.record(stream)
    for _ in range(reps):
        binding.extend_tree_candidates(sess.cfg, sess.packed, sess.k_cache, sess.v_cache, plen, ftok, fpar,
                                       len(ftok) - 1, threshold, sess.logits, cand, sess.workspace)
    e1.record(stream)
    torch.cuda.synchronize()
    step_us = e0.elapsed_time(e1) * 1e3 / reps
    steps = info["fed"]
    host_us = (dt * 1e6 - steps * step_us) / steps
    log(f"draft tree: {steps} steps in {dt * 1e3:.1f} ms, {len(tok)} nodes; one step {step_us:.1f} us on the "
        f"device, {host_us:.1f} us of host per step")
    return {
        "iterations": iterations,
        "threshold": threshold,
        "nodes": len(tok),
        "ms": round(dt * 1e3, 3),
        "step_us": round(step_us, 2),
        "host_us_per_step": round(host_us, 1),
        "what": ("one tree-decoder step per fed node (this model as the draft), its candidate summary read back "
                 "and the branch pacer on the host; step_us: one step's kernel time at the last fed node; "
                 "host_us_per_step: the rest of each step (read-back, pacer, launch)"),
    }


def concurrent_draft(sess, shape, P, parent, tok, draft_model, reps=20):
    """The speculative pipeline's overlap on one GPU (§3.4 runs draft
    generation while the target verifies): a draft model's tree-decoder steps
    issued on a second stream (default priority) while the target's
    verification passes run on the first.  Every pass is one cooperative
    launch with one workgroup per CU.  Times `reps` pairs (one verification
    pass of the workload, one draft step: node 12 of a 12-node chain at the
    same prefix length) issued one after the other on one stream, on two
    streams with the whole grid each, and on two streams with the grid split
    (the target's passes on 3/4 of the CUs, the draft's on 1/4); each alone
    for reference.  Both sessions' pass status is checked after every mode."""
    import numpy as np
    import torch

    import workloads
    from paper_2309_04255_amd import binding

    dshape = workloads.MODELS[draft_model]
    dsess = binding.Session(dshape, capacity=P + 128, max_n=32)
    dgen = workloads.make_weights(dshape, "cuda")
    dsess.load_weights(dgen)
    del dgen
    dsess.prefill(workloads.draw_tokens(P, dshape.vocab, seed=7), 0)
    dsess.check("draft prefill")
    dtok = np.asarray(workloads.draw_tokens(12, dshape.vocab, seed=8))
    dpar = np.arange(-1, 11)
    main, side = torch.cuda.current_stream(), torch.cuda.Stream()
    G = torch.cuda.get_device_properties(0).multi_processor_count
    grids = {"target": None, "draft": None}

    def with_grid(g):
        if g is None:
            os.environ.pop("LLMCAD_PASS_GRID", None)
        else:
            os.environ["LLMCAD_PASS_GRID"] = str(g)

    def verify(stream):
        with_grid(grids["target"])
        binding.verify_tree(sess.cfg, sess.packed, sess.k_cache, sess.v_cache, P, tok, parent, sess.logits,
                            sess.path, sess.accept_len, sess.next_token, sess.workspace, stream=stream)

    def step(stream):
        with_grid(grids["draft"])
        binding.extend_tree(dsess.cfg, dsess.packed, dsess.k_cache, dsess.v_cache, P, dtok, dpar, len(dtok) - 1,
                            dsess.logits, dsess.workspace, stream=stream)

    def run(mode):
        grids["target"], grids["draft"] = (3 * G // 4, G // 4) if mode == "split" else (None, None)
        for _ in range(2):  # warm-up
            verify(main)
            step(side if mode in ("concurrent", "split") else main)
        torch.cuda.synchronize()
        t = time.perf_counter()
        for _ in range(reps):
            if mode != "draft":
                verify(main)
            if mode != "target":
                step(side if mode in ("concurrent", "split") else main)
        torch.cuda.synchronize()
        ms = (time.perf_counter() - t) / reps * 1e3
        with_grid(None)
        sess.check(f"verification pass ({mode})")
        dsess.check(f"draft step ({mode})")
        return round(ms, 4)

    saved_spin = os.environ.get("LLMCAD_SPIN_LIMIT")
    os.environ["LLMCAD_SPIN_LIMIT"] = "400000"  # a pass that cannot gather its grid gives up quickly
    out = {}
    try:
        for m in ("target", "draft", "serial", "concurrent", "split"):
            try:
                out[m] = run(m)
            except binding.LlmcadPassError as e:  # (the workspace was re-initialised by the check)
                torch.cuda.synchronize()
                out[m] = f"failed: {e}"
    finally:
        if saved_spin is None:
            os.environ.pop("LLMCAD_SPIN_LIMIT", None)
        else:
            os.environ["LLMCAD_SPIN_LIMIT"] = saved_spin
        with_grid(None)
    log(f"concurrent draft ({draft_model}): {out}")
    return {
        "draft_model": draft_model,
        "ms_per_pair": out,
        "what": ("ms per (31-node verification pass of the target, one tree-decoder step of the draft): "
                 "target / draft alone, both on one stream (serial), on two streams with the whole grid each "
                 "(concurrent), on two streams with the CUs split 3/4 target, 1/4 draft (split)"),
    }


def setup_model(shape, capacity):
    """Session with the model's packed weights (seeded generator run on the GPU)."""
    import torch

    import workloads
    from paper_2309_04255_amd import binding

    t0 = time.perf_counter()
    sess = binding.Session(shape, capacity=capacity, max_n=128)
    gen = workloads.make_weights(shape, "cuda")
    binding.pack_globals(sess.cfg, gen.tok_embed(), gen.final_norm(), gen.lm_head(), sess.packed)
    pack = binding.pack_layer_q4 if sess.cfg.weight_bits == 4 else binding.pack_layer
    for l in range(shape.n_layers):
        pack(sess.cfg, l, gen.layer(l), sess.packed)
        torch.cuda.synchronize()
        if l % 8 == 7:
            log(f"packed layer {l + 1}/{shape.n_layers}")
    torch.cuda.empty_cache()
    log(f"{shape.name}: weights generated and packed in {time.perf_counter() - t0:.1f}s")
    return sess, gen


def measure(sess, gen, wl, args, headline):
    """The bench line of one workload on a session holding its model."""
    import torch

    import workloads
    from paper_2309_04255_amd import binding

    shape = wl.shape
    P = wl.prefix_len
    parent, tok = workloads.make_tree(wl.tree, shape.vocab, wl.seed)
    n = len(parent)
    t0 = time.perf_counter()
    sess.prefill(workloads.draw_tokens(P, shape.vocab, seed=wl.seed), 0)
    sess.check("prefill")
    log(f"{wl.name}: {P}-token prefill {time.perf_counter() - t0:.2f}s")

    def one_pass():
        binding.verify_tree(sess.cfg, sess.packed, sess.k_cache, sess.v_cache, P, tok, parent,
                            sess.logits, sess.path, sess.accept_len, sess.next_token, sess.workspace)

    if args.calibration_copy_mib > 0:
        src = torch.ones(args.calibration_copy_mib << 18, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    for _ in range(args.warmup):
        one_pass()
    sess.outcome()

    # The timed steps: a pass and the read-back of its result (status, path,
    # accept_len, next token: what a decode loop waits for before its next
    # tree), back to back.  Inputs (weights, KV cache, tree) are resident.
    torch.cuda.synchronize()
    step_s = []
    w0 = time.perf_counter()
    for _ in range(args.steps):
        t = time.perf_counter()
        one_pass()
        sess.outcome()
        step_s.append(time.perf_counter() - t)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    ms_per_pass = 1e3 * wall / args.steps
    value = args.steps / wall
    reps = [1e3 * sum(step_s[i:i + 50]) / len(step_s[i:i + 50]) for i in range(0, len(step_s), 50)]
    log(f"{wl.name}: timed {args.steps} passes with read-back: {wall * 1e3:.1f} ms -> {ms_per_pass:.3f} ms/pass "
        f"(per 50-pass repetition: {[round(r, 4) for r in reps]})")

    # Dominant kernel: the pass kernel itself, timed per launch with HIP events
    # recorded by the library on the stream it launches on, over the same
    # number of back-to-back passes in the same launch configuration.
    B = pass_bytes(shape, P, n)
    binding.timing_enable(binding.KERNEL_PASS, args.steps)
    stream = torch.cuda.current_stream()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record(stream)
    for _ in range(args.steps):
        one_pass()
    ev1.record(stream)
    sess.outcome()
    tot_ms, nl = binding.timing_read(binding.KERNEL_PASS)
    binding.timing_enable(-1, 0)
    back_to_back_ms = ev0.elapsed_time(ev1) / args.steps
    k_ms = tot_ms / max(nl, 1)
    k_achieved = B / (k_ms / 1e3)
    log(f"{wl.name}: pass kernel {nl} launches, mean {k_ms * 1e3:.1f} us, {k_achieved / 1e9:.0f} GB/s; "
        f"back to back {back_to_back_ms * 1e3:.1f} us per pass")

    decode = decode_loop(sess, shape, P, parent, tok) if headline and not args.no_decode_loop else None

    frac = B / (wall / args.steps) / HBM_PEAK
    traffic = load_traffic(wl.name)
    q4 = ("4-bit codes, one bf16 scale per 128 inputs (GPTQ-style symmetric groups); bf16 MFMA on the codes"
          if getattr(shape, "weight_bits", 16) == 4 else None)
    out = {
        "metric": METRIC,
        "value": round(value, 3),
        "unit": "passes/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_pass, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": ("synthetic: random-init bf16 weights (counter-hash Irwin-Hall, std 0.02), uniform tokens"
                 if q4 is None else
                 "synthetic: random-init 4-bit layer weights (uniform codes, bf16 group scales, spread 0.02), "
                 "bf16 embedding / LM head, uniform tokens"),
        "config": {
            "workload": wl.name,
            "shape": f"L{shape.n_layers} d{shape.d_model} H{shape.n_heads}x{shape.head_dim} "
                     f"F{shape.d_ffn} V{shape.vocab}",
            "weights": "bf16" if q4 is None else q4,
            "prefix_len": P,
            "tree_nodes": n,
            "tree": str(wl.tree),
        },
        "step": "one verification pass + read-back of status / path / accept_len / next token (host sync)",
        "tree_tokens_per_s": round(value * n, 1),
        "hbm_roofline_frac": round(frac, 4),
        "pass_alg_bytes": B,
        "ms_per_step_median_of_reps": round(statistics.median(reps), 4),
        "reps_ms_per_step": [round(r, 4) for r in reps],
        "ms_per_pass_back_to_back": round(back_to_back_ms, 4),
        "roofline": {
            "bound": "hbm",
            "kernel": "pass_kernel (persistent: embed, per layer QKV / attention / O / gate-up / down, LM head, walk)",
            "achieved": round(k_achieved / 1e9, 1),
            "peak": HBM_PEAK / 1e9,
            "unit": "GB/s",
            "frac": round(k_achieved / HBM_PEAK, 4),
            "traffic": traffic,
            "alg_bytes_per_launch": B,
            "mean_launch_us": round(k_ms * 1e3, 2),
        },
    }
    if decode is not None:
        out["decode_loop"] = decode
    if not args.no_cpu_baseline and (headline or args.cpu_baseline_all):
        log(f"{wl.name}: timing the CPU oracle (one whole pass)")
        out["cpu_baseline"] = cpu_baseline(gen, shape, P, parent, tok, wl.seed)
    return out


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=250)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="llama7b_p512_n31",
                    help="workload name, or several separated by commas (one JSON line each, in order)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-baseline-all", action="store_true",
                    help="time the CPU oracle for every workload, not only the first")
    ap.add_argument("--no-decode-loop", action="store_true",
                    help="skip the generate-and-verify loop measurement")
    ap.add_argument("--calibration-copy-mib", type=int, default=0,
                    help="(profiling) first copy this many MiB three times: the counter calibration")
    ap.add_argument("--concurrent-draft", metavar="DRAFT_MODEL", default=None,
                    help="also time draft steps of DRAFT_MODEL on a second stream beside the first workload's passes")
    ap.add_argument("--write-traffic", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="write the traffic file from two rocprofv3 --pmc counter CSVs and exit")
    args = ap.parse_args()
    if args.write_traffic:
        write_traffic(args.write_traffic[0], args.write_traffic[1], args.workload,
                      args.calibration_copy_mib or 1024)
        return
    if args.gpus != 1:
        print("bench.py measures a single GPU: this build has no multi-GPU path "
              "(run with --gpus 1).", file=sys.stderr)
        sys.exit(2)

    import faulthandler
    import gc

    import torch

    import workloads
    from paper_2309_04255_amd import binding

    faulthandler.enable()
    if not torch.cuda.is_available():
        print("bench.py needs a ROCm GPU", file=sys.stderr)
        sys.exit(1)
    torch.cuda.set_device(0)
    names = [w for w in args.workload.split(",") if w]
    wls = [workloads.get_workload(w) for w in names]
    sess = gen = None
    model = None
    for i, wl in enumerate(wls):
        if wl.model != model:
            sess = gen = None
            gc.collect()
            torch.cuda.empty_cache()
            cap = max(w.prefix_len for w in wls if w.model == wl.model) + 128
            sess, gen = setup_model(wl.shape, cap)
            model = wl.model
        line = measure(sess, gen, wl, args, headline=i == 0)
        if i == 0 and args.concurrent_draft:
            parent, tok = workloads.make_tree(wl.tree, wl.shape.vocab, wl.seed)
            line["concurrent_draft"] = concurrent_draft(sess, wl.shape, wl.prefix_len, parent, tok,
                                                        args.concurrent_draft)
        print(json.dumps(line), flush=True)
    # Leave nothing of the library's behind for the interpreter's exit: no
    # timing events, no device buffers, no work in flight.
    binding.timing_enable(-1, 0)
    sess = gen = None
    gc.collect()
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    log("done")


if __name__ == "__main__":
    main()
