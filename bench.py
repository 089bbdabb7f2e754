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
    """Algorithmic HBM bytes of one pass: every weight byte once (embedding: n
    rows), prefix K+V read once, tree K/V written, embedding rows, fp32 logits."""
    L, d, F, V = shape.n_layers, shape.d_model, shape.d_ffn, shape.vocab
    weights = 2 * (L * (4 * d * d + 3 * d * F + 2 * d) + V * d + d)
    return weights + 4 * L * P * d + 4 * L * n * d + 2 * n * d + 4 * n * V


def source_hash():
    h = hashlib.sha256()
    for path in KERNEL_SOURCES:
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def load_traffic(workload):
    """Measured HBM bytes per pass-kernel launch (FETCH_SIZE + WRITE_SIZE,
    calibrated against a copy kernel), or None when the counters were taken
    on other kernel sources or another workload."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("kernel_sources_sha256_16") != source_hash() or t.get("workload") != workload:
        return None
    return t.get("bytes_per_launch")


def write_traffic(fetch_csv, write_csv, workload, copy_mib):
    """From two rocprofv3 --pmc runs of `bench.py --calibration-copy-mib N`
    (one collecting FETCH_SIZE, one WRITE_SIZE; per dispatch, in KiB), the
    pass kernel's HBM bytes per launch.  Calibration: the N MiB fill that
    precedes the copy writes a known size (write factor), and the copy's
    chunks read as much as they write (read factor).  Writes TRAFFIC_FILE
    tagged with the kernel sources' hash."""
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
    # (the prefill's passes run another instance of the pass kernel, for
    # 128-row chunks; the verification passes are the most frequent one)
    passk = max((k for k in fetch if "pass_kernel" in k), key=lambda k: len(fetch[k]))
    f_kib, w_kib = statistics.mean(fetch[passk]), statistics.mean(write[passk])
    out = {
        "workload": workload, "kernel_sources_sha256_16": source_hash(), "kernel": passk[:90],
        "launches": len(fetch[passk]), "fetch_kib_mean": round(f_kib), "write_kib_mean": round(w_kib),
        "calibration": {"fill_mib": copy_mib, "fill_write_kib": fill_kib, "write_factor": round(write_factor, 4),
                        "copy_chunk_fetch_kib": chunk_fetch, "copy_chunk_write_kib": chunk_write,
                        "read_factor": round(read_factor, 4)},
        "read_bytes": round(f_kib * 1024 * read_factor), "write_bytes": round(w_kib * 1024 * write_factor),
    }
    out["bytes_per_launch"] = out["read_bytes"] + out["write_bytes"]
    with open(TRAFFIC_FILE, "w") as f:
        json.dump(out, f, indent=1)
        f.write("\n")
    print(json.dumps(out, indent=1))


def cpu_baseline(shape, P, n, seed):
    """Time the CPU oracle on a bounded sample: tree_forward with 1 and 2 of the
    model's layers (+ embedding and LM head); one pass = t1 + (L-1)(t2 - t1)."""
    import numpy as np

    import oracle
    import workloads

    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:  # threadpoolctl missing: report the visible cores
        threads = os.cpu_count() or 1
    gen = workloads.make_weights(shape, "cpu")

    def np64(t):
        return t.float().numpy().astype(np.float64)

    t0 = time.perf_counter()
    layers = {l: {k: np64(v) for k, v in gen.layer(l).items()} for l in (0, 1)}
    emb, fin, head = np64(gen.tok_embed()), np64(gen.final_norm()), np64(gen.lm_head())
    log(f"cpu baseline: weights for 2 layers converted in {time.perf_counter() - t0:.1f}s")
    rng = np.random.default_rng(seed)
    H, Dh = shape.n_heads, shape.head_dim
    pk = oracle.bf16_round(rng.standard_normal((2, P, H, Dh)))
    pv = oracle.bf16_round(rng.standard_normal((2, P, H, Dh)))
    parent, tok = workloads.make_tree(("complete", (2, 2, 2, 2)), shape.vocab, seed) \
        if n == 31 else workloads.make_tree(("random", n, 7), shape.vocab, seed)

    def run(nl):
        cfg = oracle.OracleConfig(nl, shape.d_model, shape.n_heads, shape.head_dim, shape.d_ffn,
                                  shape.vocab, shape.rms_eps, shape.rope_theta)
        w = oracle.OracleWeights(cfg, emb, fin, head, lambda l: layers[l])
        w.layer(0)
        if nl > 1:
            w.layer(1)
        t = time.perf_counter()
        oracle.tree_forward(w, pk[:nl], pv[:nl], tok, parent, rounding=True)
        return time.perf_counter() - t

    reps = []
    for _ in range(3):
        t1, t2 = run(1), run(2)
        reps.append((t1, t2))
    t1 = statistics.median(r[0] for r in reps)
    t2 = statistics.median(r[1] for r in reps)
    per_pass = t1 + (shape.n_layers - 1) * max(t2 - t1, 0.0)
    log(f"cpu baseline: 1 layer {t1:.2f}s, 2 layers {t2:.2f}s -> {per_pass:.1f}s per pass")
    return {
        "value": 1.0 / per_pass,
        "unit": "passes/s",
        "cores": int(threads),
        "kind": "oracle",
        "sample": (f"oracle.tree_forward (float64 NumPy, bf16 storage rounding) with layers 0 and 1 "
                   f"of the {shape.n_layers}-layer model plus embedding and LM head, P={P}, n={n}; "
                   f"median of 3; pass = t(1 layer) + {shape.n_layers - 1} x (t(2) - t(1)); "
                   f"host cores visible: {os.cpu_count()}"),
    }


def decode_loop(sess, shape, P, parent, tok, iterations=12, planted=4):
    """The generate-and-verify loop (verify, roll back, continue) on the bench
    workload's tree.  Before each iteration the target's own greedy
    continuation from the loop's current context is taken from one-node
    passes (plain greedy decoding, untimed), and `planted` of its tokens are
    planted along one deepest branch of the tree, the other nodes uniform.
    Timed per iteration: the verification pass, the rollback kernel and the
    read-back of accept_len / next token that the host needs for the next
    tree.  Also times the rollback kernel alone."""
    import numpy as np
    import torch

    import workloads

    n = len(parent)
    leaf = n - 1

    def greedy_from(plen, root, k):
        out = []
        for t in range(k):
            sess.verify_tree(plen + t, np.array([root]), np.array([-1]), want_logits=False)
            root = int(sess.next_token.item())
            out.append(root)
        return out

    plen, root = P, int(tok[0])
    accs, t_loop, made = [], 0.0, 0
    last = None
    for it in range(iterations + 1):  # the first iteration warms up
        cont = greedy_from(plen, root, planted + 1)
        ptok = workloads.draft_tree(parent, root, cont, planted, leaf, shape.vocab, seed=it)
        torch.cuda.synchronize()
        t = time.perf_counter()
        sess.verify_tree(plen, ptok, parent, want_logits=False)
        sess.commit(plen, n)
        acc = int(sess.accept_len.item())
        nxt = int(sess.next_token.item())
        dt = time.perf_counter() - t
        if it > 0:
            t_loop += dt
            made += acc + 1
            accs.append(acc)
        last = (plen, [int(x) for x in sess.path[: acc + 1].cpu()])
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
                  f"(one-node passes from the loop's context, untimed) planted along one depth-{planted} "
                  f"branch, the other nodes uniform"),
        "iteration": "verify pass + rollback kernel + read back accept_len / next token (host sync)",
        "commit_us": round(commit_us, 2),
        "commit_rows_moved": moved,
        "commit_bytes": commit_bytes,
        "draft_tree": draft_tree,
    }


def draft_generation(sess, plen, root, iterations, threshold=0.3):
    """Draft-side tree generation with this model as the draft (in the
    paper's LLaMA2 pair the 7B model drafts for the 13B): `iterations` fed
    nodes after the root, one tree-decoder step each, the logits row read back
    and the branch pacer run on the host between steps.  Also times one
    tree-decoder step alone (the step's launch on the stream, no read-back)."""
    import numpy as np
    import torch

    from paper_2309_04255_amd import draft

    draft.generate_tree(sess, plen, root, iterations, threshold)  # warm-up
    torch.cuda.synchronize()
    t = time.perf_counter()
    tok, par, info = draft.generate_tree(sess, plen, root, iterations, threshold)
    dt = time.perf_counter() - t
    stream = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    reps = 20
    ftok, fpar = np.asarray(tok[:info["fed"]]), np.asarray(par[:info["fed"]])
    e0.record(stream)
    for _ in range(reps):
        sess.extend(plen, ftok, fpar, len(ftok) - 1)
    e1.record(stream)
    torch.cuda.synchronize()
    step_us = e0.elapsed_time(e1) * 1e3 / reps
    log(f"draft tree: {iterations} steps in {dt * 1e3:.1f} ms, {len(tok)} nodes; one step {step_us:.1f} us")
    return {
        "iterations": iterations,
        "threshold": threshold,
        "nodes": len(tok),
        "ms": round(dt * 1e3, 3),
        "step_us": round(step_us, 2),
        "what": ("one tree-decoder step per fed node (this model as the draft), logits row read back and "
                 "threshold + branch pacer on the host; step_us: one step's kernel time at the last fed node"),
    }


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="llama7b_p512_n31")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-decode-loop", action="store_true",
                    help="skip the generate-and-verify loop measurement")
    ap.add_argument("--calibration-copy-mib", type=int, default=0,
                    help="(profiling) first copy this many MiB three times: the counter calibration")
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

    import torch

    import workloads
    from paper_2309_04255_amd import binding

    if not torch.cuda.is_available():
        print("bench.py needs a ROCm GPU", file=sys.stderr)
        sys.exit(1)
    torch.cuda.set_device(0)
    wl = workloads.get_workload(args.workload)
    shape = wl.shape
    P = wl.prefix_len
    parent, tok = workloads.make_tree(wl.tree, shape.vocab, wl.seed)
    n = len(parent)
    prefix = workloads.draw_tokens(P, shape.vocab, seed=wl.seed)

    t0 = time.perf_counter()
    sess = binding.Session(shape, capacity=P + max(n, 128), max_n=128)
    gen = workloads.make_weights(shape, "cuda")
    binding.pack_globals(sess.cfg, gen.tok_embed(), gen.final_norm(), gen.lm_head(), sess.packed)
    for l in range(shape.n_layers):
        binding.pack_layer(sess.cfg, l, gen.layer(l), sess.packed)
        torch.cuda.synchronize()
        if l % 8 == 7:
            log(f"packed layer {l + 1}/{shape.n_layers}")
    torch.cuda.empty_cache()
    sess.prefill(prefix, 0)
    torch.cuda.synchronize()
    log(f"setup (weights, packing, {P}-token prefill) {time.perf_counter() - t0:.1f}s")

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
    torch.cuda.synchronize()

    stream = torch.cuda.current_stream()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(args.steps):
        one_pass()
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    gpu_s = ev0.elapsed_time(ev1) / 1e3
    elapsed = max(wall, gpu_s)
    ms_per_pass = 1e3 * elapsed / args.steps
    value = args.steps / elapsed
    log(f"timed {args.steps} passes: wall {wall * 1e3:.1f} ms, events {gpu_s * 1e3:.1f} ms "
        f"-> {ms_per_pass:.3f} ms/pass")

    # Dominant kernel: the pass kernel itself, timed per launch with HIP events
    # recorded by the library on the stream it launches on, over the same
    # number of passes in the same launch configuration.
    B = pass_bytes(shape, P, n)
    binding.timing_enable(binding.KERNEL_PASS, args.steps)
    for _ in range(args.steps):
        one_pass()
    torch.cuda.synchronize()
    tot_ms, nl = binding.timing_read(binding.KERNEL_PASS)
    binding.timing_enable(-1, 0)
    k_ms = tot_ms / max(nl, 1)
    k_achieved = B / (k_ms / 1e3)
    log(f"pass kernel: {nl} launches, mean {k_ms * 1e3:.1f} us, {k_achieved / 1e9:.0f} GB/s")

    # Latency of a pass when the decode loop waits for the accepted path.
    lat = []
    for _ in range(min(args.steps, 20)):
        t = time.perf_counter()
        one_pass()
        sess.accept_len.cpu()
        lat.append(time.perf_counter() - t)

    decode = None if args.no_decode_loop else decode_loop(sess, shape, P, parent, tok)

    frac = B / (elapsed / args.steps) / HBM_PEAK
    traffic = load_traffic(wl.name)
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
        "data": "synthetic: random-init bf16 weights (counter-hash Irwin-Hall, std 0.02), uniform tokens",
        "config": {
            "workload": wl.name,
            "shape": f"L{shape.n_layers} d{shape.d_model} H{shape.n_heads}x{shape.head_dim} "
                     f"F{shape.d_ffn} V{shape.vocab}",
            "prefix_len": P,
            "tree_nodes": n,
            "tree": str(wl.tree),
        },
        "tree_tokens_per_s": round(value * n, 1),
        "hbm_roofline_frac": round(frac, 4),
        "pass_alg_bytes": B,
        "ms_per_pass_with_readback": round(1e3 * statistics.median(lat), 4),
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
    if not args.no_cpu_baseline:
        log("timing the CPU oracle (bounded sample)")
        out["cpu_baseline"] = cpu_baseline(shape, P, n, wl.seed)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
