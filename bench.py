#!/usr/bin/env python
"""Benchmark of the tree-verification hot path on one MI355X.

Workload: GPT-2-L shape (36 x 1280, 20 heads of 64, MLP 5120, vocab 50257),
random N(0, 0.02) bf16 weights, a synthetic 512-token prefix cache and a
32-node tree (branching 4,2,2,1 breadth-first, truncated), greedy acceptance.
One step = the whole hot path on that input: the captured verification pass
with its greedy accept (the argmax of every node taken from the LM head's
per-workgroup maxima, then the walk down the tree), and the KV commit of the
accepted path (commit rewrites the same rows past the prefix every step, and
verification never reads them, so steps repeat exactly).  `value` is the
tree tokens verified per second of timed steps.  Inputs are resident in HBM
before timing starts.

Also reported: the pass alone and its HBM roofline fraction, the tree-size x
prefix sweep (with both GEMM paths of the one-kernel-per-sub-layer pass and
their crossover), the 256-node / 2048-token stress point with its sampling
accepts timed, staged end-to-end generation (greedy and top-50 sampling),
and the CPU oracle's time on this host.

Prints one JSON line on stdout; progress goes to stderr.
"""
import argparse
import hashlib
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0
METRIC = "µs per tree-verify pass + verified tree tokens/s, GPT-2-L shape; HBM GB/s"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def pass_bytes(cfg, n, P, q8=False):
    """Algorithmic HBM bytes of one verification pass: every parameter once
    (matrices, tied LM head, vectors; the embedding rows gathered are
    negligible), the prefix K/V once, the tree K/V written once and the
    float32 logits written once.  q8: the matrices and the LM head as 8-bit
    codes plus one float32 scale per row (rows padded to 16)."""
    d, m, L, V = cfg.d_model, cfg.d_mlp, cfg.n_layer, cfg.vocab
    es = 2 if cfg.dtype == "bf16" else 4
    mats = L * (3 * d * d + d * d + m * d + d * m) * es
    head = V * d * es
    if q8:
        pad = lambda r: (r + 15) // 16 * 16
        mats = L * (3 * d * d + d * d + m * d + d * m) + L * 4 * (pad(3 * d) + pad(d) + pad(m) + pad(d))
        head = V * d + 4 * pad(V)
    vecs = (L * (2 * d + 3 * d + d + 2 * d + m + d) + 2 * d) * es
    kv_row = L * 2 * d * es
    return mats + head + vecs + kv_row * P + (kv_row + V * 4) * n


def kernel_source_hash(fused=True):
    """Hash of the sources of the dominant kernel: the persistent pass
    (fused.hip) or the per-sub-layer kernels (kernels.hip), with their shared
    header."""
    h = hashlib.sha256()
    for name in ("fused.hip" if fused else "kernels.hip", "ssd_internal.h"):
        with open(os.path.join(ROOT, "paper_2308_04623_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor()


COPY_BYTES = 256 << 20
def fc_kernel(n):
    """The MLP up-projection + GELU GEMM's kernel at n nodes (matrix cores):
    one-or-two-row-block tiles up to 64 nodes, the wide-tree kernel above."""
    return "gemm2d_kernel<2, 2, 2, 4," if n > 64 else "gemm_kernel<2, 2, 2,"
PASS_KERNEL = "pass_kernel"         # the persistent single-launch pass


def probe_traffic(sess, cfg, n, P, toks, par, fused):
    """Kernels for the HBM-traffic counters: a plain device-to-device copy of
    COPY_BYTES (reads and writes exactly that much), then the dominant kernel:
    three verification passes (persistent pass) or the MLP up-projection GEMM
    of every layer twice (one kernel per sub-layer)."""
    import torch
    src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    if fused:
        for _ in range(3):
            sess.verify(P, toks, par)
    else:
        for _ in range(2):
            for l in range(cfg.n_layer):
                sess.launch_gemm(2, l, n)
    torch.cuda.synchronize()
    log("traffic probe done")


def _counter_rows(d):
    import csv
    import glob
    files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no counter_collection.csv under {d}")
    rows = []
    for f in files:
        with open(f, newline="") as fh:
            rows += list(csv.DictReader(fh))
    return rows


def _per_kernel(rows, counter):
    """{(kernel name, grid size): [value per dispatch]} for one counter
    (values summed over the rows of a dispatch)."""
    per = {}
    for r in rows:
        if r.get("Counter_Name") != counter:
            continue
        key = (r.get("Dispatch_Id"), r.get("Kernel_Name", ""), int(r.get("Grid_Size", 0) or 0))
        per[key] = per.get(key, 0.0) + float(r["Counter_Value"])
    out = {}
    for (_, name, grid), v in per.items():
        out.setdefault((name, grid), []).append(v)
    return out


def traffic_path(fused):
    return os.path.join(ROOT, "profiles", "traffic_pass_kernel.json" if fused else "traffic_fc_gemm.json")


def write_traffic(fetch_dir, write_dir, n, fused):
    kname = PASS_KERNEL if fused else fc_kernel(n)
    out = {"kernel_source": kernel_source_hash(fused), "kernel": kname, "nodes": n, "copy_bytes": COPY_BYTES}
    for counter, d in (("FETCH_SIZE", fetch_dir), ("WRITE_SIZE", write_dir)):
        per = _per_kernel(_counter_rows(d), counter)
        # the probe's copy is the largest-grid copy kernel of the run (set-up copies are small)
        grids = [g for (k, g) in per if "copyBuffer" in k]
        copy = [v for (k, g), vs in per.items() if "copyBuffer" in k and grids and g == max(grids) for v in vs]
        kern = [v for (k, g), vs in per.items() if kname in k for v in vs]
        if not copy or not kern:
            raise SystemExit(f"{counter}: copy or {kname} dispatches missing ({sorted(per)})")
        copy_kib = sorted(copy)[len(copy) // 2]
        scale = COPY_BYTES / (copy_kib * 1024.0)  # bytes per counted KiB unit, from the copy of known size
        k_kib = sum(kern) / len(kern)
        out[counter.lower()] = {"copy_kib_per_dispatch": copy_kib, "kernel_kib_per_dispatch": round(k_kib, 1),
                                "scale": round(scale, 4), "kernel_bytes_per_launch": round(k_kib * 1024 * scale),
                                "kernel_dispatches": len(kern)}
    out["bytes_per_launch"] = (out["fetch_size"]["kernel_bytes_per_launch"]
                               + out["write_size"]["kernel_bytes_per_launch"])
    with open(traffic_path(fused), "w") as fh:
        json.dump(out, fh, indent=1)
    print(json.dumps(out))


def stored_traffic(fused, n):
    """HBM bytes per launch from the committed counter runs, or None when they
    were taken on other kernel sources or another node count."""
    path = traffic_path(fused)
    if not os.path.exists(path):
        return None
    t = json.load(open(path))
    if t.get("kernel_source") == kernel_source_hash(fused) and t.get("nodes") == n:
        return t.get("bytes_per_launch")
    return None


def write_mfma(counter_dir, trace_dir, n, P, cmd_pmc, cmd_trace):
    """Matrix-core use of the weight GEMMs from a rocprofv3 --pmc run
    (MfmaUtil, MfmaFlopsF16 per dispatch) and a --kernel-trace --stats run of
    the same command (average durations): profiles/mfma_gemm_n{n}_p{P}.md."""
    import csv
    import glob
    rows = _counter_rows(counter_dir)
    util = _per_kernel(rows, "MfmaUtil")
    flops = _per_kernel(rows, "MfmaFlopsF16")
    avg = {}
    for f in glob.glob(os.path.join(trace_dir, "**", "*kernel_stats.csv"), recursive=True):
        for r in csv.DictReader(open(f, newline="")):
            avg[r["Name"]] = float(r["AverageNs"]) * 1e-3
    lines = [f"# Matrix-core use of the weight GEMMs: GPT-2-L shape, {n} nodes, {P}-token prefix", "",
             "Commands (repo root, one MI355X; `TMPDIR=/tmp`):", "", f"    {cmd_pmc}", f"    {cmd_trace}",
             f"    python bench.py --mfma-from {counter_dir} {trace_dir} --nodes {n} --prefix {P}", "",
             "MfmaUtil = matrix-core busy cycles / (GPU active cycles x 1024 SIMDs); FLOPs are rocprofv3's "
             "MfmaFlopsF16 (512 per MOPS count). TFLOP/s = FLOPs per dispatch / the kernel's average duration "
             "in the trace run; the dense float16 peak is 2500 TFLOP/s.", "",
             "| kernel | dispatches | MfmaUtil % | GFLOP per dispatch | avg us | TFLOP/s | of peak |",
             "|---|---|---|---|---|---|---|"]
    for (name, grid), us in sorted(util.items(), key=lambda kv: -sum(kv[1])):
        fl = flops.get((name, grid), [0.0])
        f_avg = sum(fl) / len(fl)
        t = next((v for k, v in avg.items() if k.split("(")[0] == name.split("(")[0]), None)
        tf = f_avg / (t * 1e-6) / 1e12 if t else None
        short = name.split("(")[0]
        lines.append(f"| `{short}` (grid {grid}) | {len(us)} | {sum(us) / len(us):.2f} | {f_avg / 1e9:.3f} | "
                     f"{t if t is None else round(t, 2)} | {'' if tf is None else round(tf, 1)} | "
                     f"{'' if tf is None else f'{tf / 2500 * 100:.2f}%'} |")
    text = "\n".join(lines) + "\n"
    with open(os.path.join(ROOT, "profiles", f"mfma_gemm_n{n}_p{P}.md"), "w") as fh:
        fh.write(text)
    print(text)


def fc_gemm_roofline(sess, cfg, N, stream):
    """Dominant kernel of the one-kernel-per-sub-layer path: the MLP
    up-projection GEMM (13.1 MB of weights per launch), launched on its own
    for every layer in turn so its weights stream from HBM, captured in a
    graph so host launch rate does not limit it; HIP events on the stream it
    runs on."""
    import torch
    fc_graph = torch.cuda.CUDAGraph()
    cap = torch.cuda.Stream()
    cap.wait_stream(stream)
    with torch.cuda.stream(cap):
        for l in range(cfg.n_layer):  # warm-up outside the graph
            sess.launch_gemm(2, l, N)
        cap.synchronize()
        with torch.cuda.graph(fc_graph, stream=cap):
            for l in range(cfg.n_layer):
                sess.launch_gemm(2, l, N)
    torch.cuda.synchronize()
    reps = 10
    for _ in range(3):
        fc_graph.replay()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record(stream)
    for _ in range(reps):
        fc_graph.replay()
    b.record(stream)
    torch.cuda.synchronize()
    us_fc = a.elapsed_time(b) * 1e3 / (reps * cfg.n_layer)
    fc_bytes = cfg.d_mlp * cfg.d_model * 2 + N * cfg.d_model * 2 + N * cfg.d_mlp * 2
    fc_gbs = fc_bytes / us_fc / 1e3
    return {"bound": "hbm", "achieved": round(fc_gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
            "frac": round(fc_gbs / PEAK_HBM_GBS, 4), "traffic": stored_traffic(False, N),
            "kernel": "gemm (MLP up-projection + GELU), 5120x1280 bf16",
            "bytes_per_launch": fc_bytes, "us_per_launch": round(us_fc, 2)}


def end_to_end(ssd, W, cfg, model, N_NEW, PROMPT):
    """Staged greedy generation of N_NEW tokens from a PROMPT-token random
    prompt (draft: the oracle's first 4 layers; draft^2: bigram table), and
    plain greedy decoding of the same, wall clock including host work."""
    import numpy as np
    import torch
    from paper_2308_04623_amd import staged as S
    draft = model.prefix_view(4)
    prompt = W.prefix_tokens(PROMPT, cfg.vocab, seed=5)
    max_ctx = PROMPT + N_NEW + 80

    def backend(record_gaps=False):
        o = ssd.Session(model, max_ctx, S.MAX_ORACLE_NODES)
        d = ssd.Session(draft, max_ctx, 256, o.k_cache, o.v_cache)
        b = S.GpuBackend(o, d, record_gaps)
        return b, b.prefill(prompt[:-1])

    b_plain, P = backend()
    plain = S.plain_greedy(b_plain, P, int(prompt[-1]), N_NEW)
    b_st, P2 = backend()
    t0 = time.perf_counter()
    succ = S.build_bigram_gpu(b_st, cfg.vocab)
    t_bigram = time.perf_counter() - t0
    st = S.staged_greedy(b_st, P2, int(prompt[-1]), N_NEW, succ)
    agree = next((i for i, (a, b) in enumerate(zip(st.tokens, plain.tokens)) if a != b), N_NEW)
    gap = None
    if agree < N_NEW:
        # untimed replay of plain decoding up to the divergence, recording the
        # top-2 logit gap of each step: a gap under 1e-3 is a precision tie
        # between the two verification shapes, anything larger a real mismatch
        b_gap, P3 = backend(record_gaps=True)
        S.plain_greedy(b_gap, P3, int(prompt[-1]), agree + 1)
        gap = b_gap.gaps[agree]
    # the same reusing the draft's work: the oracle verifies the endorsed
    # subtree only, from layer 4 on
    b_r, P8 = backend()
    st_r = S.staged_greedy_reuse(b_r, P8, int(prompt[-1]), N_NEW, succ)
    agree_r = next((i for i, (a, b) in enumerate(zip(st_r.tokens, plain.tokens)) if a != b), N_NEW)
    log(f"end to end, greedy with draft reuse: staged {N_NEW / st_r.seconds:.1f} tok/s, accepted "
        f"{sum(st_r.accepted)} in {st_r.steps} steps, agree {agree_r}/{N_NEW}")
    # the same with top-k sampling (k = 50, T = 1): plain steps draw from the
    # oracle's top-k target; staged steps accept the draft's chosen children
    # by rejection sampling against it, so both emit that law (Sec. 2.3)
    b_ps, P4 = backend()
    plain_s = S.plain_sample(b_ps, P4, int(prompt[-1]), N_NEW, top_k=50, seed0=11)
    b_ss, P5 = backend()
    st_s = S.staged_sample(b_ss, P5, int(prompt[-1]), N_NEW, succ, top_k=50, seed0=11)
    log(f"end to end, top-50 sampling: plain {N_NEW / plain_s.seconds:.1f} tok/s, staged "
        f"{N_NEW / st_s.seconds:.1f} tok/s, accepted {sum(st_s.accepted)} in {st_s.steps} steps")
    # CDF-first sampling over the whole vocabulary at T = 1: uniforms drawn
    # first, trees assembled from the draft's inverse-CDF picks around them
    # (SSD_ACCEPT_SAMPLE_CDF); plain steps draw from the same target
    b_pc, P6 = backend()
    plain_c = S.plain_sample(b_pc, P6, int(prompt[-1]), N_NEW, top_k=0, seed0=13)
    b_sc, P7 = backend()
    st_c = S.staged_sample_cdf(b_sc, P7, int(prompt[-1]), N_NEW, succ, temperature=1.0, seed0=13)
    log(f"end to end, CDF-first sampling: plain {N_NEW / plain_c.seconds:.1f} tok/s, staged "
        f"{N_NEW / st_c.seconds:.1f} tok/s, accepted {sum(st_c.accepted)} in {st_c.steps} steps")
    log(f"end to end: plain {N_NEW / plain.seconds:.1f} tok/s, staged {N_NEW / st.seconds:.1f} tok/s, "
        f"accepted {sum(st.accepted)} in {st.steps} steps, agree {agree}/{N_NEW}"
        + ("" if gap is None else f", plain top-2 gap at the divergence {gap:.3g}"))
    return {"workload": f"greedy generation of {N_NEW} tokens from a {PROMPT}-token random prompt; draft = first 4 "
                        "layers + shared head, draft^2 = bigram table (2^15-token stream); oracle trees <= 64 nodes",
            "plain_tokens_per_s": round(N_NEW / plain.seconds, 1), "staged_tokens_per_s": round(N_NEW / st.seconds, 1),
            "staged_steps": st.steps, "accepted_tree_tokens": int(sum(st.accepted)),
            "mean_oracle_tree_nodes": round(float(np.mean(st.oracle_nodes)), 1),
            "mean_endorsed_nodes": round(float(np.mean(st.endorsed)), 2),
            "tokens_equal_to_plain": agree,
            "plain_top2_gap_at_divergence": None if gap is None else round(gap, 6),
            "bigram_build_s": round(t_bigram, 2),
            "top50_sampling": {"plain_tokens_per_s": round(N_NEW / plain_s.seconds, 1),
                               "staged_tokens_per_s": round(N_NEW / st_s.seconds, 1), "staged_steps": st_s.steps,
                               "accepted_tree_tokens": int(sum(st_s.accepted)),
                               "mean_oracle_tree_nodes": round(float(np.mean(st_s.oracle_nodes)), 1)},
            "greedy_draft_reuse": {"staged_tokens_per_s": round(N_NEW / st_r.seconds, 1), "staged_steps": st_r.steps,
                                   "accepted_tree_tokens": int(sum(st_r.accepted)),
                                   "mean_oracle_tree_nodes": round(float(np.mean(st_r.oracle_nodes)), 1),
                                   "tokens_equal_to_plain": agree_r},
            "cdf_first_sampling": {"plain_tokens_per_s": round(N_NEW / plain_c.seconds, 1),
                                   "staged_tokens_per_s": round(N_NEW / st_c.seconds, 1),
                                   "staged_steps": st_c.steps, "accepted_tree_tokens": int(sum(st_c.accepted)),
                                   "mean_oracle_tree_nodes": round(float(np.mean(st_c.oracle_nodes)), 1)}}


STAGES = ["LN1", "QKV", "ATT", "WO", "LN2", "FC", "WPR"]
CROSS_XCD = {0, 4}  # stages whose inputs come from all 8 XCDs


def stage_trace(sess, cfg, N, P, toks, par, us_pass):
    """Record one persistent pass's stage timestamps (ssd_kv_set_trace) and
    write a summary per stage to profiles/stage_trace_n{N}_p{P}.md: per XCD
    and layer (layers 2..L-2), the hand-off (last producer published -> first
    consumer's dependency met), the met skew inside the XCD, the span (first
    met -> last published) and their total; medians, with the max of the
    total."""
    import numpy as np
    import torch
    L = cfg.n_layer
    buf = torch.zeros(256 * (L + 1) * 24, dtype=torch.int64, device="cuda")
    sess.set_trace(buf)
    sess.verify(P, toks, par)
    torch.cuda.synchronize()
    sess.set_trace(None)
    t = buf.cpu().numpy().reshape(256, L + 1, 8, 3).astype(np.int64)
    x_of = np.arange(256) // 32   # trace rows are x * 32 + rank
    res = {s_: [] for s_ in range(7)}
    for l in range(2, L - 1):
        for s_ in range(7):
            pl, ps = (l, s_ - 1) if s_ else (l - 1, 6)
            for x in range(8):
                cons = x_of == x
                prod = np.ones(256, bool) if s_ in CROSS_XCD else cons
                pdone = t[prod, pl, ps, 2].max()
                met = t[cons, l, s_, 1]
                met = met[met > 0]
                if len(met) == 0:
                    continue
                done = t[cons, l, s_, 2].max()
                res[s_].append((met.min() - pdone, met.max() - met.min(), done - met.min(), done - pdone))
    period = np.median([(t[:, l + 1, 0, 0].min() - t[:, l, 0, 0].min()) * 0.01 for l in range(1, L - 1)])
    head = (t[:, L, 1, 2].max() - t[:, L, 0, 0].min()) * 0.01
    rows = []
    tot = 0.0
    for s_ in range(7):
        a = np.array(res[s_], dtype=np.float64) * 0.01
        med = np.median(a, 0)
        tot += med[3]
        rows.append(f"| {STAGES[s_]} | {'all 8 XCDs' if s_ in CROSS_XCD else 'own XCD'} | {med[0]:.2f} | "
                    f"{med[1]:.2f} | {med[2]:.2f} | {med[3]:.2f} | {a[:, 3].max():.2f} |")
    cmd = f"python bench.py --stage-trace --nodes {N} --prefix {P}"
    text = "\n".join([
        f"# Stage trace of the persistent pass: GPT-2-L shape, {N} nodes, {P}-token prefix",
        "",
        f"Command: `{cmd}` (MI355X; kernel sources {kernel_source_hash()}).",
        "",
        "One traced pass (s_memrealtime, 100 MHz, per workgroup: stage entry, dependency met, "
        "stage published). Per XCD and layer (layers 2..L-2), medians in us:",
        "hand-off = last producer published -> first consumer met; skew = first -> last consumer "
        "met inside the XCD; span = first met -> last published; total = last producer "
        "published -> last published (the stage's share of the critical path).",
        "",
        "| stage | inputs from | hand-off | met skew | span | total | max total |",
        "|---|---|---|---|---|---|---|",
        *rows,
        "",
        f"Sum of the median totals: {tot:.2f} us per layer; median layer period {period:.2f} us; "
        f"final LayerNorm + LM head {head:.1f} us; untraced pass {us_pass:.1f} us.",
        ""])
    path = os.path.join(ROOT, "profiles", f"stage_trace_n{N}_p{P}.md")
    with open(path, "w") as f:
        f.write(text)
    log(text)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--nodes", type=int, default=32)
    ap.add_argument("--prefix", type=int, default=512)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-sweep", action="store_true")
    ap.add_argument("--no-e2e", action="store_true", help="skip the staged end-to-end generation")
    ap.add_argument("--traffic-probe", action="store_true",
                    help="only run the kernels the HBM-traffic counters are read on (a 256 MiB device copy, then "
                         "the dominant kernel); meant to run under rocprofv3 --pmc")
    ap.add_argument("--traffic-from", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="read two rocprofv3 --pmc outputs (FETCH_SIZE, WRITE_SIZE) of --traffic-probe and write "
                         "profiles/traffic_pass_kernel.json (or traffic_fc_gemm.json with --kernels-path); "
                         "no GPU needed")
    ap.add_argument("--stage-trace", action="store_true",
                    help="time the pass, record one traced persistent pass and write "
                         "profiles/stage_trace_n{nodes}_p{prefix}.md")
    ap.add_argument("--mfma-probe", action="store_true",
                    help="only run three eager verification passes (for rocprofv3 --pmc MfmaUtil MfmaFlopsF16)")
    ap.add_argument("--mfma-from", nargs=2, metavar=("COUNTER_DIR", "TRACE_DIR"),
                    help="summarise a rocprofv3 --pmc MfmaUtil MfmaFlopsF16 run and a --kernel-trace --stats -f csv "
                         "run of the same command into profiles/mfma_gemm_n{nodes}_p{prefix}.md; no GPU needed")
    ap.add_argument("--q8", action="store_true",
                    help="run the timed step (and the probe modes) on the 8-bit weight model of the same weights")
    ap.add_argument("--kernels-path", action="store_true",
                    help="with --traffic-from: the counters are of the one-kernel-per-sub-layer path's GEMM")
    args = ap.parse_args()
    if args.mfma_from:
        base = f"python -u bench.py --nodes {args.nodes} --prefix {args.prefix} --mfma-probe"
        write_mfma(args.mfma_from[0], args.mfma_from[1], args.nodes, args.prefix,
                   f"rocprofv3 --pmc MfmaUtil MfmaFlopsF16 --kernel-include-regex gemm -f csv -d {args.mfma_from[0]} "
                   f"-o pmc -- {base}",
                   f"rocprofv3 --kernel-trace --stats -f csv -d {args.mfma_from[1]} -o trace -- {base}")
        return
    if args.traffic_from:
        write_traffic(args.traffic_from[0], args.traffic_from[1], args.nodes, not args.kernels_path)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for {args.gpus}): the library has no multi-GPU path "
              "(a pass would shard its heads and MLP slices over GPUs by tensor parallelism)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2308_04623_amd import ssd
    from paper_2308_04623_amd import workloads as W

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    # GPT-2-L shape with the position table extended to 2048 + 256 rows (the
    # 2048-token stress point needs them; positions are gathered, not
    # streamed, so no byte count changes)
    cfg = W.GPT2L_LONG
    N, P = args.nodes, args.prefix
    cached = max(1024, P)
    max_ctx, max_nodes = cached + 64, max(128, N)
    log("generating GPT-2-L weights")
    w = W.make_weights(cfg, 0)
    model = ssd.Model(cfg, w, q8=args.q8)
    kc, vc = W.random_kv_cache(cfg, max_ctx, cached, seed=3)
    sess = ssd.Session(model, max_ctx, max_nodes, ssd.to_device(kc, cfg), ssd.to_device(vc, cfg))
    par = W.branching_tree([4, 2, 2, 1], N)
    toks = W.tree_tokens(par, cfg.vocab, seed=2)
    logits = torch.empty((N, cfg.vocab), dtype=torch.float32, device="cuda")
    fused = sess.verify_path(N) == ssd.PASS_FUSED
    if args.traffic_probe:
        probe_traffic(sess, cfg, N, P, toks, par, fused)
        return
    if args.mfma_probe:
        # a few eager passes (no graph replays) for the matrix-core counters
        for _ in range(3):
            sess.verify(P, toks, par)
        torch.cuda.synchronize()
        log("mfma probe done")
        return
    if args.stage_trace:
        if not fused:
            raise SystemExit(f"a {N}-node pass does not run as the persistent kernel: nothing to trace")
        g = sess.capture_verify(P, toks, par, logits)
        for _ in range(5):
            g.launch()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(50):
            g.launch()
        b.record()
        torch.cuda.synchronize()
        stage_trace(sess, cfg, N, P, toks, par, a.elapsed_time(b) / 50 * 1e3)
        return
    stream = torch.cuda.current_stream()
    outs = (torch.zeros(N, dtype=torch.int32, device="cuda"), torch.zeros(1, dtype=torch.int32, device="cuda"),
            torch.zeros(1, dtype=torch.int32, device="cuda"))
    # one step: the captured pass with its greedy accept (ssd_tree_verify_greedy),
    # then the KV commit of the accepted path
    graph_step = sess.capture_verify_greedy(P, toks, par, logits, outs)

    def step():
        graph_step.launch()
        sess.commit(P, outs[0], outs[1])

    log(f"warmup {args.warmup}")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(args.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    ms_step = e0.elapsed_time(e1) / args.steps
    log(f"step {ms_step * 1e3:.1f} us")
    # a persistent pass that ended early (its logits undefined) or a float16
    # overflow counts here: the timing is only valid if none happened
    errs = sess.error_count()
    if errs:
        raise SystemExit(f"the session's error counter is {errs} after the timed steps: results invalid")

    def time_graph(g, reps):
        for _ in range(5):
            g.launch()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for _ in range(reps):
            g.launch()
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) / reps * 1e3  # us

    def time_calls(fn, reps):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for _ in range(reps):
            fn()
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) / reps * 1e3  # us

    graph = sess.capture_verify(P, toks, par, logits)
    us_pass = time_graph(graph, max(args.steps, 50))
    us_step_graph = time_graph(graph_step, 50)
    us_accept_logits = time_calls(lambda: sess.accept(toks, par, logits, out=outs), 50)
    B = pass_bytes(cfg, N, P, args.q8)
    log(f"verify pass {us_pass:.1f} us, {B / us_pass / 1e3:.0f} GB/s; pass + greedy accept {us_step_graph:.1f} us; "
        f"accept from the logits {us_accept_logits:.1f} us")
    if sess.error_count():
        raise SystemExit("the session's error counter grew during the timed passes")

    if fused:
        # dominant kernel: the persistent pass itself (the pass is this one
        # kernel; the graph adds only the ~2 KB tree upload before it), so its
        # algorithmic bytes are the pass's and its duration the graph
        # replays' on the stream they run on
        roofline = {"bound": "hbm", "achieved": round(B / us_pass / 1e3, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                    "frac": round(B / us_pass / 1e3 / PEAK_HBM_GBS, 4),
                    "traffic": None if args.q8 else stored_traffic(True, N),
                    "kernel": f"ssd::fz::pass_kernel<{min((N + 15) // 16, 2) if N <= 32 else 4}> "
                              "(persistent single-launch verification pass)",
                    "bytes_per_launch": B, "us_per_launch": round(us_pass, 2)}
    else:
        roofline = fc_gemm_roofline(sess, cfg, N, stream)

    def pass_point(n_s, p_s, s_=None, q8=None, **opts):
        s_ = s_ or sess
        q8 = args.q8 if q8 is None else q8
        tt, pp = W.best_first_tree(n_s, seed=3, vocab=cfg.vocab)
        tt[0] = int(toks[0])
        lg = torch.empty((n_s, cfg.vocab), dtype=torch.float32, device="cuda")
        with s_.options(**opts):
            path = s_.verify_path(n_s)
            g = s_.capture_verify(p_s, tt, pp, lg)
            us = time_graph(g, 30)
            g.close()
        bb = pass_bytes(cfg, n_s, p_s, q8)
        return {"nodes": n_s, "prefix": p_s, "us": round(us, 1), "GB/s": round(bb / us / 1e3, 1),
                "frac": round(bb / us / 1e3 / PEAK_HBM_GBS, 4),
                "path": "persistent" if path == ssd.PASS_FUSED else "per-sub-layer"}

    sweep, crossover = [], None
    if not args.no_sweep:
        # the size x prefix grid; each point in the default mode, and on the
        # one-kernel-per-sub-layer path with each GEMM path pinned (vector ALU
        # vs matrix cores) to locate their crossover
        grid = [(n_s, p_s) for p_s in (128, 512, 1024) for n_s in (1, 8, 16, 64, 128)]
        per_p = {}
        for n_s, p_s in grid:
            pt = pass_point(n_s, p_s)
            vec = pass_point(n_s, p_s, pass_mode=ssd.PASS_KERNELS, gemm_path=ssd.GEMM_VEC)
            mma = pass_point(n_s, p_s, pass_mode=ssd.PASS_KERNELS, gemm_path=ssd.GEMM_MFMA)
            pt["kernels_vec_us"], pt["kernels_mfma_us"] = vec["us"], mma["us"]
            sweep.append(pt)
            per_p.setdefault(p_s, []).append((n_s, vec["us"], mma["us"]))
            log(f"sweep N={n_s} P={p_s}: {pt['us']:.1f} us ({pt['path']}); per-sub-layer vec {vec['us']:.1f}, "
                f"mfma {mma['us']:.1f}")
        # smallest node count at which the matrix-core GEMMs beat the vector ALU
        crossover = {str(p_s): next((n for n, v, m in pts if m < v), None) for p_s, pts in per_p.items()}
        # latency growth with tree size at the 512-token prefix (log-log slope per step)
        row = sorted((p["nodes"], p["us"]) for p in sweep if p["prefix"] == 512)
        slopes = [round(float(np.log(b[1] / a[1]) / np.log(b[0] / a[0])), 3) for a, b in zip(row, row[1:])]
        crossover = {"smallest_nodes_mfma_faster_by_prefix": crossover, "loglog_slopes_P512": slopes,
                     "T128_over_T1_P512": round(row[-1][1] / row[0][1], 3)}
        if sess.error_count():
            raise SystemExit("the session's error counter grew during the sweep")

    stress = None
    if not args.no_sweep:
        # 256-node tree (branching 8,4,2,2,1 cut at 256) over a 2048-token
        # prefix, temperature-1 rejection sampling over the full vocabulary
        # with draft rows 0.5 x oracle softmax + 0.5 x Dirichlet(0.1) noise
        n5, p5 = 256, 2048
        kc5, vc5 = W.random_kv_cache(cfg, p5 + 8, p5, seed=5)
        s5 = ssd.Session(model, p5 + 8, n5, ssd.to_device(kc5, cfg), ssd.to_device(vc5, cfg))
        par5 = W.branching_tree([8, 4, 2, 2, 1], n5)
        tok5 = W.tree_tokens(par5, cfg.vocab, seed=6)
        lg5 = torch.empty((n5, cfg.vocab), dtype=torch.float32, device="cuda")
        g5 = s5.capture_verify(p5, tok5, par5, lg5)
        us5 = time_graph(g5, 20)
        g5.launch()
        torch.cuda.synchronize()
        gen = torch.Generator(device="cuda").manual_seed(7)
        noise = torch._standard_gamma(torch.full((n5, cfg.vocab), 0.1, device="cuda"), generator=gen)
        q5 = (0.5 * torch.softmax(lg5, 1) + 0.5 * noise / noise.sum(1, keepdim=True)).float().contiguous()
        out5 = (torch.zeros(n5, dtype=torch.int32, device="cuda"), torch.zeros(1, dtype=torch.int32, device="cuda"),
                torch.zeros(1, dtype=torch.int32, device="cuda"))
        acc = {}
        for name, kw in (("wor", dict(mode=ssd.SAMPLE_WOR, draft_probs=q5)),
                         ("wor_top50", dict(mode=ssd.SAMPLE_WOR, draft_probs=q5, top_k=50)),
                         ("chosen_top50", dict(mode=ssd.SAMPLE_DET, top_k=50)),
                         ("cdf_first", dict(mode=ssd.SAMPLE_CDF)),
                         ("greedy", dict())):
            acc[name] = round(time_calls(lambda: s5.accept(tok5, par5, lg5, out=out5, seed=3, **kw), 10), 1)
        b5 = pass_bytes(cfg, n5, p5, args.q8)
        stress = {"workload": "256-node tree (branching 8,4,2,2,1 cut at 256), 2048-token prefix, T=1 rejection "
                              "sampling over 50257 tokens, draft = 0.5 softmax + 0.5 Dirichlet(0.1)",
                  "verify_us": round(us5, 1), "GB/s": round(b5 / us5 / 1e3, 1),
                  "frac": round(b5 / us5 / 1e3 / PEAK_HBM_GBS, 4), "accept_us": acc,
                  "path": "persistent" if s5.verify_path(n5) == ssd.PASS_FUSED else "per-sub-layer"}
        log(f"stress: verify {us5:.1f} us, accept {acc}")
        if s5.error_count():
            raise SystemExit("the stress session's error counter grew")
        g5.close()
        s5.close()

    w8 = None
    if not args.no_sweep and not args.q8:
        # the same weights as 8-bit codes (ssd_model_create_q8): the pass at
        # five points on both models, the timed step at this workload, and
        # how far the 8-bit model's logits sit from the bfloat16 model's
        m8 = ssd.Model(cfg, w, q8=True)
        s8 = ssd.Session(m8, max_ctx, max_nodes, ssd.to_device(kc, cfg), ssd.to_device(vc, cfg))
        pts8 = []
        for n_s, p_s in ((1, 512), (32, 512), (64, 512), (128, 512)):
            a16, a8 = pass_point(n_s, p_s), pass_point(n_s, p_s, s_=s8, q8=True)
            pts8.append({"nodes": n_s, "prefix": p_s, "us_16bit": a16["us"], "us_8bit": a8["us"],
                         "GB/s_8bit": a8["GB/s"], "frac_8bit": a8["frac"], "path": a8["path"]})
        kc6, vc6 = W.random_kv_cache(cfg, 2048 + 8, 2048, seed=5)
        s86 = ssd.Session(m8, 2048 + 8, 256, ssd.to_device(kc6, cfg), ssd.to_device(vc6, cfg))
        s16 = ssd.Session(model, 2048 + 8, 256, ssd.to_device(kc6, cfg), ssd.to_device(vc6, cfg))
        a16, a8 = pass_point(256, 2048, s_=s16), pass_point(256, 2048, s_=s86, q8=True)
        pts8.append({"nodes": 256, "prefix": 2048, "us_16bit": a16["us"], "us_8bit": a8["us"],
                     "GB/s_8bit": a8["GB/s"], "frac_8bit": a8["frac"], "path": a8["path"]})
        s86.close()
        s16.close()
        lg8 = torch.empty_like(logits)
        outs8 = tuple(torch.zeros_like(o) for o in outs)
        g8 = s8.capture_verify_greedy(P, toks, par, lg8, outs8)

        def step8():
            g8.launch()
            s8.commit(P, outs8[0], outs8[1])

        for _ in range(args.warmup):
            step8()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for _ in range(args.steps):
            step8()
        b.record(stream)
        torch.cuda.synchronize()
        ms8 = a.elapsed_time(b) / args.steps
        g8.close()
        lg16 = sess.verify(P, toks, par).cpu().numpy()
        lq = s8.verify(P, toks, par).cpu().numpy()
        srt = np.sort(lg16, 1)
        if s8.error_count():
            raise SystemExit("the 8-bit session's error counter grew")
        w8 = {"workload": "the same GPT-2-L weights as symmetric 8-bit codes with a float32 scale per row "
                          "(matrices and LM head; float16 activations, float32 accumulation as in the "
                          "16-bit model)",
              "value": round(N / (ms8 * 1e-3), 1), "ms_per_step": round(ms8, 4),
              "pass_bytes_8bit": pass_bytes(cfg, N, P, True), "points": pts8,
              "max_abs_logit_change_vs_16bit": round(float(np.abs(lq - lg16).max()), 4),
              "greedy_tokens_equal_vs_16bit": int((lq.argmax(1) == lg16.argmax(1)).sum()),
              "greedy_tokens_compared": int(N), "top2_gap_median_16bit": round(float(np.median(srt[:, -1] - srt[:, -2])), 4)}
        log(f"8-bit weights: step {ms8 * 1e3:.1f} us; points {pts8}")
        s8.close()
        m8.close()

    reuse = None
    if not args.no_sweep:
        # the oracle pass started at layer 4 from the 4-layer draft's
        # residual stream and K/V (ssd_tree_reuse, then
        # ssd_tree_verify_from) against the pass from the embedding, on the
        # same best-first trees; eager calls both (host staging included),
        # and the hand-over's own time
        view = model.prefix_view(4)
        ds = ssd.Session(view, max_ctx, max_nodes, sess.k_cache, sess.v_cache)
        pts_r = []
        for n_s in (1, 16, 32, 64):
            tt, pp = W.best_first_tree(n_s, seed=3, vocab=cfg.vocab)
            tt[0] = int(toks[0])
            rows = np.arange(n_s, dtype=np.int32)
            lg_a = torch.empty((n_s, cfg.vocab), dtype=torch.float32, device="cuda")
            lg_b = torch.empty_like(lg_a)
            ds.verify(P, tt, pp)
            xr = ds.reuse_into(sess, rows)
            us_from = time_calls(lambda: sess.verify_from(P, tt, pp, 4, xr, logits=lg_a), 30)
            us_full = time_calls(lambda: sess.verify(P, tt, pp, logits=lg_b), 30)
            us_hand = time_calls(lambda: ds.reuse_into(sess, rows), 30)
            torch.cuda.synchronize()
            pts_r.append({"nodes": n_s, "prefix": P, "us_from_layer4": round(us_from, 1),
                          "us_from_embedding": round(us_full, 1), "us_handover": round(us_hand, 1),
                          "logits_bitwise_equal": bool(torch.equal(lg_a, lg_b)),
                          "path": "persistent" if sess.verify_path(n_s) == ssd.PASS_FUSED else "per-sub-layer"})
        if sess.error_count() or ds.error_count():
            raise SystemExit("a session's error counter grew during the reuse points")
        ds.close()
        reuse = {"workload": "oracle pass over a best-first tree the 4-layer draft already ran, started at layer 4 "
                             "from the draft's residual stream and layer 0-3 K/V, against the pass from the "
                             "embedding (eager calls)", "points": pts_r}
        log(f"draft reuse: {pts_r}")

    e2e = None
    if not args.no_e2e:
        e2e = end_to_end(ssd, W, cfg, model, N_NEW=256, PROMPT=128)

    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        threads = int(os.environ.get("OMP_NUM_THREADS", "0") or 0) or (os.cpu_count() or 1)
        om = oracle.Model(cfg, w, q8=args.q8)
        okt, ovt = om.kv(max_nodes), om.kv(max_nodes)

        def oracle_time(n_s, p_s, tt, pp, budget, reps):
            ts = []
            t_start = time.time()
            while len(ts) < reps and (time.time() - t_start) < budget:
                t0 = time.time()
                oracle.tree_verify(om, kc, vc, p_s, tt, pp, okt, ovt, threads)
                ts.append(time.time() - t0)
            return sorted(ts)[len(ts) // 2], len(ts)

        tpass, nrun = oracle_time(N, P, toks, par, 10.0, 30)
        tok64, par64 = W.best_first_tree(64, seed=3, vocab=cfg.vocab)
        tok64[0] = int(toks[0])
        t64, _ = oracle_time(64, 512, tok64, par64, 6.0, 3)
        t1, n1 = oracle_time(1, 512, np.array([int(toks[0])], np.int32), np.array([-1], np.int32), 4.0, 20)
        # the tiny fp32 model (2 x 128, vocab 512): a 15-node binary tree over 64 cached tokens
        tcfg = W.TINY
        tw = W.make_weights(tcfg, 0)
        tom = oracle.Model(tcfg, tw)
        tkc, tvc = W.random_kv_cache(tcfg, 128, 64, seed=1)
        tpar = W.complete_binary_tree(15)
        ttok = W.tree_tokens(tpar, tcfg.vocab, seed=2)
        tt0 = time.time()
        for _ in range(20):
            oracle.tree_verify(tom, tkc, tvc, 64, ttok, tpar, tom.kv(16), tom.kv(16), threads)
        t_tiny = (time.time() - tt0) / 20
        cpu = {"value": round(N / tpass, 3), "unit": "verified tree tokens/s", "cores": threads, "kind": "oracle",
               "sample": f"{nrun} full oracle verification passes of this workload (fp64, {N} nodes, "
                         f"prefix {P}), median {tpass:.2f} s each; host {cpu_model()}",
               "also": {"nodes64_prefix512_pass_s": round(t64, 3),
                        "plain_decode_tokens_per_s": round(1.0 / t1, 3),
                        "tiny_fp32_15_nodes_pass_ms": round(t_tiny * 1e3, 3)}}
        log(f"oracle pass {tpass:.2f} s on {threads} threads; 64 nodes {t64:.2f} s; plain decode {1 / t1:.2f} tok/s")

    # whole-step throughput: tree tokens verified per second of timed steps
    # (pass, greedy accept, commit)
    value = N / (ms_step * 1e-3)
    line = {
        "metric": METRIC, "value": round(value, 1), "unit": "verified tree tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "int8" if args.q8 else "bf16", "data": "synthetic",
        "config": {"workload": f"GPT-2-L shape tree verification, {N}-node tree (branching 4,2,2,1), "
                               f"{P}-token prefix, greedy accept + commit"
                               + (", 8-bit weights (symmetric codes, float32 row scales)" if args.q8 else ""),
                   "nodes": N, "prefix": P, "layers": cfg.n_layer, "d_model": cfg.d_model, "vocab": cfg.vocab},
        "verify_path": "persistent single launch" if fused else "one kernel per sub-layer",
        "us_per_verify_pass": round(us_pass, 2),
        "us_pass_plus_greedy_accept": round(us_step_graph, 2),
        "us_accept_from_logits": round(us_accept_logits, 2),
        "pass_hbm_GBs": round(B / us_pass / 1e3, 1),
        "pass_frac_of_peak": round(B / us_pass / 1e3 / PEAK_HBM_GBS, 4),
        "pass_algorithmic_bytes": B,
        "roofline": roofline,
        "cpu_baseline": cpu,
        "draft_reuse": reuse,
        "end_to_end": e2e,
        "sweep": sweep,
        "sweep_summary": crossover,
        "stress": stress,
        "weights_8bit": w8,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
