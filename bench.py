#!/usr/bin/env python3
"""Benchmark of one Clover speculate-and-verify step on one MI355X.

Workload (default): the 7B-shape bf16 model (32 layers, d_model 4096, 32 heads of
128, SwiGLU 11008, vocab 125696) with the Clover speculator (Augmenting Block + 3
heads), batch 1, a 1024-token uniform-random prompt and a 64-token verify tree
from per-depth top-k (8, 4, 2).  Weights are random-init N(0, 0.02) drawn on the
device; nothing here is a trained model, so acceptance is ~1 token per step and
only per-step costs are comparable to the paper.

A step is one clover_step call: draft (Augmenting Block state, Attention Decoder,
head MLPs, shared LM head + top-k, tree truncation), the tree-masked verify
forward, greedy acceptance and KV compaction.  The timed region runs --steps steps
after --warmup untimed ones, bracketed by device synchronisation.

Prints one JSON line with the throughput (tree tokens verified per second over
whole steps), the per-phase latencies, the streaming GEMM's achieved HBM
bandwidth against the 8 TB/s peak (HIP events around every launch in the timed
region) and the CPU oracle's throughput on a bounded sample of the same workload.
"""
import argparse
import gc
import hashlib
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0  # dense bf16 matrix-core peak of MI355X
TILED_MIN_ROWS = 129  # verify GEMMs with this many rows run the register-blocked kernel
METRIC = "verify-step latency (ms) & tree-tokens/s at 7B shape; weight-stream HBM GB/s vs peak"


def gemm_source_hash():
    """Hash of the sources that define the streaming GEMM kernel."""
    h = hashlib.sha256()
    for f in ("gemm.hip", "kernels.h", "common.h"):
        with open(os.path.join(ROOT, "paper_2405_00263_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(workload):
    """HBM bytes per verify-GEMM launch from the committed counter summary.

    The summary under profiles/ holds FETCH_SIZE + WRITE_SIZE per dispatch, each scaled
    by the factor a plain copy of known size gives for the same counter, averaged over
    the verify forward's GEMM launches, and the hash of the kernel sources it was taken
    with.  Returns None when there is no summary for the workload or the kernel has
    changed since.
    """
    path = os.path.join(ROOT, "profiles", f"gemm_verify_{workload}_traffic.md")
    if not os.path.exists(path):
        return None
    vals = {}
    with open(path) as fh:
        for line in fh:
            if ":" in line and line.split(":")[0] in ("traffic_bytes_per_launch", "gemm_source_sha256_16"):
                k, v = line.split(":", 1)
                vals[k] = v.strip()
    if vals.get("gemm_source_sha256_16") != gemm_source_hash() or "traffic_bytes_per_launch" not in vals:
        return None
    return int(float(vals["traffic_bytes_per_launch"]))


def _prompt_lengths(cfg):
    import synth
    if cfg.batch == 1:
        return [cfg.prompt_len[0]]
    return synth.make_prompt_lengths(cfg)


def _tiny_single_thread():
    """The oracle on the small fp32 workload (2 layers, d_model 256, 41-token trees,
    128-token prompt), single-threaded: prefill, then all 16 steps."""
    import synth
    import oracle
    from threadpoolctl import threadpool_limits

    cfg = synth.get_config("tiny_fp32")
    w = synth.make_weights(cfg, seed=0, device="cpu")
    o = oracle.make_oracle(cfg, w)
    prompt = synth.make_prompt(cfg, n=cfg.prompt_len[0])
    steps = 16
    with threadpool_limits(1):
        st = o.prefill(prompt)
        t0 = time.perf_counter()
        for _ in range(steps):
            o.step(st)
        dt = time.perf_counter() - t0
    return {"value": round(steps * cfg.tree_tokens / dt, 2), "unit": "tree-tokens/s", "cores": 1,
            "sample": f"{steps} oracle steps of tiny_fp32 after its {cfg.prompt_len[0]}-token prefill, one thread"}


def cpu_baseline(cfg, seed=0):
    """The oracle, as written, on a bounded sample of the workload.

    Sample: repeated oracle steps (draft over all depths, tree truncation, verify,
    accept, commit) of a 1-layer slice of the workload with a synthetic committed
    context of the workload's prompt length, plus n_layers - 1 runs of one oracle
    decoder layer over the T tree rows against that context; the mean step plus the
    layer runs is the oracle's time for one full-depth step.
    """
    import numpy as np
    import synth
    import oracle
    from oracle.model import BaseModel

    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:
        cores = os.cpu_count() or 1
    c1 = cfg.with_(n_layers=1, batch=1)
    w = synth.make_weights(c1, seed=seed, device="cpu")
    o = oracle.make_oracle(c1, w)
    del w
    rng = np.random.default_rng(1)
    L = _prompt_lengths(cfg)[0]
    prec = o.prec
    shape = (L, c1.n_kv_heads, c1.head_dim)
    kv = [(prec.store(rng.standard_normal(shape)), prec.store(rng.standard_normal(shape)))]
    ab = None if cfg.ab_kind in ("none", "mlp") else (prec.store(rng.standard_normal(shape)),
                                                       prec.store(rng.standard_normal(shape)))
    st = oracle.SeqState(tokens=list(rng.integers(0, c1.vocab, L)), kv=kv, ab_kv=ab,
                         h0=rng.standard_normal(c1.d_model), t0=int(rng.integers(0, c1.vocab)))
    # oracle steps of the 1-layer slice, repeated for a stable figure (about 6 s)
    n_step, t_steps = 0, 0.0
    while n_step < 3 or (t_steps < 6.0 and n_step < 12):
        t0 = time.perf_counter()
        o.step(st)
        t_steps += time.perf_counter() - t0
        n_step += 1
    t_step = t_steps / n_step
    # the remaining decoder layers over the tree rows against the committed context
    T = cfg.tree_tokens
    x = rng.standard_normal((T, c1.d_model))
    pos = L + np.minimum(np.arange(T), 3)
    mask = oracle.tree_mask([-1] + [0] * (T - 1))
    t0 = time.perf_counter()
    for _ in range(cfg.n_layers - 1):
        o.base.run_layer(o.base.layers[0], x, pos, kv[0][0], kv[0][1], mask)
    t_layers = time.perf_counter() - t0
    total = t_step + t_layers
    return {
        "value": round(cfg.batch * T / total, 4),
        "unit": "tree-tokens/s",
        "cores": int(cores),
        "kind": "oracle",
        "sample": (f"{n_step} oracle steps of a 1-layer slice of {cfg.name} (T={T}, context {L}), "
                   f"mean {t_step:.2f}s, + {cfg.n_layers - 1} oracle decoder layers over the "
                   f"{T} tree rows {t_layers:.2f}s = {total:.2f}s per full step (float64 NumPy)"),
        "single_thread_tiny": _tiny_single_thread(),
    }


def verify_weight_bytes(cfg):
    """Bytes of weight one verify forward streams: target layers, the Augmenting Block (or
    its configured half) and the LM head."""
    es = 2 if cfg.dtype == "bf16" else 4
    d, F, V = cfg.d_model, cfg.ffn_dim, cfg.vocab
    qd, kvd = cfg.n_heads * cfg.head_dim, cfg.n_kv_heads * cfg.head_dim
    attn_w = (qd * d + 2 * kvd * d + d * qd) * es
    layer_w = attn_w + 3 * F * d * es
    ab_w = {"full": layer_w, "none": 0, "attn": attn_w, "mlp": 3 * F * d * es}[cfg.ab_kind]
    return cfg.n_layers * layer_w + ab_w + V * d * es


def verify_kv_bytes(cfg, contexts):
    """KV-cache bytes one verify forward moves besides the weights: every committed key and
    value of each sequence read once per attention layer (the target layers, plus the
    Augmenting Block when it has an attention half), and the tree's own keys and values
    written once."""
    es = 2 if cfg.dtype == "bf16" else 4
    kvd = cfg.n_kv_heads * cfg.head_dim
    layers = cfg.n_layers + (1 if cfg.ab_kind in ("full", "attn") else 0)
    read = sum(2 * c * kvd * es for c in contexts) * layers
    write = 2 * cfg.batch * cfg.tree_tokens * kvd * es * layers
    return read + write


def measured_copy_gbps(torch, nbytes=1 << 30, reps=10):
    """Device-to-device copy rate on this GPU (bytes read + written per second), the
    achievable-bandwidth reference the roofline is also compared against."""
    src = torch.empty(nbytes // 2, dtype=torch.bfloat16, device="cuda").fill_(1.0)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    del src, dst
    torch.cuda.empty_cache()
    return 2.0 * nbytes / (ms * 1e-3) / 1e9


def _pct(v, q):
    """Percentile q (0..100) of the list v by linear interpolation."""
    v = sorted(v)
    if not v:
        return 0.0
    x = (len(v) - 1) * q / 100.0
    lo = int(x)
    hi = min(lo + 1, len(v) - 1)
    return v[lo] + (v[hi] - v[lo]) * (x - lo)


def surface(args):
    """Batch x tree-size cost surface of one step (Sec. 1 and 4.2 of the paper argue that
    speculation pays while the verify stays memory-bound and loses its edge as batch and
    tree grow towards the compute bound).

    One JSON line per cell: batch B, tree tokens T, the per-phase latencies, and the verify
    forward's weight-stream rate and matrix arithmetic rate (2 flops per weight per verify
    row).  Every cell uses the same weights, a committed context of --prompt-len tokens per
    sequence (default 1024), top-k (8, 4, 2) truncated to T (T = 128: (16, 4, 2)).
    """
    import torch
    import synth
    import paper_2405_00263_amd as P

    base = synth.get_config(args.workload)
    L0 = args.prompt_len or 1024
    batches = [int(v) for v in args.surface_batches.split(",")]
    trees = [int(v) for v in args.surface_trees.split(",")]
    cells = [("clover", B, T) for B in batches for T in trees]
    cells += [("medusa", B, 64) for B in batches]
    print(f"[surface] {len(cells)} cells on {base.name}: generating weights on device", file=sys.stderr, flush=True)
    w = synth.make_weights(base.with_(draft="clover", ab="default"), seed=args.seed, device="cuda")
    for draft, B, T in cells:
        cfg = base.with_(batch=B, tree_tokens=T, topk=(16, 4, 2) if T > 64 else (8, 4, 2), draft=draft,
                         prompt_len=(L0, L0))
        ww = {n: w[n] for n, _ in synth.weight_specs(cfg)}
        H1 = cfg.n_spec_heads + 1
        eng = P.CloverEngine(cfg, ww, max_batch=B, max_context=L0 + (args.warmup + args.steps) * H1 + T + 16)
        seqs = list(range(B))
        for b in seqs:
            eng.prefill(b, synth.make_prompt(cfg, seq=b, n=L0))
        for _ in range(args.warmup):
            eng.step(seqs)
        ph = {"draft_ms": [], "verify_ms": [], "total_ms": []}
        gc.collect()
        gc.disable()  # no garbage-collector pause inside the timed steps
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(args.steps):
            eng.step(seqs)
            tm = eng.timings()
            for k in ph:
                ph[k].append(tm[k])
        torch.cuda.synchronize()
        step_ms = 1e3 * (time.perf_counter() - t0) / args.steps
        gc.enable()
        med = {k: statistics.median(v) for k, v in ph.items()}
        wb = verify_weight_bytes(cfg)
        params = wb / (2 if cfg.dtype == "bf16" else 4)
        print(json.dumps({"surface_cell": {
            "speculator": draft, "batch": B, "tree_tokens": T, "verify_rows": B * T, "context": L0,
            "step_ms": round(step_ms, 4), "verify_ms": round(med["verify_ms"], 4),
            "draft_ms": round(med["draft_ms"], 4),
            "tree_tokens_per_s": round(B * T / (step_ms * 1e-3), 1),
            "verify_weight_GBps": round(wb / (med["verify_ms"] * 1e-3) / 1e9, 1),
            "verify_gemm_TFLOPs": round(2.0 * B * T * params / (med["verify_ms"] * 1e-3) / 1e12, 1),
        }}), flush=True)
        eng.close()
        del eng
        torch.cuda.empty_cache()


def context_grid(args):
    """Tree-size x context grid on the 7B shape at batch 1: tree sizes {16, 32, 64, 128}
    (top-k (4,2,2), (4,3,2), (8,4,2), (16,4,2), root included) x committed contexts {512,
    4096, 16384, 32768} filled by a real prefill of uniform-random tokens.  One JSON line per
    cell: whole-step throughput and latency, the verify and draft (Clover heads) latencies
    from the graph-replayed steps, then from a second pass with every launch timed by HIP
    events: the tree-masked attention's time per layer (attention kernel plus its key-split
    merge) and its rate over the algorithmic KV bytes (every committed key and value, and the
    tree's, read once per layer, plus Q and O), and the verify GEMMs' weight-stream rate."""
    import torch
    import synth
    import paper_2405_00263_amd as P

    base = synth.get_config("llama7b_b1")
    print(f"[grid] {len(synth.SWEEP_TREES) * len(synth.SWEEP_CONTEXTS)} cells: generating weights on device",
          file=sys.stderr, flush=True)
    w = synth.make_weights(base, seed=args.seed, device="cuda")
    kt = max(3, args.steps // 2)
    for T, topk in synth.SWEEP_TREES:
        for L0 in synth.SWEEP_CONTEXTS:
            cfg = base.with_(tree_tokens=T, topk=topk, prompt_len=(L0, L0))
            H1 = cfg.n_spec_heads + 1
            eng = P.CloverEngine(cfg, w, max_batch=1, max_context=L0 + (args.warmup + args.steps + kt) * H1 + T + 16)
            eng.prefill(0, synth.make_prompt(cfg, n=L0))
            for _ in range(args.warmup):
                eng.step([0])
            ph = {"draft_ms": [], "verify_ms": [], "total_ms": []}
            gc.collect()
            gc.disable()
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for _ in range(args.steps):
                eng.step([0])
                tm = eng.timings()
                for k in ph:
                    ph[k].append(tm[k])
            torch.cuda.synchronize()
            step_ms = 1e3 * (time.perf_counter() - t0) / args.steps
            gc.enable()
            eng.set_flags(P.FLAG_PROFILE)
            eng.reset_kernel_stats()
            for _ in range(kt):
                eng.step([0])
            eng.set_flags(0)
            ks = eng.kernel_stats()
            att, gv = ks["attention"], ks["gemm_verify"]
            med = {k: statistics.median(v) for k, v in ph.items()}
            print(json.dumps({"grid_cell": {
                "tree_tokens": T, "topk": list(topk), "context": L0,
                "step_ms": round(step_ms, 4), "tree_tokens_per_s": round(T / (step_ms * 1e-3), 1),
                "verify_ms": round(med["verify_ms"], 4), "draft_ms": round(med["draft_ms"], 4),
                "attention_us_per_layer": round(1e3 * att["total_ms"] / max(1, att["launches"]), 2),
                "attention_GBps": round(att["bytes"] / (att["total_ms"] * 1e-3) / 1e9, 1) if att["total_ms"] else 0.0,
                "attention_kv_MB_per_layer": round(att["bytes"] / max(1, att["launches"]) / 1e6, 2),
                "verify_gemm_GBps": round(gv["bytes"] / (gv["total_ms"] * 1e-3) / 1e9, 1) if gv["total_ms"] else 0.0,
            }}), flush=True)
            eng.close()
            del eng
            torch.cuda.empty_cache()


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="llama7b_b1")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-kernel-timing", action="store_true",
                    help="skip the second, per-launch timed pass (no roofline figure)")
    ap.add_argument("--prompt-len", type=int, default=0,
                    help="override the prompt length (context sweep cells)")
    ap.add_argument("--tree-tokens", type=int, default=0, help="override T (tree tokens, root included)")
    ap.add_argument("--topk", default="", help="override the per-depth top-k, e.g. 16,4,2")
    ap.add_argument("--draft", default="", choices=["", "clover", "medusa"],
                    help="override the speculator: Clover heads or the Medusa baseline")
    ap.add_argument("--ab", default="", choices=["", "default", "full", "attn", "mlp", "none"],
                    help="override the Augmenting Block variant (Sec. 4.3)")
    ap.add_argument("--ad-keys", default="", choices=["", "single", "two", "path"],
                    help="override the Attention Decoder's key set (Eq. 1 readings)")
    ap.add_argument("--regressive", default="", choices=["", "attention", "mlp"],
                    help="override the Clover draft's regressive block: the Attention Decoder or the "
                         "MLP over [RMSNorm(h); e] of the components ablation (Sec. 4.3)")
    ap.add_argument("--medusa-lm", default="", choices=["", "shared", "per_head"],
                    help="Medusa draft: heads share the target's LM head, or each has its own (Sec. 3.4)")
    ap.add_argument("--ab-commit", action="store_true",
                    help="run the Augmenting Block at commit over the accepted rows at every batch size")
    ap.add_argument("--temperature", type=float, default=-1.0,
                    help="override the sampling temperature (0: greedy; > 0: speculative sampling)")
    ap.add_argument("--surface", action="store_true",
                    help="batch x tree-size cost surface instead of the headline line (one JSON line per cell)")
    ap.add_argument("--context-grid", action="store_true",
                    help="tree-size x context grid at the 7B shape, batch 1 (one JSON line per cell)")
    ap.add_argument("--surface-batches", default="1,2,4,8,16")
    ap.add_argument("--surface-trees", default="4,16,32,64,128")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported "
              "(each sequence is independent, so more GPUs would each run their own batch)",
              file=sys.stderr)
        sys.exit(2)
    if args.surface:
        surface(args)
        return
    if args.context_grid:
        context_grid(args)
        return

    import torch
    import synth
    import paper_2405_00263_amd as P

    cfg = synth.get_config(args.workload)
    over = {}
    if args.prompt_len:
        over["prompt_len"] = (args.prompt_len, args.prompt_len)
    if args.tree_tokens:
        over["tree_tokens"] = args.tree_tokens
    if args.topk:
        over["topk"] = tuple(int(v) for v in args.topk.split(","))
    if args.draft:
        over["draft"] = args.draft
    if args.ab:
        over["ab"] = args.ab
    if args.ad_keys:
        over["ad_keys"] = args.ad_keys
    if args.regressive:
        over["regressive"] = args.regressive
    if args.medusa_lm:
        over["medusa_lm"] = args.medusa_lm
    if args.temperature >= 0:
        over["temperature"] = args.temperature
    if over:
        cfg = cfg.with_(**over)
    torch.cuda.set_device(0)
    lens = _prompt_lengths(cfg)
    H1 = cfg.n_spec_heads + 1
    kt_steps = 0 if args.no_kernel_timing else max(5, args.steps // 2)
    max_context = max(lens) + (args.warmup + args.steps + kt_steps) * H1 + cfg.tree_tokens + 16
    print(f"[bench] workload {cfg.name}: generating weights on device", file=sys.stderr, flush=True)
    w = synth.make_weights(cfg, seed=args.seed, device="cuda")
    base_flags = P.FLAG_AB_COMMIT if args.ab_commit else 0
    eng = P.CloverEngine(cfg, w, max_batch=cfg.batch, max_context=max_context, free_source=True, flags=base_flags)
    del w
    torch.cuda.empty_cache()
    seqs = list(range(cfg.batch))
    for b in seqs:
        eng.prefill(b, synth.make_prompt(cfg, seq=b, n=lens[b]))
    ctx_start = [eng.seq_len(b) for b in seqs]
    print(f"[bench] prefill done (context {ctx_start}); warmup {args.warmup} steps",
          file=sys.stderr, flush=True)
    for _ in range(args.warmup):
        eng.step(seqs)
    eng.reset_kernel_stats()
    phase = {"draft_ms": [], "verify_ms": [], "accept_ms": [], "total_ms": []}
    emitted = 0
    # Python's cyclic garbage collector can stop this loop for tens of milliseconds (a
    # full collection over the interpreter's objects); it runs before, not inside, the
    # timed steps
    gc.collect()
    gc.disable()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        out = eng.step(seqs)
        emitted += sum(len(o) for o in out)
        tm = eng.timings()
        for k in phase:
            phase[k].append(tm[k])
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    gc.enable()
    ms_per_step = 1e3 * elapsed / args.steps
    T = cfg.tree_tokens
    value = cfg.batch * T * args.steps / elapsed
    # second pass over the same workload with every launch timed by HIP events on the
    # context's stream (eager launches; the graph replay above cannot carry them)
    if kt_steps:
        eng.set_flags(P.FLAG_PROFILE | base_flags)
        eng.reset_kernel_stats()
        for _ in range(kt_steps):
            eng.step(seqs)
        eng.set_flags(base_flags)
    ks = eng.kernel_stats()
    g = ks["gemm_verify"]
    achieved = g["bytes"] / (g["total_ms"] * 1e-3) / 1e9 if g["total_ms"] > 0 else 0.0
    # with enough rows the verify GEMMs run on the matrix cores' compute bound: report
    # their arithmetic rate against the dense bf16 peak instead of the HBM bound
    mfma_bound = cfg.dtype == "bf16" and cfg.batch * cfg.tree_tokens >= TILED_MIN_ROWS
    tflops = g["flops"] / (g["total_ms"] * 1e-3) / 1e12 if g["total_ms"] > 0 else 0.0
    med = {k: statistics.median(v) for k, v in phase.items()}
    d, F, V = cfg.d_model, cfg.ffn_dim, cfg.vocab
    verify_wbytes = verify_weight_bytes(cfg)
    # context at the middle of the timed steps (each step commits about one token per
    # sequence with random-init heads)
    mid_ctx = [c + args.warmup + args.steps // 2 for c in ctx_start]
    verify_kvbytes = verify_kv_bytes(cfg, mid_ctx)
    copy_gbps = measured_copy_gbps(torch)
    result = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "tree-tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic: random-init N(0,0.02) weights, uniform-random prompt tokens",
        "config": {"workload": cfg.name, "speculator": cfg.draft, "augmenting_block": cfg.ab_kind, "ab_at_commit": bool(args.ab_commit),
                   "decoder_keys": cfg.ad_keys, "regressive_block": cfg.regressive,
                   "medusa_lm_heads": cfg.medusa_lm,
                   "temperature": cfg.temperature,
                   "n_layers": cfg.n_layers, "d_model": d,
                   "n_heads": cfg.n_heads, "n_kv_heads": cfg.n_kv_heads, "head_dim": cfg.head_dim,
                   "ffn_dim": F, "vocab": V, "spec_heads": cfg.n_spec_heads, "topk": list(cfg.topk),
                   "batch": cfg.batch, "tree_tokens": T, "prompt_len": lens,
                   "context_at_timed_start": [c + args.warmup for c in ctx_start]},
        "verify_ms": round(med["verify_ms"], 4),
        "draft_ms": round(med["draft_ms"], 4),
        "accept_ms": round(med["accept_ms"], 4),
        "step_ms_events": round(med["total_ms"], 4),
        "step_ms_p10_p50_p90": [round(_pct(phase["total_ms"], q), 4) for q in (10, 50, 90)],
        "verify_ms_p10_p50_p90": [round(_pct(phase["verify_ms"], q), 4) for q in (10, 50, 90)],
        "verify_weight_GBps": round(verify_wbytes / (med["verify_ms"] * 1e-3) / 1e9, 1),
        "verify_effective_GBps": round((verify_wbytes + verify_kvbytes) / (med["verify_ms"] * 1e-3) / 1e9, 1),
        "measured_copy_GBps": round(copy_gbps, 1),
        "tokens_emitted_per_step": round(emitted / (args.steps * cfg.batch), 3),
        "roofline": {
            "bound": "mfma" if mfma_bound else "hbm",
            "achieved": round(tflops, 1) if mfma_bound else round(achieved, 1),
            "peak": MFMA_BF16_PEAK_TFLOPS if mfma_bound else HBM_PEAK_GBS,
            "unit": "TFLOP/s" if mfma_bound else "GB/s",
            "frac": round(tflops / MFMA_BF16_PEAK_TFLOPS, 4) if mfma_bound else round(achieved / HBM_PEAK_GBS, 4),
            "traffic": measured_traffic(cfg.name),
            "kernel": ("verify-forward GEMMs (32x32 wide_kernel; LM head on the register-blocked tiled_kernel)"
                       if mfma_bound else "verify-forward GEMMs (streaming gemm_kernel)"),
            # the whole verify forward (GEMMs, attention, norms, fix-ups) against the HBM peak:
            # verify weight bytes over the verify's event-timed latency
            "verify_forward_frac_of_hbm_peak": round(verify_wbytes / (med["verify_ms"] * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
            "weight_stream_GBps": round(achieved, 1),
            "frac_of_measured_copy": None if mfma_bound else round(achieved / copy_gbps, 4),
            "timed_steps": kt_steps,
            "launches": g["launches"],
            "avg_launch_us": round(1e3 * g["total_ms"] / max(g["launches"], 1), 3),
            "bytes_per_launch": round(g["bytes"] / max(g["launches"], 1)),
        },
        "kernel_classes": {k: {"launches": v["launches"], "ms": round(v["total_ms"], 3),
                               "GBps": round(v["bytes"] / (v["total_ms"] * 1e-3) / 1e9, 1) if v["total_ms"] else None}
                           for k, v in ks.items()},
    }
    eng.close()
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle on a bounded sample", file=sys.stderr, flush=True)
        result["cpu_baseline"] = cpu_baseline(cfg, args.seed)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
