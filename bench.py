#!/usr/bin/env python3
"""Benchmark of the fused per-position scoring path on one MI355X.

One step = one olive_kl_masked call over one packed batch already resident in HBM:
vocabulary projection of both models (bf16 MFMA, fp32 accumulate), online
log-softmax over the full vocabulary, realised-token log-probs, masked
KL(teacher || student), greedy argmax with the exact near-tie re-decision, and
Eq. 1's per-sequence loss. Default workload: long_rollout (B=8 x L=4096,
V=151,936, d_S=2048, d_T=4096, logits x4, EOS-truncated).

Prints one JSON line: positions/s (valid positions scored per second), the
scoring kernel's achieved bf16 TFLOP/s against the MI355X dense peak, and the fp64
CPU oracle's rate on a bounded row sample.
"""
import argparse
import json
import os
import sys
import time

PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA (no sparsity)
PROFILES = os.path.join(os.path.dirname(os.path.abspath(__file__)), "profiles")


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def cpu_baseline(wl, seconds: float):
    """The fp64 oracle on a bounded, seeded sample of the workload's valid rows."""
    import numpy as np
    import torch
    from threadpoolctl import threadpool_info
    from oracle import olive_oracle as O

    def np32(t):
        return (t.float() if t.dtype == torch.bfloat16 else t).cpu().numpy()
    cu = wl["cu_seqlens"].cpu().numpy()
    cut = wl["cut"].cpu().numpy()
    vl = None if wl["valid_len"] is None else wl["valid_len"].cpu().numpy()
    m = O.masks(cu, cut, vl)
    valid_rows = np.nonzero(m["valid"])[0]
    rng = np.random.default_rng(12345)
    order = rng.permutation(valid_rows)
    ws = np32(wl["w_student"]).astype(np.float64)   # input marshalling, untimed
    wt = np32(wl["w_teacher"]).astype(np.float64)

    def run(rows):
        idx = torch.from_numpy(np.sort(rows)).cuda()
        hs = np32(wl["h_student"][idx]).astype(np.float64)
        ht = np32(wl["h_teacher"][idx]).astype(np.float64)
        y = wl["targets"][idx].cpu().numpy()
        t0 = time.perf_counter()
        # what the timed call forms: both models' log-normalisers, log-probs and greedy
        # tokens, and the forward KL (no reverse KL or top-K sets)
        O.row_scores(hs, ws, y, wl["scale_student"], ht, wt, wl["scale_teacher"],
                     extras=False)
        return time.perf_counter() - t0
    # Rows in chunks until the timed oracle work reaches `seconds` (only the oracle
    # calls are timed; gathering the rows is not).
    n, t, chunk = 0, 0.0, 16
    while t < seconds and n < len(order):
        rows = order[n:n + chunk]
        t += run(rows)
        n += len(rows)
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [os.cpu_count()])
    return dict(value=n / t, unit="positions/s", cores=int(threads), kind="oracle",
                cpu_model=cpu_model(),
                sample="%d random valid rows of the workload (seed 12345), fp64 numpy oracle "
                       "row_scores without its reverse-KL and top-K extras (both models' "
                       "log-normalisers, log-probs and greedy tokens, forward KL: what the "
                       "timed GPU call forms), weights converted to float64 before the timed "
                       "region; %.1f s" % (n, t))


def bench_library_gemm(args, wl):
    """Plain library GEMMs of the workload's contractions (torch.mm -> hipBLASLt),
    bf16 operands and bf16 results, for comparison with the fused kernels: the logits
    z_X = h_X W_X of both models over the valid rows (what an unfused path computes
    before its softmax and KL passes; it would also write and re-read the [T, V]
    logits), and the backward's products dL/dh = g W^T and dL/dW = h^T g over the
    scored rows with a bf16 logit gradient g."""
    import torch

    # Row selection only: packed rows below each sequence's valid length, and of those
    # the scored ones (from the cut, or the spans of a multi-turn batch).
    cu = wl["cu_seqlens"].tolist()
    vl = None if wl["valid_len"] is None else wl["valid_len"].tolist()
    cut = wl["cut"].tolist()
    spans = wl.get("spans")                       # per-sequence (start, end) lists
    valid_rows, scored_rows = [], []
    for b in range(len(cu) - 1):
        n = cu[b + 1] - cu[b] if vl is None else vl[b]
        valid_rows += range(cu[b], cu[b] + n)
        for lo, hi in (spans[b] if spans is not None else [(cut[b], n)]):
            scored_rows += range(cu[b] + lo, cu[b] + min(hi, n))
    dev = wl["h_student"].device
    valid = torch.tensor(valid_rows, dtype=torch.int64, device=dev)
    scored = torch.tensor(scored_rows, dtype=torch.int64, device=dev)
    V = wl["spec"].vocab

    def timed(fn, reps):
        for _ in range(2):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    res = []

    def add(name, ms, flop):
        tf = flop / ms / 1e9
        res.append(dict(gemm=name, ms=round(ms, 4), tflops=round(tf, 1),
                        frac=round(tf / PEAK_BF16_TFLOPS, 4)))
        log("%-28s %9.3f ms %8.1f TFLOP/s" % (name, ms, tf))

    reps = max(1, min(args.steps, 10))
    F = torch.nn.functional
    # Each product in both operand layouts the library takes without a copy: "nn" =
    # torch.mm(A, B) with both row-major, "nt" = F.linear(A, B^T-stored) = A B with B
    # held transposed. The fused kernels read W as [V][d] (the "nt" form of z).
    for tag, h, w in (("z_S = h_S W_S", wl["h_student"], wl["w_student"]),
                      ("z_T = h_T W_T", wl["h_teacher"], wl["w_teacher"])):
        hv = h.index_select(0, valid).contiguous()
        flop = 2.0 * hv.shape[0] * V * hv.shape[1]
        add(tag + " nn", timed(lambda: torch.mm(hv, w), reps), flop)
        wvd = w.t().contiguous()                     # [V][d]
        add(tag + " nt", timed(lambda: F.linear(hv, wvd), reps), flop)
        del hv, wvd
    w = wl["w_student"]                              # [d_S][V]
    hr = wl["h_student"].index_select(0, scored).contiguous()
    R, d = hr.shape
    g = (torch.randn(R, V, device=dev) * 1e-3).to(torch.bfloat16)
    flop = 2.0 * R * V * d
    wvd = w.t().contiguous()                         # [V][d_S]
    add("dh = g W^T nn", timed(lambda: torch.mm(g, wvd), reps), flop)
    del wvd
    add("dh = g W^T nt", timed(lambda: F.linear(g, w), reps), flop)
    hrt = hr.t().contiguous()                        # [d_S][R]
    add("dW = h^T g nn", timed(lambda: torch.mm(hrt, g), reps), flop)
    gt = g.t().contiguous()                          # [V][R]
    add("dW = h^T g nt", timed(lambda: F.linear(hrt, gt), reps), flop)
    print(json.dumps(dict(library_gemm=res, workload=args.workload, valid_rows=int(valid.numel()),
                          scored_rows=int(R), dtype="bf16", peak_tflops=PEAK_BF16_TFLOPS)),
          flush=True)


def cpu_model() -> str:
    """The host CPU's model name (lscpu, else /proc/cpuinfo)."""
    import subprocess
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for line in out.splitlines():
            if line.lower().startswith("model name"):
                return line.split(":", 1)[1].strip()
    except (OSError, subprocess.SubprocessError):
        pass
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.lower().startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawTextHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="long_rollout")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--narrow-tile", action="store_true",
                    help="score with the 256 x 128 two-model kernel (OLIVE_FLAG_NARROW_TILE) "
                         "instead of the 256 x 256 one")
    ap.add_argument("--reverse-kl", action="store_true",
                    help="also form KL(student || teacher) in the same pass (olive_score_batch)")
    ap.add_argument("--reverse-kl-only", action="store_true",
                    help="form KL(student || teacher) instead of KL(teacher || student) "
                         "(olive_score_batch with kl_reverse set and kl NULL)")
    ap.add_argument("--jsd", action="store_true",
                    help="also form the Jensen-Shannon divergence (a second pass over the "
                         "scored rows; olive_score_batch)")
    ap.add_argument("--region-only", action="store_true",
                    help="score only the region's positions (OLIVE_OUT_REGION_ONLY): the rate "
                         "and the roofline then count scored positions")
    ap.add_argument("--topk", action="store_true",
                    help="also form the top-16 statistics (overlap ratio, top-16 KL and both "
                         "index sets; OLIVE_FLAG_TOPK)")
    ap.add_argument("--backward", action="store_true",
                    help="time olive_score_backward instead (dL/dh_S and dL/dW_S of Eq. 1's "
                         "summed loss, plus --backward-kl times the summed KL)")
    ap.add_argument("--backward-kl", type=float, default=0.0, metavar="W",
                    help="KL weight of the --backward loss (default 0: Eq. 1 alone)")
    ap.add_argument("--train-step", action="store_true",
                    help="with --backward: each step is a forward call (KL, both models' "
                         "log-probs, per-sequence CE) and a backward that reuses its "
                         "normalisers (OLIVE_GRAD_REUSE_FORWARD)")
    ap.add_argument("--library-gemm", action="store_true",
                    help="only time the plain library GEMMs (torch.mm, bf16 in and out) of "
                         "the workload's contractions: each model's logits over the valid "
                         "rows and the backward's two products over the scored rows, the "
                         "unfused path's dominant cost; prints one JSON line and exits")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="only run 3 plain device copies of BYTES bytes (for scaling the "
                         "FETCH_SIZE / WRITE_SIZE counters) and exit")
    args = ap.parse_args()
    if args.copy_calibration:
        import torch
        n = args.copy_calibration // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": n * 4, "copies": 3}), flush=True)
        return
    if args.gpus != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(--gpus %d requested)" % args.gpus, file=sys.stderr)
        sys.exit(2)
    if not 1 <= args.steps <= 64:
        print("--steps must be in [1, 64]", file=sys.stderr)
        sys.exit(2)
    if args.train_step and not args.backward:
        print("--train-step applies to --backward", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2609_36246_amd import _lib as L
    from paper_2609_36246_amd import workloads as W

    L.load()
    log("generating workload", args.workload)
    t0 = time.time()
    wl = W.make_workload(args.workload, args.seed, device="cuda")
    spec = wl["spec"]
    T = wl["total_positions"]
    B = spec.num_seqs
    log("workload ready in %.1fs: T=%d" % (time.time() - t0, T))
    if args.backward:
        bench_backward(args, wl, L)
        return
    if args.library_gemm:
        bench_library_gemm(args, wl)
        return
    desc = L.make_desc(spec.vocab, spec.d_student, spec.d_teacher,
                       L.OLIVE_BF16 if spec.dtype == "bf16" else L.OLIVE_F32, L.OLIVE_W_DV,
                       wl["scale_student"], wl["scale_teacher"], max_positions=T, max_seqs=B,
                       flags=L.OLIVE_FLAG_KERNEL_TIMING |
                       (L.OLIVE_FLAG_TOPK if args.topk else 0) |
                       (L.OLIVE_FLAG_NARROW_TILE if args.narrow_tile else 0))
    stream = torch.cuda.current_stream()
    ctx = L.olive_score_init(desc, wl["w_student"], wl["w_teacher"], stream)
    dev = wl["h_student"].device
    kl = None if args.reverse_kl_only else torch.empty(T, dtype=torch.float32, device=dev)
    counts = torch.empty(2, dtype=torch.int64, device=dev)
    lps = torch.empty(T, dtype=torch.float32, device=dev)
    lpt = torch.empty(T, dtype=torch.float32, device=dev)
    ams = torch.empty(T, dtype=torch.int32, device=dev)
    amt = torch.empty(T, dtype=torch.int32, device=dev)
    ce = torch.empty(B, dtype=torch.float32, device=dev)
    klr = torch.empty(T, dtype=torch.float32, device=dev) \
        if (args.reverse_kl or args.reverse_kl_only) else None
    tk = dict(topk_overlap=torch.empty(T, dtype=torch.float32, device=dev),
              kl_topk=torch.empty(T, dtype=torch.float32, device=dev),
              topk_student=torch.empty(T, L.OLIVE_TOPK, dtype=torch.int32, device=dev),
              topk_teacher=torch.empty(T, L.OLIVE_TOPK, dtype=torch.int32, device=dev)) \
        if args.topk else {}
    jsd = torch.empty(T, dtype=torch.float32, device=dev) if args.jsd else None
    outs = L.make_outputs(kl=kl, kl_reverse=klr, jsd=jsd, counts=counts, logp_student=lps,
                          logp_teacher=lpt, argmax_student=ams, argmax_teacher=amt,
                          ce_per_seq=ce,
                          flags=L.OLIVE_OUT_REGION_ONLY if args.region_only else 0, **tk)
    use_spans = wl.get("spans") is not None       # multi-turn: teacher actions scored
    batch = L.make_batch(wl["cu_seqlens"], None if use_spans else wl["cut"], wl["targets"],
                         wl["h_student"], wl["h_teacher"], wl["valid_len"],
                         L.OLIVE_REGION_SPANS if use_spans else L.OLIVE_REGION_TEACHER)
    spans = L.make_spans(wl["span_offsets"], wl["span_pairs"]) if use_spans else None

    def step():
        if use_spans:
            L.olive_score_batch_spans(ctx, batch, spans, outs, stream)
        elif args.reverse_kl or args.reverse_kl_only or args.jsd or args.region_only or \
                args.topk:
            L.olive_score_batch(ctx, batch, outs, stream)
        else:
            L.olive_kl_masked(ctx, batch, kl, counts, lps, lpt, ams, amt, ce, stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log("warmup done")
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(args.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    ms_total = e0.elapsed_time(e1)
    ms_step = ms_total / args.steps
    kms = L.olive_score_kernel_times(ctx, args.steps)
    kernel_ms = sum(kms) / len(kms)
    stats = L.olive_score_last_stats(ctx)
    err = L.olive_score_last_error(ctx)
    n_scored, t_valid = [int(x) for x in counts.cpu().tolist()]
    rows = n_scored if args.region_only else t_valid     # positions the pass scores
    log("timed %d steps: %.3f ms/step, scoring kernel %.3f ms, stats %s, err %d"
        % (args.steps, ms_step, kernel_ms, stats, err))
    flops = 2.0 * rows * spec.vocab * (spec.d_student + spec.d_teacher)
    achieved = flops / (kernel_ms * 1e-3) / 1e12
    # the dominant kernel of the call: the 256 x 256 one, or the 256 x 128 one (both KL
    # directions, top-K, OLIVE_FLAG_NARROW_TILE)
    kernel = "score_wide" if stats.get("tile") == "256x256" else "score_mfma"
    traffic = None if (args.reverse_kl or args.reverse_kl_only or args.jsd or
                       args.region_only or args.topk) \
        else measured_traffic(args.workload, kernel)
    out = {
        "metric": "scored positions/sec and % bf16 MFMA peak, fused LM-head+logsoftmax+KL",
        "value": rows / (ms_step * 1e-3),
        "unit": "positions/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded; random hidden states and weights of the workload's shapes)",
        "config": {
            "workload": args.workload, "num_seqs": B, "total_positions": T,
            "valid_positions": t_valid, "scored_positions": n_scored, "vocab": spec.vocab,
            "d_student": spec.d_student, "d_teacher": spec.d_teacher,
            "logit_scale": spec.logit_scale, "vocab_splits": stats["splits"],
            "reverse_kl": bool(args.reverse_kl), "reverse_kl_only": bool(args.reverse_kl_only),
            "jsd": bool(args.jsd),
            "region_only": bool(args.region_only),
            "topk": bool(args.topk), "topk_filtered_pairs": stats["topk_filtered"],
            "topk_scanned_pairs": stats["topk_scanned"],
            "region": "spans" if use_spans else "teacher",
            "near_tie_rows": stats["flagged"], "grid": stats["grid"],
            "step_tflops": flops / (ms_step * 1e-3) / 1e12,
            "pct_bf16_peak_step": 100.0 * flops / (ms_step * 1e-3) / 1e12 / PEAK_BF16_TFLOPS,
            "kernel_ms": kernel_ms,
        },
        "roofline": {
            "bound": "mfma", "achieved": achieved, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
            "frac": achieved / PEAK_BF16_TFLOPS, "traffic": traffic, "kernel": kernel + "_kernel",
        },
    }
    L.olive_score_free(ctx)
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle) on a bounded sample ...")
        out["cpu_baseline"] = cpu_baseline(wl, args.cpu_seconds)
    print(json.dumps(out), flush=True)


def bench_backward(args, wl, L):
    """One olive_score_backward call per step: the forward normalisers of the scored
    rows, the logit gradient and the two products, both gradients requested. With
    --train-step, a forward call first, whose normalisers the backward reuses."""
    import torch
    spec = wl["spec"]
    T = wl["total_positions"]
    B = spec.num_seqs
    desc = L.make_desc(spec.vocab, spec.d_student, spec.d_teacher, L.OLIVE_BF16, L.OLIVE_W_DV,
                       wl["scale_student"], wl["scale_teacher"], max_positions=T, max_seqs=B,
                       flags=L.OLIVE_FLAG_BACKWARD)
    stream = torch.cuda.current_stream()
    ctx = L.olive_score_init(desc, wl["w_student"], wl["w_teacher"], stream)
    dev = wl["h_student"].device
    gh = torch.empty((T, spec.d_student), dtype=torch.float32, device=dev)
    gw = torch.empty((spec.d_student, spec.vocab), dtype=torch.float32, device=dev)
    use_spans = wl.get("spans") is not None
    batch = L.make_batch(wl["cu_seqlens"], None if use_spans else wl["cut"], wl["targets"],
                         wl["h_student"], wl["h_teacher"], wl["valid_len"],
                         L.OLIVE_REGION_SPANS if use_spans else L.OLIVE_REGION_TEACHER)
    spans = L.make_spans(wl["span_offsets"], wl["span_pairs"]) if use_spans else None
    counts = torch.zeros(2, dtype=torch.int64, device=dev)
    train = args.train_step
    g = L.make_grad_outputs(1.0, args.backward_kl, gh, gw, counts, reuse_forward=train)
    if train:
        f32 = dict(dtype=torch.float32, device=dev)
        fo = L.make_outputs(kl=torch.empty(T, **f32), logp_student=torch.empty(T, **f32),
                            logp_teacher=torch.empty(T, **f32),
                            ce_per_seq=torch.empty(B, **f32))

    def step():
        if train:
            if spans is not None:
                L.olive_score_batch_spans(ctx, batch, spans, fo, stream=stream)
            else:
                L.olive_score_batch(ctx, batch, fo, stream=stream)
        L.olive_score_backward(ctx, batch, g, spans=spans, stream=stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log("warmup done")
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(args.steps):
        step()
    e1.record(stream)
    torch.cuda.synchronize()
    ms_step = e0.elapsed_time(e1) / args.steps
    err = L.olive_score_last_error(ctx)
    L.olive_score_free(ctx)
    R = int(counts[0].item())
    Tv = int(counts[1].item())
    dt = spec.d_teacher if args.backward_kl else 0
    if train:
        # the forward projects both models over the valid rows; the backward's
        # logit-gradient pass and its two products
        flops = 2.0 * spec.vocab * (Tv * (spec.d_student + spec.d_teacher) +
                                    R * (spec.d_student + dt + 2 * spec.d_student))
    else:
        # the two products are 2 R V d_S each. A cross-entropy-only backward on the
        # 256 x 256 pipeline projects the student once (its logit-gradient pass forms the
        # normalisers); otherwise a normaliser pass and the logit-gradient pass each
        # project the models of the loss
        proj = 1 if (not args.backward_kl and not args.narrow_tile) else 2
        flops = 2.0 * R * spec.vocab * (proj * (spec.d_student + dt) + 2 * spec.d_student)
    log("timed %d %s steps: %.3f ms/step, err %d"
        % (args.steps, "training" if train else "backward", ms_step, err))
    out = {
        "metric": ("scored positions/sec, training step (forward outputs + backward reusing "
                   "its normalisers) of the masked CE" if train else
                   "scored positions/sec, backward (dL/dh_S, dL/dW_S) of the masked CE"),
        "value": R / (ms_step * 1e-3), "unit": "positions/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded; random hidden states and weights of the workload's shapes)",
        "config": {"workload": args.workload, "scored_positions": R, "vocab": spec.vocab,
                   "d_student": spec.d_student, "d_teacher": spec.d_teacher,
                   "w_ce": 1.0, "w_kl": args.backward_kl, "train_step": train,
                   "valid_positions": Tv,
                   "step_tflops": flops / (ms_step * 1e-3) / 1e12,
                   "pct_bf16_peak_step": 100.0 * flops / (ms_step * 1e-3) / 1e12 /
                   PEAK_BF16_TFLOPS},
    }
    print(json.dumps(out), flush=True)


def measured_traffic(workload: str, kernel: str):
    """HBM bytes per launch of a scoring kernel from the committed rocprofv3 counter
    summary of this workload (FETCH_SIZE and WRITE_SIZE, scaled by a plain copy's
    readings), or None when there is none for the current kernel source."""
    path = os.path.join(PROFILES, "%s_%s_traffic.txt" % (kernel, workload))
    if not os.path.exists(path):
        return None
    fields = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.startswith((" ", "#", "$")):
                k, v = line.split(":", 1)
                fields[k.strip()] = v.strip()
    if fields.get("kernel_source_sha") != kernel_source_sha(kernel):
        return None
    try:
        return float(fields["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


# Each scoring kernel's source and the headers it includes.
KERNEL_SOURCES = {
    "score_mfma": ("score_mfma.hip", "fold.hpp", "mfma_pipe.hpp", "olive_device.hpp",
                   "olive_internal.hpp", "phase_lock.hpp"),
    "score_wide": ("score_wide.hip", "wide_pipe.hpp", "fold.hpp", "mfma_pipe.hpp",
                   "olive_device.hpp", "olive_internal.hpp", "phase_lock.hpp"),
}


def kernel_source_sha(kernel: str = "score_wide") -> str:
    import hashlib
    csrc = os.path.join(os.path.dirname(os.path.abspath(__file__)), "paper_2609_36246_amd",
                        "csrc")
    h = hashlib.sha256()
    for name in KERNEL_SOURCES[kernel]:
        with open(os.path.join(csrc, name), "rb") as f:
            h.update(name.encode() + b"\0" + f.read())
    return h.hexdigest()[:16]


if __name__ == "__main__":
    main()
