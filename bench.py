#!/usr/bin/env python3
"""Benchmark of the per-layer OJBKQ quantisation path on one MI355X.

One step = the whole path for one layer: Gram and cross term over every
calibration token, damping, Cholesky and L^-1, the relaxed solution folded
into the decoder's input Rbar qbar, Klein temperatures, the batched Babai + K Klein decode of every column and
the selection, with the synthetic inputs already resident in HBM.

Default workload: the Llama-7B-shaped attention projection, W 4096 x 4096
(n = 4096 output channels, m = 4096 input features), X_ref / X_q 4096 x
262144 calibration tokens with heavy-tailed per-channel scales, 4-bit,
group 128, K = 16 Klein samples, alpha (the JTA knob) = 0.5.

Prints one JSON line.  value = n (K + 1) / layer time, i.e. candidate paths
(columns x samples) decoded per second, end to end (times the number of JTA
knobs when a workload sweeps several on one factor).  The roofline object is
for the dominant kernel, the fused Gram + cross-term contraction, timed with
HIP events on the stream it is launched on (for layers with n <= 0.4 m,
whose cross term is accumulated already multiplied by W, the accumulate call
as a whole: the Gram kernel and the two projection GEMMs).  The CPU baseline times the oracle
on a bounded sample of the same workload on this host and extrapolates.
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "layer quantize time (s) and columns×samples decoded/sec; % MFMA/HBM peak"
PEAK_F64_MFMA_TFLOPS = 78.6     # MI355X dense fp64 matrix peak
PEAK_I8_MFMA_TOPS = 5000.0      # MI355X dense int8 matrix peak (5.0 POP/s)
PEAK_HBM_GBS = 8000.0
I8_DIGIT_PRODUCTS = 13          # int8 digit products per entry and token (gram_i8.hip)


def act_order_arg(args):
    """The binding's act_order value for --act-order."""
    return {None: False, "positions": True, "static": "static"}[args.act_order]


def packing_perm(args, q):
    """The order to pack codes in: the decode order when the scale groups
    follow it, else W's own (no act order, or static groups)."""
    return q.perm if args.act_order == "positions" else None


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--config", default="c2", help="workload key (c1..c5)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-tokens", type=int, default=16384,
                    help="tokens of the oracle's timed Gram/cross sample")
    ap.add_argument("--cpu-columns", type=int, default=24,
                    help="columns of the oracle's timed solve/decode sample")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run one 1 GiB streaming negation (for scaling HBM counters)")
    ap.add_argument("--sweep-k", metavar="SHAPES", default=None,
                    help="instead of the benchmark line: one JSON line per (layer, K) with the "
                         "layer time and the mean JTA residual, on the Llama-3-8B-shaped layers "
                         "given as a comma list of l3_* keys or 'all'")
    ap.add_argument("--k-values", default="0,1,5,10,25,50", help="K values of --sweep-k")
    ap.add_argument("--sweep-mu", metavar="SHAPES", default=None,
                    help="instead of the benchmark line: one JSON line per (layer, alpha) with "
                         "the output error against the full-precision target and against the "
                         "quantized input, on one factor per layer (l3_* keys or 'all')")
    ap.add_argument("--mu-values", default="0,0.2,0.4,0.6,0.8,1", help="alpha values of --sweep-mu")
    ap.add_argument("--act-order", nargs="?", const="positions", default=None,
                    choices=("positions", "static"),
                    help="weight permutation: decide the features with the largest Hessian "
                         "diagonal first (every mode); scale groups by decode position "
                         "(default) or kept as W's own groups (static)")
    ap.add_argument("--gram", default="int8", choices=("int8", "fp64"),
                    help="arithmetic of the token sums: int8 digit products (default) or fp64")
    ap.add_argument("--scheme", default="asym", choices=("asym", "sym"),
                    help="scales and zero points: asymmetric min-max or symmetric Absmax")
    ap.add_argument("--mlp-stack", action="store_true",
                    help="instead of the benchmark line: quantize a synthetic stack of layers in "
                         "order, each on the activations of the layers already quantized (formed "
                         "with the packed-code product), and report per-layer output errors")
    ap.add_argument("--adaptive", action="store_true",
                    help="with --mlp-stack: pick lambda, alpha and K per layer on held-out tokens")
    ap.add_argument("--stack-layers", type=int, default=4)
    ap.add_argument("--stack-dim", type=int, default=4096)
    ap.add_argument("--stack-tokens", type=int, default=32768)
    return ap.parse_args()


def sweep_k(args):
    """Layer time and selected residual against K (the paper's ablation over
    K and its figure of the per-layer time increase with K), one fresh layer
    per K: Gram, factor, solves, decode and selection all rerun."""
    import torch
    import paper_2602_08376_amd as ok
    from synth import LLAMA3_8B
    from synth.workloads import activation_chunks, make_weights

    keys = list(LLAMA3_8B) if args.sweep_k == "all" else args.sweep_k.split(",")
    ks = [int(k) for k in args.k_values.split(",")]
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    ok.library()
    for key in keys:
        cfg = LLAMA3_8B[key]
        W = make_weights(cfg, device=dev)
        chunks = list(activation_chunks(cfg, device=dev))
        torch.cuda.synchronize()
        log(f"sweep {key}: inputs generated")

        def layer(K):
            s = ok.LayerSolver(cfg.m, cfg.n, cfg.bits, cfg.group, K, cfg.klein_seed,
                               cfg.lambda_rel, device=dev, scheme=args.scheme,
                               act_order=act_order_arg(args))
            s.set_timing(True)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            s.set_weights(W)
            for Xr, Xq in chunks:
                s.accumulate(Xr, Xq)
            out = s.solve(W, cfg.mu)
            torch.cuda.synchronize()
            t = time.perf_counter() - t0
            stages = s.stage_times()
            s.close()
            return t, out, stages

        layer(ks[0])   # warm-up: first launches of every kernel
        base = None
        for K in ks:
            t, out, stages = layer(K)
            res = out.residuals.double()
            mean_r = float(res.mean())
            if base is None:
                base = (t, mean_r, res)
            line = {
                "sweep": "K", "workload": f"{key}: {cfg.title}", "K": K,
                "n_out": cfg.n, "m_in": cfg.m, "tokens": cfg.T, "bits": cfg.bits,
                "group": cfg.group, "alpha": cfg.mu, "scheme": args.scheme,
                "act_order": args.act_order, "layer_time_s": t, "time_ratio_vs_first": t / base[0],
                "decode_ms": stages["decode"],
                "decode_paths_per_s": cfg.n * (K + 1) / (stages["decode"] * 1e-3),
                "mean_residual": mean_r, "residual_ratio_vs_first": mean_r / base[1],
                "columns_improved_vs_first": float((res < base[2]).double().mean()),
                "klein_wins": float((out.winner > 0).double().mean()),
            }
            print(json.dumps(line), flush=True)
            log(f"sweep {key} K={K}: {t * 1e3:.1f} ms, mean residual {mean_r:.6e}")
        del W, chunks
        torch.cuda.empty_cache()


# the sources that decide each measured kernel's traffic (its file, the shared
# device helpers and the launch constants in kernels.h)
KERNEL_SOURCES = {
    "gram_cross_kernel": ("paper_2602_08376_amd/csrc/gram.hip", "paper_2602_08376_amd/csrc/device.h",
                          "paper_2602_08376_amd/csrc/kernels.h"),
    "gram_i8": ("paper_2602_08376_amd/csrc/gram_i8.hip", "paper_2602_08376_amd/csrc/device.h",
                "paper_2602_08376_amd/csrc/kernels.h"),
}


def measured_traffic(kernel, workload):
    """HBM bytes per launch from the committed rocprofv3 FETCH_SIZE / WRITE_SIZE passes.

    Returns None when no summary covers (kernel, workload) or when the kernel's
    sources changed since the counters were taken (hash recorded in the summary).
    """
    import glob
    import hashlib
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES[kernel]:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    digest = h.hexdigest()[:16]
    for path in sorted(glob.glob(os.path.join(ROOT, "profiles", "*.md"))):
        with open(path) as f:
            for line in f:
                if not line.startswith("traffic "):
                    continue
                kv = dict(t.split("=", 1) for t in line.split()[1:])
                if (kv.get("kernel") == kernel and kv.get("workload") == workload
                        and kv.get("source_sha256_16") == digest):
                    return float(kv["bytes_per_launch"])
    return None


def workload_desc(cfg):
    return {
        "workload": f"{cfg.key}: {cfg.title}",
        "n_out": cfg.n, "m_in": cfg.m, "tokens": cfg.T, "bits": cfg.bits, "group": cfg.group,
        "K": cfg.K, "alpha": list(cfg.mus) if len(cfg.mus) > 1 else cfg.mu,
        "lambda_rel": cfg.lambda_rel, "token_chunks": cfg.chunks,
    }


def cpu_baseline(cfg, W, Xr, Xq, tokens, columns, scheme="asym"):
    """The oracle as it stands, timed stage by stage on a bounded sample, extrapolated."""
    import numpy as np
    from oracle import ojbkq as orc
    try:
        from threadpoolctl import threadpool_info
        blas_threads = max([int(i.get("num_threads", 1)) for i in threadpool_info()] or [1])
    except Exception:
        blas_threads = len(os.sched_getaffinity(0))
    Ts = min(tokens, cfg.T)
    ns = min(columns, cfg.n)
    Wn = W[:ns].cpu().numpy()
    Xrn = Xr[:, :Ts].cpu().numpy()
    Xqn = Xq[:, :Ts].cpu().numpy()
    t = {}
    t0 = time.perf_counter()
    S, Z = orc.scales_zeros(Wn, cfg.bits, cfg.group, scheme)
    t["scales"] = time.perf_counter() - t0
    t0 = time.perf_counter()
    G = orc.gram(Xqn)
    t["gram"] = time.perf_counter() - t0
    lam2 = orc.damping(G, cfg.lambda_rel)
    t0 = time.perf_counter()
    R = orc.cholesky_upper(G + lam2 * np.eye(cfg.m))
    t["cholesky"] = time.perf_counter() - t0
    t0 = time.perf_counter()
    V = orc.relaxed_solution(Wn, Xrn, Xqn, cfg.mu, lam2, R)
    t["relaxed"] = time.perf_counter() - t0
    qb = orc.centres(V, S, Z, cfg.group)
    t0 = time.perf_counter()
    orc.decode(R, qb, S, cfg.bits, cfg.group, cfg.K, cfg.klein_seed)
    t["decode"] = time.perf_counter() - t0
    sample_s = sum(t.values())
    tok_x, col_x = cfg.T / Ts, cfg.n / ns
    # the oracle's relaxed solution forms X~^T y* per column over the tokens
    layer_s = (t["gram"] * tok_x + t["cholesky"] + t["relaxed"] * tok_x * col_x
               + (t["decode"] + t["scales"]) * col_x)
    return {
        "value": cfg.n * (cfg.K + 1) / layer_s,
        "unit": "columns*samples/s",
        "cores": blas_threads,
        "kind": "oracle",
        "layer_s_extrapolated": layer_s,
        "sample_s": sample_s,
        "stage_s": {k: round(v, 4) for k, v in t.items()},
        "sample": (f"fp64 numpy oracle on this host: Gram on {Ts} of {cfg.T} tokens "
                   f"(x{tok_x:g}), damped Cholesky of the full {cfg.m}x{cfg.m} Gram, relaxed "
                   f"solution over {Ts} tokens for {ns} of {cfg.n} columns (x{tok_x * col_x:g}), "
                   f"decode of all {cfg.K + 1} candidates of {ns} columns (x{col_x:g}); "
                   f"layer time extrapolated linearly"),
    }


PEAK_F16_MFMA_TFLOPS = 2500.0   # MI355X dense fp16 matrix peak


def mlp_stack(args):
    """Layer-by-layer quantization of a synthetic stack y = W_l silu(...):
    layer l is quantized on X = the full-precision activations and X~ = the
    activations of the stack whose layers 0..l-1 are already quantized (the
    setting of the paper's JTA target), and X~ of the next layer is formed
    from the packed codes with the dequantize-and-multiply kernel.  Reports
    the relative output error of every layer for (alpha, K) in
    {1, 0.6} x {0, 16}: alpha = 1 drops the cross term (each layer fits its
    own quantized input), alpha = 0.6 is the paper's setting; and the
    dequantize-and-multiply kernel against the fp16 MFMA roofline.

    The full-precision forward pass and the SiLU between layers are the
    synthetic model, computed with torch; every quantization step and the
    quantized product run in the library."""
    import torch
    import paper_2602_08376_amd as ok
    from synth import LayerConfig
    from synth.workloads import activation_chunks, make_weights

    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    ok.library()
    d, L, T, bits, group = args.stack_dim, args.stack_layers, args.stack_tokens, 4, 128
    base = LayerConfig(key="stack", title="synthetic MLP stack", n=d, m=d, T=T, bits=bits,
                       group=group, K=16, mus=(0.6,), w_std=0.02, kind="heavy", data_seed=21,
                       noise=0.0)
    Ws = [make_weights(dataclass_replace(base, data_seed=21 + l), device=dev) for l in range(L)]
    (X0, _), = list(activation_chunks(base, device=dev))
    silu = torch.nn.functional.silu

    def product_ms(fn, reps=10):
        # one call for the output, then the mean of `reps` back-to-back calls
        st = torch.cuda.current_stream(dev)
        out = fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(st)
        for _ in range(reps):
            fn()
        e1.record(st)
        e1.synchronize()
        return out, e0.elapsed_time(e1) / reps

    for mu, K in ((1.0, 0), (1.0, 16), (0.6, 0), (0.6, 16)):
        X, Xq = X0, X0
        errs, qtimes, dq, dq_tiles = [], [], [], []
        for l, W in enumerate(Ws):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            s = ok.LayerSolver(d, d, bits, group, K, 0, 0.01, device=dev, scheme=args.scheme,
                               act_order=act_order_arg(args))
            s.set_weights(W)
            s.accumulate(X, Xq)
            q = s.solve(W, mu)
            torch.cuda.synchronize()
            qtimes.append(time.perf_counter() - t0)
            s.close()
            pp = packing_perm(args, q)                   # decode order, position groups
            P = ok.pack_codes(q.codes, bits, pp)
            Xq16 = Xq.half()
            ws = torch.empty(ok.library().ojbkq_dequant_matmul_workspace_bytes(d, d),
                             dtype=torch.uint8, device=dev)
            Yq, ms = product_ms(lambda: ok.dequant_matmul(P, q.scales, q.zeros, d, bits, group,
                                                          Xq16, pp, workspace=ws))
            dq.append(ms)
            _, ms_tiles = product_ms(lambda: ok.dequant_matmul(P, q.scales, q.zeros, d, bits,
                                                               group, Xq16, pp, workspace=False))
            dq_tiles.append(ms_tiles)
            Y = W @ X                                  # the full-precision stack
            errs.append(float((Yq - Y).norm() / Y.norm()))
            X, Xq = silu(Y), silu(Yq)
            del Y, Yq, P, Xq16
        flops = 2.0 * d * d * T
        line = {"mlp_stack": True, "alpha": mu, "K": K, "layers": L, "dim": d, "tokens": T,
                "bits": bits, "group": group, "scheme": args.scheme,
                "act_order": args.act_order, "relative_output_error": errs, "quantize_s": qtimes,
                "dequant_matmul_ms": dq,
                # the same product without a workspace (dequantized per tile)
                "dequant_matmul_per_tile_ms": dq_tiles,
                "dequant_matmul_roofline": {"bound": "mfma", "unit": "TFLOP/s",
                                            "achieved": flops / (min(dq) * 1e-3) / 1e12,
                                            "peak": PEAK_F16_MFMA_TFLOPS,
                                            "frac": flops / (min(dq) * 1e-3) / 1e12 /
                                            PEAK_F16_MFMA_TFLOPS}}
        print(json.dumps(line), flush=True)
        log(f"stack alpha={mu} K={K}: errors {[round(e, 5) for e in errs]}")


def adaptive_stack(args):
    """Per-layer knobs (the paper fixes mu, lambda and K for every layer and
    names per-layer choices as future work), on the synthetic stack of
    --mlp-stack.  The tokens are split 3:1 into a fit set, on which every
    layer is quantized, and a held-out set.  For each layer: lambda_rel in
    {0.001, 0.01, 0.1} x alpha in {0, 0.2, .., 1} at K = 0, then K in
    {0, 4, 16} at the best pair, each candidate scored by the held-out output
    error ||W_hat X~_v - W X_v|| / ||W X_v|| (the full-precision target the
    JTA objective serves); one context per layer serves the whole search
    (one Gram, one factor per lambda).  A second stack runs the fixed knobs
    (lambda_rel 0.01, alpha 0.6, K 16) on the same fit tokens; each stack
    feeds its own X~ forward.  Errors are reported on all tokens and on the
    held-out ones."""
    import torch
    import paper_2602_08376_amd as ok
    from synth import LayerConfig
    from synth.workloads import activation_chunks, make_weights

    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    ok.library()
    d, L, T, bits, group = args.stack_dim, args.stack_layers, args.stack_tokens, 4, 128
    Tf = (3 * T // 4) // 256 * 256
    base = LayerConfig(key="stack", title="synthetic MLP stack", n=d, m=d, T=T, bits=bits,
                       group=group, K=16, mus=(0.6,), w_std=0.02, kind="heavy", data_seed=21,
                       noise=0.0)
    Ws = [make_weights(dataclass_replace(base, data_seed=21 + l), device=dev) for l in range(L)]
    (X0, _), = list(activation_chunks(base, device=dev))
    silu = torch.nn.functional.silu
    lams, mus, ks = (0.001, 0.01, 0.1), (0.0, 0.2, 0.4, 0.6, 0.8, 1.0), (0, 4, 16)

    def product(q, Xq16):
        pp = packing_perm(args, q)
        P = ok.pack_codes(q.codes, bits, pp)
        return ok.dequant_matmul(P, q.scales, q.zeros, d, bits, group, Xq16, pp)

    def quantize(W, X, Xq, search):
        s = ok.LayerSolver(d, d, bits, group, max(ks), 0, 0.01, device=dev,
                           scheme=args.scheme, act_order=act_order_arg(args), keep_gram=True)
        s.set_weights(W)
        s.accumulate(X[:, :Tf], Xq[:, :Tf])
        Yv = W @ X[:, Tf:]
        nv = float(Yv.norm())
        Xv16 = Xq[:, Tf:].contiguous().half()

        def held_out(q):
            return float((product(q, Xv16) - Yv).norm()) / nv

        if not search:
            s.set_knobs(0.01, 16)
            q = s.solve(W, 0.6)
            s.close()
            return q, (0.01, 0.6, 16), None
        best, trail = None, []
        for lam in lams:
            s.set_knobs(lam, 0)
            for mu in mus:
                e = held_out(s.solve(W, mu))
                trail.append((lam, mu, 0, e))
                if best is None or e < best[3]:
                    best = (lam, mu, 0, e)
        lam, mu = best[0], best[1]
        for K in ks[1:]:
            s.set_knobs(lam, K)
            e = held_out(s.solve(W, mu))
            trail.append((lam, mu, K, e))
            if e < best[3]:
                best = (lam, mu, K, e)
        s.set_knobs(best[0], best[2])
        q = s.solve(W, best[1])
        s.close()
        return q, best[:3], trail

    for search in (False, True):
        X, Xq = X0, X0
        errs, errs_v, knobs, times = [], [], [], []
        for l, W in enumerate(Ws):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            q, kn, _ = quantize(W, X, Xq, search)
            torch.cuda.synchronize()
            times.append(time.perf_counter() - t0)
            Yq = product(q, Xq.half())
            Y = W @ X
            errs.append(float((Yq - Y).norm() / Y.norm()))
            errs_v.append(float((Yq[:, Tf:] - Y[:, Tf:]).norm() / Y[:, Tf:].norm()))
            knobs.append({"lambda_rel": kn[0], "alpha": kn[1], "K": kn[2]})
            X, Xq = silu(Y), silu(Yq)
            del Y, Yq
        line = {"mlp_stack": True, "knobs": "per-layer search" if search else "fixed",
                "layers": L, "dim": d, "tokens": T, "fit_tokens": Tf, "bits": bits,
                "group": group, "scheme": args.scheme, "act_order": args.act_order,
                "chosen": knobs, "relative_output_error": errs,
                "relative_output_error_held_out": errs_v, "quantize_and_search_s": times}
        print(json.dumps(line), flush=True)
        log(f"stack {'search' if search else 'fixed'}: errors {[round(e, 5) for e in errs]}, "
            f"knobs {knobs}")


def sweep_mu(args):
    """The JTA knob's trade-off on one layer (the paper's mu ablation): for
    each alpha the relative output errors ||W_hat X~ - W X|| / ||W X|| (the
    full-precision target, Eq. obj_mismatch) and ||(W_hat - W) X~|| / ||W X~||
    (the quantized input, Eq. obj_rt), all alpha values on one factor.  The
    errors are evaluated with torch in float32 from the dequantized weights;
    the quantization runs in the library."""
    import torch
    import paper_2602_08376_amd as ok
    from synth import LLAMA3_8B
    from synth.workloads import activation_chunks, make_weights

    keys = list(LLAMA3_8B) if args.sweep_mu == "all" else args.sweep_mu.split(",")
    mus = [float(x) for x in args.mu_values.split(",")]
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    ok.library()
    for key in keys:
        cfg = LLAMA3_8B[key]
        W = make_weights(cfg, device=dev)
        (X, Xq), = list(activation_chunks(cfg, device=dev))
        Y = W @ X
        Yq = W @ Xq
        ny, nyq = float(Y.norm()), float(Yq.norm())
        s = ok.LayerSolver(cfg.m, cfg.n, cfg.bits, cfg.group, cfg.K, cfg.klein_seed,
                           cfg.lambda_rel, device=dev, scheme=args.scheme,
                           act_order=act_order_arg(args))
        s.set_weights(W)
        s.accumulate(X, Xq)
        g = ok.num_groups(cfg.m, cfg.group)
        gs = cfg.m if cfg.group <= 0 or cfg.group >= cfg.m else cfg.group
        for mu in mus:
            q = s.solve(W, mu)
            # group of every input feature: that of its decode position
            gidx = torch.arange(cfg.m, device=dev) // gs
            if packing_perm(args, q) is not None:
                gidx = torch.empty_like(gidx).index_copy_(0, q.perm.long(), gidx)
            Sx = q.scales[:, gidx]
            Zx = q.zeros[:, gidx]
            Wh = Sx * (q.codes.float() - Zx)
            Yh = Wh @ Xq
            line = {"sweep": "alpha", "workload": f"{key}: {cfg.title}", "alpha": mu, "K": cfg.K,
                    "scheme": args.scheme, "act_order": args.act_order, "groups": g,
                    "error_vs_full_precision": float((Yh - Y).norm()) / ny,
                    "error_vs_quantized_input": float((Yh - Yq).norm()) / nyq,
                    "mean_reduced_residual": float(q.residuals.double().mean())}
            print(json.dumps(line), flush=True)
            log(f"sweep {key} alpha={mu}: {line['error_vs_full_precision']:.5f} / "
                f"{line['error_vs_quantized_input']:.5f}")
            del Sx, Zx, Wh, Yh
        s.close()
        del W, X, Xq, Y, Yq
        torch.cuda.empty_cache()


def dataclass_replace(cfg, **kw):
    import dataclasses
    return dataclasses.replace(cfg, **kw)


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}, WORLD_SIZE {world}): "
              "the path runs on a single GPU (it would shard over output columns, each GPU "
              "decoding its own columns against a replicated factor)",
              file=sys.stderr)
        sys.exit(2)
    if args.sweep_k:
        sweep_k(args)
        return
    if args.mlp_stack:
        (adaptive_stack if args.adaptive else mlp_stack)(args)
        return
    if args.sweep_mu:
        sweep_mu(args)
        return

    import torch
    import paper_2602_08376_amd as ok
    from synth import CONFIGS
    from synth.workloads import activation_chunks, make_weights

    cfg = CONFIGS[args.config]
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    ok.library()
    log(f"workload {cfg.key}: {cfg.title}")
    t0 = time.perf_counter()
    W = make_weights(cfg, device=dev)
    chunks = list(activation_chunks(cfg, device=dev))
    torch.cuda.synchronize()
    log(f"inputs generated on the GPU in {time.perf_counter() - t0:.1f} s "
        f"({sum(x.numel() * 8 for x, _ in chunks) / 2**30:.1f} GiB of activations)")

    need = ok.workspace_bytes(cfg.m, cfg.n, cfg.bits, cfg.group, cfg.K, cfg.mu, cfg.lambda_rel,
                              cfg.klein_seed, act_order=act_order_arg(args), gram=args.gram)
    ws = torch.empty(need, dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream(dev)
    log(f"workspace {need / 2**30:.2f} GiB")

    def step(record):
        s = ok.LayerSolver(cfg.m, cfg.n, cfg.bits, cfg.group, cfg.K, cfg.klein_seed,
                           cfg.lambda_rel, device=dev, workspace=ws, scheme=args.scheme,
                           act_order=act_order_arg(args), gram=args.gram)
        s.set_timing(True)                        # per-stage HIP events inside the library
        s.set_weights(W)                          # lets thin layers skip the m x m cross term
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2 * len(chunks) + 1)]
        for i, (Xr, Xq) in enumerate(chunks):
            ev[2 * i].record(stream)
            s.accumulate(Xr, Xq)              # one gram_cross launch per chunk
            ev[2 * i + 1].record(stream)
        for mu in cfg.mus:                    # one factor serves every JTA knob
            out = s.solve(W, mu)
        ev[-1].record(stream)
        stages = s.stage_times()
        s.close()
        if record is not None:
            record.append((ev, out, stages))
        return out

    for w in range(args.warmup):
        step(None)
        log(f"warmup step {w + 1}/{args.warmup} done")
    torch.cuda.synchronize()
    recs = []
    t0 = time.perf_counter()
    for k in range(args.steps):
        step(recs)
        log(f"timed step {k + 1}/{args.steps} done")
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = wall * 1e3 / args.steps

    gc_ms, solve_ms = [], []
    stage_ms = {k: sum(r[2][k] for r in recs) / len(recs) for k in ok.STAGES}
    for ev, _, _ in recs:
        for i in range(len(chunks)):
            gc_ms.append(ev[2 * i].elapsed_time(ev[2 * i + 1]))
        solve_ms.append(ev[2 * len(chunks) - 1].elapsed_time(ev[-1]))
    gc_avg = sum(gc_ms) / len(gc_ms)
    m, T = cfg.m, cfg.T
    Tc = T // cfg.chunks
    i8 = args.gram == "int8"
    projected = ok.projects_cross_term(m, cfg.n, gram=args.gram)
    # per accumulate call, the method's work: the Gram's lower half m^2 Tc,
    # plus the cross term X~^T (X - X~), 2 m^2 Tc, or (thin layers, weights
    # bound) W (X - X~) and its product with X~^T, 4 n m Tc
    flops = m * m * Tc + (4.0 * cfg.n * m * Tc if projected else 2.0 * m * m * Tc)
    achieved = flops / (gc_avg * 1e-3) / 1e12
    # the int8 digit products that carry it: 13 per entry and token, over the
    # Gram's lower triangle m (m + 1) / 2 and (unless projected) the m^2
    # cross-term entries, 2 operations per multiply-add
    i8_ops = (2.0 * I8_DIGIT_PRODUCTS * Tc *
              (m * (m + 1) / 2 + (0.0 if projected else float(m) * m)))
    i8_achieved = i8_ops / (gc_avg * 1e-3) / 1e12
    paths = cfg.n * (cfg.K + 1) * len(cfg.mus)
    dec_flops = float(m) * m * paths     # m^2 per candidate path (the strict triangle, 2 FLOP/MAC)
    out = recs[-1][1]
    result = {
        "metric": METRIC,
        "value": paths / (ms_step * 1e-3),
        "unit": "columns*samples/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "layer_time_s": ms_step * 1e-3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "i8/f64" if i8 else "f64",
        "data": "synthetic (seeded, generated on the GPU; inputs resident in HBM)",
        "config": {**workload_desc(cfg), **({"scheme": "sym"} if args.scheme == "sym" else {}),
                   **({"act_order": args.act_order} if args.act_order else {})},
        "stages_ms": {"gram_cross_per_launch": gc_avg,
                      "rest_of_path": sum(solve_ms) / len(solve_ms),
                      **{f"library_{k}": v for k, v in stage_ms.items()}},
        "roofline": ({
            "bound": "mfma",
            "kernel": ("gram_i8 (row exponents, split, int8 digit contraction, fix-up; "
                       "one accumulate call)" + (" + fp64 projection GEMMs" if projected else "")),
            "achieved": i8_achieved,
            "peak": PEAK_I8_MFMA_TOPS,
            "unit": "TOP/s",
            "frac": i8_achieved / PEAK_I8_MFMA_TOPS,
            "traffic": None if projected else measured_traffic("gram_i8", cfg.key),
            "algorithmic_ops_per_launch": i8_ops,
            "method_flops_per_launch": flops,
            "fp64_equivalent_tflops": achieved,
            # activations read twice (exponents, split), the digits written and
            # read once; G and E written
            "algorithmic_bytes_per_launch": 16.0 * m * Tc + 16.0 * m * Tc + (
                8.0 * m * m + 20.0 * cfg.n * m if projected else 16.0 * m * m),
        } if i8 else {
            "bound": "mfma",
            "kernel": ("gram_cross_kernel + projection GEMMs (accumulate call)" if projected
                       else "gram_cross_kernel"),
            "achieved": achieved,
            "peak": PEAK_F64_MFMA_TFLOPS,
            "unit": "TFLOP/s",
            "frac": achieved / PEAK_F64_MFMA_TFLOPS,
            "traffic": None if projected else measured_traffic("gram_cross_kernel", cfg.key),
            "algorithmic_flops_per_launch": flops,
            # activations read once; G (and E) written, or W read and U updated
            "algorithmic_bytes_per_launch": 8.0 * m * Tc + (
                8.0 * m * m + 20.0 * cfg.n * m if projected else 16.0 * m * m),
        }),
        "decode_roofline": {
            "bound": "mfma",
            "kernel": "decode_kernel",
            "achieved": dec_flops / (stage_ms["decode"] * 1e-3) / 1e12,
            "peak": PEAK_F64_MFMA_TFLOPS,
            "unit": "TFLOP/s",
            "frac": dec_flops / (stage_ms["decode"] * 1e-3) / 1e12 / PEAK_F64_MFMA_TFLOPS,
            "algorithmic_flops_per_step": dec_flops,
            "paths_per_s": paths / (stage_ms["decode"] * 1e-3),
        },
        "checks": {"codes_max": int(out.codes.max()),
                   "mean_winner_is_klein": float((out.winner > 0).float().mean()),
                   "mean_residual": float(out.residuals.double().mean())},
    }
    if args.copy_calibration:
        # a written source (a never-written one can read back nothing from
        # HBM), then one streaming pass over it: a negation, whose kernel no
        # other step launches, reads 1 GiB and writes 1 GiB
        a = torch.empty(1 << 28, dtype=torch.float32, device=dev).uniform_()
        b = torch.empty_like(a)
        torch.cuda.synchronize()
        torch.neg(a, out=b)
        torch.cuda.synchronize()
        result["copy_calibration_bytes"] = a.numel() * 4
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a bounded sample")
        Xr0, Xq0 = chunks[0]
        result["cpu_baseline"] = cpu_baseline(cfg, W, Xr0, Xq0, args.cpu_tokens, args.cpu_columns,
                                              args.scheme)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
