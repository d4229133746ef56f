"""Benchmark of one speculative verification step on one MI355X.

A step is the whole hot path over one batch of synthetic inputs resident in HBM:
  sr_heads_propose (heads + vocabulary projection + draft tree)
  -> sr_tree_verify_attn (tree-masked attention over the paged prefix, one layer)
  -> sr_tree_accept (exact acceptance walk).
After the timed steps, the calls around the step are timed on their own and reported beside it: the
accepted-path cache commit (sr_commit_path) of the last step's accepted paths for all 28 layers of the
7B-shaped target, the acceptance walk with nucleus truncation (top_p 0.95, as the paper's rollouts
sample), the Reflex feedback (sr_reflex_feedback) of one matured record per (trajectory,
horizon) slot on the step's own target-logit rows, head logits and draft trees, and the gated head-state
correction (the sr_reflex_correct kernel of sr_heads_propose_reflex) from the resulting memory. Finally the
whole step is timed on the other workloads (1.5B-shaped, 14B-shaped tail, and the seven points of the
7B-shaped concurrency sweep) and reported under "other_configs".
Workload: the 7B-shaped rollout step (B=128 trajectories, T=32-node trees, Hq=28, Hkv=4, D=128,
hidden 3584, 4 heads, vocab 151936, contexts uniform in [1024, 8192], bf16).

Prints one JSON line. ``--gpus`` above 1 is refused: the benchmark runs on one GPU.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "verified tree tokens/s per GPU at 7B shape; tree-attn HBM GB/s % peak"
HBM_PEAK_GBPS = 8000.0
BF16_PEAK_TFLOPS = 2500.0
CALIB_ELEMS = 1 << 28          # 1 GiB of float32 read and 1 GiB written by the calibration copy
KERNEL_SOURCE = {"sr_tree_attn": "k_attn.hip", "sr_attn_combine": "k_attn.hip", "sr_vocab_gemm": "k_heads.hip",
                 "sr_head_gemm": "k_heads.hip", "sr_clip_ln": "k_heads.hip", "sr_group_max": "k_heads.hip",
                 "sr_topm": "k_heads.hip", "sr_topm_full": "k_heads.hip", "sr_tree_build": "k_heads.hip",
                 "sr_tree_accept": "k_accept.hip", "sr_commit_path": "k_engine.hip",
                 "sr_reflex_feedback": "k_reflex.hip"}
COMMIT_LAYERS = 28             # decoder layers of the 7B-shaped target: one commit launch covers all of them


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def dev_tensor(x, device):
    import numpy as np
    import torch
    if x.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16).to(device)
    return torch.from_numpy(np.ascontiguousarray(x)).to(device)


def algorithmic(cfg, ctx_len, kernel):
    """Algorithmic bytes and flops of one launch of ``kernel`` for this workload."""
    B, T, Hq, Hkv, D, d, H, V = cfg.B, cfg.T, cfg.Hq, cfg.Hkv, cfg.D, cfg.d, cfg.H, cfg.V
    e = 2 if cfg.dtype == "bf16" else 4
    Ls = float(sum(int(x) for x in ctx_len))
    if kernel == "sr_vocab_gemm":
        M = B * H
        return dict(bytes=V * d * e + M * d * e + M * V * 4, flops=2.0 * M * V * d)
    if kernel == "sr_head_gemm":
        return dict(bytes=H * d * d * e + H * d * e + B * d * (e + 4) + B * H * d * e, flops=2.0 * B * H * d * d)
    if kernel == "sr_tree_attn":
        kv = Ls * 2 * Hkv * D * e
        return dict(bytes=kv + B * T * (Hq + 2 * Hkv) * D * e + B * T * Hq * (D + 1) * 4,
                    flops=4.0 * T * Hq * D * Ls)
    return dict(bytes=float("nan"), flops=float("nan"))


def attn_chunks(cfg, ctx_len):
    """Prefix chunks of every trajectory under the library's chunk plan (sr_tree_verify_attn): row groups of
    at most 224 query rows (bf16), chunks of 32/128/256 pages by the number of (trajectory, KV head, row
    group) triples."""
    R = cfg.T * (cfg.Hq // cfg.Hkv)
    ng = -(-R // 224) if (cfg.dtype == "bf16" and R > 224) else 1
    triples = cfg.B * cfg.Hkv * ng
    cp = 32 if triples < 64 else (128 if triples < 512 else 256)
    pages = [-(-int(L) // cfg.block_size) for L in ctx_len]
    return [max(1, -(-p_ // cp)) for p_ in pages], R


def step_kernel_work(cfg, ctx_len, max_children, rows_read):
    """Bytes and flops each step kernel moves or computes by design (one launch), for the per-kernel roofline.
    The chunk merge moves the partial results the split prefix needs (not the method's own bytes); the
    fp32-V recomputation has nothing to do on these inputs."""
    B, T, Hq, Hkv, D, d, H, V = cfg.B, cfg.T, cfg.Hq, cfg.Hkv, cfg.D, cfg.d, cfg.H, cfg.V
    e = 2 if cfg.dtype == "bf16" else 4
    mc, G = int(max_children), -(-V // 64)
    nch, R = attn_chunks(cfg, ctx_len)
    merged = [c for c in nch if c > 1]
    n_items = sum(nch) * Hkv * (-(-R // 224) if (cfg.dtype == "bf16" and R > 224) else 1)
    w = {k: algorithmic(cfg, ctx_len, k) for k in ("sr_head_gemm", "sr_vocab_gemm", "sr_tree_attn")}
    w["sr_clip_ln"] = dict(bytes=B * d * (e + 4 + 4 + e) + B, flops=12.0 * B * d)
    w["sr_topm"] = dict(bytes=B * H * (G * 4 + mc * 64 * 4 + mc * 8), flops=float(B * H * (G + mc * 64)))
    w["sr_tree_build"] = dict(bytes=B * H * mc * 8 + B * T * (4 + 4 + 4 + 8) + B * 4, flops=float(B * T * mc * 8))
    w["sr_attn_order"] = dict(bytes=B * 4 + n_items * 8, flops=0.0)
    w["sr_attn_redo"] = dict(bytes=4.0, flops=0.0)
    w["sr_attn_combine"] = dict(bytes=sum(Hkv * (c * R * (D * 4 + 8) + R * (D * 4 + 4)) for c in merged),
                                flops=float(sum(Hkv * c * R * D * 3 for c in merged)))
    w["sr_tree_accept"] = dict(bytes=float(rows_read) * V * e + B * T * 16, flops=float(rows_read) * V * 4)
    return w


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample", type=int, default=32, help="trajectories the oracle runs on")
    ap.add_argument("--no-other-configs", action="store_true",
                    help="skip the step timings of the 1.5B, 14B and concurrency-sweep workloads")
    ap.add_argument("--calib-copy", action="store_true",
                    help="run a plain 1 GiB float32 elementwise copy (negation) before the steps, as the "
                         "reference point that scales the HBM byte counters of a profiler run")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print(json.dumps({"error": "the benchmark runs on one GPU only; --gpus must be 1"}))
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2608_04962_amd as sr
    import synth

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    cfg = synth.SHAPE_7B
    t0 = time.time()
    hin = synth.heads_inputs(cfg, seed=args.seed)
    ain = synth.attn_inputs(cfg, seed=args.seed)
    cin = synth.accept_inputs(cfg, seed=args.seed)
    log(f"inputs generated in {time.time() - t0:.1f}s")

    H = {k: dev_tensor(hin[k], dev) for k in ("hidden", "corr", "active", "A", "bias", "W", "parents", "root_token",
                                              "u_tree")}
    A_ = {k: dev_tensor(ain[k], dev) for k in ("q", "k_cache", "v_cache", "block_table", "ctx_len", "k_tree", "v_tree",
                                               "parents")}
    C_ = {k: dev_tensor(cin[k], dev) for k in ("target_logits", "child_logit", "tokens", "parents", "u_acc", "u_fin")}
    B, T = cfg.B, cfg.T
    # outputs and workspaces allocated once, outside the timed region
    tok = torch.empty((B, T), dtype=torch.int32, device=dev)
    cl = torch.empty((B, T), dtype=torch.float32, device=dev)
    hws = torch.empty(sr.heads_workspace_bytes(B, cfg.d, cfg.H, cfg.V, T, hin["max_children"]), dtype=torch.uint8,
                      device=dev)
    out = torch.empty((B, T, cfg.Hq, cfg.D), dtype=torch.float32, device=dev)
    lse = torch.empty((B, T, cfg.Hq), dtype=torch.float32, device=dev)
    adesc = sr.attn_desc(A_["q"], A_["k_cache"], A_["block_table"])
    aws_n = sr.attn_workspace_bytes(adesc)
    aws = torch.empty(max(aws_n, 1), dtype=torch.uint8, device=dev)
    md = cin["max_depth"]
    outs = dict(acc_nodes=torch.empty((B, md), dtype=torch.int32, device=dev),
                out_tokens=torch.empty((B, md + 1), dtype=torch.int32, device=dev),
                out_len=torch.empty((B,), dtype=torch.int32, device=dev),
                final_kind=torch.empty((B,), dtype=torch.uint8, device=dev),
                min_margin=torch.empty((B,), dtype=torch.float32, device=dev))

    def step():
        sr.heads_propose(H["hidden"], H["corr"], H["active"], H["A"], H["bias"], H["W"], H["parents"],
                         H["root_token"], H["u_tree"], hin["max_children"], tokens=tok, child_logit=cl,
                         workspace=hws)
        sr.tree_verify_attn(A_["q"], A_["k_cache"], A_["v_cache"], A_["block_table"], A_["ctx_len"], A_["k_tree"],
                            A_["v_tree"], A_["parents"], out=out, lse=lse, workspace=aws)
        sr.tree_accept(C_["target_logits"], C_["child_logit"], C_["tokens"], C_["parents"], C_["u_acc"],
                       C_["u_fin"], md, outputs=outs)

    if args.calib_copy:
        src = torch.ones(CALIB_ELEMS, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.neg(src, out=dst)
        torch.cuda.synchronize()
        del src, dst

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    # per-kernel durations over the warm-up pattern identify the dominant kernel
    per_kernel = {}
    for name in sr.kernel_names():
        sr.prof_begin(name)
        step()
        ms, n = sr.prof_end()
        if n:
            per_kernel[name] = ms
    torch.cuda.synchronize()
    dominant = max(per_kernel, key=per_kernel.get)
    log("per-kernel ms (one step): " + ", ".join(f"{k}={v:.4f}" for k, v in per_kernel.items()))

    # timed region: K whole steps; the dominant kernel is bracketed by events on its own stream
    sr.prof_begin(dominant)
    torch.cuda.synchronize()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    marks = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]   # per-step spread
    ev0.record()
    for i in range(args.steps):
        marks[i].record()
        step()
    marks[-1].record()
    ev1.record()
    torch.cuda.synchronize()
    total_ms = ev0.elapsed_time(ev1)
    per_step = np.sort(np.array([marks[i].elapsed_time(marks[i + 1]) for i in range(args.steps)]))
    dom_ms, dom_n = sr.prof_end()
    ms_per_step = total_ms / args.steps
    dom_avg_ms = dom_ms / max(dom_n, 1)
    value = B * T / (ms_per_step / 1e3)

    alg = algorithmic(cfg, ain["ctx_len"], dominant)
    if dominant in ("sr_vocab_gemm", "sr_head_gemm") and cfg.B * cfg.H >= 312:
        bound, achieved, peak, unit = "mfma", alg["flops"] / (dom_avg_ms / 1e3) / 1e12, BF16_PEAK_TFLOPS, "TFLOP/s"
    else:
        bound, achieved, peak, unit = "hbm", alg["bytes"] / (dom_avg_ms / 1e3) / 1e9, HBM_PEAK_GBPS, "GB/s"
    attn_alg = algorithmic(cfg, ain["ctx_len"], "sr_tree_attn")
    attn_ms = per_kernel.get("sr_tree_attn", float("nan")) + per_kernel.get("sr_attn_combine", 0.0)
    attn_gbps = attn_alg["bytes"] / (attn_ms / 1e3) / 1e9

    # sanity of the step's outputs (not timed)
    kinds = outs["final_kind"].cpu().numpy()
    assert (kinds != 255).all(), "invalid trajectories in the benchmark step"
    assert torch.isfinite(out).all().item()

    # MALL (256 MB last-level cache) check: the same step with 1 GiB written between steps (outside each
    # step's event pair) against the back-to-back steps above
    flush = torch.empty(CALIB_ELEMS, dtype=torch.float32, device=dev)
    fl_ms = []
    for _ in range(20):
        flush.fill_(1.0)
        f0, f1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        f0.record()
        step()
        f1.record()
        torch.cuda.synchronize()
        fl_ms.append(f0.elapsed_time(f1))
    del flush
    torch.cuda.empty_cache()
    mall = {"flushed_step_ms_p50": float(np.median(fl_ms)), "back_to_back_step_ms_p50": float(np.percentile(per_step, 50)),
            "flush_bytes": CALIB_ELEMS * 4, "steps": len(fl_ms)}
    mall["ratio"] = mall["flushed_step_ms_p50"] / mall["back_to_back_step_ms_p50"]
    # the same steps back to back over four copies of every per-step input (activations, paged KV caches,
    # tree data, target logits; the weights stay shared, as a serving engine's do): no step finds the
    # previous step's inputs in the cache, and nothing runs between the steps
    per_set = [(A_, C_, H)]
    for r in range(3):
        a2 = {k: v.clone() for k, v in A_.items()}
        c2 = {k: v.clone() for k, v in C_.items()}
        h2 = dict(H)
        for k in ("hidden", "corr", "active", "parents", "root_token", "u_tree"):
            h2[k] = H[k].clone()
        per_set.append((a2, c2, h2))
    rot_bytes = sum(v.numel() * v.element_size() for a, c, h in per_set
                    for v in list(a.values()) + list(c.values()) + [h[k] for k in ("hidden", "corr")])

    def step_set(a, c, h):
        sr.heads_propose(h["hidden"], h["corr"], h["active"], h["A"], h["bias"], h["W"], h["parents"],
                         h["root_token"], h["u_tree"], hin["max_children"], tokens=tok, child_logit=cl,
                         workspace=hws)
        sr.tree_verify_attn(a["q"], a["k_cache"], a["v_cache"], a["block_table"], a["ctx_len"], a["k_tree"],
                            a["v_tree"], a["parents"], out=out, lse=lse, workspace=aws)
        sr.tree_accept(c["target_logits"], c["child_logit"], c["tokens"], c["parents"], c["u_acc"],
                       c["u_fin"], md, outputs=outs)

    for i in range(4):
        step_set(*per_set[i % 4])
    torch.cuda.synchronize()
    rmarks = [torch.cuda.Event(enable_timing=True) for _ in range(41)]
    for i in range(40):
        rmarks[i].record()
        step_set(*per_set[i % 4])
    rmarks[-1].record()
    torch.cuda.synchronize()
    rot_ms = [rmarks[i].elapsed_time(rmarks[i + 1]) for i in range(40)]
    del per_set
    torch.cuda.empty_cache()
    mall["rotated_step_ms_p50"] = float(np.median(rot_ms))
    mall["rotated_input_bytes"] = int(rot_bytes)
    mall["rotated_ratio"] = mall["rotated_step_ms_p50"] / mall["back_to_back_step_ms_p50"]

    # acceptance walk alone: algorithmic bytes = one target row per visited node (out_len rows per trajectory)
    sr.prof_begin("sr_tree_accept")
    for _ in range(20):
        sr.tree_accept(C_["target_logits"], C_["child_logit"], C_["tokens"], C_["parents"], C_["u_acc"],
                       C_["u_fin"], md, outputs=outs)
    acc_ms, acc_n = sr.prof_end()
    acc_avg = acc_ms / max(acc_n, 1)
    rows_read = int(outs["out_len"].sum().item())
    acc_bytes = rows_read * cfg.V * 2 + B * T * 16
    vocab = algorithmic(cfg, ain["ctx_len"], "sr_vocab_gemm")
    headg = algorithmic(cfg, ain["ctx_len"], "sr_head_gemm")
    gemms = {}
    for kname, a in (("sr_vocab_gemm", vocab), ("sr_head_gemm", headg)):
        kms = per_kernel.get(kname, float("nan"))
        gemms[kname] = {"ms": kms, "TFLOP/s": a["flops"] / (kms / 1e3) / 1e12,
                        "frac_bf16_peak": a["flops"] / (kms / 1e3) / 1e12 / BF16_PEAK_TFLOPS,
                        "GB/s": a["bytes"] / (kms / 1e3) / 1e9,
                        "frac_hbm_peak": a["bytes"] / (kms / 1e3) / 1e9 / HBM_PEAK_GBPS}

    # per-kernel roofline of one step: max(bytes / HBM peak, flops / bf16 MFMA peak) / measured time
    kwork = step_kernel_work(cfg, ain["ctx_len"], hin["max_children"], rows_read)
    kroof = {}
    for k, ms in per_kernel.items():
        wk = kwork.get(k)
        if wk is None or not ms:
            continue
        t_hbm = wk["bytes"] / (HBM_PEAK_GBPS * 1e9)
        t_mfma = wk["flops"] / (BF16_PEAK_TFLOPS * 1e12)
        kroof[k] = {"ms": ms, "bytes": wk["bytes"], "flops": wk["flops"], "bound": "hbm" if t_hbm >= t_mfma else "mfma",
                    "frac": max(t_hbm, t_mfma) / (ms / 1e3)}

    res = {
        "metric": METRIC, "value": value, "unit": "tree tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_per_step, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "7B-shape rollout verification step: B=128 trajectories, 32-node trees (depth 5), "
                               "Hq=28 Hkv=4 D=128 paged KV (block 16, contexts U[1024,8192]), hidden 3584, "
                               "4 heads, vocab 151936, one attention layer",
                   "global_batch": B, "tree_nodes": T, "parallelism": "none (1 GPU)"},
        "roofline": {"bound": bound, "achieved": achieved, "peak": peak, "unit": unit, "frac": achieved / peak,
                     "traffic": measured_traffic(dominant), "kernel": dominant, "avg_ms": dom_avg_ms, "launches": dom_n},
        "step_ms": {"p50": float(np.percentile(per_step, 50)), "p90": float(np.percentile(per_step, 90)),
                    "min": float(per_step[0]), "max": float(per_step[-1])},
        "tree_attn": {"GB/s": attn_gbps, "frac_hbm_peak": attn_gbps / HBM_PEAK_GBPS, "ms": attn_ms},
        "tree_accept": {"avg_ms": acc_avg, "launches": acc_n, "rows_read": rows_read, "algorithmic_bytes": acc_bytes,
                        "GB/s": acc_bytes / (acc_avg / 1e3) / 1e9,
                        "frac_hbm_peak": acc_bytes / (acc_avg / 1e3) / 1e9 / HBM_PEAK_GBPS},
        "head_gemms": gemms,
        "mall_check": mall,
        "kernels_ms": per_kernel,
        "kernel_roofline": kroof,
        "accepted_mean_len": float(outs["out_len"].float().mean().item()),
    }

    # the acceptance walk under the rollouts' nucleus truncation (top_p 0.95), same inputs
    nouts = {k: torch.empty_like(v) for k, v in outs.items()}
    for _ in range(2):
        sr.tree_accept(C_["target_logits"], C_["child_logit"], C_["tokens"], C_["parents"], C_["u_acc"], C_["u_fin"],
                       md, outputs=nouts, top_p=0.95)
    torch.cuda.synchronize()
    sr.prof_begin("sr_tree_accept")
    for _ in range(10):
        sr.tree_accept(C_["target_logits"], C_["child_logit"], C_["tokens"], C_["parents"], C_["u_acc"], C_["u_fin"],
                       md, outputs=nouts, top_p=0.95)
    nms, nn = sr.prof_end()
    res["accept_top_p_0.95"] = {"avg_ms": nms / max(nn, 1), "launches": nn,
                                "accepted_mean_len": float(nouts["out_len"].float().mean().item())}
    res["commit_path"] = commit_bench(sr, synth, cfg, args.seed, outs, dev)
    res["reflex_feedback"] = reflex_bench(sr, cfg, H, C_, hin, hws, dev)
    res["tree_budget"] = dict(zip(("N_t", "horizon_counts", "parents"), sr.tree_budget(B)))

    if not args.no_other_configs:
        res["other_configs"] = other_configs(sr, synth, dev, W7=H["W"], A7=H["A"], bias7=H["bias"])

    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(cfg, hin, ain, cin, args.cpu_sample)
    print(json.dumps(res), flush=True)


def other_configs(sr, synth, dev, W7=None, A7=None, bias7=None, steps=5, warmup=2):
    """Whole-step throughput of the other workloads: the 1.5B-shaped step, the 14B-shaped tail step and the
    seven points of the 7B-shaped concurrency sweep (live batch 256 -> 4, tree 8 -> 96 nodes). Values are
    drawn on the GPU with the workloads' distributions (only the timing is used); context lengths, trees and
    page tables follow the same recipe as the main workload."""
    import numpy as np
    import torch
    g = torch.Generator(device=dev).manual_seed(1)
    bf = torch.bfloat16
    rn = lambda shape, std: (torch.randn(shape, generator=g, device=dev) * std).to(bf)  # noqa: E731
    cases = [("1.5B-shape", synth.SHAPE_1P5B), ("14B-shape-tail", synth.SHAPE_14B_TAIL)]
    cases += [(f"7B-sweep-B{b}-T{t}", synth.sweep_config(b, t)) for b, t in synth.SWEEP_POINTS]
    out = {}
    for name, cfg in cases:
        B, T, Hq, Hkv, D, d, Hh, V = cfg.B, cfg.T, cfg.Hq, cfg.Hkv, cfg.D, cfg.d, cfg.H, cfg.V
        seven = d == 3584 and W7 is not None
        W = W7 if seven else rn((V, d), 0.02)
        A = A7 if seven else rn((Hh, d, d), 0.02)
        bias = bias7 if seven else rn((Hh, d), 0.02)
        hidden = rn((B, d), 1.0)
        corr = torch.randn((B, d), generator=g, device=dev) * 0.1
        active = (torch.rand((B,), generator=g, device=dev) < cfg.active_frac).to(torch.uint8)
        par_np = synth.topology(cfg)
        parents = torch.from_numpy(np.ascontiguousarray(np.broadcast_to(par_np, (B, T)))).to(dev)
        root = torch.randint(0, V, (B,), generator=g, device=dev, dtype=torch.int32)
        u_tree = torch.rand((B, T), generator=g, device=dev).clamp_(1e-6, 1 - 1e-6)
        mc = synth.max_children(par_np)
        L = synth.context_lengths(cfg, 0)
        nblk = -(-L // cfg.block_size)
        NB = int(nblk.sum())
        perm = np.random.default_rng(0).permutation(NB).astype(np.int32)
        table = np.full((B, cfg.max_blocks), -1, dtype=np.int32)
        off = 0
        for b in range(B):
            table[b, :nblk[b]] = perm[off:off + nblk[b]]
            off += nblk[b]
        q = rn((B, T, Hq, D), 1.0)
        kc, vc = rn((NB, Hkv, cfg.block_size, D), 1.0), rn((NB, Hkv, cfg.block_size, D), 1.0)
        kt, vt = rn((B, T, Hkv, D), 1.0), rn((B, T, Hkv, D), 1.0)
        bt, cl_ = torch.from_numpy(table).to(dev), torch.from_numpy(L.astype(np.int32)).to(dev)
        tl = rn((B, T, V), 4.0)
        u_acc = torch.rand((B, T), generator=g, device=dev).clamp_(1e-6, 1 - 1e-6)
        u_fin = torch.rand((B,), generator=g, device=dev).clamp_(1e-6, 1 - 1e-6)
        md = int(synth.node_depths(par_np).max()) if T > 1 else 0
        tok = torch.empty((B, T), dtype=torch.int32, device=dev)
        cl = torch.empty((B, T), dtype=torch.float32, device=dev)
        hws = torch.empty(sr.heads_workspace_bytes(B, d, Hh, V, T, mc), dtype=torch.uint8, device=dev)
        o = torch.empty((B, T, Hq, D), dtype=torch.float32, device=dev)
        lse = torch.empty((B, T, Hq), dtype=torch.float32, device=dev)
        adesc = sr.attn_desc(q, kc, bt)
        aws = torch.empty(max(sr.attn_workspace_bytes(adesc), 1), dtype=torch.uint8, device=dev)
        outs = dict(acc_nodes=torch.empty((B, max(md, 1)), dtype=torch.int32, device=dev),
                    out_tokens=torch.empty((B, md + 1), dtype=torch.int32, device=dev),
                    out_len=torch.empty((B,), dtype=torch.int32, device=dev),
                    final_kind=torch.empty((B,), dtype=torch.uint8, device=dev),
                    min_margin=torch.empty((B,), dtype=torch.float32, device=dev))

        def step():
            sr.heads_propose(hidden, corr, active, A, bias, W, parents, root, u_tree, mc, tokens=tok, child_logit=cl,
                             workspace=hws)
            sr.tree_verify_attn(q, kc, vc, bt, cl_, kt, vt, parents, out=o, lse=lse, workspace=aws)
            sr.tree_accept(tl, cl, tok, parents, u_acc, u_fin, md, outputs=outs)
        for _ in range(warmup):
            step()
        torch.cuda.synchronize()
        sr.prof_begin("sr_tree_attn")
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(steps):
            step()
        e1.record()
        torch.cuda.synchronize()
        ams, an = sr.prof_end()
        ms = e0.elapsed_time(e1) / steps
        kv = float(L.sum()) * 2 * Hkv * D * 2 + B * T * (Hq + 2 * Hkv) * D * 2 + B * T * Hq * (D + 1) * 4
        am = ams / max(an, 1)
        # per-kernel durations, one step per kernel name (outside the timed steps)
        kms = {}
        for kname in sr.kernel_names():
            sr.prof_begin(kname)
            step()
            kt_ms, kn = sr.prof_end()
            if kn:
                kms[kname] = kt_ms
        torch.cuda.synchronize()
        assert (outs["final_kind"].cpu() != 255).all(), name
        out[name] = {"B": B, "T": T, "ms_per_step": ms, "tree_tokens_per_s": B * T / (ms / 1e3),
                     "tree_attn_ms": am, "tree_attn_GB/s": kv / (am / 1e3) / 1e9, "kernels_ms": kms}
        log(f"{name}: {ms:.3f} ms/step, {B * T / (ms / 1e3):.4g} tree tokens/s, attention {kv / (am / 1e3) / 1e9:.0f} GB/s")
        del q, kc, vc, kt, vt, tl
        if not seven:
            del W, A, bias
        torch.cuda.empty_cache()
    return out


def commit_bench(sr, synth, cfg, seed, outs, dev):
    """Time sr_commit_path on the step's own accepted paths for every layer of the target (one launch)."""
    import torch
    ci = synth.commit_inputs(cfg, seed=seed, with_kv=False)
    nl, B, T, Hkv, D = COMMIT_LAYERS, cfg.B, cfg.T, cfg.Hkv, cfg.D
    g = torch.Generator(device=dev).manual_seed(seed)
    kt = torch.randn((nl, B, T, Hkv, D), generator=g, device=dev).to(torch.bfloat16)
    vt = torch.randn((nl, B, T, Hkv, D), generator=g, device=dev).to(torch.bfloat16)
    shape = (nl, ci["num_blocks"], Hkv, cfg.block_size, D)
    kc = torch.empty(shape, dtype=torch.bfloat16, device=dev)
    vc = torch.empty(shape, dtype=torch.bfloat16, device=dev)
    table = torch.from_numpy(ci["block_table"]).to(dev)
    ctx = torch.from_numpy(ci["ctx_len"]).to(dev)
    new = torch.empty((B,), dtype=torch.int32, device=dev)
    par = torch.from_numpy(ci["parents"]).to(dev)
    run = lambda: sr.commit_path(kc, vc, table, ctx, kt, vt, outs["acc_nodes"], outs["out_len"],  # noqa: E731
                                 parents=par, new_ctx_len=new)
    for _ in range(3):
        run()
    torch.cuda.synchronize()
    sr.prof_begin("sr_commit_path")
    for _ in range(20):
        run()
    ms, n = sr.prof_end()
    rows = int(outs["out_len"].sum().item())
    assert (new.cpu() >= 0).all(), "rejected trajectories in the commit benchmark"
    moved = rows * Hkv * D * 2 * 2 * nl            # K and V rows, bf16, per layer
    alg = 2 * moved + B * (4 * 3 + 4 * outs["acc_nodes"].shape[1])  # read + write, plus the small int inputs
    avg = ms / max(n, 1)
    del kc, vc, kt, vt
    torch.cuda.empty_cache()
    return {"layers": nl, "rows_per_layer": rows, "avg_ms": avg, "launches": n, "algorithmic_bytes": alg,
            "GB/s": alg / (avg / 1e3) / 1e9, "frac_hbm_peak": alg / (avg / 1e3) / 1e9 / HBM_PEAK_GBPS}


def reflex_bench(sr, cfg, H, C_, hin, hws, dev):
    """Time sr_reflex_feedback for B*H records: record (i, h) takes trajectory i's target row at its first
    depth-h node, the step's head-h logits of trajectory i, and the tokens of trajectory i's depth-h nodes
    as candidates (the realised token is the first of them)."""
    import numpy as np
    import torch
    B, T, Hh, V, d = cfg.B, cfg.T, cfg.H, cfg.V, cfg.d
    logits = torch.empty((B, Hh, V), dtype=torch.float32, device=dev)
    tok = torch.empty((B, T), dtype=torch.int32, device=dev)
    cl = torch.empty((B, T), dtype=torch.float32, device=dev)
    sr.heads_propose(H["hidden"], H["corr"], H["active"], H["A"], H["bias"], H["W"], H["parents"], H["root_token"],
                     H["u_tree"], hin["max_children"], logits=logits, tokens=tok, child_logit=cl, workspace=hws)
    torch.cuda.synchronize()
    par = hin["parents"][0]
    depth = np.zeros(T, dtype=np.int64)
    for c in range(1, T):
        depth[c] = depth[par[c]] + 1
    by_depth = [np.nonzero(depth == h)[0] for h in range(Hh + 1)]
    maxc = max(len(by_depth[h]) for h in range(1, Hh + 1))
    tk = tok.cpu().numpy()
    R = B * Hh
    cand = np.full((R, maxc), -1, dtype=np.int32)
    p_row = np.empty(R, dtype=np.int32)
    q_row = np.empty(R, dtype=np.int32)
    traj = np.empty(R, dtype=np.int32)
    hor = np.empty(R, dtype=np.int32)
    for i in range(B):
        for h in range(1, Hh + 1):
            r = i * Hh + h - 1
            nodes = by_depth[h]
            # distinct tokens of the depth-h nodes, in node order
            seen = []
            for u in nodes:
                if int(tk[i, u]) not in seen:
                    seen.append(int(tk[i, u]))
            cand[r, :len(seen)] = seen
            p_row[r] = i * T + int(nodes[0])
            q_row[r] = i * Hh + h - 1
            traj[r], hor[r] = i, h
    t = lambda x: torch.from_numpy(x).to(dev)  # noqa: E731
    args = (C_["target_logits"].view(B * T, V), t(p_row), logits.view(B * Hh, V), t(q_row), t(cand),
            t(cand[:, 0].copy()), t(traj), t(hor), H["W"])
    mem = torch.zeros((B, Hh, d), dtype=torch.float32, device=dev)
    stats = torch.empty((R, 8), dtype=torch.float32, device=dev)
    for _ in range(3):
        sr.reflex_feedback(*args, mem, stats=stats)
    torch.cuda.synchronize()
    sr.prof_begin("sr_reflex_feedback")
    for _ in range(20):
        sr.reflex_feedback(*args, mem, stats=stats)
    ms, n = sr.prof_end()
    st = stats.cpu().numpy()
    assert (st[:, 5] >= 0).all(), "invalid records in the feedback benchmark"
    # the gated head-state correction from that memory, every gate open (enough aligned evidence)
    g = torch.Generator(device=dev).manual_seed(0)
    P = torch.randn((24, d), generator=g, device=dev)
    P /= P.norm(dim=1, keepdim=True)
    align = torch.tensor([100.0, 0.9, 99 * 0.0025, 20.0], device=dev).repeat(B, Hh, 1).contiguous()
    sk = torch.empty((B, Hh, 24), dtype=torch.float32, device=dev)
    al = torch.empty((B, Hh), dtype=torch.float32, device=dev)
    run_c = lambda: sr.heads_propose_reflex(  # noqa: E731
        H["hidden"], None, None, H["A"], H["bias"], H["W"], H["parents"], H["root_token"], H["u_tree"],
        hin["max_children"], mem, align, P, tokens=tok, child_logit=cl, sketch_out=sk, alpha_out=al, workspace=hws)
    run_c()
    torch.cuda.synchronize()
    sr.prof_begin("sr_reflex_correct")
    for _ in range(20):
        run_c()
    cms, cn = sr.prof_end()
    assert (al.cpu() > 0).all(), "closed gates in the correction benchmark"
    nS = float(st[:, 4].mean())
    # per record: one target row (bf16), one head row (fp32), the support's rows of W, the memory row in/out
    alg = R * (V * 2 + V * 4 + nS * d * 2 + 2 * d * 4)
    avg = ms / max(n, 1)
    del logits
    calg = B * Hh * d * (2 + 4 + 2) + 24 * d * 4   # z in and out (bf16), memory row, P
    cavg = cms / max(cn, 1)
    return {"records": R, "mean_support": nS, "avg_ms": avg, "launches": n, "algorithmic_bytes": alg,
            "GB/s": alg / (avg / 1e3) / 1e9, "frac_hbm_peak": alg / (avg / 1e3) / 1e9 / HBM_PEAK_GBPS,
            "applied_frac": float((st[:, 5] == 1).mean()),
            "correct": {"rows": B * Hh, "avg_ms": cavg, "launches": cn, "algorithmic_bytes": calg,
                        "GB/s": calg / (cavg / 1e3) / 1e9}}


def measured_traffic(kernel):
    """HBM bytes per launch of ``kernel`` from the committed profiler record (FETCH_SIZE + WRITE_SIZE, each
    divided by what the same counter reads for the 1 GiB calibration copy), or None when there is no record
    or the kernel's source has changed since the counters were taken."""
    import hashlib
    rec = os.path.join(ROOT, "profiles", f"traffic_{kernel}_7b_step.txt")
    src = os.path.join(ROOT, "paper_2608_04962_amd", "csrc", KERNEL_SOURCE.get(kernel, ""))
    if not (os.path.isfile(rec) and os.path.isfile(src)):
        return None
    fields = {}
    for line in open(rec):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            fields[k.strip()] = v.strip()
    with open(src, "rb") as f:
        if hashlib.sha256(f.read()).hexdigest() != fields.get("source_sha256"):
            return None
    try:
        return float(fields["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def oracle_step(cfg, hin, ain, cin, rows):
    """Seconds the float64 oracle takes for the step on trajectories ``rows``: (heads + tree, attention of every
    node, acceptance)."""
    import numpy as np

    import oracle
    import synth
    dt = cfg.dtype
    f = lambda x: synth.to_f64(x, dt)  # noqa: E731
    rows = np.asarray(rows)
    A64, b64, W64 = f(hin["A"]), f(hin["bias"]), f(hin["W"])
    q, kc, vc, kt, vt = (f(ain[n]) for n in ("q", "k_cache", "v_cache", "k_tree", "v_tree"))
    t0 = time.perf_counter()
    ho = oracle.heads_forward(f(hin["hidden"])[rows], hin["corr"][rows], hin["active"][rows], A64, b64, W64,
                              cfg.clip_norm, 1e-5, round_fn=None if dt == "f32" else oracle.round_bf16)
    oracle.tree_build(ho["logits"], hin["parents"][rows], hin["root_token"][rows], hin["u_tree"][rows])
    t1 = time.perf_counter()
    oracle.tree_attention(q, kc, vc, ain["block_table"], ain["ctx_len"], kt, vt, ain["parents"], ain["scale"],
                          nodes=[(int(b), u) for b in rows for u in range(cfg.T)])
    t2 = time.perf_counter()

    class Rows:
        def __getitem__(self, b):
            return f(cin["target_logits"][b])
    oracle.tree_accept(Rows(), cin["child_logit"], cin["tokens"], cin["parents"], cin["u_acc"], cin["u_fin"], 1.0,
                       cin["max_depth"], rows=[int(b) for b in rows])
    t3 = time.perf_counter()
    return t1 - t0, t2 - t1, t3 - t2


def cpu_baseline(cfg, hin, ain, cin, k):
    """The float64 oracle on the first k trajectories of the same workload on the host cores (BLAS threads as the
    process has them), plus single-thread figures of the tiny fp32 workload (whole) and of the 1.5B-shaped one
    (two trajectories)."""
    import synth
    try:
        from threadpoolctl import threadpool_info, threadpool_limits
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:  # pragma: no cover
        threadpool_limits = None
        threads = len(os.sched_getaffinity(0))
    th, ta, tc = oracle_step(cfg, hin, ain, cin, range(k))
    secs = th + ta + tc
    res = {"value": k * cfg.T / secs, "unit": "tree tokens/s", "cores": threads, "kind": "oracle",
           "sample": f"{k} of {cfg.B} trajectories of the same workload (all {cfg.T} nodes each): heads+tree "
                     f"{th:.1f}s, attention {ta:.1f}s, acceptance {tc:.1f}s; float64 NumPy",
           "seconds": secs, "cpu_model": cpu_model(), "affinity_cpus": len(os.sched_getaffinity(0))}
    single = {}
    if threadpool_limits is not None:
        for c, n in ((synth.TINY_FP32, synth.TINY_FP32.B), (synth.SHAPE_1P5B, 2)):
            h = synth.heads_inputs(c, seed=0)
            a = synth.attn_inputs(c, seed=0)
            ac = synth.accept_inputs(c, seed=0)
            with threadpool_limits(limits=1):
                t = oracle_step(c, h, a, ac, range(n))
            single[c.name] = {"tree_tokens_per_s": n * c.T / sum(t), "trajectories": n, "seconds": sum(t),
                              "heads_tree_s": t[0], "attention_s": t[1], "acceptance_s": t[2]}
            del h, a, ac
    res["single_thread"] = single
    return res


if __name__ == "__main__":
    main()
