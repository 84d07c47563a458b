"""Benchmark of one LoPA verify step on one MI355X.

One step = lopa_build_branches + lopa_verify_forward (all k+1 branches, one
pass) + lopa_branch_confidence_select + lopa_commit_kv on the Dream-7B shape
(28 layers, hidden 3584, 28 q / 4 kv heads, head_dim 128, SwiGLU 18944, vocab
152064; random bf16 weights N(0, 0.02)), prefix 512 (block-causal prefill of a
uniform-random prompt), block 32, k = 7 (8 branches, 256 rows), tau = 0.9. The
timed state is the block's first iteration (all 32 positions masked, conf /
pred from the initial forward), replayed K times (commit rewrites the same rows).

Prints one JSON line: value = branch-tokens/s = 8 * 32 / step seconds.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0        # MI355X HBM3E
MFMA_BF16_PEAK_TFS = 2500.0  # dense bf16


def step_bytes(cfg, P, L, nb):
    """Algorithmic HBM bytes of one verify step (weights once, prefix K/V once,
    staging written, commit copy)."""
    H, F, V, d = cfg["hidden"], cfg["ffn"], cfg["vocab"], cfg["head_dim"]
    Hq, Hkv, Ly = cfg["heads"], cfg["kv_heads"], cfg["layers"]
    layer_w = (H * (Hq + 2 * Hkv) * d + Hq * d * H + 2 * F * H + F * H) * 2
    w = Ly * layer_w + V * H * 2
    kv_prefix = Ly * 2 * Hkv * P * d * 2
    staging = nb * Ly * 2 * Hkv * L * d * 2
    commit = 2 * Ly * 2 * Hkv * L * d * 2
    return w + kv_prefix + staging + commit


def step_flops(cfg, P, L, nb):
    H, F, V, d = cfg["hidden"], cfg["ffn"], cfg["vocab"], cfg["head_dim"]
    Hq, Hkv, Ly = cfg["heads"], cfg["kv_heads"], cfg["layers"]
    M = nb * L
    gemm = 2 * M * (Ly * (H * (Hq + 2 * Hkv) * d + Hq * d * H + 3 * F * H) + V * H)
    attn = Ly * 2 * 2 * M * Hq * (P + L) * d
    return gemm + attn


def gateup_launch_bytes(cfg, M):
    """Algorithmic bytes of one gate/up + SwiGLU launch: its weights, the
    normalised activations read once, the SwiGLU output written once."""
    H, F = cfg["hidden"], cfg["ffn"]
    return 2 * F * H * 2 + M * H * 2 + M * F * 2


def cpu_baseline(cfg_full, weights_dev, P, L, k, layers_sample=4):
    """Time the oracle (float64 numpy) on a bounded sample of the same step:
    `layers_sample` decoder layers of the full shape + the LM head and softmax for
    all (k+1)*L rows, against a random prefix cache; scaled to all layers."""
    import numpy as np
    import torch

    import synth
    from oracle import KVCache, OracleModel

    cfg = dict(cfg_full)
    cfg["layers"] = layers_sample
    host = {"embed": weights_dev["embed"].float().cpu(),
            "layers": [{kk: v.float().cpu() for kk, v in weights_dev["layers"][i].items()}
                       for i in range(layers_sample)],
            "final_norm": weights_dev["final_norm"].float().cpu(),
            "lm_head": weights_dev["lm_head"].float().cpu()}
    model = OracleModel(cfg, host, "pure")
    del host
    cache = KVCache(cfg, P + L)
    g = synth.irwin_hall(synth.stream_key(7, 1), cache.k[:, :, :P].size, 1.0).double().numpy()
    cache.k[:, :, :P] = g.reshape(cache.k[:, :, :P].shape)
    cache.v[:, :, :P] = -g.reshape(cache.v[:, :, :P].shape)
    nb = k + 1
    tokens = synth.prompt(cfg, nb * L, seed=3).numpy().reshape(nb, L)
    tokens[:, ::2] = cfg["mask_id"]
    threads = len(os.sched_getaffinity(0))
    torch.set_num_threads(threads)
    # layers
    t0 = time.perf_counter()
    out = model.forward_block(tokens, P, cache, n_layers=layers_sample)
    t_layers = time.perf_counter() - t0
    # LM head + softmax for every row (final norm included)
    from oracle.model import confidence, rms_norm
    t0 = time.perf_counter()
    hf = rms_norm(out["x"], model.final_norm, cfg["rms_eps"])
    confidence(hf @ model.lm_head.T, cfg["mask_id"])
    t_head = time.perf_counter() - t0
    step_s = t_layers / layers_sample * cfg_full["layers"] + t_head
    return {"value": nb * L / step_s, "unit": "branch-tokens/s", "cores": threads,
            "kind": "oracle",
            "sample": (f"float64 numpy oracle, {layers_sample} of {cfg_full['layers']} decoder layers "
                       f"+ LM head/softmax of the Dream-7B shape at {nb}x{L} rows, prefix {P}; "
                       f"measured {t_layers:.2f}s layers + {t_head:.2f}s head, scaled to "
                       f"{step_s:.1f}s per step")}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="dream7b", help="synth config name (model shape)")
    ap.add_argument("--prefix", type=int, default=512)
    ap.add_argument("--block", type=int, default=32)
    ap.add_argument("--k", type=int, default=7)
    ap.add_argument("--tau", type=float, default=0.9)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-layers", type=int, default=4)
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: this build runs on one GPU; --gpus {args.gpus} is not supported "
              "(multi-GPU branch parallelism is a design note, not built)", file=sys.stderr)
        sys.exit(2)

    import torch

    import synth
    import paper_2512_16229_amd as lp

    dev = "cuda"
    torch.cuda.set_device(0)
    cfg = synth.config(args.config)
    P, L, k, tau = args.prefix, args.block, args.k, args.tau
    nb, M = k + 1, (k + 1) * args.block
    log = lambda m: print(m, file=sys.stderr, flush=True)

    t0 = time.perf_counter()
    w = synth.model_weights(cfg, device=dev, dtype=torch.bfloat16)
    torch.cuda.synchronize()
    log(f"weights generated on the GPU in {time.perf_counter() - t0:.1f}s")
    t0 = time.perf_counter()
    model = lp.Model(cfg, w)
    log(f"model repacked in {time.perf_counter() - t0:.1f}s")
    kv = lp.KV(model, P + L, nb, L)
    dec = lp.Decoder(model, kv, L, k, tau)
    t0 = time.perf_counter()
    assert dec.prefill(synth.prompt(cfg, P, device=dev)) == P
    dec.init_block(P)
    torch.cuda.synchronize()
    log(f"prefill of {P} positions + initial forward in {time.perf_counter() - t0:.1f}s")

    i32 = dict(dtype=torch.int32, device=dev)
    tokens, conf, pred = dec.tokens.clone(), dec.conf.clone(), dec.pred.clone()
    bt = torch.empty(nb * L, **i32)
    fp = torch.empty(nb, **i32)
    va = torch.empty(nb, dtype=torch.uint8, device=dev)
    nv = torch.empty(1, **i32)
    cb = torch.empty(nb * L, dtype=torch.float32, device=dev)
    pb = torch.empty(nb * L, **i32)
    sc = torch.empty(nb, dtype=torch.float32, device=dev)
    win = torch.empty(1, **i32)
    nt, nc, npd, nu = (torch.empty(L, **i32), torch.empty(L, dtype=torch.float32, device=dev),
                       torch.empty(L, **i32), torch.empty(1, **i32))
    off = torch.empty(1, **i32)
    mask = cfg["mask_id"]

    def step():
        lp.lopa_build_branches(tokens, conf, pred, L, mask, tau, k, bt, fp, va, nv)
        lp.lopa_verify_forward(model, kv, P, bt, nb, L, cb, pb)
        lp.lopa_branch_confidence_select(bt, cb, pb, va, nb, L, mask, sc, win, nt, nc, npd, nu)
        lp.lopa_commit_kv(kv, win, P, L, off)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    ev0.record()
    for _ in range(args.steps):
        step()
    ev1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = ev0.elapsed_time(ev1) / args.steps
    log(f"{args.steps} steps: {ms:.3f} ms/step (events), {wall / args.steps * 1e3:.3f} ms/step (wall)")

    # per-kind launch times with HIP events on the library's stream
    kv.profile(lp.PROF_KINDS)
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    prof = kv.profile_read()
    kv.profile(())
    kernel_ms = {kd: (t / n if n else 0.0) for kd, (t, n) in prof.items()}
    per_step_ms = {kd: t / args.steps for kd, (t, n) in prof.items()}
    log("per-step ms by kind: " + ", ".join(f"{kd} {v:.3f}" for kd, v in per_step_ms.items()))

    gu_ms = kernel_ms["gateup"]
    gu_bytes = gateup_launch_bytes(cfg, M)
    achieved = gu_bytes / (gu_ms * 1e-3) / 1e9
    sb = step_bytes(cfg, P, L, nb)
    sf = step_flops(cfg, P, L, nb)
    result = {
        "metric": "LoPA verify-step ms & branch-tokens/s (7B shape, k=7); % HBM/MFMA roofline",
        "value": round(nb * L / (ms * 1e-3), 1),
        "unit": "branch-tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": (f"LoPA verify step, {args.config} shape ({cfg['layers']}L H{cfg['hidden']} "
                                f"{cfg['heads']}q/{cfg['kv_heads']}kv d{cfg['head_dim']} F{cfg['ffn']} "
                                f"V{cfg['vocab']}), random bf16 weights, prefix {P}, block {L}, "
                                f"k={k} ({nb} branches, {M} rows), tau {tau}"),
                   "prefix": P, "block": L, "k": k, "rows": M},
        "roofline": {"bound": "hbm", "kernel": "gate/up projection + SwiGLU (gemm_kernel<EPI_SWIGLU>)",
                     "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None,
                     "bytes_per_launch": gu_bytes, "avg_launch_ms": round(gu_ms, 4)},
        "step_roofline": {"hbm_bytes": sb, "flops": sf,
                          "hbm_frac": round(sb / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                          "mfma_frac": round(sf / (ms * 1e-3) / 1e12 / MFMA_BF16_PEAK_TFS, 4)},
        "kernel_ms_per_step": {kd: round(v, 4) for kd, v in per_step_ms.items()},
    }
    if not args.no_cpu_baseline:
        t0 = time.perf_counter()
        try:
            result["cpu_baseline"] = cpu_baseline(cfg, w, P, L, k, args.cpu_layers)
        except Exception as e:  # the GPU number stands; say why the baseline is missing
            result["cpu_baseline"] = {"value": None, "error": repr(e)}
        log(f"cpu baseline in {time.perf_counter() - t0:.1f}s")
    print(json.dumps(result))


if __name__ == "__main__":
    main()
