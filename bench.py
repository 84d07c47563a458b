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


def step_bytes(cfg, P, L, nb, precision="bf16"):
    """Algorithmic HBM bytes of one verify step (weights once, prefix K/V once,
    staging written, commit copy); FP8 modes: one byte per quantised weight."""
    H, F, V, d = cfg["hidden"], cfg["ffn"], cfg["vocab"], cfg["head_dim"]
    Hq, Hkv, Ly = cfg["heads"], cfg["kv_heads"], cfg["layers"]
    bq = 1 if precision == "fp8" else 2       # QKV and LM head
    bm = 1 if precision != "bf16" else 2      # gate / up / down
    layer_w = H * (Hq + 2 * Hkv) * d * bq + Hq * d * H * 2 + 3 * F * H * bm
    w = Ly * layer_w + V * H * bq
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


def gateup_launch_bytes(cfg, M, precision="bf16"):
    """Algorithmic bytes of one gate/up + SwiGLU launch: its weights, the
    normalised activations read once, the SwiGLU output (bf16) written once.
    FP8 modes: one byte per weight and activation value, plus the per-channel
    and per-row fp32 scales and the row maxima written for the requantisation."""
    H, F = cfg["hidden"], cfg["ffn"]
    if precision == "bf16":
        return 2 * F * H * 2 + M * H * 2 + M * F * 2
    return 2 * F * H + M * H + M * F * 2 + 2 * F * 4 + M * 4 + M * 4


def gemm_source_sha():
    """Short hash of the GEMM kernel source (the measured HBM traffic is only
    valid for the source it was taken on)."""
    import hashlib
    h = hashlib.sha256()
    for f in ("gemm.hip", "common.h"):
        with open(os.path.join(ROOT, "paper_2512_16229_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(path):
    """HBM bytes per gate/up launch from the rocprofv3 FETCH_SIZE / WRITE_SIZE
    summary in profiles/ (copy-kernel calibrated), or None when the summary is
    missing or was taken on another GEMM source."""
    try:
        txt = open(path).read()
    except OSError:
        return None
    vals = dict(l.split(":", 1) for l in txt.splitlines() if l.startswith(("sha:", "traffic_bytes:")))
    if vals.get("sha", "").strip() != gemm_source_sha():
        return None
    try:
        return int(float(vals["traffic_bytes"]))
    except (KeyError, ValueError):
        return None


class _Hip:
    """The few HIP runtime calls the torch-free counter runs need."""

    def __init__(self):
        import ctypes as C
        self.C = C
        self.rt = C.CDLL("libamdhip64.so")
        for name, args in (("hipMalloc", [C.POINTER(C.c_void_p), C.c_size_t]),
                           ("hipFree", [C.c_void_p]),
                           ("hipMemsetD16", [C.c_void_p, C.c_ushort, C.c_size_t]),
                           ("hipMemset", [C.c_void_p, C.c_int, C.c_size_t]),
                           ("hipMemcpy", [C.c_void_p, C.c_void_p, C.c_size_t, C.c_int]),
                           ("hipDeviceSynchronize", [])):
            getattr(self.rt, name).argtypes = args
            getattr(self.rt, name).restype = C.c_int

    def check(self, rc, what):
        if rc != 0:
            raise RuntimeError(f"{what} failed with hipError {rc}")

    def alloc(self, nbytes, fill16=None):
        p = self.C.c_void_p()
        self.check(self.rt.hipMalloc(self.C.byref(p), nbytes), "hipMalloc")
        if fill16 is not None:
            self.check(self.rt.hipMemsetD16(p, fill16, nbytes // 2), "hipMemsetD16")
        else:
            self.check(self.rt.hipMemset(p, 0, nbytes), "hipMemset")
        return p


def copy_calibration(nbytes=1 << 30, reps=5):
    """A plain device-to-device copy of known size (the runtime's copy kernel),
    for scaling the HBM counters. Torch-free, like hbm_counter_run."""
    hip = _Hip()
    src, dst = hip.alloc(nbytes, fill16=0x3F80), hip.alloc(nbytes)
    for _ in range(reps):
        hip.check(hip.rt.hipMemcpy(dst, src, nbytes, 3), "hipMemcpy")  # device to device
    hip.check(hip.rt.hipDeviceSynchronize(), "hipDeviceSynchronize")
    print(json.dumps({"copy_bytes": nbytes, "reps": reps}))


def hbm_counter_run(cfg, P, L, k, reps=3):
    """Torch-free verify forwards on the given shape for the HBM counter runs
    (rocprofv3 --pmc): weights are constant fills, which changes no traffic."""
    import ctypes as C
    import importlib.util
    spec = importlib.util.spec_from_file_location(
        "lopa_abi", os.path.join(ROOT, "paper_2512_16229_amd", "_abi.py"))
    abi = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(abi)
    hip = _Hip()
    H, F, V, d = cfg["hidden"], cfg["ffn"], cfg["vocab"], cfg["head_dim"]
    Hq, Hkv = cfg["heads"], cfg["kv_heads"]
    W = lambda n, v=0x3C00: hip.alloc(2 * n, fill16=v)  # bf16 0.0078 (norm weights 1.0)
    layers = (abi.lopa_layer_weights * cfg["layers"])()
    for i in range(cfg["layers"]):
        b = (lambda n: W(n)) if cfg["qkv_bias"] else (lambda n: None)
        layers[i] = abi.lopa_layer_weights(
            W(Hq * d * H), W(Hkv * d * H), W(Hkv * d * H), b(Hq * d), b(Hkv * d), b(Hkv * d),
            W(H * Hq * d), W(F * H), W(F * H), W(H * F), W(H, 0x3F80), W(H, 0x3F80))
    wp = abi.lopa_weight_ptrs(W(V * H), layers, W(H, 0x3F80), W(V * H))
    c = abi.lopa_model_cfg(cfg["layers"], H, Hq, Hkv, d, F, V, cfg["mask_id"], cfg["rms_eps"],
                           cfg["rope_theta"], 1 if cfg["qkv_bias"] else 0)
    lib = abi.lib

    def ok(rc):
        if rc != 0:
            raise RuntimeError(lib.lopa_last_error().decode())

    model, kv = C.c_void_p(), C.c_void_p()
    ok(lib.lopa_model_create(C.byref(c), C.byref(wp), None, C.byref(model)))
    nb = k + 1
    ok(lib.lopa_kv_create(model, P + L, nb, L, C.byref(kv)))
    tokens = hip.alloc(4 * nb * L)  # token 0 everywhere
    conf, pred = hip.alloc(4 * nb * L), hip.alloc(4 * nb * L)
    for _ in range(reps):
        ok(lib.lopa_verify_forward(model, kv, P, tokens, nb, L, conf, pred, None))
    hip.check(hip.rt.hipDeviceSynchronize(), "hipDeviceSynchronize")
    lib.lopa_kv_destroy(kv)
    lib.lopa_model_destroy(model)
    print(json.dumps({"verify_forwards": reps, "rows": nb * L, "prefix": P}))


def cpu_baseline(cfg_full, weights_dev, P, L, k, layers_sample=4, min_seconds=10.0, max_reps=8):
    """Time the oracle (float64 numpy) on a bounded sample of the same step:
    `layers_sample` decoder layers of the full shape + the LM head and softmax for
    all (k+1)*L rows, against a random prefix cache; the layer pass is repeated
    until about `min_seconds` of CPU work, and the mean is scaled to all layers."""
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
    # layers (repeated for a stable mean)
    t_all, reps = 0.0, 0
    while reps < max_reps and (reps == 0 or t_all < min_seconds):
        t0 = time.perf_counter()
        out = model.forward_block(tokens, P, cache, n_layers=layers_sample)
        t_all += time.perf_counter() - t0
        reps += 1
    t_layers = t_all / reps
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
                       f"mean of {reps} runs {t_layers:.2f}s layers + {t_head:.2f}s head, scaled to "
                       f"{step_s:.1f}s per step")}


def e2e_decode(lp, synth, model, cfg, prompt_len=256, gen=256, L=32, k=7, tau=0.9):
    """End-to-end LoPA decode (Alg. 1 driven block by block): a uniform-random
    prompt encoded block-causally, then gen / L blocks, each an initial forward
    plus LoPA iterations until the winner has no unfilled position, committing
    the winner's K/V every iteration. Iterations are timed one by one on the
    host (each ends with the 4-byte read of the winner's unfilled count)."""
    import torch
    kv = lp.KV(model, prompt_len + gen, k + 1, L)
    dec = lp.Decoder(model, kv, L, k, tau)
    prompt = synth.prompt(cfg, prompt_len, device="cuda")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    P = dec.prefill(prompt)
    torch.cuda.synchronize()
    t_prefill = time.perf_counter() - t0
    dec.forwards = 0
    steps, init_s = [], 0.0
    t1 = time.perf_counter()
    for _ in range(gen // L):
        ti = time.perf_counter()
        dec.init_block(P)
        torch.cuda.synchronize()
        init_s += time.perf_counter() - ti
        while True:
            ts = time.perf_counter()
            dec.step(P)
            done = int(dec.next_unfilled.item()) == 0
            steps.append(time.perf_counter() - ts)
            if done:
                break
            if len(steps) > 2 * gen:
                raise RuntimeError("decode did not converge")
        P += L
    torch.cuda.synchronize()
    t_dec = time.perf_counter() - t1
    st = sorted(steps)
    q = lambda f: st[min(len(st) - 1, int(f * len(st)))] * 1e3
    return {"workload": (f"{cfg['name']} shape, {prompt_len}-token uniform-random prompt, "
                         f"{gen} generated tokens in {gen // L} blocks of {L}, k={k}, tau {tau}"),
            "tokens_per_s": round(gen / t_dec, 1), "tokens_per_forward": round(gen / dec.forwards, 3),
            "forwards": dec.forwards, "iterations": len(steps),
            "step_ms_median": round(q(0.5), 3), "step_ms_p10": round(q(0.1), 3),
            "step_ms_p90": round(q(0.9), 3), "initial_forward_ms_mean": round(init_s / (gen // L) * 1e3, 3),
            "prefill_s": round(t_prefill, 4), "decode_s": round(t_dec, 4)}


def e2e_window_decode(lp, synth, model, cfg, prompt_len=256, gen=256, L=32, k=7, tau=0.9,
                      tau_add=0.1, tau_act=0.95, w_max=2, block_causal=False):
    """End-to-end decode with the multi-block window (Sec. 3.3, integration with
    D2F): up to w_max active blocks explored as one window, the D2F gates at the
    appendix's GSM8K setting (tau_add 0.1, tau_act 0.95, tau_conf 0.9);
    block_causal: the Ascend system's block-wise causal mask inside the window
    (Sec. 3.4) instead of full attention."""
    import torch
    kv = lp.KV(model, prompt_len + gen, k + 1, L * w_max)
    dec = lp.WindowDecoder(model, kv, L, k, tau, tau_add, tau_act, w_max, block_causal=block_causal)
    prompt = synth.prompt(cfg, prompt_len, device="cuda")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    out = dec.decode(prompt, gen)
    torch.cuda.synchronize()
    t = time.perf_counter() - t0
    return {"workload": (f"{cfg['name']} shape, {prompt_len}-token uniform-random prompt (prefill "
                         f"included), {gen} generated tokens, window of up to {w_max} blocks of {L}, "
                         f"k={k}, tau {tau}, tau_add {tau_add}, tau_act {tau_act}"
                         + (", block-causal attention inside the window" if block_causal else "")),
            "tokens_per_s": round(gen / t, 1), "tokens_per_forward": round(out["tpf"], 3),
            "forwards": out["forwards"], "iterations": out["iterations"], "seconds": round(t, 4)}


def fp8_step_figures(lp, synth, cfg, w, P, L, k, tau, steps, warmup, precision):
    """The same verify step (the block's first iteration, replayed) with the
    projections of `precision` in W8A8 E4M3 ("fp8_mlp": gate / up / down; "fp8":
    also QKV and the LM head): a second model from the same weights; ms/step,
    branch-tokens/s and per-kind times."""
    import torch
    nb, dev = k + 1, "cuda"
    model = lp.Model(cfg, w, precision=precision)
    kv = lp.KV(model, P + L, nb, L)
    dec = lp.Decoder(model, kv, L, k, tau)
    assert dec.prefill(synth.prompt(cfg, P, device=dev)) == P
    dec.init_block(P)
    i32 = dict(dtype=torch.int32, device=dev)
    tokens, conf, pred = dec.tokens.clone(), dec.conf.clone(), dec.pred.clone()
    bt, fp = torch.empty(nb * L, **i32), torch.empty(nb, **i32)
    va, nv = torch.empty(nb, dtype=torch.uint8, device=dev), torch.empty(1, **i32)
    cb, pb = torch.empty(nb * L, dtype=torch.float32, device=dev), torch.empty(nb * L, **i32)
    sc, win = torch.empty(nb, dtype=torch.float32, device=dev), torch.empty(1, **i32)
    nt, nc = torch.empty(L, **i32), torch.empty(L, dtype=torch.float32, device=dev)
    npd, nu, off = torch.empty(L, **i32), torch.empty(1, **i32), torch.empty(1, **i32)
    mask = cfg["mask_id"]

    def step():
        lp.lopa_build_branches(tokens, conf, pred, L, mask, tau, k, bt, fp, va, nv)
        lp.lopa_verify_forward(model, kv, P, bt, nb, L, cb, pb)
        lp.lopa_branch_confidence_select(bt, cb, pb, va, nb, L, mask, sc, win, nt, nc, npd, nu)
        lp.lopa_commit_kv(kv, win, P, L, off)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    kv.profile(lp.PROF_KINDS)
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    prof = kv.profile_read()
    kv.profile(())
    what = ("gate / up / down" if precision == "fp8_mlp"
            else "QKV, gate / up / down and the LM head")
    rest = ("attention, QKV / O and the LM head bf16" if precision == "fp8_mlp"
            else "attention and the output projection bf16")
    out = {"workload": f"the headline step with {what} in W8A8 E4M3 (per-channel weight "
                       f"and per-row activation scales); {rest}",
           "ms_per_step": round(ms, 4), "branch_tokens_per_s": round(nb * L / (ms * 1e-3), 1),
           "kernel_ms_per_step": {kd: round(t / steps, 4) for kd, (t, n) in prof.items()}}
    del dec, kv, model
    torch.cuda.empty_cache()
    return out


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
    ap.add_argument("--no-e2e", action="store_true", help="skip the end-to-end decode run")
    ap.add_argument("--precision", default="bf16", choices=["bf16", "fp8_mlp", "fp8"],
                    help="projection precision of the timed model (the headline is bf16; "
                         "fp8_mlp: gate / up / down in W8A8 E4M3; fp8: also QKV and the LM head)")
    ap.add_argument("--no-fp8", action="store_true", help="skip the FP8 step figures")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a 1 GiB device copy 5 times (HBM counter calibration)")
    ap.add_argument("--hbm-counters", action="store_true",
                    help="only run 3 torch-free verify forwards (for rocprofv3 --pmc)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: this build runs on one GPU; --gpus {args.gpus} is not supported "
              "(multi-GPU branch parallelism is a design note, not built)", file=sys.stderr)
        sys.exit(2)

    if args.copy_calibration:
        copy_calibration()
        return
    if args.hbm_counters:
        # the shape table of the synthetic generator, read without importing torch
        import importlib.util
        spec = importlib.util.spec_from_file_location("synth_shapes",
                                                      os.path.join(ROOT, "synth", "shapes.py"))
        shapes = importlib.util.module_from_spec(spec)
        spec.loader.exec_module(shapes)
        hbm_counter_run(shapes.config(args.config), args.prefix, args.block, args.k)
        return

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
    model = lp.Model(cfg, w, precision=args.precision)
    log(f"model repacked in {time.perf_counter() - t0:.1f}s ({args.precision})")
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

    # launch times with HIP events on the library's stream: first the gate/up
    # launches alone (the roofline kernel; one event pair per launch), then
    # every kind for the per-step breakdown
    kv.profile(("gateup",))
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    t, n = kv.profile_read()["gateup"]
    gu_ms = t / n
    kv.profile(lp.PROF_KINDS)
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    prof = kv.profile_read()
    kv.profile(())
    per_step_ms = {kd: t / args.steps for kd, (t, n) in prof.items()}
    log("per-step ms by kind: " + ", ".join(f"{kd} {v:.3f}" for kd, v in per_step_ms.items()))

    # the box's own copy bandwidth (device-to-device copy of 1 GiB, read + write
    # bytes over the event time), the reference a measured roofline is read against
    src = torch.empty(1 << 29, dtype=torch.int16, device=dev)
    dst = torch.empty_like(src)
    dst.copy_(src)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(5):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    copy_gbs = 5 * 2 * src.numel() * 2 / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del src, dst

    gu_bytes = gateup_launch_bytes(cfg, M, args.precision)
    achieved = gu_bytes / (gu_ms * 1e-3) / 1e9
    sb = step_bytes(cfg, P, L, nb, args.precision)
    sf = step_flops(cfg, P, L, nb)
    result = {
        "metric": "LoPA verify-step ms & branch-tokens/s (7B shape, k=7); % HBM/MFMA roofline",
        "value": round(nb * L / (ms * 1e-3), 1),
        "unit": "branch-tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": {"bf16": "bf16", "fp8_mlp": "bf16 + fp8(e4m3) MLP",
                  "fp8": "bf16 + fp8(e4m3) QKV/MLP/LM head"}[args.precision], "data": "synthetic",
        "config": {"workload": (f"LoPA verify step, {args.config} shape ({cfg['layers']}L H{cfg['hidden']} "
                                f"{cfg['heads']}q/{cfg['kv_heads']}kv d{cfg['head_dim']} F{cfg['ffn']} "
                                f"V{cfg['vocab']}), random bf16 weights, prefix {P}, block {L}, "
                                f"k={k} ({nb} branches, {M} rows), tau {tau}"),
                   "prefix": P, "block": L, "k": k, "rows": M},
        "roofline": {"bound": "hbm", "kernel": "gate/up projection + SwiGLU (gemm_kernel<EPI_SWIGLU>)",
                     "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": measured_traffic(os.path.join(ROOT, "profiles",
                                                              "gemm_swiglu_dream7b_hbm_traffic.md"))
                     if args.precision == "bf16" else None,
                     "bytes_per_launch": gu_bytes, "avg_launch_ms": round(gu_ms, 4),
                     "copy_gbs_measured": round(copy_gbs, 1),
                     "frac_of_measured_copy": round(achieved / copy_gbs, 4)},
        "step_roofline": {"hbm_bytes": sb, "flops": sf,
                          "hbm_frac": round(sb / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                          "mfma_frac": round(sf / (ms * 1e-3) / 1e12 / MFMA_BF16_PEAK_TFS, 4)},
        "kernel_ms_per_step": {kd: round(v, 4) for kd, v in per_step_ms.items()},
    }
    if not args.no_e2e:
        t0 = time.perf_counter()
        result["e2e_decode"] = e2e_decode(lp, synth, model, cfg, L=L, k=k, tau=tau)
        log(f"end-to-end decode in {time.perf_counter() - t0:.1f}s: "
            f"{result['e2e_decode']['tokens_per_s']} tok/s, TPF {result['e2e_decode']['tokens_per_forward']}")
        if 2 * L <= lp.MAX_BLOCK:
            t0 = time.perf_counter()
            result["e2e_window_decode"] = e2e_window_decode(lp, synth, model, cfg, L=L, k=k, tau=tau)
            log(f"end-to-end window decode in {time.perf_counter() - t0:.1f}s: "
                f"{result['e2e_window_decode']['tokens_per_s']} tok/s, "
                f"TPF {result['e2e_window_decode']['tokens_per_forward']}")
            t0 = time.perf_counter()
            result["e2e_window_decode_block_causal"] = e2e_window_decode(
                lp, synth, model, cfg, L=L, k=k, tau=tau, block_causal=True)
            log(f"end-to-end block-causal window decode in {time.perf_counter() - t0:.1f}s: "
                f"{result['e2e_window_decode_block_causal']['tokens_per_s']} tok/s, "
                f"TPF {result['e2e_window_decode_block_causal']['tokens_per_forward']}")
    if args.precision == "bf16" and not args.no_fp8:
        for prec in ("fp8_mlp", "fp8"):
            t0 = time.perf_counter()
            key = prec + "_step"
            result[key] = fp8_step_figures(lp, synth, cfg, w, P, L, k, tau, args.steps,
                                           args.warmup, prec)
            log(f"{prec} step in {time.perf_counter() - t0:.1f}s: "
                f"{result[key]['ms_per_step']} ms/step")
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
