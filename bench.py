"""Benchmark of one LoPA verify step on one MI355X.

One step = lopa_build_branches + lopa_verify_forward (all k+1 branches, one
pass) + lopa_branch_confidence_select + lopa_commit_kv on the Dream-7B shape
(28 layers, hidden 3584, 28 q / 4 kv heads, head_dim 128, SwiGLU 18944, vocab
152064; random bf16 weights N(0, 0.02)), prefix 512 (block-causal prefill of a
uniform-random prompt), block 32, k = 7 (8 branches, 256 rows), tau = 0.9. The
timed state is the block's first iteration (all 32 positions masked, conf /
pred from the initial forward), replayed K times (commit rewrites the same rows).

Prints one JSON line: value = branch-tokens/s = 8 * 32 / mean step seconds,
with the median / p10 / p90 of the per-step times (an event before every step),
per-kind launch times, the gate/up roofline, end-to-end decode figures, the
FP8 variants, three further shapes (the 2-layer tiny model at prefix 64, k = 3;
the same 7B model at prefix 2048, k = 15; the LLaDA-8B layout at prefix 1024,
k = 7) and the float64 oracle's time for the same whole step on the host CPU.
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


def hbm_counter_run(cfg, P, L, k, reps=3, precision="bf16"):
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
    prec = {"bf16": 0, "fp8_mlp": 1, "fp8": 2}[precision]  # LOPA_PRECISION_*
    ok(lib.lopa_model_create_ex(C.byref(c), C.byref(wp), prec, None, C.byref(model)))
    nb = k + 1
    ok(lib.lopa_kv_create(model, P + L, nb, L, C.byref(kv)))
    tokens = hip.alloc(4 * nb * L)  # token 0 everywhere
    conf, pred = hip.alloc(4 * nb * L), hip.alloc(4 * nb * L)
    for _ in range(reps):
        ok(lib.lopa_verify_forward(model, kv, P, tokens, nb, L, conf, pred, None))
    hip.check(hip.rt.hipDeviceSynchronize(), "hipDeviceSynchronize")
    lib.lopa_kv_destroy(kv)
    lib.lopa_model_destroy(model)
    print(json.dumps({"verify_forwards": reps, "rows": nb * L, "prefix": P, "precision": precision}))


def host_info():
    """The CPU model, the BLAS library numpy calls (and its thread count) and
    the cores this process may run on."""
    import subprocess
    model = None
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for line in out.splitlines():
            if line.startswith("Model name:"):
                model = line.split(":", 1)[1].strip()
                break
    except (OSError, subprocess.SubprocessError):
        pass
    blas = []
    try:
        import numpy  # noqa: F401  (loads the BLAS that threadpoolctl inspects)
        from threadpoolctl import threadpool_info
        blas = [{"api": i.get("internal_api"), "version": i.get("version"),
                 "threads": i.get("num_threads")}
                for i in threadpool_info() if i.get("user_api") == "blas"]
    except ImportError:
        pass
    return {"cpu_model": model, "blas": blas, "affinity_cores": len(os.sched_getaffinity(0))}


class _HostLayers:
    """The device layers as float64 host tensors, converted on access."""

    def __init__(self, layers):
        self.layers = layers

    def __len__(self):
        return len(self.layers)

    def __getitem__(self, i):
        return {kk: v.double().cpu() for kk, v in self.layers[i].items()}


def cpu_baseline(cfg, weights_dev, state, P, L, k, tau, runs=3):
    """Time the oracle (float64 numpy, as it stands) on the same step: one
    LoPA iteration (build, batched forward of all k+1 branches through every
    layer and the LM head, select, commit) from the GPU's first-iteration
    state, against a random prefix cache of length P. Median of `runs` runs.
    The weights are converted to float64 host arrays before the timed region
    when host memory allows, else one layer at a time inside it (said in the
    sample text)."""
    import numpy as np
    import psutil

    import synth
    from oracle import KVCache, OracleModel
    from oracle.lopa import lopa_step

    n_layer = sum(v.numel() for v in weights_dev["layers"][0].values())
    need = 8 * (cfg["layers"] * n_layer + weights_dev["embed"].numel() +
                weights_dev["lm_head"].numel())
    resident = psutil.virtual_memory().available > 1.25 * need + (16 << 30)
    host = {"embed": weights_dev["embed"].double().cpu(),
            "layers": _HostLayers(weights_dev["layers"]),
            "final_norm": weights_dev["final_norm"].double().cpu(),
            "lm_head": weights_dev["lm_head"].double().cpu()}
    model = OracleModel(cfg, host, "pure", keep_layers=True if resident else 1)
    del host
    t0 = time.perf_counter()
    if resident:
        for i in range(cfg["layers"]):
            model.layer(i)
    t_conv = time.perf_counter() - t0
    print(f"cpu baseline: weights {'converted' if resident else 'left bf16'} in {t_conv:.1f}s",
          file=sys.stderr, flush=True)
    cache = KVCache(cfg, P + L)
    g = synth.irwin_hall(synth.stream_key(7, 1), cache.k[:, :, :P].size, 1.0).double().numpy()
    cache.k[:, :, :P] = g.reshape(cache.k[:, :, :P].shape)
    cache.v[:, :, :P] = -g.reshape(cache.v[:, :, :P].shape)
    st = (np.asarray(state[0], dtype=np.int64), np.asarray(state[1], dtype=np.float64),
          np.asarray(state[2], dtype=np.int64))
    times = []
    for _ in range(runs):
        t0 = time.perf_counter()
        lopa_step(model, cache, P, st, k, tau)
        times.append(time.perf_counter() - t0)
        print(f"cpu baseline: oracle step {len(times)} in {times[-1]:.2f}s", file=sys.stderr,
              flush=True)
    step_s = sorted(times)[len(times) // 2]
    info = host_info()
    threads = max([b["threads"] for b in info["blas"] if b["threads"]] or [1])
    nb = k + 1
    return {"value": round(nb * L / step_s, 3), "unit": "branch-tokens/s", "cores": threads,
            "kind": "oracle", "ms_per_step": round(step_s * 1e3, 1),
            "runs_s": [round(t, 3) for t in times],
            "cpu_model": info["cpu_model"], "blas": info["blas"],
            "affinity_cores": info["affinity_cores"],
            "sample": (f"the whole step, not a sample: float64 numpy oracle, one LoPA iteration "
                       f"(build, forward of {nb}x{L} rows through all {cfg['layers']} layers + "
                       f"LM head / softmax, select, commit) on the {cfg['name']} shape, prefix {P} "
                       f"(random cache), median of {runs} runs; weights "
                       + (f"converted to float64 before the timed region ({t_conv:.1f}s)"
                          if resident else "upcast from bf16 one layer at a time inside it"))}


def cpu_tiny_step(cfg, weights_dev, state, P, L, k, tau, runs=20):
    """The oracle's step time on a small shape (median of `runs`, seconds)."""
    import numpy as np

    from oracle import KVCache, OracleModel
    from oracle.lopa import lopa_step

    host = {"embed": weights_dev["embed"].double().cpu(),
            "layers": [{kk: v.double().cpu() for kk, v in lw.items()}
                       for lw in weights_dev["layers"]],
            "final_norm": weights_dev["final_norm"].double().cpu(),
            "lm_head": weights_dev["lm_head"].double().cpu()}
    model = OracleModel(cfg, host, "pure")
    cache = KVCache(cfg, P + L)
    rng = np.random.default_rng(7)
    cache.k[:, :, :P] = rng.standard_normal(cache.k[:, :, :P].shape)
    cache.v[:, :, :P] = rng.standard_normal(cache.v[:, :, :P].shape)
    st = (np.asarray(state[0], dtype=np.int64), np.asarray(state[1], dtype=np.float64),
          np.asarray(state[2], dtype=np.int64))
    times = []
    for _ in range(runs):
        t0 = time.perf_counter()
        lopa_step(model, cache, P, st, k, tau)
        times.append(time.perf_counter() - t0)
    return sorted(times)[runs // 2]


class StepRunner:
    """The timed workload: the four calls of one LoPA iteration (build, verify
    forward of all k+1 branches, select, commit) on the block's first state
    (all L positions masked, conf / pred from the initial forward), replayed;
    the commit rewrites the same cache rows, so every replay is the same step."""

    def __init__(self, lp, synth, model, cfg, P, L, k, tau):
        import torch
        self.lp, self.model, self.cfg = lp, model, cfg
        self.P, self.L, self.k, self.tau, self.nb = P, L, k, tau, k + 1
        dev = "cuda"
        self.kv = lp.KV(model, P + L, self.nb, L)
        dec = lp.Decoder(model, self.kv, L, k, tau)
        assert dec.prefill(synth.prompt(cfg, P, device=dev)) == P
        dec.init_block(P)
        self.dec = dec
        i32 = dict(dtype=torch.int32, device=dev)
        nb = self.nb
        self.tokens, self.conf, self.pred = dec.tokens.clone(), dec.conf.clone(), dec.pred.clone()
        self.bt, self.fp = torch.empty(nb * L, **i32), torch.empty(nb, **i32)
        self.va, self.nv = torch.empty(nb, dtype=torch.uint8, device=dev), torch.empty(1, **i32)
        self.cb = torch.empty(nb * L, dtype=torch.float32, device=dev)
        self.pb = torch.empty(nb * L, **i32)
        self.sc, self.win = torch.empty(nb, dtype=torch.float32, device=dev), torch.empty(1, **i32)
        self.nt, self.nc = torch.empty(L, **i32), torch.empty(L, dtype=torch.float32, device=dev)
        self.npd, self.nu, self.off = torch.empty(L, **i32), torch.empty(1, **i32), torch.empty(1, **i32)

    def step(self):
        lp, L, k, nb, P, mask = self.lp, self.L, self.k, self.nb, self.P, self.cfg["mask_id"]
        lp.lopa_build_branches(self.tokens, self.conf, self.pred, L, mask, self.tau, k, self.bt,
                               self.fp, self.va, self.nv)
        lp.lopa_verify_forward(self.model, self.kv, P, self.bt, nb, L, self.cb, self.pb)
        lp.lopa_branch_confidence_select(self.bt, self.cb, self.pb, self.va, nb, L, mask, self.sc,
                                         self.win, self.nt, self.nc, self.npd, self.nu)
        lp.lopa_commit_kv(self.kv, self.win, P, L, self.off)

    def time(self, steps, warmup):
        """Per-step times from an event before each step and after the last:
        mean over the run (= (last - first) / steps) and the step quantiles."""
        import torch
        for _ in range(warmup):
            self.step()
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
        ev[0].record()
        for i in range(steps):
            self.step()
            ev[i + 1].record()
        torch.cuda.synchronize()
        per = sorted(ev[i].elapsed_time(ev[i + 1]) for i in range(steps))
        q = lambda f: per[min(steps - 1, int(round(f * (steps - 1))))]
        return {"mean": ev[0].elapsed_time(ev[steps]) / steps, "median": q(0.5), "p10": q(0.1),
                "p90": q(0.9), "steps": steps}

    def kinds(self, steps):
        """Per-kind launch times (HIP events on the library's stream) per step."""
        import torch
        self.kv.profile(self.lp.PROF_KINDS)
        for _ in range(steps):
            self.step()
        torch.cuda.synchronize()
        prof = self.kv.profile_read()
        self.kv.profile(())
        return {kd: round(t / steps, 4) for kd, (t, n) in prof.items()}


def blas_reference(reps_per_copy=20):
    """The same GEMM shapes (256 rows, the verify step at the 7B shape) through
    torch.matmul (the vendor BLAS, hipBLASLt / rocBLAS) in bf16, with enough
    distinct weight copies that every call streams its weights from HBM, as
    the model's layers do. The library GEMMs here carry no epilogue (no
    SwiGLU, bias, RoPE or softmax statistics)."""
    import torch
    out = {}
    for name, (M, K, N) in {"qkv": (256, 3584, 4608), "o": (256, 3584, 3584),
                            "gateup": (256, 3584, 37888), "down": (256, 18944, 3584),
                            "lmhead": (256, 3584, 152064)}.items():
        copies = max(2, int(600e6 // (K * N * 2)))
        g = torch.Generator(device="cuda").manual_seed(0)
        A = torch.randn(M, K, device="cuda", dtype=torch.bfloat16, generator=g) * 0.1
        Ws = [torch.randn(N, K, device="cuda", dtype=torch.bfloat16, generator=g) * 0.02
              for _ in range(copies)]
        for W in Ws:
            C = A @ W.t()
        torch.cuda.synchronize()
        reps = reps_per_copy * copies
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for i in range(reps):
            C = A @ Ws[i % copies].t()
        e1.record()
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) * 1e3 / reps
        out[name] = {"M": M, "K": K, "N": N, "us": round(us, 1),
                     "weight_gbs": round(K * N * 2 / us / 1e3, 1)}
        del Ws, A, C
        torch.cuda.empty_cache()
    print(json.dumps({"blas_reference": out}))


def shape_figure(lp, synth, model, cfg, P, L, k, tau, steps, warmup, what, precision="bf16"):
    """One line per further measured shape: ms/step (mean, median, p10, p90),
    branch-tokens/s, the step's algorithmic HBM bytes and FLOPs against the
    peaks, per-kind times."""
    import torch
    run = StepRunner(lp, synth, model, cfg, P, L, k, tau)
    t = run.time(steps, warmup)
    kinds = run.kinds(steps)
    nb = k + 1
    sb, sf = step_bytes(cfg, P, L, nb, precision), step_flops(cfg, P, L, nb)
    ms = t["mean"]
    out = {"workload": what, "ms_per_step": round(ms, 4),
           "ms_median": round(t["median"], 4), "ms_p10": round(t["p10"], 4),
           "ms_p90": round(t["p90"], 4), "steps": t["steps"],
           "branch_tokens_per_s": round(nb * L / (ms * 1e-3), 1),
           "step_roofline": {"hbm_bytes": sb, "flops": sf,
                             "hbm_frac": round(sb / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                             "mfma_frac": round(sf / (ms * 1e-3) / 1e12 / MFMA_BF16_PEAK_TFS, 4)},
           "kernel_ms_per_step": kinds}
    del run
    torch.cuda.empty_cache()
    return out


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
                         f"included), {gen} generated tokens, window of up to {w_max} blocks of {L} "
                         f"(gates on the device), "
                         f"k={k}, tau {tau}, tau_add {tau_add}, tau_act {tau_act}"
                         + (", block-causal attention inside the window" if block_causal else "")),
            "tokens_per_s": round(gen / t, 1), "tokens_per_forward": round(out["tpf"], 3),
            "forwards": out["forwards"], "iterations": out["iterations"], "seconds": round(t, 4)}


def fp8_step_figures(lp, synth, cfg, w, P, L, k, tau, steps, warmup, precision):
    """The same verify step (the block's first iteration, replayed) with the
    projections of `precision` in W8A8 E4M3 ("fp8_mlp": gate / up / down; "fp8":
    also QKV, O and the LM head): a second model from the same weights; ms/step,
    branch-tokens/s and per-kind times."""
    import torch
    model = lp.Model(cfg, w, precision=precision)
    what = ("gate / up / down" if precision == "fp8_mlp"
            else "QKV, O, gate / up / down and the LM head")
    rest = ("attention, QKV / O and the LM head bf16" if precision == "fp8_mlp"
            else "attention bf16")
    out = shape_figure(lp, synth, model, cfg, P, L, k, tau, steps, warmup,
                       f"the headline step with {what} in W8A8 E4M3 (per-channel weight "
                       f"and per-row activation scales); {rest}", precision)
    del model
    torch.cuda.empty_cache()
    return out


def describe(cfg, P, L, k, tau):
    nb = k + 1
    return (f"LoPA verify step, {cfg['name']} shape ({cfg['layers']}L H{cfg['hidden']} "
            f"{cfg['heads']}q/{cfg['kv_heads']}kv d{cfg['head_dim']} F{cfg['ffn']} "
            f"V{cfg['vocab']}), random bf16 weights, prefix {P}, block {L}, "
            f"k={k} ({nb} branches, {nb * L} rows), tau {tau}")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=60)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="dream7b", help="synth config name (model shape)")
    ap.add_argument("--prefix", type=int, default=512)
    ap.add_argument("--block", type=int, default=32)
    ap.add_argument("--k", type=int, default=7)
    ap.add_argument("--tau", type=float, default=0.9)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-runs", type=int, default=3)
    ap.add_argument("--no-e2e", action="store_true", help="skip the end-to-end decode runs")
    ap.add_argument("--no-shapes", action="store_true",
                    help="skip the further shapes (tiny; k=15 at prefix 2048; LLaDA-8B)")
    ap.add_argument("--precision", default="bf16", choices=["bf16", "fp8_mlp", "fp8"],
                    help="projection precision of the timed model (the headline is bf16; "
                         "fp8_mlp: gate / up / down in W8A8 E4M3; fp8: also QKV and the LM head)")
    ap.add_argument("--no-fp8", action="store_true", help="skip the FP8 step figures")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a 1 GiB device copy 5 times (HBM counter calibration)")
    ap.add_argument("--hbm-counters", action="store_true",
                    help="only run 3 torch-free verify forwards (for rocprofv3 --pmc)")
    ap.add_argument("--blas-reference", action="store_true",
                    help="only time the step's GEMM shapes through torch.matmul (vendor BLAS)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: the library runs the verify step on one GPU; --gpus {args.gpus} is "
              "not supported (branch parallelism over several GPUs is not implemented)",
              file=sys.stderr)
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
        hbm_counter_run(shapes.config(args.config), args.prefix, args.block, args.k,
                        precision=args.precision)
        return

    import torch

    if args.blas_reference:
        blas_reference()
        return

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
    t0 = time.perf_counter()
    run = StepRunner(lp, synth, model, cfg, P, L, k, tau)
    torch.cuda.synchronize()
    log(f"prefill of {P} positions + initial forward in {time.perf_counter() - t0:.1f}s")

    t0 = time.perf_counter()
    t = run.time(args.steps, args.warmup)
    wall = time.perf_counter() - t0
    ms = t["mean"]
    log(f"{args.steps} steps: {ms:.3f} ms/step mean, median {t['median']:.3f}, p10 {t['p10']:.3f}, "
        f"p90 {t['p90']:.3f} (events); {wall / (args.steps + args.warmup) * 1e3:.3f} ms/step (wall)")

    # launch times with HIP events on the library's stream: first the gate/up
    # launches alone (the roofline kernel; one event pair per launch), then
    # every kind for the per-step breakdown
    run.kv.profile(("gateup",))
    for _ in range(args.steps):
        run.step()
    torch.cuda.synchronize()
    tg, n = run.kv.profile_read()["gateup"]
    gu_ms = tg / n
    run.kv.profile(())
    per_step_ms = run.kinds(args.steps)
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
        "ms_median": round(t["median"], 4), "ms_p10": round(t["p10"], 4),
        "ms_p90": round(t["p90"], 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": {"bf16": "bf16", "fp8_mlp": "bf16 + fp8(e4m3) MLP",
                  "fp8": "bf16 + fp8(e4m3) QKV/MLP/LM head"}[args.precision], "data": "synthetic",
        "config": {"workload": describe(cfg, P, L, k, tau), "prefix": P, "block": L, "k": k,
                   "rows": M},
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
        "kernel_ms_per_step": per_step_ms,
    }
    state = (run.tokens.cpu().numpy(), run.conf.cpu().numpy(), run.pred.cpu().numpy())
    del run
    torch.cuda.empty_cache()
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
            if 4 * L <= lp.MAX_BLOCK:
                t0 = time.perf_counter()
                result["e2e_window_decode_w4"] = e2e_window_decode(lp, synth, model, cfg, L=L, k=k,
                                                                   tau=tau, w_max=4)
                log(f"end-to-end window decode (4 blocks) in {time.perf_counter() - t0:.1f}s: "
                    f"{result['e2e_window_decode_w4']['tokens_per_s']} tok/s, "
                    f"TPF {result['e2e_window_decode_w4']['tokens_per_forward']}")
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
    if not args.no_shapes and args.config == "dream7b":
        shapes = {}
        # the same model at 16 branches and a 2048-position prefix
        t0 = time.perf_counter()
        shapes["dream7b_p2048_k15"] = shape_figure(
            lp, synth, model, cfg, 2048, 32, 15, tau, args.steps, args.warmup,
            describe(cfg, 2048, 32, 15, tau))
        log(f"dream7b p2048 k15 in {time.perf_counter() - t0:.1f}s: "
            f"{shapes['dream7b_p2048_k15']['ms_per_step']} ms/step")
        # the parity workhorse: launch-bound, microseconds per step
        t0 = time.perf_counter()
        ct = synth.config("tiny")
        wt = synth.model_weights(ct, device=dev, dtype=torch.bfloat16)
        mt = lp.Model(ct, wt)
        fig = shape_figure(lp, synth, mt, ct, 64, 16, 3, tau, max(args.steps, 200),
                           args.warmup, describe(ct, 64, 16, 3, tau))
        fig["us_per_step"] = round(fig["ms_per_step"] * 1e3, 1)
        fig["us_median"] = round(fig["ms_median"] * 1e3, 1)
        if not args.no_cpu_baseline:
            rt = StepRunner(lp, synth, mt, ct, 64, 16, 3, tau)
            st = (rt.tokens.cpu().numpy(), rt.conf.cpu().numpy(), rt.pred.cpu().numpy())
            del rt
            fig["cpu_oracle_us_per_step"] = round(
                cpu_tiny_step(ct, wt, st, 64, 16, 3, tau) * 1e6, 1)
        shapes["tiny_p64_k3"] = fig
        del mt, wt
        log(f"tiny in {time.perf_counter() - t0:.1f}s: {fig['us_per_step']} us/step")
        # LLaDA-8B layout (MHA, 32 layers) at prefix 1024
        t0 = time.perf_counter()
        cl = synth.config("llada8b")
        wl = synth.model_weights(cl, device=dev, dtype=torch.bfloat16)
        ml = lp.Model(cl, wl)
        shapes["llada8b_p1024_k7"] = shape_figure(
            lp, synth, ml, cl, 1024, 32, 7, tau, args.steps, args.warmup,
            describe(cl, 1024, 32, 7, tau))
        del ml, wl
        torch.cuda.empty_cache()
        log(f"llada8b p1024 k7 in {time.perf_counter() - t0:.1f}s: "
            f"{shapes['llada8b_p1024_k7']['ms_per_step']} ms/step")
        result["shapes"] = shapes
    if not args.no_cpu_baseline:
        t0 = time.perf_counter()
        try:
            result["cpu_baseline"] = cpu_baseline(cfg, w, state, P, L, k, tau, args.cpu_runs)
        except Exception as e:  # the GPU number stands; say why the baseline is missing
            result["cpu_baseline"] = {"value": None, "error": repr(e)}
        log(f"cpu baseline in {time.perf_counter() - t0:.1f}s")
    print(json.dumps(result))


if __name__ == "__main__":
    main()
