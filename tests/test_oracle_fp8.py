"""Pins of the oracle's FP8 pieces (oracle/fp8.py), CPU only.

* E4M3 rounding against torch's independent float8_e4m3fn conversion: every
  code point, exact midpoints (ties to even), random values over the whole
  range including subnormals, and saturation at +-448.
* Per-row scaling: the largest magnitude of a row maps to +-448 exactly, a zero
  row to zeros, dequantised values within the E4M3 relative step of the input,
  and scaling a row by a power of two scales the result exactly.
* The quantised product stays within the error bound the two roundings allow,
  and the FP8 mode of the forward runs the MLP through it."""
import numpy as np
import pytest
import torch

import synth
from oracle import KVCache, OracleModel, lopa
from oracle.fp8 import E4M3_MAX, e4m3_round, fp8_matmul, quantize_rows


def torch_e4m3(x):
    t = torch.tensor(np.asarray(x, dtype=np.float32))
    return t.to(torch.float8_e4m3fn).to(torch.float32).numpy().astype(np.float64)


def all_codes():
    codes = torch.arange(256, dtype=torch.int32).to(torch.uint8).view(torch.float8_e4m3fn)
    v = codes.to(torch.float32).numpy().astype(np.float64)
    return np.unique(v[np.isfinite(v)])


def test_codes_are_fixed_points():
    v = all_codes()
    assert v.max() == E4M3_MAX and v.min() == -E4M3_MAX
    assert len(v) == 253  # 256 codes minus two NaNs, +0 and -0 merged
    assert np.array_equal(e4m3_round(v), v)


def test_midpoints_round_to_even():
    v = all_codes()
    pos = v[v >= 0]
    mid = (pos[:-1] + pos[1:]) / 2.0
    got = e4m3_round(mid)
    assert np.array_equal(got, torch_e4m3(mid))
    # ties go to the code with an even mantissa (the even index among the codes)
    idx = np.searchsorted(pos, got)
    assert np.all(idx % 2 == 0)
    assert np.array_equal(e4m3_round(-mid), -got)


def test_random_values_match_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.uniform(-448, 448, 20000),
                        rng.standard_normal(20000) * 10.0 ** rng.uniform(-4, 2, 20000),
                        rng.uniform(-2 ** -6, 2 ** -6, 5000)])
    x = x.astype(np.float32).astype(np.float64)
    assert np.array_equal(e4m3_round(x), torch_e4m3(x))


def test_saturation():
    x = np.array([448.0, 450.0, 463.9, 464.0, 500.0, 1e6, -1e6])
    assert np.array_equal(e4m3_round(x), [448, 448, 448, 448, 448, 448, -448])


def test_row_scaling_rule():
    rng = np.random.default_rng(1)
    v = rng.standard_normal((6, 300)) * np.array([1e-3, 0.1, 1, 10, 300, 0])[:, None]
    q, s = quantize_rows(v)
    for i in range(5):
        j = np.argmax(np.abs(v[i]))
        assert abs(q[i, j]) == E4M3_MAX and np.all(np.abs(q[i]) <= E4M3_MAX)
        # dequantised within half an E4M3 step (relative 2^-4) plus the subnormal step
        err = np.abs(q[i] * s[i] - v[i])
        assert np.all(err <= 2.0 ** -4 * np.abs(v[i]) + 2.0 ** -10 * s[i] * 1.0001 + 1e-12)
    assert s[5] == 0 and not np.any(q[5])
    # a power-of-two multiple of a row: the same codes, the scale times that power
    q2, s2 = quantize_rows(v[:5] * 8.0)
    assert np.array_equal(q2, q[:5]) and np.array_equal(s2, s[:5] * 8.0)


def test_quantized_product_error_bound():
    rng = np.random.default_rng(2)
    x = rng.standard_normal((8, 512))
    w = rng.standard_normal((64, 512)) * 0.02
    qw, sw = quantize_rows(w)
    y = fp8_matmul(x, qw, sw)
    exact = x @ w.T
    qx, sx = quantize_rows(x)
    # each factor within relative 2^-4 (plus its subnormal step) of its input
    ex = np.abs(qx * sx[:, None] - x)
    ew = np.abs(qw * sw[:, None] - w)
    bound = ex @ np.abs(w).T + np.abs(x) @ ew.T + ex @ ew.T
    assert np.all(np.abs(y - exact) <= bound * (1 + 1e-9) + 1e-12)
    assert np.max(np.abs(y - exact)) > 0


def test_fp8_mode_forward():
    """The FP8 mode quantises exactly the three MLP projections: its weights
    dequantise to the bf16 weights within the E4M3 step, and with a zero down
    projection (no MLP contribution) the FP8 and bf16 modes agree bit for bit,
    so nothing outside the MLP is quantised."""
    cfg = synth.config("tiny")
    w = synth.model_weights(cfg)
    f = OracleModel(cfg, w, "faithful")
    q = OracleModel(cfg, w, "fp8_mlp")
    layer = q.layers[0]
    for key in ("w_gate", "w_up", "w_down"):
        assert np.all(np.abs(layer[key + "_q"]) <= E4M3_MAX)
        err = np.abs(layer[key + "_q"] * layer[key + "_s"][:, None] - f.layers[0][key])
        assert np.all(err <= 2.0 ** -4 * np.abs(f.layers[0][key])
                      + 2.0 ** -10 * layer[key + "_s"][:, None] * 1.0001)
    cache = KVCache(cfg, 48)
    bt = np.full((2, 16), cfg["mask_id"])
    for m in (f, q):
        for lw in m.layers:
            lw["w_down"] = np.zeros_like(lw["w_down"])
            if "w_down_q" in lw:
                lw["w_down_q"] = np.zeros_like(lw["w_down_q"])
    a, b = f.forward_block(bt, 0, cache), q.forward_block(bt, 0, cache)
    assert np.array_equal(a["conf"], b["conf"]) and np.array_equal(a["k"], b["k"])


@pytest.mark.parametrize("k", [0, 3])
def test_fp8_mode_decodes(k):
    cfg = synth.config("tiny")
    q = OracleModel(cfg, synth.model_weights(cfg), "fp8_mlp")
    res = lopa.decode(q, synth.prompt(cfg, 32).numpy(), 32, 16, k, 0.9)
    assert len(res["tokens"]) == 32 and not np.any(res["tokens"] == cfg["mask_id"])


def test_fp8_full_mode_quantizes_every_projection():
    """The "fp8" mode adds the QKV projection, the output projection and the
    LM head: their weights dequantise to the bf16 weights within the E4M3
    step, and the LM head's logits are the quantised product of the
    final-normed rows."""
    cfg = synth.config("tiny")
    w = synth.model_weights(cfg)
    f = OracleModel(cfg, w, "faithful")
    q = OracleModel(cfg, w, "fp8")
    for key in ("wq", "wk", "wv", "wo"):
        l0, f0 = q.layers[0], f.layers[0]
        err = np.abs(l0[key + "_q"] * l0[key + "_s"][:, None] - f0[key])
        assert np.all(err <= 2.0 ** -4 * np.abs(f0[key]) + 2.0 ** -10 * l0[key + "_s"][:, None] * 1.0001)
    err = np.abs(q.lm_head_q * q.lm_head_s[:, None] - f.lm_head)
    assert np.all(err <= 2.0 ** -4 * np.abs(f.lm_head) + 2.0 ** -10 * q.lm_head_s[:, None] * 1.0001)
    cache = KVCache(cfg, 48)
    bt = np.full((2, 16), cfg["mask_id"])
    out = q.forward_block(bt, 0, cache, keep_hidden=True)
    np.testing.assert_allclose(out["logits"], fp8_matmul(out["hidden"], q.lm_head_q, q.lm_head_s),
                               rtol=0, atol=1e-12)
    res = lopa.decode(q, synth.prompt(cfg, 32).numpy(), 32, 16, 3, 0.9)
    assert len(res["tokens"]) == 32 and not np.any(res["tokens"] == cfg["mask_id"])


def test_fp8_output_projection_within_quantization_bound():
    """In the "fp8" mode the output projection's contribution to the residual
    stream (the value after the attention block minus the layer's input) stays
    within the error the two E4M3 roundings allow of the exact product of the
    stored attention output and the bf16 weights: each factor within relative
    2^-4 plus its subnormal step, the activation scaled per row over all heads."""
    cfg = synth.config("tiny")
    w = synth.model_weights(cfg)
    q = OracleModel(cfg, w, "fp8")
    f = OracleModel(cfg, w, "faithful")
    cache = KVCache(cfg, 48)
    bt = np.random.default_rng(3).integers(0, cfg["vocab"] - 1, (2, 16))
    trace = []
    q.forward_block(bt, 0, cache, trace=trace)
    val = {(n, li): v for n, li, v in trace}
    o = val[("o", 0)].reshape(-1, val[("o", 0)].shape[-1])
    x_in = q.embed[bt].reshape(-1, cfg["hidden"])
    got = val[("x1", 0)].reshape(-1, cfg["hidden"]) - x_in
    wo = f.layers[0]["wo"]
    exact = o @ wo.T
    s_row = np.max(np.abs(o), axis=1) / E4M3_MAX
    e_o = 2.0 ** -4 * np.abs(o) + 2.0 ** -10 * s_row[:, None] * 1.0001
    s_w = np.max(np.abs(wo), axis=1) / E4M3_MAX
    e_w = 2.0 ** -4 * np.abs(wo) + 2.0 ** -10 * s_w[:, None] * 1.0001
    bound = e_o @ np.abs(wo).T + np.abs(o) @ e_w.T + e_o @ e_w.T
    assert np.all(np.abs(got - exact) <= bound * (1 + 1e-9) + 1e-9)
    assert np.max(np.abs(got - exact)) > 0
