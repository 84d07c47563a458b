"""Python binding of liblopa, the MI355X (gfx950) LoPA branch-verification step.

Argument marshalling only: every step of the method runs in the HIP kernels
behind the C ABI declared in include/lopa.h. PyTorch supplies device memory and
the stream. The functions keep the C names:

    lopa_build_branches            Eq. 1 + top-k lookahead branches (Alg. 1 steps 1-2)
    lopa_verify_forward            one batched forward of all branches (Alg. 1 step 3)
    lopa_branch_confidence_select  Eq. 2 scores, argmax, next state (Sec. 3.2 logit reuse)
    lopa_commit_kv                 winner K/V -> static cache (Sec. 3.4)

Importing this module loads liblopa.so built in-tree by build.py (or
__graft_entry__.build()); there is no fallback: a missing library raises.
"""
from __future__ import annotations

import ctypes as C

import torch

from ._abi import (EXPORTS, LIB_PATH, LOPA_ECAPACITY, LOPA_EHIP, LOPA_EINVAL, LOPA_ENOMEM,  # noqa: F401
                   LOPA_ESHAPE, LOPA_OK, MAX_BLOCK, MAX_ROWS, METRIC_LOWEST_SEGMENT, METRIC_MEAN,
                   METRIC_WINDOW_MIN, PRECISIONS, PROF_KINDS, WINDOW_MAX_BLOCKS, LopaError, lib,
                   lopa_layer_weights, lopa_model_cfg, lopa_weight_ptrs, lopa_window)


def _check(status: int):
    if status != LOPA_OK:
        raise LopaError(status, lib.lopa_last_error().decode())


def _ptr(t, dtype=None, name="tensor"):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name}: expected a torch tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name}: must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name}: must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name}: expected {dtype}, got {t.dtype}")
    return C.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return C.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


# ------------------------------------------------------------------ handles
class Model:
    """Repacked model weights on the device (lopa_model)."""

    def __init__(self, cfg: dict, weights: dict, stream=None, precision: str = "bf16"):
        """precision: "bf16", or "fp8_mlp" (gate / up / down in W8A8 E4M3 with
        per-channel weight and per-row activation scales)."""
        if precision not in PRECISIONS:
            raise ValueError(f"precision {precision!r} not in {sorted(PRECISIONS)}")
        c = lopa_model_cfg(cfg["layers"], cfg["hidden"], cfg["heads"], cfg["kv_heads"],
                           cfg["head_dim"], cfg["ffn"], cfg["vocab"], cfg["mask_id"],
                           cfg["rms_eps"], cfg["rope_theta"], 1 if cfg["qkv_bias"] else 0)
        bf = torch.bfloat16
        n = cfg["layers"]
        arr = (lopa_layer_weights * n)()
        for i, lw in enumerate(weights["layers"]):
            f = {}
            for key in ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down", "ln1", "ln2"):
                f[key] = _ptr(lw[key], bf, key)
            for key in ("bq", "bk", "bv"):
                f[key] = _ptr(lw[key], bf, key) if cfg["qkv_bias"] else None
            arr[i] = lopa_layer_weights(**f)
        w = lopa_weight_ptrs(_ptr(weights["embed"], bf, "embed"), arr,
                             _ptr(weights["final_norm"], bf, "final_norm"),
                             _ptr(weights["lm_head"], bf, "lm_head"))
        h = C.c_void_p()
        _check(lib.lopa_model_create_ex(C.byref(c), C.byref(w), PRECISIONS[precision],
                                        _stream(stream), C.byref(h)))
        self.handle, self.cfg, self.precision = h, dict(cfg), precision

    def close(self):
        if getattr(self, "handle", None) and lib is not None:
            lib.lopa_model_destroy(self.handle)
            self.handle = None

    def __del__(self):
        self.close()


class KV:
    """Static KV cache + per-branch staging + verify workspace (lopa_kv)."""

    def __init__(self, model: Model, max_len: int, max_branches: int, max_block: int):
        h = C.c_void_p()
        _check(lib.lopa_kv_create(model.handle, max_len, max_branches, max_block, C.byref(h)))
        self.handle, self.model = h, model
        self.max_len, self.max_branches, self.max_block = max_len, max_branches, max_block

    def read(self, layer: int, start: int, length: int, stream=None):
        c = self.model.cfg
        shp = (c["kv_heads"], length, c["head_dim"])
        k = torch.empty(shp, dtype=torch.bfloat16, device="cuda")
        v = torch.empty_like(k)
        _check(lib.lopa_kv_read(self.handle, layer, start, length, _ptr(k), _ptr(v), _stream(stream)))
        return k, v

    def write(self, layer: int, start: int, k: torch.Tensor, v: torch.Tensor, stream=None):
        _check(lib.lopa_kv_write(self.handle, layer, start, k.shape[1], _ptr(k, torch.bfloat16),
                                 _ptr(v, torch.bfloat16), _stream(stream)))

    def read_staging(self, branch: int, layer: int, L: int, stream=None):
        c = self.model.cfg
        k = torch.empty((c["kv_heads"], L, c["head_dim"]), dtype=torch.bfloat16, device="cuda")
        v = torch.empty_like(k)
        _check(lib.lopa_kv_read_staging(self.handle, branch, layer, _ptr(k), _ptr(v), _stream(stream)))
        return k, v

    def set_block_causal(self, sub_block: int):
        """0: full attention inside the block; c > 0 (multiple of 16): rows of
        sub-block b see the prefix and sub-blocks 0..b of their branch."""
        _check(lib.lopa_kv_set_block_causal(self.handle, sub_block))

    def profile(self, kinds=()):
        """Time launches of the given kinds (names from PROF_KINDS) with HIP events."""
        mask = 0
        for kd in kinds:
            mask |= 1 << PROF_KINDS.index(kd)
        _check(lib.lopa_kv_profile(self.handle, mask))

    def profile_read(self) -> dict:
        """{kind: (total_ms, launches)} since the last read."""
        n = len(PROF_KINDS)
        ms = (C.c_double * n)()
        cnt = (C.c_int64 * n)()
        _check(lib.lopa_kv_profile_read(self.handle, ms, cnt))
        return {PROF_KINDS[i]: (ms[i], cnt[i]) for i in range(n)}

    def close(self):
        if getattr(self, "handle", None) and lib is not None:
            lib.lopa_kv_destroy(self.handle)
            self.handle = None

    def __del__(self):
        self.close()


# ------------------------------------------------------------- entry points
I32, F32, U8 = torch.int32, torch.float32, torch.uint8


def lopa_build_branches(tokens, conf, pred, L, mask_id, tau, k, branch_tokens, fill_pos, valid,
                        n_valid, stream=None):
    _check(lib.lopa_build_branches(_ptr(tokens, I32, "tokens"), _ptr(conf, F32, "conf"),
                                   _ptr(pred, I32, "pred"), L, mask_id, float(tau), k,
                                   _ptr(branch_tokens, I32, "branch_tokens"),
                                   _ptr(fill_pos, I32, "fill_pos"), _ptr(valid, U8, "valid"),
                                   _ptr(n_valid, I32, "n_valid"), _stream(stream)))


def lopa_build_branches_window(tokens, conf, pred, L, n_eligible, mask_id, tau, k, branch_tokens,
                               fill_pos, valid, n_valid, stream=None):
    _check(lib.lopa_build_branches_window(_ptr(tokens, I32, "tokens"), _ptr(conf, F32, "conf"),
                                          _ptr(pred, I32, "pred"), L, n_eligible, mask_id,
                                          float(tau), k, _ptr(branch_tokens, I32, "branch_tokens"),
                                          _ptr(fill_pos, I32, "fill_pos"), _ptr(valid, U8, "valid"),
                                          _ptr(n_valid, I32, "n_valid"), _stream(stream)))


def lopa_verify_forward(model: Model, kv: KV, prefix_len, branch_tokens, n_branches, L, conf, pred,
                        stream=None):
    _check(lib.lopa_verify_forward(model.handle, kv.handle, prefix_len,
                                   _ptr(branch_tokens, I32, "branch_tokens"), n_branches, L,
                                   _ptr(conf, F32, "conf"), _ptr(pred, I32, "pred"),
                                   _stream(stream)))


def lopa_verify_forward_noalloc(model: Model, kv: KV, prefix_len, branch_tokens, n_branches, L,
                                conf, pred, stream=None):
    _check(lib.lopa_verify_forward_noalloc(model.handle, kv.handle, prefix_len,
                                           _ptr(branch_tokens, I32, "branch_tokens"), n_branches,
                                           L, _ptr(conf, F32, "conf"), _ptr(pred, I32, "pred"),
                                           _stream(stream)))


def lopa_branch_confidence_select(branch_tokens, conf, pred, valid, n_branches, L, mask_id, scores,
                                  winner, next_tokens, next_conf, next_pred, next_unfilled,
                                  stream=None):
    _check(lib.lopa_branch_confidence_select(
        _ptr(branch_tokens, I32, "branch_tokens"), _ptr(conf, F32, "conf"), _ptr(pred, I32, "pred"),
        _ptr(valid, U8, "valid"), n_branches, L, mask_id, _ptr(scores, F32, "scores"),
        _ptr(winner, I32, "winner"), _ptr(next_tokens, I32, "next_tokens"),
        _ptr(next_conf, F32, "next_conf"), _ptr(next_pred, I32, "next_pred"),
        _ptr(next_unfilled, I32, "next_unfilled"), _stream(stream)))


def lopa_branch_confidence_select_metric(branch_tokens, conf, pred, valid, n_branches, L, mask_id,
                                         metric, window, eta, scores, winner, next_tokens,
                                         next_conf, next_pred, next_unfilled, stream=None):
    _check(lib.lopa_branch_confidence_select_metric(
        _ptr(branch_tokens, I32, "branch_tokens"), _ptr(conf, F32, "conf"), _ptr(pred, I32, "pred"),
        _ptr(valid, U8, "valid"), n_branches, L, mask_id, metric, window, eta,
        _ptr(scores, F32, "scores"), _ptr(winner, I32, "winner"),
        _ptr(next_tokens, I32, "next_tokens"), _ptr(next_conf, F32, "next_conf"),
        _ptr(next_pred, I32, "next_pred"), _ptr(next_unfilled, I32, "next_unfilled"),
        _stream(stream)))


def lopa_debug_hidden(model: Model, kv: KV, prefix_len, branch_tokens, n_branches, L, n_layers,
                      x_out, stream=None):
    _check(lib.lopa_debug_hidden(model.handle, kv.handle, prefix_len,
                                 _ptr(branch_tokens, I32, "branch_tokens"), n_branches, L, n_layers,
                                 _ptr(x_out, F32, "x_out"), _stream(stream)))


def lopa_commit_kv(kv: KV, winner, prefix_len, L, append_offset, stream=None):
    _check(lib.lopa_commit_kv(kv.handle, _ptr(winner, I32, "winner"), prefix_len, L,
                              _ptr(append_offset, I32, "append_offset"), _stream(stream)))


def lopa_commit_kv_rows(kv: KV, winner, prefix_len, L, n_rows, append_offset, stream=None):
    _check(lib.lopa_commit_kv_rows(kv.handle, _ptr(winner, I32, "winner"), prefix_len, L, n_rows,
                                   _ptr(append_offset, I32, "append_offset"), _stream(stream)))


# ---------------------------------------------------- multi-block window
WINDOW_WORDS = C.sizeof(lopa_window) // 4  # int32 words of the device window state


def window_state(device="cuda") -> torch.Tensor:
    """Device memory for one lopa_window (int32 words)."""
    return torch.zeros(WINDOW_WORDS, dtype=torch.int32, device=device)


def window_read(win: torch.Tensor) -> lopa_window:
    """The window state copied to the host (a synchronising read)."""
    host = win.cpu().numpy()
    return lopa_window.from_buffer_copy(host.tobytes())


def lopa_window_init(win, tokens, conf, pred, L, w_max, n_blocks, prefix_len, mask_id, tau_add,
                     tau_act, stream=None):
    _check(lib.lopa_window_init(_ptr(win, I32, "win"), _ptr(tokens, I32, "tokens"),
                                _ptr(conf, F32, "conf"), _ptr(pred, I32, "pred"), L, w_max,
                                n_blocks, prefix_len, mask_id, float(tau_add), float(tau_act),
                                _stream(stream)))


def lopa_window_update(win, tokens, conf, pred, out_tokens, stream=None):
    _check(lib.lopa_window_update(_ptr(win, I32, "win"), _ptr(tokens, I32, "tokens"),
                                  _ptr(conf, F32, "conf"), _ptr(pred, I32, "pred"),
                                  _ptr(out_tokens, I32, "out_tokens"), _stream(stream)))


def lopa_window_commit(kv: KV, winner, win, stream=None):
    _check(lib.lopa_window_commit(kv.handle, _ptr(winner, I32, "winner"), _ptr(win, I32, "win"),
                                  _stream(stream)))


from .decoder import Decoder, WindowDecoder  # noqa: E402,F401
