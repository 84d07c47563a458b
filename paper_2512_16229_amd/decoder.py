"""Host driver of the LoPA decode loop over the four C-ABI calls.

One iteration (Alg. 1) = build_branches -> verify_forward (all k+1 branches in
one pass) -> branch_confidence_select -> commit_kv, all enqueued on one
stream; the only host read per iteration is the winner's unfilled count (a
4-byte copy) that ends the block. Prompt encoding is block-causal in blocks of
L through the same verify forward with one branch, committed block by block.
"""
from __future__ import annotations

import torch

from . import (KV, MAX_BLOCK, METRIC_MEAN, WINDOW_MAX_BLOCKS, Model,
               lopa_branch_confidence_select, lopa_branch_confidence_select_metric,
               lopa_build_branches, lopa_build_branches_window, lopa_commit_kv,
               lopa_verify_forward, lopa_window_commit, lopa_window_init, lopa_window_update,
               window_read, window_state)


class Decoder:
    """metric / window / eta choose the branch confidence of the selection
    (METRIC_MEAN: Eq. 2; the alternatives of lopa_branch_confidence_select_metric)."""

    def __init__(self, model: Model, kv: KV, L: int, k: int, tau: float, metric: int = METRIC_MEAN,
                 window: int = 4, eta: float = 0.25):
        self.model, self.kv, self.L, self.k, self.tau = model, kv, L, k, float(tau)
        self.metric, self.window, self.eta = int(metric), int(window), float(eta)
        self.mask_id = model.cfg["mask_id"]
        nb = k + 1
        dev = "cuda"
        i32 = dict(dtype=torch.int32, device=dev)
        f32 = dict(dtype=torch.float32, device=dev)
        self.tokens = torch.full((L,), self.mask_id, **i32)
        self.conf = torch.zeros(L, **f32)
        self.pred = torch.zeros(L, **i32)
        self.branch_tokens = torch.empty(nb * L, **i32)
        self.fill_pos = torch.empty(nb, **i32)
        self.valid = torch.empty(nb, dtype=torch.uint8, device=dev)
        self.n_valid = torch.empty(1, **i32)
        self.conf_b = torch.empty(nb * L, **f32)
        self.pred_b = torch.empty(nb * L, **i32)
        self.scores = torch.empty(nb, **f32)
        self.winner = torch.zeros(1, **i32)
        self.next_tokens = torch.empty(L, **i32)
        self.next_conf = torch.empty(L, **f32)
        self.next_pred = torch.empty(L, **i32)
        self.next_unfilled = torch.empty(1, **i32)
        self.append_offset = torch.empty(1, **i32)
        self.zero = torch.zeros(1, **i32)
        self.forwards = 0

    # -------------------------------------------------------------- prompt
    def prefill(self, prompt: torch.Tensor) -> int:
        """Encode the prompt block-causally; returns the new prefix length."""
        prompt = prompt.to(device="cuda", dtype=torch.int32).contiguous()
        pos = 0
        conf = torch.empty(self.L, dtype=torch.float32, device="cuda")
        pred = torch.empty(self.L, dtype=torch.int32, device="cuda")
        while pos < prompt.numel():
            blk = prompt[pos:pos + self.L].contiguous()
            n = blk.numel()
            lopa_verify_forward(self.model, self.kv, pos, blk, 1, n, conf[:n], pred[:n])
            lopa_commit_kv(self.kv, self.zero, pos, n, self.append_offset)
            pos += n
        return pos

    # --------------------------------------------------------------- block
    def init_block(self, P: int):
        """All-mask block and its first forward (conf / pred of the state)."""
        self.tokens.fill_(self.mask_id)
        lopa_verify_forward(self.model, self.kv, P, self.tokens, 1, self.L, self.conf, self.pred)
        self.forwards += 1

    def step(self, P: int):
        """One LoPA iteration; the next state replaces the current one."""
        L, nb = self.L, self.k + 1
        lopa_build_branches(self.tokens, self.conf, self.pred, L, self.mask_id, self.tau, self.k,
                            self.branch_tokens, self.fill_pos, self.valid, self.n_valid)
        lopa_verify_forward(self.model, self.kv, P, self.branch_tokens, nb, L, self.conf_b,
                            self.pred_b)
        outs = (self.scores, self.winner, self.next_tokens, self.next_conf, self.next_pred,
                self.next_unfilled)
        if self.metric == METRIC_MEAN:
            lopa_branch_confidence_select(self.branch_tokens, self.conf_b, self.pred_b, self.valid,
                                          nb, L, self.mask_id, *outs)
        else:
            lopa_branch_confidence_select_metric(self.branch_tokens, self.conf_b, self.pred_b,
                                                 self.valid, nb, L, self.mask_id, self.metric,
                                                 self.window, self.eta, *outs)
        lopa_commit_kv(self.kv, self.winner, P, L, self.append_offset)
        self.tokens, self.next_tokens = self.next_tokens, self.tokens
        self.conf, self.next_conf = self.next_conf, self.conf
        self.pred, self.next_pred = self.next_pred, self.pred
        self.forwards += 1

    def decode_block(self, P: int, trace=None) -> int:
        """Run iterations until the winner has no unfilled position; returns the count.
        trace: a list that receives each iteration's snapshot and the state
        (tokens, conf, pred) the iteration started from (host copies)."""
        self.init_block(P)
        it = 0
        while True:
            state = (self.tokens.cpu(), self.conf.cpu(), self.pred.cpu()) if trace is not None else None
            self.step(P)
            it += 1
            if trace is not None:
                trace.append(dict(self.snapshot(), state=state))
            if int(self.next_unfilled.item()) == 0:
                return it
            if it > self.L:
                raise RuntimeError("block did not complete in L iterations")

    def snapshot(self) -> dict:
        nb, L = self.k + 1, self.L
        return dict(branch_tokens=self.branch_tokens.view(nb, L).cpu(),
                    fill_pos=self.fill_pos.cpu(), valid=self.valid.cpu(),
                    n_valid=int(self.n_valid.item()), conf=self.conf_b.view(nb, L).cpu(),
                    pred=self.pred_b.view(nb, L).cpu(), scores=self.scores.cpu(),
                    winner=int(self.winner.item()), tokens=self.tokens.cpu(),
                    append_offset=int(self.append_offset.item()))

    def decode(self, prompt: torch.Tensor, gen_len: int) -> dict:
        P = self.prefill(prompt)
        out, iters = [], 0
        self.forwards = 0
        for _ in range(gen_len // self.L):
            iters += self.decode_block(P)
            out.append(self.tokens.clone())
            P += self.L
        toks = torch.cat(out) if out else torch.zeros(0, dtype=torch.int32, device="cuda")
        return dict(tokens=toks, iterations=iters, forwards=self.forwards,
                    tpf=(toks.numel() / self.forwards) if self.forwards else 0.0)


class WindowDecoder:
    """LoPA over a window of up to w_max active blocks (Sec. 3.3, integration
    with D2F: the active blocks form one window for branch exploration, full
    attention inside it). The gates run on the device, in the library's
    readings (lopa_window_init / lopa_window_update / lopa_window_commit and
    the lopa_window state): blocks join while the last one is at least tau_add
    filled, become fully activated (eligible for the Eq. 1 fallback and the
    lookahead fills) once the block before is fully activated and at least
    tau_act filled, and leave with their K/V committed once they have no
    unfilled position. The host reads the window's header (a few words) once
    per iteration: the next iteration's launch shapes depend on it."""

    def __init__(self, model: Model, kv: KV, L: int, k: int, tau: float, tau_add: float,
                 tau_act: float, w_max: int, metric: int = METRIC_MEAN, window: int = 4,
                 eta: float = 0.25, block_causal: bool = False):
        if w_max * L > MAX_BLOCK or w_max > WINDOW_MAX_BLOCKS:
            raise ValueError(f"a window of {w_max} blocks of {L} exceeds the library's "
                             f"{WINDOW_MAX_BLOCKS} blocks / {MAX_BLOCK} positions")
        self.model, self.kv, self.L, self.k = model, kv, L, k
        # block_causal: the window's blocks attend block-causally (Sec. 3.4,
        # the Ascend system's mask) instead of with full attention
        self.block_causal = bool(block_causal)
        self.tau, self.tau_add, self.tau_act, self.w_max = float(tau), float(tau_add), float(tau_act), w_max
        self.metric, self.window, self.eta = int(metric), int(window), float(eta)
        self.mask_id = model.cfg["mask_id"]
        W, nb, dev = w_max * L, k + 1, "cuda"
        i32 = dict(dtype=torch.int32, device=dev)
        f32 = dict(dtype=torch.float32, device=dev)
        self.tokens = torch.empty(W, **i32)
        self.conf = torch.zeros(W, **f32)
        self.pred = torch.empty(W, **i32)
        self.bt = torch.empty(nb * W, **i32)
        self.fill_pos = torch.empty(nb, **i32)
        self.valid = torch.empty(nb, dtype=torch.uint8, device=dev)
        self.n_valid = torch.empty(1, **i32)
        self.conf_b = torch.empty(nb * W, **f32)
        self.pred_b = torch.empty(nb * W, **i32)
        self.scores = torch.empty(nb, **f32)
        self.winner = torch.zeros(1, **i32)
        self.next_tokens = torch.empty(W, **i32)
        self.next_conf = torch.empty(W, **f32)
        self.next_pred = torch.empty(W, **i32)
        self.next_unfilled = torch.empty(1, **i32)
        self.win = window_state(dev)
        self.forwards = self.iterations = 0

    def decode(self, prompt: torch.Tensor, gen_len: int, trace=None) -> dict:
        L, k, nb, mask = self.L, self.k, self.k + 1, self.mask_id
        self.kv.set_block_causal(L if self.block_causal else 0)
        P = Decoder(self.model, self.kv, L, 0, self.tau).prefill(prompt)
        n_blocks = gen_len // L
        out = torch.empty(max(1, n_blocks * L), dtype=torch.int32, device="cuda")
        lopa_window_init(self.win, self.tokens, self.conf, self.pred, L, self.w_max, n_blocks, P,
                         mask, self.tau_add, self.tau_act)
        while True:
            h = window_read(self.win)
            if h.error:
                raise RuntimeError("window commit found invalid inputs")
            if h.done:
                break
            P, Lw, n_el = h.prefix_len, h.blocks * L, h.eligible
            if h.need_initial:
                # the new first block's initial forward (the block alone)
                lopa_verify_forward(self.model, self.kv, P, self.tokens[:L], 1, L, self.conf[:L],
                                    self.pred[:L])
                self.forwards += 1
            state = ((self.tokens[:Lw].cpu(), self.conf[:Lw].cpu(), self.pred[:Lw].cpu())
                     if trace is not None else None)
            lopa_build_branches_window(self.tokens[:Lw], self.conf[:Lw], self.pred[:Lw], Lw, n_el,
                                       mask, self.tau, k, self.bt[:nb * Lw], self.fill_pos,
                                       self.valid, self.n_valid)
            lopa_verify_forward(self.model, self.kv, P, self.bt[:nb * Lw], nb, Lw,
                                self.conf_b[:nb * Lw], self.pred_b[:nb * Lw])
            outs = (self.scores, self.winner, self.next_tokens[:Lw], self.next_conf[:Lw],
                    self.next_pred[:Lw], self.next_unfilled)
            if self.metric == METRIC_MEAN:
                lopa_branch_confidence_select(self.bt[:nb * Lw], self.conf_b[:nb * Lw],
                                              self.pred_b[:nb * Lw], self.valid, nb, Lw, mask, *outs)
            else:
                lopa_branch_confidence_select_metric(self.bt[:nb * Lw], self.conf_b[:nb * Lw],
                                                     self.pred_b[:nb * Lw], self.valid, nb, Lw,
                                                     mask, self.metric, self.window, self.eta, *outs)
            self.tokens, self.next_tokens = self.next_tokens, self.tokens
            self.conf, self.next_conf = self.next_conf, self.conf
            self.pred, self.next_pred = self.next_pred, self.pred
            self.forwards += 1
            self.iterations += 1
            selected = self.tokens[:Lw].cpu() if trace is not None else None
            lopa_window_update(self.win, self.tokens, self.conf, self.pred, out)
            lopa_window_commit(self.kv, self.winner, self.win)
            if trace is not None:
                trace.append(dict(prefix_len=P, n_eligible=n_el, window_len=Lw,
                                  initial_forward=bool(h.need_initial),
                                  winner=int(self.winner.item()), tokens=selected,
                                  committed_blocks=window_read(self.win).last_commit,
                                  scores=self.scores.cpu(), state=state,
                                  branch_tokens=self.bt[:nb * Lw].view(nb, Lw).cpu(),
                                  valid=self.valid.cpu(), n_valid=int(self.n_valid.item()),
                                  conf=self.conf_b[:nb * Lw].view(nb, Lw).cpu(),
                                  pred=self.pred_b[:nb * Lw].view(nb, Lw).cpu()))
            if self.iterations > 2 * gen_len + 2 * n_blocks:
                raise RuntimeError("window decode did not converge")
        toks = out[:n_blocks * L].cpu() if n_blocks else torch.zeros(0, dtype=torch.int32)
        return dict(tokens=toks, iterations=self.iterations, forwards=self.forwards,
                    tpf=(toks.numel() / self.forwards) if self.forwards else 0.0)
