"""One draft-verify round on the GPU through libspecverify.

`DeviceRound` owns the torch device buffers of a round (inputs already resident
in HBM, outputs, workspaces) and issues the C-ABI calls on one stream. By default
(`fused`) these are sv_prepare_round -> sv_verify_attn_run -> sv_spec_accept, where
the first call does the budget, the packing and the attention work plan in one
launch. Otherwise they are the separate calls sv_alloc_budget -> sv_pack_verify ->
sv_verify_attn -> sv_spec_accept. It only moves data and marshals arguments; all
arithmetic of the round runs in the library's kernels.

The round is self-contained on the device: the budget writes qo_indptr, the packing
turns it and the committed context lengths into the key counts kv_lens = L_i + k_i
that attention reads, and acceptance reads the same qo_indptr. No per-round value
crosses to the host between the calls.
"""
from __future__ import annotations

import copy

import numpy as np
import torch

from . import binding as B
from . import synth


def to_dev(x: np.ndarray, dtype=None, device="cuda"):
    """numpy -> torch device tensor; uint16 arrays are bf16 bit patterns."""
    if x.dtype == np.uint16:
        t = torch.from_numpy(x.view(np.int16).copy()).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(x))
    if dtype is not None:
        t = t.to(dtype)
    return t.to(device)


class DeviceRound:
    """Device-resident inputs and outputs of one round of workload `cfg`.

    budget: "fixed"/"cost" run sv_alloc_budget; "given" takes k_i from the
    generator (no budget step). The target rows handed to acceptance are the
    rows of the kept positions, gathered once after the first budget call (the
    target model would have produced exactly those rows).
    """

    def __init__(self, cfg: synth.RoundConfig, kind: str = "logits", with_attn: bool = True,
                 with_accept: bool = True, fill_unused=0.0, device="cuda", kv_split: int = 0,
                 logits=None, kv=None, fused: bool = True):
        self.cfg = cfg
        self.fused = fused
        self.kind = kind
        self.device = device
        R, b, D = cfg.R, cfg.b, cfg.D
        dt_t = torch.float32 if cfg.dtype == "f32" else torch.bfloat16
        self.dt = dt_t
        self.L = synth.kv_context_lengths(cfg)
        self.lr = logits if logits is not None else (
            synth.make_logits_round(cfg, want_probs=(kind == "probs")) if with_accept or cfg.budget[0] != "given"
            else None)
        # ---- budget inputs
        mode = cfg.budget[0]
        self.mode = mode
        if mode == "given":
            self.k_given = synth.given_depths(cfg)
            self.qo_host = synth.indptr_from_depths(self.k_given)
        else:
            self.conf = to_dev(self.lr["conf"], device=device)
            if mode == "fixed":
                self.bdesc = B.budget_desc(R, b, "fixed", fixed_budget=cfg.budget[1])
            else:
                cost = synth.profiled_cost(R, b)
                self.cost = cost
                self.bdesc = B.budget_desc(R, b, "cost", ratios_pm=synth.PAPER_RATIOS_PM, cost=cost)
        self.keep = torch.empty(R, dtype=torch.int32, device=device)
        self.qo = torch.empty(R + 1, dtype=torch.int32, device=device)
        self.sel = torch.empty(2, dtype=torch.int32, device=device)
        self.scores = torch.empty(R * b, dtype=torch.float32, device=device)
        self.util = torch.empty(B.SV_MAX_RATIOS, dtype=torch.int64, device=device)
        if mode == "given":
            self.qo.copy_(torch.from_numpy(self.qo_host))
        else:
            self.run_budget()
            torch.cuda.synchronize()
            self.qo_host = self.qo.cpu().numpy()
        self.K = int(self.qo_host[-1])
        # ---- packing inputs: the committed context lengths and each request's block
        # (position 0 the certain token, then the drafts)
        self.ctx_lens = to_dev(np.asarray(self.L, np.int32), device=device)
        tok_rng = np.random.default_rng(cfg.seed + 17)
        blk = np.empty((R, b), np.int32)
        blk[:, 0] = tok_rng.integers(0, cfg.V, size=R)
        if self.lr is not None and b > 1:
            blk[:, 1:] = self.lr["draft_tokens"]
        elif b > 1:
            blk[:, 1:] = tok_rng.integers(0, cfg.V, size=(R, b - 1))
        self.block_tokens_host = blk
        self.block_tokens = to_dev(blk, device=device)
        self.pdesc = B.pack_desc(R, b, R * b)
        self.v_tokens = torch.empty(R * b, dtype=torch.int32, device=device)
        self.v_positions = torch.empty(R * b, dtype=torch.int32, device=device)
        self.kv_lens = torch.empty(R, dtype=torch.int32, device=device)
        self.run_pack()
        # ---- attention inputs (cache holds L_i + b tokens; k_i of the block are visible)
        self.with_attn = with_attn
        if with_attn:
            on_device = isinstance(kv, str) and kv == "device"
            if on_device:
                self.kv = synth.make_kv(cfg, self.L, want_cache=False)
            else:
                self.kv = kv if kv is not None else synth.make_kv(cfg, self.L, fill_unused=fill_unused)
            self.q = to_dev(synth.pack_rows(self.kv["q_full"], self.qo_host), device=device)
            if on_device:
                g = torch.Generator(device=device)
                g.manual_seed(cfg.seed)
                shape = (self.kv["num_pages"], cfg.Hkv, cfg.page, cfg.d)
                self.k_cache = torch.randn(shape, generator=g, dtype=dt_t, device=device)
                self.v_cache = torch.randn(shape, generator=g, dtype=dt_t, device=device)
            else:
                self.k_cache = to_dev(self.kv["k_cache"], device=device)
                self.v_cache = to_dev(self.kv["v_cache"], device=device)
            self.page_table = to_dev(self.kv["page_table"], device=device)
            pt = self.kv["page_table"]
            self.adesc = B.attn_desc(R, R * b, b, cfg.Hq, cfg.Hkv, cfg.d, cfg.page, pt.shape[1],
                                     self.kv["num_pages"], int(self.L.max()) + b,
                                     B.SV_F32 if cfg.dtype == "f32" else B.SV_BF16, kv_split=kv_split)
            q_rows = R * b
            self.attn_out = torch.zeros((q_rows, cfg.Hq, cfg.d), dtype=dt_t, device=device)
            self.q_full_rows = torch.zeros((q_rows, cfg.Hq, cfg.d), dtype=dt_t, device=device)
            self.q_full_rows[:self.K] = self.q
            self.q = self.q_full_rows
            self.attn_lse = torch.zeros((q_rows, cfg.Hq), dtype=torch.float32, device=device)
            nws = B.attn_workspace_size(self.adesc)
            self.attn_ws = torch.empty(max(nws, 256), dtype=torch.uint8, device=device)
        # ---- acceptance inputs
        self.with_accept = with_accept
        if with_accept:
            ua, us = synth.acceptance_uniforms(cfg)
            self.ua_host, self.us_host = ua, us
            if kind == "probs":
                tfull, dft, dt_code = self.lr["target_probs_full"], self.lr["draft_probs"], B.SV_F32
            else:
                tfull, dft = self.lr["target_full"], self.lr["draft"]
                dt_code = B.SV_F32 if cfg.dtype == "f32" else B.SV_BF16
            self.target_host = synth.pack_rows(tfull, self.qo_host)
            self.draft_host = dft
            self.target = to_dev(self.target_host, device=device)
            self.draft = to_dev(dft, device=device)
            self.tokens = to_dev(self.lr["draft_tokens"], device=device)
            self.u_accept = to_dev(ua, device=device)
            self.u_sample = to_dev(us, device=device)
            self.xdesc = B.accept_desc(R, b, cfg.V, B.SV_PROBS if kind == "probs" else B.SV_LOGITS, dt_code)
            self.accept_len = torch.empty(R, dtype=torch.int32, device=device)
            self.out_tokens = torch.empty((R, b), dtype=torch.int32, device=device)
            self.flags = torch.empty(R, dtype=torch.int32, device=device)
            self.acc_ws = torch.empty(B.accept_workspace_size(self.xdesc), dtype=torch.uint8, device=device)

    def replica(self) -> "DeviceRound":
        """Another copy of this round: every device buffer cloned (aliases kept), host
        arrays shared. Copies used in turn make every step read its inputs from HBM
        rather than from the last-level cache."""
        r = copy.copy(self)
        seen = {}
        for name, v in vars(self).items():
            if isinstance(v, torch.Tensor):
                if id(v) not in seen:
                    seen[id(v)] = v.clone()
                setattr(r, name, seen[id(v)])
        return r

    def device_bytes(self) -> int:
        """Bytes of the distinct device buffers of this round."""
        seen = {id(v): v for v in vars(self).values() if isinstance(v, torch.Tensor)}
        return int(sum(v.numel() * v.element_size() for v in seen.values()))

    # ---- the calls
    def run_budget(self, stream=None):
        if self.mode == "given":
            return
        B.alloc_budget(self.bdesc, self.conf, self.keep, self.qo, self.sel, self.scores, self.util, stream)

    def run_pack(self, stream=None):
        B.pack_verify(self.pdesc, self.block_tokens, self.ctx_lens, self.qo, self.v_tokens, self.v_positions,
                      self.kv_lens, stream)

    def run_attn(self, stream=None):
        B.verify_attn(self.adesc, self.q, self.k_cache, self.v_cache, self.page_table, self.qo, self.kv_lens,
                      self.attn_out, self.attn_lse, self.attn_ws, stream)

    def run_accept(self, stream=None):
        B.spec_accept(self.xdesc, self.target, self.draft, self.tokens, self.qo, self.u_accept, self.u_sample,
                      self.accept_len, self.out_tokens, self.flags, self.acc_ws, stream)

    def run_prepare(self, stream=None):
        """sv_prepare_round: the budget, the packing and the attention work plan, one launch."""
        B.prepare_round(self.bdesc, self.conf, self.keep, self.qo, self.sel, self.scores, self.util, self.pdesc,
                        self.block_tokens, self.ctx_lens, self.v_tokens, self.v_positions, self.kv_lens,
                        self.adesc if self.with_attn else None, self.attn_ws if self.with_attn else None, stream)

    def run_attn_planned(self, stream=None):
        """sv_verify_attn_run on the plan run_prepare left in the attention workspace."""
        B.verify_attn_run(self.adesc, self.q, self.k_cache, self.v_cache, self.page_table, self.qo, self.kv_lens,
                          self.attn_out, self.attn_lse, self.attn_ws, stream)

    def calls(self):
        """The round's calls in order, as (name, function of stream): with `fused` (and a
        budget stage) sv_prepare_round, then the attention on its plan; otherwise budget,
        packing and the attention with its own plan as separate calls."""
        out = []
        if self.fused and self.mode != "given":
            out.append(("prepare", self.run_prepare))
            if self.with_attn:
                out.append(("attention", self.run_attn_planned))
        else:
            if self.mode != "given":
                out.append(("budget", self.run_budget))
            out.append(("pack", self.run_pack))
            if self.with_attn:
                out.append(("attention", self.run_attn))
        if self.with_accept:
            out.append(("acceptance", self.run_accept))
        return out

    def run(self, stream=None):
        for _, fn in self.calls():
            fn(stream)
