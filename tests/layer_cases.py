"""Helpers for GPU-vs-oracle parity tests: build a synthetic layer, run it
through the C ABI, and compute the oracle's reference from the same seeded
inputs (the oracle never sees a value produced by the GPU path)."""
from __future__ import annotations

import numpy as np
import torch

from oracle import oracle as O
from paper_2504_15299_amd import api
from paper_2504_15299_amd import workloads as wl

DEV = torch.device("cuda:0") if torch.cuda.is_available() else None
FWD_TOL = 2e-2   # per-row max-abs-rel (bf16 operands, fp32 accumulation)


def row_max_abs_rel(got: np.ndarray, ref: np.ndarray) -> np.ndarray:
    den = np.abs(ref).max(axis=1)
    den = np.where(den > 0, den, 1.0)
    return np.abs(got - ref).max(axis=1) / den


def logit_error_bound(x: np.ndarray, Wg: np.ndarray, bias) -> np.ndarray:
    """Bound on |fp32 GPU logit - exact| for the gate kernel's summation
    (256 per-thread fma chains of ceil(d/256) terms, a 6-level shuffle tree,
    a sequential sum over 4 waves and the bias: at most ceil(d/256) + 11
    roundings per term), per token, with one rounding of slack:
    (ceil(d/256) + 12) * 2^-24 * max_e sum_c |x_c Wg_ec| (+ |bias|)."""
    d = x.shape[1]
    mag = np.abs(x.astype(np.float64)) @ np.abs(Wg.astype(np.float64)).T
    if bias is not None:
        mag = mag + np.abs(bias)[None, :]
    return (-(-d // 256) + 12) * 2.0 ** -24 * mag.max(axis=1)


def ambiguous_tokens(logits: np.ndarray, k: int, bound: np.ndarray) -> np.ndarray:
    """Tokens whose k-th and (k+1)-th logits are within 2*bound (their top-k
    set could legitimately differ between fp32 and exact logits)."""
    T, E = logits.shape
    if k >= E:
        return np.zeros(T, bool)
    s = -np.sort(-logits, axis=1)
    return (s[:, k - 1] - s[:, k]) <= 2 * bound


class Layer:
    """A synthetic MoE layer on the GPU plus everything the oracle needs."""

    def __init__(self, spec: wl.LayerSpec, layer: int = 0):
        self.spec = s = spec
        self.x = wl.activations(s, layer)
        self.Wg, self.bias = wl.gate(s, layer)
        self.req = wl.token_requests(s)
        self.W13 = [wl.expert_w13(s, e, layer) for e in range(s.E)]
        self.W2 = [wl.expert_w2(s, e, layer) for e in range(s.E)]
        self.shared = None
        if s.shared_f:
            self.SW13 = wl.shared_w13(s, layer)
            self.SW2 = wl.shared_w2(s, layer)
        # oracle routing from its own binary64 logits
        self.ref_logits = O.gate_logits(self.x, self.Wg, self.bias)
        if s.bits_mode == "hottest_first":
            probe = O.route_from_logits(self.ref_logits, s.k, self.req,
                                        np.full((s.n_requests, s.E), 8, np.uint8), s.b_min, s.b_max)
            counts = np.bincount(probe["topk_idx"].ravel(), minlength=s.E)
            self.table = wl.bit_table(s, layer, expert_counts=counts)
        else:
            self.table = wl.bit_table(s, layer)
        self.ref_route = O.route_from_logits(self.ref_logits, s.k, self.req, self.table,
                                             s.b_min, s.b_max)
        self._codes = None

    # ---- GPU side ----
    def pack(self):
        s = self.spec
        self.w13 = api.MWQ.empty(s.E, 2 * s.f, s.d, s.group, s.b_min, s.b_max, device=DEV)
        self.w2 = api.MWQ.empty(s.E, s.d, s.f, s.group, s.b_min, s.b_max, device=DEV)
        api.pack_mwq(torch.from_numpy(np.stack(self.W13)).to(DEV), self.w13)
        api.pack_mwq(torch.from_numpy(np.stack(self.W2)).to(DEV), self.w2)
        if s.shared_f:
            self.sw13 = api.MWQ.empty(1, 2 * s.shared_f, s.d, s.group, s.b_min, s.b_max, device=DEV)
            self.sw2 = api.MWQ.empty(1, s.d, s.shared_f, s.group, s.b_min, s.b_max, device=DEV)
            api.pack_mwq(torch.from_numpy(self.SW13[None]).to(DEV), self.sw13)
            api.pack_mwq(torch.from_numpy(self.SW2[None]).to(DEV), self.sw2)
            self.shared = (self.sw13, self.sw2, s.shared_bits)
        return self

    def x_dev(self):
        t = torch.from_numpy(self.x).to(DEV)
        return t.to(torch.bfloat16) if self.spec.x_dtype == "bf16" else t

    def route(self):
        s = self.spec
        self.xt = self.x_dev()
        bias = None if self.bias is None else torch.from_numpy(self.bias).to(DEV)
        self.r = api.route(self.xt, torch.from_numpy(self.Wg).to(DEV), bias, s.k,
                           torch.from_numpy(self.req).to(DEV),
                           torch.from_numpy(self.table).to(DEV), s.b_min, s.b_max)
        return self.r

    def forward(self):
        out = api.moe_forward(self.xt, self.w13, self.w2, self.r, self.spec.k, shared=self.shared)
        torch.cuda.synchronize()
        return out.float().cpu().numpy()

    # ---- oracle side ----
    def codes(self):
        if self._codes is None:
            s = self.spec
            c13 = [O.mwq_quantize(w, s.group, s.b_min, s.b_max) for w in self.W13]
            c2 = [O.mwq_quantize(w, s.group, s.b_min, s.b_max) for w in self.W2]
            sh = None
            if s.shared_f:
                sh = (O.mwq_quantize(self.SW13, s.group, s.b_min, s.b_max),
                      O.mwq_quantize(self.SW2, s.group, s.b_min, s.b_max), s.shared_bits)
            self._codes = (c13, c2, sh)
        return self._codes

    def reference(self, tokens=None):
        c13, c2, sh = self.codes()
        return O.moe_layer(self.x, self.ref_route, c13, c2, tokens=tokens, shared=sh)
