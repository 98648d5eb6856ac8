"""Workload rig: a libmoesplit context filled with seeded synthetic weights.

Shared by the GPU tests, the benchmark and the smoke check.  It allocates the
device pool with torch (plumbing only), hands the synthetic weights of
``synth`` to the library through the C ABI binding, configures per-layer
budgets and split ratios, and loads top segments.  It keeps the exact fp32
values of every tensor so that tests can give the oracle the same inputs.
"""
from __future__ import annotations

from concurrent.futures import ThreadPoolExecutor

import numpy as np
import torch

import synth
from paper_2509_08342_amd import moesplit as ms


def bf16_tensor(raw: np.ndarray, device="cuda") -> torch.Tensor:
    """bf16 bit patterns (uint16 numpy) -> torch.bfloat16 tensor on device."""
    return torch.from_numpy(raw.view(np.int16).copy()).view(torch.bfloat16).to(device)


def to_device(raw: np.ndarray, dtype: str, device="cuda") -> torch.Tensor:
    if dtype == "bf16":
        return bf16_tensor(raw, device)
    return torch.from_numpy(np.ascontiguousarray(raw, np.float32)).to(device)


class SplitRig:
    """One context for ``shape`` with ``n_sets`` distinct expert weight sets.

    Layer l uses weight set l % n_sets (ms_alias_expert for the others), so a
    deep stack does not need a distinct host blob per layer.  Routers are
    distinct per layer.  ``keep_f32`` keeps the exact fp32 copies for the
    oracle."""

    def __init__(self, shape: synth.ModelShape, *, seed=0, max_tokens=1, n_sets=None,
                 n_buffer_slots=0, budget_bytes=0, keep_f32=True, threads=8, ffn_splits=0):
        self.shape = shape
        self.seed = seed
        self.max_tokens = max_tokens
        L = shape.n_layers
        self.n_sets = L if n_sets is None else max(1, min(n_sets, L))
        self.desc = ms.model_desc(shape, max_tokens, n_buffer_slots, ffn_splits)
        self.sizes = ms.ms_query_sizes(self.desc)
        self.pool_bytes = int(self.sizes.fixed_pool_bytes) + int(budget_bytes)
        self.pool = torch.empty(self.pool_bytes, dtype=torch.uint8, device="cuda")
        self.ctx = ms.ms_create(self.desc, self.pool, self.pool_bytes, 0)
        self.keep_f32 = keep_f32
        self.routers = []        # exact fp32 [d][E] per layer
        self.biases = []         # fp32 [E] or None per layer
        self.experts = {}        # weight set -> list of E (w_gate, w_up, w_down) fp32
        self.shared = []         # per layer list of fp32 triples
        for l in range(L):
            raw, f32 = synth.router(shape, seed, l)
            bias = synth.router_bias(shape, seed, l)
            ms.ms_set_router(self.ctx, l, raw, bias)
            self.routers.append(f32)
            self.biases.append(bias)

        bits = getattr(shape, "expert_bits", 0)

        def gen(args):
            s, e = args
            if bits:
                return s, e, synth.quant_expert(shape, seed, s, e, bits)
            return s, e, synth.expert(shape, seed, s, e)

        jobs = [(s, e) for s in range(self.n_sets) for e in range(shape.n_experts)]
        with ThreadPoolExecutor(threads) as pool:
            for s, e, ex in pool.map(gen, jobs):
                if bits:
                    # b-bit experts: the oracle gets the same codes and metadata
                    ms.ms_set_expert_q(self.ctx, s, e, ex.codes, ex.meta)
                    if keep_f32:
                        self.experts.setdefault(s, [None] * shape.n_experts)[e] = ex
                else:
                    ms.ms_set_expert(self.ctx, s, e, *ex.raw)
                    if keep_f32:
                        self.experts.setdefault(s, [None] * shape.n_experts)[e] = ex.f32
                del ex
        for l in range(self.n_sets, L):
            for e in range(shape.n_experts):
                ms.ms_alias_expert(self.ctx, l, e, l % self.n_sets, e)
        # shared experts: layer l uses the shared weights of set l % n_sets
        sets_sh = []
        for s_ in range(self.n_sets if shape.n_shared else 0):
            sets_sh.append([synth.expert(shape, seed, s_, i, shared=True) for i in range(shape.n_shared)])
        for l in range(L):
            sh = []
            for i in range(shape.n_shared):
                ex = sets_sh[l % self.n_sets][i]
                ms.ms_set_shared_expert(self.ctx, l, i, *ex.raw)
                sh.append(ex.f32 if keep_f32 else None)
            self.shared.append(sh)
        self.budget_bytes = int(budget_bytes)

    # ------------------------------------------------------------------
    def layer_experts(self, layer):
        return self.experts[layer % self.n_sets]

    def configure(self, budgets, r):
        return ms.ms_configure(self.ctx, np.asarray(budgets, np.uint64), np.asarray(r, np.float32))

    def configure_uniform(self, r, total_budget=None):
        L = self.shape.n_layers
        total = self.budget_bytes if total_budget is None else total_budget
        return self.configure([total // L] * L, [r] * L)

    def load_tops(self, layer, experts):
        for e in experts:
            ms.ms_load_top(self.ctx, layer, int(e))

    def hidden(self, T, tag=0):
        raw, f32 = synth.hidden(self.shape, self.seed, T, tag)
        return to_device(raw, self.shape.dtype), f32

    def outputs(self, T):
        d, K = self.shape.d_model, self.shape.top_k
        y = torch.empty(max(T, 1), d, dtype=torch.float32, device="cuda")
        idx = torch.empty(max(T, 1), K, dtype=torch.int32, device="cuda")
        w = torch.empty(max(T, 1), K, dtype=torch.float32, device="cuda")
        return y, idx, w

    def forward(self, layer, h, T, y, idx, w, flags=0, stream=None):
        if stream is None:
            stream = torch.cuda.current_stream()
        ms.ms_forward(self.ctx, layer, h, T, y, idx, w, flags, stream)

    def close(self):
        if self.ctx is not None:
            ms.ms_sync(self.ctx)
            ms.ms_destroy(self.ctx)
            self.ctx = None
        self.pool = None

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()


def top_bytes(rig: SplitRig, r: float) -> int:
    """Bytes of one top segment at split ratio r."""
    return ms.ms_split_plan(rig.desc, 0, r)[1]
