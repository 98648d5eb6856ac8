"""Stacks of split-expert MoE layers on libmoesplit: the harness of the
multi-layer workloads (Mixtral-shaped 32-layer decode, DeepSeek-V2-Lite-
shaped 26-layer and Qwen3-30B-A3B-shaped 48-layer prefill + decode).

Each layer's input is the previous layer's output through the glue
h_{i+1} = RMSNorm(h_i + y_i) (ms_residual_norm).  Layer i's forward predicts
layer i+1 from h_i with layer i+1's router and prefetches it (Sec. 3.2); the
first layer of the next step is predicted from the last layer's input h_{L-1}
of this step (the last layer's intermediate activation, Sec. 3.2).  The cache of each layer holds the top segments of the experts
selected most often in a warm-up (ties to the lower index) until a cache
configurator chooses otherwise.  Every step of the layer runs in the
library's kernels; this module only sequences calls and moves test data.
"""
from __future__ import annotations

import numpy as np
import torch

import synth
from paper_2509_08342_amd import moesplit as ms
from workload import SplitRig, to_device, top_bytes


class Stack:
    def __init__(self, shape: synth.ModelShape, *, seed=0, n_sets=2, max_tokens=1, budget_total=0,
                 n_buffer_slots=0, keep_f32=True, threads=16):
        self.shape = shape
        self.rig = SplitRig(shape, seed=seed, max_tokens=max_tokens, n_sets=n_sets, n_buffer_slots=n_buffer_slots,
                            budget_bytes=budget_total, keep_f32=keep_f32, threads=threads)
        self.ctx = self.rig.ctx
        self.L = shape.n_layers
        dt = torch.bfloat16 if shape.dtype == "bf16" else torch.float32
        d = shape.d_model
        self.h = [torch.empty(max_tokens, d, dtype=dt, device="cuda") for _ in range(2)]
        self.y, self.idx, self.w = self.rig.outputs(max_tokens)
        self.slots = None

    # ---------------------------------------------------------- cache setup
    def configure(self, r, budget_total, budgets=None):
        """Per-layer split ratios r (scalar or list) and budgets (uniform
        split of budget_total unless given); returns the cache slots C_i."""
        L = self.L
        rs = [float(r)] * L if np.isscalar(r) else [float(x) for x in r]
        bs = [int(budget_total) // L] * L if budgets is None else [int(b) for b in budgets]
        self.slots = self.rig.configure(bs, rs)
        return self.slots

    def load_most_selected(self, counts):
        """Per layer, cache the tops of the C_i experts with the largest
        selection counts (ties to the lower index)."""
        for l in range(self.L):
            order = sorted(range(self.shape.n_experts), key=lambda e: (-int(counts[l][e]), e))
            self.rig.load_tops(l, order[:int(self.slots[l])])
        ms.ms_sync(self.ctx)

    # -------------------------------------------------------------- running
    def step(self, x, T, flags=ms.MS_FWD_PREDICT_NEXT, capture=(), counts=None, stream=None):
        """One pass of T tokens through every layer.  x: [T][d] device
        tensor in the model dtype (not modified).  capture: layers whose
        (input, y, idx, w) are copied to the host.  counts: [L][E] array of
        selection counts to accumulate.  Returns (final hidden state tensor,
        captured dict)."""
        if stream is None:
            stream = torch.cuda.current_stream()
        cap = {}
        src = x
        for l in range(self.L):
            # with MS_FWD_PREDICT_NEXT the last layer predicts layer 0 of the
            # next step from its own input, the last layer's intermediate
            # activation (Sec. 3.2)
            ms.ms_forward(self.ctx, l, src, T, self.y, self.idx, self.w, flags, stream)
            if l in capture or counts is not None:
                stream.synchronize()
                idx = self.idx[:T].cpu().numpy()
                if counts is not None:
                    np.add.at(counts[l], idx.reshape(-1), 1)
                if l in capture:
                    cap[l] = dict(h=src[:T].float().cpu().numpy(), y=self.y[:T].cpu().numpy().copy(),
                                  idx=idx.copy(), w=self.w[:T].cpu().numpy().copy())
            dst = self.h[l % 2]
            ms.ms_residual_norm(self.ctx, src, self.y, T, dst, stream)
            src = dst
        return src, cap

    def warmup_counts(self, xs, T):
        """Selection counts [L][E] over the inputs xs (device tensors)."""
        counts = np.zeros((self.L, self.shape.n_experts), np.int64)
        for x in xs:
            self.step(x, T, counts=counts)
        ms.ms_sync(self.ctx)
        return counts

    def stats(self):
        return [ms.ms_stats(self.ctx, l) for l in range(self.L)]

    def close(self):
        self.rig.close()

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()


def decode_inputs(shape, seed, steps, T, tag=0):
    """Seeded correlated token sequence (x_s = sqrt(1-eps^2) x_{s-1} + eps z_s,
    eps = 0.3): list of (device tensor, fp32 host copy)."""
    return [(to_device(raw, shape.dtype), f) for raw, f in synth.walk(shape, seed, steps, T=T, tag=tag)]


def stack_top_bytes(stack: Stack, r: float) -> int:
    return top_bytes(stack.rig, r)
