"""A whole decoder loop around the split-expert MoE layers (Sec. 2.1): per
layer the attention module, h = Norm(x + Att(x)) (Eq. (1)), then the MoE
module, x' = Norm(h + MoE(h)) (Eq. (2)); after the last layer the head, the
greedy token and its embedding, which is the next step's x^0.  Every step
runs in the library's kernels (ms_dense, ms_rope_kv, ms_attention,
ms_residual_norm, ms_forward, ms_argmax, ms_embed); this module allocates
device buffers with torch and sequences the calls.

Layer i's forward predicts layer i + 1 from h^i and prefetches it
(Sec. 3.2), so the copies run under layer i's MoE module and layer i + 1's
attention; layer 0 of the next token is predicted from the last layer's
intermediate activation h^L of the current token (Sec. 3.2, following
AdapMoE), and its copies run under the head and layer 0's attention (the
first layer's window, T_head + T_att)."""
from __future__ import annotations

import time

import numpy as np
import torch

import synth
from paper_2509_08342_amd import moesplit as ms
from stack import Stack
from workload import to_device


class Decoder:
    def __init__(self, shape: synth.ModelShape, attn: synth.AttnShape, *, seed=0, n_sets=2, max_tokens=1,
                 max_ctx=256, budget_total=0, keep_f32=True, threads=16):
        self.shape, self.attn = shape, attn
        self.stack = Stack(shape, seed=seed, n_sets=n_sets, max_tokens=max_tokens, budget_total=budget_total,
                           keep_f32=keep_f32, threads=threads)
        self.ctx = self.stack.ctx
        self.L = shape.n_layers
        self.max_ctx = max_ctx
        self.max_tokens = max_tokens
        d, V = shape.d_model, attn.vocab
        Hq, Hkv, D = attn.n_heads, attn.n_kv_heads, attn.head_dim
        self.n_qkv = (Hq + 2 * Hkv) * D
        bf = torch.bfloat16
        dev = "cuda"
        # attention weights: layer l uses weight set l % n_sets, like the experts
        self.n_sets = self.stack.rig.n_sets
        self.w_qkv, self.w_o, self.f32 = [], [], {}
        for s_ in range(self.n_sets):
            (qr, qf), (orr, of) = synth.attn_weights(shape, attn, seed, s_)
            self.w_qkv.append(to_device(qr, shape.dtype))
            self.w_o.append(to_device(orr, shape.dtype))
            if keep_f32:
                self.f32[s_] = (qf, of)
        (hr, hf), (er, ef) = synth.head_weights(shape, attn, seed)
        self.head = to_device(hr, shape.dtype)
        self.embed = to_device(er, shape.dtype)
        self.head_f32, self.embed_f32 = (hf, ef) if keep_f32 else (None, None)
        self.kc = torch.zeros(self.L, Hkv, max_ctx, D, dtype=bf, device=dev)
        self.vc = torch.zeros(self.L, Hkv, max_ctx, D, dtype=bf, device=dev)
        T = max_tokens
        self.qkv = torch.empty(T, self.n_qkv, dtype=torch.float32, device=dev)
        self.q = torch.empty(T, Hq, D, dtype=bf, device=dev)
        self.o = torch.empty(T, Hq * D, dtype=bf, device=dev)
        self.att = torch.empty(T, d, dtype=torch.float32, device=dev)
        self.x = [torch.empty(T, d, dtype=bf, device=dev) for _ in range(2)]
        self.h = torch.empty(T, d, dtype=bf, device=dev)
        self.y, self.idx, self.w = self.stack.rig.outputs(T)
        self.logits = torch.empty(1, V, dtype=torch.float32, device=dev)
        self.ids = torch.zeros(max(T, 1), dtype=torch.int32, device=dev)
        self.pos = 0

    def layer_weights(self, l):
        return self.w_qkv[l % self.n_sets], self.w_o[l % self.n_sets]

    def reset(self):
        """Forget the context (the caches are overwritten as positions fill)."""
        self.pos = 0

    # ------------------------------------------------------------- a step
    def step(self, x0, T, flags=ms.MS_FWD_PREDICT_NEXT, stream=None, capture=(), marks=None):
        """Run T tokens (x0 [T][d] bf16 device rows, at positions pos ..
        pos + T - 1) through every layer and the head of the last token.
        Returns the next token id as a 1-element device tensor.  capture:
        layers whose (x_in, h, x_out) are copied to the host; marks: list that
        receives (name, event) pairs around the attention, MoE and head parts."""
        if stream is None:
            stream = torch.cuda.current_stream()
        a = self.attn
        d, V = self.shape.d_model, a.vocab
        pos0 = self.pos
        assert pos0 + T <= self.max_ctx and T <= self.max_tokens
        cap = {}
        src = x0

        def mark(name):
            if marks is not None:
                ev = torch.cuda.Event(enable_timing=True)
                ev.record(stream)
                marks.append((name, ev))

        for l in range(self.L):
            wq, wo = self.layer_weights(l)
            mark("att")
            ms.ms_dense(src, wq, T, d, self.n_qkv, self.qkv, None, stream)
            ms.ms_rope_kv(self.qkv, T, a.n_heads, a.n_kv_heads, a.head_dim, pos0, a.rope_base, self.q,
                          self.kc[l], self.vc[l], self.max_ctx, stream)
            ms.ms_attention(self.q, self.kc[l], self.vc[l], T, a.n_heads, a.n_kv_heads, a.head_dim, pos0,
                            self.max_ctx, self.o, stream)
            ms.ms_dense(self.o, wo, T, a.n_heads * a.head_dim, d, self.att, None, stream)
            ms.ms_residual_norm(self.ctx, src, self.att, T, self.h, stream)
            mark("moe")
            # the last layer of a single-token step predicts layer 0 of the
            # next token from its own intermediate activation h (Sec. 3.2);
            # a prompt's last layer predicts from its last row below
            fl = flags if (l + 1 < self.L or T == 1) else flags & ~ms.MS_FWD_PREDICT_NEXT
            ms.ms_forward(self.ctx, l, self.h, T, self.y, self.idx, self.w, fl, stream)
            dst = self.x[l % 2]
            ms.ms_residual_norm(self.ctx, self.h, self.y, T, dst, stream)
            if l in capture:
                stream.synchronize()
                cap[l] = dict(x=src[:T].float().cpu().numpy(), h=self.h[:T].float().cpu().numpy(),
                              x_out=dst[:T].float().cpu().numpy(), idx=self.idx[:T].cpu().numpy().copy())
            src = dst
        mark("head")
        last = src[T - 1:T]
        if flags & ms.MS_FWD_PREDICT_NEXT and T > 1:
            # layer 0 of the token after the prompt, predicted from the last
            # layer's intermediate activation of the prompt's last token; its
            # copies run under the head and layer 0's attention
            order, _ = ms.ms_predict(self.ctx, 0, self.h[T - 1:T], 1, stream, self.shape.n_experts)
            ms.ms_prefetch(self.ctx, 0, order[:self.shape.top_k])
        ms.ms_dense(last, self.head, 1, d, V, self.logits, None, stream)
        ms.ms_argmax(self.logits, 1, V, self.ids, stream)
        mark("end")
        self.pos += T
        self.final = src
        return cap

    def embed_ids(self, ids_dev, T, out, stream=None):
        ms.ms_embed(ids_dev, self.embed, self.attn.vocab, T, self.shape.d_model, out, stream)

    def generate(self, prompt, n_new, flags=ms.MS_FWD_PREDICT_NEXT, stream=None, timing=False, after_prefill=None):
        """Prefill the prompt (host int32 ids), then n_new greedy decode steps.
        after_prefill: called once the first token is out.  Returns (token
        ids, ttft_ms, [per-token ms])."""
        if stream is None:
            stream = torch.cuda.current_stream()
        P = len(prompt)
        ids = torch.from_numpy(np.asarray(prompt, np.int32)).to("cuda")
        xin = torch.empty(P, self.shape.d_model, dtype=torch.bfloat16, device="cuda")
        self.embed_ids(ids, P, xin, stream)
        out = []
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        self.step(xin, P, flags, stream)
        tok = self.ids[:1].clone()
        stream.synchronize()
        ttft = (time.perf_counter() - t0) * 1e3
        out.append(int(tok.item()))
        if after_prefill is not None:
            after_prefill()
        tpot = []
        x1 = torch.empty(1, self.shape.d_model, dtype=torch.bfloat16, device="cuda")
        for _ in range(n_new - 1):
            t1 = time.perf_counter()
            self.embed_ids(self.ids, 1, x1, stream)
            self.step(x1, 1, flags, stream)
            stream.synchronize()
            tpot.append((time.perf_counter() - t1) * 1e3)
            out.append(int(self.ids[0].item()))
        return out, ttft, tpot

    def close(self):
        self.stack.close()

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()
