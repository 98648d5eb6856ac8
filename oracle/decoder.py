"""Oracle of the decoder loop around the split-expert MoE layer: a whole
layer of Sec. 2.1 (the attention module, Eq. (1), then the MoE module,
Eq. (2), each followed by the residual and Norm), the head, greedy token
choice and the embedding of the next token.

TEST INFRASTRUCTURE ONLY, like the rest of this package: plain numpy in
fp64, sharing no code with the GPU library.

The paper defers the attention module to the standard designs it cites
(scaled dot-product attention with grouped-query heads).  Readings taken
here, which the GPU side follows:
* Att(x) = o W_o^T with o the causal grouped-query attention of
  q = rope(x W_q^T), k = rope(x W_k^T), v = x W_v^T: Hq query heads of width
  D share Hkv key/value heads (query head h uses group h // (Hq / Hkv));
  scores q.k / sqrt(D), softmax over positions 0 .. p of a token at
  position p.  W_qkv is one [(Hq + 2 Hkv) D][d] matrix: the query rows, then
  the key rows, then the value rows.
* Positions enter through rotary embeddings (the Mixtral convention,
  "rotate half"): for i < D/2, angle p * base^(-2 i / D) rotates the pair
  (x_i, x_{i + D/2}).
* The key/value cache holds the model dtype (bf16): K, V and q are rounded
  to bf16 where the GPU stores them, and the attention output o is rounded
  to bf16 before W_o.
* Norm is the weightless RMSNorm of the stack (eps 1e-6), applied to the
  residual sums of Eq. (1) and (2).
* The head is logits = x^L W_head^T; the next token is the arg max (lowest
  index on ties); its embedding row is x^0 of the next step.
"""
from __future__ import annotations

import numpy as np

import oracle


def bf16_round(x):
    """Round to bf16 (nearest even) through fp32, returned as fp64."""
    f = np.ascontiguousarray(x, np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    u = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    return u.astype(np.uint32).view(np.float32).astype(np.float64)


def rope(x, pos, base):
    """Rotary embedding of x [H][D] at position pos (rotate-half pairs)."""
    x = np.asarray(x, np.float64)
    D = x.shape[-1]
    half = D // 2
    i = np.arange(half, dtype=np.float64)
    ang = pos * np.power(float(base), -2.0 * i / D)
    c, s = np.cos(ang), np.sin(ang)
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def attend(q, K, V, n_ctx):
    """Grouped-query attention of one token: q [Hq][D], K, V [Hkv][>= n_ctx][D];
    keys 0 .. n_ctx - 1.  Returns [Hq][D]."""
    q = np.asarray(q, np.float64)
    Hq, D = q.shape
    Hkv = K.shape[0]
    group = Hq // Hkv
    out = np.empty((Hq, D))
    for h in range(Hq):
        g = h // group
        s = K[g, :n_ctx] @ q[h] / np.sqrt(D)
        p = np.exp(s - s.max())
        p /= p.sum()
        out[h] = p @ V[g, :n_ctx]
    return out


class Cache:
    """Key/value cache of one layer: [Hkv][max_ctx][D] fp64 (bf16 values)."""

    def __init__(self, Hkv, max_ctx, D):
        self.K = np.zeros((Hkv, max_ctx, D))
        self.V = np.zeros((Hkv, max_ctx, D))


def attention(x, w_qkv, w_o, cache, pos0, Hq, Hkv, D, base):
    """Att(x) for T tokens at positions pos0 .. pos0 + T - 1 (appending their
    keys and values to the cache).  x [T][d] (the layer input).  Returns
    dict(att [T][d] fp64, q [T][Hq][D], o [T][Hq D])."""
    x = np.atleast_2d(np.asarray(x, np.float64))
    T = x.shape[0]
    qkv = x @ np.asarray(w_qkv, np.float64).T
    nq, nk = Hq * D, Hkv * D
    qs, os_ = [], []
    for t in range(T):
        p = pos0 + t
        q = bf16_round(rope(qkv[t, :nq].reshape(Hq, D), p, base))
        k = bf16_round(rope(qkv[t, nq:nq + nk].reshape(Hkv, D), p, base))
        v = bf16_round(qkv[t, nq + nk:].reshape(Hkv, D))
        cache.K[:, p] = k
        cache.V[:, p] = v
        qs.append(q)
    for t in range(T):
        os_.append(bf16_round(attend(qs[t], cache.K, cache.V, pos0 + t + 1).reshape(-1)))
    o = np.array(os_)
    att = o @ np.asarray(w_o, np.float64).T
    return dict(att=att, q=np.array(qs), o=o)


def rmsnorm(x, eps=1e-6):
    x = np.atleast_2d(np.asarray(x, np.float64))
    return x / np.sqrt(np.mean(x * x, axis=1, keepdims=True) + eps)


def head_argmax(x, w_head):
    """logits = x W_head^T and the arg max per row (lowest index on ties)."""
    logits = np.atleast_2d(np.asarray(x, np.float64)) @ np.asarray(w_head, np.float64).T
    return logits, np.argmax(logits, axis=1).astype(np.int32)


def layer(x, lw, cache, pos0, cfg, moe):
    """One decoder layer of Sec. 2.1: h = Norm(x + Att(x)) (Eq. (1)), then
    x' = Norm(h + MoE(h)) (Eq. (2)), with `moe(h_bf16_as_f32) -> y [T][d]`
    the MoE module (the plain layer oracle).  Activations handed between
    modules are bf16, as on the GPU.  Returns (x', h)."""
    a = attention(x, lw["w_qkv"], lw["w_o"], cache, pos0, cfg["Hq"], cfg["Hkv"], cfg["D"], cfg["base"])
    h = bf16_round(rmsnorm(np.asarray(x, np.float64) + a["att"]))
    y = moe(h)
    return bf16_round(rmsnorm(h + y)), h


def moe_from_layer_oracle(w_r, experts, K, renormalize=True, bias=None):
    """The MoE module of Eq. (2) for `layer`, from the plain layer oracle."""
    def moe(h):
        return oracle.moe_layer(np.asarray(h, np.float32), w_r, experts, K, renormalize=renormalize,
                                bias=bias)["y"]
    return moe
