"""Oracle of the split-expert MoE layer whose experts are stored as affine
b-bit codes: the HQQ-quantized MoE weights of the paper's Mixtral setting
(Sec. 5.1: attention 4-bit, MoE modules 2-bit).

TEST INFRASTRUCTURE ONLY, like the rest of this package: plain numpy in
fp64, sharing no code with the GPU library.

Format (the plain definition of the quantized weights): every matrix is
taken as [out][in] -- gate and up [F][d], down [d][F] -- and each group of 64
consecutive elements along `in` carries one fp16 scale s and one fp16 zero z;
element w = (q - z) * s with q the element's b-bit code.  Codes are packed
8 / b per byte, element i of a row at bits (i % (8 / b)) * b of byte
i // (8 / b).  Splitting, caching and streaming do not change what the layer
computes (Eq. (2)): the output is the plain MoE layer over the dequantized
experts, which is what ``moe_layer`` evaluates.
"""
from __future__ import annotations

import numpy as np

import oracle

GROUP = 64


def unpack_codes(packed, bits, n):
    """[rows][n * bits / 8] bytes -> [rows][n] integer codes."""
    packed = np.asarray(packed, np.uint8)
    per = 8 // bits
    mask = (1 << bits) - 1
    rows = packed.shape[0]
    q = np.empty((rows, n), np.int64)
    for i in range(n):
        q[:, i] = (packed[:, i // per] >> ((i % per) * bits)) & mask
    return q


def fp16_values(bits16):
    """fp16 bit patterns -> fp64 values (exact)."""
    return np.asarray(bits16, np.uint16).view(np.float16).astype(np.float64)


def dequantize(packed, meta, bits, n):
    """w[r][i] = (q[r][i] - z[r][i // 64]) * s[r][i // 64] in fp64.

    packed [rows][n * bits / 8]; meta [rows][n / 64][2] fp16 bit patterns
    (scale, zero)."""
    q = unpack_codes(packed, bits, n)
    meta = np.asarray(meta, np.uint16)
    s = fp16_values(meta[:, :, 0])
    z = fp16_values(meta[:, :, 1])
    w = np.empty(q.shape, np.float64)
    for i in range(n):
        g = i // GROUP
        w[:, i] = (q[:, i] - z[:, g]) * s[:, g]
    return w


def expert_weights(codes, meta, bits, d, F):
    """(w_gate [d][F], w_up [d][F], w_down [F][d]) in fp64 from the three
    quantized matrices ([out][in] each)."""
    wg = dequantize(codes[0], meta[0], bits, d).T
    wu = dequantize(codes[1], meta[1], bits, d).T
    wd = dequantize(codes[2], meta[2], bits, F).T
    return np.ascontiguousarray(wg), np.ascontiguousarray(wu), np.ascontiguousarray(wd)


def expert(h_t, weights):
    """SwiGLU expert in fp64: (silu(h . W_gate) * (h . W_up)) . W_down."""
    wg, wu, wd = weights
    h = np.asarray(h_t, np.float64).reshape(-1)
    g = h @ wg
    u = h @ wu
    a = g / (1.0 + np.exp(-g)) * u
    return a @ wd


def moe_layer(h, w_r, experts, K, renormalize=True, bias=None, tokens=None):
    """One MoE module over dequantized experts: routing and gate weights by
    the plain oracle (Eq. (2)), then y_t = sum_k w_tk E_{S_tk}(h_t) in fp64,
    k in selection order.  experts: list of E fp64 weight triples from
    expert_weights.  Returns dict like oracle.moe_layer."""
    h = np.ascontiguousarray(np.atleast_2d(h), np.float32)
    T, d = h.shape
    logits = oracle.router_logits(h, w_r, bias)
    idx = oracle.topk(logits, K)
    w = oracle.gate_weights(logits, idx, renormalize)
    rows = np.arange(T) if tokens is None else np.asarray(tokens, np.int64)
    y = np.zeros((len(rows), d), np.float64)
    for i, t in enumerate(rows):
        for k in range(K):
            y[i] += w[t, k] * expert(h[t], experts[int(idx[t, k])])
    return dict(logits=logits, idx=idx, w=w, y=y, tokens=rows)
