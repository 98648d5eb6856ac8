"""Oracle of the split-expert MoE layer whose experts are stored as affine
b-bit codes: the HQQ-quantized MoE weights of the paper's Mixtral setting
(Sec. 4.1: attention 4-bit, MoE modules 2-bit).

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
    """[rows][n * bits / 8] bytes -> [rows][n] integer codes: code i of a row
    is bits (i % per) * bits of byte i // per, per = 8 / bits."""
    packed = np.asarray(packed, np.uint8)
    per = 8 // bits
    mask = (1 << bits) - 1
    shifts = (np.arange(per) * bits).astype(np.uint8)
    # [rows][n / per][per]: byte i // per, position i % per
    q = (packed[:, :, None] >> shifts[None, None, :]) & mask
    return q.reshape(packed.shape[0], n)


def fp16_values(bits16):
    """fp16 bit patterns -> fp64 values (exact)."""
    return np.asarray(bits16, np.uint16).view(np.float16).astype(np.float64)


def dequantize(packed, meta, bits, n):
    """w[r][i] = (q[r][i] - z[r][i // 64]) * s[r][i // 64] in fp64.

    packed [rows][n * bits / 8]; meta [rows][n / 64][2] fp16 bit patterns
    (scale, zero)."""
    rows = np.asarray(packed).shape[0]
    q = unpack_codes(packed, bits, n).reshape(rows, n // GROUP, GROUP)
    meta = np.asarray(meta, np.uint16)
    s = fp16_values(meta[:, :, 0])[:, :, None]  # group g = i // 64 of element i
    z = fp16_values(meta[:, :, 1])[:, :, None]
    return ((q - z) * s).reshape(rows, n)


def expert_weights(codes, meta, bits, d, F):
    """(w_gate [d][F], w_up [d][F], w_down [F][d]) in fp64 from the three
    quantized matrices ([out][in] each)."""
    wg = dequantize(codes[0], meta[0], bits, d).T
    wu = dequantize(codes[1], meta[1], bits, d).T
    wd = dequantize(codes[2], meta[2], bits, F).T
    return wg, wu, wd


def expert(h_t, weights):
    """SwiGLU expert in fp64: (silu(h . W_gate) * (h . W_up)) . W_down."""
    wg, wu, wd = weights
    h = np.asarray(h_t, np.float64).reshape(-1)
    g = h @ wg
    u = h @ wu
    a = g / (1.0 + np.exp(-g)) * u
    return a @ wd


def expert_range(h_t, codes, meta, bits, d, F, lo, hi):
    """E^[lo,hi)(h_t): the expert's sum over intermediate units [lo, hi)
    (multiples of 64; Sec. 3.1's vertical split), dequantizing only those
    units' gate and up rows and down columns.  fp64."""
    assert lo % GROUP == 0 and hi % GROUP == 0 and 0 <= lo <= hi <= F
    per = 8 // bits
    wg = dequantize(np.asarray(codes[0])[lo:hi], np.asarray(meta[0])[lo:hi], bits, d)      # [hi-lo][d]
    wu = dequantize(np.asarray(codes[1])[lo:hi], np.asarray(meta[1])[lo:hi], bits, d)
    wd = dequantize(np.asarray(codes[2])[:, lo // per:hi // per], np.asarray(meta[2])[:, lo // GROUP:hi // GROUP],
                    bits, hi - lo)                                                            # [d][hi-lo]
    h = np.asarray(h_t, np.float64).reshape(-1)
    g = wg @ h
    u = wu @ h
    a = g / (1.0 + np.exp(-g)) * u
    return wd @ a


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
