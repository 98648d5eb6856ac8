"""Seeded synthetic inputs for the split-expert MoE layer.

This module is the only code shared by the GPU-side tests/benchmark and the
CPU oracle side: it draws random numbers and rounds them to the model's
storage type, and holds none of the layer's arithmetic.

Recipe (the paper's models and MMLU prompts are not available; these shapes
and distributions stand in for them):
  * every tensor comes from numpy's PCG64 seeded with
    SeedSequence([seed, kind, layer, index]);
  * expert and router weights are N(0, 0.02), token activations N(0, 1);
  * bf16 models round the fp32 draw to bf16 with round-to-nearest-even; the
    fp32 view of the rounded value (exact) is what the oracle consumes;
  * decode sequences follow x_s = sqrt(1 - eps^2) x_{s-1} + eps z_s (eps 0.3),
    which keeps every x_s marginally N(0, 1) while consecutive tokens stay
    correlated;
  * a Zipf(1.1)-skewed workload adds the router bias
    b_e = -1.1 ln(1 + pi(e)) with pi a seeded permutation of the experts, so
    softmax(b) alone is exactly Zipf(1.1) over expert ranks.
"""
from __future__ import annotations

import dataclasses
import numpy as np

KIND_GATE, KIND_UP, KIND_DOWN, KIND_ROUTER, KIND_HIDDEN = 0, 1, 2, 3, 4
KIND_SH_GATE, KIND_SH_UP, KIND_SH_DOWN, KIND_PERM, KIND_WALK = 5, 6, 7, 8, 9
KIND_QKV, KIND_O, KIND_HEAD, KIND_EMBED, KIND_TOKENS = 10, 11, 12, 13, 14

WEIGHT_STD = 0.02


@dataclasses.dataclass(frozen=True)
class ModelShape:
    name: str
    n_layers: int
    d_model: int
    d_ff: int
    n_experts: int
    top_k: int
    dtype: str = "bf16"          # "f32" or "bf16" storage of weights and h
    n_shared: int = 0
    d_ff_shared: int = 0
    renormalize: int = 1
    zipf: float = 0.0            # router-bias skew exponent (0 = none)
    expert_bits: int = 0         # 0: experts in `dtype`; 2 or 4: affine codes (see QuantExpert)

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2

    @property
    def expert_bytes(self) -> int:
        if self.expert_bits:
            # codes of three matrices plus one 4-byte (scale, zero) per group of 64
            return 3 * self.d_model * self.d_ff * self.expert_bits // 8 + 3 * (self.d_model * self.d_ff // 64) * 4
        return 3 * self.d_model * self.d_ff * self.elem_bytes


# Workload shapes: a tiny fp32 layer, and Mixtral-8x7B-, DeepSeek-V2-Lite- and
# Qwen3-30B-A3B-shaped layers (bf16 weights, fp32 accumulation).
TINY = ModelShape("tiny-f32", 1, 256, 512, 8, 2, "f32")
MIXTRAL = ModelShape("mixtral-8x7b", 1, 4096, 14336, 8, 2)
MIXTRAL_STACK = dataclasses.replace(MIXTRAL, name="mixtral-8x7b-stack", n_layers=32)
DEEPSEEK = ModelShape("deepseek-v2-lite", 26, 2048, 1408, 64, 6, n_shared=2,
                      d_ff_shared=1408)
QWEN3 = ModelShape("qwen3-30b-a3b", 48, 2048, 768, 128, 8, zipf=1.1)

# The paper's Mixtral setting stores the MoE weights as 2-bit HQQ codes.
MIXTRAL_Q2 = dataclasses.replace(MIXTRAL, name="mixtral-8x7b-q2", expert_bits=2)
MIXTRAL_Q2_STACK = dataclasses.replace(MIXTRAL_Q2, name="mixtral-8x7b-q2-stack", n_layers=32)

SHAPES = {s.name: s for s in (TINY, MIXTRAL, MIXTRAL_STACK, DEEPSEEK, QWEN3, MIXTRAL_Q2, MIXTRAL_Q2_STACK)}


def _rng(seed: int, kind: int, layer: int, index: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(
        np.random.SeedSequence([int(seed), int(kind), int(layer), int(index)])))


# ------------------------------------------------------------ bf16 storage --

def bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns (uint16), round to nearest, ties to even."""
    u = np.ascontiguousarray(x, np.float32).view(np.uint32)
    r = u >> np.uint32(16)
    r &= np.uint32(1)
    r += np.uint32(0x7FFF)
    r += u
    r >>= np.uint32(16)
    return r.astype(np.uint16)


def bf16_to_f32(b: np.ndarray) -> np.ndarray:
    """bf16 bit patterns -> fp32 (exact)."""
    return (np.ascontiguousarray(b, np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def storage(x_f32: np.ndarray, dtype: str):
    """Round an fp32 draw to the storage type.

    Returns (raw, exact_f32): ``raw`` is what the library is given (fp32 or
    bf16 bits), ``exact_f32`` the same values as fp32 for the oracle."""
    if dtype == "f32":
        x = np.ascontiguousarray(x_f32, np.float32)
        return x, x
    b = bf16_bits(x_f32)
    return b, bf16_to_f32(b)


def _normal(seed, kind, layer, index, shape, std):
    x = _rng(seed, kind, layer, index).standard_normal(shape, dtype=np.float32)
    if std != 1.0:
        x *= np.float32(std)
    return x


# ----------------------------------------------------------------- tensors --

@dataclasses.dataclass
class Expert:
    """One SwiGLU expert: w_gate, w_up [d][F]; w_down [F][d].

    ``raw`` holds the storage-typed arrays for the library, ``f32`` the exact
    fp32 values for the oracle."""
    raw: tuple
    f32: tuple


def expert(shape: ModelShape, seed: int, layer: int, e: int, shared: bool = False) -> Expert:
    d = shape.d_model
    F = shape.d_ff_shared if shared else shape.d_ff
    kinds = (KIND_SH_GATE, KIND_SH_UP, KIND_SH_DOWN) if shared else (KIND_GATE, KIND_UP, KIND_DOWN)
    shapes = ((d, F), (d, F), (F, d))
    raw, f32 = [], []
    for kind, shp in zip(kinds, shapes):
        r, x = storage(_normal(seed, kind, layer, e, shp, WEIGHT_STD), shape.dtype)
        raw.append(r)
        f32.append(x)
    return Expert(tuple(raw), tuple(f32))


# ------------------------------------------------------ quantized storage --
#
# Experts stored as affine b-bit codes in the format of HQQ (half-quadratic
# quantization), which the paper uses for its 2-bit Mixtral: each matrix is
# taken as [out][in] (gate and up: [F][d]; down: [d][F]) and every group of
# QGROUP consecutive elements along `in` has one scale and one zero, both
# fp16, with w = (q - zero) * scale.  The synthetic weights are the same
# N(0, 0.02) draws as the bf16 experts, quantized by round-to-nearest over
# each group's [min, max] (HQQ's starting point; its zero-point refinement
# changes values, not the format or the bytes moved).

QGROUP = 64


@dataclasses.dataclass
class QuantExpert:
    """codes: (gate [F][d/P], up [F][d/P], down [d][F/P]) uint8 with P = 8 /
    bits codes per byte, element i of a row at bits (i % P) * bits of byte
    i // P; meta: (gate [F][d/64][2], up [F][d/64][2], down [d][F/64][2])
    uint16 fp16 bit patterns (scale, zero)."""
    bits: int
    codes: tuple
    meta: tuple


def pack_codes(q: np.ndarray, bits: int) -> np.ndarray:
    """[rows][n] codes (0 .. 2^bits - 1) -> [rows][n * bits / 8] bytes."""
    P = 8 // bits
    q = np.asarray(q, np.uint8)
    out = np.zeros((q.shape[0], q.shape[1] // P), np.uint8)
    for j in range(P):
        out |= (q[:, j::P] << (j * bits)).astype(np.uint8)
    return out


def quantize_rows(w: np.ndarray, bits: int):
    """Round-to-nearest affine codes of w [rows][n] (n a multiple of 64):
    returns (packed codes, meta [rows][n/64][2] uint16)."""
    rows, n = w.shape
    g = np.asarray(w, np.float32).reshape(rows, n // QGROUP, QGROUP)
    lo, hi = g.min(axis=2), g.max(axis=2)
    qmax = np.float32(2 ** bits - 1)
    scale = ((hi - lo) / qmax).astype(np.float32)
    scale[scale == 0] = 1.0
    s16 = scale.astype(np.float16)
    z16 = (-lo / s16.astype(np.float32)).astype(np.float16)
    q = g / s16.astype(np.float32)[:, :, None]
    q += z16.astype(np.float32)[:, :, None]
    np.rint(q, out=q)
    np.clip(q, 0, qmax, out=q)
    q = q.astype(np.uint8).reshape(rows, n)
    meta = np.stack([s16.view(np.uint16), z16.view(np.uint16)], axis=2)
    return pack_codes(q, bits), np.ascontiguousarray(meta)


def quant_expert(shape: ModelShape, seed: int, layer: int, e: int, bits: int) -> QuantExpert:
    """Expert e of `layer` as b-bit codes: N(0, 0.02) draws in [out][in]
    order (gate, up [F][d]; down [d][F]), quantized row-group by row-group."""
    d, F = shape.d_model, shape.d_ff
    parts = []
    for kind, shp in ((KIND_GATE, (F, d)), (KIND_UP, (F, d)), (KIND_DOWN, (d, F))):
        parts.append(quantize_rows(_normal(seed, kind, layer, e, shp, WEIGHT_STD), bits))
    return QuantExpert(bits, tuple(p[0] for p in parts), tuple(p[1] for p in parts))


def router(shape: ModelShape, seed: int, layer: int):
    """Router weight [d][E] as (raw, exact_f32)."""
    x = _normal(seed, KIND_ROUTER, layer, 0, (shape.d_model, shape.n_experts), WEIGHT_STD)
    return storage(x, shape.dtype)


def router_bias(shape: ModelShape, seed: int, layer: int):
    """Zipf-skew router bias [E] (fp32), or None when the shape has no skew."""
    if shape.zipf <= 0.0:
        return None
    perm = _rng(seed, KIND_PERM, layer, 0).permutation(shape.n_experts)
    return (-shape.zipf * np.log1p(perm.astype(np.float64))).astype(np.float32)


def hidden(shape: ModelShape, seed: int, T: int, tag: int = 0):
    """Token activations [T][d] ~ N(0, 1) as (raw, exact_f32)."""
    return storage(_normal(seed, KIND_HIDDEN, tag, 0, (T, shape.d_model), 1.0), shape.dtype)


def walk(shape: ModelShape, seed: int, steps: int, T: int = 1, eps: float = 0.3, tag: int = 0):
    """Correlated decode inputs: x_s = sqrt(1-eps^2) x_{s-1} + eps z_s.

    Returns a list of (raw, exact_f32) pairs, each [T][d]."""
    rng = _rng(seed, KIND_WALK, tag, 0)
    x = rng.standard_normal((T, shape.d_model), dtype=np.float32)
    a = np.float32(np.sqrt(1.0 - eps * eps))
    out = []
    for _ in range(steps):
        out.append(storage(x, shape.dtype))
        x = a * x + np.float32(eps) * rng.standard_normal((T, shape.d_model), dtype=np.float32)
    return out


# ------------------------------------------------------------ decoder loop --

@dataclasses.dataclass(frozen=True)
class AttnShape:
    """Attention and head of a decoder around the MoE layers: Hq query heads
    and Hkv key/value heads of width D, rotary base, vocabulary size."""
    n_heads: int
    n_kv_heads: int
    head_dim: int
    rope_base: float
    vocab: int


# Mixtral-8x7B's attention (32 heads, 8 key/value heads of 128, rotary base
# 1e6) and vocabulary; a tiny one for the tests.
MIXTRAL_ATTN = AttnShape(32, 8, 128, 1e6, 32000)
TINY_ATTN = AttnShape(4, 2, 64, 1e4, 512)


def attn_weights(shape: ModelShape, attn: AttnShape, seed: int, layer: int):
    """(w_qkv [(Hq + 2 Hkv) D][d], w_o [d][Hq D]) as (raw, exact_f32) pairs,
    N(0, 0.02) rounded to the model dtype."""
    d, D = shape.d_model, attn.head_dim
    n_qkv = (attn.n_heads + 2 * attn.n_kv_heads) * D
    qkv = storage(_normal(seed, KIND_QKV, layer, 0, (n_qkv, d), WEIGHT_STD), shape.dtype)
    o = storage(_normal(seed, KIND_O, layer, 0, (d, attn.n_heads * D), WEIGHT_STD), shape.dtype)
    return qkv, o


def head_weights(shape: ModelShape, attn: AttnShape, seed: int):
    """(head [V][d] N(0, 0.02), embedding [V][d] N(0, 1)) as (raw, exact_f32)."""
    head = storage(_normal(seed, KIND_HEAD, 0, 0, (attn.vocab, shape.d_model), WEIGHT_STD), shape.dtype)
    emb = storage(_normal(seed, KIND_EMBED, 0, 0, (attn.vocab, shape.d_model), 1.0), shape.dtype)
    return head, emb


def prompt_tokens(attn: AttnShape, seed: int, n: int, tag: int = 0) -> np.ndarray:
    """A seeded prompt of n token ids, uniform over the vocabulary."""
    return _rng(seed, KIND_TOKENS, tag, 0).integers(0, attn.vocab, size=n).astype(np.int32)
