"""CPU oracle of the split-expert MoE layer (arXiv 2509.08342, "MoEpic").

TEST INFRASTRUCTURE ONLY: only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this package.  The GPU library never
calls it and must fail loudly rather than fall back to it.

Thin ctypes wrapper over ``moe_oracle.c`` (plain C, compiled here with gcc,
floating-point contraction off).  What each function computes and which
passage of the paper it follows is documented in the C source; the wrappers
only marshal numpy arrays.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "moe_oracle.c")
_LIB_PATH = os.environ.get("MOE_ORACLE_LIB") or os.path.join(_HERE, "libmoe_oracle.so")
_SAN_PATH = os.path.join(_HERE, "libmoe_oracle_san.so")
_lib = None
_lock = threading.Lock()

CHUNK_UNITS = 64  # intermediate units per chunk when rounding the split point

_f32p = np.ctypeslib.ndpointer(np.float32, flags="C_CONTIGUOUS")
_f64p = np.ctypeslib.ndpointer(np.float64, flags="C_CONTIGUOUS")
_i32p = np.ctypeslib.ndpointer(np.int32, flags="C_CONTIGUOUS")


def build_oracle(force: bool = True, sanitize: bool = False) -> str:
    """Compile moe_oracle.c into libmoe_oracle.so with gcc (no GPU toolchain);
    sanitize=True builds libmoe_oracle_san.so with AddressSanitizer and
    UndefinedBehaviorSanitizer instead (same floating-point flags)."""
    path = _SAN_PATH if sanitize else _LIB_PATH
    if force or not os.path.exists(path) or (os.path.getmtime(path) < os.path.getmtime(_SRC)):
        tmp = path + ".tmp%d" % os.getpid()
        san = ["-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
               "-fno-omit-frame-pointer"] if sanitize else []
        cmd = ["gcc", "-O2", "-std=c99", "-fPIC", "-shared", "-ffp-contract=off",
               "-fno-fast-math", "-Wall", "-Wextra", *san, "-o", tmp, _SRC, "-lm"]
        subprocess.check_call(cmd)
        os.replace(tmp, path)
    return path


def _load():
    global _lib
    with _lock:
        if _lib is not None:
            return _lib
        build_oracle(force=False)
        lib = ctypes.CDLL(_LIB_PATH)
        c_int = ctypes.c_int
        lib.orc_router_logits.argtypes = [_f32p, _f32p, ctypes.c_void_p, c_int, c_int, c_int, _f32p]
        lib.orc_router_logits.restype = c_int
        lib.orc_topk.argtypes = [_f32p, c_int, c_int, c_int, _i32p]
        lib.orc_topk.restype = None
        lib.orc_gate_weights.argtypes = [_f32p, _i32p, c_int, c_int, c_int, c_int, _f64p]
        lib.orc_gate_weights.restype = None
        lib.orc_expert_range.argtypes = [_f32p, _f32p, _f32p, _f32p, c_int, c_int, c_int, c_int, _f64p]
        lib.orc_expert_range.restype = None
        lib.orc_expert_act.argtypes = [_f32p, _f32p, _f32p, c_int, c_int, c_int, c_int, _f64p]
        lib.orc_expert_act.restype = None
        lib.orc_predict.argtypes = [_f32p, c_int, c_int, _f64p, _i32p]
        lib.orc_predict.restype = None
        lib.orc_group.argtypes = [_i32p, c_int, c_int, c_int, _i32p, _i32p]
        lib.orc_group.restype = None
        lib.orc_residual_rmsnorm.argtypes = [_f64p, _f64p, c_int, c_int, ctypes.c_double, _f64p]
        lib.orc_residual_rmsnorm.restype = None
        lib.orc_top_units.argtypes = [ctypes.c_double, c_int, c_int]
        lib.orc_top_units.restype = c_int
        _lib = lib
        return lib


def _f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


# --------------------------------------------------------------------- router

def router_logits(h, w_r, bias=None):
    """Router logits R(h) = h . w_r (+ bias) in the canonical fp32 order.

    h [T][d], w_r [d][E]; returns float32 [T][E]."""
    h = _f32(np.atleast_2d(h))
    w_r = _f32(w_r)
    T, d = h.shape
    E = w_r.shape[1]
    assert w_r.shape[0] == d
    out = np.empty((T, E), np.float32)
    b = None
    if bias is not None:
        b = _f32(bias)
        assert b.shape == (E,)
    rc = _load().orc_router_logits(h, w_r, None if b is None else b.ctypes.data, T, d, E, out)
    if rc != 0:
        raise ValueError("d must be a multiple of 64")
    return out


def topk(logits, K):
    """K largest logits per row, lowest index on ties, in selection order."""
    logits = _f32(np.atleast_2d(logits))
    T, E = logits.shape
    assert 1 <= K <= E
    idx = np.empty((T, K), np.int32)
    _load().orc_topk(logits, T, E, K, idx)
    return idx


def gate_weights(logits, idx, renormalize=True):
    """Eq. (2) gate weights (fp64): selected softmax scores, renormalised."""
    logits = _f32(np.atleast_2d(logits))
    idx = np.ascontiguousarray(idx, np.int32)
    T, E = logits.shape
    K = idx.shape[1]
    w = np.empty((T, K), np.float64)
    _load().orc_gate_weights(logits, idx, T, E, K, int(bool(renormalize)), w)
    return w


# --------------------------------------------------------------------- expert

def expert_range(h_t, w_gate, w_up, w_down, lo, hi, acc=None):
    """E^[lo,hi)(h_t) for one token, fp64, accumulated onto ``acc`` if given.

    w_gate, w_up [d][F]; w_down [F][d]."""
    h_t = _f32(h_t).reshape(-1)
    w_gate, w_up, w_down = _f32(w_gate), _f32(w_up), _f32(w_down)
    d, F = w_gate.shape
    assert h_t.shape == (d,) and w_up.shape == (d, F) and w_down.shape == (F, d)
    assert 0 <= lo <= hi <= F
    out = np.zeros(d, np.float64) if acc is None else acc
    assert out.dtype == np.float64 and out.flags.c_contiguous and out.shape == (d,)
    _load().orc_expert_range(h_t, w_gate, w_up, w_down, d, F, int(lo), int(hi), out)
    return out


def expert_act(h_t, w_gate, w_up, lo, hi):
    """SwiGLU intermediate a_f = silu(h.G_f)(h.U_f), f in [lo,hi), fp64."""
    h_t = _f32(h_t).reshape(-1)
    w_gate, w_up = _f32(w_gate), _f32(w_up)
    d, F = w_gate.shape
    a = np.empty(hi - lo, np.float64)
    _load().orc_expert_act(h_t, w_gate, w_up, d, F, int(lo), int(hi), a)
    return a


def expert(h_t, ex):
    """Full expert output E(h_t); ``ex`` is a (w_gate, w_up, w_down) triple."""
    F = ex[0].shape[1]
    return expert_range(h_t, ex[0], ex[1], ex[2], 0, F)


# ---------------------------------------------------------------------- layer

def moe_layer(h, w_r, experts, K, renormalize=True, bias=None, shared=(),
              tokens=None):
    """One MoE module (Eq. 2 without residual/Norm) on CPU.

    h [T][d]; w_r [d][E]; experts: list of E (w_gate, w_up, w_down) fp32
    triples; shared: list of always-active experts added with weight 1.
    ``tokens`` restricts the expert evaluation (the costly part) to a subset
    of token rows; routing is still returned for every token.
    Returns dict(logits f32 [T][E], idx i32 [T][K], w f64 [T][K],
    y f64 [len(tokens)][d], tokens)."""
    h = _f32(np.atleast_2d(h))
    T, d = h.shape
    logits = router_logits(h, w_r, bias)
    idx = topk(logits, K)
    w = gate_weights(logits, idx, renormalize)
    rows = np.arange(T) if tokens is None else np.asarray(tokens, np.int64)
    y = np.zeros((len(rows), d), np.float64)
    for i, t in enumerate(rows):
        for k in range(K):
            e = int(idx[t, k])
            y[i] += w[t, k] * expert(h[t], experts[e])
        for ex in shared:
            y[i] += expert(h[t], ex)
    return dict(logits=logits, idx=idx, w=w, y=y, tokens=rows)


# ----------------------------------------------------------------- prediction

def predict(h, w_r_next, bias=None):
    """Eq. (3) prediction: summed next-layer probabilities and their ranking.

    Returns (score f64 [E], order i32 [E]), order by descending score, lower
    index first on equal scores."""
    logits = router_logits(h, w_r_next, bias)
    T, E = logits.shape
    score = np.empty(E, np.float64)
    order = np.empty(E, np.int32)
    _load().orc_predict(logits, T, E, score, order)
    return score, order


# ------------------------------------------------------------------- grouping

def group(idx, E):
    """Stable token-to-expert grouping of the T*K slots: (offsets[E+1], perm)."""
    idx = np.ascontiguousarray(idx, np.int32)
    T, K = idx.shape
    offsets = np.empty(E + 1, np.int32)
    perm = np.empty(max(T * K, 1), np.int32)
    _load().orc_group(idx, T, K, E, offsets, perm)
    return offsets, perm[:T * K]


# ----------------------------------------------------------------------- glue

def residual_rmsnorm(h, y, eps=1e-6):
    """Stack glue: RMSNorm(h + y), weightless."""
    h = np.ascontiguousarray(np.atleast_2d(h), np.float64)
    y = np.ascontiguousarray(np.atleast_2d(y), np.float64)
    T, d = h.shape
    out = np.empty_like(h)
    _load().orc_residual_rmsnorm(h, y, T, d, float(eps), out)
    return out


def top_units(r, F, g=CHUNK_UNITS):
    """Intermediate units in the top segment for split ratio r (chunk-rounded)."""
    return int(_load().orc_top_units(float(r), int(F), int(g)))
