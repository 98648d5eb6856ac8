"""ctypes binding of libmoesplit (include/moesplit.h), same names as the C ABI.

Argument marshalling only: every step of the layer runs in the library's HIP
kernels.  Device buffers are passed as torch tensors (their data_ptr()) or raw
integers; streams as torch.cuda.Stream objects, raw handles or None.  The
binding raises ImportError if the built library is missing; there is no
fallback implementation.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

# MOESPLIT_LIB names another build of the same library (the sanitized host
# build of build.py --sanitize); there is no fallback when it is missing.
_LIB_PATH = os.environ.get("MOESPLIT_LIB") or os.path.join(os.path.dirname(os.path.abspath(__file__)),
                                                          "libmoesplit.so")

MS_OK, MS_E_INVALID, MS_E_BUDGET, MS_E_STATE, MS_E_HIP, MS_E_NOMEM, MS_E_UNSUPPORTED = range(7)
STATUS_NAMES = {0: "MS_OK", 1: "MS_E_INVALID", 2: "MS_E_BUDGET", 3: "MS_E_STATE", 4: "MS_E_HIP",
                5: "MS_E_NOMEM", 6: "MS_E_UNSUPPORTED"}
MS_F32, MS_BF16 = 0, 1
MS_FWD_PREDICT_NEXT = 1
MS_FWD_MATRIX_CORES = 2
MS_FWD_NO_MATRIX_CORES = 4
(MS_IV_ROUTER, MS_IV_GROUP, MS_IV_FFN_RESIDENT, MS_IV_FFN_STREAMED, MS_IV_COMBINE,
 MS_IV_COPY_MISS, MS_IV_COPY_PREFETCH, MS_IV_COPY_TOP, MS_IV_PREDICT, MS_IV_FFN_DOWN) = range(10)
INTERVAL_NAMES = ["router", "group", "ffn_resident", "ffn_streamed", "combine",
                  "copy_miss", "copy_prefetch", "copy_top", "predict", "ffn_down"]


class ms_model_desc(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "n_layers", "d_model", "d_ff", "n_experts", "top_k", "n_shared", "d_ff_shared",
        "dtype", "renormalize", "max_tokens", "n_buffer_slots", "ffn_splits", "expert_bits")]


class ms_sizes(ctypes.Structure):
    _fields_ = [("chunk_bytes", ctypes.c_uint64), ("n_chunks", ctypes.c_int32),
                ("expert_bytes", ctypes.c_uint64), ("fixed_pool_bytes", ctypes.c_uint64),
                ("buffer_bytes", ctypes.c_uint64)]


class ms_layer_stats(ctypes.Structure):
    _fields_ = [(n, ctypes.c_uint64) for n in (
        "forwards", "tokens", "selected", "experts_active", "alpha", "beta", "gamma",
        "buffer_hits", "bytes_miss", "bytes_prefetch", "bytes_prefetch_used",
        "bytes_prefetch_dropped", "predicted_hits", "predictions", "cache_inserts")]

    def as_dict(self):
        return {n: int(getattr(self, n)) for n, _ in self._fields_}


class ms_plan_problem(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("n_experts", ctypes.c_int32), ("top_k", ctypes.c_int32),
                ("expert_bytes", ctypes.c_uint64), ("t_att_us", ctypes.c_double), ("t_moe_us", ctypes.c_double),
                ("t_head_us", ctypes.c_double), ("t_load_us", ctypes.c_double),
                ("hit", ctypes.c_void_p), ("pred", ctypes.c_void_p), ("pred_hit", ctypes.c_void_p)]


MS_CACHE_STATIC, MS_CACHE_LCP, MS_CACHE_LRU, MS_CACHE_LFU, MS_CACHE_RND = range(5)
MS_COPY_KERNEL, MS_COPY_DMA = range(2)


class ms_interval(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("layer", ctypes.c_int32), ("t0_ms", ctypes.c_double),
                ("t1_ms", ctypes.c_double), ("bytes", ctypes.c_uint64)]


def _load():
    if not os.path.exists(_LIB_PATH):
        raise ImportError(
            "libmoesplit.so is not built (%s); run __graft_entry__.build() or "
            "python paper_2509_08342_amd/build.py" % _LIB_PATH)
    lib = ctypes.CDLL(_LIB_PATH)
    P, I32, U64, F32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_uint64, ctypes.c_float
    sig = {
        "ms_query_sizes": [ctypes.POINTER(ms_model_desc), ctypes.POINTER(ms_sizes)],
        "ms_split_plan": [ctypes.POINTER(ms_model_desc), U64, F32, ctypes.POINTER(I32),
                          ctypes.POINTER(U64), ctypes.POINTER(I32)],
        "ms_create": [ctypes.POINTER(ms_model_desc), P, U64, I32, ctypes.POINTER(P)],
        "ms_set_router": [P, I32, P, P],
        "ms_set_expert": [P, I32, I32, P, P, P],
        "ms_set_expert_q": [P, I32, I32, P, P, P, P, P, P],
        "ms_alias_expert": [P, I32, I32, I32, I32],
        "ms_set_shared_expert": [P, I32, I32, P, P, P],
        "ms_configure": [P, P, P, P],
        "ms_load_top": [P, I32, I32],
        "ms_evict_top": [P, I32, I32],
        "ms_residency": [P, I32, P],
        "ms_predict": [P, I32, P, I32, P, P, P],
        "ms_prefetch": [P, I32, P, I32],
        "ms_forward": [P, I32, P, I32, P, P, P, I32, P],
        "ms_forward_noalloc": [P, I32, P, I32, P, P, P, I32, P],
        "ms_sync": [P],
        "ms_drop_buffer": [P],
        "ms_stats": [P, I32, ctypes.POINTER(ms_layer_stats)],
        "ms_reset_stats": [P],
        "ms_residual_norm": [P, P, P, I32, P, P],
        "ms_plan_stats": [P, I32, P, P, P, P],
        "ms_reset_plan_stats": [P],
        "ms_lcp_priority": [P, I32, P],
        "ms_plan_solve": [ctypes.POINTER(ms_plan_problem), U64, ctypes.c_double, P, I32, P, P, P, P, P],
        "ms_cache_update": [P, P, P],
        "ms_set_cache_policy": [P, I32, ctypes.c_double, ctypes.c_double, U64],
        "ms_set_copy_engine": [P, I32],
        "ms_dense": [P, P, I32, I32, I32, P, P, P],
        "ms_rope_kv": [P, I32, I32, I32, I32, I32, ctypes.c_double, P, P, P, I32, P],
        "ms_attention": [P, P, P, I32, I32, I32, I32, I32, I32, P, P],
        "ms_argmax": [P, I32, I32, P, P],
        "ms_embed": [P, P, I32, I32, I32, P, P],
        "ms_timeline_begin": [P, P, I32],
        "ms_timeline_end": [P, ctypes.POINTER(ms_interval), I32, ctypes.POINTER(I32)],
    }
    for name, args in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = ctypes.c_int
    lib.ms_destroy.argtypes = [P]
    lib.ms_destroy.restype = None
    lib.ms_last_error.argtypes = [P]
    lib.ms_last_error.restype = ctypes.c_char_p
    return lib


lib = _load()


class MoeSplitError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__("%s: %s" % (STATUS_NAMES.get(status, status), msg))
        self.status = status


def _ptr(x):
    """Device/host address of a tensor, numpy array or integer (None -> NULL)."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if isinstance(x, np.ndarray):
        assert x.flags.c_contiguous
        return x.ctypes.data
    if hasattr(x, "data_ptr"):
        assert x.is_contiguous()
        return x.data_ptr()
    raise TypeError("cannot take the address of %r" % type(x))


def _stream(s):
    if s is None:
        return None
    if isinstance(s, int):
        return s
    return s.cuda_stream


def model_desc(shape, max_tokens, n_buffer_slots=0, ffn_splits=0):
    """ms_model_desc from a synth.ModelShape-like object."""
    return ms_model_desc(shape.n_layers, shape.d_model, shape.d_ff, shape.n_experts, shape.top_k,
                         shape.n_shared, shape.d_ff_shared,
                         MS_BF16 if shape.dtype == "bf16" else MS_F32, shape.renormalize,
                         max_tokens, n_buffer_slots, ffn_splits, getattr(shape, "expert_bits", 0))


def _check(st, ctx=None, what=""):
    if st != MS_OK:
        msg = lib.ms_last_error(ctx).decode() if ctx else what
        raise MoeSplitError(st, msg or what)


# --------------------------------------------------------------- functions

def ms_query_sizes(desc):
    out = ms_sizes()
    _check(lib.ms_query_sizes(ctypes.byref(desc), ctypes.byref(out)), what="ms_query_sizes")
    return out


def ms_split_plan(desc, budget_bytes, r):
    units, tb, slots = ctypes.c_int32(), ctypes.c_uint64(), ctypes.c_int32()
    _check(lib.ms_split_plan(ctypes.byref(desc), int(budget_bytes), float(r), ctypes.byref(units),
                             ctypes.byref(tb), ctypes.byref(slots)), what="ms_split_plan")
    return units.value, tb.value, slots.value


def ms_create(desc, dev_pool, pool_bytes, host_store_experts=0):
    h = ctypes.c_void_p()
    _check(lib.ms_create(ctypes.byref(desc), _ptr(dev_pool), int(pool_bytes), int(host_store_experts),
                         ctypes.byref(h)), what="ms_create")
    return h


def ms_destroy(ctx):
    lib.ms_destroy(ctx)


def ms_last_error(ctx):
    return lib.ms_last_error(ctx).decode()


def ms_set_router(ctx, layer, w_r, bias=None):
    w_r = np.ascontiguousarray(w_r)
    b = None if bias is None else np.ascontiguousarray(bias, np.float32)
    _check(lib.ms_set_router(ctx, layer, _ptr(w_r), _ptr(b)), ctx)


def ms_set_expert(ctx, layer, e, w_gate, w_up, w_down):
    arrs = [np.ascontiguousarray(a) for a in (w_gate, w_up, w_down)]
    _check(lib.ms_set_expert(ctx, layer, e, *[_ptr(a) for a in arrs]), ctx)


def ms_set_expert_q(ctx, layer, e, codes, meta):
    """codes: (gate [F][d*b/8], up [F][d*b/8], down [d][F*b/8]) uint8;
    meta: (gate [F][d/64][2], up, down [d][F/64][2]) uint16 fp16 patterns."""
    cs = [np.ascontiguousarray(a, np.uint8) for a in codes]
    ms_ = [np.ascontiguousarray(a, np.uint16) for a in meta]
    _check(lib.ms_set_expert_q(ctx, layer, e, _ptr(cs[0]), _ptr(ms_[0]), _ptr(cs[1]), _ptr(ms_[1]),
                               _ptr(cs[2]), _ptr(ms_[2])), ctx)


def ms_alias_expert(ctx, layer, e, src_layer, src_e):
    _check(lib.ms_alias_expert(ctx, layer, e, src_layer, src_e), ctx)


def ms_set_shared_expert(ctx, layer, s, w_gate, w_up, w_down):
    arrs = [np.ascontiguousarray(a) for a in (w_gate, w_up, w_down)]
    _check(lib.ms_set_shared_expert(ctx, layer, s, *[_ptr(a) for a in arrs]), ctx)


def ms_configure(ctx, budget_bytes, r):
    b = np.ascontiguousarray(budget_bytes, np.uint64)
    rr = np.ascontiguousarray(r, np.float32)
    slots = np.zeros(len(b), np.int32)
    _check(lib.ms_configure(ctx, _ptr(b), _ptr(rr), _ptr(slots)), ctx)
    return slots


def ms_load_top(ctx, layer, e):
    _check(lib.ms_load_top(ctx, layer, e), ctx)


def ms_evict_top(ctx, layer, e):
    _check(lib.ms_evict_top(ctx, layer, e), ctx)


def ms_residency(ctx, layer, n_experts):
    out = np.zeros(n_experts, np.uint8)
    _check(lib.ms_residency(ctx, layer, _ptr(out)), ctx)
    return out


def ms_predict(ctx, layer, h_dev, T, stream, n_experts):
    order = np.zeros(n_experts, np.int32)
    score = np.zeros(n_experts, np.float32)
    _check(lib.ms_predict(ctx, layer, _ptr(h_dev), T, _stream(stream), _ptr(order), _ptr(score)), ctx)
    return order, score


def ms_prefetch(ctx, layer, experts):
    ex = np.ascontiguousarray(experts, np.int32)
    _check(lib.ms_prefetch(ctx, layer, _ptr(ex), len(ex)), ctx)


def ms_forward(ctx, layer, h_dev, T, y_dev, idx_dev, w_dev, flags=0, stream=None):
    _check(lib.ms_forward(ctx, layer, _ptr(h_dev), T, _ptr(y_dev), _ptr(idx_dev), _ptr(w_dev), flags,
                          _stream(stream)), ctx)


def ms_forward_noalloc(ctx, layer, h_dev, T, y_dev, idx_dev, w_dev, flags=0, stream=None):
    _check(lib.ms_forward_noalloc(ctx, layer, _ptr(h_dev), T, _ptr(y_dev), _ptr(idx_dev), _ptr(w_dev), flags,
                                  _stream(stream)), ctx)


def ms_sync(ctx):
    _check(lib.ms_sync(ctx), ctx)


def ms_drop_buffer(ctx):
    _check(lib.ms_drop_buffer(ctx), ctx)


def ms_residual_norm(ctx, h_dev, y_dev, T, out_dev, stream=None):
    _check(lib.ms_residual_norm(ctx, _ptr(h_dev), _ptr(y_dev), T, _ptr(out_dev), _stream(stream)), ctx)


def ms_plan_stats(ctx, layer, n_experts):
    """(hit [N+1], pred [N], pred_hit [N][N+1], (q, q_pred)) of one layer."""
    N = n_experts
    hit = np.zeros(N + 1)
    pred = np.zeros(N)
    ph = np.zeros((N, N + 1))
    tok = np.zeros(2, np.uint64)
    _check(lib.ms_plan_stats(ctx, layer, _ptr(hit), _ptr(pred), _ptr(ph), _ptr(tok)), ctx)
    return hit, pred, ph, (int(tok[0]), int(tok[1]))


def ms_reset_plan_stats(ctx):
    _check(lib.ms_reset_plan_stats(ctx), ctx)


def ms_lcp_priority(ctx, layer, n_experts):
    out = np.zeros(n_experts)
    _check(lib.ms_lcp_priority(ctx, layer, _ptr(out)), ctx)
    return out


def ms_plan_solve(n_layers, n_experts, top_k, expert_bytes, t_att_us, t_moe_us, t_head_us, t_load_us,
                  hit, pred, pred_hit, v_e_bytes, zeta=0.01, start_budgets=None, max_iter=100000):
    """Algorithm 1 over per-layer statistics (arrays [L][N+1], [L][N],
    [L][N][N+1]); returns dict(budgets, theta, cache, exposed_us, iters)."""
    L, N = n_layers, n_experts
    hit = np.ascontiguousarray(hit, np.float64).reshape(L, N + 1)
    pred = np.ascontiguousarray(pred, np.float64).reshape(L, N)
    pred_hit = np.ascontiguousarray(pred_hit, np.float64).reshape(L, N, N + 1)
    prob = ms_plan_problem(L, N, top_k, int(expert_bytes), float(t_att_us), float(t_moe_us), float(t_head_us),
                           float(t_load_us), hit.ctypes.data, pred.ctypes.data, pred_hit.ctypes.data)
    start = None if start_budgets is None else np.ascontiguousarray(start_budgets, np.uint64)
    budgets = np.zeros(L, np.uint64)
    theta = np.zeros(L)
    cache = np.zeros(L, np.int32)
    exposed = np.zeros(L)
    iters = ctypes.c_int32()
    _check(lib.ms_plan_solve(ctypes.byref(prob), int(v_e_bytes), float(zeta), _ptr(start), int(max_iter),
                             _ptr(budgets), _ptr(theta), _ptr(cache), _ptr(exposed), ctypes.byref(iters)),
           what="ms_plan_solve")
    return dict(budgets=budgets, theta=theta, cache=cache, exposed_us=exposed, iters=iters.value)


def ms_cache_update(ctx, budgets, r):
    b = np.ascontiguousarray(budgets, np.uint64)
    rr = np.ascontiguousarray(r, np.float32)
    _check(lib.ms_cache_update(ctx, _ptr(b), _ptr(rr)), ctx)


def ms_set_cache_policy(ctx, policy, rho=0.25, omega=128.0, seed=0):
    _check(lib.ms_set_cache_policy(ctx, int(policy), float(rho), float(omega), int(seed)), ctx)


def ms_set_copy_engine(ctx, engine):
    _check(lib.ms_set_copy_engine(ctx, int(engine)), ctx)


def ms_stats(ctx, layer):
    out = ms_layer_stats()
    _check(lib.ms_stats(ctx, layer, ctypes.byref(out)), ctx)
    return out.as_dict()


def ms_reset_stats(ctx):
    _check(lib.ms_reset_stats(ctx), ctx)


def ms_timeline_begin(ctx, stream, capacity=1 << 16):
    _check(lib.ms_timeline_begin(ctx, _stream(stream), capacity), ctx)


def ms_timeline_end(ctx, cap=1 << 16):
    buf = (ms_interval * cap)()
    n = ctypes.c_int32()
    _check(lib.ms_timeline_end(ctx, buf, cap, ctypes.byref(n)), ctx)
    return [dict(kind=INTERVAL_NAMES[buf[i].kind], layer=buf[i].layer, t0_ms=buf[i].t0_ms,
                 t1_ms=buf[i].t1_ms, bytes=int(buf[i].bytes)) for i in range(n.value)]


# ------------------------------------------------- decoder loop (stateless)

def ms_dense(x, w, T, n_in, n_out, y, add=None, stream=None):
    _check(lib.ms_dense(_ptr(x), _ptr(w), int(T), int(n_in), int(n_out), _ptr(y),
                        None if add is None else _ptr(add), _stream(stream)), what="ms_dense")


def ms_rope_kv(qkv, T, Hq, Hkv, D, pos0, base, q_out, k_cache, v_cache, max_ctx, stream=None):
    _check(lib.ms_rope_kv(_ptr(qkv), int(T), int(Hq), int(Hkv), int(D), int(pos0), float(base), _ptr(q_out),
                          _ptr(k_cache), _ptr(v_cache), int(max_ctx), _stream(stream)), what="ms_rope_kv")


def ms_attention(q, k_cache, v_cache, T, Hq, Hkv, D, pos0, max_ctx, out, stream=None):
    _check(lib.ms_attention(_ptr(q), _ptr(k_cache), _ptr(v_cache), int(T), int(Hq), int(Hkv), int(D), int(pos0),
                            int(max_ctx), _ptr(out), _stream(stream)), what="ms_attention")


def ms_argmax(x, T, n, idx_out, stream=None):
    _check(lib.ms_argmax(_ptr(x), int(T), int(n), _ptr(idx_out), _stream(stream)), what="ms_argmax")


def ms_embed(ids, table, n_vocab, T, d, out, stream=None):
    _check(lib.ms_embed(_ptr(ids), _ptr(table), int(n_vocab), int(T), int(d), _ptr(out), _stream(stream)),
           what="ms_embed")
