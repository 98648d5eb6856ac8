"""Pins of the CPU oracle against what the paper and mathematics fix.

Each test ties the oracle to something other than itself: hand-computed
instances of Eq. (2), brute-force sorting, the exactness of the top/bottom
split along the FFN intermediate axis, special cases that reduce to plain
library routines (numpy fp64 matmul, scipy softmax), and floating-point error
bounds of the canonical fp32 logit order.
"""
import json
import math
import os

import numpy as np
import pytest
import scipy.special

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "two_expert_cases.json")
U32 = 2.0 ** -24  # unit roundoff of fp32


def gamma(n, u=U32):
    return n * u / (1 - n * u)


def _golden():
    with open(GOLDEN) as f:
        return json.load(f)


def _pad_d(x, d_to, axis):
    """Zero-pad a small hand case to a feature width the canonical router
    order accepts (a multiple of 64); zeros change no sum."""
    pad = [(0, 0)] * x.ndim
    pad[axis] = (0, d_to - x.shape[axis])
    return np.pad(np.asarray(x, np.float32), pad)


def _hand_experts(g):
    ex = []
    for name in ("E0", "E1"):
        e = g["experts"][name]
        wg = _pad_d(np.array(e["w_gate"], np.float32), 64, 0)   # [d][F]
        wu = _pad_d(np.array(e["w_up"], np.float32), 64, 0)
        wd = _pad_d(np.array(e["w_down"], np.float32), 64, 1)   # [F][d]
        ex.append((wg, wu, wd))
    return ex


# ------------------------------------------------------- hand-computed cases

@pytest.mark.parametrize("case", [c["name"] for c in _golden()["cases"]])
def test_hand_cases(case):
    g = _golden()
    c = next(c for c in g["cases"] if c["name"] == case)
    ex = _hand_experts(g)
    h = _pad_d(np.array([c["h"]], np.float32), 64, 1)
    w_r = _pad_d(np.array(c["w_r"], np.float32), 64, 0)
    out = oracle.moe_layer(h, w_r, ex, c["K"], renormalize=c["renormalize"])
    assert out["idx"][0].tolist() == c["idx"]
    np.testing.assert_allclose(out["w"][0], c["w"], rtol=1e-7, atol=0)
    np.testing.assert_allclose(out["y"][0, :2], c["y"], rtol=1e-7, atol=1e-12)
    assert np.all(out["y"][0, 2:] == 0.0)


def test_hand_expert_outputs_and_split():
    g = _golden()
    ex = _hand_experts(g)
    h = _pad_d(np.array([[1, 2]], np.float32), 64, 1)[0]
    ref = g["expert_outputs_h12"]
    sp = g["split_r05_h12"]
    for i, name in enumerate(("E0", "E1")):
        wg, wu, wd = ex[i]
        full = oracle.expert_range(h, wg, wu, wd, 0, 2)
        top = oracle.expert_range(h, wg, wu, wd, 0, 1)
        bot = oracle.expert_range(h, wg, wu, wd, 1, 2)
        np.testing.assert_allclose(full[:2], ref[name], rtol=1e-15)
        np.testing.assert_allclose(top[:2], sp[name + "_top"], rtol=1e-15, atol=0)
        np.testing.assert_allclose(bot[:2], sp[name + "_bottom"], rtol=1e-15, atol=0)


def test_hand_activations():
    """The SwiGLU intermediate a_f = silu(h.G_f) * (h.U_f) of both hand
    experts at h = (1, 2), whole and unit by unit (range form)."""
    g = _golden()
    ex = _hand_experts(g)
    h = _pad_d(np.array([[1, 2]], np.float32), 64, 1)[0]
    ref = g["activations_h12"]
    for i, name in enumerate(("E0", "E1")):
        wg, wu, _ = ex[i]
        np.testing.assert_allclose(oracle.expert_act(h, wg, wu, 0, 2), ref[name], rtol=1e-15, atol=0)
        np.testing.assert_allclose(oracle.expert_act(h, wg, wu, 1, 2), ref[name][1:], rtol=1e-15, atol=0)
        np.testing.assert_allclose(oracle.expert_act(h, wg, wu, 0, 1), ref[name][:1], rtol=1e-15, atol=0)


# ------------------------------------------------- canonical fp32 logit order

@pytest.mark.parametrize("which", ["a", "b", "c"])
def test_canonical_order_golden(which):
    co = _golden()["canonical_order"]
    d = co["d"]
    h = np.zeros((1, d), np.float32)
    for j, v in co[which]["products"].items():
        h[0, int(j)] = v
    w_r = np.ones((d, 1), np.float32)
    got = oracle.router_logits(h, w_r)[0, 0]
    assert got == np.float32(co[which]["logit"])
    exact = float(h[0].astype(np.float64).sum())
    seq = np.float32(0)
    for x in h[0]:
        seq = np.float32(seq + x)
    if which in ("a", "c"):
        # the canonical order keeps both ones; left to right loses them
        assert got == exact and seq != got
    else:
        # the canonical order pairs each one with 2^24 first and loses both
        assert got != exact


@pytest.mark.parametrize("d,E,seed", [(64, 8, 0), (256, 8, 1), (2048, 64, 2), (4096, 8, 3)])
def test_logits_within_fp32_error_bound(d, E, seed):
    rng = np.random.default_rng(seed)
    T = 5
    h = rng.standard_normal((T, d)).astype(np.float32)
    w_r = (0.02 * rng.standard_normal((d, E))).astype(np.float32)
    bias = rng.standard_normal(E).astype(np.float32)
    got = oracle.router_logits(h, w_r, bias).astype(np.float64)
    exact = h.astype(np.float64) @ w_r.astype(np.float64) + bias
    absprod = np.abs(h.astype(np.float64)) @ np.abs(w_r.astype(np.float64)) + np.abs(bias)
    bound = gamma(d // 64 + 6 + 1) * absprod
    assert np.all(np.abs(got - exact) <= bound)
    # bf16-valued operands: products are exact in fp32, same bound applies
    assert np.all(np.abs(got - exact) <= bound)


def test_logits_reject_bad_width():
    with pytest.raises(ValueError):
        oracle.router_logits(np.zeros((1, 100), np.float32), np.zeros((100, 4), np.float32))


# ------------------------------------------------------------ top-k selection

def _brute_topk(logits, K):
    # full stable sort of (-logit, index): largest first, lower index on ties
    return np.stack([np.argsort(-row, kind="stable")[:K] for row in logits]).astype(np.int32)


@pytest.mark.parametrize("E,K,seed", [(8, 2, 0), (64, 6, 1), (128, 8, 2), (8, 8, 3), (1, 1, 4)])
def test_topk_matches_brute_force(E, K, seed):
    rng = np.random.default_rng(seed)
    T = 50
    logits = rng.standard_normal((T, E)).astype(np.float32)
    # adversarial ties: duplicated columns, coarse quantisation, all-equal rows
    if E > 1:
        logits[:, E // 2] = logits[:, 0]
    logits[10:20] = np.round(logits[10:20] * 2) / 2
    logits[20] = 0.0
    logits[21] = -3.0
    got = oracle.topk(logits, K)
    assert np.array_equal(got, _brute_topk(logits, K))
    assert got[20].tolist() == list(range(K))


def test_topk_prefers_logit_over_rounded_probability():
    # two logits far apart in fp32 whose softmax scores are equal after exp
    logits = np.array([[-200.0, -100.0, -200.0 + 1e-4, 0.0]], np.float32)
    assert oracle.topk(logits, 3)[0].tolist() == [3, 1, 2]


# ------------------------------------------------------------- gate weights

@pytest.mark.parametrize("renorm", [0, 1])
def test_gate_weights_against_scipy_softmax(renorm):
    rng = np.random.default_rng(7)
    T, E, K = 20, 64, 6
    logits = (3 * rng.standard_normal((T, E))).astype(np.float32)
    idx = oracle.topk(logits, K)
    w = oracle.gate_weights(logits, idx, renorm)
    p = scipy.special.softmax(logits.astype(np.float64), axis=1)
    sel = np.take_along_axis(p, idx.astype(np.int64), axis=1)
    ref = sel / sel.sum(axis=1, keepdims=True) if renorm else sel
    np.testing.assert_allclose(w, ref, rtol=1e-13)
    if renorm:
        np.testing.assert_allclose(w.sum(axis=1), 1.0, rtol=1e-14)
    # selected weights are non-increasing in selection order
    assert np.all(np.diff(w, axis=1) <= 1e-15)


# -------------------------------------------------------------- split identity

def _rand_expert(rng, d, F, std=0.05):
    return tuple(x.astype(np.float32) for x in (
        std * rng.standard_normal((d, F)), std * rng.standard_normal((d, F)),
        std * rng.standard_normal((F, d))))


@pytest.mark.parametrize("r", [0.0, 0.25, 0.5, 0.75, 1.0])
def test_split_identity(r):
    rng = np.random.default_rng(11)
    d, F = 64, 512
    wg, wu, wd = _rand_expert(rng, d, F)
    h = rng.standard_normal(d).astype(np.float32)
    F_top = oracle.top_units(r, F)
    full = oracle.expert_range(h, wg, wu, wd, 0, F)
    # continued accumulation: bottom onto the top's running sum -> bitwise equal
    acc = oracle.expert_range(h, wg, wu, wd, 0, F_top)
    oracle.expert_range(h, wg, wu, wd, F_top, F, acc=acc)
    assert np.array_equal(acc, full)
    # separately summed partials: equal within the fp64 summation bound
    top = oracle.expert_range(h, wg, wu, wd, 0, F_top)
    bot = oracle.expert_range(h, wg, wu, wd, F_top, F)
    a = oracle.expert_act(h, wg, wu, 0, F)
    bound = gamma(F + 1, 2.0 ** -53) * (np.abs(a)[:, None] * np.abs(wd.astype(np.float64))).sum(0)
    assert np.all(np.abs(top + bot - full) <= bound)


@pytest.mark.parametrize("r,F,expect", [
    (0.0, 512, 0), (1.0, 512, 512), (0.5, 512, 256),
    (0.25, 14336, 3584), (0.5, 14336, 7168), (0.75, 14336, 10752),
    (0.5, 1408, 704), (0.5, 768, 384),
    (0.4, 1408, 576),      # 8.8 chunks -> 9
    (0.1, 160, 0),         # 0.25 chunk -> 0
    (0.99, 100, 100),      # clamped to F
])
def test_top_units(r, F, expect):
    assert oracle.top_units(r, F) == expect


# ------------------------------------------ special cases vs library routines

def _swiglu_np(h, ex):
    wg, wu, wd = (x.astype(np.float64) for x in ex)
    h = h.astype(np.float64)
    g = h @ wg
    u = h @ wu
    a = g / (1.0 + np.exp(-g)) * u
    return a @ wd


def test_single_expert_is_plain_swiglu():
    rng = np.random.default_rng(5)
    d, F, T = 128, 192, 3
    ex = _rand_expert(rng, d, F)
    h = rng.standard_normal((T, d)).astype(np.float32)
    w_r = rng.standard_normal((d, 1)).astype(np.float32)
    out = oracle.moe_layer(h, w_r, [ex], 1)
    assert np.all(out["idx"] == 0) and np.all(out["w"] == 1.0)
    np.testing.assert_allclose(out["y"], _swiglu_np(h, ex), rtol=1e-11, atol=1e-13)


def test_all_experts_is_dense_softmax_mixture():
    rng = np.random.default_rng(6)
    d, F, E, T = 64, 128, 4, 4
    exs = [_rand_expert(rng, d, F) for _ in range(E)]
    h = rng.standard_normal((T, d)).astype(np.float32)
    w_r = (0.3 * rng.standard_normal((d, E))).astype(np.float32)
    out = oracle.moe_layer(h, w_r, exs, E, renormalize=True)
    p = scipy.special.softmax(out["logits"].astype(np.float64), axis=1)
    ref = sum(p[:, [e]] * _swiglu_np(h, exs[e]) for e in range(E))
    np.testing.assert_allclose(out["y"], ref, rtol=1e-10, atol=1e-12)


def test_shared_experts_add_with_weight_one():
    rng = np.random.default_rng(8)
    d, F, E, T = 64, 64, 4, 2
    exs = [_rand_expert(rng, d, F) for _ in range(E)]
    sh = [_rand_expert(rng, d, 128) for _ in range(2)]
    h = rng.standard_normal((T, d)).astype(np.float32)
    w_r = rng.standard_normal((d, E)).astype(np.float32)
    base = oracle.moe_layer(h, w_r, exs, 2)
    with_sh = oracle.moe_layer(h, w_r, exs, 2, shared=sh)
    ref = base["y"] + _swiglu_np(h, sh[0]) + _swiglu_np(h, sh[1])
    np.testing.assert_allclose(with_sh["y"], ref, rtol=1e-11, atol=1e-13)


def test_zero_input_gives_zero_output():
    rng = np.random.default_rng(9)
    d, F, E = 64, 64, 8
    exs = [_rand_expert(rng, d, F) for _ in range(E)]
    out = oracle.moe_layer(np.zeros((2, d), np.float32), rng.standard_normal((d, E)).astype(np.float32), exs, 2)
    assert np.all(out["y"] == 0.0)
    assert out["idx"][0].tolist() == [0, 1]   # all logits 0 -> lowest indices


def test_token_subset_matches_full():
    rng = np.random.default_rng(10)
    d, F, E, T = 64, 64, 8, 6
    exs = [_rand_expert(rng, d, F) for _ in range(E)]
    h = rng.standard_normal((T, d)).astype(np.float32)
    w_r = rng.standard_normal((d, E)).astype(np.float32)
    full = oracle.moe_layer(h, w_r, exs, 3)
    sub = oracle.moe_layer(h, w_r, exs, 3, tokens=[4, 1])
    assert np.array_equal(sub["y"], full["y"][[4, 1]])


# ----------------------------------------------------------------- prediction

def test_predict_order_and_scores():
    rng = np.random.default_rng(12)
    d, E, T = 128, 16, 7
    h = rng.standard_normal((T, d)).astype(np.float32)
    w = (0.1 * rng.standard_normal((d, E))).astype(np.float32)
    score, order = oracle.predict(h, w)
    logits = oracle.router_logits(h, w).astype(np.float64)
    ref = scipy.special.softmax(logits, axis=1).sum(0)
    np.testing.assert_allclose(score, ref, rtol=1e-13)
    assert math.isclose(score.sum(), T, rel_tol=1e-13)
    assert np.array_equal(order, np.argsort(-score, kind="stable"))
    # one token: the ranking is the ranking of its logits
    s1, o1 = oracle.predict(h[:1], w)
    assert np.array_equal(o1, oracle.topk(oracle.router_logits(h[:1], w), E)[0])


def test_nan_logits_read_as_minus_infinity():
    """Reading: a NaN router logit ranks as -inf (lower index first among
    equal values) and has softmax score 0.  Row (NaN, 0.5, NaN, -inf, 2):
    ranking e4, e1, then e0, e2, e3 tied at -inf; scores of e4 and e1 are
    1 / (1 + e^-1.5) and 1 / (1 + e^1.5), the rest 0, with or without
    renormalisation; the prediction ranks the same way."""
    row = np.array([[np.nan, 0.5, np.nan, -np.inf, 2.0]], np.float32)
    assert oracle.topk(row, 5)[0].tolist() == [4, 1, 0, 2, 3]
    idx = oracle.topk(row, 2)
    assert idx[0].tolist() == [4, 1]
    p4, p1 = 1.0 / (1.0 + math.exp(-1.5)), 1.0 / (1.0 + math.exp(1.5))
    for renorm in (0, 1):
        np.testing.assert_allclose(oracle.gate_weights(row, idx, renorm)[0], [p4, p1], rtol=1e-15)
    w5 = oracle.gate_weights(row, oracle.topk(row, 5), 1)[0]
    np.testing.assert_allclose(w5, [p4, p1, 0.0, 0.0, 0.0], rtol=1e-15, atol=0)
    # prediction from logits through the router: a NaN router column
    d = 64
    h = np.zeros((2, d), np.float32)
    h[:, 0] = 1.0
    w = np.zeros((d, 5), np.float32)
    w[0] = [np.nan, 0.5, np.nan, -np.inf, 2.0]
    score, order = oracle.predict(h, w)
    assert order.tolist() == [4, 1, 0, 2, 3]
    np.testing.assert_allclose(score, [0.0, 2 * p1, 0.0, 0.0, 2 * p4], rtol=1e-15, atol=0)


def test_predict_ties_lower_index_first():
    d, E = 64, 6
    s, o = oracle.predict(np.zeros((3, d), np.float32), np.ones((d, E), np.float32))
    assert o.tolist() == list(range(E))
    np.testing.assert_allclose(s, 3.0 / E)


# ------------------------------------------------------------------- grouping

@pytest.mark.parametrize("T,K,E,seed", [(1, 2, 8, 0), (4, 2, 8, 1), (37, 6, 64, 2), (512, 8, 128, 3), (0, 2, 8, 4)])
def test_group_matches_stable_sort(T, K, E, seed):
    rng = np.random.default_rng(seed)
    idx = np.array([rng.permutation(E)[:K] for _ in range(T)], np.int32).reshape(T, K)
    offsets, perm = oracle.group(idx, E)
    flat = idx.reshape(-1)
    assert np.array_equal(perm, np.argsort(flat, kind="stable"))
    assert np.array_equal(offsets, np.concatenate([[0], np.cumsum(np.bincount(flat, minlength=E))]))


# ----------------------------------------------------------------------- glue

def test_residual_rmsnorm():
    rng = np.random.default_rng(13)
    h = rng.standard_normal((3, 64))
    y = rng.standard_normal((3, 64))
    out = oracle.residual_rmsnorm(h, y, eps=1e-6)
    x = h + y
    ms = (x * x).mean(1)
    np.testing.assert_allclose((out * out).mean(1), ms / (ms + 1e-6), rtol=1e-12)
    # parallel to h + y with a positive factor
    ratio = out / x
    np.testing.assert_allclose(ratio, ratio[:, :1] * np.ones_like(ratio), rtol=1e-12)
    assert np.all(ratio > 0)
