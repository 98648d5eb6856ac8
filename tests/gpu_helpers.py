"""Shared helpers of the GPU parity tests (tolerances and oracle calls)."""
import numpy as np

import oracle


def check_close(gpu, ref, dtype, what="y"):
    """Tolerance of the layer outputs: bf16 |gpu - oracle| <= 1e-2 max|oracle|
    + 1e-3; fp32 <= 1e-5 max|oracle| (max over the compared tensor)."""
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    assert gpu.shape == ref.shape, (gpu.shape, ref.shape)
    if ref.size == 0:
        return 0.0
    m = float(np.max(np.abs(ref)))
    bound = 1e-2 * m + 1e-3 if dtype == "bf16" else 1e-5 * m
    err = float(np.max(np.abs(gpu - ref)))
    assert err <= bound, "%s: max err %.3e > bound %.3e (max|ref| %.3e)" % (what, err, bound, m)
    return err / max(m, 1e-30)


def quant_weights(rig, layer):
    """fp64 dequantized experts of a b-bit rig's layer (cached on the rig)."""
    from oracle import quant
    cache = rig.__dict__.setdefault("_deq", {})
    key = layer % rig.n_sets
    if key not in cache:
        s = rig.shape
        cache[key] = [quant.expert_weights(q.codes, q.meta, q.bits, s.d_model, s.d_ff)
                      for q in rig.layer_experts(layer)]
    return cache[key]


def oracle_layer(rig, layer, h_f32, tokens=None):
    s = rig.shape
    if getattr(s, "expert_bits", 0):
        from oracle import quant
        return quant.moe_layer(h_f32, rig.routers[layer], quant_weights(rig, layer), s.top_k,
                               renormalize=s.renormalize, bias=rig.biases[layer], tokens=tokens)
    return oracle.moe_layer(h_f32, rig.routers[layer], rig.layer_experts(layer), s.top_k,
                            renormalize=s.renormalize, bias=rig.biases[layer],
                            shared=rig.shared[layer], tokens=tokens)


def check_layer(rig, layer, h_f32, y, idx, w, tokens=None):
    """idx bit-exact, w within fp32 rounding, y within the dtype tolerance."""
    ref = oracle_layer(rig, layer, h_f32, tokens)
    T = h_f32.shape[0]
    idx_g = idx[:T].cpu().numpy()
    assert np.array_equal(idx_g, ref["idx"]), "selected experts differ"
    np.testing.assert_allclose(w[:T].cpu().numpy(), ref["w"], rtol=2e-6, atol=1e-7)
    rows = ref["tokens"]
    return check_close(y[:T].cpu().numpy()[rows], ref["y"], rig.shape.dtype)


def check_prediction(order, score, ref_score, tol=2e-6):
    """The ranking is unique only where scores differ by more than rounding:
    scores match the oracle's, the order is a permutation sorted by the
    returned scores (lower index first on equal), and consistent with the
    oracle's scores up to the tolerance."""
    E = len(ref_score)
    np.testing.assert_allclose(score, ref_score, rtol=0, atol=tol * max(1.0, float(np.sum(ref_score))))
    assert sorted(order.tolist()) == list(range(E))
    for a, b in zip(order[:-1], order[1:]):
        assert score[a] > score[b] or (score[a] == score[b] and a < b)
        assert ref_score[a] >= ref_score[b] - 2 * tol * max(1.0, float(np.sum(ref_score)))
