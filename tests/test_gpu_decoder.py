"""GPU parity of the decoder loop around the MoE layer against the decoder
oracle: the dense projection, rotary embedding with the cache append,
causal grouped-query attention (every group size, several positions),
arg max and embedding gather, and a two-layer decoder (prefill then greedy
decode, prediction and prefetch on) whose every layer is checked
teacher-forced: the oracle gets each layer's GPU input and builds its own
key/value caches from them."""
import numpy as np
import pytest

import synth
from gpu_helpers import check_close

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _bf16(a):
    """(device bf16 tensor, exact fp64 values) of an fp32 array."""
    from workload import to_device
    raw, f = synth.storage(np.ascontiguousarray(a, np.float32), "bf16")
    return to_device(raw, "bf16"), f.astype(np.float64)


# T >= 16 with n_in a multiple of 32 takes the matrix-core kernel (ragged
# 64-token and 64-output tiles); the rest the fma-chain kernel
@pytest.mark.parametrize("T,n_in,n_out", [(1, 256, 13), (3, 4096, 100), (9, 512, 64), (2, 8192, 24),
                                          (16, 256, 13), (17, 1024, 70), (64, 4096, 100), (130, 512, 200),
                                          (40, 8192, 24), (20, 264, 33)])
def test_dense_matches_numpy(T, n_in, n_out):
    from paper_2509_08342_amd import moesplit as ms
    rng = np.random.default_rng(T + n_in)
    x, xf = _bf16(rng.standard_normal((T, n_in)))
    w, wf = _bf16(0.02 * rng.standard_normal((n_out, n_in)))
    add = torch.from_numpy(rng.standard_normal((T, n_out)).astype(np.float32)).cuda()
    y = torch.empty(T, n_out, dtype=torch.float32, device="cuda")
    ms.ms_dense(x, w, T, n_in, n_out, y, add, torch.cuda.current_stream())
    torch.cuda.synchronize()
    ref = xf @ wf.T + add.cpu().numpy()
    bound = 1e-5 * (np.abs(xf) @ np.abs(wf).T).max() + 1e-6
    assert np.max(np.abs(y.cpu().numpy() - ref)) <= bound


@pytest.mark.parametrize("pos0,T", [(0, 1), (7, 3), (200, 2)])
def test_rope_kv_matches_oracle(pos0, T):
    from oracle import decoder as od
    from paper_2509_08342_amd import moesplit as ms
    Hq, Hkv, D, base, max_ctx = 4, 2, 64, 1e4, 256
    rng = np.random.default_rng(pos0)
    qkv = rng.standard_normal((T, (Hq + 2 * Hkv) * D)).astype(np.float32)
    q = torch.empty(T, Hq, D, dtype=torch.bfloat16, device="cuda")
    kc = torch.zeros(Hkv, max_ctx, D, dtype=torch.bfloat16, device="cuda")
    vc = torch.zeros_like(kc)
    ms.ms_rope_kv(torch.from_numpy(qkv).cuda(), T, Hq, Hkv, D, pos0, base, q, kc, vc, max_ctx,
                  torch.cuda.current_stream())
    torch.cuda.synchronize()
    qg, kg, vg = q.float().cpu().numpy(), kc.float().cpu().numpy(), vc.float().cpu().numpy()
    for t in range(T):
        p = pos0 + t
        rq = od.bf16_round(od.rope(qkv[t, :Hq * D].reshape(Hq, D), p, base))
        rk = od.bf16_round(od.rope(qkv[t, Hq * D:(Hq + Hkv) * D].reshape(Hkv, D), p, base))
        rv = od.bf16_round(qkv[t, (Hq + Hkv) * D:].reshape(Hkv, D))
        # fp32 products against fp64: at most one bf16 rounding step apart
        for got, ref in ((qg[t], rq), (kg[:, p], rk)):
            assert np.all(np.abs(got - ref) <= 2.0 ** -7 * np.abs(ref) + 1e-30)
        assert np.array_equal(vg[:, p], rv)
    untouched = np.ones(max_ctx, bool)
    untouched[pos0:pos0 + T] = False
    assert not np.any(kg[:, untouched]) and not np.any(vg[:, untouched])


@pytest.mark.parametrize("G", [1, 2, 4, 8])
@pytest.mark.parametrize("pos0,T", [(0, 1), (5, 3), (300, 2)])
def test_attention_matches_oracle(G, pos0, T):
    from oracle import decoder as od
    from paper_2509_08342_amd import moesplit as ms
    Hkv, D, max_ctx = 2, 128, 512
    Hq = G * Hkv
    rng = np.random.default_rng(100 * G + pos0)
    q, qf = _bf16(rng.standard_normal((T, Hq, D)))
    kc, kf = _bf16(rng.standard_normal((Hkv, max_ctx, D)))
    vc, vf = _bf16(rng.standard_normal((Hkv, max_ctx, D)))
    out = torch.empty(T, Hq, D, dtype=torch.bfloat16, device="cuda")
    ms.ms_attention(q, kc, vc, T, Hq, Hkv, D, pos0, max_ctx, out, torch.cuda.current_stream())
    torch.cuda.synchronize()
    got = out.float().cpu().numpy()
    for t in range(T):
        ref = od.attend(qf[t], kf, vf, pos0 + t + 1)
        check_close(got[t], ref, "bf16", "attention t=%d" % t)


def test_attention_rejects_what_it_cannot_hold():
    from paper_2509_08342_amd import moesplit as ms
    q = torch.zeros(1, 8, 128, dtype=torch.bfloat16, device="cuda")
    kc = torch.zeros(1, 8192, 128, dtype=torch.bfloat16, device="cuda")
    out = torch.empty_like(q)
    with pytest.raises(ms.MoeSplitError) as ei:
        ms.ms_attention(q, kc, kc, 1, 8, 1, 128, 4000, 8192, out)
    assert ei.value.status == ms.MS_E_UNSUPPORTED
    with pytest.raises(ms.MoeSplitError) as ei:
        ms.ms_attention(q, kc, kc, 1, 8, 1, 128, 8192, 8192, out)
    assert ei.value.status == ms.MS_E_INVALID


def test_argmax_and_embed():
    from paper_2509_08342_amd import moesplit as ms
    x = torch.tensor([[1.0, 5.0, 5.0, -1.0], [0.0, 0.0, 0.0, 0.0], [-3.0, -2.0, -9.0, -2.0]], device="cuda")
    idx = torch.empty(3, dtype=torch.int32, device="cuda")
    ms.ms_argmax(x, 3, 4, idx)
    torch.cuda.synchronize()
    assert idx.cpu().tolist() == [1, 0, 1]
    rng = np.random.default_rng(9)
    big = torch.from_numpy(rng.standard_normal((2, 70001)).astype(np.float32)).cuda()
    ms.ms_argmax(big, 2, 70001, idx)
    torch.cuda.synchronize()
    assert idx[:2].cpu().tolist() == np.argmax(big.cpu().numpy(), axis=1).tolist()
    table, tf = _bf16(rng.standard_normal((50, 64)))
    ids = torch.tensor([3, 49, 0], dtype=torch.int32, device="cuda")
    out = torch.empty(3, 64, dtype=torch.bfloat16, device="cuda")
    ms.ms_embed(ids, table, 50, 3, 64, out)
    torch.cuda.synchronize()
    assert np.array_equal(out.float().cpu().numpy(), tf[[3, 49, 0]])


def test_decoder_layers_match_oracle():
    import oracle
    from oracle import decoder as od
    from decoder import Decoder
    from paper_2509_08342_amd import moesplit as ms
    from workload import top_bytes
    shape = synth.ModelShape("dec-tiny", 2, 256, 512, 8, 2, "bf16")
    attn = synth.TINY_ATTN
    P, n_dec = 12, 3
    with Decoder(shape, attn, seed=4, n_sets=2, max_tokens=P, max_ctx=64,
                 budget_total=2 * 8 * shape.expert_bytes) as dec:
        rig = dec.stack.rig
        dec.stack.configure(0.5, 2 * 4 * top_bytes(rig, 0.5))
        for l in range(2):
            rig.load_tops(l, [0, 1, 2, 3])
        ms.ms_sync(dec.ctx)
        cfg = dict(Hq=attn.n_heads, Hkv=attn.n_kv_heads, D=attn.head_dim, base=attn.rope_base)
        caches = [od.Cache(attn.n_kv_heads, 64, attn.head_dim) for _ in range(2)]
        prompt = synth.prompt_tokens(attn, 4, P)
        ids = torch.from_numpy(prompt).cuda()
        x = torch.empty(P, shape.d_model, dtype=torch.bfloat16, device="cuda")
        dec.embed_ids(ids, P, x)
        torch.cuda.synchronize()
        assert np.array_equal(x.float().cpu().numpy(), dec.embed_f32[prompt])
        x1 = torch.empty(1, shape.d_model, dtype=torch.bfloat16, device="cuda")
        for step in range(1 + n_dec):
            T = P if step == 0 else 1
            pos0 = dec.pos
            cap = dec.step(x if step == 0 else x1, T, capture=(0, 1))
            torch.cuda.synchronize()
            for l in range(2):
                c = cap[l]
                qf, of = dec.f32[l % dec.n_sets]
                moe = od.moe_from_layer_oracle(rig.routers[l], rig.layer_experts(l), shape.top_k, bias=rig.biases[l])
                xo, h = od.layer(c["x"], dict(w_qkv=qf, w_o=of), caches[l], pos0, cfg, moe)
                check_close(c["h"], h, "bf16", "step %d layer %d h" % (step, l))
                # routing of the GPU's own h is exact; its output within tolerance
                ref = oracle.moe_layer(c["h"].astype(np.float32), rig.routers[l], rig.layer_experts(l), shape.top_k,
                                       bias=rig.biases[l])
                assert np.array_equal(c["idx"], ref["idx"])
                check_close(c["x_out"], od.bf16_round(od.rmsnorm(c["h"] + ref["y"])), "bf16",
                            "step %d layer %d x_out" % (step, l))
            # head on the GPU's final state; the greedy token where the top two are apart
            last = dec.final[T - 1:T].float().cpu().numpy()
            logits, am = od.head_argmax(last, dec.head_f32)
            got = dec.logits.cpu().numpy()
            check_close(got, logits, "bf16", "logits")
            top2 = np.sort(logits[0])[-2:]
            if top2[1] - top2[0] > 1e-3 * np.abs(logits).max():
                assert int(dec.ids[0].item()) == int(am[0])
            dec.embed_ids(dec.ids, 1, x1)
        assert dec.pos == P + n_dec
