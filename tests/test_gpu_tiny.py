"""GPU parity on the tiny fp32 layer (d=256, F=512, E=8, top-2, T=4, r=0.5,
tops of experts 0-3 resident, seed 0), plus residency invariance, the fixed
logit order, prediction, edge cases and error codes."""
import itertools

import numpy as np
import pytest

import synth
from gpu_helpers import check_layer, check_prediction, check_close

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def rig():
    from workload import SplitRig, top_bytes
    import workload
    r = SplitRig(synth.TINY, seed=0, max_tokens=64, budget_bytes=8 * synth.TINY.expert_bytes)
    r.top_bytes = lambda ratio: top_bytes(r, ratio)
    yield r
    r.close()


def _setup(rig, r_ratio, tops, budget_tops=8):
    from paper_2509_08342_amd import moesplit as ms
    tb = rig.top_bytes(r_ratio)
    slots = rig.configure([budget_tops * tb], [r_ratio])
    rig.load_tops(0, tops)
    return slots


def _run(rig, h, T, flags=0):
    y, idx, w = rig.outputs(T)
    rig.forward(0, h, T, y, idx, w, flags)
    torch.cuda.synchronize()
    return y, idx, w


def test_tiny_layer_parity(rig):
    from paper_2509_08342_amd import moesplit as ms
    slots = _setup(rig, 0.5, [0, 1, 2, 3], budget_tops=4)
    assert slots.tolist() == [4]
    assert ms.ms_residency(rig.ctx, 0, 8).tolist() == [1, 1, 1, 1, 0, 0, 0, 0]
    h, hf = rig.hidden(4)
    y, idx, w = _run(rig, h, 4)
    check_layer(rig, 0, hf, y, idx, w)
    st = ms.ms_stats(rig.ctx, 0)
    assert st["forwards"] >= 1 and st["alpha"] + st["beta"] + st["gamma"] == st["experts_active"]


@pytest.mark.parametrize("T", [1, 3, 5, 16, 37, 64])
def test_tiny_ragged_token_counts(rig, T):
    _setup(rig, 0.5, [0, 1, 2, 3])
    h, hf = rig.hidden(T, tag=T)
    y, idx, w = _run(rig, h, T)
    check_layer(rig, 0, hf, y, idx, w)



@pytest.mark.parametrize("T", [24, 37, 64])
def test_tiny_multi_tile_experts_independent_of_residency(rig, T):
    """Experts with more tokens than one FFN tile spread their tiles over
    several work-groups, and each tile takes the shape of its real token
    count (read on the device).  Resident launches size their grid before
    the routing is known, streamed ones after it; every token's sums run in
    the same order either way, so outputs are bitwise equal across residency
    states and match the oracle."""
    h, hf = rig.hidden(T, tag=700 + T)
    outs = []
    for r, tops in ((0.5, [0, 1, 2, 3]), (0.0, []), (1.0, list(range(8))), (0.5, [4, 5, 6, 7])):
        _setup(rig, r, tops)
        y, idx, w = _run(rig, h, T)
        if not outs:
            check_layer(rig, 0, hf, y, idx, w)
            counts = np.bincount(idx.cpu().numpy()[:T].reshape(-1), minlength=8)
            assert counts.max() > 8, counts  # some expert's tokens span two tiles
            assert (counts % 8 != 0).any(), counts  # and some tile holds fewer than 8
        outs.append(y.cpu().numpy()[:T])
    for o in outs[1:]:
        assert np.array_equal(o, outs[0])

# bf16, d = 512 (8 k pieces), F = 512 (8 chunks), 4 experts, top-2: large
# enough for the matrix-core tiles' k split and column blocks, small enough
# for the oracle; at these T every expert has 12-36 rows
MT_BF16 = synth.ModelShape("multi-tile-bf16", 1, 512, 512, 4, 2, "bf16")


@pytest.mark.parametrize("T", [37, 50, 64])
def test_bf16_multi_tile_experts_independent_of_residency(T):
    """bf16 decode path (forced also where the token count would choose the
    prefill path): tiles of 5-16 rows run on the matrix cores in both
    phases, tiles of 1-4 rows on fma chains, and an expert with more rows
    than one tile spreads over several work-groups.  Outputs match the
    oracle and are bitwise equal across residency states."""
    from paper_2509_08342_amd import moesplit as ms
    from workload import SplitRig, top_bytes
    s = MT_BF16
    with SplitRig(s, seed=5, max_tokens=64, budget_bytes=s.n_experts * s.expert_bytes) as r:
        h, hf = r.hidden(T, tag=900 + T)
        outs = []
        for ratio, tops in ((0.5, [0, 1]), (0.0, []), (1.0, list(range(4))), (0.5, [2, 3]), (0.25, [1, 3])):
            r.configure([s.n_experts * top_bytes(r, ratio)], [ratio])
            r.load_tops(0, tops)
            y, idx, w = r.outputs(T)
            r.forward(0, h, T, y, idx, w, ms.MS_FWD_NO_MATRIX_CORES)
            torch.cuda.synchronize()
            if not outs:
                check_layer(r, 0, hf, y, idx, w)
                counts = np.bincount(idx.cpu().numpy()[:T].reshape(-1), minlength=4)
                assert counts.max() > 16, counts  # some expert spans two tiles
                tails = counts[counts > 0] % 16
                assert ((tails > 4) | (tails == 0)).any() and ((tails >= 1) & (tails <= 4)).any(), counts
            outs.append(y.cpu().numpy()[:T])
        for o in outs[1:]:
            assert np.array_equal(o, outs[0])


def test_tiny_outputs_independent_of_residency_and_split(rig):
    """Eq. (2) output must not depend on r or on which tops are cached: every
    residency subset at r=0.5, and several subsets at r in {0,.25,.75,1}
    (r=0: prefetch only, r=1: whole experts cached) give bitwise equal y."""
    h, hf = rig.hidden(4, tag=99)
    _setup(rig, 0.5, [0, 1, 2, 3])
    y0, idx0, w0 = _run(rig, h, 4)
    check_layer(rig, 0, hf, y0, idx0, w0)
    y0 = y0.cpu().numpy()
    cases = [(0.5, [e for e in range(8) if (m >> e) & 1]) for m in range(256)]
    rng = np.random.default_rng(1)
    for r in (0.0, 0.25, 0.75, 1.0):
        subsets = [[], list(range(8))] + [sorted(rng.choice(8, 3, replace=False).tolist()) for _ in range(3)]
        cases += [(r, s) for s in subsets]
    for r, tops in cases:
        if r == 0.0 and tops:
            continue  # no top segment exists at r = 0
        _setup(rig, r, tops)
        y, idx, w = _run(rig, h, 4)
        assert np.array_equal(idx.cpu().numpy(), idx0.cpu().numpy())
        assert np.array_equal(y.cpu().numpy(), y0), "r=%s tops=%s" % (r, tops)


def test_tiny_repeated_forwards_reuse_buffer(rig):
    from paper_2509_08342_amd import moesplit as ms
    _setup(rig, 0.5, [0, 1])
    h, hf = rig.hidden(4, tag=7)
    y1, _, _ = _run(rig, h, 4)
    ms.ms_reset_stats(rig.ctx)
    y2, idx, w = _run(rig, h, 4)
    st = ms.ms_stats(rig.ctx, 0)
    assert np.array_equal(y1.cpu().numpy(), y2.cpu().numpy())
    # the second pass finds its missing parts still in the staging buffer
    # unless more experts were active than buffer slots
    if st["beta"] + st["gamma"] <= 4:
        assert st["bytes_miss"] == 0
    check_layer(rig, 0, hf, y2, idx, w)


def test_tiny_prediction_matches_oracle(rig):
    import oracle
    from paper_2509_08342_amd import moesplit as ms
    _setup(rig, 0.5, [0, 1, 2, 3])
    for T in (1, 4, 33):
        h, hf = rig.hidden(T, tag=200 + T)
        order, score = ms.ms_predict(rig.ctx, 0, h, T, torch.cuda.current_stream(), 8)
        ref_score, ref_order = oracle.predict(hf, rig.routers[0], rig.biases[0])
        check_prediction(order, score, ref_score)


def test_tiny_predict_next_and_prefetch_keep_outputs(rig):
    from paper_2509_08342_amd import moesplit as ms
    _setup(rig, 0.5, [0, 1, 2, 3])
    steps = synth.walk(synth.TINY, 0, 12, T=2)
    ref = []
    for raw, f in steps:
        h = torch.from_numpy(raw).cuda()
        y, idx, w = _run(rig, h, 2)
        ref.append(y.cpu().numpy())
    _setup(rig, 0.5, [0, 1, 2, 3])
    ms.ms_reset_stats(rig.ctx)
    for i, (raw, f) in enumerate(steps):
        h = torch.from_numpy(raw).cuda()
        y, idx, w = _run(rig, h, 2, ms.MS_FWD_PREDICT_NEXT)
        assert np.array_equal(y.cpu().numpy(), ref[i])
    st = ms.ms_stats(rig.ctx, 0)
    assert st["predictions"] == len(steps) - 1
    # explicit prefetch of every expert, then a forward: still the same output
    ms.ms_prefetch(rig.ctx, 0, list(range(8)))
    h = torch.from_numpy(steps[0][0]).cuda()
    y, idx, w = _run(rig, h, 2)
    assert np.array_equal(y.cpu().numpy(), ref[0])


def test_tiny_copy_engines_give_equal_outputs(rig):
    """Segment copies by the copy kernel (default) and by the DMA engines
    move the same bytes: same outputs bitwise and the same copy statistics,
    over forwards with misses, prediction and prefetch."""
    from paper_2509_08342_amd import moesplit as ms
    steps = synth.walk(synth.TINY, 4, 10, T=3)
    runs = []
    for engine in (ms.MS_COPY_DMA, ms.MS_COPY_KERNEL):
        ms.ms_set_copy_engine(rig.ctx, engine)
        _setup(rig, 0.5, [1, 3])
        ms.ms_drop_buffer(rig.ctx)
        ms.ms_reset_stats(rig.ctx)
        ys = []
        for i, (raw, f) in enumerate(steps):
            h = torch.from_numpy(raw).cuda()
            y, idx, w = _run(rig, h, 3, ms.MS_FWD_PREDICT_NEXT if i % 2 else 0)
            ys.append(y.cpu().numpy().copy())
            if i == 4:
                check_layer(rig, 0, f, y, idx, w)
                ms.ms_drop_buffer(rig.ctx)
        st = ms.ms_stats(rig.ctx, 0)
        runs.append((ys, st["bytes_miss"], st["bytes_prefetch"]))
    with pytest.raises(RuntimeError):
        ms.ms_set_copy_engine(rig.ctx, 7)
    assert all(np.array_equal(a, b) for a, b in zip(runs[0][0], runs[1][0]))
    assert runs[0][1:] == runs[1][1:]
    assert runs[0][1] > 0


def test_tiny_zero_tokens_is_a_no_op(rig):
    _setup(rig, 0.5, [0])
    h, _ = rig.hidden(1)
    y, idx, w = rig.outputs(1)
    y.fill_(7.0)
    rig.forward(0, h, 0, y, idx, w)
    torch.cuda.synchronize()
    assert torch.all(y == 7.0)


def test_tiny_zero_input_selects_lowest_indices(rig):
    _setup(rig, 0.5, [0, 1, 2, 3])
    h = torch.zeros(3, 256, dtype=torch.float32, device="cuda")
    y, idx, w = _run(rig, h, 3)
    assert idx.cpu().numpy().tolist() == [[0, 1]] * 3
    assert torch.all(y == 0)
    np.testing.assert_allclose(w.cpu().numpy(), 0.5)


def test_tiny_error_codes(rig):
    from paper_2509_08342_amd import moesplit as ms
    tb = rig.top_bytes(0.5)
    rig.configure([2 * tb], [0.5])
    rig.load_tops(0, [0, 1])
    with pytest.raises(ms.MoeSplitError) as ei:
        ms.ms_load_top(rig.ctx, 0, 2)          # both cache slots taken
    assert ei.value.status == ms.MS_E_BUDGET
    with pytest.raises(ms.MoeSplitError) as ei:
        ms.ms_load_top(rig.ctx, 0, 1)          # already cached
    assert ei.value.status == ms.MS_E_STATE
    with pytest.raises(ms.MoeSplitError) as ei:
        ms.ms_evict_top(rig.ctx, 0, 5)         # not cached
    assert ei.value.status == ms.MS_E_STATE
    ms.ms_evict_top(rig.ctx, 0, 1)
    ms.ms_load_top(rig.ctx, 0, 2)
    assert ms.ms_residency(rig.ctx, 0, 8).tolist() == [1, 0, 1, 0, 0, 0, 0, 0]
    with pytest.raises(ms.MoeSplitError) as ei:
        rig.configure([rig.pool_bytes], [0.5])  # more than the pool holds
    assert ei.value.status == ms.MS_E_BUDGET
    with pytest.raises(ms.MoeSplitError) as ei:
        rig.configure([0], [1.5])
    assert ei.value.status == ms.MS_E_INVALID
    h, _ = rig.hidden(65)
    y, idx, w = rig.outputs(65)
    with pytest.raises(ms.MoeSplitError) as ei:
        rig.forward(0, h, 65, y, idx, w)       # T > max_tokens
    assert ei.value.status == ms.MS_E_INVALID
    with pytest.raises(ms.MoeSplitError) as ei:
        ms.ms_forward(rig.ctx, 3, h, 1, y, idx, w, 0, None)   # no such layer
    assert ei.value.status == ms.MS_E_INVALID


GOLDEN_D = 256  # the narrowest supported d_model; the cases use elements 0-65, the rest are zero


def _golden_router_case(which):
    """Router of two experts on d = 256 whose top-1 choice depends on the
    fixed fp32 logit order: expert 0's products follow the golden patterns of
    tests/golden/two_expert_cases.json (elements beyond them zero, which adds
    exact zeros to every residue's chain), expert 1 has one exact product."""
    h = np.zeros((1, GOLDEN_D), np.float32)
    w_r = np.zeros((GOLDEN_D, 2), np.float32)
    prods = {"a": {0: 2.0 ** 24, 1: 1.0, 65: 1.0}, "b": {0: 2.0 ** 24, 16: 1.0, 32: 1.0},
             "c": {0: 2.0 ** 24, 1: 1.0, 33: 1.0}}[which]
    for j, v in prods.items():
        h[0, j] = v
        w_r[j, 0] = 1.0
    # expert 1: h_0 * w = 2^24 + 2 exactly (a single exact product)
    w_r[0, 1] = np.float32(1.0 + 2.0 ** -23)
    # canonical expert-0 logits: a, c -> 2^24 + 2 (tie with expert 1 -> 0); b -> 2^24 (-> 1)
    expect = {"a": 0, "b": 1, "c": 0}[which]
    return h, w_r, expect


@pytest.mark.parametrize("which", ["a", "b", "c"])
def test_router_follows_fixed_logit_order(which):
    import oracle
    from workload import SplitRig
    shape = synth.ModelShape("golden-order", 1, GOLDEN_D, 64, 2, 1, "f32")
    h, w_r, expect = _golden_router_case(which)
    assert oracle.topk(oracle.router_logits(h, w_r), 1)[0, 0] == expect
    with SplitRig(shape, seed=3, max_tokens=1, budget_bytes=0) as rig:
        from paper_2509_08342_amd import moesplit as ms
        ms.ms_set_router(rig.ctx, 0, w_r)
        rig.configure([0], [0.0])
        y, idx, w = rig.outputs(1)
        rig.forward(0, torch.from_numpy(h).cuda(), 1, y, idx, w)
        torch.cuda.synchronize()
        assert int(idx[0, 0]) == expect


@pytest.mark.parametrize("splits", [1, 2, 4])
def test_tiny_every_chunk_split_matches_oracle(splits):
    """The FFN kernel's work-group split of a chunk changes only the
    summation grouping: each split passes parity and is residency-invariant."""
    from workload import SplitRig, top_bytes
    with SplitRig(synth.TINY, seed=0, max_tokens=16, budget_bytes=8 * synth.TINY.expert_bytes,
                  ffn_splits=splits) as r:
        h, hf = r.hidden(16, tag=31)
        outs = []
        for ratio, tops in ((0.5, [0, 1, 2, 3]), (1.0, list(range(8))), (0.0, [])):
            tb = top_bytes(r, ratio)
            r.configure([8 * tb], [ratio])
            r.load_tops(0, tops)
            y, idx, w = r.outputs(16)
            r.forward(0, h, 16, y, idx, w)
            torch.cuda.synchronize()
            check_layer(r, 0, hf, y, idx, w)
            outs.append(y.cpu().numpy())
        assert np.array_equal(outs[0], outs[1]) and np.array_equal(outs[0], outs[2])


def test_tiny_rewritten_expert_is_streamed_fresh():
    """Expert weights set again after forwards have streamed (and cached)
    the old ones -- the same host blob, rewritten in place: the next forward
    uses only the new weights, streamed and cached."""
    from paper_2509_08342_amd import moesplit as ms
    from workload import SplitRig, top_bytes
    with SplitRig(synth.TINY, seed=0, max_tokens=8, budget_bytes=8 * synth.TINY.expert_bytes) as r:
        r.configure([4 * top_bytes(r, 0.5)], [0.5])
        r.load_tops(0, [0, 1, 2, 3])
        h, hf = r.hidden(8, tag=61)
        for _ in range(2):
            y, idx, w = r.outputs(8)
            r.forward(0, h, 8, y, idx, w)
            torch.cuda.synchronize()
        check_layer(r, 0, hf, y, idx, w)
        for e in range(8):
            ex = synth.expert(synth.TINY, 17, 0, e)
            ms.ms_set_expert(r.ctx, 0, e, *ex.raw)
            r.experts[0][e] = ex.f32
        assert ms.ms_residency(r.ctx, 0, 8).tolist() == [1, 1, 1, 1, 0, 0, 0, 0]
        y, idx, w = r.outputs(8)
        r.forward(0, h, 8, y, idx, w)
        torch.cuda.synchronize()
        check_layer(r, 0, hf, y, idx, w)
