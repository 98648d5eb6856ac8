"""GPU parity of stacked split-expert layers: the residual-norm glue against
the oracle, and teacher-forced layer parity (each checked layer's own GPU
input fed to the oracle) on layers {0, 1, L/2, L-1} of decode and prefill
passes through Mixtral-, DeepSeek- and Qwen3-shaped stacks with cross-layer
prediction and prefetch on.  Prefill layers are checked on 16 seeded rows."""
import numpy as np
import pytest

import synth
from gpu_helpers import check_layer

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

GIB = 1 << 30
TINY_STACK = synth.ModelShape("tiny-stack-bf16", 4, 256, 512, 8, 2, "bf16")
TINY_STACK_F32 = synth.ModelShape("tiny-stack-f32", 3, 256, 512, 8, 2, "f32")


def _check_capture(stack, layer, cap, rows=None):
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a))
    return check_layer(stack.rig, layer, cap["h"], t(cap["y"]), t(cap["idx"]), t(cap["w"]), tokens=rows)


@pytest.mark.parametrize("shape", [TINY_STACK, TINY_STACK_F32], ids=lambda s: s.name)
def test_residual_norm_matches_oracle(shape):
    import oracle
    from paper_2509_08342_amd import moesplit as ms
    from workload import SplitRig, to_device
    T = 37
    with SplitRig(shape, seed=2, max_tokens=T, budget_bytes=0) as r:
        raw, hf = synth.hidden(shape, 2, T, 9)
        h = to_device(raw, shape.dtype)
        y = torch.from_numpy(np.random.default_rng(4).standard_normal((T, shape.d_model)).astype(np.float32)).cuda()
        out = torch.empty_like(h)
        ms.ms_residual_norm(r.ctx, h, y, T, out)
        ms.ms_residual_norm(r.ctx, h, y, T, h)  # in place
        torch.cuda.synchronize()
        ref = oracle.residual_rmsnorm(hf, y.cpu().numpy().astype(np.float64))
        got = out.float().cpu().numpy()
        # fp32 arithmetic, then one rounding to the model dtype
        tol = 2.0 ** -8 if shape.dtype == "bf16" else 2e-6
        assert np.all(np.abs(got - ref) <= tol * np.abs(ref) + 1e-6)
        assert np.array_equal(h.float().cpu().numpy(), got)


@pytest.mark.parametrize("shape", [TINY_STACK, TINY_STACK_F32], ids=lambda s: s.name)
def test_tiny_stack_teacher_forced(shape):
    """Warm-up counts pick the cached tops; then decode steps and a ragged
    prefill pass, every layer checked against the oracle on its own input,
    and each layer's input checked to be the glue of the previous one."""
    import oracle
    from stack import Stack, decode_inputs, stack_top_bytes
    L = shape.n_layers
    with Stack(shape, seed=1, n_sets=2, max_tokens=70, budget_total=L * 8 * shape.expert_bytes) as st:
        tb = stack_top_bytes(st, 0.5)
        st.configure(0.5, L * 2 * tb)
        xs = decode_inputs(shape, 1, 10, 1)
        counts = st.warmup_counts([x for x, _ in xs[:4]], 1)
        assert counts.sum() == 4 * L * shape.top_k
        st.load_most_selected(counts)
        for x, _ in xs[4:]:
            _, cap = st.step(x, 1, capture=range(L))
            for l in range(L):
                _check_capture(st, l, cap[l])
            for l in range(L - 1):
                glue = oracle.residual_rmsnorm(cap[l]["h"], cap[l]["y"].astype(np.float64))
                tol = 2.0 ** -8 if shape.dtype == "bf16" else 2e-6
                assert np.all(np.abs(cap[l + 1]["h"] - glue) <= tol * np.abs(glue) + 1e-6)
        h, _ = st.rig.hidden(70, tag=5)
        _, cap = st.step(h, 70, capture=range(L))
        for l in range(L):
            _check_capture(st, l, cap[l])
        st_all = st.stats()
        assert sum(s["forwards"] for s in st_all) == L * (10 + 1)
        assert sum(s["predictions"] for s in st_all) > 0


def _check_captures(st, cap, layers, rows=None):
    """The checked layers of one step against the oracle, one thread per
    layer (the oracle's loops release the interpreter lock)."""
    from concurrent.futures import ThreadPoolExecutor
    with ThreadPoolExecutor(len(layers)) as ex:
        list(ex.map(lambda l: _check_capture(st, l, cap[l], rows), layers))


def _model_stack(shape, budget, r, prefill_T, decode_T, decode_steps):
    from stack import Stack, decode_inputs
    L = shape.n_layers
    check = sorted({0, 1, L // 2, L - 1})
    rows = sorted(np.random.default_rng(7).choice(prefill_T, 16, replace=False).tolist()) if prefill_T else None
    with Stack(shape, seed=0, n_sets=2, max_tokens=max(prefill_T, decode_T), budget_total=budget) as st:
        slots = st.configure(r, budget)
        xs = decode_inputs(shape, 0, decode_steps + 2, decode_T)
        counts = st.warmup_counts([x for x, _ in xs[:2]], decode_T)
        st.load_most_selected(counts)
        if prefill_T:
            h, _ = st.rig.hidden(prefill_T, tag=11)
            _, cap = st.step(h, prefill_T, capture=check)
            _check_captures(st, cap, check, rows)
        for x, _ in xs[2:]:
            _, cap = st.step(x, decode_T, capture=check)
            _check_captures(st, cap, check)
        return st.stats(), slots


def test_mixtral_stack_decode_teacher_forced():
    _model_stack(synth.MIXTRAL_STACK, 12 * GIB, 0.5, 0, 1, 2)


def test_deepseek_stack_prefill_and_decode_teacher_forced():
    _model_stack(synth.DEEPSEEK, 4 * GIB, 0.5, 512, 1, 2)


def test_qwen_stack_prefill_and_decode16_teacher_forced():
    _model_stack(synth.QWEN3, 8 * GIB, 0.5, 2048, 16, 2)


def test_mixtral_stack_mixed_split_ratios_teacher_forced():
    """Mixtral-shaped 32-layer stack at 12 GiB with r = .25 / .5 / .75 by layer
    index mod 3 (C_i = 4 / 2 / 1 tops of the 402.7 MB per-layer budget), 16
    decode steps with cross-layer prediction and prefetch, checked on layers
    {0, 1, 16, 31} at every step."""
    rs = [(0.25, 0.5, 0.75)[l % 3] for l in range(32)]
    stats, slots = _model_stack(synth.MIXTRAL_STACK, 12 * GIB, rs, 0, 1, 16)
    assert [int(c) for c in slots[:3]] == [4, 2, 1]
    assert sum(s["bytes_prefetch"] for s in stats) > 0
    assert sum(s["beta"] for s in stats) > 0 and sum(s["gamma"] for s in stats) > 0


def test_qwen_stack_configured_by_algorithm_1_with_lcp():
    """Qwen3-shaped 48-layer stack, 8 GiB, decode batch 16: the cache
    configurator (Algorithm 1) runs on the statistics of a 16-step warm-up,
    its per-layer budgets and split ratios are applied with ms_cache_update
    (each layer then caches the C_i tops of highest priority), LCP
    replacement is switched on, and 16 more steps are checked on layers
    {0, 1, 24, 47} at every step."""
    from paper_2509_08342_amd import moesplit as ms
    from stack import Stack, decode_inputs
    shape, budget, T = synth.QWEN3, 8 * GIB, 16
    L, E, K = shape.n_layers, shape.n_experts, shape.top_k
    check = [0, 1, L // 2, L - 1]
    with Stack(shape, seed=0, n_sets=2, max_tokens=T, budget_total=budget) as st:
        st.configure(0.5, budget)
        xs = decode_inputs(shape, 0, 32, T)
        ms.ms_reset_plan_stats(st.ctx)
        st.load_most_selected(st.warmup_counts([x for x, _ in xs[:16]], T))
        stats = [ms.ms_plan_stats(st.ctx, l, E) for l in range(L)]
        plan = ms.ms_plan_solve(L, E, K, shape.expert_bytes, 0.0, 305.0, 0.0, shape.expert_bytes / 55e3,
                                np.array([s[0] for s in stats]), np.array([s[1] for s in stats]),
                                np.array([s[2] for s in stats]), budget, 0.01)
        # the budget is conserved (less the remainder of the uniform start)
        assert budget - L < int(plan["budgets"].sum()) <= budget
        ms.ms_cache_update(st.ctx, plan["budgets"], plan["theta"].astype(np.float32))
        for l in range(L):
            units, tb, c = ms.ms_split_plan(st.rig.desc, int(plan["budgets"][l]), float(plan["theta"][l]))
            assert int((ms.ms_residency(st.ctx, l, E) > 0).sum()) == min(c, E)
        ms.ms_set_cache_policy(st.ctx, ms.MS_CACHE_LCP)
        ms.ms_reset_stats(st.ctx)
        for x, _ in xs[16:]:
            _, cap = st.step(x, T, capture=check)
            _check_captures(st, cap, check)
        tot = st.stats()
        assert sum(s["forwards"] for s in tot) == 16 * L
