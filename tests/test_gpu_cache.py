"""GPU runs of the cache configurator's inputs and the online replacement
policies against the planner oracle: the statistics H, P, PH and the cache
priorities gathered by ms_forward over a token trace (exactly), the cache
update of Algorithm 1 (highest priorities cached), and LCP / LRU / LFU
replacement on misses (same residency as the oracle's simulation after
every forward) with outputs still matching the layer oracle."""
import numpy as np
import pytest

import synth
from gpu_helpers import check_layer

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _rig(max_tokens=4):
    from workload import SplitRig
    return SplitRig(synth.TINY, seed=3, max_tokens=max_tokens, budget_bytes=8 * synth.TINY.expert_bytes)


def _counts(idx, E):
    c = [0] * E
    for e in idx.reshape(-1).tolist():
        c[e] += 1
    return c


def test_plan_statistics_match_oracle():
    from oracle import planner
    from paper_2509_08342_amd import moesplit as ms
    from workload import top_bytes
    E, K = synth.TINY.n_experts, synth.TINY.top_k
    with _rig() as r:
        r.configure([4 * top_bytes(r, 0.5)], [0.5])
        r.load_tops(0, [0, 1, 2, 3])
        ref = planner.LayerStats(E, K)
        seq = synth.walk(synth.TINY, 5, 30, T=3)
        for step, (raw, _) in enumerate(seq):
            T = 1 + step % 3
            h = torch.from_numpy(np.ascontiguousarray(raw[:T])).cuda()
            order = None
            if step % 4 != 3:   # some forwards without a prediction
                order, _ = ms.ms_predict(r.ctx, 0, h, T, torch.cuda.current_stream(), E)
            y, idx, w = r.outputs(T)
            r.forward(0, h, T, y, idx, w)
            torch.cuda.synchronize()
            ref.forward(_counts(idx[:T].cpu().numpy(), E), T, None if order is None else order.tolist())
        hit, pred, ph, tok = ms.ms_plan_stats(r.ctx, 0, E)
        assert tok == (ref.q, ref.q_pred)
        assert hit.tolist() == ref.H()
        assert pred.tolist() == ref.P()
        assert ph.tolist() == ref.PH()
        prio = ms.ms_lcp_priority(r.ctx, 0, E)
        assert prio.tolist() == planner.lcp_priority(ref.mu, ref.nu)
        # the cache update of Algorithm 1: the highest priorities get the tops
        ms.ms_cache_update(r.ctx, np.array([3 * top_bytes(r, 0.5)], np.uint64), np.array([0.5], np.float32))
        top3 = [e for e in range(E) if planner.priority_ranks(prio.tolist())[e] < 3]
        assert ms.ms_residency(r.ctx, 0, E).tolist() == [1 if e in top3 else 0 for e in range(E)]
        h, hf = r.hidden(4, tag=8)
        y, idx, w = r.outputs(4)
        r.forward(0, h, 4, y, idx, w)
        torch.cuda.synchronize()
        check_layer(r, 0, hf, y, idx, w)
        ms.ms_reset_plan_stats(r.ctx)
        hit, pred, ph, tok = ms.ms_plan_stats(r.ctx, 0, E)
        assert tok == (0, 0) and not hit.any() and not ms.ms_lcp_priority(r.ctx, 0, E).any()


@pytest.mark.parametrize("policy", ["lcp", "lru", "lfu"])
def test_online_replacement_follows_the_rule(policy):
    from oracle import planner
    from paper_2509_08342_amd import moesplit as ms
    from workload import top_bytes
    code = {"lcp": ms.MS_CACHE_LCP, "lru": ms.MS_CACHE_LRU, "lfu": ms.MS_CACHE_LFU}[policy]
    E, K = synth.TINY.n_experts, synth.TINY.top_k
    with _rig(max_tokens=2) as r:
        r.configure([2 * top_bytes(r, 0.5)], [0.5])
        r.load_tops(0, [0, 1])
        ms.ms_set_cache_policy(r.ctx, code, 0.25, 8.0)   # a short window so priorities move
        ref = planner.LayerStats(E, K, rho=0.25, omega=8.0)
        last_use = [0] * E
        cached = [0, 1]
        seq = synth.walk(synth.TINY, 9, 40, T=2)
        inserts = 0
        for step, (raw, f) in enumerate(seq):
            T = 1 + step % 2
            h = torch.from_numpy(np.ascontiguousarray(raw[:T])).cuda()
            y, idx, w = r.outputs(T)
            r.forward(0, h, T, y, idx, w)
            torch.cuda.synchronize()
            if step % 5 == 0:
                check_layer(r, 0, f[:T], y, idx, w)
            counts = _counts(idx[:T].cpu().numpy(), E)
            ref.forward(counts, T, None)
            for e in range(E):
                if counts[e]:
                    last_use[e] = step + 1     # forwards of the layer so far
            before = list(cached)
            planner.replacement_step(cached, counts, planner.replacement_keys(policy, ref, last_use))
            inserts += sum(1 for a, b in zip(before, cached) if a != b)
            res = ms.ms_residency(r.ctx, 0, E).tolist()
            assert res == [1 if e in cached else 0 for e in range(E)], (step, res, cached)
        assert ms.ms_stats(r.ctx, 0)["cache_inserts"] == inserts > 0


def test_random_replacement_keeps_the_cache_size_and_outputs():
    from paper_2509_08342_amd import moesplit as ms
    from workload import top_bytes
    E = synth.TINY.n_experts
    with _rig(max_tokens=1) as r:
        r.configure([3 * top_bytes(r, 0.5)], [0.5])
        r.load_tops(0, [0, 1, 2])
        ms.ms_set_cache_policy(r.ctx, ms.MS_CACHE_RND, seed=7)
        for step, (raw, f) in enumerate(synth.walk(synth.TINY, 4, 20, T=1)):
            h = torch.from_numpy(raw).cuda()
            y, idx, w = r.outputs(1)
            r.forward(0, h, 1, y, idx, w)
            torch.cuda.synchronize()
            check_layer(r, 0, f, y, idx, w)
            assert sum(ms.ms_residency(r.ctx, 0, E)) == 3
        with pytest.raises(ms.MoeSplitError):
            ms.ms_set_cache_policy(r.ctx, 9)
        with pytest.raises(ms.MoeSplitError):
            ms.ms_set_cache_policy(r.ctx, ms.MS_CACHE_LCP, rho=1.5)
