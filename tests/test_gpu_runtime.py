"""GPU checks of the runtime's buffer and prefetch bookkeeping: dropping the
staging buffer while prefetch copies are in flight, the termination of a
queued prefetch when the layer's routing arrives (Sec. 3.2), a prefill
forward after an expert's top was evicted (one staging slot per expert), and
the seeded random replacement policy against the oracle's simulation.  Every
case also checks the layer's outputs against the oracle."""
import numpy as np
import pytest

import synth
from gpu_helpers import check_layer

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

TWO_LAYER = synth.ModelShape("tiny-2l-f32", 2, 256, 512, 8, 2, "f32")
# 12 MiB experts: a prefetch copy group is 4 MiB at most, so a whole expert
# takes four groups and a few experts queue more groups than are in flight
PF_BF16 = synth.ModelShape("pf-bf16", 2, 1024, 2048, 8, 2, "bf16")
TINY_BF16 = synth.ModelShape("tiny-bf16", 1, 256, 512, 8, 2, "bf16")


def test_drop_buffer_forgets_prefetch_in_flight():
    """ms_prefetch leaves copy groups in flight; ms_drop_buffer must forget
    them, so that the next forward's prediction still prefetches (its
    bytes_prefetch grows) and both layers still match the oracle."""
    from paper_2509_08342_amd import moesplit as ms
    from workload import SplitRig, top_bytes
    with SplitRig(TWO_LAYER, seed=4, max_tokens=1, budget_bytes=4 * TWO_LAYER.expert_bytes) as r:
        tb = top_bytes(r, 0.5)
        r.configure([2 * tb, 2 * tb], [0.5, 0.5])
        r.load_tops(0, [0, 1])
        r.load_tops(1, [0, 1])
        ms.ms_prefetch(r.ctx, 1, np.array([2, 3, 4, 5], np.int32))
        ms.ms_drop_buffer(r.ctx)
        before = ms.ms_stats(r.ctx, 1)["bytes_prefetch"]
        assert before > 0
        h, hf = r.hidden(1, tag=3)
        y, idx, w = r.outputs(1)
        r.forward(0, h, 1, y, idx, w, ms.MS_FWD_PREDICT_NEXT)
        torch.cuda.synchronize()
        check_layer(r, 0, hf, y, idx, w)
        assert ms.ms_stats(r.ctx, 1)["bytes_prefetch"] > before
        y1, idx1, w1 = r.outputs(1)
        r.forward(1, h, 1, y1, idx1, w1)
        torch.cuda.synchronize()
        check_layer(r, 1, hf, y1, idx1, w1)
        ms.ms_sync(r.ctx)


def test_prefetch_terminated_at_routing():
    """Four whole experts of layer 1 (no tops cached) are queued for prefetch
    (16 copy groups, two in flight); layer 1's forward starts at once, so most groups are
    still queued when its routing arrives and are dropped.  Every requested
    byte is either issued or dropped, some are dropped, and the layer still
    matches the oracle (groups in flight complete; what a selected expert
    still misses is copied as a miss)."""
    from paper_2509_08342_amd import moesplit as ms
    from workload import SplitRig
    s = PF_BF16
    with SplitRig(s, seed=6, max_tokens=1, budget_bytes=0) as r:
        r.configure([0, 0], [0.5, 0.5])
        for tag in range(3):
            ms.ms_drop_buffer(r.ctx)
            ms.ms_sync(r.ctx)
            ms.ms_reset_stats(r.ctx)
            h, hf = r.hidden(1, tag=40 + tag)
            y, idx, w = r.outputs(1)
            ms.ms_prefetch(r.ctx, 1, np.array([4, 5, 6, 7], np.int32))
            r.forward(1, h, 1, y, idx, w)
            torch.cuda.synchronize()
            check_layer(r, 1, hf, y, idx, w)
            ms.ms_sync(r.ctx)
            st = ms.ms_stats(r.ctx, 1)
            assert st["bytes_prefetch"] + st["bytes_prefetch_dropped"] == 4 * s.expert_bytes
            assert st["bytes_prefetch_dropped"] > 0
            assert st["bytes_prefetch"] > 0


def test_prefill_after_top_eviction_keeps_one_slot_per_expert():
    """A decode forward streams the bottoms of its two experts (tops cached);
    their tops are then evicted, so the staging slots hold only bottoms.  A
    prefill forward needs both experts whole: it must reuse their slots for
    the whole copies.  A decode forward of the first token afterwards then
    finds both whole in the buffer and copies nothing."""
    from paper_2509_08342_amd import moesplit as ms
    from workload import SplitRig, top_bytes
    s = TINY_BF16
    with SplitRig(s, seed=9, max_tokens=64, budget_bytes=s.n_experts * s.expert_bytes, n_buffer_slots=16) as r:
        tb = top_bytes(r, 0.5)
        r.configure([s.n_experts * tb], [0.5])
        r.load_tops(0, range(s.n_experts))
        h1, hf1 = r.hidden(1, tag=1)
        y, idx, w = r.outputs(1)
        r.forward(0, h1, 1, y, idx, w, ms.MS_FWD_NO_MATRIX_CORES)
        torch.cuda.synchronize()
        check_layer(r, 0, hf1, y, idx, w)
        sel = sorted(set(idx[0].cpu().numpy().tolist()))
        for e in sel:
            ms.ms_evict_top(r.ctx, 0, e)
        hp, hfp = r.hidden(64, tag=2)
        yp, idxp, wp = r.outputs(64)
        r.forward(0, hp, 64, yp, idxp, wp, ms.MS_FWD_MATRIX_CORES)
        torch.cuda.synchronize()
        check_layer(r, 0, hfp, yp, idxp, wp)
        assert set(sel) <= set(idxp[:64].cpu().numpy().reshape(-1).tolist()), "prefill did not select both"
        ms.ms_sync(r.ctx)
        miss0 = ms.ms_stats(r.ctx, 0)["bytes_miss"]
        y2, idx2, w2 = r.outputs(1)
        r.forward(0, h1, 1, y2, idx2, w2, ms.MS_FWD_NO_MATRIX_CORES)
        torch.cuda.synchronize()
        check_layer(r, 0, hf1, y2, idx2, w2)
        assert ms.ms_stats(r.ctx, 0)["bytes_miss"] == miss0


def test_random_replacement_follows_the_oracle():
    """MS_CACHE_RND: residency after every forward equals the oracle's
    simulation with the same SplitMix64 seed (keys drawn per forward, one per
    expert in index order), and the outputs match the layer oracle."""
    from oracle import planner
    from paper_2509_08342_amd import moesplit as ms
    from workload import SplitRig, top_bytes
    E, K = synth.TINY.n_experts, synth.TINY.top_k
    seed = 12345
    with SplitRig(synth.TINY, seed=3, max_tokens=2, budget_bytes=8 * synth.TINY.expert_bytes) as r:
        r.configure([2 * top_bytes(r, 0.5)], [0.5])
        r.load_tops(0, [0, 1])
        ms.ms_set_cache_policy(r.ctx, ms.MS_CACHE_RND, seed=seed)
        ref = planner.LayerStats(E, K)
        rng = planner.rnd_generator(seed)
        cached = [0, 1]
        inserts = 0
        for step, (raw, f) in enumerate(synth.walk(synth.TINY, 11, 40, T=2)):
            T = 1 + step % 2
            h = torch.from_numpy(np.ascontiguousarray(raw[:T])).cuda()
            y, idx, w = r.outputs(T)
            r.forward(0, h, T, y, idx, w)
            torch.cuda.synchronize()
            if step % 5 == 0:
                check_layer(r, 0, f[:T], y, idx, w)
            counts = [0] * E
            for e in idx[:T].cpu().numpy().reshape(-1).tolist():
                counts[e] += 1
            ref.forward(counts, T, None)
            before = list(cached)
            planner.replacement_step(cached, counts, planner.replacement_keys("rnd", ref, None, rng))
            inserts += sum(1 for a, b in zip(before, cached) if a != b)
            res = ms.ms_residency(r.ctx, 0, E).tolist()
            assert res == [1 if e in cached else 0 for e in range(E)], (step, res, cached)
        assert ms.ms_stats(r.ctx, 0)["cache_inserts"] == inserts > 0
