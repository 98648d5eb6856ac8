"""Pins of the online-replacement oracle (Sec. 3.3 with the priority of
Eq. (4)): hand-derived replacement steps, a hand-derived activation trace
under LCP, LRU and LFU, the published SplitMix64 outputs behind the random
policy, and mutants of the rule that those pins must reject."""
import json
import os

import pytest

from oracle import planner

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "replacement_cases.json")))


@pytest.mark.parametrize("case", GOLD["steps"], ids=lambda c: c["name"])
def test_replacement_step_hand_cases(case):
    cached = list(case["cached"])
    out = planner.replacement_step(cached, case["counts"], [float(k) for k in case["key"]])
    assert out is cached and cached == case["expect"]


def _trace(policy, step=planner.replacement_step, keys=planner.replacement_keys):
    g = GOLD["policy_trace"]
    N = g["N"]
    st = planner.LayerStats(N, g["K"], rho=g["rho"], omega=g["omega"])
    cached = list(g["cached"])
    last_use = [0] * N
    key = None
    for f, e in enumerate(g["activations"], start=1):
        counts = [0] * N
        counts[e] = 1
        st.forward(counts, 1, None)
        last_use[e] = f
        key = keys(policy, st, last_use)
        step(cached, counts, key)
    return cached, key


@pytest.mark.parametrize("policy", ["lcp", "lru", "lfu"])
def test_policy_trace_by_hand(policy):
    g = GOLD["policy_trace"]
    cached, key = _trace(policy)
    assert key == pytest.approx(g["keys_after"][policy], rel=1e-15, abs=0)
    assert cached == g["expect"][policy]


def test_splitmix64_published_outputs():
    g = GOLD["splitmix64"]
    gen = planner.SplitMix64(0)
    assert [gen.next() for _ in range(3)] == [int(x, 16) for x in g["state0_outputs"]]
    # the policy's seeding: state = seed XOR the increment
    gen = planner.rnd_generator(int(g["rnd_case"]["seed"], 16))
    assert gen.state == 0 and gen.next() == int(g["state0_outputs"][0], 16)


def test_random_policy_case():
    g = GOLD["splitmix64"]
    c = g["rnd_case"]
    st = planner.LayerStats(3, 1)
    rng = planner.rnd_generator(int(c["seed"], 16))
    key = planner.replacement_keys("rnd", st, [0] * 3, rng)
    assert key == [float(int(x, 16) >> 11) for x in g["state0_outputs"]]
    assert all(0.0 <= k < 2.0 ** 53 and k == int(k) for k in key)
    cached = list(c["cached"])
    assert planner.replacement_step(cached, c["counts"], key) == c["expect"]
    # the next forward draws the next three outputs
    gen = planner.SplitMix64(0)
    for _ in range(3):
        gen.next()
    assert planner.replacement_keys("rnd", st, [0] * 3, rng)[0] == float(gen.next() >> 11)


# ---------------------------------------------------------------- mutants
#
# Plausible mistakes in the rule, each as a variant of replacement_step or
# replacement_keys.  The hand-derived pins above must reject every one.

def _step_variant(evict_highest=False, victim_ties_high=False, evict_fresh=False, ascending=False,
                  missed_ties_high=False, ignore_free=False, cached_can_miss=False, first_slot_victim=False):
    def step(cached, counts, key):
        N = len(counts)
        miss = [e for e in range(N) if counts[e] > 0 and (cached_can_miss or e not in cached)]
        sgn = 1 if ascending else -1
        tie = -1 if missed_ties_high else 1
        miss.sort(key=lambda e: (sgn * key[e], tie * e))
        fresh = set()
        for e in miss[:len(cached)]:
            if -1 in cached and not ignore_free:
                slot = cached.index(-1)
            else:
                cands = [v for v in cached if v != -1 and (evict_fresh or v not in fresh)]
                if not cands:
                    break
                if first_slot_victim:
                    victim = cands[0]
                else:
                    ks = -1 if evict_highest else 1
                    vt = -1 if victim_ties_high else 1
                    victim = min(cands, key=lambda v: (ks * key[v], vt * v))
                slot = cached.index(victim)
            cached[slot] = e
            fresh.add(e)
        return cached
    return step


STEP_MUTANTS = {
    "evict_highest": dict(evict_highest=True),
    "victim_ties_to_higher_index": dict(victim_ties_high=True),
    "evicts_a_fresh_insert": dict(evict_fresh=True),
    "missed_in_ascending_key_order": dict(ascending=True),
    "missed_ties_to_higher_index": dict(missed_ties_high=True),
    "evicts_with_a_free_slot": dict(ignore_free=True),
    "cached_experts_count_as_missed": dict(cached_can_miss=True),
    "victim_is_the_first_slot": dict(first_slot_victim=True),
}


def _rejected_step(fn):
    for case in GOLD["steps"]:
        if fn(list(case["cached"]), case["counts"], [float(k) for k in case["key"]]) != case["expect"]:
            return True
    for policy in ("lcp", "lru", "lfu"):
        if _trace(policy, step=fn)[0] != GOLD["policy_trace"]["expect"][policy]:
            return True
    return False


def test_the_rule_itself_passes_the_mutant_check():
    assert not _rejected_step(planner.replacement_step)
    assert not _rejected_step(_step_variant())


@pytest.mark.parametrize("name", sorted(STEP_MUTANTS))
def test_step_mutants_are_rejected(name):
    assert _rejected_step(_step_variant(**STEP_MUTANTS[name]))


def _keys_variant(kind):
    def keys(policy, st, last_use, rng=None):
        if kind == "lru_by_count" and policy == "lru":
            return list(st.mu)
        if kind == "lfu_by_recency" and policy == "lfu":
            return [float(x) for x in last_use]
        if kind == "lcp_without_decay" and policy == "lcp":
            return list(st.mu)
        if kind == "lcp_inverted_decay" and policy == "lcp":
            return [m * st.rho ** (-n / st.omega) for m, n in zip(st.mu, st.nu)]
        if kind == "lcp_recency_only" and policy == "lcp":
            return [st.rho ** (n / st.omega) for n in st.nu]
        return planner.replacement_keys(policy, st, last_use, rng)
    return keys


@pytest.mark.parametrize("kind", ["lru_by_count", "lfu_by_recency", "lcp_without_decay", "lcp_inverted_decay",
                                  "lcp_recency_only"])
def test_key_mutants_are_rejected(kind):
    g = GOLD["policy_trace"]
    fn = _keys_variant(kind)
    rejected = False
    for policy in ("lcp", "lru", "lfu"):
        cached, key = _trace(policy, keys=fn)
        if cached != g["expect"][policy] or key != pytest.approx(g["keys_after"][policy], rel=1e-15, abs=0):
            rejected = True
    assert rejected
