"""Oracle of the cache configurator (arXiv 2509.08342, Sec. 3.3-3.4,
Eq. (4)-(11), Algorithm 1) and of the statistics it consumes.

TEST INFRASTRUCTURE ONLY, like the rest of this package: plain, slow Python
in the paper's notation and order, fp64 throughout (Python floats).  The
library's planner must reproduce these results; it shares no code with this
module.

Notation: L layers, N experts, K activated per token, U_e bytes per expert,
V_i bytes of cache budget of layer i, C_i experts whose top segments are
cached, theta_i = V_i / (C_i U_e) the split ratio.

Readings (where the paper leaves room):
* H_i(C) counts an activation as a hit of a size-C cache when the expert is
  among the C highest cache priorities (Eq. (4)) at the time of the forward,
  ties to the lower index.  C runs over 0..N here (H_i(0) = 0).
* P_i(y) and PH_i(y, C) are counted over the forwards that had a prediction
  for layer i, per token (a batch of T tokens shares one prediction ranking,
  reading of Eq. (3) for batches), and divided by those forwards' tokens.
* A batch of T tokens is one step for the activation interval nu of Eq. (4):
  nu is reset when any token of the batch activates the expert and grows by
  one otherwise; the activation frequency mu grows by the number of tokens
  that activated it.
* In the sub-problem (Eq. (11)) C runs over the sizes with theta <= 1; when
  the budget covers every expert whole, C = N and theta = 1.  Equal m: the
  smaller C.  m is clipped to [0, K].  A layer with V_i <= 0 is infeasible.
* Eq. (10) writes P_i(y, C_i); it is P_i(y) (defined in Sec. 3.4.2).
* Arg max / arg min ties in Algorithm 1 go to the lower layer index.
"""
from __future__ import annotations

import math


# ------------------------------------------------------------ statistics

def lcp_priority(mu, nu, rho=0.25, omega=128.0):
    """Eq. (4): cache priority mu * rho^(nu / omega) of each expert."""
    return [m * math.pow(rho, n / omega) for m, n in zip(mu, nu)]


def priority_ranks(prio):
    """rank[e]: position of expert e in descending priority, ties to the
    lower index (rank 0 = highest)."""
    order = sorted(range(len(prio)), key=lambda e: (-prio[e], e))
    rank = [0] * len(prio)
    for r, e in enumerate(order):
        rank[e] = r
    return rank


class LayerStats:
    """Counters of one layer (Sec. 3.4.2), fed one forward at a time."""

    def __init__(self, N, K, rho=0.25, omega=128.0):
        self.N, self.K, self.rho, self.omega = N, K, rho, omega
        self.mu = [0.0] * N
        self.nu = [0.0] * N
        self.q = 0                               # tokens
        self.q_pred = 0                          # tokens of forwards with a prediction
        self.hit_hist = [0] * N                  # activations by priority rank
        self.pred_act = [0] * N                  # tokens whose y-th prediction was activated
        self.pred_rank = [[0] * N for _ in range(N)]   # [y][rank of the y-th prediction] tokens

    def forward(self, counts, T, pred_order=None):
        """counts[e]: tokens of this forward that activated e (sum = T K);
        pred_order: the prediction's ranking of the experts, or None."""
        N = self.N
        rank = priority_ranks(lcp_priority(self.mu, self.nu, self.rho, self.omega))
        for e in range(N):
            self.hit_hist[rank[e]] += counts[e]
        if pred_order is not None:
            for y in range(N):
                e = pred_order[y]
                self.pred_act[y] += counts[e]
                self.pred_rank[y][rank[e]] += T
            self.q_pred += T
        self.q += T
        for e in range(N):
            self.mu[e] += counts[e]
            self.nu[e] = 0.0 if counts[e] > 0 else self.nu[e] + 1.0

    def H(self):
        """H_i(C), C = 0..N."""
        tot = self.q * self.K
        out, run = [0.0], 0
        for c in range(self.N):
            run += self.hit_hist[c]
            out.append(run / tot if tot else 0.0)
        return out

    def P(self):
        """P_i(y), y = 1..N (list index y - 1)."""
        return [a / self.q_pred if self.q_pred else 0.0 for a in self.pred_act]

    def PH(self):
        """PH_i(y, C), y = 1..N (index y - 1), C = 0..N."""
        out = []
        for y in range(self.N):
            row, run = [0.0], 0
            for c in range(self.N):
                run += self.pred_rank[y][c]
                row.append(run / self.q_pred if self.q_pred else 0.0)
            out.append(row)
        return out


# ---------------------------------------------------------- the planner

def subproblem(V, T_wind, H, P, PH, K, N, U_e, T_load):
    """Eq. (8)-(11): the cache size C (and theta = V / (C U_e)) maximising
    m = A_cache + sum_{y <= Y} A_pref(y), Y the prefetches that fit in
    T_wind.  Returns (theta, C, m)."""
    best = None
    for C in range(1, N + 1):
        theta = V / (C * U_e)
        if theta > 1.0:
            continue
        m = K * H[C] * theta                       # A_cache (Eq. (8) text)
        t = 0.0
        for y in range(N):
            tp = (1.0 - PH[y][C] * theta) * T_load  # Eq. (9)
            if t + tp > T_wind:
                break
            t += tp
            m += (1.0 - PH[y][C] * theta) * P[y]    # Eq. (10)
        m = min(max(m, 0.0), float(K))
        if best is None or m > best[2]:
            best = (theta, C, m)
    if best is None:                                # the budget holds every expert whole
        C, theta = N, 1.0
        m = K * H[C] * theta
        t = 0.0
        for y in range(N):
            tp = (1.0 - PH[y][C] * theta) * T_load
            if t + tp > T_wind:
                break
            t += tp
            m += (1.0 - PH[y][C] * theta) * P[y]
        best = (theta, C, min(max(m, 0.0), float(K)))
    return best


def expert_split(Vs, prm, stats):
    """Algorithm 1, ExpertSplit: per layer in order, the sub-problem's
    theta* and the exposed loading latency (Eq. (5)-(7), with
    alpha + beta theta ~ m and beta (1 - theta) + gamma ~ K - m).  Returns
    (exposed[L], theta[L], C[L], m[L]); an infeasible layer (V_i <= 0) has
    exposed latency +inf."""
    K, N, U_e = prm["K"], prm["N"], prm["U_e"]
    T_att, T_moe, T_head, T_load = prm["T_att"], prm["T_moe"], prm["T_head"], prm["T_load"]
    T_exp = T_moe / K
    T_wind = T_head + T_att
    ex, th, cs, ms = [], [], [], []
    for i, V in enumerate(Vs):
        H, P, PH = stats[i]
        if V <= 0:
            ex.append(math.inf)
            th.append(0.0)
            cs.append(0)
            ms.append(0.0)
            T_wind = T_moe + T_att
            continue
        theta, C, m = subproblem(V, T_wind, H, P, PH, K, N, U_e, T_load)
        T_hide = m * T_exp                          # Eq. (5)
        T_miss = (K - m) * T_load
        ex.append(max(0.0, T_miss - T_hide))        # Eq. (6)
        th.append(theta)
        cs.append(C)
        ms.append(m)
        T_wind = (T_moe - min(T_hide, T_miss)) + T_att   # Eq. (7)
    return ex, th, cs, ms


def vram_allocation(V_e, zeta, prm, stats, V_start=None, max_iter=100000):
    """Algorithm 1, VramAllocation: move zeta V_e of budget from the layer
    whose loss costs least to the layer whose gain is largest while the
    summed exposed latency decreases.  Budgets are integer bytes; the step
    is floor(zeta V_e).  Returns (V[L], theta[L], C[L], exposed[L], iters)."""
    L = len(stats)
    V = list(V_start) if V_start is not None else [V_e // L] * L
    step = int(math.floor(zeta * V_e))
    it = 0
    while True:
        T1, th1, c1, _ = expert_split(V, prm, stats)
        if step <= 0 or L < 2 or it >= max_iter:
            return V, th1, c1, T1, it
        T2, _, _, _ = expert_split([v + step for v in V], prm, stats)
        T3, _, _, _ = expert_split([v - step for v in V], prm, stats)
        gain = [T1[i] - T2[i] for i in range(L)]
        i1 = max(range(L), key=lambda i: (gain[i], -i))
        cost = [T3[i] - T1[i] for i in range(L)]
        i2 = min((i for i in range(L) if i != i1), key=lambda i: (cost[i], i))
        V4 = list(V)
        V4[i1] += step
        V4[i2] -= step
        T4, _, _, _ = expert_split(V4, prm, stats)
        delta = 0.0
        for i in range(L):
            delta += T4[i] - T1[i]
        if not delta < 0.0:                        # also stops on inf - inf = nan
            return V, th1, c1, T1, it
        V = V4
        it += 1


# ------------------------------------------------- online replacement

MASK64 = (1 << 64) - 1


class SplitMix64:
    """SplitMix64 (Steele, Lea and Flood, "Fast splittable pseudorandom
    number generators", OOPSLA 2014, in the 64-bit form Vigna publishes as
    splitmix64.c): the state advances by the golden-ratio increment
    0x9e3779b97f4a7c15 and each output is the state passed through the
    variant-13 mixer (shift-xor 30, multiply 0xbf58476d1ce4e5b9, shift-xor 27,
    multiply 0x94d049bb133111eb, shift-xor 31).  The random policy draws its
    keys from it; the generator is counter-based, so both sides can carry
    their own copy."""

    GAMMA = 0x9E3779B97F4A7C15

    def __init__(self, state):
        self.state = state & MASK64

    def next(self):
        self.state = (self.state + self.GAMMA) & MASK64
        z = self.state
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
        return z ^ (z >> 31)


def rnd_generator(seed):
    """The random policy's generator for a user seed: the state starts at
    seed XOR the golden-ratio increment."""
    return SplitMix64(seed ^ SplitMix64.GAMMA)


def replacement_keys(policy, st, last_use, rng=None):
    """Ranking key of each expert (larger = keep):
    LCP: the cache priority of Eq. (4) after this forward's statistics;
    LRU: last_use[e], the count of the layer's forwards up to and including
         the most recent one that activated e (0 if never);
    LFU: mu_e, the activations so far;
    RND: one draw per expert in index order, the top 53 bits of the next
         SplitMix64 output (rng, from rnd_generator), as a float."""
    if policy == "lcp":
        return lcp_priority(st.mu, st.nu, st.rho, st.omega)
    if policy == "lru":
        return [float(x) for x in last_use]
    if policy == "lfu":
        return list(st.mu)
    if policy == "rnd":
        return [float(rng.next() >> 11) for _ in range(st.N)]
    raise ValueError(policy)


def replacement_step(cached, counts, key):
    """Sec. 3.3, on a miss: the missed experts are the activated ones
    (counts[e] > 0) with no cached top.  Taken in descending key order (ties
    to the lower index), at most as many as there are cache slots, each takes
    a free slot (the lowest-numbered one) if there is one, else the slot of
    the cached expert with the lowest key (ties to the lower index) among
    those not cached in this same step.  cached: list of experts per slot
    (-1 free), updated in place and returned."""
    N = len(counts)
    missed = sorted((e for e in range(N) if counts[e] > 0 and e not in cached), key=lambda e: (-key[e], e))
    fresh = set()
    for e in missed[:len(cached)]:
        if -1 in cached:
            slot = cached.index(-1)
        else:
            cands = [v for v in cached if v not in fresh]
            if not cands:
                break
            victim = min(cands, key=lambda v: (key[v], v))
            slot = cached.index(victim)
        cached[slot] = e
        fresh.add(e)
    return cached
