"""Oracle of CacheScout's CPU control plane (test infrastructure).

Only ``tests/`` and ``bench.py``'s ``cpu_baseline`` leg may use this module.

Plain Python, following the paper's definitions in its order (arXiv
2608.14624):

* Sec. 2.2, Eq. (2): predictability R = 1 - H(A_{t+1} | A_t) / H(A_{t+1}),
  here over the observed transitions (empirical joint distribution).
* Sec. 3.2, Eq. (3): smoothed transition probability
  P_ij = (C_ij + eps) / sum_k (C_ik + eps); Eq. (4)-(5): the next-agent
  distribution is row i, the prediction its argmax.
* Sec. 3.3, Eq. (7): edge (a, b) iff P(b | a) >= tau; a breadth-first search
  from the current agent gives the hop distance E[a]; Eq. (8):
  p~(a) = 1 - min(E[a], E_max) / E_max (an agent the search cannot reach has
  E = infinity, so p~ = 0); Eq. (9): Score(b) = (p~(a_b) + delta) *
  (exp(-lambda * age(b)) + delta) * |b|, lowest score evicted first.
* Sec. 3.4, Eq. (10)-(11): when R >= R_min, warm up a* = argmax_a P(a | a_t).
* Sec. 4: among blocks of equal score, eviction prefers one whose contents are
  already resident in the CPU tier (nothing has to be copied out first).
* The runtime procedure: on a block touch, record the block's agent and
  access time; when the touching agent differs from the current one, count
  the transition, rebuild the graph and the hop table from the new agent and
  make it current.

The paper states none of eps, tau, E_max, lambda, delta, R_min numerically;
DEFAULTS are this implementation's reading.  Ties in an argmax go to the
lowest agent id, ties in an argmin to the first candidate.

Eq. (3)'s denominator sum_k (C_ik + eps) is evaluated as
(sum_k C_ik) + A * eps, the same real number; with it fixed to this fp64
expression, an edge that sits exactly on tau (likely with small counts, e.g.
P = 1.1 / 5.5 against tau = 0.2) is decided the same way by any
implementation that evaluates the same expression.
"""

import math
from collections import deque

DEFAULTS = dict(eps=0.1, tau=0.2, e_max=4, lam=0.1, delta=0.05, r_min=0.3)


def transition_prob(counts, i, j, eps):
    """Eq. (3) for an A x A list-of-lists of counts."""
    row = counts[i]
    return (row[j] + eps) / (sum(row) + len(row) * eps)


def predict_next(counts, i, eps):
    """Eq. (5): the most likely successor of agent i (lowest id on ties)."""
    n = len(counts)
    probs = [transition_prob(counts, i, j, eps) for j in range(n)]
    best = max(probs)
    return probs.index(best)


def threshold_graph(counts, eps, tau):
    """Eq. (7): adjacency lists of the edges with P(b | a) >= tau."""
    n = len(counts)
    return [[b for b in range(n) if transition_prob(counts, a, b, eps) >= tau] for a in range(n)]


def hop_distances(graph, source):
    """Breadth-first hop distance from ``source``; None where unreachable."""
    dist = [None] * len(graph)
    dist[source] = 0
    queue = deque([source])
    while queue:
        a = queue.popleft()
        for b in graph[a]:
            if dist[b] is None:
                dist[b] = dist[a] + 1
                queue.append(b)
    return dist


def survival(hops, a, e_max):
    """Eq. (8)."""
    e = hops[a]
    if e is None:
        return 0.0
    return 1.0 - min(e, e_max) / e_max


def block_score(p_surv, age, tokens, lam, delta):
    """Eq. (9)."""
    return (p_surv + delta) * (math.exp(-lam * age) + delta) * tokens


def entropy(probs):
    return -sum(p * math.log2(p) for p in probs if p > 0)


def predictability(counts):
    """Eq. (2) over the observed transitions: R = 1 - H(next | current) / H(next).

    No transitions: R = 0.  A single successor overall (H(next) = 0): R = 1.
    """
    n = len(counts)
    total = sum(sum(row) for row in counts)
    if total == 0:
        return 0.0
    next_marg = [sum(counts[i][j] for i in range(n)) / total for j in range(n)]
    h_next = entropy(next_marg)
    h_cond = 0.0
    for i in range(n):
        ri = sum(counts[i])
        if ri:
            h_cond += (ri / total) * entropy([c / ri for c in counts[i]])
    if h_next == 0.0:
        return 1.0
    return 1.0 - h_cond / h_next


class ControlPlane:
    """The runtime state and procedures, one agent id per prompt fingerprint."""

    def __init__(self, num_agents, num_blocks, **params):
        self.p = dict(DEFAULTS, **params)
        self.n = num_agents
        self.counts = [[0] * num_agents for _ in range(num_agents)]
        self.current = None
        self.hops = [None] * num_agents
        self.agent_of = [None] * num_blocks
        self.last_access = [0] * num_blocks
        self.tokens = [0] * num_blocks
        self.host_resident = [False] * num_blocks
        self.fingerprints = {}

    def agent_id(self, fingerprint):
        """Dense agent id of a prompt-prefix fingerprint (new ids in order of arrival)."""
        if fingerprint not in self.fingerprints:
            if len(self.fingerprints) == self.n:
                return None
            self.fingerprints[fingerprint] = len(self.fingerprints)
        return self.fingerprints[fingerprint]

    def observe_touch(self, block, agent, tokens, now):
        self.agent_of[block] = agent
        self.last_access[block] = now
        self.tokens[block] = tokens
        if agent != self.current:
            if self.current is not None:
                self.counts[self.current][agent] += 1
            graph = threshold_graph(self.counts, self.p["eps"], self.p["tau"])
            self.hops = hop_distances(graph, agent)
            self.current = agent

    def survival(self, agent):
        if self.current is None:
            return 0.0
        return survival(self.hops, agent, self.p["e_max"])

    def score_block(self, block, now):
        a = self.agent_of[block]
        ps = 0.0 if a is None else self.survival(a)
        return block_score(ps, now - self.last_access[block], self.tokens[block],
                           self.p["lam"], self.p["delta"])

    def set_host_resident(self, block, resident):
        self.host_resident[block] = bool(resident)

    def survival_all(self):
        return [self.survival(a) for a in range(self.n)]

    def select_victim(self, candidates, now):
        """Lowest score; among equal scores a CPU-resident block; then the first."""
        keys = [(self.score_block(b, now), 0 if self.host_resident[b] else 1) for b in candidates]
        return candidates[keys.index(min(keys))]

    def predictability(self):
        return predictability(self.counts)

    def between_step(self):
        """Eq. (10)-(11): the agent to warm up, or None when the gate is closed."""
        if self.current is None or self.predictability() < self.p["r_min"]:
            return None
        return predict_next(self.counts, self.current, self.p["eps"])
