"""Pins of the control-plane oracle: hand-computed values of Eq. (2), (3),
(8) and (9), an edge whose probability equals the threshold of Eq. (7)
exactly, closed forms of the predictability (deterministic cycle = 1,
successor independent of the current agent = 0), breadth-first hop
distances against an all-pairs shortest-path brute force, the exact survival
probability of Eq. (6) by path enumeration on small chains, the runtime
procedure on a hand trace, and planted mistakes that the pins must catch
(among them a strict comparison in Eq. (7) and the entropy of the current
agent's marginal in place of the next agent's in Eq. (2))."""

import itertools
import math
import random

import pytest

import oracle.control_plane as cp


def test_eq3_hand_values_and_rows_sum_to_one():
    counts = [[0, 3, 1], [2, 0, 0], [1, 1, 0]]
    assert cp.transition_prob(counts, 0, 1, 0.5) == pytest.approx(7 / 11, abs=1e-15)
    assert cp.transition_prob(counts, 1, 0, 0.5) == pytest.approx(5 / 7, abs=1e-15)
    assert cp.transition_prob(counts, 2, 2, 0.5) == pytest.approx(0.5 / 3.5, abs=1e-15)
    for i in range(3):
        assert sum(cp.transition_prob(counts, i, j, 0.5) for j in range(3)) == pytest.approx(1.0)


def test_prediction_is_row_argmax_with_lowest_id_on_ties():
    counts = [[0, 3, 3], [5, 0, 1], [0, 0, 0]]
    assert cp.predict_next(counts, 0, 0.1) == 1
    assert cp.predict_next(counts, 1, 0.1) == 0
    assert cp.predict_next(counts, 2, 0.1) == 0     # no data: uniform row


def test_eq2_closed_forms():
    cycle = [[0, 5, 0], [0, 0, 5], [5, 0, 0]]
    assert cp.predictability(cycle) == pytest.approx(1.0, abs=1e-12)
    independent = [[1, 2, 3], [2, 4, 6], [3, 6, 9]]
    assert cp.predictability(independent) == pytest.approx(0.0, abs=1e-12)
    # hand case: marginal (1/4, 3/4), H = 0.811278; H(next|cur) = 1/2
    r = cp.predictability([[1, 1], [0, 2]])
    h_next = -(0.25 * math.log2(0.25) + 0.75 * math.log2(0.75))
    assert r == pytest.approx(1 - 0.5 / h_next, abs=1e-12)
    assert r == pytest.approx(0.3836885, abs=1e-6)
    assert cp.predictability([[0, 0], [0, 0]]) == 0.0


def test_eq7_edge_exactly_on_tau_is_kept():
    # row 0 of five agents with counts (0, 1, 4, 0, 0): P(1 | 0) = (1 + 0.1) /
    # (5 + 5 * 0.1) = 1.1 / 5.5, exactly tau = 0.2 in float64; Eq. (7) keeps an
    # edge whose probability reaches the threshold
    counts = [[0, 1, 4, 0, 0], [0] * 5, [0] * 5, [0] * 5, [0] * 5]
    assert cp.transition_prob(counts, 0, 1, 0.1) == 0.2
    graph = cp.threshold_graph(counts, 0.1, 0.2)
    assert graph[0] == [1, 2]
    hops = cp.hop_distances(graph, 0)
    assert hops[1] == 1 and hops[2] == 1


def floyd_warshall(graph):
    n = len(graph)
    inf = float("inf")
    d = [[0 if i == j else (1 if j in graph[i] else inf) for j in range(n)] for i in range(n)]
    for k in range(n):
        for i in range(n):
            for j in range(n):
                if d[i][k] + d[k][j] < d[i][j]:
                    d[i][j] = d[i][k] + d[k][j]
    return d


@pytest.mark.parametrize("seed", range(6))
def test_bfs_hops_equal_all_pairs_shortest_paths(seed):
    rng = random.Random(seed)
    n = rng.randint(3, 9)
    counts = [[rng.choice([0, 0, 1, 2, 7]) for _ in range(n)] for _ in range(n)]
    graph = cp.threshold_graph(counts, 0.1, 0.25)
    sp = floyd_warshall(graph)
    for src in range(n):
        hops = cp.hop_distances(graph, src)
        for a in range(n):
            want = sp[src][a]
            assert (hops[a] is None) == (want == float("inf"))
            if hops[a] is not None:
                assert hops[a] == want


def test_eq8_and_eq9_hand_values():
    assert cp.survival([0, 1, 4, None, 7], 0, 4) == 1.0
    assert cp.survival([0, 1, 4, None, 7], 1, 4) == 0.75
    assert cp.survival([0, 1, 4, None, 7], 2, 4) == 0.0
    assert cp.survival([0, 1, 4, None, 7], 3, 4) == 0.0
    assert cp.survival([0, 1, 4, None, 7], 4, 4) == 0.0
    s = cp.block_score(0.75, 10, 16, 0.1, 0.05)
    assert s == pytest.approx(0.8 * (math.exp(-1.0) + 0.05) * 16, abs=1e-12)
    assert s == pytest.approx(5.348856, abs=1e-6)


def exact_survival(P, a0, a, K):
    """Eq. (6) by enumerating every path of K steps from a0."""
    n = len(P)
    total = 0.0
    for path in itertools.product(range(n), repeat=K):
        prob, prev = 1.0, a0
        for x in path:
            prob *= P[prev][x]
            prev = x
        if a in path:
            total += prob
    return total


def test_survival_approximation_orders_a_deterministic_pipeline():
    # 0 -> 1 -> 2 -> 3 -> 4 -> 0: the exact survival within K steps is 1 for
    # agents at most K hops ahead and 0 beyond; the approximation decreases
    # with the hop count, so it ranks the agents the same way
    n = 5
    counts = [[0] * n for _ in range(n)]
    for i in range(n):
        counts[i][(i + 1) % n] = 20
    P = [[cp.transition_prob(counts, i, j, 0.0) for j in range(n)] for i in range(n)]
    hops = cp.hop_distances(cp.threshold_graph(counts, 0.0, 0.5), 0)
    assert hops == [0, 1, 2, 3, 4]
    approx = [cp.survival(hops, a, 4) for a in range(1, n)]
    for K in (1, 2, 3):
        exact = [exact_survival(P, 0, a, K) for a in range(1, n)]
        assert exact == [1.0 if a <= K else 0.0 for a in range(1, n)]
    assert approx == sorted(approx, reverse=True) and approx[0] > approx[-1]


def test_survival_approximation_agrees_with_exact_on_a_stochastic_chain():
    # 0 goes to 1 (80%) or 2 (20%); 1 goes to 3; 2 goes to 3; 3 goes to 0.
    counts = [[0, 8, 2, 0], [0, 0, 0, 10], [0, 0, 0, 10], [10, 0, 0, 0]]
    P = [[cp.transition_prob(counts, i, j, 0.0) for j in range(4)] for i in range(4)]
    exact = {a: exact_survival(P, 0, a, 2) for a in (1, 2, 3)}
    assert exact[1] == pytest.approx(0.8) and exact[2] == pytest.approx(0.2)
    assert exact[3] == pytest.approx(1.0)
    hops = cp.hop_distances(cp.threshold_graph(counts, 0.0, 0.5), 0)
    # agent 2 falls below the confidence threshold: unreachable, survival 0
    assert hops[1] == 1 and hops[2] is None and hops[3] == 2
    s = {a: cp.survival(hops, a, 4) for a in (1, 2, 3)}
    assert s[1] > s[3] > s[2] == 0.0
    assert exact[1] > exact[2]


def test_runtime_procedure_on_a_hand_trace():
    plane = cp.ControlPlane(4, 10, eps=0.1, tau=0.3, e_max=3)
    trace = [(0, 0), (1, 0), (2, 1), (3, 2), (4, 0), (5, 1), (6, 2), (7, 0), (8, 1)]
    for now, (block, agent) in enumerate([(b, a) for b, a in trace]):
        plane.observe_touch(block, agent, 16, now)
    # transitions 0->1, 1->2, 2->0, 0->1, 1->2, 2->0, 0->1
    assert plane.counts[0][1] == 3 and plane.counts[1][2] == 2 and plane.counts[2][0] == 2
    assert sum(map(sum, plane.counts)) == 7
    assert plane.current == 1
    assert plane.hops[:3] == [2, 0, 1] and plane.hops[3] is None
    assert plane.survival(2) == pytest.approx(1 - 1 / 3)
    assert plane.between_step() == 2
    # the block of agent 2 touched at step 6 vs agent 3's never-touched slot
    assert plane.score_block(6, 9) > plane.score_block(9, 9)
    assert plane.select_victim([6, 9, 8], 9) == 9


def test_eviction_prefers_cpu_resident_blocks_among_equal_scores():
    plane = cp.ControlPlane(2, 4)
    for b in range(4):
        plane.observe_touch(b, 0, 16, 5)        # identical owner, age and size
    assert plane.select_victim([0, 1, 2, 3], 6) == 0
    plane.set_host_resident(2, True)
    assert plane.select_victim([0, 1, 2, 3], 6) == 2
    plane.observe_touch(3, 0, 8, 5)             # a smaller block scores lower
    assert plane.select_victim([0, 1, 2, 3], 6) == 3


def test_online_prediction_accuracy_on_a_markov_chain():
    # six agents, each with a dominant successor taken 80% of the time: the
    # online top-1 prediction approaches 0.8 once each row has a few counts
    rng = random.Random(3)
    n = 6
    succ = [3, 4, 0, 5, 1, 2]
    plane = cp.ControlPlane(n, 1)
    a, hits, total = 0, 0, 0
    for t in range(600):
        plane.observe_touch(0, a, 16, t)
        nxt = succ[a] if rng.random() < 0.8 else rng.choice([x for x in range(n) if x != succ[a]])
        if t >= 60:
            total += 1
            hits += cp.predict_next(plane.counts, a, 0.1) == nxt
        a = nxt
    assert 0.72 < hits / total < 0.88


def test_gate_closes_without_structure():
    plane = cp.ControlPlane(3, 4, r_min=0.5)
    rng = random.Random(1)
    for now in range(300):
        plane.observe_touch(0, rng.randrange(3), 16, now)
    assert plane.predictability() < 0.5
    assert plane.between_step() is None


def test_agent_ids_are_dense_in_arrival_order():
    plane = cp.ControlPlane(2, 1)
    assert plane.agent_id(0xBEEF) == 0 and plane.agent_id(0xCAFE) == 1
    assert plane.agent_id(0xBEEF) == 0 and plane.agent_id(0xF00D) is None


def _pins_hold():
    try:
        test_eq3_hand_values_and_rows_sum_to_one()
        test_eq7_edge_exactly_on_tau_is_kept()
        test_eq2_closed_forms()
        for seed in range(3):
            test_bfs_hops_equal_all_pairs_shortest_paths(seed)
        test_eq8_and_eq9_hand_values()
        test_runtime_procedure_on_a_hand_trace()
    except AssertionError:
        return False
    return True


MUTANTS = {
    "eps_only_in_numerator": ("transition_prob",
                              lambda counts, i, j, eps: (counts[i][j] + eps) / max(sum(counts[i]), 1)),
    "survival_off_by_one": ("survival",
                            lambda hops, a, e_max: 0.0 if hops[a] is None
                            else 1.0 - min(hops[a] + 1, e_max) / e_max),
    "recency_sign_flipped": ("block_score",
                             lambda p, age, tokens, lam, delta:
                             (p + delta) * (math.exp(lam * age) + delta) * tokens),
    "edge_needs_more_than_tau": ("threshold_graph",
                                 lambda counts, eps, tau: [
                                     [b for b in range(len(counts))
                                      if cp.transition_prob(counts, a, b, eps) > tau]
                                     for a in range(len(counts))]),
    "entropy_of_current_in_place_of_next": ("predictability",
                                            lambda counts: _predictability_row_marginal(counts)),
}


def _predictability_row_marginal(counts):
    """Eq. (2) with H(A_t), the current agent's marginal (row sums), taken
    for H(A_{t+1}), the next agent's marginal (column sums)."""
    n = len(counts)
    total = sum(sum(row) for row in counts)
    if total == 0:
        return 0.0
    h_wrong = cp.entropy([sum(counts[i]) / total for i in range(n)])
    h_cond = 0.0
    for i in range(n):
        ri = sum(counts[i])
        if ri:
            h_cond += (ri / total) * cp.entropy([c / ri for c in counts[i]])
    if h_wrong == 0.0:
        return 1.0
    return 1.0 - h_cond / h_wrong


def test_pins_pass_on_the_real_oracle():
    assert _pins_hold()


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_planted_mistakes_are_caught(name, monkeypatch):
    attr, bad = MUTANTS[name]
    monkeypatch.setattr(cp, attr, bad)
    assert not _pins_hold(), name
