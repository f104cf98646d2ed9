"""The C++ control plane (cs_scout_*) against the oracle, on the CPU.

Random agent traces drive both sides with the same touches; after every touch
every query is compared: integer decisions (current agent, prediction,
prefetch target, eviction victim, hop-derived survival) exactly, floating
values (Eq. (2), (3), (9)) to 1e-12 relative.  Both sides evaluate the same
fp64 expressions, so the decisions at a threshold (an edge with P exactly
tau, a gate with R exactly R_min) agree too; the small-count traces below are
built to hit such ties.
"""

import ctypes
import math
import random

import numpy as np

import pytest

import oracle.control_plane as cp

ops = pytest.importorskip("paper_2608_14624_amd.ops",
                          reason="libcachescout.so not built (run __graft_entry__.build())")

REL = 1e-12


def markov_trace(rng, num_agents, steps, noise):
    """A ring of agents with random shortcuts; `noise` is the chance of a
    uniformly random successor instead of the ring's."""
    succ = [(a + 1) % num_agents if rng.random() < 0.7 else rng.randrange(num_agents)
            for a in range(num_agents)]
    a = rng.randrange(num_agents)
    out = []
    for _ in range(steps):
        for _ in range(rng.randint(1, 3)):      # an agent touches a few blocks per turn
            out.append(a)
        a = rng.randrange(num_agents) if rng.random() < noise else succ[a]
    return out


def params_for(rng):
    return dict(eps=rng.choice([0.1, 0.5, 1.0, 0.05]), tau=rng.choice([0.1, 0.2, 0.25, 0.5]),
                e_max=rng.choice([2, 3, 4, 6]), lam=rng.choice([0.0, 0.1, 0.5]),
                delta=rng.choice([0.0, 0.05]), r_min=rng.choice([0.0, 0.3, 0.5]))


def compare_state(oracle_plane, scout, num_agents, num_blocks, now, rng):
    assert scout.current == oracle_plane.current
    for i in range(num_agents):
        for j in range(num_agents):
            want = cp.transition_prob(oracle_plane.counts, i, j, oracle_plane.p["eps"])
            assert scout.transition_prob(i, j) == pytest.approx(want, rel=REL)
    want_pred = (None if oracle_plane.current is None
                 else cp.predict_next(oracle_plane.counts, oracle_plane.current,
                                      oracle_plane.p["eps"]))
    assert scout.predict() == want_pred
    for a in range(num_agents):
        assert scout.survival(a) == oracle_plane.survival(a)
    for b in range(num_blocks):
        assert scout.score_block(b, now) == pytest.approx(oracle_plane.score_block(b, now),
                                                          rel=REL, abs=1e-300)
    assert scout.survival_all() == oracle_plane.survival_all()
    cands = rng.sample(range(num_blocks), rng.randint(1, num_blocks))
    assert scout.select_victim(cands, now) == oracle_plane.select_victim(cands, now)
    # same expressions in the same order: equal, not just close
    assert scout.predictability() == oracle_plane.predictability()
    assert scout.between_step() == oracle_plane.between_step()


@pytest.mark.parametrize("seed", range(12))
def test_random_traces_match_the_oracle(seed):
    rng = random.Random(1000 + seed)
    num_agents = rng.randint(2, 12)
    num_blocks = rng.randint(4, 40)
    prm = params_for(rng)
    oracle_plane = cp.ControlPlane(num_agents, num_blocks, **prm)
    scout = ops.Scout(num_agents, num_blocks, **prm)
    trace = markov_trace(rng, num_agents, rng.randint(20, 80), rng.choice([0.0, 0.1, 0.4]))
    for now, agent in enumerate(trace):
        block = rng.randrange(num_blocks)
        tokens = rng.choice([16, 16, 16, 7, 1])
        oracle_plane.observe_touch(block, agent, tokens, now)
        scout.observe_touch(block, agent, tokens, now)
        if rng.random() < 0.2:
            flag = rng.random() < 0.5
            oracle_plane.set_host_resident(block, flag)
            scout.set_host_resident(block, flag)
        if now % 5 == 0 or now == len(trace) - 1:
            compare_state(oracle_plane, scout, num_agents, num_blocks,
                          now + rng.randint(0, 20), rng)


@pytest.mark.parametrize("seed", range(6))
def test_threshold_ties_decided_alike(seed):
    # few agents, small counts, tau a multiple of 1/A: P == tau in exact
    # arithmetic happens often (e.g. (1 + 0.1) / (5 + 0.5) = 0.2)
    rng = random.Random(7 + seed)
    num_agents = rng.choice([2, 4, 5])
    prm = dict(eps=rng.choice([0.1, 0.5, 1.0]), tau=rng.choice([0.2, 0.25, 0.5]), e_max=3,
               lam=0.1, delta=0.05, r_min=rng.choice([0.0, 0.5, 1.0]))
    oracle_plane = cp.ControlPlane(num_agents, 4, **prm)
    scout = ops.Scout(num_agents, 4, **prm)
    for now in range(60):
        a = rng.randrange(num_agents)
        oracle_plane.observe_touch(now % 4, a, 16, now)
        scout.observe_touch(now % 4, a, 16, now)
        assert scout.current == oracle_plane.current
        for x in range(num_agents):
            assert scout.survival(x) == oracle_plane.survival(x)
        assert scout.between_step() == oracle_plane.between_step()


def test_batched_touches_equal_single_touches():
    rng = random.Random(5)
    n_agents, n_blocks = 7, 50
    trace = markov_trace(rng, n_agents, 200, 0.2)
    blocks = np.array([rng.randrange(n_blocks) for _ in trace], dtype=np.int32)
    tokens = np.array([rng.choice([16, 3]) for _ in trace], dtype=np.int32)
    now = np.arange(len(trace), dtype=np.int64) * 3
    one, many = ops.Scout(n_agents, n_blocks), ops.Scout(n_agents, n_blocks)
    for i, a in enumerate(trace):
        one.observe_touch(int(blocks[i]), a, int(tokens[i]), int(now[i]))
    many.observe_touches(blocks, np.array(trace), tokens, now)
    t = int(now[-1]) + 4
    assert many.current == one.current and many.predictability() == one.predictability()
    assert many.survival_all() == one.survival_all()
    assert [many.score_block(b, t) for b in range(n_blocks)] == \
        [one.score_block(b, t) for b in range(n_blocks)]
    # a bad entry anywhere rejects the whole batch
    fresh = ops.Scout(n_agents, n_blocks)
    bad_agents = np.array(trace)
    bad_agents[-1] = n_agents
    with pytest.raises(ops.CacheScoutError):
        fresh.observe_touches(blocks, bad_agents, tokens, now)
    assert fresh.current is None
    fresh.observe_touches(blocks[:0], bad_agents[:0], tokens[:0], now[:0])   # n = 0


def test_hand_trace_values():
    scout = ops.Scout(4, 10, eps=0.1, tau=0.3, e_max=3)
    trace = [(0, 0), (1, 0), (2, 1), (3, 2), (4, 0), (5, 1), (6, 2), (7, 0), (8, 1)]
    for now, (block, agent) in enumerate(trace):
        scout.observe_touch(block, agent, 16, now)
    assert scout.current == 1
    assert [scout.survival(a) for a in range(4)] == [1 - 2 / 3, 1.0, 1 - 1 / 3, 0.0]
    assert scout.transition_prob(0, 1) == pytest.approx(3.1 / 3.4, rel=REL)
    assert scout.predict() == 2 and scout.between_step() == 2
    assert scout.predictability() == pytest.approx(1.0)   # deterministic cycle
    assert scout.select_victim([6, 9, 8], 9) == 9


def test_fresh_plane_and_gate():
    scout = ops.Scout(3, 2)
    assert scout.current is None and scout.predict() is None and scout.between_step() is None
    assert scout.survival(0) == 0.0 and scout.predictability() == 0.0
    scout.observe_touch(0, 2, 16, 0)
    assert scout.current == 2 and scout.predictability() == 0.0   # no transition yet
    assert scout.between_step() is None                           # R = 0 < 0.3
    # a score of a never-touched block is 0 (no tokens)
    assert scout.score_block(1, 5) == 0.0


def test_agent_ids_dense_and_bounded():
    scout = ops.Scout(2, 1)
    assert scout.agent_id(0xBEEF) == 0 and scout.agent_id(0xCAFE) == 1
    assert scout.agent_id(0xBEEF) == 0 and scout.agent_id(0xF00D) is None
    assert scout.agent_id(2 ** 64 - 1) is None


def test_state_size_is_what_the_header_states():
    scout = ops.Scout(64, 1000)
    assert scout.state_bytes() == 4 * 64 * 64 + 28 * 64 + 17 * 1000
    # the paper's operating point, 24 agents: the agent-side state is small
    assert ops.Scout(24, 0).state_bytes() == 4 * 24 * 24 + 28 * 24 < 25 * 1024


def test_cpu_resident_tie_break():
    scout = ops.Scout(2, 4)
    for b in range(4):
        scout.observe_touch(b, 0, 16, 5)
    assert scout.select_victim([0, 1, 2, 3], 6) == 0
    scout.set_host_resident(2, True)
    assert scout.select_victim([0, 1, 2, 3], 6) == 2
    scout.observe_touch(3, 0, 8, 5)
    assert scout.select_victim([0, 1, 2, 3], 6) == 3
    with pytest.raises(ops.CacheScoutError):
        scout.set_host_resident(4, True)


def test_invalid_arguments_are_rejected():
    scout = ops.Scout(3, 4)
    for bad in [(4, 0, 16, 0), (-1, 0, 16, 0), (0, 3, 16, 0), (0, -1, 16, 0), (0, 0, -1, 0)]:
        with pytest.raises(ops.CacheScoutError) as e:
            scout.observe_touch(*bad)
        assert e.value.status == ops.CS_ERR_INVALID_ARG
    assert scout.current is None                     # nothing was recorded
    assert math.isnan(scout.transition_prob(3, 0)) and math.isnan(scout.survival(-1))
    assert math.isnan(scout.score_block(4, 0))
    assert scout.select_victim([0, 9], 0) is None and scout.select_victim([], 0) is None
    for kwargs in [dict(eps=0.0), dict(tau=1.5), dict(e_max=0), dict(lam=-1.0),
                   dict(delta=-0.1), dict(r_min=float("nan"))]:
        with pytest.raises(ops.CacheScoutError):
            ops.Scout(3, 4, **kwargs)
    for na, nb in [(0, 4), (5000, 4), (3, -1)]:
        with pytest.raises(ops.CacheScoutError):
            ops.Scout(na, nb)
    with pytest.raises(TypeError):
        ops.Scout(3, 4, gamma=1.0)


def test_null_handle_is_rejected():
    lib = ctypes.CDLL(ops.LIB_PATH)
    lib.cs_scout_observe_touch.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
                                           ctypes.c_int32, ctypes.c_int64]
    assert lib.cs_scout_observe_touch(None, 0, 0, 16, 0) == ops.CS_ERR_INVALID_ARG
    lib.cs_scout_predict.argtypes = [ctypes.c_void_p]
    assert lib.cs_scout_predict(None) == -1
    lib.cs_scout_destroy.argtypes = [ctypes.c_void_p]
    lib.cs_scout_destroy(None)


def test_scout_policy_targets_on_a_dispatch_cycle():
    """The policy the GPU pipeline uses, host side only: four agents served in
    a fixed cycle.  The first pass predicts from empty rows (the first turn has
    no transition, so the gate is closed); from the second pass on, every
    prediction is the next agent."""
    from paper_2608_14624_amd import workload as W
    from paper_2608_14624_amd.pipeline import ScoutPolicy
    invs = [W.Invocation(a, 5) for a in (0, 0, 1, 2, 2, 3)]
    wl = W.build_workload("cycle", 4, [64, 48, 80, 33], invs, num_q_heads=4, num_kv_heads=2,
                          head_dim=8, num_blocks=96, offpool_per_agent=1)
    order = [0, 1, 2, 3]
    pol = ScoutPolicy(wl, order)
    got = [[pol.on_turn(a) for a in order] for _ in range(3)]
    # pass 1: no transition yet (gate closed), then rows with no counts (uniform
    # row: lowest id, agent 0), which is right only for the last turn
    assert got[0] == [None, 0, 0, 0]
    assert got[1] == [1, 2, 3, 0] and got[2] == [1, 2, 3, 0]
    sc = pol.scout
    assert sc.predictability() == 1.0 and sc.current == pol.ids[3]
    # every anchor block was recorded with its owner and token count
    blocks, tokens = pol.touches[3]
    assert len(blocks) == 3 and sorted(tokens) == [1, 16, 16]
