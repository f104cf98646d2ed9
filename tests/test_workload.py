"""The seeded generator: determinism, layout round trip, poisoning, config shapes."""

import numpy as np
import pytest

from paper_2608_14624_amd import workload as W


def small():
    invs = [W.Invocation(0, 9), W.Invocation(1, 40), W.Invocation(0, 3, hit=False),
            W.Invocation(1, 16)]
    return W.build_workload("t", 3, [21, 48], invs, num_q_heads=4, num_kv_heads=2,
                            head_dim=8, num_blocks=64)


def test_bf16_rounding_is_nearest_even():
    x = np.array([1.0, 1.0 + 2**-8, 1.0 + 3 * 2**-8, -2.5, 1.0 + 2**-9], dtype=np.float32)
    got = W.f32_to_bf16_bits(x)
    # 1+2^-8 is a tie -> even (1.0); 1+3*2^-8 is a tie -> even (1+2^-6... = 0x3F82)
    assert got.tolist() == [0x3F80, 0x3F80, 0x3F82, 0xC020, 0x3F80]


def test_generator_is_deterministic():
    a, b = small(), small()
    for f in ("q", "k_pool", "v_pool", "block_tables", "prefix_lens", "cu_q_lens"):
        assert np.array_equal(getattr(a, f), getattr(b, f))


def test_layout_round_trip_and_poison():
    wl = small()
    bs = wl.block_size
    touched = np.zeros(wl.num_blocks, dtype=bool)
    for r in range(wl.batch):
        q, k, v = wl.logical_sequence(r)
        length = int(wl.kv_lens[r])
        assert k.shape[0] == length
        n = -(-length // bs)
        slots = wl.block_tables[r, :n]
        touched[slots] = True
        paged_k = wl.k_pool[slots].transpose(0, 2, 1, 3).reshape(n * bs, wl.num_kv_heads, -1)
        paged_v = wl.v_pool[slots].transpose(0, 2, 1, 3).reshape(n * bs, wl.num_kv_heads, -1)
        assert np.array_equal(paged_k[:length], k) and np.array_equal(paged_v[:length], v)
        tail = paged_k[length:]
        assert np.all((tail == W.BF16_TAIL_POS) | (tail == W.BF16_TAIL_NEG))
        c0, c1 = wl.cu_q_lens[r], wl.cu_q_lens[r + 1]
        assert np.array_equal(wl.q[c0:c1], q)
        # entries past the last block point at a NaN slot
        assert np.all(wl.k_pool[wl.block_tables[r, n:]] == W.BF16_NAN)
    assert np.all(wl.k_pool[~touched] == W.BF16_NAN)
    assert touched.sum() == wl.meta["used_blocks"]


def test_hits_share_anchor_blocks_and_misses_do_not():
    wl = small()
    # invocations 0 and 2 are agent 0 (21 tokens: 1 full block); 0 is a hit, 2 a miss
    assert wl.block_tables[0, 0] != wl.block_tables[2, 0]
    invs = [W.Invocation(0, 5), W.Invocation(0, 7)]
    wl2 = W.build_workload("s", 4, [40], invs, num_q_heads=2, num_kv_heads=1,
                           head_dim=8, num_blocks=16)
    assert np.array_equal(wl2.block_tables[0, :2], wl2.block_tables[1, :2])
    assert wl2.block_tables[0, 2] != wl2.block_tables[1, 2]      # private tail blocks


def test_tiny_config_matches_its_recipe():
    wl = W.make_config("tiny")
    assert (wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.num_blocks) == (8, 2, 64, 64)
    assert wl.prefix_lens.tolist() == [256] and wl.cu_q_lens.tolist() == [0, 64]
    assert wl.scale == 0.125
    slots = np.random.default_rng([0, 0]).permutation(64)[:20]
    assert np.array_equal(wl.block_tables[0], slots)
    assert wl.flops() == 4 * 64 * 8 * (64 * 256 + 64 * 65 // 2)


@pytest.mark.parametrize("name,flops", [("llama8b", 4.296e10), ("llama70b_prefetch", 1.168e12)])
def test_fixed_config_flops(name, flops):
    spec = W.config_spec(name)
    s = np.array([i.suffix_len for i in spec["invocations"]], dtype=np.int64)
    p = np.array([spec["anchor_lens"][i.agent] for i in spec["invocations"]], dtype=np.int64)
    f = 4 * spec["head_dim"] * spec["num_q_heads"] * np.sum(s * p + s * (s + 1) // 2)
    assert abs(f / flops - 1) < 1e-3


def test_random_config_recipes():
    ab = W.config_spec("agent_batch")
    assert len(ab["invocations"]) == 32 and len(ab["anchor_lens"]) == 4
    assert all(1536 <= a <= 3072 for a in ab["anchor_lens"])
    assert all(256 <= i.suffix_len <= 2048 for i in ab["invocations"])
    lm = W.config_spec("long_mixed")
    invs = lm["invocations"]
    assert len(invs) == 128 and sum(i.hit for i in invs) == 77
    assert all(128 <= i.suffix_len <= 4096 for i in invs)
    assert all(4096 <= a <= 8192 for a in lm["anchor_lens"])
    p70 = W.config_spec("llama70b_prefetch")
    agents = [i.agent for i in p70["invocations"]]
    assert agents == sorted(agents) and p70["offpool_per_agent"] == 64


def test_offpool_blocks_are_nan_until_prefetched():
    invs = [W.Invocation(0, 20), W.Invocation(1, 3)]
    wl = W.build_workload("off", 9, [64, 80], invs, num_q_heads=4, num_kv_heads=2,
                          head_dim=8, num_blocks=64, offpool_per_agent=2)
    assert wl.prefetch_dst.shape == (4,) and wl.host_k.shape == (4, 2, 16, 8)
    assert np.all(wl.k_pool[wl.prefetch_dst] == W.BF16_NAN)
    assert len(np.unique(wl.prefetch_dst)) == 4
    assert set(wl.prefetch_agent.tolist()) == {0, 1}


@pytest.mark.parametrize("shard,full", [("llama70b_prefetch_tp8", "llama70b_prefetch"),
                                        ("agent_batch_tp8", "agent_batch")])
def test_tp8_shard_configs_are_the_full_invocations_with_an_eighth_of_the_heads(shard, full):
    a, b = W.config_spec(shard), W.config_spec(full)
    assert a["num_q_heads"] * 8 == b["num_q_heads"] and a["num_kv_heads"] * 8 == b["num_kv_heads"]
    assert a["num_kv_heads"] == 1
    assert a["invocations"] == b["invocations"] and a["anchor_lens"] == b["anchor_lens"]
