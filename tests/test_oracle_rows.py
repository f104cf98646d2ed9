"""Pin of the row-by-row oracle against the full float64 oracle.

``oracle.prefill_paged_attn_rows`` is what the GPU tests check large
workloads with (sampled rows of the agent batch, the 70B-shape serving step,
the long mixed load, and every decode and cascade-decode test).  It has its
own row indexing and groups its samples by (invocation, KV head) for one
gather and one product per group, so it is tied here to
``oracle.prefill_paged_attn``, which the brute force, the invariants and the
golden case pin (Sec. 2.1 "Prefix caching": a hit is the last rows of a full
recompute).  The batch mixes hits and misses, prefixes that are not a
multiple of the block size, one-token suffixes and GQA groups of 1, 2 and 4;
the samples are shuffled across invocations and heads, so every group
collects rows from all over the sample list.  Two plausible mistakes planted
in the row oracle must be caught: the packed row one position early, and
the groups keyed by the invocation alone (every head of it would then read
the first sampled head's keys).
"""

import numpy as np
import pytest

import oracle
import oracle.paged_attention as pa
from paper_2608_14624_amd.workload import Invocation, build_workload


def varlen_batch(num_q_heads, num_kv_heads, seed):
    invs = [Invocation(0, 1), Invocation(1, 23), Invocation(2, 40, hit=False),
            Invocation(0, 17), Invocation(1, 1, hit=False), Invocation(2, 5)]
    # anchors of 37, 16 and 19 tokens: two of them not a multiple of 16
    return build_workload("rows", seed, [37, 16, 19], invs, num_q_heads=num_q_heads,
                          num_kv_heads=num_kv_heads, head_dim=16, num_blocks=96)


def all_rows_shuffled(wl, seed):
    rows = [(r, h, i) for r in range(wl.batch) for h in range(wl.num_q_heads)
            for i in range(int(wl.q_lens[r]))]
    order = np.random.default_rng(seed).permutation(len(rows))
    return [rows[k] for k in order]


def rows_error(wl, samples, **kw):
    full = oracle.prefill_paged_attn(wl.q, wl.k_pool, wl.v_pool, wl.block_tables,
                                     wl.prefix_lens, wl.cu_q_lens, wl.num_q_heads,
                                     wl.num_kv_heads, wl.scale)
    got = oracle.prefill_paged_attn_rows(wl.q, wl.k_pool, wl.v_pool, wl.block_tables,
                                         wl.prefix_lens, wl.cu_q_lens, wl.num_q_heads,
                                         wl.num_kv_heads, wl.scale, samples, **kw)
    want = np.stack([full[int(wl.cu_q_lens[r]) + i, h] for r, h, i in samples])
    return float(np.abs(got - want).max())


HEADS = [(2, 2), (4, 2), (8, 2)]     # GQA groups 1, 2 and 4


@pytest.mark.parametrize("hq,hkv", HEADS)
def test_rows_equal_the_full_oracle(hq, hkv):
    wl = varlen_batch(hq, hkv, seed=31)
    assert (wl.prefix_lens % 16 != 0).any() and (wl.prefix_lens == 0).any()
    assert (wl.q_lens == 1).any()
    samples = all_rows_shuffled(wl, seed=hq)
    assert rows_error(wl, samples) <= 1e-12


def test_rows_sorted_and_repeated_samples():
    # sorted order, repeated rows, and groups split over several products
    wl = varlen_batch(8, 2, seed=32)
    samples = sorted(all_rows_shuffled(wl, seed=1))
    samples = samples + samples[::7]
    assert rows_error(wl, samples) <= 1e-12
    assert rows_error(wl, samples, rows_per_product=3) <= 1e-12


ROW_MUTANTS = {
    "packed_row_one_early": ("packed_row", lambda cu, r, i: int(cu[r]) + i - 1),
    "groups_keyed_by_invocation": ("_kv_group_key", lambda r, g: r),
}


@pytest.mark.parametrize("name", sorted(ROW_MUTANTS))
def test_planted_row_mistake_is_caught(name, monkeypatch):
    attr, bad = ROW_MUTANTS[name]
    wl = varlen_batch(8, 2, seed=33)
    samples = all_rows_shuffled(wl, seed=5)
    monkeypatch.setattr(pa, attr, bad)
    assert rows_error(wl, samples) > 1e-3, f"mutation {name} was not caught"
