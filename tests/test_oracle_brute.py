"""Pin the float64 oracle against a scalar brute force on tiny inputs.

The brute force reads the logical (unpaged) token arrays and uses Python
floats with math.exp / math.fsum; the oracle reads the paged pool through the
block table with NumPy.  Agreement to 1e-12 across prefix lengths that hit
block edges (0, 1, 15, 16, 17, ...), suffix lengths, GQA group sizes, head
dims and seeds pins the gather, the head map, the mask and the softmax.
"""

import itertools

import numpy as np
import pytest

import oracle
from paper_2608_14624_amd.workload import Invocation, build_workload

GRID = [
    # (prefix, suffix, group, kv_heads, head_dim)
    (0, 1, 1, 1, 8), (0, 17, 2, 2, 8), (1, 2, 4, 1, 8), (15, 17, 2, 1, 8),
    (16, 1, 1, 2, 8), (16, 17, 4, 2, 8), (17, 2, 2, 2, 8), (17, 64, 1, 1, 8),
    (256, 2, 2, 1, 8), (256, 17, 4, 1, 8), (15, 2, 1, 1, 64), (17, 1, 2, 1, 64),
    (33, 5, 4, 1, 64),
]


def _check(wl, samples_per_seq=None):
    out = oracle.prefill_paged_attn(wl.q, wl.k_pool, wl.v_pool, wl.block_tables,
                                    wl.prefix_lens, wl.cu_q_lens, wl.num_q_heads,
                                    wl.num_kv_heads, wl.scale)
    g_size = wl.num_q_heads // wl.num_kv_heads
    for r in range(wl.batch):
        q, k, v = wl.logical_sequence(r)
        qf = oracle.bf16_bits_to_f64(q)
        kf = oracle.bf16_bits_to_f64(k)
        vf = oracle.bf16_bits_to_f64(v)
        p = int(wl.prefix_lens[r])
        c0 = int(wl.cu_q_lens[r])
        for h in range(wl.num_q_heads):
            g = h // g_size
            ref = oracle.brute_attention_rows(qf[:, h, :].tolist(), kf[:, g, :].tolist(),
                                              vf[:, g, :].tolist(), p, wl.scale)
            got = out[c0:c0 + q.shape[0], h, :]
            np.testing.assert_allclose(got, np.array(ref), rtol=0, atol=1e-12)


@pytest.mark.parametrize("seed", [0, 1, 2])
@pytest.mark.parametrize("case", GRID, ids=lambda c: "P%d_S%d_G%d_H%d_D%d" % c)
def test_oracle_matches_brute_force(case, seed):
    p, s, g, hkv, d = case
    wl = build_workload("brute", 100 + seed, [p], [Invocation(0, s)],
                        num_q_heads=g * hkv, num_kv_heads=hkv, head_dim=d,
                        num_blocks=64)
    _check(wl)


def test_oracle_matches_brute_force_varlen_batch():
    # several invocations, shared anchors, a miss, odd prefix lengths, packed queries
    invs = [Invocation(0, 5), Invocation(1, 17), Invocation(0, 1, hit=False),
            Invocation(1, 3), Invocation(0, 16)]
    wl = build_workload("brute_batch", 7, [19, 32], invs, num_q_heads=4,
                        num_kv_heads=2, head_dim=8, num_blocks=64)
    assert wl.batch == 5 and wl.prefix_lens.tolist() == [19, 32, 0, 32, 19]
    _check(wl)


def test_oracle_matches_brute_force_peaky_logits():
    # queries x8: softmax close to one-hot, exercises the max subtraction
    wl = build_workload("peaky", 11, [40], [Invocation(0, 9)], num_q_heads=2,
                        num_kv_heads=1, head_dim=16, num_blocks=32, q_gain=8.0)
    _check(wl)
