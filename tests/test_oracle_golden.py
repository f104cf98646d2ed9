"""The oracle on the hand-worked case stored in tests/golden/.

The fixture states its derivation in closed form; the test also re-derives
the closed forms with math.exp so that a typo in the stored decimals cannot
hide.
"""

import json
import math
import os

import numpy as np

import oracle
from paper_2608_14624_amd.workload import BF16_NAN, BF16_TAIL_NEG, BF16_TAIL_POS, f32_to_bf16_bits

HERE = os.path.dirname(os.path.abspath(__file__))


def load_case():
    with open(os.path.join(HERE, "golden", "hand_worked_prefix_hit.json")) as f:
        return json.load(f)


def build_pool(case, rows):
    bs, d = case["block_size"], case["head_dim"]
    pool = np.full((case["pool_num_blocks"], 1, bs, d), BF16_NAN, dtype=np.uint16)
    block = np.empty((bs, d), dtype=np.uint16)
    block[:] = np.where(np.arange(bs) % 2 == 0, BF16_TAIL_POS, BF16_TAIL_NEG)[:, None]
    block[:len(rows)] = f32_to_bf16_bits(np.array(rows, dtype=np.float32))
    pool[case["prompt_slot"], 0] = block
    return pool


def run(case, part):
    k_pool = build_pool(case, case["prompt_keys"])
    v_pool = build_pool(case, case["prompt_values"])
    sub = case[part]
    q = f32_to_bf16_bits(np.array(sub["queries"], dtype=np.float32))[:, None, :]
    s = q.shape[0]
    bt = np.array([[case["prompt_slot"]]], dtype=np.int32)
    return oracle.prefill_paged_attn(q, k_pool, v_pool, bt, np.array([sub["prefix_len"]]),
                                     np.array([0, s]), 1, 1, case["scale"])[:, 0, :]


def test_closed_forms_match_stored_decimals():
    case = load_case()
    e, e2 = math.e, math.exp(2.0)
    derived = [[e / (e + 1), 2 / (e + 1)], [(1 + 4 * e2) / (1 + 2 * e2), 6 * e2 / (1 + 2 * e2)]]
    np.testing.assert_allclose(case["hit"]["expected"], derived, rtol=0, atol=1e-15)


def test_oracle_hit_matches_hand_worked_values():
    case = load_case()
    np.testing.assert_allclose(run(case, "hit"), case["hit"]["expected"], rtol=0, atol=1e-14)


def test_oracle_miss_matches_hand_worked_values():
    case = load_case()
    np.testing.assert_allclose(run(case, "miss"), case["miss"]["expected"], rtol=0, atol=1e-14)
