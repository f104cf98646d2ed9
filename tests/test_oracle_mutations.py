"""Planted mistakes in the oracle must be caught by its pins.

Each mutation replaces one piece of the float64 oracle (on the CPU, inside
this test only) with a plausible wrong version: the mask without the
diagonal, the mask aligned to the start of the suffix, the wrong GQA head
map, the block table read in the wrong order, a dropped scale, a wrong bf16
widening.  The brute-force pin and the invariants must fail for every one of
them, which shows those pins have teeth.
"""

import numpy as np
import pytest

import oracle
import oracle.paged_attention as pa
from paper_2608_14624_amd.workload import Invocation, build_workload

from test_oracle_brute import _check
from test_oracle_golden import load_case, run


def pins_pass():
    """Run a compact set of the pins; True only if every one holds."""
    try:
        case = load_case()
        np.testing.assert_allclose(run(case, "hit"), case["hit"]["expected"], rtol=0, atol=1e-12)
        invs = [Invocation(0, 5), Invocation(1, 17), Invocation(0, 1, hit=False)]
        wl = build_workload("mut", 3, [19, 33], invs, num_q_heads=4, num_kv_heads=2,
                            head_dim=8, num_blocks=32)
        _check(wl)
    except AssertionError:
        return False
    return True


def wrong_gather_reversed_blocks(pool_bits, table_row, length, g, block_size):
    n_blocks = -(-length // block_size)
    slots = np.asarray(table_row[:n_blocks], dtype=np.int64)[::-1]
    tiles = pool_bits[slots, g]
    return oracle.bf16_bits_to_f64(tiles.reshape(n_blocks * block_size, -1)[:length])


def wrong_gather_head_axis(pool_bits, table_row, length, g, block_size):
    n_blocks = -(-length // block_size)
    slots = np.asarray(table_row[:n_blocks], dtype=np.int64)
    nb, h, bs, d = pool_bits.shape
    # reads the pool as if it were token-major [slot, token, head, D]
    tiles = pool_bits.reshape(nb, bs, h, d)[slots][:, :, g, :]
    return oracle.bf16_bits_to_f64(tiles.reshape(n_blocks * block_size, -1)[:length])


def wrong_bf16_as_fp16(bits):
    return np.asarray(bits, dtype=np.uint16).view(np.float16).astype(np.float64)


MUTATIONS = {
    "mask_drops_diagonal": ("visible_keys", lambda p, i: p + i),
    "mask_top_left": ("visible_keys", lambda p, i: i + 1),
    "gqa_modulo_head_map": ("kv_head_of", lambda h, hq, hkv: h % hkv),
    "blocks_reversed": ("gather_logical_kv", wrong_gather_reversed_blocks),
    "token_head_axes_swapped": ("gather_logical_kv", wrong_gather_head_axis),
    "scale_dropped": ("_scale64", lambda s: 1.0),
    "bf16_read_as_fp16": ("bf16_bits_to_f64", wrong_bf16_as_fp16),
}


def test_pins_pass_on_the_real_oracle():
    assert pins_pass()


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_planted_mistake_is_caught(name, monkeypatch):
    attr, bad = MUTATIONS[name]
    monkeypatch.setattr(pa, attr, bad)
    with np.errstate(all="ignore"):
        assert not pins_pass(), f"mutation {name} was not caught"
