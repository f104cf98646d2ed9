"""Pins of the write-back and offload oracles: hand-checked small cases,
round trips through the layout, untouched slots, skipped tokens."""

import numpy as np
import pytest

import oracle


def test_kv_write_hand_case():
    # 2 blocks of 4 tokens, 1 head, D = 2; tokens land at slots 5, 0, -1, 7
    pool = np.zeros((2, 1, 4, 2), dtype=np.uint16)
    k_new = np.array([[[1, 2]], [[3, 4]], [[5, 6]], [[7, 8]]], dtype=np.uint16)
    nk, nv = oracle.kv_write(k_new, k_new + 10, [5, 0, -1, 7], pool, pool)
    want = np.zeros_like(pool)
    want[1, 0, 1] = [1, 2]      # slot 5 = block 1, offset 1
    want[0, 0, 0] = [3, 4]      # slot 0
    want[1, 0, 3] = [7, 8]      # slot 7; the token with slot -1 is skipped
    assert np.array_equal(nk, want)
    assert np.array_equal(nv[want != 0], (want + 10)[want != 0])
    assert np.count_nonzero(nv) == np.count_nonzero(want)


def test_kv_write_then_gather_round_trip():
    rng = np.random.default_rng(3)
    nb, hkv, bs, d, t = 20, 3, 16, 8, 57
    k_pool = rng.integers(0, 2**16, size=(nb, hkv, bs, d), dtype=np.uint16)
    v_pool = rng.integers(0, 2**16, size=(nb, hkv, bs, d), dtype=np.uint16)
    k_new = rng.integers(0, 2**16, size=(t, hkv, d), dtype=np.uint16)
    v_new = rng.integers(0, 2**16, size=(t, hkv, d), dtype=np.uint16)
    slots = rng.choice(nb * bs, size=t, replace=False)
    slots[::7] = -1
    nk, nv = oracle.kv_write(k_new, v_new, slots, k_pool, v_pool)
    flat_k = nk.transpose(0, 2, 1, 3).reshape(nb * bs, hkv, d)
    flat_v = nv.transpose(0, 2, 1, 3).reshape(nb * bs, hkv, d)
    keep = slots >= 0
    assert np.array_equal(flat_k[slots[keep]], k_new[keep])
    assert np.array_equal(flat_v[slots[keep]], v_new[keep])
    untouched = np.setdiff1d(np.arange(nb * bs), slots[keep])
    old_k = k_pool.transpose(0, 2, 1, 3).reshape(nb * bs, hkv, d)
    assert np.array_equal(flat_k[untouched], old_k[untouched])


def test_kv_write_rejects_duplicate_slots():
    z = np.zeros((2, 1, 4, 2), dtype=np.uint16)
    with pytest.raises(AssertionError):
        oracle.kv_write(np.zeros((2, 1, 2), np.uint16), np.zeros((2, 1, 2), np.uint16), [3, 3], z, z)


def test_offload_then_prefetch_is_identity():
    rng = np.random.default_rng(4)
    k_pool = rng.integers(0, 2**16, size=(30, 2, 16, 8), dtype=np.uint16)
    v_pool = rng.integers(0, 2**16, size=(30, 2, 16, 8), dtype=np.uint16)
    ids = np.array([4, 17, 0, 29])
    hk, hv = oracle.kv_offload(ids, k_pool, v_pool)
    assert hk.shape == (4, 2, 16, 8)
    assert np.array_equal(hk[1], k_pool[17]) and np.array_equal(hv[3], v_pool[29])
    # evict (poison) and reload into the same slots: the pool is restored
    poisoned_k, poisoned_v = k_pool.copy(), v_pool.copy()
    poisoned_k[ids] = 0x7FC0
    poisoned_v[ids] = 0x7FC0
    rk, rv = oracle.kv_prefetch(hk, hv, ids, poisoned_k, poisoned_v)
    assert np.array_equal(rk, k_pool) and np.array_equal(rv, v_pool)
