"""Pins of the prefetch oracle: written slots equal the host blocks bitwise,
every other slot is untouched, the inputs are not modified."""

import numpy as np
import pytest

import oracle
from paper_2608_14624_amd.workload import make_config, Invocation, build_workload


def test_prefetch_oracle_is_a_bitwise_scatter():
    rng = np.random.default_rng(0)
    pool_k = rng.integers(0, 2**16, size=(32, 2, 16, 8), dtype=np.uint16)
    pool_v = rng.integers(0, 2**16, size=(32, 2, 16, 8), dtype=np.uint16)
    host_k = rng.integers(0, 2**16, size=(5, 2, 16, 8), dtype=np.uint16)
    host_v = rng.integers(0, 2**16, size=(5, 2, 16, 8), dtype=np.uint16)
    dst = np.array([7, 0, 31, 12, 3], dtype=np.int32)
    k0, v0 = pool_k.copy(), pool_v.copy()
    nk, nv = oracle.kv_prefetch(host_k, host_v, dst, pool_k, pool_v)
    assert np.array_equal(pool_k, k0) and np.array_equal(pool_v, v0)
    for i, s in enumerate(dst):
        assert nk[s].tobytes() == host_k[i].tobytes()
        assert nv[s].tobytes() == host_v[i].tobytes()
    others = np.setdiff1d(np.arange(32), dst)
    assert nk[others].tobytes() == pool_k[others].tobytes()
    assert nv[others].tobytes() == pool_v[others].tobytes()


def test_prefetch_oracle_rejects_duplicate_slots():
    z = np.zeros((2, 1, 16, 8), np.uint16)
    with pytest.raises(AssertionError):
        oracle.kv_prefetch(z, z, np.array([3, 3]), np.zeros((8, 1, 16, 8), np.uint16),
                           np.zeros((8, 1, 16, 8), np.uint16))


def test_prefetch_restores_off_pool_anchor_blocks():
    # off-pool anchor blocks start as NaN; after the prefetch the pool equals
    # the pool of the same workload built with every block resident
    invs = [Invocation(0, 20), Invocation(1, 3), Invocation(0, 7)]
    kw = dict(num_q_heads=4, num_kv_heads=2, head_dim=8, num_blocks=64)
    off = build_workload("off", 9, [64, 80], invs, offpool_per_agent=2, **kw)
    full = build_workload("off", 9, [64, 80], invs, **kw)
    assert off.prefetch_dst is not None and len(off.prefetch_dst) == 4
    assert not np.array_equal(off.k_pool, full.k_pool)
    nk, nv = oracle.kv_prefetch(off.host_k, off.host_v, off.prefetch_dst, off.k_pool, off.v_pool)
    assert np.array_equal(nk, full.k_pool) and np.array_equal(nv, full.v_pool)
