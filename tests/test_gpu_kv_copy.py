"""GPU tests of cs_kv_write (new tokens' K/V into pool slots) and cs_kv_offload
(pool blocks to pinned host memory): bit-exact against the NumPy oracles,
every other slot untouched, and the write-back feeding attention."""

import numpy as np
import pytest

import oracle
from paper_2608_14624_amd.workload import BF16_NAN, Invocation, build_workload

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def ops():
    from paper_2608_14624_amd import ops
    return ops


def bits(t):
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def to_dev(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()


def to_pinned(a):
    t = torch.empty(a.shape, dtype=torch.bfloat16, pin_memory=True)
    t.copy_(torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16))
    return t


@pytest.mark.parametrize("t,nb,hkv,d", [(1, 4, 1, 64), (37, 16, 2, 128), (1000, 128, 8, 128),
                                        (333, 64, 4, 64)])
def test_kv_write_is_bit_exact(ops, t, nb, hkv, d):
    print(f"[case] kv_write T={t} nb={nb} hkv={hkv} d={d}", flush=True)
    rng = np.random.default_rng(t + nb)
    kp = rng.integers(0, 2**16, size=(nb, hkv, 16, d), dtype=np.uint16)
    vp = rng.integers(0, 2**16, size=(nb, hkv, 16, d), dtype=np.uint16)
    kn = rng.integers(0, 2**16, size=(t, hkv, d), dtype=np.uint16)
    vn = rng.integers(0, 2**16, size=(t, hkv, d), dtype=np.uint16)
    slots = rng.choice(nb * 16, size=t, replace=False).astype(np.int32)
    slots[::5] = -1
    kd, vd = to_dev(kp), to_dev(vp)
    ops.cs_kv_write(to_dev(kn), to_dev(vn), torch.from_numpy(slots).cuda(), kd, vd)
    torch.cuda.synchronize()
    ek, ev = oracle.kv_write(kn, vn, slots, kp, vp)
    assert np.array_equal(bits(kd), ek) and np.array_equal(bits(vd), ev)


def test_kv_write_then_attention(ops):
    """The suffix K/V of each invocation starts NaN in the pool and arrives
    through cs_kv_write before the attention that reads it."""
    from paper_2608_14624_amd import pipeline
    invs = [Invocation(0, 70), Invocation(1, 33), Invocation(0, 5, hit=False)]
    wl = build_workload("writeback", 21, [100, 48], invs, num_q_heads=8, num_kv_heads=2,
                        head_dim=128, num_blocks=96)
    # logical positions of every suffix token and the slot it lives in
    k_rows, v_rows, slots = [], [], []
    for r in range(wl.batch):
        _, k, v = wl.logical_sequence(r)
        p = int(wl.prefix_lens[r])
        s = int(wl.q_lens[r])
        for j in range(p, p + s):
            slots.append(int(wl.block_tables[r, j // 16]) * 16 + j % 16)
            k_rows.append(k[j])
            v_rows.append(v[j])
    k_rows, v_rows = np.stack(k_rows), np.stack(v_rows)
    slots = np.array(slots, dtype=np.int32)
    full_k, full_v = wl.k_pool.copy(), wl.v_pool.copy()
    kf = wl.k_pool.transpose(0, 2, 1, 3).reshape(-1, 2, 128)
    vf = wl.v_pool.transpose(0, 2, 1, 3).reshape(-1, 2, 128)
    kf[slots] = BF16_NAN
    vf[slots] = BF16_NAN
    wl.k_pool = np.ascontiguousarray(kf.reshape(96, 16, 2, 128).transpose(0, 2, 1, 3))
    wl.v_pool = np.ascontiguousarray(vf.reshape(96, 16, 2, 128).transpose(0, 2, 1, 3))
    dw = pipeline.DeviceWorkload(wl)
    ops.cs_kv_write(to_dev(k_rows), to_dev(v_rows), torch.from_numpy(slots).cuda(),
                    dw.k_pool, dw.v_pool)
    dw.attention()
    torch.cuda.synchronize()
    assert np.array_equal(bits(dw.k_pool), full_k) and np.array_equal(bits(dw.v_pool), full_v)
    ref = oracle.prefill_paged_attn(wl.q, full_k, full_v, wl.block_tables, wl.prefix_lens,
                                    wl.cu_q_lens, 8, 2, wl.scale)
    got = oracle.bf16_bits_to_f64(dw.out_bits())
    err = np.abs(got - ref)
    assert np.isfinite(got).all() and err.max() <= 2e-2 and err.mean() <= 2e-3


@pytest.mark.parametrize("n,nb,hkv,d", [(1, 8, 1, 64), (64, 300, 8, 128), (13, 40, 2, 128)])
def test_kv_offload_is_bit_exact(ops, n, nb, hkv, d):
    print(f"[case] kv_offload n={n} nb={nb} hkv={hkv} d={d}", flush=True)
    rng = np.random.default_rng(n * 7 + nb)
    kp = rng.integers(0, 2**16, size=(nb, hkv, 16, d), dtype=np.uint16)
    vp = rng.integers(0, 2**16, size=(nb, hkv, 16, d), dtype=np.uint16)
    ids = rng.integers(0, nb, size=n).astype(np.int32)          # repeats allowed
    hk = torch.zeros((n, hkv, 16, d), dtype=torch.bfloat16, pin_memory=True)
    hv = torch.zeros((n, hkv, 16, d), dtype=torch.bfloat16, pin_memory=True)
    ops.cs_kv_offload(torch.from_numpy(ids).cuda(), to_dev(kp), to_dev(vp), hk, hv)
    torch.cuda.synchronize()
    ek, ev = oracle.kv_offload(ids, kp, vp)
    assert np.array_equal(hk.view(torch.int16).numpy().view(np.uint16), ek)
    assert np.array_equal(hv.view(torch.int16).numpy().view(np.uint16), ev)


def test_offload_then_prefetch_restores_the_pool(ops):
    rng = np.random.default_rng(9)
    kp = rng.integers(0, 2**16, size=(50, 2, 16, 128), dtype=np.uint16)
    vp = rng.integers(0, 2**16, size=(50, 2, 16, 128), dtype=np.uint16)
    kd, vd = to_dev(kp), to_dev(vp)
    ids = torch.tensor([3, 44, 17, 0], dtype=torch.int32, device="cuda")
    hk = torch.empty((4, 2, 16, 128), dtype=torch.bfloat16, pin_memory=True)
    hv = torch.empty_like(hk, pin_memory=True)
    ops.cs_kv_offload(ids, kd, vd, hk, hv)
    torch.cuda.synchronize()
    kd[ids.long()] = float("nan")
    vd[ids.long()] = float("nan")
    ops.cs_kv_prefetch(hk, hv, ids, kd, vd)
    torch.cuda.synchronize()
    assert np.array_equal(bits(kd), kp) and np.array_equal(bits(vd), vp)


def test_kv_write_debug_check_rejects_duplicate_slots(ops, monkeypatch):
    monkeypatch.setenv("CS_DEBUG_CHECK", "1")
    pool = torch.zeros((4, 1, 16, 64), dtype=torch.bfloat16, device="cuda")
    rows = torch.zeros((3, 1, 64), dtype=torch.bfloat16, device="cuda")
    slots = torch.tensor([5, -1, 5], dtype=torch.int32, device="cuda")
    with pytest.raises(ops.CacheScoutError) as ei:
        ops.cs_kv_write(rows, rows, slots, pool, pool.clone())
    assert "duplicate" in str(ei.value)
    slots = torch.tensor([5, -1, 64], dtype=torch.int32, device="cuda")
    with pytest.raises(ops.CacheScoutError):
        ops.cs_kv_write(rows, rows, slots, pool, pool.clone())
