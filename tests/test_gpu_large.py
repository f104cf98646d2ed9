"""GPU parity at the size limits (Sec. 2.1 "Prefix caching": a hit is the
last rows of a full recompute, whatever the pool and the context size).

* Blocks past 4 GiB of pool: a pool of 140,000 blocks of 8 KV heads x 16
  tokens x 128 dims holds 4.6 GB of K and as much of V (2.3e9 elements
  each, past the 2^31 a 32-bit element offset can reach).  The test's blocks
  sit at the pool's high end, so prefill (plain and with key parts), decode,
  write-back, offload and prefetch all address K/V past 2^31 elements from
  the pool base.  The expected values come from the oracle on the compact
  pool of the same workload (block ids shifted back), so they do not depend
  on the placement; copies are compared bit for bit.
* A 131,072-token prefix under a 512-token suffix (a split launch with key
  parts, and without), and the decode of that 131,584-token sequence:
  sampled rows against the row oracle (edge rows for every head).
"""

import numpy as np
import pytest

import oracle
from gpu_util import MAX_ABS, MEAN_ABS, compare_full, compare_rows, sample_rows
from paper_2608_14624_amd.workload import Invocation, build_workload, decode_view

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

HIGH_BLOCKS = 140_000     # x 8 heads x 16 x 128 = 2.29e9 elements per pool


def dev_bf16(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()


def bits(t):
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


@pytest.fixture(scope="module")
def high_pool():
    """The compact workload, and the same blocks placed at the end of a pool
    of HIGH_BLOCKS slots (slot 0 of the big pool all NaN: blocks past a
    sequence's end are loaded from there and must not leak)."""
    # few enough tiles (96) that the workspace call takes key parts
    wl = build_workload("high_slots", 23, [1000, 90], [Invocation(0, 100), Invocation(1, 41),
                                                       Invocation(0, 1)],
                        num_q_heads=32, num_kv_heads=8, head_dim=128, num_blocks=160)
    base = HIGH_BLOCKS - wl.num_blocks
    shape = (HIGH_BLOCKS,) + wl.k_pool.shape[1:]
    print(f"[case] pool of {HIGH_BLOCKS} blocks ({2 * np.prod(shape) / 2**30:.2f} GiB per pool), "
          f"the workload's {wl.num_blocks} blocks at slots {base}..", flush=True)
    kp = torch.empty(shape, dtype=torch.bfloat16, device="cuda")
    vp = torch.empty(shape, dtype=torch.bfloat16, device="cuda")
    kp[0].fill_(float("nan"))
    vp[0].fill_(float("nan"))
    kp[base:] = dev_bf16(wl.k_pool)
    vp[base:] = dev_bf16(wl.v_pool)
    bt = torch.from_numpy(wl.block_tables + base).cuda()
    yield wl, base, kp, vp, bt
    del kp, vp
    torch.cuda.empty_cache()


@pytest.mark.parametrize("workspace", [None, "auto"])
def test_prefill_with_blocks_past_4gib(high_pool, workspace):
    from paper_2608_14624_amd import ops
    wl, base, kp, vp, bt = high_pool
    if workspace:
        assert ops.prefill_workspace_bytes(wl.batch, wl.total_q, wl.max_q_len, wl.max_kv_len,
                                           wl.num_q_heads, wl.num_kv_heads, wl.head_dim) > 0
    q = dev_bf16(wl.q)
    out = torch.full_like(q, float("nan"))
    ops.cs_prefill_paged_attn(q, kp, vp, bt, torch.from_numpy(wl.prefix_lens).cuda(),
                              torch.from_numpy(wl.cu_q_lens).cuda(), out,
                              max_q_len=wl.max_q_len, max_kv_len=wl.max_kv_len, scale=wl.scale,
                              workspace=workspace)
    torch.cuda.synchronize()
    ref = oracle.prefill_paged_attn(wl.q, wl.k_pool, wl.v_pool, wl.block_tables, wl.prefix_lens,
                                    wl.cu_q_lens, wl.num_q_heads, wl.num_kv_heads, wl.scale)
    mx, mean = compare_full(bits(out), ref)
    print(f"    prefill, workspace={workspace}: max_abs={mx:.3e} mean_abs={mean:.3e}", flush=True)
    assert mx <= MAX_ABS and mean <= MEAN_ABS


def test_decode_with_blocks_past_4gib(high_pool):
    from paper_2608_14624_amd import ops
    wl, base, kp, vp, bt = high_pool
    q, seq_lens = decode_view(wl)
    qd = dev_bf16(q)
    out = torch.empty_like(qd)
    ops.cs_paged_decode_attn(qd, kp, vp, bt, torch.from_numpy(seq_lens).cuda(), out,
                             max_seq_len=int(seq_lens.max()), scale=wl.scale)
    torch.cuda.synchronize()
    b = len(seq_lens)
    ref = oracle.prefill_paged_attn_rows(q, wl.k_pool, wl.v_pool, wl.block_tables,
                                         np.asarray(seq_lens, np.int32) - 1,
                                         np.arange(b + 1, dtype=np.int32), wl.num_q_heads,
                                         wl.num_kv_heads, wl.scale,
                                         [(r, h, 0) for r in range(b) for h in range(wl.num_q_heads)])
    got = oracle.bf16_bits_to_f64(bits(out)).reshape(b * wl.num_q_heads, -1)
    err = np.abs(got - ref)
    print(f"    decode: max_abs={err.max():.3e} mean_abs={err.mean():.3e}", flush=True)
    assert np.isfinite(got).all() and err.max() <= MAX_ABS and err.mean() <= MEAN_ABS


def test_copies_with_slots_past_4gib(high_pool):
    """Write-back into the last block of the pool, offload of high blocks to
    pinned host memory, and prefetch of them back into other high slots:
    every byte as the oracle's scatters and gathers place it."""
    from paper_2608_14624_amd import ops
    wl, base, kp, vp, bt = high_pool
    hkv, bs, d = wl.k_pool.shape[1:]
    rng = np.random.default_rng(5)
    # write-back: 20 tokens into distinct positions of the last 3 slots
    t = 20
    k_new = rng.integers(0, 1 << 16, (t, hkv, d), dtype=np.uint16) & 0x7F7F   # finite bf16
    v_new = rng.integers(0, 1 << 16, (t, hkv, d), dtype=np.uint16) & 0x7F7F
    local = rng.choice(3 * bs, t, replace=False) + (wl.num_blocks - 3) * bs
    slots = torch.from_numpy((local + base * bs).astype(np.int32)).cuda()
    ops.cs_kv_write(dev_bf16(k_new), dev_bf16(v_new), slots, kp, vp)
    # offload four high blocks, then prefetch them into four other high slots
    src = np.array([wl.num_blocks - 1, wl.num_blocks - 2, 5, 7], np.int32)
    dst = np.array([wl.num_blocks - 10, wl.num_blocks - 11, 30, 31], np.int32)
    host_k = torch.empty((4, hkv, bs, d), dtype=torch.bfloat16, pin_memory=True)
    host_v = torch.empty_like(host_k, pin_memory=True)
    ops.cs_kv_offload(torch.from_numpy(src + base).cuda(), kp, vp, host_k, host_v)
    torch.cuda.synchronize()
    ops.cs_kv_prefetch(host_k, host_v, torch.from_numpy(dst + base).cuda(), kp, vp)
    torch.cuda.synchronize()
    ek, ev = oracle.kv_write(k_new, v_new, local, wl.k_pool, wl.v_pool)
    hk, hv = oracle.kv_offload(src, ek, ev)
    assert np.array_equal(bits(host_k), hk) and np.array_equal(bits(host_v), hv)
    ek, ev = oracle.kv_prefetch(hk, hv, dst, ek, ev)
    assert np.array_equal(bits(kp[base:]), ek)
    assert np.array_equal(bits(vp[base:]), ev)
    # restore the workload's blocks for any later test of this module
    kp[base:] = dev_bf16(wl.k_pool)
    vp[base:] = dev_bf16(wl.v_pool)


@pytest.fixture(scope="module")
def long_context():
    wl = build_workload("ctx128k", 29, [131_072], [Invocation(0, 512)], num_q_heads=32,
                        num_kv_heads=8, head_dim=128, num_blocks=131_072 // 16 + 64)
    print(f"[case] 128k context: prefix {int(wl.prefix_lens[0])}, suffix {int(wl.q_lens[0])}",
          flush=True)
    return wl


@pytest.mark.parametrize("workspace", [None, "auto"])
def test_prefill_128k_context_sampled(long_context, workspace):
    from paper_2608_14624_amd import ops
    wl = long_context
    if workspace:
        assert ops.prefill_workspace_bytes(wl.batch, wl.total_q, wl.max_q_len, wl.max_kv_len,
                                           wl.num_q_heads, wl.num_kv_heads, wl.head_dim) > 0
    q = dev_bf16(wl.q)
    out = torch.full_like(q, float("nan"))
    ops.cs_prefill_paged_attn(q, dev_bf16(wl.k_pool), dev_bf16(wl.v_pool),
                              torch.from_numpy(wl.block_tables).cuda(),
                              torch.from_numpy(wl.prefix_lens).cuda(),
                              torch.from_numpy(wl.cu_q_lens).cuda(), out,
                              max_q_len=wl.max_q_len, max_kv_len=wl.max_kv_len, scale=wl.scale,
                              workspace=workspace)
    torch.cuda.synchronize()
    got = bits(out)
    assert np.isfinite(oracle.bf16_bits_to_f64(got)).all()
    samples = sample_rows(wl, 48, seed=3, edge_all_heads=True)
    mx, mean = compare_rows(wl, got, samples)
    print(f"    workspace={workspace}: {len(samples)} rows max_abs={mx:.3e} mean_abs={mean:.3e}",
          flush=True)
    assert mx <= MAX_ABS and mean <= MEAN_ABS


def test_decode_128k_context(long_context):
    from paper_2608_14624_amd import ops
    wl = long_context
    q, seq_lens = decode_view(wl)
    qd = dev_bf16(q)
    out = torch.empty_like(qd)
    ops.cs_paged_decode_attn(qd, dev_bf16(wl.k_pool), dev_bf16(wl.v_pool),
                             torch.from_numpy(wl.block_tables).cuda(),
                             torch.from_numpy(seq_lens).cuda(), out,
                             max_seq_len=int(seq_lens.max()), scale=wl.scale)
    torch.cuda.synchronize()
    ref = oracle.prefill_paged_attn_rows(q, wl.k_pool, wl.v_pool, wl.block_tables,
                                         np.asarray(seq_lens, np.int32) - 1,
                                         np.arange(2, dtype=np.int32), wl.num_q_heads,
                                         wl.num_kv_heads, wl.scale,
                                         [(0, h, 0) for h in range(wl.num_q_heads)])
    got = oracle.bf16_bits_to_f64(bits(out)).reshape(wl.num_q_heads, -1)
    err = np.abs(got - ref)
    print(f"    decode of {int(seq_lens[0])} keys: max_abs={err.max():.3e} mean_abs={err.mean():.3e}",
          flush=True)
    assert np.isfinite(got).all() and err.max() <= MAX_ABS and err.mean() <= MEAN_ABS
