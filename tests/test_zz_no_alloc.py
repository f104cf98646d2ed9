"""cs_cascade_decode_attn_noalloc: the cascade decode with its partials in the
library's per-device scratch array instead of a caller workspace.

Two calls in a row through the C ABI, the second with a smaller batch, each
compared bit for bit with cs_cascade_decode_attn on the same inputs (the same
kernels in the same order, so the outputs must be identical; the float64
oracle bound holds for both).  The scratch array keeps the first call's
partials, so the second call also shows that nothing stale is read.
"""

import numpy as np
import pytest

import oracle
from gpu_util import MAX_ABS, MEAN_ABS
from paper_2608_14624_amd.workload import (Invocation, build_workload, cascade_view, decode_view,
                                           make_config)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def dev(a):
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(a).cuda()


def grouped(wl):
    cv = cascade_view(wl)
    q, seq_lens = decode_view(wl)
    o = cv["order"]
    return q[o], seq_lens[o], wl.block_tables[o], cv


def both_calls(ops, wl):
    q, seq_lens, bt, cv = grouped(wl)
    qd, kp, vp = dev(q), dev(wl.k_pool), dev(wl.v_pool)
    btd, sld = dev(bt), dev(seq_lens)
    cud, shd = dev(cv["cu_groups"]), dev(cv["shared_lens"])
    kw = dict(max_seq_len=int(seq_lens.max()), max_group_seqs=cv["max_group_seqs"],
              max_shared_len=cv["max_shared_len"], max_rest_len=cv["max_rest_len"],
              scale=wl.scale)
    need = ops.cs_cascade_decode_workspace_bytes(wl.batch, wl.num_q_heads, wl.head_dim,
                                                 cv["max_shared_len"], cv["max_rest_len"])
    print(f"[case] noalloc {wl.name}: B={wl.batch} partials {need} bytes "
          f"(scratch {ops.NOALLOC_SCRATCH_BYTES})", flush=True)
    assert 0 < need <= ops.NOALLOC_SCRATCH_BYTES
    ref = torch.full_like(qd, float("nan"))
    ops.cs_cascade_decode_attn(qd, kp, vp, btd, sld, cud, shd, ref, **kw)
    got = torch.full_like(qd, float("nan"))
    ops.cs_cascade_decode_attn_noalloc(qd, kp, vp, btd, sld, cud, shd, got, **kw)
    torch.cuda.synchronize()
    gb = got.view(torch.int16).cpu().numpy().view(np.uint16)
    rb = ref.view(torch.int16).cpu().numpy().view(np.uint16)
    return gb, rb, q, seq_lens, bt


def oracle_decode(wl, q, seq_lens, bt):
    b = len(seq_lens)
    samples = [(r, h, 0) for r in range(b) for h in range(wl.num_q_heads)]
    ref = oracle.prefill_paged_attn_rows(q, wl.k_pool, wl.v_pool, bt,
                                         np.asarray(seq_lens, np.int32) - 1,
                                         np.arange(b + 1, dtype=np.int32), wl.num_q_heads,
                                         wl.num_kv_heads, wl.scale, samples)
    return ref.reshape(b, wl.num_q_heads, -1)


def test_noalloc_matches_the_workspace_call_twice_in_a_row():
    from paper_2608_14624_amd import ops
    big = make_config("decode_batch")
    invs = [Invocation(0, 3), Invocation(1, 40), Invocation(0, 1), Invocation(1, 200),
            Invocation(2, 9, hit=False)]
    small = build_workload("noalloc_small", 45, [1100, 530, 64], invs, num_q_heads=32,
                           num_kv_heads=8, head_dim=128, num_blocks=1024)
    for wl in (big, small):
        got, ref, q, seq_lens, bt = both_calls(ops, wl)
        assert np.array_equal(got, ref), f"{wl.name}: differs from cs_cascade_decode_attn"
        err = np.abs(oracle.bf16_bits_to_f64(got) - oracle_decode(wl, q, seq_lens, bt))
        print(f"    bitwise equal; vs oracle max_abs={err.max():.3e} mean_abs={err.mean():.3e}",
              flush=True)
        assert err.max() <= MAX_ABS and err.mean() <= MEAN_ABS
