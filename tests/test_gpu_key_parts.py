"""GPU parity of cs_prefill_paged_attn_ws: launches too small to fill the GPU
split every tile's keys into parts on separate work-groups and merge the
partial results (log-sum-exp weights) in a second kernel.

Head dims 64 and 128.  Each case is compared element by element with the float64 oracle (max-abs
<= 2e-2, mean-abs <= 2e-3) and with the plain cs_prefill_paged_attn on the
same inputs; the launches are checked to really take key parts.  Cases: the
one-GPU shard of the 70B-shape serving step (8 query / 1 KV head, through
the benchmark's pipeline), parts that hold no step of a short sequence,
rows whose keys in a later part are all masked, one-token suffixes, pool
slot 0 full of NaN and NaN / Inf past the sequences' ends.
"""

import numpy as np
import pytest

import oracle
from gpu_util import MAX_ABS, MEAN_ABS, compare_full, poison_slot_zero, poison_tails
from paper_2608_14624_amd.workload import Invocation, build_workload, make_config

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def oracle_full(wl):
    kp, vp = wl.k_pool, wl.v_pool
    if wl.prefetch_dst is not None:
        kp, vp = oracle.kv_prefetch(wl.host_k, wl.host_v, wl.prefetch_dst, kp, vp)
    return oracle.prefill_paged_attn(wl.q, kp, vp, wl.block_tables, wl.prefix_lens,
                                     wl.cu_q_lens, wl.num_q_heads, wl.num_kv_heads, wl.scale)


def parts_of(ops, wl, lo=0, hi=None):
    hi = wl.batch if hi is None else hi
    cu = wl.cu_q_lens.astype(np.int64)
    q_lens = np.diff(cu[lo:hi + 1])
    kv = q_lens + wl.prefix_lens[lo:hi]
    need = ops.prefill_workspace_bytes(hi - lo, int(cu[hi] - cu[lo]), int(q_lens.max()),
                                       int(kv.max()), wl.num_q_heads, wl.num_kv_heads, wl.head_dim)
    rows = int(cu[hi] - cu[lo]) * wl.num_q_heads * (wl.head_dim + 2) * 4
    return max(1, need // rows)


def check_parts(wl, min_parts=2):
    from paper_2608_14624_amd import ops, pipeline
    p = parts_of(ops, wl)
    print(f"[case] {wl.name}: B={wl.batch} total_q={wl.total_q} Hq={wl.num_q_heads} "
          f"Hkv={wl.num_kv_heads} key parts={p}", flush=True)
    assert p >= min_parts
    dw = pipeline.DeviceWorkload(wl, workspace="auto")
    dw.prefetch_all()
    dw.out.fill_(float("nan"))
    dw.attention()
    plain = torch.full_like(dw.out, float("nan"))
    dw_plain = pipeline.DeviceWorkload(wl)
    dw_plain.prefetch_all()
    dw_plain.attention(out=plain)
    torch.cuda.synchronize()
    mx, mean = compare_full(dw.out_bits(), oracle_full(wl))
    d = (dw.out.float() - plain.float()).abs()
    print(f"    vs oracle max_abs={mx:.3e} mean_abs={mean:.3e}; vs plain call "
          f"max={d.max().item():.3e}", flush=True)
    assert mx <= MAX_ABS and mean <= MEAN_ABS
    assert d.max().item() <= MAX_ABS
    return dw


CASES = {
    # name: (anchors, invocations, Hq, Hkv)
    "one_long_sequence": ([2000], [Invocation(0, 200)], 8, 2),
    # one long sequence sets four parts; the short ones' tiles have fewer
    # steps than parts, so some parts hold no step of theirs
    "parts_without_steps": ([3000, 5], [Invocation(0, 40), Invocation(1, 3), Invocation(1, 60)], 8, 2),
    # a miss: early rows see only the first keys, masked in every later part
    "miss_rows_masked_in_later_parts": ([0, 1100], [Invocation(0, 300), Invocation(1, 1)], 8, 8),
    "single_token_suffixes": ([1500, 33], [Invocation(0, 1), Invocation(1, 1), Invocation(0, 1)], 16, 2),
    "gqa8_one_kv_head": ([4096], [Invocation(0, 512)], 8, 1),
    # tiles of 1 to 51 steps (and empty ones): parts of very unequal length
    "unequal_tiles": ([3000, 50, 700], [Invocation(i % 3, n) for i, n in
                                        enumerate([1, 37, 120, 260, 5, 90])], 8, 4),
}


@pytest.mark.parametrize("head_dim", [64, 128])
@pytest.mark.parametrize("name", sorted(CASES))
def test_key_parts_match_oracle(name, head_dim):
    anchors, invs, hq, hkv = CASES[name]
    wl = build_workload(name, 71, anchors, invs, num_q_heads=hq, num_kv_heads=hkv, head_dim=head_dim,
                        num_blocks=1024)
    check_parts(wl)


@pytest.mark.parametrize("head_dim", [64, 128])
def test_key_parts_with_peaky_logits(head_dim):
    """Queries scaled up 8x (logits in the tens of log2 units): the parts'
    maxima differ widely, and the merge's log-sum-exp weights must still
    give the oracle's result."""
    wl = build_workload("kp_peaky", 73, [2000, 300], [Invocation(0, 120), Invocation(1, 60)],
                        num_q_heads=8, num_kv_heads=2, head_dim=head_dim, num_blocks=1024,
                        q_gain=8.0)
    check_parts(wl)


@pytest.mark.parametrize("head_dim", [64, 128])
@pytest.mark.parametrize("poison", ["slot_zero_nan", "nan_inf_tails"])
def test_key_parts_ignore_poisoned_positions(poison, head_dim):
    invs = [Invocation(0, 37), Invocation(1, 90), Invocation(0, 5)]
    wl = build_workload("kp_" + poison, 6, [1061, 200], invs, num_q_heads=32, num_kv_heads=8,
                        head_dim=head_dim, num_blocks=512)
    if poison == "slot_zero_nan":
        poison_slot_zero(wl)
    else:
        assert poison_tails(wl) > 0
    check_parts(wl)


@pytest.mark.parametrize("overlap", [False, True])
def test_tp8_shard_pipeline_full(overlap):
    """One GPU's shard of the 70B-shape serving step (8 query / 1 KV head):
    the per-agent launches of up to half a round of tiles take key parts (two
    or four here), with the next agent's prefetch beside them, as the
    benchmark runs them (and with consecutive launches on two streams, each
    with its own workspace)."""
    from paper_2608_14624_amd import ops, pipeline
    wl = make_config("llama70b_prefetch_tp8")
    dw = pipeline.DeviceWorkload(wl, workspace="auto")
    pipe = pipeline.AgentPipeline(dw, overlap=overlap)
    parts = [parts_of(ops, wl, b.lo, b.hi) for b in pipe.batches]
    print(f"[case] llama70b_prefetch_tp8 key parts per agent launch: {parts}", flush=True)
    assert max(parts) >= 2
    pipe.stage_first()
    dw.out.fill_(float("nan"))
    pipe.step()
    torch.cuda.synchronize()
    mx, mean = compare_full(dw.out_bits(), oracle_full(wl))
    print(f"[case] llama70b_prefetch_tp8 pipeline: max_abs={mx:.3e} mean_abs={mean:.3e}", flush=True)
    assert mx <= MAX_ABS and mean <= MEAN_ABS


def test_key_parts_are_deterministic_and_reuse_the_workspace():
    from paper_2608_14624_amd import ops, pipeline
    invs = [Invocation(0, 200), Invocation(0, 31)]
    wl = build_workload("kp_det", 9, [1800], invs, num_q_heads=8, num_kv_heads=2, head_dim=128,
                        num_blocks=512)
    dw = pipeline.DeviceWorkload(wl)
    ws = torch.full((parts_of(ops, wl) * wl.total_q * 8 * 130 * 4,), 0xFF, dtype=torch.uint8,
                    device="cuda")
    outs = []
    for _ in range(3):
        o = torch.full_like(dw.out, float("nan"))
        ops.cs_prefill_paged_attn(dw.q, dw.k_pool, dw.v_pool, dw.block_tables, dw.prefix_lens,
                                  dw.cu_q_lens, o, max_q_len=wl.max_q_len,
                                  max_kv_len=wl.max_kv_len, scale=wl.scale, workspace=ws)
        outs.append(o)
    torch.cuda.synchronize()
    for o in outs[1:]:
        assert torch.equal(o.view(torch.int16), outs[0].view(torch.int16))
    mx, mean = compare_full(outs[0].view(torch.int16).cpu().numpy().view(np.uint16), oracle_full(wl))
    assert mx <= MAX_ABS and mean <= MEAN_ABS


def test_workspace_too_small_is_rejected():
    from paper_2608_14624_amd import ops, pipeline
    wl = build_workload("kp_small_ws", 9, [1800], [Invocation(0, 64)], num_q_heads=8,
                        num_kv_heads=2, head_dim=128, num_blocks=512)
    dw = pipeline.DeviceWorkload(wl)
    need = ops.prefill_workspace_bytes(1, wl.total_q, wl.max_q_len, wl.max_kv_len, 8, 2, 128)
    assert need > 0
    ws = torch.empty(need - 16, dtype=torch.uint8, device="cuda")
    with pytest.raises(ops.CacheScoutError) as ei:
        ops.cs_prefill_paged_attn(dw.q, dw.k_pool, dw.v_pool, dw.block_tables, dw.prefix_lens,
                                  dw.cu_q_lens, dw.out, max_q_len=wl.max_q_len,
                                  max_kv_len=wl.max_kv_len, scale=wl.scale, workspace=ws)
    assert ei.value.status == ops.CS_ERR_INVALID_ARG
