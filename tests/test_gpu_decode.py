"""GPU parity of cs_paged_decode_attn: the one-token case of the prefix-reuse
attention, compared with the float64 oracle's last row of every sequence
(max-abs <= 2e-2, mean-abs <= 2e-3), and with the prefill kernel's last row."""

import numpy as np
import pytest

import oracle
from gpu_util import MAX_ABS, MEAN_ABS
from paper_2608_14624_amd.workload import Invocation, build_workload, decode_view, make_config

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def dev_bf16(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()


def run_decode(wl):
    from paper_2608_14624_amd import ops
    q, seq_lens = decode_view(wl)
    qd = dev_bf16(q)
    out = torch.empty_like(qd)
    ops.cs_paged_decode_attn(qd, dev_bf16(wl.k_pool), dev_bf16(wl.v_pool),
                             torch.from_numpy(wl.block_tables).cuda(),
                             torch.from_numpy(seq_lens).cuda(), out,
                             max_seq_len=int(seq_lens.max()), scale=wl.scale)
    torch.cuda.synchronize()
    return oracle.bf16_bits_to_f64(out.view(torch.int16).cpu().numpy().view(np.uint16))


def oracle_last_rows(wl):
    samples = [(r, h, int(wl.q_lens[r]) - 1) for r in range(wl.batch)
               for h in range(wl.num_q_heads)]
    ref = oracle.prefill_paged_attn_rows(wl.q, wl.k_pool, wl.v_pool, wl.block_tables,
                                         wl.prefix_lens, wl.cu_q_lens, wl.num_q_heads,
                                         wl.num_kv_heads, wl.scale, samples)
    return ref.reshape(wl.batch, wl.num_q_heads, -1)


CASES = {
    # name: (anchors, [(agent, suffix)], Hq, Hkv, D)
    "len1_and_block_edges": ([0, 15, 16, 31], [(0, 1), (1, 1), (2, 1), (3, 2), (2, 17)], 8, 2, 128),
    "mha_group1": ([100], [(0, 1), (0, 33)], 4, 4, 64),
    "group2_d64": ([47, 200], [(0, 9), (1, 64), (0, 1)], 8, 4, 64),
    "group4_long": ([1000, 2049], [(0, 100), (1, 3), (1, 250)], 32, 8, 128),
    "group8": ([513], [(0, 31), (0, 32), (0, 33)], 64, 8, 128),
    "group16": ([77], [(0, 5)], 32, 2, 128),
}


@pytest.mark.parametrize("name", sorted(CASES))
def test_decode_matches_oracle(name):
    anchors, spec, hq, hkv, d = CASES[name]
    invs = [Invocation(a, s) for a, s in spec]
    wl = build_workload(name, 31, anchors, invs, num_q_heads=hq, num_kv_heads=hkv, head_dim=d,
                        num_blocks=512)
    print(f"[case] decode {name}: B={wl.batch} kv_lens={wl.kv_lens.tolist()}", flush=True)
    got = run_decode(wl)
    ref = oracle_last_rows(wl)
    err = np.abs(got - ref)
    print(f"    max_abs={err.max():.3e} mean_abs={err.mean():.3e}", flush=True)
    assert np.isfinite(got).all() and err.max() <= MAX_ABS and err.mean() <= MEAN_ABS


def test_decode_matches_prefill_last_rows():
    from paper_2608_14624_amd import pipeline
    invs = [Invocation(0, 40), Invocation(1, 1), Invocation(0, 77)]
    wl = build_workload("dec_vs_prefill", 3, [300, 64], invs, num_q_heads=32, num_kv_heads=8,
                        head_dim=128, num_blocks=256)
    got = run_decode(wl)
    dw = pipeline.DeviceWorkload(wl)
    dw.attention()
    torch.cuda.synchronize()
    pre = oracle.bf16_bits_to_f64(dw.out_bits())[wl.cu_q_lens[1:] - 1]
    assert np.abs(got - pre).max() <= MAX_ABS


def test_decode_batch_config():
    wl = make_config("decode_batch")
    print(f"[case] decode_batch B={wl.batch} max_kv={wl.max_kv_len}", flush=True)
    got = run_decode(wl)
    ref = oracle_last_rows(wl)
    err = np.abs(got - ref)
    print(f"    max_abs={err.max():.3e} mean_abs={err.mean():.3e}", flush=True)
    assert np.isfinite(got).all() and err.max() <= MAX_ABS and err.mean() <= MEAN_ABS
