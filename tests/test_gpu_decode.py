"""GPU parity of cs_paged_decode_attn: the one-token case of the prefix-reuse
attention, compared with the float64 oracle's last row of every sequence
(max-abs <= 2e-2, mean-abs <= 2e-3), and with the prefill kernel's last row."""

import numpy as np
import pytest

import oracle
from gpu_util import MAX_ABS, MEAN_ABS, poison_tails
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


# ---------------------------------------------------------------- cascade decode

def oracle_decode(q, seq_lens, block_tables, wl):
    """The oracle for a decode batch: query r is position seq_lens[r] - 1 and
    sees keys 0 .. seq_lens[r] - 1 (a one-token suffix after a prefix of
    seq_lens[r] - 1 tokens)."""
    b = len(seq_lens)
    samples = [(r, h, 0) for r in range(b) for h in range(wl.num_q_heads)]
    ref = oracle.prefill_paged_attn_rows(q, wl.k_pool, wl.v_pool, block_tables,
                                         np.asarray(seq_lens, np.int32) - 1,
                                         np.arange(b + 1, dtype=np.int32), wl.num_q_heads,
                                         wl.num_kv_heads, wl.scale, samples)
    return ref.reshape(b, wl.num_q_heads, -1)


def grouped_batch(wl):
    from paper_2608_14624_amd.workload import cascade_view
    cv = cascade_view(wl)
    q, seq_lens = decode_view(wl)
    o = cv["order"]
    return (np.ascontiguousarray(q[o]), np.ascontiguousarray(seq_lens[o]),
            np.ascontiguousarray(wl.block_tables[o]), cv)


def rest_bound(seq_lens, cu, shared):
    return max(int(seq_lens[r]) - int(shared[g]) for g in range(len(shared))
               for r in range(cu[g], cu[g + 1]))


def run_cascade(wl, q, seq_lens, bt, cu, shared, max_group_seqs, max_shared_len, workspace=None,
                max_rest_len=None, max_seq_len=None):
    from paper_2608_14624_amd import ops
    qd = dev_bf16(q)
    out = torch.full_like(qd, float("nan"))
    ops.cs_cascade_decode_attn(qd, dev_bf16(wl.k_pool), dev_bf16(wl.v_pool),
                               torch.from_numpy(bt).cuda(), torch.from_numpy(seq_lens).cuda(),
                               torch.from_numpy(np.asarray(cu, np.int32)).cuda(),
                               torch.from_numpy(np.asarray(shared, np.int32)).cuda(), out,
                               max_seq_len=(int(seq_lens.max()) if max_seq_len is None
                                            else max_seq_len),
                               max_group_seqs=max_group_seqs,
                               max_shared_len=max_shared_len,
                               max_rest_len=(rest_bound(seq_lens, cu, shared)
                                             if max_rest_len is None else max_rest_len),
                               scale=wl.scale, workspace=workspace)
    torch.cuda.synchronize()
    return oracle.bf16_bits_to_f64(out.view(torch.int16).cpu().numpy().view(np.uint16))


def check(got, ref, what):
    err = np.abs(got - ref)
    print(f"    {what}: max_abs={err.max():.3e} mean_abs={err.mean():.3e}", flush=True)
    assert np.isfinite(got).all() and err.max() <= MAX_ABS and err.mean() <= MEAN_ABS


CASCADE_CASES = {
    # name: (anchors, [(agent, suffix, hit)], Hq, Hkv, D)
    # shared prefixes of 1 .. 3 chunks with ragged tails, a miss group, an
    # anchor shorter than one block (shares nothing)
    "mixed_g4": ([1100, 530, 8, 700], [(0, 3, True), (1, 40, True), (0, 1, True), (2, 5, True),
                                      (1, 200, True), (3, 17, False), (0, 64, True),
                                      (3, 9, True)], 32, 8, 128),
    "mha_d64": ([600], [(0, 1, True), (0, 30, True)], 4, 4, 64),
    "group16": ([520], [(0, 2, True), (0, 3, True)], 32, 2, 128),
    "group8_d64": ([1030, 96], [(1, 5, True), (0, 7, True), (1, 1, True), (0, 90, True)], 16, 2, 64),
}


@pytest.mark.parametrize("name", sorted(CASCADE_CASES))
def test_cascade_decode_matches_oracle(name):
    anchors, spec, hq, hkv, d = CASCADE_CASES[name]
    invs = [Invocation(a, s, h) for a, s, h in spec]
    wl = build_workload(name, 41, anchors, invs, num_q_heads=hq, num_kv_heads=hkv, head_dim=d,
                        num_blocks=1024)
    q, seq_lens, bt, cv = grouped_batch(wl)
    print(f"[case] cascade {name}: cu={cv['cu_groups'].tolist()} shared={cv['shared_lens'].tolist()}",
          flush=True)
    got = run_cascade(wl, q, seq_lens, bt, cv["cu_groups"], cv["shared_lens"],
                      cv["max_group_seqs"], cv["max_shared_len"])
    check(got, oracle_decode(q, seq_lens, bt, wl), "vs oracle")


def test_cascade_decode_with_loose_host_bounds():
    """max_group_seqs, max_shared_len, max_rest_len and max_seq_len only need
    to bound the batch: with each well above it the launches carry row
    tiles, shared-prefix chunks and own-key segments that hold nothing (they
    leave at once) and the workspace has more partial slots than any row
    uses.  The merge takes each row's own partial count, so the result is
    bitwise the one of the exact bounds, and matches the oracle."""
    # 12 sequences of 3 agents plus a miss; G = 16, so the loosest
    # max_group_seqs (the batch) gives a second, empty row tile
    invs = [Invocation(i % 3, 1 + (i * 53) % 400) for i in range(12)] + [Invocation(1, 30, False)]
    wl = build_workload("loose_cascade", 43, [1100, 530, 700], invs, num_q_heads=32,
                        num_kv_heads=2, head_dim=128, num_blocks=1024)
    q, seq_lens, bt, cv = grouped_batch(wl)
    cu, shared = cv["cu_groups"], cv["shared_lens"]
    exact = run_cascade(wl, q, seq_lens, bt, cu, shared, cv["max_group_seqs"], cv["max_shared_len"])
    max_seq = int(seq_lens.max()) + 4096
    wide = np.zeros((len(seq_lens), -(-max_seq // 16)), np.int32)
    wide[:, :bt.shape[1]] = bt
    bounds = dict(max_group_seqs=len(seq_lens),
                  max_shared_len=cv["max_shared_len"] + 2048,
                  max_rest_len=rest_bound(seq_lens, cu, shared) + 2500, max_seq_len=max_seq)
    print(f"[case] cascade with loose bounds {bounds} (exact: {cv['max_group_seqs']}, "
          f"{cv['max_shared_len']}, {rest_bound(seq_lens, cu, shared)}, {int(seq_lens.max())})",
          flush=True)
    loose = run_cascade(wl, q, seq_lens, wide, cu, shared, bounds["max_group_seqs"],
                        bounds["max_shared_len"], max_rest_len=bounds["max_rest_len"],
                        max_seq_len=bounds["max_seq_len"])
    assert np.array_equal(loose, exact)
    check(loose, oracle_decode(q, seq_lens, bt, wl), "loose bounds vs oracle")


def test_cascade_decode_two_row_tiles_and_empty_private_part():
    # 40 sequences of one agent at G = 4: 160 stacked rows, two row tiles; one
    # sequence ends exactly where the shared prefix ends (no keys of its own),
    # and an empty group sits between two others
    invs = [Invocation(0, 1 + (i * 37) % 300) for i in range(40)] + [Invocation(1, 4)]
    wl = build_workload("rows", 43, [777, 64], invs, num_q_heads=16, num_kv_heads=4,
                        head_dim=128, num_blocks=2048)
    q, seq_lens, bt, cv = grouped_batch(wl)
    seq_lens = seq_lens.copy()
    seq_lens[5] = 768                       # = the group's shared length
    cu = [0, 40, 40, 41]
    shared = [768, 0, 64]
    print(f"[case] cascade rows: cu={cu} shared={shared}", flush=True)
    got = run_cascade(wl, q, seq_lens, bt, cu, shared, 40, 768)
    check(got, oracle_decode(q, seq_lens, bt, wl), "vs oracle")


def test_cascade_decode_long_own_parts_span_several_segments():
    # own parts of 1023, 1024, 1025 and 3000 keys: one to three 1024-key
    # segments, ragged ends, next to a group that shares 2048 keys
    invs = [Invocation(0, s) for s in (1023, 1024, 1025, 3000)] + [Invocation(1, 7)]
    wl = build_workload("segs", 44, [2048, 96], invs, num_q_heads=16, num_kv_heads=4,
                        head_dim=128, num_blocks=2048)
    q, seq_lens, bt, cv = grouped_batch(wl)
    print(f"[case] cascade segments: rest={cv['max_rest_len']}", flush=True)
    got = run_cascade(wl, q, seq_lens, bt, cv["cu_groups"], cv["shared_lens"],
                      cv["max_group_seqs"], cv["max_shared_len"])
    check(got, oracle_decode(q, seq_lens, bt, wl), "vs oracle")


def test_cascade_decode_without_sharing_equals_paged_decode():
    anchors, spec, hq, hkv, d = CASCADE_CASES["mixed_g4"]
    invs = [Invocation(a, s, h) for a, s, h in spec]
    wl = build_workload("noshare", 41, anchors, invs, num_q_heads=hq, num_kv_heads=hkv,
                        head_dim=d, num_blocks=1024)
    q, seq_lens = decode_view(wl)
    got = run_cascade(wl, q, seq_lens, wl.block_tables, [0, wl.batch], [0], 1, 0)
    ref = run_decode(wl)
    # one group sharing nothing: the same result up to rounding (the paged
    # decode kernel splits a sequence over 12 waves, a cascade segment over
    # 4, so the partial softmaxes are summed in another order): a few bf16
    # ulps apart, and both within the oracle bounds
    single = seq_lens <= 1024
    assert single.any() and (~single).any()
    diff = np.abs(got.astype(np.float64) - ref.astype(np.float64)).max()
    assert diff <= 8e-3, diff
    check(got, oracle_decode(q, seq_lens, wl.block_tables, wl), "vs oracle")
    check(ref, oracle_decode(q, seq_lens, wl.block_tables, wl), "paged decode vs oracle")


@pytest.mark.parametrize("d", [64, 128])
def test_decode_and_cascade_with_peaky_logits(d):
    """Queries scaled up 8x (logits in the tens of log2 units): the decode
    kernel's per-chunk max and rescale, and the cascade's partials merged
    with widely different maxima, stay within the bounds."""
    invs = [Invocation(0, 5), Invocation(0, 900), Invocation(1, 40), Invocation(1, 1)]
    wl = build_workload("peaky_dec", 47, [1500, 200], invs, num_q_heads=16, num_kv_heads=4,
                        head_dim=d, num_blocks=1024, q_gain=8.0)
    print(f"[case] peaky decode / cascade d={d} kv_lens={wl.kv_lens.tolist()}", flush=True)
    q, seq_lens = decode_view(wl)
    check(run_decode(wl), oracle_decode(q, seq_lens, wl.block_tables, wl), "decode vs oracle")
    q, seq_lens, bt, cv = grouped_batch(wl)
    got = run_cascade(wl, q, seq_lens, bt, cv["cu_groups"], cv["shared_lens"],
                      cv["max_group_seqs"], cv["max_shared_len"])
    check(got, oracle_decode(q, seq_lens, bt, wl), "cascade vs oracle")


def test_cascade_decode_batch_config():
    wl = make_config("decode_batch")
    q, seq_lens, bt, cv = grouped_batch(wl)
    print(f"[case] cascade decode_batch groups={len(cv['shared_lens'])}", flush=True)
    got = run_cascade(wl, q, seq_lens, bt, cv["cu_groups"], cv["shared_lens"],
                      cv["max_group_seqs"], cv["max_shared_len"])
    check(got, oracle_decode(q, seq_lens, bt, wl), "vs oracle")


def test_cascade_workspace_reuse_and_debug_checks(monkeypatch):
    from paper_2608_14624_amd import ops
    anchors, spec, hq, hkv, d = CASCADE_CASES["mixed_g4"]
    invs = [Invocation(a, s, h) for a, s, h in spec]
    wl = build_workload("dbg", 41, anchors, invs, num_q_heads=hq, num_kv_heads=hkv, head_dim=d,
                        num_blocks=1024)
    q, seq_lens, bt, cv = grouped_batch(wl)
    need = ops.cs_cascade_decode_workspace_bytes(wl.batch, hq, d, cv["max_shared_len"],
                                                 cv["max_rest_len"])
    ws = torch.full((need,), 0xFF, dtype=torch.uint8, device="cuda")   # NaN-filled scratch
    args = (wl, q, seq_lens, bt, cv["cu_groups"], cv["shared_lens"], cv["max_group_seqs"],
            cv["max_shared_len"])
    first = run_cascade(*args, workspace=ws)
    second = run_cascade(*args, workspace=ws)
    assert np.array_equal(first, second)
    monkeypatch.setenv("CS_DEBUG_CHECK", "1")
    assert np.array_equal(run_cascade(*args, workspace=ws), first)
    bad = bt.copy()
    g1 = int(cv["cu_groups"][0])
    bad[g1 + 1, 0] = (bad[g1, 0] + 1) % wl.num_blocks     # breaks the sharing of block 0
    with pytest.raises(ops.CacheScoutError, match="does not share"):
        run_cascade(wl, q, seq_lens, bad, cv["cu_groups"], cv["shared_lens"],
                    cv["max_group_seqs"], cv["max_shared_len"], workspace=ws)
    with pytest.raises(ops.CacheScoutError, match="max_group_seqs"):
        run_cascade(wl, q, seq_lens, bt, cv["cu_groups"], cv["shared_lens"], 1,
                    cv["max_shared_len"], workspace=ws)
    with pytest.raises(ops.CacheScoutError, match="max_rest_len"):
        run_cascade(wl, q, seq_lens, bt, cv["cu_groups"], cv["shared_lens"], cv["max_group_seqs"],
                    cv["max_shared_len"], workspace=ws, max_rest_len=cv["max_rest_len"] - 1)


def test_decode_and_cascade_ignore_nan_and_inf_past_the_end():
    """NaN and Inf in the pool positions past each sequence's end (inside its
    last block) must not reach the decode or cascade output."""
    invs = [Invocation(0, 3, True), Invocation(1, 40, True), Invocation(0, 17, True),
            Invocation(1, 1, True), Invocation(2, 9, False)]
    wl = build_workload("nan_tail_dec", 43, [700, 530, 90], invs, num_q_heads=32, num_kv_heads=8,
                        head_dim=128, num_blocks=1024)
    n = poison_tails(wl)
    print(f"[case] decode/cascade nan tails: {n} poisoned positions", flush=True)
    assert n > 0
    check(run_decode(wl), oracle_last_rows(wl), "decode vs oracle")
    q, seq_lens, bt, cv = grouped_batch(wl)
    got = run_cascade(wl, q, seq_lens, bt, cv["cu_groups"], cv["shared_lens"],
                      cv["max_group_seqs"], cv["max_shared_len"])
    check(got, oracle_decode(q, seq_lens, bt, wl), "cascade vs oracle")


def test_decode_private_recipe_scaled_down():
    """The decode_private recipe (every sequence its own anchor, nothing
    shared) at 12 sequences: per-sequence decode against the oracle."""
    rng = np.random.default_rng([6, 1])
    anchors = [int(x) for x in rng.integers(4096, 8192, size=12, endpoint=True)]
    hist = np.clip(np.rint(rng.lognormal(np.log(512.0), 1.0, size=12)), 128, 4096)
    invs = [Invocation(a, int(s)) for a, s in enumerate(hist)]
    wl = build_workload("decode_private_small", 6, anchors, invs, num_q_heads=32, num_kv_heads=8,
                        head_dim=128, occupancy=0.9)
    print(f"[case] decode_private scaled down: kv_lens={wl.kv_lens.tolist()}", flush=True)
    check(run_decode(wl), oracle_last_rows(wl), "decode vs oracle")


def decode_bits(q, k_pool, v_pool, bt, seq_lens, scale):
    from paper_2608_14624_amd import ops
    qd = dev_bf16(q)
    out = torch.empty_like(qd)
    ops.cs_paged_decode_attn(qd, k_pool, v_pool, torch.from_numpy(np.ascontiguousarray(bt)).cuda(),
                             torch.from_numpy(np.ascontiguousarray(seq_lens)).cuda(), out,
                             max_seq_len=int(seq_lens.max()), scale=scale)
    torch.cuda.synchronize()
    return out.view(torch.int16).cpu().numpy()


def test_decode_is_independent_of_batch_order():
    """The kernel runs the sequences longest first (every work-group ranks
    the lengths itself, ties by index): reordering the batch, with many
    equal lengths, permutes the output rows and changes no bit of them."""
    invs = [Invocation(i % 5, 1 + (i % 4) * 17) for i in range(40)]   # ten of each length class
    wl = build_workload("order", 3, [30, 61, 16, 100, 5], invs, num_q_heads=8, num_kv_heads=2,
                        head_dim=128, num_blocks=1024)
    q, seq_lens = decode_view(wl)
    assert len(np.unique(seq_lens)) < len(seq_lens)
    kp, vp = dev_bf16(wl.k_pool), dev_bf16(wl.v_pool)
    base = decode_bits(q, kp, vp, wl.block_tables, seq_lens, wl.scale)
    for seed in (1, 2):
        perm = np.random.default_rng(seed).permutation(wl.batch)
        got = decode_bits(q[perm], kp, vp, wl.block_tables[perm], seq_lens[perm], wl.scale)
        assert np.array_equal(got, base[perm])
    ref = oracle_last_rows(wl)
    out = oracle.bf16_bits_to_f64(base.view(np.uint16))
    err = np.abs(out - ref)
    assert err.max() <= MAX_ABS and err.mean() <= MEAN_ABS


def test_decode_batch_past_the_ranking_limit():
    """Batches above 1024 sequences run in dispatch order: 1100 sequences
    give bit for bit what their two halves give (each ranked)."""
    invs = [Invocation(i % 3, 1 + (7 * i) % 40) for i in range(1100)]
    wl = build_workload("big_batch", 4, [20, 33, 70], invs, num_q_heads=4, num_kv_heads=4,
                        head_dim=64, num_blocks=8192)
    q, seq_lens = decode_view(wl)
    kp, vp = dev_bf16(wl.k_pool), dev_bf16(wl.v_pool)
    whole = decode_bits(q, kp, vp, wl.block_tables, seq_lens, wl.scale)
    a = decode_bits(q[:600], kp, vp, wl.block_tables[:600], seq_lens[:600], wl.scale)
    b = decode_bits(q[600:], kp, vp, wl.block_tables[600:], seq_lens[600:], wl.scale)
    assert np.array_equal(whole, np.concatenate([a, b]))
