"""GPU parity of cs_prefill_paged_attn against the float64 oracle.

Tolerance (bf16 output vs unrounded float64 oracle): max-abs <= 2e-2 and
mean-abs <= 2e-3 over the compared elements.  Small and edge-case workloads,
the Llama-3-8B shape, the agent batch and the 70B-shape serving step (in the
launch configuration the benchmark times) are compared element by element on
their whole output; the long mixed load, whose misses make the full oracle
too slow, on sampled rows: random rows plus, for every invocation and every
query head, its first and last rows and the rows at block and tile
boundaries.
"""

import os

import numpy as np
import pytest

import oracle
from gpu_util import MAX_ABS, MEAN_ABS, compare_full, compare_rows, poison_slot_zero, poison_tails, sample_rows
from paper_2608_14624_amd.workload import Invocation, build_workload, make_config

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def P():
    from paper_2608_14624_amd import ops, pipeline
    return ops, pipeline


def run_full(P, wl):
    _, pipeline = P
    dw = pipeline.DeviceWorkload(wl)
    dw.prefetch_all()
    dw.attention()
    torch.cuda.synchronize()
    return dw


def oracle_full(wl):
    kp, vp = wl.k_pool, wl.v_pool
    if wl.prefetch_dst is not None:
        kp, vp = oracle.kv_prefetch(wl.host_k, wl.host_v, wl.prefetch_dst, kp, vp)
    return oracle.prefill_paged_attn(wl.q, kp, vp, wl.block_tables, wl.prefix_lens,
                                     wl.cu_q_lens, wl.num_q_heads, wl.num_kv_heads, wl.scale)


def check_full(P, wl):
    print(f"[case] {wl.name}: B={wl.batch} total_q={wl.total_q} Hq={wl.num_q_heads} "
          f"Hkv={wl.num_kv_heads} D={wl.head_dim}", flush=True)
    dw = run_full(P, wl)
    mx, mean = compare_full(dw.out_bits(), oracle_full(wl))
    print(f"    max_abs={mx:.3e} mean_abs={mean:.3e}", flush=True)
    assert mx <= MAX_ABS and mean <= MEAN_ABS
    return dw


def test_tiny_full(P):
    check_full(P, make_config("tiny"))


def test_llama8b_full(P):
    check_full(P, make_config("llama8b"))


EDGE = {
    # name: (anchor_lens, invocations, Hq, Hkv, D, extra)
    "single_token_suffix": ([100], [Invocation(0, 1)], 8, 2, 128, {}),
    "prefix_not_block_multiple": ([37, 5], [Invocation(0, 50), Invocation(1, 17)], 8, 2, 128, {}),
    "miss_and_hit_mix": ([70], [Invocation(0, 40), Invocation(0, 33, hit=False), Invocation(0, 1)], 8, 8, 64, {}),
    "empty_suffix_in_batch": ([48, 20], [Invocation(0, 0), Invocation(1, 70), Invocation(0, 0), Invocation(1, 3)], 4, 1, 128, {}),
    "group1_mha": ([64], [Invocation(0, 129)], 4, 4, 64, {}),
    "group2": ([33], [Invocation(0, 97)], 4, 2, 128, {}),
    "group8": ([200], [Invocation(0, 65), Invocation(0, 31)], 16, 2, 128, {}),
    "group3": ([17], [Invocation(0, 45)], 6, 2, 64, {}),
    # groups of 5, 6, 16 and 32 query heads per KV head: one, two and four
    # heads per tile (five and six split over several head tiles)
    "group5": ([23], [Invocation(0, 33)], 5, 1, 128, {}),
    "group6": ([40], [Invocation(0, 77), Invocation(0, 2)], 12, 2, 128, {}),
    "group16_mqa_d64": ([100], [Invocation(0, 50), Invocation(0, 9)], 16, 1, 64, {}),
    "group32_mqa": ([300], [Invocation(0, 40)], 32, 1, 128, {}),
    "zero_prefix_hit": ([0], [Invocation(0, 77)], 8, 2, 128, {}),
    "peaky_logits": ([90], [Invocation(0, 70)], 8, 2, 128, {"q_gain": 8.0}),
    "long_ragged_tile": ([1000], [Invocation(0, 257), Invocation(0, 129)], 32, 8, 128, {}),
    # small launches split each tile's key steps over two wave groups: one
    # step (the first group has none), rows whose keys in the second group's
    # half are all masked, and a long prefix under a short suffix
    "split_one_key": ([0], [Invocation(0, 1)], 8, 2, 128, {}),
    "split_masked_second_half": ([0], [Invocation(0, 65), Invocation(0, 130)], 8, 2, 128, {}),
    "split_long_prefix_short_suffix": ([1000], [Invocation(0, 3)], 8, 1, 64, {}),
}


@pytest.mark.parametrize("name", sorted(EDGE))
def test_edge_cases_full(P, name):
    anchors, invs, hq, hkv, d, extra = EDGE[name]
    wl = build_workload(name, 1234, anchors, invs, num_q_heads=hq, num_kv_heads=hkv,
                        head_dim=d, num_blocks=256, **extra)
    check_full(P, wl)


TAIL = {
    # ping-pong launches whose last round is at most half full: that round's
    # tiles run as split 128-row halves in the same launch
    "tail_g4": ([300, 40], [Invocation(0, 500), Invocation(1, 130), Invocation(0, 449),
                            Invocation(1, 64), Invocation(0, 1)], 32, 8, 128),
    "tail_g2_d64": ([90, 17], [Invocation(i % 2, n) for i, n in
                               enumerate([640, 600, 1, 129, 300, 0, 77])], 16, 8, 64),
    "tail_g1": ([200], [Invocation(0, 512 - 29 * i) for i in range(17)], 8, 8, 128),
    "tail_g2_d128": ([90, 17], [Invocation(i % 2, n) for i, n in
                                enumerate([640, 600, 1, 129, 300, 0, 77])], 16, 8, 128),
    # every tile needs one 64-key step: the first key half of a tail tile
    # has no step at all and the second holds every key
    "tail_one_step": ([16, 5], [Invocation(i % 2, 1 + (7 * i) % 48) for i in range(40)], 32, 8, 128),
}


@pytest.mark.parametrize("name", sorted(TAIL))
def test_ping_pong_launch_with_split_tail(P, name):
    ops, _ = P
    anchors, invs, hq, hkv, d = TAIL[name]
    wl = build_workload(name, 99, anchors, invs, num_q_heads=hq, num_kv_heads=hkv,
                        head_dim=d, num_blocks=512)
    kernel, grid, tail = ops.prefill_launch_shape(wl.batch, wl.max_q_len, hq, hkv)
    print(f"[case] {name}: grid={grid} tail work-groups={tail}", flush=True)
    assert kernel == ops.ATTN_PING_PONG and tail > 0
    check_full(P, wl)


PP_INVS = {"split": [Invocation(0, 37), Invocation(1, 90), Invocation(0, 5)],
           "ping_pong": [Invocation(i % 2, 1000 + 13 * i) for i in range(2)],
           "ping_pong_d64": [Invocation(i % 2, 1000 + 13 * i) for i in range(2)],
           "ping_pong_tail": [Invocation(i % 2, 450 + 7 * i) for i in range(5)]}


def pp_head_dim(shape):
    return 64 if shape.endswith("_d64") else 128


@pytest.mark.parametrize("shape", ["split", "ping_pong", "ping_pong_d64", "ping_pong_tail"])
def test_slot_zero_full_of_nan(P, shape):
    """Blocks past a sequence's end are loaded from pool slot 0 and then
    masked (K) or zeroed (V): with slot 0 all NaN the output stays exact."""
    ops, _ = P
    wl = build_workload("nan_slot0", 6, [61, 200], PP_INVS[shape], num_q_heads=32, num_kv_heads=8,
                        head_dim=pp_head_dim(shape), num_blocks=512)
    u = poison_slot_zero(wl)
    print(f"[case] slot 0 all NaN, {shape}: its blocks moved to slot {u}", flush=True)
    check_full(P, wl)


@pytest.mark.parametrize("shape", ["ping_pong", "ping_pong_d64", "ping_pong_tail"])
def test_peaky_logits_on_the_ping_pong_paths(P, shape):
    """Queries scaled up 8x (logits in the tens of log2 units): the large
    launches' kernels keep the scale in fp32 and stay within tolerance too."""
    ops, _ = P
    wl = build_workload("peaky_pp", 8, [61, 200], PP_INVS[shape], num_q_heads=32, num_kv_heads=8,
                        head_dim=pp_head_dim(shape), num_blocks=512, q_gain=8.0)
    kernel, grid, tail = ops.prefill_launch_shape(wl.batch, wl.max_q_len, 32, 8)
    assert kernel == ops.ATTN_PING_PONG and (tail > 0) == (shape == "ping_pong_tail")
    print(f"[case] peaky logits, {shape}: grid={grid} tail={tail}", flush=True)
    check_full(P, wl)


@pytest.mark.parametrize("shape", ["split", "ping_pong", "ping_pong_d64", "ping_pong_tail"])
def test_nan_and_inf_past_the_end_do_not_leak(P, shape):
    """Pool positions past a sequence's end inside its last block may hold
    anything (a recycled slot): NaN and Inf there must not reach the output,
    on every kernel path."""
    ops, _ = P
    wl = build_workload("nan_tail", 5, [61, 200], PP_INVS[shape], num_q_heads=32, num_kv_heads=8,
                        head_dim=pp_head_dim(shape), num_blocks=512)
    kernel, grid, tail = ops.prefill_launch_shape(wl.batch, wl.max_q_len, 32, 8)
    assert (kernel, tail > 0) == {"split": (ops.ATTN_SPLIT, False),
                                  "ping_pong": (ops.ATTN_PING_PONG, False),
                                  "ping_pong_d64": (ops.ATTN_PING_PONG, False),
                                  "ping_pong_tail": (ops.ATTN_PING_PONG, True)}[shape]
    n = poison_tails(wl)
    print(f"[case] nan tails, {shape}: {n} poisoned positions, grid={grid}", flush=True)
    assert n > 0
    check_full(P, wl)


@pytest.mark.parametrize("prefix,suffix,n_inv", [(2048, 512, 16), (0, 512, 16), (37, 300, 32)])
def test_head_dim_64_ping_pong_full(P, prefix, suffix, n_inv):
    """head_dim 64 launches of whole rounds (the direct-to-LDS ping-pong kernel
    with its eight-row LDS groups), every output element against the oracle:
    prefix hits, misses with the causal triangle only, and a prefix that is
    not a multiple of the block size with a ragged last token tile."""
    ops, _ = P
    invs = [Invocation(0, suffix - (i % 3)) for i in range(n_inv)]
    wl = build_workload("pp_d64", 17, [prefix], invs, num_q_heads=32, num_kv_heads=8,
                        head_dim=64, num_blocks=prefix // 16 + n_inv * (suffix // 16 + 2) + 64)
    kernel, grid, tail = ops.prefill_launch_shape(wl.batch, wl.max_q_len, 32, 8)
    print(f"[case] head_dim 64 ping-pong P={prefix} S={suffix} x{n_inv}: grid={grid} tail={tail}",
          flush=True)
    assert kernel == ops.ATTN_PING_PONG and tail == 0
    check_full(P, wl)


def test_agent_batch_full(P):
    _, pipeline = P
    wl = make_config("agent_batch")
    print(f"[case] agent_batch total_q={wl.total_q}", flush=True)
    dw = pipeline.DeviceWorkload(wl)
    dw.attention()
    torch.cuda.synchronize()
    mx, mean = compare_full(dw.out_bits(), oracle_full(wl))
    print(f"    all {wl.total_q * wl.num_q_heads} rows: max_abs={mx:.3e} mean_abs={mean:.3e}",
          flush=True)
    assert mx <= MAX_ABS and mean <= MEAN_ABS


def test_agent_batch_tp8_shard_full(P):
    """One GPU's shard of agent_batch under an 8-way KV-head split (4 query
    heads / 1 KV head): one launch of 1024 ping-pong tiles, all of them on
    the one KV head, called with a workspace as the benchmark calls it (a
    launch this large takes no key parts); every output element."""
    _, pipeline = P
    wl = make_config("agent_batch_tp8")
    print(f"[case] agent_batch_tp8 total_q={wl.total_q} Hq={wl.num_q_heads} Hkv={wl.num_kv_heads}",
          flush=True)
    dw = pipeline.DeviceWorkload(wl, workspace="auto")
    dw.attention()
    torch.cuda.synchronize()
    mx, mean = compare_full(dw.out_bits(), oracle_full(wl))
    print(f"    all {wl.total_q * wl.num_q_heads} rows: max_abs={mx:.3e} mean_abs={mean:.3e}",
          flush=True)
    assert mx <= MAX_ABS and mean <= MEAN_ABS


@pytest.mark.parametrize("overlap", [False, True])
def test_llama70b_prefetch_pipeline_full(P, overlap):
    """The benchmark's launch configuration: per-agent attention with the next
    agent's CPU-tier blocks prefetched on a side stream (and with consecutive
    agents' launches on two streams); every output element against the
    oracle.  The prefetched slots start as NaN, so an attention launch that
    ran before its agent's prefetch had landed would show."""
    _, pipeline = P
    wl = make_config("llama70b_prefetch")
    print(f"[case] llama70b_prefetch pipeline total_q={wl.total_q} overlap={overlap}", flush=True)
    dw = pipeline.DeviceWorkload(wl)
    pipe = pipeline.AgentPipeline(dw, overlap=overlap)
    pipe.stage_first()
    dw.out.fill_(float("nan"))
    pipe.step()
    torch.cuda.synchronize()
    kp, vp = oracle.kv_prefetch(wl.host_k, wl.host_v, wl.prefetch_dst, wl.k_pool, wl.v_pool)
    mx, mean = compare_full(dw.out_bits(), oracle_full(wl))
    print(f"    all {wl.total_q * wl.num_q_heads} rows: max_abs={mx:.3e} mean_abs={mean:.3e}",
          flush=True)
    assert mx <= MAX_ABS and mean <= MEAN_ABS
    # the pools on the device now equal the oracle's post-prefetch pools
    assert np.array_equal(dw.k_pool.view(torch.int16).cpu().numpy().view(np.uint16), kp)
    assert np.array_equal(dw.v_pool.view(torch.int16).cpu().numpy().view(np.uint16), vp)
    # every output row was written
    assert torch.isfinite(dw.out.float()).all().item()


def test_llama70b_prefetch_pipeline_driven_by_the_control_plane(P):
    """The same workload with the prefetch target chosen by the control plane
    (cs_scout_*): three passes, misses only while it learns the cycle, and
    the same outputs and pools as the oracle."""
    _, pipeline = P
    wl = make_config("llama70b_prefetch")
    print(f"[case] llama70b_prefetch scout-driven pipeline total_q={wl.total_q}", flush=True)
    dw = pipeline.DeviceWorkload(wl)
    agents = sorted({inv.agent for inv in wl.invocations})
    policy = pipeline.ScoutPolicy(wl, agents)
    # record every turn's decision of the C++ control plane
    decisions = []
    on_turn = policy.on_turn

    def recording_on_turn(a):
        t = on_turn(a)
        decisions.append((a, t))
        return t
    policy.on_turn = recording_on_turn
    pipe = pipeline.AgentPipeline(dw, policy=policy)
    pipe.stage_first()
    for p in range(3):
        dw.out.fill_(float("nan"))
        pipe.step()
        torch.cuda.synchronize()
        print(f"    pass {p}: hits={pipe.hits} misses={pipe.misses}", flush=True)
    n = len(pipe.agents)
    assert pipe.misses == n - 1 and pipe.hits == 2 * n + 1
    # the same turns replayed through the oracle control plane (Eq. (3)-(11),
    # the runtime procedure) give the same prefetch target at every turn
    import oracle.control_plane as ocp
    ref = ocp.ControlPlane(len(agents), wl.num_blocks)
    for now, (a, t) in enumerate(decisions):
        blocks, tokens = policy.touches[a]
        for b, tk in zip(blocks.tolist(), tokens.tolist()):
            ref.observe_touch(b, policy.ids[a], tk, now)
        want = ref.between_step()
        assert (None if want is None else policy.by_id.get(want)) == t, (now, a, t, want)
    print(f"    {len(decisions)} decisions equal to the oracle control plane's", flush=True)
    kp, vp = oracle.kv_prefetch(wl.host_k, wl.host_v, wl.prefetch_dst, wl.k_pool, wl.v_pool)
    samples = sample_rows(wl, 300, seed=4)
    mx, mean = compare_rows(wl, dw.out_bits(), samples, kp, vp)
    print(f"    {len(samples)} rows: max_abs={mx:.3e} mean_abs={mean:.3e}", flush=True)
    assert mx <= MAX_ABS and mean <= MEAN_ABS
    assert np.array_equal(dw.k_pool.view(torch.int16).cpu().numpy().view(np.uint16), kp)
    assert np.array_equal(dw.v_pool.view(torch.int16).cpu().numpy().view(np.uint16), vp)
    assert torch.isfinite(dw.out.float()).all().item()


@pytest.mark.slow
def test_long_mixed_sampled(P):
    _, pipeline = P
    wl = make_config("long_mixed")
    print(f"[case] long_mixed total_q={wl.total_q}", flush=True)
    dw = pipeline.DeviceWorkload(wl)
    dw.attention()
    torch.cuda.synchronize()
    samples = sample_rows(wl, 300, seed=4, edge_all_heads=True)
    mx, mean = compare_rows(wl, dw.out_bits(), samples)
    print(f"    {len(samples)} rows: max_abs={mx:.3e} mean_abs={mean:.3e}", flush=True)
    assert mx <= MAX_ABS and mean <= MEAN_ABS


def test_loaded_library_is_built_from_these_sources(P):
    """The library the GPU tests run is the build of the sources in this tree."""
    ops, _ = P
    from paper_2608_14624_amd import build
    print(f"[case] library digest {ops.source_digest()}, sources {build.source_digest()}",
          flush=True)
    assert ops.source_digest() == build.source_digest()


def small_batch():
    invs = [Invocation(0, 40), Invocation(1, 90), Invocation(0, 7), Invocation(2, 33, hit=False)]
    return build_workload("inv", 77, [61, 128, 30], invs, num_q_heads=8, num_kv_heads=2,
                          head_dim=128, num_blocks=128)


def test_block_permutation_is_bitwise_invariant(P):
    wl = small_batch()
    base = run_full(P, wl).out_bits()
    perm = np.random.default_rng(5).permutation(wl.num_blocks)
    k2 = np.empty_like(wl.k_pool)
    v2 = np.empty_like(wl.v_pool)
    k2[perm] = wl.k_pool
    v2[perm] = wl.v_pool
    wl.k_pool, wl.v_pool = k2, v2
    wl.block_tables = perm[wl.block_tables].astype(np.int32)
    moved = run_full(P, wl).out_bits()
    assert np.array_equal(base, moved)


def test_run_to_run_determinism(P):
    _, pipeline = P
    wl = make_config("llama8b")
    dw = pipeline.DeviceWorkload(wl)
    dw.attention()
    a = dw.out.clone()
    for _ in range(3):
        dw.out.zero_()
        dw.attention()
        torch.cuda.synchronize()
        assert torch.equal(a.view(torch.int16), dw.out.view(torch.int16))


@pytest.mark.parametrize("hq,hkv,d", [(32, 8, 128), (16, 8, 64), (12, 4, 128), (8, 8, 128),
                                     (24, 4, 128), (32, 2, 64)])
def test_wide_and_small_launches_agree(P, hq, hkv, d):
    """A batch large enough for the 8-wave ping-pong kernel, and its first
    invocation alone (a launch below one work-group per CU, whose tiles run
    with their key steps split over two wave groups), agree to the parity
    tolerance, and the batch matches the oracle."""
    _, pipeline = P
    invs = [Invocation(i % 3, 300 + 37 * i) for i in range(16)]
    wl = build_workload("wide", 12, [520, 77, 1200], invs, num_q_heads=hq, num_kv_heads=hkv,
                        head_dim=d, num_blocks=4096)
    print(f"[case] wide vs split launch hq={hq} hkv={hkv} d={d} total_q={wl.total_q}", flush=True)
    dw = pipeline.DeviceWorkload(wl)
    dw.attention()
    first = pipeline.SubBatch(dw, 0, 1)
    alone = torch.full_like(first.out, float("nan"))
    from paper_2608_14624_amd import ops
    ops.cs_prefill_paged_attn(first.q, dw.k_pool, dw.v_pool, first.block_tables,
                              first.prefix_lens, first.cu_q_lens, alone,
                              max_q_len=first.max_q_len, max_kv_len=first.max_kv_len,
                              scale=wl.scale)
    torch.cuda.synchronize()
    diff = (alone.float() - first.out.float()).abs()
    print(f"    alone vs batch: max_abs={diff.max().item():.3e} mean_abs={diff.mean().item():.3e}",
          flush=True)
    assert diff.max().item() <= MAX_ABS and diff.mean().item() <= MEAN_ABS
    samples = sample_rows(wl, 200, seed=5)
    mx, mean = compare_rows(wl, dw.out_bits(), samples)
    print(f"    {len(samples)} rows: max_abs={mx:.3e} mean_abs={mean:.3e}", flush=True)
    assert mx <= MAX_ABS and mean <= MEAN_ABS


LOOSE = {
    # name: (extra max_q_len, extra max_kv_len, workspace, expected kernel,
    #        key parts expected): with exact bounds this batch is a split
    #        launch of 112 tiles without parts
    "split_with_key_parts": (56, 3000, "auto", 0, True),
    "ping_pong_mostly_empty": (800, 3000, None, 1, False),
}


@pytest.mark.parametrize("name", sorted(LOOSE))
def test_loose_host_bounds(P, name):
    """max_q_len and max_kv_len only need to bound the lengths (>=): bounds
    far above them size a launch with token tiles past every suffix (they
    leave at once), may switch the kernel, and with a workspace cut key
    parts whose later ranges hold no key of any sequence.  The output still
    matches the oracle on every element."""
    from paper_2608_14624_amd import ops
    extra_q, extra_kv, workspace, want_kernel, want_parts = LOOSE[name]
    invs = [Invocation(0, 90), Invocation(1, 33), Invocation(0, 1), Invocation(1, 200)]
    wl = build_workload("loose", 77, [700, 260], invs, num_q_heads=16, num_kv_heads=4,
                        head_dim=128, num_blocks=512)
    mq, mk = wl.max_q_len + extra_q, wl.max_kv_len + extra_kv
    kernel, grid, _ = ops.prefill_launch_shape(wl.batch, mq, 16, 4)
    need = ops.prefill_workspace_bytes(wl.batch, wl.total_q, mq, mk, 16, 4, 128)
    print(f"[case] loose bounds {name}: max_q_len {wl.max_q_len}->{mq}, max_kv_len "
          f"{wl.max_kv_len}->{mk}, kernel {kernel}, grid {grid}, workspace {need} B", flush=True)
    assert kernel == want_kernel and (need > 0) == want_parts
    # the block table widened so that max_blocks_per_seq * 16 covers the bound
    bt = np.zeros((wl.batch, -(-mk // 16)), np.int32)
    bt[:, :wl.block_tables.shape[1]] = wl.block_tables
    dev = torch.device("cuda")

    def bf16(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(dev)
    q = bf16(wl.q)
    out = torch.full_like(q, float("nan"))
    ops.cs_prefill_paged_attn(q, bf16(wl.k_pool), bf16(wl.v_pool), torch.from_numpy(bt).to(dev),
                              torch.from_numpy(wl.prefix_lens).to(dev),
                              torch.from_numpy(wl.cu_q_lens).to(dev), out, max_q_len=mq,
                              max_kv_len=mk, scale=wl.scale, workspace=workspace)
    torch.cuda.synchronize()
    got = out.view(torch.int16).cpu().numpy().view(np.uint16)
    mx, mean = compare_full(got, oracle_full(wl))
    print(f"    max_abs={mx:.3e} mean_abs={mean:.3e}", flush=True)
    assert mx <= MAX_ABS and mean <= MEAN_ABS


def test_hit_rows_match_miss_rows(P):
    # the same prompt served as a hit and as a miss
    for prefix, suffix in ((256, 64), (37, 100), (1000, 1)):
        invs = [Invocation(0, suffix, hit=True, suffix_key=0),
                Invocation(0, suffix, hit=False, suffix_key=0)]
        wl = build_workload("hitmiss", 8, [prefix], invs, num_q_heads=8, num_kv_heads=2,
                            head_dim=128, num_blocks=256)
        out = oracle.bf16_bits_to_f64(run_full(P, wl).out_bits())
        hit = out[:suffix]
        miss_tail = out[suffix + prefix:]
        assert np.abs(hit - miss_tail).max() <= MAX_ABS


def test_empty_batch_is_noop(P):
    ops, _ = P
    dev = torch.device("cuda:0")
    z = torch.zeros((0, 8, 64), dtype=torch.bfloat16, device=dev)
    pool = torch.zeros((4, 2, 16, 64), dtype=torch.bfloat16, device=dev)
    bt = torch.zeros((0, 1), dtype=torch.int32, device=dev)
    pl = torch.zeros((0,), dtype=torch.int32, device=dev)
    cu = torch.zeros((1,), dtype=torch.int32, device=dev)
    ops.cs_prefill_paged_attn(z, pool, pool, bt, pl, cu, z.clone(), max_q_len=0, max_kv_len=0,
                              scale=0.125)
    torch.cuda.synchronize()


def test_debug_check_rejects_out_of_range_block(P, monkeypatch):
    ops, pipeline = P
    wl = small_batch()
    wl.block_tables[1, 3] = wl.num_blocks + 5
    dw = pipeline.DeviceWorkload(wl)
    monkeypatch.setenv("CS_DEBUG_CHECK", "1")
    with pytest.raises(ops.CacheScoutError) as ei:
        dw.attention()
    assert ei.value.status == ops.CS_ERR_INVALID_ARG
    assert "block_tables[1][3]" in str(ei.value)


def test_debug_check_accepts_valid_metadata(P, monkeypatch):
    _, pipeline = P
    monkeypatch.setenv("CS_DEBUG_CHECK", "1")
    wl = small_batch()
    dw = pipeline.DeviceWorkload(wl)
    dw.attention()
    torch.cuda.synchronize()
