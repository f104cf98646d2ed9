"""The C ABI library on the CPU: it loads, exports every declared symbol, and
its host-side validation rejects bad arguments before touching a GPU.

No kernel is launched here; every call below returns from the argument checks
(or is a documented no-op) before the first HIP runtime call.
"""

import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "cachescout.h")

ops = pytest.importorskip("paper_2608_14624_amd.ops",
                          reason="libcachescout.so not built (run __graft_entry__.build())")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(cs_[a-z_0-9]+)\s*\(", text)))


def test_header_declares_the_expected_calls():
    assert declared_functions() == sorted(ops.EXPORTED)


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(ops.LIB_PATH)
    for name in declared_functions():
        assert hasattr(lib, name), f"{name} not exported"


def test_library_is_built_from_the_sources_beside_it():
    """A library left over from an earlier edit of the sources would make every
    GPU test check stale code: the digest the build embeds must match the tree."""
    from paper_2608_14624_amd import build
    assert ops.source_digest() == build.source_digest(), (
        "libcachescout.so is stale: rebuild with python -m paper_2608_14624_amd.build")


def test_status_strings():
    assert ops.status_string(0) == "CS_OK"
    assert ops.status_string(1) == "CS_ERR_INVALID_ARG"
    assert ops.status_string(2) == "CS_ERR_UNSUPPORTED"
    assert ops.status_string(3) == "CS_ERR_HIP"
    assert ops.status_string(77) == "CS_UNKNOWN_STATUS"


FAKE = 1 << 20   # a 16-byte aligned non-null address; never dereferenced here

GOOD = dict(q=FAKE, k_pool=FAKE, v_pool=FAKE, block_tables=FAKE, prefix_lens=FAKE,
            cu_q_lens=FAKE, batch=2, total_q=10, max_q_len=8, max_kv_len=40,
            max_blocks_per_seq=3, num_blocks=64, num_q_heads=8, num_kv_heads=2, head_dim=64,
            block_size=16, scale=0.125, out=FAKE, stream=0)


def attn(**kw):
    args = dict(GOOD)
    args.update(kw)
    return ops.cs_prefill_paged_attn_raw(**args)


@pytest.mark.parametrize("kw,status", [
    (dict(batch=-1), ops.CS_ERR_INVALID_ARG),
    (dict(total_q=-5), ops.CS_ERR_INVALID_ARG),
    (dict(num_kv_heads=3), ops.CS_ERR_INVALID_ARG),
    (dict(num_q_heads=0), ops.CS_ERR_INVALID_ARG),
    (dict(head_dim=96), ops.CS_ERR_UNSUPPORTED),
    (dict(head_dim=256), ops.CS_ERR_UNSUPPORTED),
    (dict(block_size=32), ops.CS_ERR_UNSUPPORTED),
    (dict(scale=float("nan")), ops.CS_ERR_INVALID_ARG),
    (dict(scale=float("inf")), ops.CS_ERR_INVALID_ARG),
    (dict(scale=0.0), ops.CS_ERR_UNSUPPORTED),
    (dict(scale=-0.0), ops.CS_ERR_UNSUPPORTED),
    (dict(scale=-0.125), ops.CS_ERR_UNSUPPORTED),
    (dict(q=None), ops.CS_ERR_INVALID_ARG),
    (dict(out=None), ops.CS_ERR_INVALID_ARG),
    (dict(block_tables=None), ops.CS_ERR_INVALID_ARG),
    (dict(max_blocks_per_seq=2), ops.CS_ERR_INVALID_ARG),    # 2 * 16 < 40
    (dict(max_q_len=41), ops.CS_ERR_INVALID_ARG),
    (dict(num_blocks=0), ops.CS_ERR_INVALID_ARG),
    (dict(q=FAKE + 2), ops.CS_ERR_INVALID_ARG),               # misaligned
    (dict(k_pool=FAKE + 8), ops.CS_ERR_INVALID_ARG),
])
def test_attention_rejects_bad_arguments(kw, status):
    assert attn(**kw) == status
    assert ops.last_error() != ""


@pytest.mark.parametrize("kw", [dict(batch=0), dict(total_q=0), dict(max_q_len=0),
                                dict(batch=0, q=None, out=None)])
def test_attention_empty_work_is_a_noop(kw):
    assert attn(**kw) == ops.CS_OK
    assert ops.last_error() == ""


PGOOD = dict(host_k=FAKE, host_v=FAKE, dst_block_ids=FAKE, n=4, k_pool=FAKE, v_pool=FAKE,
             num_blocks=64, num_kv_heads=2, head_dim=64, block_size=16, stream=0)


def prefetch(**kw):
    args = dict(PGOOD)
    args.update(kw)
    return ops.cs_kv_prefetch_raw(**args)


@pytest.mark.parametrize("kw,status", [
    (dict(n=-1), ops.CS_ERR_INVALID_ARG),
    (dict(head_dim=80), ops.CS_ERR_UNSUPPORTED),
    (dict(block_size=8), ops.CS_ERR_UNSUPPORTED),
    (dict(num_kv_heads=0), ops.CS_ERR_INVALID_ARG),
    (dict(host_k=None), ops.CS_ERR_INVALID_ARG),
    (dict(dst_block_ids=None), ops.CS_ERR_INVALID_ARG),
    (dict(n=65), ops.CS_ERR_INVALID_ARG),
    (dict(host_v=FAKE + 4), ops.CS_ERR_INVALID_ARG),
    (dict(n=2 ** 30, num_blocks=2 ** 31 - 1), ops.CS_ERR_INVALID_ARG),   # 2 n units overflow int32
])
def test_prefetch_rejects_bad_arguments(kw, status):
    assert prefetch(**kw) == status


def test_prefetch_zero_blocks_is_a_noop():
    assert prefetch(n=0, host_k=None, host_v=None) == ops.CS_OK


WGOOD = dict(k_new=FAKE, v_new=FAKE, slot_mapping=FAKE, num_tokens=10, k_pool=FAKE, v_pool=FAKE,
             num_blocks=64, num_kv_heads=2, head_dim=128, block_size=16, stream=0)


@pytest.mark.parametrize("kw,status", [
    (dict(num_tokens=-1), ops.CS_ERR_INVALID_ARG),
    (dict(head_dim=32), ops.CS_ERR_UNSUPPORTED),
    (dict(block_size=32), ops.CS_ERR_UNSUPPORTED),
    (dict(k_new=None), ops.CS_ERR_INVALID_ARG),
    (dict(slot_mapping=None), ops.CS_ERR_INVALID_ARG),
    (dict(num_blocks=0), ops.CS_ERR_INVALID_ARG),
    (dict(v_pool=FAKE + 2), ops.CS_ERR_INVALID_ARG),
])
def test_kv_write_rejects_bad_arguments(kw, status):
    args = dict(WGOOD)
    args.update(kw)
    assert ops.cs_kv_write_raw(**args) == status


def test_kv_write_zero_tokens_is_a_noop():
    args = dict(WGOOD, num_tokens=0, k_new=None)
    assert ops.cs_kv_write_raw(**args) == ops.CS_OK


OGOOD = dict(src_block_ids=FAKE, n=4, k_pool=FAKE, v_pool=FAKE, num_blocks=64, host_k=FAKE,
             host_v=FAKE, num_kv_heads=2, head_dim=64, block_size=16, stream=0)


@pytest.mark.parametrize("kw,status", [
    (dict(n=-1), ops.CS_ERR_INVALID_ARG),
    (dict(head_dim=96), ops.CS_ERR_UNSUPPORTED),
    (dict(host_k=None), ops.CS_ERR_INVALID_ARG),
    (dict(src_block_ids=None), ops.CS_ERR_INVALID_ARG),
    (dict(host_v=FAKE + 4), ops.CS_ERR_INVALID_ARG),
    (dict(n=2 ** 30), ops.CS_ERR_INVALID_ARG),
])
def test_kv_offload_rejects_bad_arguments(kw, status):
    args = dict(OGOOD)
    args.update(kw)
    assert ops.cs_kv_offload_raw(**args) == status


def test_kv_offload_zero_blocks_is_a_noop():
    assert ops.cs_kv_offload_raw(**dict(OGOOD, n=0, host_k=None)) == ops.CS_OK


DGOOD = dict(q=FAKE, k_pool=FAKE, v_pool=FAKE, block_tables=FAKE, seq_lens=FAKE, batch=4,
             max_seq_len=100, max_blocks_per_seq=7, num_blocks=64, num_q_heads=8, num_kv_heads=2,
             head_dim=128, block_size=16, scale=0.1, out=FAKE, stream=0)


@pytest.mark.parametrize("kw,status", [
    (dict(batch=-1), ops.CS_ERR_INVALID_ARG),
    (dict(num_q_heads=64, num_kv_heads=2), ops.CS_ERR_UNSUPPORTED),   # 32 heads per KV head
    (dict(num_kv_heads=3), ops.CS_ERR_INVALID_ARG),
    (dict(head_dim=80), ops.CS_ERR_UNSUPPORTED),
    (dict(q=None), ops.CS_ERR_INVALID_ARG),
    (dict(max_blocks_per_seq=6), ops.CS_ERR_INVALID_ARG),             # 96 < 100
    (dict(max_seq_len=0), ops.CS_ERR_INVALID_ARG),
    (dict(scale=float("inf")), ops.CS_ERR_INVALID_ARG),
    (dict(scale=0.0), ops.CS_ERR_UNSUPPORTED),
    (dict(scale=-0.0), ops.CS_ERR_UNSUPPORTED),
    (dict(scale=-0.125), ops.CS_ERR_UNSUPPORTED),
])
def test_decode_rejects_bad_arguments(kw, status):
    args = dict(DGOOD)
    args.update(kw)
    assert ops.cs_paged_decode_attn_raw(**args) == status


def test_decode_empty_batch_is_a_noop():
    assert ops.cs_paged_decode_attn_raw(**dict(DGOOD, batch=0, q=None)) == ops.CS_OK


CGOOD = dict(DGOOD, cu_groups=FAKE, shared_lens=FAKE, num_groups=2, max_group_seqs=3,
             max_shared_len=64, max_rest_len=36, workspace=FAKE, workspace_bytes=1 << 20)


def test_cascade_workspace_bytes():
    # (ceil(max_shared_len / 1024) + ceil(max_rest_len / 1024)) parts x batch x Hq x (D + 2) floats
    assert ops.cs_cascade_decode_workspace_bytes(4, 8, 128, 0, 0) == 0
    assert ops.cs_cascade_decode_workspace_bytes(4, 8, 128, 64, 0) == 1 * 4 * 8 * 130 * 4
    assert ops.cs_cascade_decode_workspace_bytes(4, 8, 128, 1024, 0) == 1 * 4 * 8 * 130 * 4
    assert ops.cs_cascade_decode_workspace_bytes(4, 8, 128, 1025, 0) == 2 * 4 * 8 * 130 * 4
    assert ops.cs_cascade_decode_workspace_bytes(4, 8, 128, 1025, 1025) == 4 * 4 * 8 * 130 * 4
    assert ops.cs_cascade_decode_workspace_bytes(4, 8, 64, 0, 1) == 1 * 4 * 8 * 66 * 4
    assert ops.cs_cascade_decode_workspace_bytes(-1, 8, 128, 64, 0) == -1
    assert ops.cs_cascade_decode_workspace_bytes(4, 0, 128, 64, 0) == -1
    assert ops.cs_cascade_decode_workspace_bytes(4, 8, 128, 64, -1) == -1


@pytest.mark.parametrize("kw,status", [
    (dict(batch=-1), ops.CS_ERR_INVALID_ARG),
    (dict(head_dim=96), ops.CS_ERR_UNSUPPORTED),
    (dict(num_q_heads=64, num_kv_heads=2), ops.CS_ERR_UNSUPPORTED),
    (dict(num_groups=0), ops.CS_ERR_INVALID_ARG),
    (dict(num_groups=5), ops.CS_ERR_INVALID_ARG),           # more groups than sequences
    (dict(max_group_seqs=0), ops.CS_ERR_INVALID_ARG),
    (dict(max_group_seqs=5), ops.CS_ERR_INVALID_ARG),
    (dict(max_shared_len=101), ops.CS_ERR_INVALID_ARG),     # beyond max_seq_len
    (dict(max_shared_len=-16), ops.CS_ERR_INVALID_ARG),
    (dict(max_rest_len=101), ops.CS_ERR_INVALID_ARG),      # beyond max_seq_len
    (dict(max_seq_len=600000, max_blocks_per_seq=37500, max_shared_len=500000,
          max_rest_len=100000, workspace_bytes=1 << 40), ops.CS_ERR_UNSUPPORTED),   # 587 partials
    (dict(max_rest_len=-1), ops.CS_ERR_INVALID_ARG),
    (dict(cu_groups=None), ops.CS_ERR_INVALID_ARG),
    (dict(shared_lens=None), ops.CS_ERR_INVALID_ARG),
    (dict(workspace=None), ops.CS_ERR_INVALID_ARG),
    (dict(workspace=FAKE + 8), ops.CS_ERR_INVALID_ARG),
    (dict(workspace_bytes=100), ops.CS_ERR_INVALID_ARG),
    (dict(workspace_bytes=-1), ops.CS_ERR_INVALID_ARG),
    (dict(scale=0.0), ops.CS_ERR_UNSUPPORTED),
    (dict(scale=-0.125), ops.CS_ERR_UNSUPPORTED),
])
def test_cascade_rejects_bad_arguments(kw, status):
    args = dict(CGOOD)
    args.update(kw)
    assert ops.cs_cascade_decode_attn_raw(**args) == status


def test_cascade_empty_batch_is_a_noop():
    assert ops.cs_cascade_decode_attn_raw(**dict(CGOOD, batch=0, q=None, num_groups=0,
                                                 workspace=None)) == ops.CS_OK


def test_library_exports_only_the_declared_calls():
    import shutil
    import subprocess
    nm = shutil.which("nm")
    if nm is None:
        pytest.skip("nm not available")
    out = subprocess.run([nm, "-D", "--defined-only", ops.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    text_symbols = sorted(line.split()[-1] for line in out.splitlines()
                          if len(line.split()) == 3 and line.split()[1] == "T")
    assert text_symbols == declared_functions()


@pytest.mark.parametrize("batch,max_q,hq,hkv,expect", [
    # 256-row ping-pong tiles: T = ceil(max_q / span) * batch * head_tiles,
    # span = 32 * 8 / heads_per_wg, head_tiles = hq / heads_per_wg
    (1, 1024, 32, 8, (ops.ATTN_SPLIT, 32 * 8, 0)),          # T = 128: split 128-row tiles
    (1, 1984, 32, 8, (ops.ATTN_SPLIT, 62 * 8, 0)),          # T = 248: split
    (1, 1985, 32, 8, (ops.ATTN_PING_PONG, 256, 0)),         # T = 256: one full round
    (1, 2049, 32, 8, (ops.ATTN_PING_PONG, 256 + 2 * 8, 16)),    # T = 264: tail of 8 tiles
    (2, 1024, 32, 8, (ops.ATTN_PING_PONG, 256, 0)),         # one full round
    (5, 500, 32, 8, (ops.ATTN_PING_PONG, 256 + 2 * 64, 128)),   # T = 320: tail of 64 tiles
    (3, 1024, 32, 8, (ops.ATTN_PING_PONG, 256 + 2 * 128, 256)),  # T = 384: tail of 128
    (7, 512, 32, 8, (ops.ATTN_PING_PONG, 448, 0)),          # T = 448: tail over half a round
    (7, 640, 16, 8, (ops.ATTN_PING_PONG, 256 + 2 * 24, 48)),    # G = 2: span 128, T = 280
    (17, 512, 8, 8, (ops.ATTN_PING_PONG, 256 + 2 * 16, 32)),    # G = 1: span 256, T = 272
    (11, 512, 12, 3, (ops.ATTN_PING_PONG, 11 * 2 * 12, 0)),     # 3 KV heads: no tail
    (0, 512, 32, 8, (ops.ATTN_SPLIT, 0, 0)),
    (4, 0, 32, 8, (ops.ATTN_SPLIT, 0, 0)),
])
def test_prefill_launch_shape(batch, max_q, hq, hkv, expect):
    assert ops.prefill_launch_shape(batch, max_q, hq, hkv, num_cus=256) == expect


@pytest.mark.parametrize("cus,expect", [
    # 128 ping-pong tiles: a full round on 128 CUs, under one on 256 or 160
    (128, (ops.ATTN_PING_PONG, 128, 0)),
    (160, (ops.ATTN_SPLIT, 256, 0)),
    (256, (ops.ATTN_SPLIT, 256, 0)),
    (120, (ops.ATTN_PING_PONG, 120 + 2 * 8, 16)),      # tail of 8 tiles after a round of 120
])
def test_prefill_launch_shape_follows_the_cu_count(cus, expect):
    assert ops.prefill_launch_shape(1, 1024, 32, 8, num_cus=cus) == expect


@pytest.mark.parametrize("args", [(-1, 64, 8, 2, 256), (1, -1, 8, 2, 256), (1, 64, 0, 2, 256),
                                  (1, 64, 8, 3, 256), (1, 64, 8, 0, 256), (1, 64, 8, 2, -1)])
def test_prefill_launch_shape_rejects_bad_arguments(args):
    with pytest.raises(ops.CacheScoutError) as ei:
        ops.prefill_launch_shape(*args)
    assert ei.value.args[0].startswith("CS_ERR_INVALID_ARG")


def cascade_noalloc(**kw):
    args = {k: v for k, v in CGOOD.items() if k not in ("workspace", "workspace_bytes")}
    args.update(kw)
    return ops.cs_cascade_decode_attn_noalloc_raw(**args)


@pytest.mark.parametrize("kw,status", [
    (dict(batch=-1), ops.CS_ERR_INVALID_ARG),
    (dict(head_dim=96), ops.CS_ERR_UNSUPPORTED),
    (dict(num_groups=0), ops.CS_ERR_INVALID_ARG),
    (dict(cu_groups=None), ops.CS_ERR_INVALID_ARG),
    (dict(scale=0.0), ops.CS_ERR_UNSUPPORTED),
    # 128 sequences x 32 heads x (D + 2) x 4 B x (8 + 8) partials = 34 MB > 32 MiB
    (dict(batch=128, num_q_heads=32, num_kv_heads=8, max_seq_len=16384, max_blocks_per_seq=1024,
          num_groups=8, max_group_seqs=16, max_shared_len=8192, max_rest_len=8192),
     ops.CS_ERR_UNSUPPORTED),
])
def test_cascade_noalloc_rejects_bad_arguments_before_any_gpu_call(kw, status):
    assert cascade_noalloc(**kw) == status
    if status == ops.CS_ERR_UNSUPPORTED and kw.get("batch") == 128:
        need = ops.cs_cascade_decode_workspace_bytes(128, 32, 128, 8192, 8192)
        assert need > ops.NOALLOC_SCRATCH_BYTES
        assert "scratch" in ops.last_error()


def test_cascade_noalloc_empty_batch_is_a_noop():
    assert cascade_noalloc(batch=0, q=None, num_groups=0) == ops.CS_OK


def test_noalloc_scratch_size_matches_the_header():
    text = open(HEADER).read()
    m = re.search(r"#define CS_NOALLOC_SCRATCH_BYTES \((\d+) \* (\d+) \* (\d+)\)", text)
    assert m and int(m[1]) * int(m[2]) * int(m[3]) == ops.NOALLOC_SCRATCH_BYTES


@pytest.mark.parametrize("args,expect", [
    # one GPU's shard of a 70B-shape agent launch: 4 x 512 tokens, 8 / 1 heads:
    # 128 split tiles on 256 CUs -> 2 key parts of fp32 (D + 2) per row
    ((4, 2048, 512, 4608, 8, 1, 128, 256), 2 * 2048 * 8 * 130 * 4),
    # 8 tiles -> 4 parts (the cap)
    ((1, 100, 100, 1000, 8, 2, 128, 256), 4 * 100 * 8 * 130 * 4),
    # 3 parts when 85 tiles (4 heads x 32 tokens) leave room for three
    ((1, 2720, 2720, 2720, 4, 1, 128, 256), 3 * 2720 * 4 * 130 * 4),
    ((1, 1024, 1024, 3072, 32, 8, 128, 256), 0),        # a full round of tiles: no parts
    ((1, 100, 100, 1000, 8, 2, 64, 256), 4 * 100 * 8 * 66 * 4),   # head_dim 64: (D + 2) = 66
    ((1, 100, 100, 100, 8, 2, 128, 256), 0),            # two key steps: no parts
    ((0, 0, 0, 0, 8, 2, 128, 256), 0),
    ((-1, 100, 100, 1000, 8, 2, 128, 256), -1),
    ((1, 100, 100, 1000, 8, 3, 128, 256), -1),
    ((1, 100, 100, 1000, 8, 2, 96, 256), -1),
])
def test_prefill_workspace_bytes(args, expect):
    assert ops.prefill_workspace_bytes(*args) == expect


def attn_ws(**kw):
    args = dict(GOOD, workspace=FAKE, workspace_bytes=1 << 20)
    args.update(kw)
    return ops.cs_prefill_paged_attn_ws_raw(**args)


@pytest.mark.parametrize("kw,status", [
    (dict(batch=-1), ops.CS_ERR_INVALID_ARG),
    (dict(head_dim=96), ops.CS_ERR_UNSUPPORTED),
    (dict(scale=0.0), ops.CS_ERR_UNSUPPORTED),
    (dict(q=None), ops.CS_ERR_INVALID_ARG),
    (dict(workspace_bytes=-1), ops.CS_ERR_INVALID_ARG),
])
def test_prefill_ws_rejects_bad_arguments_before_any_gpu_call(kw, status):
    assert attn_ws(**kw) == status


def test_prefill_ws_empty_batch_is_a_noop():
    assert attn_ws(batch=0, q=None, workspace=None, workspace_bytes=0) == ops.CS_OK
