"""Python binding of libcachescout.so (argument marshalling only).

The functions keep the C names.  They take PyTorch tensors for device memory,
pinned host memory and streams, pass raw pointers and sizes to the C ABI and
raise :class:`CacheScoutError` on a non-zero status.  All computation happens
in the HIP kernels; there is no fallback path: if the shared library is
missing or fails to load, importing this module raises.
"""

import ctypes
import os

import torch

# CACHESCOUT_LIB names another build of the same library (the host-sanitized
# one from build_sanitized.py); by default the in-tree build is loaded
_LIB_PATH = os.environ.get("CACHESCOUT_LIB") or os.path.join(
    os.path.dirname(os.path.abspath(__file__)), "libcachescout.so")

CS_OK = 0
CS_ERR_INVALID_ARG = 1
CS_ERR_UNSUPPORTED = 2
CS_ERR_HIP = 3

# every symbol the C header declares
EXPORTED = ("cs_prefill_paged_attn", "cs_kv_prefetch", "cs_kv_write", "cs_kv_offload",
            "cs_paged_decode_attn", "cs_status_string", "cs_last_error",
            "cs_scout_default_params", "cs_scout_create", "cs_scout_destroy",
            "cs_scout_agent_id", "cs_scout_observe_touch", "cs_scout_current",
            "cs_scout_transition_prob", "cs_scout_predict", "cs_scout_survival",
            "cs_scout_score_block", "cs_scout_select_victim", "cs_scout_predictability",
            "cs_scout_between_step", "cs_scout_state_bytes", "cs_scout_set_host_resident",
            "cs_scout_survival_all", "cs_scout_observe_touches", "cs_cascade_decode_attn",
            "cs_cascade_decode_workspace_bytes", "cs_prefill_paged_attn_launch_shape",
            "cs_source_digest", "cs_cascade_decode_attn_noalloc", "cs_prefill_paged_attn_ws",
            "cs_prefill_paged_attn_workspace_bytes")

# bytes of the device scratch array behind cs_cascade_decode_attn_noalloc
NOALLOC_SCRATCH_BYTES = 32 * 1024 * 1024


class ScoutParams(ctypes.Structure):
    """``cs_scout_params``: the control plane's hyperparameters."""
    _fields_ = [("eps", ctypes.c_double), ("tau", ctypes.c_double), ("e_max", ctypes.c_int32),
                ("lam", ctypes.c_double), ("delta", ctypes.c_double),
                ("r_min", ctypes.c_double)]


class CacheScoutError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(f"{status_string(status)}: {message}")
        self.status = status


def _load():
    if not os.path.exists(_LIB_PATH):
        raise ImportError(
            f"{_LIB_PATH} is missing: build it with `python -m paper_2608_14624_amd.build` "
            "(or __graft_entry__.build()); there is no non-HIP fallback")
    lib = ctypes.CDLL(_LIB_PATH)
    i32, vp, f32 = ctypes.c_int32, ctypes.c_void_p, ctypes.c_float
    lib.cs_prefill_paged_attn.argtypes = [vp, vp, vp, vp, vp, vp, i32, i32, i32, i32, i32, i32,
                                          i32, i32, i32, i32, f32, vp, vp]
    lib.cs_prefill_paged_attn.restype = ctypes.c_int
    lib.cs_prefill_paged_attn_ws.argtypes = [vp, vp, vp, vp, vp, vp, i32, i32, i32, i32, i32, i32,
                                             i32, i32, i32, i32, f32, vp, ctypes.c_int64, vp, vp]
    lib.cs_prefill_paged_attn_ws.restype = ctypes.c_int
    lib.cs_prefill_paged_attn_workspace_bytes.argtypes = [i32, i32, i32, i32, i32, i32, i32, i32]
    lib.cs_prefill_paged_attn_workspace_bytes.restype = ctypes.c_int64
    lib.cs_kv_prefetch.argtypes = [vp, vp, vp, i32, vp, vp, i32, i32, i32, i32, vp]
    lib.cs_kv_prefetch.restype = ctypes.c_int
    lib.cs_kv_write.argtypes = [vp, vp, vp, i32, vp, vp, i32, i32, i32, i32, vp]
    lib.cs_kv_write.restype = ctypes.c_int
    lib.cs_kv_offload.argtypes = [vp, i32, vp, vp, i32, vp, vp, i32, i32, i32, vp]
    lib.cs_kv_offload.restype = ctypes.c_int
    lib.cs_paged_decode_attn.argtypes = [vp, vp, vp, vp, vp, i32, i32, i32, i32, i32, i32, i32,
                                         i32, f32, vp, vp]
    lib.cs_paged_decode_attn.restype = ctypes.c_int
    lib.cs_cascade_decode_attn.argtypes = [vp, vp, vp, vp, vp, i32, i32, i32, i32, vp, vp, i32,
                                           i32, i32, i32, i32, i32, i32, i32, f32, vp,
                                           ctypes.c_int64, vp, vp]
    lib.cs_cascade_decode_attn.restype = ctypes.c_int
    lib.cs_cascade_decode_attn_noalloc.argtypes = [vp, vp, vp, vp, vp, i32, i32, i32, i32, vp, vp,
                                                   i32, i32, i32, i32, i32, i32, i32, i32, f32,
                                                   vp, vp]
    lib.cs_cascade_decode_attn_noalloc.restype = ctypes.c_int
    lib.cs_cascade_decode_workspace_bytes.argtypes = [i32, i32, i32, i32, i32]
    lib.cs_cascade_decode_workspace_bytes.restype = ctypes.c_int64
    lib.cs_status_string.argtypes = [ctypes.c_int]
    lib.cs_status_string.restype = ctypes.c_char_p
    lib.cs_last_error.argtypes = []
    lib.cs_last_error.restype = ctypes.c_char_p
    lib.cs_source_digest.argtypes = []
    lib.cs_source_digest.restype = ctypes.c_char_p
    i64, u64, f64, h = ctypes.c_int64, ctypes.c_uint64, ctypes.c_double, ctypes.c_void_p
    sigs = {
        "cs_scout_default_params": ([ctypes.POINTER(ScoutParams)], None),
        "cs_scout_create": ([i32, i32, ctypes.POINTER(ScoutParams), ctypes.POINTER(h)],
                            ctypes.c_int),
        "cs_scout_destroy": ([h], None),
        "cs_scout_agent_id": ([h, u64], i32),
        "cs_scout_observe_touch": ([h, i32, i32, i32, i64], ctypes.c_int),
        "cs_scout_current": ([h], i32),
        "cs_scout_transition_prob": ([h, i32, i32], f64),
        "cs_scout_predict": ([h], i32),
        "cs_scout_survival": ([h, i32], f64),
        "cs_scout_score_block": ([h, i32, i64], f64),
        "cs_scout_select_victim": ([h, ctypes.POINTER(i32), i32, i64], i32),
        "cs_scout_predictability": ([h], f64),
        "cs_scout_between_step": ([h], i32),
        "cs_scout_state_bytes": ([h], i64),
        "cs_scout_set_host_resident": ([h, i32, i32], ctypes.c_int),
        "cs_scout_survival_all": ([h, ctypes.POINTER(f64)], ctypes.c_int),
        "cs_scout_observe_touches": ([h, vp, vp, vp, vp, i32], ctypes.c_int),
        "cs_prefill_paged_attn_launch_shape": ([i32, i32, i32, i32, i32, ctypes.POINTER(i32),
                                                ctypes.POINTER(i64), ctypes.POINTER(i64)],
                                               ctypes.c_int),
    }
    for name, (args, res) in sigs.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    return lib


_lib = _load()
LIB_PATH = _LIB_PATH


def status_string(status):
    return _lib.cs_status_string(int(status)).decode()


def last_error():
    return _lib.cs_last_error().decode()


def source_digest():
    """Digest of the sources the loaded library was built from."""
    return _lib.cs_source_digest().decode()


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream_handle(stream, device):
    if stream is None:
        stream = torch.cuda.current_stream(device)
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _check(status):
    if status != CS_OK:
        raise CacheScoutError(status, last_error())


def cs_prefill_paged_attn_raw(q, k_pool, v_pool, block_tables, prefix_lens, cu_q_lens, batch,
                              total_q, max_q_len, max_kv_len, max_blocks_per_seq, num_blocks,
                              num_q_heads, num_kv_heads, head_dim, block_size, scale, out,
                              stream=0):
    """The C call with raw pointers (ints or None); returns the status code."""
    return _lib.cs_prefill_paged_attn(q, k_pool, v_pool, block_tables, prefix_lens, cu_q_lens,
                                      batch, total_q, max_q_len, max_kv_len, max_blocks_per_seq,
                                      num_blocks, num_q_heads, num_kv_heads, head_dim,
                                      block_size, ctypes.c_float(scale), out, stream)


def cs_kv_prefetch_raw(host_k, host_v, dst_block_ids, n, k_pool, v_pool, num_blocks,
                       num_kv_heads, head_dim, block_size, stream=0):
    """The C call with raw pointers (ints or None); returns the status code."""
    return _lib.cs_kv_prefetch(host_k, host_v, dst_block_ids, n, k_pool, v_pool, num_blocks,
                               num_kv_heads, head_dim, block_size, stream)


def _require(cond, msg):
    if not cond:
        raise CacheScoutError(CS_ERR_INVALID_ARG, msg)


ATTN_SPLIT, ATTN_PING_PONG = 0, 1


def prefill_launch_shape(batch, max_q_len, num_q_heads, num_kv_heads, num_cus=0):
    """``(kernel, grid, tail_work_groups)`` of a cs_prefill_paged_attn call
    (host-only): kernel is ATTN_SPLIT or ATTN_PING_PONG.  ``num_cus`` sizes
    the launch for that many compute units; 0 takes the current device's."""
    kernel, grid, tail = ctypes.c_int32(), ctypes.c_int64(), ctypes.c_int64()
    _check(_lib.cs_prefill_paged_attn_launch_shape(batch, max_q_len, num_q_heads, num_kv_heads,
                                                   num_cus, ctypes.byref(kernel),
                                                   ctypes.byref(grid), ctypes.byref(tail)))
    return kernel.value, grid.value, tail.value


def cs_prefill_paged_attn_ws_raw(q, k_pool, v_pool, block_tables, prefix_lens, cu_q_lens, batch,
                                 total_q, max_q_len, max_kv_len, max_blocks_per_seq, num_blocks,
                                 num_q_heads, num_kv_heads, head_dim, block_size, scale, workspace,
                                 workspace_bytes, out, stream=0):
    """The C call with a workspace, raw pointers (ints or None); returns the status code."""
    return _lib.cs_prefill_paged_attn_ws(q, k_pool, v_pool, block_tables, prefix_lens, cu_q_lens,
                                         batch, total_q, max_q_len, max_kv_len, max_blocks_per_seq,
                                         num_blocks, num_q_heads, num_kv_heads, head_dim,
                                         block_size, ctypes.c_float(scale), workspace,
                                         workspace_bytes, out, stream)


def prefill_workspace_bytes(batch, total_q, max_q_len, max_kv_len, num_q_heads, num_kv_heads,
                            head_dim, num_cus=0):
    """Bytes of workspace ``cs_prefill_paged_attn_ws`` takes (0: the launch
    does not split its keys into parts)."""
    return int(_lib.cs_prefill_paged_attn_workspace_bytes(batch, total_q, max_q_len, max_kv_len,
                                                          num_q_heads, num_kv_heads, head_dim,
                                                          num_cus))


def _prefill_args(q, k_pool, v_pool, block_tables, prefix_lens, cu_q_lens, out, max_q_len,
                  max_kv_len, scale):
    """Validate a prefill attention call's tensors; the C arguments up to the
    scale, the output pointer and the device."""
    dev = q.device
    for name, t, dt in (("q", q, torch.bfloat16), ("k_pool", k_pool, torch.bfloat16),
                        ("v_pool", v_pool, torch.bfloat16), ("out", out, torch.bfloat16),
                        ("block_tables", block_tables, torch.int32),
                        ("prefix_lens", prefix_lens, torch.int32),
                        ("cu_q_lens", cu_q_lens, torch.int32)):
        _require(t.device == dev and t.is_cuda, f"{name} must be on {dev}")
        _require(t.dtype == dt, f"{name} must be {dt}")
        _require(t.is_contiguous(), f"{name} must be contiguous")
    _require(q.dim() == 3 and out.shape == q.shape, "q and out must be [total_q, Hq, D]")
    _require(k_pool.dim() == 4 and v_pool.shape == k_pool.shape,
             "pools must be [num_blocks, Hkv, block_size, D]")
    _require(block_tables.dim() == 2, "block_tables must be [B, max_blocks]")
    total_q, hq, d = q.shape
    num_blocks, hkv, bs, d2 = k_pool.shape
    _require(d == d2, "head_dim of q and pools differ")
    batch = block_tables.shape[0]
    _require(prefix_lens.numel() == batch and cu_q_lens.numel() == batch + 1,
             "prefix_lens must have B entries and cu_q_lens B + 1")
    args = (_ptr(q), _ptr(k_pool), _ptr(v_pool), _ptr(block_tables), _ptr(prefix_lens),
            _ptr(cu_q_lens), batch, total_q, int(max_q_len), int(max_kv_len),
            block_tables.shape[1], num_blocks, hq, hkv, d, bs, ctypes.c_float(scale))
    return args, _ptr(out), dev


def _resolve_workspace(workspace, args, dev):
    """None: the call without a workspace.  "auto": a new uint8 GPU tensor of
    the size the call needs (None if it needs none).  A tensor: used as is."""
    if workspace is None or (isinstance(workspace, str) and workspace == "auto"):
        if workspace is None:
            return None
        batch, total_q, max_q, max_kv = args[6], args[7], args[8], args[9]
        hq, hkv, d = args[12], args[13], args[14]
        need = prefill_workspace_bytes(batch, total_q, max_q, max_kv, hq, hkv, d)
        _require(need >= 0, "no workspace size for these arguments")
        if need == 0:
            return None
        return torch.empty(need, dtype=torch.uint8, device=dev)
    _require(workspace.is_cuda and workspace.device == dev, f"workspace must be on {dev}")
    return workspace


def cs_prefill_paged_attn(q, k_pool, v_pool, block_tables, prefix_lens, cu_q_lens, out, *,
                          max_q_len, max_kv_len, scale, workspace=None, stream=None):
    """Enqueue paged prefill attention on ``stream`` (default: the current stream).

    Tensors: ``q``/``out`` bf16 ``[total_q, Hq, D]``; pools bf16
    ``[num_blocks, Hkv, 16, D]``; ``block_tables`` int32 ``[B, max_blocks]``;
    ``prefix_lens`` int32 ``[B]``; ``cu_q_lens`` int32 ``[B+1]``; all on the
    same GPU and contiguous.  ``max_q_len``/``max_kv_len`` are host integers
    bounding the suffix and total lengths.  ``workspace``: None (the plain
    call), "auto" (``cs_prefill_paged_attn_ws`` with a workspace allocated
    here when the launch splits its keys), or a uint8 GPU tensor for it.
    """
    args, outp, dev = _prefill_args(q, k_pool, v_pool, block_tables, prefix_lens, cu_q_lens, out,
                                    max_q_len, max_kv_len, scale)
    ws = _resolve_workspace(workspace, args, dev)
    handle = _stream_handle(stream, dev)
    if workspace is None:
        _check(_lib.cs_prefill_paged_attn(*args, outp, handle))
    else:
        _check(_lib.cs_prefill_paged_attn_ws(*args, _ptr(ws),
                                             0 if ws is None else ws.numel(), outp, handle))


class PrefillCall:
    """A prefill attention call with its tensors validated once.

    Serving loops launch the same attention over the same buffers again and
    again; this keeps the argument checks and pointer extraction out of the
    per-launch path, so each launch costs one C call.  The tensors must stay
    alive and unchanged in shape while the object is used.  ``workspace`` as
    for :func:`cs_prefill_paged_attn` ("auto" allocates it once, here).
    """

    def __init__(self, q, k_pool, v_pool, block_tables, prefix_lens, cu_q_lens, out, *,
                 max_q_len, max_kv_len, scale, workspace=None):
        args, outp, dev = _prefill_args(q, k_pool, v_pool, block_tables, prefix_lens, cu_q_lens,
                                        out, max_q_len, max_kv_len, scale)
        self.device = dev
        self.workspace = _resolve_workspace(workspace, args, dev)
        self._keep = (q, k_pool, v_pool, block_tables, prefix_lens, cu_q_lens, out)
        if workspace is None:
            self._fn = _lib.cs_prefill_paged_attn
            self._args = args + (outp,)
        else:
            ws = self.workspace
            self._fn = _lib.cs_prefill_paged_attn_ws
            self._args = args + (_ptr(ws), 0 if ws is None else ws.numel(), outp)

    def __call__(self, stream=None):
        _check(self._fn(*self._args, _stream_handle(stream, self.device)))


def cs_kv_prefetch(host_k, host_v, dst_block_ids, k_pool, v_pool, *, stream=None):
    """Enqueue the host-to-pool block copy on ``stream`` (default: current stream).

    ``host_k``/``host_v``: pinned CPU bf16 tensors ``[n, Hkv, 16, D]``;
    ``dst_block_ids``: int32 GPU tensor ``[n]``; pools as for attention.
    """
    dev = k_pool.device
    _require(host_k.device.type == "cpu" and host_v.device.type == "cpu",
             "host blocks must be CPU tensors")
    _require(host_k.is_pinned() and host_v.is_pinned(), "host blocks must be pinned")
    _require(host_k.dtype == torch.bfloat16 and host_v.dtype == torch.bfloat16,
             "host blocks must be bf16")
    _require(host_k.is_contiguous() and host_v.is_contiguous(), "host blocks must be contiguous")
    _require(dst_block_ids.dtype == torch.int32 and dst_block_ids.device == dev,
             "dst_block_ids must be int32 on the pool's device")
    _require(k_pool.shape == v_pool.shape and k_pool.dtype == torch.bfloat16,
             "pools must match and be bf16")
    n = dst_block_ids.numel()
    _require(host_k.shape[0] >= n and host_v.shape[0] >= n, "fewer host blocks than ids")
    _require(tuple(host_k.shape[1:]) == tuple(k_pool.shape[1:]), "host block shape != pool block shape")
    num_blocks, hkv, bs, d = k_pool.shape
    status = cs_kv_prefetch_raw(_ptr(host_k), _ptr(host_v), _ptr(dst_block_ids), n,
                                _ptr(k_pool), _ptr(v_pool), num_blocks, hkv, d, bs,
                                _stream_handle(stream, dev))
    _check(status)


def cs_kv_write_raw(k_new, v_new, slot_mapping, num_tokens, k_pool, v_pool, num_blocks,
                    num_kv_heads, head_dim, block_size, stream=0):
    """The C call with raw pointers (ints or None); returns the status code."""
    return _lib.cs_kv_write(k_new, v_new, slot_mapping, num_tokens, k_pool, v_pool, num_blocks,
                            num_kv_heads, head_dim, block_size, stream)


def cs_kv_offload_raw(src_block_ids, n, k_pool, v_pool, num_blocks, host_k, host_v,
                      num_kv_heads, head_dim, block_size, stream=0):
    """The C call with raw pointers (ints or None); returns the status code."""
    return _lib.cs_kv_offload(src_block_ids, n, k_pool, v_pool, num_blocks, host_k, host_v,
                              num_kv_heads, head_dim, block_size, stream)


def cs_kv_write(k_new, v_new, slot_mapping, k_pool, v_pool, *, stream=None):
    """Enqueue the write of new tokens' K/V into their pool slots.

    ``k_new``/``v_new``: bf16 GPU tensors ``[T, Hkv, D]``; ``slot_mapping``:
    int32 GPU tensor ``[T]`` (block * 16 + offset, negative = skip); pools as
    for attention.
    """
    dev = k_pool.device
    for name, t, dt in (("k_new", k_new, torch.bfloat16), ("v_new", v_new, torch.bfloat16),
                        ("slot_mapping", slot_mapping, torch.int32),
                        ("k_pool", k_pool, torch.bfloat16), ("v_pool", v_pool, torch.bfloat16)):
        _require(t.is_cuda and t.device == dev, f"{name} must be on {dev}")
        _require(t.dtype == dt, f"{name} must be {dt}")
        _require(t.is_contiguous(), f"{name} must be contiguous")
    _require(k_new.shape == v_new.shape and k_new.dim() == 3, "k_new/v_new must be [T, Hkv, D]")
    _require(k_pool.shape == v_pool.shape, "pools must match")
    num_blocks, hkv, bs, d = k_pool.shape
    _require(tuple(k_new.shape[1:]) == (hkv, d), "token rows must match the pool's heads and dims")
    n = k_new.shape[0]
    _require(slot_mapping.numel() == n, "slot_mapping must have one entry per token")
    _check(cs_kv_write_raw(_ptr(k_new), _ptr(v_new), _ptr(slot_mapping), n, _ptr(k_pool),
                           _ptr(v_pool), num_blocks, hkv, d, bs, _stream_handle(stream, dev)))


def cs_kv_offload(src_block_ids, k_pool, v_pool, host_k, host_v, *, stream=None):
    """Enqueue the copy of pool blocks ``src_block_ids`` into pinned host buffers."""
    dev = k_pool.device
    _require(host_k.device.type == "cpu" and host_v.device.type == "cpu",
             "host blocks must be CPU tensors")
    _require(host_k.is_pinned() and host_v.is_pinned(), "host blocks must be pinned")
    _require(host_k.dtype == torch.bfloat16 and host_v.dtype == torch.bfloat16,
             "host blocks must be bf16")
    _require(host_k.is_contiguous() and host_v.is_contiguous(), "host blocks must be contiguous")
    _require(src_block_ids.dtype == torch.int32 and src_block_ids.device == dev,
             "src_block_ids must be int32 on the pool's device")
    _require(k_pool.shape == v_pool.shape and k_pool.dtype == torch.bfloat16,
             "pools must match and be bf16")
    n = src_block_ids.numel()
    _require(host_k.shape[0] >= n and host_v.shape[0] >= n, "fewer host blocks than ids")
    _require(tuple(host_k.shape[1:]) == tuple(k_pool.shape[1:]), "host block shape != pool block shape")
    num_blocks, hkv, bs, d = k_pool.shape
    _check(cs_kv_offload_raw(_ptr(src_block_ids), n, _ptr(k_pool), _ptr(v_pool), num_blocks,
                             _ptr(host_k), _ptr(host_v), hkv, d, bs, _stream_handle(stream, dev)))


def cs_paged_decode_attn_raw(q, k_pool, v_pool, block_tables, seq_lens, batch, max_seq_len,
                             max_blocks_per_seq, num_blocks, num_q_heads, num_kv_heads, head_dim,
                             block_size, scale, out, stream=0):
    """The C call with raw pointers (ints or None); returns the status code."""
    return _lib.cs_paged_decode_attn(q, k_pool, v_pool, block_tables, seq_lens, batch,
                                     max_seq_len, max_blocks_per_seq, num_blocks, num_q_heads,
                                     num_kv_heads, head_dim, block_size, ctypes.c_float(scale),
                                     out, stream)


def cs_paged_decode_attn(q, k_pool, v_pool, block_tables, seq_lens, out, *, max_seq_len, scale,
                         stream=None):
    """Enqueue paged decode attention: ``q``/``out`` bf16 ``[B, Hq, D]``,
    ``seq_lens`` int32 ``[B]``, pools and block tables as for prefill."""
    dev = q.device
    for name, t, dt in (("q", q, torch.bfloat16), ("k_pool", k_pool, torch.bfloat16),
                        ("v_pool", v_pool, torch.bfloat16), ("out", out, torch.bfloat16),
                        ("block_tables", block_tables, torch.int32),
                        ("seq_lens", seq_lens, torch.int32)):
        _require(t.is_cuda and t.device == dev, f"{name} must be on {dev}")
        _require(t.dtype == dt, f"{name} must be {dt}")
        _require(t.is_contiguous(), f"{name} must be contiguous")
    _require(q.dim() == 3 and out.shape == q.shape, "q and out must be [B, Hq, D]")
    _require(k_pool.shape == v_pool.shape and k_pool.dim() == 4, "pools must match")
    batch, hq, d = q.shape
    num_blocks, hkv, bs, d2 = k_pool.shape
    _require(d == d2, "head_dim of q and pools differ")
    _require(block_tables.dim() == 2 and block_tables.shape[0] == batch, "block_tables must be [B, max_blocks]")
    _require(seq_lens.numel() == batch, "seq_lens must have B entries")
    _check(cs_paged_decode_attn_raw(_ptr(q), _ptr(k_pool), _ptr(v_pool), _ptr(block_tables),
                                    _ptr(seq_lens), batch, int(max_seq_len), block_tables.shape[1],
                                    num_blocks, hq, hkv, d, bs, float(scale), _ptr(out),
                                    _stream_handle(stream, dev)))


def cs_cascade_decode_attn_raw(q, k_pool, v_pool, block_tables, seq_lens, batch, max_seq_len,
                               max_blocks_per_seq, num_blocks, cu_groups, shared_lens, num_groups,
                               max_group_seqs, max_shared_len, max_rest_len, num_q_heads,
                               num_kv_heads, head_dim, block_size, scale, workspace,
                               workspace_bytes, out, stream=0):
    """The C call with raw pointers (ints or None); returns the status code."""
    return _lib.cs_cascade_decode_attn(q, k_pool, v_pool, block_tables, seq_lens, batch,
                                       max_seq_len, max_blocks_per_seq, num_blocks, cu_groups,
                                       shared_lens, num_groups, max_group_seqs, max_shared_len,
                                       max_rest_len, num_q_heads, num_kv_heads, head_dim,
                                       block_size, ctypes.c_float(scale), workspace,
                                       workspace_bytes, out, stream)


def cs_cascade_decode_attn_noalloc_raw(q, k_pool, v_pool, block_tables, seq_lens, batch,
                                       max_seq_len, max_blocks_per_seq, num_blocks, cu_groups,
                                       shared_lens, num_groups, max_group_seqs, max_shared_len,
                                       max_rest_len, num_q_heads, num_kv_heads, head_dim,
                                       block_size, scale, out, stream=0):
    """The allocation-free C call with raw pointers (ints or None); returns the status."""
    return _lib.cs_cascade_decode_attn_noalloc(q, k_pool, v_pool, block_tables, seq_lens, batch,
                                               max_seq_len, max_blocks_per_seq, num_blocks,
                                               cu_groups, shared_lens, num_groups,
                                               max_group_seqs, max_shared_len, max_rest_len,
                                               num_q_heads, num_kv_heads, head_dim, block_size,
                                               ctypes.c_float(scale), out, stream)


def cs_cascade_decode_workspace_bytes(batch, num_q_heads, head_dim, max_shared_len, max_rest_len):
    return int(_lib.cs_cascade_decode_workspace_bytes(batch, num_q_heads, head_dim,
                                                      max_shared_len, max_rest_len))


def cs_cascade_decode_attn(q, k_pool, v_pool, block_tables, seq_lens, cu_groups, shared_lens,
                           out, *, max_seq_len, max_group_seqs, max_shared_len, max_rest_len,
                           scale, workspace=None, stream=None):
    """Enqueue cascade decode attention.  Tensors as for
    :func:`cs_paged_decode_attn`, plus ``cu_groups`` int32 ``[G+1]`` and
    ``shared_lens`` int32 ``[G]`` on the device.  ``workspace``: a uint8 GPU
    tensor of at least :func:`cs_cascade_decode_workspace_bytes` bytes, or
    None to allocate one here (the C call itself allocates nothing)."""
    dev = q.device
    for name, t, dt in (("q", q, torch.bfloat16), ("k_pool", k_pool, torch.bfloat16),
                        ("v_pool", v_pool, torch.bfloat16), ("out", out, torch.bfloat16),
                        ("block_tables", block_tables, torch.int32),
                        ("seq_lens", seq_lens, torch.int32), ("cu_groups", cu_groups, torch.int32),
                        ("shared_lens", shared_lens, torch.int32)):
        _require(t.is_cuda and t.device == dev, f"{name} must be on {dev}")
        _require(t.dtype == dt, f"{name} must be {dt}")
        _require(t.is_contiguous(), f"{name} must be contiguous")
    _require(q.dim() == 3 and out.shape == q.shape, "q and out must be [B, Hq, D]")
    _require(k_pool.shape == v_pool.shape and k_pool.dim() == 4, "pools must match")
    batch, hq, d = q.shape
    num_blocks, hkv, bs, d2 = k_pool.shape
    _require(d == d2, "head_dim of q and pools differ")
    _require(block_tables.dim() == 2 and block_tables.shape[0] == batch, "block_tables must be [B, max_blocks]")
    _require(seq_lens.numel() == batch, "seq_lens must have B entries")
    num_groups = shared_lens.numel()
    _require(cu_groups.numel() == num_groups + 1, "cu_groups must have G + 1 entries")
    need = cs_cascade_decode_workspace_bytes(batch, hq, d, int(max_shared_len), int(max_rest_len))
    if workspace is None:
        workspace = torch.empty(max(need, 16), dtype=torch.uint8, device=dev)
    _require(workspace.is_cuda and workspace.device == dev, f"workspace must be on {dev}")
    _check(cs_cascade_decode_attn_raw(
        _ptr(q), _ptr(k_pool), _ptr(v_pool), _ptr(block_tables), _ptr(seq_lens), batch,
        int(max_seq_len), block_tables.shape[1], num_blocks, _ptr(cu_groups), _ptr(shared_lens),
        num_groups, int(max_group_seqs), int(max_shared_len), int(max_rest_len), hq, hkv, d, bs,
        float(scale),
        _ptr(workspace), workspace.numel() * workspace.element_size(), _ptr(out),
        _stream_handle(stream, dev)))


def cs_cascade_decode_attn_noalloc(q, k_pool, v_pool, block_tables, seq_lens, cu_groups,
                                   shared_lens, out, *, max_seq_len, max_group_seqs,
                                   max_shared_len, max_rest_len, scale, stream=None):
    """Enqueue cascade decode attention with the partials in the library's
    per-device scratch array (no workspace, nothing allocated; calls on one
    device must not overlap).  Tensors as for :func:`cs_cascade_decode_attn`."""
    dev = q.device
    for name, t, dt in (("q", q, torch.bfloat16), ("k_pool", k_pool, torch.bfloat16),
                        ("v_pool", v_pool, torch.bfloat16), ("out", out, torch.bfloat16),
                        ("block_tables", block_tables, torch.int32),
                        ("seq_lens", seq_lens, torch.int32), ("cu_groups", cu_groups, torch.int32),
                        ("shared_lens", shared_lens, torch.int32)):
        _require(t.is_cuda and t.device == dev, f"{name} must be on {dev}")
        _require(t.dtype == dt, f"{name} must be {dt}")
        _require(t.is_contiguous(), f"{name} must be contiguous")
    _require(q.dim() == 3 and out.shape == q.shape, "q and out must be [B, Hq, D]")
    _require(k_pool.shape == v_pool.shape and k_pool.dim() == 4, "pools must match")
    batch, hq, d = q.shape
    num_blocks, hkv, bs, d2 = k_pool.shape
    _require(d == d2, "head_dim of q and pools differ")
    _require(block_tables.dim() == 2 and block_tables.shape[0] == batch, "block_tables must be [B, max_blocks]")
    _require(seq_lens.numel() == batch, "seq_lens must have B entries")
    num_groups = shared_lens.numel()
    _require(cu_groups.numel() == num_groups + 1, "cu_groups must have G + 1 entries")
    _check(cs_cascade_decode_attn_noalloc_raw(
        _ptr(q), _ptr(k_pool), _ptr(v_pool), _ptr(block_tables), _ptr(seq_lens), batch,
        int(max_seq_len), block_tables.shape[1], num_blocks, _ptr(cu_groups), _ptr(shared_lens),
        num_groups, int(max_group_seqs), int(max_shared_len), int(max_rest_len), hq, hkv, d, bs,
        float(scale), _ptr(out), _stream_handle(stream, dev)))


def scout_default_params():
    p = ScoutParams()
    _lib.cs_scout_default_params(ctypes.byref(p))
    return p


class Scout:
    """Owner of a ``cs_scout`` handle: the host-side control plane (transition
    learner, survival scorer, prefetch coordinator).  Methods map one to one
    onto the ``cs_scout_*`` calls; -1 from the C side becomes ``None``."""

    def __init__(self, num_agents, num_blocks, **params):
        prm = scout_default_params()
        for k, v in params.items():
            if not hasattr(prm, k):
                raise TypeError(f"unknown control-plane parameter {k!r}")
            setattr(prm, k, v)
        handle = ctypes.c_void_p()
        _check(_lib.cs_scout_create(int(num_agents), int(num_blocks), ctypes.byref(prm),
                                    ctypes.byref(handle)))
        self._h = handle
        self._destroy = _lib.cs_scout_destroy   # still reachable at interpreter exit
        self.num_agents = int(num_agents)
        self.num_blocks = int(num_blocks)
        self.params = prm

    def close(self):
        if getattr(self, "_h", None):
            self._destroy(self._h)
            self._h = None

    def __del__(self):
        self.close()

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    @staticmethod
    def _opt(v):
        return None if v < 0 else v

    def agent_id(self, fingerprint):
        return self._opt(_lib.cs_scout_agent_id(self._h, fingerprint & 0xFFFFFFFFFFFFFFFF))

    def observe_touch(self, block, agent, tokens, now):
        _check(_lib.cs_scout_observe_touch(self._h, block, agent, tokens, now))

    def observe_touches(self, blocks, agents, tokens, now):
        """Batched touches from four equal-length int32/int32/int32/int64
        numpy arrays (C-contiguous)."""
        import numpy as np
        arrs = [np.ascontiguousarray(blocks, dtype=np.int32),
                np.ascontiguousarray(agents, dtype=np.int32),
                np.ascontiguousarray(tokens, dtype=np.int32),
                np.ascontiguousarray(now, dtype=np.int64)]
        n = len(arrs[0])
        if any(len(a) != n for a in arrs):
            raise CacheScoutError(CS_ERR_INVALID_ARG, "touch arrays differ in length")
        _check(_lib.cs_scout_observe_touches(self._h, *(a.ctypes.data for a in arrs), n))

    @property
    def current(self):
        return self._opt(_lib.cs_scout_current(self._h))

    def transition_prob(self, i, j):
        return _lib.cs_scout_transition_prob(self._h, i, j)

    def predict(self):
        return self._opt(_lib.cs_scout_predict(self._h))

    def survival(self, agent):
        return _lib.cs_scout_survival(self._h, agent)

    def score_block(self, block, now):
        return _lib.cs_scout_score_block(self._h, block, now)

    def set_host_resident(self, block, resident):
        _check(_lib.cs_scout_set_host_resident(self._h, block, 1 if resident else 0))

    def survival_all(self):
        out = (ctypes.c_double * self.num_agents)()
        _check(_lib.cs_scout_survival_all(self._h, out))
        return list(out)

    def select_victim(self, candidates, now):
        arr = (ctypes.c_int32 * len(candidates))(*candidates)
        return self._opt(_lib.cs_scout_select_victim(self._h, arr, len(candidates), now))

    def predictability(self):
        return _lib.cs_scout_predictability(self._h)

    def between_step(self):
        return self._opt(_lib.cs_scout_between_step(self._h))

    def state_bytes(self):
        return _lib.cs_scout_state_bytes(self._h)
