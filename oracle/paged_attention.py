"""Float64 oracle of paged prefix-reuse prefill attention (test infrastructure).

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s ``cpu_baseline``
may use this module; see the package docstring.

The operation (arXiv 2608.14624, Sec. 2.1 "Prefix caching"; Sec. 4 on the
unchanged attention kernels): invocation ``r`` has a cached prefix of ``P_r``
tokens whose K/V already sit in a paged pool, and ``S_r`` new suffix tokens
whose K/V have been written to the pool as well.  Its ``S_r`` suffix queries
attend over all ``L_r = P_r + S_r`` keys with a causal mask aligned to the end
of the prompt: suffix row ``i`` is prompt position ``P_r + i`` and sees keys
``0 .. P_r + i``.  Because a prefix hit reuses the prefix KV instead of
recomputing it, this is exactly the last ``S_r`` rows of causal attention over
the whole prompt; a miss is the case ``P_r = 0``.

Layouts (all arrays are NumPy):

* ``q``            uint16 bf16 bit patterns ``[total_q, Hq, D]``; the suffix
                   tokens of the invocations packed one after another.
* ``k_pool``,
  ``v_pool``       uint16 bf16 bit patterns ``[num_blocks, Hkv, block_size, D]``.
* ``block_tables`` int ``[B, max_blocks]``; row ``r`` maps logical block
                   ``b`` (tokens ``b*block_size ..``) to a pool slot, for
                   ``b < ceil(L_r / block_size)``.  Later entries are never read.
* ``prefix_lens``  int ``[B]`` (``P_r``); ``cu_q_lens`` int ``[B+1]``, prefix
                   sums of ``S_r``.

Query head ``h`` reads KV head ``h // (Hq // Hkv)`` (consecutive grouping).
All bf16 inputs are widened exactly to float64; the scale is the float32 value
the kernel receives, widened exactly; logits, softmax and the weighted sum of
values are float64 and the result is returned unrounded.
"""

import numpy as np


def bf16_bits_to_f64(bits):
    """Widen bf16 bit patterns (uint16) exactly to float64.

    A bf16 number is the upper half of the float32 with the same sign,
    exponent and leading mantissa bits, so the widening is a 16-bit shift.
    """
    b = np.asarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def kv_head_of(h, num_q_heads, num_kv_heads):
    """KV head read by query head ``h`` under grouped-query attention.

    ``G = Hq / Hkv`` consecutive query heads share one KV head.
    """
    group = num_q_heads // num_kv_heads
    return h // group


def visible_keys(prefix_len, i):
    """Number of keys suffix row ``i`` may attend to: positions ``0 .. P + i``."""
    return prefix_len + i + 1


def gather_logical_kv(pool_bits, table_row, length, g, block_size):
    """Logical K (or V) rows ``0 .. length-1`` of one sequence for KV head ``g``.

    Token ``j`` lives in pool slot ``table_row[j // block_size]`` at offset
    ``j % block_size``.  Only the ``ceil(length / block_size)`` slots the
    sequence covers are read, and positions at or beyond ``length`` inside the
    last block are dropped.  Returns float64 ``[length, D]``.
    """
    if length == 0:
        return np.zeros((0, pool_bits.shape[-1]), dtype=np.float64)
    n_blocks = -(-length // block_size)
    slots = np.asarray(table_row[:n_blocks], dtype=np.int64)
    tiles = pool_bits[slots, g]                      # [n_blocks, block_size, D]
    rows = tiles.reshape(n_blocks * block_size, -1)[:length]
    return bf16_bits_to_f64(rows)


def _softmax_weighted_sum(logits, values):
    """Row-wise softmax of ``logits`` (masked entries are -inf) applied to ``values``."""
    m = logits.max(axis=-1, keepdims=True)
    w = np.exp(logits - m)
    return (w @ values) / w.sum(axis=-1, keepdims=True)


def _scale64(scale):
    return float(np.float32(scale))


def packed_row(cu_q_lens, r, i):
    """Row of the packed ``[total_q, ...]`` arrays that holds suffix token ``i``
    of invocation ``r``: the invocations' suffixes are stored one after
    another, so it is ``cu_q_lens[r] + i``."""
    return int(cu_q_lens[r]) + i


def _kv_group_key(r, g):
    """Gathered K/V depend on the invocation (its block table and length) and
    on the KV head, so sampled rows share a gather only when both agree."""
    return (r, g)


def prefill_paged_attn(q, k_pool, v_pool, block_tables, prefix_lens, cu_q_lens,
                       num_q_heads, num_kv_heads, scale, block_size=16):
    """Full float64 output ``[total_q, Hq, D]`` of paged prefill attention."""
    q = np.asarray(q)
    total_q, hq, d = q.shape
    assert hq == num_q_heads and num_q_heads % num_kv_heads == 0
    cu = np.asarray(cu_q_lens, dtype=np.int64)
    pl = np.asarray(prefix_lens, dtype=np.int64)
    s64 = _scale64(scale)
    out = np.zeros((total_q, hq, d), dtype=np.float64)
    for r in range(len(pl)):
        s_len = int(cu[r + 1] - cu[r])
        if s_len == 0:
            continue
        p_len = int(pl[r])
        length = p_len + s_len
        # key j is visible to suffix row i iff j < visible_keys(P, i)
        rows_i = np.arange(s_len)[:, None]
        keys_j = np.arange(length)[None, :]
        allowed = keys_j < visible_keys(p_len, rows_i)
        for g in range(num_kv_heads):
            kk = gather_logical_kv(k_pool, block_tables[r], length, g, block_size)
            vv = gather_logical_kv(v_pool, block_tables[r], length, g, block_size)
            for h in range(hq):
                if kv_head_of(h, num_q_heads, num_kv_heads) != g:
                    continue
                qq = bf16_bits_to_f64(q[cu[r]:cu[r] + s_len, h, :])
                logits = s64 * (qq @ kk.T)
                logits = np.where(allowed, logits, -np.inf)
                out[cu[r]:cu[r] + s_len, h, :] = _softmax_weighted_sum(logits, vv)
    return out


def prefill_paged_attn_rows(q, k_pool, v_pool, block_tables, prefix_lens, cu_q_lens,
                            num_q_heads, num_kv_heads, scale, samples, block_size=16,
                            rows_per_product=1024):
    """Float64 output rows for sampled ``(r, h, i)`` triples, shape ``[n, D]``.

    Row ``(r, h, i)`` is query head ``h`` of suffix token ``i`` of invocation
    ``r``, i.e. output row ``cu_q_lens[r] + i``; it attends over keys
    ``0 .. P_r + i`` of its invocation (the same definition as
    ``prefill_paged_attn``), so this serves workloads too large for the full
    oracle.  The samples are grouped by (invocation, KV head): each group's
    K/V are gathered once and its rows' logits come from one product with
    the group's stacked queries (at most ``rows_per_product`` rows at a time),
    each row masked to its own visible keys.
    """
    cu = np.asarray(cu_q_lens, dtype=np.int64)
    pl = np.asarray(prefix_lens, dtype=np.int64)
    s64 = _scale64(scale)
    d = q.shape[-1]
    res = np.zeros((len(samples), d), dtype=np.float64)
    groups = {}
    for n, (r, h, i) in enumerate(samples):
        r, h, i = int(r), int(h), int(i)
        assert 0 <= i < int(cu[r + 1] - cu[r])
        g = kv_head_of(h, num_q_heads, num_kv_heads)
        groups.setdefault(_kv_group_key(r, g), []).append((n, r, g, h, i))
    for members in groups.values():
        _, r, g, _, _ = members[0]
        p_len = int(pl[r])
        length = p_len + int(cu[r + 1] - cu[r])
        kk = gather_logical_kv(k_pool, block_tables[r], length, g, block_size)
        vv = gather_logical_kv(v_pool, block_tables[r], length, g, block_size)
        keys_j = np.arange(length)[None, :]
        for c0 in range(0, len(members), rows_per_product):
            part = members[c0:c0 + rows_per_product]
            qq = bf16_bits_to_f64(np.stack([q[packed_row(cu, r, i), h, :]
                                            for _, _, _, h, i in part]))
            nvis = np.array([visible_keys(p_len, i) for _, _, _, _, i in part])[:, None]
            logits = np.where(keys_j < nvis, s64 * (qq @ kk.T), -np.inf)
            out = _softmax_weighted_sum(logits, vv)
            for k, (n, _, _, _, _) in enumerate(part):
                res[n] = out[k]
    return res
