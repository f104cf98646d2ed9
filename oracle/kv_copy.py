"""Oracles of the KV write-back scatter and the KV offload (test infrastructure).

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s ``cpu_baseline``
leg may use this module.

* Write-back: the K/V that a forward pass produces for new prompt tokens is
  stored into the paged pool before attention reads it (arXiv 2608.14624,
  Sec. 2.1: prefill computes KV tensors for every prompt token and caches them
  in 16-token blocks; Sec. 4: a warmup produces the same KV blocks as a
  normal invocation).  Token ``t`` goes to slot ``s = slot_mapping[t]``: pool
  block ``s // block_size``, offset ``s % block_size``; a negative slot means
  the token is not stored.
* Offload: a block leaving the GPU pool is copied to the CPU tier (Sec. 4:
  eviction prefers blocks already resident in the CPU tier; the CPU-offload
  connector and LMCache hold them), the reverse of the prefetch.

Both are byte copies, so the oracles are NumPy scatters and gathers.
"""

import numpy as np


def kv_write(k_new, v_new, slot_mapping, k_pool, v_pool):
    """Return ``(k_pool', v_pool')`` with each new token written to its slot.

    ``k_new``/``v_new``: ``[T, Hkv, D]``; pools ``[NB, Hkv, bs, D]``;
    ``slot_mapping``: ``[T]`` ints, distinct among the non-negative entries.
    """
    k_out = np.array(k_pool, copy=True)
    v_out = np.array(v_pool, copy=True)
    bs = k_pool.shape[2]
    slots = np.asarray(slot_mapping, dtype=np.int64)
    used = slots[slots >= 0]
    assert len(np.unique(used)) == len(used), "slots must be distinct"
    for t, s in enumerate(slots):
        if s < 0:
            continue
        k_out[s // bs, :, s % bs, :] = k_new[t]
        v_out[s // bs, :, s % bs, :] = v_new[t]
    return k_out, v_out


def kv_offload(src_block_ids, k_pool, v_pool):
    """Return the host copies ``(host_k, host_v)`` ``[n, Hkv, bs, D]`` of the named blocks."""
    ids = np.asarray(src_block_ids, dtype=np.int64)
    return np.array(k_pool[ids], copy=True), np.array(v_pool[ids], copy=True)
