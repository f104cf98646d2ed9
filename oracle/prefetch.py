"""Oracle of the KV prefetch (test infrastructure).

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s ``cpu_baseline``
may use this module.

The prefetch reloads an anchor's KV blocks from the CPU tier into free slots
of the GPU pool (arXiv 2608.14624: architecture figure of Sec. 3, reload from
external KV pools when present; Sec. 4, the CPU-offload connector and
LMCache).  A reloaded block must hold exactly the bytes a normal invocation
would have produced (Sec. 4), so the operation is a bit copy:
``pool'[dst[i]] = host[i]`` for every ``i < n`` and ``pool'[s] = pool[s]`` for
every slot ``s`` not named in ``dst``.
"""

import numpy as np


def kv_prefetch(host_k, host_v, dst_block_ids, k_pool, v_pool):
    """Return ``(k_pool', v_pool')`` after copying host blocks into their slots.

    ``host_k``/``host_v``: ``[n, Hkv, block_size, D]``; pools
    ``[num_blocks, Hkv, block_size, D]``; ``dst_block_ids``: ``[n]`` unique slot
    ids.  Arrays are copied, never modified in place; any dtype is handled as
    raw elements, so the copy is bitwise.
    """
    dst = np.asarray(dst_block_ids, dtype=np.int64)
    assert len(np.unique(dst)) == len(dst), "destination slots must be unique"
    k_new = np.array(k_pool, copy=True)
    v_new = np.array(v_pool, copy=True)
    for i, slot in enumerate(dst):
        k_new[slot] = host_k[i]
        v_new[slot] = host_v[i]
    return k_new, v_new
