"""CPU oracle for the paged prefix-reuse prefill attention and the KV prefetch.

TEST INFRASTRUCTURE ONLY.  Nothing here is part of the product path.  Only the
test suite (``tests/``), ``__graft_entry__.smoke()`` and the ``cpu_baseline``
leg of ``bench.py`` may import, call or run anything in this package.  The HIP
library and its Python binding never import it, and this package imports
nothing from them: the two sides share no kernels, helpers, tables or
constants.  Inputs reach both sides from the seeded generator
``paper_2608_14624_amd.workload``, which contains none of the arithmetic
below.

What the paper fixes, and what this package therefore computes
(arXiv 2608.14624, "Learning Agent Execution for KV-Cache Management in
Agentic Serving"):

* Sec. 2.1 (Background, "Prefix caching"): a request whose prompt shares a
  prefix with an earlier one reuses that prefix's KV tensors instead of
  recomputing them; vLLM keeps them in 16-token blocks.  Reuse is exact, so a
  prefix hit must produce the same attention output as a full recompute of
  the whole prompt.
* Sec. 3.4 and Sec. 4: the warmup of a predicted agent yields the same KV
  blocks as a normal invocation, the attention kernels are unchanged, and the
  anchor is reloaded from the CPU / external KV tier when it is present
  there (the architecture figure of Sec. 3).  Reload is a byte copy of whole
  blocks into pool slots.

The paper states nothing about the attention arithmetic itself, so the
attention oracle is the plain definition of scaled dot-product attention with
a causal mask aligned to the end of the prompt, evaluated in float64
(``paged_attention.py``), pinned by a scalar brute force (``brute.py``) and by
the invariants and closed forms in ``tests/test_oracle_*.py``.  The prefetch
oracle is a NumPy scatter (``prefetch.py``); the write-back of new tokens'
K/V through a slot mapping and the offload of blocks to the CPU tier are
NumPy scatters and gathers too (``kv_copy.py``).

The host-side control plane (Sec. 3.2-3.4, Eq. (2)-(11), the runtime
workflow algorithm) is plain Python in ``control_plane.py``, pinned by hand
values, closed forms, breadth-first distances against all-pairs shortest
paths, the exact survival probability by path enumeration, and planted
mistakes (``tests/test_control_plane_oracle.py``).

Every function here is pinned; none is "parity unpinned".  The full
attention oracle is pinned by the brute force, the invariants, the closed
forms and the golden case (``tests/test_oracle_*.py``); the row-by-row
oracle ``prefill_paged_attn_rows`` is pinned to the full oracle on shuffled
varlen samples, with planted indexing and grouping mistakes
(``tests/test_oracle_rows.py``); the copies by round trips and per-slot
checks; the control plane as listed above.
"""

from .paged_attention import (  # noqa: F401
    bf16_bits_to_f64,
    gather_logical_kv,
    kv_head_of,
    prefill_paged_attn,
    prefill_paged_attn_rows,
    visible_keys,
)
from .prefetch import kv_prefetch  # noqa: F401
from .kv_copy import kv_offload, kv_write  # noqa: F401
from .brute import brute_attention_rows  # noqa: F401
