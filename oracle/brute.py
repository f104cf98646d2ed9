"""Scalar brute force of prefix-hit attention (test infrastructure).

Only ``tests/`` may use this module; it exists to pin the NumPy oracle in
``paged_attention.py`` on tiny inputs.  It works on the *logical* token
arrays of one sequence (no pool, no block table, no NumPy): plain Python
floats, ``math.exp`` and correctly rounded sums (``math.fsum``).

Definition followed (arXiv 2608.14624, Sec. 2.1 "Prefix caching": a hit
reuses the prefix KV, so its output equals recomputing the whole prompt):
suffix row ``i`` sits at prompt position ``P + i`` and its output is the
softmax-weighted mean of the values of keys ``0 .. P + i``, with logits
``scale * <q_i, k_j>``.
"""

import math


def brute_attention_rows(q_rows, keys, values, prefix_len, scale):
    """Attention output of every suffix row, as lists of Python floats.

    ``q_rows``  : S rows of D floats (the suffix queries of one head).
    ``keys``    : L = P + S rows of D floats (prefix keys, then suffix keys).
    ``values``  : L rows of D floats.
    ``prefix_len``: P.  ``scale``: a Python float.
    """
    out = []
    for i, qv in enumerate(q_rows):
        n_visible = prefix_len + i + 1
        logits = []
        for j in range(n_visible):
            logits.append(scale * math.fsum(qv[d] * keys[j][d] for d in range(len(qv))))
        top = max(logits)
        weights = [math.exp(x - top) for x in logits]
        denom = math.fsum(weights)
        row = []
        for d in range(len(values[0])):
            row.append(math.fsum(weights[j] * values[j][d] for j in range(n_visible)) / denom)
        out.append(row)
    return out
