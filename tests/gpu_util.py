"""Helpers for the GPU tests: tolerances, sampling and comparison against the oracle."""

import numpy as np

import oracle

# float tolerance on bf16 outputs against the unrounded float64 oracle
MAX_ABS = 2e-2
MEAN_ABS = 2e-3


def bits_to_f64(bits):
    return oracle.bf16_bits_to_f64(bits)


def compare_full(got_bits, ref):
    """Max-abs / mean-abs error of a full bf16 output against the float64 oracle."""
    got = bits_to_f64(got_bits)
    assert got.shape == ref.shape
    assert np.isfinite(got).all(), "non-finite output"
    err = np.abs(got - ref)
    return float(err.max()), float(err.mean())


def sample_rows(wl, n_random, seed, edge=True, edge_all_heads=False):
    """(r, h, i) triples: random rows plus, per invocation, its first and last
    rows and the rows around block and 32-row tile boundaries (for one random
    query head each, or for every head with ``edge_all_heads``)."""
    rng = np.random.default_rng(seed)
    q_lens = wl.q_lens
    out = set()
    nonempty = [r for r in range(wl.batch) if q_lens[r] > 0]
    for _ in range(n_random):
        r = int(rng.choice(nonempty))
        out.add((r, int(rng.integers(wl.num_q_heads)), int(rng.integers(q_lens[r]))))
    if edge:
        for r in nonempty:
            s = int(q_lens[r])
            for i in {0, 1, 15, 16, 31, 32, 63, 64, s // 2, s - 2, s - 1}:
                if 0 <= i < s:
                    if edge_all_heads:
                        out.update((r, h, i) for h in range(wl.num_q_heads))
                    else:
                        out.add((r, int(rng.integers(wl.num_q_heads)), i))
    return sorted(out)


def compare_rows(wl, got_bits, samples, k_pool=None, v_pool=None):
    """Errors of sampled output rows against the oracle computed row by row."""
    kp = wl.k_pool if k_pool is None else k_pool
    vp = wl.v_pool if v_pool is None else v_pool
    ref = oracle.prefill_paged_attn_rows(wl.q, kp, vp, wl.block_tables,
                                         wl.prefix_lens, wl.cu_q_lens, wl.num_q_heads,
                                         wl.num_kv_heads, wl.scale, samples)
    cu = wl.cu_q_lens
    got = np.stack([bits_to_f64(got_bits[int(cu[r]) + i, h]) for r, h, i in samples])
    assert np.isfinite(got).all(), "non-finite output"
    err = np.abs(got - ref)
    return float(err.max()), float(err.mean())


BF16_QNAN, BF16_POS_INF = 0x7FC0, 0x7F80


def poison_tails(wl, bits=(BF16_QNAN, BF16_POS_INF)):
    """Fill the pool positions past the end of every sequence's last block
    (K and V, all heads) with NaN and Inf, alternating by position, where no
    sequence reads them as keys.  Returns the number of positions poisoned."""
    kv = wl.prefix_lens.astype(np.int64) + wl.q_lens.astype(np.int64)
    bs = wl.block_size
    # first position of each slot that some sequence reads as a key
    limit = {}
    for r in range(wl.batch):
        L = int(kv[r])
        for b in range(-(-L // bs)):
            slot = int(wl.block_tables[r, b])
            limit[slot] = max(limit.get(slot, 0), min(bs, L - b * bs))
    n = 0
    for slot, used in limit.items():
        for pos in range(used, bs):
            v = np.uint16(bits[pos % len(bits)])
            wl.k_pool[slot, :, pos, :] = v
            wl.v_pool[slot, :, pos, :] = v
            n += 1
    return n


def poison_slot_zero(wl, bits=BF16_QNAN):
    """Move whatever pool slot 0 holds to a slot no sequence reads, rename it
    in the block tables, and fill slot 0 with NaN (K and V, all heads): the
    kernels load slot 0 in place of blocks past a sequence's end, and those
    loads must stay masked (K) or zeroed (V).  Returns the slot used."""
    used = set(int(x) for r in range(wl.batch)
               for x in wl.block_tables[r, :-(-int(wl.prefix_lens[r] + wl.q_lens[r]) // wl.block_size)])
    free = [s for s in range(1, wl.num_blocks) if s not in used]
    assert free, "the pool needs a slot no sequence reads"
    u = free[0]
    for pool in (wl.k_pool, wl.v_pool):
        pool[u] = pool[0]
        pool[0] = np.uint16(bits)
    bt = wl.block_tables
    bt[bt == 0] = u
    return u

