"""Seeded synthetic workloads for paged prefix-reuse prefill attention.

This module only *builds inputs*: bf16 queries, the paged K/V pools, block
tables, lengths and the host-side prefetch buffers.  It contains no attention
arithmetic and no copy kernels, and it serves both the HIP path (through the
Python binding) and the CPU oracle (through the tests), which otherwise share
no code.

Shapes follow the paper's setting (arXiv 2608.14624):

* agents with a fixed reusable prompt prefix, the "agent anchor" (Sec. 2.1),
  making up roughly half of the prompt tokens (Sec. 1 reports 53-62%) and
  reused by every invocation of that agent (Sec. 2.2);
* 16-token KV blocks in a paged pool (Sec. 2.1, vLLM's default);
* the Llama-3.1-8B attention shape, 32 query / 8 KV heads of dimension 128
  (Sec. 5 setup), plus a 64/8 shape for a 70B-class model;
* on a prefix hit only the suffix queries run; a miss recomputes the whole
  prompt (prefix length 0);
* the predicted next agent's anchor blocks may sit in the CPU tier and are
  reloaded into free pool slots before use (Sec. 3.4, Sec. 4).

Values are N(0, 1) in bf16, stored as uint16 bit patterns, drawn by inverse
transform sampling: a uniform 16-bit integer ``u`` selects the bf16 value
(nearest-even) of the standard normal quantile at ``(u + 0.5) / 65536``.
bf16 itself has only 65536 codes, so this is a faithful N(0, 1) at bf16
resolution (tails clipped at +/-4.31), and about six times faster than
rounding float32 normal draws, which matters for the 3 GB configurations.
Every random stream is keyed by ``(seed, kind, index)`` so that an agent's
anchor content does not depend on how many invocations were drawn before
it.

Pool conventions:

* unreferenced slots hold bf16 NaN (0x7FC0), so any read of them shows up;
* positions past the end of a sequence inside its last block hold +/-29952
  (a large *finite* bf16), so a kernel that masks them correctly is not
  poisoned by ``0 * NaN`` while one that forgets the mask is visibly wrong;
* block-table entries past a sequence's last block point at a NaN slot;
* an agent's full anchor blocks are shared by all its hit invocations; the
  anchor's partial last block (``P mod 16`` tokens) is copied into a private
  block of each invocation, followed by its first suffix tokens.
"""

from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

BLOCK_SIZE = 16
BF16_NAN = np.uint16(0x7FC0)
# +29952 and -29952 in bf16: large and finite
BF16_TAIL_POS = np.uint16(0x46EA)
BF16_TAIL_NEG = np.uint16(0xC6EA)

# stream kinds for np.random.default_rng([seed, kind, index])
_K_SLOTS, _K_ANCHOR_KV, _K_ANCHOR_Q, _K_SUFFIX, _K_SPEC, _K_OFFPOOL = range(6)


def f32_to_bf16_bits(x):
    """Round float32 values to nearest-even bf16 and return the uint16 bit patterns.

    Inputs are finite (they are normal draws), so no NaN handling is needed.
    """
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


_NORMAL_TABLE = None


def normal_bf16_table():
    """bf16 codes of the N(0, 1) quantiles at the midpoints of 65536 equal bins."""
    global _NORMAL_TABLE
    if _NORMAL_TABLE is None:
        from scipy.special import ndtri
        mid = (np.arange(65536, dtype=np.float64) + 0.5) / 65536.0
        _NORMAL_TABLE = f32_to_bf16_bits(ndtri(mid).astype(np.float32))
    return _NORMAL_TABLE


def _normal_bf16(rng, shape):
    n = int(np.prod(shape))
    codes = rng.integers(0, 65536, size=n, dtype=np.uint16)
    out = np.empty(n, dtype=np.uint16)
    table = normal_bf16_table()
    step = 1 << 20        # bounded index temporaries
    for a in range(0, n, step):
        np.take(table, codes[a:a + step], out=out[a:a + step])
    return out.reshape(shape)


@dataclass
class Invocation:
    """One agent invocation: its agent, its suffix length and hit/miss."""
    agent: int
    suffix_len: int
    hit: bool = True
    # invocations with the same key get the same suffix tokens (Q, K, V)
    suffix_key: Optional[int] = None


@dataclass
class Workload:
    name: str
    seed: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    block_size: int
    scale: float                      # a float32 value held as a Python float
    anchor_lens: List[int]
    invocations: List[Invocation]
    q: np.ndarray                     # uint16 [total_q, Hq, D]
    k_pool: np.ndarray                # uint16 [num_blocks, Hkv, bs, D]
    v_pool: np.ndarray
    block_tables: np.ndarray          # int32 [B, max_blocks_per_seq]
    prefix_lens: np.ndarray           # int32 [B]
    cu_q_lens: np.ndarray             # int32 [B + 1]
    # blocks that start in the CPU tier (pool slot still NaN) and their sources
    host_k: Optional[np.ndarray] = None   # uint16 [n, Hkv, bs, D]
    host_v: Optional[np.ndarray] = None
    prefetch_dst: Optional[np.ndarray] = None    # int32 [n]
    prefetch_agent: Optional[np.ndarray] = None  # int32 [n]
    q_gain: float = 1.0
    meta: dict = field(default_factory=dict)

    # -- sizes the C ABI takes as host integers -------------------------
    @property
    def batch(self):
        return len(self.invocations)

    @property
    def total_q(self):
        return int(self.cu_q_lens[-1])

    @property
    def q_lens(self):
        return np.diff(self.cu_q_lens.astype(np.int64))

    @property
    def kv_lens(self):
        return self.prefix_lens.astype(np.int64) + self.q_lens

    @property
    def max_q_len(self):
        return int(self.q_lens.max()) if self.batch else 0

    @property
    def max_kv_len(self):
        return int(self.kv_lens.max()) if self.batch else 0

    @property
    def max_blocks_per_seq(self):
        return int(self.block_tables.shape[1])

    @property
    def num_blocks(self):
        return int(self.k_pool.shape[0])

    def pairs(self):
        """Visible (query, key) pairs per query head: sum_r S_r*P_r + S_r(S_r+1)/2."""
        s = self.q_lens
        p = self.prefix_lens.astype(np.int64)
        return int(np.sum(s * p + s * (s + 1) // 2))

    def flops(self):
        """Algorithmic FLOP of the attention: 4 * D * Hq * pairs (QK^T and PV)."""
        return 4 * self.head_dim * self.num_q_heads * self.pairs()

    def prefetch_bytes(self):
        if self.prefetch_dst is None:
            return 0
        return int(self.host_k.nbytes + self.host_v.nbytes)

    # -- logical (unpaged) content, regenerated from the seeds ----------
    def logical_sequence(self, r):
        """Unpaged ``(q [S, Hq, D], k [L, Hkv, D], v [L, Hkv, D])`` of invocation r.

        For a hit, ``q`` holds the suffix queries and ``k``/``v`` the anchor
        followed by the suffix; for a miss ``q`` covers the whole prompt.
        """
        inv = self.invocations[r]
        ak, av, aq = _anchor_content(self, inv.agent, need_q=not inv.hit)
        sq, sk, sv = _suffix_content(self, inv)
        k = np.concatenate([ak, sk], axis=0)
        v = np.concatenate([av, sv], axis=0)
        q = sq if inv.hit else np.concatenate([aq, sq], axis=0)
        return _apply_gain(q, self.q_gain), k, v


def _apply_gain(q_bits, gain):
    if gain == 1.0:
        return q_bits
    as_f32 = (q_bits.astype(np.uint32) << np.uint32(16)).view(np.float32)
    return f32_to_bf16_bits(as_f32 * np.float32(gain))


def _anchor_content(wl, a, need_q):
    rng = np.random.default_rng([wl.seed, _K_ANCHOR_KV, a])
    p = wl.anchor_lens[a]
    k = _normal_bf16(rng, (p, wl.num_kv_heads, wl.head_dim))
    v = _normal_bf16(rng, (p, wl.num_kv_heads, wl.head_dim))
    q = None
    if need_q:
        rq = np.random.default_rng([wl.seed, _K_ANCHOR_Q, a])
        q = _normal_bf16(rq, (p, wl.num_q_heads, wl.head_dim))
    return k, v, q


def _suffix_content(wl, inv):
    rng = np.random.default_rng([wl.seed, _K_SUFFIX, inv.suffix_key])
    s = inv.suffix_len
    k = _normal_bf16(rng, (s, wl.num_kv_heads, wl.head_dim))
    v = _normal_bf16(rng, (s, wl.num_kv_heads, wl.head_dim))
    q = _normal_bf16(rng, (s, wl.num_q_heads, wl.head_dim))
    return q, k, v


def build_workload(name, seed, anchor_lens, invocations, num_q_heads, num_kv_heads,
                   head_dim, num_blocks=None, occupancy=None, offpool_per_agent=0,
                   scale=None, q_gain=1.0):
    """Build pools, tables and queries for the given agents and invocations.

    ``num_blocks`` fixes the pool size; otherwise the pool is sized so the
    referenced blocks fill ``occupancy`` of it (at least one slot stays free).
    ``offpool_per_agent`` anchor blocks of every agent with a hit are left out
    of the pool (their slots stay NaN) and returned as prefetch sources.
    ``q_gain`` multiplies the queries before rounding (peaky softmax tests).
    """
    bs = BLOCK_SIZE
    invs = []
    for idx, inv in enumerate(invocations):
        key = idx if inv.suffix_key is None else inv.suffix_key
        invs.append(Invocation(inv.agent, int(inv.suffix_len), bool(inv.hit), key))
    n_agents = len(anchor_lens)
    hit_agents = sorted({inv.agent for inv in invs if inv.hit})

    # logical layout: which logical blocks each sequence has and which are shared
    shared_blocks = {a: anchor_lens[a] // bs for a in hit_agents}
    seq_len, pre_len, q_len, private_from = [], [], [], []
    for inv in invs:
        p_a = anchor_lens[inv.agent]
        total = p_a + inv.suffix_len
        seq_len.append(total)
        if inv.hit:
            pre_len.append(p_a)
            q_len.append(inv.suffix_len)
            private_from.append(shared_blocks[inv.agent])
        else:
            pre_len.append(0)
            q_len.append(total)
            private_from.append(0)
    n_blocks_seq = [-(-t // bs) for t in seq_len]
    used = sum(shared_blocks.values()) + sum(n - f for n, f in zip(n_blocks_seq, private_from))
    if num_blocks is None:
        occ = 0.9 if occupancy is None else occupancy
        num_blocks = max(int(np.ceil(used / occ)), used + 1)
    if used + 1 > num_blocks:
        raise ValueError(f"pool of {num_blocks} blocks cannot hold {used} blocks plus a free slot")

    slots = np.random.default_rng([seed, _K_SLOTS]).permutation(num_blocks).astype(np.int32)
    cursor = 0
    agent_slots = {}
    for a in hit_agents:
        agent_slots[a] = slots[cursor:cursor + shared_blocks[a]]
        cursor += shared_blocks[a]
    inv_slots = []
    for n, f in zip(n_blocks_seq, private_from):
        inv_slots.append(slots[cursor:cursor + (n - f)])
        cursor += n - f
    free_slot = int(slots[cursor])

    hkv, hq, d = num_kv_heads, num_q_heads, head_dim
    k_pool = np.full((num_blocks, hkv, bs, d), BF16_NAN, dtype=np.uint16)
    v_pool = np.full((num_blocks, hkv, bs, d), BF16_NAN, dtype=np.uint16)
    max_blocks = max(n_blocks_seq) if invs else 1
    block_tables = np.full((len(invs), max_blocks), free_slot, dtype=np.int32)

    if scale is None:
        scale = float(np.float32(1.0 / np.sqrt(head_dim)))
    wl = Workload(name=name, seed=seed, num_q_heads=hq, num_kv_heads=hkv, head_dim=d,
                  block_size=bs, scale=float(np.float32(scale)),
                  anchor_lens=list(anchor_lens), invocations=invs,
                  q=np.zeros((0, hq, d), np.uint16), k_pool=k_pool, v_pool=v_pool,
                  block_tables=block_tables,
                  prefix_lens=np.asarray(pre_len, dtype=np.int32),
                  cu_q_lens=np.concatenate([[0], np.cumsum(q_len)]).astype(np.int32))

    def blocked(x, n_blk):
        # [T, H, D] -> [n_blk, H, bs, D] with poisoned tail positions
        t = x.shape[0]
        buf = np.empty((n_blk * bs, x.shape[1], d), dtype=np.uint16)
        buf[:t] = x
        tail = np.arange(n_blk * bs - t)
        buf[t:] = np.where(tail % 2 == 0, BF16_TAIL_POS, BF16_TAIL_NEG)[:, None, None]
        return buf.reshape(n_blk, bs, x.shape[1], d).transpose(0, 2, 1, 3)

    # shared anchor blocks (and the CPU-tier copies of the off-pool ones)
    anchors = {}
    off_k, off_v, off_dst, off_agent = [], [], [], []
    for a in hit_agents:
        ak, av, _ = _anchor_content(wl, a, need_q=False)
        anchors[a] = (ak, av)
        nf = shared_blocks[a]
        if nf == 0:
            continue
        kb = blocked(ak[:nf * bs], nf)
        vb = blocked(av[:nf * bs], nf)
        resident = np.ones(nf, dtype=bool)
        if offpool_per_agent:
            pick = np.random.default_rng([seed, _K_OFFPOOL, a]).choice(
                nf, size=min(offpool_per_agent, nf), replace=False)
            pick.sort()
            resident[pick] = False
            off_k.append(kb[pick])
            off_v.append(vb[pick])
            off_dst.append(agent_slots[a][pick])
            off_agent.append(np.full(len(pick), a, dtype=np.int32))
        k_pool[agent_slots[a][resident]] = kb[resident]
        v_pool[agent_slots[a][resident]] = vb[resident]

    # per-invocation private blocks and queries, written in place
    anchor_q = {}
    cu_all = wl.cu_q_lens.astype(np.int64)
    q_all = np.empty((int(cu_all[-1]), hq, d), dtype=np.uint16)
    for r, inv in enumerate(invs):
        sq, sk, sv = _suffix_content(wl, inv)
        if inv.agent not in anchors:
            ak, av, _ = _anchor_content(wl, inv.agent, need_q=False)
            anchors[inv.agent] = (ak, av)
        ak, av = anchors[inv.agent]
        f = private_from[r]
        n = n_blocks_seq[r]
        kk = np.concatenate([ak[f * bs:], sk], axis=0)
        vv = np.concatenate([av[f * bs:], sv], axis=0)
        k_pool[inv_slots[r]] = blocked(kk, n - f)
        v_pool[inv_slots[r]] = blocked(vv, n - f)
        if f:
            block_tables[r, :f] = agent_slots[inv.agent]
        block_tables[r, f:n] = inv_slots[r]
        c0, c1 = int(cu_all[r]), int(cu_all[r + 1])
        if inv.hit:
            q_all[c0:c1] = sq
        else:
            if inv.agent not in anchor_q:
                rq = np.random.default_rng([seed, _K_ANCHOR_Q, inv.agent])
                anchor_q[inv.agent] = _normal_bf16(rq, (anchor_lens[inv.agent], hq, d))
            pa = anchor_lens[inv.agent]
            q_all[c0:c0 + pa] = anchor_q[inv.agent]
            q_all[c0 + pa:c1] = sq
    wl.q = q_all
    wl.q_gain = float(q_gain)
    wl.q = _apply_gain(wl.q, wl.q_gain)
    if off_dst:
        wl.host_k = np.ascontiguousarray(np.concatenate(off_k))
        wl.host_v = np.ascontiguousarray(np.concatenate(off_v))
        wl.prefetch_dst = np.concatenate(off_dst).astype(np.int32)
        wl.prefetch_agent = np.concatenate(off_agent)
    wl.meta = {"used_blocks": int(used), "free_slot": free_slot,
               "anchor_share": _anchor_share(anchor_lens, invs)}
    return wl


def _anchor_share(anchor_lens, invs):
    """Fraction of prompt tokens that belong to the agent anchors."""
    anchor = sum(anchor_lens[i.agent] for i in invs)
    total = sum(anchor_lens[i.agent] + i.suffix_len for i in invs)
    return anchor / total if total else 0.0


# --------------------------------------------------------------------------
# The named configurations
# --------------------------------------------------------------------------

CONFIG_NAMES = ("tiny", "llama8b", "agent_batch", "llama70b_prefetch", "long_mixed",
                "decode_batch", "decode_private", "llama70b_prefetch_tp8", "agent_batch_tp8")

# one GPU's shard of a configuration split 8 ways by KV head (tensor
# parallelism): the same invocations with Hq / 8 query and Hkv / 8 KV heads
_TP8_OF = {"llama70b_prefetch_tp8": "llama70b_prefetch", "agent_batch_tp8": "agent_batch"}


def config_spec(name):
    """Agents, invocations and shapes of a named configuration (no arrays)."""
    if name in _TP8_OF:
        spec = config_spec(_TP8_OF[name])
        spec["num_q_heads"] //= 8
        spec["num_kv_heads"] //= 8
        return spec
    if name == "tiny":
        # 1 request: 256-token cached prefix + 64-token suffix, 8/2 heads, D=64,
        # pool of 64 blocks, scale 1/sqrt(64)
        return dict(seed=0, anchor_lens=[256], invocations=[Invocation(0, 64)],
                    num_q_heads=8, num_kv_heads=2, head_dim=64, num_blocks=64, scale=0.125)
    if name == "llama8b":
        # Llama-3-8B attention shape: prefix 2048 + suffix 1024, pool of 16384 blocks
        return dict(seed=1, anchor_lens=[2048], invocations=[Invocation(0, 1024)],
                    num_q_heads=32, num_kv_heads=8, head_dim=128, num_blocks=16384)
    if name == "agent_batch":
        # 32 invocations over 4 agents, anchors U[1536, 3072], suffixes U[256, 2048]
        rng = np.random.default_rng([2, _K_SPEC])
        anchors = [int(x) for x in rng.integers(1536, 3072, size=4, endpoint=True)]
        agents = rng.integers(0, 4, size=32)
        sfx = rng.integers(256, 2048, size=32, endpoint=True)
        invs = [Invocation(int(a), int(s)) for a, s in zip(agents, sfx)]
        return dict(seed=2, anchor_lens=anchors, invocations=invs,
                    num_q_heads=32, num_kv_heads=8, head_dim=128, num_blocks=16384)
    if name == "llama70b_prefetch":
        # 16 invocations over 4 agents, 64/8 heads, prefix 4096 + suffix 512;
        # 64 of each agent's 256 anchor blocks start in the CPU tier.
        # Invocations are packed grouped by agent (dispatch order), so that
        # each agent's batch is a contiguous slice of the queries.
        rng = np.random.default_rng([3, _K_SPEC])
        agents = sorted(int(a) for a in rng.integers(0, 4, size=16))
        invs = [Invocation(a, 512) for a in agents]
        return dict(seed=3, anchor_lens=[4096] * 4, invocations=invs,
                    num_q_heads=64, num_kv_heads=8, head_dim=128, num_blocks=16384,
                    offpool_per_agent=64)
    if name == "long_mixed":
        # 128 invocations over 8 agents, anchors U[4096, 8192], suffix lengths
        # lognormal (median 512, sigma 1) clipped to [128, 4096]; 77 hits and
        # 51 misses; pool at 90% occupancy
        rng = np.random.default_rng([4, _K_SPEC])
        anchors = [int(x) for x in rng.integers(4096, 8192, size=8, endpoint=True)]
        agents = rng.integers(0, 8, size=128)
        sfx = np.clip(np.rint(rng.lognormal(np.log(512.0), 1.0, size=128)), 128, 4096)
        hits = np.array([True] * 77 + [False] * 51)
        rng.shuffle(hits)
        invs = [Invocation(int(a), int(s), bool(h)) for a, s, h in zip(agents, sfx, hits)]
        return dict(seed=4, anchor_lens=anchors, invocations=invs,
                    num_q_heads=32, num_kv_heads=8, head_dim=128, occupancy=0.9)
    if name == "decode_batch":
        # decode after the agent turns: 128 sequences over 8 agents, each the
        # agent's anchor U[4096, 8192] + its own history (lognormal, median
        # 512, clipped to [128, 4096]) ending in the token being decoded
        rng = np.random.default_rng([5, _K_SPEC])
        anchors = [int(x) for x in rng.integers(4096, 8192, size=8, endpoint=True)]
        agents = rng.integers(0, 8, size=128)
        hist = np.clip(np.rint(rng.lognormal(np.log(512.0), 1.0, size=128)), 128, 4096)
        invs = [Invocation(int(a), int(s)) for a, s in zip(agents, hist)]
        return dict(seed=5, anchor_lens=anchors, invocations=invs,
                    num_q_heads=32, num_kv_heads=8, head_dim=128, occupancy=0.9)
    if name == "decode_private":
        # the same length mix with nothing shared: 128 sequences, each its own
        # agent with an anchor U[4096, 8192] + history as in decode_batch, so
        # every key of every sequence is a distinct pool block
        rng = np.random.default_rng([6, _K_SPEC])
        anchors = [int(x) for x in rng.integers(4096, 8192, size=128, endpoint=True)]
        hist = np.clip(np.rint(rng.lognormal(np.log(512.0), 1.0, size=128)), 128, 4096)
        invs = [Invocation(a, int(s)) for a, s in enumerate(hist)]
        return dict(seed=6, anchor_lens=anchors, invocations=invs,
                    num_q_heads=32, num_kv_heads=8, head_dim=128, occupancy=0.9)
    raise KeyError(name)


def decode_view(wl):
    """The last suffix token of every invocation as a decode batch.

    Returns ``(q [B, Hq, D], seq_lens [B])``: row ``r`` is the query of the
    last prompt position of invocation ``r``, which sees all ``P_r + S_r``
    keys.  The pools and block tables of ``wl`` serve unchanged.
    """
    last = wl.cu_q_lens[1:].astype(np.int64) - 1
    assert np.all(wl.q_lens > 0), "every invocation needs a token to decode"
    return np.ascontiguousarray(wl.q[last]), wl.kv_lens.astype(np.int32)


def cascade_view(wl):
    """The decode batch of ``wl`` ordered for cascade attention.

    Sequences of an agent with a prefix hit share the anchor's full blocks
    (the same pool slots); they become one group whose shared length is those
    blocks' tokens.  Sequences without a hit form one last group sharing
    nothing.  Returns a dict with ``order`` (the batch permutation: row ``i``
    of the grouped batch is sequence ``order[i]``), ``cu_groups``,
    ``shared_lens``, ``max_group_seqs`` (over groups that share something, at
    least 1), ``max_shared_len`` and ``max_rest_len`` (the most keys of its
    own any sequence has beyond its group's shared part).
    """
    bs = wl.block_size
    by_agent = {}
    misses = []
    for r, inv in enumerate(wl.invocations):
        if inv.hit and wl.anchor_lens[inv.agent] >= bs:
            by_agent.setdefault(inv.agent, []).append(r)
        else:
            misses.append(r)
    order, cu, shared = [], [0], []
    for a in sorted(by_agent):
        order += by_agent[a]
        cu.append(len(order))
        shared.append(wl.anchor_lens[a] // bs * bs)
    if misses:
        order += misses
        cu.append(len(order))
        shared.append(0)
    sizes = [cu[i + 1] - cu[i] for i in range(len(shared)) if shared[i] > 0]
    kv = wl.kv_lens
    rest = [int(kv[order[k]]) - shared[gi] for gi in range(len(shared))
            for k in range(cu[gi], cu[gi + 1])]
    return dict(order=np.asarray(order, dtype=np.int64),
                cu_groups=np.asarray(cu, dtype=np.int32),
                shared_lens=np.asarray(shared, dtype=np.int32),
                max_group_seqs=max(sizes + [1]),
                max_shared_len=max(shared + [0]),
                max_rest_len=max(rest + [0]))


def make_config(name):
    """Build the named configuration's arrays."""
    spec = config_spec(name)
    seed = spec.pop("seed")
    anchors = spec.pop("anchor_lens")
    invs = spec.pop("invocations")
    return build_workload(name, seed, anchors, invs, **spec)
