"""Device-resident workloads and the prefetch/attention stream pipeline.

``DeviceWorkload`` moves a generated workload into GPU memory (PyTorch
tensors: bf16 pools and queries, int32 metadata) and its CPU-tier blocks into
pinned host memory.  ``AgentPipeline`` runs the serving order of the paper's
background prefetch (arXiv 2608.14624, Sec. 3.4: while the current agent is
served, the anchor of the predicted next agent, Eq. (10), is brought in off
the critical path): for each agent in dispatch order,

    side stream : wait until the target's last attention has finished,
                  cs_kv_prefetch(target agent's CPU-tier blocks), record event
    main stream : cs_prefill_paged_attn(this agent's invocations)
    main stream : wait for the event before the next agent's attention

The target is the next agent in dispatch order (the known-order protocol),
or, with a :class:`ScoutPolicy`, the control plane's between-step decision
(Eq. (10)-(11)); a wrong or withheld prediction is a miss, and the next
agent's blocks are then brought in on the main stream, on the critical path.
A prefetch rewrites only its target's slots, after the target's last reader
has finished, so the attention in flight never sees a slot being written.
Only the C calls do work; this module orders them.
"""

import hashlib

import numpy as np
import torch

from . import ops


def _to_device_bf16(bits, device):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).to(device)


def _to_pinned_bf16(bits):
    src = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16)
    dst = torch.empty(src.shape, dtype=torch.bfloat16, pin_memory=True)
    dst.copy_(src)
    return dst


def _i32(x, device):
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.int32)).to(device)


class SubBatch:
    """Invocations ``[lo, hi)`` of a workload as their own attention call."""

    def __init__(self, dw, lo, hi):
        wl = dw.wl
        cu = wl.cu_q_lens.astype(np.int64)
        self.lo, self.hi = lo, hi
        self.q0, self.q1 = int(cu[lo]), int(cu[hi])
        self.q = dw.q[self.q0:self.q1]
        self.out = dw.out[self.q0:self.q1]
        self.block_tables = dw.block_tables[lo:hi]
        self.prefix_lens = dw.prefix_lens[lo:hi]
        self.cu_q_lens = _i32(cu[lo:hi + 1] - cu[lo], dw.device)
        qlens = np.diff(cu[lo:hi + 1])
        kvlens = qlens + wl.prefix_lens[lo:hi].astype(np.int64)
        self.max_q_len = int(qlens.max()) if hi > lo else 0
        self.max_kv_len = int(kvlens.max()) if hi > lo else 0
        self.flops = 4 * wl.head_dim * wl.num_q_heads * int(
            np.sum(qlens * wl.prefix_lens[lo:hi] + qlens * (qlens + 1) // 2))
        self.dw = dw
        self._call = None
        if hi > lo:
            self._call = ops.PrefillCall(self.q, dw.k_pool, dw.v_pool, self.block_tables,
                                         self.prefix_lens, self.cu_q_lens, self.out,
                                         max_q_len=self.max_q_len, max_kv_len=self.max_kv_len,
                                         scale=wl.scale, workspace=dw.workspace)

    def attention(self, stream=None):
        if self._call is not None:
            self._call(stream)


class DeviceWorkload:
    """GPU copies of a :class:`~paper_2608_14624_amd.workload.Workload`."""

    def __init__(self, wl, device="cuda:0", workspace=None):
        """``workspace``: None for the plain attention call, "auto" for the
        call with a workspace (allocated per launch shape when it splits
        small launches' keys over more work-groups)."""
        self.wl = wl
        self.workspace = workspace
        self.device = torch.device(device)
        self.q = _to_device_bf16(wl.q, self.device)
        self.k_pool = _to_device_bf16(wl.k_pool, self.device)
        self.v_pool = _to_device_bf16(wl.v_pool, self.device)
        self.block_tables = _i32(wl.block_tables, self.device)
        self.prefix_lens = _i32(wl.prefix_lens, self.device)
        self.cu_q_lens = _i32(wl.cu_q_lens, self.device)
        self.out = torch.empty_like(self.q)
        self._call = ops.PrefillCall(self.q, self.k_pool, self.v_pool, self.block_tables,
                                     self.prefix_lens, self.cu_q_lens, self.out,
                                     max_q_len=wl.max_q_len, max_kv_len=wl.max_kv_len,
                                     scale=wl.scale, workspace=workspace)
        self.host_k = self.host_v = self.prefetch_dst = None
        if wl.prefetch_dst is not None:
            self.host_k = _to_pinned_bf16(wl.host_k)
            self.host_v = _to_pinned_bf16(wl.host_v)
            self.prefetch_dst = _i32(wl.prefetch_dst, self.device)

    def attention(self, stream=None, out=None):
        if out is None:
            self._call(stream)
            return
        wl = self.wl
        ops.cs_prefill_paged_attn(self.q, self.k_pool, self.v_pool, self.block_tables,
                                  self.prefix_lens, self.cu_q_lens, out,
                                  max_q_len=wl.max_q_len, max_kv_len=wl.max_kv_len,
                                  scale=wl.scale, workspace=self.workspace, stream=stream)

    def prefetch_all(self, stream=None):
        if self.prefetch_dst is None:
            return
        ops.cs_kv_prefetch(self.host_k, self.host_v, self.prefetch_dst, self.k_pool,
                           self.v_pool, stream=stream)

    def out_bits(self):
        """The output as uint16 bf16 bit patterns on the host."""
        return self.out.view(torch.int16).cpu().numpy().view(np.uint16)


def agent_fingerprint(block_ids):
    """64-bit fingerprint of an agent from its anchor's leading block ids (the
    block pool's prefix hashes play this role in a serving engine, Sec. 4)."""
    digest = hashlib.blake2b(np.ascontiguousarray(block_ids, dtype=np.int32).tobytes(),
                             digest_size=8).digest()
    return int.from_bytes(digest, "little")


class ScoutPolicy:
    """Prefetch targets from the control plane (cs_scout_*).

    Every turn reports the agent's prefix-block touches (the block pool's
    prefix match, one call per turn) and then asks the between-step decision
    for the agent to warm up next.  Host-only; usable without a GPU.
    """

    def __init__(self, wl, agents, **params):
        self.scout = ops.Scout(max(len(agents), 1), wl.num_blocks, **params)
        self.ids, self.by_id, self.touches = {}, {}, {}
        for a in agents:
            invs = [r for r, inv in enumerate(wl.invocations) if inv.agent == a]
            blocks, tokens = [], []
            for r in invs:
                p = int(wl.prefix_lens[r])
                nb = -(-p // 16)
                blocks.append(wl.block_tables[r, :nb])
                tokens.append(np.minimum(16, p - 16 * np.arange(nb)))
            blocks = np.concatenate(blocks) if blocks else np.zeros(0, np.int32)
            tokens = np.concatenate(tokens) if tokens else np.zeros(0, np.int32)
            blocks, first = np.unique(blocks, return_index=True)
            lead = wl.block_tables[invs[0], :4] if invs else np.zeros(0, np.int32)
            aid = self.scout.agent_id(agent_fingerprint(lead))
            if aid in self.by_id:
                raise ValueError(f"agents {self.by_id[aid]} and {a} share a fingerprint")
            self.ids[a], self.by_id[aid] = aid, a
            self.touches[a] = (blocks.astype(np.int32), tokens[first].astype(np.int32))
        self.now = 0

    def on_turn(self, a):
        """Record agent ``a``'s turn; return the agent to prefetch, or None."""
        blocks, tokens = self.touches[a]
        n = len(blocks)     # an agent with no cached prefix touches nothing
        self.scout.observe_touches(blocks, np.full(n, self.ids[a], np.int32), tokens,
                                   np.full(n, self.now, np.int64))
        self.now += 1
        t = self.scout.between_step()
        return None if t is None else self.by_id.get(t)


class AgentPipeline:
    """Per-agent attention with a prefetch overlapped on a side stream.

    Requires the invocations to be packed grouped by agent (each agent's
    invocations contiguous) and at least two agents.  ``policy``: None for the
    known dispatch order, or a :class:`ScoutPolicy`.  ``overlap`` (known order
    only): consecutive agents' attention launches alternate between the
    current stream and a second one, so that one launch's last round can run
    beside the next launch's first; each still waits only for its own
    prefetch, and the pass ends on the current stream.
    """

    def __init__(self, dw, side_stream=None, policy=None, overlap=False):
        wl = dw.wl
        agents = [inv.agent for inv in wl.invocations]
        order = []
        for a in agents:
            if not order or order[-1] != a:
                order.append(a)
        if len(order) != len(set(order)):
            raise ValueError("invocations must be grouped by agent")
        if len(order) < 2:
            raise ValueError("the pipeline needs at least two agents")
        self.dw = dw
        self.agents = order
        self.policy = policy
        self.batches = []
        lo = 0
        for a in order:
            hi = lo
            while hi < len(agents) and agents[hi] == a:
                hi += 1
            self.batches.append(SubBatch(dw, lo, hi))
            lo = hi
        # each agent's CPU-tier blocks, as contiguous pinned slices
        self.prefetch = {}
        if dw.prefetch_dst is not None:
            pa = wl.prefetch_agent
            for a in order:
                idx = np.nonzero(pa == a)[0]
                if len(idx) == 0:
                    continue
                i0, i1 = int(idx[0]), int(idx[-1]) + 1
                assert i1 - i0 == len(idx), "prefetch blocks must be grouped by agent"
                self.prefetch[a] = (dw.host_k[i0:i1], dw.host_v[i0:i1], dw.prefetch_dst[i0:i1])
        self.side = side_stream if side_stream is not None else torch.cuda.Stream(dw.device)
        self.overlap = overlap and policy is None
        self.alt = torch.cuda.Stream(dw.device) if self.overlap else None
        self.events = {a: torch.cuda.Event() for a in order}       # prefetch done
        self.attn_done = {a: torch.cuda.Event() for a in order}    # last reader done
        # known order only: the previous pass ended / the first agent's
        # attention of this pass is done (the only readers a prefetch can race)
        self.pass_done = torch.cuda.Event()
        self.first_done = torch.cuda.Event()
        self.flops = sum(b.flops for b in self.batches)
        self.prefetch_bytes = sum(int(k.numel() * 2 + v.numel() * 2)
                                  for k, v, _ in self.prefetch.values())
        self.hits = self.misses = 0

    def prefetch_agent(self, a, stream):
        if a in self.prefetch:
            hk, hv, dst = self.prefetch[a]
            ops.cs_kv_prefetch(hk, hv, dst, self.dw.k_pool, self.dw.v_pool, stream=stream)

    def stage_first(self):
        """Bring the first agent's blocks in before the loop starts."""
        main = torch.cuda.current_stream(self.dw.device)
        self.prefetch_agent(self.agents[0], main)

    def step(self, timing=None):
        """One pass over all agents; each turn's prefetch overlaps its attention.

        With the known order the last turn prefetches the first agent again
        (for the next pass), so every pass moves every agent's CPU-tier blocks
        once.  ``timing``: optional per-turn ``((p0, p1), (a0, a1))`` timing
        events recorded around the side-stream prefetch and the attention.
        """
        main = torch.cuda.current_stream(self.dw.device)
        n = len(self.agents)
        known = self.policy is None

        def turn_stream(t):
            return self.alt if self.overlap and t % 2 == 1 else main

        if self.overlap:
            self.alt.wait_stream(main)      # work enqueued before this pass
        for k, a in enumerate(self.agents):
            s_k = turn_stream(k)
            nxt = self.agents[(k + 1) % n]
            target = nxt if known else self.policy.on_turn(a)
            (p0, p1), (a0, a1) = timing[k] if timing is not None else ((None, None),) * 2
            if target is not None and target != a:
                # wait for the last attention that read the target's slots.
                # Known order: for turns 0 .. n-2 that was in the previous
                # pass (one wait at turn 0 covers them); the last turn's
                # target is the first agent, read at turn 0 of this pass.
                # Two cross-stream events per pass instead of one per turn.
                if not known:
                    self.side.wait_event(self.attn_done[target])
                elif k == 0:
                    self.side.wait_event(self.pass_done)
                elif k == n - 1:
                    self.side.wait_event(self.first_done)
                with torch.cuda.stream(self.side):
                    if p0 is not None:
                        p0.record(self.side)
                    self.prefetch_agent(target, self.side)
                    if p1 is not None:
                        p1.record(self.side)
                    self.events[target].record(self.side)
            elif p0 is not None:
                # no prefetch this turn: an empty interval keeps the events recorded
                p0.record(self.side)
                p1.record(self.side)
            if a0 is not None:
                a0.record(s_k)
            self.batches[k].attention(stream=s_k)
            if a1 is not None:
                a1.record(s_k)
            if not known:
                self.attn_done[a].record(main)
            elif k == 0:
                self.first_done.record(s_k)
            if known and k == n - 1:
                if self.overlap:
                    main.wait_stream(self.alt)   # the pass ends with every launch
                self.pass_done.record(main)
            if target == nxt:
                self.hits += 1
                turn_stream((k + 1) % n).wait_event(self.events[nxt])
            else:
                # a miss: the next agent's blocks come in on the critical path
                # (after any side-stream write still in flight)
                self.misses += 1
                main.wait_stream(self.side)
                self.prefetch_agent(nxt, main)
