/*
 * cachescout.h - C ABI of libcachescout.so: paged prefix-reuse prefill
 * attention and KV prefetch for AMD Instinct MI355X (gfx950).
 *
 * The calls are the GPU work behind agent-aware KV-cache reuse (arXiv
 * 2608.14624, "Learning Agent Execution for KV-Cache Management in Agentic
 * Serving"):
 *
 *   cs_prefill_paged_attn  - an agent invocation that hits its cached prompt
 *                            prefix (the "agent anchor", Sec. 2.1) runs
 *                            attention for its new suffix tokens over the
 *                            anchor's KV, which sits in 16-token blocks of a
 *                            paged GPU pool (Sec. 2.1 "Prefix caching"), plus
 *                            the suffix's own causal KV.  A miss is the same
 *                            call with prefix length 0.
 *   cs_kv_prefetch         - the predicted next agent's anchor blocks
 *                            (Sec. 3.4, Eq. (10) picks that agent) are
 *                            reloaded from the CPU tier into free pool slots
 *                            (architecture figure of Sec. 3; Sec. 4), as a
 *                            bit-exact block copy.
 *   cs_kv_write            - the K/V of new tokens is stored into pool slots
 *                            through a slot mapping (the write that precedes
 *                            attention, Sec. 2.1 and Sec. 4).
 *   cs_kv_offload          - whole blocks are copied from the pool to the
 *                            CPU tier (Sec. 4), the reverse of the prefetch.
 *   cs_paged_decode_attn   - one new token per sequence attends over its whole
 *                            paged KV (the decode that follows a prefill).
 *   cs_cascade_decode_attn - the same decode with each agent's shared anchor
 *                            attended once for all of its sequences.
 *
 * Conventions shared by all calls
 *   - Every pointer is caller-owned.  The GPU calls allocate no device or
 *     host memory and keep no state beyond a per-process cache of device
 *     properties (the compute-unit count of each device, read once, which
 *     sizes the attention launch) and the fixed device array of
 *     cs_cascade_decode_attn_noalloc; they are reentrant and may run
 *     concurrently on different streams (except that allocation-free call,
 *     whose calls on one GPU share that array).
 *   - The attention launch orders its work-groups for MI355X's 8 XCDs
 *     (consecutive work-groups dealt round-robin to the XCDs, one L2 each);
 *     on a part with another XCD count the result is the same, only the L2
 *     reuse differs.  The control plane (cs_scout_*, at the end of this file) is
 *     host-only and owns the host memory behind its handle.
 *   - Every call enqueues its kernels on `stream` (NULL = the legacy default
 *     stream of the current device) and returns without synchronizing.  Device
 *     metadata is read by the kernels, never by the host, so the calls can be
 *     captured in a HIP graph (unless CS_DEBUG_CHECK=1, see below).
 *   - The device is the caller's current HIP device; every device pointer
 *     must belong to it.
 *   - bf16 means IEEE-754 binary32 truncated to its upper 16 bits (bfloat16),
 *     stored little-endian as 2 bytes.
 *   - Return value: CS_OK, or one of the error codes below.  Arguments are
 *     validated synchronously before anything is enqueued; on an error
 *     nothing is launched.  cs_last_error() gives a message for the calling
 *     thread's last failure.
 *   - Values that live in device memory (block ids, lengths) are NOT checked
 *     in normal operation; out-of-range or inconsistent values are undefined
 *     behaviour.  With the environment variable CS_DEBUG_CHECK=1 the library
 *     copies that metadata to the host, synchronizing the stream, and
 *     validates it first (CS_ERR_INVALID_ARG on a violation).
 */
#ifndef CACHESCOUT_H
#define CACHESCOUT_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* A HIP stream handle (hipStream_t) passed through as an opaque pointer. */
typedef struct ihipStream_t *cs_stream_t;

enum cs_status {
    CS_OK = 0,
    CS_ERR_INVALID_ARG = 1,  /* a null pointer, negative size, inconsistent
                                sizes, misaligned buffer, non-pinned host
                                buffer, or (debug mode) bad device metadata */
    CS_ERR_UNSUPPORTED = 2,  /* valid but not implemented: head_dim other
                                than 64 or 128, block_size other than 16,
                                more than 16 query heads per KV head (decode) */
    CS_ERR_HIP = 3           /* the HIP runtime reported an error */
};

/*
 * Paged prefill attention with a reused prefix (GQA, variable length).
 *
 * Operation (Sec. 2.1 "Prefix caching": a hit reuses the prefix KV instead
 * of recomputing it, so the result equals a full recompute): for every
 * invocation r < batch, query head h < num_q_heads, suffix row
 * i < S_r = cu_q_lens[r+1] - cu_q_lens[r] and feature d < head_dim,
 *
 *   P = prefix_lens[r],  g = h / (num_q_heads / num_kv_heads)
 *   K_r[j] = k_pool[block_tables[r][j / 16]][g][j % 16][:]   (V_r likewise)
 *   s_j    = scale * dot(q[cu_q_lens[r] + i][h][:], K_r[j])   for j <= P + i
 *   out[cu_q_lens[r] + i][h][d] = sum_j softmax(s)_j * V_r[j][d]
 *
 * i.e. suffix row i is prompt position P + i and sees keys 0 .. P + i (the
 * causal mask is aligned to the end of the prompt).  Every key, prefix or
 * suffix, is read through the block table: the suffix's own K/V must already
 * be in the pool.  Arithmetic: bf16 products with float32 accumulation,
 * float32 softmax; the probabilities are rounded to bf16 before the product
 * with V; the output is rounded to nearest-even bf16.
 *
 * Arguments
 *   q             device, bf16 [total_q][num_q_heads][head_dim], the suffix
 *                 tokens of all invocations packed in invocation order;
 *                 16-byte aligned.
 *   k_pool,
 *   v_pool        device, bf16 [num_blocks][num_kv_heads][block_size][head_dim]
 *                 (one (block, head) tile is contiguous); 16-byte aligned.
 *   block_tables  device, int32 [batch][max_blocks_per_seq]; row r maps logical
 *                 block b to a pool slot in [0, num_blocks) for
 *                 b < ceil((P_r + S_r) / block_size); later entries are not read.
 *                 Rows may share slots (a shared anchor).
 *   prefix_lens   device, int32 [batch], P_r >= 0 (0 = a miss).
 *   cu_q_lens     device, int32 [batch + 1], cu_q_lens[0] = 0, non-decreasing,
 *                 cu_q_lens[batch] = total_q.  S_r = 0 is allowed.
 *   batch, total_q          as above.
 *   max_q_len     >= every S_r (host value; sizes the launch).
 *   max_kv_len    >= every P_r + S_r; max_blocks_per_seq * block_size must be
 *                 >= max_kv_len.
 *   num_blocks    pool slots.
 *   num_q_heads, num_kv_heads  num_q_heads % num_kv_heads == 0.
 *   head_dim      64 or 128.   block_size  16.
 *   scale         logit scale, finite and > 0 (typically 1/sqrt(head_dim));
 *                 NaN or Inf -> CS_ERR_INVALID_ARG, 0 or negative ->
 *                 CS_ERR_UNSUPPORTED (the kernels track the running maximum
 *                 of the unscaled logits, which orders them only for a
 *                 positive scale).
 *   out           device, bf16 [total_q][num_q_heads][head_dim], 16-byte
 *                 aligned, must not overlap the inputs.
 *   stream        HIP stream.
 *
 * batch == 0, total_q == 0 or max_q_len == 0 is a no-op returning CS_OK.
 */
int cs_prefill_paged_attn(const void *q, const void *k_pool, const void *v_pool,
                          const int32_t *block_tables, const int32_t *prefix_lens,
                          const int32_t *cu_q_lens, int32_t batch, int32_t total_q,
                          int32_t max_q_len, int32_t max_kv_len,
                          int32_t max_blocks_per_seq, int32_t num_blocks,
                          int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                          int32_t block_size, float scale, void *out,
                          cs_stream_t stream);

/*
 * The same attention with a caller workspace, for launches too small to fill
 * the device (Sec. 2.1 "Prefix caching", as cs_prefill_paged_attn).
 *
 * When a call of cs_prefill_paged_attn would run its split kernel on at most
 * half as many 128-row tiles as there are compute units, this call cuts
 * every tile's key steps into `parts` contiguous pieces (2 to 4: as many as
 * fit one round of one work-group per CU, each at least four 64-key steps
 * of the longest sequence, which must have at least 16) that run on
 * separate work-groups; each writes its rows' partial result (O relative to
 * its running maximum m, m, and the probability sum l, in fp32) to the
 * workspace, and a second kernel combines the parts of every (token, query
 * head) row with log-sum-exp weights into the bf16 output.  The result
 * equals cs_prefill_paged_attn's up to rounding order.  Other launches (more tiles, or fewer than 16 key steps) ignore
 * the workspace and run exactly as cs_prefill_paged_attn.
 *
 * Arguments as in cs_prefill_paged_attn, plus
 *   workspace        device, 16-byte aligned, caller-owned scratch of at least
 *                    cs_prefill_paged_attn_workspace_bytes(batch, total_q,
 *                    max_q_len, max_kv_len, num_q_heads, num_kv_heads,
 *                    head_dim, 0) bytes (may be NULL when that is 0); its
 *                    contents are undefined after the call; calls that share
 *                    a workspace must be ordered on one stream.
 *   workspace_bytes  its size; smaller than required -> CS_ERR_INVALID_ARG.
 */
int cs_prefill_paged_attn_ws(const void *q, const void *k_pool, const void *v_pool,
                             const int32_t *block_tables, const int32_t *prefix_lens,
                             const int32_t *cu_q_lens, int32_t batch, int32_t total_q,
                             int32_t max_q_len, int32_t max_kv_len, int32_t max_blocks_per_seq,
                             int32_t num_blocks, int32_t num_q_heads, int32_t num_kv_heads,
                             int32_t head_dim, int32_t block_size, float scale, void *workspace,
                             int64_t workspace_bytes, void *out, cs_stream_t stream);

/* Workspace bytes cs_prefill_paged_attn_ws needs: parts * total_q *
 * num_q_heads * (head_dim + 2) * 4, or 0 when the launch takes no key parts.
 * num_cus: compute units to size for, 0 = the current device's (-1 if there
 * is none).  -1 for a negative size, bad head counts or a head_dim other
 * than 64 or 128. */
int64_t cs_prefill_paged_attn_workspace_bytes(int32_t batch, int32_t total_q, int32_t max_q_len,
                                              int32_t max_kv_len, int32_t num_q_heads,
                                              int32_t num_kv_heads, int32_t head_dim,
                                              int32_t num_cus);

/*
 * Launch shape of cs_prefill_paged_attn for a batch: a host-only query (no
 * GPU work, no device pointers) for profilers and tests that need to know
 * which kernel a call runs.
 *
 *   *kernel      CS_ATTN_SPLIT: 128-row tiles, each run by 8 waves over two
 *                halves of its keys (launches of fewer 256-row tiles than
 *                compute units, less than one round); CS_ATTN_PING_PONG:
 *                256-row tiles, where the last *tail_work_groups work-groups
 *                run the tiles of a last round at most half full as split
 *                128-row halves.
 *   *grid        work-groups of the launch (0 for a no-op call).
 *   *tail_work_groups  0 unless *kernel is CS_ATTN_PING_PONG.
 *
 * num_cus: the compute units to size the launch for (256 on MI355X), or 0
 * for those of the caller's current device (the count cs_prefill_paged_attn
 * uses; the runtime is then queried once per device, CS_ERR_HIP if it has
 * no device).  Other arguments as in cs_prefill_paged_attn; batch,
 * max_q_len, num_cus >= 0, head counts positive with num_q_heads %
 * num_kv_heads == 0, else CS_ERR_INVALID_ARG.  Output pointers must be
 * non-null.
 */
enum { CS_ATTN_SPLIT = 0, CS_ATTN_PING_PONG = 1 };
int cs_prefill_paged_attn_launch_shape(int32_t batch, int32_t max_q_len, int32_t num_q_heads,
                                       int32_t num_kv_heads, int32_t num_cus, int32_t *kernel,
                                       int64_t *grid, int64_t *tail_work_groups);

/*
 * KV prefetch: copy whole blocks from pinned host memory into pool slots.
 *
 * Operation (reload of an anchor from the CPU tier, Sec. 3 architecture
 * figure and Sec. 4; the reloaded blocks are the ones a normal invocation
 * produces, so the copy is bit-exact): for every i < n,
 *   k_pool[dst_block_ids[i]] = host_k_blocks[i]
 *   v_pool[dst_block_ids[i]] = host_v_blocks[i]
 * byte for byte; no other slot is written.  The kernel reads the host
 * buffers directly over the host link.
 *
 * Arguments
 *   host_k_blocks,
 *   host_v_blocks  pinned, device-mapped host memory (hipHostMalloc, or a
 *                  PyTorch pin_memory tensor), bf16
 *                  [n][num_kv_heads][block_size][head_dim], 16-byte aligned.
 *                  Anything else -> CS_ERR_INVALID_ARG.
 *   dst_block_ids  device, int32 [n]; unique, each in [0, num_blocks).
 *   n              number of blocks, at most min(num_blocks, 2^30 - 1); 0 is a
 *                  no-op returning CS_OK.
 *   k_pool, v_pool device, as in cs_prefill_paged_attn, 16-byte aligned.
 *   num_blocks, num_kv_heads, head_dim (64 or 128), block_size (16).
 *   stream         HIP stream, typically a side stream.  The destination
 *                  slots must not be read or written by any kernel still in
 *                  flight; order the consumer with an event recorded after
 *                  this call.  The host buffers must stay alive and unchanged
 *                  until the copy has completed.
 */
int cs_kv_prefetch(const void *host_k_blocks, const void *host_v_blocks,
                   const int32_t *dst_block_ids, int32_t n, void *k_pool, void *v_pool,
                   int32_t num_blocks, int32_t num_kv_heads, int32_t head_dim,
                   int32_t block_size, cs_stream_t stream);

/*
 * Paged decode attention: one query token per sequence over all its keys.
 *
 * Operation (the one-token case of cs_prefill_paged_attn, i.e. P = L - 1,
 * S = 1: the per-turn latency of Sec. 5 includes the decode that follows
 * the prefill): for every sequence r < batch, query head h and d,
 *   L = seq_lens[r],  g = h / (num_q_heads / num_kv_heads)
 *   out[r][h][d] = sum_{j < L} softmax_j(scale * dot(q[r][h], K_r[j])) V_r[j][d]
 * with K_r, V_r read through block_tables as in cs_prefill_paged_attn.  The
 * token's own K/V must already be in the pool (cs_kv_write).  Same
 * arithmetic conventions as cs_prefill_paged_attn.
 *
 * Arguments
 *   q, out         device, bf16 [batch][num_q_heads][head_dim], 16-byte aligned.
 *   block_tables   device, int32 [batch][max_blocks_per_seq].
 *   seq_lens       device, int32 [batch], each in [1, max_seq_len].
 *   num_q_heads / num_kv_heads <= 16; head_dim 64 or 128; block_size 16.
 *   scale          finite and > 0, as in cs_prefill_paged_attn.
 *   batch == 0 is a no-op returning CS_OK.
 */
int cs_paged_decode_attn(const void *q, const void *k_pool, const void *v_pool,
                         const int32_t *block_tables, const int32_t *seq_lens, int32_t batch,
                         int32_t max_seq_len, int32_t max_blocks_per_seq, int32_t num_blocks,
                         int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                         int32_t block_size, float scale, void *out, cs_stream_t stream);

/*
 * Cascade (shared-prefix) decode: the same result as cs_paged_decode_attn,
 * computed so that a prefix shared by a group of sequences is read once.
 *
 * Operation (Sec. 2.1, "Agent anchor": every invocation of an agent starts
 * with the same prompt prefix; Sec. 2.2: anchor blocks are the most reused
 * KV blocks, read by every invocation of the agent): the sequences are
 * partitioned into num_groups groups of consecutive sequences, group g being
 * sequences
 * cu_groups[g] .. cu_groups[g+1]-1, whose first shared_lens[g] keys are the
 * same pool blocks (identical block-table entries).  For each group and KV
 * head the queries of all its sequences (and of the query heads of that KV
 * head) are stacked and attend once over the shared keys, in chunks of 1024
 * keys; each chunk leaves a partial result (O relative to its running max m,
 * m and the sum l) in the workspace.  Each sequence's own keys
 * shared_lens[g] .. seq_lens[r]-1 are attended in segments of 1024 keys,
 * each leaving a partial too, and a last launch merges all partials of a
 * row with log-sum-exp weights.  The output equals cs_paged_decode_attn's up
 * to rounding order.
 *
 * Arguments (those of cs_paged_decode_attn, plus)
 *   cu_groups       device, int32 [num_groups + 1]: 0 = cu_groups[0] <= ...
 *                   <= cu_groups[num_groups] = batch.
 *   shared_lens     device, int32 [num_groups]: multiples of 16, each at most
 *                   max_shared_len and at most every seq_lens of its group
 *                   (0: the group shares nothing).
 *   num_groups      in [1, batch] (when batch > 0).
 *   max_group_seqs  host bound on the sequences of a group with a nonzero
 *                   shared_lens, in [1, batch] (groups sharing nothing may be
 *                   larger).
 *   max_shared_len  host bound on shared_lens, <= max_seq_len; sizes the launch
 *                   and the workspace.
 *   max_rest_len    host bound on every sequence's own keys,
 *                   seq_lens[r] - shared_lens[g] <= max_rest_len <= max_seq_len.
 *                   ceil(max_shared_len / 1024) + ceil(max_rest_len / 1024)
 *                   above 512 is CS_ERR_UNSUPPORTED.
 *   workspace       device, 16-byte aligned, caller-owned scratch of at least
 *                   cs_cascade_decode_workspace_bytes(batch, num_q_heads,
 *                   head_dim, max_shared_len, max_rest_len) bytes; its contents
 *                   are undefined after the call.  Calls that share a
 *                   workspace must be ordered on one stream.
 * With CS_DEBUG_CHECK=1 the group structure, the shared block ids and the
 * decode metadata are validated on the host first.
 */
int cs_cascade_decode_attn(const void *q, const void *k_pool, const void *v_pool,
                           const int32_t *block_tables, const int32_t *seq_lens, int32_t batch,
                           int32_t max_seq_len, int32_t max_blocks_per_seq, int32_t num_blocks,
                           const int32_t *cu_groups, const int32_t *shared_lens,
                           int32_t num_groups, int32_t max_group_seqs, int32_t max_shared_len,
                           int32_t max_rest_len, int32_t num_q_heads, int32_t num_kv_heads,
                           int32_t head_dim, int32_t block_size, float scale, void *workspace,
                           int64_t workspace_bytes, void *out, cs_stream_t stream);

/*
 * Cascade decode without a workspace, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation).
 *
 * The same operation, arguments, results and kernels as
 * cs_cascade_decode_attn, minus workspace / workspace_bytes: the partial
 * results go to a scratch array of CS_NOALLOC_SCRATCH_BYTES bytes that the
 * library holds in each device's memory from the time it is loaded until the
 * process ends.  The call allocates nothing (no hipMalloc, no host buffer).
 *   - A call whose cs_cascade_decode_workspace_bytes(batch, num_q_heads,
 *     head_dim, max_shared_len, max_rest_len) exceeds
 *     CS_NOALLOC_SCRATCH_BYTES returns CS_ERR_UNSUPPORTED before anything
 *     is enqueued (e.g. 128 sequences x 32 query heads at head_dim 128 and
 *     16 partials per row need 34 MB: use cs_cascade_decode_attn).
 *   - Every call on a device shares that device's array: calls that may
 *     overlap on one device (different streams without ordering, or
 *     different threads) race and give undefined results.  Order them on one
 *     stream or with events.  Nothing in the array needs to start at zero:
 *     every partial a call reads is written earlier in the same call.
 *   - The first call on each device asks the runtime for the array's device
 *     address once (make that first call outside a stream capture if the
 *     runtime cannot answer during one); later calls only launch kernels.
 *   - CS_DEBUG_CHECK is ignored here (its checks copy metadata to host
 *     buffers).
 */
#define CS_NOALLOC_SCRATCH_BYTES (32 * 1024 * 1024)
int cs_cascade_decode_attn_noalloc(const void *q, const void *k_pool, const void *v_pool,
                                   const int32_t *block_tables, const int32_t *seq_lens,
                                   int32_t batch, int32_t max_seq_len,
                                   int32_t max_blocks_per_seq, int32_t num_blocks,
                                   const int32_t *cu_groups, const int32_t *shared_lens,
                                   int32_t num_groups, int32_t max_group_seqs,
                                   int32_t max_shared_len, int32_t max_rest_len,
                                   int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                                   int32_t block_size, float scale, void *out,
                                   cs_stream_t stream);

/* Workspace bytes cs_cascade_decode_attn needs:
 * (ceil(max_shared_len / 1024) + ceil(max_rest_len / 1024)) * batch *
 * num_q_heads * (head_dim + 2) * 4; -1 for a negative size or a zero head
 * count or head_dim. */
int64_t cs_cascade_decode_workspace_bytes(int32_t batch, int32_t num_q_heads, int32_t head_dim,
                                          int32_t max_shared_len, int32_t max_rest_len);

/*
 * KV write-back: store the K/V rows of new tokens into their pool slots.
 *
 * Operation (Sec. 2.1: prefill computes the KV of every prompt token and the
 * prefix cache keeps it in 16-token blocks; Sec. 4: a warmup produces the
 * same KV blocks as a normal invocation): for every token t < num_tokens with
 * s = slot_mapping[t] >= 0 and every KV head h,
 *   k_pool[s / block_size][h][s % block_size][:] = k_new[t][h][:]
 *   v_pool[s / block_size][h][s % block_size][:] = v_new[t][h][:]
 * byte for byte.  Tokens with a negative slot are skipped.  This is the
 * write that puts a suffix's own K/V into the pool before
 * cs_prefill_paged_attn reads it.
 *
 * Arguments
 *   k_new, v_new   device, bf16 [num_tokens][num_kv_heads][head_dim], 16-byte
 *                  aligned.
 *   slot_mapping   device, int32 [num_tokens]; the non-negative entries are
 *                  distinct and < num_blocks * block_size.
 *   k_pool, v_pool device, as in cs_prefill_paged_attn.
 *   num_tokens == 0 is a no-op returning CS_OK.
 */
int cs_kv_write(const void *k_new, const void *v_new, const int32_t *slot_mapping,
                int32_t num_tokens, void *k_pool, void *v_pool, int32_t num_blocks,
                int32_t num_kv_heads, int32_t head_dim, int32_t block_size,
                cs_stream_t stream);

/*
 * KV offload: copy whole pool blocks to pinned host memory.
 *
 * Operation (Sec. 4: blocks are kept in the CPU tier, and eviction prefers
 * blocks already resident there; the reverse of cs_kv_prefetch): for every
 * i < n, host_k_blocks[i] = k_pool[src_block_ids[i]] and host_v_blocks[i] =
 * v_pool[src_block_ids[i]], byte for byte.  The kernel writes the host
 * buffers directly over the host link.
 *
 * Arguments
 *   src_block_ids  device, int32 [n], each in [0, num_blocks) (repeats allowed).
 *   k_pool, v_pool device, as in cs_prefill_paged_attn.
 *   host_k_blocks,
 *   host_v_blocks  pinned, device-mapped host memory, bf16
 *                  [n][num_kv_heads][block_size][head_dim], 16-byte aligned;
 *                  anything else -> CS_ERR_INVALID_ARG.  Read them only after
 *                  the stream has passed this call.
 *   n <= 2^30 - 1; n == 0 is a no-op returning CS_OK.
 */
int cs_kv_offload(const int32_t *src_block_ids, int32_t n, const void *k_pool,
                  const void *v_pool, int32_t num_blocks, void *host_k_blocks,
                  void *host_v_blocks, int32_t num_kv_heads, int32_t head_dim,
                  int32_t block_size, cs_stream_t stream);

/* ------------------------------------------------------------------------
 * Control plane (host only): the agent-transition learner, the survival
 * scorer and the prefetch coordinator of Sec. 3.2-3.4, driven as in the
 * runtime workflow algorithm of Sec. 3 (a block touch updates the block's
 * metadata; a touch by another agent than the current one is a dispatch:
 * the transition is counted, the thresholded graph and the hop table are
 * rebuilt from the new agent, and it becomes current).
 *
 * Agents are dense ids in [0, num_agents) (cs_scout_agent_id maps a
 * prompt-prefix fingerprint to one); blocks are pool slots in
 * [0, num_blocks).  Times are caller-defined integer ticks (the paper uses
 * scheduler steps); ages are `now - last access`.
 *
 * A handle is not thread-safe: calls on one handle must not overlap.
 * Handles are independent of each other and of the GPU calls.  Functions
 * that return a status fail with CS_ERR_INVALID_ARG (message in
 * cs_last_error()); queries with an out-of-range argument return -1 (ids)
 * or NaN (probabilities, scores).  A NULL handle is CS_ERR_INVALID_ARG,
 * -1 or NaN likewise.
 * ------------------------------------------------------------------------ */

typedef struct cs_scout cs_scout;

/* Hyperparameters.  The paper names them without values; the defaults are
 * this library's reading. */
typedef struct cs_scout_params {
    double eps;     /* Eq. (3) additive smoothing, > 0            (0.1)  */
    double tau;     /* Eq. (7) edge confidence threshold, [0, 1]  (0.2)  */
    int32_t e_max;  /* Eq. (8) hop horizon E_max, > 0             (4)    */
    double lambda;  /* Eq. (9) recency decay per tick, >= 0       (0.1)  */
    double delta;   /* Eq. (9) floor of both factors, >= 0        (0.05) */
    double r_min;   /* Eq. (11) predictability gate, finite       (0.3)  */
} cs_scout_params;

/* Fill *out with the defaults above. */
void cs_scout_default_params(cs_scout_params *out);

/* Create a control plane for up to num_agents agents (1..4096) and
 * num_blocks pool slots (>= 0).  params NULL = defaults.  On success *out
 * owns O(num_agents^2 + num_blocks) host memory (cs_scout_state_bytes);
 * release it with cs_scout_destroy.  On failure *out is NULL. */
int cs_scout_create(int32_t num_agents, int32_t num_blocks,
                    const cs_scout_params *params, cs_scout **out);

/* Release a handle (NULL is a no-op). */
void cs_scout_destroy(cs_scout *s);

/* Dense agent id of a prompt-prefix fingerprint (the agent anchor's hash,
 * Sec. 3.1): a known fingerprint returns its id, a new one the next free
 * id in arrival order, or -1 once num_agents ids are taken. */
int32_t cs_scout_agent_id(cs_scout *s, uint64_t fingerprint);

/* Record that `agent` touched pool slot `block` holding `tokens` tokens
 * (>= 0) at time `now`.  If `agent` differs from the current agent this is
 * a dispatch: C[current][agent] += 1 (when there is a current agent), the
 * hop table is rebuilt by breadth-first search from `agent` over the edges
 * of Eq. (7), and `agent` becomes current.  O(1) without a dispatch,
 * O(num_agents^2) with one. */
int cs_scout_observe_touch(cs_scout *s, int32_t block, int32_t agent,
                           int32_t tokens, int64_t now);

/* cs_scout_observe_touch for touches i = 0..n-1 in order (host arrays of n
 * entries): the block pool's prefix match of one request touches all its
 * prefix blocks at once.  Every entry is validated before any is applied;
 * on an error nothing changes. */
int cs_scout_observe_touches(cs_scout *s, const int32_t *blocks, const int32_t *agents,
                             const int32_t *tokens, const int64_t *now, int32_t n);

/* The current agent, -1 before the first touch. */
int32_t cs_scout_current(const cs_scout *s);

/* Eq. (3): P(j | i) = (C_ij + eps) / (sum_k C_ik + num_agents * eps). */
double cs_scout_transition_prob(const cs_scout *s, int32_t i, int32_t j);

/* Eq. (5): argmax_j P(j | current), lowest id on ties; -1 before the first
 * touch. */
int32_t cs_scout_predict(const cs_scout *s);

/* Eq. (8): 1 - min(E[a], e_max) / e_max with E[a] the hop distance from the
 * current agent in the graph of Eq. (7); 0 if unreachable or before the
 * first touch. */
double cs_scout_survival(const cs_scout *s, int32_t agent);

/* Eq. (8) for every agent into out[0..num_agents) (host array): the table
 * the paper computes once per scheduler step (Sec. 4). */
int cs_scout_survival_all(const cs_scout *s, double *out);

/* Eq. (9): (survival(owner) + delta) * (exp(-lambda * (now - last access))
 * + delta) * tokens, for the block's last toucher (survival 0 for a block
 * never touched, whose tokens are 0 as well). */
double cs_scout_score_block(const cs_scout *s, int32_t block, int64_t now);

/* Mark whether a block's contents are also resident in the CPU tier (e.g.
 * after cs_kv_offload); eviction prefers such blocks among equal scores
 * (Sec. 4).  resident: 0 or non-zero. */
int cs_scout_set_host_resident(cs_scout *s, int32_t block, int32_t resident);

/* The eviction victim among candidates[0..n) (host array): the block with
 * the lowest score; among equal scores a CPU-resident one; then the first.
 * -1 if n <= 0, candidates is NULL or any candidate is out of range. */
int32_t cs_scout_select_victim(const cs_scout *s, const int32_t *candidates,
                               int32_t n, int64_t now);

/* Eq. (2) over the observed transitions: 1 - H(next | current) / H(next)
 * of their empirical joint distribution; 0 with no transition, 1 when
 * every transition has the same successor. */
double cs_scout_predictability(const cs_scout *s);

/* Eq. (10)-(11), the between-step decision: the agent whose anchor to
 * prefetch (cs_scout_predict) when predictability >= r_min, else -1. */
int32_t cs_scout_between_step(const cs_scout *s);

/* Host bytes of the decision state: transition counts, row and column
 * totals, row entropies, hop table and the per-block tables (excludes the
 * fingerprint map): 4 A^2 + 28 A + 17 num_blocks for A = num_agents. */
int64_t cs_scout_state_bytes(const cs_scout *s);

/* Static, NUL-terminated name of a status code ("CS_OK", ...). */
const char *cs_status_string(int status);

/* Message describing the calling thread's most recent failed call; "" if none.
 * The pointer stays valid until the thread's next call into the library. */
const char *cs_last_error(void);

/* Static, NUL-terminated digest of the sources the library was built from
 * (16 hex digits of a SHA-256 over the names and bytes of the kernel
 * sources, internal headers and this header, as the package's build step
 * computes it), or "unknown" for a build that did not define it.  Lets a
 * caller check that a built library matches the sources beside it. */
const char *cs_source_digest(void);

#ifdef __cplusplus
}
#endif

#endif /* CACHESCOUT_H */
