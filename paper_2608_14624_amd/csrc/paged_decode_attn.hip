// Paged decode attention for gfx950: one new token per sequence attends over
// all keys of its sequence in the paged pool.
//
// This is the one-token case of the prefix-reuse attention (arXiv
// 2608.14624, Sec. 2.1: a request reuses the cached KV of its prefix; the
// per-turn latency the paper reports includes the decode that follows the
// prefill, Sec. 5): the query of sequence r is its last position L_r - 1 and
// sees every key 0 .. L_r - 1.  Decode reads each key once per KV head and
// does G = Hq / Hkv dot products with it, so it is bound by HBM bandwidth,
// not by the matrix cores.
//
// Kernel design
//   * One work-group = W wave64s = one (sequence, KV head), W = 12 (4 in
//     cascade mode); the G query heads of the group are the N = 16 columns
//     of v_mfma_f32_16x16x32_bf16 (G <= 16).
//   * The W waves split the key range in 32-key chunks (wave w takes chunks
//     w, w+W, ...) and run independent online softmaxes, so there is no
//     synchronisation in the loop; the W partial results are merged in LDS
//     at the end (log-sum-exp weights), so no workspace is needed.
//   * S^T = K Q^T with K fragments loaded from HBM straight into the MFMA A
//     operand (16 B per lane), Q^T kept in VGPRs.  O^T = V^T P^T reads V^T
//     with ds_read_b64_tr_b16 from a per-wave LDS tile that the wave itself
//     wrote (LDS operations of one wave complete in order, so no barrier).
//   * The K/V loads of a wave's next chunk are issued before the math of the
//     current one, so each wave keeps 16 KiB in flight.
//   * Work-groups are ordered KV head fastest, so each XCD serves one head.
//
// Cascade mode: a sequence belongs to a group whose shared prefix (its first
// shared_len keys) is attended by the stacked prefill kernel, which leaves
// one partial result (O relative to its running max m, the max m and the sum
// l) per 1024-key chunk in a workspace.  Here a work-group takes one KV head
// and one 1024-key segment of a sequence's own keys shared_len .. L - 1, so
// a long history spreads over several work-groups, and leaves its partial
// in the workspace too; cascade_merge_kernel then combines every partial of
// a row with log-sum-exp weights exp2((m_i - max) * c).
#include "internal.h"

#include <math.h>

namespace cs {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

constexpr int kBlock = 16;
constexpr int kChunk = 32;           // keys per wave step (2 pool blocks)
// waves per work-group: 12 for plain decode (one work-group fills a CU at
// three waves per SIMD, so a CU's last, longest sequence runs on all of its
// wave slots instead of a third of them), 4 for the cascade's 1024-key
// segments
constexpr int kDecodeWaves = 12;
constexpr int kCascadeWaves = 4;
constexpr int kThreads = 256;        // the merge kernel
constexpr int kMaxGroup = 16;
// plain decode batches up to this size run longest sequence first
constexpr int kLptMaxBatch = 1024;
constexpr float kLog2e = 1.4426950408889634f;

struct DecParams {
  const uint16_t* q;          // [B][Hq][D]
  const uint16_t* k_pool;
  const uint16_t* v_pool;
  const int32_t* block_tables;
  const int32_t* seq_lens;
  uint16_t* out;              // [B][Hq][D]
  int max_blocks_per_seq;
  int num_q_heads;
  int num_kv_heads;
  int group;
  float scale_log2;
  // cascade mode only
  const int32_t* cu_groups;     // [num_groups + 1], cu_groups[0] = 0, last = batch
  const int32_t* shared_lens;   // [num_groups]
  int num_groups;
  int batch;
  int chunk_keys;               // keys per partial of the shared prefix
  int chunks;                   // shared-prefix partials per row (upper bound)
  int segments;                 // own-key partials per row (upper bound)
  float* ws_o;                  // [chunks + segments][batch * num_q_heads][D]
  float* ws_ml;                 // [chunks + segments][batch * num_q_heads][2]
  int ws_rows;
};

// first key of sequence r that its group does not share
__device__ __forceinline__ int shared_len_of(const DecParams& p, int r) {
  int lo = 0, hi = p.num_groups - 1;   // the last group gr with cu_groups[gr] <= r
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (p.cu_groups[mid] <= r) lo = mid; else hi = mid - 1;
  }
  return p.shared_lens[lo];
}

template <int D, int W>
struct DecLds {
  // V tile of one wave: 32 keys x D, rows padded by 32 B so that the 32 lanes
  // of a transposing read (8 keys x 32 B) fall on distinct banks.
  static constexpr int vStride = D + 16;
  union {
    uint16_t v[W][kChunk * vStride];
    struct {
      float m[W][kMaxGroup];
      float l[W][kMaxGroup];
      float o[W][kMaxGroup][D];
    } merge;
  };
};

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8, v); }

template <int D, bool kCascade>
__global__ __launch_bounds__(64 * (kCascade ? kCascadeWaves : kDecodeWaves)) void paged_decode_attn_kernel(DecParams p) {
  constexpr int kWaves = kCascade ? kCascadeWaves : kDecodeWaves;
  constexpr int kWGThreads = 64 * kWaves;
  __shared__ DecLds<D, kWaves> sm;
  constexpr int vStride = DecLds<D, kWaves>::vStride;
  constexpr int DC = D / 32;         // 32-wide k-steps of the QK^T product
  constexpr int DT = D / 16;         // 16-row output tiles over the head dim
  constexpr int kRowChunks = D / 8;  // 16-byte chunks per key row
  constexpr int kVLoads = kChunk * kRowChunks / 64;

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int j = lane & 15;           // MFMA column: query head within the group
  const int qd = lane >> 4;          // lane group: k-slots 8*qd .. +7

  const int g = blockIdx.x % p.num_kv_heads;
  int r, seg = 0;
  if constexpr (kCascade) {
    r = (blockIdx.x / p.num_kv_heads) % p.batch;
    seg = blockIdx.x / p.num_kv_heads / p.batch;
  } else {
    // Longest sequence first: the work-groups of one wave of dispatch take
    // the sequences of ranks w / num_kv_heads in decreasing length (ties by
    // index), so the last of the launch's rounds holds the shortest ones
    // and the CUs run out of work together.  Every work-group ranks the
    // lengths itself (each thread a few candidates against all of them, in
    // LDS): the order is a permutation whatever the lengths hold, so every
    // (sequence, head) is still computed exactly once, and each output is
    // the same as in any other order.
    r = blockIdx.x / p.num_kv_heads;
    if (p.batch <= kLptMaxBatch) {
      __shared__ int lens[kLptMaxBatch];
      __shared__ int pick;
      for (int s = threadIdx.x; s < p.batch; s += kWGThreads) lens[s] = p.seq_lens[s];
      if (threadIdx.x == 0) pick = r;
      __syncthreads();
      for (int s = threadIdx.x; s < p.batch; s += kWGThreads) {
        const int ls = lens[s];
        int rank = 0;
        for (int t = 0; t < p.batch; ++t) {
          const int lt = lens[t];
          rank += (lt > ls) || (lt == ls && t < s);
        }
        if (rank == r) pick = s;
      }
      __syncthreads();
      r = pick;
    }
  }
  const int L = p.seq_lens[r];
  int start = 0;       // keys start .. end - 1 are this work-group's
  int end = L;
  if constexpr (kCascade) {
    start = shared_len_of(p, r) + seg * kCascadeSegmentKeys;
    end = min(L, start + kCascadeSegmentKeys);
    if (start >= end) return;          // nothing of this sequence's own here
  }
  const int n_blk = (end + kBlock - 1) / kBlock;
  const int first_chunk = start / kChunk;
  const int ch_end = (end + kChunk - 1) / kChunk;
  const size_t tile_elems = (size_t)kBlock * D;
  const size_t slot_elems = (size_t)p.num_kv_heads * tile_elems;
  const uint16_t* kbase = p.k_pool + (size_t)g * tile_elems;
  const uint16_t* vbase = p.v_pool + (size_t)g * tile_elems;
  const __attribute__((address_space(4))) int32_t* bt =
      (const __attribute__((address_space(4))) int32_t*)(p.block_tables +
                                                          (size_t)r * p.max_blocks_per_seq);

  // ---- Q^T operand: column j = query head g*G + j, dims 32*dc + 8*qd .. +7
  const bool head_valid = j < p.group;
  const int h = g * p.group + (head_valid ? j : 0);
  bf16x8 qreg[DC];
#pragma unroll
  for (int dc = 0; dc < DC; ++dc) {
    uint4 v = make_uint4(0, 0, 0, 0);
    if (head_valid)
      v = *reinterpret_cast<const uint4*>(p.q + ((size_t)r * p.num_q_heads + h) * D + 32 * dc + 8 * qd);
    qreg[dc] = as_bf16x8(v);
  }

  // ---- loads of one chunk: K fragments (A operand) and V rows (to LDS) --
  uint4 kreg[2][DC];
  uint4 vreg[kVLoads];
  auto load_chunk = [&](int ch) {
    const int b0 = 2 * ch;
    const int id0 = b0 < n_blk ? bt[b0] : -1;
    const int id1 = b0 + 1 < n_blk ? bt[b0 + 1] : -1;
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
      const int id = mt ? id1 : id0;
#pragma unroll
      for (int dc = 0; dc < DC; ++dc) {
        kreg[mt][dc] = make_uint4(0, 0, 0, 0);
        if (id >= 0)
          kreg[mt][dc] = *reinterpret_cast<const uint4*>(kbase + (size_t)id * slot_elems + j * D + 32 * dc + 8 * qd);
      }
    }
#pragma unroll
    for (int u = 0; u < kVLoads; ++u) {
      const int c = lane + 64 * u;
      const int key = c / kRowChunks;           // 0..31, uniform block per u
      const int id = key < kBlock ? id0 : id1;
      vreg[u] = make_uint4(0, 0, 0, 0);
      if (id >= 0)
        vreg[u] = *reinterpret_cast<const uint4*>(vbase + (size_t)id * slot_elems + (key % kBlock) * D + (c % kRowChunks) * 8);
    }
  };

  // V^T fragment (16 dims x 32 keys) for output tile dt: the slot s of lane
  // group qd is key 16*(s/4) + 4*qd + s%4, matching the S^T accumulator
  // layout (tile s/4, register s%4).  ds_read_b64_tr_b16 hands lane j of a
  // 16-lane group M[4e + j/4][j%4] of the 8-byte rows its lanes address; lane
  // 16*qd + i addresses key 4*qd + i/4, dims 16*dt + 4*(i%4).
  const uint16_t* vt = sm.v[wave];
  const int tr_off = (4 * qd + (j >> 2)) * vStride + 4 * (j & 3);
  auto v_frag = [&](int dt) -> bf16x8 {
    const uint16_t* base = vt + tr_off + 16 * dt;
    const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(base));
    const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(base + 16 * vStride));
    const i16x4 lohi[2] = {lo, hi};
    return __builtin_bit_cast(bf16x8, lohi);
  };

  f32x4 oacc[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) oacc[dt] = f32x4{};
  float m_run = -INFINITY;
  float l_run = 0.f;
  const float c = p.scale_log2;

  int ch = first_chunk + wave;
  if (ch < ch_end) load_chunk(ch);
  for (; ch < ch_end; ch += kWaves) {
    // V rows of this chunk into the wave's LDS tile
#pragma unroll
    for (int u = 0; u < kVLoads; ++u) {
      const int cc = lane + 64 * u;
      *reinterpret_cast<uint4*>(&sm.v[wave][(cc / kRowChunks) * vStride + (cc % kRowChunks) * 8]) = vreg[u];
    }
    // rows past the end of the sequence (inside its last block) overwritten
    // with zeros: their probabilities are 0, but 0 times a stale NaN or Inf
    // in the pool is NaN
    if ((ch + 1) * kChunk > end) {
#pragma unroll
      for (int u = 0; u < kVLoads; ++u) {
        const int cc = lane + 64 * u;
        if (ch * kChunk + cc / kRowChunks >= end)
          *reinterpret_cast<uint4*>(&sm.v[wave][(cc / kRowChunks) * vStride + (cc % kRowChunks) * 8]) =
              make_uint4(0, 0, 0, 0);
      }
    }
    // S^T = K Q^T: two 16-key tiles
    f32x4 s[2] = {f32x4{}, f32x4{}};
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
      for (int dc = 0; dc < DC; ++dc)
        s[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(kreg[mt][dc]), qreg[dc], s[mt], 0, 0, 0);
    if (ch + kWaves < ch_end) load_chunk(ch + kWaves);     // in flight during the math

    // mask keys past the end; register r of tile mt holds key 32*ch + 16*mt + 4*qd + r
    const int kbase_idx = ch * kChunk;
    float mloc = -INFINITY;
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const int key = kbase_idx + 16 * mt + 4 * qd + rr;
        s[mt][rr] = (key < end && key >= start) ? s[mt][rr] : -INFINITY;
        mloc = fmaxf(mloc, s[mt][rr]);
      }
    mloc = fmaxf(mloc, __shfl_xor(mloc, 16));
    mloc = fmaxf(mloc, __shfl_xor(mloc, 32));
    const float m_new = fmaxf(m_run, mloc);
    const float alpha = __builtin_amdgcn_exp2f((m_run - m_new) * c);
    m_run = m_new;
    l_run *= alpha;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) oacc[dt] *= alpha;
    const float mc = m_new * c;
    bf16x8 pb;
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const float e = __builtin_amdgcn_exp2f(__builtin_fmaf(s[mt][rr], c, -mc));
        pb[4 * mt + rr] = (__bf16)e;
        l_run += (float)pb[4 * mt + rr];
      }
    // O^T += V^T P^T
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
      oacc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(v_frag(dt), pb, oacc[dt], 0, 0, 0);
  }

  // ---- merge the waves' partial softmaxes -----------------------------
  l_run += __shfl_xor(l_run, 16);
  l_run += __shfl_xor(l_run, 32);
  __syncthreads();                     // every wave is done with its V tile
  if (qd == 0) {
    sm.merge.m[wave][j] = m_run;
    sm.merge.l[wave][j] = l_run;
  }
  // accumulator register rr of tile dt holds dim 16*dt + 4*qd + rr of head j
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int rr = 0; rr < 4; ++rr) sm.merge.o[wave][j][16 * dt + 4 * qd + rr] = oacc[dt][rr];
  __syncthreads();
  for (int idx = threadIdx.x; idx < p.group * D; idx += kWGThreads) {
    const int hj = idx / D;
    const int d = idx % D;
    const size_t row = (size_t)r * p.num_q_heads + g * p.group + hj;
    float mx = -INFINITY;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) mx = fmaxf(mx, sm.merge.m[w][hj]);
    float num = 0.f, den = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const float wt = __builtin_amdgcn_exp2f((sm.merge.m[w][hj] - mx) * c);   // 0 for idle waves
      num += wt * sm.merge.o[w][hj][d];
      den += wt * sm.merge.l[w][hj];
    }
    if constexpr (kCascade) {
      // this segment's partial: O relative to mx, mx, and the sum
      const size_t widx = (size_t)(p.chunks + seg) * p.ws_rows + row;
      p.ws_o[widx * D + d] = num;
      if (d == 0) {
        p.ws_ml[2 * widx] = mx;
        p.ws_ml[2 * widx + 1] = den;
      }
    } else {
      p.out[row * D + d] = __builtin_bit_cast(uint16_t, (__bf16)(num / den));
    }
  }
}

// One work-group per (sequence, KV head): the final output of cascade decode
// from every partial of the row (shared-prefix chunks, own-key segments).
// The maxima and sums of all partials are gathered into LDS by all threads
// at once, turned into per-partial weights, and every thread then sums its
// output elements over the partials with the loads issued together.
template <int D>
__global__ __launch_bounds__(kThreads) void cascade_merge_kernel(DecParams p) {
  extern __shared__ float wsm[];            // [group][parts]: maxima, then weights
  const int g = blockIdx.x % p.num_kv_heads;
  const int r = blockIdx.x / p.num_kv_heads;
  const int L = p.seq_lens[r];
  const int shared = shared_len_of(p, r);
  const int n_shared = (shared + p.chunk_keys - 1) / p.chunk_keys;
  const int n_own = (L - shared + kCascadeSegmentKeys - 1) / kCascadeSegmentKeys;
  const int n = n_shared + n_own;
  const int stride = p.chunks + p.segments;     // row length of wsm
  float* m_s = wsm;
  float* l_s = wsm + p.group * stride;
  const float c = p.scale_log2;
  const size_t row0 = (size_t)r * p.num_q_heads + g * p.group;
  auto part_of = [&](int i) { return i < n_shared ? i : p.chunks + (i - n_shared); };
  for (int t = threadIdx.x; t < p.group * n; t += kThreads) {
    const int hj = t / n, i = t % n;
    const float2 ml = *reinterpret_cast<const float2*>(p.ws_ml + 2 * ((size_t)part_of(i) * p.ws_rows + row0 + hj));
    m_s[hj * stride + i] = ml.x;
    l_s[hj * stride + i] = ml.y;
  }
  __syncthreads();
  if ((int)threadIdx.x < p.group) {
    const int hj = threadIdx.x;
    float mx = -INFINITY;
    for (int i = 0; i < n; ++i) mx = fmaxf(mx, m_s[hj * stride + i]);
    float den = 0.f;
    for (int i = 0; i < n; ++i) {
      const float wt = __builtin_amdgcn_exp2f((m_s[hj * stride + i] - mx) * c);
      m_s[hj * stride + i] = wt;              // the maximum becomes the weight
      den += wt * l_s[hj * stride + i];
    }
    const float inv = 1.f / den;
    for (int i = 0; i < n; ++i) m_s[hj * stride + i] *= inv;
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < p.group * D; idx += kThreads) {
    const int hj = idx / D;
    const int d = idx % D;
    const size_t row = row0 + hj;
    float acc = 0.f;
    int i = 0;
    for (; i + 4 <= n; i += 4) {
      float o[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) o[u] = p.ws_o[((size_t)part_of(i + u) * p.ws_rows + row) * D + d];
#pragma unroll
      for (int u = 0; u < 4; ++u) acc += m_s[hj * stride + i + u] * o[u];
    }
    for (; i < n; ++i) acc += m_s[hj * stride + i] * p.ws_o[((size_t)part_of(i) * p.ws_rows + row) * D + d];
    p.out[row * D + d] = __builtin_bit_cast(uint16_t, (__bf16)acc);
  }
}

}  // namespace

hipError_t launch_paged_decode_attn(const DecodeLaunch& a, hipStream_t stream) {
  DecParams p;
  p.q = a.q;
  p.k_pool = a.k_pool;
  p.v_pool = a.v_pool;
  p.block_tables = a.block_tables;
  p.seq_lens = a.seq_lens;
  p.out = a.out;
  p.max_blocks_per_seq = a.max_blocks_per_seq;
  p.num_q_heads = a.num_q_heads;
  p.num_kv_heads = a.num_kv_heads;
  p.group = a.num_q_heads / a.num_kv_heads;
  p.scale_log2 = a.scale * kLog2e;
  p.batch = a.batch;
  const dim3 grid((unsigned)((long long)a.batch * a.num_kv_heads)), block(64 * kDecodeWaves);
  if (a.head_dim == 128) {
    hipLaunchKernelGGL((paged_decode_attn_kernel<128, false>), grid, block, 0, stream, p);
  } else {
    hipLaunchKernelGGL((paged_decode_attn_kernel<64, false>), grid, block, 0, stream, p);
  }
  return hipGetLastError();
}

hipError_t launch_cascade_decode_rest(const CascadeLaunch& a, hipStream_t stream) {
  const CascadeGeometry geo = cascade_geometry(a.num_groups, a.max_group_seqs, a.max_shared_len,
                                               a.max_rest_len, a.num_q_heads, a.num_kv_heads);
  DecParams p = {};
  p.q = a.q;
  p.k_pool = a.k_pool;
  p.v_pool = a.v_pool;
  p.block_tables = a.block_tables;
  p.seq_lens = a.seq_lens;
  p.out = a.out;
  p.max_blocks_per_seq = a.max_blocks_per_seq;
  p.num_q_heads = a.num_q_heads;
  p.num_kv_heads = a.num_kv_heads;
  p.group = a.num_q_heads / a.num_kv_heads;
  p.scale_log2 = a.scale * kLog2e;
  p.cu_groups = a.cu_groups;
  p.shared_lens = a.shared_lens;
  p.num_groups = a.num_groups;
  p.batch = a.batch;
  p.chunk_keys = geo.chunk_keys;
  p.chunks = geo.chunks;
  p.segments = geo.segments;
  p.ws_o = a.ws_o;
  p.ws_ml = a.ws_ml;
  p.ws_rows = a.batch * a.num_q_heads;
  const long long rows = (long long)a.batch * a.num_kv_heads;
  if (geo.segments > 0) {
    const dim3 grid((unsigned)(rows * geo.segments)), block(64 * kCascadeWaves);
    if (a.head_dim == 128) {
      hipLaunchKernelGGL((paged_decode_attn_kernel<128, true>), grid, block, 0, stream, p);
    } else {
      hipLaunchKernelGGL((paged_decode_attn_kernel<64, true>), grid, block, 0, stream, p);
    }
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  const size_t lds = 2 * sizeof(float) * (size_t)p.group * (geo.chunks + geo.segments);
  if (a.head_dim == 128) {
    hipLaunchKernelGGL(cascade_merge_kernel<128>, dim3((unsigned)rows), dim3(kThreads), lds, stream, p);
  } else {
    hipLaunchKernelGGL(cascade_merge_kernel<64>, dim3((unsigned)rows), dim3(kThreads), lds, stream, p);
  }
  return hipGetLastError();
}

}  // namespace cs
