// KV write-back scatter and KV offload for gfx950.
//
// Write-back (arXiv 2608.14624, Sec. 2.1: prefill computes the KV of every
// prompt token and the cache keeps it in 16-token blocks; Sec. 4: a warmup
// produces the same blocks as a normal invocation): the K/V rows a forward
// pass produced for new tokens are stored into their pool slots before the
// attention reads them.  One wave moves one token: its Hkv x D row is
// contiguous in the source, and lands as Hkv runs of D elements (one per KV
// head) in the pool.  HBM bound: every byte is read once and written once.
//
// Offload (Sec. 4: blocks leaving the GPU are kept in the CPU tier): whole
// blocks are copied from pool slots to pinned host memory, the reverse of
// the prefetch, by the same few persistent work-groups (block_copy.h): 16-byte
// loads from HBM and non-temporal 16-byte stores that go over the host link
// through the buffer's device mapping.
#include "block_copy.h"
#include "internal.h"

namespace cs {
namespace {

constexpr int kThreads = 256;
constexpr int kTokensPerWG = kThreads / 64;

__global__ __launch_bounds__(kThreads) void kv_write_kernel(
    const u32x4* __restrict__ k_new, const u32x4* __restrict__ v_new,
    const int32_t* __restrict__ slot_mapping, int num_tokens, u32x4* __restrict__ k_pool,
    u32x4* __restrict__ v_pool, int num_kv_heads, int vecs_per_head_row, int block_size) {
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * kTokensPerWG + (threadIdx.x >> 6);
  if (t >= num_tokens) return;
  const int slot = slot_mapping[t];
  if (slot < 0) return;                       // token not stored
  const size_t blk = (size_t)(slot / block_size);
  const int off = slot % block_size;
  const int vecs = num_kv_heads * vecs_per_head_row;   // 16-byte chunks per token row
  const u32x4* ks = k_new + (size_t)t * vecs;
  const u32x4* vs = v_new + (size_t)t * vecs;
  for (int c = lane; c < vecs; c += 64) {
    const int h = c / vecs_per_head_row;
    const int w = c % vecs_per_head_row;
    const size_t dst = ((blk * num_kv_heads + h) * block_size + off) * vecs_per_head_row + w;
    const u32x4 kv = ks[c];
    const u32x4 vv = vs[c];
    k_pool[dst] = kv;
    v_pool[dst] = vv;
  }
}

__global__ __launch_bounds__(kCopyThreads) void kv_offload_kernel(
    const int32_t* __restrict__ src_ids, const u32x4* __restrict__ k_pool,
    const u32x4* __restrict__ v_pool, u32x4* __restrict__ host_k, u32x4* __restrict__ host_v,
    int units, long long vecs_per_block) {
  copy_units<false, true>(
      units, vecs_per_block,
      [=](int u) { return ((u & 1) ? v_pool : k_pool) + (size_t)src_ids[u >> 1] * vecs_per_block; },
      [=](int u) { return ((u & 1) ? host_v : host_k) + (size_t)(u >> 1) * vecs_per_block; });
}

}  // namespace

hipError_t launch_kv_write(const KvWriteLaunch& a, hipStream_t stream) {
  const dim3 grid((unsigned)((a.num_tokens + kTokensPerWG - 1) / kTokensPerWG)), block(kThreads);
  hipLaunchKernelGGL(kv_write_kernel, grid, block, 0, stream,
                     reinterpret_cast<const u32x4*>(a.k_new), reinterpret_cast<const u32x4*>(a.v_new),
                     a.slot_mapping, a.num_tokens, reinterpret_cast<u32x4*>(a.k_pool),
                     reinterpret_cast<u32x4*>(a.v_pool), a.num_kv_heads, a.head_dim / 8,
                     a.block_size);
  return hipGetLastError();
}

hipError_t launch_kv_offload(const KvOffloadLaunch& a, hipStream_t stream) {
  const int units = 2 * a.n;
  hipLaunchKernelGGL(kv_offload_kernel, dim3(copy_grid(units)), dim3(kCopyThreads), 0, stream,
                     a.src_ids, reinterpret_cast<const u32x4*>(a.k_pool),
                     reinterpret_cast<const u32x4*>(a.v_pool), reinterpret_cast<u32x4*>(a.host_k),
                     reinterpret_cast<u32x4*>(a.host_v), units, a.block_bytes / 16);
  return hipGetLastError();
}

}  // namespace cs
