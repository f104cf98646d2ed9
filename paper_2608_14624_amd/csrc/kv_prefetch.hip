// KV prefetch for gfx950: copy whole KV blocks from pinned host memory into
// pool slots (arXiv 2608.14624: the predicted agent's anchor is reloaded from
// the CPU tier, Sec. 3 architecture figure and Sec. 4; the reloaded bytes
// are exactly those of a normal invocation, so the copy is bit-exact).
//
// The kernel reads the host buffers directly through their device mapping,
// so the bytes cross the host link once and land in HBM without a staging
// buffer.  One work-group moves one contiguous block (all KV heads, K or V:
// 32 KiB at 8 KV heads x 16 tokens x 128 dims), and every lane keeps eight
// 16-byte reads in flight before it writes, which puts 32 KiB per work-group
// on the link at once; a launch of 2n work-groups covers the link's latency
// with few waves per CU, so the copy leaves room for attention running
// concurrently on another stream.  Writes are plain 16-byte vector stores.
#include "internal.h"

namespace cs {
namespace {

constexpr int kThreads = 256;
constexpr int kUnroll = 8;

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(kThreads) void kv_prefetch_kernel(
    const u32x4* __restrict__ host_k, const u32x4* __restrict__ host_v,
    const int32_t* __restrict__ dst, u32x4* __restrict__ k_pool,
    u32x4* __restrict__ v_pool, long long vecs_per_block) {
  const int i = blockIdx.x >> 1;            // block index in the request
  const bool is_v = blockIdx.x & 1;
  const u32x4* src = (is_v ? host_v : host_k) + (size_t)i * vecs_per_block;
  const size_t slot = (size_t)dst[i];
  u32x4* out = (is_v ? v_pool : k_pool) + slot * vecs_per_block;
  for (long long base = 0; base < vecs_per_block; base += (long long)kThreads * kUnroll) {
    u32x4 v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const long long idx = base + (long long)u * kThreads + threadIdx.x;
      if (idx < vecs_per_block) v[u] = __builtin_nontemporal_load(src + idx);
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const long long idx = base + (long long)u * kThreads + threadIdx.x;
      if (idx < vecs_per_block) out[idx] = v[u];
    }
  }
}

}  // namespace

hipError_t launch_kv_prefetch(const PrefetchLaunch& a, hipStream_t stream) {
  const long long vecs = a.block_bytes / 16;
  const dim3 grid((unsigned)(2LL * a.n)), block(kThreads);
  hipLaunchKernelGGL(kv_prefetch_kernel, grid, block, 0, stream,
                     reinterpret_cast<const u32x4*>(a.host_k),
                     reinterpret_cast<const u32x4*>(a.host_v), a.dst,
                     reinterpret_cast<u32x4*>(a.k_pool), reinterpret_cast<u32x4*>(a.v_pool),
                     vecs);
  return hipGetLastError();
}

}  // namespace cs
