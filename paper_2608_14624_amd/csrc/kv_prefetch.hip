// KV prefetch for gfx950: copy whole KV blocks from pinned host memory into
// pool slots (arXiv 2608.14624: the predicted agent's anchor is reloaded from
// the CPU tier, Sec. 3 architecture figure and Sec. 4; the reloaded bytes
// are exactly those of a normal invocation, so the copy is bit-exact).
//
// The kernel reads the host buffers directly through their device mapping,
// so the bytes cross the host link once and land in HBM without a staging
// buffer.  It is built lean (block_copy.h): its waves need so few registers
// that they fit beside the attention work-groups running on another stream,
// on the same CUs, instead of holding CUs the attention would use; enough
// work-groups keep enough reads in flight to fill the link.  Writes are
// plain 16-byte vector stores.
#include "block_copy.h"
#include "internal.h"

namespace cs {
namespace {

__global__ __launch_bounds__(kCopyThreads) __attribute__((amdgpu_num_vgpr(kLeanVgprs)))
void kv_prefetch_kernel(const u32x4* __restrict__ host_k, const u32x4* __restrict__ host_v,
                        const int32_t* __restrict__ dst, u32x4* __restrict__ k_pool,
                        u32x4* __restrict__ v_pool, int units, int vecs_per_block) {
  copy_units_lean<true, false>(
      units, vecs_per_block,
      [=](int u) { return ((u & 1) ? host_v : host_k) + (size_t)(u >> 1) * vecs_per_block; },
      [=](int u) { return ((u & 1) ? v_pool : k_pool) + (size_t)dst[u >> 1] * vecs_per_block; });
}

}  // namespace

hipError_t launch_kv_prefetch(const PrefetchLaunch& a, hipStream_t stream) {
  const int vecs = (int)(a.block_bytes / 16);
  const int units = 2 * a.n;
  hipLaunchKernelGGL(kv_prefetch_kernel, dim3(lean_copy_grid(units)), dim3(kCopyThreads), 0, stream,
                     reinterpret_cast<const u32x4*>(a.host_k),
                     reinterpret_cast<const u32x4*>(a.host_v), a.dst,
                     reinterpret_cast<u32x4*>(a.k_pool), reinterpret_cast<u32x4*>(a.v_pool),
                     units, vecs);
  return hipGetLastError();
}

}  // namespace cs
