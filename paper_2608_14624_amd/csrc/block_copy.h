// Whole-block copies between the pool and pinned host memory (prefetch and
// offload), shared by both directions.
//
// The copy crosses the host link, so its speed is set by the bytes kept in
// flight, not by the number of CUs: a few persistent work-groups that each
// keep 2 units x 8 x 16 bytes per lane in flight (64 KiB per work-group)
// fill the link, and leave every other CU to attention running concurrently
// on another stream.  A unit is one block's K or V: unit u is block u / 2,
// K for even u and V for odd u.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cs {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kCopyThreads = 256;
constexpr int kCopyGroups = 16;    // work-groups per launch (fewer when there is less work)
constexpr int kCopyUnroll = 8;     // 16-byte vectors per lane per unit and step
constexpr int kCopyUnits = 2;      // units in flight per work-group

inline unsigned copy_grid(long long units) {
  return (unsigned)(units < kCopyGroups ? units : kCopyGroups);
}

// Work-group blockIdx.x copies units blockIdx.x + k * gridDim.x.  src_of(u)
// and dst_of(u) give the unit's first vector; a unit is `vecs` vectors.
// kNtLoad / kNtStore mark the side that crosses the host link (read once,
// never reused on the GPU) as non-temporal.
template <bool kNtLoad, bool kNtStore, class SrcOf, class DstOf>
__device__ __forceinline__ void copy_units(int units, long long vecs, SrcOf src_of, DstOf dst_of) {
  const int stride = gridDim.x;
  for (int u0 = blockIdx.x; u0 < units; u0 += stride * kCopyUnits) {
    for (long long base = 0; base < vecs; base += (long long)kCopyThreads * kCopyUnroll) {
      u32x4 v[kCopyUnits][kCopyUnroll];
#pragma unroll
      for (int j = 0; j < kCopyUnits; ++j) {
        const int u = u0 + j * stride;
        if (u >= units) continue;
        const u32x4* src = src_of(u);
#pragma unroll
        for (int e = 0; e < kCopyUnroll; ++e) {
          const long long idx = base + (long long)e * kCopyThreads + threadIdx.x;
          if (idx < vecs) v[j][e] = kNtLoad ? __builtin_nontemporal_load(src + idx) : src[idx];
        }
      }
#pragma unroll
      for (int j = 0; j < kCopyUnits; ++j) {
        const int u = u0 + j * stride;
        if (u >= units) continue;
        u32x4* dst = dst_of(u);
#pragma unroll
        for (int e = 0; e < kCopyUnroll; ++e) {
          const long long idx = base + (long long)e * kCopyThreads + threadIdx.x;
          if (idx < vecs) {
            if (kNtStore)
              __builtin_nontemporal_store(v[j][e], dst + idx);
            else
              dst[idx] = v[j][e];
          }
        }
      }
    }
  }
}

}  // namespace cs
