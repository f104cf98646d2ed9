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

// Lean variant for a copy that runs beside attention: at most kLeanVgprs
// registers per lane (two 16-byte vectors in flight), so its waves fit in the
// registers an attention work-group leaves free on a CU (two waves of at most
// 248 VGPRs per SIMD) and run on the same CUs instead of taking CUs of their
// own.  kLeanGroups work-groups keep 128 KiB in flight, which still fills the
// host link (52 GB/s measured): more (64 work-groups, 512 KiB) slowed the
// attention running beside the copy by 14% instead of 9%, fewer (8) left
// the link at 41 GB/s.
constexpr int kLeanGroups = 16;
constexpr int kLeanVgprs = 16;

inline unsigned lean_copy_grid(long long units) {
  return (unsigned)(units < kLeanGroups ? units : kLeanGroups);
}

template <bool kNtLoad, bool kNtStore, class SrcOf, class DstOf>
__device__ __forceinline__ void copy_units_lean(int units, int vecs, SrcOf src_of, DstOf dst_of) {
  for (int u = blockIdx.x; u < units; u += gridDim.x) {
    const u32x4* src = src_of(u);
    u32x4* dst = dst_of(u);
    for (int i = threadIdx.x; i < vecs; i += 2 * kCopyThreads) {
      const int i1 = i + kCopyThreads;
      const u32x4 a = kNtLoad ? __builtin_nontemporal_load(src + i) : src[i];
      u32x4 b = a;
      if (i1 < vecs) b = kNtLoad ? __builtin_nontemporal_load(src + i1) : src[i1];
      if (kNtStore) __builtin_nontemporal_store(a, dst + i); else dst[i] = a;
      if (i1 < vecs) {
        if (kNtStore) __builtin_nontemporal_store(b, dst + i1); else dst[i1] = b;
      }
    }
  }
}

}  // namespace cs
