// C ABI of libcachescout.so: argument validation, pinned-pointer resolution,
// optional metadata checks (CS_DEBUG_CHECK=1) and kernel launches.  The
// operations themselves are described in include/cachescout.h.
#include "cachescout.h"
#include "error.h"
#include "internal.h"

#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <atomic>
#include <vector>

namespace {
thread_local char g_last_error[512];

// compute units per device ordinal, 0 until read
constexpr int kMaxDevices = 64;
std::atomic<int> g_device_cus[kMaxDevices];
}  // namespace

namespace cs {

int fail(int status, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return status;
}

int ok() {
  g_last_error[0] = '\0';
  return CS_OK;
}

hipError_t current_device_cus(int* cus) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  const bool cached = dev >= 0 && dev < kMaxDevices;
  if (cached) {
    const int c = g_device_cus[dev].load(std::memory_order_relaxed);
    if (c > 0) {
      *cus = c;
      return hipSuccess;
    }
  }
  int c = 0;
  e = hipDeviceGetAttribute(&c, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  if (c <= 0) return hipErrorInvalidDevice;
  if (cached) g_device_cus[dev].store(c, std::memory_order_relaxed);
  *cus = c;
  return hipSuccess;
}

}  // namespace cs

namespace {

using cs::fail;
using cs::ok;

int hip_fail(hipError_t e, const char* what) {
  return fail(CS_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

// the block copies index the K and V units of a call (2 n) with 32-bit ints
constexpr int32_t kMaxCopyBlocks = (1 << 30) - 1;

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

bool debug_checks_enabled() {
  const char* v = getenv("CS_DEBUG_CHECK");
  return v != nullptr && v[0] == '1';
}

template <typename T>
hipError_t copy_to_host(std::vector<T>& dst, const T* src, size_t count, hipStream_t stream) {
  dst.resize(count);
  if (count == 0) return hipSuccess;
  hipError_t e = hipMemcpyAsync(dst.data(), src, count * sizeof(T), hipMemcpyDeviceToHost, stream);
  if (e != hipSuccess) return e;
  return hipStreamSynchronize(stream);
}

int debug_check_attn(const int32_t* block_tables, const int32_t* prefix_lens,
                     const int32_t* cu_q_lens, int batch, int total_q, int max_q_len,
                     int max_kv_len, int max_blocks_per_seq, int num_blocks,
                     hipStream_t stream) {
  std::vector<int32_t> cu, pl, bt;
  hipError_t e = copy_to_host(cu, cu_q_lens, (size_t)batch + 1, stream);
  if (e == hipSuccess) e = copy_to_host(pl, prefix_lens, (size_t)batch, stream);
  if (e == hipSuccess) e = copy_to_host(bt, block_tables, (size_t)batch * max_blocks_per_seq, stream);
  if (e != hipSuccess) return hip_fail(e, "CS_DEBUG_CHECK metadata copy");
  if (cu[0] != 0) return fail(CS_ERR_INVALID_ARG, "cu_q_lens[0] = %d, expected 0", cu[0]);
  if (cu[batch] != total_q)
    return fail(CS_ERR_INVALID_ARG, "cu_q_lens[batch] = %d but total_q = %d", cu[batch], total_q);
  for (int r = 0; r < batch; ++r) {
    const long long s = (long long)cu[r + 1] - cu[r];
    if (s < 0) return fail(CS_ERR_INVALID_ARG, "cu_q_lens decreases at %d", r);
    if (s > max_q_len) return fail(CS_ERR_INVALID_ARG, "S_%d = %lld exceeds max_q_len %d", r, s, max_q_len);
    if (pl[r] < 0) return fail(CS_ERR_INVALID_ARG, "prefix_lens[%d] = %d is negative", r, pl[r]);
    const long long len = s + pl[r];
    if (len > max_kv_len)
      return fail(CS_ERR_INVALID_ARG, "P_%d + S_%d = %lld exceeds max_kv_len %d", r, r, len, max_kv_len);
    const long long nb = (len + 15) / 16;
    for (long long b = 0; b < nb; ++b) {
      const int32_t slot = bt[(size_t)r * max_blocks_per_seq + b];
      if (slot < 0 || slot >= num_blocks)
        return fail(CS_ERR_INVALID_ARG, "block_tables[%d][%lld] = %d outside [0, %d)", r, b, slot, num_blocks);
    }
  }
  return CS_OK;
}

int debug_check_prefetch(const int32_t* dst, int n, int num_blocks, hipStream_t stream) {
  std::vector<int32_t> ids;
  hipError_t e = copy_to_host(ids, dst, (size_t)n, stream);
  if (e != hipSuccess) return hip_fail(e, "CS_DEBUG_CHECK metadata copy");
  std::vector<unsigned char> seen((size_t)num_blocks, 0);
  for (int i = 0; i < n; ++i) {
    if (ids[i] < 0 || ids[i] >= num_blocks)
      return fail(CS_ERR_INVALID_ARG, "dst_block_ids[%d] = %d outside [0, %d)", i, ids[i], num_blocks);
    if (seen[ids[i]]) return fail(CS_ERR_INVALID_ARG, "dst_block_ids[%d] = %d is a duplicate", i, ids[i]);
    seen[ids[i]] = 1;
  }
  return CS_OK;
}

int debug_check_slots(const int32_t* slots, int n, long long num_slots, hipStream_t stream) {
  std::vector<int32_t> ids;
  hipError_t e = copy_to_host(ids, slots, (size_t)n, stream);
  if (e != hipSuccess) return hip_fail(e, "CS_DEBUG_CHECK metadata copy");
  std::vector<unsigned char> seen((size_t)num_slots, 0);
  for (int i = 0; i < n; ++i) {
    if (ids[i] < 0) continue;
    if (ids[i] >= num_slots)
      return fail(CS_ERR_INVALID_ARG, "slot_mapping[%d] = %d outside [0, %lld)", i, ids[i], num_slots);
    if (seen[ids[i]]) return fail(CS_ERR_INVALID_ARG, "slot_mapping[%d] = %d is a duplicate", i, ids[i]);
    seen[ids[i]] = 1;
  }
  return CS_OK;
}

int debug_check_block_ids(const int32_t* ids_d, int n, int num_blocks, hipStream_t stream) {
  std::vector<int32_t> ids;
  hipError_t e = copy_to_host(ids, ids_d, (size_t)n, stream);
  if (e != hipSuccess) return hip_fail(e, "CS_DEBUG_CHECK metadata copy");
  for (int i = 0; i < n; ++i)
    if (ids[i] < 0 || ids[i] >= num_blocks)
      return fail(CS_ERR_INVALID_ARG, "src_block_ids[%d] = %d outside [0, %d)", i, ids[i], num_blocks);
  return CS_OK;
}

int debug_check_decode(const int32_t* block_tables, const int32_t* seq_lens, int batch,
                       int max_seq_len, int max_blocks_per_seq, int num_blocks,
                       hipStream_t stream) {
  std::vector<int32_t> sl, bt;
  hipError_t e = copy_to_host(sl, seq_lens, (size_t)batch, stream);
  if (e == hipSuccess) e = copy_to_host(bt, block_tables, (size_t)batch * max_blocks_per_seq, stream);
  if (e != hipSuccess) return hip_fail(e, "CS_DEBUG_CHECK metadata copy");
  for (int r = 0; r < batch; ++r) {
    if (sl[r] < 1 || sl[r] > max_seq_len)
      return fail(CS_ERR_INVALID_ARG, "seq_lens[%d] = %d outside [1, %d]", r, sl[r], max_seq_len);
    for (int b = 0; b < (sl[r] + 15) / 16; ++b) {
      const int32_t slot = bt[(size_t)r * max_blocks_per_seq + b];
      if (slot < 0 || slot >= num_blocks)
        return fail(CS_ERR_INVALID_ARG, "block_tables[%d][%d] = %d outside [0, %d)", r, b, slot, num_blocks);
    }
  }
  return CS_OK;
}

// Groups partition the batch in order; each shared prefix is whole blocks
// that every sequence of the group holds, through identical block ids.
int debug_check_groups(const int32_t* block_tables, const int32_t* seq_lens,
                       const int32_t* cu_groups, const int32_t* shared_lens, int batch,
                       int num_groups, int max_group_seqs, int max_shared_len, int max_rest_len,
                       int max_blocks_per_seq, hipStream_t stream) {
  std::vector<int32_t> sl, bt, cu, sh;
  hipError_t e = copy_to_host(sl, seq_lens, (size_t)batch, stream);
  if (e == hipSuccess) e = copy_to_host(bt, block_tables, (size_t)batch * max_blocks_per_seq, stream);
  if (e == hipSuccess) e = copy_to_host(cu, cu_groups, (size_t)num_groups + 1, stream);
  if (e == hipSuccess) e = copy_to_host(sh, shared_lens, (size_t)num_groups, stream);
  if (e != hipSuccess) return hip_fail(e, "CS_DEBUG_CHECK metadata copy");
  if (cu[0] != 0 || cu[num_groups] != batch)
    return fail(CS_ERR_INVALID_ARG, "cu_groups must start at 0 and end at batch = %d", batch);
  for (int g = 0; g < num_groups; ++g) {
    const int n = cu[g + 1] - cu[g];
    if (n < 0) return fail(CS_ERR_INVALID_ARG, "cu_groups decreases at %d", g);
    if (sh[g] > 0 && n > max_group_seqs)
      return fail(CS_ERR_INVALID_ARG, "group %d has %d sequences (max_group_seqs %d)", g, n, max_group_seqs);
    if (sh[g] < 0 || sh[g] % 16 != 0 || sh[g] > max_shared_len)
      return fail(CS_ERR_INVALID_ARG, "shared_lens[%d] = %d is not a multiple of 16 in [0, %d]", g,
                  sh[g], max_shared_len);
    for (int r = cu[g]; r < cu[g + 1]; ++r) {
      if (sh[g] > sl[r])
        return fail(CS_ERR_INVALID_ARG, "shared_lens[%d] = %d exceeds seq_lens[%d] = %d", g, sh[g], r, sl[r]);
      if (sl[r] - sh[g] > max_rest_len)
        return fail(CS_ERR_INVALID_ARG, "sequence %d has %d own keys (max_rest_len %d)", r,
                    sl[r] - sh[g], max_rest_len);
      for (int b = 0; b < sh[g] / 16; ++b) {
        if (bt[(size_t)r * max_blocks_per_seq + b] != bt[(size_t)cu[g] * max_blocks_per_seq + b])
          return fail(CS_ERR_INVALID_ARG, "sequence %d does not share block %d of group %d", r, b, g);
      }
    }
  }
  return CS_OK;
}

// Device-visible address of a pinned, device-mapped host buffer, or null.
const void* mapped_host_pointer(const void* host, const char* name, int* status) {
  hipPointerAttribute_t attr;
  memset(&attr, 0, sizeof(attr));
  hipError_t e = hipPointerGetAttributes(&attr, host);
  if (e != hipSuccess) {
    (void)hipGetLastError();   // clear the sticky error of the failed query
    *status = fail(CS_ERR_INVALID_ARG, "%s is not pinned host memory (%s)", name, hipGetErrorString(e));
    return nullptr;
  }
  if (attr.type != hipMemoryTypeHost || attr.devicePointer == nullptr || attr.hostPointer == nullptr) {
    *status = fail(CS_ERR_INVALID_ARG, "%s is not pinned, device-mapped host memory", name);
    return nullptr;
  }
  const char* base_h = static_cast<const char*>(attr.hostPointer);
  const char* base_d = static_cast<const char*>(attr.devicePointer);
  *status = CS_OK;
  return base_d + (static_cast<const char*>(host) - base_h);
}

}  // namespace

namespace {

// Argument checks shared by the decode calls; *noop is set for an empty batch.
int validate_decode(const void* q, const void* k_pool, const void* v_pool,
                    const int32_t* block_tables, const int32_t* seq_lens, int32_t batch,
                    int32_t max_seq_len, int32_t max_blocks_per_seq, int32_t num_blocks,
                    int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                    int32_t block_size, float scale, const void* out, bool* noop) {
  *noop = false;
  if (batch < 0 || max_seq_len < 0 || max_blocks_per_seq < 0 || num_blocks < 0)
    return fail(CS_ERR_INVALID_ARG, "negative size argument");
  if (num_q_heads <= 0 || num_kv_heads <= 0 || head_dim <= 0 || block_size <= 0)
    return fail(CS_ERR_INVALID_ARG, "head counts, head_dim and block_size must be positive");
  if (num_q_heads % num_kv_heads != 0)
    return fail(CS_ERR_INVALID_ARG, "num_q_heads %d is not a multiple of num_kv_heads %d",
                num_q_heads, num_kv_heads);
  if (num_q_heads / num_kv_heads > 16)
    return fail(CS_ERR_UNSUPPORTED, "more than 16 query heads per KV head");
  if (head_dim != 64 && head_dim != 128)
    return fail(CS_ERR_UNSUPPORTED, "head_dim %d (supported: 64, 128)", head_dim);
  if (block_size != 16) return fail(CS_ERR_UNSUPPORTED, "block_size %d (supported: 16)", block_size);
  if (!isfinite(scale)) return fail(CS_ERR_INVALID_ARG, "scale is not finite");
  if (!(scale > 0.f)) return fail(CS_ERR_UNSUPPORTED, "scale %g (supported: > 0)", (double)scale);
  if (batch == 0) {
    *noop = true;
    return CS_OK;
  }
  if (!q || !k_pool || !v_pool || !block_tables || !seq_lens || !out)
    return fail(CS_ERR_INVALID_ARG, "null pointer argument");
  if (num_blocks == 0 || max_seq_len == 0)
    return fail(CS_ERR_INVALID_ARG, "num_blocks and max_seq_len must be positive");
  if ((long long)max_blocks_per_seq * block_size < max_seq_len)
    return fail(CS_ERR_INVALID_ARG, "max_blocks_per_seq * block_size < max_seq_len");
  if (!aligned16(q) || !aligned16(k_pool) || !aligned16(v_pool))
    return fail(CS_ERR_INVALID_ARG, "q, k_pool and v_pool must be 16-byte aligned");
  if ((long long)batch * num_kv_heads > 0x7fffffffLL) return fail(CS_ERR_INVALID_ARG, "launch too large");
  return CS_OK;
}

}  // namespace

namespace {

// Workspace bytes of a launch with key parts: per part, an fp32 O row and
// (m, l) for every (token, query head); 0 without parts.
int64_t key_part_bytes(const cs::AttnGeometry& geo, int32_t total_q, int32_t num_q_heads,
                       int32_t head_dim) {
  if (geo.parts <= 1) return 0;
  return (int64_t)geo.parts * total_q * num_q_heads * (head_dim + 2) * (int64_t)sizeof(float);
}

// cs_prefill_paged_attn, and with a workspace (has_ws) the variant whose
// launches that would leave CUs idle split their keys into parts
int prefill_paged_attn(const void* q, const void* k_pool, const void* v_pool,
                       const int32_t* block_tables, const int32_t* prefix_lens,
                       const int32_t* cu_q_lens, int32_t batch, int32_t total_q, int32_t max_q_len,
                       int32_t max_kv_len, int32_t max_blocks_per_seq, int32_t num_blocks,
                       int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                       int32_t block_size, float scale, bool has_ws, void* workspace,
                       int64_t workspace_bytes, void* out, cs_stream_t stream) {
  if (batch < 0 || total_q < 0 || max_q_len < 0 || max_kv_len < 0 || max_blocks_per_seq < 0 ||
      num_blocks < 0)
    return fail(CS_ERR_INVALID_ARG, "negative size argument");
  if (num_q_heads <= 0 || num_kv_heads <= 0 || head_dim <= 0 || block_size <= 0)
    return fail(CS_ERR_INVALID_ARG, "head counts, head_dim and block_size must be positive");
  if (num_q_heads % num_kv_heads != 0)
    return fail(CS_ERR_INVALID_ARG, "num_q_heads %d is not a multiple of num_kv_heads %d",
                num_q_heads, num_kv_heads);
  if (head_dim != 64 && head_dim != 128)
    return fail(CS_ERR_UNSUPPORTED, "head_dim %d (supported: 64, 128)", head_dim);
  if (block_size != 16) return fail(CS_ERR_UNSUPPORTED, "block_size %d (supported: 16)", block_size);
  if (!isfinite(scale)) return fail(CS_ERR_INVALID_ARG, "scale is not finite");
  if (!(scale > 0.f)) return fail(CS_ERR_UNSUPPORTED, "scale %g (supported: > 0)", (double)scale);
  if (batch == 0 || total_q == 0 || max_q_len == 0) return ok();
  if (!q || !k_pool || !v_pool || !block_tables || !prefix_lens || !cu_q_lens || !out)
    return fail(CS_ERR_INVALID_ARG, "null pointer argument");
  if (num_blocks == 0) return fail(CS_ERR_INVALID_ARG, "num_blocks is 0");
  if (max_q_len > max_kv_len) return fail(CS_ERR_INVALID_ARG, "max_q_len exceeds max_kv_len");
  if ((long long)max_blocks_per_seq * block_size < max_kv_len)
    return fail(CS_ERR_INVALID_ARG, "max_blocks_per_seq * block_size < max_kv_len");
  if (!aligned16(q) || !aligned16(k_pool) || !aligned16(v_pool) || !aligned16(out))
    return fail(CS_ERR_INVALID_ARG, "q, k_pool, v_pool and out must be 16-byte aligned");
  if (has_ws && workspace_bytes < 0) return fail(CS_ERR_INVALID_ARG, "negative workspace_bytes");
  int cus = 0;
  hipError_t ecu = cs::current_device_cus(&cus);
  if (ecu != hipSuccess) return hip_fail(ecu, "compute-unit count of the current device");
  const cs::AttnGeometry geo = cs::attn_geometry(batch, max_q_len, max_kv_len, num_q_heads,
                                                 num_kv_heads, head_dim, cus, has_ws);
  if (geo.grid > 0x7fffffffLL) return fail(CS_ERR_INVALID_ARG, "launch too large");
  const int64_t need = key_part_bytes(geo, total_q, num_q_heads, head_dim);
  if (need > 0) {
    if (!workspace || !aligned16(workspace))
      return fail(CS_ERR_INVALID_ARG, "workspace must be a 16-byte aligned device buffer");
    if (workspace_bytes < need)
      return fail(CS_ERR_INVALID_ARG, "workspace_bytes %lld < %lld required", (long long)workspace_bytes,
                  (long long)need);
  }

  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  if (debug_checks_enabled()) {
    int st = debug_check_attn(block_tables, prefix_lens, cu_q_lens, batch, total_q, max_q_len,
                              max_kv_len, max_blocks_per_seq, num_blocks, s);
    if (st != CS_OK) return st;
  }
  cs::AttnLaunch a;
  a.q = static_cast<const uint16_t*>(q);
  a.k_pool = static_cast<const uint16_t*>(k_pool);
  a.v_pool = static_cast<const uint16_t*>(v_pool);
  a.block_tables = block_tables;
  a.prefix_lens = prefix_lens;
  a.cu_q_lens = cu_q_lens;
  a.out = static_cast<uint16_t*>(out);
  a.batch = batch;
  a.max_q_len = max_q_len;
  a.max_blocks_per_seq = max_blocks_per_seq;
  a.num_q_heads = num_q_heads;
  a.num_kv_heads = num_kv_heads;
  a.head_dim = head_dim;
  a.scale = scale;
  a.cus = cus;
  a.max_kv_len = max_kv_len;
  a.total_q = total_q;
  a.workspace = need > 0 ? workspace : nullptr;
  hipError_t e = cs::launch_prefill_paged_attn(a, s);
  if (e != hipSuccess) return hip_fail(e, "prefill_paged_attn launch");
  return ok();
}

}  // namespace

// Device scratch of cs_cascade_decode_attn_noalloc (the cascade's partial
// results), one array per device for the life of the process.  Host code
// never passes this name to a kernel: it uses the address the runtime
// reports for the current device (scratch_address).
static __device__ __align__(256) unsigned char scratch[CS_NOALLOC_SCRATCH_BYTES];

namespace {

std::atomic<void*> g_scratch_address[kMaxDevices];

// Device address of `scratch` on the current device, asked of the runtime on
// the first call on each device and kept.
hipError_t scratch_address(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  void* p = g_scratch_address[dev].load(std::memory_order_acquire);
  if (p == nullptr) {
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    g_scratch_address[dev].store(p, std::memory_order_release);
  }
  *out = p;
  return hipSuccess;
}

// cs_cascade_decode_attn with the caller's workspace, or (use_scratch) with
// this device's scratch array, in which case the metadata debug checks,
// which copy to host buffers, are skipped.
int cascade_decode(const void* q, const void* k_pool, const void* v_pool,
                   const int32_t* block_tables, const int32_t* seq_lens, int32_t batch,
                   int32_t max_seq_len, int32_t max_blocks_per_seq, int32_t num_blocks,
                   const int32_t* cu_groups, const int32_t* shared_lens, int32_t num_groups,
                   int32_t max_group_seqs, int32_t max_shared_len, int32_t max_rest_len,
                   int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                   int32_t block_size, float scale, void* workspace, int64_t workspace_bytes,
                   bool use_scratch, void* out, cs_stream_t stream) {
  bool noop;
  int st0 = validate_decode(q, k_pool, v_pool, block_tables, seq_lens, batch, max_seq_len,
                            max_blocks_per_seq, num_blocks, num_q_heads, num_kv_heads, head_dim,
                            block_size, scale, out, &noop);
  if (st0 != CS_OK) return st0;
  if (num_groups < 0 || max_group_seqs < 0 || max_shared_len < 0 || max_rest_len < 0 ||
      workspace_bytes < 0)
    return fail(CS_ERR_INVALID_ARG, "negative size argument");
  if (noop) return ok();
  if (num_groups < 1 || num_groups > batch)
    return fail(CS_ERR_INVALID_ARG, "num_groups %d outside [1, batch = %d]", num_groups, batch);
  if (max_group_seqs < 1 || max_group_seqs > batch)
    return fail(CS_ERR_INVALID_ARG, "max_group_seqs %d outside [1, batch = %d]", max_group_seqs, batch);
  if (max_shared_len > max_seq_len)
    return fail(CS_ERR_INVALID_ARG, "max_shared_len %d exceeds max_seq_len %d", max_shared_len, max_seq_len);
  if (max_rest_len > max_seq_len)
    return fail(CS_ERR_INVALID_ARG, "max_rest_len %d exceeds max_seq_len %d", max_rest_len, max_seq_len);
  if (!cu_groups || !shared_lens) return fail(CS_ERR_INVALID_ARG, "null pointer argument");
  const int64_t need = cs_cascade_decode_workspace_bytes(batch, num_q_heads, head_dim, max_shared_len,
                                                         max_rest_len);
  if (use_scratch) {
    if (need > (int64_t)CS_NOALLOC_SCRATCH_BYTES)
      return fail(CS_ERR_UNSUPPORTED, "this call needs %lld bytes of scratch; the allocation-free "
                  "entry point holds %lld (use cs_cascade_decode_attn with a workspace)",
                  (long long)need, (long long)CS_NOALLOC_SCRATCH_BYTES);
    hipError_t e = scratch_address(&workspace);
    if (e != hipSuccess) return hip_fail(e, "scratch address on the current device");
    workspace_bytes = CS_NOALLOC_SCRATCH_BYTES;
  }
  if (need > 0) {
    if (!workspace || !aligned16(workspace))
      return fail(CS_ERR_INVALID_ARG, "workspace must be a 16-byte aligned device buffer");
    if (workspace_bytes < need)
      return fail(CS_ERR_INVALID_ARG, "workspace_bytes %lld < %lld required", (long long)workspace_bytes,
                  (long long)need);
  }
  const cs::CascadeGeometry geo = cs::cascade_geometry(num_groups, max_group_seqs, max_shared_len,
                                                       max_rest_len, num_q_heads, num_kv_heads);
  if (geo.grid > 0x7fffffffLL || (long long)batch * num_kv_heads * geo.segments > 0x7fffffffLL)
    return fail(CS_ERR_INVALID_ARG, "launch too large");
  if (geo.chunks + geo.segments > cs::kCascadeMaxParts)
    return fail(CS_ERR_UNSUPPORTED, "%d partials per row (max %d): max_shared_len / 1024 + "
                "max_rest_len / 1024 too large", geo.chunks + geo.segments, cs::kCascadeMaxParts);
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  if (!use_scratch && debug_checks_enabled()) {
    int st = debug_check_decode(block_tables, seq_lens, batch, max_seq_len, max_blocks_per_seq,
                                num_blocks, s);
    if (st == CS_OK)
      st = debug_check_groups(block_tables, seq_lens, cu_groups, shared_lens, batch, num_groups,
                              max_group_seqs, max_shared_len, max_rest_len, max_blocks_per_seq, s);
    if (st != CS_OK) return st;
  }
  cs::CascadeLaunch a;
  a.q = static_cast<const uint16_t*>(q);
  a.k_pool = static_cast<const uint16_t*>(k_pool);
  a.v_pool = static_cast<const uint16_t*>(v_pool);
  a.block_tables = block_tables;
  a.seq_lens = seq_lens;
  a.cu_groups = cu_groups;
  a.shared_lens = shared_lens;
  a.out = static_cast<uint16_t*>(out);
  a.ws_o = static_cast<float*>(workspace);
  a.ws_ml = a.ws_o + (size_t)(geo.chunks + geo.segments) * batch * num_q_heads * head_dim;
  a.batch = batch;
  a.max_blocks_per_seq = max_blocks_per_seq;
  a.num_groups = num_groups;
  a.max_group_seqs = max_group_seqs;
  a.max_shared_len = max_shared_len;
  a.max_rest_len = max_rest_len;
  a.num_q_heads = num_q_heads;
  a.num_kv_heads = num_kv_heads;
  a.head_dim = head_dim;
  a.scale = scale;
  hipError_t e = cs::launch_shared_prefix_partials(a, s);
  if (e != hipSuccess) return hip_fail(e, "shared-prefix attention launch");
  e = cs::launch_cascade_decode_rest(a, s);
  if (e != hipSuccess) return hip_fail(e, "cascade decode launch");
  return ok();
}

}  // namespace

// the C ABI is the only thing the library exports (built with -fvisibility=hidden)
#pragma GCC visibility push(default)
extern "C" {

const char* cs_status_string(int status) {
  switch (status) {
    case CS_OK: return "CS_OK";
    case CS_ERR_INVALID_ARG: return "CS_ERR_INVALID_ARG";
    case CS_ERR_UNSUPPORTED: return "CS_ERR_UNSUPPORTED";
    case CS_ERR_HIP: return "CS_ERR_HIP";
    default: return "CS_UNKNOWN_STATUS";
  }
}

const char* cs_last_error(void) { return g_last_error; }

#ifndef CS_SOURCE_DIGEST
#define CS_SOURCE_DIGEST "unknown"
#endif
const char* cs_source_digest(void) { return CS_SOURCE_DIGEST; }

int cs_prefill_paged_attn(const void* q, const void* k_pool, const void* v_pool,
                          const int32_t* block_tables, const int32_t* prefix_lens,
                          const int32_t* cu_q_lens, int32_t batch, int32_t total_q,
                          int32_t max_q_len, int32_t max_kv_len, int32_t max_blocks_per_seq,
                          int32_t num_blocks, int32_t num_q_heads, int32_t num_kv_heads,
                          int32_t head_dim, int32_t block_size, float scale, void* out,
                          cs_stream_t stream) {
  return prefill_paged_attn(q, k_pool, v_pool, block_tables, prefix_lens, cu_q_lens, batch, total_q,
                            max_q_len, max_kv_len, max_blocks_per_seq, num_blocks, num_q_heads,
                            num_kv_heads, head_dim, block_size, scale, false, nullptr, 0, out, stream);
}

int cs_prefill_paged_attn_ws(const void* q, const void* k_pool, const void* v_pool,
                             const int32_t* block_tables, const int32_t* prefix_lens,
                             const int32_t* cu_q_lens, int32_t batch, int32_t total_q,
                             int32_t max_q_len, int32_t max_kv_len, int32_t max_blocks_per_seq,
                             int32_t num_blocks, int32_t num_q_heads, int32_t num_kv_heads,
                             int32_t head_dim, int32_t block_size, float scale, void* workspace,
                             int64_t workspace_bytes, void* out, cs_stream_t stream) {
  return prefill_paged_attn(q, k_pool, v_pool, block_tables, prefix_lens, cu_q_lens, batch, total_q,
                            max_q_len, max_kv_len, max_blocks_per_seq, num_blocks, num_q_heads,
                            num_kv_heads, head_dim, block_size, scale, true, workspace,
                            workspace_bytes, out, stream);
}

int64_t cs_prefill_paged_attn_workspace_bytes(int32_t batch, int32_t total_q, int32_t max_q_len,
                                              int32_t max_kv_len, int32_t num_q_heads,
                                              int32_t num_kv_heads, int32_t head_dim,
                                              int32_t num_cus) {
  if (batch < 0 || total_q < 0 || max_q_len < 0 || max_kv_len < 0 || num_cus < 0 ||
      num_q_heads <= 0 || num_kv_heads <= 0 || num_q_heads % num_kv_heads != 0 ||
      (head_dim != 64 && head_dim != 128))
    return -1;
  if (batch == 0 || total_q == 0 || max_q_len == 0) return 0;
  int cus = num_cus;
  if (cus == 0 && cs::current_device_cus(&cus) != hipSuccess) return -1;
  const cs::AttnGeometry geo = cs::attn_geometry(batch, max_q_len, max_kv_len, num_q_heads,
                                                 num_kv_heads, head_dim, cus, true);
  return key_part_bytes(geo, total_q, num_q_heads, head_dim);
}

int cs_prefill_paged_attn_launch_shape(int32_t batch, int32_t max_q_len, int32_t num_q_heads,
                                       int32_t num_kv_heads, int32_t num_cus, int32_t* kernel,
                                       int64_t* grid, int64_t* tail_work_groups) {
  if (!kernel || !grid || !tail_work_groups) return fail(CS_ERR_INVALID_ARG, "null output pointer");
  if (batch < 0 || max_q_len < 0 || num_cus < 0) return fail(CS_ERR_INVALID_ARG, "negative size argument");
  if (num_q_heads <= 0 || num_kv_heads <= 0 || num_q_heads % num_kv_heads != 0)
    return fail(CS_ERR_INVALID_ARG, "num_q_heads %d, num_kv_heads %d", num_q_heads, num_kv_heads);
  int cus = num_cus;
  if (cus == 0) {
    hipError_t e = cs::current_device_cus(&cus);
    if (e != hipSuccess) return hip_fail(e, "compute-unit count of the current device");
  }
  const cs::AttnGeometry geo = cs::attn_geometry(batch, max_q_len, max_q_len, num_q_heads, num_kv_heads,
                                                 128, cus, false);
  const bool pp = geo.waves == 8;
  *kernel = pp ? CS_ATTN_PING_PONG : CS_ATTN_SPLIT;
  *grid = (batch == 0 || max_q_len == 0) ? 0 : geo.grid;
  *tail_work_groups = pp && *grid ? geo.grid - geo.pp_grid : 0;
  return ok();
}

int cs_kv_prefetch(const void* host_k_blocks, const void* host_v_blocks,
                   const int32_t* dst_block_ids, int32_t n, void* k_pool, void* v_pool,
                   int32_t num_blocks, int32_t num_kv_heads, int32_t head_dim, int32_t block_size,
                   cs_stream_t stream) {
  if (n < 0 || num_blocks < 0) return fail(CS_ERR_INVALID_ARG, "negative size argument");
  if (n > kMaxCopyBlocks) return fail(CS_ERR_INVALID_ARG, "n = %d exceeds 2^30 - 1 blocks", n);
  if (num_kv_heads <= 0 || head_dim <= 0 || block_size <= 0)
    return fail(CS_ERR_INVALID_ARG, "num_kv_heads, head_dim and block_size must be positive");
  if (head_dim != 64 && head_dim != 128)
    return fail(CS_ERR_UNSUPPORTED, "head_dim %d (supported: 64, 128)", head_dim);
  if (block_size != 16) return fail(CS_ERR_UNSUPPORTED, "block_size %d (supported: 16)", block_size);
  if (n == 0) return ok();
  if (!host_k_blocks || !host_v_blocks || !dst_block_ids || !k_pool || !v_pool)
    return fail(CS_ERR_INVALID_ARG, "null pointer argument");
  if (n > num_blocks) return fail(CS_ERR_INVALID_ARG, "n = %d exceeds num_blocks = %d", n, num_blocks);
  if (!aligned16(host_k_blocks) || !aligned16(host_v_blocks) || !aligned16(k_pool) ||
      !aligned16(v_pool))
    return fail(CS_ERR_INVALID_ARG, "host buffers and pools must be 16-byte aligned");
  int st = CS_OK;
  const void* dk = mapped_host_pointer(host_k_blocks, "host_k_blocks", &st);
  if (st != CS_OK) return st;
  const void* dv = mapped_host_pointer(host_v_blocks, "host_v_blocks", &st);
  if (st != CS_OK) return st;

  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  if (debug_checks_enabled()) {
    st = debug_check_prefetch(dst_block_ids, n, num_blocks, s);
    if (st != CS_OK) return st;
  }
  cs::PrefetchLaunch a;
  a.host_k = static_cast<const uint16_t*>(dk);
  a.host_v = static_cast<const uint16_t*>(dv);
  a.dst = dst_block_ids;
  a.n = n;
  a.k_pool = static_cast<uint16_t*>(k_pool);
  a.v_pool = static_cast<uint16_t*>(v_pool);
  a.block_bytes = (long long)num_kv_heads * block_size * head_dim * 2;
  hipError_t e = cs::launch_kv_prefetch(a, s);
  if (e != hipSuccess) return hip_fail(e, "kv_prefetch launch");
  return ok();
}

int cs_paged_decode_attn(const void* q, const void* k_pool, const void* v_pool,
                         const int32_t* block_tables, const int32_t* seq_lens, int32_t batch,
                         int32_t max_seq_len, int32_t max_blocks_per_seq, int32_t num_blocks,
                         int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                         int32_t block_size, float scale, void* out, cs_stream_t stream) {
  bool noop;
  int st0 = validate_decode(q, k_pool, v_pool, block_tables, seq_lens, batch, max_seq_len,
                            max_blocks_per_seq, num_blocks, num_q_heads, num_kv_heads, head_dim,
                            block_size, scale, out, &noop);
  if (st0 != CS_OK) return st0;
  if (noop) return ok();
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  if (debug_checks_enabled()) {
    int st = debug_check_decode(block_tables, seq_lens, batch, max_seq_len, max_blocks_per_seq,
                                num_blocks, s);
    if (st != CS_OK) return st;
  }
  cs::DecodeLaunch a;
  a.q = static_cast<const uint16_t*>(q);
  a.k_pool = static_cast<const uint16_t*>(k_pool);
  a.v_pool = static_cast<const uint16_t*>(v_pool);
  a.block_tables = block_tables;
  a.seq_lens = seq_lens;
  a.out = static_cast<uint16_t*>(out);
  a.batch = batch;
  a.max_blocks_per_seq = max_blocks_per_seq;
  a.num_q_heads = num_q_heads;
  a.num_kv_heads = num_kv_heads;
  a.head_dim = head_dim;
  a.scale = scale;
  hipError_t e = cs::launch_paged_decode_attn(a, s);
  if (e != hipSuccess) return hip_fail(e, "paged_decode_attn launch");
  return ok();
}

int64_t cs_cascade_decode_workspace_bytes(int32_t batch, int32_t num_q_heads, int32_t head_dim,
                                           int32_t max_shared_len, int32_t max_rest_len) {
  if (batch < 0 || num_q_heads <= 0 || head_dim <= 0 || max_shared_len < 0 || max_rest_len < 0)
    return -1;
  const long long chunk = (long long)cs::kCascadeChunkSteps * 64;
  const long long parts = (max_shared_len + chunk - 1) / chunk +
                          (max_rest_len + cs::kCascadeSegmentKeys - 1) / cs::kCascadeSegmentKeys;
  return (int64_t)(parts * batch * num_q_heads * (head_dim + 2) * (long long)sizeof(float));
}

int cs_cascade_decode_attn(const void* q, const void* k_pool, const void* v_pool,
                           const int32_t* block_tables, const int32_t* seq_lens, int32_t batch,
                           int32_t max_seq_len, int32_t max_blocks_per_seq, int32_t num_blocks,
                           const int32_t* cu_groups, const int32_t* shared_lens,
                           int32_t num_groups, int32_t max_group_seqs, int32_t max_shared_len,
                           int32_t max_rest_len, int32_t num_q_heads, int32_t num_kv_heads,
                           int32_t head_dim, int32_t block_size, float scale, void* workspace,
                           int64_t workspace_bytes, void* out, cs_stream_t stream) {
  return cascade_decode(q, k_pool, v_pool, block_tables, seq_lens, batch, max_seq_len,
                        max_blocks_per_seq, num_blocks, cu_groups, shared_lens, num_groups,
                        max_group_seqs, max_shared_len, max_rest_len, num_q_heads, num_kv_heads,
                        head_dim, block_size, scale, workspace, workspace_bytes, false, out,
                        stream);
}

int cs_cascade_decode_attn_noalloc(const void* q, const void* k_pool, const void* v_pool,
                                   const int32_t* block_tables, const int32_t* seq_lens,
                                   int32_t batch, int32_t max_seq_len,
                                   int32_t max_blocks_per_seq, int32_t num_blocks,
                                   const int32_t* cu_groups, const int32_t* shared_lens,
                                   int32_t num_groups, int32_t max_group_seqs,
                                   int32_t max_shared_len, int32_t max_rest_len,
                                   int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                                   int32_t block_size, float scale, void* out,
                                   cs_stream_t stream) {
  return cascade_decode(q, k_pool, v_pool, block_tables, seq_lens, batch, max_seq_len,
                        max_blocks_per_seq, num_blocks, cu_groups, shared_lens, num_groups,
                        max_group_seqs, max_shared_len, max_rest_len, num_q_heads, num_kv_heads,
                        head_dim, block_size, scale, nullptr, 0, true, out, stream);
}

int cs_kv_write(const void* k_new, const void* v_new, const int32_t* slot_mapping,
                int32_t num_tokens, void* k_pool, void* v_pool, int32_t num_blocks,
                int32_t num_kv_heads, int32_t head_dim, int32_t block_size, cs_stream_t stream) {
  if (num_tokens < 0 || num_blocks < 0) return fail(CS_ERR_INVALID_ARG, "negative size argument");
  if (num_kv_heads <= 0 || head_dim <= 0 || block_size <= 0)
    return fail(CS_ERR_INVALID_ARG, "num_kv_heads, head_dim and block_size must be positive");
  if (head_dim != 64 && head_dim != 128)
    return fail(CS_ERR_UNSUPPORTED, "head_dim %d (supported: 64, 128)", head_dim);
  if (block_size != 16) return fail(CS_ERR_UNSUPPORTED, "block_size %d (supported: 16)", block_size);
  if (num_tokens == 0) return ok();
  if (!k_new || !v_new || !slot_mapping || !k_pool || !v_pool)
    return fail(CS_ERR_INVALID_ARG, "null pointer argument");
  if (num_blocks == 0) return fail(CS_ERR_INVALID_ARG, "num_blocks is 0");
  if (!aligned16(k_new) || !aligned16(v_new) || !aligned16(k_pool) || !aligned16(v_pool))
    return fail(CS_ERR_INVALID_ARG, "k_new, v_new and the pools must be 16-byte aligned");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  if (debug_checks_enabled()) {
    int st = debug_check_slots(slot_mapping, num_tokens, (long long)num_blocks * block_size, s);
    if (st != CS_OK) return st;
  }
  cs::KvWriteLaunch a;
  a.k_new = static_cast<const uint16_t*>(k_new);
  a.v_new = static_cast<const uint16_t*>(v_new);
  a.slot_mapping = slot_mapping;
  a.num_tokens = num_tokens;
  a.k_pool = static_cast<uint16_t*>(k_pool);
  a.v_pool = static_cast<uint16_t*>(v_pool);
  a.num_kv_heads = num_kv_heads;
  a.head_dim = head_dim;
  a.block_size = block_size;
  hipError_t e = cs::launch_kv_write(a, s);
  if (e != hipSuccess) return hip_fail(e, "kv_write launch");
  return ok();
}

int cs_kv_offload(const int32_t* src_block_ids, int32_t n, const void* k_pool, const void* v_pool,
                  int32_t num_blocks, void* host_k_blocks, void* host_v_blocks,
                  int32_t num_kv_heads, int32_t head_dim, int32_t block_size, cs_stream_t stream) {
  if (n < 0 || num_blocks < 0) return fail(CS_ERR_INVALID_ARG, "negative size argument");
  if (n > kMaxCopyBlocks) return fail(CS_ERR_INVALID_ARG, "n = %d exceeds 2^30 - 1 blocks", n);
  if (num_kv_heads <= 0 || head_dim <= 0 || block_size <= 0)
    return fail(CS_ERR_INVALID_ARG, "num_kv_heads, head_dim and block_size must be positive");
  if (head_dim != 64 && head_dim != 128)
    return fail(CS_ERR_UNSUPPORTED, "head_dim %d (supported: 64, 128)", head_dim);
  if (block_size != 16) return fail(CS_ERR_UNSUPPORTED, "block_size %d (supported: 16)", block_size);
  if (n == 0) return ok();
  if (!src_block_ids || !k_pool || !v_pool || !host_k_blocks || !host_v_blocks)
    return fail(CS_ERR_INVALID_ARG, "null pointer argument");
  if (num_blocks == 0) return fail(CS_ERR_INVALID_ARG, "num_blocks is 0");
  if (!aligned16(host_k_blocks) || !aligned16(host_v_blocks) || !aligned16(k_pool) ||
      !aligned16(v_pool))
    return fail(CS_ERR_INVALID_ARG, "host buffers and pools must be 16-byte aligned");
  int st = CS_OK;
  const void* dk = mapped_host_pointer(host_k_blocks, "host_k_blocks", &st);
  if (st != CS_OK) return st;
  const void* dv = mapped_host_pointer(host_v_blocks, "host_v_blocks", &st);
  if (st != CS_OK) return st;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  if (debug_checks_enabled()) {
    st = debug_check_block_ids(src_block_ids, n, num_blocks, s);
    if (st != CS_OK) return st;
  }
  cs::KvOffloadLaunch a;
  a.src_ids = src_block_ids;
  a.n = n;
  a.k_pool = static_cast<const uint16_t*>(k_pool);
  a.v_pool = static_cast<const uint16_t*>(v_pool);
  a.host_k = const_cast<uint16_t*>(static_cast<const uint16_t*>(dk));
  a.host_v = const_cast<uint16_t*>(static_cast<const uint16_t*>(dv));
  a.block_bytes = (long long)num_kv_heads * block_size * head_dim * 2;
  hipError_t e = cs::launch_kv_offload(a, s);
  if (e != hipSuccess) return hip_fail(e, "kv_offload launch");
  return ok();
}

}  // extern "C"
#pragma GCC visibility pop
