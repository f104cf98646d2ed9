// Internal declarations shared by the C ABI layer (api.hip) and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace cs {

// Everything the attention kernel needs, already validated by the ABI layer.
struct AttnLaunch {
  const uint16_t* q;
  const uint16_t* k_pool;
  const uint16_t* v_pool;
  const int32_t* block_tables;
  const int32_t* prefix_lens;
  const int32_t* cu_q_lens;
  uint16_t* out;
  int batch;
  int max_q_len;
  int max_blocks_per_seq;
  int num_q_heads;
  int num_kv_heads;
  int head_dim;
  float scale;
  int cus;            // compute units of the device (sizes the rounds)
  int max_kv_len;
  int total_q;
  void* workspace;    // null: no key parts (see attn_geometry)
};

// most key parts a split launch takes (work-groups per tile), the fewest
// 64-key steps of the longest sequence per part, and the fewest steps of
// the longest sequence for a launch to take parts at all
constexpr int kMaxKeyParts = 4;
constexpr int kMinPartSteps = 4;
constexpr int kMinPartedSteps = 16;

// Compute units of the caller's current device, read from the runtime once
// per device and cached (a host-only query, safe during stream capture).
hipError_t current_device_cus(int* cus);

// Launch geometry of the attention kernel (host-side, for tests and tuning).
struct AttnGeometry {
  int waves;          // row waves per work-group: 8 (ping-pong kernel), or 4
                      // (each tile run by 8 waves over two halves of its keys)
  int heads_per_wg;   // query heads of one GQA group handled by one work-group
  int span;           // suffix tokens handled by one work-group
  int token_tiles;    // span-sized token tiles per invocation (upper bound)
  int head_tiles;     // num_q_heads / heads_per_wg
  long long grid;     // work-groups launched
  long long pp_grid;  // ping-pong work-groups; the rest of the grid (ping-pong
                      // launches only) runs the half tiles of the last round
  int parts;          // key parts per split tile (1: none; then grid = tiles)
  long long split_tiles;  // split launches: tiles per key part
};

// cus: compute units of the device.  The work-group order assumes the
// dispatcher deals consecutive work-groups round-robin to 8 XCDs (MI355X);
// any other count of XCDs changes only which L2 serves a tile, not the result.
// allow_parts: the caller gave a workspace, so a split launch that would
// leave at least half the CUs idle takes its tiles' keys in up to
// kMaxKeyParts parts on separate work-groups, whose partials
// a merge kernel combines.
AttnGeometry attn_geometry(int batch, int max_q_len, int max_kv_len, int num_q_heads, int num_kv_heads,
                           int head_dim, int cus, bool allow_parts);
hipError_t launch_prefill_paged_attn(const AttnLaunch& a, hipStream_t stream);

struct PrefetchLaunch {
  const uint16_t* host_k;   // device-visible addresses of the pinned host buffers
  const uint16_t* host_v;
  const int32_t* dst;
  int n;
  uint16_t* k_pool;
  uint16_t* v_pool;
  long long block_bytes;    // num_kv_heads * block_size * head_dim * 2
};

hipError_t launch_kv_prefetch(const PrefetchLaunch& a, hipStream_t stream);

struct KvWriteLaunch {
  const uint16_t* k_new;    // [num_tokens][num_kv_heads][head_dim]
  const uint16_t* v_new;
  const int32_t* slot_mapping;
  int num_tokens;
  uint16_t* k_pool;
  uint16_t* v_pool;
  int num_kv_heads;
  int head_dim;
  int block_size;
};

hipError_t launch_kv_write(const KvWriteLaunch& a, hipStream_t stream);

struct KvOffloadLaunch {
  const int32_t* src_ids;
  int n;
  const uint16_t* k_pool;
  const uint16_t* v_pool;
  uint16_t* host_k;         // device-visible addresses of the pinned host buffers
  uint16_t* host_v;
  long long block_bytes;
};

hipError_t launch_kv_offload(const KvOffloadLaunch& a, hipStream_t stream);

struct DecodeLaunch {
  const uint16_t* q;        // [batch][num_q_heads][head_dim]
  const uint16_t* k_pool;
  const uint16_t* v_pool;
  const int32_t* block_tables;
  const int32_t* seq_lens;
  uint16_t* out;
  int batch;
  int max_blocks_per_seq;
  int num_q_heads;
  int num_kv_heads;
  int head_dim;
  float scale;
};

hipError_t launch_paged_decode_attn(const DecodeLaunch& a, hipStream_t stream);

// Cascade decode: the shared prefix of each group of sequences is attended
// once with the group's queries stacked (shared_prefix_partials_kernel), in
// chunks of kCascadeChunkSteps * 64 keys whose partial results go to a
// workspace; the decode kernel attends each sequence's own keys in segments
// of kCascadeSegmentKeys, also as partials; a merge kernel combines them.
constexpr int kCascadeChunkSteps = 16;
// keys of a sequence's own part per work-group of the rest-of-sequence launch
constexpr int kCascadeSegmentKeys = 1024;
// partials per row the merge stages in LDS (16 heads x 512 x 8 B = 64 KiB)
constexpr int kCascadeMaxParts = 512;

struct CascadeGeometry {
  int chunk_keys;     // keys per chunk of a shared prefix
  int chunks;         // chunks of the longest shared prefix
  int segments;       // own-key segments of the longest rest of a sequence
  int row_tiles;      // 128-row tiles of the largest group
  long long grid;     // work-groups of the shared-prefix launch
};

CascadeGeometry cascade_geometry(int num_groups, int max_group_seqs, int max_shared_len,
                                 int max_rest_len, int num_q_heads, int num_kv_heads);

struct CascadeLaunch {
  const uint16_t* q;        // [batch][num_q_heads][head_dim]
  const uint16_t* k_pool;
  const uint16_t* v_pool;
  const int32_t* block_tables;
  const int32_t* seq_lens;
  const int32_t* cu_groups;     // [num_groups + 1]
  const int32_t* shared_lens;   // [num_groups]
  uint16_t* out;
  float* ws_o;                  // [chunks + segments][batch * num_q_heads][head_dim]
  float* ws_ml;                 // [chunks + segments][batch * num_q_heads][2]
  int batch;
  int max_blocks_per_seq;
  int num_groups;
  int max_group_seqs;
  int max_shared_len;
  int max_rest_len;
  int num_q_heads;
  int num_kv_heads;
  int head_dim;
  float scale;
};

hipError_t launch_shared_prefix_partials(const CascadeLaunch& a, hipStream_t stream);
hipError_t launch_cascade_decode_rest(const CascadeLaunch& a, hipStream_t stream);

}  // namespace cs
