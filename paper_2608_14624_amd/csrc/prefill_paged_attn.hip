// Paged prefix-reuse prefill attention for gfx950 (CDNA4).
//
// What it computes (arXiv 2608.14624, Sec. 2.1 "Prefix caching"): the suffix
// queries of each agent invocation attend over the KV of the cached prefix
// (the agent anchor) and of the suffix itself, all of it stored in 16-token
// blocks of a paged pool and reached through the invocation's block table;
// suffix row i is prompt position P + i and sees keys 0 .. P + i.
//
// Kernel design
//   * Each wave owns 32 query rows (one head x 32 consecutive suffix tokens
//     of one invocation), and the waves of a work-group share one KV head:
//     every K/V tile staged in LDS serves several heads of its GQA group
//     (all of them when the group has at least 4), or consecutive token
//     tiles of fewer heads.
//   * The contractions run on bf16 MFMA (v_mfma_f32_32x32x16_bf16) in the
//     transposed orientation S^T = K Q^T and O^T = V^T P^T.  In that
//     orientation a lane owns one query: the row max and row sum of the
//     online softmax are in-lane reductions plus one exchange between the two
//     lane halves, and the probabilities leave the S^T accumulator already in
//     the register layout of the B operand of the PV product.
//   * Keys are consumed 64 at a time (4 pool blocks, block ids read from the
//     block table with scalar loads a step ahead).  K and V go from HBM
//     straight into LDS (buffer loads with the LDS flag) as padded,
//     XOR-swizzled [key][d] rows; the A operand of the PV product (V^T) comes
//     from two transposing 8-byte LDS reads (ds_read_b64_tr_b16).
//   * Masking is a select to -inf (never an additive mask), so K positions
//     past the end of a sequence inside its last block never contribute
//     whatever they hold; the V rows there are overwritten with zeros in LDS
//     (their probabilities are 0, and 0 times a NaN would not be), and whole
//     blocks past the end are never loaded.
//   * Softmax runs in base 2 with log2(e) folded into the scale.
//
// Work-group order: the KV head varies fastest, so with 8 KV heads the 8 XCDs
// each serve one KV head and its K/V stays in that XCD's L2; then head tiles,
// then the token tiles of an invocation from the last (most keys) to the
// first, then invocations, so the 32 CUs of an XCD work on one or two
// invocations at a time and their K/V fits the XCD's 4 MB L2 (with
// invocations varying before token tiles, a 32-invocation batch kept 16
// invocations' K/V in flight per XCD and ran 9% slower).
//
// Ping-pong kernel (launches of at least a round of its tiles): 8 waves,
// 256 query rows per work-group, and the two waves of a SIMD are offset by
// half a step: waves 0-3 run an iteration as [MFMAs: PV of the previous step
// + QK^T of this one][softmax of this step], waves 4-7 as [softmax of the
// previous step][the same MFMAs], so one wave's matrix work overlaps the
// other's vector work between two barriers.  One work-group per CU at head
// dim 128, two at 64.
//
// Split tiles (launches of less than a round of ping-pong tiles): a 128-row
// tile of four waves alone on a CU would leave one wave per SIMD, with
// nothing to hide its softmax behind.  Instead 8 waves run each tile: waves
// w and w + 4 own the same rows, waves 0-3 take the first half of the key
// steps and waves 4-7 the second, each half with its own LDS ring, and at
// the end waves 4-7 hand (O, m, l) to waves 0-3 through LDS, which merge
// them with the log-sum-exp weights.  A ping-pong launch whose last round
// would be at most half full runs that round's tiles the same way, as two
// 128-row halves each, so it occupies every CU.  Launches that leave half
// the CUs idle even so can take a tile's keys in parts on more work-groups,
// whose partial results a merge kernel combines (the workspace call).
//
// Stacked mode (the shared-prefix half of cascade attention): the query rows
// of a work-group are any 128 (sequence, query head) pairs of one group of
// sequences that share a prefix and one KV head; they attend, without a
// causal limit, over one 64-key-aligned chunk of the shared prefix, and the
// work-group writes its unnormalized partial result (O, running max m, sum
// l) to a workspace instead of the output.  The other half (each sequence's
// own keys) and the log-sum-exp merge run in the decode kernel.  This kernel
// stages K and V through registers into a double-buffered LDS tile.
#include "internal.h"

#include <math.h>

#include <algorithm>
#include <type_traits>

namespace cs {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

constexpr int kBlock = 16;    // tokens per pool block
constexpr int kBN = 64;       // keys per step
constexpr int kNQ = 32;       // query rows per wave
constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr int kPPWaves = 8;             // ping-pong kernel: two groups of four waves
constexpr int kPPThreads = 64 * kPPWaves;
constexpr float kLog2e = 1.4426950408889634f;

struct Params {
  const uint16_t* q;
  const uint16_t* k_pool;
  const uint16_t* v_pool;
  const int32_t* block_tables;
  const int32_t* prefix_lens;
  const int32_t* cu_q_lens;
  uint16_t* out;
  int batch;
  int max_blocks_per_seq;
  int num_q_heads;
  int num_kv_heads;
  int group;          // query heads per KV head
  int heads_per_wg;
  int span;
  int token_tiles;
  int head_tiles;
  float scale_log2;   // scale * log2(e)
  // ping-pong launches: work-groups below pp_grid take ping-pong tiles; the
  // rest take the two 128-row halves of the tiles pp_grid, pp_grid + 1, ...
  // (span = the ping-pong tile's tokens)
  long long pp_grid;
  // shared_prefix_partials_kernel only (ws_o / ws_ml: also the key parts)
  const int32_t* cu_groups;     // [num_groups + 1] sequence range of each group
  const int32_t* shared_lens;   // [num_groups] shared prefix tokens (multiple of 16)
  int row_tiles;                // 128-row tiles of the largest group
  int chunk_steps;              // 64-key steps per chunk of the shared prefix
  int chunks;                   // chunks of the longest shared prefix
  float* ws_o;                  // [chunks][batch * num_q_heads][D] partial O
  float* ws_ml;                 // [chunks][batch * num_q_heads][2] partial (m, l)
  int ws_rows;                  // batch * num_q_heads
  // split launches with key parts (partial results in a workspace): work-group
  // wg takes key part wg / split_tiles of tile wg % split_tiles; the partials
  // go to ws_o / ws_ml as [parts][total_q * num_q_heads][D] and [..][2]
  int parts;
  int split_tiles;
  long long part_rows;          // total_q * num_q_heads
};

template <int D>
struct Lds {
  static constexpr int kStride = D + 8;       // K rows: [key][d], 16 B pad
  // V rows [key][d] padded by 64 B: a transposing read serves 32 lanes per
  // cycle from 64 banks, and those lanes cover 4 keys x 64 bytes; with rows
  // 64 bytes apart modulo 256 they hit every bank once.
  static constexpr int vStride = D + 32;
  uint16_t k[2][kBN * kStride];               // K of steps j (even/odd buffer)
  uint16_t v[2][kBN * vStride];               // V of steps j
};

// Direct-to-LDS staging (the ppd kernels).  buffer_load_dwordx4 with the
// LDS flag writes lane i's 16 bytes at the instruction's LDS address + 16 i,
// so one load moves 1 KB of a (block, head) tile: four 256-byte rows at
// D = 128, eight 128-byte rows at D = 64 (a "group").  Which 16-byte chunk
// each lane fetches is free, so the layout inside a group is any
// permutation of its chunks.  A buffer holds one 64-key step as 16 (D = 128)
// or 8 (D = 64) groups.
//   D = 128: groups 4 D + 8 elements apart (16 bytes of padding); chunk s of
//            row d holds the row's chunk s ^ 4d.
//   D = 64:  groups 8 D + 16 elements apart (32 bytes); chunk s of row d
//            holds the row's chunk s ^ y(d), y(d) = 4 ((d / 2) % 2) + d / 4.
// The K operand reads (ds_read_b128: 16 lanes, one chunk of 16 rows, per
// pass) and the transposing V reads (32 lanes, 64 bytes of 4 rows, per pass)
// are then free of bank conflicts at 64 banks (checked element by element,
// with the bank of every access, in the host layout test), and every
// per-lane address is one register plus a constant.  Buffer loads rather
// than global_load_lds: the compiler's wait insertion counts a global load
// into LDS as a flat access and then makes every LDS read wait for all loads
// in flight; with buffer loads it keeps exact counts.
template <int D>
struct DirectLayout;
template <>
struct DirectLayout<128> {
  static constexpr int kRows = 4;                 // rows per 1 KB group
  static constexpr int kGrp = 4 * 128 + 8;        // elements from group to group
  static __device__ __forceinline__ int swz(int d) { return 4 * d; }
};
template <>
struct DirectLayout<64> {
  static constexpr int kRows = 8;
  static constexpr int kGrp = 8 * 64 + 16;
  static __device__ __forceinline__ int swz(int d) { return 4 * ((d >> 1) & 1) + (d >> 2); }
};
//
// Word 3 of a raw buffer descriptor on gfx9-family parts: 32-bit data format
// (DATA_FORMAT = 4), no swizzle, no index stride.
constexpr int kRawBufferWord3 = 0x00020000;
// s_waitcnt immediates (gfx9 layout: vmcnt[3:0], expcnt[6:4], lgkmcnt[11:8],
// vmcnt[5:4] at [15:14]; a field at its maximum does not wait)
constexpr int kWaitVmcnt0 = 0x0F70;
constexpr int kWaitVmcnt2 = 0x0F72;
constexpr int kWaitVmcnt4 = 0x0F74;
constexpr int kWaitLgkmcnt0 = 0xC07F;

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8, v); }

// Lanes l and l ^ 32 hold the same query row (the two halves of its keys).
// v_permlane32_swap exchanges the upper lane half of its first operand with
// the lower lane half of its second, in VALU without an LDS round trip; with
// both operands holding x, the first then holds (x_lo, x_lo) and the second
// (x_hi, x_hi), so every lane sees its own value and its partner's.  The
// clang builtin of this ROCm returns the first operand for both results, so
// the instruction is written out; the s_nops cover the VALU-write /
// permlane-read hazard the compiler cannot see inside inline asm.
__device__ __forceinline__ void pair_swap(float x, float& a, float& b) {
  a = x;
  b = x;
  asm volatile("s_nop 1\n\tv_permlane32_swap_b32 %0, %1\n\ts_nop 1" : "+v"(a), "+v"(b));
}
__device__ __forceinline__ float pair_max(float x) {
  float a, b;
  pair_swap(x, a, b);
  return fmaxf(a, b);
}
__device__ __forceinline__ float pair_sum(float x) {
  float a, b;
  pair_swap(x, a, b);
  return a + b;
}

constexpr int kRowsPerWG = kNQ * kWaves;

// One 128-row tile of stacked rows against one chunk of a group's shared
// prefix: four waves of 32 rows, K and V staged through two register stages
// into a double-buffered LDS tile; writes the chunk's partial result.
template <int D>
__device__ __forceinline__ void stacked_tile(const Params& p, Lds<D>& sm, const int wg) {
  constexpr int kStride = Lds<D>::kStride;
  constexpr int vStride = Lds<D>::vStride;
  constexpr int KS = D / 16;     // MFMA k-steps over the head dim
  constexpr int DT = D / 32;     // 32-wide output tiles over the head dim

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;                  // row owner within the work-group
  const int qi = lane & 31;
  const int half = lane >> 5;

  // ---- work tile -----------------------------------------------------
  // Work-groups are dealt to the 8 XCDs round-robin, so the KV head is the
  // fastest-varying index (with 8 KV heads every XCD serves exactly one and
  // keeps its K/V in its own L2); then row tiles, chunks of the shared
  // prefix, groups.  Stacked row rho of a group is query head
  // g * group + rho % group of its sequence rho / group.
  const int g = wg % p.num_kv_heads;
  int rest = wg / p.num_kv_heads;
  const int rt = rest % p.row_tiles;
  rest /= p.row_tiles;
  const int chunk = rest % p.chunks;
  const int gr = rest / p.chunks;
  const int s0 = p.cu_groups[gr];
  const int n_rows = (p.cu_groups[gr + 1] - s0) * p.group;
  const int SH = p.shared_lens[gr];
  const int kb = chunk * p.chunk_steps * kBN;
  if (rt * kRowsPerWG >= n_rows || kb >= SH) return;
  const int ke = min(SH, kb + p.chunk_steps * kBN);
  const int qpos = ke - 1;                               // every row sees the whole chunk
  const int rho = rt * kRowsPerWG + wave * kNQ + qi;
  const bool row_valid = rho < n_rows;                   // this lane holds a real row
  const int rr = row_valid ? rho : 0;
  const int seq = s0 + rr / p.group;
  const int h = g * p.group + rr % p.group;
  const size_t qrow = ((size_t)seq * p.num_q_heads + h) * D;   // element offset in q
  const int j0 = kb / kBN;                               // first 64-key step
  const int n_steps = (ke - kb + kBN - 1) / kBN;
  const int n_blk = SH / kBlock;                         // shared prefixes are whole blocks
  const int32_t* bt = p.block_tables + (size_t)s0 * p.max_blocks_per_seq;   // the group's shared blocks
  const size_t tile_elems = (size_t)kBlock * D;             // one (block, head)
  const size_t slot_elems = (size_t)p.num_kv_heads * tile_elems;
  const uint16_t* kbase = p.k_pool + (size_t)g * tile_elems;
  const uint16_t* vbase = p.v_pool + (size_t)g * tile_elems;

  // ---- Q^T operand: lane holds query qi, dims ks*16 + half*8 .. +7 -----
  bf16x8 qreg[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    uint4 v = make_uint4(0, 0, 0, 0);
    if (row_valid) v = *reinterpret_cast<const uint4*>(p.q + qrow + ks * 16 + half * 8);
    qreg[ks] = as_bf16x8(v);
  }

  // ---- staging: wave w moves pool block (4*step + w) of the key range ----
  // The block id is wave-uniform and read with a scalar load one step ahead,
  // so the vector loads of a step never wait on a block-table lookup.  K and
  // V tiles are both moved row-major: lane l moves chunks c = l + 64u, token
  // c / (D/8), dims (c % (D/8))*8 .. +7.
  constexpr int kChunksPerRow = D / 8;
  constexpr int kKLoads = kBlock * kChunksPerRow / 64;             // 4 (D=128), 2 (D=64)
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);
  const __attribute__((address_space(4))) int32_t* bt_c =
      (const __attribute__((address_space(4))) int32_t*)bt;
  auto block_id = [&](int step) -> int {
    const int lb = (j0 + step) * (kBN / kBlock) + wave_u;
    return lb < n_blk ? bt_c[lb] : -1;                               // -1: past the end
  };

  // Iteration j reads K_j and V_j from buffer j&1 and, after the barrier
  // that ends iteration j-1's reads of buffer (j+1)&1, writes K_{j+1} and
  // V_{j+1} there, so one barrier per step separates every write from the
  // reads it must follow.  Two register stages: the loads of step j+3 are
  // issued at iteration j into the stage whose data (step j+1) was just
  // stored, so every global load has two steps to arrive.
  using Stage = uint4[kKLoads];
  uint4 kreg[2][kKLoads];
  uint4 vreg[2][kKLoads];
  auto load_tile = [&](Stage& dst, const uint16_t* base, int id) {
    if (id >= 0) {
      const uint16_t* src = base + (size_t)id * slot_elems;
#pragma unroll
      for (int u = 0; u < kKLoads; ++u) {
        const int c = lane + 64 * u;
        dst[u] = *reinterpret_cast<const uint4*>(src + (c / kChunksPerRow) * D + (c % kChunksPerRow) * 8);
      }
    } else {
#pragma unroll
      for (int u = 0; u < kKLoads; ++u) dst[u] = make_uint4(0, 0, 0, 0);
    }
  };
  auto store_tile = [&](const Stage& src, uint16_t* buf, int stride) {
#pragma unroll
    for (int u = 0; u < kKLoads; ++u) {
      const int c = lane + 64 * u;
      const int key = wave_u * kBlock + c / kChunksPerRow;
      *reinterpret_cast<uint4*>(&buf[key * stride + (c % kChunksPerRow) * 8]) = src[u];
    }
  };
  // V^T fragment for keys 16*ks2 .. +15 and dims 32*dt .. +31 from two
  // transposing reads.  ds_read_b64_tr_b16 treats the 8-byte rows addressed
  // by the 16 lanes of a group as a 16 x 4 matrix M and hands lane j of the
  // group M[4e + j/4][j%4], e = 0..3.  Lane 16g + i addresses key
  // 4*(g/2) + i/4 and dims 16*(g%2) + 4*(i%4) .. +3, so lane l receives
  // V[4*(l/32) + e][32*dt + l%32], e = 0..3: the A-operand slots 0..3 (keys
  // 4*half + e); the second read, 8 keys further, fills slots 4..7.
  const int tr_row = 4 * (lane >> 5) + ((lane & 15) >> 2);
  const int tr_col = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
  auto v_frag = [&](const uint16_t* vbuf, int ks2, int dt) -> bf16x8 {
    const uint16_t* base = &vbuf[(16 * ks2 + tr_row) * vStride + 32 * dt + tr_col];
    const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(base));
    const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(base + 8 * vStride));
    const i16x4 lohi[2] = {lo, hi};
    return __builtin_bit_cast(bf16x8, lohi);
  };

  // S^T = K Q^T for the 64 keys in kbuf: two 32-key tiles
  auto logits = [&](const uint16_t* kbuf, f32x16* sacc) {
    sacc[0] = f32x16{};
    sacc[1] = f32x16{};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
      for (int mt = 0; mt < 2; ++mt) {
        const uint4 a = *reinterpret_cast<const uint4*>(&kbuf[(mt * 32 + qi) * kStride + ks * 16 + half * 8]);
        sacc[mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(a), qreg[ks], sacc[mt], 0, 0, 0);
      }
    }
  };

  f32x16 oacc[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) oacc[dt] = f32x16{};
  float m_run = -INFINITY;     // running max of the raw (unscaled) logits
  const float c = p.scale_log2;

  // ---- prologue: step 0 in LDS buffer 0; steps 1 and 2 in registers ----
  float l_part[4] = {0.f, 0.f, 0.f, 0.f};     // partial row sums (short add chains)
  {
    const int id0 = block_id(0);
    load_tile(kreg[0], kbase, id0);
    load_tile(vreg[0], vbase, id0);
    store_tile(kreg[0], sm.k[0], kStride);
    store_tile(vreg[0], sm.v[0], vStride);
    if (n_steps > 1) {
      const int id1 = block_id(1);
      load_tile(kreg[1], kbase, id1);
      load_tile(vreg[1], vbase, id1);
    }
    if (n_steps > 2) {
      const int id2 = block_id(2);
      load_tile(kreg[0], kbase, id2);
      load_tile(vreg[0], vbase, id2);
    }
  }
  int id_next = block_id(3);   // block id of step j+3, read at iteration j

  // One step: stage j+1 into LDS, issue the loads of step j+3, then the
  // logits, softmax and PV product of step j.
  auto step = [&](const int j, Stage& kst, Stage& vst) {
    const int kstart = (j0 + j) * kBN;
    const int cur = j & 1;
    __syncthreads();   // iteration j-1's reads are done and its writes visible
    if (j + 1 < n_steps) {
      store_tile(kst, sm.k[cur ^ 1], kStride);     // K_{j+1}, V_{j+1}
      store_tile(vst, sm.v[cur ^ 1], vStride);
    }
    if (j + 3 < n_steps) {                          // in flight for two steps
      load_tile(kst, kbase, id_next);
      load_tile(vst, vbase, id_next);
    }
    id_next = block_id(j + 4);

    // The two waves of a SIMD (one per work-group) alternate between MFMA
    // bursts and softmax VALU work.  A wave raises its priority while it
    // issues MFMAs, so the matrix core is fed first and the other wave's
    // VALU work fills the gaps instead of delaying it.
    f32x16 s_cur[2];
    __builtin_amdgcn_s_setprio(1);
    logits(sm.k[cur], s_cur);
    __builtin_amdgcn_s_setprio(0);

    // ---- mask: keys past the chunk's end (a last step that is not full)
    // accumulator register rr of tile mt holds key
    //   kstart + 32*mt + 8*(rr/4) + 4*half + rr%4   for query qi
    if (kstart + kBN - 1 > qpos) {
#pragma unroll
      for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
        for (int rr = 0; rr < 16; ++rr) {
          const int kj = kstart + mt * 32 + 8 * (rr >> 2) + 4 * half + (rr & 3);
          s_cur[mt][rr] = (kj <= qpos) ? s_cur[mt][rr] : -INFINITY;
        }
      }
    }
    float mloc = -INFINITY;
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
      for (int rr = 0; rr < 16; ++rr) mloc = fmaxf(mloc, s_cur[mt][rr]);
    }
    mloc = pair_max(mloc);
    // ---- lazy rescale: move the reference max only when a row's max grew
    // by more than 2^8 in probability; otherwise keep it (p <= 256 then)
    const bool grow = (mloc - m_run) * c > 8.f;      // true for every row at step 0
    if (__builtin_amdgcn_ballot_w64(grow) != 0) {
      const float m_new = grow ? mloc : m_run;
      const float alpha = __builtin_amdgcn_exp2f((m_run - m_new) * c);
      m_run = m_new;
#pragma unroll
      for (int u = 0; u < 4; ++u) l_part[u] *= alpha;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) oacc[dt] *= alpha;
    }

    const float mc = m_run * c;
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
      for (int rr = 0; rr < 16; ++rr)
        s_cur[mt][rr] = __builtin_amdgcn_exp2f(__builtin_fmaf(s_cur[mt][rr], c, -mc));
    }

    // ---- O^T += V^T P^T: four 16-key MFMA steps --------------------
    const uint16_t* vbuf = sm.v[cur];
    __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int ks2 = 0; ks2 < kBN / 16; ++ks2) {
      const int mt = ks2 >> 1;
      const int rb = (ks2 & 1) * 8;
      bf16x8 b;
#pragma unroll
      for (int s2 = 0; s2 < 8; ++s2) b[s2] = (__bf16)s_cur[mt][rb + s2];
      // row sum over the same bf16 probabilities the PV product uses,
      // two per instruction
      const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
      l_part[0] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(b, b, 0, 1), ones, l_part[0], false);
      l_part[1] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(b, b, 2, 3), ones, l_part[1], false);
      l_part[2] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(b, b, 4, 5), ones, l_part[2], false);
      l_part[3] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(b, b, 6, 7), ones, l_part[3], false);
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
        oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(v_frag(vbuf, ks2, dt), b, oacc[dt], 0, 0, 0);
    }
    __builtin_amdgcn_s_setprio(0);
  };

  // unrolled by two so the register stage of each step is a constant
  for (int j = 0; j < n_steps; j += 2) {
    step(j, kreg[1], vreg[1]);
    if (j + 1 < n_steps) step(j + 1, kreg[0], vreg[0]);
  }
  const float l_run = (l_part[0] + l_part[1]) + (l_part[2] + l_part[3]);

  const float l_tot = pair_sum(l_run);
  // ---- partial result: O (relative to m_run), m_run, l ---------------
  if (row_valid) {
    const size_t widx = (size_t)chunk * p.ws_rows + qrow / D;
    float* orow = p.ws_o + widx * D;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
#pragma unroll
      for (int rg = 0; rg < 4; ++rg) {
        const float4 o = make_float4(oacc[dt][rg * 4], oacc[dt][rg * 4 + 1], oacc[dt][rg * 4 + 2],
                                     oacc[dt][rg * 4 + 3]);
        *reinterpret_cast<float4*>(orow + dt * 32 + 8 * rg + 4 * half) = o;
      }
    }
    if (half == 0) *reinterpret_cast<float2*>(p.ws_ml + 2 * widx) = make_float2(m_run, l_tot);
  }
}

template <int D>
__global__ __launch_bounds__(kThreads) void shared_prefix_partials_kernel(Params p) {
  __shared__ Lds<D> sm;
  stacked_tile<D>(p, sm, blockIdx.x);
}

// Split tile with direct-to-LDS staging: 8 waves over one tile of span rows
// (a launch of less than a round of ping-pong tiles), or over one half
// (span / 2 rows) of a ping-pong tile in a launch's last round (kTailTile).
// Waves 0-3 take the first half of the tile's 64-key steps, waves 4-7 the
// second; each wave loads one block of K and one of V per step straight into
// a two-deep ring of its half (k0/k1, v0/v1 or k2/k3, v2/v3), one iteration
// ahead (an iteration takes about 2 us, ample for a load), and the halves
// merge through LDS at the end.  Per step the arithmetic of a row is that of
// the ping-pong kernel (logits, mask, lazy rescale, exp2, bf16 P, row sums
// over the same bf16 values, PV), in the same order.
template <int D, bool kTailTile, bool kPartial = false>
__device__ __forceinline__ void ppd_split_tile(const Params& p, const int wg, uint16_t* k0, uint16_t* k1,
                                               uint16_t* k2, uint16_t* k3, uint16_t* v0, uint16_t* v1,
                                               uint16_t* v2, uint16_t* v3) {
  constexpr int KS = D / 16;     // MFMA k-steps over the head dim
  constexpr int DT = D / 32;     // 32-wide output tiles over the head dim
  using DL = DirectLayout<D>;
  constexpr int kGrp = DL::kGrp;
  constexpr int kLoads = kBlock / DL::kRows;           // 1 KB loads per block
  constexpr int kGroupElems = DL::kRows * D;           // (a local constant, as in the ppd kernel)
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = (tid >> 6) & 3;                 // row owner within the half
  const int split_half = __builtin_amdgcn_readfirstlane(tid >> 8);
  const int qi = lane & 31;
  const int half = lane >> 5;

  // ---- work tile (the order of the ping-pong kernel, with 128-row tiles);
  // the halves of a ping-pong tile are num_kv_heads work-groups apart, so
  // both run on the XCD that holds their KV head
  const int tiles_per_kv = p.head_tiles / p.num_kv_heads;
  int tile = wg;
  int sub_half = 0;
  int span = p.span;
  int part = 0;
  if constexpr (kPartial) {
    part = wg / p.split_tiles;
    tile = wg - part * p.split_tiles;
  }
  if constexpr (kTailTile) {
    const long long jt = wg - p.pp_grid;
    const int kvh = (int)(jt % p.num_kv_heads);
    const long long rj = jt / p.num_kv_heads;
    sub_half = (int)(rj & 1);
    tile = (int)(p.pp_grid + (rj >> 1) * p.num_kv_heads + kvh);
    span = p.span / 2;
  }
  const int g = tile % p.num_kv_heads;
  const int sub = tile / p.num_kv_heads;
  const int head_tile = g * tiles_per_kv + sub % tiles_per_kv;
  const int rest = sub / tiles_per_kv;
  const int r = rest / p.token_tiles;
  const int token_tile = p.token_tiles - 1 - rest % p.token_tiles;
  const int q0 = p.cu_q_lens[r];
  const int S = p.cu_q_lens[r + 1] - q0;
  const int t0 = token_tile * p.span + sub_half * span;
  if (t0 >= S) return;
  const int P = p.prefix_lens[r];
  const int L = P + S;
  const int h = head_tile * p.heads_per_wg + wave % p.heads_per_wg;
  const int t = t0 + (wave / p.heads_per_wg) * kNQ + qi;   // this lane's suffix row
  const bool row_valid = t < S;
  const size_t qrow = ((size_t)(q0 + (row_valid ? t : 0)) * p.num_q_heads + h) * D;
  const int qpos = row_valid ? P + t : L - 1;               // last visible key
  const int kv_end = P + min(S, t0 + span);                 // keys the tile needs
  const int n_all = (kv_end + kBN - 1) / kBN;
  // this work-group's key steps [s0, s1): all of them, or one of p.parts
  // contiguous parts (a part may be empty)
  int s0 = 0, s1 = n_all;
  if constexpr (kPartial) {
    s0 = (int)((long long)n_all * part / p.parts);
    s1 = (int)((long long)n_all * (part + 1) / p.parts);
  }
  const int n_part = s1 - s0;
  const int n_iter = n_part - n_part / 2;                   // both halves run as many iterations
  const int j0 = s0 + (split_half ? n_part / 2 : 0);
  const int n_steps = split_half ? n_part - n_part / 2 : n_part / 2;
  const int n_blk = (L + kBlock - 1) / kBlock;
  const int32_t* bt = p.block_tables + (size_t)r * p.max_blocks_per_seq;
  const int wave_qmin = P + min(t0 + (wave / p.heads_per_wg) * kNQ, S - 1);
  const size_t tile_elems = (size_t)kBlock * D;             // one (block, head)
  const size_t slot_elems = (size_t)p.num_kv_heads * tile_elems;

  // ---- Q^T operand: lane holds query qi, dims ks*16 + half*8 .. +7 -----
  bf16x8 qreg[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    uint4 v = make_uint4(0, 0, 0, 0);
    if (row_valid) v = *reinterpret_cast<const uint4*>(p.q + qrow + ks * 16 + half * 8);
    qreg[ks] = as_bf16x8(v);
  }

  // ---- staging: wave w loads pool block 4*step + w of its half's steps,
  // K and V, in the direct-to-LDS layout
  const int slot_u = __builtin_amdgcn_readfirstlane(wave);
  const uint16_t* kbase = p.k_pool + (size_t)g * tile_elems;
  const uint16_t* vbase = p.v_pool + (size_t)g * tile_elems;
  const __attribute__((address_space(4))) int32_t* bt_c =
      (const __attribute__((address_space(4))) int32_t*)bt;
  auto block_id = [&](int step) __attribute__((always_inline)) -> int {
    const int lb = (j0 + step) * (kBN / kBlock) + slot_u;
    return (step < n_steps && lb < n_blk) ? bt_c[lb] : -1;          // -1: past the end
  };
  // staging and operand addressing as in the ppd kernel (DirectLayout<D>)
  const int dma_d = lane / (D / 8);
  const int dma_off = dma_d * D + 8 * ((lane % (D / 8)) ^ DL::swz(dma_d));
  auto dma = [&](uint16_t* buf, const uint16_t* base, int id) __attribute__((always_inline)) {
    const uint16_t* blk = base + (size_t)(id >= 0 ? id : 0) * slot_elems;
    const __amdgpu_buffer_rsrc_t rs =
        __builtin_amdgcn_make_buffer_rsrc((void*)blk, (short)0, (int)(tile_elems * sizeof(uint16_t)), kRawBufferWord3);
#pragma unroll
    for (int u = 0; u < kLoads; ++u)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (__attribute__((address_space(3))) void*)(buf + (kLoads * slot_u + u) * kGrp),
                                               16, 2 * dma_off, 2 * u * kGroupElems, 0, 0);
  };
  auto zero_tail = [&](uint16_t* buf, int key0) __attribute__((always_inline)) {
    if (key0 + kBlock > L) {
#pragma unroll
      for (int u = 0; u < kLoads; ++u) {
        if (key0 + DL::kRows * u + dma_d >= L)
          *reinterpret_cast<uint4*>(&buf[(kLoads * slot_u + u) * kGrp + 8 * lane]) = make_uint4(0, 0, 0, 0);
      }
    }
  };
  constexpr int kKoff = D == 128 ? 4 : KS;
  int koff[kKoff];
#pragma unroll
  for (int k2i = 0; k2i < kKoff; ++k2i) {
    if constexpr (D == 128)
      koff[k2i] = (qi >> 2) * kGrp + (qi & 3) * D + 8 * half + 32 * (k2i ^ (qi & 3));
    else
      koff[k2i] = (qi >> 3) * kGrp + (qi & 7) * D + 8 * ((2 * k2i + half) ^ DL::swz(qi & 7));
  }
  auto k_addr = [&](const uint16_t* kbuf, int ks, int mt) __attribute__((always_inline)) -> const uint16_t* {
    if constexpr (D == 128) return &kbuf[mt * 8 * kGrp + 16 * (ks & 1) + koff[ks >> 1]];
    else return &kbuf[mt * 4 * kGrp + koff[ks]];
  };
  const int tr_row = 4 * (lane >> 5) + ((lane & 15) >> 2);
  int voff[DT];
  if constexpr (D == 128) {
    const int tr_d = tr_row & 3;
    const int tr_base = (tr_row >> 2) * kGrp + tr_d * D + 8 * (2 * ((lane >> 4) & 1) + ((lane & 3) >> 1)) + 4 * (lane & 1);
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) voff[dt] = tr_base + 32 * (dt ^ tr_d);
  } else {
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
      voff[dt] = tr_row * D + 8 * ((4 * dt + 2 * ((lane >> 4) & 1) + ((lane & 3) >> 1)) ^ DL::swz(tr_row)) + 4 * (lane & 1);
  }
  constexpr int kSliceGroups = 16 / DL::kRows;        // groups per 16-key slice
  auto v_frag = [&](const uint16_t* vbuf, int ks2, int dt) __attribute__((always_inline)) -> bf16x8 {
    const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(vbuf + kSliceGroups * ks2 * kGrp + voff[dt]));
    const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (lds_i16x4*)(vbuf + kSliceGroups * ks2 * kGrp + (kSliceGroups / 2) * kGrp + voff[dt]));
    const i16x4 lohi[2] = {lo, hi};
    return __builtin_bit_cast(bf16x8, lohi);
  };

  f32x16 oacc[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) oacc[dt] = f32x16{};
  float m_run = -INFINITY;     // running max of the raw (unscaled) logits
  float l_part[4] = {0.f, 0.f, 0.f, 0.f};
  const float c = p.scale_log2;

  // logits, mask, online softmax and PV product of step j
  auto step = [&](const int j, const uint16_t* kbuf, const uint16_t* vbuf) __attribute__((always_inline)) {
    const int kstart = (j0 + j) * kBN;
    f32x16 s_cur[2];
    s_cur[0] = f32x16{};
    s_cur[1] = f32x16{};
    __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
      for (int mt = 0; mt < 2; ++mt) {
        const uint4 a = *reinterpret_cast<const uint4*>(k_addr(kbuf, ks, mt));
        s_cur[mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(a), qreg[ks], s_cur[mt], 0, 0, 0);
      }
    }
    // interleave, the K reads two k-steps ahead of their MFMAs
    __builtin_amdgcn_sched_group_barrier(0x100, 4, 2);
#pragma unroll
    for (int ks = 2; ks < KS; ++ks) {
      __builtin_amdgcn_sched_group_barrier(0x008, 2, 2);
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 2);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 4, 2);
    __builtin_amdgcn_s_setprio(0);
    // accumulator register rr of tile mt holds key
    //   kstart + 32*mt + 8*(rr/4) + 4*half + rr%4   for query qi
    if (kstart + kBN - 1 > wave_qmin) {
      // key kj <= qpos  <=>  its constant offset in the step <= lim
      const int lim = qpos - kstart - 4 * half;
#pragma unroll
      for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
        for (int rr = 0; rr < 16; ++rr)
          s_cur[mt][rr] = (mt * 32 + 8 * (rr >> 2) + (rr & 3) <= lim) ? s_cur[mt][rr] : -INFINITY;
      }
    }
    float mloc = -INFINITY;
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
      for (int rr = 0; rr < 16; ++rr) mloc = fmaxf(mloc, s_cur[mt][rr]);
    }
    mloc = pair_max(mloc);
    // lazy rescale (a row whose keys so far were all masked keeps
    // m_run = -inf: possible only in the second half)
    const bool grow = (mloc - m_run) * c > 8.f;
    if (__builtin_amdgcn_ballot_w64(grow) != 0) {
      const float m_new = grow ? mloc : m_run;
      const float alpha = (m_new == m_run) ? 1.f : __builtin_amdgcn_exp2f((m_run - m_new) * c);
      m_run = m_new;
#pragma unroll
      for (int u = 0; u < 4; ++u) l_part[u] *= alpha;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) oacc[dt] *= alpha;
    }
    const float mc = (m_run == -INFINITY) ? 0.f : m_run * c;
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
      for (int rr = 0; rr < 16; ++rr)
        s_cur[mt][rr] = __builtin_amdgcn_exp2f(__builtin_fmaf(s_cur[mt][rr], c, -mc));
    }
    __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int ks2 = 0; ks2 < kBN / 16; ++ks2) {
      const int mt = ks2 >> 1;
      const int rb = (ks2 & 1) * 8;
      bf16x8 b;
#pragma unroll
      for (int s2 = 0; s2 < 8; ++s2) b[s2] = (__bf16)s_cur[mt][rb + s2];
      const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
      l_part[0] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(b, b, 0, 1), ones, l_part[0], false);
      l_part[1] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(b, b, 2, 3), ones, l_part[1], false);
      l_part[2] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(b, b, 4, 5), ones, l_part[2], false);
      l_part[3] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(b, b, 6, 7), ones, l_part[3], false);
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
        oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(v_frag(vbuf, ks2, dt), b, oacc[dt], 0, 0, 0);
    }
    // interleave, the V reads two fragments ahead of their MFMAs
    __builtin_amdgcn_sched_group_barrier(0x100, 4, 3);
#pragma unroll
    for (int f = 2; f < DT * (kBN / 16); ++f) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 3);
      __builtin_amdgcn_sched_group_barrier(0x100, 2, 3);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 2, 3);
    __builtin_amdgcn_s_setprio(0);
  };

  // iteration j: this step's loads have landed (nothing newer is in flight),
  // V past the end zeroed, barrier; then the loads of step j+1 into the
  // other buffer, read last in iteration j-1, and step j
  auto run = [&](uint16_t* kr0, uint16_t* kr1, uint16_t* vr0, uint16_t* vr1) __attribute__((always_inline)) {
    int id = block_id(0);
    if (n_steps > 0) {
      dma(kr0, kbase, id);
      dma(vr0, vbase, id);
    }
    id = block_id(1);
    auto iteration = [&](const int j, uint16_t* kcur, uint16_t* vcur, uint16_t* knext,
                         uint16_t* vnext) __attribute__((always_inline)) {
      __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
      if (j < n_steps) zero_tail(vcur, (j0 + j) * kBN + slot_u * kBlock);
      __builtin_amdgcn_s_waitcnt(kWaitLgkmcnt0);
      asm volatile("s_barrier" ::: "memory");
      if (j + 1 < n_steps) {
        dma(knext, kbase, id);
        dma(vnext, vbase, id);
      }
      if (j < n_steps) step(j, kcur, vcur);
      id = block_id(j + 2);
    };
    for (int j = 0; j < n_iter; j += 2) {
      iteration(j, kr0, vr0, kr1, vr1);
      if (j + 1 < n_iter) iteration(j + 1, kr1, vr1, kr0, vr0);
    }
  };
  if (split_half) run(k2, k3, v2, v3);
  else run(k0, k1, v0, v1);

  const float l_run = (l_part[0] + l_part[1]) + (l_part[2] + l_part[3]);
  float l_tot = pair_sum(l_run);
  // ---- merge: wave w of the second half hands (O, m, l) of its rows to
  // wave w of the first through one staging buffer (16640 bytes at head_dim
  // 128, 8448 at 64: exactly what it takes): value e of lane l at word
  // 64 e + l, m and l of query qi at words kMl + qi and kMl + 32 + qi
  constexpr int kMl = DT * 16 * 64;
  static_assert(kMl + 64 <= (kBN / DL::kRows) * DL::kGrp / 2, "merge exchange exceeds a staging buffer");
  float* x = reinterpret_cast<float*>(wave == 0 ? k0 : wave == 1 ? k1 : wave == 2 ? v0 : v1);
  __syncthreads();
  if (split_half == 1) {
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
#pragma unroll
      for (int rr = 0; rr < 16; ++rr) x[(dt * 16 + rr) * 64 + lane] = oacc[dt][rr];
    x[kMl + 32 * half + qi] = half ? l_tot : m_run;
  }
  __syncthreads();
  if (split_half == 1) return;
  const float m1 = x[kMl + qi];
  const float l1 = x[kMl + 32 + qi];
  const float mx = fmaxf(m_run, m1);
  const float w0 = m_run == -INFINITY ? 0.f : __builtin_amdgcn_exp2f((m_run - mx) * c);
  const float w1 = m1 == -INFINITY ? 0.f : __builtin_amdgcn_exp2f((m1 - mx) * c);
#pragma unroll
  for (int dt = 0; dt < DT; ++dt)
#pragma unroll
    for (int rr = 0; rr < 16; ++rr) oacc[dt][rr] = w0 * oacc[dt][rr] + w1 * x[(dt * 16 + rr) * 64 + lane];
  l_tot = w0 * l_tot + w1 * l1;
  if constexpr (kPartial) {
    // partial result of this key part: O relative to mx, mx and l (a row
    // whose keys in this part are all masked stores O = 0, -inf, 0)
    if (row_valid) {
      const size_t prow = (size_t)part * p.part_rows + (size_t)(q0 + t) * p.num_q_heads + h;
      float* orow = p.ws_o + prow * D;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
#pragma unroll
        for (int rg = 0; rg < 4; ++rg)
          *reinterpret_cast<float4*>(orow + dt * 32 + 8 * rg + 4 * half) =
              make_float4(oacc[dt][rg * 4], oacc[dt][rg * 4 + 1], oacc[dt][rg * 4 + 2], oacc[dt][rg * 4 + 3]);
      }
      if (half == 0) *reinterpret_cast<float2*>(p.ws_ml + 2 * prow) = make_float2(mx, l_tot);
    }
    return;
  }
  const float inv = 1.f / l_tot;
  if (row_valid) {
    uint16_t* orow = p.out + qrow;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
#pragma unroll
      for (int rg = 0; rg < 4; ++rg) {
        bf16x4 o;
#pragma unroll
        for (int u = 0; u < 4; ++u) o[u] = (__bf16)(oacc[dt][rg * 4 + u] * inv);
        *reinterpret_cast<uint2*>(orow + dt * 32 + 8 * rg + 4 * half) = __builtin_bit_cast(uint2, o);
      }
    }
  }
}

// The ping-pong kernel (D = 128 and 64).  K and V go straight from HBM into
// LDS, with no round trip through registers, and the loads of a step have
// two iterations to land in a three-deep ring of K and V buffers.  kTail:
// the work-groups from pp_grid on take the 128-row halves of the tiles of
// the launch's last round (split tiles).
// At head_dim 64 the kernel holds at most 128 VGPRs (at least four waves per
// SIMD) and 50,688 bytes of LDS (67,584 with the tail's two more buffers),
// so two work-groups share a CU.
template <int D, bool kTail>
__global__ __launch_bounds__(kPPThreads, D == 64 ? 4 : 2) void prefill_paged_attn_ppd_kernel(Params p) {
  using DL = DirectLayout<D>;
  // K and V of three steps, each in its own array so that the compiler can
  // tell a read of one from a direct load in flight into another
  constexpr int kBuf = (kBN / DL::kRows) * DL::kGrp;
  __shared__ __attribute__((aligned(16))) uint16_t k0[kBuf], k1[kBuf], k2[kBuf];
  __shared__ __attribute__((aligned(16))) uint16_t v0[kBuf], v1[kBuf], v2[kBuf];
  const int wg = blockIdx.x;
  if constexpr (kTail) {
    if (wg >= p.pp_grid) {
      // the tail's two-deep rings take two more buffers
      __shared__ __attribute__((aligned(16))) uint16_t k3[kBuf], v3[kBuf];
      ppd_split_tile<D, true>(p, wg, k0, k1, k2, k3, v0, v1, v2, v3);
      return;
    }
  }
  constexpr int KS = D / 16;     // MFMA k-steps over the head dim
  constexpr int DT = D / 32;     // 32-wide output tiles over the head dim

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int qi = lane & 31;
  const int half = lane >> 5;
  // group A (waves 0-3) runs MFMA-first, group B (waves 4-7) VALU-first; the
  // two waves of a SIMD belong to different groups
  const bool group_b = __builtin_amdgcn_readfirstlane(wave) >= 4;

  // ---- work tile: KV head fastest, then head tiles, then token tiles from
  // the last to the first, then invocations
  const int tiles_per_kv = p.head_tiles / p.num_kv_heads;
  const int g = wg % p.num_kv_heads;
  const int sub = wg / p.num_kv_heads;
  const int head_tile = g * tiles_per_kv + sub % tiles_per_kv;
  const int rest = sub / tiles_per_kv;
  const int r = rest / p.token_tiles;
  const int token_tile = p.token_tiles - 1 - rest % p.token_tiles;
  const int q0 = p.cu_q_lens[r];
  const int S = p.cu_q_lens[r + 1] - q0;
  const int t0 = token_tile * p.span;
  if (t0 >= S) return;
  const int P = p.prefix_lens[r];
  const int L = P + S;
  const int h = head_tile * p.heads_per_wg + wave % p.heads_per_wg;
  const int t = t0 + (wave / p.heads_per_wg) * kNQ + qi;   // this lane's suffix row
  const bool row_valid = t < S;
  const size_t qrow = ((size_t)(q0 + (row_valid ? t : 0)) * p.num_q_heads + h) * D;
  const int qpos = row_valid ? P + t : L - 1;               // last visible key
  const int kv_end = P + min(S, t0 + p.span);               // keys the tile needs
  const int n_steps = (kv_end + kBN - 1) / kBN;
  const int n_blk = (L + kBlock - 1) / kBlock;
  const int32_t* bt = p.block_tables + (size_t)r * p.max_blocks_per_seq;
  // first key position some row of this wave cannot see
  const int wave_qmin = P + min(t0 + (wave / p.heads_per_wg) * kNQ, S - 1);
  const size_t tile_elems = (size_t)kBlock * D;             // one (block, head)
  const size_t slot_elems = (size_t)p.num_kv_heads * tile_elems;

  // ---- Q^T operand: lane holds query qi, dims ks*16 + half*8 .. +7 -----
  bf16x8 qreg[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) {
    uint4 v = make_uint4(0, 0, 0, 0);
    if (row_valid) v = *reinterpret_cast<const uint4*>(p.q + qrow + ks * 16 + half * 8);
    qreg[ks] = as_bf16x8(v);
  }

  // ---- staging: waves 0-3 move K, waves 4-7 move V, straight from global
  // memory into LDS in the direct-to-LDS layout; wave w moves pool block
  // 4*step + (w & 3), kLoads groups of rows
  constexpr int kGrp = DL::kGrp;                       // elements from group to group
  constexpr int kLoads = kBlock / DL::kRows;           // 1 KB loads per block
  // (a local constant: with the dependent DL::kRows written into the
  // builtin's argument, this hipcc's host pass drops the kernel's launch
  // stubs without a diagnostic)
  constexpr int kGroupElems = DL::kRows * D;           // elements of one group's rows
  const int slot_u = __builtin_amdgcn_readfirstlane(wave & 3);
  const uint16_t* my_base = (group_b ? p.v_pool : p.k_pool) + (size_t)g * tile_elems;
  const __attribute__((address_space(4))) int32_t* bt_c =
      (const __attribute__((address_space(4))) int32_t*)bt;
  auto block_id = [&](int step) __attribute__((always_inline)) -> int {
    const int lb = step * (kBN / kBlock) + slot_u;
    return (step < n_steps && lb < n_blk) ? bt_c[lb] : -1;          // -1: past the end
  };
  // lane i of a load: row d = i / (D / 8) of the group, stored chunk
  // i % (D / 8), which holds the row's chunk (i % (D / 8)) ^ swz(d)
  const int dma_d = lane / (D / 8);
  const int dma_off = dma_d * D + 8 * ((lane % (D / 8)) ^ DL::swz(dma_d));
  // a block past the end loads pool slot 0 (any valid slot): its K logits
  // are masked and its V rows zeroed
  auto dma = [&](uint16_t* buf, int id) __attribute__((always_inline)) {
    const uint16_t* blk = my_base + (size_t)(id >= 0 ? id : 0) * slot_elems;
    // a buffer descriptor over the one (block, head) tile: the loads cannot leave it
    const __amdgpu_buffer_rsrc_t rs =
        __builtin_amdgcn_make_buffer_rsrc((void*)blk, (short)0, (int)(tile_elems * sizeof(uint16_t)), kRawBufferWord3);
#pragma unroll
    for (int u = 0; u < kLoads; ++u)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (__attribute__((address_space(3))) void*)(buf + (kLoads * slot_u + u) * kGrp),
                                               16, 2 * dma_off, 2 * u * kGroupElems, 0, 0);
  };
  // V rows past the end of the sequence (inside its last block, or whole
  // blocks past it) overwritten with zeros once their load has landed:
  // their probabilities are 0, but 0 times a stale NaN or Inf is NaN
  auto zero_tail = [&](uint16_t* buf, int key0) __attribute__((always_inline)) {
    if (key0 + kBlock > L) {
#pragma unroll
      for (int u = 0; u < kLoads; ++u) {
        if (key0 + DL::kRows * u + dma_d >= L)
          *reinterpret_cast<uint4*>(&buf[(kLoads * slot_u + u) * kGrp + 8 * lane]) = make_uint4(0, 0, 0, 0);
      }
    }
  };
  // K operand: row mt*32 + qi, chunk 2 ks + half.  D = 128: group 8 mt +
  // qi/4, row qi%4, stored at chunk half + 2 (ks%2) + 4 ((ks/2) ^ (qi%4));
  // D = 64: group 4 mt + qi/8, row qi%8, stored at chunk (2 ks + half) ^ y(qi%8)
  constexpr int kKoff = D == 128 ? 4 : KS;
  int koff[kKoff];
#pragma unroll
  for (int k2 = 0; k2 < kKoff; ++k2) {
    if constexpr (D == 128)
      koff[k2] = (qi >> 2) * kGrp + (qi & 3) * D + 8 * half + 32 * (k2 ^ (qi & 3));
    else
      koff[k2] = (qi >> 3) * kGrp + (qi & 7) * D + 8 * ((2 * k2 + half) ^ DL::swz(qi & 7));
  }
  auto k_addr = [&](const uint16_t* kbuf, int ks, int mt) __attribute__((always_inline)) -> const uint16_t* {
    if constexpr (D == 128) return &kbuf[mt * 8 * kGrp + 16 * (ks & 1) + koff[ks >> 1]];
    else return &kbuf[mt * 4 * kGrp + koff[ks]];
  };
  // V^T fragment for keys 16*ks2 .. +15 and dims 32*dt .. +31 from two
  // transposing reads; lane 16e + i addresses key 4*(e/2) + i/4 and dims
  // 16*(e%2) + 4*(i%4) .. +3, an 8-byte half of chunk 4 dt + jc with
  // jc = 2 (e%2) + (i%4)/2, stored at chunk 4 (dt ^ d) + jc of its row d
  // (D = 64: key 16 ks2 + tr_row of the lo read is row tr_row of group 2 ks2,
  // the hi read's the same row of group 2 ks2 + 1; the lane's 8 bytes are
  // half (lane % 2) of chunk 4 dt + 2 ((lane / 16) % 2) + (lane % 4) / 2)
  const int tr_row = 4 * (lane >> 5) + ((lane & 15) >> 2);
  int voff[DT];
  if constexpr (D == 128) {
    const int tr_d = tr_row & 3;
    const int tr_base = (tr_row >> 2) * kGrp + tr_d * D + 8 * (2 * ((lane >> 4) & 1) + ((lane & 3) >> 1)) + 4 * (lane & 1);
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) voff[dt] = tr_base + 32 * (dt ^ tr_d);
  } else {
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
      voff[dt] = tr_row * D + 8 * ((4 * dt + 2 * ((lane >> 4) & 1) + ((lane & 3) >> 1)) ^ DL::swz(tr_row)) + 4 * (lane & 1);
  }
  constexpr int kSliceGroups = 16 / DL::kRows;        // groups per 16-key slice
  auto v_frag = [&](const uint16_t* vbuf, int ks2, int dt) __attribute__((always_inline)) -> bf16x8 {
    const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(vbuf + kSliceGroups * ks2 * kGrp + voff[dt]));
    const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (lds_i16x4*)(vbuf + kSliceGroups * ks2 * kGrp + (kSliceGroups / 2) * kGrp + voff[dt]));
    const i16x4 lohi[2] = {lo, hi};
    return __builtin_bit_cast(bf16x8, lohi);
  };

  auto run = [&](auto group_tag) __attribute__((always_inline)) {
    constexpr bool kB = decltype(group_tag)::value;
    f32x16 oacc[DT];
  #pragma unroll
    for (int dt = 0; dt < DT; ++dt) oacc[dt] = f32x16{};
    f32x16 s_acc[2];             // logits of the step whose softmax is pending
    bf16x8 pb[kBN / 16];         // probabilities of the step whose PV is pending
    float m_run = -INFINITY;     // running max of the raw (unscaled) logits
    float l_part[4] = {0.f, 0.f, 0.f, 0.f};
    const float c = p.scale_log2;

    // M phase of iteration j: S_j = K_j Q^T, then O += P_{j-1} V_{j-1} (the
    // softmax of S_j can start while the PV MFMAs drain; at normal priority,
    // measured 0.5-1% faster than the other order with the priority raised)
    auto mfma_phase = [&](int j, const uint16_t* kbuf_cur, const uint16_t* vbuf_prev) __attribute__((always_inline)) {
      if (j < n_steps) {
        const uint16_t* kbuf = kbuf_cur;
        s_acc[0] = f32x16{};
        s_acc[1] = f32x16{};
  #pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
  #pragma unroll
          for (int mt = 0; mt < 2; ++mt) {
            const uint4 a = *reinterpret_cast<const uint4*>(k_addr(kbuf, ks, mt));
            s_acc[mt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(as_bf16x8(a), qreg[ks], s_acc[mt], 0, 0, 0);
          }
        }
        __builtin_amdgcn_sched_group_barrier(0x100, 4, 1);
#pragma unroll
        for (int ks = 2; ks < KS; ++ks) {
          __builtin_amdgcn_sched_group_barrier(0x008, 2, 1);
          __builtin_amdgcn_sched_group_barrier(0x100, 2, 1);
        }
        __builtin_amdgcn_sched_group_barrier(0x008, 4, 1);
      }
      __builtin_amdgcn_sched_barrier(0);
      if (j >= 1) {
        const uint16_t* vbuf = vbuf_prev;
  #pragma unroll
        for (int ks2 = 0; ks2 < kBN / 16; ++ks2) {
  #pragma unroll
          for (int dt = 0; dt < DT; ++dt)
            oacc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(v_frag(vbuf, ks2, dt), pb[ks2], oacc[dt], 0, 0, 0);
        }
        // interleave, the reads two fragments ahead of their MFMAs (12 VGPRs
        // of V fragments live instead of a whole 16-key slice's 32)
        __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
#pragma unroll
        for (int f = 2; f < DT * (kBN / 16); ++f) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
        }
        __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
      }
    };

    // V phase for step x: mask, online softmax, P_x in bf16, row sums
    auto valu_phase = [&](int x) __attribute__((always_inline)) {
      if (x < 0 || x >= n_steps) return;
      const int kstart = x * kBN;
      // accumulator register rr of tile mt holds key
      //   kstart + 32*mt + 8*(rr/4) + 4*half + rr%4   for query qi
      if (kstart + kBN - 1 > wave_qmin) {
        // key kj <= qpos  <=>  its constant offset in the step <= lim
        const int lim = qpos - kstart - 4 * half;
  #pragma unroll
        for (int mt = 0; mt < 2; ++mt) {
  #pragma unroll
          for (int rr = 0; rr < 16; ++rr)
            s_acc[mt][rr] = (mt * 32 + 8 * (rr >> 2) + (rr & 3) <= lim) ? s_acc[mt][rr] : -INFINITY;
        }
      }
      float mloc = -INFINITY;
  #pragma unroll
      for (int mt = 0; mt < 2; ++mt) {
  #pragma unroll
        for (int rr = 0; rr < 16; ++rr) mloc = fmaxf(mloc, s_acc[mt][rr]);
      }
      mloc = pair_max(mloc);
      // lazy rescale: move the reference max only when a row's max grew by
      // more than 2^8 in probability (true for every row at the first step)
      const bool grow = (mloc - m_run) * c > 8.f;
      if (__builtin_amdgcn_ballot_w64(grow) != 0) {
        const float m_new = grow ? mloc : m_run;
        const float alpha = __builtin_amdgcn_exp2f((m_run - m_new) * c);
        m_run = m_new;
  #pragma unroll
        for (int u = 0; u < 4; ++u) l_part[u] *= alpha;
  #pragma unroll
        for (int dt = 0; dt < DT; ++dt) oacc[dt] *= alpha;
      }
      const float mc = m_run * c;
      const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
  #pragma unroll
      for (int ks2 = 0; ks2 < kBN / 16; ++ks2) {
        const int mt = ks2 >> 1;
        const int rb = (ks2 & 1) * 8;
  #pragma unroll
        for (int s2 = 0; s2 < 8; ++s2)
          pb[ks2][s2] = (__bf16)__builtin_amdgcn_exp2f(__builtin_fmaf(s_acc[mt][rb + s2], c, -mc));
        // row sum over the same bf16 probabilities the PV product uses
        l_part[0] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pb[ks2], pb[ks2], 0, 1), ones, l_part[0], false);
        l_part[1] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pb[ks2], pb[ks2], 2, 3), ones, l_part[1], false);
        l_part[2] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pb[ks2], pb[ks2], 4, 5), ones, l_part[2], false);
        l_part[3] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_shufflevector(pb[ks2], pb[ks2], 6, 7), ones, l_part[3], false);
      }
    };

    // ---- prologue ------------------------------------------------------
    // K waves load K_0 and K_1, V waves V_0.  Iteration j reads K_j and
    // V_{j-1} and issues K_{j+2} (K waves) or V_{j+1} (V waves) into the
    // buffer of the step three back, read in iteration j-1; every wave issues
    // exactly kLoads loads per iteration (a step past the last loads slot 0
    // into a buffer nothing reads again), so waiting until at most kLoads are
    // in flight before the barrier completes the loads of the data read next.
    int id_next;     // block of the step the next iteration loads, read ahead
    if (!kB) {
      dma(k0, block_id(0));
      dma(k1, block_id(1));
      id_next = block_id(2);
    } else {
      dma(v0, block_id(0));
      id_next = block_id(1);
    }

    auto iteration = [&](const int j, uint16_t* kcur, uint16_t* knext2, uint16_t* vprev,
                         uint16_t* vnext) __attribute__((always_inline)) {
      // loads issued two iterations back have landed (vmcnt <= kLoads); the
      // V block read in this iteration gets its tail zeroed; then the barrier
      __builtin_amdgcn_s_waitcnt(D == 128 ? kWaitVmcnt4 : kWaitVmcnt2);
      if (kB && j >= 1) zero_tail(vprev, (j - 1) * kBN + slot_u * kBlock);
      __builtin_amdgcn_s_waitcnt(kWaitLgkmcnt0);
      asm volatile("s_barrier" ::: "memory");
      const int id = id_next;
      __builtin_amdgcn_sched_barrier(0);
      if (!kB) dma(knext2, id);                            // K_{j+2}
      else dma(vnext, id);                                 // V_{j+1}
      __builtin_amdgcn_sched_barrier(0);
      if (!kB) {
        mfma_phase(j, kcur, vprev);
        __builtin_amdgcn_sched_barrier(0);
        valu_phase(j);
      } else {
        valu_phase(j - 1);
        __builtin_amdgcn_sched_barrier(0);
        mfma_phase(j, kcur, vprev);
      }
      __builtin_amdgcn_sched_barrier(0);
      id_next = block_id(kB ? j + 2 : j + 3);
    };
    // buffers of iteration j: K_j in kb[j%3], K_{j+2} into kb[(j+2)%3],
    // V_{j-1} in vb[(j+2)%3], V_{j+1} into vb[(j+1)%3]; unrolled by three so
    // that every buffer is a constant
    int j = 0;
    for (; j + 2 <= n_steps; j += 3) {
      iteration(j, k0, k2, v2, v1);
      iteration(j + 1, k1, k0, v0, v2);
      iteration(j + 2, k2, k1, v1, v0);
    }
    if (j <= n_steps) iteration(j, k0, k2, v2, v1);
    if (j + 1 <= n_steps) iteration(j + 1, k1, k0, v0, v2);
    const float l_run = (l_part[0] + l_part[1]) + (l_part[2] + l_part[3]);
    const float l_tot = pair_sum(l_run);
    const float inv = 1.f / l_tot;
    if (row_valid) {
      uint16_t* orow = p.out + qrow;
  #pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
  #pragma unroll
        for (int rg = 0; rg < 4; ++rg) {
          bf16x4 o;
  #pragma unroll
          for (int u = 0; u < 4; ++u) o[u] = (__bf16)(oacc[dt][rg * 4 + u] * inv);
          *reinterpret_cast<uint2*>(orow + dt * 32 + 8 * rg + 4 * half) = __builtin_bit_cast(uint2, o);
        }
      }
    }

  };
  if (group_b) run(std::true_type{});
  else run(std::false_type{});
}

// Launches of less than one round of ping-pong tiles: split tiles (128 rows x
// 8 waves over two halves of the keys) with direct-to-LDS staging.  At head
// dim 64, 128 VGPRs and 67,584 bytes of LDS: two work-groups per CU.
template <int D, bool kPartial>
__global__ __launch_bounds__(kPPThreads, D == 64 ? 4 : 2) void prefill_paged_attn_ppd_split_kernel(Params p) {
  using DL = DirectLayout<D>;
  constexpr int kBuf = (kBN / DL::kRows) * DL::kGrp;
  __shared__ __attribute__((aligned(16))) uint16_t k0[kBuf], k1[kBuf], k2[kBuf], k3[kBuf];
  __shared__ __attribute__((aligned(16))) uint16_t v0[kBuf], v1[kBuf], v2[kBuf], v3[kBuf];
  ppd_split_tile<D, false, kPartial>(p, blockIdx.x, k0, k1, k2, k3, v0, v1, v2, v3);
}

// The output of a split launch with key parts: each (token, head) row
// combines its parts' partial results with the log-sum-exp weights in base
// 2 (the kernels' own units): w_p = 2^{(m_p - max m) c}, out = sum_p w_p O_p /
// sum_p w_p l_p, rounded to bf16.  Part 0 holds key 0, which every row sees,
// so the sum of weights is never empty.  D / 4 threads per row, four
// consecutive features each.
template <int D>
__global__ __launch_bounds__(kThreads) void prefill_split_merge_kernel(Params p) {
  constexpr int kTpr = D / 4;
  constexpr int kRowsPerBlock = kThreads / kTpr;
  const long long row = (long long)blockIdx.x * kRowsPerBlock + threadIdx.x / kTpr;
  if (row >= p.part_rows) return;
  const int d0 = (threadIdx.x % kTpr) * 4;
  const float c = p.scale_log2;
  float mx = -INFINITY;
  for (int q = 0; q < p.parts; ++q) mx = fmaxf(mx, p.ws_ml[2 * ((size_t)q * p.part_rows + row)]);
  float den = 0.f;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int q = 0; q < p.parts; ++q) {
    const size_t prow = (size_t)q * p.part_rows + row;
    const float2 ml = *reinterpret_cast<const float2*>(p.ws_ml + 2 * prow);
    const float w = ml.x == -INFINITY ? 0.f : __builtin_amdgcn_exp2f((ml.x - mx) * c);
    const float4 o = *reinterpret_cast<const float4*>(p.ws_o + prow * D + d0);
    den += w * ml.y;
    acc.x += w * o.x;
    acc.y += w * o.y;
    acc.z += w * o.z;
    acc.w += w * o.w;
  }
  const float inv = 1.f / den;
  bf16x4 r;
  r[0] = (__bf16)(acc.x * inv);
  r[1] = (__bf16)(acc.y * inv);
  r[2] = (__bf16)(acc.z * inv);
  r[3] = (__bf16)(acc.w * inv);
  *reinterpret_cast<uint2*>(p.out + row * D + d0) = __builtin_bit_cast(uint2, r);
}

}  // namespace

AttnGeometry attn_geometry(int batch, int max_q_len, int max_kv_len, int num_q_heads, int num_kv_heads,
                           int head_dim, int cus, bool allow_parts) {
  // one round = one ping-pong (or split) work-group per CU
  const long long kCUs = cus;
  AttnGeometry geo;
  geo.parts = 1;
  const int group = num_q_heads / num_kv_heads;
  geo.heads_per_wg = (group % 4 == 0) ? 4 : (group % 2 == 0) ? 2 : 1;
  geo.head_tiles = num_q_heads / geo.heads_per_wg;
  // ping-pong tiles of 256 rows
  geo.waves = kPPWaves;
  geo.span = kNQ * (kPPWaves / geo.heads_per_wg);
  geo.token_tiles = (max_q_len + geo.span - 1) / geo.span;
  const long long tiles = (long long)geo.token_tiles * batch * geo.head_tiles;
  geo.grid = geo.pp_grid = tiles;
  if (tiles < kCUs) {
    // less than a round: 128-row split tiles on twice as many work-groups
    // (measured faster than the ping-pong tiles up to a full round)
    geo.waves = kWaves;
    geo.span = kNQ * (kWaves / geo.heads_per_wg);
    geo.token_tiles = (max_q_len + geo.span - 1) / geo.span;
    geo.grid = (long long)geo.token_tiles * batch * geo.head_tiles;
    geo.pp_grid = 0;
    geo.split_tiles = geo.grid;
    // with a workspace, a launch that leaves at least half the CUs idle and
    // whose longest sequence has at least kMinPartedSteps key steps cuts each
    // tile's keys into parts on separate work-groups, as many as fit one
    // round (at most kMaxKeyParts), each part at least kMinPartSteps steps of
    // the longest sequence.  (Single small launches of 5-12 steps ran 0.4-1.5
    // us slower with parts, the merge launch unpaid for; 17 steps ran 22%
    // faster.)
    // (Choosing the parts by the rounds they take, so that launches of more
    // than half a round split too, was slower: a part's fixed costs of Q
    // loads, pipeline fill, half merge and partial store outweigh it.)
    const long long steps = ((long long)max_kv_len + kBN - 1) / kBN;
    if (allow_parts && geo.grid > 0 && steps >= kMinPartedSteps) {
      long long parts = std::min<long long>(kCUs / geo.grid, kMaxKeyParts);
      parts = std::min<long long>(parts, steps / kMinPartSteps);
      if (parts > 1) {
        geo.parts = (int)parts;
        geo.grid *= parts;
      }
    }
    return geo;
  }
  // a last round at most half full runs as split half tiles (whose pairs
  // must stay num_kv_heads work-groups apart, so the rounds must hold whole
  // groups of KV heads)
  const long long tail = tiles % kCUs;
  if (tiles > kCUs && tail <= kCUs / 2 && kCUs % num_kv_heads == 0) {
    geo.pp_grid = tiles - tail;
    geo.grid = geo.pp_grid + 2 * tail;
  }
  return geo;
}

hipError_t launch_prefill_paged_attn(const AttnLaunch& a, hipStream_t stream) {
  const AttnGeometry geo = attn_geometry(a.batch, a.max_q_len, a.max_kv_len, a.num_q_heads, a.num_kv_heads,
                                         a.head_dim, a.cus, a.workspace != nullptr);
  Params p;
  p.q = a.q;
  p.k_pool = a.k_pool;
  p.v_pool = a.v_pool;
  p.block_tables = a.block_tables;
  p.prefix_lens = a.prefix_lens;
  p.cu_q_lens = a.cu_q_lens;
  p.out = a.out;
  p.batch = a.batch;
  p.max_blocks_per_seq = a.max_blocks_per_seq;
  p.num_q_heads = a.num_q_heads;
  p.num_kv_heads = a.num_kv_heads;
  p.group = a.num_q_heads / a.num_kv_heads;
  p.heads_per_wg = geo.heads_per_wg;
  p.span = geo.span;
  p.token_tiles = geo.token_tiles;
  p.head_tiles = geo.head_tiles;
  p.scale_log2 = a.scale * kLog2e;
  p.pp_grid = geo.pp_grid;
  p.parts = geo.parts;
  p.split_tiles = (int)geo.split_tiles;
  p.part_rows = (long long)a.total_q * a.num_q_heads;
  p.ws_o = static_cast<float*>(a.workspace);
  p.ws_ml = p.ws_o ? p.ws_o + (size_t)geo.parts * p.part_rows * a.head_dim : nullptr;
  const dim3 grid((unsigned)geo.grid);
  if (geo.parts > 1) {
    // key parts on more work-groups, then the merge of their partials
    const long long rows_per_block = kThreads / (a.head_dim / 4);
    const dim3 mgrid((unsigned)((p.part_rows + rows_per_block - 1) / rows_per_block));
    if (a.head_dim == 128) {
      hipLaunchKernelGGL((prefill_paged_attn_ppd_split_kernel<128, true>), grid, dim3(kPPThreads), 0, stream, p);
      hipLaunchKernelGGL(prefill_split_merge_kernel<128>, mgrid, dim3(kThreads), 0, stream, p);
    } else {
      hipLaunchKernelGGL((prefill_paged_attn_ppd_split_kernel<64, true>), grid, dim3(kPPThreads), 0, stream, p);
      hipLaunchKernelGGL(prefill_split_merge_kernel<64>, mgrid, dim3(kThreads), 0, stream, p);
    }
    return hipGetLastError();
  }
  if (geo.waves == kPPWaves) {
    const bool tail = geo.grid > geo.pp_grid;
    if (a.head_dim == 128) {
      if (tail) {
        hipLaunchKernelGGL((prefill_paged_attn_ppd_kernel<128, true>), grid, dim3(kPPThreads), 0, stream, p);
      } else {
        hipLaunchKernelGGL((prefill_paged_attn_ppd_kernel<128, false>), grid, dim3(kPPThreads), 0, stream, p);
      }
    } else if (tail) {
      hipLaunchKernelGGL((prefill_paged_attn_ppd_kernel<64, true>), grid, dim3(kPPThreads), 0, stream, p);
    } else {
      hipLaunchKernelGGL((prefill_paged_attn_ppd_kernel<64, false>), grid, dim3(kPPThreads), 0, stream, p);
    }
  } else if (a.head_dim == 128) {
    // fewer than one ping-pong work-group per CU: 128-row tiles, each run
    // by 8 waves over two halves of its keys
    hipLaunchKernelGGL((prefill_paged_attn_ppd_split_kernel<128, false>), grid, dim3(kPPThreads), 0, stream, p);
  } else {
    hipLaunchKernelGGL((prefill_paged_attn_ppd_split_kernel<64, false>), grid, dim3(kPPThreads), 0, stream, p);
  }
  return hipGetLastError();
}

CascadeGeometry cascade_geometry(int num_groups, int max_group_seqs, int max_shared_len,
                                 int max_rest_len, int num_q_heads, int num_kv_heads) {
  CascadeGeometry geo;
  const int group = num_q_heads / num_kv_heads;
  geo.chunk_keys = kCascadeChunkSteps * kBN;
  geo.chunks = (max_shared_len + geo.chunk_keys - 1) / geo.chunk_keys;
  geo.segments = (max_rest_len + kCascadeSegmentKeys - 1) / kCascadeSegmentKeys;
  geo.row_tiles = ((long long)max_group_seqs * group + kRowsPerWG - 1) / kRowsPerWG;
  geo.grid = (long long)num_kv_heads * geo.row_tiles * geo.chunks * num_groups;
  return geo;
}

hipError_t launch_shared_prefix_partials(const CascadeLaunch& a, hipStream_t stream) {
  const CascadeGeometry geo = cascade_geometry(a.num_groups, a.max_group_seqs, a.max_shared_len,
                                               a.max_rest_len, a.num_q_heads, a.num_kv_heads);
  if (geo.grid == 0) return hipSuccess;
  Params p = {};
  p.q = a.q;
  p.k_pool = a.k_pool;
  p.v_pool = a.v_pool;
  p.block_tables = a.block_tables;
  p.batch = a.batch;
  p.max_blocks_per_seq = a.max_blocks_per_seq;
  p.num_q_heads = a.num_q_heads;
  p.num_kv_heads = a.num_kv_heads;
  p.group = a.num_q_heads / a.num_kv_heads;
  p.scale_log2 = a.scale * kLog2e;
  p.cu_groups = a.cu_groups;
  p.shared_lens = a.shared_lens;
  p.row_tiles = geo.row_tiles;
  p.chunk_steps = kCascadeChunkSteps;
  p.chunks = geo.chunks;
  p.ws_o = a.ws_o;
  p.ws_ml = a.ws_ml;
  p.ws_rows = a.batch * a.num_q_heads;
  const dim3 grid((unsigned)geo.grid), block(kThreads);
  if (a.head_dim == 128) {
    hipLaunchKernelGGL((shared_prefix_partials_kernel<128>), grid, block, 0, stream, p);
  } else {
    hipLaunchKernelGGL((shared_prefix_partials_kernel<64>), grid, block, 0, stream, p);
  }
  return hipGetLastError();
}

}  // namespace cs
