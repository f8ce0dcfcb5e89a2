// Internal declarations shared by the kernels (vtoken_kernels.hip, vtoken_copy.hip,
// vtoken_attention.hip, vtoken_planner.hip, vtoken_layout.hip) and the C ABI front end
// (vtoken_abi.hip). Not installed; the public interface is include/vtoken.h.
#pragma once

#include <stdint.h>
#include <hip/hip_runtime.h>

#include "vtoken.h"

namespace vtoken {

// Launch geometry of the metadata kernels (one workgroup per request each).
constexpr int kCountThreads = 512;
constexpr int kCountThreadsShort = 128;   // for requests averaging < kLongRequestTokens
constexpr int kPlanThreads = 1024;
constexpr int kPlanBallots = 8;                            // ballots per wave per tile
constexpr int kPlanTile = kPlanThreads * kPlanBallots;     // tokens per tile (8192)
constexpr int kPlanHead = 8192;   // free-list entries a plan workgroup holds in LDS (32 KiB)
// Batches of more than kFusedAdmitReqs requests (kFusedAdmitShortReqs when their requests
// average fewer than kLongRequestTokens tokens) run the admission once, in a launch of its
// own, instead of in every plan workgroup; it stages the first kAdmitStage live counts and
// table lengths in LDS, and their plan workgroups have kPlanThreadsSplit threads.
constexpr int kFusedAdmitReqs = 512;
constexpr int kFusedAdmitShortReqs = 256;
constexpr int kLongRequestTokens = 1024;
constexpr int kAdmitStage = 4096;
constexpr int kPlanThreadsSplit = 256;
// Batches this small are planned by one workgroup in one launch (they are bound by launch
// latency); larger ones by a count launch and a plan launch of one workgroup per request.
constexpr int kSmallReqs = 24;
constexpr int kSmallTokens = 8192;
constexpr int kFreeThreads = 256;

// Copy kernel geometry: 256 threads, each moving 16-byte units.
constexpr int kCopyThreads = 256;

// The plan's mode word (plan->counters[4]), written by the kernels that build a plan and
// checked by the copy and the freed list that consume it.
constexpr int32_t kPlanOutOfPlace = 1;   // vtoken_build_token_table
constexpr int32_t kPlanInPlace = 2;      // vtoken_build_token_table_inplace
constexpr int32_t kPlanPartial = 3;      // vtoken_plan_partial: the out-of-place copy; its
                                         // released blocks are the planner state's sources

struct MetaArgs {
  // batch
  const int32_t* seq_lens;
  const int32_t* tok_indptr;
  const int32_t* bt_indptr;
  const int32_t* block_ids;
  const uint8_t* live;
  const int32_t* free_list;
  int32_t num_reqs;
  int32_t num_tokens;
  int32_t num_bt_entries;
  int32_t free_len;
  // cache geometry
  int32_t block_size;
  int32_t num_blocks;
  // plan
  int32_t* token_slot;
  int32_t* live_count;
  int32_t* admitted;
  int32_t* dst_indptr;
  int32_t* new_bt_indptr;
  int32_t* new_block_ids;
  int32_t* src_plan;
  int32_t* freed_indptr;
  int32_t* counters;
  int64_t new_bt_capacity;
  int64_t src_plan_capacity;
  int32_t inplace;          // 1: destinations are each request's own leading blocks
};

struct CopyArgs {
  uint8_t* kv;
  int64_t plane_bytes;      // num_blocks * S * row_bytes
  int64_t row_bytes;        // H * D * elem_bytes, a multiple of 16
  int32_t num_planes;       // 2 * L
  int32_t block_size;       // S
  int32_t num_blocks;
  int32_t num_slots;        // num_blocks * S
  int32_t row_units;        // row_bytes / 16
  int32_t chunk_units;      // S * row_units
  int32_t max_used;         // upper bound on counters[0] the buffers can hold
  uint32_t row_magic;       // floor(2^32 / row_units) + 1 (0 if row_units == 1)
  int32_t order;            // 1 plane-major, otherwise block-major work order
  const int32_t* src_plan;
  const int32_t* free_list;
  int32_t* counters;        // read; the status word is set if the plan's mode does not match
  int32_t copy_grid;        // workgroups of the copy (set by the launch)
  // the freed list in the same launch (vtoken_repack_free): the num_reqs workgroups after the
  // copy's write request r's released blocks; num_reqs == 0: none (vtoken_repack). freed may be
  // null when the batch has no table entries (nothing to write)
  int32_t num_reqs;
  int64_t num_bt_entries;
  const int32_t* bt_indptr;
  const int32_t* block_ids;
  const int32_t* admitted;
  const int32_t* freed_indptr;
  int32_t* freed;
  int64_t freed_capacity;
};

// The released blocks of request r, written to freed[freed_indptr[r] ..): the last
// freed_indptr[r+1] - freed_indptr[r] entries of its old table (all of it out of place, the
// part past the new table in place), for an admitted request; nothing for the others. The
// threads of the calling workgroup share the copy; ranges are checked before any access.
__device__ inline void write_freed_blocks(int r, const int32_t* admitted,
                                          const int32_t* bt_indptr, const int32_t* freed_indptr,
                                          const int32_t* block_ids, int64_t num_bt_entries,
                                          int32_t* freed, int64_t capacity) {
  if (!admitted[r]) return;
  const int b0 = bt_indptr[r];
  const int m = bt_indptr[r + 1] - b0;
  const int64_t o = freed_indptr[r];
  const int n = freed_indptr[r + 1] - freed_indptr[r];
  if (b0 < 0 || m < 0 || (int64_t)b0 + m > num_bt_entries || o < 0 || n < 0 || n > m) return;
  const int first = b0 + m - n;
  for (int j = threadIdx.x; j < n; j += blockDim.x) {
    if (o + j < capacity) freed[o + j] = block_ids[first + j];
  }
}

// Arguments of the in-place copy: one workgroup per (request, plane) chain.
struct InplaceArgs {
  uint8_t* kv;
  int64_t plane_bytes;
  int64_t row_bytes;
  int32_t num_planes;
  int32_t block_size;
  int32_t num_blocks;
  int32_t num_slots;
  int32_t row_units;
  int32_t chunk_units;
  uint32_t row_magic;
  int32_t num_reqs;
  int64_t src_plan_capacity;
  int64_t new_bt_capacity;
  const int32_t* src_plan;
  const int32_t* new_block_ids;
  const int32_t* dst_indptr;
  const int32_t* new_bt_indptr;
  const int32_t* admitted;
  int32_t* counters;        // read; the status word is set if the plan's mode does not match
};

// Largest chunk (S * row_bytes) the in-place copy stages through LDS.
constexpr int64_t kMaxInplaceChunkBytes = 64 * 1024;

// Slot mapping (live tokens' slots per request, logical order).
struct SlotMapArgs {
  int32_t num_reqs;
  int32_t num_tokens;
  const int32_t* tok_indptr;
  const int32_t* token_slot;
  const int32_t* live_count;
  const int32_t* counters;
  int32_t* slot_indptr;
  int32_t* slots;
  int64_t slots_capacity;
  int32_t reserve;        // extra room per request (slot table); 0 for a packed mapping
  int32_t* slot_count;    // slot table counts, or null
};

struct AppendArgs {
  int32_t num_reqs;
  const int32_t* append_indptr;
  const int32_t* append_slots;
  const int32_t* slot_start;
  int32_t* slot_count;
  int32_t* slots;
  int32_t* status;
};

// Paged decode attention of one layer through a slot mapping.
struct AttnArgs {
  const uint8_t* kv;
  int64_t plane_bytes;
  int64_t row_bytes;
  int32_t num_kv_heads;
  int32_t num_q_heads;
  int32_t head_dim;
  int32_t layer;
  int32_t kv_kind;   // 0 fp16, 1 bf16, 2 fp8 e4m3
  int32_t num_slots;
  int32_t num_reqs;
  int32_t splits;    // split records per (request, query head) in the workspace
  int32_t split_tokens;  // tokens per split: decode_split_tokens_w(head_dim, elem bytes, waves)
  float scale;
  const float* q;
  float* out;
  float* workspace;
  const int32_t* slot_indptr;
  const int32_t* slots;
  const int32_t* slot_count;  // null: counts from slot_indptr
};

// Arguments of the partial reclamation pass (vtoken_plan_partial).
struct PlannerArgs {
  int32_t num_reqs;
  int32_t num_tokens;
  int32_t num_bt_entries;
  int32_t block_size;
  int32_t num_blocks;
  int32_t num_slots;
  int32_t free_len;
  int32_t theta_num, theta_den;
  int32_t max_live;
  int32_t min_eligible;
  int32_t free_watermark;
  int64_t max_sources;
  const int32_t* seq_lens;
  const int32_t* tok_indptr;
  const int32_t* bt_indptr;
  const int32_t* block_ids;
  const uint8_t* live;
  const int32_t* slot_in;
  const int32_t* free_list;
  const uint8_t* pinned;  // may be null
  uint64_t* live_bits;
  int32_t* refs;
  int32_t* n_b;
  int32_t* selected;
  int32_t* elig_cum;
  int32_t* src_count;
  int32_t* sources;
  int64_t* stats;
  int32_t* token_slot;
  int32_t* live_count;
  int32_t* admitted;
  int32_t* dst_indptr;
  int32_t* new_bt_indptr;
  int32_t* new_block_ids;
  int32_t* src_plan;
  int32_t* freed_indptr;
  int32_t* counters;
  int64_t new_bt_capacity;
  int64_t src_plan_capacity;
};

hipError_t launch_planner(const PlannerArgs& a, hipStream_t stream);

hipError_t launch_slot_mapping(const SlotMapArgs& a, hipStream_t stream);
hipError_t launch_append_slots(const AppendArgs& a, hipStream_t stream);
hipError_t launch_paged_decode(const AttnArgs& a, hipStream_t stream);
// The library-held decode workspace (vtoken_paged_decode_noalloc): its size, and its address
// on the device of `stream` (looked up on the first call per device; allocates nothing).
constexpr int64_t kDecodeScratchBytes = VTOKEN_DECODE_SCRATCH_BYTES;
hipError_t decode_scratch(hipStream_t stream, float** out);
// Decode split geometry. Each wave of a split workgroup covers 8 KiB of K (and of V) of one
// KV head: 128 bytes per lane and operand. A workgroup has 4 waves, or 8 for 16-bit caches
// with GQA groups of 8, whose per-workgroup work (query operands, the merge of the waves, a
// split record of 8 heads) is then spread over twice the tokens (measured +11%; 8 waves were
// slower for fp8, whose waves already cover twice the tokens). 16-bit caches at smaller
// groups take 8 waves too when the batch's longest request spans kDecodeLongSplits 4-wave
// splits or more (half the split records: Llama-3-70B bf16, requests of 16-64K tokens, G = 1,
// 2, 4 faster by 4.8%, 4.4%, 2.8%; on the Llama-3-8B batches, ~27 splits, 8 waves were 0-4%
// slower: fewer, longer workgroups leave a longer tail).
constexpr int kDecodeWaveBytes = 8192;
constexpr int kDecodeLongSplits = 64;
constexpr int decode_split_waves(int elem_bytes, int group) {
  return elem_bytes == 2 && group == 8 ? 8 : 4;
}
// Tokens one split workgroup of `waves` waves covers (head_dim 32, 64, 128, 256 -> 512, 256,
// 128, 64 tokens for 16-bit caches with 4 waves; twice as many with 8 waves or at 1 byte per
// element).
constexpr int decode_split_tokens_w(int head_dim, int elem_bytes, int waves) {
  return waves * kDecodeWaveBytes / (head_dim * elem_bytes);
}
constexpr int decode_split_tokens(int head_dim, int elem_bytes, int group) {
  return decode_split_tokens_w(head_dim, elem_bytes, decode_split_waves(elem_bytes, group));
}
// Waves per split workgroup for a batch whose requests hold at most max_tokens slots.
constexpr int decode_waves_for(int head_dim, int elem_bytes, int group, int64_t max_tokens) {
  return elem_bytes == 2 && decode_split_waves(elem_bytes, group) == 4 &&
                 max_tokens >= (int64_t)kDecodeLongSplits *
                                   decode_split_tokens_w(head_dim, elem_bytes, 4)
             ? 8
             : decode_split_waves(elem_bytes, group);
}
// The smallest split over the element sizes and groups: the workspace bound of the C ABI.
constexpr int decode_min_split_tokens(int head_dim) {
  return decode_split_tokens(head_dim, 2, 1);
}
// Split slots per (request, KV head) in the split launch's grid. Workgroups are handed to the
// 8 XCDs in turn, so with an even count and few splits the requests' first splits, which hold
// the work, fall on the same XCDs (Llama-3-8B Random, 20 splits: one XCD 12% above the mean);
// rounding a count below 64 up to an odd one spreads them evenly (measured: that call 5%
// faster). With more splits per request the counts even out by themselves, and the odd count
// measured 0.2-0.7% slower (Llama-3-70B, 78 splits), so those keep theirs.
__host__ __device__ constexpr int decode_grid_splits(int splits) {
  return splits < 64 ? (splits | 1) : splits;
}

hipError_t launch_build(const MetaArgs& a, hipStream_t stream);
// variant: 0 default, 1 LDS double buffer, 2 LDS single buffer, 3 registers
hipError_t launch_repack_inplace(const InplaceArgs& a, int variant, hipStream_t stream);
hipError_t launch_free(const MetaArgs& a, int32_t* freed, int64_t freed_capacity,
                       hipStream_t stream);
// The layout check (vtoken_layout.hip): words[0] is the flag word, words[1 ..] one bit per
// block; layout_words() words in all.
struct LayoutArgs {
  const int32_t* block_ids;
  const int32_t* free_list;
  int64_t num_bt_entries;
  int64_t free_len;
  int32_t num_blocks;
  int64_t num_words;
  uint32_t* words;
  int32_t* status;
};
int64_t layout_words(int32_t num_blocks);
hipError_t launch_check_layout(const LayoutArgs& a, hipStream_t stream);
// variant/grid/order as in vtoken_repack_options; returns hipErrorInvalidValue for an
// unknown variant or order.
hipError_t launch_repack(const CopyArgs& a, int variant, int grid, int order,
                         hipStream_t stream);
int num_repack_variants();

// Largest chunk (S * row_bytes / 16 units) and row (row_bytes / 16 units) the copy kernel's
// multiply-high division is exact for.
constexpr int64_t kMaxChunkUnits = (1 << 20) - 1;
constexpr int64_t kMaxRowUnits = 1 << 12;

// ---- device helpers shared by the metadata kernels (vtoken_kernels.hip, vtoken_planner.hip,
// which bring them in with `using namespace vtoken::meta`)
namespace meta {

__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }

// Number of set bits of a wave-wide ballot in the lanes below this one.
__device__ __forceinline__ int lanes_below(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(mask >> 32),
                                   __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(mask), 0u));
}

// Lane i of each 16-lane row receives lane i - kN of its row, 0 for i < kN (DPP row shift).
template <int kN>
__device__ __forceinline__ int row_shr(int x) {
  static_assert(kN > 0 && kN < 16, "row shift");
  return __builtin_amdgcn_update_dpp(0, x, 0x110 + kN, 0xF, 0xF, true);
}

// Inclusive prefix sum over the 64 lanes (every lane active): within each 16-lane row by DPP
// row shifts (no LDS), then each row adds the totals of the rows below it, read from lanes
// 15, 31 and 47.
__device__ __forceinline__ int wave_inclusive_scan(int v) {
  v += row_shr<1>(v);
  v += row_shr<2>(v);
  v += row_shr<4>(v);
  v += row_shr<8>(v);
  const int t0 = __builtin_amdgcn_readlane(v, 15);
  const int t1 = __builtin_amdgcn_readlane(v, 31);
  const int t2 = __builtin_amdgcn_readlane(v, 47);
  const int row = lane_id() >> 4;
  return v + (row >= 1 ? t0 : 0) + (row >= 2 ? t1 : 0) + (row >= 3 ? t2 : 0);
}

// Inclusive prefix sum over lanes 0-15 (the first DPP row); the other rows scan their own.
__device__ __forceinline__ int row_inclusive_scan(int v) {
  v += row_shr<1>(v);
  v += row_shr<2>(v);
  v += row_shr<4>(v);
  return v + row_shr<8>(v);
}

// Exclusive scan of NV values per thread across the workgroup (at most 16 waves); total[k] is
// the sum. A wave whose values are all zero (requests past the batch's end) skips its own
// scan. The wave totals go through LDS once: lane w of every wave reads wave w's total and a
// 16-lane scan gives each wave its offset.
template <int NV>
__device__ __forceinline__ void block_exclusive_scan(int (&v)[NV], int (&total)[NV],
                                                     int (*lds)[NV]) {
  const int lane = lane_id();
  const int wave = threadIdx.x >> 6;
  const int nwaves = blockDim.x >> 6;
  int any = 0;
#pragma unroll
  for (int k = 0; k < NV; ++k) any |= v[k];
  int incl[NV];
  if (__ballot(any != 0) != 0) {
#pragma unroll
    for (int k = 0; k < NV; ++k) incl[k] = wave_inclusive_scan(v[k]);
  } else {
#pragma unroll
    for (int k = 0; k < NV; ++k) incl[k] = 0;
  }
  if (lane == 63) {
#pragma unroll
    for (int k = 0; k < NV; ++k) lds[wave][k] = incl[k];
  }
  __syncthreads();
#pragma unroll
  for (int k = 0; k < NV; ++k) {
    const int wt = row_inclusive_scan(lane < nwaves ? lds[lane][k] : 0);
    const int off = wave > 0 ? __builtin_amdgcn_readlane(wt, wave - 1) : 0;
    total[k] = __builtin_amdgcn_readlane(wt, nwaves - 1);
    v[k] = off + incl[k] - v[k];
  }
  __syncthreads();
}

// Nonzero bytes of a 32-bit word: each byte's bits are folded into its lowest bit (the bits
// shifted in from the next byte land at offsets >= 1 and are masked off).
__device__ __forceinline__ int nonzero_bytes(uint32_t w) {
  w |= w >> 4;
  w |= w >> 2;
  w |= w >> 1;
  return __popc(w & 0x01010101u);
}

// Division and remainder of non-negative positions and ranks by the block size S: shifts and
// masks when S is a power of two (the kernels that divide per token are instantiated for both).
template <bool kPow2>
struct BlockDiv {
  int s, sh;
  __device__ explicit BlockDiv(int S) : s(S), sh(__ffs(S) - 1) {}
  __device__ int div(int x) const { return kPow2 ? x >> sh : x / s; }
  __device__ int mod(int x) const { return kPow2 ? x & (s - 1) : x % s; }
};

}  // namespace meta

}  // namespace vtoken
