// The copies of the vToken repack for CDNA4 (gfx950, wave64): they consume a plan built by
// the metadata kernels (vtoken_kernels.hip) or the partial planner (vtoken_planner.hip).
//
//   repack_direct_kernel        the out-of-place gather-repack (Sec. 3.3, 3.3.4): every live
//                               K/V row of every admitted request into packed destination
//                               blocks, all layers, K and V, all KV heads in one launch
//   repack_inplace_kernel,      in-place compaction: one workgroup walks each (request, plane)
//   repack_inplace_pipe_kernel  chain in block order (the hazard rule below)
//
// Both read the status word plan->counters[3] and do nothing when it is set, and check the
// plan's mode word plan->counters[4]. No MFMA, no arithmetic on the payload: byte movement.
#include "vtoken_internal.h"

namespace vtoken {
namespace {

// A copy handed a plan built for the other mode copies nothing and reports it in the status
// word (first error wins), so the later calls of the pass do nothing either.
__device__ __forceinline__ void plan_mode_error(int32_t* counters) {
  if (blockIdx.x == 0 && threadIdx.x == 0) atomicCAS(&counters[3], 0, VTOKEN_ERR_PLAN_MODE);
}

// Number of set bits of a wave-wide ballot in the lanes below this one.
__device__ __forceinline__ int lanes_below(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(mask >> 32),
                                   __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(mask), 0u));
}

// ------------------------------------------------------------------------------------------
// Step 2: the gather-repack. Destination block g of a plane is one contiguous chunk of
// S*row_bytes bytes at block free_list[g], whose row j comes from the source slot
// src_plan[g*S + j]. A work item is (part of destination block g, plane), a part being one
// round of kCopyThreads*kV 16-byte units (32 KiB at kV = 8): every workgroup moves one round
// whatever the block size, and a chunk of several rounds (S = 32 or 48 at 2 KiB rows) is
// spread over several workgroups. A thread loads its kV units before storing any, so every
// wave keeps kV*1 KiB of reads in flight. Rows are head_dim-contiguous, so a wave's 64 lanes
// read and write 1 KiB of consecutive bytes per instruction (a whole 2 KiB row takes two).
//
// Source slots of one destination block: with S <= 64, lane j of every wave holds
// src_plan[g*S + j] and rows are picked with a cross-lane shuffle; otherwise each unit reads
// its entry from memory. The copy is branch-free so the compiler can keep every load of a
// round in flight (a conditional load or store would force a full wait on the vector
// memory counter): lanes of padding rows (src_plan -1, the tail of a request's last block)
// load the part's first row, which the workgroup reads anyway, and their stores go through a
// buffer resource spanning only the destination chunk with an out-of-range offset, which the
// hardware drops. Padding rows are a suffix of the block, so a part whose first row is
// padding is all padding and is skipped.
// ------------------------------------------------------------------------------------------
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr uint32_t kBufferDword3 = 0x00020000u;  // raw buffer, 32-bit data format (gfx9)
constexpr uint32_t kDropOffset = 0x80000000u;    // beyond every chunk: store discarded

// Cache policies of the copy (CDNA4 cache-policy bits: sc0 = 1, nt = 2, sc1 = 16).
struct Policy {
  bool load_nt;
  int store_aux;
};
constexpr Policy kPolicies[] = {
    {true, 16},   // 0: default - non-temporal loads, sc1 stores (as 4)
    {false, 0},   // 1: plain loads, plain stores
    {true, 2},    // 2: non-temporal loads and stores
    {true, 0},    // 3: non-temporal loads, plain stores
    {true, 16},   // 4: non-temporal loads, sc1 stores
    {true, 17},   // 5: non-temporal loads, sc0 sc1 stores
    {true, 18},   // 6: non-temporal loads, sc1 nt stores
};
constexpr int kNumPolicies = sizeof(kPolicies) / sizeof(kPolicies[0]);

template <bool kNT>
__device__ __forceinline__ u32x4 load16(const u32x4* p) {
  if constexpr (kNT) {
    return __builtin_nontemporal_load(p);
  } else {
    return *p;
  }
}

// The destination pointer is the same for the whole workgroup; say so, so that the
// buffer resource lives in scalar registers.
__device__ __forceinline__ uint8_t* uniform_ptr(uint8_t* p) {
  const uint64_t x = reinterpret_cast<uint64_t>(p);
  const uint32_t lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(x));
  const uint32_t hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(x >> 32));
  return reinterpret_cast<uint8_t*>((static_cast<uint64_t>(hi) << 32) | lo);
}

template <int kPolicy, bool kSmallS, int kV>
__global__ __launch_bounds__(kCopyThreads) void repack_direct_kernel(CopyArgs a) {
  constexpr Policy pol = kPolicies[kPolicy];
  constexpr int kRound = kCopyThreads * kV;  // units of one part
  if (a.counters[3] != 0) return;
  // plans of the full pass; plans of the partial pass too, but not with the freed list of
  // vtoken_repack_free (a partial pass releases its selected sources, not table tails)
  const int mode = a.counters[4];
  if (mode != kPlanOutOfPlace && (mode != kPlanPartial || a.num_reqs > 0)) {
    plan_mode_error(a.counters);
    return;
  }
  if (static_cast<int>(blockIdx.x) >= a.copy_grid) {   // the freed list (vtoken_repack_free)
    write_freed_blocks(static_cast<int>(blockIdx.x) - a.copy_grid, a.admitted, a.bt_indptr,
                       a.freed_indptr, a.block_ids, a.num_bt_entries, a.freed,
                       a.freed_capacity);
    return;
  }
  int used = a.counters[0];
  used = used < 0 ? 0 : (used > a.max_used ? a.max_used : used);
  if (used == 0) return;
  const int P = a.num_planes;
  const int chunk = a.chunk_units;
  const int parts = (chunk + kRound - 1) / kRound;
  // gp = g * parts + part: the parts of a destination block are consecutive in both orders
  const int used_parts = used * parts;
  const int64_t items = (int64_t)used_parts * P;
  const int S = a.block_size;
  const uint32_t chunk_bytes = static_cast<uint32_t>(chunk) * 16u;
  const int U = a.row_units;
  // j = u / U as a multiply-high with floor(2^32/U)+1: exact for u < 2^20 and
  // 2 <= U <= 2^12 (checked on the host)
  const uint32_t magic = a.row_magic;
  const bool unit_rows = U == 1;  // 16-byte rows: j = u (the constant would not fit)
  const int lane = threadIdx.x & 63;
  const int tid = static_cast<int>(threadIdx.x);
  // (hi, lo) = (plane, gp) for the plane-major order, (gp, plane) for the block-major order
  const bool plane_major = a.order == 1;
  const int inner = plane_major ? used_parts : P;
  int64_t w = blockIdx.x;
  if (items < a.copy_grid) {
    // fewer items than workgroups: item k runs in workgroup floor(k * grid / items), so the
    // workgroups without an item are spread through the launch, where the dispatcher has time
    // to spare, instead of trailing it (Llama-3-8B Random: 103K of 524K, 12 us)
    const int64_t k = (w * items + a.copy_grid - 1) / a.copy_grid;
    if (k >= items || (k * a.copy_grid) / items != w) return;
    w = k;
  }
  if (w >= items) return;
  int hi = static_cast<int>(w / inner);
  int lo = static_cast<int>(w - (int64_t)hi * inner);
  const int grid = a.copy_grid;
  const int step_hi = grid / inner;
  const int step_lo = grid - step_hi * inner;

  // prefetch of the next item's destination block and plan entry (lanes >= S read entry
  // S-1 and never use it; the loads are unconditional so no branch splits the copy loop)
  const int plan_lane = lane < S ? lane : S - 1;
  int next_gp = plane_major ? lo : hi;
  int next_g = next_gp / parts;
  int next_dblk = a.free_list[next_g];
  int next_pv = kSmallS ? a.src_plan[(int64_t)next_g * S + plan_lane] : -1;

  for (; w < items; w += grid) {
    const int plane = plane_major ? hi : lo;
    const int g = next_g;
    const int part = next_gp - g * parts;
    const int dblk = __builtin_amdgcn_readfirstlane(next_dblk);
    const int pv = next_pv;
    lo += step_lo;
    hi += step_hi;
    if (lo >= inner) {
      lo -= inner;
      ++hi;
    }
    // past the last item the prefetch re-reads item 0's entries (in bounds, unused)
    next_gp = (w + grid < items) ? (plane_major ? lo : hi) : 0;
    next_g = next_gp / parts;
    next_dblk = a.free_list[next_g];
    if (kSmallS) next_pv = a.src_plan[(int64_t)next_g * S + plan_lane];

    const bool dst_ok = static_cast<unsigned>(dblk) < static_cast<unsigned>(a.num_blocks);
    const uint8_t* pbase = a.kv + (int64_t)plane * a.plane_bytes;
    uint8_t* dptr = uniform_ptr(a.kv + (int64_t)plane * a.plane_bytes +
                                (dst_ok ? (int64_t)dblk * S * a.row_bytes : 0));
    const __amdgpu_buffer_rsrc_t drsrc =
        __builtin_amdgcn_make_buffer_rsrc(dptr, 0, dst_ok ? chunk_bytes : 0u, kBufferDword3);
    const int32_t* plan = a.src_plan + (int64_t)g * S;
    const int u0 = part * kRound;
    const int j0 =
        unit_rows ? u0 : static_cast<int>(__umulhi(static_cast<uint32_t>(u0), magic));
    const int s0 = kSmallS ? __builtin_amdgcn_readlane(pv, j0)
                           : __builtin_amdgcn_readfirstlane(plan[j0]);
    // the part's first row is padding: so is the rest of the part
    if (static_cast<unsigned>(s0) >= static_cast<unsigned>(a.num_slots)) continue;
    {
      int src[kV];
      int col[kV];
      uint32_t off[kV];
#pragma unroll
      for (int v = 0; v < kV; ++v) {
        const int u = u0 + v * kCopyThreads + tid;
        const int j = unit_rows ? u : static_cast<int>(__umulhi(static_cast<uint32_t>(u), magic));
        col[v] = u - j * U;
        int s;
        if (kSmallS) {
          s = __shfl(pv, j & 63, 64);
        } else {
          s = u < chunk ? plan[j] : -1;
        }
        const bool ok =
            (u < chunk) && static_cast<unsigned>(s) < static_cast<unsigned>(a.num_slots);
        src[v] = ok ? s : s0;
        off[v] = ok ? static_cast<uint32_t>(u) * 16u : kDropOffset;
      }
      u32x4 buf[kV];
#pragma unroll
      for (int v = 0; v < kV; ++v) {
        buf[v] = load16<pol.load_nt>(
            reinterpret_cast<const u32x4*>(pbase + (int64_t)src[v] * a.row_bytes) + col[v]);
      }
#pragma unroll
      for (int v = 0; v < kV; ++v) {
        __builtin_amdgcn_raw_buffer_store_b128(buf[v], drsrc, off[v], 0, pol.store_aux);
      }
    }
  }
}

// Default launch: one workgroup per work item, for as many items as the buffers can hold
// (the device-side count is not known on the host), capped at kMaxCopyGrid workgroups; the
// kernel's grid-stride loop covers the rest, and with fewer items than workgroups it spreads
// the items over the grid (the workgroups left without one exit at once). Measured on
// MI355X, one item per workgroup beats a persistent grid sized from occupancy: the hardware
// dispatcher refills CUs as workgroups retire, while a persistent wave has to drain its
// stores before its next item's loads.
constexpr int64_t kMaxCopyGrid = 1 << 19;

template <void (*kKernel)(CopyArgs)>
hipError_t launch_kernel(const CopyArgs& a_in, int64_t items, int grid, hipStream_t stream) {
  if (grid <= 0) grid = static_cast<int>(items < kMaxCopyGrid ? items : kMaxCopyGrid);
  CopyArgs a = a_in;
  a.copy_grid = grid;
  // the freed list's workgroups follow the copy's
  const int64_t total = (int64_t)grid + a.num_reqs;
  if (total <= 0) return hipSuccess;
  hipLaunchKernelGGL(kKernel, dim3(static_cast<unsigned>(total)), dim3(kCopyThreads), 0, stream,
                     a);
  return hipGetLastError();
}

template <int kPolicy, int kV>
hipError_t launch_direct(const CopyArgs& a, int grid, hipStream_t stream) {
  // work items: every (part of a destination block, plane) the buffers can hold; the kernel
  // indexes parts with 32-bit integers
  const int64_t parts = (a.chunk_units + kCopyThreads * kV - 1) / (kCopyThreads * kV);
  if ((int64_t)a.max_used * parts > 0x7fffffff) return hipErrorInvalidValue;
  const int64_t items = (int64_t)a.max_used * parts * a.num_planes;
  if (a.block_size <= 64) {
    return launch_kernel<repack_direct_kernel<kPolicy, true, kV>>(a, items, grid, stream);
  }
  return launch_kernel<repack_direct_kernel<kPolicy, false, kV>>(a, items, grid, stream);
}

template <int kPolicy>
hipError_t launch_policy(const CopyArgs& a, int grid, hipStream_t stream) {
  // enough 16-byte units per thread to cover one chunk, at most 8
  const int per_thread = a.chunk_units / kCopyThreads;
  if (per_thread >= 8) return launch_direct<kPolicy, 8>(a, grid, stream);
  if (per_thread >= 4) return launch_direct<kPolicy, 4>(a, grid, stream);
  if (per_thread >= 2) return launch_direct<kPolicy, 2>(a, grid, stream);
  return launch_direct<kPolicy, 1>(a, grid, stream);
}

// ------------------------------------------------------------------------------------------
// In-place copy. Destination block b of request r is r's own b-th block, and the token of
// rank k sits at position p >= k, so the sources of destination block b lie in blocks >= b
// of the same request: block b may be written only after every read for blocks <= b.
// One workgroup walks one (request, plane) chain in block order: it stages the rows of
// block b that move (rows already in place are skipped) into LDS with direct 16-byte
// global->LDS loads, waits for them, synchronises, and writes them back from LDS. Reads for
// block b+1 touch blocks >= b+1 only, so they may start while block b is being written.
// With two LDS buffers one barrier per block suffices: a thread stages block b+1 into buffer
// (b+1)%2 only after passing barrier b, and every thread reaches barrier b only after its
// writes of block b-1, the last use of that buffer. With one buffer a second barrier after
// the writes protects it.
// ------------------------------------------------------------------------------------------
typedef __attribute__((address_space(3))) void* lds_ptr_t;

// kStage: 0 LDS double buffer, 1 LDS single buffer, 2 registers (no LDS; the barrier alone
// orders a block's reads before its writes, since every thread holds its own rows).
enum InplaceStage { kLdsDouble = 0, kLdsSingle = 1, kRegisters = 2 };

template <int kV, bool kSmallS, int kStage>
__global__ __launch_bounds__(kCopyThreads) void repack_inplace_kernel(InplaceArgs a) {
  extern __shared__ __attribute__((aligned(16))) uint8_t stage[];
  if (a.counters[3] != 0) return;
  if (a.counters[4] != kPlanInPlace) {
    plan_mode_error(a.counters);
    return;
  }
  const int P = a.num_planes;
  const int r = static_cast<int>(blockIdx.x / P);
  const int plane = static_cast<int>(blockIdx.x - (int64_t)r * P);
  if (r >= a.num_reqs || !a.admitted[r]) return;
  const int g0 = a.dst_indptr[r];
  const int need = a.dst_indptr[r + 1] - g0;
  const int nb0 = a.new_bt_indptr[r];
  const int S = a.block_size;
  if (g0 < 0 || need <= 0 || nb0 < 0 || (int64_t)(g0 + need) * S > a.src_plan_capacity ||
      (int64_t)nb0 + need > a.new_bt_capacity) {
    return;
  }
  const int U = a.row_units;
  const int chunk = a.chunk_units;
  const uint32_t magic = a.row_magic;
  const bool unit_rows = U == 1;
  const int tid = static_cast<int>(threadIdx.x);
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  uint8_t* pbase = a.kv + (int64_t)plane * a.plane_bytes;
  const int chunk_bytes = chunk * 16;
  const int plan_lane = lane < S ? lane : S - 1;
  // the next block's table entry and plan entry are fetched one block ahead; the barrier
  // that ends each block has retired them by the time they are used
  int next_pv = kSmallS ? a.src_plan[(int64_t)g0 * S + plan_lane] : -1;
  int next_dblk = a.new_block_ids[nb0];
  int phase = 0;

  for (int b = 0; b < need; ++b) {
    const int dblk = __builtin_amdgcn_readfirstlane(next_dblk);
    const int pv = next_pv;
    const int bn = b + 1 < need ? b + 1 : b;
    next_dblk = a.new_block_ids[nb0 + bn];
    if (kSmallS) next_pv = a.src_plan[(int64_t)(g0 + bn) * S + plan_lane];
    if (static_cast<unsigned>(dblk) >= static_cast<unsigned>(a.num_blocks)) continue;
    const int dslot0 = dblk * S;
    if (kSmallS) {
      // every wave holds the same plan row, so this ballot is uniform over the workgroup:
      // a block whose rows are all in place needs no copy and no barrier
      const bool row_moves = lane < S && static_cast<unsigned>(pv) <
                             static_cast<unsigned>(a.num_slots) && pv != dslot0 + lane;
      if (__ballot(row_moves) == 0) continue;
    }
    const int32_t* plan = a.src_plan + (int64_t)(g0 + b) * S;
    // LDS buffer of this block (offsets into `stage`: the direct-load builtin needs an
    // address derived from the shared array itself)
    const int buf = kStage == kLdsDouble ? phase * chunk_bytes : 0;
    phase ^= 1;
    int src[kV];
    int col[kV];
    bool mv[kV];
#pragma unroll
    for (int v = 0; v < kV; ++v) {
      const int u = v * kCopyThreads + tid;
      const int j = unit_rows ? u : static_cast<int>(__umulhi(static_cast<uint32_t>(u), magic));
      col[v] = u - j * U;
      if (kSmallS) {
        src[v] = __shfl(pv, j & 63, 64);
      } else {
        src[v] = u < chunk ? plan[j] : -1;
      }
      // rows already in place (source slot == destination slot) are not copied
      mv[v] = (u < chunk) && static_cast<unsigned>(src[v]) < static_cast<unsigned>(a.num_slots) &&
              src[v] != dslot0 + j;
    }
    u32x4 regs[kStage == kRegisters ? kV : 1];
#pragma unroll
    for (int v = 0; v < kV; ++v) {
      if (mv[v]) {
        // addresses in locals of non-dependent type: a template-dependent argument makes
        // the host pass drop the kernel without a diagnostic
        const uint8_t* gsrc = pbase + (int64_t)src[v] * a.row_bytes + col[v] * 16;
        if (kStage == kRegisters) {
          regs[kStage == kRegisters ? v : 0] = load16<true>(reinterpret_cast<const u32x4*>(gsrc));
        } else {
          // lane i of a wave lands at the wave's base + 16 i
          const int loff = buf + (v * kCopyThreads + wave * 64) * 16;
          __builtin_amdgcn_global_load_lds(gsrc, (lds_ptr_t)(stage + loff), 16, 0, 0);
        }
      }
    }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
#pragma unroll
    for (int v = 0; v < kV; ++v) {
      if (mv[v]) {
        const int u = v * kCopyThreads + tid;
        const u32x4 val = kStage == kRegisters
                              ? regs[kStage == kRegisters ? v : 0]
                              : *reinterpret_cast<const u32x4*>(stage + buf + u * 16);
        *reinterpret_cast<u32x4*>(pbase + (int64_t)dslot0 * a.row_bytes + (int64_t)u * 16) = val;
      }
    }
    if (kStage == kLdsSingle) __syncthreads();
  }
}

// s_waitcnt immediate (gfx9 encoding): wait until at most n vector-memory operations are
// outstanding, without waiting on the other counters.
constexpr int vmcnt_imm(int n) {
  return (n & 0xF) | (((n >> 4) & 3) << 14) | (0x7 << 4) | (0xF << 8);
}

// Pipelined in-place copy (S <= 64): the reads of the next moving block are in flight while
// the current block is written. Vector-memory counters retire in order, so a wait for a
// block's reads is only cheap when nothing after them is waited for too: the plan rows and
// destination blocks of 32 blocks at a time are staged in LDS first (one drain per 32 blocks),
// the blocks whose rows move are listed there, and the listed blocks are walked with exactly
// kV reads and kV writes per thread each, so every wait count is static: a unit that does not
// move (a row already in place inside a moving block, a padding row, past the block) reads
// the plane's first 16 bytes (one cached line) and its store goes to a dropped buffer offset.
// Hazards: the sources of destination block b lie at table positions >= b, so the reads of a
// later listed block never touch the block being written; a block is written only after the
// barrier that every thread reaches once its own reads of that block have returned, and the
// reads of earlier blocks that touched it returned before earlier barriers. Blocks left out
// of the list have all their rows in place: nothing reads from them for another block.
constexpr int kLongestFirstMaxReqs = 256;

template <int kV>
__global__ __launch_bounds__(kCopyThreads) void repack_inplace_pipe_kernel(InplaceArgs a) {
  constexpr int kChunkBlocks = 32;
  constexpr int kWaves = kCopyThreads / 64;
  __shared__ int plan_s[kChunkBlocks * 64];
  __shared__ int dblk_s[kChunkBlocks];
  __shared__ int flag_s[kChunkBlocks];
  __shared__ int list_s[kChunkBlocks];
  __shared__ int nlist_s;
  __shared__ int r_s;
  if (a.counters[3] != 0) return;
  if (a.counters[4] != kPlanInPlace) {
    plan_mode_error(a.counters);
    return;
  }
  if (a.counters[1] == 0) return;   // nothing admitted
  const int P = a.num_planes;
  // longest chains first: workgroup k*P + plane takes the request with the k-th longest
  // chain (ties by index), so the last workgroups to start are short ones and the tail of the
  // launch is short; the ranking costs O(R) per thread, so it is done for R <= 256 only
  const int k = static_cast<int>(blockIdx.x / P);
  const int plane = static_cast<int>(blockIdx.x - (int64_t)k * P);
  if (k >= a.num_reqs) return;
  int r = k;
  if (a.num_reqs <= kLongestFirstMaxReqs) {
    if (threadIdx.x == 0) r_s = k;
    __syncthreads();
    for (int i = threadIdx.x; i < a.num_reqs; i += kCopyThreads) {
      const int ni = a.admitted[i] ? a.dst_indptr[i + 1] - a.dst_indptr[i] : 0;
      int rank = 0;
      for (int j = 0; j < a.num_reqs; ++j) {
        const int nj = a.admitted[j] ? a.dst_indptr[j + 1] - a.dst_indptr[j] : 0;
        rank += (nj > ni) || (nj == ni && j < i);
      }
      if (rank == k) r_s = i;
    }
    __syncthreads();
    r = r_s;
  }
  if (!a.admitted[r]) return;
  const int g0 = a.dst_indptr[r];
  const int need = a.dst_indptr[r + 1] - g0;
  const int nb0 = a.new_bt_indptr[r];
  const int S = a.block_size;
  if (g0 < 0 || need <= 0 || nb0 < 0 || (int64_t)(g0 + need) * S > a.src_plan_capacity ||
      (int64_t)nb0 + need > a.new_bt_capacity) {
    return;
  }
  const int U = a.row_units;
  const int chunk = a.chunk_units;
  const uint32_t chunk_bytes = static_cast<uint32_t>(chunk) * 16u;
  const uint32_t magic = a.row_magic;
  const bool unit_rows = U == 1;
  const int tid = static_cast<int>(threadIdx.x);
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const uint8_t* pbase = a.kv + (int64_t)plane * a.plane_bytes;

  // kV reads per thread of listed block lb (index within the chunk, or -1 for none): the
  // moving rows, and for the other units the plane's first 16 bytes; returns which of the kV
  // units move
  auto load_block = [&](int lb, u32x4 (&regs)[kV]) -> uint32_t {
    const int dslot0 = lb >= 0 ? dblk_s[lb] * S : 0;
    const int pv = lb >= 0 ? plan_s[lb * S + (lane < S ? lane : S - 1)] : -1;
    uint32_t moving = 0;
#pragma unroll
    for (int v = 0; v < kV; ++v) {
      const int u = v * kCopyThreads + tid;
      const int j = unit_rows ? u : static_cast<int>(__umulhi(static_cast<uint32_t>(u), magic));
      const int col = u - j * U;
      const int src = __shfl(pv, j & 63, 64);
      const bool mv = u < chunk &&
                      static_cast<unsigned>(src) < static_cast<unsigned>(a.num_slots) &&
                      src != dslot0 + j;
      const int64_t off = mv ? (int64_t)src * a.row_bytes + col * 16 : 0;
      regs[v] = load16<true>(reinterpret_cast<const u32x4*>(pbase + off));
      moving |= mv ? 1u << v : 0u;
    }
    return moving;
  };
  auto store_block = [&](int lb, const u32x4 (&regs)[kV], uint32_t moving) {
    uint8_t* dptr = uniform_ptr(a.kv + (int64_t)plane * a.plane_bytes +
                                (int64_t)dblk_s[lb] * S * a.row_bytes);
    const __amdgpu_buffer_rsrc_t rsrc =
        __builtin_amdgcn_make_buffer_rsrc(dptr, 0, chunk_bytes, kBufferDword3);
#pragma unroll
    for (int v = 0; v < kV; ++v) {
      const int u = v * kCopyThreads + tid;
      const uint32_t off = (moving >> v) & 1u ? static_cast<uint32_t>(u) * 16u : kDropOffset;
      __builtin_amdgcn_raw_buffer_store_b128(regs[v], rsrc, off, 0, 16);
    }
  };

  for (int c0 = 0; c0 < need; c0 += kChunkBlocks) {
    const int nb = need - c0 < kChunkBlocks ? need - c0 : kChunkBlocks;
    __syncthreads();  // the previous chunk is done with the LDS arrays
    for (int i = tid; i < nb * S; i += kCopyThreads) {
      plan_s[i] = a.src_plan[(int64_t)(g0 + c0) * S + i];
    }
    if (tid < nb) dblk_s[tid] = a.new_block_ids[nb0 + c0 + tid];
    __syncthreads();
    // which blocks move (a block with an invalid destination is left alone)
    for (int b = wave; b < nb; b += kWaves) {
      const int dblk = dblk_s[b];
      const int pv = lane < S ? plan_s[b * S + lane] : -1;
      const bool row_moves = static_cast<unsigned>(dblk) < static_cast<unsigned>(a.num_blocks) &&
                             lane < S && static_cast<unsigned>(pv) <
                             static_cast<unsigned>(a.num_slots) && pv != dblk * S + lane;
      const uint64_t m = __ballot(row_moves);
      if (lane == 0) flag_s[b] = m != 0;
    }
    __syncthreads();
    if (wave == 0) {
      const bool f = lane < nb && flag_s[lane] != 0;
      const uint64_t m = __ballot(f);
      if (f) list_s[lanes_below(m)] = lane;
      if (lane == 0) nlist_s = __popcll(m);
    }
    __syncthreads();
    const int nl = nlist_s;
    if (nl == 0) continue;
    u32x4 ra[kV], rb[kV];
    uint32_t ma = load_block(list_s[0], ra), mb;
    // vector-memory operations retire in order (stores included): after issuing the next
    // block's kV reads, waiting until kV remain means this block's reads (and the previous
    // block's stores) are done. Past the end of the list the "next" reads are of no block
    // (-1: every unit reads the plane's first 16 bytes), so every wait count stays static.
    for (int i = 0; i < nl; i += 2) {
      mb = load_block(i + 1 < nl ? list_s[i + 1] : -1, rb);
      __builtin_amdgcn_s_waitcnt(vmcnt_imm(kV));
      __syncthreads();
      store_block(list_s[i], ra, ma);
      if (i + 1 < nl) {
        ma = load_block(i + 2 < nl ? list_s[i + 2] : -1, ra);
        __builtin_amdgcn_s_waitcnt(vmcnt_imm(kV));
        __syncthreads();
        store_block(list_s[i + 1], rb, mb);
      }
    }
  }
}

template <int kV, bool kSmallS>
hipError_t launch_inplace_v(const InplaceArgs& a, int variant, hipStream_t stream) {
  const int64_t grid = (int64_t)a.num_reqs * a.num_planes;
  const int64_t chunk_bytes = (int64_t)a.chunk_units * 16;
  // default: pipelined registers for S <= 64, else registers (measured fastest); LDS double
  // buffer when asked and two fit
  int stage = variant == 1 ? kLdsDouble : variant == 2 ? kLdsSingle : kRegisters;
  if (stage == kLdsDouble && chunk_bytes * 2 > kMaxInplaceChunkBytes) stage = kLdsSingle;
  const dim3 g(static_cast<unsigned>(grid));
  const dim3 t(kCopyThreads);
  if constexpr (kSmallS) {
    if (variant == 4 || variant == 0) {
      auto kernel = repack_inplace_pipe_kernel<kV>;
      hipLaunchKernelGGL(kernel, g, t, 0, stream, a);
      return hipGetLastError();
    }
  }
  if (stage == kLdsDouble) {
    auto kernel = repack_inplace_kernel<kV, kSmallS, kLdsDouble>;
    hipLaunchKernelGGL(kernel, g, t, static_cast<size_t>(2 * chunk_bytes), stream, a);
  } else if (stage == kLdsSingle) {
    auto kernel = repack_inplace_kernel<kV, kSmallS, kLdsSingle>;
    hipLaunchKernelGGL(kernel, g, t, static_cast<size_t>(chunk_bytes), stream, a);
  } else {
    auto kernel = repack_inplace_kernel<kV, kSmallS, kRegisters>;
    hipLaunchKernelGGL(kernel, g, t, 0, stream, a);
  }
  return hipGetLastError();
}

template <bool kSmallS>
hipError_t launch_inplace_s(const InplaceArgs& a, int variant, hipStream_t stream) {
  // units per thread that cover one chunk (at most 16: chunks are at most 64 KiB)
  const int per_thread = (a.chunk_units + kCopyThreads - 1) / kCopyThreads;
  if (per_thread <= 1) return launch_inplace_v<1, kSmallS>(a, variant, stream);
  if (per_thread <= 2) return launch_inplace_v<2, kSmallS>(a, variant, stream);
  if (per_thread <= 4) return launch_inplace_v<4, kSmallS>(a, variant, stream);
  if (per_thread <= 8) return launch_inplace_v<8, kSmallS>(a, variant, stream);
  return launch_inplace_v<16, kSmallS>(a, variant, stream);
}

}  // namespace

hipError_t launch_repack_inplace(const InplaceArgs& a, int variant, hipStream_t stream) {
  if (variant < 0 || variant > 4) return hipErrorInvalidValue;
  if ((int64_t)a.num_reqs * a.num_planes <= 0) return hipSuccess;
  if ((int64_t)a.chunk_units * 16 > kMaxInplaceChunkBytes) return hipErrorInvalidValue;
  return a.block_size <= 64 ? launch_inplace_s<true>(a, variant, stream)
                            : launch_inplace_s<false>(a, variant, stream);
}

hipError_t launch_repack(const CopyArgs& a_in, int variant, int grid, int order,
                         hipStream_t stream) {
  if (order < 0 || order > 2) return hipErrorInvalidValue;
  CopyArgs a = a_in;
  a.order = order;
  switch (variant) {
    case 0: return launch_policy<0>(a, grid, stream);
    case 1: return launch_policy<1>(a, grid, stream);
    case 2: return launch_policy<2>(a, grid, stream);
    case 3: return launch_policy<3>(a, grid, stream);
    case 4: return launch_policy<4>(a, grid, stream);
    case 5: return launch_policy<5>(a, grid, stream);
    case 6: return launch_policy<6>(a, grid, stream);
    default: return hipErrorInvalidValue;
  }
}

int num_repack_variants() { return kNumPolicies; }

}  // namespace vtoken
