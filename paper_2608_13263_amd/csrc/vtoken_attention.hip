// Consumer side of the repack on CDNA4 (gfx950): the attention slot mapping and a paged
// decode attention that reads the (repacked) KV cache through it.
//
//   slot_indptr_kernel   exclusive scan of the live counts (one workgroup)
//   slot_map_kernel      one workgroup per request: wave-ballot compaction of token_slot,
//                        the live tokens' slots in logical order (Sec. 3.4: the slot mapping
//                        is built through the token table, once per token)
//   decode_split_kernel  one workgroup per (request, KV head, split of 32 KiB of K: 32768 /
//                        (D * element bytes) tokens): scores and the weighted sum of V of the
//                        G query heads that share the KV head, both on the matrix cores, with
//                        a split-local softmax (flash-decoding partials)
//   decode_combine_kernel  one workgroup per (request, query head): merges the splits
//
// Decode attention is HBM-bound (2G flops per byte of K/V). Both products are small dense
// contractions (16 tokens x D x the G heads of a KV head, and their transposes) and run on
// MFMA, which leaves the vector ALUs to the softmax and the operand conversions.
#include <math.h>

#include <atomic>
#include <mutex>

#include "vtoken_internal.h"

namespace vtoken {
namespace {


__device__ __forceinline__ int lanes_below(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(mask >> 32),
                                   __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(mask), 0u));
}

// ------------------------------------------------------------------------------------------
// Slot mapping.
// ------------------------------------------------------------------------------------------
__global__ __launch_bounds__(1024) void slot_indptr_kernel(SlotMapArgs a) {
  __shared__ int wave_tot[16];
  if (a.counters[3] != 0) return;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  int carry = 0;
  for (int base = 0; base < a.num_reqs; base += 1024) {
    const int r = base + tid;
    int live = r < a.num_reqs ? a.live_count[r] : 0;
    live = live < 0 ? 0 : live;
    if (r < a.num_reqs && a.slot_count != nullptr) a.slot_count[r] = live;
    int v = r < a.num_reqs ? live + a.reserve : 0;
    int incl = v;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const int t = __shfl_up(incl, d, 64);
      if (lane >= d) incl += t;
    }
    if (lane == 63) wave_tot[wave] = incl;
    __syncthreads();
    int off = carry, tot = 0;
    for (int w = 0; w < 16; ++w) {
      off += w < wave ? wave_tot[w] : 0;
      tot += wave_tot[w];
    }
    if (r < a.num_reqs) a.slot_indptr[r] = off + incl - v;
    carry += tot;
    __syncthreads();
  }
  if (tid == 0) a.slot_indptr[a.num_reqs] = carry;
}

// One workgroup per request compacts its live token slots in logical order: tiles of
// 16 waves x kSlotBallots x 64 tokens, every token_slot load of a tile in flight before its
// ballots, one pair of barriers per tile.
constexpr int kSlotBallots = 8;

__global__ __launch_bounds__(1024) void slot_map_kernel(SlotMapArgs a) {
  __shared__ int wave_tot[16];
  if (a.counters[3] != 0) return;
  const int r = blockIdx.x;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int t0 = a.tok_indptr[r];
  const int n = a.tok_indptr[r + 1] - t0;
  const int o = a.slot_indptr[r];
  if (t0 < 0 || n < 0 || (int64_t)t0 + n > a.num_tokens || o < 0) return;
  const int32_t* ts = a.token_slot + t0;
  int carry = 0;
  for (int base = 0; base < n; base += 1024 * kSlotBallots) {
    // wave w holds positions base + w*64*kSlotBallots + k*64 + lane
    const int wbase = base + wave * (64 * kSlotBallots);
    int s[kSlotBallots];
#pragma unroll
    for (int k = 0; k < kSlotBallots; ++k) {
      const int p = wbase + k * 64 + lane;
      s[k] = p < n ? ts[p] : -1;
    }
    int rank[kSlotBallots];
    int local = 0;
#pragma unroll
    for (int k = 0; k < kSlotBallots; ++k) {
      const uint64_t m = __ballot(s[k] >= 0);
      rank[k] = local + lanes_below(m);
      local += __popcll(m);
    }
    if (lane == 0) wave_tot[wave] = local;
    __syncthreads();
    int off = carry, tot = 0;
    for (int w = 0; w < 16; ++w) {
      off += w < wave ? wave_tot[w] : 0;
      tot += wave_tot[w];
    }
#pragma unroll
    for (int k = 0; k < kSlotBallots; ++k) {
      const int64_t dst = (int64_t)o + off + rank[k];
      if (s[k] >= 0 && dst < a.slots_capacity) a.slots[dst] = s[k];
    }
    carry += tot;
    __syncthreads();
  }
}

// Append-only growth of a slot table: one workgroup per request copies its new slots after
// its current ones if its region has room.
__global__ __launch_bounds__(256) void append_status_kernel(AppendArgs a) {
  if (threadIdx.x == 0) a.status[0] = 0;
}

__global__ __launch_bounds__(256) void append_slots_kernel(AppendArgs a) {
  const int r = blockIdx.x;
  const int a0 = a.append_indptr[r];
  const int n = a.append_indptr[r + 1] - a0;
  if (n <= 0) return;
  const int start = a.slot_start[r];
  const int cap = a.slot_start[r + 1] - start;
  const int cnt = a.slot_count[r];
  if (a0 < 0 || cnt < 0 || (int64_t)cnt + n > cap) {
    if (threadIdx.x == 0) atomicCAS(a.status, 0, VTOKEN_ERR_CAPACITY);
    return;
  }
  for (int i = threadIdx.x; i < n; i += 256) a.slots[start + cnt + i] = a.append_slots[a0 + i];
  __syncthreads();
  if (threadIdx.x == 0) a.slot_count[r] = cnt + n;
}

// ------------------------------------------------------------------------------------------
// Paged decode attention.
// ------------------------------------------------------------------------------------------
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kPer = 8;  // elements of a head row per lane

// Eight consecutive elements of a K or V head row: 16 bytes of fp16 / bf16, 8 bytes of fp8.
template <int kKind>
struct Piece {
  typedef u32x4 type;
};
template <>
struct Piece<2> {
  typedef u32x2 type;
};

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// The matrix-core operand type of the scores: fp16 caches multiply in fp16, bf16 and fp8
// caches in bf16 (every e4m3 value is exact in bf16).
template <int kKind>
struct ScoreOp {
  typedef bf16x8 type;
  typedef __bf16 elem;
};
template <>
struct ScoreOp<0> {
  typedef f16x8 type;
  typedef _Float16 elem;
};

template <int kKind>
__device__ __forceinline__ f32x4 score_mfma(typename ScoreOp<kKind>::type k,
                                            typename ScoreOp<kKind>::type q, f32x4 acc) {
  if constexpr (kKind == 0) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(k, q, acc, 0, 0, 0);
  } else {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(k, q, acc, 0, 0, 0);
  }
}

// Eight K elements as a matrix-core operand: the 16 loaded bytes as they are (fp16, bf16), or
// 8 fp8 bytes widened to bf16 by the gfx950 conversion instruction (scale 1).
template <int kKind>
__device__ __forceinline__ typename ScoreOp<kKind>::type k_operand(
    typename Piece<kKind>::type w) {
  if constexpr (kKind == 2) {
    bf16x8 o;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const bf16x2 a = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(static_cast<int>(w[i]), 1.f,
                                                                 false);
      const bf16x2 b = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(static_cast<int>(w[i]), 1.f,
                                                                 true);
      o[4 * i] = a.x;
      o[4 * i + 1] = a.y;
      o[4 * i + 2] = b.x;
      o[4 * i + 3] = b.y;
    }
    return o;
  } else {
    return __builtin_bit_cast(typename ScoreOp<kKind>::type, w);
  }
}

typedef short i16x4 __attribute__((ext_vector_type(4)));

// Eight V elements as 16-bit values of the matrix-core type: fp16 / bf16 as loaded, fp8
// widened to bf16 (exact).
template <int kKind>
__device__ __forceinline__ u32x4 v_row16(typename Piece<kKind>::type w) {
  if constexpr (kKind == 2) {
    return __builtin_bit_cast(u32x4, k_operand<2>(w));
  } else {
    return w;
  }
}

// LDS transpose read of gfx950 (ds_read_b64_tr_b16): in each group of 16 lanes, lane
// 4a + b receives element b of the four 16-bit values addressed by lanes a, a+4, a+8 and
// a+12 of its group (in that order).
__device__ __forceinline__ i16x4 lds_read_tr16(const uint8_t* lds_addr) {
  typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (lds_i16x4*)(reinterpret_cast<uintptr_t>(lds_addr)));
}

// Cross-lane steps of the decode without the LDS crossbar (ds_bpermute): DPP rotations inside
// 16-lane rows and the gfx950 row swaps (v_permlane16_swap, v_permlane32_swap). Every lane of
// the wave must be active.
//
// Lane i of each 16-lane row receives lane (i - kN) mod 16 of its row.
template <int kN>
__device__ __forceinline__ float row_ror(float x) {
  static_assert(kN > 0 && kN < 16, "row rotation");
  return __int_as_float(
      __builtin_amdgcn_update_dpp(0, __float_as_int(x), 0x120 + kN, 0xF, 0xF, false));
}

// x combined with the value of lane i ^ 16 (kDist 16) or i ^ 32 (kDist 32): the swap leaves
// the even rows' values in one result and the odd rows' (the low half's and the high half's)
// in the other, in every lane.
template <int kDist, bool kMax>
__device__ __forceinline__ float xor_combine(float x) {
  const uint32_t u = __float_as_uint(x);
  float a, b;
  if constexpr (kDist == 16) {
    const auto r = __builtin_amdgcn_permlane16_swap(u, u, false, false);
    a = __uint_as_float(r[0]);
    b = __uint_as_float(r[1]);
  } else {
    static_assert(kDist == 32, "16 or 32");
    const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
    a = __uint_as_float(r[0]);
    b = __uint_as_float(r[1]);
  }
  return kMax ? fmaxf(a, b) : a + b;
}

// Sum (or maximum) over the lanes i, i + kStride, i + 2 kStride, ... of the wave (kStride a
// power of two below 64); every lane receives its class's result.
template <int kStride, bool kMax>
__device__ __forceinline__ float lanes_reduce(float x) {
  if constexpr (kStride <= 1) x = kMax ? fmaxf(x, row_ror<1>(x)) : x + row_ror<1>(x);
  if constexpr (kStride <= 2) x = kMax ? fmaxf(x, row_ror<2>(x)) : x + row_ror<2>(x);
  if constexpr (kStride <= 4) x = kMax ? fmaxf(x, row_ror<4>(x)) : x + row_ror<4>(x);
  if constexpr (kStride <= 8) x = kMax ? fmaxf(x, row_ror<8>(x)) : x + row_ror<8>(x);
  if constexpr (kStride <= 16) x = xor_combine<16, kMax>(x);
  return xor_combine<32, kMax>(x);
}

// Minimum waves per SIMD the decode kernels are compiled for. The fp8 geometries with
// head_dim 64 or 128, and the 16-bit ones up to head_dim 128, come out a few registers above
// the four-wave budget (128 registers); held to it they do not spill (fp8: 5-10% faster).
// Elsewhere the compiler's choice stands (fp8 with head_dim 32 or 256 would spill).
constexpr int decode_min_waves(int kind, int head_dim) {
  return kind == 2 ? (head_dim == 64 || head_dim == 128 ? 4 : 1) : (head_dim <= 128 ? 4 : 1);
}

// Split kernel of the paged decode, both products on the matrix cores.
//
// kKind: element type; kD: head_dim (32, 64, 128, 256); kG: query heads per KV head (1, 2,
// 4, 8; smaller groups leave operand columns as zero padding).
//
// One workgroup (kWaves = 4 waves, 8 for 16-bit caches at kG = 8) covers kSplit = kWaves *
// 8192 / (kD * element bytes) tokens of one (request, KV head); wave w owns tokens
// [w*kTW, (w+1)*kTW), kTW = kSplit / kWaves, and computes
// for them, on the matrix cores (MFMA 16x16x32, fp16 for fp16 caches, bf16 otherwise; fp8
// widened to bf16):
//   scores  S[token][col] = K_tile (16 x kD) . Q2^T (kD x 16). The float32 query is split into
//           high and low 16-bit parts (q = hi + lo to ~2^-17): column c < 8 of Q2 is the high
//           part of head c, column c + 8 its low part (zero for c >= kG), so one product
//           carries both and the score of head c is S[.][c] + S[.][c + 8] (float32 accuracy);
//   weights p = exp(score - m_w) with the wave's own maximum m_w per head, l_w = sum of p;
//   values  O2[row][d] = P2 (16 x 32 tokens) . V (32 tokens x 16 elements) per 16-element
//           chunk, row c < 8 of P2 the high part of head c's weights, row c + 8 their low
//           part, so O_w[c] = O2[c] + O2[c + 8]. V goes through a per-wave LDS window of 32
//           rows, one 32-token k-step at a time (16-bit rows, padded by 32 bytes against bank
//           conflicts), and comes back in operand layout by transpose reads. The operand
//           layout fixes which tokens a lane holds: lane l has column l%16 and, of each
//           32-token chunk, tokens 4*(l/16)..+3 of its first 16-token tile and the same of its
//           second; the V rows are read in that order.
// The waves are merged with the usual max-rescaling into the split's record.
// Every thread issues all of its K and V loads (128 + 128 bytes) before any arithmetic.
// Non-finite K or V values are outside the contract (a zero weight times an infinite value
// gives NaN).
template <int kKind, int kD, int kG, int kWaves>
__global__ __launch_bounds__(64 * kWaves)
__attribute__((amdgpu_waves_per_eu(decode_min_waves(kKind, kD))))
void decode_split_kernel(AttnArgs a) {
  using PieceT = typename Piece<kKind>::type;
  using OpT = typename ScoreOp<kKind>::type;
  using ElemT = typename ScoreOp<kKind>::elem;
  constexpr int kElem = kKind == 2 ? 1 : 2;
  constexpr int kChunks = kD / 32;                   // score k-steps
  constexpr int kSplit = decode_split_tokens_w(kD, kElem, kWaves);
  constexpr int kThreads = 64 * kWaves;
  constexpr int kTW = kSplit / kWaves;               // tokens per wave: 16 .. 256
  constexpr int kTiles = kTW / 16;                   // 16-token score tiles per wave
  constexpr int kKC = (kTiles + 1) / 2;              // 32-token value k-steps per wave
  constexpr int kDC = kD / 16;                       // 16-element value chunks
  constexpr int kPerV = kKind == 2 ? 16 : kPer;      // V elements per lane load: 16 bytes
  constexpr int kLanesV = kD / kPerV;                // V load: lanes per token row
  constexpr int kTokV = 64 / kLanesV;                // V load: tokens per wave pass
  constexpr int kItV = kTW / kTokV;                  // V load: pieces per lane
  constexpr int kWin = kTW < 32 ? kTW : 32;          // V rows a wave stages per k-step
  constexpr int kItW = kWin / kTokV;                 // V pieces per lane per k-step
  constexpr int kRowB = kD * 2 + 32;                 // LDS bytes per V row
  static_assert(kTiles * 16 == kTW && kItW * kKC == kItV && kItW * kTokV == kWin,
                "split geometry");
  static_assert(kG >= 1 && kG <= 8, "the high and low parts fill the 16 operand columns");
  constexpr int kVB = kWaves * kWin * kRowB;
  constexpr int kMergeB = kWaves * kG * (kD + 2) * 4;
  constexpr int kLdsB = kVB > kMergeB ? kVB : kMergeB;
  __shared__ __attribute__((aligned(16))) uint8_t lds[kLdsB];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  // the grid holds decode_grid_splits(a.splits) split slots per (request, KV head); one past
  // a.splits (a count rounded up to an odd one) returns at once
  const int gs = decode_grid_splits(a.splits);
  const int split = blockIdx.x % gs;
  const int h = (blockIdx.x / gs) % a.num_kv_heads;
  const int r = blockIdx.x / (gs * a.num_kv_heads);
  if (r >= a.num_reqs || split >= a.splits) return;
  const int s0 = a.slot_indptr[r];
  const int c = a.slot_count != nullptr ? a.slot_count[r] : a.slot_indptr[r + 1] - s0;
  const int t0 = split * kSplit;
  if (t0 >= c || s0 < 0) return;
  const int nt = c - t0 < kSplit ? c - t0 : kSplit;
  const int* slots = a.slots + s0 + t0;
  const uint8_t* kplane = a.kv + (int64_t)(2 * a.layer) * a.plane_bytes;
  const uint8_t* vplane = kplane + a.plane_bytes;
  const int64_t head0 = (int64_t)h * kD * kElem;
  const int grp = lane >> 4;    // operand k-group / result row group
  const int row = lane & 15;    // token of a tile (K operand) / column (Q) / row (P)
  const int wt0 = wave * kTW;   // first token of this wave

  const bool low = row >= 8;          // this lane's column / P row holds low parts
  const bool real = (row & 7) < kG;   // column / P row of a query head (else zero padding)
  // The query operand of column `row` is head row % 8 (padding columns re-read head 0: the
  // load is unconditional, since a conditional load would wait for every outstanding K/V
  // load). Every wave needs the same operands: they are built once per workgroup into LDS and
  // read after a barrier.
  // The head dims of a k-chunk's lane group: any assignment gives the same dot products as
  // long as q and K use the same one. fp8 pairs the chunks (2c, 2c+1) so that a lane's two
  // 8-byte K pieces are 16 contiguous bytes, read by one load.
  constexpr bool kPairK = kKind == 2 && kChunks % 2 == 0;
  auto head_dim_of = [&](int ch, int e) {
    return kPairK ? (ch >> 1) * 64 + grp * 16 + (ch & 1) * 8 + e : ch * 32 + grp * kPer + e;
  };
  __shared__ OpT q_s[kChunks][64];
  // ---- loads in two rounds: the query values and every slot index this lane needs, then
  // (once the slots are in) every K and V load back to back; the query operands are built
  // while those are in flight. The vector-memory counter retires loads in order, so a slot
  // read issued after a K load would hold that slot's K pieces until the earlier K load
  // returned: interleaving slot reads with K and V loads cost a round trip per tile.
  constexpr int kQC = (kChunks + kWaves - 1) / kWaves;   // query chunks a wave builds
  const float* qrow =
      a.q + ((int64_t)r * a.num_q_heads + h * kG + (real ? row & 7 : 0)) * kD;
  float qraw[kQC][kPer];
#pragma unroll
  for (int c = 0; c < kQC; ++c) {
    // unconditional (a chunk past the last re-reads the last one, unused)
    const int ch = wave + c * kWaves < kChunks ? wave + c * kWaves : kChunks - 1;
#pragma unroll
    for (int e = 0; e < kPer; ++e) qraw[c][e] = qrow[head_dim_of(ch, e)];
  }
  // slot indices of this lane's K tiles and V pieces; tokens past the split's end re-read
  // its last token
  int ksl[kTiles];
#pragma unroll
  for (int i = 0; i < kTiles; ++i) {
    const int t = wt0 + i * 16 + row;
    ksl[i] = slots[t < nt ? t : nt - 1];
  }
  const int vpiece = lane % kLanesV;
  int vsl[kItV];
#pragma unroll
  for (int i = 0; i < kItV; ++i) {
    const int t = wt0 + lane / kLanesV + i * kTokV;
    vsl[i] = slots[t < nt ? t : nt - 1];
  }
  // (the scheduler keeps these reads ahead of the K and V loads, and those ahead of the query
  // operands' arithmetic)
  __builtin_amdgcn_sched_barrier(0);

  // ---- all K and V loads
  PieceT kw[kTiles][kChunks];
  bool kok[kTiles];
#pragma unroll
  for (int i = 0; i < kTiles; ++i) {
    const int sl = ksl[i];
    kok[i] = static_cast<unsigned>(sl) < static_cast<unsigned>(a.num_slots);
    const uint8_t* row_base = kplane + (int64_t)(kok[i] ? sl : 0) * a.row_bytes + head0;
    if constexpr (kPairK) {
#pragma unroll
      for (int p = 0; p < kChunks / 2; ++p) {
        const u32x4 w = *reinterpret_cast<const u32x4*>(row_base + p * 64 + grp * 16);
        kw[i][2 * p] = PieceT{w.x, w.y};
        kw[i][2 * p + 1] = PieceT{w.z, w.w};
      }
    } else {
      const uint8_t* base = row_base + grp * kPer * kElem;
#pragma unroll
      for (int ch = 0; ch < kChunks; ++ch) {
        kw[i][ch] = *reinterpret_cast<const PieceT*>(base + ch * 32 * kElem);
      }
    }
  }
  // V rows: 16 bytes per lane (8 elements at 16 bits, 16 fp8), a whole head row per kLanesV
  // lanes, read with non-temporal loads (each line is used by one instruction; measured
  // +2-6% over plain loads). The K pieces above stay plain: in the matrix-core operand order
  // a row's line is split over two instructions, and non-temporal K loads were slower.
  u32x4 vw[kItV];
#pragma unroll
  for (int i = 0; i < kItV; ++i) {
    const int sl = vsl[i];
    const bool ok = static_cast<unsigned>(sl) < static_cast<unsigned>(a.num_slots);
    vw[i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(
        vplane + (int64_t)(ok ? sl : 0) * a.row_bytes + head0 + vpiece * 16));
  }

  __builtin_amdgcn_sched_barrier(0);
  // ---- query operands (column `row` = head row % 8, scaled; its high part for row < 8, its
  // low part for row >= 8): wave w builds chunks w, w + kWaves, ... for all 64 lanes into LDS
#pragma unroll
  for (int c = 0; c < kQC; ++c) {
    const int ch = wave + c * kWaves;
    if (ch < kChunks) {
      OpT qv8;
#pragma unroll
      for (int e = 0; e < kPer; ++e) {
        const float q = real ? qraw[c][e] * a.scale : 0.f;
        const ElemT hi = static_cast<ElemT>(q);
        qv8[e] = low ? static_cast<ElemT>(q - static_cast<float>(hi)) : hi;
      }
      q_s[ch][lane] = qv8;
    }
  }

  // ---- scores of this wave's tiles: lane holds tokens wt0 + 16i + 4*grp + j of head row % 8
  // (columns row and row ^ 8 summed: lanes row and row + 8 then hold the same scores); the
  // K/V loads above stay in flight across the barrier
  __syncthreads();  // query operands in LDS
  OpT qop[kChunks];
#pragma unroll
  for (int ch = 0; ch < kChunks; ++ch) qop[ch] = q_s[ch][lane];
  f32x4 sc[kTiles];
#pragma unroll
  for (int i = 0; i < kTiles; ++i) {
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ch = 0; ch < kChunks; ++ch) {
      acc = score_mfma<kKind>(k_operand<kKind>(kw[i][ch]), qop[ch], acc);
    }
    // a slot outside the pool (its row was read at slot 0) poisons the request: NaN score;
    // tokens past the split's end get weight zero
    const uint64_t okm = __ballot(kok[i]);            // bit k: token k of the tile
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      acc[j] += row_ror<8>(acc[j]);
      if (!((okm >> (4 * grp + j)) & 1)) acc[j] = __builtin_nanf("");
      if (wt0 + 16 * i + 4 * grp + j >= nt) acc[j] = -INFINITY;
    }
    sc[i] = acc;
  }

  // ---- V rows of k-step kc into this wave's LDS window
  uint8_t* vwin = lds + wave * kWin * kRowB;
  auto stage_v = [&](int kc) {
#pragma unroll
    for (int ii = 0; ii < kItW; ++ii) {
      const u32x4 w = vw[kc * kItW + ii];
      uint8_t* dst = vwin + (lane / kLanesV + ii * kTokV) * kRowB + vpiece * kPerV * 2;
      if constexpr (kKind == 2) {   // 16 fp8 values -> 16 bf16 values (32 bytes)
        *reinterpret_cast<u32x4*>(dst) = v_row16<kKind>(u32x2{w.x, w.y});
        *reinterpret_cast<u32x4*>(dst + 16) = v_row16<kKind>(u32x2{w.z, w.w});
      } else {
        *reinterpret_cast<u32x4*>(dst) = w;
      }
    }
  };
  stage_v(0);

  // ---- wave-local softmax per head (the four lanes of a column share `row`)
  float m = -INFINITY;
#pragma unroll
  for (int i = 0; i < kTiles; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) m = fmaxf(m, sc[i][j]);
  m = lanes_reduce<16, true>(m);
  const float msafe = m == -INFINITY ? 0.f : m;   // a wave with no valid token
  float l = 0.f;
#pragma unroll
  for (int i = 0; i < kTiles; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      sc[i][j] = __expf(sc[i][j] - msafe);
      l += sc[i][j];
    }
  l = lanes_reduce<16, false>(l);

  // ---- O_w = P . V on the matrix cores, one 32-token k-step at a time; the V rows of a
  // k-step go through this wave's LDS window (rows past the split's end weigh zero), the first
  // k-step's before the softmax above
  f32x4 o[kDC];
#pragma unroll
  for (int dc = 0; dc < kDC; ++dc) o[dc] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int kc = 0; kc < kKC; ++kc) {
    if (kc > 0) {
      __syncthreads();  // the previous k-step's reads of the window are done
      stage_v(kc);
    }
    __syncthreads();  // V rows written (each wave reads only its own window)
    // A operand: row `row` (head row % 8, high or low part), tokens 4*grp..+3 of tile 2kc
    // then of tile 2kc+1 (zero if absent)
    OpT pop;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int tile = 2 * kc + (j >> 2);
      const float p = tile < kTiles ? sc[tile < kTiles ? tile : 0][j & 3] : 0.f;
      const ElemT hi = static_cast<ElemT>(p);
      pop[j] = low ? static_cast<ElemT>(p - static_cast<float>(hi)) : hi;
    }
    // B operand rows: lane 16*grp + rho supplies the row of token 4*grp + rho/4 of the first
    // tile (then of the second), elements 4*(rho%4)..+3 of the 16-element chunk
    const int t1 = 4 * grp + row / 4;                                  // window rows
    const int t2 = (2 * kc + 1 < kTiles ? 16 : 0) + 4 * grp + row / 4;
    const uint8_t* r1 = vwin + t1 * kRowB + (row % 4) * 8;
    const uint8_t* r2 = vwin + t2 * kRowB + (row % 4) * 8;
#pragma unroll
    for (int dc = 0; dc < kDC; ++dc) {
      const i16x4 x1 = lds_read_tr16(r1 + dc * 32);
      const i16x4 x2 = lds_read_tr16(r2 + dc * 32);
      typedef short i16x8 __attribute__((ext_vector_type(8)));
      const i16x8 xv = {x1[0], x1[1], x1[2], x1[3], x2[0], x2[1], x2[2], x2[3]};
      const OpT vop = __builtin_bit_cast(OpT, xv);
      o[dc] = score_mfma<kKind>(pop, vop, o[dc]);
    }
  }
  // result rows 4*grp + j: high parts in lane groups 0, 1 (heads 0-7), low parts 32 lanes up
#pragma unroll
  for (int dc = 0; dc < kDC; ++dc)
#pragma unroll
    for (int j = 0; j < 4; ++j) o[dc][j] = xor_combine<32, false>(o[dc][j]);
  __syncthreads();  // the LDS rows are reused for the merge

  // ---- merge the waves: [m_w, l_w] and O_w[head][d] per wave into LDS
  float* mrg = reinterpret_cast<float*>(lds);        // [wave][head][kD + 2]
  if (grp == 0 && row < kG) {
    mrg[(wave * kG + row) * (kD + 2)] = m;
    mrg[(wave * kG + row) * (kD + 2) + 1] = l;
  }
  if (grp < 2) {
#pragma unroll
    for (int dc = 0; dc < kDC; ++dc)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int g = 4 * grp + j;                     // result row = head
        if (g < kG) mrg[(wave * kG + g) * (kD + 2) + 2 + dc * 16 + row] = o[dc][j];
      }
  }
  __syncthreads();
  for (int i = tid; i < kG * kD; i += kThreads) {
    const int g = i / kD, d = i - g * kD;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) M = fmaxf(M, mrg[(w * kG + g) * (kD + 2)]);
    float v = 0.f, L = 0.f;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const float* wr = mrg + (w * kG + g) * (kD + 2);
      const float f = wr[0] == -INFINITY ? 0.f : __expf(wr[0] - M);
      v += wr[2 + d] * f;
      L += wr[1] * f;
    }
    float* rec = a.workspace +
                 (((int64_t)r * a.num_q_heads + h * kG + g) * a.splits + split) * (kD + 2);
    rec[2 + d] = v;
    if (d == 0) {
      rec[0] = M;
      rec[1] = L;
    }
  }
}

// Merge of the split partials of one (request, query head): M = max of the split maxima,
// weights w_s = exp(m_s - M), out = sum_s w_s acc_s / sum_s w_s l_s. The splits are spread
// over the threads (maxima, weights) and the head elements over the threads (weighted sum,
// 128 splits per chunk with their weights in LDS), so no thread walks the splits alone.
// Each thread reads the (m_s, l_s) pair of its first split once, and the values of the first
// kCombinePre splits are loaded before the two reductions, so that the call waits for about
// two dependent rounds of loads instead of four; the remaining splits go 8, then 4 at a time.
constexpr int kCombineThreads = 128;
constexpr int kCombinePre = 8;

template <bool kMax>
__device__ __forceinline__ float block_reduce(float v, float* red) {
  v = lanes_reduce<1, kMax>(v);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  v = red[0];
#pragma unroll
  for (int w = 1; w < kCombineThreads / 64; ++w) v = kMax ? fmaxf(v, red[w]) : v + red[w];
  __syncthreads();
  return v;
}

__global__ __launch_bounds__(kCombineThreads) void decode_combine_kernel(AttnArgs a) {
  __shared__ float red[kCombineThreads / 64];
  __shared__ float w_s[kCombineThreads];
  const int qh = blockIdx.x % a.num_q_heads;
  const int r = blockIdx.x / a.num_q_heads;
  if (r >= a.num_reqs) return;
  const int tid = threadIdx.x;
  const int s0 = a.slot_indptr[r];
  const int c = a.slot_count != nullptr ? a.slot_count[r] : a.slot_indptr[r + 1] - s0;
  const int D = a.head_dim;
  const int64_t rs = D + 2;  // record stride
  float* out = a.out + ((int64_t)r * a.num_q_heads + qh) * D;
  const int ns = c <= 0 ? 0 : (c + a.split_tokens - 1) / a.split_tokens;
  // a malformed slot range (the split kernel computed nothing for it), or more slots than
  // max_tokens (the splits past the workspace were never computed): NaN
  if (s0 < 0 || c < 0 || ns > a.splits) {
    for (int d = tid; d < D; d += kCombineThreads) out[d] = __builtin_nanf("");
    return;
  }
  if (ns == 0) {
    for (int d = tid; d < D; d += kCombineThreads) out[d] = 0.f;
    return;
  }
  const float* rec0 = a.workspace + ((int64_t)r * a.num_q_heads + qh) * a.splits * rs;
  // each thread owns head elements d = tid, tid + 128 (head_dim <= 256)
  const int d0 = tid, d1 = tid + kCombineThreads;
  float p0[kCombinePre], p1[kCombinePre];
#pragma unroll
  for (int j = 0; j < kCombinePre; ++j) {
    p0[j] = j < ns && d0 < D ? rec0[j * rs + 2 + d0] : 0.f;
    p1[j] = j < ns && d1 < D ? rec0[j * rs + 2 + d1] : 0.f;
  }
  // (m_s, l_s) of split s = tid, both issued before either is used
  float m0 = -INFINITY, l0 = 0.f;
  if (tid < ns) {
    m0 = rec0[tid * rs];
    l0 = rec0[tid * rs + 1];
  }
  float m = m0;
  for (int s = tid + kCombineThreads; s < ns; s += kCombineThreads) m = fmaxf(m, rec0[s * rs]);
  const float M = block_reduce<true>(m, red);
  const float w0 = tid < ns ? __expf(m0 - M) : 0.f;
  float l = tid < ns ? l0 * w0 : 0.f;
  for (int s = tid + kCombineThreads; s < ns; s += kCombineThreads) {
    l += rec0[s * rs + 1] * __expf(rec0[s * rs] - M);
  }
  const float L = block_reduce<false>(l, red);
  const float inv = 1.f / L;
  float v0 = 0.f, v1 = 0.f;
  for (int base = 0; base < ns; base += kCombineThreads) {
    const int n = ns - base < kCombineThreads ? ns - base : kCombineThreads;
    if (tid < n) w_s[tid] = base == 0 ? w0 : __expf(rec0[(base + tid) * rs] - M);
    __syncthreads();
    const float* rb = rec0 + (int64_t)base * rs + 2;
    int j = 0;
    if (base == 0) {
#pragma unroll
      for (int i = 0; i < kCombinePre; ++i) {
        if (i < n) {
          v0 += p0[i] * w_s[i];
          v1 += p1[i] * w_s[i];
        }
      }
      j = n < kCombinePre ? n : kCombinePre;
    }
    for (; j + 8 <= n; j += 8) {
      if (d0 < D) {
        float x[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) x[u] = rb[(j + u) * rs + d0];
#pragma unroll
        for (int u = 0; u < 8; ++u) v0 += x[u] * w_s[j + u];
      }
      if (d1 < D) {
        float x[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) x[u] = rb[(j + u) * rs + d1];
#pragma unroll
        for (int u = 0; u < 8; ++u) v1 += x[u] * w_s[j + u];
      }
    }
    for (; j + 4 <= n; j += 4) {
      if (d0 < D) {
        v0 += rb[j * rs + d0] * w_s[j] + rb[(j + 1) * rs + d0] * w_s[j + 1] +
              rb[(j + 2) * rs + d0] * w_s[j + 2] + rb[(j + 3) * rs + d0] * w_s[j + 3];
      }
      if (d1 < D) {
        v1 += rb[j * rs + d1] * w_s[j] + rb[(j + 1) * rs + d1] * w_s[j + 1] +
              rb[(j + 2) * rs + d1] * w_s[j + 2] + rb[(j + 3) * rs + d1] * w_s[j + 3];
      }
    }
    for (; j < n; ++j) {
      if (d0 < D) v0 += rb[j * rs + d0] * w_s[j];
      if (d1 < D) v1 += rb[j * rs + d1] * w_s[j];
    }
    __syncthreads();
  }
  if (d0 < D) out[d0] = v0 * inv;
  if (d1 < D) out[d1] = v1 * inv;
}

template <int kKind, int kD, int kG, int kWaves>
hipError_t launch_split_w(const AttnArgs& a, hipStream_t stream) {
  const dim3 grid(
      static_cast<unsigned>((int64_t)a.num_reqs * a.num_kv_heads * decode_grid_splits(a.splits)));
  auto kernel = decode_split_kernel<kKind, kD, kG, kWaves>;
  hipLaunchKernelGGL(kernel, grid, dim3(64 * kWaves), 0, stream, a);
  return hipGetLastError();
}

// the split size the host chose (decode_waves_for) selects the workgroup's waves
template <int kKind, int kD, int kG>
hipError_t launch_split(const AttnArgs& a, hipStream_t stream) {
  constexpr int kElem = kKind == 2 ? 1 : 2;
  constexpr int kBase = decode_split_waves(kElem, kG);
  if constexpr (kElem == 2 && kBase == 4) {
    if (a.split_tokens == decode_split_tokens_w(kD, kElem, 8)) {
      return launch_split_w<kKind, kD, kG, 8>(a, stream);
    }
  }
  return launch_split_w<kKind, kD, kG, kBase>(a, stream);
}

template <int kKind, int kD>
hipError_t launch_decode_g(const AttnArgs& a, hipStream_t stream) {
  switch (a.num_q_heads / a.num_kv_heads) {
    case 1: return launch_split<kKind, kD, 1>(a, stream);
    case 2: return launch_split<kKind, kD, 2>(a, stream);
    case 4: return launch_split<kKind, kD, 4>(a, stream);
    case 8: return launch_split<kKind, kD, 8>(a, stream);
    default: return hipErrorInvalidValue;
  }
}

template <int kKind>
hipError_t launch_decode_k(const AttnArgs& a, hipStream_t stream) {
  switch (a.head_dim) {
    case 32: return launch_decode_g<kKind, 32>(a, stream);
    case 64: return launch_decode_g<kKind, 64>(a, stream);
    case 128: return launch_decode_g<kKind, 128>(a, stream);
    case 256: return launch_decode_g<kKind, 256>(a, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_append_slots(const AppendArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL(append_status_kernel, dim3(1), dim3(64), 0, stream, a);
  if (a.num_reqs > 0) {
    hipLaunchKernelGGL(append_slots_kernel, dim3(a.num_reqs), dim3(256), 0, stream, a);
  }
  return hipGetLastError();
}

hipError_t launch_slot_mapping(const SlotMapArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL(slot_indptr_kernel, dim3(1), dim3(1024), 0, stream, a);
  if (a.num_reqs > 0) {
    hipLaunchKernelGGL(slot_map_kernel, dim3(a.num_reqs), dim3(1024), 0, stream, a);
  }
  return hipGetLastError();
}

hipError_t launch_paged_decode(const AttnArgs& a, hipStream_t stream) {
  if (a.num_reqs <= 0) return hipSuccess;
  const int elem = a.kv_kind == 2 ? 1 : 2;
  const int group = a.num_q_heads / a.num_kv_heads;
  if (a.split_tokens != decode_split_tokens(a.head_dim, elem, group) &&
      (elem != 2 || a.split_tokens != decode_split_tokens_w(a.head_dim, elem, 8))) {
    return hipErrorInvalidValue;
  }
  hipError_t e;
  switch (a.kv_kind) {
    case 0: e = launch_decode_k<0>(a, stream); break;
    case 1: e = launch_decode_k<1>(a, stream); break;
    case 2: e = launch_decode_k<2>(a, stream); break;
    default: return hipErrorInvalidValue;
  }
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(decode_combine_kernel, dim3(static_cast<unsigned>(
                         (int64_t)a.num_reqs * a.num_q_heads)), dim3(kCombineThreads), 0,
                     stream, a);
  return hipGetLastError();
}

// Split partials of vtoken_paged_decode_noalloc: a library-held workspace for callers that
// cannot allocate. Each GPU that loads the library holds its own copy of the array until the
// process ends; its address on a device is looked up once, with that device current, and kept.
// The name below stands for the array only in device code: host code uses the address.
static __device__ __align__(256) float scratch[kDecodeScratchBytes / 4];

namespace {
constexpr int kMaxScratchDevices = 64;
std::atomic<void*> g_scratch_ptr[kMaxScratchDevices];
std::mutex g_scratch_mu;
}  // namespace

hipError_t decode_scratch(hipStream_t stream, float** out) {
  int cur = 0;
  hipError_t e = hipGetDevice(&cur);
  if (e != hipSuccess) return e;
  int dev = cur;
  if (stream != nullptr) {
    e = hipStreamGetDevice(stream, &dev);
    if (e != hipSuccess) return e;
  }
  if (dev < 0 || dev >= kMaxScratchDevices) return hipErrorInvalidDevice;
  void* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (p == nullptr) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    p = g_scratch_ptr[dev].load(std::memory_order_relaxed);
    if (p == nullptr) {
      // the lookup is per device and needs the stream's device current
      if (dev != cur && (e = hipSetDevice(dev)) != hipSuccess) return e;
      e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
      if (dev != cur) {
        const hipError_t back = hipSetDevice(cur);
        if (e == hipSuccess) e = back;
      }
      if (e != hipSuccess) return e;
      if (p == nullptr) return hipErrorInvalidSymbol;
      g_scratch_ptr[dev].store(p, std::memory_order_release);
    }
  }
  *out = static_cast<float*>(p);
  return hipSuccess;
}

}  // namespace vtoken
