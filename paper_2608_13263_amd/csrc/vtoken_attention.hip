// Consumer side of the repack on CDNA4 (gfx950): the attention slot mapping and a paged
// decode attention that reads the (repacked) KV cache through it.
//
//   slot_indptr_kernel   exclusive scan of the live counts (one workgroup)
//   slot_map_kernel      one workgroup per request: wave-ballot compaction of token_slot,
//                        the live tokens' slots in logical order (Sec. 3.4: the slot mapping
//                        is built through the token table, once per token)
//   decode_split_kernel  one workgroup per (request, KV head, split of 16384/D tokens):
//                        scores of the G query heads that share the KV head on the matrix
//                        cores, split-local softmax, partial weighted sum of V on the vector
//                        ALUs (flash-decoding partials)
//   decode_combine_kernel  one workgroup per (request, query head): merges the splits
//
// Decode attention is HBM-bound up to GQA groups of about 4 (2G flops per byte of K/V);
// the score product is a small dense contraction (16 tokens x D x the G heads of a KV head)
// and runs on MFMA, which leaves the vector ALUs to the softmax and the weighted V sum, where
// a head's D elements are read by D/8 consecutive lanes, 8 elements (16 bytes of fp16 / bf16,
// 8 of fp8) each.
#include <math.h>

#include "vtoken_internal.h"

namespace vtoken {
namespace {

constexpr int kAttnThreads = 256;

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
    int v = r < a.num_reqs ? a.live_count[r] : 0;
    v = v < 0 ? 0 : v;
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
  int carry = 0;
  for (int base = 0; base < n; base += 1024) {
    const int p = base + tid;
    const int s = p < n ? a.token_slot[t0 + p] : -1;
    const bool live = s >= 0;
    const uint64_t m = __ballot(live);
    if (lane == 0) wave_tot[wave] = __popcll(m);
    __syncthreads();
    int off = carry, tot = 0;
    for (int w = 0; w < 16; ++w) {
      off += w < wave ? wave_tot[w] : 0;
      tot += wave_tot[w];
    }
    const int64_t k = (int64_t)o + off + lanes_below(m);
    if (live && k < a.slots_capacity) a.slots[k] = s;
    carry += tot;
    __syncthreads();
  }
}

// ------------------------------------------------------------------------------------------
// Paged decode attention.
// ------------------------------------------------------------------------------------------
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

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

__device__ __forceinline__ float half_bits_to_float(uint32_t h) {
  _Float16 x;
  const uint16_t s = static_cast<uint16_t>(h);
  __builtin_memcpy(&x, &s, 2);
  return static_cast<float>(x);
}

// kind 0 fp16, 1 bf16 (widening by shifts), 2 fp8: the gfx950 conversion instruction, which
// reads OCP e4m3 (no infinities, 0x7F / 0xFF are NaN).
template <int kKind>
__device__ __forceinline__ void piece_to_float(typename Piece<kKind>::type w, float* out) {
  if constexpr (kKind == 2) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const f32x2 lo = __builtin_amdgcn_cvt_pk_f32_fp8(static_cast<int>(w[i]), false);
      const f32x2 hi = __builtin_amdgcn_cvt_pk_f32_fp8(static_cast<int>(w[i]), true);
      out[4 * i] = lo.x;
      out[4 * i + 1] = lo.y;
      out[4 * i + 2] = hi.x;
      out[4 * i + 3] = hi.y;
    }
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      if constexpr (kKind == 1) {
        out[2 * i] = __uint_as_float(w[i] << 16);
        out[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
      } else {
        out[2 * i] = half_bits_to_float(w[i] & 0xFFFFu);
        out[2 * i + 1] = half_bits_to_float(w[i] >> 16);
      }
    }
  }
}

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

// kKind: element type; kD: head_dim (32, 64, 128, 256); kG: query heads per KV head (1-8).
//
// One workgroup (4 waves) covers kSplit = 16384 / kD tokens of one (request, KV head).
// Scores on the matrix cores: for a tile of 16 tokens, S[token][head] = K_tile (16 x kD) times
// Q^T (kD x 16, the kG query heads of this KV head, zero-padded), as kD/32 MFMA 16x16x32 steps;
// the float32 query is split into a high and a low 16-bit part (q = hi + lo to about 2^-17
// relative) and both are multiplied, so the scores keep float32 accuracy. Lane l holds token
// l%16 and elements 8*(l/16)..+7 of each 32-element chunk (the operand layout of the
// instruction), and receives the scores of tokens 4*(l/16)..+3 for head l%16.
// Weighted V sum on the vector ALUs: kD/8 lanes per token, 8 elements each.
// Every thread issues all of its K and V loads (8 + 8 pieces) before any arithmetic.
template <int kKind, int kD, int kG>
__global__ __launch_bounds__(kAttnThreads) void decode_split_kernel(AttnArgs a) {
  using PieceT = typename Piece<kKind>::type;
  using OpT = typename ScoreOp<kKind>::type;
  using ElemT = typename ScoreOp<kKind>::elem;
  constexpr int kElem = kKind == 2 ? 1 : 2;
  constexpr int kChunks = kD / 32;
  constexpr int kSplit = decode_split_tokens(kD);
  constexpr int kWaves = kAttnThreads / 64;
  constexpr int kTilesPerWave = kSplit / 16 / kWaves;
  constexpr int kLanes = kD / kPer;                  // V: lanes per token row
  constexpr int kTokPerPass = kAttnThreads / kLanes;
  constexpr int kIters = kSplit / kTokPerPass;       // V: tokens per thread
  static_assert(kTilesPerWave * 16 * kWaves == kSplit && kIters == kDecodeTokensPerThread,
                "split geometry");
  __shared__ float p_s[kG][kSplit];
  __shared__ float red_s[kWaves][kG];
  __shared__ float acc_s[kWaves][kG][kD];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int split = blockIdx.x % a.splits;
  const int h = (blockIdx.x / a.splits) % a.num_kv_heads;
  const int r = blockIdx.x / (a.splits * a.num_kv_heads);
  if (r >= a.num_reqs) return;
  const int s0 = a.slot_indptr[r];
  const int c = a.slot_indptr[r + 1] - s0;
  const int t0 = split * kSplit;
  if (t0 >= c || s0 < 0) return;
  const int nt = c - t0 < kSplit ? c - t0 : kSplit;
  const int* slots = a.slots + s0 + t0;
  const uint8_t* kplane = a.kv + (int64_t)(2 * a.layer) * a.plane_bytes;
  const uint8_t* vplane = kplane + a.plane_bytes;
  const int64_t head0 = (int64_t)h * kD * kElem;

  // ---- all loads first; tokens past the split's end re-read its last token (dropped later)
  const int grp = lane >> 4;    // which 8 elements of each 32-element chunk (scores)
  const int row = lane & 15;    // token of the tile (scores) / query head (operand, result)
  // query operand first (needed first): head `row` (zero past kG), scaled, split into high
  // and low parts
  OpT qh[kChunks], ql[kChunks];
  {
    const bool real = row < kG;
    const float* qrow = a.q + ((int64_t)r * a.num_q_heads + h * kG + (real ? row : 0)) * kD;
#pragma unroll
    for (int ch = 0; ch < kChunks; ++ch) {
#pragma unroll
      for (int e = 0; e < kPer; ++e) {
        // unconditional load (a padded head re-reads head 0), then a select: a conditional
        // load would wait for every outstanding K/V load
        const float qv = qrow[ch * 32 + grp * kPer + e] * a.scale;
        const float q = real ? qv : 0.f;
        const ElemT hi = static_cast<ElemT>(q);
        qh[ch][e] = hi;
        ql[ch][e] = static_cast<ElemT>(q - static_cast<float>(hi));
      }
    }
  }

  PieceT kw[kTilesPerWave][kChunks];
  bool kok[kTilesPerWave];
#pragma unroll
  for (int i = 0; i < kTilesPerWave; ++i) {
    const int t = (wave * kTilesPerWave + i) * 16 + row;
    const int sl = slots[t < nt ? t : nt - 1];
    kok[i] = static_cast<unsigned>(sl) < static_cast<unsigned>(a.num_slots);
    const uint8_t* base = kplane + (int64_t)(kok[i] ? sl : 0) * a.row_bytes + head0 +
                          grp * kPer * kElem;
#pragma unroll
    for (int ch = 0; ch < kChunks; ++ch) {
      kw[i][ch] = *reinterpret_cast<const PieceT*>(base + ch * 32 * kElem);
    }
  }
  const int piece = tid % kLanes;
  const int tg = tid / kLanes;
  PieceT vw[kIters];
  bool vok[kIters];
#pragma unroll
  for (int i = 0; i < kIters; ++i) {
    const int t = tg + i * kTokPerPass;
    const int sl = slots[t < nt ? t : nt - 1];
    vok[i] = static_cast<unsigned>(sl) < static_cast<unsigned>(a.num_slots);
    vw[i] = *reinterpret_cast<const PieceT*>(vplane + (int64_t)(vok[i] ? sl : 0) * a.row_bytes +
                                             head0 + piece * kPer * kElem);
  }

  // ---- scores
#pragma unroll
  for (int i = 0; i < kTilesPerWave; ++i) {
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ch = 0; ch < kChunks; ++ch) {
      PieceT w = kw[i][ch];
      if (!kok[i]) w = PieceT{};
      const OpT kop = k_operand<kKind>(w);
      acc = score_mfma<kKind>(kop, qh[ch], acc);
      acc = score_mfma<kKind>(kop, ql[ch], acc);
    }
    if (row < kG) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int t = (wave * kTilesPerWave + i) * 16 + grp * 4 + j;
        if (t < nt) p_s[row][t] = acc[j];
      }
    }
  }
  __syncthreads();

  // ---- split-local softmax: max and sum of exp per query head
  float m_g[kG], l_g[kG];
#pragma unroll
  for (int g = 0; g < kG; ++g) {
    float m = -INFINITY;
    for (int t = tid; t < nt; t += kAttnThreads) m = fmaxf(m, p_s[g][t]);
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) m = fmaxf(m, __shfl_xor(m, d, 64));
    if (lane == 0) red_s[wave][g] = m;
  }
  __syncthreads();
#pragma unroll
  for (int g = 0; g < kG; ++g) {
    float m = red_s[0][g];
    for (int w = 1; w < kWaves; ++w) m = fmaxf(m, red_s[w][g]);
    m_g[g] = m;
  }
  __syncthreads();
#pragma unroll
  for (int g = 0; g < kG; ++g) {
    float l = 0.f;
    for (int t = tid; t < nt; t += kAttnThreads) {
      const float e = __expf(p_s[g][t] - m_g[g]);
      p_s[g][t] = e;
      l += e;
    }
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) l += __shfl_xor(l, d, 64);
    if (lane == 0) red_s[wave][g] = l;
  }
  __syncthreads();
#pragma unroll
  for (int g = 0; g < kG; ++g) {
    float l = 0.f;
    for (int w = 0; w < kWaves; ++w) l += red_s[w][g];
    l_g[g] = l;
  }

  // ---- weighted sum of V from the registers (kG * 8 <= 64 accumulators per thread)
  float acc[kG][kPer];
#pragma unroll
  for (int g = 0; g < kG; ++g)
#pragma unroll
    for (int e = 0; e < kPer; ++e) acc[g][e] = 0.f;
#pragma unroll
  for (int i = 0; i < kIters; ++i) {
    const int t = tg + i * kTokPerPass;
    if (t < nt) {
      float vf[kPer];
      PieceT w = vw[i];
      if (!vok[i]) w = PieceT{};
      piece_to_float<kKind>(w, vf);
#pragma unroll
      for (int g = 0; g < kG; ++g) {
        const float p = p_s[g][t];
#pragma unroll
        for (int e = 0; e < kPer; ++e) acc[g][e] += p * vf[e];
      }
    }
  }
  // reduce over the token groups: inside the wave (lanes with the same piece), then across
  // waves through LDS
#pragma unroll
  for (int g = 0; g < kG; ++g)
#pragma unroll
    for (int e = 0; e < kPer; ++e)
#pragma unroll
      for (int d = kLanes; d < 64; d <<= 1) acc[g][e] += __shfl_xor(acc[g][e], d, 64);
  if (lane < kLanes) {
#pragma unroll
    for (int g = 0; g < kG; ++g)
#pragma unroll
      for (int e = 0; e < kPer; ++e) acc_s[wave][g][piece * kPer + e] = acc[g][e];
  }
  __syncthreads();
  // partial record per (request, query head, split): [m, l, acc[D]]
  for (int i = tid; i < kG * kD; i += kAttnThreads) {
    const int g = i / kD, d = i - g * kD;
    float v = 0.f;
    for (int w = 0; w < kWaves; ++w) v += acc_s[w][g][d];
    float* rec = a.workspace +
                 (((int64_t)r * a.num_q_heads + h * kG + g) * a.splits + split) * (kD + 2);
    rec[2 + d] = v;
    if (d == 0) {
      rec[0] = m_g[g];
      rec[1] = l_g[g];
    }
  }
}

// Merge of the split partials of one (request, query head): M = max of the split maxima,
// weights w_s = exp(m_s - M), out = sum_s w_s acc_s / sum_s w_s l_s. The splits are spread
// over the threads (maxima, weights) and the head elements over the threads (weighted sum,
// 128 splits per chunk with their weights in LDS), so no thread walks the splits alone.
constexpr int kCombineThreads = 128;

__device__ __forceinline__ float block_reduce(float v, bool is_max, float* red) {
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const float o = __shfl_xor(v, d, 64);
    v = is_max ? fmaxf(v, o) : v + o;
  }
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  v = red[0];
#pragma unroll
  for (int w = 1; w < kCombineThreads / 64; ++w) v = is_max ? fmaxf(v, red[w]) : v + red[w];
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
  const int c = a.slot_indptr[r + 1] - a.slot_indptr[r];
  const int D = a.head_dim;
  const int64_t rs = D + 2;  // record stride
  float* out = a.out + ((int64_t)r * a.num_q_heads + qh) * D;
  int ns = c <= 0 ? 0 : (c + a.split_tokens - 1) / a.split_tokens;
  ns = ns < a.splits ? ns : a.splits;  // the workspace holds a.splits records
  if (ns == 0) {
    for (int d = tid; d < D; d += kCombineThreads) out[d] = 0.f;
    return;
  }
  const float* rec0 = a.workspace + ((int64_t)r * a.num_q_heads + qh) * a.splits * rs;
  float m = -INFINITY;
  for (int s = tid; s < ns; s += kCombineThreads) m = fmaxf(m, rec0[s * rs]);
  const float M = block_reduce(m, true, red);
  float l = 0.f;
  for (int s = tid; s < ns; s += kCombineThreads) l += rec0[s * rs + 1] * __expf(rec0[s * rs] - M);
  const float L = block_reduce(l, false, red);
  const float inv = 1.f / L;
  // each thread owns head elements d = tid, tid + 128 (head_dim <= 256)
  float v0 = 0.f, v1 = 0.f;
  const int d0 = tid, d1 = tid + kCombineThreads;
  for (int base = 0; base < ns; base += kCombineThreads) {
    const int n = ns - base < kCombineThreads ? ns - base : kCombineThreads;
    if (tid < n) w_s[tid] = __expf(rec0[(base + tid) * rs] - M);
    __syncthreads();
    const float* rb = rec0 + (int64_t)base * rs + 2;
    int j = 0;
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

template <int kKind, int kD, int kG>
hipError_t launch_split(const AttnArgs& a, hipStream_t stream) {
  const dim3 grid(static_cast<unsigned>((int64_t)a.num_reqs * a.num_kv_heads * a.splits));
  auto kernel = decode_split_kernel<kKind, kD, kG>;
  hipLaunchKernelGGL(kernel, grid, dim3(kAttnThreads), 0, stream, a);
  return hipGetLastError();
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

hipError_t launch_slot_mapping(const SlotMapArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL(slot_indptr_kernel, dim3(1), dim3(1024), 0, stream, a);
  if (a.num_reqs > 0) {
    hipLaunchKernelGGL(slot_map_kernel, dim3(a.num_reqs), dim3(1024), 0, stream, a);
  }
  return hipGetLastError();
}

hipError_t launch_paged_decode(const AttnArgs& a, hipStream_t stream) {
  if (a.num_reqs <= 0) return hipSuccess;
  if (a.split_tokens != decode_split_tokens(a.head_dim)) return hipErrorInvalidValue;
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

}  // namespace vtoken
