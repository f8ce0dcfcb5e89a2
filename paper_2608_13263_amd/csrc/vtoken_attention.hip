// Consumer side of the repack on CDNA4 (gfx950): the attention slot mapping and a paged
// decode attention that reads the (repacked) KV cache through it.
//
//   slot_indptr_kernel   exclusive scan of the live counts (one workgroup)
//   slot_map_kernel      one workgroup per request: wave-ballot compaction of token_slot,
//                        the live tokens' slots in logical order (Sec. 3.4: the slot mapping
//                        is built through the token table, once per token)
//   decode_split_kernel  one workgroup per (request, KV head, 256-token split): scores of the
//                        G query heads that share the KV head, split-local softmax, partial
//                        weighted sum of V (flash-decoding partials)
//   decode_combine_kernel  one workgroup per (request, query head): merges the splits
//
// Decode attention is HBM-bound (about G flops per byte of K/V), so the dot products run on
// the fp32 vector ALUs; K/V rows are read as 16-byte pieces, a head's D elements by a group
// of D*e/16 consecutive lanes.
#include <math.h>

#include "vtoken_internal.h"

namespace vtoken {
namespace {

constexpr int kAttnThreads = 256;
constexpr int kAttnSplit = 256;   // tokens per split workgroup

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

// OCP e4m3 (fp8, no infinities): sign, 4 exponent bits with bias 7, 3 mantissa bits.
__device__ __forceinline__ float fp8e4m3_to_float(uint32_t b) {
  const uint32_t sign = (b & 0x80u) << 24;
  const uint32_t e = (b >> 3) & 0xFu;
  const uint32_t m = b & 0x7u;
  if (e == 0xFu && m == 0x7u) return __uint_as_float(0x7FC00000u | sign);
  if (e == 0) {
    const float v = static_cast<float>(m) * 0.001953125f;  // m * 2^-9
    return sign ? -v : v;
  }
  return __uint_as_float(sign | ((e + 120u) << 23) | (m << 20));
}

__device__ __forceinline__ float half_bits_to_float(uint32_t h) {
  _Float16 x;
  const uint16_t s = static_cast<uint16_t>(h);
  __builtin_memcpy(&x, &s, 2);
  return static_cast<float>(x);
}

// A 16-byte piece of a K or V row as float: 8 values (2-byte types) or 16 (fp8); kind
// 0 fp16, 1 bf16, 2 fp8 e4m3.
template <int kKind>
__device__ __forceinline__ void piece_to_float(u32x4 w, float* out) {
  const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    if (kKind == 1) {
      out[2 * i] = __uint_as_float(ws[i] << 16);
      out[2 * i + 1] = __uint_as_float(ws[i] & 0xFFFF0000u);
    } else if (kKind == 0) {
      out[2 * i] = half_bits_to_float(ws[i] & 0xFFFFu);
      out[2 * i + 1] = half_bits_to_float(ws[i] >> 16);
    } else {
#pragma unroll
      for (int k = 0; k < 4; ++k) out[4 * i + k] = fp8e4m3_to_float((ws[i] >> (8 * k)) & 0xFFu);
    }
  }
}

// kKind: element type; kLanes: lanes per head row (D*e/16, a power of two <= 64);
// kG: query heads per KV head (GQA group), at most 8.
template <int kKind, int kLanes, int kG>
__global__ __launch_bounds__(kAttnThreads) void decode_split_kernel(AttnArgs a) {
  constexpr int kPer = kKind == 2 ? 16 : 8;          // elements per 16-byte piece
  constexpr int kD = kLanes * kPer;                  // head_dim
  constexpr int kTokPerPass = kAttnThreads / kLanes; // tokens processed per pass
  __shared__ float q_s[kG][kD];
  __shared__ float p_s[kG][kAttnSplit];
  __shared__ float red_s[kAttnThreads / 64][kG];
  __shared__ float acc_s[kAttnThreads / 64][kG][kD];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int split = blockIdx.x % a.splits;
  const int h = (blockIdx.x / a.splits) % a.num_kv_heads;
  const int r = blockIdx.x / (a.splits * a.num_kv_heads);
  if (r >= a.num_reqs) return;
  const int s0 = a.slot_indptr[r];
  const int c = a.slot_indptr[r + 1] - s0;
  const int t0 = split * kAttnSplit;
  if (t0 >= c || s0 < 0) return;
  const int nt = c - t0 < kAttnSplit ? c - t0 : kAttnSplit;
  const int* slots = a.slots + s0 + t0;

  // the G query rows of this KV head
  for (int i = tid; i < kG * kD; i += kAttnThreads) {
    const int g = i / kD, d = i - g * kD;
    q_s[g][d] = a.q[((int64_t)r * a.num_q_heads + h * kG + g) * kD + d];
  }
  __syncthreads();

  const int piece = tid % kLanes;       // which 16-byte piece of the head row
  const int tg = tid / kLanes;          // token group
  const uint8_t* kplane = a.kv + (int64_t)(2 * a.layer) * a.plane_bytes;
  const uint8_t* vplane = kplane + a.plane_bytes;
  const int64_t head_off = (int64_t)h * kD * (kKind == 2 ? 1 : 2) + piece * 16;

  // scores
  for (int t = tg; t < nt; t += kTokPerPass) {
    const int s = slots[t];
    float kf[kPer];
    const bool ok = static_cast<unsigned>(s) < static_cast<unsigned>(a.num_slots);
    u32x4 w = {0u, 0u, 0u, 0u};
    if (ok) w = *reinterpret_cast<const u32x4*>(kplane + (int64_t)s * a.row_bytes + head_off);
    piece_to_float<kKind>(w, kf);
#pragma unroll
    for (int g = 0; g < kG; ++g) {
      float acc = 0.f;
#pragma unroll
      for (int i = 0; i < kPer; ++i) acc += q_s[g][piece * kPer + i] * kf[i];
#pragma unroll
      for (int d = 1; d < kLanes; d <<= 1) acc += __shfl_xor(acc, d, 64);
      if (piece == 0) p_s[g][t] = acc * a.scale;
    }
  }
  __syncthreads();

  // split-local softmax: max and sum of exp per query head
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
    for (int w = 1; w < kAttnThreads / 64; ++w) m = fmaxf(m, red_s[w][g]);
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
    for (int w = 0; w < kAttnThreads / 64; ++w) l += red_s[w][g];
    l_g[g] = l;
  }

  // weighted sum of V over this split, kGB query heads at a time (at most 64 accumulators
  // per thread; a second pass re-reads the split's V rows from cache)
  constexpr int kGB = kG * kPer <= 64 ? kG : (64 / kPer);
  for (int g0 = 0; g0 < kG; g0 += kGB) {
    float acc[kGB][kPer];
#pragma unroll
    for (int g = 0; g < kGB; ++g)
#pragma unroll
      for (int i = 0; i < kPer; ++i) acc[g][i] = 0.f;
    for (int t = tg; t < nt; t += kTokPerPass) {
      const int s = slots[t];
      float vf[kPer];
      const bool ok = static_cast<unsigned>(s) < static_cast<unsigned>(a.num_slots);
      u32x4 w = {0u, 0u, 0u, 0u};
      if (ok) w = *reinterpret_cast<const u32x4*>(vplane + (int64_t)s * a.row_bytes + head_off);
      piece_to_float<kKind>(w, vf);
#pragma unroll
      for (int g = 0; g < kGB; ++g) {
        const float p = p_s[g0 + g][t];
#pragma unroll
        for (int i = 0; i < kPer; ++i) acc[g][i] += p * vf[i];
      }
    }
    // reduce over the token groups: inside the wave (lanes with the same piece), then across
    // waves through LDS
#pragma unroll
    for (int g = 0; g < kGB; ++g)
#pragma unroll
      for (int i = 0; i < kPer; ++i)
#pragma unroll
        for (int d = kLanes; d < 64; d <<= 1) acc[g][i] += __shfl_xor(acc[g][i], d, 64);
    if (lane < kLanes) {
#pragma unroll
      for (int g = 0; g < kGB; ++g)
#pragma unroll
        for (int i = 0; i < kPer; ++i) acc_s[wave][g0 + g][piece * kPer + i] = acc[g][i];
    }
  }
  __syncthreads();
  // partial record per (request, query head, split): [m, l, acc[D]]
  for (int i = tid; i < kG * kD; i += kAttnThreads) {
    const int g = i / kD, d = i - g * kD;
    float v = 0.f;
    for (int w = 0; w < kAttnThreads / 64; ++w) v += acc_s[w][g][d];
    float* rec = a.workspace +
                 (((int64_t)r * a.num_q_heads + h * kG + g) * a.splits + split) * (kD + 2);
    rec[2 + d] = v;
    if (d == 0) {
      rec[0] = m_g[g];
      rec[1] = l_g[g];
    }
  }
}

__global__ __launch_bounds__(64) void decode_combine_kernel(AttnArgs a) {
  const int qh = blockIdx.x % a.num_q_heads;
  const int r = blockIdx.x / a.num_q_heads;
  if (r >= a.num_reqs) return;
  const int c = a.slot_indptr[r + 1] - a.slot_indptr[r];
  const int D = a.head_dim;
  float* out = a.out + ((int64_t)r * a.num_q_heads + qh) * D;
  int ns = c <= 0 ? 0 : (c + kAttnSplit - 1) / kAttnSplit;
  ns = ns < a.splits ? ns : a.splits;  // the workspace holds a.splits records
  const float* rec0 = a.workspace + ((int64_t)r * a.num_q_heads + qh) * a.splits * (D + 2);
  float M = -INFINITY;
  for (int s = 0; s < ns; ++s) M = fmaxf(M, rec0[(int64_t)s * (D + 2)]);
  float L = 0.f;
  for (int s = 0; s < ns; ++s) {
    const float* rec = rec0 + (int64_t)s * (D + 2);
    L += rec[1] * __expf(rec[0] - M);
  }
  for (int d = threadIdx.x; d < D; d += 64) {
    float v = 0.f;
    for (int s = 0; s < ns; ++s) {
      const float* rec = rec0 + (int64_t)s * (D + 2);
      v += rec[2 + d] * __expf(rec[0] - M);
    }
    out[d] = ns ? v / L : 0.f;
  }
}

template <int kKind, int kLanes, int kG>
hipError_t launch_split(const AttnArgs& a, hipStream_t stream) {
  const dim3 grid(static_cast<unsigned>((int64_t)a.num_reqs * a.num_kv_heads * a.splits));
  auto kernel = decode_split_kernel<kKind, kLanes, kG>;
  hipLaunchKernelGGL(kernel, grid, dim3(kAttnThreads), 0, stream, a);
  return hipGetLastError();
}

template <int kKind, int kLanes>
hipError_t launch_decode_g(const AttnArgs& a, hipStream_t stream) {
  switch (a.num_q_heads / a.num_kv_heads) {
    case 1: return launch_split<kKind, kLanes, 1>(a, stream);
    case 2: return launch_split<kKind, kLanes, 2>(a, stream);
    case 4: return launch_split<kKind, kLanes, 4>(a, stream);
    case 8: return launch_split<kKind, kLanes, 8>(a, stream);
    default: return hipErrorInvalidValue;
  }
}

template <int kKind>
hipError_t launch_decode_k(const AttnArgs& a, hipStream_t stream) {
  const int lanes = a.head_dim * (kKind == 2 ? 1 : 2) / 16;
  switch (lanes) {
    case 4: return launch_decode_g<kKind, 4>(a, stream);
    case 8: return launch_decode_g<kKind, 8>(a, stream);
    case 16: return launch_decode_g<kKind, 16>(a, stream);
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

int attention_split_tokens() { return kAttnSplit; }

hipError_t launch_paged_decode(const AttnArgs& a, hipStream_t stream) {
  if (a.num_reqs <= 0) return hipSuccess;
  hipError_t e;
  switch (a.kv_kind) {
    case 0: e = launch_decode_k<0>(a, stream); break;
    case 1: e = launch_decode_k<1>(a, stream); break;
    case 2: e = launch_decode_k<2>(a, stream); break;
    default: return hipErrorInvalidValue;
  }
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(decode_combine_kernel, dim3(static_cast<unsigned>(
                         (int64_t)a.num_reqs * a.num_q_heads)), dim3(64), 0, stream, a);
  return hipGetLastError();
}

}  // namespace vtoken
