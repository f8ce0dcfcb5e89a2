// The paper's partial reclamation pass (Sec. 3.3) on CDNA4 (gfx950): per-block liveness,
// the waste-ratio trigger, low-utilisation sources under a bound B, the move list and the
// token-table update. The copy itself is the same gather kernel as the full pass (a source
// plan per destination block), launched by vtoken_repack.
//
//   pl_clear_kernel    zero the per-block live bitmaps and reference counts, the statistics
//                      and the counters
//   pl_count_kernel    references of every block over all tables; one bit per live slot
//                      (a slot held live by several requests of a shared prefix counts once)
//   pl_blocks_request_kernel  two kinds of workgroups in one launch: up to 128 compute
//                      n_b = live bits of each allocated block (Sec. 2.3.1, Sec. 3.3.1) and
//                      the totals behind the waste ratio F; one per request finds its live
//                      count and its candidate blocks (unshared, unpinned, n_b <= max_live) in
//                      table order with their cumulative live tokens
//   pl_admit_kernel    one workgroup: the trigger (F > theta_F, enough candidates, free list at
//                      or below the watermark, Sec. 3.3.2), the bound B over the candidates in
//                      request order, T_live, ceil(T_live / S), strict gain, admission against
//                      the free list, and every CSR offset (Sec. 3.3.3); one wave with wave
//                      scans for at most 64 requests
//   pl_table_kernel    one workgroup per request: selected sources, new block table (kept
//                      blocks then destinations), released sources, and the move list in
//                      logical order written as token slots and the per-destination source
//                      plan (Sec. 3.3.3, Sec. 3.2 apply_moves); tokens in tiles of 8192 with
//                      every load of a tile in flight before its ballots
//
// Every kernel after pl_count_kernel does nothing once plan->counters[3] holds an error;
// every dereference of caller data is bounds-checked.
#include "vtoken_internal.h"

namespace vtoken {
namespace {

using namespace vtoken::meta;

constexpr int kPlThreads = 256;
constexpr int kPlWaves = kPlThreads / 64;
constexpr int kPlAdmitThreads = 1024;
constexpr int kPlAdmitWaves = kPlAdmitThreads / 64;
constexpr int kPlTableThreads = 1024;
constexpr int kPlTableWaves = kPlTableThreads / 64;
constexpr int kPlBallots = 8;                          // 64-token ballots per wave per tile
constexpr int kPlTile = kPlTableThreads * kPlBallots;  // tokens per tile (8192)
constexpr int kPlDestLds = 4096;   // destinations of a request held in LDS (16 KiB)

__device__ __forceinline__ void pl_error(int32_t* counters, int code) {
  atomicCAS(&counters[3], 0, code);
}

// Rank of `flag` among the flagged threads of the workgroup (kWaves waves; ballots), and
// their count.
template <int kWaves = kPlWaves>
__device__ __forceinline__ int pl_rank(bool flag, int* total, int* lds) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const uint64_t m = __ballot(flag);
  if (lane == 0) lds[wave] = __popcll(m);
  __syncthreads();
  int off = 0, t = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    const int x = lds[w];
    off += w < wave ? x : 0;
    t += x;
  }
  __syncthreads();
  *total = t;
  return off + lanes_below(m);
}

// n_b of block b if it is a candidate source (unshared, unpinned, n_b <= max_live), else -1;
// n_b from the block's live bits, so that it does not wait for pl_blocks (the same launch)
__device__ __forceinline__ int pl_candidate_live(const PlannerArgs& a, int b) {
  if (b < 0 || b >= a.num_blocks) return -1;
  if (a.refs[b] != 1) return -1;                         // shared-prefix blocks never move
  if (a.pinned != nullptr && a.pinned[b] != 0) return -1;
  const int n = __popcll(a.live_bits[b]);
  return n <= a.max_live ? n : -1;
}

__global__ __launch_bounds__(256) void pl_clear_kernel(PlannerArgs a) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < a.num_blocks;
       i += stride) {
    a.live_bits[i] = 0ull;
    a.refs[i] = 0;
  }
  if (blockIdx.x == 0 && threadIdx.x < 8) a.stats[threadIdx.x] = 0;
  // the plan's mode word: the partial pass's plan is copied by the out-of-place copy, and its
  // released blocks are the state's sources (vtoken_free_blocks refuses it)
  if (blockIdx.x == 0 && threadIdx.x < 5) {
    a.counters[threadIdx.x] = threadIdx.x == 4 ? kPlanPartial : 0;
  }
}

// OR over the 64 lanes (every lane active): DPP row rotations, then the gfx950 row swaps.
__device__ __forceinline__ uint32_t wave_or(uint32_t x) {
  x |= static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(x), 0x121, 0xF,
                                                         0xF, false));
  x |= static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(x), 0x122, 0xF,
                                                         0xF, false));
  x |= static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(x), 0x124, 0xF,
                                                         0xF, false));
  x |= static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(x), 0x128, 0xF,
                                                         0xF, false));
  const auto r16 = __builtin_amdgcn_permlane16_swap(x, x, false, false);
  x = r16[0] | r16[1];
  const auto r32 = __builtin_amdgcn_permlane32_swap(x, x, false, false);
  return r32[0] | r32[1];
}

// References of every table entry's block; one bit per live slot. Tokens go 64 to a wave:
// the bits of the wave's tokens that fall in one block are ORed across the wave and set with
// one atomic (up to 8 blocks per wave; a wave's remaining tokens set their bits one by one).
template <bool kPow2>
__global__ __launch_bounds__(256) void pl_count_kernel(PlannerArgs a) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < a.num_bt_entries;
       i += stride) {
    const int b = a.block_ids[i];
    if (b < 0 || b >= a.num_blocks) {
      pl_error(a.counters, VTOKEN_ERR_BLOCK_RANGE);
    } else {
      atomicAdd(&a.refs[b], 1);
    }
  }
  const BlockDiv<kPow2> bd(a.block_size);
  const int lane = threadIdx.x & 63;
  const int64_t waves = stride / 64;
  for (int64_t w0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) / 64 * 64;
       w0 < a.num_tokens; w0 += waves * 64) {
    const int64_t t = w0 + lane;
    const bool lv = t < a.num_tokens && a.live[t] != 0;
    const int s = lv ? a.slot_in[t] : -1;
    const bool bad = lv && (s < 0 || s >= a.num_slots);
    if (bad) pl_error(a.counters, VTOKEN_ERR_SLOT);
    const bool ok = lv && !bad;
    const int blk = ok ? bd.div(s) : -1;
    const int off = ok ? bd.mod(s) : 0;
    uint64_t pending = __ballot(ok);
    for (int it = 0; it < 8 && pending != 0; ++it) {
      const int leader = __builtin_ctzll(pending);
      const int lb = __builtin_amdgcn_readlane(blk, leader);
      const bool mine = ok && blk == lb;
      const uint32_t lo = wave_or(mine && off < 32 ? 1u << off : 0u);
      const uint32_t hi = wave_or(mine && off >= 32 ? 1u << (off - 32) : 0u);
      if (lane == leader) {
        atomicOr(reinterpret_cast<unsigned long long*>(&a.live_bits[lb]),
                 (static_cast<unsigned long long>(hi) << 32) | lo);
      }
      pending &= ~__ballot(mine);
    }
    if ((pending >> lane) & 1) {
      atomicOr(reinterpret_cast<unsigned long long*>(&a.live_bits[blk]), 1ull << off);
    }
  }
}

// n_b of every block and the totals behind F, by workgroups wg of nwg
__device__ __forceinline__ void pl_blocks(const PlannerArgs& a, int wg, int nwg) {
  __shared__ int64_t red[2][4];
  const int64_t stride = (int64_t)nwg * blockDim.x;
  int64_t live = 0, alloc = 0;
  for (int64_t b = (int64_t)wg * blockDim.x + threadIdx.x; b < a.num_blocks; b += stride) {
    const bool held = a.refs[b] > 0;
    const int n = held ? __popcll(a.live_bits[b]) : 0;
    a.n_b[b] = n;
    live += n;
    alloc += held ? 1 : 0;
  }
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    live += __shfl_xor(live, d, 64);
    alloc += __shfl_xor(alloc, d, 64);
  }
  const int wave = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    red[0][wave] = live;
    red[1][wave] = alloc;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int64_t l = 0, al = 0;
    for (int w = 0; w < 4; ++w) {
      l += red[0][w];
      al += red[1][w];
    }
    if (l) atomicAdd(reinterpret_cast<unsigned long long*>(&a.stats[0]),
                     static_cast<unsigned long long>(l));
    if (al) atomicAdd(reinterpret_cast<unsigned long long*>(&a.stats[1]),
                      static_cast<unsigned long long>(al));
  }
}

// request r: live count and candidate blocks
__device__ __forceinline__ void pl_request(const PlannerArgs& a, int r) {
  __shared__ int lds2[kPlWaves][2];
  __shared__ int wave_sum[kPlWaves];
  const int tid = threadIdx.x;
  const int n = a.seq_lens[r];
  const int t0 = a.tok_indptr[r], t1 = a.tok_indptr[r + 1];
  const int b0 = a.bt_indptr[r], b1 = a.bt_indptr[r + 1];
  if (n < 0 || t0 < 0 || t1 > a.num_tokens || (int64_t)t1 - t0 != n) {
    if (tid == 0) {
      pl_error(a.counters, VTOKEN_ERR_TOK_LEN);
      a.src_count[r] = 0;
    }
    return;
  }
  if (b0 < 0 || b1 > a.num_bt_entries || b1 < b0) {
    if (tid == 0) {
      pl_error(a.counters, VTOKEN_ERR_BT_LEN);
      a.src_count[r] = 0;
    }
    return;
  }
  // live count of the request: 16-byte loads over the 16-byte-aligned middle of its mask,
  // bytes at the ends
  const uint8_t* lv = a.live + t0;
  const int lead = static_cast<int>((16 - (reinterpret_cast<uintptr_t>(lv) & 15)) & 15);
  const int head = lead < n ? lead : n;
  const int words = (n - head) / 16;
  const int tail0 = head + words * 16;
  int lc = 0;
  if (tid < head) lc += lv[tid] != 0;
  if (tail0 + tid < n) lc += lv[tail0 + tid] != 0;
  const uint4* w16 = reinterpret_cast<const uint4*>(lv + head);
  for (int w = tid; w < words; w += kPlThreads) {
    const uint4 x = w16[w];
    lc += nonzero_bytes(x.x) + nonzero_bytes(x.y) + nonzero_bytes(x.z) + nonzero_bytes(x.w);
  }
  lc = wave_inclusive_scan(lc);
  if ((tid & 63) == 63) wave_sum[tid >> 6] = lc;
  __syncthreads();
  if (tid == 0) {
    int c = 0;
#pragma unroll
    for (int w = 0; w < kPlWaves; ++w) c += wave_sum[w];
    a.live_count[r] = c;
  }

  // candidates in table order, with the cumulative live tokens of the candidates so far (one
  // workgroup scan per chunk gives both the rank and the live prefix)
  int carry = 0;
  int live_carry = 0;
  for (int base = 0; base < b1 - b0; base += kPlThreads) {
    const int j = base + tid;
    const int b = j < b1 - b0 ? a.block_ids[b0 + j] : -1;
    const int cl = j < b1 - b0 ? pl_candidate_live(a, b) : -1;
    const bool cand = cl >= 0;
    const int nb = cand ? cl : 0;
    int v[2] = {cand ? 1 : 0, nb}, tot[2];
    block_exclusive_scan<2>(v, tot, lds2);
    if (cand) a.elig_cum[b0 + carry + v[0]] = live_carry + v[1] + nb;
    carry += tot[0];
    live_carry += tot[1];
  }
  if (tid == 0) {
    a.src_count[r] = carry;
    if (carry) atomicAdd(reinterpret_cast<unsigned long long*>(&a.stats[2]),
                         static_cast<unsigned long long>(carry));
  }
}

// Steps 2 and 3 of the planner in one launch: workgroups [0, blocks_grid) count the live
// bits of every block (pl_blocks), the rest take one request each (pl_request). Both read only
// what pl_count_kernel wrote.
__global__ __launch_bounds__(kPlThreads) void pl_blocks_request_kernel(PlannerArgs a,
                                                                       int blocks_grid) {
  const int wg = static_cast<int>(blockIdx.x);
  if (wg < blocks_grid) {
    pl_blocks(a, wg, blocks_grid);
  } else {
    pl_request(a, wg - blocks_grid);
  }
}

__global__ __launch_bounds__(kPlAdmitThreads) void pl_admit_kernel(PlannerArgs a) {
  __shared__ int lds6[kPlAdmitWaves][6];
  if (a.counters[3] != 0) return;
  const int tid = threadIdx.x;
  const int S = a.block_size;
  const int64_t L = a.stats[0], A = a.stats[1], E = a.stats[2];
  const int64_t cap = A * S;
  const bool trig = cap > 0 && (cap - L) * a.theta_den > (int64_t)a.theta_num * cap &&
                    E >= a.min_eligible &&
                    (a.free_watermark < 0 || a.free_len <= a.free_watermark);
  // the totals, written by thread 0 (the capacity check first)
  auto finish = [&](int64_t c_dst, int64_t c_len, int64_t c_free, int64_t s_k,
                    int64_t s_moved, int64_t n_adm) {
    a.dst_indptr[a.num_reqs] = static_cast<int32_t>(c_dst);
    a.new_bt_indptr[a.num_reqs] = static_cast<int32_t>(c_len);
    a.freed_indptr[a.num_reqs] = static_cast<int32_t>(c_free);
    a.stats[3] = trig ? 1 : 0;
    if (c_dst * S > a.src_plan_capacity || c_len > a.new_bt_capacity) {
      a.counters[3] = VTOKEN_ERR_CAPACITY;
      return;
    }
    a.counters[0] = static_cast<int32_t>(c_dst);
    a.counters[1] = static_cast<int32_t>(n_adm);
    a.counters[2] = static_cast<int32_t>(c_free);
    a.stats[4] = s_k;
    a.stats[5] = s_moved;
    a.stats[6] = c_free;
    a.stats[7] = c_dst;
  };
  if (a.num_reqs <= 64) {
    // one wave holds every request: the same rules with wave scans and no barrier. Every sum
    // over the requests is bounded by num_bt_entries or num_tokens and fits 32 bits.
    if (tid >= 64) return;
    const int r = tid;
    const bool in = r < a.num_reqs;
    const int m = in ? a.bt_indptr[r + 1] - a.bt_indptr[r] : 0;
    const int e = in && trig ? a.src_count[r] : 0;
    const int ce = wave_inclusive_scan(e) - e;              // candidates of earlier requests
    const int64_t room = a.max_sources - ce;                // bound B over the candidates
    const int64_t k = room <= 0 ? 0 : (e < room ? e : room);
    const int64_t T = k > 0 ? a.elig_cum[a.bt_indptr[r] + k - 1] : 0;
    const int64_t need = (T + S - 1) / S;
    const bool prof = k > 0 && need < k;                    // strict block reduction (I4)
    const int pn = prof ? static_cast<int>(need) : 0;
    const int o = wave_inclusive_scan(pn) - pn;
    const bool adm = prof && o + need <= a.free_len;
    const int y0 = adm ? static_cast<int>(need) : 0;
    const int y1 = adm ? m - static_cast<int>(k) + static_cast<int>(need) : m;
    const int y2 = adm ? static_cast<int>(k) : 0;
    const int i0 = wave_inclusive_scan(y0), i1 = wave_inclusive_scan(y1);
    const int i2 = wave_inclusive_scan(y2);
    const int ik = wave_inclusive_scan(static_cast<int>(k));
    const int im = wave_inclusive_scan(adm ? static_cast<int>(T) : 0);
    if (in) {
      a.src_count[r] = static_cast<int32_t>(k);
      a.admitted[r] = adm ? 1 : 0;
      a.dst_indptr[r] = i0 - y0;
      a.new_bt_indptr[r] = i1 - y1;
      a.freed_indptr[r] = i2 - y2;
    }
    const int t0 = __builtin_amdgcn_readlane(i0, 63), t1 = __builtin_amdgcn_readlane(i1, 63);
    const int t2 = __builtin_amdgcn_readlane(i2, 63), tk = __builtin_amdgcn_readlane(ik, 63);
    const int tm = __builtin_amdgcn_readlane(im, 63);
    const int na = __popcll(__ballot(adm));
    if (tid == 0) finish(t0, t1, t2, tk, tm, na);
    return;
  }
  // carries over the chunks: candidates of earlier requests, needs of earlier profitable
  // requests, destinations, new table entries, released sources; and the totals. The scans
  // are 32-bit (DPP wave scans): every sum is bounded by num_bt_entries or num_tokens.
  int64_t c_e = 0, c_o = 0, c_dst = 0, c_len = 0, c_free = 0;
  int64_t s_k = 0, s_moved = 0, n_adm = 0;
  for (int base = 0; base < a.num_reqs; base += kPlAdmitThreads) {
    const int r = base + tid;
    const bool in = r < a.num_reqs;
    const int m = in ? a.bt_indptr[r + 1] - a.bt_indptr[r] : 0;
    const int e = in && trig ? a.src_count[r] : 0;
    int v1[1] = {e}, t1[1];
    block_exclusive_scan<1>(v1, t1, reinterpret_cast<int (*)[1]>(lds6));
    const int64_t room = a.max_sources - (c_e + v1[0]);    // bound B over the candidates
    const int64_t k = room <= 0 ? 0 : (e < room ? e : room);
    c_e += t1[0];
    const int64_t T = k > 0 ? a.elig_cum[a.bt_indptr[r] + k - 1] : 0;
    const int64_t need = (T + S - 1) / S;
    const bool prof = k > 0 && need < k;                   // strict block reduction (I4)
    v1[0] = prof ? static_cast<int>(need) : 0;
    block_exclusive_scan<1>(v1, t1, reinterpret_cast<int (*)[1]>(lds6));
    const bool adm = prof && c_o + v1[0] + need <= a.free_len;
    c_o += t1[0];
    int y[6] = {adm ? static_cast<int>(need) : 0,
                adm ? m - static_cast<int>(k) + static_cast<int>(need) : m,
                adm ? static_cast<int>(k) : 0, static_cast<int>(k),
                adm ? static_cast<int>(T) : 0, adm ? 1 : 0};
    int ty[6];
    block_exclusive_scan<6>(y, ty, lds6);
    if (in) {
      a.src_count[r] = static_cast<int32_t>(k);
      a.admitted[r] = adm ? 1 : 0;
      a.dst_indptr[r] = static_cast<int32_t>(c_dst + y[0]);
      a.new_bt_indptr[r] = static_cast<int32_t>(c_len + y[1]);
      a.freed_indptr[r] = static_cast<int32_t>(c_free + y[2]);
    }
    c_dst += ty[0];
    c_len += ty[1];
    c_free += ty[2];
    s_k += ty[3];
    s_moved += ty[4];
    n_adm += ty[5];
  }
  if (tid == 0) finish(c_dst, c_len, c_free, s_k, s_moved, n_adm);
}

// One 1024-thread workgroup per request. The sources and the new table first (table entries
// in rounds of 1024); the request's destinations are read into LDS (when they fit). Then the
// tokens in tiles of 8192: every lane issues the mask bytes and slots of its eight tokens,
// then the selection flags of their blocks, before any ballot; ranks of the moving tokens come
// from wave ballots and one LDS scan of the wave totals per tile.
template <bool kPow2>
__global__ __launch_bounds__(kPlTableThreads) void pl_table_kernel(PlannerArgs a) {
  __shared__ int lds_rank[kPlTableWaves];
  __shared__ int wave_total[kPlTableWaves];
  __shared__ int32_t dest_s[kPlDestLds];
  if (a.counters[3] != 0) return;
  const int r = blockIdx.x;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int S = a.block_size;
  const BlockDiv<kPow2> bd(S);
  const int t0 = a.tok_indptr[r], n = a.tok_indptr[r + 1] - t0;
  const int b0 = a.bt_indptr[r], m = a.bt_indptr[r + 1] - b0;
  const bool adm = a.admitted[r] != 0;
  const int k = adm ? a.src_count[r] : 0;
  const int d0 = a.dst_indptr[r];
  const int need = a.dst_indptr[r + 1] - d0;
  const int nb0 = a.new_bt_indptr[r];
  const int f0 = a.freed_indptr[r];
  const bool dest_lds = need <= kPlDestLds;
  if (dest_lds) {
    for (int i = tid; i < need; i += kPlTableThreads) dest_s[i] = a.free_list[d0 + i];
  }

  // sources: the first k candidates in table order; kept blocks and released sources
  int cand_carry = 0, keep_carry = 0, sel_carry = 0;
  for (int base = 0; base < m; base += kPlTableThreads) {
    const int j = base + tid;
    const bool in = j < m;
    const int b = in ? a.block_ids[b0 + j] : -1;
    const bool cand = in && adm && pl_candidate_live(a, b) >= 0;
    int cnt;
    const int crank = cand_carry + pl_rank<kPlTableWaves>(cand, &cnt, lds_rank);
    cand_carry += cnt;
    const bool sel = cand && crank < k;
    if (in && b >= 0 && b < a.num_blocks) a.selected[b] = sel ? 1 : 0;
    int nkeep;
    const int krank = keep_carry + pl_rank<kPlTableWaves>(in && !sel, &nkeep, lds_rank);
    keep_carry += nkeep;
    int nsel;
    const int srank = sel_carry + pl_rank<kPlTableWaves>(sel, &nsel, lds_rank);
    sel_carry += nsel;
    if (in && !sel && nb0 + krank < a.new_bt_capacity) a.new_block_ids[nb0 + krank] = b;
    if (sel) a.sources[f0 + srank] = b;
  }
  __syncthreads();  // selected[] of this request's blocks and the LDS destinations
  for (int i = tid; i < need; i += kPlTableThreads) {
    a.new_block_ids[nb0 + keep_carry + i] = dest_lds ? dest_s[i] : a.free_list[d0 + i];
  }

  // move list in logical order: live tokens whose slot lies in a selected source
  const int64_t plan0 = (int64_t)d0 * S;
  const int64_t plan_n = (int64_t)need * S;
  int q_carry = 0;
  bool overflow = false;
  for (int base = 0; base < n; base += kPlTile) {
    const int wbase = base + wave * (64 * kPlBallots);
    // unconditional loads (positions clamped to the last token), all in flight together
    uint8_t lv[kPlBallots];
    int sl[kPlBallots];
#pragma unroll
    for (int q = 0; q < kPlBallots; ++q) {
      const int pc = min(wbase + q * 64 + lane, n - 1);
      lv[q] = a.live[t0 + pc];
      sl[q] = a.slot_in[t0 + pc];
    }
    int sel[kPlBallots];
#pragma unroll
    for (int q = 0; q < kPlBallots; ++q) {
      const bool valid = sl[q] >= 0 && sl[q] < a.num_slots;
      sel[q] = a.selected[valid ? bd.div(sl[q]) : 0];
    }
    int rank[kPlBallots];
    int local = 0;
#pragma unroll
    for (int q = 0; q < kPlBallots; ++q) {
      const int p = wbase + q * 64 + lane;
      const bool valid = sl[q] >= 0 && sl[q] < a.num_slots;
      const bool mv = adm && p < n && lv[q] != 0 && valid && sel[q] != 0;
      const uint64_t mk = __ballot(mv);
      rank[q] = mv ? local + lanes_below(mk) : -1;
      local += __popcll(mk);
    }
    if (lane == 0) wave_total[wave] = local;
    __syncthreads();
    int off = q_carry, tile = 0;
#pragma unroll
    for (int w = 0; w < kPlTableWaves; ++w) {
      const int x = wave_total[w];
      off += w < wave ? x : 0;
      tile += x;
    }
#pragma unroll
    for (int q = 0; q < kPlBallots; ++q) {
      const int p = wbase + q * 64 + lane;
      if (p >= n) continue;
      const int s = sl[q];
      const bool valid = s >= 0 && s < a.num_slots;
      int out = lv[q] != 0 && valid ? s : -1;
      if (rank[q] >= 0) {
        const int qq = off + rank[q];
        if (qq < plan_n) {
          const int g = bd.div(qq);
          const int dblk = dest_lds ? dest_s[g] : a.free_list[d0 + g];
          out = dblk * S + bd.mod(qq);
          a.src_plan[plan0 + qq] = s;
        } else {
          overflow = true;
        }
      }
      a.token_slot[t0 + p] = out;
    }
    q_carry += tile;
    __syncthreads();
  }
  if (adm) {
    // the moved tokens must be exactly the live tokens counted in the sources
    const int expect = k > 0 ? a.elig_cum[b0 + k - 1] : 0;
    if (overflow || (tid == 0 && q_carry != expect)) pl_error(a.counters, VTOKEN_ERR_SLOT);
    for (int64_t q = q_carry + tid; q < plan_n; q += kPlTableThreads) a.src_plan[plan0 + q] = -1;
  }
}

}  // namespace

hipError_t launch_planner(const PlannerArgs& a, hipStream_t stream) {
  auto grid_for = [](int64_t n) {
    int64_t g = (n + 255) / 256;
    g = g < 1 ? 1 : g;
    return static_cast<unsigned>(g < 2048 ? g : 2048);
  };
  hipLaunchKernelGGL(pl_clear_kernel, dim3(grid_for(a.num_blocks)), dim3(256), 0, stream, a);
  const bool pow2 = (a.block_size & (a.block_size - 1)) == 0;
  hipLaunchKernelGGL(pow2 ? pl_count_kernel<true> : pl_count_kernel<false>,
                     dim3(grid_for((int64_t)a.num_bt_entries + a.num_tokens)), dim3(256), 0,
                     stream, a);
  // at most 128 workgroups: each adds its totals with two atomics on the same two words
  const unsigned blocks_grid = grid_for(a.num_blocks) < 128u ? grid_for(a.num_blocks) : 128u;
  hipLaunchKernelGGL(pl_blocks_request_kernel,
                     dim3(blocks_grid + static_cast<unsigned>(a.num_reqs > 0 ? a.num_reqs : 0)),
                     dim3(kPlThreads), 0, stream, a, static_cast<int>(blocks_grid));
  hipLaunchKernelGGL(pl_admit_kernel, dim3(1), dim3(kPlAdmitThreads), 0, stream, a);
  if (a.num_reqs > 0) {
    hipLaunchKernelGGL(pow2 ? pl_table_kernel<true> : pl_table_kernel<false>, dim3(a.num_reqs),
                       dim3(kPlTableThreads), 0, stream, a);
  }
  return hipGetLastError();
}

}  // namespace vtoken
