// HIP kernels of the vToken repack's metadata steps for CDNA4 (gfx950, wave64).
//
//   count_kernel   one workgroup per request (512 threads, 128 for short requests):
//                  validates the request's CSR ranges and block ids and counts its live
//                  tokens (16-byte loads of the live mask).
//   admit_kernel   large batches (over 512 requests; over 256 of short ones): the admission
//                  over all requests (destination need ceil(live/S), strict gain, prefix
//                  admission against the free list: Sec. 3.3.2, 3.3.3, I4 of Sec. 3.5) in
//                  one workgroup.
//   plan_kernel    one workgroup per request: the admission (each workgroup over all
//                  requests, or read from admit_kernel's outputs), then the request's new
//                  block table, token slots (slot = block * S + offset, Sec. 3.4; ranks by
//                  wave ballots, the order-preserving fill of Sec. 3.3.3) and
//                  per-destination source plan.
//   plan_small_kernel  both steps in one workgroup and one launch for batches of at most
//                  24 requests and 8,192 tokens.
//   free_kernel    the freed list: old blocks of admitted requests (Sec. 3.3.4); the same
//                  work runs in the copy's launch for vtoken_repack_free.
//
// Scans across a wave use DPP row shifts and lane reads, never the LDS-routed shuffles
// (vtoken_internal.h). The copies that consume the plan are in vtoken_copy.hip. Kernels
// after the plan read the status word plan->counters[3] and do nothing when it is set; every
// dereference of caller data is bounds-checked.
#include <limits.h>

#include "vtoken_internal.h"

namespace vtoken {
namespace {

using namespace vtoken::meta;

static_assert(kPlanThreads % 64 == 0 && kPlanThreads <= 1024,
              "the workgroup scans take at most 16 waves");
static_assert(kPlanThreadsSplit % 64 == 0 && kPlanThreadsSplit <= kPlanThreads,
              "plan workgroups of whole waves");


// ------------------------------------------------------------------------------------------
// Step 1a: per request, validation of its CSR ranges and block ids, and its live count
// (Sec. 3.2: the token table's liveness bits). A request with an error stores the (negative)
// error code as its live count, which the plan kernel picks up.
// ------------------------------------------------------------------------------------------
template <int kThreads>
__global__ __launch_bounds__(kThreads) void count_kernel(MetaArgs a) {
  __shared__ int wave_sum[kThreads / 64];
  const int r = blockIdx.x;
  const int tid = threadIdx.x;
  const int S = a.block_size;
  const int n = a.seq_lens[r];
  const int t0 = a.tok_indptr[r], t1 = a.tok_indptr[r + 1];
  const int b0 = a.bt_indptr[r], b1 = a.bt_indptr[r + 1];

  int code = 0;
  if (n < 0 || t0 < 0 || t1 > a.num_tokens || (int64_t)t1 - t0 != n) {
    code = VTOKEN_ERR_TOK_LEN;
  } else if (b0 < 0 || b1 > a.num_bt_entries ||
             (int64_t)b1 - b0 != ((int64_t)n + S - 1) / S) {
    code = VTOKEN_ERR_BT_LEN;
  }
  if (code != 0) {   // uniform: every thread read the same entries
    if (tid == 0) a.live_count[r] = code;
    return;
  }
  // the block ids (validated) and the mask (counted) are read in the same loop, so that their
  // loads are in flight together; 16-byte loads over the 16-byte-aligned middle of the mask,
  // bytes at its ends
  const uint8_t* lv = a.live + t0;
  const int lead = static_cast<int>((16 - (reinterpret_cast<uintptr_t>(lv) & 15)) & 15);
  const int head = lead < n ? lead : n;
  const int words = (n - head) / 16;
  const int tail0 = head + words * 16;
  const int m = b1 - b0;
  const int iters = words > m ? words : m;
  int cnt = 0, bad = 0;
  if (tid < head) cnt += lv[tid] != 0;
  if (tail0 + tid < n) cnt += lv[tail0 + tid] != 0;
  const uint4* w16 = reinterpret_cast<const uint4*>(lv + head);
  for (int w = tid; w < iters; w += kThreads) {
    const int blk = w < m ? a.block_ids[b0 + w] : 0;
    const uint4 x = w < words ? w16[w] : make_uint4(0, 0, 0, 0);
    bad |= (blk < 0) | (blk >= a.num_blocks);
    cnt += nonzero_bytes(x.x) + nonzero_bytes(x.y) + nonzero_bytes(x.z) + nonzero_bytes(x.w);
  }
  if (__syncthreads_or(bad)) {
    if (tid == 0) a.live_count[r] = VTOKEN_ERR_BLOCK_RANGE;
    return;
  }
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) cnt += __shfl_xor(cnt, d, 64);
  if ((tid & 63) == 0) wave_sum[tid >> 6] = cnt;
  __syncthreads();
  if (tid == 0) {
    int c = 0;
#pragma unroll
    for (int w = 0; w < kThreads / 64; ++w) c += wave_sum[w];
    a.live_count[r] = c;
  }
}

// The admission over all requests, every thread of the workgroup taking part (R/1024 rounds of
// two workgroup scans; one wave alone, with wave scans, when R <= 64): destination need
// ceil(live/S), strict gain (Sec. 3.3.3, I4 of Sec. 3.5), prefix admission against the free
// list (Sec. 3.3.2). count(i) is request i's live count
// (a negative error code for a request the validation rejected), blocks(i) the length of its
// old table; visit(i, admitted, destination offset, new-table offset, freed offset) is called
// once per request by the thread holding it.
struct Admission {
  int used, n_new, n_freed, n_admitted, first_error;
};

template <class Count, class Blocks, class Visit>
__device__ __forceinline__ Admission admit_requests(const MetaArgs& a, Count count,
                                                    Blocks blocks, Visit visit,
                                                    int (*lds)[4], int* first_error_req) {
  const int tid = threadIdx.x;
  const int R = a.num_reqs;
  const int S = a.block_size;
  if (R <= 64) {
    // one wave holds every request: the same rules with wave scans only, no workgroup
    // barrier until the totals are published
    if (tid < 64) {
      const int i = tid;
      const bool valid = i < R;
      const int c = valid ? count(i) : 0;
      const int m = valid ? blocks(i) : 0;
      const uint64_t errors = __ballot(valid && c < 0);
      const int need = c > 0 ? (c + S - 1) / S : 0;
      const bool profitable = valid && c >= 0 && need < m;
      const int e = profitable ? need : 0;
      const int o = wave_inclusive_scan(e) - e;
      const bool adm = profitable && (a.inplace || o + need <= a.free_len);
      const int n_free = adm ? (a.inplace ? m - need : m) : 0;
      const int d = adm ? need : 0, nb = adm ? need : m;
      const int di = wave_inclusive_scan(d);
      const int ni = wave_inclusive_scan(nb);
      const int fi = wave_inclusive_scan(n_free);
      if (valid) visit(i, adm ? 1 : 0, di - d, ni - nb, fi - n_free);
      const int used = __builtin_amdgcn_readlane(di, 63);
      const int n_new = __builtin_amdgcn_readlane(ni, 63);
      const int n_freed = __builtin_amdgcn_readlane(fi, 63);
      const int n_adm = __popcll(__ballot(adm));
      if (tid == 0) {
        lds[0][0] = used;
        lds[0][1] = n_new;
        lds[0][2] = n_freed;
        lds[0][3] = n_adm;
        *first_error_req = errors != 0 ? __builtin_ctzll(errors) : INT_MAX;
      }
    }
    __syncthreads();
    return Admission{lds[0][0], lds[0][1], lds[0][2], lds[0][3], *first_error_req};
  }
  if (tid == 0) *first_error_req = INT_MAX;
  __syncthreads();
  int carry_e = 0, carry_dst = 0, carry_new = 0, carry_freed = 0, n_admitted = 0;
  for (int base = 0; base < R; base += kPlanThreads) {
    const int i = base + tid;
    const bool valid = i < R;
    const int c = valid ? count(i) : 0;
    if (valid && c < 0) atomicMin(first_error_req, i);
    const int m = valid ? blocks(i) : 0;
    const int need = c > 0 ? (c + S - 1) / S : 0;
    const bool profitable = valid && c >= 0 && need < m;
    // position of this request's destinations in the free list: needs of every earlier
    // profitable request (admitted or not - once one is deferred all later ones are)
    int s1[1] = {profitable ? need : 0};
    int t1[1];
    block_exclusive_scan<1>(s1, t1, reinterpret_cast<int (*)[1]>(lds));
    // in place the destinations are the request's own blocks: nothing to wait for
    const bool adm = profitable && (a.inplace || carry_e + s1[0] + need <= a.free_len);
    // freed: all old blocks out of place, the blocks past the need in place
    const int n_free = adm ? (a.inplace ? m - need : m) : 0;
    int s2[4] = {adm ? need : 0, adm ? need : m, n_free, adm ? 1 : 0};
    int t2[4];
    block_exclusive_scan<4>(s2, t2, lds);
    if (valid) visit(i, adm ? 1 : 0, carry_dst + s2[0], carry_new + s2[1], carry_freed + s2[2]);
    carry_e += t1[0];
    carry_dst += t2[0];
    carry_new += t2[1];
    carry_freed += t2[2];
    n_admitted += t2[3];
  }
  __syncthreads();
  return Admission{carry_dst, carry_new, carry_freed, n_admitted, *first_error_req};
}

// The pass's status after the admission: the first rejected request's code, else a capacity
// shortfall, else (checked by the workgroup that reports) a consumed free-list entry outside
// the pool; head[0 .. head_len) is a copy of the free list's first entries in LDS, checked
// there. The reporting workgroup writes the offsets' ends and the counters.
__device__ __forceinline__ int admission_status(const MetaArgs& a, const Admission& adm,
                                                int request_error, bool report,
                                                const int32_t* head = nullptr,
                                                int head_len = 0) {
  const int tid = threadIdx.x;
  const int S = a.block_size;
  int status = request_error;
  if (status == 0 && ((int64_t)adm.n_new > a.new_bt_capacity ||
                      (int64_t)adm.used * S > a.src_plan_capacity ||
                      (!a.inplace && adm.used > a.free_len))) {
    status = VTOKEN_ERR_CAPACITY;
  }
  if (!report) return status;
  if (status == 0 && !a.inplace) {
    // every consumed free-list entry must be a block of the pool (eight loads in flight per
    // thread)
    int bad = 0;
    const int in_head = adm.used < head_len ? adm.used : head_len;
    for (int j = tid; j < in_head; j += kPlanThreads) {
      bad |= (head[j] < 0) | (head[j] >= a.num_blocks);
    }
    for (int j0 = in_head; j0 < adm.used; j0 += 8 * kPlanThreads) {
      int blk[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const int j = j0 + k * kPlanThreads + tid;
        blk[k] = j < adm.used ? a.free_list[j] : 0;
      }
#pragma unroll
      for (int k = 0; k < 8; ++k) bad |= (blk[k] < 0) | (blk[k] >= a.num_blocks);
    }
    if (__syncthreads_or(bad)) status = VTOKEN_ERR_BLOCK_RANGE;
  }
  if (tid == 0) {
    const int R = a.num_reqs;
    a.dst_indptr[R] = adm.used;
    a.new_bt_indptr[R] = adm.n_new;
    a.freed_indptr[R] = adm.n_freed;
    a.counters[0] = status == 0 ? adm.used : 0;
    a.counters[1] = status == 0 ? adm.n_admitted : 0;
    a.counters[2] = status == 0 ? adm.n_freed : 0;
    a.counters[3] = status;
    a.counters[4] = a.inplace ? kPlanInPlace : kPlanOutOfPlace;
  }
  return status;
}

// ------------------------------------------------------------------------------------------
// Step 1b, large batches: the admission alone, in one workgroup (destination need
// ceil(live/S), strict gain, prefix admission; Sec. 3.3.2, 3.3.3, I4 of Sec. 3.5). It writes
// every request's admitted flag and CSR offsets, the offsets' ends, the totals and the status
// word, which plan_kernel<kPow2, true, ...> then reads instead of repeating the admission in
// each of its R workgroups (R/1024 rounds of workgroup scans each, O(R^2) over the launch). The live
// counts and table lengths of the first kAdmitStage requests are staged in LDS, all of their
// loads in flight at once.
// ------------------------------------------------------------------------------------------
__global__ __launch_bounds__(kPlanThreads) void admit_kernel(MetaArgs a) {
  __shared__ int lds[kPlanThreads / 64][4];
  __shared__ int first_error_req;
  __shared__ int count_s[kAdmitStage];
  __shared__ int blocks_s[kAdmitStage];
  const int tid = threadIdx.x;
  const int R = a.num_reqs;
  const int staged = min(R, kAdmitStage);
  int c[kAdmitStage / kPlanThreads], m[kAdmitStage / kPlanThreads];
#pragma unroll
  for (int q = 0; q < kAdmitStage / kPlanThreads; ++q) {
    const int i = q * kPlanThreads + tid;
    c[q] = i < staged ? a.live_count[i] : 0;
    m[q] = i < staged ? a.bt_indptr[i + 1] - a.bt_indptr[i] : 0;
  }
#pragma unroll
  for (int q = 0; q < kAdmitStage / kPlanThreads; ++q) {
    const int i = q * kPlanThreads + tid;
    if (i < staged) {
      count_s[i] = c[q];
      blocks_s[i] = m[q];
    }
  }
  // (the admission's first barrier orders these LDS writes before every read)
  const Admission adm = admit_requests(
      a, [&](int i) { return i < kAdmitStage ? count_s[i] : a.live_count[i]; },
      [&](int i) {
        return i < kAdmitStage ? blocks_s[i] : a.bt_indptr[i + 1] - a.bt_indptr[i];
      },
      [&](int i, int ad, int dst, int nb, int fr) {
        a.admitted[i] = ad;
        a.dst_indptr[i] = dst;
        a.new_bt_indptr[i] = nb;
        a.freed_indptr[i] = fr;
      },
      lds, &first_error_req);
  admission_status(a, adm, adm.first_error == INT_MAX ? 0 : a.live_count[adm.first_error], true);
}

// ------------------------------------------------------------------------------------------
// Step 1b: the plan. For batches of at most kFusedAdmitReqs requests (kFusedAdmitShortReqs of
// short ones) every workgroup first runs the admission over all requests itself (each reads
// the R live counts; one round of two workgroup scans, one wave alone for R <= 64):
// destination need ceil(live/S), strict gain
// (Sec. 3.3.3, I4 of Sec. 3.5), prefix admission against the free list (Sec. 3.3.2), and the
// CSR offsets of its own request; the workgroup of request 0 also writes the totals and the
// status word. No workgroup waits for another, so the admission costs one extra pass per
// workgroup instead of a launch. Larger batches (kAdmitted) take their request's offsets and
// the status word from admit_kernel, the launch before. Then workgroup r builds request r's
// part of the bulk apply_moves (Sec. 3.2): its new block table, the slot of every token (slot =
// block * S + offset, Sec. 3.4; ranks from wave ballots and lane prefix counts over the live
// mask, the order-preserving fill of Sec. 3.3.3) and its rows of the per-destination source
// plan.
// ------------------------------------------------------------------------------------------
template <bool kPow2, bool kAdmitted, int kThreads>
__global__ __launch_bounds__(kThreads) void plan_kernel(MetaArgs a) {
  // With the admission done before, a workgroup only builds its request's table and holds no
  // free-list head in LDS: kPlanThreadsSplit threads, so that more requests are in progress at
  // once (the admission in the workgroup takes all kPlanThreads; with 1024 threads per request
  // the plan of 257 short requests takes 4-5 us longer than that of 256, one per CU).
  static_assert(kAdmitted || kThreads == kPlanThreads, "the admission takes 16 waves");
  constexpr int kWaves = kThreads / 64;
  constexpr int kTile = kThreads * kPlanBallots;   // tokens per tile
  __shared__ int lds[kWaves][4];
  __shared__ int wave_total[kWaves];
  __shared__ int first_error_req;
  __shared__ int mine[4];   // admitted, destination offset, new-table offset, freed offset
  __shared__ int32_t head[kAdmitted ? 1 : kPlanHead];   // free_list[0 .. P)
  const int r = blockIdx.x;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int R = a.num_reqs;
  const int S = a.block_size;
  const BlockDiv<kPow2> bd(S);

  // Loads that depend on nothing are issued first, so that they are in flight together with
  // the request's own CSR entries: the admission's inputs for the first 1024 requests, and the
  // head of the free list (out of place), from which destinations are looked up in LDS
  // instead of by a load after the admission. (With the admission done before, the request's
  // own offsets and the status word instead; its destinations are read from the free list.)
  int c_pre = 0, m_pre = 0;
  int my_adm = 0, my_dst = 0, my_new = 0, pre_status = 0;
  if constexpr (kAdmitted) {
    if (r < R) {
      my_adm = a.admitted[r];
      my_dst = a.dst_indptr[r];
      my_new = a.new_bt_indptr[r];
    }
    pre_status = a.counters[3];
  } else if (tid < R) {
    c_pre = a.live_count[tid];
    m_pre = a.bt_indptr[tid + 1] - a.bt_indptr[tid];
  }
  const int P = kAdmitted || a.inplace ? 0 : min(a.free_len, kPlanHead);
  int32_t fl[kPlanHead / kThreads];
  if constexpr (!kAdmitted) {
#pragma unroll
    for (int q = 0; q < kPlanHead / kThreads; ++q) {
      const int j = q * kThreads + tid;
      fl[q] = j < P ? a.free_list[j] : 0;
    }
  }

  // this request's first tile of live bits and the block-table entries of its positions do not
  // depend on the admission: they are loaded first and arrive during it (ranges checked here,
  // so even a request the count kernel rejected reads only inside the batch's arrays)
  int n = 0, t0 = 0, b0 = 0;
  if (r < R) {
    n = a.seq_lens[r];
    t0 = a.tok_indptr[r];
    b0 = a.bt_indptr[r];
  }
  const bool in_range = r < R && n >= 0 && t0 >= 0 && (int64_t)t0 + n <= a.num_tokens &&
                        b0 >= 0 && (int64_t)b0 + ((int64_t)n + S - 1) / S <= a.num_bt_entries;
  const uint8_t* lv = a.live + t0;
  const int32_t* bt = a.block_ids + b0;
  uint8_t live0[kPlanBallots];
  int phys0[kPlanBallots];
#pragma unroll
  for (int k = 0; k < kPlanBallots; ++k) {
    const int pos = wave * (64 * kPlanBallots) + k * 64 + lane;
    const bool ok = in_range && pos < n;
    live0[k] = ok ? lv[pos] : 0;
    phys0[k] = ok ? bt[bd.div(pos)] : 0;
  }

  if constexpr (!kAdmitted) {
#pragma unroll
    for (int q = 0; q < kPlanHead / kThreads; ++q) {
      const int j = q * kThreads + tid;
      if (j < P) head[j] = fl[q];
    }
  }
  int status = pre_status;
  if constexpr (!kAdmitted) {
    // (the admission's first barrier orders these LDS writes before every read)
    const Admission adm = admit_requests(
        a, [&](int i) { return i < kPlanThreads ? c_pre : a.live_count[i]; },
        [&](int i) { return i < kPlanThreads ? m_pre : a.bt_indptr[i + 1] - a.bt_indptr[i]; },
        [&](int i, int ad, int dst, int nb, int fr) {
          if (i == r) {
            mine[0] = ad;
            mine[1] = dst;
            mine[2] = nb;
            mine[3] = fr;
          }
        },
        lds, &first_error_req);
    status =
        admission_status(a, adm, adm.first_error == INT_MAX ? 0 : a.live_count[adm.first_error],
                         r == 0, head, P);
    if (r >= R) return;   // the one workgroup of an empty batch
    my_adm = mine[0];
    my_dst = mine[1];
    my_new = mine[2];
    if (tid == 0) {
      a.admitted[r] = my_adm;
      a.dst_indptr[r] = my_dst;
      a.new_bt_indptr[r] = my_new;
      a.freed_indptr[r] = mine[3];
    }
  }
  // an error anywhere: the status word (request 0's workgroup, or the admission launch)
  // reports it, nothing is built
  if (status != 0) return;

  int32_t* ts = a.token_slot + t0;
  int32_t* nbt = a.new_block_ids + my_new;
  if (!my_adm) {
    // unchanged: the old table, every live token at its positional slot
    const int m = a.bt_indptr[r + 1] - b0;
    for (int j = tid; j < m; j += kThreads) nbt[j] = bt[j];
    for (int base = 0; base < n; base += kTile) {
      if (base > 0) {   // later tiles: unconditional loads, positions clamped
#pragma unroll
        for (int k = 0; k < kPlanBallots; ++k) {
          const int pc = min(base + wave * (64 * kPlanBallots) + k * 64 + lane, n - 1);
          live0[k] = lv[pc];
          phys0[k] = bt[bd.div(pc)];
        }
      }
#pragma unroll
      for (int k = 0; k < kPlanBallots; ++k) {
        const int p = base + wave * (64 * kPlanBallots) + k * 64 + lane;
        if (p < n) ts[p] = live0[k] != 0 ? phys0[k] * S + bd.mod(p) : -1;
      }
    }
    return;
  }
  const int o = my_dst;
  const int c = a.live_count[r];
  const int need = (c + S - 1) / S;
  // this request's destinations: read from the LDS head of the free list when they lie in it
  const bool dest_lds = !a.inplace && o + need <= P;
  const int32_t* dest = a.inplace ? bt : a.free_list + o;
  const int32_t* dest_s = head + o;
  int32_t* plan = a.src_plan + (int64_t)o * S;
  for (int j = tid; j < need; j += kThreads) nbt[j] = dest_lds ? dest_s[j] : dest[j];
  if (need == 0) {
    // no live token (every block is released): only dead slots to write
    for (int p = tid; p < n; p += kThreads) ts[p] = -1;
    return;
  }
  int carry = 0;
  for (int base = 0; base < n; base += kTile) {
    const int wbase = base + wave * (64 * kPlanBallots);
    // the tile's live bytes and table entries: the first tile's were loaded before the
    // admission; later tiles load theirs here, unconditionally (positions clamped to the
    // request's last token), so all of them are in flight together
    if (base > 0) {
#pragma unroll
      for (int k = 0; k < kPlanBallots; ++k) {
        const int pc = min(wbase + k * 64 + lane, n - 1);
        live0[k] = lv[pc];
        phys0[k] = bt[bd.div(pc)];
      }
    }
    int rank[kPlanBallots];
    int local = 0;
#pragma unroll
    for (int k = 0; k < kPlanBallots; ++k) {
      const int p = wbase + k * 64 + lane;
      const bool l = (p < n) && live0[k] != 0;
      const uint64_t mk = __ballot(l);
      rank[k] = l ? local + lanes_below(mk) : -1;
      local += __popcll(mk);
    }
    if (lane == 0) wave_total[wave] = local;
    __syncthreads();
    int off = carry, tile = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      const int x = wave_total[w];
      off += (w < wave) ? x : 0;
      tile += x;
    }
    // every lane's destination blocks first, one unconditional read each (a dead or absent
    // token re-reads the first destination), so the eight reads are in flight together
    int dblk[kPlanBallots];
    if (dest_lds) {
#pragma unroll
      for (int k = 0; k < kPlanBallots; ++k) {
        dblk[k] = dest_s[bd.div(rank[k] >= 0 ? off + rank[k] : 0)];
      }
    } else {
#pragma unroll
      for (int k = 0; k < kPlanBallots; ++k) {
        dblk[k] = dest[bd.div(rank[k] >= 0 ? off + rank[k] : 0)];
      }
    }
#pragma unroll
    for (int k = 0; k < kPlanBallots; ++k) {
      const int p = wbase + k * 64 + lane;
      if (p < n) {
        if (rank[k] >= 0) {
          const int kk = off + rank[k];
          plan[kk] = phys0[k] * S + bd.mod(p);
          ts[p] = dblk[k] * S + bd.mod(kk);
        } else {
          ts[p] = -1;
        }
      }
    }
    carry += tile;
    __syncthreads();
  }
  // destination slots past the last live token: nothing to copy
  for (int k = c + tid; k < need * S; k += kThreads) plan[k] = -1;
}

// ------------------------------------------------------------------------------------------
// Steps 1a and 1b in one workgroup, for small batches (at most kSmallReqs requests and
// kSmallTokens tokens), where the pass is bound by launch latency: one launch instead of two.
// Wave w validates and counts requests w, w + 16, ... (64-token ballots, eight in flight), the
// workgroup runs the admission over the counts held in LDS, and wave w builds the same requests'
// tables, token slots and source plans (wave-level ballots and lane prefix counts). The first
// tile of a wave's first request stays in registers from the counting to the build, and the
// head of the free list is read once into LDS, so that a small pass waits for few dependent
// loads.
// ------------------------------------------------------------------------------------------
template <bool kPow2>
__global__ __launch_bounds__(kPlanThreads) void plan_small_kernel(MetaArgs a) {
  __shared__ int lds[kPlanThreads / 64][4];
  __shared__ int first_error_req;
  __shared__ int count_s[kSmallReqs];
  __shared__ int meta_s[kSmallReqs][4];   // tokens, first token, first table entry, blocks
  __shared__ int plan_s[kSmallReqs][4];   // admitted, destination, new-table and freed offsets
  __shared__ int32_t head[kPlanHead];     // free_list[0 .. P)
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  constexpr int kWaves = kPlanThreads / 64;
  constexpr int kTile = 64 * kPlanBallots;
  const int R = a.num_reqs;
  const int S = a.block_size;
  const BlockDiv<kPow2> bd(S);

  // the head of the free list (out of place), loaded first and written to LDS after the
  // counting: destinations and the consumed-entry range check read it there
  const int P = a.inplace ? 0 : min(a.free_len, kPlanHead);
  int32_t fl[kPlanHead / kPlanThreads];
#pragma unroll
  for (int q = 0; q < kPlanHead / kPlanThreads; ++q) {
    const int j = q * kPlanThreads + tid;
    fl[q] = j < P ? a.free_list[j] : 0;
  }

  // validation and live count per request; the first tile of the wave's first request (mask
  // bytes and table entries) stays in registers for the build below
  uint8_t keep_l[kPlanBallots] = {};
  int keep_b[kPlanBallots] = {};
  for (int r = wave; r < R; r += kWaves) {
    const int n = a.seq_lens[r];
    const int t0 = a.tok_indptr[r], t1 = a.tok_indptr[r + 1];
    const int b0 = a.bt_indptr[r], b1 = a.bt_indptr[r + 1];
    int code = 0;
    if (n < 0 || t0 < 0 || t1 > a.num_tokens || (int64_t)t1 - t0 != n) {
      code = VTOKEN_ERR_TOK_LEN;
    } else if (b0 < 0 || b1 > a.num_bt_entries ||
               (int64_t)b1 - b0 != ((int64_t)n + S - 1) / S) {
      code = VTOKEN_ERR_BT_LEN;
    }
    int c = code;
    if (code == 0) {
      const uint8_t* lv = a.live + t0;
      const int32_t* bt = a.block_ids + b0;
      const int m = b1 - b0;
      // the first block ids and the first tile's mask bytes and table entries are in flight
      // together (positions clamped to the last token; the ranges were checked above)
      const int bid = lane < m ? bt[lane] : 0;
      uint8_t l[kPlanBallots] = {};
      int blk[kPlanBallots] = {};
      if (n > 0) {
#pragma unroll
        for (int k = 0; k < kPlanBallots; ++k) {
          const int pc = min(k * 64 + lane, n - 1);
          l[k] = lv[pc];
          blk[k] = bt[bd.div(pc)];
        }
      }
      bool bad = lane < m && (bid < 0 || bid >= a.num_blocks);
      for (int j = 64 + lane; j < m; j += 64) {
        const int x = bt[j];
        bad |= x < 0 || x >= a.num_blocks;
      }
      c = 0;
#pragma unroll
      for (int k = 0; k < kPlanBallots; ++k) {
        c += __popcll(__ballot(k * 64 + lane < n && l[k] != 0));
      }
      if (r == wave) {
#pragma unroll
        for (int k = 0; k < kPlanBallots; ++k) {
          keep_l[k] = l[k];
          keep_b[k] = blk[k];
        }
      }
      for (int base = kTile; base < n; base += kTile) {
        // unconditional loads (positions clamped to the last token) keep all eight in flight
#pragma unroll
        for (int k = 0; k < kPlanBallots; ++k) l[k] = lv[min(base + k * 64 + lane, n - 1)];
#pragma unroll
        for (int k = 0; k < kPlanBallots; ++k) {
          c += __popcll(__ballot(base + k * 64 + lane < n && l[k] != 0));
        }
      }
      if (__ballot(bad) != 0) c = VTOKEN_ERR_BLOCK_RANGE;
    }
    if (lane == 0) {
      a.live_count[r] = c;
      count_s[r] = c;
      meta_s[r][0] = n;
      meta_s[r][1] = t0;
      meta_s[r][2] = b0;
      meta_s[r][3] = b1 - b0;
    }
  }
#pragma unroll
  for (int q = 0; q < kPlanHead / kPlanThreads; ++q) {
    const int j = q * kPlanThreads + tid;
    if (j < P) head[j] = fl[q];
  }
  __syncthreads();

  const Admission adm = admit_requests(
      a, [&](int i) { return count_s[i]; }, [&](int i) { return meta_s[i][3]; },
      [&](int i, int ad, int dst, int nb, int fr) {
        a.admitted[i] = ad;
        a.dst_indptr[i] = dst;
        a.new_bt_indptr[i] = nb;
        a.freed_indptr[i] = fr;
        plan_s[i][0] = ad;
        plan_s[i][1] = dst;
        plan_s[i][2] = nb;
        plan_s[i][3] = fr;
      },
      lds, &first_error_req);
  const int status = admission_status(
      a, adm, adm.first_error == INT_MAX ? 0 : count_s[adm.first_error], true, head, P);
  if (status != 0) return;

  for (int r = wave; r < R; r += kWaves) {
    const int n = meta_s[r][0];
    const uint8_t* lv = a.live + meta_s[r][1];
    const int32_t* bt = a.block_ids + meta_s[r][2];
    int32_t* ts = a.token_slot + meta_s[r][1];
    int32_t* nbt = a.new_block_ids + plan_s[r][2];
    const bool kept = r == wave;   // first tile in registers
    uint8_t l[kPlanBallots];
    int blk[kPlanBallots];
    auto tile = [&](int base) {
      if (base == 0 && kept) {
#pragma unroll
        for (int k = 0; k < kPlanBallots; ++k) {
          l[k] = keep_l[k];
          blk[k] = keep_b[k];
        }
      } else {
#pragma unroll
        for (int k = 0; k < kPlanBallots; ++k) {
          const int pc = min(base + k * 64 + lane, n - 1);
          l[k] = lv[pc];
          blk[k] = bt[bd.div(pc)];
        }
      }
    };
    if (!plan_s[r][0]) {
      // unchanged: the old table, every live token at its positional slot
      const int m = meta_s[r][3];
      for (int j = lane; j < m; j += 64) nbt[j] = bt[j];
      for (int base = 0; base < n; base += kTile) {
        tile(base);
#pragma unroll
        for (int k = 0; k < kPlanBallots; ++k) {
          const int p = base + k * 64 + lane;
          if (p < n) ts[p] = l[k] != 0 ? blk[k] * S + bd.mod(p) : -1;
        }
      }
      continue;
    }
    const int o = plan_s[r][1];
    const int c = count_s[r];
    const int need = (c + S - 1) / S;
    // destinations: the LDS head of the free list when they lie in it
    const bool dest_lds = !a.inplace && o + need <= P;
    const int32_t* dest = a.inplace ? bt : a.free_list + o;
    const int32_t* dest_s = head + o;
    int32_t* plan = a.src_plan + (int64_t)o * S;
    for (int j = lane; j < need; j += 64) nbt[j] = dest_lds ? dest_s[j] : dest[j];
    if (need == 0) {
      // no live token (every block is released): only dead slots to write
      for (int p = lane; p < n; p += 64) ts[p] = -1;
      continue;
    }
    int carry = 0;
    for (int base = 0; base < n; base += kTile) {
      tile(base);
      // ranks first, then every lane's destination block with one unconditional read each (a
      // dead or absent token re-reads the first destination): the reads are in flight together
      int rank[kPlanBallots];
#pragma unroll
      for (int k = 0; k < kPlanBallots; ++k) {
        const int p = base + k * 64 + lane;
        const bool live = p < n && l[k] != 0;
        const uint64_t mk = __ballot(live);
        rank[k] = live ? carry + lanes_below(mk) : -1;
        carry += __popcll(mk);
      }
      int dblk[kPlanBallots];
      if (dest_lds) {
#pragma unroll
        for (int k = 0; k < kPlanBallots; ++k) {
          dblk[k] = dest_s[bd.div(rank[k] >= 0 ? rank[k] : 0)];
        }
      } else {
#pragma unroll
        for (int k = 0; k < kPlanBallots; ++k) {
          dblk[k] = dest[bd.div(rank[k] >= 0 ? rank[k] : 0)];
        }
      }
#pragma unroll
      for (int k = 0; k < kPlanBallots; ++k) {
        const int p = base + k * 64 + lane;
        if (p < n) {
          if (rank[k] >= 0) {
            plan[rank[k]] = blk[k] * S + bd.mod(p);
            ts[p] = dblk[k] * S + bd.mod(rank[k]);
          } else {
            ts[p] = -1;
          }
        }
      }
    }
    // destination slots past the last live token: nothing to copy
    for (int k = c + lane; k < need * S; k += 64) plan[k] = -1;
  }
}

// ------------------------------------------------------------------------------------------
// Step 3: freed list.
// ------------------------------------------------------------------------------------------
__global__ __launch_bounds__(kFreeThreads) void free_kernel(MetaArgs a, int32_t* freed,
                                                            int64_t capacity) {
  if (a.counters[3] != 0) return;
  const int mode = a.counters[4];
  if (mode != kPlanOutOfPlace && mode != kPlanInPlace) {
    // a partial pass's plan (its released blocks are the planner state's sources): nothing is
    // written and the status word says so
    if (blockIdx.x == 0 && threadIdx.x == 0) atomicCAS(&a.counters[3], 0, VTOKEN_ERR_PLAN_MODE);
    return;
  }
  write_freed_blocks(blockIdx.x, a.admitted, a.bt_indptr, a.freed_indptr, a.block_ids,
                     a.num_bt_entries, freed, capacity);
}

}  // namespace

hipError_t launch_build(const MetaArgs& a, hipStream_t stream) {
  const bool pow2 = (a.block_size & (a.block_size - 1)) == 0;
  if (a.num_reqs <= kSmallReqs && a.num_tokens <= kSmallTokens) {
    hipLaunchKernelGGL(pow2 ? plan_small_kernel<true> : plan_small_kernel<false>, dim3(1),
                       dim3(kPlanThreads), 0, stream, a);
    return hipGetLastError();
  }
  // requests averaging fewer than kLongRequestTokens tokens need one 16-byte load per thread
  // even at kCountThreadsShort threads, and smaller workgroups are resident more at a time
  const bool long_reqs = a.num_reqs > 0 && a.num_tokens / a.num_reqs >= kLongRequestTokens;
  if (a.num_reqs > 0) {
    if (long_reqs) {
      hipLaunchKernelGGL(count_kernel<kCountThreads>, dim3(a.num_reqs), dim3(kCountThreads), 0,
                         stream, a);
    } else {
      hipLaunchKernelGGL(count_kernel<kCountThreadsShort>, dim3(a.num_reqs),
                         dim3(kCountThreadsShort), 0, stream, a);
    }
  }
  if (a.num_reqs > kFusedAdmitReqs || (a.num_reqs > kFusedAdmitShortReqs && !long_reqs)) {
    hipLaunchKernelGGL(admit_kernel, dim3(1), dim3(kPlanThreads), 0, stream, a);
    const auto plan = pow2 ? plan_kernel<true, true, kPlanThreadsSplit>
                           : plan_kernel<false, true, kPlanThreadsSplit>;
    hipLaunchKernelGGL(plan, dim3(a.num_reqs), dim3(kPlanThreadsSplit), 0, stream, a);
    return hipGetLastError();
  }
  // at least one workgroup: an empty batch still writes the offsets' ends and the counters
  const auto plan =
      pow2 ? plan_kernel<true, false, kPlanThreads> : plan_kernel<false, false, kPlanThreads>;
  hipLaunchKernelGGL(plan, dim3(a.num_reqs > 0 ? a.num_reqs : 1), dim3(kPlanThreads), 0, stream,
                     a);
  return hipGetLastError();
}

hipError_t launch_free(const MetaArgs& a, int32_t* freed, int64_t freed_capacity,
                       hipStream_t stream) {
  if (a.num_reqs > 0) {
    hipLaunchKernelGGL(free_kernel, dim3(a.num_reqs), dim3(kFreeThreads), 0, stream, a, freed,
                       freed_capacity);
  }
  return hipGetLastError();
}

}  // namespace vtoken
