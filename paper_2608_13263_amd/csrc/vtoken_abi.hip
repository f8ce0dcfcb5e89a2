// C ABI of the vToken repack (include/vtoken.h): host-side argument validation and launch.
// Nothing here allocates, synchronises or keeps pointers; each call enqueues kernels on the
// caller's stream and returns.
#include <stdint.h>

#include "vtoken_internal.h"

namespace {

constexpr int64_t kInt32Limit = 2147483647LL;

// The HIP error behind the calling thread's most recent VTOKEN_ERR_HIP.
thread_local int32_t g_last_hip_error = 0;

vtoken_status hip_status(hipError_t e) {
  if (e == hipSuccess) return VTOKEN_OK;
  g_last_hip_error = static_cast<int32_t>(e);
  return VTOKEN_ERR_HIP;
}

vtoken_status check_cache(const vtoken_cache* c) {
  if (c == nullptr || c->kv == nullptr) return VTOKEN_ERR_NULL;
  if (c->num_layers <= 0 || c->num_kv_heads <= 0 || c->head_dim <= 0 || c->block_size <= 0 ||
      c->num_blocks <= 0) {
    return VTOKEN_ERR_SHAPE;
  }
  if (c->elem_bytes != 1 && c->elem_bytes != 2) return VTOKEN_ERR_SHAPE;
  const int64_t row = (int64_t)c->num_kv_heads * c->head_dim * c->elem_bytes;
  if (row % 16 != 0 || row > kInt32Limit) return VTOKEN_ERR_SHAPE;
  if ((int64_t)c->num_blocks * c->block_size > kInt32Limit) return VTOKEN_ERR_SHAPE;
  if (row / 16 > vtoken::kMaxRowUnits) return VTOKEN_ERR_SHAPE;
  if ((int64_t)c->block_size * (row / 16) > vtoken::kMaxChunkUnits) return VTOKEN_ERR_SHAPE;
  return VTOKEN_OK;
}

vtoken_status check_batch(const vtoken_batch* b) {
  if (b == nullptr) return VTOKEN_ERR_NULL;
  if (b->num_reqs < 0 || b->num_tokens < 0 || b->num_bt_entries < 0 || b->free_len < 0) {
    return VTOKEN_ERR_SHAPE;
  }
  if (b->num_tokens > kInt32Limit || b->num_bt_entries > kInt32Limit ||
      (int64_t)b->num_reqs + 1 > kInt32Limit) {
    return VTOKEN_ERR_SHAPE;
  }
  if (b->tok_indptr == nullptr || b->bt_indptr == nullptr) return VTOKEN_ERR_NULL;
  if (b->num_reqs > 0 && b->seq_lens == nullptr) return VTOKEN_ERR_NULL;
  if (b->num_tokens > 0 && b->live == nullptr) return VTOKEN_ERR_NULL;
  if (b->num_bt_entries > 0 && b->block_ids == nullptr) return VTOKEN_ERR_NULL;
  if (b->free_len > 0 && b->free_list == nullptr) return VTOKEN_ERR_NULL;
  return VTOKEN_OK;
}

int64_t min_src_plan_capacity(const vtoken_batch* b, int32_t block_size, bool inplace) {
  // at most min(free_len, M) destinations out of place; at most M in place
  const int64_t f = inplace || b->num_bt_entries < b->free_len ? b->num_bt_entries : b->free_len;
  return f * block_size;
}

vtoken_status check_plan(const vtoken_plan* p, const vtoken_batch* b, int32_t block_size,
                         bool inplace) {
  if (p == nullptr) return VTOKEN_ERR_NULL;
  if (p->dst_indptr == nullptr || p->new_bt_indptr == nullptr || p->freed_indptr == nullptr ||
      p->counters == nullptr) {
    return VTOKEN_ERR_NULL;
  }
  if (b->num_tokens > 0 && p->token_slot == nullptr) return VTOKEN_ERR_NULL;
  if (b->num_reqs > 0 && (p->live_count == nullptr || p->admitted == nullptr)) {
    return VTOKEN_ERR_NULL;
  }
  if (b->num_bt_entries > 0 && p->new_block_ids == nullptr) return VTOKEN_ERR_NULL;
  const int64_t plan_min = min_src_plan_capacity(b, block_size, inplace);
  if (plan_min > 0 && p->src_plan == nullptr) return VTOKEN_ERR_NULL;
  if (p->new_bt_capacity < b->num_bt_entries) return VTOKEN_ERR_CAPACITY;
  if (p->src_plan_capacity < plan_min) return VTOKEN_ERR_CAPACITY;
  return VTOKEN_OK;
}

vtoken::MetaArgs meta_args(const vtoken_cache* c, const vtoken_batch* b, const vtoken_plan* p) {
  vtoken::MetaArgs a;
  a.seq_lens = b->seq_lens;
  a.tok_indptr = b->tok_indptr;
  a.bt_indptr = b->bt_indptr;
  a.block_ids = b->block_ids;
  a.live = b->live;
  a.free_list = b->free_list;
  a.num_reqs = b->num_reqs;
  a.num_tokens = static_cast<int32_t>(b->num_tokens);
  a.num_bt_entries = static_cast<int32_t>(b->num_bt_entries);
  a.free_len = b->free_len;
  a.block_size = c->block_size;
  a.num_blocks = c->num_blocks;
  a.token_slot = p->token_slot;
  a.live_count = p->live_count;
  a.admitted = p->admitted;
  a.dst_indptr = p->dst_indptr;
  a.new_bt_indptr = p->new_bt_indptr;
  a.new_block_ids = p->new_block_ids;
  a.src_plan = p->src_plan;
  a.freed_indptr = p->freed_indptr;
  a.counters = p->counters;
  a.new_bt_capacity = p->new_bt_capacity;
  a.src_plan_capacity = p->src_plan_capacity;
  a.inplace = 0;
  return a;
}

}  // namespace

extern "C" {

vtoken_status vtoken_build_token_table(const vtoken_cache* cache, const vtoken_batch* batch,
                                       const vtoken_plan* plan, hipStream_t stream) {
  vtoken_status s = check_cache(cache);
  if (s != VTOKEN_OK) return s;
  if ((s = check_batch(batch)) != VTOKEN_OK) return s;
  if ((s = check_plan(plan, batch, cache->block_size, false)) != VTOKEN_OK) return s;
  vtoken::MetaArgs a = meta_args(cache, batch, plan);
  a.inplace = 0;
  return hip_status(vtoken::launch_build(a, stream));
}

vtoken_status vtoken_build_token_table_inplace(const vtoken_cache* cache,
                                               const vtoken_batch* batch,
                                               const vtoken_plan* plan, hipStream_t stream) {
  vtoken_status s = check_cache(cache);
  if (s != VTOKEN_OK) return s;
  if ((s = check_batch(batch)) != VTOKEN_OK) return s;
  if ((s = check_plan(plan, batch, cache->block_size, true)) != VTOKEN_OK) return s;
  vtoken::MetaArgs a = meta_args(cache, batch, plan);
  a.inplace = 1;
  a.free_list = nullptr;
  a.free_len = 0;
  return hip_status(vtoken::launch_build(a, stream));
}

vtoken_status vtoken_repack_inplace(const vtoken_cache* cache, const vtoken_batch* batch,
                                    const vtoken_plan* plan, hipStream_t stream) {
  return vtoken_repack_inplace_ex(cache, batch, plan, nullptr, stream);
}

vtoken_status vtoken_repack_inplace_ex(const vtoken_cache* cache, const vtoken_batch* batch,
                                       const vtoken_plan* plan,
                                       const vtoken_repack_options* options,
                                       hipStream_t stream) {
  const int variant = options != nullptr ? options->variant : 0;
  if (variant < 0 || variant > 4 || (options != nullptr && (options->grid != 0 ||
                                                            options->order != 0))) {
    return VTOKEN_ERR_ARGUMENT;
  }
  vtoken_status s = check_cache(cache);
  if (s != VTOKEN_OK) return s;
  if ((s = check_batch(batch)) != VTOKEN_OK) return s;
  if ((s = check_plan(plan, batch, cache->block_size, true)) != VTOKEN_OK) return s;
  const int64_t row = (int64_t)cache->num_kv_heads * cache->head_dim * cache->elem_bytes;
  if ((int64_t)cache->block_size * row > vtoken::kMaxInplaceChunkBytes) return VTOKEN_ERR_SHAPE;
  if ((int64_t)batch->num_reqs * 2 * cache->num_layers > kInt32Limit) return VTOKEN_ERR_SHAPE;
  vtoken::InplaceArgs a;
  a.kv = static_cast<uint8_t*>(cache->kv);
  a.row_bytes = row;
  a.plane_bytes = (int64_t)cache->num_blocks * cache->block_size * row;
  a.num_planes = 2 * cache->num_layers;
  a.block_size = cache->block_size;
  a.num_blocks = cache->num_blocks;
  a.num_slots = cache->num_blocks * cache->block_size;
  a.row_units = static_cast<int32_t>(row / 16);
  a.chunk_units = cache->block_size * a.row_units;
  a.row_magic = a.row_units > 1 ? static_cast<uint32_t>((1ULL << 32) / a.row_units + 1) : 0u;
  a.num_reqs = batch->num_reqs;
  a.src_plan_capacity = plan->src_plan_capacity;
  a.new_bt_capacity = plan->new_bt_capacity;
  a.src_plan = plan->src_plan;
  a.new_block_ids = plan->new_block_ids;
  a.dst_indptr = plan->dst_indptr;
  a.new_bt_indptr = plan->new_bt_indptr;
  a.admitted = plan->admitted;
  a.counters = plan->counters;
  return hip_status(vtoken::launch_repack_inplace(a, variant, stream));
}

}  // extern "C"

namespace {
// The out-of-place copy, and with with_free the freed list in the same launch.
// with_free: vtoken_repack_free, the freed list written by workgroups of the copy's launch
vtoken_status repack_out_of_place(const vtoken_cache* cache, const vtoken_batch* batch,
                                  const vtoken_plan* plan, const vtoken_repack_options* options,
                                  bool with_free, int32_t* freed, int64_t freed_capacity,
                                  hipStream_t stream) {
  vtoken_status s = check_cache(cache);
  if (s != VTOKEN_OK) return s;
  if ((s = check_batch(batch)) != VTOKEN_OK) return s;
  if (plan == nullptr || plan->counters == nullptr) return VTOKEN_ERR_NULL;
  const int64_t plan_min = min_src_plan_capacity(batch, cache->block_size, false);
  if (plan_min > 0 && plan->src_plan == nullptr) return VTOKEN_ERR_NULL;
  if (plan->src_plan_capacity < plan_min) return VTOKEN_ERR_CAPACITY;
  int variant = 0, grid = 0, order = 0;
  if (options != nullptr) {
    variant = options->variant;
    grid = options->grid;
    order = options->order;
  }
  if (variant < 0 || variant >= vtoken::num_repack_variants() || grid < 0 || order < 0 ||
      order > 2) {
    return VTOKEN_ERR_ARGUMENT;
  }
  // the copy never needs more destination blocks than the free list or the plan holds
  const int64_t by_plan = plan->src_plan_capacity / cache->block_size;
  int64_t max_used = batch->free_len < by_plan ? batch->free_len : by_plan;
  // nothing can have been copied (the freed-list workgroups still run: requests with no live
  // token may release blocks, and they check the plan's mode)
  if (max_used == 0 && (!with_free || batch->num_reqs == 0)) return VTOKEN_OK;
  vtoken::CopyArgs a = {};
  a.kv = static_cast<uint8_t*>(cache->kv);
  a.row_bytes = (int64_t)cache->num_kv_heads * cache->head_dim * cache->elem_bytes;
  a.plane_bytes = (int64_t)cache->num_blocks * cache->block_size * a.row_bytes;
  a.num_planes = 2 * cache->num_layers;
  a.block_size = cache->block_size;
  a.num_blocks = cache->num_blocks;
  a.num_slots = cache->num_blocks * cache->block_size;
  a.row_units = static_cast<int32_t>(a.row_bytes / 16);
  a.chunk_units = cache->block_size * a.row_units;
  a.max_used = static_cast<int32_t>(max_used);
  a.row_magic = a.row_units > 1 ? static_cast<uint32_t>((1ULL << 32) / a.row_units + 1) : 0u;
  a.order = order;
  a.src_plan = plan->src_plan;
  a.free_list = batch->free_list;
  a.counters = plan->counters;
  if (with_free) {
    a.num_reqs = batch->num_reqs;
    a.num_bt_entries = batch->num_bt_entries;
    a.bt_indptr = batch->bt_indptr;
    a.block_ids = batch->block_ids;
    a.admitted = plan->admitted;
    a.freed_indptr = plan->freed_indptr;
    a.freed = freed;
    a.freed_capacity = freed_capacity;
  }
  return hip_status(vtoken::launch_repack(a, variant, grid, order, stream));
}
}  // namespace

extern "C" {

vtoken_status vtoken_repack_ex(const vtoken_cache* cache, const vtoken_batch* batch,
                               const vtoken_plan* plan, const vtoken_repack_options* options,
                               hipStream_t stream) {
  return repack_out_of_place(cache, batch, plan, options, false, nullptr, 0, stream);
}

vtoken_status vtoken_repack_free(const vtoken_cache* cache, const vtoken_batch* batch,
                                 const vtoken_plan* plan, int32_t* freed,
                                 int64_t freed_capacity, hipStream_t stream) {
  vtoken_status s = check_batch(batch);
  if (s != VTOKEN_OK) return s;
  if (plan == nullptr || plan->counters == nullptr || plan->freed_indptr == nullptr) {
    return VTOKEN_ERR_NULL;
  }
  if (batch->num_reqs > 0 && plan->admitted == nullptr) return VTOKEN_ERR_NULL;
  if (freed_capacity < batch->num_bt_entries) return VTOKEN_ERR_CAPACITY;
  if (batch->num_bt_entries > 0 && freed == nullptr) return VTOKEN_ERR_NULL;
  return repack_out_of_place(cache, batch, plan, nullptr, true, freed, freed_capacity, stream);
}

vtoken_status vtoken_repack(const vtoken_cache* cache, const vtoken_batch* batch,
                            const vtoken_plan* plan, hipStream_t stream) {
  return vtoken_repack_ex(cache, batch, plan, nullptr, stream);
}

vtoken_status vtoken_free_blocks(const vtoken_batch* batch, const vtoken_plan* plan,
                                 int32_t* freed, int64_t freed_capacity, hipStream_t stream) {
  vtoken_status s = check_batch(batch);
  if (s != VTOKEN_OK) return s;
  if (plan == nullptr || plan->counters == nullptr || plan->freed_indptr == nullptr) {
    return VTOKEN_ERR_NULL;
  }
  if (batch->num_reqs > 0 && plan->admitted == nullptr) return VTOKEN_ERR_NULL;
  if (freed_capacity < batch->num_bt_entries) return VTOKEN_ERR_CAPACITY;
  if (batch->num_bt_entries > 0 && freed == nullptr) return VTOKEN_ERR_NULL;
  vtoken::MetaArgs a = {};
  a.bt_indptr = batch->bt_indptr;
  a.block_ids = batch->block_ids;
  a.num_reqs = batch->num_reqs;
  a.num_bt_entries = static_cast<int32_t>(batch->num_bt_entries);
  a.admitted = plan->admitted;
  a.freed_indptr = plan->freed_indptr;
  a.counters = plan->counters;
  return hip_status(vtoken::launch_free(a, freed, freed_capacity, stream));
}

namespace {

vtoken_status build_slots(const vtoken_batch* batch, const vtoken_plan* plan, int32_t reserve,
                          int32_t* slot_indptr, int32_t* slot_count, int32_t* slots,
                          int64_t slots_capacity, hipStream_t stream) {
  vtoken_status s = check_batch(batch);
  if (s != VTOKEN_OK) return s;
  if (plan == nullptr || plan->counters == nullptr || slot_indptr == nullptr) {
    return VTOKEN_ERR_NULL;
  }
  if (batch->num_reqs > 0 && plan->live_count == nullptr) return VTOKEN_ERR_NULL;
  if (batch->num_tokens > 0 && (plan->token_slot == nullptr || slots == nullptr)) {
    return VTOKEN_ERR_NULL;
  }
  if (reserve < 0) return VTOKEN_ERR_ARGUMENT;
  const int64_t need = batch->num_tokens + (int64_t)batch->num_reqs * reserve;
  if (need > kInt32Limit) return VTOKEN_ERR_SHAPE;
  if (slots_capacity < need) return VTOKEN_ERR_CAPACITY;
  if (need > 0 && slots == nullptr) return VTOKEN_ERR_NULL;
  vtoken::SlotMapArgs a;
  a.num_reqs = batch->num_reqs;
  a.num_tokens = static_cast<int32_t>(batch->num_tokens);
  a.tok_indptr = batch->tok_indptr;
  a.token_slot = plan->token_slot;
  a.live_count = plan->live_count;
  a.counters = plan->counters;
  a.slot_indptr = slot_indptr;
  a.slots = slots;
  a.slots_capacity = slots_capacity;
  a.reserve = reserve;
  a.slot_count = slot_count;
  return hip_status(vtoken::launch_slot_mapping(a, stream));
}

}  // namespace

vtoken_status vtoken_build_slot_mapping(const vtoken_batch* batch, const vtoken_plan* plan,
                                        int32_t* slot_indptr, int32_t* slots,
                                        int64_t slots_capacity, hipStream_t stream) {
  return build_slots(batch, plan, 0, slot_indptr, nullptr, slots, slots_capacity, stream);
}

vtoken_status vtoken_build_slot_table(const vtoken_batch* batch, const vtoken_plan* plan,
                                      int32_t reserve, int32_t* slot_start, int32_t* slot_count,
                                      int32_t* slots, int64_t slots_capacity,
                                      hipStream_t stream) {
  if (batch != nullptr && batch->num_reqs > 0 && slot_count == nullptr) return VTOKEN_ERR_NULL;
  return build_slots(batch, plan, reserve, slot_start, slot_count, slots, slots_capacity,
                     stream);
}

vtoken_status vtoken_append_slots(int32_t num_reqs, const int32_t* append_indptr,
                                  const int32_t* append_slots, const int32_t* slot_start,
                                  int32_t* slot_count, int32_t* slots, int32_t* status,
                                  hipStream_t stream) {
  if (num_reqs < 0) return VTOKEN_ERR_SHAPE;
  if (status == nullptr || append_indptr == nullptr) return VTOKEN_ERR_NULL;
  if (num_reqs > 0 && (append_slots == nullptr || slot_start == nullptr ||
                       slot_count == nullptr || slots == nullptr)) {
    return VTOKEN_ERR_NULL;
  }
  vtoken::AppendArgs a;
  a.num_reqs = num_reqs;
  a.append_indptr = append_indptr;
  a.append_slots = append_slots;
  a.slot_start = slot_start;
  a.slot_count = slot_count;
  a.slots = slots;
  a.status = status;
  return hip_status(vtoken::launch_append_slots(a, stream));
}

int64_t vtoken_decode_workspace_bytes(int32_t num_reqs, int32_t num_q_heads, int32_t head_dim,
                                      int32_t max_tokens) {
  if (num_reqs < 0 || num_q_heads <= 0 || max_tokens < 0) return -1;
  if (head_dim != 32 && head_dim != 64 && head_dim != 128 && head_dim != 256) return -1;
  const int64_t split = vtoken::decode_min_split_tokens(head_dim);
  const int64_t splits = max_tokens > 0 ? (max_tokens + split - 1) / split : 1;
  return (int64_t)num_reqs * num_q_heads * splits * (head_dim + 2) * 4;
}

}  // extern "C"

namespace {

// The paged decode with its split partials in `workspace` (the caller's, or the library-held
// array of the no-alloc entry point; nullptr: the caller's, from *d).
vtoken_status paged_decode(const vtoken_cache* cache, const vtoken_decode* d, int32_t num_reqs,
                           const int32_t* slot_indptr, const int32_t* slots,
                           hipStream_t stream, bool library_workspace) {
  vtoken_status s = check_cache(cache);
  if (s != VTOKEN_OK) return s;
  if (d == nullptr || slot_indptr == nullptr) return VTOKEN_ERR_NULL;
  if (num_reqs < 0 || d->layer < 0 || d->layer >= cache->num_layers || d->max_tokens < 0) {
    return VTOKEN_ERR_SHAPE;
  }
  if (num_reqs == 0) return VTOKEN_OK;
  if (d->q == nullptr || d->out == nullptr || slots == nullptr ||
      (!library_workspace && d->workspace == nullptr)) {
    return VTOKEN_ERR_NULL;
  }
  const int kind = d->kv_dtype;
  if (kind < 0 || kind > 2 || (kind == 2) != (cache->elem_bytes == 1)) return VTOKEN_ERR_SHAPE;
  const int g = cache->num_kv_heads > 0 ? d->num_q_heads / cache->num_kv_heads : 0;
  if (d->num_q_heads <= 0 || d->num_q_heads % cache->num_kv_heads != 0 ||
      (g != 1 && g != 2 && g != 4 && g != 8)) {
    return VTOKEN_ERR_SHAPE;
  }
  const int D = cache->head_dim;
  if (D != 32 && D != 64 && D != 128 && D != 256) return VTOKEN_ERR_SHAPE;
  const int64_t need = vtoken_decode_workspace_bytes(num_reqs, d->num_q_heads, cache->head_dim,
                                                     d->max_tokens);
  if (need < 0) return VTOKEN_ERR_SHAPE;
  if (need > (library_workspace ? vtoken::kDecodeScratchBytes : d->workspace_bytes)) {
    return VTOKEN_ERR_CAPACITY;
  }
  vtoken::AttnArgs a;
  a.kv = static_cast<const uint8_t*>(cache->kv);
  a.row_bytes = (int64_t)cache->num_kv_heads * cache->head_dim * cache->elem_bytes;
  a.plane_bytes = (int64_t)cache->num_blocks * cache->block_size * a.row_bytes;
  a.num_kv_heads = cache->num_kv_heads;
  a.num_q_heads = d->num_q_heads;
  a.head_dim = cache->head_dim;
  a.layer = d->layer;
  a.kv_kind = kind;
  a.num_slots = cache->num_blocks * cache->block_size;
  a.num_reqs = num_reqs;
  const int split = vtoken::decode_split_tokens_w(
      D, cache->elem_bytes, vtoken::decode_waves_for(D, cache->elem_bytes, g, d->max_tokens));
  a.split_tokens = split;
  // in 64 bits: max_tokens may lie within one split of INT32_MAX
  a.splits = d->max_tokens > 0
                 ? static_cast<int32_t>(((int64_t)d->max_tokens + split - 1) / split)
                 : 1;
  const int64_t grid_splits = vtoken::decode_grid_splits(a.splits);
  if ((int64_t)num_reqs * cache->num_kv_heads * grid_splits > INT32_MAX ||
      (int64_t)num_reqs * d->num_q_heads > INT32_MAX) {
    return VTOKEN_ERR_SHAPE;
  }
  a.scale = d->scale;
  a.q = d->q;
  a.out = d->out;
  a.workspace = d->workspace;
  if (library_workspace) {
    // the array's address on the stream's device (no allocation; first call per device)
    const hipError_t e = vtoken::decode_scratch(stream, &a.workspace);
    if (e != hipSuccess) return hip_status(e);
  }
  a.slot_indptr = slot_indptr;
  a.slots = slots;
  a.slot_count = d->slot_count;
  return hip_status(vtoken::launch_paged_decode(a, stream));
}

}  // namespace

extern "C" {

vtoken_status vtoken_paged_decode(const vtoken_cache* cache, const vtoken_decode* d,
                                  int32_t num_reqs, const int32_t* slot_indptr,
                                  const int32_t* slots, hipStream_t stream) {
  return paged_decode(cache, d, num_reqs, slot_indptr, slots, stream, false);
}

vtoken_status vtoken_paged_decode_noalloc(const vtoken_cache* cache, const vtoken_decode* d,
                                          int32_t num_reqs, const int32_t* slot_indptr,
                                          const int32_t* slots, hipStream_t stream) {
  return paged_decode(cache, d, num_reqs, slot_indptr, slots, stream, true);
}

vtoken_status vtoken_plan_partial(const vtoken_cache* cache, const vtoken_batch* batch,
                                  const int32_t* slot_in, const vtoken_planner_params* params,
                                  const vtoken_planner_state* st, const vtoken_plan* plan,
                                  hipStream_t stream) {
  vtoken_status s = check_cache(cache);
  if (s != VTOKEN_OK) return s;
  if ((s = check_batch(batch)) != VTOKEN_OK) return s;
  if (params == nullptr || st == nullptr || plan == nullptr) return VTOKEN_ERR_NULL;
  const int S = cache->block_size;
  if (S > 64) return VTOKEN_ERR_SHAPE;
  if (params->theta_den <= 0 || params->max_sources < 0 || params->min_eligible < 0 ||
      params->reserved != 0) {
    return VTOKEN_ERR_ARGUMENT;
  }
  const int32_t R = batch->num_reqs;
  const int64_t T = batch->num_tokens, M = batch->num_bt_entries;
  if (st->live_bits == nullptr || st->refs == nullptr || st->n_b == nullptr ||
      st->selected == nullptr || st->stats == nullptr || plan->counters == nullptr ||
      plan->dst_indptr == nullptr || plan->new_bt_indptr == nullptr ||
      plan->freed_indptr == nullptr) {
    return VTOKEN_ERR_NULL;
  }
  if (R > 0 && (st->src_count == nullptr || plan->live_count == nullptr ||
                plan->admitted == nullptr)) {
    return VTOKEN_ERR_NULL;
  }
  if (T > 0 && (slot_in == nullptr || plan->token_slot == nullptr)) return VTOKEN_ERR_NULL;
  if (M > 0 && (st->elig_cum == nullptr || st->sources == nullptr ||
                plan->new_block_ids == nullptr)) {
    return VTOKEN_ERR_NULL;
  }
  if (plan->new_bt_capacity < M) return VTOKEN_ERR_CAPACITY;
  const int64_t plan_min = (batch->free_len < M ? batch->free_len : M) * (int64_t)S;
  if (plan_min > 0 && plan->src_plan == nullptr) return VTOKEN_ERR_NULL;
  if (plan->src_plan_capacity < plan_min) return VTOKEN_ERR_CAPACITY;
  vtoken::PlannerArgs a = {};
  a.num_reqs = R;
  a.num_tokens = static_cast<int32_t>(T);
  a.num_bt_entries = static_cast<int32_t>(M);
  a.block_size = S;
  a.num_blocks = cache->num_blocks;
  a.num_slots = cache->num_blocks * S;
  a.free_len = batch->free_len;
  a.theta_num = params->theta_num;
  a.theta_den = params->theta_den;
  if (params->max_live_per_source >= 0) {
    a.max_live = params->max_live_per_source;
  } else {
    // largest n with n * den < (den - num) * S: the block's own waste exceeds theta_F
    const int64_t lim = ((int64_t)params->theta_den - params->theta_num) * S;
    a.max_live = lim > 0 ? static_cast<int32_t>((lim - 1) / params->theta_den) : -1;
  }
  a.min_eligible = params->min_eligible;
  a.free_watermark = params->free_watermark;
  a.max_sources = params->max_sources;
  a.seq_lens = batch->seq_lens;
  a.tok_indptr = batch->tok_indptr;
  a.bt_indptr = batch->bt_indptr;
  a.block_ids = batch->block_ids;
  a.live = batch->live;
  a.slot_in = slot_in;
  a.free_list = batch->free_list;
  a.pinned = st->pinned;
  a.live_bits = st->live_bits;
  a.refs = st->refs;
  a.n_b = st->n_b;
  a.selected = st->selected;
  a.elig_cum = st->elig_cum;
  a.src_count = st->src_count;
  a.sources = st->sources;
  a.stats = st->stats;
  a.token_slot = plan->token_slot;
  a.live_count = plan->live_count;
  a.admitted = plan->admitted;
  a.dst_indptr = plan->dst_indptr;
  a.new_bt_indptr = plan->new_bt_indptr;
  a.new_block_ids = plan->new_block_ids;
  a.src_plan = plan->src_plan;
  a.freed_indptr = plan->freed_indptr;
  a.counters = plan->counters;
  a.new_bt_capacity = plan->new_bt_capacity;
  a.src_plan_capacity = plan->src_plan_capacity;
  return hip_status(vtoken::launch_planner(a, stream));
}

int64_t vtoken_check_layout_workspace_bytes(int32_t num_blocks) {
  if (num_blocks <= 0) return -1;
  return 4 * vtoken::layout_words(num_blocks);
}

vtoken_status vtoken_check_layout(const vtoken_cache* cache, const vtoken_batch* batch,
                                  void* workspace, int64_t workspace_bytes, int32_t* status,
                                  hipStream_t stream) {
  vtoken_status s = check_cache(cache);
  if (s != VTOKEN_OK) return s;
  if ((s = check_batch(batch)) != VTOKEN_OK) return s;
  if (workspace == nullptr || status == nullptr) return VTOKEN_ERR_NULL;
  if (workspace_bytes < vtoken_check_layout_workspace_bytes(cache->num_blocks)) {
    return VTOKEN_ERR_CAPACITY;
  }
  vtoken::LayoutArgs a;
  a.block_ids = batch->block_ids;
  a.free_list = batch->free_list;
  a.num_bt_entries = batch->num_bt_entries;
  a.free_len = batch->free_len;
  a.num_blocks = cache->num_blocks;
  a.num_words = vtoken::layout_words(cache->num_blocks);
  a.words = static_cast<uint32_t*>(workspace);
  a.status = status;
  return hip_status(vtoken::launch_check_layout(a, stream));
}

int32_t vtoken_last_hip_error(void) { return g_last_hip_error; }

const char* vtoken_status_string(int32_t status) {
  switch (status) {
    case VTOKEN_OK: return "VTOKEN_OK";
    case VTOKEN_ERR_NULL: return "VTOKEN_ERR_NULL: a required pointer is NULL";
    case VTOKEN_ERR_SHAPE: return "VTOKEN_ERR_SHAPE: invalid cache geometry or batch sizes";
    case VTOKEN_ERR_CAPACITY: return "VTOKEN_ERR_CAPACITY: an output buffer is too small";
    case VTOKEN_ERR_HIP: return "VTOKEN_ERR_HIP: the HIP runtime reported an error";
    case VTOKEN_ERR_ARGUMENT: return "VTOKEN_ERR_ARGUMENT: invalid repack option";
    case VTOKEN_ERR_BLOCK_RANGE: return "VTOKEN_ERR_BLOCK_RANGE: block id outside the pool";
    case VTOKEN_ERR_BT_LEN: return "VTOKEN_ERR_BT_LEN: block table length != ceil(len/S)";
    case VTOKEN_ERR_TOK_LEN: return "VTOKEN_ERR_TOK_LEN: token range != sequence length";
    case VTOKEN_ERR_SLOT: return "VTOKEN_ERR_SLOT: a live token's slot is invalid for its table";
    case VTOKEN_ERR_LAYOUT: return "VTOKEN_ERR_LAYOUT: a block id is held twice";
    case VTOKEN_ERR_PLAN_MODE:
      return "VTOKEN_ERR_PLAN_MODE: the plan was built for another mode of the pass";
    default: return "unknown vtoken status";
  }
}

int32_t vtoken_version(void) { return 200; }

const char* vtoken_build_id(void) {
#if defined(VTOKEN_SRC_SHA0) && defined(VTOKEN_SRC_SHA1) && defined(VTOKEN_SRC_SHA2) && \
    defined(VTOKEN_SRC_SHA3)
  // the four 64-bit words of the sources' SHA-256, as 64 hex digits (a constant string)
  static const char* id = [] {
    static char buf[65];
    const unsigned long long w[4] = {VTOKEN_SRC_SHA0, VTOKEN_SRC_SHA1, VTOKEN_SRC_SHA2,
                                     VTOKEN_SRC_SHA3};
    const char* hex = "0123456789abcdef";
    for (int i = 0; i < 4; ++i)
      for (int j = 0; j < 16; ++j) buf[16 * i + j] = hex[(w[i] >> (60 - 4 * j)) & 0xF];
    buf[64] = 0;
    return buf;
  }();
  return id;
#else
  return "unknown";
#endif
}

}  // extern "C"
