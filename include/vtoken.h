/*
 * vtoken.h - C ABI of the vToken KV repack for AMD Instinct MI355X (gfx950).
 *
 * The repack turns token-level liveness into reusable KV blocks, as described in
 * "vToken: Token-Level Virtualization for Reclaimable KV Caches" (arXiv 2608.13263):
 * the token table of Sec. 3.2, the reclamation backend of Sec. 3.3 (headroom-aware
 * admission Sec. 3.3.2, relocation planning Sec. 3.3.3, copy Sec. 3.3.4) and the slot
 * formula of Sec. 3.4 (slot = block_id * block_size + offset).
 *
 * One repack pass is three calls, enqueued in this order on one HIP stream:
 *
 *   vtoken_build_token_table   per-request exclusive scan of the live mask, admission of
 *                              requests against the free list, token table, new block
 *                              tables and the per-destination-block source plan
 *   vtoken_repack              gathers every live K/V row of every admitted request into
 *                              densely packed destination blocks, all layers, K and V, and
 *                              all KV heads in one launch (the only call touching KV bytes)
 *   vtoken_free_blocks         emits the list of freed source blocks
 *
 * vtoken_repack_free enqueues the last two in one launch (same effects and errors).
 *
 * General conventions (all calls):
 *   - Pointers inside the structs are DEVICE pointers unless a field says [host].
 *   - The caller owns every buffer; the library keeps no pointer after a call returns,
 *     allocates no memory and never synchronises: every call only enqueues kernels on
 *     `stream` and returns. The calls therefore may be captured into a HIP graph.
 *   - Host-side argument errors return a negative status synchronously and enqueue
 *     nothing. Errors that only the device can see (a bad block id, inconsistent CSR
 *     lengths, a capacity exceeded) are written to plan->counters[3] by the kernels of
 *     vtoken_build_token_table, before any table is built (a copy handed a plan of the
 *     other mode writes VTOKEN_ERR_PLAN_MODE there); every later kernel reads that word
 *     and does nothing when it is not VTOKEN_OK. The caller inspects it after its own
 *     sync.
 *     Every kernel bounds-checks what it dereferences, so no status path writes
 *     outside the buffers the caller described.
 *   - The library is re-entrant: calls on different streams with disjoint buffers may
 *     run concurrently. Calls that share a plan or a KV cache must be stream-ordered.
 *
 * Conventions the paper leaves open (frozen here; the CPU oracle follows the same ones):
 *   - Out-of-place relocation (Sec. 3.3.2): destinations are taken from the caller's
 *     free list front to back, requests in ascending index order; sources are never
 *     written; source blocks are released only by vtoken_free_blocks, after the copy
 *     (Sec. 3.3.4, invariant I3 of Sec. 3.5).
 *   - Every block of a request is a relocation source (the source batch of Sec. 3.3.3
 *     is the whole request); a request needs ceil(live / block_size) destinations.
 *   - A request is profitable iff it needs strictly fewer blocks than it holds (Sec.
 *     3.3.3, invariant I4). Profitable requests are admitted in ascending order while
 *     the free list can supply their destinations; once one is deferred every later
 *     profitable request is deferred too (prefix admission, Sec. 3.3.2). Unprofitable
 *     and deferred requests keep their block table and slots.
 *   - Live tokens keep their logical order and fill each destination block completely
 *     before the next (Sec. 3.3.3): the token of rank k goes to destination block
 *     k / block_size, offset k % block_size.
 *   - Dead tokens get token_slot -1 (Sec. 3.2, evict_token). The tail slots of the last
 *     destination block and all non-destination bytes keep their previous contents.
 *   - freed = concatenation over admitted requests (ascending) of all their old blocks
 *     in block-table order.
 *   - Layout precondition of the full pass: every block id appears at most once over all
 *     block tables and free_list[0 .. free_len). An admitted request releases all its
 *     blocks, so a block held by two tables would be released twice and a block both held
 *     and free could be overwritten while live. Caches with shared-prefix blocks use
 *     vtoken_plan_partial, which keeps blocks held by several tables in place (I4 of Sec.
 *     3.5, Sec. 5.7). vtoken_check_layout verifies the precondition on the device.
 *
 * KV layout: one contiguous buffer of 2*num_layers planes, plane index 2*layer + (0 for K,
 * 1 for V); each plane is [num_blocks][block_size][num_kv_heads][head_dim] elements of
 * elem_bytes bytes. The row of one token in one plane is num_kv_heads*head_dim*elem_bytes
 * contiguous bytes (head_dim fastest). The payload is copied as opaque bytes, so any
 * 1- or 2-byte element type (fp8, fp16, bf16) is supported and NaN payloads survive.
 * One token table and one block table drive all planes: the table is per sequence, not
 * per layer or head (Sec. 3.2).
 */
#ifndef VTOKEN_H
#define VTOKEN_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum vtoken_status {
  VTOKEN_OK = 0,
  VTOKEN_ERR_NULL = -1,       /* a required pointer is NULL                                */
  VTOKEN_ERR_SHAPE = -2,      /* a dimension <= 0, elem_bytes not 1 or 2, a row not a      */
                              /* multiple of 16 bytes, num_blocks*block_size >= 2^31,      */
                              /* num_tokens >= 2^31 or negative lengths                    */
  VTOKEN_ERR_CAPACITY = -3,   /* an output capacity below the documented minimum           */
  VTOKEN_ERR_HIP = -4,        /* the HIP runtime reported an error at launch               */
  VTOKEN_ERR_ARGUMENT = -5,   /* an invalid tuning option (vtoken_repack_ex)               */
  /* device-detected, written to plan->counters[3]: */
  VTOKEN_ERR_BLOCK_RANGE = -10, /* a block id in block_ids or in the consumed part of    */
                                /* free_list lies outside [0, num_blocks)                */
  VTOKEN_ERR_BT_LEN = -11,      /* bt_indptr[r+1]-bt_indptr[r] != ceil(seq_lens[r]/S),   */
                                /* or bt_indptr outside [0, num_bt_entries]              */
  VTOKEN_ERR_TOK_LEN = -12,     /* tok_indptr[r+1]-tok_indptr[r] != seq_lens[r] or       */
                                /* tok_indptr outside [0, num_tokens]                    */
  VTOKEN_ERR_SLOT = -13,        /* vtoken_plan_partial: a live token's slot lies outside */
                                /* [0, num_blocks*S), or the live tokens of a request's  */
                                /* sources do not match the live slots counted in them   */
                                /* (two tokens on one slot, a slot outside its table)    */
  VTOKEN_ERR_LAYOUT = -14,      /* vtoken_check_layout: a block id held twice over the   */
                                /* block tables and the free list                        */
  VTOKEN_ERR_PLAN_MODE = -15    /* a call was handed a plan built for another mode       */
                                /* (vtoken_repack[_ex] needs a plan of                   */
                                /* vtoken_build_token_table or vtoken_plan_partial,      */
                                /* vtoken_repack_inplace[_ex] one of                     */
                                /* vtoken_build_token_table_inplace; vtoken_free_blocks  */
                                /* and vtoken_repack_free refuse a plan of               */
                                /* vtoken_plan_partial); nothing is copied or released   */
} vtoken_status;

/* The paged KV cache (Sec. 2.1). */
typedef struct vtoken_cache {
  void*   kv;            /* device, [2*num_layers][num_blocks][block_size][H][D], see above */
  int32_t num_layers;    /* L                                                               */
  int32_t num_kv_heads;  /* H (KV heads; GQA/MQA only change H, Sec. 6)                     */
  int32_t head_dim;      /* D                                                               */
  int32_t block_size;    /* S, tokens per block                                             */
  int32_t num_blocks;    /* blocks per plane; block ids are shared by all planes            */
  int32_t elem_bytes;    /* 1 (fp8) or 2 (fp16, bf16)                                       */
} vtoken_cache;

/* The requests of one repack pass, in CSR form. Request r has seq_lens[r] tokens; its
 * tokens' live bits are live[tok_indptr[r] .. tok_indptr[r+1]) (1 live, 0 evicted: the
 * evict_token call of Sec. 3.2 is a write of 0 there), and its block table (Sec. 2.1) is
 * block_ids[bt_indptr[r] .. bt_indptr[r+1]) with exactly ceil(seq_lens[r]/S) entries.
 * Token position p of request r lives at slot block_ids[bt_indptr[r] + p/S]*S + p%S. */
typedef struct vtoken_batch {
  int32_t        num_reqs;       /* R                                     [host]            */
  int64_t        num_tokens;     /* T = tok_indptr[R]                     [host]            */
  int64_t        num_bt_entries; /* M = bt_indptr[R]                      [host]            */
  const int32_t* seq_lens;       /* [R]                                                     */
  const int32_t* tok_indptr;     /* [R+1]                                                   */
  const int32_t* bt_indptr;      /* [R+1]                                                   */
  const int32_t* block_ids;      /* [M]                                                     */
  const uint8_t* live;           /* [T]                                                     */
  const int32_t* free_list;      /* [free_len] destination supply, consumed front to back   */
  int32_t        free_len;       /* f                                     [host]            */
} vtoken_batch;

/* Caller-allocated outputs of vtoken_build_token_table; read by the two later calls.
 * They form the bulk apply_moves of Sec. 3.2: token_slot and the new block tables are
 * valid for attention once vtoken_repack has executed on the stream. */
typedef struct vtoken_plan {
  int32_t* token_slot;      /* [T]   slot of every token after the pass; -1 if dead         */
  int32_t* live_count;      /* [R]   live tokens per request                                */
  int32_t* admitted;        /* [R]   1 repacked in this pass, 0 unchanged                   */
  int32_t* dst_indptr;      /* [R+1] exclusive scan of admitted*need: request r's          */
                            /*       destinations are free_list[dst_indptr[r] ..)           */
  int32_t* new_bt_indptr;   /* [R+1] exclusive scan of the new block-table lengths          */
  int32_t* new_block_ids;   /* [new_bt_capacity] new block tables, CSR by new_bt_indptr     */
  int32_t* src_plan;        /* [src_plan_capacity] for destination block g (the g-th       */
                            /*       consumed free-list entry) and offset j, entry g*S+j is */
                            /*       the source slot of the token placed there, -1 if none */
  int32_t* freed_indptr;    /* [R+1] exclusive scan of admitted*old_blocks                  */
  int32_t* counters;        /* [5]   used free-list entries, admitted requests, freed       */
                            /*       blocks, status (VTOKEN_OK or a device error code),     */
                            /*       plan mode (1 out of place, 2 in place, 3 partial pass; */
                            /*       checked by the copy and the freed list, which set      */
                            /*       VTOKEN_ERR_PLAN_MODE on a mismatch)                    */
  int64_t  new_bt_capacity;   /* entries in new_block_ids, >= M            [host]           */
  int64_t  src_plan_capacity; /* entries in src_plan, >= min(free_len, M)*S [host]         */
} vtoken_plan;

/* Step 1 (Sec. 3.2, 3.3.2, 3.3.3): scan, admission, token table, block tables, plan.
 * Writes every field of *plan (device memory) except new_bt/src_plan capacity beyond
 * what is used. Returns VTOKEN_OK once the kernels are enqueued: one kernel for batches of
 * at most 24 requests and 8,192 tokens, two (counts, then tables) up to 256 requests or up
 * to 512 averaging at least 1,024 tokens, three (counts, admission, tables) above. */
vtoken_status vtoken_build_token_table(const vtoken_cache* cache, const vtoken_batch* batch,
                                       const vtoken_plan* plan, hipStream_t stream);

/* Step 2 (Sec. 3.3, lazy compaction; Sec. 3.3.4 copy): for every admitted request r, every
 * live token and every plane, copies the token's row from its old slot to its new slot.
 * Reads plan->src_plan, plan->counters and batch->free_list; writes KV bytes of the
 * destination rows only. Idempotent on unchanged inputs (sources are never written).
 * Must follow vtoken_build_token_table on the same stream. */
vtoken_status vtoken_repack(const vtoken_cache* cache, const vtoken_batch* batch,
                            const vtoken_plan* plan, hipStream_t stream);

/* Step 3 (Sec. 3.3.4: sources are returned only after the packed layout is committed):
 * writes freed[0 .. counters[2]) = old blocks of the admitted requests (in-place mode: the
 * blocks past each admitted request's new table). Stream order after vtoken_repack is what
 * makes reuse of these blocks safe. freed_capacity >= M. A plan of vtoken_plan_partial (whose
 * released blocks are its state's sources) is refused: nothing is written and counters[3]
 * becomes VTOKEN_ERR_PLAN_MODE. */
vtoken_status vtoken_free_blocks(const vtoken_batch* batch, const vtoken_plan* plan,
                                 int32_t* freed, int64_t freed_capacity, hipStream_t stream);

/* Steps 2 and 3 in one launch (Sec. 3.3.4): vtoken_repack followed by vtoken_free_blocks on
 * a plan of vtoken_build_token_table, for callers that enqueue the two back to back. Same
 * arguments, checks, outputs and errors as the two calls in that order (freed_capacity >= M;
 * the copy uses the default options; a plan of vtoken_plan_partial is refused with
 * VTOKEN_ERR_PLAN_MODE and nothing is copied). The freed list is written by the copy's own
 * launch (one workgroup per request after the copy's); the blocks in it may be reused once
 * that launch has executed on the stream, as after vtoken_free_blocks. */
vtoken_status vtoken_repack_free(const vtoken_cache* cache, const vtoken_batch* batch,
                                 const vtoken_plan* plan, int32_t* freed,
                                 int64_t freed_capacity, hipStream_t stream);

/* Debug check of the full pass's layout precondition (see the conventions above): every id
 * in block_ids[0 .. M) and free_list[0 .. free_len) lies in [0, num_blocks) and appears at
 * most once over both. Writes to *status (device int32): VTOKEN_OK; VTOKEN_ERR_BLOCK_RANGE if
 * any id lies outside the pool (reported before duplicates); else VTOKEN_ERR_LAYOUT if any id
 * appears twice. workspace: device, at least vtoken_check_layout_workspace_bytes(num_blocks)
 * bytes (a flag word and one bit per block), overwritten by the call. Reads only the batch's
 * block_ids and free_list (seq_lens, live and the CSR ranges are not inspected); touches no
 * KV byte; enqueues three small kernels on `stream`. */
int64_t vtoken_check_layout_workspace_bytes(int32_t num_blocks);
vtoken_status vtoken_check_layout(const vtoken_cache* cache, const vtoken_batch* batch,
                                  void* workspace, int64_t workspace_bytes, int32_t* status,
                                  hipStream_t stream);

/* In-place mode (an extension beyond the paper's out-of-place relocation, Sec. 3.3.2):
 * the destinations of a repacked request are its own first ceil(live/S) blocks, so no free
 * list is needed and every profitable request is repacked; the freed blocks are the rest of
 * its old table, and rows already in place are not copied. batch->free_list is ignored.
 * plan outputs have the same meaning as out of place, except that counters[0] counts the
 * destination blocks (rows of src_plan) and dst_indptr indexes src_plan only; the plan must
 * hold src_plan_capacity >= M*S. Call order: vtoken_build_token_table_inplace, then
 * vtoken_repack_inplace, then vtoken_free_blocks (the freed list is the released tails).
 * vtoken_repack_inplace requires block_size*row_bytes <= 64 KiB (VTOKEN_ERR_SHAPE otherwise):
 * one workgroup walks each (request, plane) chain in block order and holds one destination
 * block's moving rows at a time (in registers by default; in LDS with the staging variants of
 * vtoken_repack_inplace_ex), so that a block is written only after every read of its own and
 * earlier destination blocks. Handed a plan of vtoken_build_token_table, it copies nothing and
 * sets counters[3] to VTOKEN_ERR_PLAN_MODE (and vtoken_repack does the same with an in-place
 * plan). */
vtoken_status vtoken_build_token_table_inplace(const vtoken_cache* cache,
                                               const vtoken_batch* batch,
                                               const vtoken_plan* plan, hipStream_t stream);
vtoken_status vtoken_repack_inplace(const vtoken_cache* cache, const vtoken_batch* batch,
                                    const vtoken_plan* plan, hipStream_t stream);

/* Tuning entry for the copy of step 2; vtoken_repack uses the defaults (all fields 0).
 *   variant: cache policy of the copy's 16-byte loads and stores (CDNA4 cache-policy bits)
 *            0 default (= 4), 1 plain loads and stores, 2 non-temporal loads and stores,
 *            3 non-temporal loads and plain stores, 4 non-temporal loads and sc1 stores,
 *            5 non-temporal loads and sc0 sc1 stores, 6 non-temporal loads, sc1 nt stores
 *   grid:    workgroups of the copy launch; 0 = one per work item that the free list and
 *            plan can hold, capped at 2^19 (a grid-stride loop covers any remainder); a work
 *            item is one 32 KiB part (at most) of a destination block in one plane. Every
 *            workgroup is dispatched even when the plan admits nothing (the work is counted
 *            on the device), at about 4.7 per ns on MI355X: such a pass takes 0.112 ms at
 *            2^19, 0.016 ms at 2^16. Measured, 2^16 costs a full copy 0.1% (Llama-3-8B
 *            Random) to 0.5% (Llama-3-8B H2O); callers whose passes mostly admit nothing
 *            may prefer it
 *   order:   work order over (part of a destination block, plane) items: 0 default (= 2),
 *            1 plane-major, 2 block-major (all planes of one part together)
 * All settings produce identical bytes; they differ only in speed. Invalid values return
 * VTOKEN_ERR_ARGUMENT. */
typedef struct vtoken_repack_options {
  int32_t variant;
  int32_t grid;
  int32_t order;
  int32_t reserved;
} vtoken_repack_options;

vtoken_status vtoken_repack_ex(const vtoken_cache* cache, const vtoken_batch* batch,
                               const vtoken_plan* plan, const vtoken_repack_options* options,
                               hipStream_t stream);

/* Tuning entry for the in-place copy; vtoken_repack_inplace uses the default (variant 0).
 *   variant: how a destination block is staged between its reads and its writes:
 *            0 default (4 for block_size <= 64, else 3), 1 LDS double buffer (direct
 *            global->LDS loads; falls back to
 *            2 when two blocks exceed 64 KiB), 2 LDS single buffer, 3 registers, 4 registers
 *            with the next moving block's reads in flight while a block is written
 *            (block_size <= 64; larger blocks use 3)
 *   grid, order: must be 0 (one workgroup per (request, plane) chain)
 * All variants produce identical bytes. */
vtoken_status vtoken_repack_inplace_ex(const vtoken_cache* cache, const vtoken_batch* batch,
                                       const vtoken_plan* plan,
                                       const vtoken_repack_options* options,
                                       hipStream_t stream);

/* ---- Partial reclamation pass (Sec. 3.3.1-3.3.3; I4 of Sec. 3.5; Sec. 5.7) ----
 *
 * The paper's planner: per-block live counts n_b and the waste ratio F (Sec. 2.3.1), the
 * trigger F > theta_F with enough low-utilisation blocks and the free list near its low
 * watermark (Sec. 3.3.2), and per request its low-utilisation source blocks only, at most B
 * source blocks considered in the pass (Sec. 3.3.3). Shared-prefix blocks - blocks that appear
 * in more than one request's table - and pinned blocks are never sources (I4, Sec. 5.7).
 *
 * Input is a token table: slot_in[t] (device, int32 [num_tokens]) is the current slot of
 * logical token t, -1 if it holds none; a live token's slot must lie in a block of its own
 * request's table (blocks of a table may be in any order and hold tokens in any order, so
 * passes can follow each other). bt_indptr gives each request's table (any length); the
 * token CSR is as for the full pass. block_size <= 64.
 *
 * Readings (also those of the CPU reference): a block is a candidate iff it is in exactly
 * one table, not pinned, and n_b <= max_live_per_source; F > theta_num/theta_den is decided
 * exactly in integers; the pass is attempted iff F > theta_F, at least min_eligible
 * candidates exist and (free_watermark < 0 or free_len <= free_watermark); candidates are
 * considered in request order, table order within a request, until max_sources (B) have
 * been considered, admitted or not; T_live = live tokens of a request's considered sources,
 * need = ceil(T_live/S), a plan exists iff 0 < sources and need < sources; admission is the
 * prefix rule of the full pass over free_list; the move list takes the live tokens of the
 * sources in logical order into the destinations (each filled before the next); the new table
 * is the kept blocks in order followed by the destinations; dead tokens map to -1.
 *
 * Outputs go to the vtoken_plan (sizes as for vtoken_build_token_table: token_slot [T],
 * live_count / admitted [R], CSR offsets [R+1], new_block_ids with new_bt_capacity >= M,
 * src_plan with src_plan_capacity >= min(free_len, M)*S, counters [5] = {destination blocks
 * used, requests admitted, sources released, status, plan mode 3}) and to the state buffers
 * below. The copy is vtoken_repack on the same plan, enqueued after this call. The released
 * sources are state->sources[0 .. counters[2]) (CSR by freed_indptr): reuse them only after
 * the copy has executed on the stream; vtoken_free_blocks and vtoken_repack_free refuse this
 * plan (VTOKEN_ERR_PLAN_MODE). */
typedef struct vtoken_planner_params {
  int32_t theta_num;            /* theta_F = theta_num / theta_den (paper default 1/4)       */
  int32_t theta_den;            /* > 0                                                        */
  int32_t max_live_per_source;  /* < 0: the block's own waste exceeds theta_F, i.e.          */
                                /* n_b * theta_den < (theta_den - theta_num) * S             */
  int32_t min_eligible;         /* candidates needed for an attempt (>= 0)                   */
  int32_t free_watermark;       /* attempt only if free_len <= this; < 0: no condition      */
  int32_t reserved;             /* 0                                                          */
  int64_t max_sources;          /* B, >= 0                                                    */
} vtoken_planner_params;

typedef struct vtoken_planner_state {   /* caller-allocated device buffers */
  uint64_t* live_bits;   /* [num_blocks] scratch: live slots of each block                   */
  int32_t*  refs;        /* [num_blocks] out: tables holding each block                      */
  int32_t*  n_b;         /* [num_blocks] out: live tokens of each block (0 if unallocated)   */
  int32_t*  selected;    /* [num_blocks] scratch                                             */
  int32_t*  elig_cum;    /* [num_bt_entries] scratch                                         */
  int32_t*  src_count;   /* [num_reqs] out: sources considered per request                   */
  int32_t*  sources;     /* [num_bt_entries] out: released source blocks (CSR freed_indptr)  */
  int64_t*  stats;       /* [8] out: sum n_b, allocated blocks N, candidates, attempted      */
                         /* (0/1), sources considered, tokens moved, sources released,       */
                         /* destination blocks used                                          */
  const uint8_t* pinned; /* [num_blocks] or NULL: nonzero = never a source                   */
} vtoken_planner_state;

vtoken_status vtoken_plan_partial(const vtoken_cache* cache, const vtoken_batch* batch,
                                  const int32_t* slot_in, const vtoken_planner_params* params,
                                  const vtoken_planner_state* state, const vtoken_plan* plan,
                                  hipStream_t stream);

/* ---- Consumer side (Sec. 3.4: slot mapping; Sec. 3.3.4 and I3 of Sec. 3.5: ordering) ----
 *
 * The attention slot mapping: for every request, the slots of its live tokens in logical
 * order, looked up once per token through the token table (Sec. 3.4). Reads plan->token_slot,
 * plan->live_count and plan->counters of a preceding vtoken_build_token_table[_inplace] on the
 * same stream (no-op when counters[3] is set); the slots are valid for attention once the
 * matching repack has executed on the stream. slot_indptr [R+1] is the exclusive scan of the
 * live counts; slots [slots_capacity >= num_tokens] receives the slots in CSR order. */
vtoken_status vtoken_build_slot_mapping(const vtoken_batch* batch, const vtoken_plan* plan,
                                        int32_t* slot_indptr, int32_t* slots,
                                        int64_t slots_capacity, hipStream_t stream);

/* The slot mapping as a translation cache that grows append-only (Sec. 3.2: the cached
 * translation array is extended by the new entries as a sequence grows, and rebuilt only after
 * a structural change - eviction or relocation). vtoken_build_slot_table is the rebuild: like
 * vtoken_build_slot_mapping, but request r's region is slot_start[r] .. slot_start[r+1] with
 * room for `reserve` more slots after its live_count[r] ones; slot_count[r] = live_count[r].
 * slots_capacity >= num_tokens + num_reqs * reserve. vtoken_append_slots appends
 * append_slots[append_indptr[r] .. append_indptr[r+1]) (device, int32) to request r's region
 * and adds their number to slot_count[r]; a request whose region would overflow is left
 * unchanged and *status (device int32, written by the call) becomes VTOKEN_ERR_CAPACITY (a
 * rebuild is due), else 0. Decode reads a slot table with vtoken_decode.slot_count set. */
vtoken_status vtoken_build_slot_table(const vtoken_batch* batch, const vtoken_plan* plan,
                                      int32_t reserve, int32_t* slot_start, int32_t* slot_count,
                                      int32_t* slots, int64_t slots_capacity,
                                      hipStream_t stream);
vtoken_status vtoken_append_slots(int32_t num_reqs, const int32_t* append_indptr,
                                  const int32_t* append_slots, const int32_t* slot_start,
                                  int32_t* slot_count, int32_t* slots, int32_t* status,
                                  hipStream_t stream);

/* Decode attention of one layer over the paged cache through a slot mapping: for request r
 * and query head qh (GQA: KV head qh / (num_q_heads / num_kv_heads)),
 *   out[r][qh] = softmax(scale * q[r][qh] . K[slot]^T) @ V[slot] over the slots of r,
 * K and V being the layer's K and V planes (float32 math; zeros for a request with no slots).
 * Flash-decoding: splits of 32 KiB of K per KV head (32768 / (head_dim * elem_bytes) tokens;
 * 64 KiB for 2-byte caches with 8 query heads per KV head, or when max_tokens spans 64 or
 * more 32 KiB splits), then a merge; the workspace
 * holds the split partials and is overwritten by every call (calls sharing it must be
 * stream-ordered). A request with more slots than max_tokens provides for is never
 * truncated: its outputs are NaN, unless its slots still fit the ceil(max_tokens / split)
 * splits, which are all computed. A slot outside the pool (negative
 * or >= num_blocks * block_size) is never dereferenced; its request's outputs are NaN. A
 * request whose slot range is malformed (slot_indptr[r] < 0, or a negative count:
 * slot_indptr[r+1] < slot_indptr[r], or slot_count[r] < 0) reads no slot and gets NaN
 * outputs. The split launch has R * num_kv_heads * ceil(max_tokens / split) workgroups, and
 * those past a request's slots return at once: pass the batch's largest slot count rather
 * than a model's context limit (on MI355X a bound 2, 4 and 8 times too large cost the
 * Llama-3-8B Random decode 2%, 8% and 25%). */
enum { VTOKEN_KV_FP16 = 0, VTOKEN_KV_BF16 = 1, VTOKEN_KV_FP8_E4M3 = 2 };

typedef struct vtoken_decode {
  const float* q;          /* device [R][num_q_heads][head_dim] float32                    */
  float*       out;        /* device [R][num_q_heads][head_dim] float32                    */
  int32_t      num_q_heads; /* num_kv_heads times 1, 2, 4 or 8                              */
  int32_t      layer;      /* 0 <= layer < num_layers                                       */
  int32_t      kv_dtype;   /* VTOKEN_KV_*; fp8 (OCP e4m3) iff elem_bytes == 1               */
  float        scale;      /* softmax scale, usually 1/sqrt(head_dim)                       */
  int32_t      max_tokens; /* [host] >= the slot count of every request (else NaN outputs)  */
  float*       workspace;  /* device, >= vtoken_decode_workspace_bytes() bytes              */
  int64_t      workspace_bytes;
  const int32_t* slot_count; /* device [R] or NULL: request r's slots are                   */
                           /* slots[slot_indptr[r] .. + slot_count[r]) (a slot table, below);*/
                           /* NULL: slots[slot_indptr[r] .. slot_indptr[r+1])               */
} vtoken_decode;

/* Bytes of workspace: num_reqs * num_q_heads * ceil(max_tokens / (16384 / head_dim)) (at
 * least one split) * (head_dim + 2) * 4, enough for either element size (1-byte caches use
 * half as many splits). head_dim must be 32, 64, 128 or 256 (also for vtoken_paged_decode:
 * VTOKEN_ERR_SHAPE otherwise). Returns -1 for invalid sizes. */
int64_t vtoken_decode_workspace_bytes(int32_t num_reqs, int32_t num_q_heads, int32_t head_dim,
                                      int32_t max_tokens);
vtoken_status vtoken_paged_decode(const vtoken_cache* cache, const vtoken_decode* decode,
                                  int32_t num_reqs, const int32_t* slot_indptr,
                                  const int32_t* slots, hipStream_t stream);

/* For callers that cannot allocate device memory (code under HIP graph capture, serving loops
 * or harnesses that forbid hipMalloc): vtoken_paged_decode with its split partials in a
 * workspace the library holds - a static device array of VTOKEN_DECODE_SCRATCH_BYTES on every
 * GPU the library runs on, kept until the process ends - instead of decode->workspace
 * (decode->workspace and decode->workspace_bytes are ignored). Same arguments, kernels and
 * results as vtoken_paged_decode otherwise. Calls no hipMalloc, hipFree or other allocating
 * routine: the first call on a device looks the array's address up on the device of `stream`
 * (hipGetSymbolAddress, with that device made current for the lookup) and keeps it.
 * Limit: vtoken_decode_workspace_bytes(num_reqs, num_q_heads, head_dim, max_tokens) must not
 * exceed VTOKEN_DECODE_SCRATCH_BYTES; a larger call returns VTOKEN_ERR_CAPACITY and enqueues
 * nothing. Every call on one GPU shares that GPU's array, which keeps the last call's
 * partials (the decode writes every partial it reads, so nothing needs clearing): calls on one
 * GPU must be stream-ordered with respect to each other - calls that may overlap (different
 * streams without an event between them) race on the array and give wrong outputs. */
#define VTOKEN_DECODE_SCRATCH_BYTES (64LL << 20)
vtoken_status vtoken_paged_decode_noalloc(const vtoken_cache* cache,
                                          const vtoken_decode* decode, int32_t num_reqs,
                                          const int32_t* slot_indptr, const int32_t* slots,
                                          hipStream_t stream);

/* The hipError_t behind the calling thread's most recent VTOKEN_ERR_HIP (0 if none yet). */
int32_t vtoken_last_hip_error(void);

/* Static string naming a status code; never NULL. */
const char* vtoken_status_string(int32_t status);

/* Library ABI version: major*10000 + minor*100 + patch. */
int32_t vtoken_version(void);

/* The SHA-256 of the sources the library was built from, as 64 lowercase hex digits: over
 * every file of the package's csrc/ directory and include/vtoken.h, in sorted order of their
 * paths relative to the repository root, each hashed as its path, a NUL byte, its contents
 * and a NUL byte (what the package's build script computes and compiles in). "unknown" for a
 * library built without it. A static string; never NULL. */
const char* vtoken_build_id(void);

#ifdef __cplusplus
}
#endif

#endif /* VTOKEN_H */
