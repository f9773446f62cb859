/*
 * talaria_sp_attn -- session-prefill (SP) attention over a paged KV pool on
 * one AMD Instinct MI355X (gfx950).
 *
 * The operation.  SP admission (paper Section 3.4, cold-pool scheduling)
 * batch-prefills continuations of agent sessions whose prefix KV is already
 * resident on the device; only the new tail is computed (Section 4.3, Host KV
 * Registry: restore the agreed prefix into device slots, recompute only the
 * unconfirmed tail).  For one attention layer and a batch of B sequences,
 * sequence b has P_b cached tokens (its committed KV length, Section 4.1)
 * and S_b new tokens.  New token i of sequence b sits at absolute position
 * P_b + i and attends causally to keys 0 .. P_b + i:
 *
 *     o[b,i,h] = sum_j softmax_j( sigma * <q[b,i,h], k[b,j,g]> ) v[b,j,g],
 *     lse[b,i,h] = ln sum_j exp( sigma * <q[b,i,h], k[b,j,g]> ),
 *
 * with g = h / (Hq / Hkv) (grouped-query attention) and sigma the softmax
 * scale (default 1/sqrt(head_dim)).  Keys j < P_b come from the cached
 * prefix; keys P_b .. P_b + S_b - 1 are the new tokens, which
 * talaria_sp_attn_append_kv first writes into their pool slots.
 *
 * Memory.  The caller owns every buffer (pools, block tables, inputs,
 * outputs, workspace); the library never allocates, frees or moves device
 * memory and keeps no pointer across calls, so pool pages keep stable
 * addresses (the stable-HBM-layout contract of Section 4.2).  Pages are
 * allocated by the caller: block_tables[b][p] names the physical page that
 * holds logical tokens p*page_size .. (p+1)*page_size - 1 of sequence b.
 * Device arrays of bf16 rows (q, out, k_new, v_new, the pools, gather
 * outputs) and workspaces must be 16-byte aligned, block tables and lse
 * 4-byte aligned (hipMalloc returns 256-byte aligned memory), and so must
 * the HKVR caches and slab; the attention, append, gather and HKVR calls
 * return TALARIA_SP_EINVAL otherwise, before launching anything.
 *
 * Layouts (all bf16 tensors are raw 16-bit bfloat16, row-major):
 *   q, out      [T][Hq][head_dim]             T = sum_b S_b, sequences in order
 *   k_new,v_new [T][Hkv][head_dim]
 *   lse         [T][Hq] float32 (natural log)
 *   k_pool      [num_pages][Hkv][page_size][head_dim]
 *   v_pool      [num_pages][Hkv][head_dim][page_size]   (token index innermost)
 *   block_tables[num_seqs][max_pages_per_seq] int32 (device memory)
 * One pool pair holds one layer (layer-first device layout, Appendix C).
 * V pages keep tokens innermost so that the PV contraction, which reduces
 * over tokens, reads its operands contiguously.
 *
 * Ordering.  Every call that takes a stream only enqueues work on it and
 * returns; nothing synchronises.  For one batch: plan (host only), then
 * append_kv, then prefill, on one stream (or with the caller's own
 * ordering).  A plan is plain host data: it may be reused for any number of
 * calls and copied freely.
 *
 * Errors.  Every call returns TALARIA_SP_OK (0) or a negative status and
 * launches nothing on error; talaria_sp_last_error() then describes the
 * failure (thread-local, valid until the next failing call on the thread).
 * No C++ exception crosses this interface.
 */
#ifndef TALARIA_SP_ATTN_H
#define TALARIA_SP_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define TALARIA_SP_API __attribute__((visibility("default")))

#define TALARIA_SP_OK 0
#define TALARIA_SP_EINVAL (-1)       /* null pointer, negative length, bad geometry, short table */
#define TALARIA_SP_EUNSUPPORTED (-2) /* head_dim, page_size, group size or batch size not built */
#define TALARIA_SP_ENOSPACE (-3)     /* workspace smaller than the plan needs */
#define TALARIA_SP_EHIP (-4)         /* the HIP runtime rejected a launch */

/* Largest batch one plan describes (the plan travels as a kernel argument). */
#define TALARIA_SP_MAX_SEQS 128
/* Size of the opaque plan storage in 64-bit words. */
#define TALARIA_SP_PLAN_WORDS 448

/* Attention geometry of one layer's pool (the slab shape, page size and
 * dtype of the KV layout descriptor, Appendix C).  Supported: head_dim 64
 * or 128; page_size a power of two in [8, 256]; num_q_heads a multiple of
 * num_kv_heads with num_q_heads / num_kv_heads <= 256. */
typedef struct {
    int32_t num_q_heads;
    int32_t num_kv_heads;
    int32_t head_dim;
    int32_t page_size;
    int32_t num_pages;
} talaria_sp_geom;

/* Caller-owned plan storage, filled by talaria_sp_attn_plan. */
typedef struct {
    uint64_t opaque[TALARIA_SP_PLAN_WORDS];
} talaria_sp_plan;

/*
 * Plan one SP batch (host only; touches no device state).  The batch is the
 * bounded set of continuations that one SP opportunity admits (Section 3.4);
 * each brings its committed prefix length (the device-resident KV of Section
 * 4.1) and its new-token count, and the batch's prefill is the T_pf of that
 * opportunity.
 *
 * geom                 pool geometry (host pointer).
 * num_seqs             sequences in the batch, 0 .. TALARIA_SP_MAX_SEQS.
 * prefix_lens          host int32[num_seqs]: cached tokens P_b >= 0.
 * suffix_lens          host int32[num_seqs]: new tokens S_b >= 0 (0 = no-op).
 * max_pages_per_seq    row stride of block_tables; must be at least
 *                      ceil((P_b + S_b) / page_size) for every b.
 * kv_splits            0 lets the planner split long key ranges across
 *                      compute units; k > 0 forces exactly min(k, tiles)
 *                      splits per query tile (tests use this).
 * workspace_bytes      out: device workspace talaria_sp_attn_prefill needs
 *                      (may be 0).
 * plan                 out: the plan.
 *
 * The planner cuts every (sequence, KV head) into query tiles and splits
 * each tile's visible key range into near-equal pieces, so a ragged batch
 * spreads over all compute units; split results are merged by a
 * log-sum-exp combine inside talaria_sp_attn_prefill.  A batch that takes
 * several rounds of the GPU is cut finer and launched longest items first.
 * Neither choice changes what is computed.
 */
TALARIA_SP_API int talaria_sp_attn_plan(const talaria_sp_geom* geom, int32_t num_seqs,
                         const int32_t* prefix_lens, const int32_t* suffix_lens,
                         int32_t max_pages_per_seq, int32_t kv_splits,
                         size_t* workspace_bytes, talaria_sp_plan* plan);

/*
 * Opt-in host validation of block tables (for debugging and for callers that
 * keep a host copy of their tables; host only, nothing is launched).  The
 * kernels trust the tables: an id outside the pool is an out-of-bounds
 * device access, and two sequences appending into one page corrupt each
 * other.  host_block_tables is the host image of the block_tables the
 * device calls take, int32[num_seqs][max_pages_per_seq].  For every
 * sequence b and logical page p < ceil((P_b + S_b) / page_size) (the
 * entries the calls read) it returns TALARIA_SP_EINVAL, naming the first
 * offending entry, when:
 *   - the id is outside [0, num_pages);
 *   - the sequence names one physical page at two logical positions;
 *   - a page that append writes (one holding some position
 *     P_b .. P_b + S_b - 1) is named by any other entry of the batch.
 * Pages that only hold cached prefix positions may be shared between
 * sequences (read-only).  Entries past a sequence's last page are ignored.
 */
TALARIA_SP_API int talaria_sp_attn_check_tables(const talaria_sp_plan* plan,
                                                const int32_t* host_block_tables);

/*
 * Append: write the K and V rows of every new token into its pool slot
 * (Section 4.3: the returning request's new tail goes into newly allocated
 * device slots).  Token i of sequence b (row off_b + i of k_new / v_new)
 * goes to logical position P_b + i, i.e. page
 * block_tables[b][(P_b+i) / page_size], slot (P_b+i) mod page_size.  The
 * copy is bit-exact; no other pool slot is written.  The caller guarantees
 * that the pages named for positions P_b .. P_b+S_b-1 are distinct across
 * the batch and below num_pages.
 *
 * k_new, v_new   device bf16 [T][Hkv][head_dim]
 * k_pool, v_pool device bf16 pools (layouts above), written in place
 * block_tables   device int32 [num_seqs][max_pages_per_seq]
 * stream         hipStream_t (NULL = default stream)
 */
TALARIA_SP_API int talaria_sp_attn_append_kv(const talaria_sp_plan* plan, const void* k_new, const void* v_new,
                              void* k_pool, void* v_pool, const int32_t* block_tables,
                              void* stream);

/*
 * Prefill: causal attention of every new token over its sequence's cached
 * prefix plus the new tokens (the batched prefill T_pf of an SP step,
 * Section 3.4), reading K/V through the block tables.  append_kv for the
 * same plan must have been enqueued first.  Pool slots past P_b + S_b in a
 * sequence's last page, and block-table entries past its last page, are
 * never read, so stale contents there (even NaN) do not matter.
 *
 * q              device bf16 [T][Hq][head_dim] (positional encoding applied)
 * k_pool, v_pool device bf16 pools holding positions 0 .. P_b+S_b-1
 * block_tables   device int32 [num_seqs][max_pages_per_seq]
 * sm_scale       softmax scale sigma; <= 0 selects 1/sqrt(head_dim)
 * out            device bf16 [T][Hq][head_dim] (round to nearest even)
 * lse            device float32 [T][Hq] or NULL
 * workspace      device buffer of at least workspace_bytes from the plan
 *                (NULL allowed when that is 0); contents are scratch
 * stream         hipStream_t (NULL = default stream)
 *
 * For a fixed plan the result is bitwise deterministic.
 */
TALARIA_SP_API int talaria_sp_attn_prefill(const talaria_sp_plan* plan, const void* q, const void* k_pool,
                            const void* v_pool, const int32_t* block_tables, float sm_scale,
                            void* out, float* lse, void* workspace, size_t workspace_bytes,
                            void* stream);

/*
 * Allocation-free prefill, for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): talaria_sp_attn_prefill without the workspace argument.  Same
 * plan, inputs, outputs, kernels and results (bit-identical to
 * talaria_sp_attn_prefill on the same plan).  Split partials go to a
 * scratch array inside the library instead: TALARIA_SP_NOALLOC_SCRATCH_BYTES
 * (64 MiB) of device memory on every GPU the library runs on, held until the
 * process ends.  A plan whose workspace_bytes exceeds that returns
 * TALARIA_SP_ENOSPACE before anything is launched.  The call allocates
 * nothing; its first call on a device looks up that device's scratch
 * address once (no allocation, no stream work).
 *
 * Every call on one GPU shares that GPU's scratch, and the scratch keeps the
 * last call's contents: calls that overlap on one GPU (other streams, other
 * threads) race and must be ordered by the caller.
 */
#define TALARIA_SP_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
TALARIA_SP_API int talaria_sp_attn_prefill_noalloc(const talaria_sp_plan* plan, const void* q,
                                                   const void* k_pool, const void* v_pool,
                                                   const int32_t* block_tables, float sm_scale,
                                                   void* out, float* lse, void* stream);
/* TALARIA_SP_NOALLOC_SCRATCH_BYTES as the built library has it. */
TALARIA_SP_API size_t talaria_sp_attn_noalloc_scratch_bytes(void);

/*
 * Decode: the S_b = 1 case of prefill -- each sequence's one new token (at
 * position P_b, its K/V appended first) attends to keys 0 .. P_b -- with a
 * kernel built for it: the D phase that resumes after an SP batch (Section
 * 3.4) reads every cached K/V byte once for only `group` query rows, so it
 * is bound by HBM, not by the matrix cores.  Same plan (made with suffix
 * lengths of 0 or 1), arguments, layouts and workspace as prefill.
 * EINVAL if some suffix length exceeds 1; EUNSUPPORTED if more than 32
 * query heads share a KV head.
 */
TALARIA_SP_API int talaria_sp_attn_decode(const talaria_sp_plan* plan, const void* q,
                                          const void* k_pool, const void* v_pool,
                                          const int32_t* block_tables, float sm_scale, void* out,
                                          float* lse, void* workspace, size_t workspace_bytes,
                                          void* stream);

/*
 * Gather: copy positions 0 .. P_b+S_b-1 of every sequence out of the pool
 * into contiguous token-major rows -- the block-table page walk that the
 * prefill kernel performs internally, as a standalone copy (the layer-first
 * page view of Appendix C turned into a flat per-sequence view).
 *
 * k_out, v_out   device bf16 [sum_b (P_b+S_b)][Hkv][head_dim], sequences in order
 */
TALARIA_SP_API int talaria_sp_attn_gather_kv(const talaria_sp_plan* plan, const void* k_pool,
                              const void* v_pool, const int32_t* block_tables, void* k_out,
                              void* v_out, void* stream);

/* Introspection of a plan's work list (host only).  Writes up to max_items
 * records of 8 int32 each: {sequence, kv_head, first_token, num_tokens,
 * key_begin, key_end, split, num_splits}, in launch order; sequence is the
 * caller's index and keys are absolute positions.
 * Returns the number of work items (>= 0) or a negative status. */
TALARIA_SP_API int talaria_sp_attn_plan_items(const talaria_sp_plan* plan, int32_t* items, int32_t max_items);

/* ---- XCD placement ------------------------------------------------------
 *
 * Workgroup i of a launch runs on XCD i % 8, and the XCDs of one MI355X
 * differ in speed by several percent, steadily from launch to launch.  With
 * one round of equal-cost items the slowest XCD therefore sets the end of
 * the call.  Once an XCD order is set, every prefill plan made afterwards
 * that is one round of at most 256 items (and not a decode batch) places
 * its longest items on the fastest XCDs.  Placement only changes which
 * compute unit runs an item: results are bit-identical with or without it.
 *
 * talaria_sp_attn_calibrate_xcd measures the order on the caller's own
 * batch: it runs one prefill of `plan` (outputs land in out / workspace as
 * for talaria_sp_attn_prefill with the default scale and no LSE) with each
 * workgroup recording its XCD and main-loop time into `stamps` (device
 * memory, 32 bytes per work item), synchronises `stream`, ranks the XCDs by
 * mean time per key tile and sets the order (also written to `order`,
 * int32[8], unless NULL).  It synchronises and copies to the host, so it
 * belongs in set-up, not in the serving loop.  The plan needs at least 8
 * work items and a timed item on every XCD (a full-GPU batch, e.g. one
 * 25K-token continuation, is a good calibration batch).  Returns EINVAL,
 * ENOSPACE (stamps too small) or EHIP as the other calls do.
 *
 * talaria_sp_set_xcd_order sets the order directly (order[g] = the XCD that
 * takes the g-th longest block; a permutation of 0..7) or, with NULL,
 * clears it.  talaria_sp_get_xcd_order copies the order into order[8] and
 * returns 1, or returns 0 when none is set.  The order is process-wide;
 * plans already made keep their placement.  Host only.
 */
TALARIA_SP_API int talaria_sp_attn_calibrate_xcd(const talaria_sp_plan* plan, const void* q,
                                                 const void* k_pool, const void* v_pool,
                                                 const int32_t* block_tables, void* out,
                                                 void* workspace, size_t workspace_bytes,
                                                 void* stamps, size_t stamps_bytes,
                                                 int32_t* order, void* stream);
TALARIA_SP_API int talaria_sp_set_xcd_order(const int32_t* order);
TALARIA_SP_API int talaria_sp_get_xcd_order(int32_t* order);

/* ---- HKVR page transfer (host KV registry restore / checkpoint) ----------
 *
 * A returning session's prefix may live in pinned host memory instead of the
 * device cache.  Restoring it places the agreed prefix pages into newly
 * allocated device pages before the unconfirmed tail is recomputed (Section
 * 4.3); checkpointing copies device pages out when a turn ends.  The two
 * layouts are the layer-first device cache and the page-first host slab of
 * Appendix C:
 *
 *   k_cache  [num_layers][num_pages][Hkv][page_size][head_dim]   (device)
 *   v_cache  [num_layers][num_pages][Hkv][head_dim][page_size]   (device)
 *   slab     [num_slab_pages][num_layers][2][Hkv*page_size*head_dim] (host)
 *
 * Layer l of the cache is the single-layer pool pair the attention calls
 * above take (k_cache + l * num_pages * Hkv * page_size * head_dim, and
 * likewise for V).  Slab block [p][l][0] is device page page_ids[p] of layer
 * l's K pool and [p][l][1] the same page of its V pool, each in the device
 * page's own element order, so a transfer moves whole page blocks and
 * reorders no element.  Whole pages only: restored prefixes are page
 * aligned.
 *
 * The slab must be pinned host memory that the device can address directly
 * (hipHostMalloc, or a torch tensor allocated with pin_memory=True); the
 * copy kernels read or write it through that address over the host link.
 * page_ids is a device int32 array of num_slab_pages entries (typically the
 * first entries of the sequence's block-table row); an entry outside
 * [0, num_pages) moves nothing.  Entries should be distinct: two slab pages
 * naming one device page race on restore.  Stream-ordered like the calls
 * above; nothing synchronises.
 */
typedef struct {
    int32_t num_layers;    /* 1 .. 65535 */
    int32_t num_kv_heads;
    int32_t head_dim;      /* 64 or 128 */
    int32_t page_size;     /* power of two in [8, 256] */
    int32_t num_pages;     /* device pages per layer */
} talaria_kv_cache;

/* Host slab -> device cache (H2D restore of num_slab_pages pages, all layers). */
TALARIA_SP_API int talaria_hkvr_restore(const talaria_kv_cache* cache, int32_t num_slab_pages,
                                        const void* slab, const int32_t* page_ids,
                                        void* k_cache, void* v_cache, void* stream);

/* Device cache -> host slab (D2H checkpoint of num_slab_pages pages, all layers). */
TALARIA_SP_API int talaria_hkvr_checkpoint(const talaria_kv_cache* cache, int32_t num_slab_pages,
                                           const void* k_cache, const void* v_cache,
                                           const int32_t* page_ids, void* slab, void* stream);

/* ---- D2D-staged weight switching (staging guard and gather) -------------
 *
 * The next model's weights are pre-staged in fixed-size chunks in unused
 * high-address HBM of the KV region while the current model serves; at the
 * switch, staged clean chunks are copied device to device and the rest is
 * reloaded from host (Section 4.4).  A staged chunk becomes dirty when a KV
 * allocation takes pages overlapping its staging range.
 *
 * Regions (byte addresses, 16-byte aligned):
 *   staging       device, staging_bytes: the region the staged copies sit in;
 *                 also the region whose pages the KV allocator hands out
 *                 (page p = bytes [p*page_bytes, (p+1)*page_bytes)).
 *   weights       device, weight_bytes: the target model's weight region.
 *   host_weights  pinned host memory with the same layout as weights.
 * Chunk i (talaria_stage_chunk, device array) moves `bytes` bytes to
 * weights + weight_offset, from staging + stage_offset when bit i of `staged`
 * is set and bit i of `dirty` is clear, else from host_weights +
 * weight_offset.  Sizes and offsets are multiples of 16.  A chunk whose
 * weight range leaves the weight region is skipped; a staged range outside
 * the staging region falls back to the host copy.  Bitmaps are device
 * uint32 arrays, bit i = word i/32, bit i%32.
 */
typedef struct {
    int64_t stage_offset;   /* byte offset of the staged copy in `staging` */
    int64_t weight_offset;  /* byte offset in `weights` (and `host_weights`) */
    int64_t bytes;          /* chunk size, a positive multiple of 16 */
} talaria_stage_chunk;

/* dirty bit i = 1 iff some page p with bit p of used_pages set overlaps
 * chunk i's staging range (pages >= num_pages are not tracked).  Writes all
 * ceil(num_chunks/32) words of dirty. */
TALARIA_SP_API int talaria_stage_mark_dirty(const talaria_stage_chunk* chunks, int32_t num_chunks,
                                            const uint32_t* used_pages, int64_t num_pages,
                                            int64_t page_bytes, uint32_t* dirty, void* stream);

/* Assemble the weight region from clean staged chunks (D2D) and host copies
 * (H2D) in one kernel. */
TALARIA_SP_API int talaria_stage_gather(const talaria_stage_chunk* chunks, int32_t num_chunks,
                                        const uint32_t* staged, const uint32_t* dirty,
                                        const void* staging, int64_t staging_bytes,
                                        const void* host_weights, void* weights,
                                        int64_t weight_bytes, void* stream);

/* ---- SP batch selection (host) -------------------------------------------
 *
 * Each SP opportunity takes a bounded set of the waiting continuations,
 * sized so that its predicted cost (attention time, page restore time,
 * device pages) stays inside what the slot has left once decode is served;
 * the others wait (Section 3.4).  talaria_sp_select scans candidates in
 * queue order and admits each one that still fits all bounds (first fit),
 * skipping the rest.
 *
 * Predicted cost of a candidate (host-resident prefixes are restored page
 * aligned, their partial last page recomputed with the suffix, Appendix B:
 * P' = floor(P/ps)*ps, S' = S + P - P'; device-resident ones keep P, S):
 *   seconds = 4*d*Hq*layers*(S*P + S*(S+1)/2) / attn_flops_per_s
 *           + S * per_token_s
 *           + (host-resident) (P/ps) * 2*Hkv*ps*d*2*layers bytes / restore_bytes_per_s
 *   pages   = ceil((P+S)/ps) - (device-resident ? ceil(P/ps) : 0)
 * plus batch_overhead_s once per non-empty batch.  Candidates with S <= 0
 * or P < 0 are never admitted.
 *
 * selected          out: indices of admitted candidates, in queue order
 *                   (room for max_batch entries)
 * plan_prefix_lens, plan_suffix_lens
 *                   out (may be NULL): the admitted candidates' P and S as
 *                   talaria_sp_attn_plan takes them (after the alignment above)
 * predicted_seconds, predicted_pages
 *                   out (may be NULL): the batch's predicted totals
 * Returns the number admitted (>= 0) or a negative status.  Host only.
 */
typedef struct {
    int32_t prefix_len;     /* P: committed (device) or checkpointed (host) tokens */
    int32_t suffix_len;     /* S: new tokens to prefill */
    int32_t host_resident;  /* nonzero: the prefix must be restored from host */
} talaria_sp_candidate;

typedef struct {
    int32_t num_layers, num_q_heads, num_kv_heads, head_dim, page_size;
    double attn_flops_per_s;    /* sustained SP attention FLOP/s */
    double per_token_s;         /* other prefill work per new token */
    double restore_bytes_per_s; /* host -> device restore rate */
    double batch_overhead_s;    /* fixed cost of one SP batch */
} talaria_sp_cost_model;

typedef struct {
    double time_budget_s;   /* prefill + restore time left in the slot */
    int64_t free_pages;     /* device pages the batch may allocate */
    int32_t max_batch;      /* 0 .. TALARIA_SP_MAX_SEQS */
} talaria_sp_budget;

TALARIA_SP_API int talaria_sp_select(const talaria_sp_candidate* cands, int32_t num_cands,
                                     const talaria_sp_cost_model* model,
                                     const talaria_sp_budget* budget, int32_t* selected,
                                     int32_t* plan_prefix_lens, int32_t* plan_suffix_lens,
                                     double* predicted_seconds, int64_t* predicted_pages);

/* Message for the last failing call on this thread ("" if none). */
TALARIA_SP_API const char* talaria_sp_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* TALARIA_SP_ATTN_H */
