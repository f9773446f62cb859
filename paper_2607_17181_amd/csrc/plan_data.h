// Internal plan representation shared by the host planner and the kernels.
//
// A plan is plain data: per-sequence descriptors plus batch-wide constants.
// It is handed to every kernel by value (as a kernel argument), so planning
// never writes device memory and nothing has to be uploaded before a launch.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "talaria_sp_attn.h"

#if defined(__HIPCC__)
#define TSP_HD __host__ __device__ __forceinline__
#else
#define TSP_HD inline
#endif

namespace tsp {

constexpr uint32_t kPlanMagic = 0x54535041u;  // "TSPA"
constexpr uint32_t kPlanVersion = 3;

// Work decomposition of the prefill kernel.
constexpr int kRowsPerTile = 256;   // query rows (token x head-in-group) per work item
constexpr int kKeysPerTile = 64;    // keys per K/V tile staged in LDS
constexpr int kMaxSplits = 64;      // key-range splits per query tile
constexpr int kXcds = 8;            // XCDs; workgroup i of a launch runs on XCD i % 8
constexpr int kMappedItems = 256;   // plans of at most this many items may be XCD-placed

struct SeqDesc {
    int32_t prefix_len;  // P_b
    int32_t suffix_len;  // S_b
    int32_t tok_off;     // first row of this sequence in q / out / k_new
    int32_t item_off;    // first work item of this sequence
    int32_t part_off;    // first partial-result slot (split sequences only)
};

struct PlanData {
    uint32_t magic;
    uint32_t version;
    int32_t num_q_heads;
    int32_t num_kv_heads;
    int32_t head_dim;
    int32_t page_size;
    int32_t page_shift;      // log2(page_size)
    int32_t num_pages;
    int32_t num_seqs;
    int32_t bt_stride;       // max_pages_per_seq
    int32_t group;           // Hq / Hkv
    int32_t tile_tokens;     // tokens per query tile: kRowsPerTile / group
    int32_t total_tokens;    // T
    int32_t total_kv_tokens; // sum_b (P_b + S_b)
    int32_t num_items;       // prefill work items
    int32_t num_part_items;  // items that write partial results
    int32_t max_suffix_pages;   // most logical pages any suffix touches
    int32_t max_seq_pages;      // most logical pages any sequence holds
    int64_t ws_lse_offset;      // byte offset of partial LSE in the workspace
    int64_t ws_bytes;           // workspace bytes needed
    int32_t wg_mapped;          // 1: prefill workgroup i runs item item_of_wg[i]
    int32_t pad0;
    uint64_t stamps;            // device address of per-workgroup timing records, or 0
    uint8_t item_of_wg[kMappedItems];  // XCD placement (wg_mapped only)
    int32_t kv_off[TALARIA_SP_MAX_SEQS + 1];  // gather output row offsets
    SeqDesc seq[TALARIA_SP_MAX_SEQS + 1];     // entry num_seqs: sentinel
    // Sequences are held in launch order (see the planner); seq_orig[i] is
    // the caller's index of sequence i, i.e. its block-table row.  Token and
    // gather offsets (tok_off, kv_off) are the caller's layout already.
    uint8_t seq_orig[TALARIA_SP_MAX_SEQS];
};

static_assert(sizeof(PlanData) <= sizeof(talaria_sp_plan), "plan storage too small");
static_assert(sizeof(PlanData) <= 3584, "plan must fit a kernel argument");
static_assert(TALARIA_SP_MAX_SEQS <= 256, "seq_orig holds sequence indices in a byte");
static_assert(offsetof(PlanData, item_of_wg) % 4 == 0 && offsetof(PlanData, seq_orig) % 4 == 0 &&
                  kMappedItems % 4 == 0 && TALARIA_SP_MAX_SEQS % 4 == 0,
              "plan byte arrays are read as aligned 32-bit words");

struct WorkItem {
    int32_t seq;
    int32_t kv_head;
    int32_t q_tile;
    int32_t split;
    int32_t num_splits;
    int32_t first_token;  // first new token (suffix index) of the query tile
    int32_t num_tokens;   // tokens in the query tile
    int32_t tile_begin;   // first key tile (of kKeysPerTile keys) of this split
    int32_t tile_end;     // one past the last key tile
    int32_t part_index;   // partial-result slot, or -1 when the tile is not split
};

TSP_HD int32_t ceil_div(int32_t a, int32_t b) { return (a + b - 1) / b; }

TSP_HD int32_t num_q_tiles(const PlanData& p, int32_t b) {
    return ceil_div(p.seq[b].suffix_len, p.tile_tokens);
}

// Splits per query tile of sequence b (uniform inside a sequence).
TSP_HD int32_t num_splits_of(const PlanData& p, int32_t b) {
    int32_t items = p.seq[b + 1].item_off - p.seq[b].item_off;
    int32_t per = num_q_tiles(p, b) * p.num_kv_heads;
    return per > 0 ? items / per : 1;
}

// Sequence that owns work item `id` (binary search over item offsets).
TSP_HD int32_t seq_of_item(const PlanData& p, int32_t id) {
    int32_t lo = 0, hi = p.num_seqs - 1;
    while (lo < hi) {
        int32_t mid = (lo + hi + 1) >> 1;
        if (p.seq[mid].item_off <= id)
            lo = mid;
        else
            hi = mid - 1;
    }
    return lo;
}

// Byte i of a 4-byte-aligned byte array, read as its aligned 32-bit word:
// kernels then load plan bytes with scalar (not per-lane) loads.
TSP_HD uint32_t plan_byte(const uint8_t* a, int32_t i) {
    const uint32_t word = reinterpret_cast<const uint32_t*>(a)[i >> 2];
    return (word >> (8 * (i & 3))) & 0xffu;
}

// Block-table row of (launch-order) sequence b.
TSP_HD int64_t bt_row_index(const PlanData& p, int32_t b) { return plan_byte(p.seq_orig, b); }

// Decode a work item.  Inside a sequence the split index varies fastest,
// then the KV head, then the query tile in reverse order (the query tiles
// with the longest causal key range start first).
TSP_HD WorkItem decode_item(const PlanData& p, int32_t id) {
    WorkItem w;
    int32_t b = seq_of_item(p, id);
    const SeqDesc& s = p.seq[b];
    int32_t nqt = num_q_tiles(p, b);
    int32_t nsp = num_splits_of(p, b);
    int32_t r = id - s.item_off;
    w.seq = b;
    w.split = r % nsp;
    r /= nsp;
    w.kv_head = r % p.num_kv_heads;
    w.q_tile = nqt - 1 - r / p.num_kv_heads;
    w.num_splits = nsp;
    w.first_token = w.q_tile * p.tile_tokens;
    int32_t left = s.suffix_len - w.first_token;
    w.num_tokens = left < p.tile_tokens ? left : p.tile_tokens;
    // Keys visible to the last token of the tile: 0 .. P + first + num - 1.
    int32_t nkeys = s.prefix_len + w.first_token + w.num_tokens;
    int32_t ntiles = ceil_div(nkeys, kKeysPerTile);
    w.tile_begin = (int32_t)(((int64_t)ntiles * w.split) / nsp);
    w.tile_end = (int32_t)(((int64_t)ntiles * (w.split + 1)) / nsp);
    w.part_index = nsp > 1 ? s.part_off + (id - s.item_off) : -1;
    return w;
}

}  // namespace tsp
