// Host planner for SP attention: argument validation, ragged offsets, and
// the split of every query tile's key range into work items.
//
// The planner follows the shape of an SP step (Section 3.4): a bounded
// batch of admitted continuations, each with its own committed prefix
// length and new-token count.  It produces one flat work list that the
// prefill kernel walks by block index:
//
//   sequence b  ->  query tiles of kRowsPerTile rows (tile_tokens tokens x
//                   group query heads that share one KV head)
//               ->  per KV head
//               ->  num_splits near-equal ranges of the tile's visible keys
//
// The number of splits per sequence is chosen so that the whole batch fills
// the GPU's 256 compute units with items of similar cost: long prefixes
// are cut into more pieces, short ones are not cut at all.
#include <hip/hip_runtime.h>

#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <vector>

#include "common.h"

namespace tsp {

namespace {
thread_local char g_error[512] = "";

// Work items that run at once: one per compute unit of an MI355X.
constexpr int kConcurrentItems = 256;
// Never cut a key range below this many key tiles.
constexpr int kMinTilesPerSplit = 8;
// Decode batches: two decode workgroups fit on a CU (LDS bound), so a decode
// batch is cut for twice as many concurrent items; and the shortest key
// range worth a split.
constexpr int kDecodeItemsPerCU = 2;
constexpr int kMinTilesPerDecodeSplit = 4;
// A batch that takes several rounds is cut into items of at most this
// fraction of one compute unit's share of its key tiles, so that, started
// longest first, no item can form a long tail.
constexpr double kMultiRoundShare = 0.25;
}  // namespace

int fail(int code, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_error, sizeof g_error, fmt, ap);
    va_end(ap);
    return code;
}

const PlanData* checked_plan(const talaria_sp_plan* plan, int* status) {
    if (!plan) {
        *status = fail(TALARIA_SP_EINVAL, "plan is NULL");
        return nullptr;
    }
    const PlanData* p = reinterpret_cast<const PlanData*>(plan);
    if (p->magic != kPlanMagic || p->version != kPlanVersion) {
        *status = fail(TALARIA_SP_EINVAL, "plan was not produced by talaria_sp_attn_plan");
        return nullptr;
    }
    *status = TALARIA_SP_OK;
    return p;
}

int launch_status(const char* what) {
    hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return fail(TALARIA_SP_EHIP, "%s launch failed: %s", what, hipGetErrorString(e));
    return TALARIA_SP_OK;
}

}  // namespace tsp

using namespace tsp;

extern "C" const char* talaria_sp_last_error(void) { return g_error; }

namespace {

// XCD order for placement, fastest XCD first (process-wide; see
// talaria_sp_set_xcd_order).
std::mutex g_xcd_mutex;
bool g_xcd_set = false;
int32_t g_xcd_order[tsp::kXcds];

bool xcd_order_snapshot(int32_t* out) {
    std::lock_guard<std::mutex> lock(g_xcd_mutex);
    if (g_xcd_set)
        memcpy(out, g_xcd_order, sizeof g_xcd_order);
    return g_xcd_set;
}

}  // namespace

extern "C" int talaria_sp_set_xcd_order(const int32_t* order) {
    if (!order) {
        std::lock_guard<std::mutex> lock(g_xcd_mutex);
        g_xcd_set = false;
        return TALARIA_SP_OK;
    }
    bool seen[kXcds] = {};
    for (int g = 0; g < kXcds; ++g) {
        if (order[g] < 0 || order[g] >= kXcds || seen[order[g]])
            return fail(TALARIA_SP_EINVAL, "xcd order must be a permutation of 0..%d", kXcds - 1);
        seen[order[g]] = true;
    }
    std::lock_guard<std::mutex> lock(g_xcd_mutex);
    memcpy(g_xcd_order, order, sizeof g_xcd_order);
    g_xcd_set = true;
    return TALARIA_SP_OK;
}

extern "C" int talaria_sp_get_xcd_order(int32_t* order) {
    if (!order)
        return fail(TALARIA_SP_EINVAL, "order must not be NULL");
    int32_t o[kXcds];
    if (!xcd_order_snapshot(o))
        return 0;
    memcpy(order, o, sizeof o);
    return 1;
}

extern "C" int talaria_sp_attn_plan(const talaria_sp_geom* geom, int32_t num_seqs,
                                    const int32_t* prefix_lens, const int32_t* suffix_lens,
                                    int32_t max_pages_per_seq, int32_t kv_splits,
                                    size_t* workspace_bytes, talaria_sp_plan* plan) {
    if (!geom || !plan || !workspace_bytes)
        return fail(TALARIA_SP_EINVAL, "geom, plan and workspace_bytes must not be NULL");
    const int32_t hq = geom->num_q_heads, hkv = geom->num_kv_heads, d = geom->head_dim;
    const int32_t ps = geom->page_size;
    if (hq <= 0 || hkv <= 0 || hq % hkv != 0)
        return fail(TALARIA_SP_EINVAL, "num_q_heads (%d) must be a positive multiple of "
                    "num_kv_heads (%d)", hq, hkv);
    if (geom->num_pages <= 0)
        return fail(TALARIA_SP_EINVAL, "num_pages must be positive (got %d)", geom->num_pages);
    if (d != 64 && d != 128)
        return fail(TALARIA_SP_EUNSUPPORTED, "head_dim %d not supported (64 or 128)", d);
    if (ps < 8 || ps > 256 || (ps & (ps - 1)) != 0)
        return fail(TALARIA_SP_EUNSUPPORTED, "page_size %d not supported (power of two in "
                    "[8, 256])", ps);
    if ((int64_t)hkv * ps * d * 2 > INT32_MAX)
        return fail(TALARIA_SP_EUNSUPPORTED, "one page of all %d KV heads exceeds 2 GiB", hkv);
    if (hq / hkv > kRowsPerTile)
        return fail(TALARIA_SP_EUNSUPPORTED, "query group %d exceeds %d", hq / hkv, kRowsPerTile);
    if (num_seqs < 0)
        return fail(TALARIA_SP_EINVAL, "num_seqs must be >= 0 (got %d)", num_seqs);
    if (num_seqs > TALARIA_SP_MAX_SEQS)
        return fail(TALARIA_SP_EUNSUPPORTED, "num_seqs %d exceeds %d; split the batch",
                    num_seqs, TALARIA_SP_MAX_SEQS);
    if (num_seqs > 0 && (!prefix_lens || !suffix_lens))
        return fail(TALARIA_SP_EINVAL, "prefix_lens and suffix_lens must not be NULL");
    if (kv_splits < 0)
        return fail(TALARIA_SP_EINVAL, "kv_splits must be >= 0 (got %d)", kv_splits);
    if (max_pages_per_seq < 0)
        return fail(TALARIA_SP_EINVAL, "max_pages_per_seq must be >= 0");

    PlanData p;
    memset(&p, 0, sizeof p);
    p.magic = kPlanMagic;
    p.version = kPlanVersion;
    p.num_q_heads = hq;
    p.num_kv_heads = hkv;
    p.head_dim = d;
    p.page_size = ps;
    p.page_shift = __builtin_ctz((unsigned)ps);
    p.num_pages = geom->num_pages;
    p.num_seqs = num_seqs;
    p.bt_stride = max_pages_per_seq;
    p.group = hq / hkv;
    p.tile_tokens = kRowsPerTile / p.group;

    // Lengths, offsets and the cost of one unsplit item per sequence.
    int64_t tok = 0, kvtok = 0;
    int32_t tiles[TALARIA_SP_MAX_SEQS];
    int32_t qtiles[TALARIA_SP_MAX_SEQS];
    int32_t tok_off[TALARIA_SP_MAX_SEQS], kv_off[TALARIA_SP_MAX_SEQS];
    double total_cost = 0.0;
    int64_t base_items = 0;
    for (int32_t b = 0; b < num_seqs; ++b) {
        const int64_t P = prefix_lens[b], S = suffix_lens[b];
        if (P < 0 || S < 0)
            return fail(TALARIA_SP_EINVAL, "sequence %d: negative length (P=%lld, S=%lld)", b,
                        (long long)P, (long long)S);
        if (P + S > INT32_MAX / 2)
            return fail(TALARIA_SP_EINVAL, "sequence %d: P+S too large", b);
        const int64_t pages = (P + S + ps - 1) / ps;
        if (pages > max_pages_per_seq)
            return fail(TALARIA_SP_EINVAL, "sequence %d needs %lld pages but the block-table "
                        "stride is %d", b, (long long)pages, max_pages_per_seq);
        tok_off[b] = (int32_t)tok;
        kv_off[b] = (int32_t)kvtok;
        tok += S;
        kvtok += P + S;
        if (tok > INT32_MAX / 2 || kvtok > INT32_MAX / 2)
            return fail(TALARIA_SP_EINVAL, "batch too large");
        qtiles[b] = (int32_t)((S + p.tile_tokens - 1) / p.tile_tokens);
        tiles[b] = S > 0 ? (int32_t)((P + S + kKeysPerTile - 1) / kKeysPerTile) : 0;
        base_items += (int64_t)qtiles[b] * hkv;
        total_cost += (double)qtiles[b] * hkv * tiles[b];
        if (S > 0) {
            const int32_t first_page = (int32_t)(P / ps), last_page = (int32_t)((P + S - 1) / ps);
            p.max_suffix_pages = std::max(p.max_suffix_pages, last_page - first_page + 1);
        }
        p.max_seq_pages = std::max(p.max_seq_pages, (int32_t)pages);
    }
    p.total_tokens = (int32_t)tok;
    p.total_kv_tokens = (int32_t)kvtok;
    p.kv_off[num_seqs] = (int32_t)kvtok;

    // Target key tiles per item: the per-CU share of the batch when the
    // batch alone cannot fill the GPU (one round of equal items), a quarter
    // of it otherwise (kMultiRoundShare).
    //
    // A decode batch (every suffix at most one token) streams K/V for very
    // few query rows: its items are HBM-bound and cheap in compute, so it is
    // cut kDecodeItemsPerCU times finer to keep every resident slot busy.
    bool decode_batch = true;
    for (int32_t b = 0; b < num_seqs; ++b)
        decode_batch = decode_batch && suffix_lens[b] <= 1;
    const int concurrent = decode_batch ? kDecodeItemsPerCU * kConcurrentItems : kConcurrentItems;
    double share = total_cost / concurrent;
    const bool multi_round = base_items >= concurrent;
    if (multi_round)
        share *= kMultiRoundShare;
    double target = std::max<double>(decode_batch ? kMinTilesPerDecodeSplit : kMinTilesPerSplit,
                                     share);
    auto splits_of = [&](int32_t b, double tgt) {
        if (tiles[b] <= 0)
            return 1;
        const int32_t n = kv_splits > 0 ? kv_splits : (int32_t)ceil(tiles[b] / tgt * 0.999);
        return std::max(1, std::min({n, tiles[b], kMaxSplits}));
    };
    // One round of items: every sequence rounds its split count up, which can
    // push the total past the resident slots and leave a second round of
    // items running alone at the end.  Raise the target (the fewest splits
    // that fit) until the items fit; at `target` >= the longest key range
    // every sequence has one split per query tile, i.e. base_items < slots.
    if (kv_splits == 0 && base_items < concurrent) {
        auto count = [&](double tgt) {
            int64_t n = 0;
            for (int32_t b = 0; b < num_seqs; ++b)
                n += (int64_t)qtiles[b] * hkv * splits_of(b, tgt);
            return n;
        };
        if (count(target) > concurrent) {
            double lo = target, hi = 2.0 * target;
            while (count(hi) > concurrent)
                hi *= 2.0;
            for (int i = 0; i < 40 && hi - lo > 1e-3; ++i) {
                const double mid = 0.5 * (lo + hi);
                (count(mid) > concurrent ? lo : hi) = mid;
            }
            target = hi;
        }
    }

    // Launch order.  Workgroups start in item order as compute units free
    // up, so a batch that takes several rounds runs its longest items first
    // (sequences ranked by their longest item, which bounds the tail to
    // about one short item); inside a sequence the longest query tiles
    // already come first.  One-round and decode plans keep the caller's
    // order.  The order changes which compute unit runs an item and when,
    // never what it computes.
    int32_t launch[TALARIA_SP_MAX_SEQS];
    for (int32_t b = 0; b < num_seqs; ++b)
        launch[b] = b;
    if (multi_round && !decode_batch) {
        int32_t longest[TALARIA_SP_MAX_SEQS];
        for (int32_t b = 0; b < num_seqs; ++b)
            longest[b] = qtiles[b] > 0 ? ceil_div(tiles[b], splits_of(b, target)) : -1;
        std::stable_sort(launch, launch + num_seqs,
                         [&](int32_t a, int32_t c) { return longest[a] > longest[c]; });
    }

    int64_t items = 0, part_items = 0;
    for (int32_t i = 0; i < num_seqs; ++i) {
        const int32_t b = launch[i];
        const int32_t nsp = splits_of(b, target);
        p.seq[i].prefix_len = prefix_lens[b];
        p.seq[i].suffix_len = suffix_lens[b];
        p.seq[i].tok_off = tok_off[b];
        p.kv_off[i] = kv_off[b];
        p.seq_orig[i] = (uint8_t)b;
        p.seq[i].item_off = (int32_t)items;
        p.seq[i].part_off = (int32_t)part_items;
        const int64_t n = (int64_t)qtiles[b] * hkv * nsp;
        items += n;
        if (nsp > 1)
            part_items += n;
        if (items > INT32_MAX / 2)
            return fail(TALARIA_SP_EINVAL, "too many work items");
    }
    p.seq[num_seqs].item_off = (int32_t)items;
    p.seq[num_seqs].part_off = (int32_t)part_items;
    p.seq[num_seqs].tok_off = (int32_t)tok;
    p.num_items = (int32_t)items;
    p.num_part_items = (int32_t)part_items;

    // XCD placement.  Workgroup i of a launch runs on XCD i % kXcds, and
    // XCDs of one part differ in speed by several percent, steadily.  Once an
    // XCD order is set (fastest first, as talaria_sp_attn_calibrate_xcd
    // measures it), a prefill plan that is one round of at most kMappedItems
    // items is placed so that each XCD reads a narrow band of keys and the
    // longest items run on the fastest XCDs:
    //  - items are sorted by the keys they read (sequence, KV head, middle
    //    of the key-tile range) and cut into kXcds contiguous groups, one per
    //    XCD, so each XCD's L2 streams one band of K/V instead of all of it;
    //  - the groups are ranked by their longest item and dealt to the XCDs
    //    fastest first (among XCDs with the same number of workgroups).
    // Placement changes which compute unit runs an item, never what it
    // computes.
    int32_t order[kXcds];
    if (!decode_batch && items > 0 && items <= kMappedItems && xcd_order_snapshot(order)) {
        const int32_t n = (int32_t)items;
        int32_t by_key[kMappedItems], cost[kMappedItems];
        int64_t key[kMappedItems];
        uint8_t uses[kMappedItems] = {};
        for (int32_t i = 0; i < n; ++i) {
            const WorkItem w = decode_item(p, i);
            cost[i] = w.tile_end - w.tile_begin;
            key[i] = (((int64_t)w.seq * p.num_kv_heads + w.kv_head) << 32) +
                     (int64_t)w.tile_begin + w.tile_end;
            by_key[i] = i;
        }
        std::sort(by_key, by_key + n, [&](int32_t a, int32_t b) {
            return key[a] != key[b] ? key[a] < key[b] : a < b;
        });
        // Workgroups per XCD: XCD x runs workgroups x, x + kXcds, ...
        int32_t slots[kXcds];
        for (int x = 0; x < kXcds; ++x)
            slots[x] = x < n ? (n - x + kXcds - 1) / kXcds : 0;
        // Group g (in key order) gets the size of the XCD at speed rank g
        // after sorting ranks by size (larger first), which keeps sizes
        // matched; then groups of one size are ranked by their longest item.
        int32_t by_speed[kXcds];
        for (int g = 0; g < kXcds; ++g)
            by_speed[g] = order[g];
        std::stable_sort(by_speed, by_speed + kXcds,
                         [&](int32_t a, int32_t b) { return slots[a] > slots[b]; });
        int32_t gbeg[kXcds + 1], gmax[kXcds], gidx[kXcds];
        gbeg[0] = 0;
        for (int g = 0; g < kXcds; ++g) {
            gbeg[g + 1] = gbeg[g] + slots[by_speed[g]];
            gmax[g] = 0;
            for (int32_t k = gbeg[g]; k < gbeg[g + 1]; ++k)
                gmax[g] = std::max(gmax[g], cost[by_key[k]]);
            gidx[g] = g;
        }
        std::stable_sort(gidx, gidx + kXcds, [&](int32_t a, int32_t b) {
            const int32_t sa = gbeg[a + 1] - gbeg[a], sb = gbeg[b + 1] - gbeg[b];
            return sa != sb ? sa > sb : gmax[a] > gmax[b];
        });
        for (int g = 0; g < kXcds; ++g) {
            const int32_t x = by_speed[g], grp = gidx[g];
            int32_t k = gbeg[grp];
            for (int32_t wg = x; wg < n; wg += kXcds) {
                p.item_of_wg[wg] = (uint8_t)by_key[k];
                ++uses[by_key[k++]];
            }
            if (k != gbeg[grp + 1])
                return fail(TALARIA_SP_EINVAL, "internal error: XCD group size mismatch");
        }
        for (int32_t i = 0; i < n; ++i)
            if (uses[i] != 1)
                return fail(TALARIA_SP_EINVAL, "internal error: XCD placement is not one-to-one");
        p.wg_mapped = 1;
    }

    // Split partials: normalised outputs in f16 (each is a convex combination
    // of bf16 V rows, so f16 keeps 3 more mantissa bits than the bf16 result)
    // and base-2 LSE in fp32.
    const int64_t part_o = part_items * kRowsPerTile * (int64_t)d * 2;
    const int64_t part_lse = part_items * kRowsPerTile * 4;
    p.ws_lse_offset = (part_o + 255) & ~(int64_t)255;
    p.ws_bytes = part_items ? p.ws_lse_offset + part_lse : 0;

    memset(plan, 0, sizeof *plan);
    memcpy(plan, &p, sizeof p);
    *workspace_bytes = (size_t)p.ws_bytes;
    return TALARIA_SP_OK;
}

extern "C" int talaria_sp_attn_check_tables(const talaria_sp_plan* plan,
                                            const int32_t* host_block_tables) {
    int status;
    const PlanData* p = checked_plan(plan, &status);
    if (!p)
        return status;
    if (p->num_seqs > 0 && !host_block_tables)
        return fail(TALARIA_SP_EINVAL, "check_tables: host_block_tables is NULL");
    // last[page]: the last sequence that named the page (-1: none yet).
    std::vector<int32_t> last((size_t)p->num_pages, -1);
    std::vector<uint8_t> written((size_t)p->num_pages, 0);
    // Sequences are visited in the caller's order (row b of the tables).
    std::vector<int32_t> at((size_t)p->num_seqs);
    for (int32_t i = 0; i < p->num_seqs; ++i)
        at[p->seq_orig[i]] = i;
    // Pass 1: range, duplicates inside one sequence, and the written pages.
    for (int32_t b = 0; b < p->num_seqs; ++b) {
        const int64_t P = p->seq[at[b]].prefix_len, S = p->seq[at[b]].suffix_len;
        const int64_t pages = (P + S + p->page_size - 1) >> p->page_shift;
        const int32_t* row = host_block_tables + (int64_t)b * p->bt_stride;
        for (int64_t lp = 0; lp < pages; ++lp) {
            const int32_t id = row[lp];
            if (id < 0 || id >= p->num_pages)
                return fail(TALARIA_SP_EINVAL, "check_tables: sequence %d, logical page %lld: "
                            "id %d outside [0, %d)", b, (long long)lp, id, p->num_pages);
            if (last[id] == b)
                return fail(TALARIA_SP_EINVAL, "check_tables: sequence %d names page %d at two "
                            "logical positions (second at %lld)", b, id, (long long)lp);
            last[id] = b;
            if (S > 0 && lp >= (P >> p->page_shift) && lp <= ((P + S - 1) >> p->page_shift))
                written[id] = 1;
        }
    }
    // Pass 2: a written page must be named exactly once in the whole batch.
    std::vector<int32_t> count((size_t)p->num_pages, 0);
    for (int32_t b = 0; b < p->num_seqs; ++b) {
        const int64_t P = p->seq[at[b]].prefix_len, S = p->seq[at[b]].suffix_len;
        const int64_t pages = (P + S + p->page_size - 1) >> p->page_shift;
        const int32_t* row = host_block_tables + (int64_t)b * p->bt_stride;
        for (int64_t lp = 0; lp < pages; ++lp)
            if (written[row[lp]] && ++count[row[lp]] > 1)
                return fail(TALARIA_SP_EINVAL, "check_tables: page %d receives appended tokens "
                            "and is also named by sequence %d, logical page %lld", row[lp], b,
                            (long long)lp);
    }
    return TALARIA_SP_OK;
}

extern "C" int talaria_sp_attn_plan_items(const talaria_sp_plan* plan, int32_t* items,
                                          int32_t max_items) {
    int status;
    const PlanData* p = checked_plan(plan, &status);
    if (!p)
        return status;
    if (max_items < 0 || (max_items > 0 && !items))
        return fail(TALARIA_SP_EINVAL, "items must hold max_items records");
    const int32_t n = std::min(max_items, p->num_items);
    for (int32_t i = 0; i < n; ++i) {
        const WorkItem w = decode_item(*p, i);
        const int32_t P = p->seq[w.seq].prefix_len;
        const int32_t kend_all = P + w.first_token + w.num_tokens;
        int32_t* r = items + 8 * i;
        r[0] = p->seq_orig[w.seq];
        r[1] = w.kv_head;
        r[2] = w.first_token;
        r[3] = w.num_tokens;
        r[4] = std::min(w.tile_begin * kKeysPerTile, kend_all);
        r[5] = std::min(w.tile_end * kKeysPerTile, kend_all);
        r[6] = w.split;
        r[7] = w.num_splits;
    }
    return p->num_items;
}
