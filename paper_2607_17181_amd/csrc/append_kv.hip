// Append the new tokens' K/V into their pool pages (bit-exact copy).
//
// Section 4.3 of the paper: a returning session gets newly allocated device
// slots and only its unconfirmed tail is recomputed; this kernel writes that
// tail's K/V into the slots.  New token i of sequence b lands at logical
// position P_b + i, i.e. page block_tables[b][(P_b+i) / page_size], slot
// (P_b+i) mod page_size.  A suffix may start and end in the middle of a
// page; slots outside [P_b, P_b + S_b) are never written.
//
// Work unit: one workgroup per (logical page touched by the suffix,
// sequence, KV head).  K rows move as 16-byte chunks (page rows are
// contiguous in both layouts).  V pages are stored tokens-innermost, so V
// is transposed through LDS: the page's new V rows arrive with 16-byte loads
// (token-major, each row padded by 16 bytes so that the column reads below
// spread over the banks), and each thread then assembles 8 consecutive slots
// of one feature row from LDS and writes them with one 16-byte store, a
// wave's stores covering whole feature rows.  Groups of 8 slots that the
// suffix only partly covers are written slot by slot.  The new rows are read
// once, so their loads are non-temporal; the pool stores stay cached for the
// prefill that follows.
#include <hip/hip_runtime.h>

#include "common.h"

namespace tsp {

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <int D>
__global__ __launch_bounds__(256) void append_kv_kernel(PlanData p, const uint16_t* __restrict__ k_new,
                                                        const uint16_t* __restrict__ v_new,
                                                        uint16_t* __restrict__ k_pool,
                                                        uint16_t* __restrict__ v_pool,
                                                        const int32_t* __restrict__ bt) {
    const int b = blockIdx.y;
    const int g = blockIdx.z;
    const SeqDesc s = p.seq[b];
    if (s.suffix_len == 0)
        return;
    const int ps = p.page_size;
    const int lp = (s.prefix_len >> p.page_shift) + (int)blockIdx.x;
    const int end = s.prefix_len + s.suffix_len;
    if (lp * ps >= end)
        return;
    const int pos_lo = max(s.prefix_len, lp * ps);
    const int pos_hi = min(end, (lp + 1) * ps);
    const int64_t page = bt[bt_row_index(p, b) * p.bt_stride + lp];
    const int hkv = p.num_kv_heads;

    // K: token rows of D bf16 = D/8 chunks of 16 bytes.
    constexpr int CH = D / 8;
    const int ntok = pos_hi - pos_lo;
    for (int c = threadIdx.x; c < ntok * CH; c += 256) {
        const int pos = pos_lo + c / CH;
        const int col = c % CH;
        const int64_t row = s.tok_off + (pos - s.prefix_len);
        const u32x4* src = reinterpret_cast<const u32x4*>(k_new + (row * hkv + g) * D) + col;
        u32x4* dst = reinterpret_cast<u32x4*>(
                         k_pool + ((page * hkv + g) * ps + (pos & (ps - 1))) * D) + col;
        *dst = __builtin_nontemporal_load(src);
    }

    // V: new rows -> LDS tile [ps][D] (row stride 2D + 16 bytes) -> page
    // block [D][ps] in groups of 8 slots of one feature row.
    extern __shared__ __attribute__((aligned(16))) char vt[];
    constexpr int kRow = 2 * D + 16;
    const int slot_lo = pos_lo - lp * ps, slot_hi = pos_hi - lp * ps;
    const int64_t row0 = s.tok_off + (lp * ps - s.prefix_len);  // row of slot 0 (may be < tok_off)
    for (int c = threadIdx.x; c < ntok * CH; c += 256) {
        const int sl = slot_lo + c / CH, col = c % CH;
        const u32x4* src = reinterpret_cast<const u32x4*>(v_new + ((row0 + sl) * hkv + g) * D) + col;
        *reinterpret_cast<u32x4*>(vt + sl * kRow + col * 16) = __builtin_nontemporal_load(src);
    }
    __syncthreads();
    const int grp_lo = slot_lo >> 3, grp_hi = (slot_hi + 7) >> 3;
    const int ngrp = grp_hi - grp_lo;
    uint16_t* vpage = v_pool + (page * hkv + g) * (int64_t)D * ps;
    for (int c = threadIdx.x; c < ngrp * D; c += 256) {
        const int d = c / ngrp;
        const int s0 = (grp_lo + c % ngrp) * 8;
        const char* col = vt + d * 2;
        uint16_t* dst = vpage + (int64_t)d * ps + s0;
        if (s0 >= slot_lo && s0 + 8 <= slot_hi) {
            union {
                u32x4 v;
                uint16_t h[8];
            } u;
#pragma unroll
            for (int e = 0; e < 8; ++e)
                u.h[e] = *reinterpret_cast<const uint16_t*>(col + (s0 + e) * kRow);
            *reinterpret_cast<u32x4*>(dst) = u.v;
        } else {
            for (int e = 0; e < 8; ++e) {
                const int sl = s0 + e;
                if (sl >= slot_lo && sl < slot_hi)
                    dst[e] = *reinterpret_cast<const uint16_t*>(col + sl * kRow);
            }
        }
    }
}

}  // namespace
}  // namespace tsp

using namespace tsp;

extern "C" int talaria_sp_attn_append_kv(const talaria_sp_plan* plan, const void* k_new,
                                         const void* v_new, void* k_pool, void* v_pool,
                                         const int32_t* block_tables, void* stream) {
    int status;
    const PlanData* p = checked_plan(plan, &status);
    if (!p)
        return status;
    if (p->total_tokens == 0)
        return TALARIA_SP_OK;
    if (!k_new || !v_new || !k_pool || !v_pool || !block_tables)
        return fail(TALARIA_SP_EINVAL, "append_kv: k_new, v_new, k_pool, v_pool and "
                    "block_tables must not be NULL");
    if (!aligned16(k_new) || !aligned16(v_new) || !aligned16(k_pool) || !aligned16(v_pool) ||
        ((uintptr_t)block_tables & 3u) != 0)
        return fail(TALARIA_SP_EINVAL, "append_kv: k_new, v_new, k_pool and v_pool must be "
                    "16-byte aligned, block_tables 4-byte aligned");
    dim3 grid(p->max_suffix_pages, p->num_seqs, p->num_kv_heads);
    hipStream_t st = reinterpret_cast<hipStream_t>(stream);
    auto kn = static_cast<const uint16_t*>(k_new);
    auto vn = static_cast<const uint16_t*>(v_new);
    auto kp = static_cast<uint16_t*>(k_pool);
    auto vp = static_cast<uint16_t*>(v_pool);
    // LDS: one page of new V rows, padded.
    const size_t lds = (size_t)p->page_size * (2 * p->head_dim + 16);
    if (p->head_dim == 128)
        hipLaunchKernelGGL(append_kv_kernel<128>, grid, dim3(256), lds, st, *p, kn, vn, kp, vp,
                           block_tables);
    else
        hipLaunchKernelGGL(append_kv_kernel<64>, grid, dim3(256), lds, st, *p, kn, vn, kp, vp,
                           block_tables);
    return launch_status("append_kv");
}
