// Standalone block-table page gather: copy logical positions
// 0 .. P_b+S_b-1 of every sequence out of the paged pool into contiguous
// token-major rows.
//
// This is the page walk that the prefill kernel performs for every key tile,
// run on its own so that its bandwidth can be measured and its addressing
// checked bit for bit.  It is the device-side half of turning the
// layer-first page layout into a flat per-sequence view (Appendix C).
//
// Work unit: one workgroup per (logical page, sequence, KV head).  K page
// rows are contiguous and move as 16-byte chunks.  V page blocks are stored
// tokens-innermost, so V is transposed through LDS: each thread reads 8
// slots of one feature row with one 16-byte load and writes them into a
// token-major LDS tile, then reads 8 consecutive features of one token and
// writes them to the output row with one 16-byte store.  Pool and output
// bytes stream through once: loads and stores are non-temporal.
#include <hip/hip_runtime.h>

#include "common.h"

namespace tsp {

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <int D>
__global__ __launch_bounds__(256) void gather_kv_kernel(PlanData p, const uint16_t* __restrict__ k_pool,
                                                        const uint16_t* __restrict__ v_pool,
                                                        const int32_t* __restrict__ bt,
                                                        uint16_t* __restrict__ k_out,
                                                        uint16_t* __restrict__ v_out) {
    const int b = blockIdx.y;
    const int g = blockIdx.z;
    const SeqDesc s = p.seq[b];
    const int n = s.prefix_len + s.suffix_len;
    const int ps = p.page_size;
    const int lp = blockIdx.x;
    if (lp * ps >= n)
        return;
    const int ntok = min(ps, n - lp * ps);
    const int64_t page = bt[bt_row_index(p, b) * p.bt_stride + lp];
    const int hkv = p.num_kv_heads;
    const int64_t out0 = (int64_t)p.kv_off[b] + lp * ps;  // output row of slot 0

    constexpr int CH = D / 8;
    for (int c = threadIdx.x; c < ntok * CH; c += 256) {
        const int sl = c / CH, col = c % CH;
        const u32x4* src = reinterpret_cast<const u32x4*>(
                               k_pool + ((page * hkv + g) * ps + sl) * D) + col;
        u32x4* dst = reinterpret_cast<u32x4*>(k_out + ((out0 + sl) * hkv + g) * D) + col;
        __builtin_nontemporal_store(__builtin_nontemporal_load(src), dst);
    }

    // V: page block [D][ps] -> LDS tile [ps][D] (token-major, rows padded by
    // 4 bytes so the 2-byte column writes spread over the banks) -> output
    // rows in 16-byte chunks.
    extern __shared__ __attribute__((aligned(16))) char vt[];
    constexpr int kRow = 2 * D + 4;
    const uint16_t* vpage = v_pool + (page * hkv + g) * (int64_t)D * ps;
    const int ngrp = (ntok + 7) >> 3;
    for (int c = threadIdx.x; c < ngrp * D; c += 256) {
        const int d = c % D;
        const int s0 = (c / D) * 8;
        union {
            u32x4 v;
            uint16_t h[8];
        } u;
        u.v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(vpage + (int64_t)d * ps + s0));
#pragma unroll
        for (int e = 0; e < 8; ++e)
            *reinterpret_cast<uint16_t*>(vt + (s0 + e) * kRow + d * 2) = u.h[e];
    }
    __syncthreads();
    for (int c = threadIdx.x; c < ntok * CH; c += 256) {
        const int sl = c / CH, col = c % CH;
        union {
            u32x4 v;
            uint32_t w[4];
        } u;
        const uint32_t* src = reinterpret_cast<const uint32_t*>(vt + sl * kRow + col * 16);
#pragma unroll
        for (int e = 0; e < 4; ++e)
            u.w[e] = src[e];
        __builtin_nontemporal_store(
            u.v, reinterpret_cast<u32x4*>(v_out + ((out0 + sl) * hkv + g) * D) + col);
    }
}

}  // namespace
}  // namespace tsp

using namespace tsp;

extern "C" int talaria_sp_attn_gather_kv(const talaria_sp_plan* plan, const void* k_pool,
                                         const void* v_pool, const int32_t* block_tables,
                                         void* k_out, void* v_out, void* stream) {
    int status;
    const PlanData* p = checked_plan(plan, &status);
    if (!p)
        return status;
    if (p->total_kv_tokens == 0)
        return TALARIA_SP_OK;
    if (!k_pool || !v_pool || !block_tables || !k_out || !v_out)
        return fail(TALARIA_SP_EINVAL, "gather_kv: pointers must not be NULL");
    if (!aligned16(k_pool) || !aligned16(v_pool) || !aligned16(k_out) || !aligned16(v_out) ||
        ((uintptr_t)block_tables & 3u) != 0)
        return fail(TALARIA_SP_EINVAL, "gather_kv: k_pool, v_pool, k_out and v_out must be "
                    "16-byte aligned, block_tables 4-byte aligned");
    dim3 grid(p->max_seq_pages, p->num_seqs, p->num_kv_heads);
    hipStream_t st = reinterpret_cast<hipStream_t>(stream);
    auto kp = static_cast<const uint16_t*>(k_pool);
    auto vp = static_cast<const uint16_t*>(v_pool);
    auto ko = static_cast<uint16_t*>(k_out);
    auto vo = static_cast<uint16_t*>(v_out);
    // LDS: one page of V, token-major, rows padded by 4 bytes (8-slot groups
    // rounded up: a partial last group still writes whole groups).
    const size_t lds = (size_t)((p->page_size + 7) & ~7) * (2 * p->head_dim + 4);
    if (p->head_dim == 128)
        hipLaunchKernelGGL(gather_kv_kernel<128>, grid, dim3(256), lds, st, *p, kp, vp,
                           block_tables, ko, vo);
    else
        hipLaunchKernelGGL(gather_kv_kernel<64>, grid, dim3(256), lds, st, *p, kp, vp,
                           block_tables, ko, vo);
    return launch_status("gather_kv");
}
