// Decode-phase paged attention: one new token per sequence attends to its
// whole cached context (P_b cached tokens plus itself, appended first), the D
// phase that resumes for every in-flight session after an SP batch (paper
// Section 3.4).  It is the S_b = 1 case of the SP prefill, but bound by HBM:
// every K/V byte of the context is read once for only `group` query rows.
//
// Work decomposition: the prefill plan's items (sequence, KV head, key-range
// split); one workgroup of 4 waves per item.  The item's key range is cut
// into 32-key steps dealt round-robin to the waves.  A wave streams a step's
// K rows into its own LDS buffer with the buffer form of the direct-to-LDS
// load (each instruction moves 1 KB of whole rows of one page), from where
// they are read in the row order that makes S^T land in the PV B-operand
// layout; V feature rows go straight to registers as 16-byte runs of 8 keys
// (tokens are innermost in V pages, so each V instruction also reads 1 KB
// contiguous).  K buffers and V registers are double-buffered: the next
// step's loads are in flight while the current step computes.  Page numbers
// are wave-uniform scalar reads, made one step ahead of the loads that use
// them, so no load waits on its own page lookup.  Each wave keeps
// its own online-softmax state for the <= 32 query rows (one 32-row MFMA
// block); the four states are merged through LDS at the end, and split items
// go through the same log-sum-exp combine as the prefill.  Keys past the end
// are read from clamped in-range addresses and masked (K) or zeroed (V), so
// stale slots -- even NaN -- cannot reach the output.
#include <hip/hip_runtime.h>

#include <math.h>
#include <string.h>

#include "common.h"

namespace tsp {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(1))) const char gbl_char;

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kRescaleThreshold = 8.0f;  // log2 units
constexpr int kWaves = 4;
constexpr int kStep = 32;  // keys per wave step
// Buffer descriptor of a page: no range clamp that a page offset could reach,
// 32-bit data format (the raw-buffer setting).
constexpr int kRsrcRecords = 0x7fffffff;
constexpr int kRsrcFlags = 0x00020000;

// s_waitcnt immediate that waits until at most N vector-memory operations of
// the wave are outstanding (gfx9 encoding: vmcnt in bits 3:0 and 15:14,
// expcnt and lgkmcnt left at their maximum).
template <int N>
constexpr int vmcnt_only() {
    static_assert(N >= 0 && N < 64, "vmcnt out of range");
    return (N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8);
}

// One 1 KB direct-to-LDS load: each lane moves the 16 bytes at base + off
// into LDS bytes [16 lane, 16 lane + 16) of dst.
__device__ __forceinline__ void load_lds_16(const gbl_char* base, uint32_t off, char* dst) {
    const __amdgpu_buffer_rsrc_t rsrc =
        __builtin_amdgcn_make_buffer_rsrc((void*)base, 0, kRsrcRecords, kRsrcFlags);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (lds_void*)dst, 16, off, 0, 0, 0);
}

// Waits until at most N vector-memory operations of the wave are outstanding
// (a compiler-visible wait).
template <int N>
__device__ __forceinline__ void wait_vmem() {
    __builtin_amdgcn_s_waitcnt(vmcnt_only<N>());
}

__device__ __forceinline__ int pi_row(int i) {
    return (i & ~12) | ((i & 4) << 1) | ((i & 8) >> 1);
}
// 16-byte chunk swizzle of K rows in LDS (conflict-free MFMA operand reads).
template <int D>
__device__ __forceinline__ int kswz(int row) {
    return D == 128 ? (row & 15) : ((row & 3) | ((row >> 1) & 4));
}
__device__ __forceinline__ float xhalf_max(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x),
                                                    false, false);
    return __builtin_elementwise_maximum(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float xhalf_sum(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x),
                                                    false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

template <int D>
__global__ __launch_bounds__(256) void decode_kernel(PlanData p, const uint16_t* __restrict__ q,
                                                     const uint16_t* __restrict__ k_pool,
                                                     const uint16_t* __restrict__ v_pool,
                                                     const int32_t* __restrict__ bt, float sm_scale,
                                                     uint16_t* __restrict__ out,
                                                     float* __restrict__ lse,
                                                     _Float16* __restrict__ part_o,
                                                     float* __restrict__ part_lse) {
    constexpr int KS = D / 16, DB = D / 32;
    // Per-wave double-buffered K steps during the loop; the merge reuses the
    // same bytes for the waves' O tiles afterwards.
    constexpr int KBYTES = kWaves * 2 * kStep * D * 2;
    constexpr int OBYTES = kWaves * 32 * (D + 1) * 4;
    __shared__ __attribute__((aligned(1024))) char s_raw[KBYTES > OBYTES ? KBYTES : OBYTES];
    auto s_k = reinterpret_cast<uint16_t(*)[2][kStep * D]>(s_raw);
    auto s_o = reinterpret_cast<float(*)[32][D + 1]>(s_raw);
    __shared__ float s_m[kWaves][32], s_l[kWaves][32];

    const WorkItem w = decode_item(p, blockIdx.x);
    const SeqDesc s = p.seq[w.seq];
    const int G = p.group;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // uniform: scalar page reads
    const int lq = lane & 31, lh = lane >> 5;
    const int ps = p.page_size, shift = p.page_shift, hkv = p.num_kv_heads, g = w.kv_head;
    const int32_t* bt_row = bt + bt_row_index(p, w.seq) * p.bt_stride;
    const int kv_len = s.prefix_len + s.suffix_len;
    const int key_lo = w.tile_begin * kKeysPerTile;
    const int key_hi = min(w.tile_end * kKeysPerTile, kv_len);
    const int last_grp = ((kv_len - 1) >> 3) << 3;  // last 8-key group holding a key

    // Q fragments of row lq (query head g*G + lq); rows >= G are zero.
    const bool qvalid = lq < G;
    const uint16_t* qsrc =
        q + ((int64_t)(s.tok_off + w.first_token) * p.num_q_heads + g * G + (qvalid ? lq : 0)) * D +
        lh * 8;
    bf16x8 qf[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
        const u32x4 x = qvalid ? *reinterpret_cast<const u32x4*>(qsrc + ks * 16) : u32x4{0, 0, 0, 0};
        qf[ks] = __builtin_bit_cast(bf16x8, x);
    }

    const float scale = sm_scale * kLog2e;
    f32x16 o[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db)
        o[db] = f32x16{};
    float m_run = -INFINITY, l_run = 0.f;

    // K steps go HBM -> LDS with direct-to-LDS loads (1 KB contiguous per
    // instruction, KRL whole rows of one page), double-buffered per wave; V
    // goes to registers, also double-buffered.  The next step's loads are
    // issued before the current step computes.
    constexpr int KRL = 1024 / (2 * D);  // K rows per 1 KB load
    constexpr int KLOADS = kStep / KRL;  // loads per K step
    constexpr int KCH = D / 8;           // 16-byte chunks per K row
    char* const kbuf = reinterpret_cast<char*>(&s_k[wave][0][0]);
    const int last_krow_grp = ((kv_len - 1) / KRL) * KRL;
    const uint32_t page_bytes = (uint32_t)(hkv * ps * D * 2);  // < 2^31 (planner)
    const gbl_char* const kpool_g = (const gbl_char*)(const char*)k_pool + (int64_t)g * ps * D * 2;
    // Lane l fills LDS bytes [16 l, 16 l + 16) of a load: row l / KCH of the
    // load's row group, physical chunk l % KCH, which holds the row's logical
    // chunk (l % KCH) ^ kswz(row).
    uint32_t koff[KLOADS];
#pragma unroll
    for (int li = 0; li < KLOADS; ++li)
        koff[li] = (uint32_t)(((lane / KCH) * D + ((lane % KCH) ^ kswz<D>(li * KRL + lane / KCH)) * 8) * 2);
    // Pages of a step's four 8-key groups (keys k0, k0+8, k0+16, k0+24, each
    // clamped to the last group holding a key).  A K load's rows and a V
    // load's 8 keys lie in one such group, clamped the same way.
    auto pages = [&](int k0, uint32_t (&pg)[4]) {
#pragma unroll
        for (int j = 0; j < 4; ++j)
            pg[j] = (uint32_t)bt_row[min(k0 + 8 * j, last_grp) >> shift];
    };
    auto issue = [&](int k0, int b, u32x4 (&va)[2][DB], const uint32_t (&pg)[4]) {
        char* kb = kbuf + b * (kStep * D * 2);
#pragma unroll
        for (int li = 0; li < KLOADS; ++li) {
            // Groups past the end re-read the last one (masked below).
            const int key = min(k0 + li * KRL, last_krow_grp);
            const gbl_char* base = kpool_g + (uint64_t)pg[(li * KRL) >> 3] * page_bytes +
                                   (uint32_t)((key & (ps - 1)) * (D * 2));
            load_lds_16(base, koff[li], kb + li * 1024);
        }
#pragma unroll
        for (int ks2 = 0; ks2 < 2; ++ks2) {
            // The two half-waves' 8-key groups.
            const int kg0 = min(k0 + 16 * ks2, last_grp), kg1 = min(k0 + 16 * ks2 + 8, last_grp);
            const uint32_t pg0 = pg[2 * ks2], pg1 = pg[2 * ks2 + 1];
            const int kg = lh ? kg1 : kg0;
            const uint16_t* vb = v_pool + ((int64_t)(lh ? pg1 : pg0) * hkv + g) * D * ps +
                                 (kg & (ps - 1));
#pragma unroll
            for (int db = 0; db < DB; ++db)
                va[ks2][db] = *reinterpret_cast<const u32x4*>(vb + (int64_t)(db * 32 + lq) * ps);
        }
    };
    // S^T = K Q^T over the step's 32 keys (K rows read in pi_row order).
    auto qk = [&](int b) {
        const char* kb = kbuf + b * (kStep * D * 2);
        f32x16 sc = f32x16{};
        const int row = pi_row(lq);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            const int lc = 2 * ks + lh;
            const u32x4 a = *reinterpret_cast<const u32x4*>(kb + row * (2 * D) +
                                                            ((lc ^ kswz<D>(row)) << 4));
            sc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), qf[ks], sc,
                                                         0, 0, 0);
        }
        return sc;
    };
    // Softmax step and O^T += V^T P^T for the step at k0.
    auto rest = [&](int k0, f32x16 sc, u32x4 (&va)[2][DB]) {
        // V slots past the end: zero, whatever they hold.  Only the step
        // holding the end needs it (a wave-uniform test); inside it the mask
        // is applied branch-free.
        if (k0 + kStep > kv_len) {
#pragma unroll
            for (int ks2 = 0; ks2 < 2; ++ks2) {
                const int kg = min(k0 + 16 * ks2 + 8 * lh, last_grp);
#pragma unroll
                for (int db = 0; db < DB; ++db)
#pragma unroll
                    for (int e = 0; e < 8; e += 2) {
                        const uint32_t keep = (kg + e < kv_len ? 0x0000FFFFu : 0u) |
                                              (kg + e + 1 < kv_len ? 0xFFFF0000u : 0u);
                        va[ks2][db][e / 2] &= keep;
                    }
            }
        }
        // Keys outside this item's range (or past the end): -inf.
        float m = -INFINITY;
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            const int key = k0 + 16 * (j >> 3) + 8 * lh + (j & 7);
            if (key >= key_hi)
                sc[j] = -INFINITY;
            m = __builtin_elementwise_maximum(m, sc[j]);
        }
        const float mt = xhalf_max(m) * scale;
        if (__any(mt > m_run + kRescaleThreshold)) {
            const float mn = __builtin_fmaxf(m_run, mt);
            const float a = (m_run == -INFINITY) ? 1.f : __builtin_amdgcn_exp2f(m_run - mn);
            m_run = mn;
            l_run *= a;
#pragma unroll
            for (int db = 0; db < DB; ++db)
                o[db] *= a;
        }
        const float mb = (m_run == -INFINITY) ? 0.f : m_run;
        bf16x8 pf[2];
#pragma unroll
        for (int ks2 = 0; ks2 < 2; ++ks2)
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const float pv = __builtin_amdgcn_exp2f(fmaf(sc[ks2 * 8 + e], scale, -mb));
                l_run += pv;
                pf[ks2][e] = (__bf16)pv;
            }
        // O^T += V^T P^T.
#pragma unroll
        for (int ks2 = 0; ks2 < 2; ++ks2)
#pragma unroll
            for (int db = 0; db < DB; ++db)
                o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, va[ks2][db]),
                                                                pf[ks2], o[db], 0, 0, 0);
    };
    // One pipelined step on buffer b: wait for this step's K, read it from
    // LDS for S = K Q^T, then issue the step after it into the other buffer
    // (so no LDS read runs while a load into LDS is in flight, which would
    // make the compiler wait for every load), wait for this step's V and
    // finish the step.
    // The pages of the step after the next are read here too, while the
    // current step computes.
    constexpr int kStride = kWaves * kStep;
    u32x4 va0[2][DB], va1[2][DB];
    uint32_t pga[4], pgb[4];
    auto run = [&](int k0, int b, u32x4 (&va_this)[2][DB], u32x4 (&va_next)[2][DB],
                   const uint32_t (&pg_next)[4], uint32_t (&pg_after)[4]) {
        // The waits are compiler-visible (wait_vmem), so after the
        // branches join the compiler knows this step's loads are complete on
        // both paths and adds no drain of its own.
        wait_vmem<2 * DB>();
        const f32x16 sc = qk(b);
        if (k0 + kStride < key_hi) {
            issue(k0 + kStride, b ^ 1, va_next, pg_next);
            pages(k0 + 2 * kStride, pg_after);
            wait_vmem<KLOADS + 2 * DB>();
        } else {
            wait_vmem<0>();
        }
        rest(k0, sc, va_this);
    };
    int k0 = key_lo + wave * kStep;
    if (k0 < key_hi) {
        pages(k0, pga);
        issue(k0, 0, va0, pga);
        pages(k0 + kStride, pgb);
    }
    for (; k0 < key_hi; k0 += 2 * kStride) {
        run(k0, 0, va0, va1, pgb, pga);
        if (k0 + kStride >= key_hi)
            break;
        run(k0 + kStride, 1, va1, va0, pga, pgb);
    }
    __syncthreads();  // every wave is done with its K buffers (s_o aliases them)

    // Merge the four waves' states (rows lq < G) through LDS.
    const float l_row = xhalf_sum(l_run);
    if (lh == 0) {
        s_m[wave][lq] = m_run;
        s_l[wave][lq] = l_row;
    }
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r)
            s_o[wave][lq][db * 32 + 8 * (r >> 2) + 4 * lh + (r & 3)] = o[db][r];
    __syncthreads();
    constexpr int TPR = 256 / 32;  // threads per row
    constexpr int DPT = D / TPR;   // features per thread
    const int row = threadIdx.x / TPR, sub = threadIdx.x % TPR;
    if (row >= G)
        return;
    float mx = -INFINITY;
#pragma unroll
    for (int v = 0; v < kWaves; ++v)
        mx = __builtin_fmaxf(mx, s_m[v][row]);
    float wv[kWaves], l = 0.f;
#pragma unroll
    for (int v = 0; v < kWaves; ++v) {
        wv[v] = s_m[v][row] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(s_m[v][row] - mx);
        l += wv[v] * s_l[v][row];
    }
    const float inv = l > 0.f ? 1.f / l : 0.f;
    const float lse2 = l > 0.f ? mx + __log2f(l) : -INFINITY;
    float acc[DPT];
#pragma unroll
    for (int e = 0; e < DPT; ++e) {
        float a = 0.f;
#pragma unroll
        for (int v = 0; v < kWaves; ++v)
            a += wv[v] * s_o[v][row][sub * DPT + e];
        acc[e] = a * inv;
    }
    if (w.part_index < 0) {
        const int64_t orow = (int64_t)(s.tok_off + w.first_token) * p.num_q_heads + g * G + row;
        uint16_t* dst = out + orow * D + sub * DPT;
#pragma unroll
        for (int e = 0; e < DPT; e += 4) {
            bf16x4 b;
#pragma unroll
            for (int i = 0; i < 4; ++i)
                b[i] = (__bf16)acc[e + i];
            *reinterpret_cast<bf16x4*>(dst + e) = b;
        }
        if (lse && sub == 0)
            lse[orow] = lse2 * kLn2;
    } else {
        _Float16* dst = part_o + ((int64_t)w.part_index * kRowsPerTile + row) * D + sub * DPT;
#pragma unroll
        for (int e = 0; e < DPT; e += 4)
            *reinterpret_cast<f16x4*>(dst + e) = f16x4{(_Float16)acc[e], (_Float16)acc[e + 1],
                                                       (_Float16)acc[e + 2], (_Float16)acc[e + 3]};
        if (sub == 0)
            part_lse[(int64_t)w.part_index * kRowsPerTile + row] = lse2;
    }
}

}  // namespace
}  // namespace tsp

using namespace tsp;

extern "C" int talaria_sp_attn_decode(const talaria_sp_plan* plan, const void* q,
                                      const void* k_pool, const void* v_pool,
                                      const int32_t* block_tables, float sm_scale, void* out,
                                      float* lse, void* workspace, size_t workspace_bytes,
                                      void* stream) {
    int status;
    const PlanData* p = checked_plan(plan, &status);
    if (!p)
        return status;
    for (int32_t b = 0; b < p->num_seqs; ++b)
        if (p->seq[b].suffix_len > 1)
            return fail(TALARIA_SP_EINVAL, "decode: sequence %d has %d new tokens (at most 1)", b,
                        p->seq[b].suffix_len);
    if (p->group > 32)
        return fail(TALARIA_SP_EUNSUPPORTED, "decode: %d query heads per KV head (at most 32)",
                    p->group);
    if (p->num_items == 0)
        return TALARIA_SP_OK;
    if (!q || !k_pool || !v_pool || !block_tables || !out)
        return fail(TALARIA_SP_EINVAL, "decode: q, k_pool, v_pool, block_tables and out must "
                    "not be NULL");
    uint32_t scale_bits;
    memcpy(&scale_bits, &sm_scale, sizeof scale_bits);
    if ((scale_bits & 0x7f800000u) == 0x7f800000u)
        return fail(TALARIA_SP_EINVAL, "decode: sm_scale must be finite");
    if (!aligned16(q) || !aligned16(k_pool) || !aligned16(v_pool) || !aligned16(out) ||
        !aligned16(workspace) || ((uintptr_t)lse & 3u) != 0 || ((uintptr_t)block_tables & 3u) != 0)
        return fail(TALARIA_SP_EINVAL, "decode: q, k_pool, v_pool, out and workspace must be "
                    "16-byte aligned, lse and block_tables 4-byte aligned");
    if (sm_scale <= 0.f)
        sm_scale = 1.f / sqrtf((float)p->head_dim);
    if ((size_t)p->ws_bytes > workspace_bytes || (p->ws_bytes > 0 && !workspace))
        return fail(TALARIA_SP_ENOSPACE, "decode: workspace of %zu bytes, plan needs %lld",
                    workspace_bytes, (long long)p->ws_bytes);
    hipStream_t st = reinterpret_cast<hipStream_t>(stream);
    char* ws = static_cast<char*>(workspace);
    _Float16* part_o = reinterpret_cast<_Float16*>(ws);
    float* part_lse = ws ? reinterpret_cast<float*>(ws + p->ws_lse_offset) : nullptr;
    auto qq = static_cast<const uint16_t*>(q);
    auto kp = static_cast<const uint16_t*>(k_pool);
    auto vp = static_cast<const uint16_t*>(v_pool);
    auto o = static_cast<uint16_t*>(out);
    if (p->head_dim == 128)
        hipLaunchKernelGGL(decode_kernel<128>, dim3(p->num_items), dim3(256), 0, st, *p, qq, kp, vp,
                           block_tables, sm_scale, o, lse, part_o, part_lse);
    else
        hipLaunchKernelGGL(decode_kernel<64>, dim3(p->num_items), dim3(256), 0, st, *p, qq, kp, vp,
                           block_tables, sm_scale, o, lse, part_o, part_lse);
    status = launch_status("decode");
    if (status != TALARIA_SP_OK)
        return status;
    return launch_combine(*p, part_o, part_lse, o, lse, st);
}
