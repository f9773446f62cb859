// SP prefill attention on gfx950: causal attention of each continuation's new
// tokens over its cached prefix plus themselves, reading K/V from the paged
// pool through the block tables (the batched prefill of an SP step, paper
// Section 3.3, over the device-resident prefix of Section 4.3).
//
// One workgroup (4 waves, 256 threads) runs one work item of the plan: a
// query tile of 256 rows -- tile_tokens new tokens times the `group` query
// heads that share one KV head, so every K/V byte staged in LDS serves all
// of them -- against one contiguous range of 64-key tiles.  Each wave owns
// 64 rows as two 32-row MFMA blocks.
//
// Per key tile:
//   * page walk + 16-byte global loads of the next tile into registers
//     (keys at or past P_b + S_b are zero-filled, never loaded);
//   * S^T = K Q^T on v_mfma_f32_32x32x16_bf16 (K from LDS, Q in registers);
//   * causal mask only on tiles that cross the diagonal;
//   * online softmax in base 2 with a lazy rescale: the running maximum is
//     only moved (and O rescaled) when some row's new maximum exceeds it by
//     more than 2^8, so exp2 arguments stay <= 8;
//   * O^T += V^T P^T on the same MFMA, P converted to bf16 in registers
//     (the S^T accumulator layout already is the B-operand layout);
//   * the registers of the next tile go to the other LDS buffer.
//
// Items whose query tile is split over several key ranges write normalised
// fp32 partials and base-2 LSE to the workspace; the combine kernel merges
// them in a fixed order (bitwise deterministic).
#include <hip/hip_runtime.h>

#include <math.h>

#include "common.h"

namespace tsp {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kRescaleThreshold = 8.0f;  // log2 units

template <int D>
struct Smem {
    static constexpr int KSTR = D + 8;  // K tile row stride (elements): 16-byte pad
    static constexpr int VSTR = kKeysPerTile + 8;  // V^T tile row stride (elements)
    uint16_t k[2][kKeysPerTile * KSTR];
    uint16_t v[2][D * VSTR];
};

// Position of key `kk` (0..15) inside its 16-key group in the V^T tile.
// The S^T accumulator gives lane half h the keys {4h..4h+3, 8+4h..8+4h+3}
// of each 16-key group; storing the middle two quarters swapped makes those
// 8 keys contiguous, so the PV A-operand is one 16-byte LDS read.
__device__ __forceinline__ int vt_pos(int kk) {
    const int q = kk >> 2;
    const int qs = (q == 1) ? 2 : (q == 2) ? 1 : q;
    return (qs << 2) | (kk & 3);
}

template <int D>
struct TileRegs {
    static constexpr int NK = (kKeysPerTile * D / 8) / 256;  // 16-byte K chunks per thread
    static constexpr int NV = NK;                             // 16-byte V chunks per thread
    u32x4 k[NK];
    u32x4 v[NV];
};

struct ItemCtx {
    const int32_t* bt_row;  // block-table row of the sequence
    int64_t kv_head_off;    // g * (ps * D): offset of the head inside a page
    int kv_len;             // P_b + S_b
    int page_shift;
    int ps;
    int hkv;
};

// Issue the global loads of key tile `kt` into registers.
template <int D>
__device__ __forceinline__ void load_tile(TileRegs<D>& r, const ItemCtx& c, int kt,
                                          const uint16_t* __restrict__ k_pool,
                                          const uint16_t* __restrict__ v_pool) {
    const int tid = threadIdx.x;
    const int k0 = kt * kKeysPerTile;
    constexpr int CH = D / 8;
#pragma unroll
    for (int i = 0; i < TileRegs<D>::NK; ++i) {
        const int ch = tid + 256 * i;
        const int pos = k0 + ch / CH;
        const int col = ch % CH;
        if (pos < c.kv_len) {
            const int64_t page = c.bt_row[pos >> c.page_shift];
            const uint16_t* src = k_pool + (page * c.hkv) * ((int64_t)c.ps * D) + c.kv_head_off +
                                  (int64_t)(pos & (c.ps - 1)) * D + col * 8;
            r.k[i] = *reinterpret_cast<const u32x4*>(src);
        } else {
            r.k[i] = u32x4{0, 0, 0, 0};
        }
    }
    // V chunk = 8 consecutive keys of one feature row inside one page.
    const int span = c.ps < kKeysPerTile ? c.ps : kKeysPerTile;  // keys of one page in the tile
    const int gpp = span >> 3;                                   // 8-key groups per page row
#pragma unroll
    for (int i = 0; i < TileRegs<D>::NV; ++i) {
        const int ch = tid + 256 * i;
        const int grp = ch % gpp;
        const int d = (ch / gpp) % D;
        const int pj = ch / (gpp * D);
        const int pos = k0 + pj * span + grp * 8;
        if (pos < c.kv_len) {
            const int64_t page = c.bt_row[pos >> c.page_shift];
            const uint16_t* src = v_pool + (page * c.hkv) * ((int64_t)c.ps * D) + c.kv_head_off +
                                  (int64_t)d * c.ps + (pos & (c.ps - 1));
            u32x4 x = *reinterpret_cast<const u32x4*>(src);
            const int valid = c.kv_len - pos;  // zero slots at or past the end
            if (valid < 8) {
#pragma unroll
                for (int w = 0; w < 4; ++w) {
                    const int e = 2 * w;
                    uint32_t m = (e < valid ? 0x0000FFFFu : 0u) | (e + 1 < valid ? 0xFFFF0000u : 0u);
                    x[w] &= m;
                }
            }
            r.v[i] = x;
        } else {
            r.v[i] = u32x4{0, 0, 0, 0};
        }
    }
}

template <int D>
__device__ __forceinline__ void store_tile(Smem<D>& sm, int buf, const TileRegs<D>& r,
                                           const ItemCtx& c) {
    const int tid = threadIdx.x;
    constexpr int CH = D / 8;
#pragma unroll
    for (int i = 0; i < TileRegs<D>::NK; ++i) {
        const int ch = tid + 256 * i;
        const int key = ch / CH, col = ch % CH;
        *reinterpret_cast<u32x4*>(&sm.k[buf][key * Smem<D>::KSTR + col * 8]) = r.k[i];
    }
    const int span = c.ps < kKeysPerTile ? c.ps : kKeysPerTile;
    const int gpp = span >> 3;
#pragma unroll
    for (int i = 0; i < TileRegs<D>::NV; ++i) {
        const int ch = tid + 256 * i;
        const int grp = ch % gpp;
        const int d = (ch / gpp) % D;
        const int pj = ch / (gpp * D);
        const int key0 = pj * span + grp * 8;  // multiple of 8
        const int base = (key0 & ~15);
        const int kk = key0 & 15;  // 0 or 8
        uint16_t* row = &sm.v[buf][d * Smem<D>::VSTR + base];
        *reinterpret_cast<u32x2*>(row + vt_pos(kk)) = u32x2{r.v[i][0], r.v[i][1]};
        *reinterpret_cast<u32x2*>(row + vt_pos(kk + 4)) = u32x2{r.v[i][2], r.v[i][3]};
    }
}

__device__ __forceinline__ float wave_xor32(float x) {
    return __shfl_xor(x, 32);
}

template <int D>
__global__ __launch_bounds__(256, 1) void prefill_kernel(PlanData p, const uint16_t* __restrict__ q,
                                                         const uint16_t* __restrict__ k_pool,
                                                         const uint16_t* __restrict__ v_pool,
                                                         const int32_t* __restrict__ bt,
                                                         float sm_scale, uint16_t* __restrict__ out,
                                                         float* __restrict__ lse,
                                                         float* __restrict__ part_o,
                                                         float* __restrict__ part_lse) {
    __shared__ Smem<D> sm;
    constexpr int KS = D / 16;  // MFMA k-steps over the head dimension
    constexpr int DB = D / 32;  // 32-wide output blocks over the head dimension

    const WorkItem w = decode_item(p, blockIdx.x);
    const SeqDesc s = p.seq[w.seq];
    const int G = p.group;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int lq = lane & 31;
    const int lh = lane >> 5;

    ItemCtx c;
    c.bt_row = bt + (int64_t)w.seq * p.bt_stride;
    c.kv_head_off = (int64_t)w.kv_head * p.page_size * D;
    c.kv_len = s.prefix_len + s.suffix_len;
    c.page_shift = p.page_shift;
    c.ps = p.page_size;
    c.hkv = p.num_kv_heads;

    // Query rows of this lane: one per 32-row block.
    const int rows_used = p.tile_tokens * G;
    int qtok[2];   // token index inside the tile, or -1 for a padding row
    int qhead[2];
    bf16x8 qf[2][KS];
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
        const int r = wave * 64 + qb * 32 + lq;
        const int t = r / G;
        const bool valid = r < rows_used && t < w.num_tokens;
        qtok[qb] = valid ? t : -1;
        qhead[qb] = w.kv_head * G + r % G;
        const uint16_t* src = q + ((int64_t)(s.tok_off + w.first_token + t) * p.num_q_heads +
                                   qhead[qb]) * D + lh * 8;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            u32x4 x = valid ? *reinterpret_cast<const u32x4*>(src + ks * 16) : u32x4{0, 0, 0, 0};
            qf[qb][ks] = __builtin_bit_cast(bf16x8, x);
        }
    }
    // Absolute position of each row's token (padding rows: the tile's last).
    int qpos[2];
#pragma unroll
    for (int qb = 0; qb < 2; ++qb)
        qpos[qb] = s.prefix_len + w.first_token + (qtok[qb] >= 0 ? qtok[qb] : w.num_tokens - 1);
    const int tile_first_pos = s.prefix_len + w.first_token;

    const float scale = sm_scale * kLog2e;  // logits in base-2 units
    f32x16 o[2][DB];
#pragma unroll
    for (int qb = 0; qb < 2; ++qb)
#pragma unroll
        for (int db = 0; db < DB; ++db)
            o[qb][db] = f32x16{};
    float m_run[2] = {-INFINITY, -INFINITY};  // running max of scaled logits
    float l_run[2] = {0.f, 0.f};              // this lane's partial row sum

    TileRegs<D> regs;
    if (w.tile_begin < w.tile_end) {
        load_tile<D>(regs, c, w.tile_begin, k_pool, v_pool);
        store_tile<D>(sm, 0, regs, c);
    }
    __syncthreads();

    for (int kt = w.tile_begin; kt < w.tile_end; ++kt) {
        const int cur = (kt - w.tile_begin) & 1;
        const bool has_next = kt + 1 < w.tile_end;
        if (has_next)
            load_tile<D>(regs, c, kt + 1, k_pool, v_pool);

        // S^T = K Q^T: acc[qb][kb] holds 32 keys x 32 queries.
        f32x16 sacc[2][2];
#pragma unroll
        for (int qb = 0; qb < 2; ++qb)
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
                sacc[qb][kb] = f32x16{};
        const uint16_t* ktile = sm.k[cur];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
                const u32x4 a = *reinterpret_cast<const u32x4*>(
                    &ktile[(kb * 32 + lq) * Smem<D>::KSTR + ks * 16 + lh * 8]);
                const bf16x8 af = __builtin_bit_cast(bf16x8, a);
#pragma unroll
                for (int qb = 0; qb < 2; ++qb)
                    sacc[qb][kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af, qf[qb][ks],
                                                                           sacc[qb][kb], 0, 0, 0);
            }
        }

        // Causal mask, only on tiles that cross the diagonal.
        const int k0 = kt * kKeysPerTile;
        if (k0 + kKeysPerTile - 1 > tile_first_pos) {
#pragma unroll
            for (int qb = 0; qb < 2; ++qb)
#pragma unroll
                for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                    for (int j = 0; j < 16; ++j) {
                        const int key = k0 + kb * 32 + 8 * (j >> 2) + 4 * lh + (j & 3);
                        if (key > qpos[qb])
                            sacc[qb][kb][j] = -INFINITY;
                    }
        }

        // Row maxima in base-2 units (each row's 64 keys live in lanes lq
        // and lq+32; the scale is positive, so it commutes with max).
        float mt[2];
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) {
            float m = sacc[qb][0][0];
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int j = 0; j < 16; ++j)
                    m = fmaxf(m, sacc[qb][kb][j]);
            mt[qb] = fmaxf(m, wave_xor32(m)) * scale;
        }
        // Lazy rescale: only when some row's max grew by more than the threshold.
        const bool grow = (mt[0] > m_run[0] + kRescaleThreshold) ||
                          (mt[1] > m_run[1] + kRescaleThreshold);
        if (__any(grow)) {
#pragma unroll
            for (int qb = 0; qb < 2; ++qb) {
                const float mn = fmaxf(m_run[qb], mt[qb]);
                const float alpha = (mn == -INFINITY) ? 1.f : __builtin_amdgcn_exp2f(m_run[qb] - mn);
                m_run[qb] = mn;
                l_run[qb] *= alpha;
#pragma unroll
                for (int db = 0; db < DB; ++db)
                    o[qb][db] *= alpha;
            }
        }

        // P = exp2(S - m) in bf16, laid out as the B operand of O^T += V^T P^T.
        bf16x8 pf[2][4];
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) {
            const float mb = (m_run[qb] == -INFINITY) ? 0.f : m_run[qb];
            float ls = 0.f;
#pragma unroll
            for (int ks2 = 0; ks2 < 4; ++ks2) {
                bf16x8 v;
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const float pe = __builtin_amdgcn_exp2f(
                        fmaf(sacc[qb][ks2 >> 1][(ks2 & 1) * 8 + e], scale, -mb));
                    ls += pe;
                    v[e] = (__bf16)pe;
                }
                pf[qb][ks2] = v;
            }
            l_run[qb] += ls;
        }

        // O^T += V^T P^T.
        const uint16_t* vtile = sm.v[cur];
#pragma unroll
        for (int ks2 = 0; ks2 < 4; ++ks2) {
#pragma unroll
            for (int db = 0; db < DB; ++db) {
                const u32x4 a = *reinterpret_cast<const u32x4*>(
                    &vtile[(db * 32 + lq) * Smem<D>::VSTR + ks2 * 16 + lh * 8]);
                const bf16x8 af = __builtin_bit_cast(bf16x8, a);
#pragma unroll
                for (int qb = 0; qb < 2; ++qb)
                    o[qb][db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af, pf[qb][ks2],
                                                                        o[qb][db], 0, 0, 0);
            }
        }

        if (has_next)
            store_tile<D>(sm, cur ^ 1, regs, c);
        __syncthreads();
    }

    // Epilogue: full row sums, normalise, write.
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
        const float l = l_run[qb] + wave_xor32(l_run[qb]);
        const float inv = l > 0.f ? 1.f / l : 0.f;
        const float lse2 = l > 0.f ? m_run[qb] + log2f(l) : -INFINITY;
        if (qtok[qb] < 0)
            continue;
        const int r = wave * 64 + qb * 32 + lq;
        if (w.part_index < 0) {
            const int64_t row = (int64_t)(s.tok_off + w.first_token + qtok[qb]) * p.num_q_heads +
                                qhead[qb];
            uint16_t* dst = out + row * D;
#pragma unroll
            for (int db = 0; db < DB; ++db)
#pragma unroll
                for (int j4 = 0; j4 < 4; ++j4) {
                    bf16x4 v;
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        v[e] = (__bf16)(o[qb][db][j4 * 4 + e] * inv);
                    *reinterpret_cast<bf16x4*>(dst + db * 32 + j4 * 8 + lh * 4) = v;
                }
            if (lse && lh == 0)
                lse[row] = lse2 * kLn2;
        } else {
            float* dst = part_o + ((int64_t)w.part_index * kRowsPerTile + r) * D;
#pragma unroll
            for (int db = 0; db < DB; ++db)
#pragma unroll
                for (int j4 = 0; j4 < 4; ++j4) {
                    f32x4 v;
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        v[e] = o[qb][db][j4 * 4 + e] * inv;
                    *reinterpret_cast<f32x4*>(dst + db * 32 + j4 * 8 + lh * 4) = v;
                }
            if (lh == 0)
                part_lse[(int64_t)w.part_index * kRowsPerTile + r] = lse2;
        }
    }
}

// Merge the split partials of one query tile (launched per work item; only
// split 0 of a split tile does work).  Base-2 LSE merge in split order.
template <int D>
__global__ __launch_bounds__(256) void combine_kernel(PlanData p, const float* __restrict__ part_o,
                                                      const float* __restrict__ part_lse,
                                                      uint16_t* __restrict__ out,
                                                      float* __restrict__ lse) {
    const WorkItem w = decode_item(p, blockIdx.x);
    if (w.part_index < 0 || w.split != 0)
        return;
    const SeqDesc s = p.seq[w.seq];
    const int G = p.group;
    const int n = w.num_splits;
    constexpr int TPR = D / 4;            // threads per row (4 features each)
    constexpr int RPP = 256 / TPR;        // rows per pass
    const int sub = threadIdx.x % TPR;
    const int rows = w.num_tokens * G;
    for (int r = threadIdx.x / TPR; r < rows; r += RPP) {
        float mx = -INFINITY;
        for (int k = 0; k < n; ++k)
            mx = fmaxf(mx, part_lse[(int64_t)(w.part_index + k) * kRowsPerTile + r]);
        float acc[4] = {0.f, 0.f, 0.f, 0.f};
        float wsum = 0.f;
        for (int k = 0; k < n; ++k) {
            const float lk = part_lse[(int64_t)(w.part_index + k) * kRowsPerTile + r];
            const float wk = (lk == -INFINITY) ? 0.f : exp2f(lk - mx);
            wsum += wk;
            const f32x4 v = *reinterpret_cast<const f32x4*>(
                part_o + ((int64_t)(w.part_index + k) * kRowsPerTile + r) * D + sub * 4);
#pragma unroll
            for (int e = 0; e < 4; ++e)
                acc[e] += wk * v[e];
        }
        const float inv = 1.f / wsum;
        const int t = r / G;
        const int64_t row = (int64_t)(s.tok_off + w.first_token + t) * p.num_q_heads +
                            w.kv_head * G + r % G;
        bf16x4 v;
#pragma unroll
        for (int e = 0; e < 4; ++e)
            v[e] = (__bf16)(acc[e] * inv);
        *reinterpret_cast<bf16x4*>(out + row * D + sub * 4) = v;
        if (lse && sub == 0)
            lse[row] = (mx + log2f(wsum)) * kLn2;
    }
}

template <int D>
int launch_prefill(const PlanData& p, const uint16_t* q, const uint16_t* kp, const uint16_t* vp,
                   const int32_t* bt, float sm_scale, uint16_t* out, float* lse, char* ws,
                   hipStream_t st) {
    float* part_o = reinterpret_cast<float*>(ws);
    float* part_lse = ws ? reinterpret_cast<float*>(ws + p.ws_lse_offset) : nullptr;
    hipLaunchKernelGGL(prefill_kernel<D>, dim3(p.num_items), dim3(256), 0, st, p, q, kp, vp, bt,
                       sm_scale, out, lse, part_o, part_lse);
    int status = launch_status("prefill");
    if (status != TALARIA_SP_OK || p.num_part_items == 0)
        return status;
    hipLaunchKernelGGL(combine_kernel<D>, dim3(p.num_items), dim3(256), 0, st, p, part_o,
                       part_lse, out, lse);
    return launch_status("combine");
}

}  // namespace
}  // namespace tsp

using namespace tsp;

extern "C" int talaria_sp_attn_prefill(const talaria_sp_plan* plan, const void* q,
                                       const void* k_pool, const void* v_pool,
                                       const int32_t* block_tables, float sm_scale, void* out,
                                       float* lse, void* workspace, size_t workspace_bytes,
                                       void* stream) {
    int status;
    const PlanData* p = checked_plan(plan, &status);
    if (!p)
        return status;
    if (p->num_items == 0)
        return TALARIA_SP_OK;
    if (!q || !k_pool || !v_pool || !block_tables || !out)
        return fail(TALARIA_SP_EINVAL, "prefill: q, k_pool, v_pool, block_tables and out must "
                    "not be NULL");
    if (!(sm_scale == sm_scale) || isinf(sm_scale))
        return fail(TALARIA_SP_EINVAL, "prefill: sm_scale must be finite");
    if (sm_scale <= 0.f)
        sm_scale = 1.f / sqrtf((float)p->head_dim);
    if ((size_t)p->ws_bytes > workspace_bytes || (p->ws_bytes > 0 && !workspace))
        return fail(TALARIA_SP_ENOSPACE, "prefill: workspace of %zu bytes, plan needs %lld",
                    workspace_bytes, (long long)p->ws_bytes);
    hipStream_t st = reinterpret_cast<hipStream_t>(stream);
    auto qq = static_cast<const uint16_t*>(q);
    auto kp = static_cast<const uint16_t*>(k_pool);
    auto vp = static_cast<const uint16_t*>(v_pool);
    auto o = static_cast<uint16_t*>(out);
    auto ws = static_cast<char*>(workspace);
    if (p->head_dim == 128)
        return launch_prefill<128>(*p, qq, kp, vp, block_tables, sm_scale, o, lse, ws, st);
    return launch_prefill<64>(*p, qq, kp, vp, block_tables, sm_scale, o, lse, ws, st);
}
