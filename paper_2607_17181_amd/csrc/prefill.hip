// SP prefill attention on gfx950: causal attention of each continuation's new
// tokens over its cached prefix plus themselves, reading K/V from the paged
// pool through the block tables (the batched prefill of an SP step, paper
// Section 3.4, over the device-resident prefix of Section 4.3).
//
// One workgroup (8 waves, 512 threads, two waves per SIMD) runs one work item
// of the plan: a query tile of 256 rows -- tile_tokens new tokens times the
// `group` query heads that share one KV head, so every K/V byte staged in
// LDS serves all of them -- against one contiguous range of 64-key tiles.
// Each wave owns 32 query rows, as two 16-row MFMA blocks.
//
// Matrix cores.  Both products run on v_mfma_f32_16x16x32_bf16 in
// accumulation chains: S^T(16 keys x 16 queries) chains over the head
// dimension, O^T(16 features x 16 queries) over the keys.  On random bf16
// operands this shape, chained, retires about 20% more work per second than
// 32x32x16 under the part's power limit (the clock the part holds is set by
// the operand switching, not by the issue rate).  Every K or V operand read
// from LDS feeds the same chain position of both query blocks.
//
// Data movement.  K/V tiles move HBM -> LDS with the buffer form of the
// direct-to-LDS load (no register staging) into two rings, K four tiles deep
// and V five: all of a wave's loads of one tile stay inside one page, so its
// page id is one wave-uniform block-table load and the per-lane part of each
// address is loop-invariant.  Keys at or past P_b + S_b are never fetched
// from unowned pages; V entries past the end are zeroed in LDS so stale
// slots (even NaN) cannot reach the output.
//   K tile in LDS: 64 keys x D, natural key order, 16-byte chunks XOR-swizzled
//                  by key.
//   V tile in LDS: per page, [D][span] (tokens innermost, as in the pool),
//                  chunks XOR-swizzled by feature row.
// The QK^T A-operand of key block kb reads, for accumulator row r, the key
// 32 (kb / 2) + 8 (r / 4) + 4 (kb % 2) + r % 4.  With that order the S^T
// accumulators of blocks 2j and 2j+1 give lane group g (lanes 16g..16g+15)
// the 8 consecutive keys 32j + 8g .. +7 of each query: exactly the B operand
// of the PV MFMA over keys 32j .. 32j+31, so P goes from accumulator to
// operand in registers and V needs no transpose.
//
// Pipeline (per wave, one iteration per key tile t):
//     P(t) = softmax step on S(t)  VALU: fma, exp2, cvt_pk_bf16, fp32 row
//                                  sums (and, when needed, the row max
//                                  across the four lanes of a row)
//     O   += V(t-1)^T P(t-1)      D/4 x v_mfma_f32_16x16x32_bf16
//     S(t+1) = K(t+1) Q^T          D/4 x MFMA
// The two waves of a SIMD are one phase apart, so one wave's softmax runs
// while the other's MFMAs do; the MFMA phase runs at raised wave priority.
// The running maximum is lazy: O and l are rescaled only when some row's
// maximum grows by more than 2^8, so exp2 arguments stay <= 8.  Unmasked
// tiles first try the step with the running max as it stands and fall back
// to the full step (with the row max) only when some P value could exceed
// 2^8.
//
// Items whose query tile is split over several key ranges write normalised
// f16 partials and fp32 base-2 LSE to the workspace; the combine kernel
// merges them in a fixed order (bitwise deterministic).
#include <hip/hip_runtime.h>

#include <math.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <type_traits>
#include <vector>

#include "common.h"

namespace tsp {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(1))) const char gbl_char;

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kRescaleThreshold = 8.0f;  // log2 units
constexpr float kMaxLazyP = 256.0f;        // 2^kRescaleThreshold
static_assert(kRescaleThreshold == 8.0f && kMaxLazyP == 256.0f,
              "the optimistic softmax bound must equal 2^kRescaleThreshold");
constexpr int kKStages = 4;  // K tile ring depth
// Buffer descriptor of a page: no range clamp that a page offset could reach,
// 32-bit data format (the raw-buffer setting).
constexpr int kRsrcRecords = 0x7fffffff;
constexpr int kRsrcFlags = 0x00020000;
constexpr int kVStages = 5;  // V tile ring depth
constexpr int kQB = 2;       // 16-row query blocks per wave
// Combine: features per thread (one 16-byte f16 load per split, one 16-byte
// bf16 store).
constexpr int kCombineFeatures = 8;
typedef _Float16 f16xc __attribute__((ext_vector_type(kCombineFeatures)));
typedef float f32xc __attribute__((ext_vector_type(kCombineFeatures)));
typedef __bf16 bf16xc __attribute__((ext_vector_type(kCombineFeatures)));

struct NoMask {
    static constexpr bool value = false;
};
struct WithMask {
    static constexpr bool value = true;
};

template <int D, int SPAN>
struct Geo {
    static constexpr int NW = kRowsPerTile / (16 * kQB);     // waves per workgroup
    static constexpr int NT = 64 * NW;                       // threads per workgroup
    static constexpr int TILE_BYTES = kKeysPerTile * D * 2;  // one K (or V) tile
    static constexpr int LOADS = TILE_BYTES / 1024 / NW;     // wave-loads per wave per tile
    static constexpr int K_CH = D / 8;                       // 16-byte chunks per K row
    static constexpr int K_RPL = 1024 / (2 * D);             // K rows per wave-load
    static constexpr int V_CH = SPAN / 8;                    // chunks per V block row
    static constexpr int V_RPL = 1024 / (2 * SPAN);          // V block rows per wave-load
    static constexpr int V_BLOCK = 2 * D * SPAN;             // bytes of one page block
    static constexpr int V_LPB = V_BLOCK / 1024;             // wave-loads per page block
    static constexpr int KS = D / 32;                        // QK^T k-steps (chain length)
    static constexpr int DB = D / 16;                        // 16-wide output blocks
    static_assert(V_LPB >= 1, "page block smaller than one wave-load");
    static_assert(LOADS >= 1, "fewer wave-loads than waves");
    static_assert(NW == 8, "the ping-pong schedule needs 8 waves");
};

// Chunk swizzles.  A ds_read_b128 on gfx950 serves each half-wave in two
// passes, lanes {0-7, 24-31} and {8-15, 16-23} (and the same blocks +32), and
// is conflict free when the 16 lanes of a pass land on 16 distinct 16-byte
// slots of a 256-byte bank row (measured with the LDS bank-conflict counter).
// K: lane (r, g) reads chunk 4 ks + g of the key key_of(kb, r); the XOR with
// bits 0-1 and 3-4 of the key (= r) spreads every pass over all 16 slots.
template <int D>
__device__ __forceinline__ int kswz(int key) {
    return D == 128 ? ((key & 3) | ((key >> 1) & 12)) : (((key >> 1) & 1) | ((key >> 2) & 6));
}
// V: lane (r, g) reads feature row d = 16 db + r, key chunk g of the 32-key
// step.  Rows that share a bank row inside one pass get different chunks.
template <int SPAN>
__device__ __forceinline__ int vswz(int d) {
    if (SPAN <= 16)
        return 0;
    if (SPAN == 32)
        return (d >> 1) & 2;
    return d & 6;
}
// Key (tile-relative) in accumulator row r of S^T block kb.
__device__ __forceinline__ int key_of(int kb, int r) {
    return 32 * (kb >> 1) + 8 * (r >> 2) + 4 * (kb & 1) + (r & 3);
}

// Maximum / sum over the four lanes l, l^16, l^32, l^48 that hold one query
// row's keys.
__device__ __forceinline__ float quad_max(float x) {
    auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false,
                                              false);
    x = __builtin_elementwise_maximum(__uint_as_float(r[0]), __uint_as_float(r[1]));
    r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __builtin_elementwise_maximum(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float quad_sum(float x) {
    auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false,
                                              false);
    x = __uint_as_float(r[0]) + __uint_as_float(r[1]);
    r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Workgroup barrier without a memory fence.  A fenced barrier also waits for
// every direct-to-LDS load still in flight (the loads issued for tiles
// three and four ahead), which would expose their whole latency at every
// tile.  Ordering is explicit instead: each wave waits for its own loads of
// the tile that will be read (vmcnt) and for its LDS writes (lgkmcnt) before
// the barrier; the empty asm statements keep the compiler from moving memory
// accesses across it.
__device__ __forceinline__ void lds_barrier() {
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

__device__ __forceinline__ void wait_vmem_all() {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}
// Wait until at most N vector-memory loads of this wave are outstanding
// (loads complete in issue order).
template <int N>
__device__ __forceinline__ void wait_vmem_n() {
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

struct Ctx {
    const gbl_char* kpool_g;  // K pool + head offset (bytes)
    const gbl_char* vpool_g;  // V pool + head offset (bytes)
    const int32_t* bt_row;    // block-table row of the sequence
    uint32_t page_bytes;      // bytes per page (all heads); the planner bounds it below 2^31
    uint32_t last_page;       // block-table index of the sequence's last page
    int kv_len;               // P_b + S_b
    int page_shift;
    int ps;
};

// Direct-to-LDS tile loads of one wave.  Wave w's K wave-loads cover tile
// keys 8w .. 8w+7 and its V wave-loads cover the page block holding key 8w,
// so for every supported page size (>= 8) all of a wave's loads of one tile
// fall in the single page that holds key k0 + 8w: one block-table lookup
// and one base address per wave and tile; the per-lane parts are
// loop-invariant.
template <int D, int SPAN>
struct Loader {
    using G = Geo<D, SPAN>;
    uint32_t koff[G::LOADS];  // per-lane byte offsets inside the page
    uint32_t voff[G::LOADS];
    int wave;

    __device__ __forceinline__ void init(int w, int lane, int ps) {
        wave = w;
#pragma unroll
        for (int i = 0; i < G::LOADS; ++i) {
            const int li = w * G::LOADS + i;
            const int row0 = li * G::K_RPL;  // first tile key of the wave-load
            const int row = row0 + lane / G::K_CH;
            const int lc = (lane % G::K_CH) ^ kswz<D>(row);
            koff[i] = (uint32_t)((((row0 & (ps - 1)) + lane / G::K_CH) * D + lc * 8) * 2);
            const int bl = li % G::V_LPB;
            const int d = bl * G::V_RPL + lane / G::V_CH;
            const int vlc = (lane % G::V_CH) ^ vswz<SPAN>(d);
            voff[i] = (uint32_t)(((bl * G::V_RPL + lane / G::V_CH) * ps + vlc * 8) * 2);
        }
    }

    // Block-table index of this wave's page for the tile at k0, clamped to
    // the sequence's last page (a tile past the end then reads keys that are
    // masked (K) or zeroed afterwards (V), from a page the sequence owns).
    __device__ __forceinline__ uint32_t page_index(uint32_t k0, const Ctx& c) const {
        return min((k0 + 8u * (uint32_t)wave) >> c.page_shift, c.last_page);
    }

    // The loads use the buffer form of the direct-to-LDS load: a descriptor
    // built (in scalar registers) for the wave's page, plus the per-lane
    // 32-bit offset.  Unlike the global form, the compiler counts these loads
    // on the vector-memory counter only, so LDS reads issued while they are
    // in flight keep exact (not drain-all) waits.
    __device__ __forceinline__ void issue(const gbl_char* pool, const uint32_t (&off)[G::LOADS],
                                          uint32_t in_page, char* buf, uint32_t page,
                                          const Ctx& c) const {
        const gbl_char* base = pool + (uint64_t)page * c.page_bytes + in_page;
        const __amdgpu_buffer_rsrc_t rsrc =
            __builtin_amdgcn_make_buffer_rsrc((void*)base, 0, kRsrcRecords, kRsrcFlags);
#pragma unroll
        for (int i = 0; i < G::LOADS; ++i)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                rsrc, (lds_void*)(buf + (wave * G::LOADS + i) * 1024), 16, off[i], 0, 0, 0);
    }
    __device__ __forceinline__ void issue_k(char* buf, uint32_t k0, uint32_t page,
                                            const Ctx& c) const {
        issue(c.kpool_g, koff, (k0 & (uint32_t)(c.ps - 1)) * (D * 2), buf, page, c);
    }
    __device__ __forceinline__ void issue_v(char* buf, uint32_t k0, uint32_t page,
                                            const Ctx& c) const {
        issue(c.vpool_g, voff, (k0 & (uint32_t)(c.ps - 1)) * 2, buf, page, c);
    }
};

// Per-lane LDS byte offsets of the MFMA operand reads, fixed for the whole
// kernel.  Lane l reads row r = l % 16 of a 16-row operand block and the
// 16-byte chunk g = l / 16 of its 32-wide k-step.
//   K: one offset per k-step; the four key blocks sit at constant offsets
//      (the swizzle of key_of(kb, r) does not depend on kb).
//   V: feature row d = 16 db + r, keys 32 ks2 + 8 g .. +7.  The 16-feature
//      blocks and (for page blocks of at most 32 keys) the 32-key steps are
//      constant strides; 64-key blocks swizzle the key chunk by feature row,
//      so each step has its own offset.
template <int D, int SPAN>
struct OperandOffsets {
    using G = Geo<D, SPAN>;
    static constexpr bool V_UNIFORM_STEP = SPAN <= 32;
    static constexpr int VN = V_UNIFORM_STEP ? 1 : 2;
    uint32_t k[G::KS];
    uint32_t v[VN];

    __device__ __forceinline__ void init(int r, int g) {
        const int row = key_of(0, r);
#pragma unroll
        for (int ks = 0; ks < G::KS; ++ks)
            k[ks] = (uint32_t)(row * (2 * D) + (((4 * ks + g) ^ kswz<D>(row)) << 4));
#pragma unroll
        for (int j = 0; j < VN; ++j) {
            // Feature row d = 16 db + r has the swizzle of r (the swizzles
            // only look at the low four bits of d).
            const int key = 32 * j + 8 * g;
            const int pj = key / SPAN, lc = (key % SPAN) >> 3;
            v[j] = (uint32_t)(pj * G::V_BLOCK + r * (SPAN * 2) + ((lc ^ vswz<SPAN>(r)) << 4));
        }
    }
    static constexpr uint32_t kblock(int kb) {
        return (uint32_t)((32 * (kb >> 1) + 4 * (kb & 1)) * (2 * D));
    }
    // Offset of the V operand of 32-key step ks2 and feature block db.
    __device__ __forceinline__ const char* vptr(const char* vt, int ks2, int db) const {
        if (V_UNIFORM_STEP)
            return vt + v[0] + ks2 * (32 / SPAN) * G::V_BLOCK + db * 16 * SPAN * 2;
        return vt + v[ks2] + db * 16 * SPAN * 2;
    }
};

// Zero the V entries of keys kv_len .. k0+63 of the V tile in `vbuf`.
template <int D, int SPAN>
__device__ __forceinline__ void zero_v_tail(char* vbuf, int k0, int kv_len) {
    using G = Geo<D, SPAN>;
    const int first = kv_len - k0;  // first key (tile-relative) past the end
    if (first >= kKeysPerTile)
        return;
    const int ntail = kKeysPerTile - first;
    uint16_t* v = reinterpret_cast<uint16_t*>(vbuf);
    for (int e = threadIdx.x; e < D * ntail; e += G::NT) {
        const int d = e / ntail;
        const int key = first + e % ntail;
        const int pj = key / SPAN, inb = key % SPAN;
        const int phys = (inb >> 3) ^ vswz<SPAN>(d);
        v[(pj * G::V_BLOCK + d * SPAN * 2 + phys * 16) / 2 + (inb & 7)] = 0;
    }
}

__device__ __forceinline__ f32x4 mfma16(const bf16x8& a, const bf16x8& b, const f32x4& c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// S^T = K Q^T for the wave's two 16-row query blocks: per key block, the
// K operands of all k-steps, then one chain per query block.
template <int D, int SPAN>
__device__ __forceinline__ void qk_tile(f32x4 (&s)[kQB][4], const char* kbuf,
                                        const bf16x8 (&qf)[kQB][D / 32],
                                        const OperandOffsets<D, SPAN>& oo) {
    constexpr int KS = D / 32;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
        bf16x8 a[KS];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
            a[ks] = __builtin_bit_cast(
                bf16x8, *reinterpret_cast<const u32x4*>(kbuf + oo.k[ks] +
                                                        OperandOffsets<D, SPAN>::kblock(kb)));
#pragma unroll
        for (int qb = 0; qb < kQB; ++qb) {
            f32x4 acc = mfma16(a[0], qf[qb][0], f32x4{});
#pragma unroll
            for (int ks = 1; ks < KS; ++ks)
                acc = mfma16(a[ks], qf[qb][ks], acc);
            s[qb][kb] = acc;
        }
    }
}

// O^T += V^T P^T for the wave's two query blocks: per 16-feature block, the
// V operands of both 32-key steps, then one chain of two per query block.
template <int D, int SPAN>
__device__ __forceinline__ void pv_tile(f32x4 (&o)[kQB][D / 16], const char* vt,
                                        const bf16x8 (&pf)[kQB][2],
                                        const OperandOffsets<D, SPAN>& oo) {
#pragma unroll
    for (int db = 0; db < D / 16; ++db) {
        const bf16x8 a0 =
            __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(oo.vptr(vt, 0, db)));
        const bf16x8 a1 =
            __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(oo.vptr(vt, 1, db)));
#pragma unroll
        for (int qb = 0; qb < kQB; ++qb)
            o[qb][db] = mfma16(a1, pf[qb][1], mfma16(a0, pf[qb][0], o[qb][db]));
    }
}

// NaN-propagating maximum: gfx950 v_maximum3_f32 on MFMA results with no
// quieting step (no score is NaN: masked scores are -inf before the max).
__device__ __forceinline__ float max3f(float a, float b, float c) {
    return __builtin_elementwise_maximum(a, __builtin_elementwise_maximum(b, c));
}

// P(t) of one query block from S(t) with the row offset mb: two bf16x8 PV
// operands (keys 32 j + 8 g .. +7 from blocks 2j and 2j+1) and this lane's
// partial row sum (four independent partial sums, one per key block).
__device__ __forceinline__ float p_block(const f32x4 (&s)[4], bf16x8 (&pf)[2], float scale,
                                         float mb) {
    float ls[4];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
        float p[4];
#pragma unroll
        for (int j = 0; j < 4; ++j)
            p[j] = __builtin_amdgcn_exp2f(fmaf(s[kb][j], scale, -mb));
        ls[kb] = (p[0] + p[1]) + (p[2] + p[3]);
#pragma unroll
        for (int j = 0; j < 4; ++j)
            pf[kb >> 1][4 * (kb & 1) + j] = (__bf16)p[j];
    }
    return (ls[0] + ls[1]) + (ls[2] + ls[3]);
}

// One online-softmax step on S(t): returns P(t) as bf16 B-operands, updates
// the running max / row sums, and reports whether O must be rescaled by
// alpha before P(t) is accumulated.
template <bool MASK>
__device__ __forceinline__ bool softmax_tile(f32x4 (&s)[kQB][4], bf16x8 (&pf)[kQB][2],
                                             float (&m_run)[kQB], float (&l_run)[kQB],
                                             float (&alpha)[kQB], float scale, int k0,
                                             const int (&qpos)[kQB], int g) {
    if (MASK) {
#pragma unroll
        for (int qb = 0; qb < kQB; ++qb)
#pragma unroll
            for (int kb = 0; kb < 4; ++kb)
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int key = k0 + 32 * (kb >> 1) + 8 * g + 4 * (kb & 1) + j;
                    if (key > qpos[qb])
                        s[qb][kb][j] = -INFINITY;
                }
    }
    float mt[kQB];
    bool grow = false;
#pragma unroll
    for (int qb = 0; qb < kQB; ++qb) {
        float m = max3f(s[qb][0][0], s[qb][0][1], s[qb][0][2]);
        m = max3f(m, s[qb][0][3], s[qb][1][0]);
        m = max3f(m, s[qb][1][1], s[qb][1][2]);
        m = max3f(m, s[qb][1][3], s[qb][2][0]);
        m = max3f(m, s[qb][2][1], s[qb][2][2]);
        m = max3f(m, s[qb][2][3], s[qb][3][0]);
        m = max3f(m, s[qb][3][1], s[qb][3][2]);
        m = __builtin_elementwise_maximum(m, s[qb][3][3]);
        mt[qb] = quad_max(m) * scale;
        grow = grow || (mt[qb] > m_run[qb] + kRescaleThreshold);
    }
    const bool resc = __any(grow);
    if (resc) {
#pragma unroll
        for (int qb = 0; qb < kQB; ++qb) {
            const float mn = __builtin_fmaxf(m_run[qb], mt[qb]);
            alpha[qb] = (mn == -INFINITY) ? 1.f : __builtin_amdgcn_exp2f(m_run[qb] - mn);
            m_run[qb] = mn;
            l_run[qb] *= alpha[qb];
        }
    }
#pragma unroll
    for (int qb = 0; qb < kQB; ++qb) {
        const float mb = (m_run[qb] == -INFINITY) ? 0.f : m_run[qb];
        l_run[qb] += p_block(s[qb], pf[qb], scale, mb);
    }
    return resc;
}

// Optimistic softmax step for a tile without masked keys: P(t) with the
// running max as it stands, skipping the row maximum.  softmax_tile would
// leave the max where it is exactly when no P value exceeds 2^8, and then
// both compute the same P and row sums.  A lane's partial row sum bounds its
// P values, so the step is accepted when no lane's sum exceeds 2^8 (and
// every row already has a finite running max); otherwise the caller redoes
// the tile with softmax_tile.  Returns whether the step was accepted.
__device__ __forceinline__ bool softmax_fast(const f32x4 (&s)[kQB][4], bf16x8 (&pf)[kQB][2],
                                             const float (&m_run)[kQB], float (&l_run)[kQB],
                                             float scale) {
    bool bad = false;
    float lsum[kQB];
#pragma unroll
    for (int qb = 0; qb < kQB; ++qb) {
        bad = bad || (m_run[qb] == -INFINITY);
        lsum[qb] = p_block(s[qb], pf[qb], scale, m_run[qb]);
        bad = bad || !(lsum[qb] <= kMaxLazyP);
    }
    if (__any(bad))
        return false;
#pragma unroll
    for (int qb = 0; qb < kQB; ++qb)
        l_run[qb] += lsum[qb];
    return true;
}

template <int D, int SPAN>
__global__ __launch_bounds__(512, 1) void prefill_kernel(
    PlanData p, const uint16_t* __restrict__ q, const uint16_t* __restrict__ k_pool,
    const uint16_t* __restrict__ v_pool, const int32_t* __restrict__ bt, float sm_scale,
    uint16_t* __restrict__ out, float* __restrict__ lse, _Float16* __restrict__ part_o,
    float* __restrict__ part_lse) {
    using G = Geo<D, SPAN>;
    static_assert(G::NT == 512, "launch bounds mismatch");
    __shared__ __attribute__((aligned(1024))) char smem[(kKStages + kVStages) * G::TILE_BYTES];

    // Workgroup i runs on XCD i % 8; an XCD-placed plan names its item.
    const WorkItem w =
        decode_item(p, p.wg_mapped ? (int32_t)plan_byte(p.item_of_wg, blockIdx.x)
                                   : (int32_t)blockIdx.x);
    const SeqDesc s = p.seq[w.seq];
    const int Gq = p.group;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int lr = lane & 15;  // operand / accumulator column (query) of this lane
    const int lg = lane >> 4;  // lane group: k-chunk of operands, row quad of accumulators

    Ctx c;
    c.page_bytes = (uint32_t)(p.num_kv_heads * p.page_size * D * 2);
    c.kpool_g = (const gbl_char*)(const char*)k_pool + (int64_t)w.kv_head * p.page_size * D * 2;
    c.vpool_g = (const gbl_char*)(const char*)v_pool + (int64_t)w.kv_head * p.page_size * D * 2;
    c.bt_row = bt + bt_row_index(p, w.seq) * p.bt_stride;
    c.kv_len = s.prefix_len + s.suffix_len;
    c.page_shift = p.page_shift;
    c.last_page = (uint32_t)(c.kv_len - 1) >> p.page_shift;
    c.ps = p.page_size;

    Loader<D, SPAN> ld;
    ld.init(wave, lane, c.ps);
    OperandOffsets<D, SPAN> oo;
    oo.init(lr, lg);

    const int tb = w.tile_begin, te = w.tile_end;
    // Ring slots: K tile t in kbuf(t), V tile t in vbuf(t).  Inside the main
    // loop the slots in use are carried as byte offsets and stepped once per
    // tile (no modulo per access).
    constexpr uint32_t TB = G::TILE_BYTES;
    constexpr uint32_t KRING = kKStages * TB;
    static_assert((KRING & (KRING - 1)) == 0, "K ring size must be a power of two");
    auto kslot = [&](int t) -> uint32_t { return (uint32_t)(t % kKStages) * TB; };
    auto vslot = [&](int t) -> uint32_t { return KRING + (uint32_t)(t % kVStages) * TB; };
    auto kbuf = [&](int t) -> char* { return smem + kslot(t); };
    auto vbuf = [&](int t) -> char* { return smem + vslot(t); };
    auto knext = [](uint32_t x) -> uint32_t { return (x + TB) & (KRING - 1); };
    auto vnext = [](uint32_t x) -> uint32_t {
        return x + TB == KRING + kVStages * TB ? KRING : x + TB;
    };

    // Load schedule.  In iteration t every wave issues its share of
    // K(t + kd) and V(t + vd), kd = 3 / vd = 2, at the start of the
    // iteration, which in both groups falls between barriers t-1 and t.  The
    // prologue loads the tiles the first iterations need.  No tile at or past
    // te is loaded, so the workgroup never ends with a direct-to-LDS load in
    // flight.
    const bool group_b = wave >= G::NW / 2;
    constexpr int kd = 3, vd = 2;
    // Query rows of this lane, one per 16-row block, loaded first: they
    // need no block-table lookup, so they are in flight while the page ids
    // of the first tiles are read.
    const int rows_used = p.tile_tokens * Gq;
    int qtok[kQB], qhead[kQB], qpos[kQB];
    bf16x8 qf[kQB][D / 32];
#pragma unroll
    for (int qb = 0; qb < kQB; ++qb) {
        const int r = (wave * kQB + qb) * 16 + lr;
        const int t = r / Gq;
        const bool valid = r < rows_used && t < w.num_tokens;
        qtok[qb] = valid ? t : -1;
        qhead[qb] = w.kv_head * Gq + r % Gq;
        qpos[qb] = s.prefix_len + w.first_token + (valid ? t : w.num_tokens - 1);
        const uint16_t* src = q + ((int64_t)(s.tok_off + w.first_token + t) * p.num_q_heads +
                                   qhead[qb]) * D + lg * 8;
#pragma unroll
        for (int ks = 0; ks < D / 32; ++ks) {
            u32x4 x = valid ? *reinterpret_cast<const u32x4*>(src + ks * 32) : u32x4{0, 0, 0, 0};
            qf[qb][ks] = __builtin_bit_cast(bf16x8, x);
        }
    }

    // Then K(tb), K(tb+1) -- which the prologue and the first iteration
    // read -- and K(tb+2), V(tb), V(tb+1), which the prologue does not wait
    // for.
#pragma unroll
    for (int k = 0; k < 4; ++k)
        if (k < kd && tb + k < te)
            ld.issue_k(kbuf(tb + k), (tb + k) * kKeysPerTile,
                       c.bt_row[ld.page_index((tb + k) * kKeysPerTile, c)], c);
#pragma unroll
    for (int k = 0; k < 3; ++k)
        if (k < vd && tb + k < te)
            ld.issue_v(vbuf(tb + k), (tb + k) * kKeysPerTile,
                       c.bt_row[ld.page_index((tb + k) * kKeysPerTile, c)], c);
    uint32_t pgk_next = c.bt_row[ld.page_index((tb + kd) * kKeysPerTile, c)];
    uint32_t pgv_next = c.bt_row[ld.page_index((tb + vd) * kKeysPerTile, c)];

    const float scale = sm_scale * kLog2e;  // logits in base-2 units
    f32x4 o[kQB][D / 16];
#pragma unroll
    for (int qb = 0; qb < kQB; ++qb)
#pragma unroll
        for (int db = 0; db < D / 16; ++db)
            o[qb][db] = f32x4{};
    float m_run[kQB], l_run[kQB], alpha[kQB];
#pragma unroll
    for (int qb = 0; qb < kQB; ++qb) {
        m_run[qb] = -INFINITY;
        l_run[qb] = 0.f;  // this lane's partial row sum
        alpha[qb] = 1.f;
    }
    bool resc = false;

    {
        // The V slot that PV(tb-1) reads: zero, so 0 * V stays 0.
        u32x4* vz = reinterpret_cast<u32x4*>(vbuf(tb - 1 + kVStages));
        for (int i = threadIdx.x; i < G::TILE_BYTES / 16; i += G::NT)
            vz[i] = u32x4{0, 0, 0, 0};
    }
    // Loads complete in issue order: with all five tiles issued, at most
    // the last three tiles' loads may still be in flight.
    if (te - tb >= kd)
        wait_vmem_n<3 * G::LOADS>();
    else
        wait_vmem_all();
    lds_barrier();

    f32x4 sc[kQB][4];
    bf16x8 pf[kQB][2];
#pragma unroll
    for (int qb = 0; qb < kQB; ++qb)
#pragma unroll
        for (int k = 0; k < 2; ++k)
            pf[qb][k] = bf16x8{};
    if (tb < te)
        qk_tile<D, SPAN>(sc, kbuf(tb), qf, oo);

    // tmask = smallest t with t * 64 + 63 > tile_first_pos (first tile that
    // can hold keys past some row of the query tile).
    const int tile_first_pos = s.prefix_len + w.first_token;
    const int tmask = tile_first_pos < kKeysPerTile - 1
                          ? 0 : (tile_first_pos - (kKeysPerTile - 1)) / kKeysPerTile + 1;

    // Ping-pong.  Every wave runs the same iteration -- softmax(t), then the
    // MFMA phase PV(t-1) + QK(t+1) -- and passes one workgroup barrier per
    // tile.  Waves of group B (the second wave on each SIMD) take that
    // barrier between their two phases, group A after both, so B trails A by
    // one phase: one wave's softmax runs while the other wave's MFMAs run.
    // Between barriers t-1 and t the waves read K(t), K(t+1), V(t-2) and
    // V(t-1); K(j) occupies its ring slot from barrier j-4 to j, V(j) from
    // barrier j-3 to j+2.  A barrier waits only for the loads issued before
    // the previous barrier (the 2 * LOADS issued since may stay in flight).
    // Invariant at the start of iteration t: sc = S(t), pf = P(t-1); a pending
    // rescale (resc, alpha) from softmax(t-1) is applied to O just before
    // P(t-1) is accumulated.  Slots: k_rd holds K(t+1), k_wr receives
    // K(t+kd), v_rd holds V(t-1), v_wr receives V(t+vd).
    uint32_t k_rd = kslot(tb + 1), k_wr = kslot(tb + kd);
    uint32_t v_rd = vslot(tb - 1 + kVStages), v_wr = vslot(tb + vd);
    // Loads for tiles at or past te are not issued, so in the last kd
    // iterations fewer than 2 * LOADS loads are younger than the ones a
    // barrier must see; there it waits for every load.  The loop therefore
    // ends with no load in flight.
    auto sync_point = [&](int t) {
        if (t + kd < te)
            wait_vmem_n<2 * G::LOADS>();
        else
            wait_vmem_all();
        lds_barrier();
    };
    // Operand reads and MFMAs of one MFMA phase (PV then QK).
    constexpr int kReads = 2 * (D / 16) + 4 * (D / 32);  // V: 2 per feature block; K: 4 x KS
    constexpr int kMfmas = 2 * kReads;
    constexpr int kAhead = 6;  // operand reads issued ahead of the MFMAs
    auto iteration = [&](int t, auto mask_tag, const bf16x8 (&pf)[kQB][2],
                         bf16x8 (&pn)[kQB][2]) __attribute__((always_inline)) {
        constexpr bool MASK = decltype(mask_tag)::value;
        // Pages of the next iteration's loads.  The scalar loads are issued
        // here and waited for after the softmax (which has no LDS traffic):
        // while a scalar load is outstanding every LDS wait must drain all
        // LDS reads, which would serialise the MFMA phase's operand reads.
        const uint32_t pk = c.bt_row[ld.page_index((uint32_t)(t + 1 + kd) * kKeysPerTile, c)];
        const uint32_t pv = c.bt_row[ld.page_index((uint32_t)(t + 1 + vd) * kKeysPerTile, c)];
        float an[kQB];
        // This iteration's tile loads, issued before the softmax so that the
        // MFMA phase holds only operand reads and MFMAs.
        if (t + kd < te)
            ld.issue_k(smem + k_wr, (uint32_t)(t + kd) * kKeysPerTile, pgk_next, c);
        if (t + vd < te)
            ld.issue_v(smem + v_wr, (uint32_t)(t + vd) * kKeysPerTile, pgv_next, c);
        bool rn = false;
        if (MASK || !softmax_fast(sc, pn, m_run, l_run, scale))
            rn = softmax_tile<MASK>(sc, pn, m_run, l_run, an, scale, t * kKeysPerTile, qpos, lg);
        // The whole softmax step completes here, ahead of the MFMA phase (the
        // compiler would otherwise sink its exp/convert/sum tail past it).
#pragma unroll
        for (int qb = 0; qb < kQB; ++qb) {
#pragma unroll
            for (int k = 0; k < 2; ++k)
                asm volatile("" ::"v"(pn[qb][k]));
            asm volatile("" ::"v"(l_run[qb]));
        }
        asm volatile("" ::"s"(pk), "s"(pv));
        if (group_b)
            sync_point(t);
        __builtin_amdgcn_sched_barrier(0);
        // The MFMA phase runs at raised wave priority: its SIMD partner is in
        // its softmax, and without this the partner's VALU stream (an older
        // wave for group B) wins issue slots and stretches the MFMA phase.
        __builtin_amdgcn_s_setprio(1);
        if (resc) {
#pragma unroll
            for (int qb = 0; qb < kQB; ++qb)
#pragma unroll
                for (int db = 0; db < D / 16; ++db)
                    o[qb][db] *= alpha[qb];
        }
        // MFMA phase, unconditional: P(tb-1) = 0 over a zeroed V stage, and
        // S(te) comes from a slot K(te) was never loaded into and is never
        // used.
        pv_tile<D, SPAN>(o, smem + v_rd, pf, oo);
        qk_tile<D, SPAN>(sc, smem + k_rd, qf, oo);
        // Operand reads run kAhead reads ahead of the MFMAs that use them,
        // across the PV / QK boundary: each read feeds two MFMAs.
        __builtin_amdgcn_sched_group_barrier(0x100, kAhead, 0);
#pragma unroll
        for (int i = 0; i < kReads - kAhead; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
        __builtin_amdgcn_sched_group_barrier(0x008, kMfmas - 2 * (kReads - kAhead), 0);
        __builtin_amdgcn_s_setprio(0);
        pgk_next = pk;
        pgv_next = pv;
        k_rd = knext(k_rd);
        k_wr = knext(k_wr);
        v_rd = vnext(v_rd);
        v_wr = vnext(v_wr);
#pragma unroll
        for (int qb = 0; qb < kQB; ++qb)
            alpha[qb] = an[qb];
        resc = rn;
        if (!group_b)
            sync_point(t);
    };

    // P alternates between two register sets, two iterations per loop trip,
    // so that no copy is needed: at the start of a trip P(t-1) is in pf.
    bf16x8 pn[kQB][2];
    auto run = [&](int t0, int t1, auto mask_tag) __attribute__((always_inline)) {
        int t = t0;
        for (; t + 1 < t1; t += 2) {
            iteration(t, mask_tag, pf, pn);
            iteration(t + 1, mask_tag, pn, pf);
        }
        if (t < t1) {
            iteration(t, mask_tag, pf, pn);
#pragma unroll
            for (int qb = 0; qb < kQB; ++qb)
#pragma unroll
                for (int k = 0; k < 2; ++k)
                    pf[qb][k] = pn[qb][k];
        }
    };
    const int split = tmask < tb ? tb : (tmask > te ? te : tmask);
    // Calibration launches record the main loop's duration per workgroup.
    const uint64_t loop_t0 = p.stamps ? __builtin_amdgcn_s_memrealtime() : 0;
    run(tb, split, NoMask{});
    run(split, te, WithMask{});
    if (p.stamps && threadIdx.x == 0) {
        uint64_t* rec = reinterpret_cast<uint64_t*>(p.stamps) + 4 * (uint64_t)blockIdx.x;
        rec[0] = __builtin_amdgcn_s_getreg((3 << 11) | 20);  // XCC id (HW_REG_XCC_ID[3:0])
        rec[1] = (uint64_t)(te - tb);
        rec[2] = loop_t0;
        rec[3] = __builtin_amdgcn_s_memrealtime();
    }

    if (tb < te) {
        // Of this item's tiles only the last one can reach past the sequence's
        // end (every earlier tile ends below the item's visible key count,
        // which is at most P_b + S_b), and it is read only here: clear its V
        // entries past the end once, now that it has landed.
        if (te * kKeysPerTile > c.kv_len) {
            wait_vmem_all();
            __syncthreads();
            zero_v_tail<D, SPAN>(vbuf(te - 1), (te - 1) * kKeysPerTile, c.kv_len);
            __syncthreads();
        }
        if (resc) {
#pragma unroll
            for (int qb = 0; qb < kQB; ++qb)
#pragma unroll
                for (int db = 0; db < D / 16; ++db)
                    o[qb][db] *= alpha[qb];
        }
        pv_tile<D, SPAN>(o, vbuf(te - 1), pf, oo);
    }

    // Epilogue: full row sums, normalise, write.  Lane group g holds features
    // 16 db + 4 g .. +3 of its query row.
#pragma unroll
    for (int qb = 0; qb < kQB; ++qb) {
        const float l = quad_sum(l_run[qb]);
        const float inv = l > 0.f ? 1.f / l : 0.f;
        const float lse2 = l > 0.f ? m_run[qb] + __log2f(l) : -INFINITY;
        if (qtok[qb] < 0)
            continue;
        const int r = (wave * kQB + qb) * 16 + lr;
        if (w.part_index < 0) {
            const int64_t row = (int64_t)(s.tok_off + w.first_token + qtok[qb]) * p.num_q_heads +
                                qhead[qb];
            uint16_t* dst = out + row * D + lg * 4;
#pragma unroll
            for (int db = 0; db < D / 16; ++db) {
                bf16x4 v;
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    v[e] = (__bf16)(o[qb][db][e] * inv);
                *reinterpret_cast<bf16x4*>(dst + db * 16) = v;
            }
            if (lse && lg == 0)
                lse[row] = lse2 * kLn2;
        } else {
            // Device-scope stores: they write through this XCD's L2, so the
            // partials reach memory while the kernel runs and the end of the
            // launch has none of them left to write back for the combine.
            _Float16* dst = part_o + ((int64_t)w.part_index * kRowsPerTile + r) * D + lg * 4;
#pragma unroll
            for (int db = 0; db < D / 16; ++db)
                __hip_atomic_store(reinterpret_cast<uint64_t*>(dst + db * 16),
                                   __builtin_bit_cast(uint64_t, __builtin_convertvector(
                                                                    o[qb][db] * inv, f16x4)),
                                   __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (lg == 0)
                __hip_atomic_store(part_lse + (int64_t)w.part_index * kRowsPerTile + r, lse2,
                                   __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    }
}

// Merge the split partials of one query tile, 256 / (D / kCombineFeatures)
// rows per workgroup.  Only
// split query tiles are launched (blocks past a sequence's own tile count,
// or of sequences without splits, exit at once): a grid over every work
// item spent most of its time dispatching blocks with nothing to do.
// Base-2 LSE merge in split order, KB splits per round of loads (8, 16 or
// 32, the fewest rounds for the plan's most-split tile: a decode batch's
// longest sequences take up to 64 splits).
template <int D, int KB>
__global__ __launch_bounds__(256) void combine_kernel(PlanData p,
                                                      const _Float16* __restrict__ part_o,
                                                      const float* __restrict__ part_lse,
                                                      uint16_t* __restrict__ out,
                                                      float* __restrict__ lse) {
    // Grid: (split query tile of the sequence, row block, sequence); the
    // tile's split 0 item is item_off + tile * splits.
    const int32_t b = blockIdx.z;
    const int32_t nsp = num_splits_of(p, b);
    if (nsp <= 1 || (int32_t)blockIdx.x >= num_q_tiles(p, b) * p.num_kv_heads)
        return;
    const WorkItem w = decode_item(p, p.seq[b].item_off + (int32_t)blockIdx.x * nsp);
    constexpr int TPR = D / kCombineFeatures;  // threads per row
    constexpr int RPB = 256 / TPR;             // rows per block
    const int r = blockIdx.y * RPB + threadIdx.x / TPR;
    const int G = p.group;
    if (r >= w.num_tokens * G)
        return;
    const SeqDesc s = p.seq[w.seq];
    const int n = w.num_splits;
    const int sub = threadIdx.x % TPR;
    const float* lse_k = part_lse + (int64_t)w.part_index * kRowsPerTile + r;
    const _Float16* o_k =
        part_o + ((int64_t)w.part_index * kRowsPerTile + r) * D + sub * kCombineFeatures;
    constexpr int64_t kStrideO = (int64_t)kRowsPerTile * D;
    // Online merge in split order, KB splits per round of loads (all issued
    // before any is used): the running maximum only grows, and the sums are
    // rescaled when a later round raises it.  KB follows from the plan, so
    // for a fixed plan every result bit is fixed.
    float mx = -INFINITY;
    f32xc acc = {};
    float wsum = 0.f;
    for (int k0 = 0; k0 < n; k0 += KB) {
        float lk[KB];
        f16xc v[KB];  // converted where used: the raw halves take half the registers
#pragma unroll
        for (int k = 0; k < KB; ++k) {
            lk[k] = -INFINITY;
            if (k0 + k < n) {
                lk[k] = lse_k[(k0 + k) * kRowsPerTile];
                v[k] = *reinterpret_cast<const f16xc*>(o_k + (k0 + k) * kStrideO);
            }
        }
        float cm = mx;
#pragma unroll
        for (int k = 0; k < KB; ++k)
            cm = fmaxf(cm, lk[k]);
        if (cm > mx) {
            const float a = __builtin_amdgcn_exp2f(mx - cm);  // 0 while mx is -inf
            wsum *= a;
            acc *= a;
            mx = cm;
        }
#pragma unroll
        for (int k = 0; k < KB; ++k)
            if (k0 + k < n) {
                const float wk = (lk[k] == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f(lk[k] - mx);
                wsum += wk;
                acc += wk * __builtin_convertvector(v[k], f32xc);
            }
    }
    const float inv = 1.f / wsum;
    const int t = r / G;
    const int64_t row = (int64_t)(s.tok_off + w.first_token + t) * p.num_q_heads +
                        w.kv_head * G + r % G;
    bf16xc v;
#pragma unroll
    for (int e = 0; e < kCombineFeatures; ++e)
        v[e] = (__bf16)(acc[e] * inv);
    *reinterpret_cast<bf16xc*>(out + row * D + sub * kCombineFeatures) = v;
    if (lse && sub == 0)
        lse[row] = (mx + __log2f(wsum)) * kLn2;
}

template <int D, int SPAN>
void launch_prefill_kernel(const PlanData& p, const uint16_t* q, const uint16_t* kp,
                           const uint16_t* vp, const int32_t* bt, float sm_scale, uint16_t* out,
                           float* lse, _Float16* part_o, float* part_lse, hipStream_t st) {
    hipLaunchKernelGGL((prefill_kernel<D, SPAN>), dim3(p.num_items), dim3(Geo<D, SPAN>::NT), 0,
                       st, p, q, kp, vp, bt, sm_scale, out, lse,
                       part_o, part_lse);
}

template <int D>
int launch_prefill(const PlanData& p, const uint16_t* q, const uint16_t* kp, const uint16_t* vp,
                   const int32_t* bt, float sm_scale, uint16_t* out, float* lse, char* ws,
                   hipStream_t st) {
    _Float16* part_o = reinterpret_cast<_Float16*>(ws);
    float* part_lse = ws ? reinterpret_cast<float*>(ws + p.ws_lse_offset) : nullptr;
    switch (p.page_size) {
    case 8:
        launch_prefill_kernel<D, 8>(p, q, kp, vp, bt, sm_scale, out, lse, part_o, part_lse, st);
        break;
    case 16:
        launch_prefill_kernel<D, 16>(p, q, kp, vp, bt, sm_scale, out, lse, part_o, part_lse, st);
        break;
    case 32:
        launch_prefill_kernel<D, 32>(p, q, kp, vp, bt, sm_scale, out, lse, part_o, part_lse, st);
        break;
    default:
        launch_prefill_kernel<D, 64>(p, q, kp, vp, bt, sm_scale, out, lse, part_o, part_lse, st);
        break;
    }
    int status = launch_status("prefill");
    if (status != TALARIA_SP_OK)
        return status;
    return launch_combine(p, part_o, part_lse, out, lse, st);
}

}  // namespace

int launch_combine(const PlanData& p, const _Float16* part_o, const float* part_lse,
                   uint16_t* out, float* lse, hipStream_t st) {
    if (p.num_part_items == 0)
        return TALARIA_SP_OK;
    // The grid covers only split query tiles: per sequence, as many tiles as
    // the longest split sequence has, and the rows of the tallest split tile
    // (a decode batch's split tiles hold `group` rows, not kRowsPerTile).
    int32_t rows = 0, tiles = 0, max_splits = 0;
    for (int32_t b = 0; b < p.num_seqs; ++b)
        if (num_splits_of(p, b) > 1) {
            max_splits = max_splits > num_splits_of(p, b) ? max_splits : num_splits_of(p, b);
            const int32_t t = p.seq[b].suffix_len < p.tile_tokens ? p.seq[b].suffix_len
                                                                  : p.tile_tokens;
            rows = rows > t * p.group ? rows : t * p.group;
            const int32_t n = num_q_tiles(p, b) * p.num_kv_heads;
            tiles = tiles > n ? tiles : n;
        }
    if (rows == 0)
        return TALARIA_SP_OK;
    auto launch = [&](auto d_tag, auto kb_tag) {
        constexpr int D = decltype(d_tag)::value, KB = decltype(kb_tag)::value;
        const dim3 grid(tiles, ceil_div(rows, 256 / (D / kCombineFeatures)), p.num_seqs);
        hipLaunchKernelGGL((combine_kernel<D, KB>), grid, dim3(256), 0, st, p, part_o, part_lse,
                           out, lse);
    };
    auto with_kb = [&](auto d_tag) {
        if (max_splits > 16)
            launch(d_tag, std::integral_constant<int, 32>{});
        else if (max_splits > 8)
            launch(d_tag, std::integral_constant<int, 16>{});
        else
            launch(d_tag, std::integral_constant<int, 8>{});
    };
    if (p.head_dim == 128)
        with_kb(std::integral_constant<int, 128>{});
    else
        with_kb(std::integral_constant<int, 64>{});
    return launch_status("combine");
}

}  // namespace tsp

using namespace tsp;

namespace {

// Argument checks and launch shared by the prefill call and the XCD
// calibration call.
int prefill_impl(const PlanData& pd, const void* q, const void* k_pool, const void* v_pool,
                 const int32_t* block_tables, float sm_scale, void* out, float* lse,
                 void* workspace, size_t workspace_bytes, void* stream) {
    const PlanData* p = &pd;
    if (p->num_items == 0)
        return TALARIA_SP_OK;
    if (!q || !k_pool || !v_pool || !block_tables || !out)
        return fail(TALARIA_SP_EINVAL, "prefill: q, k_pool, v_pool, block_tables and out must "
                    "not be NULL");
    uint32_t scale_bits;
    memcpy(&scale_bits, &sm_scale, sizeof scale_bits);
    if ((scale_bits & 0x7f800000u) == 0x7f800000u)
        return fail(TALARIA_SP_EINVAL, "prefill: sm_scale must be finite");
    if (!aligned16(q) || !aligned16(k_pool) || !aligned16(v_pool) || !aligned16(out) ||
        !aligned16(workspace) || ((uintptr_t)lse & 3u) != 0 || ((uintptr_t)block_tables & 3u) != 0)
        return fail(TALARIA_SP_EINVAL, "prefill: q, k_pool, v_pool, out and workspace must be "
                    "16-byte aligned, lse and block_tables 4-byte aligned");
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

}  // namespace

extern "C" int talaria_sp_attn_prefill(const talaria_sp_plan* plan, const void* q,
                                       const void* k_pool, const void* v_pool,
                                       const int32_t* block_tables, float sm_scale, void* out,
                                       float* lse, void* workspace, size_t workspace_bytes,
                                       void* stream) {
    int status;
    const PlanData* p = checked_plan(plan, &status);
    if (!p)
        return status;
    return prefill_impl(*p, q, k_pool, v_pool, block_tables, sm_scale, out, lse, workspace,
                        workspace_bytes, stream);
}

// ---- Allocation-free prefill ---------------------------------------------
//
// Split partials of talaria_sp_attn_prefill_noalloc go to this array instead
// of a caller workspace.  Every GPU the library runs on holds its own copy
// for the life of the process.  In host code `scratch` names a host-side
// stand-in, not device memory: its device address is looked up once per
// device (hipGetSymbolAddress, that device current) and only that address is
// passed to kernels.
constexpr size_t kScratchBytes = TALARIA_SP_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) char scratch[kScratchBytes];

namespace {

constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxScratchDevices] = {};

// Device address of `scratch` on the device that owns `stream`.
int scratch_for_stream(hipStream_t stream, void** out) {
    int dev = -1;
    hipError_t e = hipStreamGetDevice(stream, &dev);
    if (e != hipSuccess)
        return fail(TALARIA_SP_EHIP, "prefill_noalloc: hipStreamGetDevice: %s",
                    hipGetErrorString(e));
    if (dev < 0 || dev >= kMaxScratchDevices)
        return fail(TALARIA_SP_EUNSUPPORTED, "prefill_noalloc: device %d out of range", dev);
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (!g_scratch_ptr[dev]) {
        int cur = -1;
        e = hipGetDevice(&cur);
        if (e == hipSuccess && cur != dev)
            e = hipSetDevice(dev);
        void* ptr = nullptr;
        if (e == hipSuccess)
            e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (cur >= 0 && cur != dev) {
            const hipError_t e2 = hipSetDevice(cur);
            if (e == hipSuccess)
                e = e2;
        }
        if (e != hipSuccess || !ptr)
            return fail(TALARIA_SP_EHIP, "prefill_noalloc: scratch address on device %d: %s",
                        dev, hipGetErrorString(e));
        g_scratch_ptr[dev] = ptr;
    }
    *out = g_scratch_ptr[dev];
    return TALARIA_SP_OK;
}

}  // namespace

extern "C" size_t talaria_sp_attn_noalloc_scratch_bytes(void) { return kScratchBytes; }

extern "C" int talaria_sp_attn_prefill_noalloc(const talaria_sp_plan* plan, const void* q,
                                               const void* k_pool, const void* v_pool,
                                               const int32_t* block_tables, float sm_scale,
                                               void* out, float* lse, void* stream) {
    int status;
    const PlanData* p = checked_plan(plan, &status);
    if (!p)
        return status;
    if ((size_t)p->ws_bytes > kScratchBytes)
        return fail(TALARIA_SP_ENOSPACE, "prefill_noalloc: the plan needs %lld bytes of "
                    "scratch, the library holds %zu per GPU; use talaria_sp_attn_prefill with "
                    "a workspace", (long long)p->ws_bytes, kScratchBytes);
    if (p->num_items == 0)
        return TALARIA_SP_OK;
    if (!q || !k_pool || !v_pool || !block_tables || !out)
        return fail(TALARIA_SP_EINVAL, "prefill_noalloc: q, k_pool, v_pool, block_tables and "
                    "out must not be NULL");
    void* ws = nullptr;
    if (p->ws_bytes > 0) {
        status = scratch_for_stream(reinterpret_cast<hipStream_t>(stream), &ws);
        if (status != TALARIA_SP_OK)
            return status;
    }
    return prefill_impl(*p, q, k_pool, v_pool, block_tables, sm_scale, out, lse, ws,
                        kScratchBytes, stream);
}

extern "C" int talaria_sp_attn_calibrate_xcd(const talaria_sp_plan* plan, const void* q,
                                             const void* k_pool, const void* v_pool,
                                             const int32_t* block_tables, void* out,
                                             void* workspace, size_t workspace_bytes,
                                             void* stamps, size_t stamps_bytes, int32_t* order,
                                             void* stream) {
    int status;
    const PlanData* p = checked_plan(plan, &status);
    if (!p)
        return status;
    const int32_t n = p->num_items;
    if (n < kXcds)
        return fail(TALARIA_SP_EINVAL, "calibrate_xcd: the plan has %d work items; at least "
                    "%d (one per XCD) are needed", n, kXcds);
    if (!stamps || stamps_bytes < (size_t)n * 32)
        return fail(TALARIA_SP_ENOSPACE, "calibrate_xcd: stamps needs %lld bytes",
                    (long long)n * 32);
    PlanData c = *p;
    c.wg_mapped = 0;
    c.stamps = reinterpret_cast<uint64_t>(stamps);
    status = prefill_impl(c, q, k_pool, v_pool, block_tables, 0.f, out, nullptr, workspace,
                          workspace_bytes, stream);
    if (status != TALARIA_SP_OK)
        return status;
    hipStream_t st = reinterpret_cast<hipStream_t>(stream);
    std::vector<uint64_t> rec((size_t)n * 4);
    hipError_t e = hipStreamSynchronize(st);
    if (e == hipSuccess)
        e = hipMemcpy(rec.data(), stamps, rec.size() * sizeof(uint64_t), hipMemcpyDeviceToHost);
    if (e != hipSuccess)
        return fail(TALARIA_SP_EHIP, "calibrate_xcd: %s", hipGetErrorString(e));
    // Mean main-loop time per key tile on each XCD (the real-time counter
    // ticks at 100 MHz), then the XCDs from fastest to slowest.
    double ns[kXcds] = {}, cnt[kXcds] = {};
    for (int32_t i = 0; i < n; ++i) {
        const uint64_t x = rec[4 * i] & 15, tiles = rec[4 * i + 1];
        if (x < (uint64_t)kXcds && tiles > 0 && rec[4 * i + 3] >= rec[4 * i + 2]) {
            ns[x] += 10.0 * (double)(rec[4 * i + 3] - rec[4 * i + 2]) / (double)tiles;
            cnt[x] += 1.0;
        }
    }
    int32_t ord[kXcds];
    for (int x = 0; x < kXcds; ++x) {
        if (cnt[x] == 0)
            return fail(TALARIA_SP_EINVAL, "calibrate_xcd: no timed work item ran on XCD %d", x);
        ns[x] /= cnt[x];
        ord[x] = x;
    }
    std::stable_sort(ord, ord + kXcds, [&](int32_t a, int32_t b) { return ns[a] < ns[b]; });
    status = talaria_sp_set_xcd_order(ord);
    if (status == TALARIA_SP_OK && order)
        memcpy(order, ord, sizeof ord);
    return status;
}
