// D2D-staged switching: the next model's weights are pre-staged in fixed-size
// chunks in the free high-address tail of the KV region while the current
// model serves; at the switch, clean staged chunks are copied device to
// device and dirty or missing ones are reloaded from host (paper Section
// 4.4).  A staged chunk turns dirty when a KV allocation takes pages that
// overlap its staging range -- those bytes may now hold KV rows, so the
// guard must not copy them.
//
// Two kernels:
//   mark_dirty  one thread per chunk: is any page in use whose bytes overlap
//               the chunk's staging range?  Sets the chunk's bit.
//   gather      kSplits workgroups per chunk stream its bytes with 16-byte
//               non-temporal accesses, from the staging copy when the chunk
//               is staged and clean, else from the pinned host copy.
#include <hip/hip_runtime.h>

#include "common.h"

namespace tsp {

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kSplits = 8;     // workgroups per chunk in the gather
constexpr int kUnroll = 4;     // 16-byte chunks in flight per thread

__device__ __forceinline__ bool bit(const uint32_t* bits, int64_t i) {
    return (bits[i >> 5] >> (i & 31)) & 1u;
}

// A chunk's destination (and its host copy, same offsets) must lie in the
// weight region; its staged copy must lie in the staging region to be used.
__device__ __forceinline__ bool weight_range_ok(const talaria_stage_chunk& c, int64_t weight_bytes) {
    return c.bytes > 0 && ((c.bytes | c.weight_offset) & 15) == 0 && c.weight_offset >= 0 &&
           c.weight_offset + c.bytes <= weight_bytes;
}
__device__ __forceinline__ bool stage_range_ok(const talaria_stage_chunk& c, int64_t stage_bytes) {
    return (c.stage_offset & 15) == 0 && c.stage_offset >= 0 &&
           c.stage_offset + c.bytes <= stage_bytes;
}

__global__ __launch_bounds__(256) void mark_dirty_kernel(const talaria_stage_chunk* __restrict__ chunks,
                                                         int32_t num_chunks,
                                                         const uint32_t* __restrict__ used_pages,
                                                         int64_t num_pages, int64_t page_bytes,
                                                         uint32_t* __restrict__ dirty) {
    const int i = blockIdx.x * 256 + threadIdx.x;
    bool d = false;
    if (i < num_chunks) {
        const talaria_stage_chunk c = chunks[i];
        if (c.bytes > 0 && c.stage_offset >= 0) {
            const int64_t first = c.stage_offset / page_bytes;
            const int64_t last = min((c.stage_offset + c.bytes - 1) / page_bytes, num_pages - 1);
            for (int64_t p = first; p <= last && !d; ++p) {
                // whole 32-page words at a time where possible
                if ((p & 31) == 0 && p + 31 <= last) {
                    d = used_pages[p >> 5] != 0;
                    p += 31;
                } else {
                    d = bit(used_pages, p);
                }
            }
        }
    }
    // One word of the bitmap per 32 chunks: combine the wave's bits.
    const uint64_t ballot = __ballot(d);
    const int lane = threadIdx.x & 63;
    if (lane == 0 || lane == 32) {
        const int w = (blockIdx.x * 256 + (threadIdx.x & ~31)) >> 5;
        if (w * 32 < num_chunks)
            dirty[w] = (uint32_t)(ballot >> lane);
    }
}

__global__ __launch_bounds__(256) void stage_gather_kernel(const talaria_stage_chunk* __restrict__ chunks,
                                                           const uint32_t* __restrict__ staged,
                                                           const uint32_t* __restrict__ dirty,
                                                           const u32x4* __restrict__ staging,
                                                           int64_t stage_bytes,
                                                           const u32x4* __restrict__ host,
                                                           u32x4* __restrict__ weights,
                                                           int64_t weight_bytes) {
    const talaria_stage_chunk c = chunks[blockIdx.x];
    if (!weight_range_ok(c, weight_bytes))
        return;  // malformed entry: nothing is copied
    const bool from_stage = bit(staged, blockIdx.x) && !bit(dirty, blockIdx.x) &&
                            stage_range_ok(c, stage_bytes);
    const u32x4* src = from_stage ? staging + c.stage_offset / 16 : host + c.weight_offset / 16;
    u32x4* dst = weights + c.weight_offset / 16;
    const int64_t n = c.bytes / 16;
    const int64_t per = (n + kSplits - 1) / kSplits;
    const int64_t lo = blockIdx.y * per, hi = min(n, lo + per);
    for (int64_t i = lo + threadIdx.x; i < hi; i += 256 * kUnroll) {
        u32x4 v[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u)
            if (i + u * 256 < hi)
                v[u] = __builtin_nontemporal_load(src + i + u * 256);
#pragma unroll
        for (int u = 0; u < kUnroll; ++u)
            if (i + u * 256 < hi)
                __builtin_nontemporal_store(v[u], dst + i + u * 256);
    }
}

}  // namespace
}  // namespace tsp

using namespace tsp;

extern "C" int talaria_stage_mark_dirty(const talaria_stage_chunk* chunks, int32_t num_chunks,
                                        const uint32_t* used_pages, int64_t num_pages,
                                        int64_t page_bytes, uint32_t* dirty, void* stream) {
    if (num_chunks < 0 || num_pages < 0 || page_bytes <= 0)
        return fail(TALARIA_SP_EINVAL, "stage_mark_dirty: negative count or page size");
    if (num_chunks == 0)
        return TALARIA_SP_OK;
    if (!chunks || !dirty || (num_pages > 0 && !used_pages))
        return fail(TALARIA_SP_EINVAL, "stage_mark_dirty: pointers must not be NULL");
    if (num_pages == 0)
        return fail(TALARIA_SP_EINVAL, "stage_mark_dirty: num_pages must be positive");
    hipLaunchKernelGGL(mark_dirty_kernel, dim3((num_chunks + 255) / 256), dim3(256), 0,
                       reinterpret_cast<hipStream_t>(stream), chunks, num_chunks, used_pages,
                       num_pages, page_bytes, dirty);
    return launch_status("stage_mark_dirty");
}

extern "C" int talaria_stage_gather(const talaria_stage_chunk* chunks, int32_t num_chunks,
                                    const uint32_t* staged, const uint32_t* dirty,
                                    const void* staging, int64_t staging_bytes,
                                    const void* host_weights, void* weights,
                                    int64_t weight_bytes, void* stream) {
    if (num_chunks < 0 || staging_bytes < 0 || weight_bytes < 0)
        return fail(TALARIA_SP_EINVAL, "stage_gather: negative count or size");
    if (num_chunks == 0)
        return TALARIA_SP_OK;
    if (!chunks || !staged || !dirty || !host_weights || !weights ||
        (staging_bytes > 0 && !staging))
        return fail(TALARIA_SP_EINVAL, "stage_gather: pointers must not be NULL");
    if (((uintptr_t)staging | (uintptr_t)host_weights | (uintptr_t)weights) & 15)
        return fail(TALARIA_SP_EINVAL, "stage_gather: regions must be 16-byte aligned");
    hipLaunchKernelGGL(stage_gather_kernel, dim3(num_chunks, kSplits), dim3(256), 0,
                       reinterpret_cast<hipStream_t>(stream), chunks, staged, dirty,
                       static_cast<const u32x4*>(staging), staging_bytes,
                       static_cast<const u32x4*>(host_weights), static_cast<u32x4*>(weights),
                       weight_bytes);
    return launch_status("stage_gather");
}
