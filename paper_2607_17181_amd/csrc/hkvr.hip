// HKVR page transfer: the host KV registry keeps a session's prefix in pinned
// host memory in a page-first layout and restores it into newly allocated
// device pages of the layer-first device cache (paper Section 4.3, restore
// of the agreed prefix before the tail is recomputed; Appendix C, the
// layer-first and page-first views of the same pages).  Checkpointing is the
// reverse copy, taken when a turn ends.
//
//   device (layer-first): k_cache [L][num_pages][Hkv][ps][d]
//                         v_cache [L][num_pages][Hkv][d][ps]
//   host   (page-first):  slab [n][L][2][Hkv * ps * d]   (K block, V block)
//
// A slab block holds one device page of one layer in the device page's own
// element order, so moving it is a straight 16-byte copy: no element is
// reordered, only whole page blocks are placed.  Work unit: one workgroup per
// (slab page, layer); 256 threads copy the K and V blocks with 16-byte
// non-temporal loads and stores, the host side read or written directly
// through its device-visible pinned address.
#include <hip/hip_runtime.h>

#include "common.h"

namespace tsp {

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// to_device: slab -> cache (restore); otherwise cache -> slab (checkpoint).
template <bool to_device>
__global__ __launch_bounds__(256) void hkvr_copy_kernel(const int32_t* __restrict__ page_ids,
                                                        int32_t num_pages, int32_t num_layers,
                                                        int64_t block_chunks,
                                                        u32x4* __restrict__ k_cache,
                                                        u32x4* __restrict__ v_cache,
                                                        u32x4* __restrict__ slab) {
    const int p = blockIdx.x;
    const int l = blockIdx.y;
    const int32_t page = page_ids[p];
    if (page < 0 || page >= num_pages)
        return;  // not a page of this cache: nothing is moved
    const int64_t dev = ((int64_t)l * num_pages + page) * block_chunks;
    u32x4* sk = slab + ((int64_t)p * num_layers + l) * 2 * block_chunks;
    u32x4* sv = sk + block_chunks;
    for (int64_t c = threadIdx.x; c < block_chunks; c += 256) {
        if (to_device) {
            const u32x4 k = __builtin_nontemporal_load(sk + c);
            const u32x4 v = __builtin_nontemporal_load(sv + c);
            __builtin_nontemporal_store(k, k_cache + dev + c);
            __builtin_nontemporal_store(v, v_cache + dev + c);
        } else {
            const u32x4 k = __builtin_nontemporal_load(k_cache + dev + c);
            const u32x4 v = __builtin_nontemporal_load(v_cache + dev + c);
            __builtin_nontemporal_store(k, sk + c);
            __builtin_nontemporal_store(v, sv + c);
        }
    }
}

int check_cache(const talaria_kv_cache* cache, int32_t num_slab_pages, const char* what) {
    if (!cache)
        return fail(TALARIA_SP_EINVAL, "%s: cache is NULL", what);
    const talaria_kv_cache& c = *cache;
    if (c.num_layers <= 0 || c.num_kv_heads <= 0 || c.num_pages <= 0 || num_slab_pages < 0)
        return fail(TALARIA_SP_EINVAL, "%s: layers, KV heads and pages must be positive", what);
    if (c.num_layers > 65535)
        return fail(TALARIA_SP_EUNSUPPORTED, "%s: at most 65535 layers", what);
    if (c.head_dim != 64 && c.head_dim != 128)
        return fail(TALARIA_SP_EUNSUPPORTED, "%s: head_dim %d not supported", what, c.head_dim);
    if (c.page_size < 8 || c.page_size > 256 || (c.page_size & (c.page_size - 1)))
        return fail(TALARIA_SP_EUNSUPPORTED, "%s: page_size %d not supported", what, c.page_size);
    return TALARIA_SP_OK;
}

template <bool to_device>
int launch_copy(const talaria_kv_cache* cache, int32_t n, const int32_t* page_ids, void* k_cache,
                void* v_cache, void* slab, void* stream, const char* what) {
    int status = check_cache(cache, n, what);
    if (status != TALARIA_SP_OK)
        return status;
    if (n == 0)
        return TALARIA_SP_OK;
    if (!page_ids || !k_cache || !v_cache || !slab)
        return fail(TALARIA_SP_EINVAL, "%s: pointers must not be NULL", what);
    if (!aligned16(k_cache) || !aligned16(v_cache) || !aligned16(slab) ||
        ((uintptr_t)page_ids & 3u) != 0)
        return fail(TALARIA_SP_EINVAL, "%s: k_cache, v_cache and slab must be 16-byte aligned, "
                    "page_ids 4-byte aligned", what);
    const int64_t block_chunks =
        (int64_t)cache->num_kv_heads * cache->page_size * cache->head_dim * 2 / 16;
    hipLaunchKernelGGL(hkvr_copy_kernel<to_device>, dim3(n, cache->num_layers), dim3(256), 0,
                       reinterpret_cast<hipStream_t>(stream), page_ids, cache->num_pages,
                       cache->num_layers, block_chunks, static_cast<u32x4*>(k_cache),
                       static_cast<u32x4*>(v_cache), static_cast<u32x4*>(slab));
    return launch_status(what);
}

}  // namespace
}  // namespace tsp

using namespace tsp;

extern "C" int talaria_hkvr_restore(const talaria_kv_cache* cache, int32_t num_slab_pages,
                                    const void* slab, const int32_t* page_ids, void* k_cache,
                                    void* v_cache, void* stream) {
    return launch_copy<true>(cache, num_slab_pages, page_ids, k_cache, v_cache,
                             const_cast<void*>(slab), stream, "hkvr_restore");
}

extern "C" int talaria_hkvr_checkpoint(const talaria_kv_cache* cache, int32_t num_slab_pages,
                                       const void* k_cache, const void* v_cache,
                                       const int32_t* page_ids, void* slab, void* stream) {
    return launch_copy<false>(cache, num_slab_pages, page_ids, const_cast<void*>(k_cache),
                              const_cast<void*>(v_cache), slab, stream, "hkvr_checkpoint");
}
