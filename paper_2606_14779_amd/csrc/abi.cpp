// extern "C" entry points: argument checks, error codes and the thread-local
// error message.  No C++ exception crosses this boundary.

#include <new>
#include <string>
#include <vector>

#include "internal.hpp"

namespace kvp {
Pool *pool_create(const kvp_region_desc *, const uint64_t *, uint32_t, const kvp_kv_spec *, int,
                  const char *const *);
void pool_destroy(Pool *);
void pool_place(Pool &, uint64_t, uint32_t, kvp_loc *);
void pool_extend(Pool &, uint64_t, uint32_t, kvp_loc *);
void pool_lookup(Pool &, uint64_t, uint32_t, kvp_loc *);
void pool_lookup_vector(Pool &, uint64_t, uint32_t, std::vector<kvp_loc> &);
void pool_release(Pool &, uint64_t);
void pool_transfer(Pool &, const kvp_loc *, uint32_t, const int32_t *, uint32_t, uint32_t, uint32_t,
                   void *const *, void *const *, void *, bool, bool = false);
void pool_region_info(const Pool &, uint32_t, kvp_region_info *);
void pool_region_read(Pool &, uint32_t, uint64_t, uint64_t, void *);
void pool_set_launch(Pool &, uint32_t, uint32_t, uint32_t, uint32_t);
void pool_set_copy_ring(Pool &, uint64_t);
void pool_set_file_ring(Pool &, uint64_t);
void pool_set_timing(Pool &, int);
void pool_last_timing(Pool &, kvp_timing *);
void pool_timing_summary(Pool &, kvp_timing_summary *);
void pool_measure(Pool &, uint64_t, uint32_t, uint64_t *);
void pool_set_bandwidths(Pool &, const uint64_t *);
}  // namespace kvp

struct kvp_pool {
    kvp::Pool *impl;
};

namespace {

thread_local std::string g_last_error;
thread_local const char *g_fixed_error = nullptr;   // set when the message itself could not be stored

// Record the message of a failure without throwing: a message that cannot be
// copied (out of host memory) is replaced by a fixed one; the code returned is
// the failure's own either way.
void set_error(const char *msg) noexcept
{
    try {
        g_last_error = msg;
        g_fixed_error = nullptr;
    } catch (...) {
        g_last_error.clear();
        g_fixed_error = "out of host memory (the error message could not be stored)";
    }
}

template <class F>
int guarded(F &&f) noexcept
{
    try {
        f();
        g_last_error.clear();
        g_fixed_error = nullptr;
        return KVP_OK;
    } catch (const kvp::Error &e) {
        set_error(e.msg.c_str());
        return e.code;
    } catch (const std::bad_alloc &) {
        set_error("host allocation failed");
        return KVP_ERR_NOMEM;
    } catch (const std::exception &e) {
        set_error(e.what());
        return KVP_ERR_INVALID;
    } catch (...) {
        set_error("unknown error");
        return KVP_ERR_INVALID;
    }
}

kvp::Pool &impl(kvp_pool *p)
{
    if (!p || !p->impl) kvp::fail(KVP_ERR_INVALID, "null pool");
    return *p->impl;
}

}  // namespace

extern "C" {

int kv_pool_create(const kvp_region_desc *regions, const uint64_t *bandwidths, uint32_t n_regions,
                   const kvp_kv_spec *spec, int hip_device, kvp_pool **out)
{
    return guarded([&] {
        if (!out) kvp::fail(KVP_ERR_INVALID, "out is null");
        *out = nullptr;
        kvp::Pool *p = kvp::pool_create(regions, bandwidths, n_regions, spec, hip_device, nullptr);
        try {
            *out = new kvp_pool{p};
        } catch (...) {
            kvp::pool_destroy(p);
            throw;
        }
    });
}

int kv_pool_create_files(const kvp_region_desc *regions, const uint64_t *bandwidths, uint32_t n_regions,
                         const kvp_kv_spec *spec, int hip_device, const char *const *paths, kvp_pool **out)
{
    return guarded([&] {
        if (!out) kvp::fail(KVP_ERR_INVALID, "out is null");
        *out = nullptr;
        kvp::Pool *p = kvp::pool_create(regions, bandwidths, n_regions, spec, hip_device, paths);
        try {
            *out = new kvp_pool{p};
        } catch (...) {
            kvp::pool_destroy(p);
            throw;
        }
    });
}

int kv_pool_place(kvp_pool *pool, uint64_t request_id, uint32_t n_blocks, kvp_loc *map_out)
{
    return guarded([&] { kvp::pool_place(impl(pool), request_id, n_blocks, map_out); });
}

int kv_pool_extend(kvp_pool *pool, uint64_t request_id, uint32_t n_new, kvp_loc *map_out)
{
    return guarded([&] { kvp::pool_extend(impl(pool), request_id, n_new, map_out); });
}

int kv_pool_lookup(kvp_pool *pool, uint64_t request_id, uint32_t n_blocks, kvp_loc *map_out)
{
    return guarded([&] { kvp::pool_lookup(impl(pool), request_id, n_blocks, map_out); });
}

int kv_pool_store(kvp_pool *pool, const kvp_loc *map, uint32_t n_blocks, const int32_t *src_block_table,
                  uint32_t src_num_slots, void *const *k_layers, void *const *v_layers, void *stream)
{
    return guarded([&] {
        kvp::Pool &p = impl(pool);
        kvp::pool_transfer(p, map, n_blocks, src_block_table, src_num_slots, 0, p.spec.num_layers, k_layers,
                           v_layers, stream, false);
    });
}

int kv_pool_store_layers(kvp_pool *pool, const kvp_loc *map, uint32_t n_blocks, const int32_t *src_block_table,
                         uint32_t src_num_slots, uint32_t layer_begin, uint32_t layer_end, void *const *k_layers,
                         void *const *v_layers, void *stream)
{
    return guarded([&] {
        kvp::pool_transfer(impl(pool), map, n_blocks, src_block_table, src_num_slots, layer_begin, layer_end,
                           k_layers, v_layers, stream, false);
    });
}

int kv_pool_retrieve(kvp_pool *pool, const kvp_loc *map, uint32_t n_blocks, const int32_t *dst_block_table,
                     uint32_t dst_num_slots, void *const *k_layers, void *const *v_layers, void *stream)
{
    return guarded([&] {
        kvp::Pool &p = impl(pool);
        kvp::pool_transfer(p, map, n_blocks, dst_block_table, dst_num_slots, 0, p.spec.num_layers, k_layers,
                           v_layers, stream, true);
    });
}

int kv_pool_retrieve_noalloc(kvp_pool *pool, const kvp_loc *map, uint32_t n_blocks, const int32_t *dst_block_table,
                             uint32_t dst_num_slots, void *const *k_layers, void *const *v_layers, void *stream)
{
    return guarded([&] {
        kvp::Pool &p = impl(pool);
        kvp::pool_transfer(p, map, n_blocks, dst_block_table, dst_num_slots, 0, p.spec.num_layers, k_layers,
                           v_layers, stream, true, true);
    });
}

int kv_pool_retrieve_layers(kvp_pool *pool, const kvp_loc *map, uint32_t n_blocks, const int32_t *dst_block_table,
                            uint32_t dst_num_slots, uint32_t layer_begin, uint32_t layer_end,
                            void *const *k_layers, void *const *v_layers, void *stream)
{
    return guarded([&] {
        kvp::pool_transfer(impl(pool), map, n_blocks, dst_block_table, dst_num_slots, layer_begin, layer_end,
                           k_layers, v_layers, stream, true);
    });
}

int kv_pool_retrieve_request(kvp_pool *pool, uint64_t request_id, uint32_t n_blocks,
                             const int32_t *dst_block_table, uint32_t dst_num_slots, void *const *k_layers,
                             void *const *v_layers, void *stream)
{
    return guarded([&] {
        kvp::Pool &p = impl(pool);
        std::vector<kvp_loc> map;
        kvp::pool_lookup_vector(p, request_id, n_blocks, map);
        kvp::pool_transfer(p, map.data(), n_blocks, dst_block_table, dst_num_slots, 0, p.spec.num_layers,
                           k_layers, v_layers, stream, true);
    });
}

int kv_pool_release(kvp_pool *pool, uint64_t request_id)
{
    return guarded([&] { kvp::pool_release(impl(pool), request_id); });
}

void kv_pool_destroy(kvp_pool *pool)
{
    if (!pool) return;
    (void)guarded([&] { kvp::pool_destroy(pool->impl); });
    delete pool;
}

const char *kv_pool_last_error(void) { return g_fixed_error ? g_fixed_error : g_last_error.c_str(); }

int kv_pool_region_info(const kvp_pool *pool, uint32_t region, kvp_region_info *out)
{
    return guarded([&] {
        if (!pool || !pool->impl) kvp::fail(KVP_ERR_INVALID, "null pool");
        kvp::pool_region_info(*pool->impl, region, out);
    });
}

int kv_pool_region_read(kvp_pool *pool, uint32_t region, uint64_t offset, uint64_t bytes, void *host_dst)
{
    return guarded([&] { kvp::pool_region_read(impl(pool), region, offset, bytes, host_dst); });
}

int kv_pool_counts(const uint64_t *bandwidths, uint32_t n_regions, uint64_t n, uint64_t *counts_out)
{
    return guarded([&] {
        if (!bandwidths || !counts_out) kvp::fail(KVP_ERR_INVALID, "null argument");
        kvp::target_counts(bandwidths, n_regions, n, counts_out);
    });
}

int kv_pool_measure_bandwidth(kvp_pool *pool, uint64_t probe_bytes, uint32_t flags, uint64_t *mbps_out)
{
    return guarded([&] { kvp::pool_measure(impl(pool), probe_bytes, flags, mbps_out); });
}

int kv_pool_set_bandwidths(kvp_pool *pool, const uint64_t *bandwidths)
{
    return guarded([&] { kvp::pool_set_bandwidths(impl(pool), bandwidths); });
}

int kv_pool_set_launch(kvp_pool *pool, uint32_t cls, uint32_t op, uint32_t grid, uint32_t flags)
{
    return guarded([&] { kvp::pool_set_launch(impl(pool), cls, op, grid, flags); });
}

int kv_pool_set_copy_ring(kvp_pool *pool, uint64_t slot_bytes)
{
    return guarded([&] { kvp::pool_set_copy_ring(impl(pool), slot_bytes); });
}

int kv_pool_set_file_ring(kvp_pool *pool, uint64_t slot_bytes)
{
    return guarded([&] { kvp::pool_set_file_ring(impl(pool), slot_bytes); });
}

int kv_pool_set_timing(kvp_pool *pool, int enable)
{
    return guarded([&] { kvp::pool_set_timing(impl(pool), enable); });
}

int kv_pool_last_timing(kvp_pool *pool, kvp_timing *out)
{
    return guarded([&] { kvp::pool_last_timing(impl(pool), out); });
}

int kv_pool_timing_summary(kvp_pool *pool, kvp_timing_summary *out)
{
    return guarded([&] { kvp::pool_timing_summary(impl(pool), out); });
}

int kv_probe_copy_kernel(void *dst, const void *src, uint64_t bytes, uint32_t grid, uint32_t flags, void *stream)
{
    return guarded([&] {
        if (!dst || !src) kvp::fail(KVP_ERR_INVALID, "null pointer");
        if ((reinterpret_cast<uintptr_t>(dst) | reinterpret_cast<uintptr_t>(src) | bytes) & 15)
            kvp::fail(KVP_ERR_INVALID, "pointers and size must be multiples of 16");
        if (flags & ~(KVP_LAUNCH_NT_LOAD | KVP_LAUNCH_NT_STORE | KVP_LAUNCH_SPLIT2))
            kvp::fail(KVP_ERR_INVALID, "unknown flags");
        if (grid > (1u << 20)) kvp::fail(KVP_ERR_INVALID, "grid too large");
        kvp::check_hip(kvp::launch_probe_copy(dst, src, bytes, grid, flags, static_cast<hipStream_t>(stream)),
                       "probe kernel launch");
    });
}

int kv_probe_memcpy(void *dst, const void *src, uint64_t bytes, void *stream)
{
    return guarded([&] {
        kvp::check_hip(hipMemcpyAsync(dst, src, bytes, hipMemcpyDefault, static_cast<hipStream_t>(stream)),
                       "hipMemcpyAsync");
    });
}

}  // extern "C"
