// A plain C++ client of libkvpool.so: no Python, no PyTorch.  Creates a pool
// of one host and one HBM staging region, places a request, stores a source
// cache filled with a per-element tag, retrieves it into a destination cache
// under a permuted block table, and checks every element on the host.  Then
// it retrieves again through the copy-engine transport with one-block ring
// slots, in two layer ranges, and checks again.  Last, a second pool made by
// kv_pool_create_files with a host and a file region (a file created in a
// temporary directory) stores and retrieves the request through the storage
// tier and is checked the same way; a resize of its file ring that cannot
// allocate (forced below) is reported as NOMEM, file transfers are refused
// until a later resize succeeds, and then work again; destroying the pool
// removes the file.
// With the argument "exit-open" it instead leaves the pool open with a
// retrieve still enqueued and returns from main: the process must end
// cleanly (the library registers nothing that runs at exit).
// Built by the package build step; run by tests/test_abi_client.py (GPU).
#include <dlfcn.h>
#include <hip/hip_runtime.h>
#include <sys/stat.h>
#include <unistd.h>

#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <string>
#include <vector>

#include "kvpool.h"

#define TRY(x)                                                                               \
    do {                                                                                     \
        int rc_ = (x);                                                                       \
        if (rc_ != KVP_OK) {                                                                 \
            std::fprintf(stderr, "%s failed: %d (%s)\n", #x, rc_, kv_pool_last_error());     \
            return 1;                                                                        \
        }                                                                                    \
    } while (0)
#define HIPTRY(x)                                                                            \
    do {                                                                                     \
        if ((x) != hipSuccess) {                                                             \
            std::fprintf(stderr, "%s failed\n", #x);                                         \
            return 1;                                                                        \
        }                                                                                    \
    } while (0)

// Pinned host allocations larger than this fail (0: none do).  This
// executable's hipHostMalloc takes the library's references to the runtime's
// (the build exports it), so a ring resize can be made to fail on any machine.
static size_t g_fail_pinned_above = 0;

extern "C" hipError_t hipHostMalloc(void **ptr, size_t size, unsigned int flags)
{
    using Fn = hipError_t (*)(void **, size_t, unsigned int);
    static const Fn real = reinterpret_cast<Fn>(dlvsym(RTLD_NEXT, "hipHostMalloc", "hip_4.2"));
    if (g_fail_pinned_above && size > g_fail_pinned_above) return hipErrorOutOfMemory;
    return real ? real(ptr, size, flags) : hipErrorNotInitialized;
}

int main(int argc, char **argv)
{
    const bool exit_open = argc > 1 && std::strcmp(argv[1], "exit-open") == 0;
    const uint32_t L = 4, H = 2, bs = 16, D = 64, n = 37, slots = 45;
    const uint64_t chunk_elems = uint64_t(H) * bs * D;                 // bf16 words per (layer, K/V) chunk
    const uint64_t layer_bytes = uint64_t(slots) * chunk_elems * 2;
    kvp_kv_spec spec = {L, H, D, bs, 2, 0};
    const uint64_t block_bytes = 2ull * L * chunk_elems * 2;
    kvp_region_desc regions[2] = {{KVP_REGION_HOST, -1, 64 * block_bytes, KVP_HOST_DEFAULT, 0},
                                  {KVP_REGION_STAGING, -1, 64 * block_bytes, 0, 0}};
    uint64_t bw[2] = {3, 1};
    kvp_pool *pool = nullptr;
    TRY(kv_pool_create(regions, bw, 2, &spec, 0, &pool));

    // engine caches: one buffer per layer and K/V
    std::vector<void *> src(2 * L), dst(2 * L);
    std::vector<uint16_t> host(slots * chunk_elems);
    for (uint32_t i = 0; i < 2 * L; ++i) {
        HIPTRY(hipMalloc(&src[i], layer_bytes));
        HIPTRY(hipMalloc(&dst[i], layer_bytes));
        for (uint64_t e = 0; e < host.size(); ++e) host[e] = uint16_t(e * 2654435761u + i * 40503u);
        HIPTRY(hipMemcpy(src[i], host.data(), layer_bytes, hipMemcpyHostToDevice));
        HIPTRY(hipMemset(dst[i], 0xA5, layer_bytes));
    }
    std::vector<void *> k_src(L), v_src(L), k_dst(L), v_dst(L);
    for (uint32_t l = 0; l < L; ++l) {
        k_src[l] = src[2 * l];
        v_src[l] = src[2 * l + 1];
        k_dst[l] = dst[2 * l];
        v_dst[l] = dst[2 * l + 1];
    }

    std::vector<kvp_loc> map(n);
    TRY(kv_pool_place(pool, 42, n, map.data()));
    std::vector<int32_t> src_table(n), dst_table(n);
    for (uint32_t b = 0; b < n; ++b) {
        src_table[b] = int32_t((b * 7 + 3) % slots);      // 7 is invertible mod 45: distinct slots
        dst_table[b] = int32_t((b * 11 + 5) % slots);
    }
    hipStream_t stream;
    HIPTRY(hipStreamCreate(&stream));
    TRY(kv_pool_store(pool, map.data(), n, src_table.data(), slots, k_src.data(), v_src.data(), stream));
    TRY(kv_pool_retrieve_request(pool, 42, n, dst_table.data(), slots, k_dst.data(), v_dst.data(), stream));
    if (exit_open) {   // pool, streams and buffers left alive, work possibly still running
        std::printf("exiting with the pool open\n");
        return 0;
    }
    HIPTRY(hipStreamSynchronize(stream));

    std::vector<uint16_t> got(slots * chunk_elems), want(slots * chunk_elems);
    std::vector<char> used(slots, 0);
    for (uint32_t b = 0; b < n; ++b) used[dst_table[b]] = 1;
    uint64_t bad = 0;
    auto check = [&]() -> int {
        for (uint32_t i = 0; i < 2 * L; ++i) {
            HIPTRY(hipMemcpy(got.data(), dst[i], layer_bytes, hipMemcpyDeviceToHost));
            for (uint64_t e = 0; e < want.size(); ++e) want[e] = uint16_t(e * 2654435761u + i * 40503u);
            for (uint32_t b = 0; b < n; ++b)
                bad += std::memcmp(&got[dst_table[b] * chunk_elems], &want[src_table[b] * chunk_elems],
                                   chunk_elems * 2) != 0;
            for (uint32_t sl = 0; sl < slots; ++sl)
                if (!used[sl])
                    for (uint64_t e = 0; e < chunk_elems; ++e) bad += got[sl * chunk_elems + e] != 0xA5A5;
        }
        return 0;
    };
    if (check()) return 1;   // store and retrieve fit the small-call launch (work list in the kernel arguments)

    // the same request through the upload path: work list uploaded, one launch per region class
    for (uint32_t i = 0; i < 2 * L; ++i) HIPTRY(hipMemset(dst[i], 0xA5, layer_bytes));
    TRY(kv_pool_set_launch(pool, KVP_CLASS_HOST, KVP_OP_RETRIEVE, 0, KVP_LAUNCH_UPLOAD));
    TRY(kv_pool_retrieve(pool, map.data(), n, dst_table.data(), slots, k_dst.data(), v_dst.data(), stream));
    HIPTRY(hipStreamSynchronize(stream));
    if (check()) return 1;

    // the same request by the allocation-free entry point (work list in the static scratch)
    for (uint32_t i = 0; i < 2 * L; ++i) HIPTRY(hipMemset(dst[i], 0xA5, layer_bytes));
    TRY(kv_pool_retrieve_noalloc(pool, map.data(), n, dst_table.data(), slots, k_dst.data(), v_dst.data(), stream));
    HIPTRY(hipStreamSynchronize(stream));
    if (check()) return 1;

    // the same request through the copy engines: ring slots of one block, two layer ranges
    for (uint32_t i = 0; i < 2 * L; ++i) HIPTRY(hipMemset(dst[i], 0xA5, layer_bytes));
    TRY(kv_pool_set_copy_ring(pool, 64 << 10));
    TRY(kv_pool_set_launch(pool, KVP_CLASS_HOST, KVP_OP_RETRIEVE, 0, KVP_LAUNCH_SDMA));
    TRY(kv_pool_retrieve_layers(pool, map.data(), n, dst_table.data(), slots, 0, 1, k_dst.data(), v_dst.data(), stream));
    TRY(kv_pool_retrieve_layers(pool, map.data(), n, dst_table.data(), slots, 1, L, k_dst.data(), v_dst.data(), stream));
    HIPTRY(hipStreamSynchronize(stream));
    if (check()) return 1;
    // store through the copy engines too (ring to host region), after clearing the host region's copy,
    // then retrieve by the kernel path: the pool bytes the engines wrote reach the cache unchanged
    TRY(kv_pool_set_launch(pool, KVP_CLASS_HOST, KVP_OP_STORE, 0, KVP_LAUNCH_SDMA));
    kvp_region_info info;
    TRY(kv_pool_region_info(pool, 0, &info));
    std::memset(info.host_ptr, 0, info.capacity_bytes);
    TRY(kv_pool_store(pool, map.data(), n, src_table.data(), slots, k_src.data(), v_src.data(), stream));
    for (uint32_t i = 0; i < 2 * L; ++i) HIPTRY(hipMemset(dst[i], 0xA5, layer_bytes));
    TRY(kv_pool_set_launch(pool, KVP_CLASS_HOST, KVP_OP_RETRIEVE, 0, KVP_LAUNCH_UPLOAD));
    TRY(kv_pool_retrieve(pool, map.data(), n, dst_table.data(), slots, k_dst.data(), v_dst.data(), stream));
    HIPTRY(hipStreamSynchronize(stream));
    if (check()) return 1;
    TRY(kv_pool_release(pool, 42));

    // a request extended by two more offload sets: lookup returns the three maps in order
    std::vector<kvp_loc> a(5), b(1), c(3), all(9);
    TRY(kv_pool_place(pool, 77, 5, a.data()));
    TRY(kv_pool_extend(pool, 77, 1, b.data()));
    TRY(kv_pool_extend(pool, 77, 3, c.data()));
    TRY(kv_pool_lookup(pool, 77, 9, all.data()));
    std::vector<kvp_loc> cat(a);
    cat.insert(cat.end(), b.begin(), b.end());
    cat.insert(cat.end(), c.begin(), c.end());
    for (uint32_t i = 0; i < 9; ++i)
        bad += all[i].region != cat[i].region || all[i].gen != cat[i].gen || all[i].offset != cat[i].offset;
    if (kv_pool_extend(pool, 78, 1, b.data()) != KVP_ERR_NOTFOUND) ++bad;
    TRY(kv_pool_release(pool, 77));
    kv_pool_destroy(pool);

    // the storage tier: a host region and a file region, weights 1:2, ring slots of four blocks
    char dir_tmpl[] = "/tmp/kvpool-abi-XXXXXX";
    if (!::mkdtemp(dir_tmpl)) {
        std::fprintf(stderr, "mkdtemp failed\n");
        return 1;
    }
    const std::string file_path = std::string(dir_tmpl) + "/region1.bin";
    kvp_region_desc fregions[2] = {{KVP_REGION_HOST, -1, 64 * block_bytes, KVP_HOST_DEFAULT, 0},
                                   {KVP_REGION_FILE, -1, 64 * block_bytes, 0, 0}};
    const char *paths[2] = {nullptr, file_path.c_str()};
    uint64_t fbw[2] = {1, 2};
    kvp_pool *fpool = nullptr;
    TRY(kv_pool_create_files(fregions, fbw, 2, &spec, 0, paths, &fpool));
    TRY(kv_pool_set_file_ring(fpool, 4 * block_bytes));
    TRY(kv_pool_place(fpool, 5, n, map.data()));
    uint32_t on_file = 0;
    for (uint32_t b = 0; b < n; ++b) on_file += map[b].region == 1;
    for (uint32_t i = 0; i < 2 * L; ++i) HIPTRY(hipMemset(dst[i], 0xA5, layer_bytes));
    TRY(kv_pool_store(fpool, map.data(), n, src_table.data(), slots, k_src.data(), v_src.data(), stream));
    TRY(kv_pool_retrieve_request(fpool, 5, n, dst_table.data(), slots, k_dst.data(), v_dst.data(), stream));
    HIPTRY(hipStreamSynchronize(stream));
    if (check()) return 1;
    struct stat st;
    if (on_file == 0 || ::stat(file_path.c_str(), &st) != 0 || uint64_t(st.st_size) != 64 * block_bytes) ++bad;
    // a ring resize that cannot allocate: NOMEM; file transfers and the file measurement refused with
    // NOMEM; a resize that fits brings them back
    g_fail_pinned_above = 64u << 20;
    if (kv_pool_set_file_ring(fpool, 128u << 20) != KVP_ERR_NOMEM) ++bad;
    g_fail_pinned_above = 0;
    if (hipGetLastError() != hipSuccess) ++bad;   // no HIP error left behind
    if (kv_pool_retrieve(fpool, map.data(), n, dst_table.data(), slots, k_dst.data(), v_dst.data(), stream) !=
        KVP_ERR_NOMEM)
        ++bad;
    if (kv_pool_store(fpool, map.data(), n, src_table.data(), slots, k_src.data(), v_src.data(), stream) != KVP_ERR_NOMEM)
        ++bad;
    uint64_t mbps[2] = {0, 0};
    if (kv_pool_measure_bandwidth(fpool, 1u << 20, 0, mbps) != KVP_ERR_NOMEM) ++bad;
    TRY(kv_pool_set_file_ring(fpool, 2 * block_bytes));
    for (uint32_t i = 0; i < 2 * L; ++i) HIPTRY(hipMemset(dst[i], 0xA5, layer_bytes));
    TRY(kv_pool_retrieve(fpool, map.data(), n, dst_table.data(), slots, k_dst.data(), v_dst.data(), stream));
    HIPTRY(hipStreamSynchronize(stream));
    if (check()) return 1;
    kv_pool_destroy(fpool);
    if (::stat(file_path.c_str(), &st) == 0) ++bad;     // the pool removes the file it created
    ::rmdir(dir_tmpl);
    HIPTRY(hipStreamDestroy(stream));
    for (void *p : src) HIPTRY(hipFree(p));
    for (void *p : dst) HIPTRY(hipFree(p));
    if (bad) {
        std::fprintf(stderr, "abi client: %llu mismatching chunks or elements\n", (unsigned long long)bad);
        return 1;
    }
    std::printf("abi client: %u blocks stored and retrieved exactly (small-call launch, upload path, allocation-free call, copy engines both ways, file region, file ring that cannot allocate)\n",
                n);
    return 0;
}
