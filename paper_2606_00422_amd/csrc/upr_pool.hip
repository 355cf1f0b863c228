// Cross-process KV-cache pool: one device allocation of slot caches, shared
// with other processes through a HIP IPC handle (paper Sec. 3, "KV-cache
// sharing across stages").
#include <atomic>
#include <cstdio>
#include <cstring>
#include <string>

#include "upr_internal.h"

// The handle is a file format: its size is part of the interface.
static_assert(sizeof(upr_kv_pool_handle) == 120, "upr_kv_pool_handle layout");

struct upr_kv_pool {
    upr_config cfg;
    int32_t slots = 0;
    int64_t capacity_rows = 0;
    size_t slot_bytes = 0;
    size_t bytes = 0;
    void* base = nullptr;
    bool owner = false;                 // created here (hipFree) or opened (close the mapping)
    hipIpcMemHandle_t ipc;
    std::atomic<uint32_t> next{0};
};

namespace {

size_t cache_bytes(const upr_config& c, int64_t rows) {
    const size_t es = (c.dtype == UPR_F32) ? 4 : 2;
    return (size_t)c.n_layers * 2 * c.n_heads * (size_t)rows * c.head_dim * es;
}

// A pool's size, or 0 with the error recorded.
upr_status pool_bytes(const upr_config* cfg, int32_t slots, int64_t rows, size_t* slot_bytes,
                      size_t* bytes) {
    upr_status st = upr::validate_config(cfg);
    if (st != UPR_OK) return st;
    if (slots < 1 || rows < 1)
        return upr::report_error(UPR_ERR_LIMIT, "pool needs slots >= 1 and capacity_rows >= 1 "
                                 "(got %d, %lld)", slots, (long long)rows);
    *slot_bytes = cache_bytes(*cfg, rows);
    if (*slot_bytes > UPR_KV_POOL_MAX_BYTES || (size_t)slots > UPR_KV_POOL_MAX_BYTES / *slot_bytes)
        return upr::report_error(UPR_ERR_LIMIT, "pool of %d slots x %zu bytes exceeds %zu bytes",
                                 slots, *slot_bytes, (size_t)UPR_KV_POOL_MAX_BYTES);
    // slots start on 256-byte boundaries (cache rows are 64- or 128-byte
    // multiples, the planes of a slot are whole rows)
    *slot_bytes = (*slot_bytes + 255) & ~size_t(255);
    *bytes = *slot_bytes * (size_t)slots;
    if (*bytes > UPR_KV_POOL_MAX_BYTES)
        return upr::report_error(UPR_ERR_LIMIT, "pool of %zu bytes exceeds %zu bytes", *bytes,
                                 (size_t)UPR_KV_POOL_MAX_BYTES);
    return UPR_OK;
}

}  // namespace

extern "C" {

upr_status upr_kv_pool_create(const upr_config* cfg, int32_t slots, int64_t capacity_rows,
                              upr_kv_pool** out) {
    if (!out) return upr::report_error(UPR_ERR_NULL, "out is NULL");
    size_t slot_bytes = 0, bytes = 0;
    upr_status st = pool_bytes(cfg, slots, capacity_rows, &slot_bytes, &bytes);
    if (st != UPR_OK) return st;
    void* base = nullptr;
    hipError_t e = hipMalloc(&base, bytes);
    if (e != hipSuccess)
        return upr::report_error(UPR_ERR_HIP, "hipMalloc(%zu) for the pool failed: %s", bytes,
                                 hipGetErrorString(e));
    hipIpcMemHandle_t h;
    e = hipIpcGetMemHandle(&h, base);
    if (e != hipSuccess) {
        (void)hipFree(base);
        return upr::report_error(UPR_ERR_HIP, "hipIpcGetMemHandle failed: %s", hipGetErrorString(e));
    }
    upr_kv_pool* p = new upr_kv_pool();
    p->cfg = *cfg;
    p->slots = slots;
    p->capacity_rows = capacity_rows;
    p->slot_bytes = slot_bytes;
    p->bytes = bytes;
    p->base = base;
    p->owner = true;
    p->ipc = h;
    *out = p;
    return upr::report_ok();
}

upr_status upr_kv_pool_export(const upr_kv_pool* pool, upr_kv_pool_handle* out) {
    if (!pool || !out) return upr::report_error(UPR_ERR_NULL, "pool or out is NULL");
    static_assert(sizeof(hipIpcMemHandle_t) == sizeof(out->ipc), "IPC handle size");
    upr_kv_pool_handle h{};
    h.magic = UPR_KV_POOL_MAGIC;
    h.slots = pool->slots;
    h.capacity_rows = pool->capacity_rows;
    h.bytes = pool->bytes;
    h.cfg = pool->cfg;
    std::memcpy(h.ipc, &pool->ipc, sizeof(h.ipc));
    *out = h;
    return upr::report_ok();
}

upr_status upr_kv_pool_export_file(const upr_kv_pool* pool, const char* path) {
    if (!path) return upr::report_error(UPR_ERR_NULL, "path is NULL");
    upr_kv_pool_handle h;
    upr_status st = upr_kv_pool_export(pool, &h);
    if (st != UPR_OK) return st;
    const std::string tmp = std::string(path) + ".tmp";
    FILE* f = std::fopen(tmp.c_str(), "wb");
    if (!f) return upr::report_error(UPR_ERR_LIMIT, "cannot write %s", tmp.c_str());
    const bool ok = std::fwrite(&h, sizeof(h), 1, f) == 1;
    if (std::fclose(f) != 0 || !ok || std::rename(tmp.c_str(), path) != 0) {
        std::remove(tmp.c_str());
        return upr::report_error(UPR_ERR_LIMIT, "cannot write the handle file %s", path);
    }
    return upr::report_ok();
}

upr_status upr_kv_pool_open(const upr_kv_pool_handle* handle, upr_kv_pool** out) {
    if (!handle || !out) return upr::report_error(UPR_ERR_NULL, "handle or out is NULL");
    if (handle->magic != UPR_KV_POOL_MAGIC)
        return upr::report_error(UPR_ERR_CONFIG, "not a pool handle (magic %08x)", handle->magic);
    size_t slot_bytes = 0, bytes = 0;
    upr_status st = pool_bytes(&handle->cfg, handle->slots, handle->capacity_rows, &slot_bytes, &bytes);
    if (st != UPR_OK) return st;
    if (bytes != handle->bytes)
        return upr::report_error(UPR_ERR_CONFIG, "handle says %llu bytes, its shape needs %zu",
                                 (unsigned long long)handle->bytes, bytes);
    hipIpcMemHandle_t h;
    std::memcpy(&h, handle->ipc, sizeof(h));
    void* base = nullptr;
    const hipError_t e = hipIpcOpenMemHandle(&base, h, hipIpcMemLazyEnablePeerAccess);
    if (e != hipSuccess)
        return upr::report_error(UPR_ERR_HIP, "hipIpcOpenMemHandle failed: %s", hipGetErrorString(e));
    upr_kv_pool* p = new upr_kv_pool();
    p->cfg = handle->cfg;
    p->slots = handle->slots;
    p->capacity_rows = handle->capacity_rows;
    p->slot_bytes = slot_bytes;
    p->bytes = bytes;
    p->base = base;
    p->owner = false;
    p->ipc = h;
    *out = p;
    return upr::report_ok();
}

upr_status upr_kv_pool_open_file(const char* path, upr_kv_pool** out) {
    if (!path) return upr::report_error(UPR_ERR_NULL, "path is NULL");
    upr_kv_pool_handle h;
    FILE* f = std::fopen(path, "rb");
    if (!f) return upr::report_error(UPR_ERR_LIMIT, "cannot read the handle file %s", path);
    const bool ok = std::fread(&h, sizeof(h), 1, f) == 1;
    std::fclose(f);
    if (!ok) return upr::report_error(UPR_ERR_CONFIG, "handle file %s is truncated", path);
    return upr_kv_pool_open(&h, out);
}

upr_status upr_kv_pool_slot(const upr_kv_pool* pool, int32_t slot, upr_kv_cache* out) {
    if (!pool || !out) return upr::report_error(UPR_ERR_NULL, "pool or out is NULL");
    if (slot < 0 || slot >= pool->slots)
        return upr::report_error(UPR_ERR_LIMIT, "slot %d outside [0, %d)", slot, pool->slots);
    out->data = static_cast<char*>(pool->base) + (size_t)slot * pool->slot_bytes;
    out->capacity_rows = pool->capacity_rows;
    return upr::report_ok();
}

int32_t upr_kv_pool_next_slot(upr_kv_pool* pool) {
    if (!pool) return -1;
    return (int32_t)(pool->next.fetch_add(1, std::memory_order_relaxed) % (uint32_t)pool->slots);
}

upr_status upr_kv_pool_info(const upr_kv_pool* pool, upr_config* cfg, int32_t* slots,
                            int64_t* capacity_rows) {
    if (!pool) return upr::report_error(UPR_ERR_NULL, "pool is NULL");
    if (cfg) *cfg = pool->cfg;
    if (slots) *slots = pool->slots;
    if (capacity_rows) *capacity_rows = pool->capacity_rows;
    return upr::report_ok();
}

void upr_kv_pool_destroy(upr_kv_pool* pool) {
    if (!pool) return;
    if (pool->owner)
        (void)hipFree(pool->base);
    else
        (void)hipIpcCloseMemHandle(pool->base);
    delete pool;
}

}  // extern "C"
