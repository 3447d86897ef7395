// C ABI of the edge-feature join library: argument validation, the device document store, and
// launch geometry. The kernels live in join_kernels.hip.
#include <stdint.h>
#include <string.h>

#include <atomic>
#include <mutex>
#include <new>

#include <hip/hip_runtime.h>

#include "cc_join.h"
#include "join_internal.h"

static_assert(CC_SORT_AUTO == ccj::kSortAuto && CC_SORT_MERGE == ccj::kSortMerge &&
                  CC_SORT_RADIX == ccj::kSortRadix &&
                  CC_SORT_RADIX_MIN_RECORDS == ccj::kSortRadixMinRecords,
              "sort method values of the header and the kernels agree");

struct cc_store {
    int device;
    int64_t n_docs;
    int64_t capacity;                // rows allocated (n_docs for a store without an id map)
    int32_t doc_row_bytes;
    int64_t *d_author;               // [capacity]
    int32_t *d_author32;             // [capacity] the same ids in 32 bits, or null
    bool compact;                    // every stored author id fits in 32 bits: joins read d_author32
    uint8_t *d_rows;                 // [capacity][doc_row_bytes]
    unsigned long long *d_invalid;   // invalid-position counter
    uint8_t *d_zero;                 // ccj::kZeroRowBytes zero bytes, read in place of absent rows
    ccj::MapEntry *d_map;            // document-id map, or null (store without ids)
    int64_t *h_counts;               // pinned host copy of an ingestion batch's counts
    int64_t map_groups;              // probe groups in d_map (a power of two)
};

namespace {

thread_local int g_last_device_error = 0;

cc_status device_error(hipError_t e) {
    g_last_device_error = (int)e;
    return CC_ERR_DEVICE;
}

bool aligned(const void *p, uintptr_t a) { return ((uintptr_t)p & (a - 1)) == 0; }

bool mul_ok(int64_t a, int64_t b, int64_t *r) { return !__builtin_mul_overflow(a, b, r); }

bool overlaps(const void *a, int64_t na, const void *b, int64_t nb) {
    const uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
    return na > 0 && nb > 0 && x < y + (uintptr_t)nb && y < x + (uintptr_t)na;
}

// Keeps the store's device current for the duration of a call.
class DeviceGuard {
public:
    explicit DeviceGuard(int dev) {
        err_ = hipGetDevice(&prev_);
        if (err_ == hipSuccess && prev_ != dev) {
            err_ = hipSetDevice(dev);
            switched_ = err_ == hipSuccess;
        }
    }
    ~DeviceGuard() {
        if (switched_)
            (void)hipSetDevice(prev_);
    }
    hipError_t error() const { return err_; }

private:
    int prev_ = 0;
    hipError_t err_ = hipSuccess;
    bool switched_ = false;
};

cc_status join_impl(const cc_store *store, int32_t n_viewers, const int64_t *cand_offsets,
                    const int64_t *cand_idx, const int64_t *cand_author, int64_t total_cand,
                    const int64_t *key_offsets,
                    const int64_t *edge_keys, int64_t total_keys, const void *edge_feats,
                    int32_t edge_row_bytes, const void *default_row, int32_t n_lookups,
                    const int64_t *extra, void *out, int64_t out_row_stride, int8_t *hit_mask,
                    int64_t n_max, int8_t *valid_mask, const cc_tuning *tuning,
                    hipStream_t stream) {
    // n_max > 0 selects the padded layout (n_viewers * n_max output slots); 0 the CSR layout.
    // ---- host-side validation; nothing touches the device before it passes ----
    if (!store || n_viewers < 0 || total_cand < 0 || total_keys < 0)
        return CC_ERR_INVALID_ARGUMENT;
    if (edge_row_bytes <= 0 || (edge_row_bytes & 15) || edge_row_bytes > ccj::kMaxRowBytes)
        return CC_ERR_INVALID_ARGUMENT;
    if (n_lookups != 1 && n_lookups != 2)
        return CC_ERR_INVALID_ARGUMENT;
    const int64_t width = (int64_t)store->doc_row_bytes + (int64_t)n_lookups * edge_row_bytes;
    if (out_row_stride < width || (out_row_stride & 15))
        return CC_ERR_INVALID_ARGUMENT;
    int64_t bytes = 0;
    if (!mul_ok(total_cand, out_row_stride, &bytes) || !mul_ok(total_keys, edge_row_bytes, &bytes) ||
        !mul_ok(total_cand, n_lookups, &bytes))
        return CC_ERR_INVALID_ARGUMENT;
    const bool padded = n_max > 0;
    int64_t slots = 0;
    if (n_max < 0)
        return CC_ERR_INVALID_ARGUMENT;
    if (padded) {
        if (!mul_ok(n_viewers, n_max, &slots) || !mul_ok(slots, out_row_stride, &bytes) ||
            !mul_ok(slots, n_lookups, &bytes))
            return CC_ERR_INVALID_ARGUMENT;
        if (slots > 0 && (!out || !hit_mask || !valid_mask || !cand_offsets))
            return CC_ERR_INVALID_ARGUMENT;
    }
    if (n_viewers > 0 && cand_offsets == nullptr && key_offsets == nullptr) {
        // single-viewer form (cc_join): offsets are implicit
    } else if (n_viewers > 0 && (!cand_offsets || !key_offsets)) {
        return CC_ERR_INVALID_ARGUMENT;
    }
    if (total_cand > 0 && (n_viewers == 0 || !cand_idx || !out || !hit_mask))
        return CC_ERR_INVALID_ARGUMENT;
    if (total_keys > 0 && (!edge_keys || !edge_feats))
        return CC_ERR_INVALID_ARGUMENT;
    if (n_lookups == 2 && total_cand > 0 && !extra)
        return CC_ERR_INVALID_ARGUMENT;
    if (!aligned(out, 16) || !aligned(edge_feats, 16) || !aligned(default_row, 16) ||
        !aligned(cand_idx, 8) || !aligned(edge_keys, 8) || !aligned(cand_offsets, 8) ||
        !aligned(key_offsets, 8) || !aligned(extra, 8) || !aligned(cand_author, 8))
        return CC_ERR_INVALID_ARGUMENT;
    {
        // The outputs must not overlap any input or each other.
        const int64_t rows = padded ? slots : total_cand;
        const int64_t nv1 = cand_offsets ? (int64_t)n_viewers + 1 : 0;
        const struct { const void *p; int64_t n; } in[] = {
            {cand_idx, total_cand * 8}, {edge_keys, total_keys * 8},
            {edge_feats, total_keys * edge_row_bytes}, {extra, extra ? total_cand * 8 : 0},
            {cand_author, cand_author ? total_cand * 8 : 0},
            {cand_offsets, nv1 * 8}, {key_offsets, nv1 * 8},
            {default_row, default_row ? edge_row_bytes : 0}};
        const struct { const void *p; int64_t n; } outs[] = {
            {out, rows * out_row_stride}, {hit_mask, rows * n_lookups},
            {valid_mask, padded ? slots : 0}};
        for (const auto &o : outs) {
            for (const auto &i : in)
                if (overlaps(o.p, o.n, i.p, i.n))
                    return CC_ERR_INVALID_ARGUMENT;
        }
        if (overlaps(outs[0].p, outs[0].n, outs[1].p, outs[1].n) ||
            overlaps(outs[0].p, outs[0].n, outs[2].p, outs[2].n) ||
            overlaps(outs[1].p, outs[1].n, outs[2].p, outs[2].n))
            return CC_ERR_INVALID_ARGUMENT;
    }
    // Up to 16 fences per candidate of a segment: a larger table costs bulk reads from L2,
    // while a longer window between fences costs every lookup another dependent line.
    int32_t lds_cap = ccj::kDefaultLdsKeys, stride = 0, wgs = 0;
    const int32_t budget = 16;
    bool one_wave = false, lds_auto = true;
    const int64_t viewers = cand_offsets ? n_viewers : 1;
    if (viewers > 0 && total_keys / viewers > ccj::kLongListKeys) {
        lds_cap = ccj::kMaxLdsKeys;
        one_wave = true;
    }
    if (tuning) {
        if (tuning->fence_stride < 0 || tuning->lds_keys < 0 || tuning->workgroups < 0 ||
            tuning->lds_keys > ccj::kMaxLdsKeys || tuning->workgroups > (1 << 30))
            return CC_ERR_INVALID_ARGUMENT;
        if (tuning->fence_stride & (tuning->fence_stride - 1))
            return CC_ERR_INVALID_ARGUMENT;
        if (tuning->lds_keys) {
            lds_cap = tuning->lds_keys;
            lds_auto = false;
        }
        stride = tuning->fence_stride;
        wgs = tuning->workgroups;
    }
    if (total_cand == 0 && slots == 0)
        return CC_OK;

    DeviceGuard guard(store->device);
    if (guard.error() != hipSuccess)
        return device_error(guard.error());

    ccj::JoinArgs a;
    a.author = store->d_author;
    // The caller's author ids are read by the 64-bit form of the kernel.
    a.author32 = store->compact && !cand_author ? store->d_author32 : nullptr;
    a.cand_author = cand_author;
    a.doc = store->d_rows;
    a.n_docs = store->n_docs;
    a.doc_bytes = store->doc_row_bytes;
    a.edge_bytes = edge_row_bytes;
    a.cand_offsets = cand_offsets;
    a.cand_idx = cand_idx;
    a.total_cand = total_cand;
    a.key_offsets = key_offsets;
    a.keys = edge_keys;
    a.total_keys = total_keys;
    a.edge = static_cast<const uint8_t *>(edge_feats);
    a.def_row = static_cast<const uint8_t *>(default_row);
    a.zero_row = store->d_zero;
    a.extra = extra;
    a.out = static_cast<uint8_t *>(out);
    a.out_stride = out_row_stride;
    a.hit = hit_mask;
    a.n_max = n_max;
    a.invalid_counter = store->d_invalid;
    a.n_viewers = cand_offsets ? n_viewers : 1;
    a.fence_stride = stride;
    a.fence_budget = budget;
    a.one_wave = one_wave;
    a.lds_auto = lds_auto && !one_wave;
    // Weighted ranges for CSR batches of 2 to kBalanceViewers viewers (each workgroup scans
    // every viewer's offsets once).
    a.balanced = cand_offsets != nullptr && n_viewers > 1 && n_viewers <= ccj::kBalanceViewers;
    // The LDS table never needs more entries than the largest viewer has keys.
    a.lds_keys = (int32_t)(total_keys < lds_cap ? (total_keys > 0 ? total_keys : 1) : lds_cap);

    hipError_t e = hipSuccess;
    if (total_cand > 0)
        e = ccj::launch_join(a, n_lookups, wgs, store->device, stream);
    if (e == hipSuccess && padded)
        e = ccj::launch_pad_fill(a, n_lookups, valid_mask, stream);
    if (e != hipSuccess)
        return device_error(e);
    return CC_OK;
}

}  // namespace

extern "C" {

namespace {

// The current device, if it is a gfx950.
cc_status current_gfx950(int *dev) {
    hipError_t e = hipGetDevice(dev);
    if (e != hipSuccess)
        return e == hipErrorNoDevice ? CC_ERR_NOT_SUPPORTED : device_error(e);
    hipDeviceProp_t prop;
    e = hipGetDeviceProperties(&prop, *dev);
    if (e != hipSuccess)
        return device_error(e);
    if (strncmp(prop.gcnArchName, "gfx950", 6) != 0)
        return CC_ERR_NOT_SUPPORTED;
    return CC_OK;
}

void free_store(cc_store *s) {
    (void)hipFree(s->d_author);
    (void)hipFree(s->d_author32);
    (void)hipFree(s->d_rows);
    (void)hipFree(s->d_invalid);
    (void)hipFree(s->d_zero);
    (void)hipFree(s->d_map);
    (void)hipHostFree(s->h_counts);
    delete s;
}

cc_status alloc_failure(cc_store *s, hipError_t err) {
    free_store(s);
    if (err == hipErrorOutOfMemory || err == hipErrorMemoryAllocation) {
        g_last_device_error = (int)err;
        (void)hipGetLastError();
        return CC_ERR_OUT_OF_MEMORY;
    }
    return device_error(err);
}

// A store with room for `capacity` rows (and an id map when with_map), counters cleared.
cc_status new_store(int64_t capacity, int32_t doc_row_bytes, bool with_map, hipStream_t stream,
                    cc_store **out) {
    int64_t row_total = 0, id_total = 0, map_total = 0;
    const int64_t groups = with_map ? ccj::map_groups_for(capacity) : 0;
    if (!mul_ok(capacity, doc_row_bytes, &row_total) || !mul_ok(capacity, 8, &id_total) ||
        !mul_ok(groups, ccj::kGroup * (int64_t)sizeof(ccj::MapEntry), &map_total))
        return CC_ERR_INVALID_ARGUMENT;
    int dev = 0;
    cc_status st = current_gfx950(&dev);
    if (st != CC_OK)
        return st;
    cc_store *s = new (std::nothrow) cc_store();
    if (!s)
        return CC_ERR_OUT_OF_MEMORY;
    s->device = dev;
    s->capacity = capacity;
    s->doc_row_bytes = doc_row_bytes;
    s->map_groups = groups;
    hipError_t e;
    if ((e = hipMalloc(&s->d_author, (size_t)(id_total > 0 ? id_total : 256))) != hipSuccess)
        return alloc_failure(s, e);
    if ((e = hipMalloc(&s->d_rows, (size_t)(row_total > 0 ? row_total : 256))) != hipSuccess)
        return alloc_failure(s, e);
    if ((e = hipMalloc(&s->d_invalid, sizeof(unsigned long long))) != hipSuccess)
        return alloc_failure(s, e);
    if ((e = hipMalloc(&s->d_zero, ccj::kZeroRowBytes)) != hipSuccess)
        return alloc_failure(s, e);
    if (with_map && (e = hipMalloc(&s->d_map, (size_t)map_total)) != hipSuccess)
        return alloc_failure(s, e);
    if (with_map) {
        // Ingestion keeps the 32-bit author column next to the 64-bit one while every id fits.
        if ((e = hipMalloc(&s->d_author32, (size_t)(capacity > 0 ? capacity * 4 : 256))) != hipSuccess)
            return alloc_failure(s, e);
        s->compact = true;
        if ((e = hipHostMalloc(&s->h_counts, ccj::kUpsertCounts * sizeof(int64_t),
                               hipHostMallocDefault)) != hipSuccess)
            return alloc_failure(s, e);
    }
    if ((e = hipMemsetAsync(s->d_invalid, 0, sizeof(unsigned long long), stream)) != hipSuccess)
        return alloc_failure(s, e);
    if ((e = hipMemsetAsync(s->d_zero, 0, ccj::kZeroRowBytes, stream)) != hipSuccess)
        return alloc_failure(s, e);
    if (with_map && (e = ccj::launch_map_init(s->d_map, groups, stream)) != hipSuccess)
        return alloc_failure(s, e);
    *out = s;
    return CC_OK;
}

}  // namespace

cc_status cc_store_create(cc_store **out_store, int64_t n_docs, const int64_t *author_ids,
                          const void *doc_rows, int32_t doc_row_bytes, uint32_t flags,
                          hipStream_t stream) {
    if (!out_store)
        return CC_ERR_INVALID_ARGUMENT;
    *out_store = nullptr;
    if (n_docs < 0 || doc_row_bytes <= 0 || (doc_row_bytes & 15) ||
        doc_row_bytes > ccj::kMaxRowBytes)
        return CC_ERR_INVALID_ARGUMENT;
    if (flags != CC_SRC_HOST && flags != CC_SRC_DEVICE)
        return CC_ERR_INVALID_ARGUMENT;
    if (n_docs > 0 && (!author_ids || !doc_rows))
        return CC_ERR_INVALID_ARGUMENT;
    int64_t row_total = 0, id_total = 0;
    if (!mul_ok(n_docs, doc_row_bytes, &row_total) || !mul_ok(n_docs, 8, &id_total))
        return CC_ERR_INVALID_ARGUMENT;
    cc_store *s = nullptr;
    cc_status st = new_store(n_docs, doc_row_bytes, false, stream, &s);
    if (st != CC_OK)
        return st;
    s->n_docs = n_docs;
    const hipMemcpyKind kind = flags == CC_SRC_HOST ? hipMemcpyHostToDevice
                                                    : hipMemcpyDeviceToDevice;
    hipError_t e;
    unsigned long long *d_wide = nullptr;
    unsigned long long wide = 1;
    if (n_docs > 0) {
        if ((e = hipMemcpyAsync(s->d_author, author_ids, (size_t)id_total, kind, stream)) != hipSuccess)
            return alloc_failure(s, e);
        if ((e = hipMemcpyAsync(s->d_rows, doc_rows, (size_t)row_total, kind, stream)) != hipSuccess)
            return alloc_failure(s, e);
        // Keep a 32-bit copy of the author column when every id fits: it spans half as many
        // cache lines, so more of it stays in L2 under the join's random author reads. The copy
        // is optional: if it cannot be allocated the store keeps to its 64-bit column.
        void *a32 = nullptr, *w = nullptr;
        bool ok = hipMalloc(&a32, (size_t)(n_docs * 4)) == hipSuccess;
        if (ok)
            s->d_author32 = static_cast<int32_t *>(a32);
        ok = ok && hipMalloc(&w, sizeof(unsigned long long)) == hipSuccess;
        if (ok)
            d_wide = static_cast<unsigned long long *>(w);
        if (ok) {
            e = hipMemsetAsync(d_wide, 0, sizeof(unsigned long long), stream);
            if (e == hipSuccess)
                e = ccj::launch_narrow_authors(s->d_author, s->d_author32, n_docs, d_wide, stream);
            if (e == hipSuccess)
                e = hipMemcpyAsync(&wide, d_wide, sizeof(wide), hipMemcpyDeviceToHost, stream);
            if (e != hipSuccess) {
                (void)hipStreamSynchronize(stream);
                (void)hipFree(d_wide);
                return alloc_failure(s, e);
            }
        } else {
            (void)hipGetLastError();              // an allocation failure is not sticky
        }
    }
    // Every path synchronises once: the copies and the counter clears have completed when the
    // call returns, so the sources may be freed and any stream may use the store.
    e = hipStreamSynchronize(stream);
    (void)hipFree(d_wide);
    if (e != hipSuccess)
        return alloc_failure(s, e);
    if (wide == 0) {
        s->compact = true;
    } else if (s->d_author32) {
        (void)hipFree(s->d_author32);
        s->d_author32 = nullptr;
    }
    *out_store = s;
    return CC_OK;
}

cc_status cc_store_create_indexed(cc_store **out_store, int64_t capacity, int32_t doc_row_bytes,
                                  hipStream_t stream) {
    if (!out_store)
        return CC_ERR_INVALID_ARGUMENT;
    *out_store = nullptr;
    if (capacity < 0 || capacity > INT32_MAX || doc_row_bytes <= 0 || (doc_row_bytes & 15) ||
        doc_row_bytes > ccj::kMaxRowBytes)
        return CC_ERR_INVALID_ARGUMENT;
    cc_store *s = nullptr;
    cc_status st = new_store(capacity, doc_row_bytes, true, stream, &s);
    if (st != CC_OK)
        return st;
    // The map is cleared on `stream`; synchronise so that any stream may use the store.
    const hipError_t e = hipStreamSynchronize(stream);
    if (e != hipSuccess)
        return alloc_failure(s, e);
    *out_store = s;
    return CC_OK;
}

// Bound on the device-side waits of an ingestion batch (cc_set_ingestion_wait_limit).
static std::atomic<int32_t> g_wait_polls{ccj::kDefaultWaitPolls};

cc_status cc_set_ingestion_wait_limit(int32_t polls) {
    g_wait_polls.store(polls < 0 ? ccj::kDefaultWaitPolls : polls, std::memory_order_relaxed);
    return CC_OK;
}

int64_t cc_upsert_workspace_bytes(int64_t n_records) {
    return ccj::upsert_workspace_bytes(n_records);
}

cc_status cc_store_upsert(cc_store *store, int64_t n_records, const int64_t *doc_ids,
                          const int64_t *author_ids, const void *doc_rows, void *workspace,
                          int64_t workspace_bytes, int64_t *n_new, int64_t *n_rejected,
                          hipStream_t stream) {
    if (!store || n_records < 0 || n_records > ccj::kMaxBatch)
        return CC_ERR_INVALID_ARGUMENT;
    if (!store->d_map)
        return CC_ERR_NOT_SUPPORTED;
    if (n_new)
        *n_new = 0;
    if (n_rejected)
        *n_rejected = 0;
    if (n_records == 0)
        return CC_OK;
    const int64_t rb = store->doc_row_bytes;
    if (!doc_ids || !author_ids || !doc_rows || !workspace)
        return CC_ERR_INVALID_ARGUMENT;
    if (!aligned(doc_ids, 8) || !aligned(author_ids, 8) || !aligned(doc_rows, 16) ||
        !aligned(workspace, 16))
        return CC_ERR_INVALID_ARGUMENT;
    if (workspace_bytes < ccj::upsert_workspace_bytes(n_records))
        return CC_ERR_INVALID_ARGUMENT;
    if (overlaps(workspace, workspace_bytes, doc_ids, n_records * 8) ||
        overlaps(workspace, workspace_bytes, author_ids, n_records * 8) ||
        overlaps(workspace, workspace_bytes, doc_rows, n_records * rb))
        return CC_ERR_INVALID_ARGUMENT;
    DeviceGuard guard(store->device);
    if (guard.error() != hipSuccess)
        return device_error(guard.error());
    hipError_t e = ccj::launch_upsert_claim(store->d_map, store->map_groups, doc_ids, n_records,
                                            workspace,
                                            g_wait_polls.load(std::memory_order_relaxed), stream);
    if (e == hipSuccess)
        e = ccj::launch_upsert_finish(store->d_map, n_records, workspace, store->n_docs,
                                      store->capacity, author_ids, doc_rows,
                                      store->doc_row_bytes, store->d_author, store->d_author32,
                                      store->d_rows, stream);
    int64_t *counts = store->h_counts;        // pinned: the read-back is one small DMA
    if (e == hipSuccess)
        e = hipMemcpyAsync(counts, ccj::upsert_counts(workspace, n_records),
                           ccj::kUpsertCounts * sizeof(int64_t), hipMemcpyDeviceToHost, stream);
    if (e == hipSuccess)
        e = hipStreamSynchronize(stream);
    if (e != hipSuccess)
        return device_error(e);
    const int64_t fresh = counts[0], rejected = counts[1], unplaced = counts[2];
    if (counts[5] > 0)
        return CC_ERR_TIMEOUT;               // a bounded device wait gave up; rolled back
    if (unplaced > 0 || store->n_docs + fresh > store->capacity)
        return CC_ERR_STORE_FULL;            // rolled back on the device: the store is unchanged
    store->n_docs += fresh;
    if (counts[3] > 0)
        store->compact = false;              // an author id wider than 32 bits arrived
    if (n_new)
        *n_new = fresh;
    if (n_rejected)
        *n_rejected = rejected;
    return CC_OK;
}

cc_status cc_store_read(const cc_store *store, int64_t first, int64_t count, int64_t *author_out,
                        void *rows_out, hipStream_t stream) {
    if (!store || first < 0 || count < 0 || first > store->n_docs || count > store->n_docs - first)
        return CC_ERR_INVALID_ARGUMENT;
    if ((author_out && !aligned(author_out, 8)) || (rows_out && !aligned(rows_out, 16)))
        return CC_ERR_INVALID_ARGUMENT;
    if (count == 0)
        return CC_OK;
    DeviceGuard guard(store->device);
    if (guard.error() != hipSuccess)
        return device_error(guard.error());
    const int64_t rb = store->doc_row_bytes;
    hipError_t e = hipSuccess;
    if (author_out)
        e = hipMemcpyAsync(author_out, store->d_author + first, (size_t)(count * 8),
                           hipMemcpyDeviceToDevice, stream);
    if (e == hipSuccess && rows_out)
        e = hipMemcpyAsync(rows_out, store->d_rows + first * rb, (size_t)(count * rb),
                           hipMemcpyDeviceToDevice, stream);
    return e == hipSuccess ? CC_OK : device_error(e);
}

cc_status cc_resolve_ids(const cc_store *store, const int64_t *doc_ids, int64_t n,
                         int64_t *positions, hipStream_t stream) {
    if (!store || n < 0)
        return CC_ERR_INVALID_ARGUMENT;
    if (!store->d_map)
        return CC_ERR_NOT_SUPPORTED;
    if (n == 0)
        return CC_OK;
    int64_t bytes = 0;
    if (!doc_ids || !positions || !aligned(doc_ids, 8) || !aligned(positions, 8) ||
        !mul_ok(n, 8, &bytes))
        return CC_ERR_INVALID_ARGUMENT;
    if (doc_ids != positions && overlaps(doc_ids, bytes, positions, bytes))
        return CC_ERR_INVALID_ARGUMENT;
    DeviceGuard guard(store->device);
    if (guard.error() != hipSuccess)
        return device_error(guard.error());
    hipError_t e = ccj::launch_resolve(store->d_map, store->map_groups, doc_ids, n, positions,
                                       stream);
    return e == hipSuccess ? CC_OK : device_error(e);
}

cc_status cc_store_destroy(cc_store *store) {
    if (!store)
        return CC_OK;
    DeviceGuard guard(store->device);
    free_store(store);
    return CC_OK;
}

cc_status cc_store_info(const cc_store *store, int64_t *n_docs, int32_t *doc_row_bytes) {
    if (!store)
        return CC_ERR_INVALID_ARGUMENT;
    if (n_docs)
        *n_docs = store->n_docs;
    if (doc_row_bytes)
        *doc_row_bytes = store->doc_row_bytes;
    return CC_OK;
}

cc_status cc_store_layout(const cc_store *store, int32_t *author_id_bytes, int64_t *capacity) {
    if (!store)
        return CC_ERR_INVALID_ARGUMENT;
    if (author_id_bytes)
        *author_id_bytes = store->compact ? 4 : 8;
    if (capacity)
        *capacity = store->capacity;
    return CC_OK;
}

cc_status cc_store_invalid_count(const cc_store *store, int64_t *count, hipStream_t stream) {
    if (!store || !count)
        return CC_ERR_INVALID_ARGUMENT;
    DeviceGuard guard(store->device);
    if (guard.error() != hipSuccess)
        return device_error(guard.error());
    unsigned long long v = 0;
    hipError_t e = hipMemcpyAsync(&v, store->d_invalid, sizeof(v), hipMemcpyDeviceToHost, stream);
    if (e == hipSuccess)
        e = hipStreamSynchronize(stream);
    if (e != hipSuccess)
        return device_error(e);
    *count = (int64_t)v;
    return CC_OK;
}

cc_status cc_store_reset_invalid_count(cc_store *store, hipStream_t stream) {
    if (!store)
        return CC_ERR_INVALID_ARGUMENT;
    DeviceGuard guard(store->device);
    if (guard.error() != hipSuccess)
        return device_error(guard.error());
    const hipError_t e = ccj::launch_clear_counter(store->d_invalid, stream);
    return e == hipSuccess ? CC_OK : device_error(e);
}

cc_status cc_join(const cc_store *store, const int64_t *cand_idx, int64_t n_cand,
                  const int64_t *edge_keys, int64_t n_keys, const void *edge_feats,
                  int32_t edge_row_bytes, const void *default_row, void *out,
                  int64_t out_row_stride, int8_t *hit_mask, hipStream_t stream) {
    return join_impl(store, 1, nullptr, cand_idx, nullptr, n_cand, nullptr, edge_keys, n_keys,
                     edge_feats,
                     edge_row_bytes, default_row, 1, nullptr, out, out_row_stride, hit_mask, 0,
                     nullptr, nullptr, stream);
}

cc_status cc_join_batched_tuned(const cc_store *store, int32_t n_viewers,
                                const int64_t *cand_offsets, const int64_t *cand_idx,
                                int64_t total_cand, const int64_t *key_offsets,
                                const int64_t *edge_keys, int64_t total_keys,
                                const void *edge_feats, int32_t edge_row_bytes,
                                const void *default_row, int32_t n_lookups,
                                const int64_t *const *extra_keys, void *out,
                                int64_t out_row_stride, int8_t *hit_mask,
                                const cc_tuning *tuning, hipStream_t stream) {
    if (n_viewers > 0 && (!cand_offsets || !key_offsets))
        return CC_ERR_INVALID_ARGUMENT;
    if (n_lookups == 2 && !extra_keys)
        return CC_ERR_INVALID_ARGUMENT;
    const int64_t *extra = (n_lookups == 2) ? extra_keys[0] : nullptr;
    return join_impl(store, n_viewers, cand_offsets, cand_idx, nullptr, total_cand, key_offsets,
                     edge_keys, total_keys, edge_feats, edge_row_bytes, default_row, n_lookups,
                     extra, out, out_row_stride, hit_mask, 0, nullptr, tuning, stream);
}

cc_status cc_join_batched_padded(const cc_store *store, int32_t n_viewers,
                                 const int64_t *cand_offsets, const int64_t *cand_idx,
                                 int64_t total_cand, const int64_t *key_offsets,
                                 const int64_t *edge_keys, int64_t total_keys,
                                 const void *edge_feats, int32_t edge_row_bytes,
                                 const void *default_row, int32_t n_lookups,
                                 const int64_t *const *extra_keys, int64_t n_max, void *out,
                                 int64_t out_row_stride, int8_t *hit_mask, int8_t *valid_mask,
                                 hipStream_t stream) {
    if (n_viewers > 0 && (!cand_offsets || !key_offsets || n_max < 1))
        return CC_ERR_INVALID_ARGUMENT;
    if (n_lookups == 2 && !extra_keys)
        return CC_ERR_INVALID_ARGUMENT;
    const int64_t *extra = (n_lookups == 2) ? extra_keys[0] : nullptr;
    if (n_viewers == 0)
        return join_impl(store, 0, cand_offsets, cand_idx, nullptr, total_cand, key_offsets,
                         edge_keys, total_keys, edge_feats, edge_row_bytes, default_row, n_lookups,
                         extra, out, out_row_stride, hit_mask, 0, nullptr, nullptr, stream);
    return join_impl(store, n_viewers, cand_offsets, cand_idx, nullptr, total_cand, key_offsets,
                     edge_keys, total_keys, edge_feats, edge_row_bytes, default_row, n_lookups,
                     extra, out, out_row_stride, hit_mask, n_max, valid_mask, nullptr, stream);
}

cc_status cc_join_batched_authors(const cc_store *store, int32_t n_viewers,
                                  const int64_t *cand_offsets, const int64_t *cand_idx,
                                  const int64_t *author_ids, int64_t total_cand,
                                  const int64_t *key_offsets, const int64_t *edge_keys,
                                  int64_t total_keys, const void *edge_feats,
                                  int32_t edge_row_bytes, const void *default_row,
                                  int32_t n_lookups, const int64_t *const *extra_keys, void *out,
                                  int64_t out_row_stride, int8_t *hit_mask, hipStream_t stream) {
    if (n_viewers > 0 && (!cand_offsets || !key_offsets))
        return CC_ERR_INVALID_ARGUMENT;
    if (n_lookups == 2 && !extra_keys)
        return CC_ERR_INVALID_ARGUMENT;
    if (total_cand > 0 && !author_ids)
        return CC_ERR_INVALID_ARGUMENT;
    const int64_t *extra = (n_lookups == 2) ? extra_keys[0] : nullptr;
    return join_impl(store, n_viewers, cand_offsets, cand_idx, author_ids, total_cand,
                     key_offsets, edge_keys, total_keys, edge_feats, edge_row_bytes, default_row,
                     n_lookups, extra, out, out_row_stride, hit_mask, 0, nullptr, nullptr,
                     stream);
}

cc_status cc_join_batched(const cc_store *store, int32_t n_viewers, const int64_t *cand_offsets,
                          const int64_t *cand_idx, int64_t total_cand,
                          const int64_t *key_offsets, const int64_t *edge_keys,
                          int64_t total_keys, const void *edge_feats, int32_t edge_row_bytes,
                          const void *default_row, int32_t n_lookups,
                          const int64_t *const *extra_keys, void *out, int64_t out_row_stride,
                          int8_t *hit_mask, hipStream_t stream) {
    return cc_join_batched_tuned(store, n_viewers, cand_offsets, cand_idx, total_cand,
                                 key_offsets, edge_keys, total_keys, edge_feats, edge_row_bytes,
                                 default_row, n_lookups, extra_keys, out, out_row_stride,
                                 hit_mask, nullptr, stream);
}

int64_t cc_sort_workspace_bytes(int64_t total_keys, int32_t n_viewers) {
    return ccj::sort_workspace_bytes(total_keys, n_viewers);
}


cc_status cc_sort_affinity_method(int32_t method, int32_t key_bits, int32_t n_viewers,
                                  const int64_t *key_offsets, const int64_t *keys_in,
                                  const void *rows_in, int32_t row_bytes, int64_t total_keys,
                                  int64_t max_keys, int64_t *keys_out, void *rows_out,
                                  void *workspace, int64_t workspace_bytes, hipStream_t stream) {
    if (method != CC_SORT_AUTO && method != CC_SORT_MERGE && method != CC_SORT_RADIX)
        return CC_ERR_INVALID_ARGUMENT;
    if (key_bits < 0 || key_bits > 64)
        return CC_ERR_INVALID_ARGUMENT;
    if (n_viewers < 0 || total_keys < 0 || total_keys >= ((int64_t)1 << 32) || max_keys < 0)
        return CC_ERR_INVALID_ARGUMENT;
    if (row_bytes <= 0 || (row_bytes & 15) || row_bytes > ccj::kMaxRowBytes)
        return CC_ERR_INVALID_ARGUMENT;
    if (n_viewers > 0 && !key_offsets)
        return CC_ERR_INVALID_ARGUMENT;
    if (total_keys == 0 || n_viewers == 0)
        return CC_OK;
    const int64_t need = ccj::sort_workspace_bytes(total_keys, n_viewers);
    if (!keys_in || !rows_in || !keys_out || !rows_out || !workspace || workspace_bytes < need)
        return CC_ERR_INVALID_ARGUMENT;
    if (!aligned(key_offsets, 8) || !aligned(keys_in, 8) || !aligned(keys_out, 8) ||
        !aligned(rows_in, 16) || !aligned(rows_out, 16) || !aligned(workspace, 16))
        return CC_ERR_INVALID_ARGUMENT;
    const int64_t kbytes = total_keys * 8, rbytes = total_keys * (int64_t)row_bytes;
    if (overlaps(keys_out, kbytes, keys_in, kbytes) || overlaps(keys_out, kbytes, rows_in, rbytes) ||
        overlaps(rows_out, rbytes, keys_in, kbytes) || overlaps(rows_out, rbytes, rows_in, rbytes) ||
        overlaps(keys_out, kbytes, workspace, need) || overlaps(rows_out, rbytes, workspace, need) ||
        overlaps(keys_out, kbytes, rows_out, rbytes))
        return CC_ERR_INVALID_ARGUMENT;
    hipError_t e = ccj::launch_sort(n_viewers, key_offsets, keys_in, rows_in, row_bytes,
                                    total_keys, max_keys, keys_out, rows_out, workspace, method,
                                    key_bits, stream);
    return e == hipSuccess ? CC_OK : device_error(e);
}

cc_status cc_sort_affinity(int32_t n_viewers, const int64_t *key_offsets, const int64_t *keys_in,
                           const void *rows_in, int32_t row_bytes, int64_t total_keys,
                           int64_t max_keys, int64_t *keys_out, void *rows_out, void *workspace,
                           int64_t workspace_bytes, hipStream_t stream) {
    return cc_sort_affinity_method(CC_SORT_AUTO, 0, n_viewers, key_offsets, keys_in, rows_in,
                                   row_bytes, total_keys, max_keys, keys_out, rows_out, workspace,
                                   workspace_bytes, stream);
}

cc_status cc_sort_affinity_noalloc(int32_t n_viewers, const int64_t *key_offsets,
                                   const int64_t *keys_in, const void *rows_in, int32_t row_bytes,
                                   int64_t total_keys, int64_t max_keys, int64_t *keys_out,
                                   void *rows_out, hipStream_t stream) {
    if (n_viewers < 0 || total_keys < 0 || max_keys < 0)
        return CC_ERR_INVALID_ARGUMENT;
    if (row_bytes <= 0 || (row_bytes & 15) || row_bytes > ccj::kMaxRowBytes)
        return CC_ERR_INVALID_ARGUMENT;
    if (n_viewers > 0 && !key_offsets)
        return CC_ERR_INVALID_ARGUMENT;
    if (total_keys > ccj::kSortScratchRecords || n_viewers > ccj::kSortScratchViewers)
        return CC_ERR_TOO_LARGE;
    if (total_keys == 0 || n_viewers == 0)
        return CC_OK;
    if (!keys_in || !rows_in || !keys_out || !rows_out)
        return CC_ERR_INVALID_ARGUMENT;
    if (!aligned(key_offsets, 8) || !aligned(keys_in, 8) || !aligned(keys_out, 8) ||
        !aligned(rows_in, 16) || !aligned(rows_out, 16))
        return CC_ERR_INVALID_ARGUMENT;
    const int64_t kbytes = total_keys * 8, rbytes = total_keys * (int64_t)row_bytes;
    if (overlaps(keys_out, kbytes, keys_in, kbytes) || overlaps(keys_out, kbytes, rows_in, rbytes) ||
        overlaps(rows_out, rbytes, keys_in, kbytes) || overlaps(rows_out, rbytes, rows_in, rbytes) ||
        overlaps(keys_out, kbytes, rows_out, rbytes))
        return CC_ERR_INVALID_ARGUMENT;
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    void *scratch = nullptr;
    if (e == hipSuccess)
        e = ccj::sort_scratch(dev, &scratch);
    if (e == hipSuccess)
        e = ccj::launch_sort(n_viewers, key_offsets, keys_in, rows_in, row_bytes, total_keys,
                             max_keys, keys_out, rows_out, scratch, ccj::kSortAuto, 0, stream);
    return e == hipSuccess ? CC_OK : device_error(e);
}

cc_status cc_validate_keys(const int64_t *key_offsets, const int64_t *edge_keys,
                           int32_t n_viewers, int64_t total_keys, int64_t *first_bad_viewer,
                           hipStream_t stream) {
    if (!first_bad_viewer || n_viewers < 0 || total_keys < 0)
        return CC_ERR_INVALID_ARGUMENT;
    *first_bad_viewer = -1;
    if (n_viewers > 0 && !key_offsets)
        return CC_ERR_INVALID_ARGUMENT;
    if (total_keys > 0 && !edge_keys)
        return CC_ERR_INVALID_ARGUMENT;
    if (!aligned(key_offsets, 8) || !aligned(edge_keys, 8))
        return CC_ERR_INVALID_ARGUMENT;
    if (n_viewers == 0 || total_keys == 0)
        return CC_OK;
    // One flag buffer per device, allocated on the first call there and kept; the lock
    // serialises the calls that share it (each call synchronises before it returns).
    static std::mutex mu;
    static unsigned long long *flag[ccj::kMaxScratchDevices] = {};
    std::lock_guard<std::mutex> lock(mu);
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return device_error(e);
    if (dev < 0 || dev >= ccj::kMaxScratchDevices)
        return device_error(hipErrorInvalidDevice);
    if (!flag[dev] && (e = hipMalloc(&flag[dev], sizeof(unsigned long long))) != hipSuccess) {
        flag[dev] = nullptr;
        return device_error(e);
    }
    unsigned long long *d_bad = flag[dev];
    unsigned long long bad = ~0ull;
    e = hipMemcpyAsync(d_bad, &bad, sizeof(bad), hipMemcpyHostToDevice, stream);
    if (e == hipSuccess)
        e = ccj::launch_validate_keys(key_offsets, edge_keys, n_viewers, total_keys, d_bad, stream);
    if (e == hipSuccess)
        e = hipMemcpyAsync(&bad, d_bad, sizeof(bad), hipMemcpyDeviceToHost, stream);
    if (e == hipSuccess)
        e = hipStreamSynchronize(stream);
    if (e != hipSuccess)
        return device_error(e);
    if (bad != ~0ull) {
        *first_bad_viewer = (int64_t)bad;
        return CC_ERR_UNSORTED_KEYS;
    }
    return CC_OK;
}

// An int, not the enum: C callers may pass any value, and a C++ enum parameter outside the
// enumerators' range would be undefined behaviour here.
const char *cc_status_string(int status) {
    switch (status) {
    case CC_OK: return "CC_OK";
    case CC_ERR_INVALID_ARGUMENT: return "CC_ERR_INVALID_ARGUMENT";
    case CC_ERR_OUT_OF_MEMORY: return "CC_ERR_OUT_OF_MEMORY";
    case CC_ERR_DEVICE: return "CC_ERR_DEVICE";
    case CC_ERR_UNSORTED_KEYS: return "CC_ERR_UNSORTED_KEYS";
    case CC_ERR_NOT_SUPPORTED: return "CC_ERR_NOT_SUPPORTED";
    case CC_ERR_STORE_FULL: return "CC_ERR_STORE_FULL";
    case CC_ERR_TOO_LARGE: return "CC_ERR_TOO_LARGE";
    case CC_ERR_TIMEOUT: return "CC_ERR_TIMEOUT";
    }
    return "CC_UNKNOWN_STATUS";
}

int cc_last_device_error(void) { return g_last_device_error; }

}  // extern "C"
