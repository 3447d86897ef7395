// Internal interface between the C ABI layer (cc_api.hip) and the kernels (join_kernels.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ccj {

constexpr int kBlock = 256;          // threads per workgroup = candidates per sub-tile
constexpr int kBalanceViewers = 4 * kBlock;   // CSR batches up to this size get weighted ranges
constexpr int kWindow = 15;          // keys between two fences read from L2 in one step
constexpr int kMaxLdsKeys = 18432;   // LDS key table limit: 144 KiB + at most 12 KiB of static
                                     // tables stays within the 160 KiB a workgroup may use
constexpr int kDefaultLdsKeys = 8192;   // 64 KiB: within the register-limited occupancy
// Table capacity when the grid is one workgroup per CU (occupancy is then set by the grid, not
// by LDS): lists of up to 16,384 keys are staged whole, with no window read per lookup.
constexpr int kWideLdsKeys = 16384;
// Average key-list length above which a launch uses the whole LDS table and one resident wave
// of workgroups (one per CU): the larger table keeps each lookup's window of keys within one
// 64-byte sector, and one wave leaves no half-empty last wave.
constexpr int64_t kLongListKeys = 4 * (int64_t)kDefaultLdsKeys;
// Largest row (document, edge or affinity record) in bytes. Copy loops count a tile's row
// chunks in 32 bits: 256 rows (or 4096 sort records) of this many bytes stay far below 2^31.
constexpr int32_t kMaxRowBytes = 1 << 20;
constexpr int kZeroRowBytes = 1024;    // >= the widest row of a compile-time specialisation

struct JoinArgs {
    const int64_t *author;       // store: author id per position
    const int32_t *author32;     // store: the same ids narrowed to 32 bits, or nullptr
    const uint8_t *doc;          // store: rows, doc_bytes each
    int64_t n_docs;
    int32_t doc_bytes;
    int32_t edge_bytes;
    const int64_t *cand_offsets; // [B+1] or nullptr for one viewer
    const int64_t *cand_idx;
    const int64_t *cand_author;  // [total_cand] author id per candidate, or nullptr: the store's
    int64_t total_cand;
    const int64_t *key_offsets;  // [B+1] or nullptr for one viewer
    const int64_t *keys;
    int64_t total_keys;
    const uint8_t *edge;
    const uint8_t *def_row;      // nullptr = zero bytes
    const uint8_t *zero_row;     // kZeroRowBytes of zeros in device memory (store-owned)
    const int64_t *extra;        // keys of lookup 1 (n_lookups == 2)
    uint8_t *out;
    int64_t out_stride;
    int8_t *hit;
    int64_t n_max;               // > 0: padded layout, n_max output rows per viewer
    unsigned long long *invalid_counter;
    int32_t n_viewers;
    int32_t lds_keys;            // capacity of the dynamic LDS key table
    int32_t fence_stride;        // 0 = chosen per viewer segment
    int32_t fence_budget;        // fences staged per candidate of a segment (automatic stride)
    bool one_wave;               // automatic grid: one resident wave (long key lists)
    bool lds_auto;               // lds_keys chosen by the library (not by a tuning)
    bool balanced;               // CSR ranges weighted by an estimated cost per candidate
    int32_t n_wg;                // workgroups launched (a multiple of 8); set by launch_join
    int64_t per_wg;              // candidates per workgroup (multiple of kBlock); set by launch_join
};

// Enqueue the join kernel matching the row widths and lookup count on `device` (current).
// `workgroups` > 0 fixes the grid; 0 sizes it from the kernel's occupancy. Returns the HIP
// error of the launch.
hipError_t launch_join(JoinArgs &args, int n_lookups, int32_t workgroups, int device,
                       hipStream_t stream);

// Enqueue the pad fill of the padded layout: valid mask of every slot, zero rows and hit bits
// for pad slots.
hipError_t launch_pad_fill(const JoinArgs &args, int n_lookups, int8_t *valid_mask,
                           hipStream_t stream);

// Workspace bytes of the affinity-record sort for `total` records in `n_viewers` viewers.
int64_t sort_workspace_bytes(int64_t total, int32_t n_viewers);

// Largest call of the allocation-free sort: its workspace is a fixed device array of
// sort_workspace_bytes(kSortScratchRecords, kSortScratchViewers) bytes.
constexpr int64_t kSortScratchRecords = (int64_t)1 << 20;
constexpr int32_t kSortScratchViewers = 1 << 16;
constexpr int kMaxScratchDevices = 64;

// Device address of the allocation-free sort's fixed scratch on `device`, which must be the
// current device. Resolved on the first call per device, then cached.
hipError_t sort_scratch(int device, void **ptr);

// Sort methods (the values of CC_SORT_AUTO, CC_SORT_MERGE, CC_SORT_RADIX) and the call size
// from which the automatic choice takes the radix method.
constexpr int32_t kSortAuto = 0;
constexpr int32_t kSortMerge = 1;
constexpr int32_t kSortRadix = 2;
constexpr int64_t kSortRadixMinRecords = (int64_t)1 << 20;

// Enqueue the per-viewer stable sort of affinity records (keys + rows) into keys_out/rows_out
// with `method` (kSortAuto: by call size). max_keys > 0 bounds the records of any one viewer;
// key_bits > 0 bounds the bit length of (largest key - smallest key); 0 = unknown.
hipError_t launch_sort(int32_t n_viewers, const int64_t *key_offsets, const int64_t *keys_in,
                       const void *rows_in, int32_t row_bytes, int64_t total, int64_t max_keys,
                       int64_t *keys_out, void *rows_out, void *workspace, int32_t method,
                       int32_t key_bits, hipStream_t stream);

// Enqueue a kernel that sets *counter (device) to zero.
hipError_t launch_clear_counter(unsigned long long *counter, hipStream_t stream);

// Enqueue the key-order check; *first_bad (device) must hold UINT64_MAX beforehand.
hipError_t launch_validate_keys(const int64_t *key_offsets, const int64_t *keys,
                                int32_t n_viewers, int64_t total_keys,
                                unsigned long long *first_bad, hipStream_t stream);

// Narrow an author column to 32 bits: dst[i] = (int32_t)src[i]; *wide counts the ids outside
// the int32 range (dst is then not usable).
hipError_t launch_narrow_authors(const int64_t *src, int32_t *dst, int64_t n,
                                 unsigned long long *wide, hipStream_t stream);

// ---- document-id map (id -> store position), open addressing over 64-byte groups ----

struct MapEntry {
    int64_t key;    // document id; kEmptyKey marks a free entry
    int32_t pos;    // store position >= 0; while a batch is applied, -(3 + first record index)
    int32_t aux;    // while a batch is applied: last record index with this id; else -1
};
static_assert(sizeof(MapEntry) == 16, "map entries are 16 bytes");
constexpr int kGroup = 4;                        // entries per probe group (64 bytes)
constexpr int64_t kEmptyKey = INT64_MIN;         // reserved: cannot be stored
constexpr int32_t kNoPos = INT32_MIN;            // pos of a free entry
constexpr int64_t kMaxBatch = (int64_t)1 << 30;  // records per ingestion batch

// Probe groups for a store of `capacity` documents (load factor <= 1/2), a power of two.
int64_t map_groups_for(int64_t capacity);
hipError_t launch_map_init(MapEntry *map, int64_t n_groups, hipStream_t stream);
hipError_t launch_resolve(const MapEntry *map, int64_t n_groups, const int64_t *ids, int64_t n,
                          int64_t *pos, hipStream_t stream);

// Ingestion batch in two launches: claim (map entries for every id, first/last occurrence,
// ranks of the new ids, and kUpsertCounts counts at upsert_counts(ws, n): n_new, n_rejected,
// n_unplaced, n_wide_authors, the scan's tile counter, waits that reached their bound),
// then finish: when the batch fits (nothing unplaced, no bounded wait given up and
// n_old + n_new <= capacity) scatter the rows and commit the map, otherwise roll the claim
// back. The decision is taken on the device from the counts.
constexpr int kUpsertCounts = 6;
constexpr int32_t kDefaultWaitPolls = 1 << 16;   // bound on each device-side wait of a batch
int64_t upsert_workspace_bytes(int64_t n);
int64_t *upsert_counts(void *workspace, int64_t n);
hipError_t launch_upsert_claim(MapEntry *map, int64_t n_groups, const int64_t *ids, int64_t n,
                               void *workspace, int32_t max_polls, hipStream_t stream);
hipError_t launch_upsert_finish(MapEntry *map, int64_t n, void *workspace, int64_t n_old,
                                int64_t capacity, const int64_t *author_in, const void *rows_in,
                                int32_t row_bytes, int64_t *author, int32_t *author32,
                                uint8_t *rows, hipStream_t stream);

}  // namespace ccj
