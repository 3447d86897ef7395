/*
 * cc_join.h -- C ABI of the MI355X edge-feature join library (libccjoin.so).
 *
 * The operation is the edge-feature join of Connected Content Retriever (§3.1, Eq. 1 and
 * Alg. 1): every candidate document carries an author id; the viewer's affinity records are
 * a sorted list of author ids with one feature row each; a candidate whose author id is in
 * the list receives that feature row, otherwise the zero row. The library fuses this with the
 * gather of the candidate's own document-feature row from a device-resident store (§6.3: the
 * document features live in GPU memory and are resolved by position), so that one call writes
 * the model-input slice
 *
 *      out[j] = [ doc_rows[cand_idx[j]] | edge row of lookup 0 | edge row of lookup 1 ... ]
 *
 * and a hit mask. All row data are opaque byte strings: the library never converts, rounds or
 * canonicalises a value (NaN payloads, signed zeros and subnormals are copied bit for bit).
 *
 * General conventions
 *   - Every per-call array is caller-owned device memory unless stated otherwise; it must
 *     stay alive until the work enqueued on `stream` has completed.
 *   - The join calls enqueue work on `stream` and return; they never synchronise and never
 *     allocate. Host-checkable argument errors return before anything is enqueued.
 *   - Data-dependent conditions that a check would need a synchronisation to see have
 *     defined, memory-safe outcomes instead of errors (see cc_join_batched).
 *   - No C++ exception crosses this interface.
 *   - A store is read-only for the joins: concurrent joins on one store, from any threads
 *     and streams, are safe. Ingestion (cc_store_upsert) is the one writer; it must not overlap
 *     any other call on the same store (the paper's read-write lock per index, §6.3.1: joins
 *     and id resolution hold the read side, an ingestion batch the write side).
 */
#ifndef CC_JOIN_H
#define CC_JOIN_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#if defined(__GNUC__) || defined(__clang__)
#define CC_API __attribute__((visibility("default")))
#else
#define CC_API
#endif

#ifdef __cplusplus
extern "C" {
#endif

typedef struct cc_store cc_store;   /* opaque; device-resident document store */

typedef enum cc_status {
    CC_OK = 0,
    CC_ERR_INVALID_ARGUMENT = 1,   /* a host-checkable argument is wrong; nothing enqueued   */
    CC_ERR_OUT_OF_MEMORY = 2,      /* device allocation failed (store creation only)        */
    CC_ERR_DEVICE = 3,             /* a HIP call failed; see cc_last_device_error()         */
    CC_ERR_UNSORTED_KEYS = 4,      /* only from cc_validate_keys                            */
    CC_ERR_NOT_SUPPORTED = 5,      /* no usable gfx950 device, or a store without an id map */
    CC_ERR_STORE_FULL = 6,         /* an ingestion batch does not fit; the store is unchanged */
    CC_ERR_TOO_LARGE = 7,          /* a size exceeds the fixed scratch of an allocation-free
                                      entry point; nothing enqueued                          */
    CC_ERR_TIMEOUT = 8             /* a bounded wait between the workgroups of an ingestion
                                      batch gave up; the batch was rolled back, the store is
                                      unchanged                                              */
} cc_status;

/* Where cc_store_create reads its source arrays from. */
#define CC_SRC_HOST 1u
#define CC_SRC_DEVICE 2u

/*
 * cc_store_create -- copy a document store into library-owned device memory.
 *
 * §6.3 (Eq. 5): each document's feature tensors are stored in GPU memory and addressed by the
 * document's position. Position p holds author_ids[p] and the row doc_rows[p].
 *
 *   out_store      receives the new store handle (set to NULL on error).
 *   n_docs         number of documents, >= 0.
 *   author_ids     [n_docs] int64 author id of each document (any int64 value).
 *   doc_rows       [n_docs][doc_row_bytes] row-major document-feature rows.
 *   doc_row_bytes  bytes per row; a positive multiple of 16, at most 2^20 (1 MiB).
 *   flags          CC_SRC_HOST (sources are host memory) or CC_SRC_DEVICE (device memory).
 *   stream         the copies are enqueued on this stream, which is synchronised once before
 *                  the call returns (also to learn whether every author id fits in 32 bits);
 *                  the sources may then be freed and any stream may use the store.
 *
 * The store is created on the current HIP device and stays on it. Layout in HBM: author ids
 * as one int64 column, rows as one row-major array, both 256-byte aligned, plus an 8-byte
 * counter of invalid candidate positions seen by joins. When every author id fits in 32 bits
 * the store also keeps a 32-bit copy of the author column, which the joins read instead
 * (cc_store_layout reports it): the column then spans half as many cache lines, so more of
 * it stays in the L2 cache. Results never depend on it.
 * Errors: CC_ERR_INVALID_ARGUMENT, CC_ERR_OUT_OF_MEMORY (nothing leaked), CC_ERR_DEVICE,
 * CC_ERR_NOT_SUPPORTED.
 */
CC_API cc_status cc_store_create(cc_store **out_store, int64_t n_docs, const int64_t *author_ids,
                          const void *doc_rows, int32_t doc_row_bytes, uint32_t flags,
                          hipStream_t stream);

/* Free a store. The caller guarantees that no join using it is still in flight.
 * NULL is accepted and ignored. */
CC_API cc_status cc_store_destroy(cc_store *store);

/* Report a store's size. Either output pointer may be NULL. */
CC_API cc_status cc_store_info(const cc_store *store, int64_t *n_docs, int32_t *doc_row_bytes);

/*
 * cc_store_layout -- how a store holds its author ids and how many documents it can hold.
 *   author_id_bytes  4 when every stored author id fits in 32 bits (the store then keeps a
 *                    32-bit copy of the column, which the joins read: a 128-byte cache line
 *                    holds 32 ids instead of 16), else 8.
 *   capacity         rows allocated (n_docs for a store from cc_store_create).
 * Either output may be NULL. Errors: CC_ERR_INVALID_ARGUMENT.
 */
CC_API cc_status cc_store_layout(const cc_store *store, int32_t *author_id_bytes,
                                 int64_t *capacity);

/* Read the number of invalid candidate positions (outside [0, n_docs)) that joins on this
 * store have met since creation or the last reset. The id -> position resolution of §6.3.1
 * (Eq. 6) returns -1 for a document id that is not in the index; such positions reach the join
 * as candidates and are counted here (their output rows are defined in cc_join_batched).
 * Synchronises `stream` (debug/metrics). Errors: CC_ERR_INVALID_ARGUMENT, CC_ERR_DEVICE. */
CC_API cc_status cc_store_invalid_count(const cc_store *store, int64_t *count, hipStream_t stream);

/* Reset that counter to zero, ordered on `stream` (no synchronisation). A kernel clears it, so
 * the call may be captured into a HIP graph. Errors: CC_ERR_INVALID_ARGUMENT, CC_ERR_DEVICE. */
CC_API cc_status cc_store_reset_invalid_count(cc_store *store, hipStream_t stream);

/*
 * cc_join -- one viewer: Eq. 1 for N candidates against K affinity records (§3.1, Alg. 1
 * Steps 2-4; the keys arrive already sorted, i.e. after Alg. 1 Step 1).
 *
 *   store          document store (author id and doc row per position).
 *   cand_idx       [n_cand] int64 candidate positions in the store (the output of the
 *                  id -> position resolution of §6.3.1, where -1 means "not found").
 *   n_cand         number of candidates, >= 0.
 *   edge_keys      [n_keys] int64 viewer's affinity author ids, ascending in signed order.
 *   n_keys         K >= 0; K = 0 makes every candidate a miss.
 *   edge_feats     [n_keys][edge_row_bytes] feature row of each key (row i belongs to key i).
 *   edge_row_bytes bytes per edge row; a positive multiple of 16, at most 2^20 (1 MiB).
 *   default_row    [edge_row_bytes] row written on a miss, or NULL for zero bytes.
 *   out            [n_cand][out_row_stride] output; row j gets
 *                  [doc row (doc_row_bytes) | edge row or default (edge_row_bytes)];
 *                  bytes past that width in each row are not written.
 *   out_row_stride bytes between output rows; a multiple of 16, >= doc_row_bytes +
 *                  edge_row_bytes.
 *   hit_mask       [n_cand] int8: 1 when the author id was found, else 0.
 *   stream         work is enqueued here.
 *
 * Alignment: edge_feats, default_row and out must be 16-byte aligned; cand_idx and
 * edge_keys 8-byte aligned. This is cc_join_batched with one viewer and one lookup.
 */
CC_API cc_status cc_join(const cc_store *store,
                  const int64_t *cand_idx, int64_t n_cand,
                  const int64_t *edge_keys, int64_t n_keys,
                  const void *edge_feats, int32_t edge_row_bytes,
                  const void *default_row,
                  void *out, int64_t out_row_stride,
                  int8_t *hit_mask,
                  hipStream_t stream);

/*
 * cc_join_batched -- B viewers in one launch, in CSR form (Alg. 1 is stated for a batch of B
 * requests; ragged sizes are kept as offsets instead of padding), with one or two lookups per
 * candidate.
 *
 *   n_viewers      B >= 0.
 *   cand_offsets   [B+1] int64 device: viewer v owns candidates [cand_offsets[v],
 *                  cand_offsets[v+1]); cand_offsets[0] = 0, non-decreasing,
 *                  cand_offsets[B] = total_cand.
 *   cand_idx       [total_cand] int64 candidate positions.
 *   total_cand     host copy of cand_offsets[B].
 *   key_offsets    [B+1] int64 device: viewer v owns keys/edge rows [key_offsets[v],
 *                  key_offsets[v+1]); same rules, key_offsets[B] = total_keys.
 *   edge_keys      [total_keys] int64, ascending within each viewer.
 *   total_keys     host copy of key_offsets[B].
 *   edge_feats     [total_keys][edge_row_bytes].
 *   default_row    [edge_row_bytes] or NULL (zero bytes).
 *   n_lookups      L in {1, 2}. Lookup 0 uses the store's author id of the candidate; lookup 1
 *                  uses extra_keys[0][j] (e.g. the first-degree member who engaged with the
 *                  post). Both search the same viewer's keys.
 *   extra_keys     host array of L-1 device pointers, each [total_cand] int64; NULL when L=1.
 *   out            [total_cand][out_row_stride]; row j = [doc row | lookup 0 row | lookup 1
 *                  row]; out_row_stride is a multiple of 16 and >= doc_row_bytes +
 *                  L * edge_row_bytes.
 *   hit_mask       [total_cand][L] int8.
 * out and hit_mask must not overlap each other or any input (checked: CC_ERR_INVALID_ARGUMENT).
 *
 * Defined outcomes for data the host cannot check without synchronising:
 *   - cand_idx[j] outside [0, n_docs): doc segment = zero bytes, every edge segment = the
 *     default row, hit bits 0, and the store's invalid counter is incremented.
 *   - Keys that are non-decreasing with repeats: the leftmost equal key's row is used.
 *   - Keys that are not sorted, or offsets that break the rules above: the result is
 *     unspecified but every memory access stays inside the arrays whose sizes total_cand and
 *     total_keys describe (offsets are clamped to those sizes).
 * Errors: CC_ERR_INVALID_ARGUMENT (null or misaligned pointers, bad sizes, L not in {1,2}),
 * CC_ERR_DEVICE (the launch failed).
 */
CC_API cc_status cc_join_batched(const cc_store *store, int32_t n_viewers,
                          const int64_t *cand_offsets, const int64_t *cand_idx,
                          int64_t total_cand,
                          const int64_t *key_offsets, const int64_t *edge_keys,
                          int64_t total_keys,
                          const void *edge_feats, int32_t edge_row_bytes,
                          const void *default_row,
                          int32_t n_lookups, const int64_t *const *extra_keys,
                          void *out, int64_t out_row_stride, int8_t *hit_mask,
                          hipStream_t stream);

/*
 * cc_join_batched_authors -- cc_join_batched with each candidate's author id supplied by the
 * caller, the input form of Alg. 1 (§3.1: every candidate document arrives with its author
 * id), in place of the store's author column at the candidate's position.
 *   author_ids     [total_cand] int64 device, 8-byte aligned, not overlapping an output:
 *                  lookup 0 searches author_ids[j] for candidate j. The doc row still comes
 *                  from the store at cand_idx[j]; a position outside [0, n_docs) still gives
 *                  the zero doc segment, default edge segments and hit bits 0 (its author id
 *                  is not looked up) and is counted as invalid.
 * Other arguments, alignment rules, output and errors as in cc_join_batched; author_ids may be
 * NULL only when total_cand == 0.
 */
CC_API cc_status cc_join_batched_authors(const cc_store *store, int32_t n_viewers,
                                         const int64_t *cand_offsets, const int64_t *cand_idx,
                                         const int64_t *author_ids, int64_t total_cand,
                                         const int64_t *key_offsets, const int64_t *edge_keys,
                                         int64_t total_keys,
                                         const void *edge_feats, int32_t edge_row_bytes,
                                         const void *default_row,
                                         int32_t n_lookups, const int64_t *const *extra_keys,
                                         void *out, int64_t out_row_stride, int8_t *hit_mask,
                                         hipStream_t stream);

/*
 * cc_join_batched_padded -- cc_join_batched writing the padded batch layout of §6.3 (batching
 * and padding for variable-length requests, where requests with n_v candidates are scattered
 * into one [B, n_max, features] tensor and padded slots are masked downstream).
 *
 * Viewer v's candidate i (i < min(n_v, n_max)) is written to row v * n_max + i of `out` and
 * `hit_mask`; every other slot (a pad slot) gets zero bytes over the row width
 * (doc_row_bytes + n_lookups * edge_row_bytes) and hit bits 0. valid_mask[v * n_max + i] is 1
 * for a candidate's slot and 0 for a pad slot. A viewer with more than n_max candidates keeps
 * its first n_max; the others produce no output and are not counted as invalid.
 *
 *   n_max          slots per viewer (>= 1 when n_viewers > 0).
 *   out            [n_viewers][n_max][out_row_stride]
 *   hit_mask       [n_viewers][n_max][n_lookups] int8
 *   valid_mask     [n_viewers][n_max] int8
 * Other arguments, alignment rules and errors as in cc_join_batched.
 */
CC_API cc_status cc_join_batched_padded(const cc_store *store, int32_t n_viewers,
                                        const int64_t *cand_offsets, const int64_t *cand_idx,
                                        int64_t total_cand,
                                        const int64_t *key_offsets, const int64_t *edge_keys,
                                        int64_t total_keys,
                                        const void *edge_feats, int32_t edge_row_bytes,
                                        const void *default_row,
                                        int32_t n_lookups, const int64_t *const *extra_keys,
                                        int64_t n_max, void *out, int64_t out_row_stride,
                                        int8_t *hit_mask, int8_t *valid_mask,
                                        hipStream_t stream);

/*
 * Launch tuning for cc_join_batched_tuned. A zero field means "choose automatically".
 *   fence_stride   power of two >= 1: the search keeps every fence_stride-th key of a viewer
 *                  in LDS and finishes with one read of the keys between two fences
 *                  (1 = the whole key list in LDS).
 *   lds_keys       capacity of the LDS key table, in keys (<= 18432, i.e. 144 KiB).
 *   workgroups     number of workgroups of the launch (<= 2^30; rounded up to a multiple of 8).
 * Results never depend on these values, only speed does.
 */
typedef struct cc_tuning {
    int32_t fence_stride;
    int32_t lds_keys;
    int32_t workgroups;
    int32_t reserved;
} cc_tuning;

/* cc_join_batched with explicit launch tuning (NULL = automatic). Same contract. */
CC_API cc_status cc_join_batched_tuned(const cc_store *store, int32_t n_viewers,
                                const int64_t *cand_offsets, const int64_t *cand_idx,
                                int64_t total_cand,
                                const int64_t *key_offsets, const int64_t *edge_keys,
                                int64_t total_keys,
                                const void *edge_feats, int32_t edge_row_bytes,
                                const void *default_row,
                                int32_t n_lookups, const int64_t *const *extra_keys,
                                void *out, int64_t out_row_stride, int8_t *hit_mask,
                                const cc_tuning *tuning, hipStream_t stream);

/*
 * cc_store_create_indexed -- an empty document store with an id map, for ingestion (§6.2) and
 * document-id resolution (§6.3.1, Eq. 6).
 *
 *   out_store      receives the new store handle (set to NULL on error).
 *   capacity       documents the store can hold, 0 <= capacity <= 2^31 - 1. Rows, author ids
 *                  and the id map are allocated for this many documents up front.
 *   doc_row_bytes  bytes per document row; a positive multiple of 16, at most 2^20 (1 MiB).
 *   stream         the map is cleared on this stream, which is synchronised before the call
 *                  returns; any stream may then use the store.
 *
 * Layout in HBM: author ids [capacity] int64, rows [capacity][doc_row_bytes], and the id map:
 * an open-addressing table of 16-byte entries {id, position} in 64-byte probe groups, sized
 * to at least twice the capacity (load factor <= 1/2), so that inserts never rebuild it.
 * The store starts with n_docs = 0; cc_store_upsert fills it. All join entry points accept it.
 * Errors: CC_ERR_INVALID_ARGUMENT, CC_ERR_OUT_OF_MEMORY, CC_ERR_NOT_SUPPORTED, CC_ERR_DEVICE.
 */
CC_API cc_status cc_store_create_indexed(cc_store **out_store, int64_t capacity,
                                         int32_t doc_row_bytes, hipStream_t stream);

/*
 * cc_store_upsert -- apply one ingestion batch (§6.2, bootstrap protocol: identify new and
 * stored ids, prefix-sum positions for the new ones, scatter the rows, update the map only
 * after the rows are written).
 *
 * The result is that of applying the records one at a time in batch order: a stored id has
 * its author id and row overwritten in place (the last record with that id wins); a new id
 * takes the next free position n_docs, n_docs + 1, ... in order of its first record. The id
 * INT64_MIN is reserved: its records are skipped and counted in *n_rejected.
 *
 *   store          a store from cc_store_create_indexed (else CC_ERR_NOT_SUPPORTED).
 *   n_records      records in the batch, 0 <= n_records <= 2^30.
 *   doc_ids        [n_records] int64 device, 8-byte aligned.
 *   author_ids     [n_records] int64 device, 8-byte aligned.
 *   doc_rows       [n_records][doc_row_bytes] device, 16-byte aligned.
 *   workspace      device scratch of cc_upsert_workspace_bytes(n_records) bytes, 16-byte
 *                  aligned, caller-owned, not overlapping the inputs.
 *   n_new, n_rejected  host outputs (may be NULL): ids added, records skipped.
 *
 * Synchronises `stream` once, at the end (whether the batch fits is decided on the device, and
 * the rows, the map or the rollback are all enqueued before the wait). When the new ids do not
 * fit in the remaining capacity, or an id cannot be placed within the map's probe
 * limit (64 groups; not expected below load 1/2), the batch is undone and CC_ERR_STORE_FULL is
 * returned with the store unchanged. Errors: CC_ERR_INVALID_ARGUMENT, CC_ERR_NOT_SUPPORTED,
 * CC_ERR_STORE_FULL, CC_ERR_TIMEOUT (a bounded device-side wait gave up, see
 * cc_set_ingestion_wait_limit; the batch is undone and the store unchanged), CC_ERR_DEVICE.
 */
/*
 * cc_set_ingestion_wait_limit -- the bound, in polls (each about a microsecond), on every wait
 * inside an ingestion batch: a record waiting for the store that put its id into the map in
 * the same batch, and a scan tile waiting for the counts of earlier tiles. Those waits are on
 * work of running workgroups and end within microseconds; the bound keeps every wave's exit
 * certain. A batch in which a wait gives up is rolled back and cc_store_upsert returns
 * CC_ERR_TIMEOUT with the store unchanged. For tests of that path: 0 makes every such wait give
 * up at once (a batch that repeats an id new to the store is then always refused). polls < 0
 * restores the default (65,536). Process-wide; applies to batches enqueued afterwards.
 * Returns CC_OK.
 */
CC_API cc_status cc_set_ingestion_wait_limit(int32_t polls);
/* Workspace bytes cc_store_upsert needs for n_records; 0 when n_records <= 0 or > 2^30 (a
 * batch the upsert rejects). */
CC_API int64_t cc_upsert_workspace_bytes(int64_t n_records);
CC_API cc_status cc_store_upsert(cc_store *store, int64_t n_records, const int64_t *doc_ids,
                                 const int64_t *author_ids, const void *doc_rows, void *workspace,
                                 int64_t workspace_bytes, int64_t *n_new, int64_t *n_rejected,
                                 hipStream_t stream);

/*
 * cc_store_read -- copy positions [first, first + count) of a store out: author ids into
 * author_out [count] int64 and rows into rows_out [count][doc_row_bytes] (either may be NULL).
 * Device buffers, 8- and 16-byte aligned. Requires 0 <= first, first + count <= n_docs.
 * Asynchronous on `stream`; must not overlap an ingestion batch. Errors:
 * CC_ERR_INVALID_ARGUMENT, CC_ERR_DEVICE.
 */
CC_API cc_status cc_store_read(const cc_store *store, int64_t first, int64_t count,
                               int64_t *author_out, void *rows_out, hipStream_t stream);

/*
 * cc_resolve_ids -- document id to store position (§6.3.1, Eq. 6): positions[i] = the
 * position of doc_ids[i] in the store, or -1 when the id is not stored. The output is what
 * cc_join / cc_join_batched take as cand_idx (a -1 there yields the defined invalid row).
 *
 *   store          a store from cc_store_create_indexed (else CC_ERR_NOT_SUPPORTED).
 *   doc_ids        [n] int64 device, 8-byte aligned.
 *   positions      [n] int64 device, 8-byte aligned; may be doc_ids itself (in place), must
 *                  not overlap it otherwise.
 * Asynchronous on `stream`; never allocates. Errors: CC_ERR_INVALID_ARGUMENT,
 * CC_ERR_NOT_SUPPORTED, CC_ERR_DEVICE.
 */
CC_API cc_status cc_resolve_ids(const cc_store *store, const int64_t *doc_ids, int64_t n,
                                int64_t *positions, hipStream_t stream);

/*
 * cc_sort_affinity -- Alg. 1 Step 1 (§3.1) on the device: sort each viewer's affinity records
 * by author id (signed int64, ascending) and move each record's feature row with it. The sort
 * is stable: records with equal ids keep their input order, so the join's leftmost-equal-key
 * rule picks the record that came first (the reading of Alg. 1's unspecified tie order).
 *
 *   n_viewers      B >= 0.
 *   key_offsets    [B+1] int64 device, CSR offsets as in cc_join_batched (records of viewer v
 *                  are [key_offsets[v], key_offsets[v+1]); sorted within that range).
 *   keys_in        [total_keys] int64 device, any order within a viewer.
 *   rows_in        [total_keys][row_bytes] device.
 *   row_bytes      positive multiple of 16, at most 2^20 (1 MiB).
 *   total_keys     host copy of key_offsets[B]; < 2^32.
 *   max_keys       host upper bound on any one viewer's record count (fewer merge rounds and
 *                  narrower sort elements), or 0 if unknown. A viewer with more records than a
 *                  nonzero max_keys is not sorted: its keys and rows are copied to the output
 *                  in their input order (cc_validate_keys reports it unless its input was
 *                  already in order); every other viewer is sorted as usual.
 *   keys_out       [total_keys] int64 device (sorted keys, same CSR offsets).
 *   rows_out       [total_keys][row_bytes] device (rows in the sorted order).
 *   workspace      device scratch of at least cc_sort_workspace_bytes(total_keys, n_viewers)
 *                  bytes, 16-byte aligned, owned by the caller (the library allocates nothing).
 * Outputs must not overlap inputs or the workspace. Alignment: rows 16 bytes, keys and
 * offsets 8 bytes. Offsets that break the CSR rules give unspecified output, but they are
 * clamped to [0, total_keys] and every access stays inside the buffers. Asynchronous on
 * `stream`. Errors: CC_ERR_INVALID_ARGUMENT, CC_ERR_DEVICE.
 */
/* Workspace bytes cc_sort_affinity needs; 0 when there is nothing to sort or total_keys >=
 * 2^32 (counts the sort rejects). */
CC_API int64_t cc_sort_workspace_bytes(int64_t total_keys, int32_t n_viewers);
CC_API cc_status cc_sort_affinity(int32_t n_viewers, const int64_t *key_offsets,
                                  const int64_t *keys_in, const void *rows_in, int32_t row_bytes,
                                  int64_t total_keys, int64_t max_keys, int64_t *keys_out,
                                  void *rows_out, void *workspace, int64_t workspace_bytes,
                                  hipStream_t stream);

/*
 * cc_sort_affinity_method -- cc_sort_affinity with the sorting method named by the caller, and
 * an optional bound on the keys' span (cc_sort_affinity is CC_SORT_AUTO with key_bits 0). Every
 * method gives the same output; they differ in speed:
 *   CC_SORT_MERGE  per-tile sorts in LDS, then merge rounds within each viewer (a number of
 *                  kernels that grows with log2 of the largest viewer); the last round writes
 *                  the keys and copies the rows. Fewer launches: the faster method for small
 *                  calls.
 *   CC_SORT_RADIX  least-significant-digit radix passes of up to 9 bits over the span of the
 *                  call's keys (decoupled look-back between a viewer's tiles), then one gather
 *                  of the rows. Moves fewer bytes per record: the faster method for large calls.
 *                  A tile waits only for earlier tiles held by running workgroups, with a bound
 *                  of 8,192 polls so that every wave exits; a wait that reached it (not
 *                  expected) would leave the call's output undefined, every output row still a
 *                  copy of one of the call's input rows (memory-safe).
 *   CC_SORT_AUTO   CC_SORT_RADIX from CC_SORT_RADIX_MIN_RECORDS records on, else CC_SORT_MERGE.
 *   key_bits       0, or an upper bound on the bit length of (largest key - smallest key) over
 *                  the call (at most 64): the radix method then launches only the passes such a
 *                  span needs (ceil(key_bits / 9), e.g. 3 for author ids below 2^27), where it
 *                  otherwise launches all 8 and lets the unneeded ones return at once. A call
 *                  whose keys span more bits than key_bits still writes, for every viewer, a
 *                  permutation of its records with their rows (memory-safe), in an order that
 *                  is then unspecified (cc_validate_keys flags it). The merge method ignores
 *                  key_bits.
 * Other arguments, the workspace and the errors are those of cc_sort_affinity; a method other
 * than these three, or key_bits outside [0, 64], is CC_ERR_INVALID_ARGUMENT.
 */
#define CC_SORT_AUTO 0
#define CC_SORT_MERGE 1
#define CC_SORT_RADIX 2
#define CC_SORT_RADIX_MIN_RECORDS (1 << 20)
CC_API cc_status cc_sort_affinity_method(int32_t method, int32_t key_bits, int32_t n_viewers,
                                         const int64_t *key_offsets, const int64_t *keys_in,
                                         const void *rows_in, int32_t row_bytes,
                                         int64_t total_keys, int64_t max_keys, int64_t *keys_out,
                                         void *rows_out, void *workspace, int64_t workspace_bytes,
                                         hipStream_t stream);

/*
 * cc_sort_affinity_noalloc -- cc_sort_affinity for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, hosts that forbid allocation): the same
 * sort, whose workspace is a fixed device array that the library holds on each device it runs
 * on until the process ends, instead of a caller-provided buffer. The call allocates nothing
 * and never synchronises; its first call on a device resolves that device's array once.
 *
 * Limits: total_keys <= CC_SORT_NOALLOC_MAX_RECORDS and n_viewers <=
 * CC_SORT_NOALLOC_MAX_VIEWERS; larger calls return CC_ERR_TOO_LARGE before anything is
 * enqueued. The array is shared by every call on one device and keeps the last call's
 * contents (nothing in it needs clearing between calls): calls that overlap on one device,
 * from any threads or streams, race and must be serialised by the caller.
 * Other arguments, the result and the errors are those of cc_sort_affinity, on the current
 * HIP device.
 */
#define CC_SORT_NOALLOC_MAX_RECORDS (1 << 20)
#define CC_SORT_NOALLOC_MAX_VIEWERS (1 << 16)
CC_API cc_status cc_sort_affinity_noalloc(int32_t n_viewers, const int64_t *key_offsets,
                                          const int64_t *keys_in, const void *rows_in,
                                          int32_t row_bytes, int64_t total_keys,
                                          int64_t max_keys, int64_t *keys_out, void *rows_out,
                                          hipStream_t stream);

/*
 * cc_validate_keys -- debug helper: check that each viewer's keys are strictly increasing
 * (the precondition under which the join result is unique, §3.1 Alg. 1 Step 1 output).
 * Synchronises `stream`. Returns CC_OK, or CC_ERR_UNSORTED_KEYS with *first_bad_viewer set to
 * the lowest offending viewer (otherwise it is set to -1). Offsets must satisfy the rules of
 * cc_join_batched (they are clamped to total_keys). The result flag lives in an 8-byte device
 * buffer that the library allocates on the first call per device and keeps; calls are
 * serialised by the library (one at a time per process).
 */
CC_API cc_status cc_validate_keys(const int64_t *key_offsets, const int64_t *edge_keys,
                           int32_t n_viewers, int64_t total_keys, int64_t *first_bad_viewer,
                           hipStream_t stream);

/* Static string naming a status code. Takes any int (a cc_status converts implicitly): a
 * value that names no status gives "CC_UNKNOWN_STATUS". */
CC_API const char *cc_status_string(int status);

/* The hipError_t of the last CC_ERR_DEVICE returned on the calling thread (0 if none). */
CC_API int cc_last_device_error(void);

#ifdef __cplusplus
}
#endif

#endif /* CC_JOIN_H */
