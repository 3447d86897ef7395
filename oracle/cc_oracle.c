/*
 * CPU oracle for the edge-feature join -- TEST INFRASTRUCTURE ONLY.
 *
 * Only the test suite, the smoke check and the benchmark's CPU-baseline leg load this file's
 * library. The product path never calls it; it shares no code, header or constant with the
 * device library.
 *
 * What it computes (Connected Content Retriever, §3.1, Eq. 1, extended to the full model-input
 * row and to many viewers):
 *
 *   For every candidate j of viewer v, with c = cand_idx[j]:
 *     if 0 <= c < n_docs:
 *       out[j][0 : Wd]                  = doc_rows[c]
 *       for each lookup l in [0, L):
 *         key  = (l == 0) ? author_id[c] : extra_keys[l-1][j]
 *         hit  = some i in [key_offsets[v], key_offsets[v+1]) has keys[i] == key
 *         out[j][Wd + l*We : Wd+(l+1)*We] = hit ? edge_rows[i_min] : default_row
 *         hit_mask[j*L + l] = hit
 *       (i_min is the smallest such i)
 *     else (an invalid position, the "-1" of the id-resolution map, §6.3.1 Eq. 6):
 *       doc segment = zero bytes, every edge segment = default_row, every hit bit = 0,
 *       and the candidate is counted in the returned invalid count.
 *   default_row == NULL means a row of zero bytes (the Zeros of Eq. 1 / Alg. 1 Step 4).
 *
 * Rows are opaque byte strings; nothing is converted, so the result is a pure copy and
 * equality is byte equality.
 *
 * Three interchangeable ways to find i_min (method argument):
 *   CCOR_LOWER_BOUND: textbook binary search for the leftmost position whose key is not less
 *                     than the query (the "searchsorted" of Alg. 1 Step 2), then the equality
 *                     test of Alg. 1 Step 3. Needs keys sorted ascending (signed int64).
 *   CCOR_SCAN:        the naive scan over all K records that §3.1 describes before Alg. 1;
 *                     first equal key wins. Works for any key order.
 *   CCOR_HASH:        open-addressing hash table from key to its first index, built per viewer
 *                     in index order. Works for any key order.
 * For sorted keys (duplicates allowed) all three return the same i_min.
 *
 * Also here: the stable per-viewer sort of Alg. 1 Step 1 (ccor_sort_affinity), the document-id
 * map of §6.3.1 Eq. 6 (ccor_resolve) and the sequential replay of ingestion batches of §6.2
 * (ccor_upsert).
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

enum { CCOR_LOWER_BOUND = 0, CCOR_SCAN = 1, CCOR_HASH = 2 };

/* Leftmost index in keys[0..n) whose value is >= x; n when every key is < x. */
static int64_t lower_bound(const int64_t *keys, int64_t n, int64_t x)
{
    int64_t lo = 0, hi = n;
    while (lo < hi) {
        int64_t mid = lo + (hi - lo) / 2;
        if (keys[mid] < x)
            lo = mid + 1;
        else
            hi = mid;
    }
    return lo;
}

/* Index of the first key equal to x, or -1. */
static int64_t find_by_lower_bound(const int64_t *keys, int64_t n, int64_t x)
{
    int64_t p = lower_bound(keys, n, x);
    if (p < n && keys[p] == x)
        return p;
    return -1;
}

static int64_t find_by_scan(const int64_t *keys, int64_t n, int64_t x)
{
    for (int64_t i = 0; i < n; i++)
        if (keys[i] == x)
            return i;
    return -1;
}

/* ---- hash table: key -> first index, linear probing, capacity a power of two ---- */
typedef struct {
    int64_t *key;
    int64_t *idx;      /* -1 marks an empty slot */
    uint64_t mask;
} table_t;

/* The 64-bit finalizer of MurmurHash3 (fmix64, Austin Appleby): a bijective mixer, so keys that
 * differ in any bit spread over the slots. */
static uint64_t mix64(uint64_t z)
{
    z ^= z >> 33;
    z *= 0xff51afd7ed558ccdULL;
    z ^= z >> 33;
    z *= 0xc4ceb9fe1a85ec53ULL;
    z ^= z >> 33;
    return z;
}

/* An empty table with room for at least n keys at load factor <= 1/2. */
static int table_init(table_t *t, int64_t n)
{
    uint64_t cap = 16;
    while (cap < (uint64_t)n * 2)
        cap <<= 1;
    t->key = (int64_t *)malloc(cap * sizeof(int64_t));
    t->idx = (int64_t *)malloc(cap * sizeof(int64_t));
    if (!t->key || !t->idx) {
        free(t->key);
        free(t->idx);
        return -1;
    }
    t->mask = cap - 1;
    for (uint64_t s = 0; s < cap; s++)
        t->idx[s] = -1;
    return 0;
}

/* Insert key -> i unless the key is present already (then the earlier index stays). */
static void table_insert(table_t *t, int64_t key, int64_t i)
{
    uint64_t s = mix64((uint64_t)key) & t->mask;
    while (t->idx[s] >= 0 && t->key[s] != key)
        s = (s + 1) & t->mask;
    if (t->idx[s] < 0) {          /* first occurrence keeps its index */
        t->key[s] = key;
        t->idx[s] = i;
    }
}

static int table_build(table_t *t, const int64_t *keys, int64_t n)
{
    if (table_init(t, n) != 0)
        return -1;
    for (int64_t i = 0; i < n; i++)
        table_insert(t, keys[i], i);
    return 0;
}

static int64_t table_find(const table_t *t, int64_t x)
{
    uint64_t s = mix64((uint64_t)x) & t->mask;
    while (t->idx[s] >= 0) {
        if (t->key[s] == x)
            return t->idx[s];
        s = (s + 1) & t->mask;
    }
    return -1;
}

static void table_free(table_t *t)
{
    free(t->key);
    free(t->idx);
}

/*
 * The join. Returns the number of invalid candidates, or -1 on an argument error
 * (null array where data is needed, negative sizes, out-of-range offsets).
 *
 * Layout: author_id[n_docs]; doc_rows[n_docs][doc_bytes]; cand_offsets[n_viewers+1] and
 * key_offsets[n_viewers+1] are running offsets into cand_idx / keys / edge_rows;
 * edge_rows[total_keys][edge_bytes]; extra_keys[(n_lookups-1) * total_cand] holds the
 * per-candidate keys of lookups 1.. in lookup-major order; out[total_cand][out_stride];
 * hit_mask[total_cand][n_lookups].
 */
int64_t ccor_join(int method,
                  int64_t n_docs, const int64_t *author_id, const uint8_t *doc_rows,
                  int64_t doc_bytes,
                  int64_t n_viewers, const int64_t *cand_offsets, const int64_t *cand_idx,
                  const int64_t *key_offsets, const int64_t *keys,
                  const uint8_t *edge_rows, int64_t edge_bytes,
                  const uint8_t *default_row,
                  int64_t n_lookups, const int64_t *extra_keys,
                  uint8_t *out, int64_t out_stride, int8_t *hit_mask)
{
    if (n_docs < 0 || doc_bytes < 0 || edge_bytes < 0 || n_viewers < 0 || n_lookups < 1)
        return -1;
    if (out_stride < doc_bytes + n_lookups * edge_bytes)
        return -1;
    if (n_viewers > 0 && (!cand_offsets || !key_offsets))
        return -1;
    int64_t total_cand = n_viewers > 0 ? cand_offsets[n_viewers] : 0;
    int64_t invalid = 0;

    for (int64_t v = 0; v < n_viewers; v++) {
        int64_t c0 = cand_offsets[v], c1 = cand_offsets[v + 1];
        int64_t k0 = key_offsets[v], k1 = key_offsets[v + 1];
        if (c0 < 0 || c1 < c0 || k0 < 0 || k1 < k0)
            return -1;
        const int64_t *vkeys = keys ? keys + k0 : NULL;
        int64_t K = k1 - k0;
        if (K > 0 && (!keys || !edge_rows))
            return -1;

        table_t table = {NULL, NULL, 0};
        if (method == CCOR_HASH && table_build(&table, vkeys, K) != 0)
            return -1;

        for (int64_t j = c0; j < c1; j++) {
            uint8_t *row = out + j * out_stride;
            int64_t c = cand_idx[j];
            int valid = (c >= 0 && c < n_docs);
            if (valid)
                memcpy(row, doc_rows + c * doc_bytes, (size_t)doc_bytes);
            else {
                memset(row, 0, (size_t)doc_bytes);
                invalid++;
            }
            for (int64_t l = 0; l < n_lookups; l++) {
                uint8_t *seg = row + doc_bytes + l * edge_bytes;
                int64_t i = -1;
                if (valid) {
                    int64_t key = (l == 0) ? author_id[c] : extra_keys[(l - 1) * total_cand + j];
                    if (method == CCOR_LOWER_BOUND)
                        i = find_by_lower_bound(vkeys, K, key);
                    else if (method == CCOR_SCAN)
                        i = find_by_scan(vkeys, K, key);
                    else
                        i = table_find(&table, key);
                }
                if (i >= 0)
                    memcpy(seg, edge_rows + (k0 + i) * edge_bytes, (size_t)edge_bytes);
                else if (default_row)
                    memcpy(seg, default_row, (size_t)edge_bytes);
                else
                    memset(seg, 0, (size_t)edge_bytes);
                hit_mask[j * n_lookups + l] = (int8_t)(i >= 0);
            }
        }
        if (method == CCOR_HASH)
            table_free(&table);
    }
    return invalid;
}

/*
 * Alg. 1 Step 1 (§3.1): sort each viewer's affinity records by author id (signed int64,
 * ascending) and move the feature rows with them. The sort is stable: records with equal ids
 * keep their input order, so the leftmost-equal-key rule of the join picks the record that came
 * first. Plain top-down merge sort of record indices, one viewer at a time.
 * Returns 0, or -1 on an argument error.
 */
static void merge_sort_idx(const int64_t *keys, int64_t *idx, int64_t *tmp, int64_t n)
{
    if (n < 2)
        return;
    int64_t h = n / 2;
    merge_sort_idx(keys, idx, tmp, h);
    merge_sort_idx(keys, idx + h, tmp, n - h);
    int64_t i = 0, j = h, k = 0;
    while (i < h && j < n) {
        if (keys[idx[j]] < keys[idx[i]])       /* strictly less: ties keep the left element */
            tmp[k++] = idx[j++];
        else
            tmp[k++] = idx[i++];
    }
    while (i < h)
        tmp[k++] = idx[i++];
    while (j < n)
        tmp[k++] = idx[j++];
    memcpy(idx, tmp, (size_t)n * sizeof(int64_t));
}

int ccor_sort_affinity(int64_t n_viewers, const int64_t *key_offsets, const int64_t *keys_in,
                       const uint8_t *rows_in, int64_t row_bytes, int64_t *keys_out,
                       uint8_t *rows_out)
{
    if (n_viewers < 0 || row_bytes < 0 || (n_viewers > 0 && !key_offsets))
        return -1;
    for (int64_t v = 0; v < n_viewers; v++) {
        int64_t k0 = key_offsets[v], k1 = key_offsets[v + 1];
        if (k0 < 0 || k1 < k0)
            return -1;
        int64_t K = k1 - k0;
        if (K == 0)
            continue;
        int64_t *idx = (int64_t *)malloc((size_t)K * sizeof(int64_t));
        int64_t *tmp = (int64_t *)malloc((size_t)K * sizeof(int64_t));
        if (!idx || !tmp) {
            free(idx);
            free(tmp);
            return -1;
        }
        for (int64_t i = 0; i < K; i++)
            idx[i] = i;
        merge_sort_idx(keys_in + k0, idx, tmp, K);
        for (int64_t i = 0; i < K; i++) {
            keys_out[k0 + i] = keys_in[k0 + idx[i]];
            memcpy(rows_out + (k0 + i) * row_bytes, rows_in + (k0 + idx[i]) * row_bytes,
                   (size_t)row_bytes);
        }
        free(idx);
        free(tmp);
    }
    return 0;
}

/*
 * Eq. 6 (§6.3.1): pos(q) = H[q] when q is a stored document id, else -1. The index is given as
 * the id stored at each position, index_ids[0, n_index) (ids unique), and H is built from it.
 * Returns 0, or -1 on an argument error.
 */
int ccor_resolve(int64_t n_index, const int64_t *index_ids, int64_t n_q, const int64_t *queries,
                 int64_t *pos_out)
{
    if (n_index < 0 || n_q < 0 || (n_index > 0 && !index_ids) || (n_q > 0 && (!queries || !pos_out)))
        return -1;
    table_t t;
    if (table_build(&t, index_ids, n_index) != 0)
        return -1;
    for (int64_t j = 0; j < n_q; j++)
        pos_out[j] = table_find(&t, queries[j]);
    table_free(&t);
    return 0;
}

/*
 * Ingestion into the index (§6.2, bootstrap protocol), as its sequential replay: the records of
 * a batch are applied one at a time in batch order. A stored id has its author id and row
 * overwritten in place; a new id takes the next free position (n_docs, n_docs + 1, ...) and is
 * added to H. The id INT64_MIN is reserved (it cannot be stored): such records are skipped and
 * counted in *n_rejected. A batch whose new ids would not fit in capacity changes nothing.
 *
 * State (caller-owned): ids_by_pos, author [capacity], rows [capacity][row_bytes], *n_docs.
 * Returns the number of new ids, -2 when the batch does not fit, or -1 on an argument error.
 */
int64_t ccor_upsert(int64_t capacity, int64_t *n_docs, int64_t *ids_by_pos, int64_t *author,
                    uint8_t *rows, int64_t row_bytes, int64_t n, const int64_t *ids,
                    const int64_t *authors_in, const uint8_t *rows_in, int64_t *n_rejected)
{
    if (!n_docs || *n_docs < 0 || *n_docs > capacity || n < 0 || row_bytes < 0 || !n_rejected)
        return -1;
    if (n > 0 && (!ids || !authors_in || !rows_in))
        return -1;
    table_t t;
    if (table_init(&t, *n_docs + n) != 0)
        return -1;
    for (int64_t p = 0; p < *n_docs; p++)
        table_insert(&t, ids_by_pos[p], p);
    /* count the distinct new ids first, so that a batch that does not fit changes nothing */
    int64_t n_new = 0, rejected = 0;
    table_t seen;
    if (table_init(&seen, n) != 0) {
        table_free(&t);
        return -1;
    }
    for (int64_t i = 0; i < n; i++) {
        if (ids[i] == INT64_MIN) {
            rejected++;
            continue;
        }
        if (table_find(&t, ids[i]) < 0 && table_find(&seen, ids[i]) < 0) {
            table_insert(&seen, ids[i], i);
            n_new++;
        }
    }
    table_free(&seen);
    if (*n_docs + n_new > capacity) {
        table_free(&t);
        return -2;
    }
    for (int64_t i = 0; i < n; i++) {
        if (ids[i] == INT64_MIN)
            continue;
        int64_t p = table_find(&t, ids[i]);
        if (p < 0) {
            p = (*n_docs)++;
            table_insert(&t, ids[i], p);
            ids_by_pos[p] = ids[i];
        }
        author[p] = authors_in[i];
        memcpy(rows + p * row_bytes, rows_in + i * row_bytes, (size_t)row_bytes);
    }
    table_free(&t);
    *n_rejected = rejected;
    return n_new;
}
