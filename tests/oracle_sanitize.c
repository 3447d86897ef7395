/*
 * Memory and undefined-behaviour check of the CPU oracle (test infrastructure).
 *
 * Built with gcc's address and undefined-behaviour sanitizers together with
 * oracle/cc_oracle.c by tests/test_oracle_sanitizers.py. Every buffer is allocated at its exact
 * size, so a read or write one element past any array stops the program. The cases also
 * cross-check the oracle's parts against each other and against plain loops written here:
 *   - the join's three search methods give byte-identical rows, hit bits and invalid counts,
 *     and the hit bits match a membership loop (Eq. 1);
 *   - the sort is ordered and stable, and moves each record's row with its key (Alg. 1 Step 1);
 *   - resolution returns each stored id's position and -1 for absent ids (Eq. 6);
 *   - ingestion matches a replay over plain arrays, including repeats, the reserved id and a
 *     batch that does not fit (§6.2).
 * Prints "ok" and exits 0, or names the failed check and exits 1.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int64_t ccor_join(int method, int64_t n_docs, const int64_t *author_id, const uint8_t *doc_rows,
                  int64_t doc_bytes, int64_t n_viewers, const int64_t *cand_offsets,
                  const int64_t *cand_idx, const int64_t *key_offsets, const int64_t *keys,
                  const uint8_t *edge_rows, int64_t edge_bytes, const uint8_t *default_row,
                  int64_t n_lookups, const int64_t *extra_keys, uint8_t *out, int64_t out_stride,
                  int8_t *hit_mask);
int ccor_sort_affinity(int64_t n_viewers, const int64_t *key_offsets, const int64_t *keys_in,
                       const uint8_t *rows_in, int64_t row_bytes, int64_t *keys_out,
                       uint8_t *rows_out);
int ccor_resolve(int64_t n_index, const int64_t *index_ids, int64_t n_q, const int64_t *queries,
                 int64_t *pos_out);
int64_t ccor_upsert(int64_t capacity, int64_t *n_docs, int64_t *ids_by_pos, int64_t *author,
                    uint8_t *rows, int64_t row_bytes, int64_t n, const int64_t *ids,
                    const int64_t *authors_in, const uint8_t *rows_in, int64_t *n_rejected);

static uint64_t rng_state;

static uint64_t rnd(void)   /* xorshift64* */
{
    rng_state ^= rng_state >> 12;
    rng_state ^= rng_state << 25;
    rng_state ^= rng_state >> 27;
    return rng_state * 0x2545F4914F6CDD1DULL;
}

static int64_t ri(int64_t lo, int64_t hi)   /* uniform in [lo, hi] */
{
    return lo + (int64_t)(rnd() % (uint64_t)(hi - lo + 1));
}

/* Exact-size allocation; a zero-size request still returns a distinct pointer. */
static void *xmalloc(size_t n)
{
    void *p = malloc(n ? n : 1);
    if (!p) {
        fprintf(stderr, "out of memory\n");
        exit(2);
    }
    return p;
}

static void fill(uint8_t *p, size_t n)
{
    for (size_t i = 0; i < n; i++)
        p[i] = (uint8_t)rnd();
}

#define CHECK(cond, what)                                                     \
    do {                                                                      \
        if (!(cond)) {                                                        \
            fprintf(stderr, "FAILED: %s (case %d)\n", what, case_no);         \
            exit(1);                                                          \
        }                                                                     \
    } while (0)

static int case_no;

static int cmp_i64(const void *a, const void *b)
{
    int64_t x = *(const int64_t *)a, y = *(const int64_t *)b;
    return (x > y) - (x < y);
}

/* A key drawn from a small pool, so that lookups hit; the pool includes the int64 extremes. */
static int64_t pool_key(void)
{
    switch (ri(0, 9)) {
    case 0: return INT64_MIN;
    case 1: return INT64_MAX;
    case 2: return -ri(1, 5);
    default: return ri(0, 30);
    }
}

static void join_case(void)
{
    const int64_t n_docs = ri(0, 40), db = 16 * ri(0, 2), eb = 16 * ri(0, 2);
    const int64_t B = ri(0, 4), L = ri(1, 2);
    int64_t *author = xmalloc((size_t)n_docs * 8);
    uint8_t *docs = xmalloc((size_t)(n_docs * db));
    for (int64_t i = 0; i < n_docs; i++)
        author[i] = pool_key();
    fill(docs, (size_t)(n_docs * db));
    int64_t *co = xmalloc((size_t)(B + 1) * 8), *ko = xmalloc((size_t)(B + 1) * 8);
    co[0] = ko[0] = 0;
    for (int64_t v = 0; v < B; v++) {
        co[v + 1] = co[v] + ri(0, 30);
        ko[v + 1] = ko[v] + (ri(0, 4) == 0 ? 0 : ri(1, 12));
    }
    const int64_t nc = co[B], nk = ko[B];
    int64_t *cand = xmalloc((size_t)nc * 8), *keys = xmalloc((size_t)nk * 8);
    int64_t *extra = xmalloc((size_t)((L - 1) * nc) * 8);
    uint8_t *edge = xmalloc((size_t)(nk * eb)), *def = xmalloc((size_t)eb);
    for (int64_t j = 0; j < nc; j++)
        cand[j] = ri(-2, n_docs + 1);
    for (int64_t i = 0; i < nk; i++)
        keys[i] = pool_key();
    for (int64_t v = 0; v < B; v++)   /* sorted per viewer, duplicates allowed */
        qsort(keys + ko[v], (size_t)(ko[v + 1] - ko[v]), 8, cmp_i64);
    for (int64_t j = 0; j < (L - 1) * nc; j++)
        extra[j] = pool_key();
    fill(edge, (size_t)(nk * eb));
    fill(def, (size_t)eb);
    const uint8_t *dflt = ri(0, 1) ? def : NULL;
    const int64_t stride = db + L * eb + 16 * ri(0, 1);
    uint8_t *out[3];
    int8_t *hit[3];
    int64_t inv[3];
    for (int m = 0; m < 3; m++) {
        out[m] = xmalloc((size_t)(nc * stride));
        hit[m] = xmalloc((size_t)(nc * L));
        memset(out[m], 0xA5, (size_t)(nc * stride));
        inv[m] = ccor_join(m, n_docs, author, docs, db, B, co, cand, ko, keys, edge, eb, dflt, L,
                           extra, out[m], stride, hit[m]);
        CHECK(inv[m] >= 0, "join returned an error");
    }
    for (int m = 1; m < 3; m++) {
        CHECK(inv[m] == inv[0], "invalid counts differ between methods");
        CHECK(memcmp(out[m], out[0], (size_t)(nc * stride)) == 0, "rows differ between methods");
        CHECK(memcmp(hit[m], hit[0], (size_t)(nc * L)) == 0, "hit bits differ between methods");
    }
    int64_t n_inv = 0;
    for (int64_t v = 0; v < B; v++) {
        for (int64_t j = co[v]; j < co[v + 1]; j++) {
            const int64_t c = cand[j];
            const int ok = c >= 0 && c < n_docs;
            n_inv += !ok;
            for (int64_t l = 0; l < L; l++) {
                int member = 0;
                if (ok) {
                    const int64_t x = l == 0 ? author[c] : extra[(l - 1) * nc + j];
                    for (int64_t i = ko[v]; i < ko[v + 1]; i++)
                        member |= keys[i] == x;
                }
                CHECK(hit[0][j * L + l] == member, "hit bit disagrees with membership");
            }
        }
    }
    CHECK(n_inv == inv[0], "invalid count disagrees with a direct count");
    for (int m = 0; m < 3; m++) {
        free(out[m]);
        free(hit[m]);
    }
    free(author); free(docs); free(co); free(ko); free(cand); free(keys); free(extra);
    free(edge); free(def);
}

static void sort_case(void)
{
    const int64_t B = ri(0, 4), rb = 16 * ri(1, 2);
    int64_t *ko = xmalloc((size_t)(B + 1) * 8);
    ko[0] = 0;
    for (int64_t v = 0; v < B; v++)
        ko[v + 1] = ko[v] + ri(0, 40);
    const int64_t n = ko[B];
    int64_t *kin = xmalloc((size_t)n * 8), *kout = xmalloc((size_t)n * 8);
    uint8_t *rin = xmalloc((size_t)(n * rb)), *rout = xmalloc((size_t)(n * rb));
    for (int64_t i = 0; i < n; i++) {
        kin[i] = pool_key();
        memset(rin + i * rb, 0, (size_t)rb);
        memcpy(rin + i * rb, &i, 8);   /* the record's input index, to check stability */
        fill(rin + i * rb + 8, (size_t)(rb - 8));
    }
    CHECK(ccor_sort_affinity(B, ko, kin, rin, rb, kout, rout) == 0, "sort returned an error");
    for (int64_t v = 0; v < B; v++) {
        for (int64_t i = ko[v]; i < ko[v + 1]; i++) {
            int64_t src;
            memcpy(&src, rout + i * rb, 8);
            CHECK(src >= ko[v] && src < ko[v + 1], "a row left its viewer");
            CHECK(kout[i] == kin[src], "a key was separated from its row");
            CHECK(memcmp(rout + i * rb, rin + src * rb, (size_t)rb) == 0, "a row was altered");
            if (i > ko[v]) {
                int64_t prev;
                memcpy(&prev, rout + (i - 1) * rb, 8);
                CHECK(kout[i - 1] < kout[i] || (kout[i - 1] == kout[i] && prev < src),
                      "not sorted, or equal keys out of input order");
            }
        }
    }
    free(ko); free(kin); free(kout); free(rin); free(rout);
}

static void resolve_case(void)
{
    const int64_t n = ri(0, 60), q = ri(0, 80);
    int64_t *ids = xmalloc((size_t)n * 8), *qs = xmalloc((size_t)q * 8);
    int64_t *pos = xmalloc((size_t)q * 8);
    for (int64_t i = 0; i < n; i++)   /* distinct ids, some negative and extreme */
        ids[i] = (i % 7 == 3) ? INT64_MAX - i : (i % 5 == 1) ? -1000 - i : 3 * i + 1;
    for (int64_t j = 0; j < q; j++)
        qs[j] = (n > 0 && ri(0, 1)) ? ids[ri(0, n - 1)] : pool_key();
    CHECK(ccor_resolve(n, ids, q, qs, pos) == 0, "resolve returned an error");
    for (int64_t j = 0; j < q; j++) {
        int64_t want = -1;
        for (int64_t i = 0; i < n; i++)
            if (ids[i] == qs[j])
                want = i;
        CHECK(pos[j] == want, "resolved position disagrees with a scan");
    }
    free(ids); free(qs); free(pos);
}

static void upsert_case(void)
{
    const int64_t cap = ri(0, 30), rb = 16;
    int64_t n_docs = 0, m_docs = 0;
    int64_t *ids = xmalloc((size_t)cap * 8), *auth = xmalloc((size_t)cap * 8);
    uint8_t *rows = xmalloc((size_t)(cap * rb));
    int64_t *mids = xmalloc((size_t)cap * 8), *mauth = xmalloc((size_t)cap * 8);
    uint8_t *mrows = xmalloc((size_t)(cap * rb));
    for (int batch = 0; batch < 6; batch++) {
        const int64_t n = ri(0, 10);
        int64_t *bid = xmalloc((size_t)n * 8), *bau = xmalloc((size_t)n * 8);
        uint8_t *brow = xmalloc((size_t)(n * rb));
        for (int64_t i = 0; i < n; i++) {
            bid[i] = ri(0, 9) == 0 ? INT64_MIN : ri(0, 15) * 7 - 20;
            bau[i] = pool_key();
        }
        fill(brow, (size_t)(n * rb));
        /* the model: plain arrays and linear search, applied in batch order */
        int64_t fresh = 0, rejected = 0;
        for (int64_t i = 0; i < n; i++) {
            int seen = 0;
            if (bid[i] == INT64_MIN) {
                rejected++;
                continue;
            }
            for (int64_t p = 0; p < m_docs; p++)
                seen |= mids[p] == bid[i];
            for (int64_t k = 0; k < i; k++)
                seen |= bid[k] == bid[i];
            fresh += !seen;
        }
        int64_t n_rej = -1;
        const int64_t got = ccor_upsert(cap, &n_docs, ids, auth, rows, rb, n, bid, bau, brow,
                                        &n_rej);
        if (m_docs + fresh > cap) {
            CHECK(got == -2 && n_docs == m_docs, "a batch that does not fit changed the state");
        } else {
            for (int64_t i = 0; i < n; i++) {
                if (bid[i] == INT64_MIN)
                    continue;
                int64_t p = -1;
                for (int64_t k = 0; k < m_docs; k++)
                    if (mids[k] == bid[i])
                        p = k;
                if (p < 0) {
                    p = m_docs++;
                    mids[p] = bid[i];
                }
                mauth[p] = bau[i];
                memcpy(mrows + p * rb, brow + i * rb, (size_t)rb);
            }
            CHECK(got == fresh && n_rej == rejected, "new and rejected counts");
            CHECK(n_docs == m_docs, "document count");
            CHECK(memcmp(ids, mids, (size_t)n_docs * 8) == 0, "ids by position");
            CHECK(memcmp(auth, mauth, (size_t)n_docs * 8) == 0, "author ids");
            CHECK(memcmp(rows, mrows, (size_t)(n_docs * rb)) == 0, "rows");
        }
        free(bid); free(bau); free(brow);
    }
    free(ids); free(auth); free(rows); free(mids); free(mauth); free(mrows);
}

int main(int argc, char **argv)
{
    const int n = argc > 1 ? atoi(argv[1]) : 400;
    rng_state = 0x9E3779B97F4A7C15ULL;
    for (case_no = 0; case_no < n; case_no++) {
        join_case();
        sort_case();
        resolve_case();
        upsert_case();
    }
    printf("ok\n");
    return 0;
}
