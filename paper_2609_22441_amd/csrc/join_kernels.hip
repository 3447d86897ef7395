// Edge-feature join kernels for gfx950 (CDNA4).
//
// Operation: Connected Content Retriever §3.1, Eq. 1 with the search of Alg. 1 Steps 2-4,
// fused with the gather of the candidate's document row (§6.3). The path is a memory-bound
// search-and-copy: no matrix cores, no arithmetic on the row payloads.
//
// Work decomposition
//   * The flattened candidate array [0, total_cand) is cut into n_wg contiguous ranges: of
//     per_wg candidates each, or, for CSR batches of up to kBalanceViewers viewers, of equal
//     estimated cost (balanced_range). Hardware dispatches workgroup b to XCD b % 8, so the
//     range index is (b % 8) * (n_wg / 8) + b / 8: each XCD walks one contiguous eighth of the
//     candidates, which keeps a viewer's keys and edge rows in a single XCD's L2.
//   * A range is split at viewer boundaries into segments. For each segment the workgroup
//     stages every S-th key of the viewer ("fences") into LDS; S = 1 stages the whole list.
//   * Sub-tiles of kBlock candidates: each thread resolves one candidate (position check,
//     author id, search), then the workgroup copies the sub-tile's output rows as 16-byte
//     chunks, consecutive lanes on consecutive chunks of the output (coalesced stores; 8
//     lanes share one 128-byte doc row read).
//
// Search for key x in a viewer's keys k[0..K) with fences f[i] = k[i*S], i < M = ceil(K/S):
//   g = #{ i : f[i] < x }            branch-free lower bound in LDS, ceil(log2 M) probes.
//   S == 1 : the lower bound is g.
//   S  > 1 : k[(g-1)*S] < x <= k[g*S], so the lower bound lies in [(g-1)*S+1, min(g*S, K)];
//            read S keys covering that window from global memory (L2) in one step, as
//            16-byte loads, and count.
//   hit    : some key equal to x in the inspected window; because keys ascend, the lower
//            bound is then the leftmost equal key.
#include <atomic>
#include <map>
#include <mutex>
#include <utility>

#include "join_internal.h"

namespace ccj {
namespace {

// Workgroup barrier that orders LDS accesses only. The barriers here protect the LDS tables;
// global loads and stores may stay in flight across them (a full __syncthreads() would
// drain every outstanding global access first).
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// 16-byte chunk as a native vector (HIP's uint4 is a struct wrapper that the compiler may keep
// in scratch memory when it sits in an array).
typedef unsigned int chunk_t __attribute__((ext_vector_type(4)));

// s_waitcnt operand for "vector memory count 0", leaving the export and LDS/scalar counters
// unconstrained (gfx9 encoding: vmcnt in bits 3:0 and 15:14, expcnt 6:4, lgkmcnt 11:8).
constexpr int kWaitVmcnt0 = (0x7 << 4) | (0xF << 8);

__device__ __forceinline__ int64_t clamp64(int64_t v, int64_t hi) {
    return v < 0 ? 0 : (v > hi ? hi : v);
}

// Number of entries of t[0..n) (ascending, n >= 1) that are < x; ceil(log2 n) iterations,
// trip count independent of x so a wavefront never diverges here.
__device__ __forceinline__ int64_t count_less(const int64_t *t, int64_t n, int64_t x) {
    const int64_t *b = t;
    while (n > 1) {
        const int64_t half = n >> 1;
        b = (b[half] < x) ? b + half : b;
        n -= half;
    }
    return (b - t) + (*b < x ? 1 : 0);
}

// Inspect keys lo .. lo+W-1 (indices clamped to K-1, so every load is in bounds and all W
// loads are issued together): count those < x among the first len, and note any equal to x.
// A clamped repeat of k[K-1] adds no false match: if k[K-1] == x it lies inside the window.
template <int W>
__device__ __forceinline__ void scan_window(const int64_t *gk, int64_t K, int64_t lo, int64_t len,
                                            int64_t x, int64_t &cnt, bool &eq) {
    int64_t k[W];
#pragma unroll
    for (int t = 0; t < W; ++t)
        k[t] = gk[min(lo + t, K - 1)];
#pragma unroll
    for (int t = 0; t < W; ++t) {
        cnt += (t < len && k[t] < x) ? 1 : 0;
        eq |= (k[t] == x);
    }
}

// Inspect the W keys gk[w0 .. w0 + W), all in bounds: count those < x and note any equal to x.
// The keys are read as W / 2 loads of 16 bytes each at the list's 8-byte alignment (global
// loads need only dword alignment), half the load instructions of one load per key. A lane's
// loads reach scattered lines, so the vector memory unit's cost grows with the instruction
// count rather than the bytes.
template <int W>
__device__ __forceinline__ void scan_block(const int64_t *gk, int64_t w0, int64_t x, int64_t &cnt,
                                           bool &eq) {
    typedef long long pair_t __attribute__((ext_vector_type(2)));
    pair_t k[W / 2];
#pragma unroll
    for (int t = 0; t < W / 2; ++t)
        __builtin_memcpy(&k[t], gk + w0 + 2 * t, sizeof(pair_t));
#pragma unroll
    for (int t = 0; t < W / 2; ++t) {
        cnt += (k[t].x < x ? 1 : 0) + (k[t].y < x ? 1 : 0);
        eq |= (k[t].x == x) | (k[t].y == x);
    }
}

// Index in [0, K) of the leftmost key equal to x, or -1.
__device__ __forceinline__ int64_t find_key(int64_t x, const int64_t *tab, int64_t M, int S,
                                            const int64_t *gk, int64_t K) {
    if (K <= 0)
        return -1;
    const int64_t g = count_less(tab, M, x);
    if (S == 1)
        return (g < K && tab[g] == x) ? g : -1;
    if (g == 0)
        return tab[0] == x ? 0 : -1;
    // k[(g-1)S] < x <= k[gS]: the lower bound lies in [lo, min(gS, K)].
    int64_t lo = (g - 1) * S + 1;
    int64_t cnt = 0;
    bool eq = false;
    if (S <= 16 && K >= S) {
        // Read S keys from w0 = min(lo, K - S): the window [lo, lo + S) moved back, if needed,
        // to end at K. Every key before lo is <= k[(g-1)S] < x, so the keys < x in the window
        // number (lower bound - w0) either way, and a key equal to x, if any, is in the window.
        const int64_t w0 = min(lo, K - S);
        switch (S) {
        case 2: scan_block<2>(gk, w0, x, cnt, eq); break;
        case 4: scan_block<4>(gk, w0, x, cnt, eq); break;
        case 8: scan_block<8>(gk, w0, x, cnt, eq); break;
        default: scan_block<16>(gk, w0, x, cnt, eq); break;
        }
        return eq ? w0 + cnt : -1;
    }
    // Strides beyond 16 (only when K exceeds 16x the LDS table), or a list shorter than a forced
    // stride: narrow in global memory, then inspect the last few keys with clamped loads.
    int64_t len = min(g * (int64_t)S, K) - lo;
    const int64_t *w = gk + lo;
    while (len > kWindow) {
        const int64_t half = len >> 1;
        w = (w[half] < x) ? w + half : w;
        len -= half;
    }
    lo = w - gk;
    scan_window<kWindow + 1>(gk, K, lo, len, x, cnt, eq);
    return eq ? lo + cnt : -1;
}

// Two windows of W keys, gk[w0 ..) for x0 and gk[w1 ..) for x1 (both in bounds): all loads are
// issued before the first compare, so the two reads cost one round trip.
template <int W>
__device__ __forceinline__ void scan_block_pair(const int64_t *gk, int64_t w0, int64_t x0,
                                                int64_t w1, int64_t x1, int64_t &c0, bool &e0,
                                                int64_t &c1, bool &e1) {
    typedef long long pair_t __attribute__((ext_vector_type(2)));
    pair_t k0[W / 2], k1[W / 2];
#pragma unroll
    for (int t = 0; t < W / 2; ++t) {
        __builtin_memcpy(&k0[t], gk + w0 + 2 * t, sizeof(pair_t));
        __builtin_memcpy(&k1[t], gk + w1 + 2 * t, sizeof(pair_t));
    }
#pragma unroll
    for (int t = 0; t < W / 2; ++t) {
        c0 += (k0[t].x < x0 ? 1 : 0) + (k0[t].y < x0 ? 1 : 0);
        e0 |= (k0[t].x == x0) | (k0[t].y == x0);
        c1 += (k1[t].x < x1 ? 1 : 0) + (k1[t].y < x1 ? 1 : 0);
        e1 |= (k1[t].x == x1) | (k1[t].y == x1);
    }
}

// Both lookups of one candidate (the same viewer's keys): r0 and r1 as find_key gives them, or
// -1 when !valid. With a fence stride of 2 to 8 and K >= S, both LDS searches run first and
// both key windows are then read together, every load from an index in bounds whatever the
// lane's values: the window starts at w = clamp((g - 1) S + 1, 0, K - S). For g = 0 that is
// the list's first S keys, none below x (x <= k[0]), so the count is 0 and an equal key can
// only be k[0]: the same answer as the g = 0 rule of find_key. (Two windows of 16 keys would
// hold 64 registers; two-lookup launches run two workgroups per CU, which needs at most 256.)
__device__ __forceinline__ void find_key_pair(int64_t x0, int64_t x1, bool valid,
                                              const int64_t *tab, int64_t M, int S,
                                              const int64_t *gk, int64_t K, int64_t &r0,
                                              int64_t &r1) {
    if (S >= 2 && S <= 8 && K >= S) {
        const int64_t g0 = count_less(tab, M, x0);
        const int64_t g1 = count_less(tab, M, x1);
        const int64_t w0 = clamp64((g0 - 1) * S + 1, K - S);
        const int64_t w1 = clamp64((g1 - 1) * S + 1, K - S);
        int64_t c0 = 0, c1 = 0;
        bool e0 = false, e1 = false;
        switch (S) {
        case 2: scan_block_pair<2>(gk, w0, x0, w1, x1, c0, e0, c1, e1); break;
        case 4: scan_block_pair<4>(gk, w0, x0, w1, x1, c0, e0, c1, e1); break;
        default: scan_block_pair<8>(gk, w0, x0, w1, x1, c0, e0, c1, e1); break;
        }
        r0 = valid && e0 ? w0 + c0 : -1;
        r1 = valid && e1 ? w1 + c1 : -1;
        return;
    }
    r0 = valid ? find_key(x0, tab, M, S, gk, K) : -1;
    r1 = valid ? find_key(x1, tab, M, S, gk, K) : -1;
}

// Fence stride for one segment: the smallest power of two whose fence count fits the LDS
// table and is not much larger than the number of candidates that will use it.
__device__ __forceinline__ int choose_stride(int64_t K, int64_t seg_len, int32_t cap,
                                             int32_t forced, int32_t per_cand) {
    int64_t budget = forced > 0 ? cap : min<int64_t>(cap, max<int64_t>(512, per_cand * seg_len));
    int S = forced > 0 ? forced : 1;
    while ((K + S - 1) / S > budget)
        S <<= 1;
    return S;
}

// Author id of candidate j at store position c: the caller's id for the candidate when the
// call supplies them (Alg. 1's input form), else the store's, from the 32-bit column when the
// store has one (every id fits in 32 bits, so a 64-byte sector holds 16 ids instead of 8) or the
// 64-bit column. The column is a compile-time choice: a branch in the prefetch would split the
// pipeline's basic blocks and cost more than the narrower reads save; the caller's ids share
// the 64-bit form, by address (one unconditional load either way).
template <bool A32>
__device__ __forceinline__ int64_t author_of(const JoinArgs &a, int64_t c, int64_t j) {
    if constexpr (A32)
        return (int64_t)a.author32[c];
    else
        return *(a.cand_author ? a.cand_author + j : a.author + c);
}

__device__ __forceinline__ int64_t range_index(int b, int n) {
    const int per_xcd = n >> 3;
    return (int64_t)(b & 7) * per_xcd + (b >> 3);
}

// Estimated cost of one candidate of a viewer with K keys when the LDS table holds T keys, in
// units of about 1/60 ns (a candidate of a 3,000-key list costs about 1,050). Fitted to
// per-workgroup clocks of ragged 64-viewer batches (1.92M candidates, K from 100 to 30,000):
// a candidate costs about 17% less when its list is short (its viewer's in-network candidates
// then come from few authors, whose rows stay in the caches), grows with log K while the list
// fits the table, and steps up by about 20% once K exceeds it (each lookup then reads a key
// window from L2). Only the split of the work depends on it, never the result.
__device__ __forceinline__ int64_t cand_cost(int64_t K, int64_t T) {
    K = K < 1 ? 1 : min<int64_t>(K, (int64_t)1 << 24);
    const int64_t k = min(K, T < 1 ? (int64_t)1 : T);
    // 16 * log2(k), linear between powers of two.
    const int l = 63 - __clzll((unsigned long long)k);
    const int64_t l16 = 16 * l + (((k - ((int64_t)1 << l)) << 4) >> l);
    int64_t c = 830 + 45 * max<int64_t>(l16 - 106, 0) / 16;      // 106 = 16 * log2(100)
    if (K > T)
        c += 100 + (K - T) * 11 / 2000;
    return c;
}

__device__ __forceinline__ int64_t wave_scan_incl(int64_t x) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const int64_t y = __shfl_up(x, d);
        if (lane >= d)
            x += y;
    }
    return x;
}

// Weighted ranges for a CSR batch of at most kBalanceViewers viewers. Candidate i of viewer v
// weighs w_v = cand_cost(K_v) (in the padded layout only its first n_max candidates, the ones
// joined, count); with prefix weights P, logical range r of n covers the candidates
// whose weight starts in [T_r, T_{r+1}), T_r = floor(r * W / n), W the total. Every workgroup
// computes the same prefix, so the ranges tile the candidates. Ranges of equal weight take
// fewer candidates of long lists, which would otherwise finish last. (A cost for starting a
// viewer, charged to the range that holds its first candidate, helped ragged batches by 1% but
// slowed batches of equal viewers, whose ranges start exactly at viewer starts, by 2%.) Returns
// the range and the viewer holding its first candidate; s is kBlock entries of LDS scratch.
__device__ __forceinline__ void balanced_range(const JoinArgs &a, int64_t r, int64_t n,
                                               int64_t *s, int64_t &begin, int64_t &end,
                                               int32_t &v_first) {
    constexpr int R = kBalanceViewers / kBlock;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int32_t B = a.n_viewers;
    int64_t w[R], vb[R], c[R];
    int64_t mine = 0;
#pragma unroll
    for (int i = 0; i < R; ++i) {
        const int64_t v = (int64_t)i * kBlock + tid;
        w[i] = 0;
        vb[i] = 0;
        c[i] = 1;
        if (v < B) {
            vb[i] = clamp64(a.cand_offsets[v], a.total_cand);
            const int64_t ve = clamp64(a.cand_offsets[v + 1], a.total_cand);
            const int64_t kb = clamp64(a.key_offsets[v], a.total_keys);
            const int64_t ke = max(kb, clamp64(a.key_offsets[v + 1], a.total_keys));
            c[i] = cand_cost(ke - kb, a.lds_keys);
            int64_t nv = max<int64_t>(ve - vb[i], 0);
            if (a.n_max > 0)                      // the padded layout joins the first n_max
                nv = min(nv, a.n_max);
            w[i] = nv * c[i];
        }
        mine += w[i];
    }
    // Total weight.
    int64_t t = mine;
#pragma unroll
    for (int d = 32; d > 0; d >>= 1)
        t += __shfl_xor(t, d);
    if (lane == 0)
        s[wave] = t;
    if (tid == 0) {
        s[8] = a.total_cand;                      // range start, if no viewer holds T_r
        s[9] = B;                                 // its viewer
        s[10] = a.total_cand;                     // range end, if no viewer holds T_{r+1}
    }
    lds_barrier();
    const int64_t W = s[0] + s[1] + s[2] + s[3];
    const int64_t q = W / n, m = W % n;
    const int64_t t0 = q * r + m * r / n, t1 = q * (r + 1) + m * (r + 1) / n;
    lds_barrier();
    // Prefix weights in viewer order, one chunk of kBlock viewers at a time.
    int64_t carry = 0;
#pragma unroll
    for (int i = 0; i < R; ++i) {
        if (i * kBlock >= B)                      // uniform: the same for every thread
            break;
        const int64_t inc = wave_scan_incl(w[i]);
        if (lane == 63)
            s[wave] = inc;
        lds_barrier();
        int64_t pre = carry + inc - w[i];
        for (int k = 0; k < wave; ++k)
            pre += s[k];
        carry += s[0] + s[1] + s[2] + s[3];
        if (w[i] > 0) {
            if (t0 >= pre && t0 < pre + w[i]) {
                s[8] = vb[i] + (t0 - pre + c[i] - 1) / c[i];
                s[9] = (int64_t)i * kBlock + tid;
            }
            if (t1 >= pre && t1 < pre + w[i])
                s[10] = vb[i] + (t1 - pre + c[i] - 1) / c[i];
        }
        lds_barrier();
    }
    begin = s[8];
    v_first = (int32_t)s[9];
    end = s[10];
    lds_barrier();                                // s is reused by the caller
}

// Copy a full sub-tile (kBlock rows) whose widths are compile-time chunk counts. Thread tid
// takes chunks e = i * kBlock + tid of the sub-tile's output, i.e. row e / CH, 16-byte column
// e % CH, so each wavefront store covers 1 KiB of contiguous output (whole 128-byte lines: a
// line split between two stores with the streaming hint would be written back twice). Every
// load and store is unconditional (absent rows are read from the store's zero row), so each
// thread has all CH loads in flight before its first store. `between()` runs after the loads
// are issued and before the stores (the caller issues the next sub-tile's dependent loads
// there). Output rows are written with the non-temporal hint: they are not read again, and
// keeping them out of the caches leaves room for the author column, keys and edge rows.
template <int DOC_CH, int EDGE_CH, int NL, typename Between>
__device__ __forceinline__ void copy_full_tile(const JoinArgs &a, const int64_t *s_src,
                                               const int64_t (*s_row)[kBlock], int64_t t0,
                                               const uint8_t *miss_row, Between between) {
    constexpr int CH = DOC_CH + NL * EDGE_CH;
    const int tid = threadIdx.x;
    chunk_t v[CH];
#pragma unroll
    for (int i = 0; i < CH; ++i) {
        const int e = i * kBlock + tid;
        const int row = e / CH, k = e % CH;
        const bool is_doc = k < DOC_CH;
        const int kk = is_doc ? 0 : k - DOC_CH;
        const int l = kk / EDGE_CH, q = kk % EDGE_CH;
        const int64_t d = s_src[row];
        const int64_t r = s_row[l][row];
        const uint8_t *pd = d >= 0 ? a.doc + d * (DOC_CH * 16) + k * 16 : a.zero_row + k * 16;
        const uint8_t *pe = r >= 0 ? a.edge + r * (EDGE_CH * 16) + q * 16 : miss_row + q * 16;
        v[i] = *reinterpret_cast<const chunk_t *>(is_doc ? pd : pe);
    }
    between();
    uint8_t *o = a.out + t0 * a.out_stride;
    if (a.out_stride == CH * 16) {
        // Packed rows: chunk e sits at byte 16 * e of the sub-tile.
        chunk_t *po = reinterpret_cast<chunk_t *>(o) + tid;
#pragma unroll
        for (int i = 0; i < CH; ++i)
            __builtin_nontemporal_store(v[i], po + i * kBlock);
    } else {
#pragma unroll
        for (int i = 0; i < CH; ++i) {
            const int e = i * kBlock + tid;
            const int row = e / CH, k = e % CH;
            __builtin_nontemporal_store(
                v[i], reinterpret_cast<chunk_t *>(o + row * a.out_stride + k * 16));
        }
    }
}

// Copy the first n rows of a sub-tile (any widths). Used for segments shorter than a sub-tile
// and for row widths without a compile-time specialisation, so it favours few live registers
// over loads in flight. DOC_CH / EDGE_CH are row widths in 16-byte chunks (0 = read them from
// the arguments).
template <int DOC_CH, int EDGE_CH, int NL>
__device__ __forceinline__ void copy_rows(const JoinArgs &a, const int64_t *s_src,
                                          const int64_t (*s_row)[kBlock], int64_t t0, int n) {
    const int tid = threadIdx.x;
    const int dch = DOC_CH > 0 ? DOC_CH : (a.doc_bytes >> 4);
    const int ech = EDGE_CH > 0 ? EDGE_CH : (a.edge_bytes >> 4);
    const int dbytes = dch * 16, ebytes = ech * 16;
    const int ch = dch + NL * ech;
    const int total = n * ch;
    constexpr int U = 4;
    for (int base = 0; base < total; base += U * kBlock) {
        chunk_t v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int e = base + u * kBlock + tid;
            v[u] = chunk_t{0u, 0u, 0u, 0u};
            if (e < total) {
                const int row = e / ch, k = e - (e / ch) * ch;
                const chunk_t *src = nullptr;
                if (k < dch) {
                    const int64_t c = s_src[row];
                    if (c >= 0)
                        src = reinterpret_cast<const chunk_t *>(a.doc + c * dbytes) + k;
                } else {
                    const int kk = k - dch;
                    const int l = kk / ech;
                    const int q = kk - l * ech;
                    const int64_t r = s_row[l][row];
                    if (r >= 0)
                        src = reinterpret_cast<const chunk_t *>(a.edge + r * ebytes) + q;
                    else if (a.def_row)
                        src = reinterpret_cast<const chunk_t *>(a.def_row) + q;
                }
                if (src)
                    v[u] = *src;
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int e = base + u * kBlock + tid;
            if (e < total) {
                const int row = e / ch, k = e - (e / ch) * ch;
                reinterpret_cast<chunk_t *>(a.out + (t0 + row) * a.out_stride)[k] = v[u];
            }
        }
    }
}

// Copy the fences f[i] = gk[i * S], i < M, into LDS, 16 loads in flight per thread (indices
// clamped to M - 1; the repeated writes of the last fence store the same value).
__device__ __forceinline__ void stage_fences(int64_t *s_tab, const int64_t *gk, int64_t M, int S) {
    const int tid = threadIdx.x;
    constexpr int U = 16;
    for (int64_t i0 = 0; i0 < M; i0 += U * kBlock) {
        int64_t f[U];
#pragma unroll
        for (int u = 0; u < U; ++u)
            f[u] = gk[min(i0 + u * kBlock + tid, M - 1) * S];
#pragma unroll
        for (int u = 0; u < U; ++u)
            s_tab[min(i0 + u * kBlock + tid, M - 1)] = f[u];
    }
}

// Resolve one sub-tile starting at candidate tb: per thread, the candidate's position check and
// search(es). Writes the doc position (or -1) to src[tid] and the global edge row per lookup (or
// -1) to row[l][tid], stores the hit bytes (output row = candidate + shift), and counts invalid
// positions of rows tid >= fresh.
template <int NL>
__device__ __forceinline__ void resolve_tile(const JoinArgs &a, int64_t *src,
                                             int64_t (*row)[kBlock], unsigned int *s_invalid,
                                             const int64_t *s_tab, int64_t M, int S,
                                             const int64_t *gk, int64_t K, int64_t kb, int64_t tb,
                                             int64_t shift, int fresh, int64_t c, int64_t x0,
                                             int64_t x1) {
    const int tid = threadIdx.x;
    const int64_t j = tb + tid + shift;
    const bool valid = c >= 0 && c < a.n_docs;
    src[tid] = valid ? c : -1;
    if (!valid && tid >= fresh)
        atomicAdd(s_invalid, 1u);
    if constexpr (NL == 2) {
        int64_t r[2];
        find_key_pair(x0, x1, valid, s_tab, M, S, gk, K, r[0], r[1]);
#pragma unroll
        for (int l = 0; l < 2; ++l) {
            row[l][tid] = r[l] >= 0 ? kb + r[l] : -1;
            a.hit[j * NL + l] = (int8_t)(r[l] >= 0 ? 1 : 0);
        }
    } else {
        int64_t r = -1;
        if (valid)
            r = find_key(x0, s_tab, M, S, gk, K);
        row[0][tid] = r >= 0 ? kb + r : -1;
        a.hit[j] = (int8_t)(r >= 0 ? 1 : 0);
    }
}

// Process candidates [s0, s1) of one viewer segment (s1 - s0 >= kBlock) in full sub-tiles.
// Sub-tile k starts at base(k) = min(s0 + k * kBlock, s1 - kBlock): the last one is moved back
// to end at s1 and overlaps its predecessor (those rows are rewritten with the same bytes, and
// `fresh` keeps them out of the invalid count).
//
// Software pipeline. A thread's dependent chain per candidate is position -> author id ->
// search -> row copy. Iteration k issues sub-tile k's copy loads, then searches sub-tile k+1
// into the other half of the double-buffered LDS tables, then issues the loads for later
// sub-tiles (positions of k+3, author ids of k+2), then stores sub-tile k. Vector-memory
// completions are counted in issue order, so a search's key-window loads, issued after the
// copy loads, never wait for stores younger than the previous iteration's. The last iteration
// searches its own sub-tile once more (identical hit bytes; `fresh` = kBlock counts nothing)
// so that the loop body has no branch. All loads are unconditional from clamped indices: a
// load under a branch, or a second path into the loop latch, would leave the compiler unable
// to count outstanding loads, and it would then wait for every store of a sub-tile first.
template <int DOC_CH, int EDGE_CH, int NL, bool A32, typename Stage>
__device__ __forceinline__ void full_tiles(const JoinArgs &a, int64_t (*s_src)[kBlock],
                                           int64_t (*s_row)[NL][kBlock],
                                           unsigned int *s_invalid, const int64_t *s_tab,
                                           int64_t M, int S, const int64_t *gk, int64_t K,
                                           int64_t kb, int64_t s0, int64_t s1, int64_t shift,
                                           const uint8_t *miss_row, Stage stage) {
    const int tid = threadIdx.x;
    const int64_t last_doc = a.n_docs > 0 ? a.n_docs - 1 : 0;
    const int64_t ntiles = (s1 - s0 + kBlock - 1) / kBlock;
    auto base = [&](int64_t k) { return min(s0 + k * kBlock, s1 - kBlock); };
    auto fresh = [&](int64_t k) { return (int)min<int64_t>(s0 + k * kBlock - base(k), kBlock); };
    auto extra = [&](int64_t k) -> int64_t {
        if constexpr (NL == 2)
            return a.extra[base(k) + tid];
        return 0;
    };
    int64_t c1 = a.cand_idx[base(1) + tid];
    int64_t c2 = a.cand_idx[base(2) + tid];
    int64_t e1 = extra(1);
    int64_t x1;
    {
        const int64_t c0 = a.cand_idx[base(0) + tid];
        const int64_t e0 = extra(0);
        const int64_t x0 = author_of<A32>(a, clamp64(c0, last_doc), base(0) + tid);
        x1 = author_of<A32>(a, clamp64(c1, last_doc), base(1) + tid);
        stage();
        resolve_tile<NL>(a, s_src[0], s_row[0], s_invalid, s_tab, M, S, gk, K, kb, base(0),
                         shift, fresh(0), c0, x0, e0);
    }
    // Let the prologue loads land here (once per segment). Otherwise, where the loop entry and
    // the back edge meet, the compiler keeps the prologue's short distances and waits for the
    // previous sub-tile's stores before every search.
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
    lds_barrier();
    for (int64_t k = 0; k < ntiles; ++k) {
        const int p = (int)(k & 1);
        copy_full_tile<DOC_CH, EDGE_CH, NL>(
            a, s_src[p], s_row[p], base(k) + shift, miss_row, [&]() {
                resolve_tile<NL>(a, s_src[p ^ 1], s_row[p ^ 1], s_invalid, s_tab, M, S, gk, K,
                                 kb, base(k + 1), shift, fresh(k + 1), c1, x1, e1);
                const int64_t c3 = a.cand_idx[base(k + 3) + tid];
                const int64_t e2 = extra(k + 2);
                const int64_t x2 = author_of<A32>(a, clamp64(c2, last_doc), base(k + 2) + tid);
                c1 = c2;
                c2 = c3;
                x1 = x2;
                e1 = e2;
            });
        lds_barrier();
    }
}

// BATCHED selects the CSR form (viewer offsets in device memory); the single-viewer form has
// one implicit viewer and skips the offset lookups.
template <int DOC_CH, int EDGE_CH, int NL, bool BATCHED, bool A32>
__global__ __launch_bounds__(kBlock) void join_kernel(JoinArgs a) {
    extern __shared__ int64_t s_tab[];            // fence table, a.lds_keys entries
    __shared__ int64_t s_src[2][kBlock];          // doc position of each sub-tile row, or -1
    __shared__ int64_t s_row[2][NL][kBlock];      // global edge row per lookup, or -1
                                                  // (two buffers: sub-tiles k and k+1)
    __shared__ unsigned int s_invalid;

    const int tid = threadIdx.x;
    constexpr bool batched = BATCHED;
    const int32_t B = batched ? a.n_viewers : 1;
    const int64_t rng = range_index(blockIdx.x, gridDim.x);
    int64_t begin, end;
    int32_t v = 0;                                // first viewer that may hold `begin`
    if (batched && a.balanced) {
        balanced_range(a, rng, gridDim.x, s_src[0], begin, end, v);
    } else {
        begin = rng * a.per_wg;
        end = min(begin + a.per_wg, a.total_cand);
        if (batched && begin < end) {
            // First viewer whose candidate range ends after `begin`.
            int32_t lo = 0, hi = B;
            while (lo < hi) {
                const int32_t mid = (lo + hi) >> 1;
                if (clamp64(a.cand_offsets[mid + 1], a.total_cand) <= begin)
                    lo = mid + 1;
                else
                    hi = mid;
            }
            v = lo;
        }
    }
    if (begin >= end)
        return;
    if (tid == 0)
        s_invalid = 0;
    const uint8_t *miss_row = a.def_row ? a.def_row : a.zero_row;

    for (; v < B && begin < end; ++v) {
        int64_t vb = 0, ve = a.total_cand, kb = 0, ke = a.total_keys;
        int64_t shift = 0;                        // output row = candidate index + shift
        if (batched) {
            vb = clamp64(a.cand_offsets[v], a.total_cand);
            ve = clamp64(a.cand_offsets[v + 1], a.total_cand);
            kb = clamp64(a.key_offsets[v], a.total_keys);
            ke = max(kb, clamp64(a.key_offsets[v + 1], a.total_keys));
            if (a.n_max > 0) {                    // padded layout: first n_max candidates
                ve = min(ve, vb + a.n_max);
                shift = (int64_t)v * a.n_max - vb;
            }
        }
        const int64_t s0 = max(begin, vb);
        const int64_t s1 = min(end, ve);
        if (s1 <= s0)
            continue;
        begin = s1;

        const int64_t K = ke - kb;
        const int64_t *gk = a.keys + kb;
        const int S = choose_stride(K, s1 - s0, a.lds_keys, a.fence_stride, a.fence_budget);
        const int64_t M = (K + S - 1) / S;
        // Stage the fences into LDS (after the previous segment's readers are done). Full
        // segments stage after issuing their first loads, so the two latencies overlap.
        auto stage = [&]() {
            lds_barrier();
            stage_fences(s_tab, gk, M, S);
            lds_barrier();
        };
        const int64_t seg = s1 - s0;
        if constexpr (DOC_CH > 0) {
            if (seg >= kBlock) {
                full_tiles<DOC_CH, EDGE_CH, NL, A32>(a, s_src, s_row, &s_invalid, s_tab, M, S, gk, K,
                                                kb, s0, s1, shift, miss_row, stage);
                continue;
            }
        }
        // A segment shorter than a sub-tile (or widths without a specialisation): guarded
        // sub-tiles, one candidate per thread.
        stage();
        for (int64_t t0 = s0; t0 < s1; t0 += kBlock) {
            const int n = (int)min<int64_t>(kBlock, s1 - t0);
            if (tid < n) {
                const int64_t c = a.cand_idx[t0 + tid];
                const bool ok = c >= 0 && c < a.n_docs;
                const int64_t x0 = ok ? author_of<A32>(a, c, t0 + tid) : 0;
                const int64_t x1 = NL == 2 ? a.extra[t0 + tid] : 0;
                resolve_tile<NL>(a, s_src[0], s_row[0], &s_invalid, s_tab, M, S, gk, K, kb, t0,
                                 shift, 0, c, x0, x1);
            }
            lds_barrier();
            copy_rows<DOC_CH, EDGE_CH, NL>(a, s_src[0], s_row[0], t0 + shift, n);
            lds_barrier();
        }
    }
    lds_barrier();
    if (tid == 0 && s_invalid)
        atomicAdd(a.invalid_counter, (unsigned long long)s_invalid);
}

constexpr int kMaxDevices = 64;

// Multiprocessor count per device (cached; devices are few).
int cu_count(int device) {
    static std::atomic<int> cache[kMaxDevices];
    if (device >= 0 && device < kMaxDevices) {
        int v = cache[device].load(std::memory_order_relaxed);
        if (v > 0)
            return v;
    }
    int v = 0;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, device) != hipSuccess ||
        v <= 0)
        v = 256;
    if (device >= 0 && device < kMaxDevices)
        cache[device].store(v, std::memory_order_relaxed);
    return v;
}

// Resident workgroups per CU for one kernel at one dynamic LDS size (registers and LDS both
// count), cached.
int resident_per_cu(const void *fn, size_t lds) {
    static std::mutex mu;
    static std::map<std::pair<const void *, size_t>, int> cache;
    std::lock_guard<std::mutex> lock(mu);
    auto it = cache.find({fn, lds});
    if (it != cache.end())
        return it->second;
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, fn, kBlock, lds) != hipSuccess || n < 1)
        n = 1;
    cache[{fn, lds}] = n;
    return n;
}

template <int D, int E, int L, bool BATCHED, bool A32>
hipError_t launch_one(JoinArgs &a, int32_t workgroups, int device, hipStream_t stream) {
    // The largest LDS table plus the kernel's static tables must fit a workgroup's 160 KiB.
    static_assert(kMaxLdsKeys * sizeof(int64_t) + (2 + 2 * L) * kBlock * sizeof(int64_t) +
                          sizeof(unsigned int) <= 160 * 1024,
                  "LDS budget exceeded");
    const void *fn = reinterpret_cast<const void *>(&join_kernel<D, E, L, BATCHED, A32>);
    const int64_t tiles = (a.total_cand + kBlock - 1) / kBlock;
    const int64_t cus = cu_count(device);
    // One workgroup per CU (below): the LDS table may then hold up to kWideLdsKeys keys at no
    // cost in occupancy, so that longer lists are staged whole.
    if (a.lds_auto && workgroups <= 0 && L == 1 && tiles >= 2 * cus)
        a.lds_keys = (int32_t)(a.total_keys < kWideLdsKeys ? (a.total_keys > 0 ? a.total_keys : 1)
                                                          : kWideLdsKeys);
    const size_t lds = (size_t)max(1, a.lds_keys) * sizeof(int64_t);
    // Raise the kernel's dynamic LDS limit once per device (the attribute is per device).
    static std::once_flag lds_limit[kMaxDevices];
    if (device < 0 || device >= kMaxDevices)
        return hipErrorInvalidDevice;
    hipError_t err = hipSuccess;
    std::call_once(lds_limit[device], [&] {
        err = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize,
                                  kMaxLdsKeys * (int)sizeof(int64_t));
    });
    if (err != hipSuccess)
        return err;
    // Grid: each workgroup owns a contiguous range of whole sub-tiles; the count is rounded to
    // a multiple of 8 so that each XCD gets an equal share.
    //   * Long key lists: one resident wave (the whole LDS table allows one workgroup per CU).
    //   * At least two sub-tiles per CU: one workgroup per CU. Fewer, longer ranges pay the
    //     fence staging and the pipeline's fill and drain once per CU; on launches of 300k to
    //     3.2M candidates this beat every larger grid, by up to 17% at 400k. Two lookups per
    //     candidate double the dependent search chain per sub-tile: two workgroups per CU then
    //     hide it better (64 requests of 100,000 candidates: 9% faster than one).
    //   * Smaller launches: about 1.5 resident waves, at most one workgroup per sub-tile.
    int64_t n_wg = workgroups;
    if (n_wg <= 0) {
        if (a.one_wave)
            n_wg = cus * resident_per_cu(fn, lds);
        else if (tiles >= 2 * cus)
            n_wg = cus * (L == 2 ? min(2, resident_per_cu(fn, lds)) : 1);
        else
            n_wg = cus * resident_per_cu(fn, lds) * 3 / 2;
    }
    if (n_wg > tiles)
        n_wg = tiles;
    if (n_wg < 1)
        n_wg = 1;
    const int64_t tiles_per_wg = (tiles + n_wg - 1) / n_wg;
    a.per_wg = tiles_per_wg * kBlock;
    if (!a.balanced)                      // equal ranges of whole sub-tiles, none left empty
        n_wg = (a.total_cand + a.per_wg - 1) / a.per_wg;
    n_wg = (n_wg + 7) & ~int64_t(7);
    a.n_wg = (int32_t)n_wg;
    hipLaunchKernelGGL((join_kernel<D, E, L, BATCHED, A32>), dim3(a.n_wg), dim3(kBlock), lds, stream,
                       a);
    return hipGetLastError();
}

template <int D, int E, int L>
hipError_t launch_form(JoinArgs &a, int32_t wgs, int device, hipStream_t stream) {
    if (a.author32)
        return a.cand_offsets ? launch_one<D, E, L, true, true>(a, wgs, device, stream)
                              : launch_one<D, E, L, false, true>(a, wgs, device, stream);
    return a.cand_offsets ? launch_one<D, E, L, true, false>(a, wgs, device, stream)
                          : launch_one<D, E, L, false, false>(a, wgs, device, stream);
}

template <int L>
hipError_t dispatch_widths(JoinArgs &a, int32_t wgs, int device, hipStream_t stream) {
    const int d = a.doc_bytes >> 4, e = a.edge_bytes >> 4;
    if (d == 4 && e == 2) return launch_form<4, 2, L>(a, wgs, device, stream);
    if (d == 8 && e == 4) return launch_form<8, 4, L>(a, wgs, device, stream);
    if (d == 8 && e == 8) return launch_form<8, 8, L>(a, wgs, device, stream);
    return launch_form<0, 0, L>(a, wgs, device, stream);
}

// Padded layout: slot r = v * n_max + i is a candidate's slot when i < min(n_v, n_max). Writes
// the valid mask of every slot; a pad slot also gets zero bytes over the row width and hit 0.
__global__ void pad_fill_kernel(JoinArgs a, int NL, int width_chunks, int8_t *valid) {
    const int64_t slots = (int64_t)a.n_viewers * a.n_max;
    for (int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; r < slots;
         r += (int64_t)gridDim.x * blockDim.x) {
        const int64_t v = r / a.n_max, i = r - v * a.n_max;
        const int64_t nv = clamp64(a.cand_offsets[v + 1], a.total_cand) -
                           clamp64(a.cand_offsets[v], a.total_cand);
        const bool used = i < nv;
        valid[r] = used ? 1 : 0;
        if (!used) {
            for (int l = 0; l < NL; ++l)
                a.hit[r * NL + l] = 0;
            chunk_t *o = reinterpret_cast<chunk_t *>(a.out + r * a.out_stride);
            for (int q = 0; q < width_chunks; ++q)
                o[q] = chunk_t{0u, 0u, 0u, 0u};
        }
    }
}

__global__ void validate_keys_kernel(const int64_t *key_offsets, const int64_t *keys,
                                     int32_t n_viewers, int64_t total_keys,
                                     unsigned long long *first_bad) {
    for (int32_t v = blockIdx.x; v < n_viewers; v += gridDim.x) {
        const int64_t kb = clamp64(key_offsets[v], total_keys);
        const int64_t ke = max(kb, clamp64(key_offsets[v + 1], total_keys));
        bool bad = false;
        for (int64_t i = kb + 1 + threadIdx.x; i < ke; i += blockDim.x)
            bad |= !(keys[i - 1] < keys[i]);
        if (bad)
            atomicMin(first_bad, (unsigned long long)v);
    }
}

}  // namespace

hipError_t launch_join(JoinArgs &a, int n_lookups, int32_t workgroups, int device,
                       hipStream_t stream) {
    return n_lookups == 2 ? dispatch_widths<2>(a, workgroups, device, stream)
                          : dispatch_widths<1>(a, workgroups, device, stream);
}

hipError_t launch_pad_fill(const JoinArgs &a, int n_lookups, int8_t *valid_mask,
                           hipStream_t stream) {
    const int64_t slots = (int64_t)a.n_viewers * a.n_max;
    if (slots <= 0)
        return hipSuccess;
    const int64_t blocks = (slots + 255) / 256;
    const int grid = (int)(blocks < 8192 ? blocks : 8192);
    const int width_chunks = (a.doc_bytes + n_lookups * a.edge_bytes) / 16;
    hipLaunchKernelGGL(pad_fill_kernel, dim3(grid), dim3(256), 0, stream, a, n_lookups,
                       width_chunks, valid_mask);
    return hipGetLastError();
}

hipError_t launch_validate_keys(const int64_t *key_offsets, const int64_t *keys,
                                int32_t n_viewers, int64_t total_keys,
                                unsigned long long *first_bad, hipStream_t stream) {
    if (n_viewers <= 0)
        return hipSuccess;
    const int grid = n_viewers < 4096 ? n_viewers : 4096;
    hipLaunchKernelGGL(validate_keys_kernel, dim3(grid), dim3(256), 0, stream, key_offsets, keys,
                       n_viewers, total_keys, first_bad);
    return hipGetLastError();
}

}  // namespace ccj
